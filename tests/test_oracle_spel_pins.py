"""Pins of the SPEL oracle (Sec. 3.3, Eqs. 4-7) and of its PolarExpress
schedule against closed forms and invariants."""
import numpy as np
import pytest

from oracle import polar_schedule as ps
from oracle import spel


def _orth(rng, n, m):
    q, _ = np.linalg.qr(rng.standard_normal((n, m)))
    return q


def _blockJ(r):
    J = np.zeros((r, r))
    for i in range(0, r, 2):
        J[i, i + 1] = 1.0
        J[i + 1, i] = -1.0
    return J


# ---------------------------------------------------------------- P7 invariants
@pytest.mark.parametrize("mode", ["exact", "pe"])
def test_stiefel_invariants(mode):
    rng = np.random.default_rng(31)
    d, r = 40, 8
    U = _orth(rng, d, r)
    G = rng.standard_normal((d, r))
    gR = spel.tangent_project(U, G)
    S = U.T @ gR
    assert np.abs(S + S.T).max() < 1e-12  # U^T g_R is skew-symmetric
    M = np.zeros((d, r))
    Un, Mn, D, _ = spel.stiefel_step(U, G, M, 1e-2, 0.95, mode=mode)
    assert np.abs(Un.T @ Un - np.eye(r)).max() < 1e-10
    P = Un @ Un.T
    assert np.abs(P @ P - P).max() < 1e-10
    # momentum of Eq. 5 from zero state
    assert np.abs(Mn - 0.05 * gR).max() < 1e-15


def test_tangent_projection_is_a_projection():
    rng = np.random.default_rng(32)
    U = _orth(rng, 30, 6)
    G = rng.standard_normal((30, 6))
    g1 = spel.tangent_project(U, G)
    g2 = spel.tangent_project(U, g1)
    assert np.abs(g1 - g2).max() < 1e-12
    # the removed part U sym(U^T G) is orthogonal (Frobenius) to the tangent part
    assert abs(np.sum((G - g1) * g1)) < 1e-10


# ---------------------------------------------------------------- P8 closed-form step
def test_closed_form_step_skew_gradient_exact():
    """G = U K with K = blockdiag(theta_i J2): g_R = U K, polar(M) = U J and
    U_1 = U (I - alpha J) / sqrt(1 + alpha^2)."""
    rng = np.random.default_rng(33)
    d, r, alpha = 24, 6, 0.03
    U = _orth(rng, d, r)
    J = _blockJ(r)
    thetas = np.repeat(rng.uniform(0.5, 2.0, r // 2), 2)
    K = J * thetas[:, None]
    G = U @ K
    Un, _, D, gR = spel.stiefel_step(U, G, np.zeros((d, r)), alpha, 0.9, mode="exact")
    assert np.abs(gR - G).max() < 1e-12
    assert np.abs(D - U @ J).max() < 1e-12
    assert np.abs(Un - U @ (np.eye(r) - alpha * J) / np.sqrt(1 + alpha ** 2)).max() < 1e-12


def test_closed_form_step_skew_gradient_pe():
    """Same gradient with equal thetas, PolarExpress mode: M / ||M||_F has every
    singular value 1/sqrt(r), so D = c U J with c = the LMO schedule composed
    at 1/sqrt(r); U - alpha D has every singular value sqrt(1 + alpha^2 c^2),
    the retraction normalises it to exactly orthonormal and keeps it there."""
    rng = np.random.default_rng(34)
    d, r, alpha = 24, 6, 0.03
    U = _orth(rng, d, r)
    J = _blockJ(r)
    G = 1.7 * (U @ J)
    Un, M1, D, _ = spel.stiefel_step(U, G, np.zeros((d, r)), alpha, 0.9, mode="pe")
    nrm = np.linalg.norm(M1)  # = 0.1 * 1.7 * sqrt(r)
    sv = (nrm / np.sqrt(r)) / (nrm + spel.LMO_EPS)
    c = ps.compose(ps.greedy_schedule(spel.LMO_LOWER, 5)[0], np.array([sv]))[0]
    assert np.abs(D - c * U @ J).max() < 1e-12
    c_ret = ps.compose(ps.greedy_schedule(spel.RETRACT_LOWER, 7)[0], np.array([1.0]))[0]
    expect = U @ (np.eye(r) - alpha * c * J) / np.sqrt(1 + alpha ** 2 * c ** 2) * c_ret
    assert np.abs(Un - expect).max() < 1e-12


def test_symmetric_gradient_leaves_U_unchanged():
    """G = U S with S symmetric lies in the normal space: g_R = 0 (up to
    rounding), the zero rule maps the LMO to 0, and U_1 = U."""
    rng = np.random.default_rng(35)
    d, r = 30, 6
    U = _orth(rng, d, r)
    S = rng.standard_normal((r, r))
    G = U @ (S + S.T)
    Un, _, D, gR = spel.stiefel_step(U, G, np.zeros((d, r)), 1e-2, 0.95, mode="exact")
    assert np.abs(gR).max() < 1e-13
    assert np.abs(Un - U).max() < 1e-12
    Un2, _, _, _ = spel.stiefel_step(U, G, np.zeros((d, r)), 1e-2, 0.95, mode="pe")
    assert np.abs(Un2 - U).max() < 1e-8


def test_fp32_symmetric_gradient_zero_rule():
    """G = U S (S symmetric) stored in fp32, as the GPU receives it: the
    stored G keeps a tangent residue of a few 1e-8 of ||G||_F, far below
    fp32 resolution.  The iteration-matched step maps such a momentum to
    D = 0 (||M||_F <= 2^-20 ||G||_F), so U moves only by the retraction's
    rounding; without the rule the residue would be blown up to a full
    lr-sized step.  A small but resolvable tangent gradient (1e-4 of ||G||)
    still takes the full step."""
    rng = np.random.default_rng(37)
    d, r, lr = 256, 64, 1e-2
    U = _orth(rng, d, r).astype(np.float32).astype(np.float64)
    S = rng.standard_normal((r, r))
    G = (U @ (S + S.T)).astype(np.float32).astype(np.float64)
    gR = spel.tangent_project(U, G)
    res = np.linalg.norm(gR) / np.linalg.norm(G)
    assert 1e-9 < res < 1e-6, res
    Un, Mn, D, _ = spel.stiefel_step(U, G, np.zeros((d, r)), lr, 0.95, mode="pe")
    assert np.abs(D).max() == 0.0
    assert np.abs(Un - U).max() < 1e-6
    # without the rule (the bare normalisation) the step is lr-sized
    D_raw = spel.lmo_pe(Mn, 5)
    assert np.linalg.norm(D_raw) > 0.5 * np.sqrt(r)
    # a resolvable tangent part is not suppressed
    K = rng.standard_normal((r, r))
    Gt = G + 1e-4 * np.linalg.norm(G) / np.linalg.norm(K) * U @ (K - K.T) / np.sqrt(2)
    Un2, _, D2, _ = spel.stiefel_step(U, Gt, np.zeros((d, r)), lr, 0.95, mode="pe")
    assert np.linalg.norm(D2) > 0.5 * np.sqrt(r)
    assert np.abs(Un2 - U).max() > 1e-3


# ---------------------------------------------------------------- P9 beta independence
@pytest.mark.parametrize("mode", ["exact", "pe"])
def test_first_step_independent_of_beta(mode):
    """From M = 0 the first momentum is (1 - beta) g_R and the polar factor is
    scale-invariant, so beta drops out.  PolarExpress normalises by
    ||M||_F + 1e-7, so there the independence holds up to that 1e-7 (the
    gradient is scaled to make it invisible)."""
    rng = np.random.default_rng(36)
    U = _orth(rng, 20, 4)
    G = 1e4 * rng.standard_normal((20, 4))
    a = spel.stiefel_step(U, G, np.zeros((20, 4)), 1e-2, 0.5, mode=mode)[0]
    b = spel.stiefel_step(U, G, np.zeros((20, 4)), 1e-2, 0.99, mode=mode)[0]
    assert np.abs(a - b).max() < (1e-12 if mode == "exact" else 1e-10)


# ---------------------------------------------------------------- P10 spectral pin of PolarExpress
def test_polar_express_acts_on_singular_values():
    rng = np.random.default_rng(37)
    d, r = 30, 7
    W = _orth(rng, d, r)
    V = _orth(rng, r, r)
    sig = np.array([3.0, 1.0, 0.5, 0.1, 0.02, 0.004, 0.0005])
    M = W @ np.diag(sig) @ V.T
    D = spel.lmo_pe(M, 5)
    y = ps.compose(ps.greedy_schedule(spel.LMO_LOWER, 5)[0], sig / (np.linalg.norm(sig) + spel.LMO_EPS))
    assert np.abs(D - W @ np.diag(y) @ V.T).max() < 1e-12


def test_pe_converges_to_exact_polar():
    rng = np.random.default_rng(38)
    M = rng.standard_normal((50, 10))
    D = spel.lmo_pe(M, 12)
    assert np.abs(D - spel.polar_exact(M)).max() < 1e-10


# ---------------------------------------------------------------- schedule pins
@pytest.mark.parametrize("lo,hi", [(1e-3, 1.0), (0.0354, 1.9646), (0.5, 1.0), (0.9, 1.1)])
def test_minimax_quintic_equioscillates(lo, hi):
    """Odd quintics span a Chebyshev system on (0, inf); the best approximation
    of 1 on [lo, hi] is characterised by 4 alternating extrema of equal size.
    Check that on a dense grid, and that no random nearby polynomial does
    better (local optimality)."""
    a, b, c, E = ps.minimax_quintic(lo, hi)
    xs = np.linspace(lo, hi, 200001)
    err = 1 - ps._poly((a, b, c), xs)
    assert abs(np.abs(err).max() - E) <= 1e-9 * max(E, 1e-12) + 1e-14
    assert abs(err[0] - E) < 1e-12  # 1 - p(lo) = +E
    # four alternating extrema
    crit = ps._critical_points((a, b, c), lo, hi)
    pts = np.array([lo] + crit + [hi])
    e = 1 - ps._poly((a, b, c), pts)
    assert np.allclose(np.abs(e), E, rtol=1e-9, atol=1e-15)
    assert np.all(np.sign(e) == np.array([1, -1, 1, -1]))
    rng = np.random.default_rng(0)
    for _ in range(200):
        p = np.array([a, b, c]) * (1 + 1e-4 * rng.standard_normal(3))
        assert np.abs(1 - ps._poly(p, xs)).max() >= E * (1 - 1e-9)


def test_schedule_intervals_chain_and_contact_polynomial():
    coefs, iv = ps.greedy_schedule(1e-3, 8)
    for t in range(len(coefs) - 1):
        lo, hi = iv[t]
        xs = np.linspace(lo, hi, 100001)
        ys = ps._poly(coefs[t], xs)
        # the image of [lo, hi] is the next design interval
        assert abs(ys.min() - iv[t + 1][0]) < 1e-9 and abs(ys.max() - iv[t + 1][1]) < 1e-9
    # once the interval has collapsed, p(1) = 1, p'(1) = 0, p''(1) = 0
    a, b, c = coefs[-1]
    assert abs(a + b + c - 1) < 1e-15
    assert abs(a + 3 * b + 5 * c) < 1e-12
    assert abs(6 * b + 20 * c) < 1e-12


def test_schedule_worst_case_error_decreases():
    xs = np.geomspace(1e-3, 1, 5001)
    errs = [np.abs(1 - ps.compose(ps.greedy_schedule(1e-3, n)[0], xs)).max() for n in range(1, 9)]
    assert all(e2 < e1 for e1, e2 in zip(errs, errs[1:]) if e1 > 1e-12)
    assert errs[-1] < 1e-12
    xs2 = np.linspace(0.5, 1, 5001)
    assert np.abs(1 - ps.compose(ps.greedy_schedule(0.5, 7)[0], xs2)).max() < 1e-14


def test_batched_step_equals_loop():
    rng = np.random.default_rng(39)
    P, d, r = 3, 12, 4
    U = np.stack([_orth(rng, d, r) for _ in range(P)])
    G = rng.standard_normal((P, d, r))
    M = rng.standard_normal((P, d, r)) * 0.1
    Un, Mn = spel.stiefel_step_batched(U, G, M, 1e-2, 0.9, mode="pe")
    for p in range(P):
        u, m, _, _ = spel.stiefel_step(U[p], G[p], M[p], 1e-2, 0.9, mode="pe")
        assert np.array_equal(u, Un[p]) and np.array_equal(m, Mn[p])
