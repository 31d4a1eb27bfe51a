"""Float64 oracle of the SPEL projector update (test infrastructure).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use
this module (see oracle/__init__).

Sec. 3.3, Eqs. 4-7 (and the projector-update half of Alg. 1), for one
projector U in St(d, r) with Euclidean gradient G, momentum M, rate alpha,
momentum coefficient beta:

    g_R = G - U sym(U^T G),  sym(S) = (S + S^T) / 2        (Eq. 4)
    M   = beta M + (1 - beta) g_R                            (Eq. 5)
    D   = polar(M)                                           (Eq. 6, LMO)
    U   = polar(U - alpha D)                                 (Eq. 7, retraction)

polar(Y) is the orthogonal polar factor W V^T of the thin SVD Y = W S V^T,
which PolarExpress approximates.  Two modes:

  mode="exact": polar by SVD (the definition).  A matrix whose Frobenius norm
                is at most 1e-12 max(||G||_F, 1) is treated as zero and maps
                to zero (the polar factor of a rounding-noise matrix is
                meaningless; in exact arithmetic such an M is 0).
  mode="pe":    the PolarExpress iteration X <- a X + X (b S + c S^2),
                S = X^T X, with the greedy minimax schedule of
                oracle.polar_schedule, carried out in float64:
                  LMO:        X0 = M / (||M||_F + 1e-7), schedule
                              designed for [1e-3, 1]; D = 0 when
                              ||M||_F <= 2^-20 ||G||_F (zero rule below);
                  retraction: X0 = Y / nu, nu = sqrt(max_i sum_j |(Y^T Y)_ij|)
                              (an upper bound of sigma_max(Y)), schedule
                              designed for [0.5, 1].
                polar(cY) = polar(Y) for c > 0, so both normalisations leave
                the limit unchanged; they fix where the finite schedule is
                accurate.

Zero rule of the LMO (a reading of Eq. 6, where the paper is silent on a
vanishing momentum).  The linear minimisation over the spectral-norm ball
has no unique answer at M = 0; D = 0 is taken there.  Gradients reach the
step as fp32 values, so a tangent part below the fp32 resolution of G is
indistinguishable from zero: G = U S with S symmetric, stored in fp32,
keeps a tangent residue of about 3e-8 ||G||_F, and the scale-invariant polar
factor would blow that residue up to a full unit-singular-value step.  The
iteration-matched mode therefore maps M to D = 0 whenever
||M||_F <= 2^-20 ||G||_F (about 16 fp32 units of G's norm).
"""
import numpy as np

from . import polar_schedule

LMO_LOWER = 1e-3
RETRACT_LOWER = 0.5
LMO_EPS = 1e-7
LMO_ZERO_REL = 2.0 ** -20


def sym(S):
    return 0.5 * (S + S.T)


def tangent_project(U, G):
    """Eq. 4: the Riemannian gradient on St(d, r) (embedded metric)."""
    U = np.asarray(U, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    return G - U @ sym(U.T @ G)


def momentum(M, gR, beta):
    """Eq. 5: heavy-ball momentum."""
    return beta * np.asarray(M, dtype=np.float64) + (1.0 - beta) * gR


def polar_exact(Y, zero_tol=0.0):
    """Orthogonal polar factor W V^T of Y = W S V^T (thin SVD)."""
    Y = np.asarray(Y, dtype=np.float64)
    if np.linalg.norm(Y) <= zero_tol:
        return np.zeros_like(Y)
    W, _, Vt = np.linalg.svd(Y, full_matrices=False)
    return W @ Vt


def pe_iterate(X, coefs):
    """PolarExpress steps X <- a X + X (b S + c S^2), S = X^T X (float64)."""
    for a, b, c in coefs:
        S = X.T @ X
        X = a * X + X @ (b * S + c * (S @ S))
    return X


def lmo_pe(M, steps, zero_below=0.0):
    """Eq. 6 with PolarExpress: D = PE_steps(M / (||M||_F + 1e-7)), and
    D = 0 when ||M||_F <= zero_below (the zero rule above)."""
    coefs, _ = polar_schedule.greedy_schedule(LMO_LOWER, steps)
    M = np.asarray(M, dtype=np.float64)
    if np.linalg.norm(M) <= zero_below:
        return np.zeros_like(M)
    X0 = M / (np.linalg.norm(M) + LMO_EPS)
    return pe_iterate(X0, coefs)


def retract_pe(Y, steps):
    """Eq. 7 with PolarExpress: U = PE_steps(Y / nu)."""
    coefs, _ = polar_schedule.greedy_schedule(RETRACT_LOWER, steps)
    Y = np.asarray(Y, dtype=np.float64)
    S = Y.T @ Y
    nu = np.sqrt(np.abs(S).sum(axis=1).max())
    return pe_iterate(Y / nu, coefs)


def stiefel_step(U, G, M, lr, beta, mode="exact", lmo_steps=5, retract_steps=7):
    """One SPEL step for one projector.  Returns (U_new, M_new, D, g_R)."""
    U = np.asarray(U, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    gR = tangent_project(U, G)
    Mn = momentum(M, gR, beta)
    if mode == "exact":
        zt = 1e-12 * max(np.linalg.norm(G), 1.0)
        D = polar_exact(Mn, zero_tol=zt)
        Un = polar_exact(U - lr * D)
    elif mode == "pe":
        D = lmo_pe(Mn, lmo_steps, zero_below=LMO_ZERO_REL * np.linalg.norm(G))
        Un = retract_pe(U - lr * D, retract_steps)
    else:
        raise ValueError(mode)
    return Un, Mn, D, gR


def stiefel_step_batched(U, G, M, lr, beta, mode="exact", lmo_steps=5, retract_steps=7):
    """Apply stiefel_step to every projector of [P,d,r] stacks."""
    U = np.asarray(U, dtype=np.float64)
    Un = np.empty_like(U)
    Mn = np.empty_like(U)
    for p in range(U.shape[0]):
        Un[p], Mn[p], _, _ = stiefel_step(U[p], G[p], M[p], lr, beta, mode, lmo_steps, retract_steps)
    return Un, Mn
