"""Pins of the float64 codec oracle against facts fixed by the paper and by
mathematics (not against the oracle itself).

Eq. 1 / Eq. 2 of Sec. 3.2 with an orthonormal projector; RVQ of Sec. 3.5."""
import itertools

import numpy as np
import pytest

from oracle import codec, precision
from paper_2606_05484_amd import synth


def _orth(rng, n, m):
    q, _ = np.linalg.qr(rng.standard_normal((n, m)))
    return q


# ---------------------------------------------------------------- P1 identity
@pytest.mark.parametrize("with_anchor", [False, True])
def test_roundtrip_identity_full_rank(with_anchor):
    """r = d, no RVQ: Eq. 2 inverts Eq. 1 exactly when U is square orthogonal
    and both sides use the same anchor (or none)."""
    rng = np.random.default_rng(11)
    T, d, V, k = 37, 24, 50, 5
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, d)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k)) if with_anchor else np.zeros((V, k))
    B = rng.standard_normal((k, d))
    Z = codec.encode(X, ids, U, A, B)
    Xh = codec.decode(Z, ids, U, A, B)
    assert np.abs(Xh - X).max() < 1e-12


@pytest.mark.parametrize("with_rvq", [False, True])
def test_roundtrip_identity_full_rank_coord(with_rvq):
    """Coordinate-space anchor (Eq. 1-2 with the anchor removed after the
    projection and added back before the lift): with r = d and the same
    anchor on both sides, decode(encode(X)) = X.  With RVQ the codebook
    holds every token's Z0 exactly (plus a zero codeword), so the codes
    reproduce Z0 and the round trip is still the identity.  Dropping the
    anchor add-back, or adding it after the lift, breaks the identity by the
    size of the anchor term (checked to be large)."""
    rng = np.random.default_rng(15)
    T, d, V, k = 29, 20, 40, 6
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, d)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k))
    B = rng.standard_normal((k, d))   # coord: B is [k, r] and r = d
    Z0 = codec.encode(X, ids, U, A, B, anchor_space="coord")
    if with_rvq:
        C = np.zeros((2, T + 1, d))
        C[0, 1:] = Z0
        C[1, 1:] = 3.0 + rng.standard_normal((T, d))
        codes, _, rs = codec.rvq_encode(Z0, C)
        assert np.array_equal(codes[:, 0], np.arange(1, T + 1)) and np.all(codes[:, 1] == 0)
        Xh = codec.decode(codes, ids, U, A, B, C, anchor_space="coord")
    else:
        Xh = codec.decode(Z0, ids, U, A, B, anchor_space="coord")
    assert np.abs(Xh - X).max() < 1e-12
    anchor_term = (A[ids] @ B) @ U.T
    assert np.abs(anchor_term).max() > 0.5
    # the ambient reading adds a B (not a B U^T): a different map here
    Xh_amb = codec.decode(Z0, ids, U, A, B, anchor_space="ambient")
    assert np.abs(Xh_amb - X).max() > 0.1


def test_roundtrip_identity_no_anchor_k0():
    rng = np.random.default_rng(12)
    X = rng.standard_normal((9, 16))
    U = _orth(rng, 16, 16)
    ids = np.zeros(9, dtype=int)
    A = np.zeros((4, 0))
    B = np.zeros((0, 16))
    Xh = codec.decode(codec.encode(X, ids, U, A, B), ids, U, A, B)
    assert np.abs(Xh - X).max() < 1e-12


# ---------------------------------------------------------------- P2 idempotence
def test_roundtrip_idempotent_low_rank():
    """With r < d and the same anchor on both sides, x -> (x - aB)UU^T + aB is
    an affine projection: applying it twice equals applying it once."""
    rng = np.random.default_rng(13)
    T, d, r, V, k = 41, 32, 7, 20, 6
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k))
    B = rng.standard_normal((k, d))
    f = lambda Y: codec.decode(codec.encode(Y, ids, U, A, B), ids, U, A, B)
    Y1 = f(X)
    Y2 = f(Y1)
    assert np.abs(Y2 - Y1).max() < 1e-12
    # and it is not the identity
    assert np.abs(Y1 - X).max() > 1e-2
    # the residual it removes is orthogonal to span(U)
    R = (X - Y1)
    assert np.abs(R @ U).max() < 1e-12


def test_encode_coord_vs_ambient_relation():
    """coord reading with B_r = B_d U equals the ambient Eq. 1."""
    rng = np.random.default_rng(14)
    T, d, r, V, k = 15, 12, 5, 9, 3
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k))
    Bd = rng.standard_normal((k, d))
    z_amb = codec.encode(X, ids, U, A, Bd, anchor_space="ambient")
    z_crd = codec.encode(X, ids, U, A, Bd @ U, anchor_space="coord")
    # brute force: per-token loop
    z_bf = np.array([(X[t] - A[ids[t]] @ Bd) @ U for t in range(T)])
    assert np.abs(z_amb - z_bf).max() < 1e-12
    assert np.abs(z_crd - z_bf).max() < 1e-12


def test_anchor_gather_range_check():
    A = np.zeros((4, 2))
    with pytest.raises(IndexError):
        codec.anchor(A, np.array([0, 4]))


# ---------------------------------------------------------------- P3 brute-force argmin
def _bruteforce_rvq(Z0, C):
    """Pure-Python loops: the nearest codeword by explicit squared differences,
    first index on ties."""
    T, r = Z0.shape
    L, K, _ = C.shape
    codes = np.zeros((T, L), dtype=int)
    for t in range(T):
        res = [float(v) for v in Z0[t]]
        for l in range(L):
            best, bj = None, -1
            for j in range(K):
                s = 0.0
                for c in range(r):
                    diff = res[c] - float(C[l, j, c])
                    s += diff * diff
                if best is None or s < best:
                    best, bj = s, j
            codes[t, l] = bj
            res = [res[c] - float(C[l, bj, c]) for c in range(r)]
    return codes


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_rvq_matches_bruteforce(seed):
    rng = np.random.default_rng(100 + seed)
    T, r, L, K = 23, 6, 3, 9
    Z0 = rng.standard_normal((T, r))
    C = rng.standard_normal((L, K, r)) * 0.7
    C[:, 0] = 0.0
    codes_e, _, _ = codec.rvq_encode(Z0, C)
    codes_d, _, _ = codec.rvq_encode(Z0, C, direct=True)
    codes_b = _bruteforce_rvq(Z0, C)
    assert np.array_equal(codes_e, codes_b)
    assert np.array_equal(codes_d, codes_b)


# ---------------------------------------------------------------- P4 monotone error
def test_rvq_error_non_increasing_with_zero_codeword():
    rng = np.random.default_rng(7)
    T, r, L, K = 300, 8, 5, 16
    Z0 = rng.standard_normal((T, r))
    C = rng.standard_normal((L, K, r))
    C[:, 0] = 0.0
    _, _, rs = codec.rvq_encode(Z0, C)
    assert np.all(np.diff(rs, axis=1) <= 1e-12)
    # the last column is exactly the reconstruction error
    Zh = codec.rvq_decode(codec.rvq_encode(Z0, C)[0], C)
    assert np.allclose(rs[:, -1], ((Z0 - Zh) ** 2).sum(1), rtol=0, atol=1e-12)


# ---------------------------------------------------------------- P5 planted codewords
def test_rvq_planted_codewords_and_tie_break():
    rng = np.random.default_rng(8)
    T, r, L, K = 12, 5, 3, 10
    Z0 = rng.standard_normal((T, r))
    C = 5.0 + rng.standard_normal((L, K, r))  # far from the data
    C[:, 0] = 0.0
    planted = {3: 4, 7: 9, 0: 2}
    for t, j in planted.items():
        C[0, j] = Z0[t]
    # duplicate of codeword 4 at index 6 -> tie, lowest index (4) must win
    C[0, 6] = C[0, 4]
    codes, gap, rs = codec.rvq_encode(Z0, C, direct=True)
    for t, j in planted.items():
        assert codes[t, 0] == j
        assert rs[t, 1] == 0.0
        assert np.all(codes[t, 1:] == 0)
    assert gap[3, 0] == 0.0  # an exact tie is reported as a zero gap


def test_rvq_top2_gap_hand_computed():
    """The near-tie measure of the comparison rule, on numbers worked out by
    hand: gap = (second-smallest - smallest squared distance) / ||R||^2,
    where ||R||^2 is the round's residual norm (the distance to the zero
    codeword).  Codewords on a line: (0,0), (1,0), (2,0), (5,0).

      token a, R0 = (3,0): distances 9, 4, 1, 4  -> code 2, gap (4-1)/9 = 1/3
               R1 = (1,0): distances 1, 0, 1, 16 -> code 1, gap (1-0)/1 = 1
      token b, R0 = (0,2): distances 4, 5, 8, 29 -> code 0, gap (5-4)/4 = 1/4
               R1 = (0,2): same                  -> code 0, gap 1/4
      token c, R0 = (1.5,0): distances 2.25, 0.25, 0.25, 12.25 -> tie of 1
               and 2, lowest index 1, gap 0; R1 = (0.5,0): distances 0.25,
               0.25, 2.25, 20.25 -> code 0, gap 0

    A denominator of the smallest distance instead of ||R||^2 would give 3
    for token a's first round; a gap measured from the zero codeword would
    give (9-1)/9."""
    C = np.zeros((2, 4, 2))
    C[:, :, 0] = [0.0, 1.0, 2.0, 5.0]
    Z0 = np.array([[3.0, 0.0], [0.0, 2.0], [1.5, 0.0]])
    codes, gap, rs = codec.rvq_encode(Z0, C, direct=True)
    assert codes.tolist() == [[2, 1], [0, 0], [1, 0]]
    assert np.allclose(gap, [[1 / 3, 1.0], [0.25, 0.25], [0.0, 0.0]], rtol=0, atol=1e-15)
    assert np.allclose(rs, [[9.0, 1.0, 0.0], [4.0, 4.0, 4.0], [2.25, 0.25, 0.25]], rtol=0, atol=1e-15)
    codes_e, gap_e, _ = codec.rvq_encode(Z0, C)
    assert np.array_equal(codes_e, codes) and np.allclose(gap_e, gap, rtol=0, atol=1e-14)


# ---------------------------------------------------------------- P6 adjoints and finite differences
@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_backward_adjoint_identities(space):
    rng = np.random.default_rng(21)
    T, d, r, V, k = 19, 14, 5, 11, 3
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k))
    B = rng.standard_normal((k, d if space == "ambient" else r))
    # encode is affine in X: J_X = right-multiplication by U
    dZ = rng.standard_normal((T, r))
    dX, _ = codec.encode_bwd(dZ, X, ids, U, A, B, anchor_space=space)
    dlt = rng.standard_normal((T, d))
    lin = codec.encode(X + dlt, ids, U, A, B, anchor_space=space) - codec.encode(X, ids, U, A, B, anchor_space=space)
    assert abs(np.sum(dZ * lin) - np.sum(dX * dlt)) < 1e-10
    # decode is affine in Zhat
    Z = rng.standard_normal((T, r))
    dXh = rng.standard_normal((T, d))
    dZh, _ = codec.decode_bwd(dXh, Z, ids, U, A, B, anchor_space=space)
    dz = rng.standard_normal((T, r))
    lin2 = codec.decode(Z + dz, ids, U, A, B, anchor_space=space) - codec.decode(Z, ids, U, A, B, anchor_space=space)
    assert abs(np.sum(dXh * lin2) - np.sum(dZh * dz)) < 1e-10


@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_dU_central_differences_through_chain(space):
    """L = 0: Xhat(U) = decode(encode(X; U); U).  The directional derivative of
    <G, Xhat(U)> along an arbitrary (unconstrained) Delta equals
    <dU_enc + dU_dec, Delta>, where dU_enc uses dZ = G U (the chain rule)."""
    rng = np.random.default_rng(22)
    T, d, r, V, k = 13, 10, 4, 7, 3
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k))
    B = rng.standard_normal((k, d if space == "ambient" else r))
    G = rng.standard_normal((T, d))
    Dl = rng.standard_normal((d, r))

    def f(Um):
        return np.sum(G * codec.decode(codec.encode(X, ids, Um, A, B, anchor_space=space), ids, Um, A, B,
                                       anchor_space=space))

    eps = 1e-5
    fd = (f(U + eps * Dl) - f(U - eps * Dl)) / (2 * eps)
    Z = codec.encode(X, ids, U, A, B, anchor_space=space)
    dZh, dU_dec = codec.decode_bwd(G, Z, ids, U, A, B, anchor_space=space)
    _, dU_enc = codec.encode_bwd(dZh, X, ids, U, A, B, anchor_space=space)
    an = np.sum((dU_enc + dU_dec) * Dl)
    assert abs(fd - an) <= 1e-7 * max(1.0, abs(an))


def test_straight_through_ignores_quantiser():
    """STE: with codebooks the backward calls are those of L = 0 evaluated at
    the decoded coordinates (the quantiser passes gradients unchanged)."""
    rng = np.random.default_rng(23)
    T, d, r, V, k, L, K = 9, 8, 3, 5, 2, 2, 4
    U = _orth(rng, d, r)
    ids = rng.integers(0, V, T)
    A = rng.standard_normal((V, k))
    B = rng.standard_normal((k, d))
    C = rng.standard_normal((L, K, r))
    codes = rng.integers(0, K, (T, L))
    dXh = rng.standard_normal((T, d))
    dZ1, dU1 = codec.decode_bwd(dXh, codes, ids, U, A, B, C)
    Zh = codec.rvq_decode(codes, C)
    dZ2, dU2 = codec.decode_bwd(dXh, Zh, ids, U, A, B, None)
    assert np.array_equal(dZ1, dZ2) and np.array_equal(dU1, dU2)


# ---------------------------------------------------------------- precision helpers
def test_bf16_rounding_known_values():
    """bf16 keeps 8 significant bits: 1 + 2^-8 is a tie and rounds to even (1),
    1 + 3*2^-8 rounds up to 1 + 2^-6, and the largest bf16 below 2 is 2 - 2^-7."""
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 2 - 2 ** -8, -3.0, 0.0])
    y = precision.round_bf16(x)
    assert list(y) == [1.0, 1.0, 1.0 + 2 ** -6, 2.0, -3.0, 0.0]
    assert precision.round_bf16(np.array([2 - 2 ** -7]))[0] == 2 - 2 ** -7


def test_bf16_matches_generator_and_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(10000) * 10.0 ** rng.integers(-8, 8, 10000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(precision.round_bf16(x.astype(np.float64)), ref)
    assert np.array_equal(synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(x)).astype(np.float64), ref)


# ---------------------------------------------------------------- P12 energy diagnostic
def test_retained_energy_equals_cumulative_energy():
    """Sec. 3.1 / Sec. 3.4: for U = top-r right singular vectors of the
    anchor-free residual, ||X_res U||^2 / ||X_res||^2 = E(r)."""
    x = synth.codec_inputs(None, seed=9, T=600, d=64, r=16, V=100, k=4, L=0, K=0, dtype="f32",
                           alpha=0.8, n_out=2, cb_sigma=0.0, gscale=1.0)
    X = x["X"].astype(np.float64)
    A = x["A"].astype(np.float64)
    B = x["B"].astype(np.float64)
    Xres = X - A[x["ids"]] @ B
    _, s, Vt = np.linalg.svd(Xres, full_matrices=False)
    for r in (1, 8, 16, 40):
        U = Vt[:r].T
        Z = codec.encode(X, x["ids"], U, A, B)
        e_proj = (Z ** 2).sum() / (Xres ** 2).sum()
        e_spec = (s[:r] ** 2).sum() / (s ** 2).sum()
        assert abs(e_proj - e_spec) < 1e-12
