"""Pins of the gradient-quantisation oracle (Sec. 3.5: the quantiser also
compresses the backward gradients; the gradient crossing back is the r-dim
dZhat = dXhat U of Eq. 2's backward)."""
import numpy as np

from oracle import codec


def _orth(rng, n, m):
    q, _ = np.linalg.qr(rng.standard_normal((n, m)))
    return q


def test_grad_quantize_matches_per_token_bruteforce():
    """Per token, in plain loops: the gradient row dXhat[t] U, then for each
    round the codeword with the smallest explicit squared difference (lowest
    index on ties), then the residual update."""
    rng = np.random.default_rng(40)
    T, d, r, L, K = 17, 12, 5, 2, 7
    dXh = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    Cg = rng.standard_normal((L, K, r))
    Cg[:, 0] = 0.0
    codes, _, _ = codec.grad_quantize(dXh, U, Cg)
    for t in range(T):
        res = [sum(dXh[t, i] * U[i, c] for i in range(d)) for c in range(r)]
        for l in range(L):
            dist = [sum((res[c] - Cg[l, j, c]) ** 2 for c in range(r)) for j in range(K)]
            j = int(np.argmin(dist))
            assert codes[t, l] == j
            res = [res[c] - Cg[l, j, c] for c in range(r)]


def test_planted_gradient_codebook_round_trip_is_exact():
    """When the gradient codebook holds every token's gradient row (and the
    zero codeword), the codes reproduce the rows, the reconstruction is the
    exact gradient, and the sender's backward (Eq. 1's dX and dU) is the
    unquantised one."""
    rng = np.random.default_rng(41)
    T, d, r, V, k = 11, 16, 6, 9, 3
    dXh = rng.standard_normal((T, d))
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    ids = rng.integers(0, V, T)
    A, B = rng.standard_normal((V, k)), rng.standard_normal((k, d))
    dZ0 = dXh @ U
    Cg = np.zeros((2, T + 1, r))
    Cg[0, 1:] = dZ0
    Cg[1, 1:] = 4.0 + rng.standard_normal((T, r))
    codes, _, rs = codec.grad_quantize(dXh, U, Cg)
    assert np.array_equal(codes[:, 0], np.arange(1, T + 1)) and np.all(codes[:, 1] == 0)
    dZq = codec.grad_dequantize(codes, Cg)
    assert np.abs(dZq - dZ0).max() < 1e-14
    dX_q, dU_q = codec.encode_bwd(dZq, X, ids, U, A, B)
    dX_0, dU_0 = codec.encode_bwd(dZ0, X, ids, U, A, B)
    assert np.abs(dX_q - dX_0).max() < 1e-12 and np.abs(dU_q - dU_0).max() < 1e-12
    # the gradient quantised is the decoder backward's dZhat, not dXhat itself
    dZ_dec, _ = codec.decode_bwd(dXh, np.zeros((T, r)), ids, U, A, B)
    assert np.abs(dZ_dec - dZ0).max() < 1e-14
