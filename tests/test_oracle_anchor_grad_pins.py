"""Pins of the anchor-table gradient oracle (Eq. 3: E_small is trainable;
it enters Eq. 1 on the sender and Eq. 2 on the receiver).  The loss is
linear in the table, so a central difference of the loss through the
codec's forward (encode / decode, themselves pinned) equals the directional
derivative <dA, delta> exactly."""
import numpy as np
import pytest

from oracle import codec
from oracle.precision import round_bf16


def _orth(rng, n, m):
    q, _ = np.linalg.qr(rng.standard_normal((n, m)))
    return q


def _setup(seed, space, d=14, r=5, V=9, k=3, T=23):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, d))
    U = _orth(rng, d, r)
    ids = np.concatenate([[0, 0, 0], rng.integers(0, V, T - 3)])  # a repeated (hot) id
    A = rng.standard_normal((V, k))
    B = rng.standard_normal((k, d if space == "ambient" else r))
    return rng, X, U, ids, A, B


@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_sender_table_gradient_matches_central_difference(space):
    rng, X, U, ids, A, B = _setup(50, space)
    dZ = rng.standard_normal((X.shape[0], U.shape[1]))
    dA = codec.anchor_grad(dZ, ids, U, B, A.shape[0], "sender", space)
    for _ in range(3):
        delta = rng.standard_normal(A.shape)
        eps = 1e-3
        lp = np.sum(dZ * codec.project(X, ids, U, A + eps * delta, B, space))
        lm = np.sum(dZ * codec.project(X, ids, U, A - eps * delta, B, space))
        assert abs((lp - lm) / (2 * eps) - np.sum(dA * delta)) < 1e-9


@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_receiver_table_gradient_matches_central_difference(space):
    rng, X, U, ids, A, B = _setup(51, space)
    T, r = X.shape[0], U.shape[1]
    Zh = rng.standard_normal((T, r))
    dXh = rng.standard_normal(X.shape)
    dY = dXh if space == "ambient" else dXh @ U
    dA = codec.anchor_grad(dY, ids, U, B, A.shape[0], "receiver", space)
    for _ in range(3):
        delta = rng.standard_normal(A.shape)
        eps = 1e-3
        lp = np.sum(dXh * codec.decode(Zh, ids, U, A + eps * delta, B, None, space))
        lm = np.sum(dXh * codec.decode(Zh, ids, U, A - eps * delta, B, None, space))
        assert abs((lp - lm) / (2 * eps) - np.sum(dA * delta)) < 1e-9


def test_absent_ids_get_zero_rows_and_bf16_factor_matches_encoder():
    """Rows of ids no token carries are zero; with bf16 operands the sender's
    factor is the encoder's rounded (B U~)~, so the gradient is that of the
    bf16 encoder's forward (checked by central difference through project
    with operand bf16)."""
    rng, X, U, ids, A, B = _setup(52, "ambient", V=40)
    dZ = rng.standard_normal((X.shape[0], U.shape[1]))
    dA = codec.anchor_grad(dZ, ids, U, B, 40, "sender", "ambient", "bf16")
    absent = np.setdiff1d(np.arange(40), ids)
    assert absent.size > 0 and np.all(dA[absent] == 0)
    delta = rng.standard_normal(A.shape)
    eps = 1e-3
    lp = np.sum(dZ * codec.project(X, ids, U, A + eps * delta, B, "ambient", "bf16"))
    lm = np.sum(dZ * codec.project(X, ids, U, A - eps * delta, B, "ambient", "bf16"))
    assert abs((lp - lm) / (2 * eps) - np.sum(dA * delta)) < 1e-9
    # and it differs from the unrounded factor's gradient
    dA_exact = codec.anchor_grad(dZ, ids, U, B, 40, "sender", "ambient", "exact")
    assert np.abs(dA - dA_exact).max() > 1e-6
