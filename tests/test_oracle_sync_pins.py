"""Pins of the streaming codebook synchronisation oracle (Sec. 3.5, App. F):
facts fixed by the protocol itself, not by the oracle's code."""
import numpy as np

from oracle import codebook_sync as cs


def test_one_fifth_per_micro_batch():
    """K = 1024 codewords in 5 parts (the paper's 1/5 refresh): parts of 205
    and 204 codewords, together every index exactly once."""
    perm = np.random.default_rng(0).permutation(1024)
    parts = cs.partition(perm, 5)
    assert [len(p) for p in parts] == [205, 205, 205, 205, 204]
    assert np.array_equal(np.sort(np.concatenate(parts)), np.arange(1024))


def test_full_cycle_reproduces_static_codebook_bitwise():
    """With a static sender codebook, one cycle of the partition makes the
    receiver's copy identical; after m < parts micro-batches exactly the
    codewords of the first m parts are fresh."""
    rng = np.random.default_rng(1)
    L, K, r, parts = 2, 1024, 16, 5
    C = rng.standard_normal((L, K, r)).astype(np.float32)
    perms = [rng.permutation(K) for _ in range(L)]
    recv = np.full_like(C, np.nan)
    sent = 0
    for m in range(parts):
        rows = np.stack([cs.partition(perms[l], parts)[m] for l in range(L)])
        recv = cs.unpack(recv, cs.pack(C, rows), rows)
        sent += rows.shape[1]
        assert np.isnan(recv).any(axis=2).sum() == L * (K - sent)
    assert np.array_equal(recv, C)


def test_staleness_bounded_by_cycle():
    """A codebook that changes every micro-batch: after each full cycle every
    receiver codeword equals the sender's version of at most parts - 1
    micro-batches earlier (the staleness the protocol accepts)."""
    rng = np.random.default_rng(2)
    L, K, r, parts = 1, 60, 4, 5
    perm = rng.permutation(K)
    recv = np.zeros((L, K, r))
    history = []
    C = rng.standard_normal((L, K, r))
    for m in range(3 * parts):
        C = C + 0.01 * rng.standard_normal(C.shape)
        history.append(C.copy())
        rows = cs.partition(perm, parts)[m % parts][None, :]
        recv = cs.unpack(recv, cs.pack(C, rows), rows)
        if m >= parts - 1:
            age = np.full(K, -1)
            for j in range(K):
                for a in range(parts):
                    if np.array_equal(recv[0, j], history[m - a][0, j]):
                        age[j] = a
                        break
            assert (age >= 0).all() and age.max() <= parts - 1
