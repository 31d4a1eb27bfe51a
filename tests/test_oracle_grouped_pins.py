"""Pins of the grouped RVQ oracle (Sec. 3.5, coordinates decomposed into
groups; App. E: K = 256 codewords, R = 2 rounds, group dimension 2)."""
import json
import os

import numpy as np

from oracle import codec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_grouped_matches_per_group_bruteforce():
    """Pure-Python loops: for every token and every group of two coordinates,
    round by round, the codeword whose two coordinates are nearest (explicit
    squared differences, lowest index on ties)."""
    rng = np.random.default_rng(60)
    T, r, L, K, gd = 9, 6, 2, 7, 2
    Z0 = rng.standard_normal((T, r))
    C = rng.standard_normal((L, K, r))
    C[:, 0] = 0.0
    codes, _, _ = codec.grouped_rvq_encode(Z0, C, gd)
    for t in range(T):
        for g in range(r // gd):
            res = [float(Z0[t, gd * g + c]) for c in range(gd)]
            for l in range(L):
                best, bj = None, -1
                for j in range(K):
                    s = sum((res[c] - float(C[l, j, gd * g + c])) ** 2 for c in range(gd))
                    if best is None or s < best:
                        best, bj = s, j
                assert codes[t, l, g] == bj
                res = [res[c] - float(C[l, bj, gd * g + c]) for c in range(gd)]


def test_group_of_the_whole_vector_is_plain_rvq():
    rng = np.random.default_rng(61)
    Z0 = rng.standard_normal((40, 8))
    C = rng.standard_normal((3, 11, 8))
    C[:, 0] = 0
    a, ga, ra = codec.grouped_rvq_encode(Z0, C, 8)
    b, gb, rb = codec.rvq_encode(Z0, C)
    assert np.array_equal(a[:, :, 0], b) and np.allclose(ra[:, :, 0], rb)
    # the same gaps, measured against ||Z0||^2 instead of each round's ||R_l||^2
    assert np.allclose(ga[:, :, 0], gb * rb[:, :3] / rb[:, :1])


def test_planted_group_codewords_reconstruct_exactly_and_error_never_grows():
    """Codeword j + 1 of round 0 holds token j's coordinates in every group,
    so the codes reproduce the tokens and the decode is exact; with random
    codebooks that contain the zero codeword, every group's residual norm is
    non-increasing over the rounds."""
    rng = np.random.default_rng(62)
    T, r = 12, 10
    Z0 = rng.standard_normal((T, r))
    C = np.zeros((2, T + 1, r))
    C[0, 1:] = Z0
    C[1, 1:] = 3 + rng.standard_normal((T, r))
    codes, _, _ = codec.grouped_rvq_encode(Z0, C, 2)
    assert np.all(codes[:, 0, :] == np.arange(1, T + 1)[:, None]) and np.all(codes[:, 1, :] == 0)
    assert np.abs(codec.grouped_rvq_decode(codes, C, 2) - Z0).max() == 0.0
    C2 = rng.standard_normal((4, 16, r))
    C2[:, 0] = 0
    _, _, rs = codec.grouped_rvq_encode(Z0, C2, 2)
    assert np.all(np.diff(rs, axis=1) <= 1e-12)


def test_paper_vq_payload_bytes():
    """Table 1's MAPL+VQ rows: 256 bytes per token at every scale (8x, 12x,
    16x against the bf16 boundary), from App. E's setting at r = 256: r / 2
    groups, R = 2 rounds of one-byte codes (K = 256)."""
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "paper_bytes_per_token.json")))
    for row in g["mapl_vq"]:
        groups = row["r"] // row["group_dim"]
        bits = int(np.log2(row["K"]))
        assert groups * row["R"] * bits // 8 == row["bytes"]
        assert 2 * row["d"] // row["bytes"] == row["compression"]


def test_grouped_gap_is_relative_to_the_groups_energy():
    """Hand-worked: one group, Z0 = (3, 0), codewords (0,0), (1,0), (2,0),
    (5,0).  Round 0: distances 9, 4, 1, 4 -> code 2, top-2 gap 3; round 1
    (residual (1, 0)): distances 1, 0, 1, 16 -> code 1, gap 1.  Both gaps are
    divided by the group's unquantised energy ||Z0||^2 = 9: 1/3 and 1/9."""
    C = np.zeros((2, 4, 2))
    C[:, :, 0] = [0.0, 1.0, 2.0, 5.0]
    codes, gap, rs = codec.grouped_rvq_encode(np.array([[3.0, 0.0]]), C, 2)
    assert codes[0, :, 0].tolist() == [2, 1]
    assert np.allclose(gap[0, :, 0], [1 / 3, 1 / 9], rtol=0, atol=1e-15)
    assert np.allclose(rs[0, :, 0], [9.0, 1.0, 0.0], rtol=0, atol=1e-15)
