"""GPU parity of the grouped RVQ (Sec. 3.5, the coordinates decomposed into
groups; App. E: group dimension 2, K = 256, R = 2), through the whole chain:
codes bit-exact per (token, group) except near ties (counted), Xhat, dZ, dX
and dU within the path's tolerance."""
import numpy as np
import pytest

from oracle import codec as ocodec
from paper_2606_05484_amd import mapl, synth
from _helpers import (Dev, chain, check_chain, codes_np, compare_codes, descr, f64, grouped_stress_codebooks,
                      operand, run_encode, torch)

pytestmark = pytest.mark.gpu

BASE = dict(V=500, dtype="bf16", alpha=0.8, n_out=4, cb_sigma=None, gscale=1.0, group_dim=2)


@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("r,L,K,T", [(64, 1, 64, 1000), (256, 2, 256, 1537), (128, 4, 96, 777), (512, 8, 256, 300),
                                     (64, 3, 32, 1)],
                         ids=["r64L1", "r256L2K256", "r128L4", "r512L8", "T1"])
def test_grouped_chain_bf16(r, L, K, T, space):
    """Ragged token counts, one to eight rounds (the wider ones with fewer
    groups per workgroup), stress codebooks drawn from the data."""
    x = synth.codec_inputs(None, seed=600 + r + L, T=T, d=max(512, r), r=r, k=16, L=L, K=K, anchor_space=space,
                           **BASE)
    C = grouped_stress_codebooks(x, 700 + r) if T >= K else x["C"]
    print("grouped", r, L, K, T, space, flush=True)
    check_chain(x, chain(x, C=C), C=C)


@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_grouped_chain_fp32(space):
    x = synth.codec_inputs("c1", anchor_space=space, group_dim=2)
    print("grouped fp32", space, flush=True)
    check_chain(x, chain(x))


def test_grouped_planted_and_tied_codewords():
    """Codeword 1 + j of round 0 holds token j's coordinates in every group:
    those tokens pick it in every group (residual 0, then the zero codeword
    in round 1); codeword 40 is overwritten with a duplicate of codeword 7,
    and token 6 resolves the tie to the lower index in every group."""
    x = synth.codec_inputs(None, seed=610, T=300, d=512, r=128, k=16, L=2, K=64, **BASE)
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), "ambient", operand(x))
    C = np.zeros((2, 64, 128), dtype=np.float32)
    C[0, 1:] = Z0[:63].astype(np.float32)
    C[0, 40] = C[0, 7]  # duplicate of codeword 7 (token 6)
    C[1, 1:] = (9 + np.random.default_rng(1).standard_normal((63, 128))).astype(np.float32)
    D = descr(x)
    g = Dev(x, C)
    codes = codes_np(run_encode(x, D, g), D)
    for j in range(63):
        if j == 39:  # its codeword was overwritten
            continue
        assert np.all(codes[j, 0] == 1 + j), (j, codes[j, 0][:8])
        assert np.all(codes[j, 1] == 0)


@pytest.mark.slow
def test_c6_full_size():
    """The paper's VQ setting at the 150M boundary (T = 8192, d = 1024,
    r = 256, group dimension 2, K = 256, R = 2: 256 bytes per token) with
    the generator's codebooks (2-D Gaussian codewords of the data's spread:
    every code in use), the whole chain against the oracle."""
    x = synth.codec_inputs("c6")
    res = chain(x)
    used = len(np.unique(codes_np(res["payload"], res["D"])[:, 0, :]))
    print("c6 distinct round-0 codes", used, flush=True)
    assert used > 200
    check_chain(x, res)
