"""mapl_encode_noalloc (no workspace argument: the library's static device
scratch) against mapl_encode, through the C ABI.  Two calls in a row, the
second with a smaller input, each equal to mapl_encode's output on the same
inputs bit for bit (the same kernels run); cases cover the fused r = 256
encoder (projection + RVQ, codebook copies in the scratch), the two-launch
r = 128 encoder (fp32 Z0 in the scratch as well) and the unquantised
payload."""
import numpy as np
import pytest

from paper_2606_05484_amd import mapl, synth
from _helpers import Dev, codes_np, descr, run_encode, stress_codebooks, torch

pytestmark = pytest.mark.gpu

BASE = dict(dtype="bf16", alpha=0.7, n_out=16, cb_sigma=None, gscale=1.0)


def _pair(x, C):
    t = torch()
    D = descr(x)
    g = Dev(x, C)
    ref = run_encode(x, D, g)
    if D.L:
        out = t.full_like(ref, -1 if ref.dtype == t.int16 else 255)
    else:
        out = t.full_like(ref, float("nan"))
    mapl.encode_noalloc(D, g.X, g.ids, g.U, g.A, g.B, g.C, out)
    t.cuda.synchronize()
    if D.L:
        a, b = codes_np(out, D), codes_np(ref, D)
    else:
        a, b = out.view(t.int16).cpu().numpy(), ref.view(t.int16).cpu().numpy()
    return a, b


@pytest.mark.parametrize("r,L,K", [(256, 2, 1024), (128, 2, 256), (256, 0, 0)], ids=["fused", "two-launch", "L0"])
def test_noalloc_matches_encode_two_calls(r, L, K):
    for i, T in enumerate((8192 + 77, 1500)):
        print("noalloc", r, L, K, "call", i, "T", T, flush=True)
        x = synth.codec_inputs(None, seed=80 + i, T=T, d=2048, r=r, V=32000, k=128, L=L, K=K, **BASE)
        C = stress_codebooks(x, 180 + i) if L else None
        a, b = _pair(x, C)
        assert np.array_equal(a, b), (r, L, K, T)
