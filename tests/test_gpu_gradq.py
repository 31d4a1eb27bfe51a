"""GPU parity of the quantised backward message (Sec. 3.5: the quantiser
compresses the backward gradients too).  mapl_decode_bwd_q RVQ-encodes the
r-dim gradient dXhat U over its own codebooks while computing dU as
mapl_decode_bwd; mapl_grad_dequantize rebuilds the gradient on the sending
side, which feeds mapl_encode_bwd.  Gradient codes bit-exact except near
ties (counted), dU and the rebuilt gradient within the path's tolerance."""
import numpy as np
import pytest

from oracle import codec as ocodec
from paper_2606_05484_amd import mapl, synth
from _helpers import (BF16_TOL, Dev, codes_np, compare_codes, descr, dev, f64, grad_codebooks, host_f64, operand,
                      rel_fro, run_encode, stress_codebooks, tol, torch)

pytestmark = pytest.mark.gpu

BASE = dict(V=500, dtype="bf16", alpha=0.8, n_out=4, cb_sigma=None, gscale=1.0)


def _gradq(x, C, Lg, Kg, Cg):
    """encode (codes or Z) -> decode_bwd_q -> grad_dequantize -> encode_bwd."""
    t = torch()
    D = descr(x)
    g = Dev(x, C)
    payload = run_encode(x, D, g)
    ws = mapl.workspace(max(mapl.decode_bwd_q_workspace_bytes(D, Lg, Kg),
                            mapl.workspace_bytes(D, mapl.CALL_ENCODE_BWD)))
    gdt = t.uint8 if Kg <= 256 else t.int16
    gcodes = t.full((x["T"], Lg), -1 if Kg > 256 else 255, dtype=gdt, device="cuda")
    dU = t.full((x["d"], x["r"]), float("nan"), device="cuda")
    Cgg = dev(Cg, "f32")
    mapl.decode_bwd_q(D, g.dXhat, payload, g.ids, g.U, g.A, g.B, g.C, Lg, Kg, Cgg, gcodes, dU, 0, ws)
    dU_dec = dU.clone()
    dZq = t.full((x["T"], x["r"]), float("nan"), dtype=g.tdt, device="cuda")
    mapl.grad_dequantize(x["T"], x["r"], Lg, Kg, gcodes, Cgg, dZq, out_dtype=x["dtype"])
    dX = t.full((x["T"], x["d"]), float("nan"), dtype=g.tdt, device="cuda")
    mapl.encode_bwd(D, dZq, g.X, g.ids, g.U, g.A, g.B, dX, dU, 1, ws)
    t.cuda.synchronize()
    gc = gcodes.cpu().numpy()
    gc = (gc.view(np.uint16) if Kg > 256 else gc).astype(np.int64)
    pay = codes_np(payload, D) if x["L"] else host_f64(payload)
    return dict(D=D, gcodes=gc, payload=pay, dU_dec=host_f64(dU_dec), dU=host_f64(dU), dZq=host_f64(dZq),
                dX=host_f64(dX))


def _check(x, C, Lg, Kg, Cg, res):
    op, sp = operand(x), x["anchor_space"]
    X, A, B = f64(x, "X"), f64(x, "A"), f64(x, "B")
    Cref = C if x["L"] else None
    codes_ref, gap, _ = ocodec.grad_quantize(f64(x, "dXhat"), x["U"], Cg, op)
    bad, ex = compare_codes(res["gcodes"], codes_ref, gap)
    print("gradient codes: mismatched", bad, "exempt", ex, "of", x["T"], "distinct",
          [len(np.unique(res["gcodes"][:, l])) for l in range(Lg)])
    assert bad == 0
    _, dUd = ocodec.decode_bwd(f64(x, "dXhat"), res["payload"], x["ids"], x["U"], A, B, Cref, sp, op)
    e = rel_fro(res["dU_dec"], dUd)
    dZq_ref = ocodec.grad_dequantize(res["gcodes"], Cg)
    e2 = rel_fro(res["dZq"], dZq_ref)
    dX_ref, dUe = ocodec.encode_bwd(dZq_ref, X, x["ids"], x["U"], A, B, sp, op)
    e3, e4 = rel_fro(res["dX"], dX_ref), rel_fro(res["dU"], dUd + dUe)
    print("dU_dec rel err", e, "dequantised gradient rel err", e2, "dX rel err", e3, "dU rel err", e4)
    assert max(e, e2, e3, e4) <= tol(x)


@pytest.mark.parametrize("r,Lg,Kg,L", [(64, 2, 96, 0), (128, 3, 256, 2), (256, 2, 1024, 2), (256, 1, 64, 0)],
                         ids=["r64", "r128L3", "r256K1024", "r256Lg1"])
def test_decode_bwd_q_bf16(r, Lg, Kg, L):
    """Ragged token counts; the fused GEMM + RVQ at r = 256, the two-launch
    path below it; u8 and u16 gradient codes; activation codes or an
    unquantised payload upstream."""
    x = synth.codec_inputs(None, seed=100 + r + Lg, T=1537, d=512, r=r, k=16, L=L, K=64 if L else 0, **BASE)
    C = stress_codebooks(x, 300 + r) if L else x["C"]
    Cg = grad_codebooks(x, Lg, Kg, 400 + r)
    print("gradq bf16 r", r, "Lg", Lg, "Kg", Kg, flush=True)
    _check(x, C, Lg, Kg, Cg, _gradq(x, C, Lg, Kg, Cg))


@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_decode_bwd_q_fp32(space):
    x = synth.codec_inputs("c1", anchor_space=space)
    Cg = grad_codebooks(x, 2, 64, 410)
    print("gradq fp32", space, flush=True)
    _check(x, x["C"], 2, 64, Cg, _gradq(x, x["C"], 2, 64, Cg))


@pytest.mark.slow
def test_decode_bwd_q_c4_full_size():
    """The benchmark workload's backward with a K = 1024, two-round gradient
    quantiser (u16 codes, the fused GEMM + RVQ): gradient codes on every
    token against the oracle, dU in full."""
    x = synth.codec_inputs("c4")
    C = stress_codebooks(x, 104)
    Cg = grad_codebooks(x, 2, 1024, 420)
    print("gradq c4", flush=True)
    _check(x, C, 2, 1024, Cg, _gradq(x, C, 2, 1024, Cg))
