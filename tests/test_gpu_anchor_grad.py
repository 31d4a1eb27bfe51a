"""GPU parity of the anchor-table gradient (Eq. 3: E_small is trainable;
the sender's table enters Eq. 1, the receiver's Eq. 2) against the float64
oracle: relative Frobenius error <= 2e-2 (bf16) / 1e-5 (fp32), rows of ids
no token carries exactly 0, repeated calls bit-identical (the per-id sums
run in a fixed order), accumulate adds.  Zipf(1.1) ids put a seventh of the
tokens on id 0, so one row sums thousands of token rows at full size."""
import numpy as np
import pytest

from oracle import codec as ocodec
from paper_2606_05484_amd import mapl, synth
from _helpers import dev, f64, operand, rel_fro, tol, torch

pytestmark = pytest.mark.gpu

SIDES = {"sender": mapl.SENDER, "receiver": mapl.RECEIVER}


def _dY(x, side):
    """The incoming gradient of each case: dZ (sender), dXhat (receiver,
    ambient) or dZhat = dXhat U~ (receiver, coord; bf16-rounded as
    mapl_decode_bwd writes it)."""
    if side == "sender":
        return x["dZ"], x["dtype"]
    if x["anchor_space"] == "ambient":
        return x["dXhat"], x["dtype"]
    dzh = f64(x, "dXhat") @ ocodec._projector(x["U"], operand(x))
    if x["dtype"] == "bf16":
        return synth.f32_to_bf16_bits(dzh.astype(np.float32)), "bf16"
    return dzh.astype(np.float32), "f32"


def _run(x, side, accumulate_into=None):
    t = torch()
    D = mapl.desc(T=x["T"], d=x["d"], r=x["r"], V=x["V"], k=x["k"], x_dtype=x["dtype"],
                  anchor_space=x["anchor_space"])
    dY, dt = _dY(x, side)
    ws = mapl.workspace(mapl.anchor_bwd_workspace_bytes(D, SIDES[side]))
    if accumulate_into is None:
        dA = t.full((x["V"], x["k"]), float("nan"), device="cuda")
        acc = 0
    else:
        dA = dev(accumulate_into.astype(np.float32), "f32")
        acc = 1
    mapl.anchor_bwd(D, SIDES[side], dev(dY, dt), dev(x["ids"], "i32"), dev(x["U"], "f32"), dev(x["B"], x["dtype"]),
                    dA, acc, ws)
    t.cuda.synchronize()
    return dA.cpu().numpy().astype(np.float64), dY, dt


def _ref(x, side, dY, dt):
    return ocodec.anchor_grad(synth.as_f64(dY, dt) if dt == "bf16" else np.asarray(dY, np.float64), x["ids"],
                              x["U"], f64(x, "B"), x["V"], side, x["anchor_space"], operand(x))


CASES = [
    dict(T=1537, d=512, r=128, V=500, k=16),     # one radix pass, k below the 64-wide tile
    dict(T=1537, d=512, r=128, V=32000, k=48),   # two radix passes, k not a multiple of 32
    dict(T=5000, d=256, r=64, V=70000, k=128),   # three radix passes
    dict(T=1, d=256, r=64, V=1, k=16),           # one token, a one-row table
]


@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("side", ["sender", "receiver"])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_anchor_grad_bf16(case, side, space):
    c = CASES[case]
    print("anchor grad", side, space, c, flush=True)
    x = synth.codec_inputs(None, seed=500 + case, anchor_space=space, dtype="bf16", alpha=0.8, n_out=4,
                           cb_sigma=None, gscale=1.0, L=0, K=0, **c)
    got, dY, dt = _run(x, side)
    ref = _ref(x, side, dY, dt)
    e = rel_fro(got, ref)
    absent = np.setdiff1d(np.arange(x["V"]), x["ids"])
    print("dA rel err", e, "absent rows", absent.size)
    assert np.isfinite(got).all() and e <= tol(x)
    assert np.all(got[absent] == 0)
    again, _, _ = _run(x, side)
    assert np.array_equal(got, again)


@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("side", ["sender", "receiver"])
def test_anchor_grad_fp32_and_accumulate(side, space):
    x = synth.codec_inputs("c1", anchor_space=space)
    got, dY, dt = _run(x, side)
    ref = _ref(x, side, dY, dt)
    e = rel_fro(got, ref)
    print("fp32", side, space, "dA rel err", e)
    assert e <= tol(x)
    base = np.random.default_rng(3).standard_normal(got.shape)
    got2, _, _ = _run(x, side, accumulate_into=base)
    assert np.abs(got2 - (base + got)).max() <= 1e-6 * np.abs(got).max()


@pytest.mark.slow
@pytest.mark.parametrize("side", ["sender", "receiver"])
def test_anchor_grad_c4_full_size(side):
    """The benchmark workload (T = 32768, V = 32000, k = 128; the receiver's
    rows come from dXhat [T, 2048]): the whole table, and the ten hottest
    rows one by one."""
    x = synth.codec_inputs("c4")
    got, dY, dt = _run(x, side)
    ref = _ref(x, side, dY, dt)
    e = rel_fro(got, ref)
    ids, cnt = np.unique(x["ids"], return_counts=True)
    hot = ids[np.argsort(-cnt)[:10]]
    worst = max(rel_fro(got[v], ref[v]) for v in hot)
    print("c4", side, "dA rel err", e, "hottest rows: tokens", sorted(cnt)[-3:], "worst row rel err", worst)
    assert e <= tol(x) and worst <= tol(x)
