"""GPU parity of the anchor path (Eqs. 1-2: E_small[ids] P removed by the
sender, the receiver's own E_small[ids] P added back).

- Bit-exact gathers: with a zero payload (decode) or zero activations
  (encode), unit-vector rows in B and an identity projector, the anchor rows
  pass through every product exactly, so the outputs must equal +-A[ids]
  bit for bit; through the fused projection + RVQ encoder the gathered rows
  are read back through planted codewords.
- Anchor-dominant parity: B with orthonormal rows and A ~ N(0,1), distinct
  sender and receiver tables, all four calls, both anchor spaces; each case
  also shows (on the CPU) that a wrong-row gather or the sender's table on
  the receiving side would move the outputs by >= 5x the tolerance."""
import numpy as np
import pytest

from paper_2606_05484_amd import mapl, synth
from _helpers import (ANCHOR_CASES, BF16_TOL, anchor_case, anchor_discrimination, chain, check_chain, codes_np,
                      dev, host_f64, torch)

pytestmark = pytest.mark.gpu

SHAPES = {
    "small": dict(T=1000, d=256, r=64, k=16, V=500),
    "k48": dict(T=555, d=512, r=128, k=48, V=900),       # anchor width not a multiple of the 32/64 K step
    "c4width": dict(T=4096 + 37, d=2048, r=256, k=128, V=32000),
}


def _bits(x):
    """bf16 tensor -> uint16 bit patterns on the host."""
    t = torch()
    return x.view(t.int16).cpu().numpy().view(np.uint16)


def _gather_inputs(s, space, seed):
    rng = np.random.default_rng(seed)
    T, d, r, k, V = s["T"], s["d"], s["r"], s["k"], s["V"]
    A = synth.f32_to_bf16_bits(rng.standard_normal((V, k)).astype(np.float32))
    ids = synth.zipf_ids(rng, V, T)
    cols = d if space == "ambient" else r
    B = np.zeros((k, cols), dtype=np.float32)
    B[:, :k] = np.eye(k)
    U = np.zeros((d, r), dtype=np.float32)
    U[:r, :r] = np.eye(r)
    return A, ids, synth.f32_to_bf16_bits(B), U


@pytest.mark.parametrize("L", [0, 2])
@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("shape", sorted(SHAPES))
def test_decode_gathers_anchor_rows_bit_exact(shape, space, L):
    """Zero payload, B_r = [I_k | 0], U = [I_r ; 0]: Xhat[t, :k] = A_r[ids[t]]
    exactly and the other columns are 0 (codes into an all-zero codebook
    give the same zero payload through the codeword gather-sum)."""
    t = torch()
    s = SHAPES[shape]
    print("decode gather", shape, space, "L", L, flush=True)
    A, ids, B, U = _gather_inputs(s, space, 301)
    T, d, r, k = s["T"], s["d"], s["r"], s["k"]
    D = mapl.desc(T=T, d=d, r=r, V=s["V"], k=k, L=L, K=64 if L else 0, anchor_space=space)
    if L:
        payload = t.zeros((T, L), dtype=t.uint8, device="cuda")
        C = t.zeros((L, 64, r), device="cuda")
    else:
        payload = t.zeros((T, r), dtype=t.bfloat16, device="cuda")
        C = None
    Xh = t.full((T, d), float("nan"), dtype=t.bfloat16, device="cuda")
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_DECODE))
    mapl.decode(D, payload, dev(ids, "i32"), dev(U, "f32"), dev(A, "bf16"), dev(B, "bf16"), C, Xh, ws)
    t.cuda.synchronize()
    got = _bits(Xh)
    assert np.array_equal(got[:, :k], A[ids])
    assert (host_f64(Xh)[:, k:] == 0).all()


@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("shape", sorted(SHAPES))
def test_encode_gathers_anchor_rows_bit_exact(shape, space):
    """X = 0, B_s = [I_k | 0], U = [I_r ; 0], no RVQ: Z[t, :k] = -A_s[ids[t]]
    exactly and the other columns are 0."""
    t = torch()
    s = SHAPES[shape]
    print("encode gather", shape, space, flush=True)
    A, ids, B, U = _gather_inputs(s, space, 302)
    T, d, r, k = s["T"], s["d"], s["r"], s["k"]
    D = mapl.desc(T=T, d=d, r=r, V=s["V"], k=k, anchor_space=space)
    X = t.zeros((T, d), dtype=t.bfloat16, device="cuda")
    Z = t.full((T, r), float("nan"), dtype=t.bfloat16, device="cuda")
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_ENCODE))
    mapl.encode(D, X, dev(ids, "i32"), dev(U, "f32"), dev(A, "bf16"), dev(B, "bf16"), None, Z, ws)
    t.cuda.synchronize()
    got = _bits(Z)
    assert np.array_equal(got[:, :k], A[ids] ^ np.uint16(0x8000))
    assert (host_f64(Z)[:, k:] == 0).all()


@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("d,k", [(512, 64), (2048, 128), (512, 48)])
def test_fused_encoder_gathers_anchor_rows_exactly(d, k, space):
    """The fused projection + RVQ encoder (r = 256) gathers the anchor rows
    in its K loop.  X = 0, B_s = [I_k | 0], U = [I_r ; 0] make Z0 = -A_s[ids]
    exactly; codeword 1 + v of round 0 is -A_s[v], so the first code must be
    1 + ids[t] (a row gathered for the wrong id lands on another codeword),
    and the zero residual then picks the zero codeword in round 1."""
    t = torch()
    V, r, K, T = 63, 256, 64, 1037
    s = dict(T=T, d=d, r=r, k=k, V=V)
    print("fused gather", d, k, space, flush=True)
    A, ids, B, U = _gather_inputs(s, space, 303)
    C = np.zeros((2, K, r), dtype=np.float32)
    C[0, 1:, :k] = -synth.bf16_bits_to_f32(A)
    C[1, 1:] = 5.0 + np.random.default_rng(4).standard_normal((K - 1, r)).astype(np.float32)
    D = mapl.desc(T=T, d=d, r=r, V=V, k=k, L=2, K=K, anchor_space=space)
    X = t.zeros((T, d), dtype=t.bfloat16, device="cuda")
    codes = t.full((T, 2), 255, dtype=t.uint8, device="cuda")
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_ENCODE))
    mapl.encode(D, X, dev(ids, "i32"), dev(U, "f32"), dev(A, "bf16"), dev(B, "bf16"), dev(C, "f32"), codes, ws)
    t.cuda.synchronize()
    got = codes_np(codes, D)
    assert np.array_equal(got[:, 0], 1 + ids.astype(np.int64))
    assert (got[:, 1] == 0).all()


@pytest.mark.parametrize("name", sorted(ANCHOR_CASES))
def test_anchor_dominant_chain(name):
    """encode (sender tables) -> decode -> decode_bwd (receiver tables) ->
    encode_bwd against the oracle with the same tables; the anchor term is
    as large as the activations, so a wrong-row gather, a dropped anchor or
    the wrong side's table fails the gate (shown per case)."""
    print("anchor-dominant chain", name, flush=True)
    x, rx, C = anchor_case(name)
    res = chain(x, C, rx=rx)
    check_chain(x, res, C, rx)
    pay = codes_np(res["payload"], res["D"]) if x["L"] else host_f64(res["payload"])
    disc = anchor_discrimination(x, pay, C, rx)
    print("discrimination", {k_: round(v, 3) for k_, v in disc.items()})
    assert min(disc.values()) >= 5 * BF16_TOL
