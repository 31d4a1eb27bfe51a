"""GPU parity of the boundary codec against the float64 oracle.

Every comparison: relative Frobenius error <= 2e-2 (bf16 paths) or 1e-5
(fp32 path); RVQ codes bit-exact except tokens whose oracle top-2 gap is
under 1e-4 relative (counted).  Workloads come from the seeded generator;
sizes span several tiles with ragged tails."""
import numpy as np
import pytest

from oracle import codec as ocodec
from paper_2606_05484_amd import mapl, synth
from _helpers import (BF16_TOL, F32_TOL, Dev, chain as _chain, check_chain as _check_chain, codes_np,
                      compare_codes, descr, dev, f64, host_f64, operand, oracle_encode, rel_fro, run_encode,
                      stress_codebooks, tol, torch)

pytestmark = pytest.mark.gpu

SMALL = dict(T=1000, d=256, r=64, V=500, k=16, L=0, K=0, dtype="bf16", alpha=0.8, n_out=4, cb_sigma=None,
             gscale=1.0)


def _x(name=None, seed=None, **over):
    print("workload", name, seed, over, flush=True)
    return synth.codec_inputs(name, seed=seed, **over)


@pytest.mark.parametrize("r", [64, 128, 256, 512])
def test_c2_projection_only(r):
    x = _x("c2_r%d" % r)
    _check_chain(x, _chain(x))


def test_c1_fp32_with_rvq():
    x = _x("c1")
    _check_chain(x, _chain(x))


def test_c1_fp32_no_rvq():
    x = _x("c1")
    _check_chain(x, _chain(x, L=0, K=0))


def test_c3_rvq_official_codebooks():
    x = _x("c3")
    _check_chain(x, _chain(x))


def test_c3_rvq_stress_codebooks():
    x = _x("c3")
    C = stress_codebooks(x, 103)
    _check_chain(x, _chain(x, C=C), C=C)


@pytest.mark.parametrize("space", ["ambient", "coord"])
@pytest.mark.parametrize("L,K", [(0, 0), (2, 96)])
def test_ragged_small_both_anchor_spaces(space, L, K):
    x = _x(None, seed=7, anchor_space=space, **dict(SMALL, L=L, K=K))
    C = stress_codebooks(x, 107) if L else None
    _check_chain(x, _chain(x, C=C), C=C)


@pytest.mark.parametrize("space", ["ambient", "coord"])
def test_fp32_ragged_odd_tokens(space):
    """fp32 operands with an odd token count: the fp32 products that
    contract over tokens (dU) take the general element-load GEMM (K not a
    multiple of 4), the others the pipelined 16-byte-load GEMM with a
    ragged last tile."""
    x = _x(None, seed=11, anchor_space=space, **dict(SMALL, T=509, dtype="f32", L=2, K=64))
    _check_chain(x, _chain(x))


@pytest.mark.parametrize("over", [
    dict(T=257, d=256, r=32, k=16, L=8, K=64),      # the most rounds, the smallest rank
    dict(T=130, d=128, r=96, k=0, L=1, K=2048),     # a rank the bf16 path refuses, a large codebook
], ids=["L8r32", "r96K2048"])
def test_fp32_limits(over):
    """The fp32 path at shapes the bf16 kernels do not take (r = 32, 96) and
    at the most rounds: the whole chain against the oracle at the fp32
    tolerance."""
    x = _x(None, seed=12, **dict(SMALL, dtype="f32", **over))
    _check_chain(x, _chain(x))


def test_fp32_coord_anchor():
    x = _x("c1", anchor_space="coord")
    _check_chain(x, _chain(x))


def test_no_anchor_k0():
    x = _x(None, seed=8, **dict(SMALL, k=0, T=333))
    _check_chain(x, _chain(x))


def test_empty_batch():
    t = torch()
    x = _x(None, seed=11, **dict(SMALL, T=0, L=2, K=64))
    D = descr(x)
    g = Dev(x)
    codes = t.empty((0, 2), dtype=t.uint8, device="cuda")
    run_encode(x, D, g, codes)
    dU = t.full((x["d"], x["r"]), 3.0, device="cuda")
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_DECODE_BWD))
    dZ = t.empty((0, x["r"]), dtype=g.tdt, device="cuda")
    mapl.decode_bwd(D, g.dXhat, codes, g.ids, g.U, g.A, g.B, g.C, dZ, dU, 0, ws)
    t.cuda.synchronize()
    assert float(dU.abs().max()) == 0.0  # overwrite with an empty sum


def test_accumulate_flag_adds():
    t = torch()
    x = _x(None, seed=12, **SMALL)
    D = descr(x)
    g = Dev(x)
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_ENCODE_BWD))
    dX = t.empty((x["T"], x["d"]), dtype=g.tdt, device="cuda")
    dU0 = t.zeros((x["d"], x["r"]), device="cuda")
    mapl.encode_bwd(D, g.dZ, g.X, g.ids, g.U, g.A, g.B, dX, dU0, 0, ws)
    base = t.randn((x["d"], x["r"]), device="cuda")
    dU1 = base.clone()
    mapl.encode_bwd(D, g.dZ, g.X, g.ids, g.U, g.A, g.B, dX, dU1, 1, ws)
    t.cuda.synchronize()
    assert t.equal(dU1, base + dU0) or float((dU1 - base - dU0).abs().max()) <= 1e-6 * float(dU0.abs().max())


def test_deterministic_repeat():
    x = _x(None, seed=13, **dict(SMALL, L=2, K=64))
    C = stress_codebooks(x, 113)
    a = _chain(x, C=C)
    b = _chain(x, C=C)
    for key in ("Xh", "dZ", "dU", "dX"):
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(codes_np(a["payload"], a["D"]), codes_np(b["payload"], b["D"]))


def test_planted_codewords_and_duplicate_tie():
    """Codewords planted at oracle coordinates of chosen tokens are picked
    (residual 0, later rounds pick the zero codeword); a duplicated codeword
    resolves to the lower index."""
    x = _x(None, seed=14, **dict(SMALL, L=2, K=64))
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), "ambient", "bf16")
    C = np.zeros((2, 64, x["r"]), dtype=np.float32)
    rng = np.random.default_rng(0)
    C[:, 1:] = (5 + rng.standard_normal((2, 63, x["r"]))).astype(np.float32)
    plant = {5: 7, 300: 12, 999: 40}
    for t_, j in plant.items():
        C[0, j] = Z0[t_].astype(np.float32)
    C[0, 50] = C[0, 12]  # duplicate of 12
    D = descr(x)
    g = Dev(x, C)
    codes = codes_np(run_encode(x, D, g), D)
    for t_, j in plant.items():
        assert codes[t_, 0] == j, (t_, codes[t_])
        assert codes[t_, 1] == 0


@pytest.mark.parametrize("T,k,L,K", [(1037, 64, 2, 96), (1037, 48, 1, 64), (1037, 0, 3, 128), (1, 16, 2, 32),
                                     (129, 64, 1, 32)])
def test_fused_encoder_r256(T, k, L, K):
    """At r = 256 the projection and the RVQ run as one launch (Z0 stays on
    chip): ragged token counts (one token; one block and one token), anchors
    whose width is and is not a multiple of the 64-wide K stage, no anchor,
    one to three rounds, codebooks whose last 64-codeword chunk is half empty
    (K = 32: the only chunk), stress codebooks."""
    x = _x(None, seed=40 + k + L, **dict(SMALL, T=T, d=512, r=256, k=k, L=L, K=K))
    C = stress_codebooks(x, 211 + L) if T >= K else None
    _check_chain(x, _chain(x, C=C), C=C)


def test_fused_encoder_planted_and_tied_r256():
    """The fused encoder's exact fp32 rescoring of ambiguous tokens: codewords
    planted at oracle coordinates are picked (later rounds then pick the zero
    codeword); a duplicated codeword (an exact tie) resolves to the lower
    index."""
    x = _x(None, seed=15, **dict(SMALL, T=700, d=512, r=256, L=2, K=128))
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), "ambient", "bf16")
    C = np.zeros((2, 128, x["r"]), dtype=np.float32)
    rng = np.random.default_rng(1)
    C[:, 1:] = (5 + rng.standard_normal((2, 127, x["r"]))).astype(np.float32)
    plant = {3: 9, 130: 70, 699: 127}
    for t_, j in plant.items():
        C[0, j] = Z0[t_].astype(np.float32)
    C[0, 120] = C[0, 70]  # duplicate of 70
    C[0, 110] = C[0, 9]  # duplicate of 9
    D = descr(x)
    g = Dev(x, C)
    codes = codes_np(run_encode(x, D, g), D)
    for t_, j in plant.items():
        assert codes[t_, 0] == j, (t_, codes[t_])
        assert codes[t_, 1] == 0


@pytest.mark.parametrize("over", [
    dict(T=300, d=512, r=256, k=16, L=8, K=64),        # the most rounds (fused encoder)
    dict(T=513, d=256, r=64, k=0, L=1, K=65536),       # the largest codebook, u16 codes
    dict(T=257, d=1024, r=64, k=512, L=2, K=96),       # the widest anchor
    dict(T=130, d=16384, r=64, k=16, L=1, K=32, rotate=False),  # the widest activations, smallest codebook
    dict(T=300, d=512, r=192, k=16, L=0, K=0),         # a rank between the 128- and 256-wide tiles
    dict(T=200, d=1024, r=1024, k=64, L=0, K=0),       # the largest rank
    dict(T=1, d=64, r=64, k=16, L=1, K=32),            # the smallest of everything
], ids=["L8", "K65536", "k512", "d16384", "r192", "r1024", "min"])
def test_extreme_shapes(over):
    """The limits the library accepts (L <= 8, K <= 65536, k <= 512,
    d <= 16384), each with ragged token counts: the whole chain against the
    oracle (stress codebooks where there are enough tokens to draw them)."""
    x = _x(None, seed=50, **dict(SMALL, **over))
    C = stress_codebooks(x, 223) if x["L"] and x["T"] >= x["K"] else None
    _check_chain(x, _chain(x, C=C), C=C)


@pytest.mark.slow
def test_c4_full_size_sampled():
    """The benchmark workload (T=32768, d=2048, r=256, k=128, L=2, K=1024)
    in the launch configuration the benchmark times: codes on every token
    against the oracle, Xhat / dZ / dX on 512 sampled tokens, dU in full."""
    t = torch()
    x = _x("c4")
    res = _chain(x)
    D = res["D"]
    X, A, B = f64(x, "X"), f64(x, "A"), f64(x, "B")
    Z0 = ocodec.project(X, x["ids"], x["U"], A, B, "ambient", "bf16")
    codes_ref, gap, _ = ocodec.rvq_encode(Z0, x["C"])
    cg = codes_np(res["payload"], D)
    bad, ex = compare_codes(cg, codes_ref, gap)
    print("c4 codes: mismatched", bad, "exempt", ex)
    assert bad == 0
    rows = np.random.default_rng(4).choice(x["T"], 512, replace=False)
    Xh_ref = ocodec.decode(cg[rows], x["ids"][rows], x["U"], A, B, x["C"], "ambient", "bf16")
    assert rel_fro(res["Xh"][rows], Xh_ref) <= BF16_TOL
    dXh = f64(x, "dXhat")
    dZ_ref = dXh[rows] @ ocodec._projector(x["U"], "bf16")
    assert rel_fro(res["dZ"][rows], dZ_ref) <= BF16_TOL
    dX_ref = f64(x, "dZ")[rows] @ ocodec._projector(x["U"], "bf16").T
    assert rel_fro(res["dX"][rows], dX_ref) <= BF16_TOL
    _, dUd = ocodec.decode_bwd(dXh, cg, x["ids"], x["U"], A, B, x["C"], "ambient", "bf16")
    _, dUe = ocodec.encode_bwd(f64(x, "dZ"), X, x["ids"], x["U"], A, B, "ambient", "bf16")
    e = rel_fro(res["dU"], dUd + dUe)
    print("c4 dU rel err", e)
    assert e <= BF16_TOL


@pytest.mark.slow
def test_c4_full_size_stress_codebooks():
    """The benchmark workload with codebooks drawn from the oracle's own
    residuals (codeword 0 = 0, the others residual rows plus 5 % noise):
    every code is in use, so the fused encoder decides near-ambiguous tokens
    by exact fp32 rescoring in every workgroup, with the 16-chunk codebook
    ring and u16 codes.  Codes on every token against the oracle (exempt
    tokens counted), Xhat / dZ / dX on 512 sampled tokens, dU (with a
    non-zero Zhat, so both halves) in full."""
    x = _x("c4")
    C = stress_codebooks(x, 104)
    res = _chain(x, C=C)
    D = res["D"]
    X, A, B = f64(x, "X"), f64(x, "A"), f64(x, "B")
    Z0 = ocodec.project(X, x["ids"], x["U"], A, B, "ambient", "bf16")
    codes_ref, gap, _ = ocodec.rvq_encode(Z0, C)
    cg = codes_np(res["payload"], D)
    bad, ex = compare_codes(cg, codes_ref, gap)
    used = [len(np.unique(cg[:, l])) for l in range(D.L)]
    print("c4 stress codes: mismatched", bad, "exempt", ex, "of", x["T"], "distinct codes per round", used)
    assert bad == 0
    assert min(used) > 0.8 * x["K"]
    rows = np.random.default_rng(6).choice(x["T"], 512, replace=False)
    Xh_ref = ocodec.decode(cg[rows], x["ids"][rows], x["U"], A, B, C, "ambient", "bf16")
    e = rel_fro(res["Xh"][rows], Xh_ref)
    print("Xhat rel err", e)
    assert e <= BF16_TOL
    P = ocodec._projector(x["U"], "bf16")
    assert rel_fro(res["dZ"][rows], f64(x, "dXhat")[rows] @ P) <= BF16_TOL
    assert rel_fro(res["dX"][rows], f64(x, "dZ")[rows] @ P.T) <= BF16_TOL
    _, dUd = ocodec.decode_bwd(f64(x, "dXhat"), cg, x["ids"], x["U"], A, B, C, "ambient", "bf16")
    _, dUe = ocodec.encode_bwd(f64(x, "dZ"), X, x["ids"], x["U"], A, B, "ambient", "bf16")
    e1, e2 = rel_fro(res["dU_dec"], dUd), rel_fro(res["dU"], dUd + dUe)
    print("c4 stress dU_dec rel err", e1, "dU rel err", e2, "|dU_dec|/|dU_enc|",
          np.linalg.norm(dUd) / np.linalg.norm(dUe))
    assert e1 <= BF16_TOL and e2 <= BF16_TOL


@pytest.mark.parametrize("d,r", [(512, 128), (512, 256)])
def test_rvq_candidate_overflow_full_rescan(d, r):
    """More codewords within the screening margin of one token than its
    candidate list holds (16): that token is decided by a full fp32 rescan
    of the codebook.  20 codewords are planted around token 5's Z0 at
    squared distances (1e-3 + 5e-4 j) ||Z0||^2, j = 0..19 (all within the
    margin, yet 5e-4 ||Z0||^2 apart: no near-tie); the nearest sits at the
    highest of their indices, so a truncated list would miss it."""
    x = _x(None, seed=16, **dict(SMALL, T=300, d=d, r=r, k=16, L=2, K=64))
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), "ambient", "bf16")
    rng = np.random.default_rng(2)
    C = np.zeros((2, 64, r), dtype=np.float32)
    C[:, 1:] = (5 + rng.standard_normal((2, 63, r))).astype(np.float32)
    z = Z0[5]
    n2 = float(z @ z)
    for j in range(20):
        u = rng.standard_normal(r)
        u /= np.linalg.norm(u)
        C[0, 59 - j] = (z + np.sqrt((1e-3 + 5e-4 * j) * n2) * u).astype(np.float32)
    codes_ref, gap, _ = ocodec.rvq_encode(Z0, C)
    assert codes_ref[5, 0] == 59 and gap[5, 0] > 2e-4
    D = descr(x)
    g = Dev(x, C)
    cg = codes_np(run_encode(x, D, g), D)
    bad, ex = compare_codes(cg, codes_ref, gap)
    print("overflow: token 5 codes", cg[5], "mismatched", bad, "exempt", ex)
    assert cg[5, 0] == 59
    assert bad == 0


@pytest.mark.parametrize("r", [64, 128, 256])
def test_rvq_every_token_undecided(r):
    """Every token of every workgroup undecided after the first pass, and
    every candidate list overflowing: each round's codebook is four distinct
    codewords repeated (C[l, j] = C[l, j % 4], K = 128), so each token's
    nearest row has 31 bitwise-identical copies, an exact tie that the lowest
    index breaks.  The second pass then lists all 128 tokens of a workgroup
    (four compacted tiles) and the rescoring falls back to the full codebook
    for each.  Codes must be the lowest index of the nearest distinct
    codeword; tokens whose two nearest distinct codewords nearly tie are
    exempt, as everywhere."""
    x = _x(None, seed=21, **dict(SMALL, T=300, d=512, r=r, k=16, L=2, K=128))
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), "ambient", "bf16")
    rng = np.random.default_rng(5)
    sig = float(np.sqrt(np.mean(Z0 ** 2)))
    base = np.zeros((2, 4, r), dtype=np.float32)
    base[0, 1:] = (Z0[rng.choice(300, 3, replace=False)] + 0.05 * sig * rng.standard_normal((3, r))).astype(np.float32)
    base[1, 1:] = (0.3 * sig * rng.standard_normal((3, r))).astype(np.float32)
    C = np.stack([np.tile(base[l], (32, 1)) for l in range(2)])
    assert C.shape == (2, 128, r) and np.array_equal(C[:, 4], C[:, 0])
    codes_ref, _, _ = ocodec.rvq_encode(Z0, C)          # lowest index among the copies
    codes_4, gap4, _ = ocodec.rvq_encode(Z0, base)      # the near-tie measure among distinct rows
    assert np.array_equal(codes_ref, codes_4)
    D = descr(x)
    g = Dev(x, C)
    mapl.profile(2)
    cg = codes_np(run_encode(x, D, g), D)
    st = mapl.profile_report()
    mapl.profile(0)
    bad, ex = compare_codes(cg, codes_ref, gap4)
    ovf = st.get("rvq:list_overflows", (0, 0))[0]
    print("every token undecided, r=%d: mismatched %d exempt %d list overflows %d" % (r, bad, ex, ovf))
    assert bad == 0
    assert ovf == 2 * 300  # every (token, round) list overflowed into the full rescan


@pytest.mark.parametrize("r", [64, 128, 256])
def test_short_k_many_tiles(r):
    """Decode and encode_bwd at d=2048 with enough tokens (8192 + a ragged
    77) that each workgroup walks several output tiles: the K depths
    r + k = 128, 192, 320 (decode) and r = 128, 256 (encode_bwd) of the
    register-resident token operand, besides the benchmark's 384 and 256."""
    x = _x("c4", T=8192 + 77, r=r, k=64, L=0, K=0)
    _check_chain(x, _chain(x))


@pytest.mark.parametrize("k", [0, 64])
@pytest.mark.parametrize("L,K", [(1, 256), (2, 256), (2, 1024)])
def test_decode_gathers_codewords_bit_exact(L, K, k):
    """Where the decoder's product walks several output tiles per workgroup
    (here 8192 + 77 tokens at d = 2048) it gathers the codewords by code
    inside its token-operand load instead of reading an assembled Zhat.
    With U = [I_r ; 0] and B_r rows = unit vectors e_{r+i}, Xhat[:, :r] must
    equal bf16(sum_l C_l[code_l]) (fp32 sum in l order, rounded once) and
    Xhat[:, r:r+k] must equal A_r[ids], bit for bit; u8 and u16 codes, one
    and two rounds, codes 0 and K-1 included, a ragged last block."""
    t = torch()
    T, d, r, V = 8192 + 77, 2048, 256, 3000
    print("decode codeword gather", L, K, k, flush=True)
    rng = np.random.default_rng(1000 + 10 * L + K + k)
    C = rng.standard_normal((L, K, r)).astype(np.float32)
    codes = rng.integers(0, K, size=(T, L))
    codes[:5] = K - 1
    codes[5:9] = 0
    cdt = np.uint8 if K <= 256 else np.uint16
    U = np.zeros((d, r), dtype=np.float32)
    U[:r, :r] = np.eye(r)
    A = synth.f32_to_bf16_bits(rng.standard_normal((V, max(k, 1))).astype(np.float32))[:, :k]
    ids = synth.zipf_ids(rng, V, T)
    B = np.zeros((k, d), dtype=np.float32)
    B[np.arange(k), r + np.arange(k)] = 1.0
    D = mapl.desc(T=T, d=d, r=r, V=V, k=k, L=L, K=K)
    payload = t.from_numpy(codes.astype(cdt).astype(np.int16 if cdt == np.uint16 else np.uint8)).cuda()
    Xh = t.full((T, d), float("nan"), dtype=t.bfloat16, device="cuda")
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_DECODE))
    mapl.decode(D, payload, dev(ids, "i32") if k else None, dev(U, "f32"), dev(A, "bf16") if k else None,
                dev(synth.f32_to_bf16_bits(B), "bf16") if k else None, t.from_numpy(C).cuda(), Xh, ws)
    t.cuda.synchronize()
    zsum = np.zeros((T, r), dtype=np.float32)
    for l in range(L):
        zsum = (zsum + C[l][codes[:, l]]).astype(np.float32)
    want = synth.f32_to_bf16_bits(zsum)
    got = Xh.view(t.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got[:, :r], want), int((got[:, :r] != want).sum())
    if k:
        assert np.array_equal(got[:, r:r + k], A[ids])
    assert (host_f64(Xh)[:, r + k:] == 0).all()


@pytest.mark.slow
def test_large_ragged_tail_sampled():
    """A token count that is not a multiple of the 128-token tile at the
    benchmark's widths (d=2048, r=256, k=128; no RVQ): the products that walk
    many output tiles per workgroup (decode, encode_bwd) run in the same
    launch configuration as at full size, with a partial last tile.  Every
    row of the last tile and 256 others are checked against the oracle."""
    x = _x("c4", T=32768 - 37, L=0, K=0)
    res = _chain(x)
    X, A, B = f64(x, "X"), f64(x, "A"), f64(x, "B")
    T = x["T"]
    last = np.arange(T - T % 128, T)
    rows = np.concatenate([last, np.random.default_rng(5).choice(T - T % 128, 256, replace=False)])
    Z_ref = ocodec.project(X[rows], x["ids"][rows], x["U"], A, B, "ambient", "bf16")
    Zg = host_f64(res["payload"])
    assert rel_fro(Zg[rows], Z_ref) <= BF16_TOL
    Xh_ref = ocodec.decode(Zg[rows], x["ids"][rows], x["U"], A, B, None, "ambient", "bf16")
    e = rel_fro(res["Xh"][rows], Xh_ref)
    print("Xhat rel err", e)
    assert np.isfinite(res["Xh"]).all() and e <= BF16_TOL
    P = ocodec._projector(x["U"], "bf16")
    assert rel_fro(res["dZ"][rows], f64(x, "dXhat")[rows] @ P) <= BF16_TOL
    e = rel_fro(res["dX"][rows], f64(x, "dZ")[rows] @ P.T)
    print("dX rel err", e)
    assert np.isfinite(res["dX"]).all() and e <= BF16_TOL
