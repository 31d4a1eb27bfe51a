"""Shared helpers for the GPU parity tests: device transfer, the library
call sequence, oracle references and the comparison rules (relative
Frobenius error; bit-exact codes except near-tie tokens)."""
import numpy as np

from oracle import codec as ocodec
from paper_2606_05484_amd import mapl, synth

BF16_TOL = 2e-2  # relative Frobenius error, bf16 paths
F32_TOL = 1e-5   # relative Frobenius error, fp32 paths
TIE_GAP = 1e-4   # relative top-2 gap under which a token is exempt


def torch():
    import torch as t
    return t


def dev(arr, dtype):
    """NumPy (bf16 bits as uint16, or float32/int32) -> CUDA tensor."""
    t = torch()
    a = np.ascontiguousarray(arr)
    if dtype == "bf16":
        return t.from_numpy(a.view(np.int16)).cuda().view(t.bfloat16)
    return t.from_numpy(a).cuda()


def host_f64(x):
    t = torch()
    if x.dtype == t.bfloat16:
        return x.float().cpu().numpy().astype(np.float64)
    return x.cpu().numpy().astype(np.float64)


def rel_fro(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(got - ref) / (den if den > 0 else 1.0)


def tol(x):
    return BF16_TOL if x["dtype"] == "bf16" else F32_TOL


def operand(x):
    return "bf16" if x["dtype"] == "bf16" else "exact"


def f64(x, key):
    return synth.as_f64(x[key], x["dtype"]) if key in ("X", "A", "B", "dXhat", "dZ") else \
        np.asarray(x[key], dtype=np.float64)


def descr(x, L=None, K=None):
    L = x["L"] if L is None else L
    K = x["K"] if K is None else K
    return mapl.desc(T=x["T"], d=x["d"], r=x["r"], V=x["V"], k=x["k"], L=L, K=K, x_dtype=x["dtype"],
                     anchor_space=x["anchor_space"], code_dtype=None if L else "u8",
                     group_dim=x.get("group_dim", 0) if L else 0)


class Dev:
    """Device copies of one workload's inputs."""

    def __init__(self, x, C=None):
        t = torch()
        dt = x["dtype"]
        self.X = dev(x["X"], dt)
        self.U = dev(x["U"], "f32")
        self.A = dev(x["A"], dt)
        self.B = dev(x["B"], dt)
        self.ids = dev(x["ids"], "i32")
        Cn = x["C"] if C is None else C
        self.C = dev(np.ascontiguousarray(Cn, dtype=np.float32), "f32") if Cn.size else None
        self.dXhat = dev(x["dXhat"], dt)
        self.dZ = dev(x["dZ"], dt)
        self.tdt = t.bfloat16 if dt == "bf16" else t.float32


def run_encode(x, D, g, payload=None):
    t = torch()
    if payload is None:
        if D.L == 0:
            payload = t.full((x["T"], x["r"]), float("nan"), dtype=g.tdt, device="cuda")
        elif D.group_dim == 2:
            payload = t.full((x["T"], D.L, x["r"] // 2), 255, dtype=t.uint8, device="cuda")
        else:
            payload = t.full((x["T"], D.L), -1 if D.code_dtype == mapl.U16 else 255,
                             dtype=t.int16 if D.code_dtype == mapl.U16 else t.uint8, device="cuda")
    ws = mapl.workspace(mapl.workspace_bytes(D, mapl.CALL_ENCODE))
    mapl.encode(D, g.X, g.ids, g.U, g.A, g.B, g.C, payload, ws)
    return payload


def codes_np(payload, D):
    a = payload.cpu().numpy()
    if D.code_dtype == mapl.U16:
        a = a.view(np.uint16)
    return a.astype(np.int64)


def compare_codes(gpu_codes, ref_codes, gap):
    """Returns (n_mismatch_nonexempt, n_exempt).  Whole-vector codes [T, L]:
    a token is exempt when any round has an oracle top-2 gap under TIE_GAP;
    for the rest every round must match.  Grouped codes [T, L, G] (gap
    relative to the group's unquantised energy): each (token, group) is
    compared round by round up to its first near-tie round, every decision
    before it must match; n_exempt counts the decisions not compared."""
    if gpu_codes.ndim == 3:
        L = ref_codes.shape[1]
        near = gap < TIE_GAP
        first = np.where(near.any(axis=1), near.argmax(axis=1), L)  # [T, G]
        compared = np.arange(L)[None, :, None] < first[:, None, :]
        bad = int(((gpu_codes != ref_codes) & compared).sum())
        return bad, int((~compared).sum())
    exempt = (gap < TIE_GAP).any(axis=1)
    bad = (gpu_codes != ref_codes).any(axis=1) & ~exempt
    return int(bad.sum()), int(exempt.sum())


def oracle_encode(x, C=None, rows=None):
    Cn = x["C"] if C is None else C
    sel = slice(None) if rows is None else rows
    X = f64(x, "X")[sel]
    ids = x["ids"][sel]
    return ocodec.encode(X, ids, x["U"], f64(x, "A"), f64(x, "B"), Cn if Cn.size else None,
                         anchor_space=x["anchor_space"], operand=operand(x))


def stress_codebooks(x, seed):
    """Codewords drawn from the oracle's own residuals plus 5% noise, with
    codeword 0 = 0, so that every code is in use (the generator's Gaussian
    codebooks leave the zero codeword winning almost every token)."""
    rng = np.random.default_rng(seed)
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), x["anchor_space"],
                        operand(x))
    L, K, r, T = x["L"], x["K"], x["r"], x["T"]
    C = np.zeros((L, K, r), dtype=np.float32)
    R = Z0.copy()
    for l in range(L):
        sig = np.sqrt(np.mean(R ** 2))
        idx = rng.choice(T, K - 1, replace=False)
        C[l, 1:] = (R[idx] + 0.05 * sig * rng.standard_normal((K - 1, r))).astype(np.float32)
        codes, _, _ = ocodec.rvq_encode(R, C[l:l + 1].astype(np.float64))
        R = R - C[l].astype(np.float64)[codes[:, 0]]
    return C


def chain(x, C=None, L=None, K=None, rx=None):
    """encode -> decode -> decode_bwd -> encode_bwd on the GPU; returns host
    results.  The sender's anchor tables (A, B of x) serve encode and
    encode_bwd; the receiver's (those of rx, default x) serve decode and
    decode_bwd, as in Eq. 2 where the next stage adds its own anchor."""
    t = torch()
    D = descr(x, L, K)
    g = Dev(x, C)
    rx = x if rx is None else rx
    Ar, Br = dev(rx["A"], x["dtype"]), dev(rx["B"], x["dtype"])
    payload = run_encode(x, D, g)
    Xh = t.full((x["T"], x["d"]), float("nan"), dtype=g.tdt, device="cuda")
    ws = mapl.workspace(max(mapl.workspace_bytes(D, c) for c in range(4)))
    mapl.decode(D, payload, g.ids, g.U, Ar, Br, g.C, Xh, ws)
    dZ = t.full((x["T"], x["r"]), float("nan"), dtype=g.tdt, device="cuda")
    dU = t.full((x["d"], x["r"]), float("nan"), dtype=t.float32, device="cuda")
    mapl.decode_bwd(D, g.dXhat, payload, g.ids, g.U, Ar, Br, g.C, dZ, dU, 0, ws)
    dU_dec = dU.clone()
    dX = t.full((x["T"], x["d"]), float("nan"), dtype=g.tdt, device="cuda")
    mapl.encode_bwd(D, g.dZ, g.X, g.ids, g.U, g.A, g.B, dX, dU, 1, ws)
    t.cuda.synchronize()
    return dict(D=D, payload=payload, Xh=host_f64(Xh), dZ=host_f64(dZ), dU_dec=host_f64(dU_dec),
                dU=host_f64(dU), dX=host_f64(dX))


def chain_refs(x, payload, C=None, rx=None, ids=None):
    """Oracle results of the four calls for the given payload (the one the
    GPU produced: decode is judged on what it was handed).  ids overrides
    the token ids of every anchor gather (used to show that a wrong-row
    gather would be caught)."""
    Cn = x["C"] if C is None else C
    Cref = Cn if (Cn is not None and Cn.size and payload.dtype.kind in "iu") else None
    rx = x if rx is None else rx
    op, sp = operand(x), x["anchor_space"]
    X, As, Bs = f64(x, "X"), f64(x, "A"), f64(x, "B")
    Ar, Br = f64(rx, "A"), f64(rx, "B")
    ids = x["ids"] if ids is None else ids
    out = dict(Z0=ocodec.project(X, ids, x["U"], As, Bs, sp, op))
    out["Xh"] = ocodec.decode(payload, ids, x["U"], Ar, Br, Cref, sp, op)
    out["dZ"], out["dU_dec"] = ocodec.decode_bwd(f64(x, "dXhat"), payload, ids, x["U"], Ar, Br, Cref, sp, op)
    out["dX"], out["dU_enc"] = ocodec.encode_bwd(f64(x, "dZ"), X, ids, x["U"], As, Bs, sp, op)
    out["dU"] = out["dU_dec"] + out["dU_enc"]
    return out


def anchor_discrimination(x, payload, C=None, rx=None, seed=0):
    """How far the oracle's outputs move when every anchor row is gathered
    for the wrong token (ids permuted), and when the sender's table is used
    on the receiving side: {quantity: relative Frobenius change}.  A parity
    test of the anchor path can only fail for such a bug when the change is
    well above its tolerance."""
    rng = np.random.default_rng(seed)
    ids = x["ids"]
    perm = ids[rng.permutation(len(ids))]
    true = chain_refs(x, payload, C, rx)
    wrong = chain_refs(x, payload, C, rx, ids=perm)
    # coord: dU_enc = X^T dZ has no anchor term; dU_dec does
    keys = ["Xh", "dU"] + (["Z0"] if x["L"] == 0 else [])
    keys.append("dU_dec" if x["anchor_space"] == "coord" else "dU_enc")
    out = {"perm_" + k: rel_fro(wrong[k], true[k]) for k in keys}
    if rx is not None:
        swap = chain_refs(x, payload, C, rx=x)
        out["swap_Xh"] = rel_fro(swap["Xh"], true["Xh"])
    return out


def check_chain(x, res, C=None, rx=None):
    """Every output of chain() against the oracle, fed the same inputs the
    GPU call saw: codes bit-exact except near-tie tokens, the rest within
    the relative Frobenius tolerance of the path."""
    Cn = x["C"] if C is None else C
    D = res["D"]
    if D.L == 0:
        Zg = host_f64(res["payload"])
        assert np.isfinite(Zg).all()
        pay = Zg  # decode is checked on the payload the GPU produced
    else:
        cg = codes_np(res["payload"], D)
        pay = cg
    ref = chain_refs(x, pay, Cn, rx)
    if D.L == 0:
        e = rel_fro(Zg, ref["Z0"])
        print("Z rel err", e)
        assert e <= tol(x)
    else:
        gd = x.get("group_dim", 0)
        codes_ref, gap, _ = (ocodec.grouped_rvq_encode(ref["Z0"], Cn, gd) if gd else ocodec.rvq_encode(ref["Z0"], Cn))
        bad, ex = compare_codes(cg, codes_ref, gap)
        print("codes: mismatched non-exempt", bad, "exempt", ex, "of", cg.size if gd else x["T"])
        assert bad == 0
    e = rel_fro(res["Xh"], ref["Xh"])
    print("Xhat rel err", e)
    assert np.isfinite(res["Xh"]).all() and e <= tol(x)
    e1, e2 = rel_fro(res["dZ"], ref["dZ"]), rel_fro(res["dU_dec"], ref["dU_dec"])
    print("dZ rel err", e1, "dU_dec rel err", e2)
    assert e1 <= tol(x) and e2 <= tol(x)
    e3, e4 = rel_fro(res["dX"], ref["dX"]), rel_fro(res["dU"], ref["dU"])
    print("dX rel err", e3, "dU (enc+dec) rel err", e4)
    assert e3 <= tol(x) and e4 <= tol(x)
    return ref


# Anchor-dominant workloads: B with orthonormal rows (the frozen random
# orthonormal companion of Eq. 3), A ~ N(0,1), so the anchor term is as large
# as the activations; the receiver's tables (seed + 1) differ from the
# sender's.  Each is (generator keywords, codebook kind).
ANCHOR_CASES = {
    "small_amb": (dict(seed=70, T=1000, d=256, r=64, V=500, k=16, L=0, K=0), None),
    "small_coord": (dict(seed=71, T=1000, d=256, r=64, V=500, k=16, L=0, K=0, anchor_space="coord"), None),
    "small_amb_rvq": (dict(seed=72, T=1000, d=256, r=128, V=500, k=32, L=2, K=96), "stress"),
    "small_coord_rvq": (dict(seed=73, T=777, d=256, r=64, V=300, k=16, L=2, K=64, anchor_space="coord"),
                        "stress"),
    "fused_r256_amb": (dict(seed=74, T=1037, d=512, r=256, V=700, k=64, L=2, K=128), "stress"),
    "fused_r256_coord": (dict(seed=75, T=1037, d=512, r=256, V=700, k=48, L=2, K=128, anchor_space="coord"),
                         "stress"),
    "c4width_amb": (dict(seed=76, T=4096 + 37, d=2048, r=256, V=32000, k=128, L=0, K=0), None),
    "c4width_coord": (dict(seed=77, T=4096 + 37, d=2048, r=256, V=32000, k=128, L=0, K=0,
                           anchor_space="coord"), None),
}
_ANCHOR_BASE = dict(dtype="bf16", alpha=0.8, n_out=4, cb_sigma=None, gscale=1.0)


def anchor_case(name):
    """(sender workload, receiver workload, codebooks or None) of a case."""
    kw, cb = ANCHOR_CASES[name]
    kw = dict(kw)
    seed = kw.pop("seed")
    x = synth.codec_inputs(None, seed=seed, anchor="orthonormal", **dict(_ANCHOR_BASE, **kw))
    rx = synth.codec_inputs(None, seed=seed + 1000, anchor="orthonormal", **dict(_ANCHOR_BASE, **kw))
    C = stress_codebooks(x, seed + 2000) if cb == "stress" else None
    return x, rx, C


def oracle_payload(x, C=None):
    """The payload the oracle itself would send: bf16-rounded Z0, or codes."""
    Cn = x["C"] if C is None else C
    Z0 = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), x["anchor_space"], operand(x))
    if x["L"] == 0:
        from oracle.precision import round_bf16
        return round_bf16(Z0)
    return ocodec.rvq_encode(Z0, Cn)[0]


def grad_codebooks(x, Lg, Kg, seed):
    """Gradient codebooks drawn like the stress codebooks, from the oracle's
    own gradient rows dXhat U (codeword 0 = 0, the others residual rows plus
    5 % noise), so every code is in use."""
    rng = np.random.default_rng(seed)
    R = f64(x, "dXhat") @ ocodec._projector(x["U"], operand(x))
    T, r = R.shape
    C = np.zeros((Lg, Kg, r), dtype=np.float32)
    for l in range(Lg):
        sig = np.sqrt(np.mean(R ** 2))
        idx = rng.choice(T, Kg - 1, replace=False)
        C[l, 1:] = (R[idx] + 0.05 * sig * rng.standard_normal((Kg - 1, r))).astype(np.float32)
        codes, _, _ = ocodec.rvq_encode(R, C[l:l + 1].astype(np.float64))
        R = R - C[l].astype(np.float64)[codes[:, 0]]
    return C


def grouped_stress_codebooks(x, seed):
    """Stress codebooks for grouped RVQ: codeword rows drawn from the oracle's
    residual rows plus 5 % noise (codeword 0 = 0), the residual updated group
    by group after each round."""
    gd = x["group_dim"]
    rng = np.random.default_rng(seed)
    R = ocodec.project(f64(x, "X"), x["ids"], x["U"], f64(x, "A"), f64(x, "B"), x["anchor_space"], operand(x))
    L, K, r, T = x["L"], x["K"], x["r"], x["T"]
    C = np.zeros((L, K, r), dtype=np.float32)
    for l in range(L):
        sig = np.sqrt(np.mean(R ** 2))
        idx = rng.choice(T, K - 1, replace=False)
        C[l, 1:] = (R[idx] + 0.05 * sig * rng.standard_normal((K - 1, r))).astype(np.float32)
        codes, _, _ = ocodec.grouped_rvq_encode(R, C[l:l + 1].astype(np.float64), gd)
        R = R - ocodec.grouped_rvq_decode(codes, C[l:l + 1].astype(np.float64), gd)
    return C
