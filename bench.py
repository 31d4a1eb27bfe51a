"""Benchmark of the MAPL boundary codec on one MI355X.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5]

One step is the codec chain of one pipeline boundary over one micro-batch
with inputs resident in HBM: encode (Eq. 1 + RVQ) -> decode (Eq. 2) ->
decode_bwd (dZhat, dU) -> encode_bwd (dX, dU accumulated), the r-dim
gradient of decode_bwd feeding encode_bwd as it would cross the pipeline.
Workload: the 1B-shaped boundary T = 16 x 2048 = 32768 tokens, d = 2048,
r = 256, anchor rank k = 128 over V = 32000, L = 2 RVQ stages of K = 1024
codewords, bf16 activations, synthetic seeded inputs.

Prints one JSON line: tokens/s of the chain, the chain's fraction of its
MFMA/HBM roofline, a live per-kernel roofline for the dominant kernel
(HIP events on the launch stream), the SPEL step timed at its own
configuration (16 projectors [2048,512]) and once for this boundary's
projector, and the float64 oracle timed on a bounded token sample on the
host cores (rank 0, N = 1 only).
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "boundary codec tokens/sec (enc+dec fwd+bwd) and % MFMA/HBM roofline, 1 MI355X"
PEAK_BF16 = 2516.6e12   # dense bf16 MFMA, FLOP/s
PEAK_F32 = 157.3e12     # dense fp32 MFMA, FLOP/s
PEAK_HBM = 8.0e12       # HBM3E, B/s


def per_call_counts(T, d, r, k, L, K, payload):
    """Algorithmic flops / bytes per call (per micro-batch), ambient anchor.

    enc: 2dr + 2kr + 2LrK flop, 2d + 4 + 2k + payload bytes per token
    dec: 2rd + 2kd flop,        payload + 4 + 2k + 2d bytes
    dec_bwd: 4dr flop,          2d + payload + 2r bytes
    enc_bwd: 4dr + 2kr flop,    2r + 4d + 4 + 2k bytes
    """
    c = {
        "encode": (2 * d * r + 2 * k * r + 2 * L * r * K, 2 * d + 4 + 2 * k + payload),
        "decode": (2 * r * d + 2 * k * d, payload + 4 + 2 * k + 2 * d),
        "decode_bwd": (4 * d * r, 2 * d + payload + 2 * r),
        "encode_bwd": (4 * d * r + 2 * k * r, 2 * r + 4 * d + 4 + 2 * k),
    }
    return {n: (f * T, b * T) for n, (f, b) in c.items()}


def kernel_counts(T, d, r, k, L, K):
    """Algorithmic (flops, bytes, bound) per launch of the codec's main kernels.

    Bytes count each kernel's compulsory HBM inputs and outputs at the
    element sizes the kernel uses (bf16 activations, fp32 Z0 / partials)."""
    return {
        "enc:gemm_tn": (2 * T * r * (d + k), T * (2 * d + 4 + 2 * k) + T * r * 4),
        "enc:rvq": (2 * T * L * r * K, T * r * 4 + T * L * 2),
        "dec:gemm_tn": (2 * T * d * (r + k), T * (2 * r + 4 + 2 * k) + T * d * 2),
        "dec:assemble": (T * L * r, T * L * 2 + T * r * 2),
        "dec_bwd:gemm_tn": (2 * T * d * r, T * d * 2 + T * r * 2),
        "dec_bwd:wgrad": (2 * T * d * r, T * d * 2 + T * r * 2),
        "enc_bwd:gemm_tn": (2 * T * d * r, T * r * 2 + T * d * 2),
        "enc_bwd:wgrad": (2 * T * (d + k) * r, T * d * 2 + T * r * 2 + T * (4 + 2 * k)),
    }


def _src_sha(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2606_05484_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "enc:gemm_tn": ["k_gemm_bf16.hip", "common.hpp"], "dec:gemm_tn": ["k_gemm_bf16.hip", "common.hpp"],
    "dec_bwd:gemm_tn": ["k_gemm_bf16.hip", "common.hpp"], "enc_bwd:gemm_tn": ["k_gemm_bf16.hip", "common.hpp"],
    "enc:rvq": ["k_rvq.hip", "common.hpp"], "dec_bwd:wgrad": ["k_wgrad.hip", "common.hpp"],
    "enc_bwd:wgrad": ["k_wgrad.hip", "common.hpp"], "dec:assemble": ["k_prep.hip", "common.hpp"],
}


def traffic_for(kernel):
    """HBM bytes per launch from committed rocprofv3 counter summaries, or None.

    profiles/traffic_c4.txt holds lines 'kernel source_sha bytes_per_launch';
    a line counts only while the kernel's sources still hash to source_sha."""
    path = os.path.join(ROOT, "profiles", "traffic_c4.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        parts = line.split()
        if len(parts) == 3 and parts[0] == kernel and not line.startswith("#"):
            if parts[1] == _src_sha(KERNEL_SOURCES.get(kernel, [])):
                return float(parts[2])
    return None


def cpu_baseline(x, budget_s=15.0):
    """Time the float64 oracle's four codec calls on a token sample."""
    from oracle import codec as oc
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    from paper_2606_05484_amd import synth
    f64 = lambda k, sel: synth.as_f64(x[k][sel], "bf16")
    A, B = synth.as_f64(x["A"], "bf16"), synth.as_f64(x["B"], "bf16")

    def run(n):
        sel = slice(0, n)
        X, dXh, dZ = f64("X", sel), f64("dXhat", sel), f64("dZ", sel)
        ids = x["ids"][sel]
        t0 = time.perf_counter()
        codes, _, _ = oc.encode(X, ids, x["U"], A, B, x["C"], operand="bf16")
        oc.decode(codes, ids, x["U"], A, B, x["C"], operand="bf16")
        oc.decode_bwd(dXh, codes, ids, x["U"], A, B, x["C"], operand="bf16")
        oc.encode_bwd(dZ, X, ids, x["U"], A, B, operand="bf16")
        return time.perf_counter() - t0

    n = 512
    dt = run(n)
    while dt < budget_s / 3 and n < x["T"]:
        n = min(x["T"], n * 4)
        dt = run(n)
    return {"value": n / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": "first %d of %d tokens of the same workload, float64 NumPy, the four codec calls "
                      "(%.1f s)" % (n, x["T"], dt)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stress", action="store_true", help="data-drawn codebooks (every code in use)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU; --gpus %d is not supported (the codec shards over "
              "tokens and the SPEL step over projectors, see DESIGN.md)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_05484_amd import mapl, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    print("generating workload c4", file=sys.stderr, flush=True)
    x = synth.codec_inputs("c4")
    T, d, r, V, k, L, K = (x[n] for n in ("T", "d", "r", "V", "k", "L", "K"))
    C = x["C"]
    if args.stress:
        from oracle import codec as oc
        Z0 = oc.project(synth.as_f64(x["X"][:8192], "bf16"), x["ids"][:8192], x["U"],
                        synth.as_f64(x["A"], "bf16"), synth.as_f64(x["B"], "bf16"), "ambient", "bf16")
        rng = np.random.default_rng(104)
        C = np.zeros_like(x["C"])
        C[0, 1:] = Z0[rng.choice(8192, K - 1, replace=False)]
        C[1, 1:] = 0.3 * Z0[rng.choice(8192, K - 1, replace=False)]
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    X, A, B, dXh = bf(x["X"]), bf(x["A"]), bf(x["B"]), bf(x["dXhat"])
    U = torch.from_numpy(x["U"]).cuda()
    ids = torch.from_numpy(x["ids"]).cuda()
    Cg = torch.from_numpy(np.ascontiguousarray(C)).cuda()
    D = mapl.desc(T=T, d=d, r=r, V=V, k=k, L=L, K=K)
    ws = mapl.workspace(max(mapl.workspace_bytes(D, c) for c in range(4)))
    codes = torch.empty((T, L), dtype=torch.int16, device="cuda")
    Xh = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    dZ = torch.empty((T, r), dtype=torch.bfloat16, device="cuda")
    dX = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    dU = torch.empty((d, r), device="cuda")

    calls = ["encode", "decode", "decode_bwd", "encode_bwd"]

    def step(ev=None):
        if ev: ev[0].record()
        mapl.encode(D, X, ids, U, A, B, Cg, codes, ws)
        if ev: ev[1].record()
        mapl.decode(D, codes, ids, U, A, B, Cg, Xh, ws)
        if ev: ev[2].record()
        mapl.decode_bwd(D, dXh, codes, ids, U, A, B, Cg, dZ, dU, 0, ws)
        if ev: ev[3].record()
        mapl.encode_bwd(D, dZ, X, ids, U, A, B, dX, dU, 1, ws)
        if ev: ev[4].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("timing %d steps" % args.steps, file=sys.stderr, flush=True)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for _ in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    value = T / (ms * 1e-3)

    # per-call times (events between calls) and per-kernel times (library trace)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    mapl.profile(True)
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    mapl.profile(False)
    prof = mapl.profile_report()
    per_call = {c: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) * 1e3 for i, c in enumerate(calls)}

    payload = L * 2
    cc = per_call_counts(T, d, r, k, L, K, payload)
    roof_calls = {n: max(f / PEAK_BF16, b / PEAK_HBM) for n, (f, b) in cc.items()}
    roof_chain = sum(roof_calls.values())
    Fsum, Bsum = sum(f for f, _ in cc.values()), sum(b for _, b in cc.values())
    chain_frac = roof_chain / (ms * 1e-3)

    kc = kernel_counts(T, d, r, k, L, K)
    kern = {n: (cnt, tot / cnt * 1e3) for n, (cnt, tot) in prof.items()}  # name -> (launches, avg us)
    dom = max((n for n in kern if n in kc), key=lambda n: kern[n][0] * kern[n][1])
    f, b = kc[dom]
    avg_s = kern[dom][1] * 1e-6
    if f / PEAK_BF16 >= b / PEAK_HBM:
        roof = {"bound": "mfma", "achieved": f / avg_s / 1e12, "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": b / avg_s / 1e9, "peak": PEAK_HBM / 1e9, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = traffic_for(dom)
    roof["kernel"] = dom
    roof["avg_us"] = kern[dom][1]

    # SPEL step: its own configuration (16 x [2048,512]) and this boundary's projector
    def time_spel(P, dd, rr, reps):
        st = synth.stiefel_inputs(None, seed=55, P=P, d=dd, r=rr, gscale=1e-3, lr=1e-2, beta=0.95, steps=1)
        Ug, Gg, Mg = (torch.from_numpy(st[n]).cuda() for n in ("U", "G", "M"))
        w = mapl.workspace(mapl.workspace_bytes(None, mapl.CALL_STIEFEL, P, dd, rr))
        for _ in range(2):
            mapl.stiefel_step(P, dd, rr, Ug, Gg, Mg, 1e-2, 0.95, 5, 7, w)
        a, bb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            mapl.stiefel_step(P, dd, rr, Ug, Gg, Mg, 1e-2, 0.95, 5, 7, w)
        bb.record()
        torch.cuda.synchronize()
        return a.elapsed_time(bb) / reps

    def spel_flops(P, dd, rr):
        it = 4 * dd * rr * rr + 2 * rr ** 3
        return P * (4 * dd * rr * rr + 12 * it)

    spel_c5 = time_spel(16, 2048, 512, 5)
    spel_b = time_spel(1, d, r, 10)
    spel = {"config": "16 projectors [2048,512], PolarExpress 5 + 7 steps", "ms_per_step": spel_c5,
            "tflops": spel_flops(16, 2048, 512) / (spel_c5 * 1e-3) / 1e12,
            "roofline_frac_fp32": spel_flops(16, 2048, 512) / PEAK_F32 / (spel_c5 * 1e-3),
            "boundary_projector_ms": spel_b}
    amort = 128  # micro-batches per optimizer step: global batch 512 / micro-batch 4
    alg1 = T / ((ms + spel_b / amort) * 1e-3)

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "1B-shaped boundary (c4): T=32768 tokens (16x2048), d=2048, r=256, "
                               "anchor k=128 over V=32000 (Zipf 1.1 ids), RVQ L=2 x K=1024, u16 codes, "
                               "ambient anchor, enc+dec fwd+bwd per step" + (", data-drawn codebooks" if args.stress else ""),
                   "global_batch": T, "seq_len": 2048, "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "chain_roofline": {"frac": chain_frac, "roofline_us": roof_chain * 1e6, "measured_us": ms * 1e3,
                           "flops": Fsum, "bytes": Bsum},
        "per_call_us": per_call,
        "per_kernel_us": {n: round(v[1], 2) for n, v in sorted(kern.items())},
        "spel": spel,
        "alg1_tokens_per_s": alg1,
    }
    if not args.no_cpu_baseline:
        print("timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(x)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
