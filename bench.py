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
        "enc:gemm_rvq": (2 * T * r * (d + k) + 2 * T * L * r * K, T * (2 * d + 4 + 2 * k) + T * L * 2),
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


_SRC_BY_KERNEL = {"gemm_tn": "k_gemm_bf16.hip", "bu_gemm": "k_gemm_bf16.hip", "rvq": "k_rvq.hip",
                  "gemm_rvq": "k_rvq.hip",
                  "wgrad": "k_wgrad.hip", "reduce": "k_wgrad.hip", "reduce_corr": "k_wgrad.hip",
                  "anchor_reduce": "k_wgrad.hip", "bu_reduce": "k_wgrad.hip"}


def kernel_sources(name):
    """Source files whose text decides a chain kernel's code and launch shape."""
    short = name.split(":")[-1]
    return [_SRC_BY_KERNEL.get(short, "k_prep.hip"), "tn_gemm.hpp", "common.hpp", "kernels.hpp", "mapl_api.cpp"]


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
            if parts[1] == _src_sha(kernel_sources(kernel)):
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

    # grow the token sample until one run takes a third of the budget; if the
    # whole micro-batch is faster than that, repeat it until the budget is used
    n = 512
    dt = run(n)
    while dt < budget_s / 3 and n < x["T"]:
        n = min(x["T"], n * 4)
        dt = run(n)
    reps, total = 1, dt
    while total < budget_s / 2 and n == x["T"]:
        total += run(n)
        reps += 1
    return {"value": n * reps / total, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": "%s%d of %d tokens of the same workload, float64 NumPy, the four codec calls, "
                      "%d run(s) in %.1f s" % ("" if n == x["T"] else "first ", n, x["T"], reps, total)}


def _csvs(d, suffix):
    import glob
    return sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))


def _dispatches(d, suffix):
    """[(dispatch_id, kernel_name, row)] of every CSV under d ending in suffix."""
    import csv
    out = {}
    for f in _csvs(d, suffix):
        for row in csv.DictReader(open(f)):
            did = int(row["Dispatch_Id"])
            e = out.setdefault(did, {"name": row["Kernel_Name"], "row": row, "ctr": {}})
            if "Counter_Name" in row:
                e["ctr"][row["Counter_Name"]] = e["ctr"].get(row["Counter_Name"], 0.0) + float(row["Counter_Value"])
    return [(k, v["name"], v) for k, v in sorted(out.items())]


def _chain_map(disp, order, chains):
    """Name each library dispatch of the first `chains` codec chains (warm-up,
    timed and profiled steps; the SPEL timing follows them) by its position."""
    lib = [x for x in disp if "mapl::" in x[1]]
    n = len(order)
    if n == 0 or len(lib) < n * chains:
        raise SystemExit("summarize: %d library dispatches, fewer than %d chains of %d" % (len(lib), chains, n))
    lib = lib[:n * chains]
    named = []
    for i, (did, sym, e) in enumerate(lib):
        named.append((order[i % n], sym, e))
    # every position must always be the same kernel symbol
    for j in range(n):
        syms = {named[i][1] for i in range(j, len(named), n)}
        if len(syms) != 1:
            raise SystemExit("summarize: chain position %d (%s) maps to several kernels" % (j, order[j]))
    return named


def _short(sym):
    import re
    s = sym.replace("(anonymous namespace)::", "").replace("mapl::", "").replace("void ", "")
    return re.sub(r"\(.*", "", s)


def _counter_table(d, order, agg):
    """Mean of every counter of one rocprofv3 --pmc run per chain kernel; with
    MfmaFlopsBF16 / MfmaFlopsF32 also the matrix rate they imply over the
    kernel's trace duration, against the dense MFMA peak of its type."""
    disp = _dispatches(d, "_counter_collection.csv")
    named = _chain_map(disp, order, len([x for x in disp if "mapl::" in x[1]]) // len(order))
    acc = {}
    for name, _, e in named:
        for c, v in e["ctr"].items():
            acc.setdefault(name, {}).setdefault(c, []).append(v)
    ctrs = sorted({c for v in acc.values() for c in v})
    rate = [c for c in ("MfmaFlopsBF16", "MfmaFlopsF32") if c in ctrs]
    out = ["", "# rocprofv3 --pmc %s (mean per launch; percentages as rocprofv3 derives them)" % " ".join(ctrs)]
    if rate:
        out.append("# TFLOP/s = counted matrix flops over the kernel's trace duration; frac against the dense "
                   "peak of that type (bf16 2516.6, fp32 157.3)")
    hdr = "%-24s" % "kernel" + "".join(" %16s" % c for c in ctrs) + ("  %9s %6s" % ("TFLOP/s", "frac") if rate else "")
    out.append(hdr)
    for name in order:
        v = acc.get(name, {})
        row = "%-24s" % name + "".join(" %16.4g" % np.mean(v[c]) if c in v else " %16s" % "-" for c in ctrs)
        if rate:
            us = agg[name][2] / agg[name][1]
            fl = {c: np.mean(v[c]) for c in rate if c in v}
            best = max(fl, key=fl.get) if fl else None
            if best and fl[best] > 0:
                tf = fl[best] / us / 1e6
                row += "  %9.1f %6.3f" % (tf, tf * 1e12 / (PEAK_BF16 if best == "MfmaFlopsBF16" else PEAK_F32))
            else:
                row += "  %9s %6s" % ("-", "-")
        out.append(row)
    return out


def summarize(paths, write_traffic):
    bench = json.loads(open(paths[0]).read().strip().splitlines()[-1])
    order = bench["kernel_order"]
    lines = ["# c4 codec chain (T=32768, d=2048, r=256, k=128, L=2, K=1024, bf16): per-kernel durations",
             "# from the rocprofv3 kernel trace of a bench.py run; each library dispatch is named by its",
             "# position in the repeated 4-call chain; bench.py's own HIP-event average beside it.", ""]
    disp = _dispatches(paths[1], "_kernel_trace.csv")
    named = _chain_map(disp, order, bench["warmup"] + 2 * bench["steps"])
    agg = {}
    for name, sym, e in named:
        row = e["row"]
        a = agg.setdefault(name, [sym, 0, 0.0])
        a[1] += 1
        a[2] += (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3
    lines.append("%-24s %-36s %8s %10s %10s" % ("kernel", "symbol", "launches", "trace_us", "bench_us"))
    for name in order:
        sym, n, tot = agg[name]
        lines.append("%-24s %-36s %8d %10.2f %10s" % (name, _short(sym)[:36], n, tot / n,
                                                     "%.2f" % bench["per_kernel_us"].get(name, float("nan"))))
    chain_us = sum(agg[nm][2] / agg[nm][1] for nm in order)
    lines.append("%-24s %-36s %8s %10.2f %10.2f" % ("sum over the chain", "", "", chain_us, bench["ms_per_step"] * 1e3))
    stats = _csvs(paths[1], "_kernel_stats.csv")
    if stats:
        import csv
        lines += ["", "# rocprofv3 --stats (all dispatches of the run, by kernel symbol)"]
        rows = list(csv.DictReader(open(stats[0])))
        for row in rows[:16]:
            lines.append("%-48s calls %6s  avg_us %10.2f  total_pct %6s" % (
                _short(row.get("Name", "?"))[:48], row.get("Calls", "?"), float(row.get("AverageNs", 0)) / 1e3,
                row.get("Percentage", "?")[:6]))
    traffic = {}
    if len(paths) >= 4:
        calib = bench.get("calib_copy_bytes")
        fd, wd = _dispatches(paths[2], "_counter_collection.csv"), _dispatches(paths[3], "_counter_collection.csv")
        cf = [e["ctr"]["FETCH_SIZE"] for _, nm, e in fd if "copyBuffer" in nm]
        cw = [e["ctr"]["WRITE_SIZE"] for _, nm, e in wd if "copyBuffer" in nm]
        if not calib or not cf or not cw:
            raise SystemExit("summarize: counter runs need --calib-copy (a copyBuffer dispatch)")
        ff, fw = calib / (cf[-1] * 1024.0), calib / (cw[-1] * 1024.0)
        lines += ["", "# HBM traffic per launch from two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE, KiB per",
                  "# dispatch), each scaled by what the same counter reads for a plain %d-byte device copy:" % calib,
                  "#   FETCH_SIZE %.0f KiB -> factor %.4f;  WRITE_SIZE %.0f KiB -> factor %.4f" % (cf[-1], ff, cw[-1], fw),
                  "# GB/s = traffic over the kernel's trace duration above; frac = GB/s over 8000 GB/s",
                  "%-24s %12s %12s %14s %14s %7s %8s %6s" % ("kernel", "fetch_KiB", "write_KiB", "traffic_B",
                                                           "algorithmic_B", "ratio", "GB/s", "frac")]
        fn = _chain_map(fd, order, len([x for x in fd if "mapl::" in x[1]]) // len(order))
        wn = _chain_map(wd, order, len([x for x in wd if "mapl::" in x[1]]) // len(order))
        kc = kernel_counts(32768, 2048, 256, 128, 2, 1024)
        acc = {}
        for (name, _, e) in fn:
            acc.setdefault(name, [[], []])[0].append(e["ctr"]["FETCH_SIZE"])
        for (name, _, e) in wn:
            acc.setdefault(name, [[], []])[1].append(e["ctr"]["WRITE_SIZE"])
        for name in order:
            fk, wk = np.mean(acc[name][0]), np.mean(acc[name][1])
            tb = fk * 1024 * ff + wk * 1024 * fw
            alg = kc[name][1] if name in kc else None
            traffic[name] = tb
            gbs = tb / (agg[name][2] / agg[name][1]) / 1e3
            lines.append("%-24s %12.0f %12.0f %14.0f %14s %7s %8.0f %6.3f" % (
                name, fk, wk, tb, "%.0f" % alg if alg else "-", "%.2f" % (tb / alg) if alg else "-", gbs,
                gbs * 1e9 / PEAK_HBM))
    for d in paths[4:]:
        lines += _counter_table(d, order, agg)
    print("\n".join(lines))
    if write_traffic and traffic:
        path = os.path.join(ROOT, "profiles", "traffic_c4.txt")
        with open(path, "w") as fh:
            fh.write("# kernel source_sha256[:16] hbm_bytes_per_launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated);\n"
                     "# written by bench.py --summarize --write-traffic; a line counts only while the kernel's\n"
                     "# sources hash to the recorded value\n")
            for name in order:
                fh.write("%s %s %.0f\n" % (name, _src_sha(kernel_sources(name)), traffic[name]))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stress", action="store_true", help="data-drawn codebooks (every code in use)")
    ap.add_argument("--no-spel", action="store_true", help="skip the SPEL step timing")
    ap.add_argument("--calib-copy", action="store_true",
                    help="end with one plain 256 MiB device copy (calibrates FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--summarize", nargs="+", metavar="PATH",
                    help="no GPU: BENCH_JSON TRACE_DIR [FETCH_DIR WRITE_DIR [PMC_DIR ...]] -> kernel summary on "
                         "stdout (each PMC_DIR: one more rocprofv3 --pmc run, every counter tabulated)")
    ap.add_argument("--write-traffic", action="store_true",
                    help="with --summarize and counter dirs: rewrite profiles/traffic_c4.txt")
    args = ap.parse_args()
    if args.summarize:
        summarize(args.summarize, args.write_traffic)
        return
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

    spel, alg1 = None, None
    if not args.no_spel:
        spel_c5 = time_spel(16, 2048, 512, 5)
        spel_b = time_spel(1, d, r, 10)
        spel = {"config": "16 projectors [2048,512], PolarExpress 5 + 7 steps", "ms_per_step": spel_c5,
                "tflops": spel_flops(16, 2048, 512) / (spel_c5 * 1e-3) / 1e12,
                "roofline_frac_fp32": spel_flops(16, 2048, 512) / PEAK_F32 / (spel_c5 * 1e-3),
                "boundary_projector_ms": spel_b}
        amort = 128  # micro-batches per optimizer step: global batch 512 / micro-batch 4
        alg1 = T / ((ms + spel_b / amort) * 1e-3)
    calib = None
    if args.calib_copy:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        calib = src.numel()

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
        "kernel_order": list(kern),
        "spel": spel,
        "alg1_tokens_per_s": alg1,
    }
    if calib:
        out["calib_copy_bytes"] = calib
    if not args.no_cpu_baseline:
        print("timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(x)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
