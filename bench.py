"""Benchmark of the MAPL boundary codec on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--graph] [--no-extra]

One step is the codec chain of one pipeline boundary over one micro-batch
with inputs resident in HBM: encode (Eq. 1 + RVQ) -> decode (Eq. 2) ->
decode_bwd (dZhat, dU) -> encode_bwd (dX, dU accumulated), the r-dim
gradient of decode_bwd feeding encode_bwd as it would cross the pipeline.
Headline workload: the 1B-shaped boundary T = 16 x 2048 = 32768 tokens,
d = 2048, r = 256, anchor rank k = 128 over V = 32000, L = 2 RVQ stages of
K = 1024 codewords, bf16 activations, synthetic seeded inputs.

Prints one JSON line: tokens/s of the chain (warm-up steps, then the mean
over a block of `steps` steps between two events; the median of `steps`
event-separated steps beside it), eager and replayed as one HIP graph; the
chain's fraction of its MFMA/HBM roofline; a live per-kernel roofline for
the dominant kernel (HIP events around each launch on its stream); the same
chain with data-drawn codebooks ("stress": every code in use) with the RVQ
encoder's decision counters; every other workload (c1, c2 for r = 64..512,
c3) with its tokens/s, roofline fraction and the oracle's tokens/s; the SPEL
step (16 projectors [2048,512], and this boundary's projector); and the
float64 oracle timed on the host cores (rank 0, N = 1 only).
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
    """Time the float64 oracle's four codec calls on a token sample of
    workload x, with its BLAS limited to the host cores this process may run
    on (len(os.sched_getaffinity(0)))."""
    from oracle import codec as oc
    from paper_2606_05484_amd import synth
    cores = len(os.sched_getaffinity(0))
    blas, ctl = "unknown", None
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = "%s %s" % (info[0].get("internal_api", "?"), info[0].get("version", ""))
        ctl = threadpool_limits(limits=cores, user_api="blas")
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = None
    dt = x["dtype"]
    op = "bf16" if dt == "bf16" else "exact"
    f64 = lambda k, sel: synth.as_f64(x[k][sel], dt)
    A, B = synth.as_f64(x["A"], dt), synth.as_f64(x["B"], dt)
    C = x["C"] if x["L"] else None

    def run(n):
        sel = slice(0, n)
        X, dXh, dZ = f64("X", sel), f64("dXhat", sel), f64("dZ", sel)
        ids = x["ids"][sel]
        t0 = time.perf_counter()
        enc = oc.encode(X, ids, x["U"], A, B, C, operand=op)
        pay = enc[0] if C is not None else enc
        oc.decode(pay, ids, x["U"], A, B, C, operand=op)
        oc.decode_bwd(dXh, pay, ids, x["U"], A, B, C, operand=op)
        oc.encode_bwd(dZ, X, ids, x["U"], A, B, operand=op)
        return time.perf_counter() - t0

    try:
        # grow the token sample until one run takes a third of the budget; if
        # the whole micro-batch is faster than that, repeat it until the
        # budget is used
        n = min(512, x["T"])
        dt_ = run(n)
        while dt_ < budget_s / 3 and n < x["T"]:
            n = min(x["T"], n * 4)
            dt_ = run(n)
        reps, total = 1, dt_
        while total < budget_s / 2 and n == x["T"]:
            total += run(n)
            reps += 1
    finally:
        if ctl is not None:
            ctl.unregister() if hasattr(ctl, "unregister") else None
    return {"value": n * reps / total, "unit": "tokens/s", "cores": cores, "blas_threads": threads, "blas": blas,
            "kind": "oracle",
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
    # the chains may follow a few set-up dispatches (e.g. the data-drawn
    # codebooks' projection): the first offset at which every chain position
    # is always the same kernel symbol
    for off in range(0, 8):
        body = lib[off:]
        m = min(chains, len(body) // n) if n else 0
        if m < 1:
            break
        body = body[:n * m]
        if all(len({body[i][1] for i in range(j, len(body), n)}) == 1 for j in range(n)):
            return [(order[i % n], sym, e) for i, (did, sym, e) in enumerate(body)]
    raise SystemExit("summarize: no offset maps the %d library dispatches onto chains of %d" % (len(lib), n))


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
    named = _chain_map(disp, order, len([x for x in disp if "mapl::" in x[1]]) // len(order))
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


GROUP_DIST_FLOPS = 5  # (x - cx)^2 + (y - cy)^2: two subtractions, two products, one sum


def chain_counts(x):
    """Per-call algorithmic (matrix flops, vector-ALU flops, bytes) of
    workload x (see per_call_counts).  Whole-vector RVQ distances are matrix
    products (2 r K per token and round); the grouped quantiser's 2-D
    distances are vector work (5 flops per codeword, group and round)."""
    es = 4 if x["dtype"] == "f32" else 2
    T, d, r, k, L, K = (x[n] for n in ("T", "d", "r", "k", "L", "K"))
    gd = x.get("group_dim", 0) if L else 0
    if gd:
        pay = L * (r // gd)
        rvq_m, rvq_a = 0, GROUP_DIST_FLOPS * L * (r // gd) * K
    else:
        pay = (L * (1 if K <= 256 else 2)) if L else r * es
        rvq_m, rvq_a = 2 * L * r * K, 0
    c = {
        "encode": (2 * d * r + 2 * k * r + rvq_m, rvq_a, es * d + 4 + es * k + pay),
        "decode": (2 * r * d + 2 * k * d, 0, pay + 4 + es * k + es * d),
        "decode_bwd": (4 * d * r, 0, es * d + pay + es * r),
        "encode_bwd": (4 * d * r + 2 * k * r, 0, es * r + 2 * es * d + 4 + es * k),
    }
    return {n: (fm * T, fa * T, b * T) for n, (fm, fa, b) in c.items()}


def roofline_of(x, ms):
    """Chain roofline: sum over calls of max(Fm / mfma peak + Fa / fp32
    vector peak, B / HBM) against the measured ms per step (matrix peak:
    bf16 or fp32 MFMA by the workload's type)."""
    peak = PEAK_F32 if x["dtype"] == "f32" else PEAK_BF16
    cc = chain_counts(x)
    per = {n: max(fm / peak + fa / PEAK_F32, b / PEAK_HBM) for n, (fm, fa, b) in cc.items()}
    bound = {n: (("mfma" if fm / peak >= fa / PEAK_F32 else "alu") if fm / peak + fa / PEAK_F32 >= b / PEAK_HBM
                 else "hbm") for n, (fm, fa, b) in cc.items()}
    roof = sum(per.values())
    return {"frac": roof / (ms * 1e-3), "roofline_us": roof * 1e6, "measured_us": ms * 1e3,
            "flops": sum(fm + fa for fm, fa, _ in cc.values()), "bytes": sum(b for _, _, b in cc.values()),
            "bound_per_call": bound}


class Chain:
    """Device buffers of one workload and its four-call chain (encode ->
    decode -> decode_bwd -> encode_bwd, the decoder's dZ feeding the
    encoder's backward as it would cross the pipeline)."""

    def __init__(self, torch, mapl, x, C):
        self.torch = torch
        self.mapl = mapl
        dt = x["dtype"]
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32

        def put(a):
            a = np.ascontiguousarray(a)
            if dt == "bf16":
                return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
            return torch.from_numpy(a).cuda()

        T, d, r, L, K = (x[n] for n in ("T", "d", "r", "L", "K"))
        self.X, self.A, self.B, self.dXh = put(x["X"]), put(x["A"]), put(x["B"]), put(x["dXhat"])
        self.U = torch.from_numpy(x["U"]).cuda()
        self.ids = torch.from_numpy(x["ids"]).cuda()
        self.C = torch.from_numpy(np.ascontiguousarray(C, dtype=np.float32)).cuda() if L else None
        self.D = mapl.desc(T=T, d=d, r=r, V=x["V"], k=x["k"], L=L, K=K, x_dtype=dt,
                           group_dim=x.get("group_dim", 0) if L else 0)
        self.ws = mapl.workspace(max(mapl.workspace_bytes(self.D, c) for c in range(4)))
        if L and self.D.group_dim:
            self.payload = torch.empty((T, L, r // self.D.group_dim), dtype=torch.uint8, device="cuda")
        elif L:
            self.payload = torch.empty((T, L), dtype=torch.uint8 if K <= 256 else torch.int16, device="cuda")
        else:
            self.payload = torch.empty((T, r), dtype=tdt, device="cuda")
        self.Xh = torch.empty((T, d), dtype=tdt, device="cuda")
        self.dZ = torch.empty((T, r), dtype=tdt, device="cuda")
        self.dX = torch.empty((T, d), dtype=tdt, device="cuda")
        self.dU = torch.empty((d, r), device="cuda")
        self.T = T

    def step(self, ev=None):
        m, D = self.mapl, self.D
        if ev: ev[0].record()
        m.encode(D, self.X, self.ids, self.U, self.A, self.B, self.C, self.payload, self.ws)
        if ev: ev[1].record()
        m.decode(D, self.payload, self.ids, self.U, self.A, self.B, self.C, self.Xh, self.ws)
        if ev: ev[2].record()
        m.decode_bwd(D, self.dXh, self.payload, self.ids, self.U, self.A, self.B, self.C, self.dZ, self.dU, 0,
                     self.ws)
        if ev: ev[3].record()
        m.encode_bwd(D, self.dZ, self.X, self.ids, self.U, self.A, self.B, self.dX, self.dU, 1, self.ws)
        if ev: ev[4].record()

    def capture(self):
        """The chain captured once into a graph (its launches only: the
        library records no memset and no synchronisation)."""
        torch = self.torch
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step()
        torch.cuda.synchronize()
        return g


def time_steps(torch, run, warmup, steps):
    """warmup untimed runs, then `steps` runs between two events (mean ms per
    step over the block: the throughput figure), then `steps` more runs with
    an event between consecutive runs (median ms per step)."""
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        run()
    t1.record()
    torch.cuda.synchronize()
    mean = t0.elapsed_time(t1) / steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        run()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return mean, float(np.median(per))


def library_stress_codebooks(torch, mapl, x, seed=104, n=8192):
    """Data-drawn codebooks (every code in use) from the library's own
    projection of the first n tokens: codeword 0 = 0, round 0's other
    codewords are projected tokens, round 1's are 0.3 times projected
    tokens.  Only the seeded choice of tokens is drawn here."""
    n = min(n, x["T"])
    sub = dict(x, T=n, X=x["X"][:n], ids=x["ids"][:n], dXhat=x["dXhat"][:n], L=0, K=0)
    ch = Chain(torch, mapl, sub, np.zeros((0,)))
    mapl.encode(ch.D, ch.X, ch.ids, ch.U, ch.A, ch.B, None, ch.payload, ch.ws)
    torch.cuda.synchronize()
    Z = ch.payload.float().cpu().numpy()
    rng = np.random.default_rng(seed)
    C = np.zeros((x["L"], x["K"], x["r"]), dtype=np.float32)
    C[0, 1:] = Z[rng.choice(n, x["K"] - 1, replace=False)]
    for l in range(1, x["L"]):
        C[l, 1:] = 0.3 * Z[rng.choice(n, x["K"] - 1, replace=False)]
    return C


def next_rows(torch, mapl, x, Cs, args):
    """Timings of the calls beside the four-call chain at the c4 widths,
    each against its own roofline: decode_bwd with the returned gradient
    quantised (K = 1024, two rounds; Sec. 3.5), the anchor-table gradient on
    both sides (Eq. 3) and the streaming codebook sync (1/5 of the codewords
    per micro-batch)."""
    T, d, r, V, k, L, K = (x[n] for n in ("T", "d", "r", "V", "k", "L", "K"))
    ch = Chain(torch, mapl, x, Cs)
    ch.step()
    out = {}
    # gradient codebooks: the library's own gradient rows dXhat U~ of the first 8192 tokens
    n = 8192
    sub = dict(x, T=n, X=x["dXhat"][:n], ids=x["ids"][:n], dXhat=x["dXhat"][:n], L=0, K=0, k=0)
    cg = Chain(torch, mapl, sub, np.zeros((0,)))
    mapl.encode(cg.D, cg.X, None, cg.U, None, None, None, cg.payload, cg.ws)
    torch.cuda.synchronize()
    G = cg.payload.float().cpu().numpy()
    rng = np.random.default_rng(105)
    Lg, Kg = 2, 1024
    Cg = np.zeros((Lg, Kg, r), dtype=np.float32)
    Cg[0, 1:] = G[rng.choice(n, Kg - 1, replace=False)]
    Cg[1, 1:] = 0.3 * G[rng.choice(n, Kg - 1, replace=False)]
    Cgg = torch.from_numpy(Cg).cuda()
    del cg
    wsq = mapl.workspace(mapl.decode_bwd_q_workspace_bytes(ch.D, Lg, Kg))
    gcodes = torch.empty((T, Lg), dtype=torch.int16, device="cuda")
    run = lambda: mapl.decode_bwd_q(ch.D, ch.dXh, ch.payload, ch.ids, ch.U, ch.A, ch.B, ch.C, Lg, Kg, Cgg, gcodes,
                                    ch.dU, 0, wsq)
    q_ms, q_med = time_steps(torch, run, 3, args.steps)
    runb = lambda: mapl.decode_bwd(ch.D, ch.dXh, ch.payload, ch.ids, ch.U, ch.A, ch.B, ch.C, ch.dZ, ch.dU, 0, ch.ws)
    b_ms, b_med = time_steps(torch, runb, 3, args.steps)
    fq = T * (4 * d * r + 2 * Lg * r * Kg)
    bq = T * (2 * d + 2 * L + 2 * Lg)
    roofq = max(fq / PEAK_BF16, bq / PEAK_HBM)
    out["decode_bwd_q"] = {"gradient_codebooks": "Lg=2 x Kg=1024 drawn from the library's own dXhat U~ rows",
                           "median_us": q_med * 1e3, "decode_bwd_median_us": b_med * 1e3,
                           "tokens_per_s": T / (q_med * 1e-3), "roofline_us": roofq * 1e6,
                           "roofline_frac": roofq / (q_med * 1e-3),
                           "bytes_per_token_returned": 2 * Lg, "bytes_per_token_unquantised": 2 * r}
    # anchor-table gradient, both sides
    for side, name in ((mapl.SENDER, "sender"), (mapl.RECEIVER, "receiver")):
        wsa = mapl.workspace(mapl.anchor_bwd_workspace_bytes(ch.D, side))
        dA = torch.empty((V, k), device="cuda")
        dY = ch.dZ if side == mapl.SENDER else ch.dXh
        runa = lambda: mapl.anchor_bwd(ch.D, side, dY, ch.ids, ch.U, ch.B, dA, 0, wsa)
        a_ms, a_med = time_steps(torch, runa, 3, args.steps)
        width = r if side == mapl.SENDER else d
        ba = T * (2 * width + 4) + V * k * 4
        fa = T * 2 * width * k
        roofa = max(fa / PEAK_BF16, ba / PEAK_HBM)
        mapl.profile(1)
        runa()
        torch.cuda.synchronize()
        mapl.profile(0)
        kp = mapl.profile_report()
        out["anchor_bwd_" + name] = {"median_us": a_med * 1e3, "roofline_us": roofa * 1e6,
                                     "roofline_frac": roofa / (a_med * 1e-3),
                                     "bound": "mfma" if fa / PEAK_BF16 >= ba / PEAK_HBM else "hbm",
                                     "per_kernel_us": {nm: round(v[1] / v[0] * 1e3, 2) for nm, v in kp.items()}}
        del wsa, dA
    # streaming codebook sync: one part of five per micro-batch
    parts = 5
    nrow = (K + parts - 1) // parts
    rows = torch.from_numpy(np.stack([np.random.default_rng(l).permutation(K)[:nrow] for l in range(L)])
                            .astype(np.int32)).cuda()
    buf = torch.empty((L, nrow, r), device="cuda")
    recv = ch.C.clone()
    runs = lambda: (mapl.codebook_pack(L, K, r, ch.C, rows, nrow, buf),
                    mapl.codebook_unpack(L, K, r, buf, rows, nrow, recv))
    s_ms, s_med = time_steps(torch, runs, 3, args.steps)
    bs = 4 * L * nrow * r * 4 + 2 * L * nrow * 4
    out["codebook_sync"] = {"rows_per_round": nrow, "parts": parts, "median_us": s_med * 1e3,
                            "bytes_moved": bs, "roofline_us": bs / PEAK_HBM * 1e6,
                            "roofline_frac": bs / PEAK_HBM / (s_med * 1e-3),
                            "bytes_on_the_wire": L * nrow * r * 4}
    return out


def spel_step_timing(torch, mapl, synth, P, dd, rr, reps):
    """(mean, median) ms of one SPEL step on P projectors [dd, rr] (seed 55)."""
    stq = synth.stiefel_inputs(None, seed=55, P=P, d=dd, r=rr, gscale=1e-3, lr=1e-2, beta=0.95, steps=1)
    Ug, Gg, Mg = (torch.from_numpy(stq[n]).cuda() for n in ("U", "G", "M"))
    w = mapl.workspace(mapl.workspace_bytes(None, mapl.CALL_STIEFEL, P, dd, rr))
    run = lambda: mapl.stiefel_step(P, dd, rr, Ug, Gg, Mg, 1e-2, 0.95, 5, 7, w)
    return time_steps(torch, run, 2, reps)


# Segments of the r x r PolarExpress iteration at the 5 / 7 schedule the
# bench runs (consecutive steps whose linear coefficients multiply to at
# most 2048): one segment each.
SPEL_SEGMENTS = {"lmo": (5,), "retraction": (7,)}


def spel_flop_split(P, dd, rr):
    """(fp32-MFMA flops, split-product flops) of one SPEL step as the library
    computes it: Eq. 4's two products and the Gram product of Y on the fp32
    matrix units; per PolarExpress segment of n steps a Gram product of its
    start (the LMO's first: of M), n polynomials, n - 1 updates
    S <- Q (S Q), n - 1 products of Q's and one d x r x r product forming X.
    Every product counted in full (the symmetric ones compute half)."""
    big, small = 2 * dd * rr * rr, 2 * rr ** 3
    f32 = 2 * big + big  # U^T G, G - U sym(S), Y^T Y
    split = 0
    for name, segs in SPEL_SEGMENTS.items():
        for k, n in enumerate(segs):
            gram = 0 if (name == "retraction" and k == 0) else big  # Y^T Y is the fp32 one
            split += gram + n * small + (n - 1) * 2 * small + (n - 1) * small + big
    return P * f32, P * split


def spel_flops(P, dd, rr):
    return sum(spel_flop_split(P, dd, rr))


def spel_roofline_s(P, dd, rr):
    """The fp32 products at the fp32 matrix peak; the split products as three
    fp16 products per flop at the 16-bit matrix peak (fp16 and bf16 dense
    peaks are equal)."""
    f32, split = spel_flop_split(P, dd, rr)
    return f32 / PEAK_F32 + split * 3 / PEAK_BF16


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="headline from the chain replayed as one HIP graph (default: eager calls; both are "
                         "reported)")
    ap.add_argument("--no-extra", action="store_true",
                    help="only the c4 headline (no stress, per-config or SPEL blocks)")
    ap.add_argument("--spel-only", action="store_true",
                    help="only the SPEL step (16 projectors [2048,512]): one JSON line, for profiling")
    ap.add_argument("--codebooks", choices=("official", "stress"), default="official",
                    help="codebooks of the headline chain: the workload's own (default), or data-drawn ones "
                         "(every code in use; for profiling the RVQ's second pass and rescoring)")
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
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    if args.spel_only:
        ms_, med_ = spel_step_timing(torch, mapl, synth, 16, 2048, 512, args.steps)
        print(json.dumps({"config": "SPEL step, 16 projectors [2048,512], PolarExpress 5 + 7 steps",
                          "ms_per_step": ms_, "median_ms_per_step": med_,
                          "roofline_ms": spel_roofline_s(16, 2048, 512) * 1e3,
                          "roofline_frac": spel_roofline_s(16, 2048, 512) / (med_ * 1e-3)}))
        return
    log("generating workload c4")
    x = synth.codec_inputs("c4")
    T, d, r, V, k, L, K = (x[n] for n in ("T", "d", "r", "V", "k", "L", "K"))
    C_head = x["C"] if args.codebooks == "official" else library_stress_codebooks(torch, mapl, x)
    ch = Chain(torch, mapl, x, C_head)
    calls = ["encode", "decode", "decode_bwd", "encode_bwd"]

    # ---- the c4 headline: every c4 chain with the official codebooks runs
    # first (eager, then graph replays, then the traced pass), so that a
    # profiler can name the library's dispatches by position
    log("timing %d eager steps" % args.steps)
    eager_ms, eager_med = time_steps(torch, ch.step, args.warmup, args.steps)
    log("capturing the chain and timing %d graph replays" % args.steps)
    g = ch.capture()
    graph_ms, graph_med = time_steps(torch, g.replay, args.warmup, args.steps)
    ms, med = (graph_ms, graph_med) if args.graph else (eager_ms, eager_med)
    value = T / (ms * 1e-3)

    # per-call times (events between calls) and per-kernel times (library
    # trace: HIP events around each launch on its stream), eager
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    mapl.profile(True)
    for i in range(args.steps):
        ch.step(evs[i])
    torch.cuda.synchronize()
    mapl.profile(False)
    prof = mapl.profile_report()
    per_call = {c: float(np.median([e[i].elapsed_time(e[i + 1]) for e in evs])) * 1e3 for i, c in enumerate(calls)}
    chain_runs = 2 * args.warmup + 4 * args.steps + 2 + args.steps  # eager, capture warm-up, graph, traced

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
    del g

    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "1B-shaped boundary (c4): T=32768 tokens (16x2048), d=2048, r=256, "
                               "anchor k=128 over V=32000 (Zipf 1.1 ids), RVQ L=2 x K=1024, u16 codes, "
                               "ambient anchor, enc+dec fwd+bwd per step, %s%s" %
                               ("the 4-call chain replayed as one HIP graph" if args.graph else "eager calls",
                                "" if args.codebooks == "official" else ", data-drawn codebooks"),
                   "global_batch": T, "seq_len": 2048, "parallelism": "none (1 GPU)"},
        "roofline": roof,
        "median_ms_per_step": med,
        "eager_ms_per_step": eager_ms, "eager_median_ms_per_step": eager_med,
        "graph_ms_per_step": graph_ms, "graph_median_ms_per_step": graph_med,
        "chain_roofline": roofline_of(x, ms),
        "per_call_us": per_call,
        "per_kernel_us": {n: round(v[1], 2) for n, v in sorted(kern.items())},
        "kernel_order": list(kern),
        "c4_chain_runs": chain_runs,
    }

    if not args.no_extra:
        # ---- c4 with data-drawn codebooks: every code in use, so the encoder
        # rescoring (and, where needed, second screening passes) run
        log("c4 with data-drawn codebooks")
        Cs = library_stress_codebooks(torch, mapl, x)
        chs = Chain(torch, mapl, x, Cs)
        s_ms, s_med = time_steps(torch, chs.step, args.warmup, args.steps)
        # kernel times from an events-only traced pass, then the decision
        # counters from a separate pass (counting adds atomics and a sync)
        mapl.profile(1)
        for i in range(10):
            chs.step()
        torch.cuda.synchronize()
        mapl.profile(0)
        sp = mapl.profile_report()
        enc_us = sp["enc:gemm_rvq"][1] / sp["enc:gemm_rvq"][0] * 1e3 if "enc:gemm_rvq" in sp else None
        mapl.profile(2)
        for i in range(5):
            chs.step()
        torch.cuda.synchronize()
        mapl.profile(0)
        st = {n: v[0] for n, v in mapl.profile_report().items() if n.startswith("rvq:")}
        out["stress"] = {
            "codebooks": "codeword 0 = 0; round 0: projected tokens (the library's own L=0 encode of the first "
                         "8192 tokens, seed 104); round 1: 0.3 x projected tokens",
            "tokens_per_s": T / (s_ms * 1e-3), "ms_per_step": s_ms, "median_ms_per_step": s_med,
            "workload": "as the headline, eager calls",
            "chain_roofline_frac": roofline_of(x, s_ms)["frac"],
            "enc_gemm_rvq_us": enc_us,
            "encode_vs_headline": (enc_us / kern["enc:gemm_rvq"][1]) if enc_us and "enc:gemm_rvq" in kern else None,
            "rvq_tokens_rescored_frac": st.get("rvq:tokens_rescored", 0) / (5.0 * T * L),
            "rvq_candidates_per_rescored_token": st.get("rvq:candidates", 0) / max(1, st.get("rvq:tokens_rescored", 0)),
            "rvq_second_pass_frac": st.get("rvq:second_pass_blocks", 0) / max(1, st.get("rvq:blocks", 0)),
            "rvq_list_overflows": st.get("rvq:list_overflows", 0),
        }
        del chs

        # ---- the other workloads: tokens/s and chain roofline (graph replay),
        # the oracle beside each on the host
        out["configs"] = {}
        for name in ["c1", "c2_r64", "c2_r128", "c2_r256", "c2_r512", "c3", "c6"]:
            log("workload", name)
            xc = synth.codec_inputs(name)
            cc = Chain(torch, mapl, xc, xc["C"])
            c_ms, c_med = time_steps(torch, cc.step, args.warmup, args.steps)
            gc = cc.capture()
            g_ms, g_med = time_steps(torch, gc.replay, args.warmup, args.steps)
            del gc
            c_med = min(c_med, g_med)
            rf = roofline_of(xc, c_med)
            blk = {"T": xc["T"], "d": xc["d"], "r": xc["r"], "k": xc["k"], "L": xc["L"], "K": xc["K"],
                   "group_dim": xc.get("group_dim", 0),
                   "dtype": xc["dtype"], "tokens_per_s": xc["T"] / (c_med * 1e-3), "median_ms_per_step": c_med,
                   "mean_ms_per_step": c_ms, "graph_median_ms_per_step": g_med,
                   "chain_roofline_frac": rf["frac"], "roofline_us": rf["roofline_us"],
                   "bound_per_call": rf["bound_per_call"]}
            if xc.get("group_dim", 0):
                # the grouped quantiser alone: vector-ALU work against the fp32 vector peak
                mapl.profile(1)
                for _ in range(10):
                    cc.step()
                torch.cuda.synchronize()
                mapl.profile(0)
                kp = mapl.profile_report()
                if "enc:grvq" in kp:
                    us = kp["enc:grvq"][1] / kp["enc:grvq"][0] * 1e3
                    fa = GROUP_DIST_FLOPS * xc["T"] * xc["L"] * (xc["r"] // 2) * xc["K"]
                    blk["grvq_kernel"] = {"bound": "alu", "avg_us": us, "achieved": fa / (us * 1e-6) / 1e12,
                                          "peak": PEAK_F32 / 1e12, "unit": "TFLOP/s",
                                          "frac": fa / (us * 1e-6) / PEAK_F32,
                                          "per_kernel_us": {n: round(v[1] / v[0] * 1e3, 2) for n, v in kp.items()}}
            if not args.no_cpu_baseline:
                blk["cpu_baseline"] = cpu_baseline(xc, budget_s=4.0)
            out["configs"][name] = blk
            del cc

        # ---- the rows beside the chain, at the c4 widths
        log("gradient quantisation, anchor-table gradient, codebook sync")
        out["next"] = next_rows(torch, mapl, x, Cs, args)

        # ---- SPEL step: its own configuration (16 x [2048,512]) and this
        # boundary's projector
        log("SPEL step")
        spel_c5, spel_c5_med = spel_step_timing(torch, mapl, synth, 16, 2048, 512, 10)
        spel_b, _ = spel_step_timing(torch, mapl, synth, 1, d, r, 20)
        out["spel"] = {"config": "16 projectors [2048,512], PolarExpress 5 + 7 steps", "ms_per_step": spel_c5,
                       "median_ms_per_step": spel_c5_med,
                       "tflops": spel_flops(16, 2048, 512) / (spel_c5_med * 1e-3) / 1e12,
                       "roofline_ms": spel_roofline_s(16, 2048, 512) * 1e3,
                       "roofline_frac": spel_roofline_s(16, 2048, 512) / (spel_c5_med * 1e-3),
                       "boundary_projector_ms": spel_b}
        amort = 128  # micro-batches per optimizer step: global batch 512 / micro-batch 4
        out["alg1_tokens_per_s"] = T / ((ms + spel_b / amort) * 1e-3)

    if args.calib_copy:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = src.numel()
    if not args.no_cpu_baseline:
        log("timing the oracle on the host")
        out["cpu_baseline"] = cpu_baseline(x)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
