"""Benchmark of fused message passing on one MI355X.

Headline workload: the power-law CSR graph with 50M nodes and 1e9 edges
(in-degrees Zipf(2.1) capped at 1e6, uniform sources, x fp32 [N, 16], edge
weights fp32), weighted-sum forward.  One step = one call of
tiga_mp_csr_fwd: the degree plan followed by the fused gather-reduce and the
split-row merge, inputs resident in HBM.

Printed: one JSON line with GEdges/s, the roofline of the dominant kernel
(the gather-reduce, timed with HIP events on its own stream), the CPU oracle
timed on a bounded sample of the same graph, and per-path figures for the
other relations (power-law CSR sum/max forward and backward, radius forward
and backward including the cell build, dense all-pairs).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# FP32 vector issue: 256 CUs x 4 SIMDs x 16 lanes x 2 flops (FMA) x 2.4 GHz;
# packed FP32 instructions are disabled in this build.
VALU_PEAK_TFLOPS = 78.6
# the published FP32 vector peak counts packed (two-wide) FP32 instructions, which this build does not use
VALU_PACKED_PEAK_TFLOPS = 157.3


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--scale", type=float, default=1.0, help="shrink the headline graph (testing only)")
    p.add_argument("--no-paths", action="store_true", help="skip the per-path figures")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-ceilings", action="store_true", help="skip the hardware-ceiling probe")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--check-rows", type=int, default=400)
    p.add_argument("--profile-pass", nargs="?", const="csr", choices=["csr", "csr2", "radius", "dense", "attention", "knn", "edgenn"],
                   help="for rocprofv3 counter runs: csr = a 4 GiB plain copy (calibration) then 3 headline steps; "
                        "csr2 = the calibration copy, then each config-2 call (sum / max forward, atomic and gather "
                        "backward) twice; "
                        "radius / dense / attention = 3 forward calls on the radius (1M points) / dense (65536 points) / "
                        "attention (16 heads x 16384 tokens x 128, binary16, triangular) workload; knn = 3 calls on "
                        "131072 uniform points, k = 16; edgenn = 3 forward + backward calls of the edge MLP on 35947 "
                        "surface points (feat 8)")
    p.add_argument("--paths-only", action="store_true", help="only the per-path figures (for kernel traces)")
    p.add_argument("--summarize", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                   help="print the markdown summary of three rocprofv3 runs (kernel trace, FETCH_SIZE, WRITE_SIZE)")
    p.add_argument("--summarize-csr2", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="markdown summary of the FETCH_SIZE and WRITE_SIZE runs of --profile-pass csr2")
    p.add_argument("--summarize-kernels", nargs="+", metavar="DIR",
                   help="markdown table of a kernel-trace run (first DIR) and the per-kernel averages of the "
                        "counters in further --pmc run directories")
    p.add_argument("--match", default="", help="with --summarize-kernels: only kernels whose name contains this")
    return p.parse_args()


PROFILE_MD = os.path.join(ROOT, "profiles", "gather_reduce_csr_powerlaw_1b_f16.md")
CSR2_MD = os.path.join(ROOT, "profiles", "csr_powerlaw_1m_16m_f64_paths.md")
# the dominant kernel of each config-2 call, as rocprofv3 names it (template arguments: float4 units,
# 16 lanes per edge, reducer, weight mode, buffer table, non-temporal, fused edge gradient)
CSR2_KERNELS = {
    "sum_fwd": "gather_reduce_kernel<4, 16, 0, 1, true, false, false>",
    "max_fwd": "gather_reduce_kernel<4, 16, 1, 1, true, false, false>",
    "sum_bwd_atomic": "edge_kernel<4, 16, 0, true, true>",
    "max_bwd_atomic": "edge_kernel<4, 16, 1, true, true>",
    "sum_bwd_gather": "gather_reduce_kernel<4, 16, 0, 2, true, false, true>",
    "max_bwd_gather": "gather_reduce_kernel<4, 16, 0, 3, true, false, true>",
}
CSR_SOURCES = ["include/tiga_mp.h", "paper_2609_24802_amd/csrc/common.hpp", "paper_2609_24802_amd/csrc/csr_common.hpp",
               "paper_2609_24802_amd/csrc/csr_fwd.hpp", "paper_2609_24802_amd/csrc/csr_fwd.hip",
               "paper_2609_24802_amd/csrc/csr_plan.hip", "paper_2609_24802_amd/csrc/csr_bwd.hpp",
               "paper_2609_24802_amd/csrc/csr_bwd.hip", "paper_2609_24802_amd/csrc/csr_util.hip"]
VALU_LANE_OPS_PER_S = 256 * 4 * 16 * 2.4e9  # CUs * SIMDs * lanes per cycle * clock
VALU_INSTR_PER_PAIR = 12
MFMA16_PEAK_TFLOPS = 2500.0  # dense fp16 / bf16 MFMA peak
# edges per page of the paged CSR forward on the headline graph
PAGE_EDGES = 1 << 26
# input widths of the edge-MLP workload (the first is profiled)
EDGENN_FEATS = [8, 32]
# exact kNN workload sizes (the largest is profiled)
KNN_SIZES = [1024, 16384, 131072]
# (tokens, heads, width, dtype, relation); the first is the profiled attention workload
ATTENTION_CASES = [(16384, 16, 128, "f16", "triangular"), (16384, 16, 64, "f16", "triangular"),
                   (16384, 16, 128, "bf16", "dense")]
KERNEL_KEY = "gather_reduce_kernel"
COPY_BYTES = 1 << 32


# The translation unit of the gather-reduce kernel (and the plan it consumes).
KERNEL_SOURCES = ["include/tiga_mp.h", "paper_2609_24802_amd/csrc/common.hpp",
                  "paper_2609_24802_amd/csrc/csr_common.hpp", "paper_2609_24802_amd/csrc/csr_fwd.hpp",
                  "paper_2609_24802_amd/csrc/csr_fwd.hip", "paper_2609_24802_amd/csrc/csr_plan.hip"]


def source_hash(files=None):
    """sha256 over the sources of the gather-reduce kernel (or of `files`): a committed counter summary
    applies only to the kernel it measured."""
    import hashlib
    h = hashlib.sha256()
    for f in files or KERNEL_SOURCES:
        h.update(os.path.basename(f).encode())
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def committed_csr2_bytes():
    """Per-dispatch memory-side bytes (calibrated FETCH_SIZE + WRITE_SIZE: what the L2s read from and write
    to the memory side, i.e. the 256 MB memory-side cache in front of HBM, so an upper bound on HBM traffic)
    of each config-2 call's dominant kernel, from the committed summary, if the CSR sources are unchanged
    since it was taken."""
    if not os.path.exists(CSR2_MD):
        return None
    vals = {}
    for line in open(CSR2_MD):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].strip().split(": ", 1)
            vals[k.strip("` ")] = v.strip("` ")
    if vals.get("csr_source_hash") != source_hash(CSR_SOURCES) or "memside_bytes_per_dispatch" not in vals:
        return None
    try:
        return json.loads(vals["memside_bytes_per_dispatch"])
    except ValueError:
        return None


def committed_traffic():
    """Per-launch HBM bytes of the gather-reduce kernel from the committed summary, if still current."""
    if not os.path.exists(PROFILE_MD):
        return None
    vals = {}
    for line in open(PROFILE_MD):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].strip().split(": ", 1)
            vals[k.strip("` ")] = v.strip("` ")
    if vals.get("source_hash") != source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _db(d):
    import glob
    import sqlite3
    fs = glob.glob(os.path.join(d, "**", "*_results.db"), recursive=True)
    if not fs:
        raise SystemExit(f"no rocprofv3 database under {d}")
    return sqlite3.connect(fs[0])


def summarize(trace_dir, fetch_dir, write_dir):
    """Markdown summary: per-kernel durations and the scaled HBM traffic of the dominant kernel."""
    cur = _db(trace_dir).cursor()
    rows = cur.execute("select name, duration from kernels").fetchall()
    agg = {}
    for name, dur in rows:
        a = agg.setdefault(name, [0, 0.0])
        a[0] += 1
        a[1] += dur
    out = ["| kernel | calls | total ms | avg ms |", "|---|---|---|---|"]
    for name, (n, d) in sorted(agg.items(), key=lambda kv: -kv[1][1])[:8]:
        out.append(f"| `{name[:90]}` | {n} | {d / 1e6:.3f} | {d / n / 1e6:.4f} |")
    dom = [(n, d) for name, (n, d) in agg.items() if KERNEL_KEY in name]
    avg_ms = dom[0][1] / dom[0][0] / 1e6 if dom else float("nan")

    def counter(d, cname):
        c = _db(d).cursor()
        vals = c.execute("select kernel_name, value from counters_collection where counter_name = ?",
                         (cname,)).fetchall()
        copy = [v for k, v in vals if "copy" in k.lower() or "elementwise" in k.lower()]
        kern = [v for k, v in vals if KERNEL_KEY in k]
        return (max(copy) if copy else float("nan")), (sum(kern) / len(kern) if kern else float("nan"))

    fcopy, fk = counter(fetch_dir, "FETCH_SIZE")
    wcopy, wk = counter(write_dir, "WRITE_SIZE")
    fscale = COPY_BYTES / (fcopy * 1024)
    wscale = COPY_BYTES / (wcopy * 1024)
    fetch_b = fk * 1024 * fscale
    write_b = wk * 1024 * wscale
    out += [
        "",
        f"- kernel_avg_ms: {avg_ms:.4f}",
        f"- copy_calibration: a {COPY_BYTES} B device copy reads FETCH_SIZE {fcopy:.1f} KiB "
        f"(scale {fscale:.3f}) and WRITE_SIZE {wcopy:.1f} KiB (scale {wscale:.3f})",
        f"- fetch_bytes_per_launch: {fetch_b:.4g}",
        f"- write_bytes_per_launch: {write_b:.4g}",
        f"- hbm_bytes_per_launch: {fetch_b + write_b:.6g}",
        f"- source_hash: {source_hash()}",
    ]
    print("\n".join(out))


def summarize_csr2(fetch_dir, write_dir):
    """Calibrated HBM bytes per dispatch of the config-2 calls' dominant kernels (--profile-pass csr2)."""
    def per_kernel(d, cname):
        c = _db(d).cursor()
        vals = c.execute("select kernel_name, value from counters_collection where counter_name = ?",
                         (cname,)).fetchall()
        copy = [v for k, v in vals if "copy" in k.lower() or "elementwise" in k.lower()]
        out = {}
        for case, key in CSR2_KERNELS.items():
            got = [v for k, v in vals if key in k]
            out[case] = sum(got) / len(got) if got else float("nan")
        return (max(copy) if copy else float("nan")), out
    fcopy, fk = per_kernel(fetch_dir, "FETCH_SIZE")
    wcopy, wk = per_kernel(write_dir, "WRITE_SIZE")
    fscale = COPY_BYTES / (fcopy * 1024)
    wscale = COPY_BYTES / (wcopy * 1024)
    rows = ["| call | dominant kernel | FETCH bytes | WRITE bytes |", "|---|---|---|---|"]
    total = {}
    for case, key in CSR2_KERNELS.items():
        fb, wb = fk[case] * 1024 * fscale, wk[case] * 1024 * wscale
        total[case] = fb + wb
        rows.append(f"| {case} | `{key}` | {fb:.4g} | {wb:.4g} |")
    rows += ["",
             f"- copy_calibration: a {COPY_BYTES} B device copy reads FETCH_SIZE {fcopy:.1f} KiB (scale {fscale:.3f}) "
             f"and WRITE_SIZE {wcopy:.1f} KiB (scale {wscale:.3f})",
             f"- memside_bytes_per_dispatch: {json.dumps({k: round(v) for k, v in total.items()})}",
             f"- csr_source_hash: {source_hash(CSR_SOURCES)}"]
    print("\n".join(rows))


def summarize_kernels(dirs, match):
    """Markdown: kernel durations of a trace run, then per-kernel counter averages of --pmc runs."""
    cur = _db(dirs[0]).cursor()
    agg = {}
    for name, dur in cur.execute("select name, duration from kernels").fetchall():
        if match in name:
            a = agg.setdefault(name, [0, 0.0])
            a[0] += 1
            a[1] += dur
    out = ["| kernel | calls | total ms | avg ms |", "|---|---|---|---|"]
    for name, (n, d) in sorted(agg.items(), key=lambda kv: -kv[1][1])[:16]:
        out.append(f"| `{name[:110]}` | {n} | {d / 1e6:.3f} | {d / n / 1e6:.4f} |")
    for d in dirs[1:]:
        c = _db(d).cursor()
        per = {}
        for k, cn, v in c.execute("select kernel_name, counter_name, value from counters_collection").fetchall():
            if match in k:
                per.setdefault(k, {}).setdefault(cn, []).append(v)
        if not per:
            continue
        names = sorted({cn for v in per.values() for cn in v})
        out += ["", f"Counters ({os.path.basename(os.path.normpath(d))}), mean per dispatch:", "",
                "| kernel | " + " | ".join(names) + " |", "|---" * (len(names) + 1) + "|"]
        for k, v in sorted(per.items()):
            cells = [f"{sum(v[cn]) / len(v[cn]):.4g}" if cn in v else "" for cn in names]
            out.append(f"| `{k[:70]}` | " + " | ".join(cells) + " |")
    print("\n".join(out))


class Timer:
    """HIP events around the dominant kernel of each call, plus whole-step events."""

    def __init__(self, torch, tb, steps):
        self.torch, self.tb = torch, tb
        self.k = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        s = torch.cuda.current_stream()
        for a, b in self.k:  # materialize the underlying hipEvents
            a.record(s)
            b.record(s)
        torch.cuda.synchronize()

    def arm(self, i):
        a, b = self.k[i]
        self.tb.tiga_mp_set_kernel_events(a, b)

    def kernel_ms(self):
        return [a.elapsed_time(b) for a, b in self.k]


def time_steps(torch, tb, fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    tm = Timer(torch, tb, steps)
    s0 = torch.cuda.Event(enable_timing=True)
    s1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    s0.record()
    for i in range(steps):
        tm.arm(i)
        fn()
    s1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    return dict(step_ms=s0.elapsed_time(s1) / steps, wall_ms=wall / steps, kernel_ms=tm.kernel_ms())


def headline(args, torch, tb, synth, oracle):
    t = time.time()
    g = synth.config5(scale=args.scale)
    rp, col, x, w, n = g["row_ptr"], g["col"], g["x"], g["w"], g["num_dst"]
    E, F = int(rp[-1]), x.shape[1]
    log(f"generated {n} nodes / {E} edges in {time.time() - t:.1f} s")
    dev = lambda a: torch.from_numpy(a).cuda()
    rel = tb.Csr(dev(rp), dev(col), n)
    xd, wd = dev(x), dev(w)
    y = torch.empty(n, F, dtype=torch.float32, device="cuda")
    ws = torch.empty(tb.load().tiga_mp_csr_fwd_workspace(rel.ref, F, tb.REDUCE_SUM), dtype=torch.uint8,
                     device="cuda")
    torch.cuda.synchronize()
    log("inputs resident on the device")

    fn = lambda: tb.tiga_mp_csr_fwd(rel, xd, wd, y=y, ws=ws)
    r = time_steps(torch, tb, fn, args.steps, args.warmup)
    log(f"step {r['step_ms']:.3f} ms, gather-reduce {np.mean(r['kernel_ms']):.3f} ms")

    # sampled parity of what was timed
    deg = np.diff(rp)
    rows = np.unique(np.concatenate([np.argsort(-deg, kind="stable")[:4],
                                     np.random.default_rng(1).integers(0, n, args.check_rows)]))
    yh = y[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    ref, mag = oracle.csr_sum_fwd(rp, col, x, w, rows=rows)
    parity_ok = bool(np.all(np.abs(yh - ref) <= 1e-5 * mag))
    log(f"sampled parity ({rows.size} rows): {'ok' if parity_ok else 'FAILED'}")

    kernel_ms = float(np.mean(r["kernel_ms"]))
    bytes_alg = E * (4 + 4 + 4 * F) + n * (8 + 4 * F)
    achieved = bytes_alg / (kernel_ms * 1e-3) / 1e9
    out = dict(E=E, n=n, F=F, step_ms=r["step_ms"], kernel_ms=kernel_ms, bytes_alg=bytes_alg,
               achieved=achieved, parity_ok=parity_ok, kernel_ms_all=r["kernel_ms"])

    if not args.no_paths:
        # the paged forward on the same graph: relation and weights in pinned host memory, staged in
        # pages of whole rows through a bounded device workspace (x and y stay resident)
        del rel, wd, ws
        torch.cuda.empty_cache()
        t = time.time()
        rel_h = tb.HostCsr(torch.from_numpy(rp).pin_memory(), torch.from_numpy(col).pin_memory(), n)
        w_h = torch.from_numpy(w).pin_memory()
        log(f"relation pinned in host memory in {time.time() - t:.1f} s")
        wsp = tb._workspace(tb.load().tiga_mp_csr_fwd_paged_workspace(F, tb.REDUCE_SUM, PAGE_EDGES), xd.device)
        yp = {}
        rp_ = time_steps(torch, tb, lambda: yp.update(y=tb.tiga_mp_csr_fwd_paged(
            rel_h, xd, w_h, page_edges=PAGE_EDGES, ws=wsp)[0]), 2, 1)
        copied = E * 8 + (n + 1) * 8 + (E // PAGE_EDGES + 1) * 8
        out["paged"] = dict(ms=rp_["step_ms"], gedges_per_s=E / rp_["step_ms"] / 1e6, page_edges=PAGE_EDGES,
                            device_ws_bytes=int(wsp.numel()), host_to_device_gbs=copied / rp_["step_ms"] / 1e6,
                            equal_to_resident=bool(torch.equal(yp["y"], y)))
        log(f"paged: {rp_['step_ms']:.1f} ms, equal to resident: {out['paged']['equal_to_resident']}")
        del rel_h, w_h, wsp, yp
    else:
        del rel, wd, ws
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(args, oracle, rp, col, x, w)
    del xd, y
    torch.cuda.empty_cache()
    return out, cpu


def host_cpu():
    """The host the CPU baseline runs on: usable cores (this process's affinity; nproc), logical CPUs of
    the machine and the processor model (/proc/cpuinfo, what lscpu reports as the model name)."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.lower().startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count()
    return dict(nproc=nproc, logical_cpus=os.cpu_count(), model=model)


def cpu_baseline(args, oracle, rp, col, x, w):
    """The oracle (untuned, fp64) on the first rows of the same graph."""
    n = rp.size - 1
    # grow the sample until it takes a measurable time, then size it for about cpu_seconds
    edges = 2_000_000
    while True:
        k = max(1, min(int(np.searchsorted(rp, edges)), n))
        t = time.perf_counter()
        oracle.csr_sum_fwd(rp, col, x, w, rows=np.arange(k))
        dt = time.perf_counter() - t
        if dt > 0.5 or k == n:
            break
        edges *= 4
    rate = (rp[k] - rp[0]) / max(dt, 1e-6)
    k = max(1, min(int(np.searchsorted(rp, int(rate * args.cpu_seconds))), n))
    rows = np.arange(k)
    t = time.perf_counter()
    oracle.csr_sum_fwd(rp, col, x, w, rows=rows)
    dt = time.perf_counter() - t
    edges = int(rp[k] - rp[0])
    log(f"cpu oracle: {edges} edges in {dt:.2f} s on {oracle.threads()} threads")
    hc = host_cpu()
    return dict(value=edges / dt / 1e9, unit="GEdges/s", cores=oracle.threads(), kind="oracle",
                sample=f"weighted-sum forward of rows [0, {k}) of the 1e9-edge graph ({edges} edges), "
                       f"fp64 accumulation, {dt:.1f} s",
                threads=oracle.threads(), nproc=hc["nproc"], logical_cpus=hc["logical_cpus"], cpu_model=hc["model"])


def cpu_baseline_config1(oracle, synth):
    """The oracle on config 1 (weighted-sum forward and backward, 1,024 nodes, 8,192 edges), single-
    threaded and on all host threads: one warmup, then the median of three calls."""
    g = synth.csr_uniform_small()
    rp, col, x, w, dy = g["row_ptr"], g["col"], g["x"], g["w"], g["dy"]

    def once():
        oracle.csr_sum_fwd(rp, col, x, w)
        oracle.csr_sum_bwd(rp, col, x, w, dy, g["num_src"])

    out = {}
    for label, nt in (("single_thread", 1), ("all_threads", 0)):
        oracle.set_threads(nt)
        once()
        ts = []
        for _ in range(3):
            t = time.perf_counter()
            once()
            ts.append(time.perf_counter() - t)
        out[f"{label}_us"] = sorted(ts)[1] * 1e6
        out[f"{label}_threads"] = oracle.threads()
    oracle.set_threads(0)
    hc = host_cpu()
    out.update(kind="oracle", sample="config 1 weighted-sum forward + backward (dx, dw), fp64 accumulation",
               nproc=hc["nproc"], cpu_model=hc["model"])
    log(f"cpu oracle config 1: {out['single_thread_us']:.0f} us on 1 thread, {out['all_threads_us']:.0f} us "
        f"on {out['all_threads_threads']}")
    return out


def radius_candidate_tests(pos, radius, max_cells=None):
    """(destination, candidate) predicate tests the radius consume kernel performs: every point of a cell
    is tested against every point of the 27 cells around it.  The cell grid is the library's own recipe
    (cells of h = max(r (1 + 2^-10), cbrt(box volume / n)), grown by 1.25 until at most n + 64 cells),
    replayed here in fp64 for reporting only."""
    n = pos.shape[0]
    max_cells = max_cells or n + 64
    lo = pos.min(0).astype(np.float64)
    ext = np.maximum(pos.max(0).astype(np.float64) - lo, 0.0)
    h = max(float(radius) * (1.0 + 1.0 / 1024.0), float(np.cbrt(np.prod(ext) / max(n, 1))))
    while True:
        dims = (np.floor(ext / h) + 1.0).astype(np.int64)
        if np.prod(dims.astype(np.float64)) <= max_cells:
            break
        h *= 1.25
    inv = 1.0 / h
    c = np.clip(np.floor((pos.astype(np.float64) - lo) * inv), 0, dims - 1).astype(np.int64)
    cnt = np.zeros(tuple(dims[::-1]), np.int64)
    np.add.at(cnt, (c[:, 2], c[:, 1], c[:, 0]), 1)
    nb = np.zeros_like(cnt)
    pad = np.pad(cnt, 1)
    for dz in range(3):
        for dy in range(3):
            for dx in range(3):
                nb += pad[dz:dz + dims[2], dy:dy + dims[1], dx:dx + dims[0]]
    return int((cnt * nb).sum())


def paths(args, torch, tb, synth):
    """Per-path figures on the other workloads (each timed with HIP events)."""
    res = {}
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    steps, warm = max(5, args.steps // 2), 2

    # config 1 (1,024 nodes, 8,192 uniform edges, F = 16): bound by launch latency (0.66 MB of traffic
    # is 83 ns at the HBM peak), so the figure is microseconds per call, from HIP events and from the
    # host clock (launch overhead included)
    g = synth.csr_uniform_small()
    rp1, col1 = g["row_ptr"], g["col"]
    E1 = int(rp1[-1])
    rel1 = tb.Csr(dev(rp1), dev(col1), g["num_dst"])
    x1, w1, dy1 = dev(g["x"]), dev(g["w"]), dev(g["dy"])
    rev1 = tb.tiga_csr_transpose(rel1)
    c1 = {"sum_fwd": lambda: tb.tiga_mp_csr_fwd(rel1, x1, w1),
          "sum_bwd_gather": lambda: tb.tiga_mp_csr_bwd(rel1, dy1, x1, w1, rev=rev1),
          "sum_fwd_bwd": lambda: (tb.tiga_mp_csr_fwd(rel1, x1, w1), tb.tiga_mp_csr_bwd(rel1, dy1, x1, w1, rev=rev1))}
    for key, fn in c1.items():
        r = time_steps(torch, tb, fn, 200, 20)
        res[f"csr_uniform_1024n_8192e_f16_{key}"] = dict(us_per_call=r["step_ms"] * 1e3,
                                                        wall_us_per_call=r["wall_ms"] * 1e3,
                                                        gedges_per_s=E1 / r["step_ms"] / 1e6)
        log(f"config 1 {key}: {r['step_ms'] * 1e3:.1f} us")
    # the same forward + backward captured once in a HIP graph and replayed: the launch-bound step
    # without the per-call host work (the library issues fill kernels, not memsets, and never syncs)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(3):
            c1["sum_fwd_bwd"]()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        c1["sum_fwd_bwd"]()
    for _ in range(20):
        graph.replay()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(200):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / 200 * 1e3
    res["csr_uniform_1024n_8192e_f16_sum_fwd_bwd_graph_replay"] = dict(us_per_call=us, gedges_per_s=E1 / us / 1e3)
    log(f"config 1 fwd+bwd graph replay: {us:.1f} us")
    del rel1, x1, w1, dy1, rev1, graph

    # the paper's own latency workloads on this path: stored CSR, weighted neighbour sum, degree 32,
    # F = 32 at 8,192 / 32,768 / 131,072 nodes, forward; and the generated radius relation (scalar
    # distance-weighted sum, nominal degree 32, 131,072 uniform points, rebuilt every call), forward
    for nn in (8192, 32768, 131072):
        g = synth.csr_fixed_degree(nn, 32, 32)
        relp = tb.Csr(dev(g["row_ptr"]), dev(g["col"]), nn)
        xp, wp = dev(g["x"]), dev(g["w"])
        r = time_steps(torch, tb, lambda: tb.tiga_mp_csr_fwd(relp, xp, wp), 50, 5)
        res[f"csr_degree32_{nn}n_f32_sum_fwd"] = dict(ms=r["step_ms"], gedges_per_s=nn * 32 / r["step_ms"] / 1e6)
        log(f"degree-32 CSR {nn}: {r['step_ms']:.4f} ms")
        del relp, xp, wp
    nr = 131072
    posr = dev(synth.uniform_f32(nr * 3, 0.0, 1.0, (10, 0)).reshape(nr, 3))
    xr = dev(synth.normal_f32(nr, (10, 1)).reshape(nr, 1))
    rr_ = synth.radius_for_mean_degree(nr)
    _, cntr = tb.tiga_mp_radius_fwd(posr, xr, rr_, np.float32(rr_ / np.float32(2)))
    pairs_r = int(cntr.long().sum().item())
    r = time_steps(torch, tb, lambda: tb.tiga_mp_radius_fwd(posr, xr, rr_, np.float32(rr_ / np.float32(2)),
                                                            want_count=False), 50, 5)
    res["radius_131072_f1_fwd_with_build"] = dict(ms=r["step_ms"], accepted_pairs=pairs_r,
                                                  gedges_per_s=pairs_r / r["step_ms"] / 1e6)
    log(f"radius 131072 F=1: {r['step_ms']:.4f} ms")
    del posr, xr, cntr

    g = synth.config2()
    rp, col, n = g["row_ptr"], g["col"], g["num_dst"]
    E = int(rp[-1])
    rel = tb.Csr(dev(rp), dev(col), n)
    xd, wd, dyd = dev(g["x"]), dev(g["w"]), dev(g["dy"])
    F = xd.shape[1]
    rev = tb.tiga_csr_transpose(rel)
    _, am = tb.tiga_mp_csr_fwd(rel, xd, wd, reducer=tb.REDUCE_MAX)
    cases = {
        "csr_powerlaw_1m_16m_f64_sum_fwd": lambda: tb.tiga_mp_csr_fwd(rel, xd, wd),
        "csr_powerlaw_1m_16m_f64_max_fwd": lambda: tb.tiga_mp_csr_fwd(rel, xd, wd, reducer=tb.REDUCE_MAX),
        "csr_powerlaw_1m_16m_f64_sum_bwd_atomic": lambda: tb.tiga_mp_csr_bwd(rel, dyd, xd, wd),
        "csr_powerlaw_1m_16m_f64_sum_bwd_gather": lambda: tb.tiga_mp_csr_bwd(rel, dyd, xd, wd, rev=rev),
        "csr_powerlaw_1m_16m_f64_max_bwd_atomic": lambda: tb.tiga_mp_csr_bwd(rel, dyd, xd, wd,
                                                                             reducer=tb.REDUCE_MAX, argmax=am),
        "csr_powerlaw_1m_16m_f64_max_bwd_gather": lambda: tb.tiga_mp_csr_bwd(rel, dyd, xd, wd,
                                                                             reducer=tb.REDUCE_MAX, argmax=am,
                                                                             rev=rev),
    }
    # algorithmic HBM bytes: forward = per edge (col, w, x row) + per row (row_ptr, y row [, argmax row]);
    # sum backward, atomic mode = per edge (col, w, x row for dw, dw, dy row added into dx) + dy rows + dx rows;
    # sum backward, gather mode (one traversal of the reverse incidence) = per edge (edge id, destination,
    # w, dy row, dw) + per source (src_ptr, x row, dx row)
    ns = int(g["x"].shape[0])
    alg = {"sum_fwd": E * (8 + 4 * F) + n * (8 + 4 * F),
           "max_fwd": E * (8 + 4 * F) + n * (8 + 8 * F),
           "sum_bwd_atomic": E * (12 + 8 * F) + n * (8 + 4 * F) + ns * 4 * F,
           "sum_bwd_gather": E * (16 + 4 * F) + ns * (8 + 8 * F)}
    # the reverse incidence is topology set-up (built once, reused by every gather-mode backward)
    cases["csr_powerlaw_1m_16m_f64_transpose"] = lambda: tb.tiga_csr_transpose(rel)
    dram = committed_csr2_bytes()
    for name, fn in cases.items():
        r = time_steps(torch, tb, fn, steps, warm)
        d = dict(ms=r["step_ms"], gedges_per_s=E / r["step_ms"] / 1e6)
        key = name.split("f64_")[1]
        akey = key
        if akey in alg:
            d.update(alg_bytes=alg[akey], alg_gbs=alg[akey] / r["step_ms"] / 1e6,
                     frac_hbm=alg[akey] / r["step_ms"] / 1e6 / HBM_PEAK_GBS)
        if key in CSR2_KERNELS:
            # the dominant kernel of the call (HIP events around it); its rocprofv3-measured memory-side
            # bytes (calibrated FETCH_SIZE + WRITE_SIZE per dispatch: L2 misses and write-backs, served by
            # the 256 MB memory-side cache or HBM) come from the committed summary while the CSR sources are
            # unchanged, else null
            k = float(np.mean(r["kernel_ms"]))
            d.update(kernel=CSR2_KERNELS[key], kernel_ms=k)
            if akey in alg:
                d.update(kernel_alg_gbs=alg[akey] / k / 1e6, kernel_frac_hbm=alg[akey] / k / 1e6 / HBM_PEAK_GBS)
            b = dram.get(key) if dram else None
            d.update(memside_bytes=b, memside_gbs=(b / k / 1e6) if b else None,
                     memside_frac_hbm=(b / k / 1e6 / HBM_PEAK_GBS) if b else None)
        res[name] = d
        log(f"{name}: {d['ms']:.3f} ms")
    del rel, xd, wd, dyd, rev, am
    torch.cuda.empty_cache()

    g = synth.config3()
    pd, xd, dyd = dev(g["pos"]), dev(g["x"]), dev(g["dy"])
    r, s = g["radius"], g["sigma"]
    _, cnt = tb.tiga_mp_radius_fwd(pd, xd, r, s)
    pairs = int(cnt.long().sum().item())
    npt, Fr = int(g["x"].shape[0]), int(g["x"].shape[1])
    # unique HBM bytes of the consume kernel: records, x rows, y rows (fwd); records, positions, x, dy, dx,
    # dpos rows (bwd).  Accepted pairs re-read rows from the caches, so this sits far below the HBM peak:
    # the kernel is bound by candidate tests (VALU) and gather latency instead.
    uniq = {"fwd": npt * (16 + 8 * Fr), "bwd": npt * (16 + 12 + 12 * Fr + 12)}
    tests = radius_candidate_tests(g["pos"], r)
    # useful FP32 work per accepted pair (each transcendental counted as one flop):
    #   forward: squared distance 8 (3 differences, 3 squares, 2 sums) + exponent argument 1 + exp 1
    #            + weighted accumulation 2F                                    = 2F + 10
    #   backward: squared distance 8 + argument 1 + exp 1 + dx accumulation 2F + the two inner products
    #            <dy_i, x_j> + <dy_j, x_i> 4F + their sum 1 + coefficient 2k/sigma^2 2 + 3 (mul + add) 6
    #                                                                          = 6F + 19
    # and, as scheme overhead, 8 flops per (destination, candidate) predicate test of rejected candidates
    useful = {"fwd": pairs * (2 * Fr + 10), "bwd": pairs * (6 * Fr + 19)}
    for name, fn in {"radius_1m_f32_fwd_with_build": lambda: tb.tiga_mp_radius_fwd(pd, xd, r, s, want_count=False),
                     "radius_1m_f32_bwd_with_build": lambda: tb.tiga_mp_radius_bwd(pd, xd, dyd, r, s)}.items():
        rr = time_steps(torch, tb, fn, steps, warm)
        k = float(np.mean(rr["kernel_ms"]))
        ph = "fwd" if "_fwd_" in name else "bwd"
        u = uniq[ph]
        tf = useful[ph] / (k * 1e-3) / 1e12
        res[name] = dict(ms=rr["step_ms"], gedges_per_s=pairs / rr["step_ms"] / 1e6, accepted_pairs=pairs,
                         consume_kernel_ms=k, consume_gedges_per_s=pairs / k / 1e6,
                         candidate_tests=tests, useful_flops=useful[ph], useful_tflops=tf,
                         frac_valu_packed=tf / VALU_PACKED_PEAK_TFLOPS, frac_valu=tf / VALU_PEAK_TFLOPS,
                         overhead_tflops=(tests - pairs) * 8 / (k * 1e-3) / 1e12,
                         kernel_unique_gbs=u / k / 1e6, kernel_frac_hbm=u / k / 1e6 / HBM_PEAK_GBS)
        log(f"{name}: {rr['step_ms']:.3f} ms (consume {k:.3f} ms, {tf:.1f} useful TFLOP/s)")
    del pd, xd, dyd
    g = synth.config4()
    pd, qd = dev(g["pos"]), dev(g["q"])
    nn = pd.shape[0]
    rr = time_steps(torch, tb, lambda: tb.tiga_mp_dense_fwd(pd, qd, g["eps"]), steps, warm)
    k = float(np.mean(rr["kernel_ms"]))
    tf = nn * (nn - 1) * 20 / (k * 1e-3) / 1e12
    # issue floor: 12 non-transcendental VALU instructions per pair (the reciprocal square root issues
    # alongside); a wave64 VALU instruction occupies a SIMD for 4 cycles: 1024 SIMDs * 2.4 GHz / 4 * 64 lanes.
    # The measured kernel time sits within a few per cent of this floor, on either side (clock variation).
    floor_ms = nn * (nn - 1) * VALU_INSTR_PER_PAIR / VALU_LANE_OPS_PER_S * 1e3
    res["dense_65536_fwd"] = dict(ms=rr["step_ms"], gpairs_per_s=nn * (nn - 1) / rr["step_ms"] / 1e6, kernel_ms=k,
                                  tflops_20_per_pair=tf, frac_valu=tf / VALU_PEAK_TFLOPS,
                                  valu_issue_floor_ms=floor_ms)
    log(f"dense: {rr['step_ms']:.3f} ms ({tf:.1f} TFLOP/s)")
    del pd, qd

    # edge-local MLP message on the radius relation (35,947 surface points, r = 0.015, hidden 32, 3
    # outputs): forward and its VJP (all six gradients), each rebuilding the relation
    for F in EDGENN_FEATS:
        g = synth.edgenn_inputs(feat=F)
        pd, xd, dyd = dev(g["pos"]), dev(g["x"]), dev(g["dy"])
        W = [dev(g[k]) for k in ("W1", "b1", "W2", "b2")]
        nn_, H, O = pd.shape[0], W[0].shape[0], W[2].shape[0]
        ws = tb._workspace(tb.load().tiga_mp_edgenn_workspace(nn_, F, H, O), pd.device)
        rf = time_steps(torch, tb, lambda: tb.tiga_mp_edgenn_fwd(pd, xd, g["radius"], *W, ws=ws), steps, warm)
        rb = time_steps(torch, tb, lambda: tb.tiga_mp_edgenn_bwd(pd, xd, g["radius"], *W, dyd, ws=ws), steps, warm)
        res[f"edgenn_surface_{nn_}_f{F}_h{H}_o{O}"] = dict(
            fwd_ms=rf["step_ms"], fwd_kernel_ms=float(np.mean(rf["kernel_ms"])), bwd_ms=rb["step_ms"],
            bwd_kernel_ms=float(np.mean(rb["kernel_ms"])), total_ms=rf["step_ms"] + rb["step_ms"])
        log(f"edgenn F={F}: fwd {rf['step_ms']:.3f} ms, bwd {rb['step_ms']:.3f} ms")
        del pd, xd, dyd, W, ws

    # exact kNN relation with the neighbour sum (k = 16, scalar features): the build (curve order, tile
    # boxes) plus the select-and-sum kernel; pairs = n (n - 1) ordered pairs the relation decides over
    for nk in KNN_SIZES:
        g = synth.knn_inputs(nk)
        pd, xd = dev(g["pos"]), dev(g["x"])
        ws = tb._workspace(tb.load().tiga_mp_knn_workspace(nk), pd.device)
        rr = time_steps(torch, tb, lambda: tb.tiga_mp_knn_fwd(pd, xd, g["k"], ws=ws), steps, warm)
        k = float(np.mean(rr["kernel_ms"]))
        # queries answered and (query, neighbour) pairs selected per second; the select kernel evaluates
        # only the candidates its exact box tests cannot exclude (at most about 8,800 per query at
        # 131,072 points, bounded by the scalar-load counter in the kNN profile), not all n (n - 1) pairs
        res[f"knn_{nk}_k16_f1"] = dict(ms=rr["step_ms"], select_kernel_ms=k,
                                        queries_per_s=nk / (rr["step_ms"] * 1e-3),
                                        selected_pairs_per_s=nk * g["k"] / (rr["step_ms"] * 1e-3))
        log(f"knn {nk}: {rr['step_ms']:.3f} ms (select {k:.3f} ms)")
        del pd, xd, ws

    # online-softmax reducer over the implicit triangular / dense relation (streaming attention forward):
    # 4 * width flops per admitted (query, key) pair (two products of 2 * width), against the dense
    # 16-bit MFMA peak
    for (nt, H, D, dt, rel) in ATTENTION_CASES:
        inp = synth.attention_inputs(nt, H, D, dt)
        tdt = torch.float16 if dt == "f16" else torch.bfloat16
        q, kk, v = (dev(inp[a].view(np.int16)).view(tdt) for a in ("q", "k", "v"))
        rr = time_steps(torch, tb, lambda: tb.tiga_mp_attention_fwd(q, kk, v, None, rel), steps, warm)
        k = float(np.mean(rr["kernel_ms"]))
        pairs = nt * (nt + 1) // 2 if rel == "triangular" else nt * nt
        tf = 4 * D * H * pairs / (k * 1e-3) / 1e12
        name = f"attention_{rel}_{nt}_h{H}_d{D}_{dt}"
        res[name] = dict(ms=rr["step_ms"], kernel_ms=k, pairs=pairs * H, tflops=tf, frac_mfma=tf / MFMA16_PEAK_TFLOPS)
        log(f"{name}: {k:.3f} ms ({tf:.1f} TFLOP/s)")
        del q, kk, v
    return res


def profile_pass(args, torch, tb, synth):
    """Workload for counter runs: a plain copy of known size, then three steps (csr); or three calls on one of the
    other workloads (radius: forward and backward)."""
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    if args.profile_pass == "csr2":
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1.0)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        g = synth.config2()
        rel = tb.Csr(dev(g["row_ptr"]), dev(g["col"]), g["num_dst"])
        xd, wd, dyd = dev(g["x"]), dev(g["w"]), dev(g["dy"])
        rev = tb.tiga_csr_transpose(rel)
        _, am = tb.tiga_mp_csr_fwd(rel, xd, wd, reducer=tb.REDUCE_MAX)
        for _ in range(2):
            tb.tiga_mp_csr_fwd(rel, xd, wd)
            tb.tiga_mp_csr_fwd(rel, xd, wd, reducer=tb.REDUCE_MAX)
            tb.tiga_mp_csr_bwd(rel, dyd, xd, wd)
            tb.tiga_mp_csr_bwd(rel, dyd, xd, wd, reducer=tb.REDUCE_MAX, argmax=am)
            tb.tiga_mp_csr_bwd(rel, dyd, xd, wd, rev=rev)
            tb.tiga_mp_csr_bwd(rel, dyd, xd, wd, reducer=tb.REDUCE_MAX, argmax=am, rev=rev)
        torch.cuda.synchronize()
        log("profile pass done")
        return
    if args.profile_pass == "radius":
        g = synth.config3()
        pd, xd, dyd = dev(g["pos"]), dev(g["x"]), dev(g["dy"])
        for _ in range(3):
            tb.tiga_mp_radius_fwd(pd, xd, g["radius"], g["sigma"])
            tb.tiga_mp_radius_bwd(pd, xd, dyd, g["radius"], g["sigma"])
        torch.cuda.synchronize()
        log("profile pass done")
        return
    if args.profile_pass == "edgenn":
        g = synth.edgenn_inputs(feat=EDGENN_FEATS[0])
        pd, xd, dyd = dev(g["pos"]), dev(g["x"]), dev(g["dy"])
        W = [dev(g[k]) for k in ("W1", "b1", "W2", "b2")]
        for _ in range(3):
            tb.tiga_mp_edgenn_fwd(pd, xd, g["radius"], *W)
            tb.tiga_mp_edgenn_bwd(pd, xd, g["radius"], *W, dyd)
        torch.cuda.synchronize()
        log("profile pass done")
        return
    if args.profile_pass == "knn":
        g = synth.knn_inputs(KNN_SIZES[-1])
        pd, xd = dev(g["pos"]), dev(g["x"])
        for _ in range(3):
            tb.tiga_mp_knn_fwd(pd, xd, g["k"])
        torch.cuda.synchronize()
        log("profile pass done")
        return
    if args.profile_pass == "attention":
        nt, H, D, dt, rel = ATTENTION_CASES[0]
        inp = synth.attention_inputs(nt, H, D, dt)
        q, kk, v = (dev(inp[a].view(np.int16)).view(torch.float16) for a in ("q", "k", "v"))
        for _ in range(3):
            tb.tiga_mp_attention_fwd(q, kk, v, None, rel)
        torch.cuda.synchronize()
        log("profile pass done")
        return
    if args.profile_pass == "dense":
        g = synth.config4()
        pd, qd = dev(g["pos"]), dev(g["q"])
        for _ in range(3):
            tb.tiga_mp_dense_fwd(pd, qd, g["eps"])
        torch.cuda.synchronize()
        log("profile pass done")
        return
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    g = synth.config5(scale=args.scale)
    dev = lambda a: torch.from_numpy(a).cuda()
    rel = tb.Csr(dev(g["row_ptr"]), dev(g["col"]), g["num_dst"])
    xd, wd = dev(g["x"]), dev(g["w"])
    for _ in range(3):
        tb.tiga_mp_csr_fwd(rel, xd, wd)
    torch.cuda.synchronize()
    log("profile pass done")


def ceilings():
    """Measured hardware ceilings (stream read/copy, random row gathers, VALU), from the probe binary."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2609_24802_amd", "ceilings", "tiga_ceilings")
    if not os.path.exists(exe):
        log("ceiling probe not built")
        return None
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        log(f"ceiling probe failed: {r.stderr.strip()[-200:]}")
        return None
    c = json.loads(r.stdout.strip().splitlines()[-1])
    log(f"ceilings: {c}")
    return c


def main():
    args = parse()
    if args.summarize:
        summarize(*args.summarize)
        return
    if args.summarize_kernels:
        summarize_kernels(args.summarize_kernels, args.match)
        return
    if args.summarize_csr2:
        summarize_csr2(*args.summarize_csr2)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import oracle
    from paper_2609_24802_amd import binding as tb
    from paper_2609_24802_amd import synth

    if not os.path.exists(tb.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    tb.load()
    if args.profile_pass:
        profile_pass(args, torch, tb, synth)
        return
    if args.paths_only:
        print(json.dumps(paths(args, torch, tb, synth)), flush=True)
        return
    ceil = None if args.no_ceilings else ceilings()
    h, cpu = headline(args, torch, tb, synth, oracle)
    extra = {} if args.no_paths else paths(args, torch, tb, synth)
    if "paged" in h:
        extra[f"csr_paged_host_relation_{h['n']}n_{h['E']}e_f{h['F']}"] = h["paged"]
    if not args.no_paths and not args.no_cpu:
        extra["csr_uniform_1024n_8192e_f16_cpu_oracle"] = cpu_baseline_config1(oracle, synth)
    value = h["E"] / (h["step_ms"] * 1e-3) / 1e9
    line = {
        "metric": "GEdges/s fused fwd(+bwd) and achieved HBM GB/s vs peak, 1 MI355X",
        "value": value,
        "unit": "GEdges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["step_ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded power-law CSR, Zipf(2.1) in-degrees, uniform sources)",
        "config": {"workload": f"csr_powerlaw_{h['n']}n_{h['E']}e_f{h['F']}_sum_fwd", "num_nodes": h["n"],
                   "num_edges": h["E"], "feat": h["F"], "reducer": "sum", "message": "w_e * x_src",
                   "scale": args.scale},
        "roofline": {"bound": "hbm", "achieved": h["achieved"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": h["achieved"] / HBM_PEAK_GBS, "traffic": committed_traffic(),
                     "kernel": "gather_reduce_kernel", "kernel_ms": h["kernel_ms"],
                     "kernel_ms_median": float(np.median(h["kernel_ms_all"])),
                     "kernel_ms_range": [float(np.min(h["kernel_ms_all"])), float(np.max(h["kernel_ms_all"]))],
                     "bytes_per_launch": h["bytes_alg"],
                     "frac_of_measured_gather_ceiling": (h["E"] / (h["kernel_ms"] * 1e-3)) / ceil["gather64_rows_per_s"]
                     if ceil else None,
                     "target_frac": 0.60, "target_met": bool(h["achieved"] / HBM_PEAK_GBS >= 0.60)},
        "cpu_baseline": cpu,
        "ceilings": ceil,
        "parity_sampled": h["parity_ok"],
        "paths": extra,
    }
    print(json.dumps(line), flush=True)
    if not h["parity_ok"]:
        log("sampled parity of the timed result FAILED")
        sys.exit(1)


if __name__ == "__main__":
    main()
