"""Benchmark of the DORA deployment hot path on one MI355X.

One step = one pass of the whole path over one batch:
    dora_select_pack_plan     (top-k with CLS pinned + cu_seqlens + packed
                               gather, and the attention work queue of the
                               packed layout, in one launch)
    dora_varlen_attn_execute  (varlen attention, bf16 MFMA)
on synthetic inputs already resident in HBM.  Prints one JSON line.  Beside
the step it also times, on the same batch, the adjacent entry points:
dora_select_pack_residual (the kept rows of tokens + attention output), the
actor decode (dora_actor_gate + dora_actor_decode), dora_lc1_readout,
dora_trajectory_flops and dora_pl_sample.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, GB/s
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense matrix peaks, TFLOP/s
METRIC = "packed tokens/s + varlen-attn TFLOP/s (% MFMA peak), DeiT-B shape, B=256"


def plan_items(w: W.Workload, keep: np.ndarray) -> int:
    """Attention work items: one per (image, head, chunk of 192 queries)."""
    return w.H * int(np.sum((keep.astype(np.int64) + 191) // 192))


def select_pack_bytes(w: W.Workload, keep: np.ndarray, n_in: np.ndarray) -> int:
    """Algorithmic HBM bytes of select/pack with its attention plan: read scores
    and keep, read and write each kept row once, write the kept indices,
    cu_seqlens, the plan's items (8 bytes each) and its 2 KB header."""
    sk = int(keep.sum())
    return 2 * sk * w.C * w.elt + 4 * (int(n_in.sum()) + sk + 2 * w.B + 1) + 8 * plan_items(w, keep) + 2048


def residual_bytes(w: W.Workload, keep: np.ndarray, n_in: np.ndarray) -> int:
    """Algorithmic HBM bytes of select/pack after the attention residual: read
    scores and keep, read the kept rows of the tokens and of the attention
    output, write each packed row once, write the kept indices and cu_seqlens."""
    sk = int(keep.sum())
    return 3 * sk * w.C * w.elt + 4 * (int(n_in.sum()) + sk + 2 * w.B + 1)


def lc1_bytes(w: W.Workload, keep: np.ndarray) -> int:
    """Algorithmic HBM bytes of the LC1 readout input: read every packed row
    once, cu_seqlens, gamma and beta; write B x 2C fp32."""
    return int(keep.sum()) * w.C * w.elt + 4 * (w.B + 1) + 8 * w.C + 8 * w.B * w.C


def attn_flops(w: W.Workload, keep: np.ndarray) -> float:
    k = keep.astype(np.float64)
    return 4.0 * w.H * W.HEAD_DIM * float(np.sum(k * k))


def attn_bytes(w: W.Workload, keep: np.ndarray) -> int:
    return 4 * int(keep.sum()) * w.H * W.HEAD_DIM * w.elt   # Q, K, V read once, O written once


KERNEL_SOURCES = {"lc1": "paper_2609_34325_amd/csrc/lc1_readout.hip",
                  "attn": "paper_2609_34325_amd/csrc/varlen_attn.hip",
                  "select_pack": "paper_2609_34325_amd/csrc/select_pack.hip",
                  "residual": "paper_2609_34325_amd/csrc/select_pack.hip"}
KERNEL_NAMES = {"attn": ("attn_fwd_bf16_kernel", "attn_fwd_f32_kernel"),
                "select_pack": ("select_pack_kernel",),
                "residual": ("select_pack_residual_kernel",),
                "actor": ("actor_gate_kernel", "actor_decode_kernel"),
                "pl": ("pl_kernel",),
                "lc1": ("lc1_readout_kernel", "lc1_combine_kernel"),
                "flops": ("trajectory_flops_kernel",),
                "plan": ("attn_plan_kernel",)}


def source_digest(rel: str) -> str:
    """Hash of a kernel source with comments and blank lines removed, so that
    stored counter readings go stale when the code changes, not its comments."""
    import hashlib
    import re
    text = open(os.path.join(ROOT, rel)).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    code = "\n".join(l.rstrip() for l in text.splitlines() if l.strip())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def load_traffic(path: str, workload: str) -> dict:
    """HBM bytes per launch measured by hardware counters, per kernel; a kernel
    whose source changed since the counters were taken gets None."""
    try:
        entry = json.load(open(path)).get(workload, {})
    except (OSError, ValueError):
        return {}
    out = {}
    for k, rel in KERNEL_SOURCES.items():
        e = entry.get(k)
        out[k] = e["bytes_per_launch"] if e and e.get("source_sha") == source_digest(rel) else None
    return out


def _kernel_key(name: str):
    for k, pats in KERNEL_NAMES.items():
        if any(p in name for p in pats):
            return k
    return None


def summarize_profile(d: str, workload: str, traffic_json: str, calib_mib: int) -> int:
    """Reads the rocprofv3 CSV output of three runs of this script under
    DIR/stats (--kernel-trace --stats), DIR/fetch (--pmc FETCH_SIZE) and
    DIR/write (--pmc WRITE_SIZE), each run with --calibrate-copy; scales the
    counters by what they read for the plain calibration copy; prints a
    markdown summary and stores the per-launch bytes in the traffic file."""
    import csv
    import collections
    lines = []
    stats = os.path.join(d, "stats", "run_kernel_stats.csv")
    if os.path.exists(stats):
        lines += ["| Kernel | Calls | Average (ns) | Min (ns) | Max (ns) | Share |", "|---|---|---|---|---|---|"]
        for r in csv.DictReader(open(stats)):
            name = r["Name"].replace("dora::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
            lines.append(f"| {name} | {r['Calls']} | {float(r['AverageNs']):,.0f} | {int(r['MinNs']):,} | "
                         f"{int(r['MaxNs']):,} | {float(r['Percentage']):.1f} % |")
        lines.append("")
    calib_kib = calib_mib * 1024.0
    measured = collections.defaultdict(dict)
    factors = {}
    for counter, sub in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
        f = os.path.join(d, sub, "run_counter_collection.csv")
        if not os.path.exists(f):
            continue
        per = collections.defaultdict(lambda: collections.defaultdict(float))
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter:
                per[r["Kernel_Name"]][int(r["Dispatch_Id"])] += float(r["Counter_Value"])
        copies = [v for name, ds in per.items() if "copyBuffer" in name for v in ds.values()]
        ref = max(copies) if copies else 0.0
        if ref <= 0:
            continue
        factors[counter] = calib_kib / ref
        lines.append(f"{counter}: the {calib_mib} MiB calibration copy reads {ref:,.0f} KiB "
                     f"(scale factor {factors[counter]:.3f})")
        for name, ds in per.items():
            k = _kernel_key(name)
            if k is None:
                continue
            vals = [ds[i] for i in sorted(ds)]
            vals = vals[2:] if len(vals) > 3 else vals   # skip the first launches (cold caches)
            kib = sum(vals) / len(vals)
            # kernels of one entry point add up (one launch of each per call)
            prev = measured[k].get(counter, (0.0, 0.0, 0))
            measured[k][counter] = (prev[0] + kib, prev[1] + kib * 1024.0 * factors[counter], len(vals))
    lines.append("")
    if measured:
        lines += ["| Kernel | FETCH_SIZE KiB/launch | WRITE_SIZE KiB/launch | scaled HBM bytes/launch |",
                  "|---|---|---|---|"]
    try:
        allt = json.load(open(traffic_json))
    except (OSError, ValueError):
        allt = {}
    entry = allt.setdefault(workload, {})
    for k, m in sorted(measured.items()):
        if "FETCH_SIZE" not in m or "WRITE_SIZE" not in m:
            continue
        total = m["FETCH_SIZE"][1] + m["WRITE_SIZE"][1]
        lines.append(f"| {k} | {m['FETCH_SIZE'][0]:,.0f} | {m['WRITE_SIZE'][0]:,.0f} | {total:,.0f} |")
        if k in KERNEL_SOURCES:
            entry[k] = {"bytes_per_launch": total, "fetch_bytes": m["FETCH_SIZE"][1],
                        "write_bytes": m["WRITE_SIZE"][1], "source_sha": source_digest(KERNEL_SOURCES[k]),
                        "fetch_factor": factors["FETCH_SIZE"], "write_factor": factors["WRITE_SIZE"]}
    with open(traffic_json, "w") as fh:
        json.dump(allt, fh, indent=1, sort_keys=True)
        fh.write("\n")
    print("\n".join(lines))
    return 0


N_XCD = 8             # MI355X: GRBM_GUI_ACTIVE comes summed over its 8 accelerator complex dies
N_SIMD = 256 * 4      # 256 CUs x 4 SIMDs


def summarize_pmc(d: str, workload: str) -> int:
    """Reads rocprofv3 --pmc CSV output of runs of this script under DIR/*/
    and prints, per kernel, the matrix-unit and LDS counters the attention
    kernel is measured by: MFMA busy share (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE x SIMDs, rocprofv3's MfmaUtil), bf16 MFMA flops executed
    (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) against the algorithmic flops, and
    LDS bank conflicts per LDS access cycle.  Averages are per dispatch, over
    the launches after the first two."""
    import csv
    import collections
    w = W.WORKLOADS[workload]
    keep = W.generate(w, parts=("keep",))[0].keep
    alg = {"attn": attn_flops(w, keep)}
    per = collections.defaultdict(lambda: collections.defaultdict(lambda: collections.defaultdict(float)))
    dur = collections.defaultdict(dict)
    for sub in sorted(os.listdir(d)):
        f = os.path.join(d, sub, "run_counter_collection.csv")
        if not os.path.exists(f):
            continue
        for r in csv.DictReader(open(f)):
            k = _kernel_key(r["Kernel_Name"])
            if k is None:
                continue
            disp = (sub, int(r["Dispatch_Id"]))
            per[k][r["Counter_Name"]][disp] += float(r["Counter_Value"])
            dur[k][disp] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9

    def mean(vals):
        vals = [vals[i] for i in sorted(vals)]
        vals = vals[2:] if len(vals) > 3 else vals
        return sum(vals) / len(vals) if vals else float("nan")

    lines = ["| Kernel | Counter / derived | Per launch |", "|---|---|---|"]
    for k in sorted(per):
        c = {name: mean(v) for name, v in per[k].items()}
        t = mean(dur[k])
        for name in sorted(c):
            lines.append(f"| {k} | {name} | {c[name]:,.0f} |")
        lines.append(f"| {k} | duration under the counters (us) | {t * 1e6:,.1f} |")
        grbm = c.get("GRBM_GUI_ACTIVE")
        if grbm:
            lines.append(f"| {k} | clock = GRBM_GUI_ACTIVE / {N_XCD} / duration (GHz) | {grbm / N_XCD / t / 1e9:.2f} |")
        if grbm and "SQ_VALU_MFMA_BUSY_CYCLES" in c:
            util = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (grbm / N_XCD * N_SIMD)
            lines.append(f"| {k} | MFMA busy = MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / {N_XCD} x {N_SIMD} SIMDs) | "
                         f"{100 * util:.1f} % |")
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in c and k in alg:
            ex = c["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
            lines.append(f"| {k} | bf16 MFMA flops executed / algorithmic | {ex / 1e9:,.2f} G / {alg[k] / 1e9:,.2f} G "
                         f"= {ex / alg[k]:.2f} |")
            lines.append(f"| {k} | executed bf16 MFMA rate over the duration | {ex / t / 1e12:,.0f} TFLOP/s "
                         f"({100 * ex / t / 1e12 / MFMA_PEAK_TFLOPS['bf16']:.1f} % of peak) |")
        if "SQ_LDS_BANK_CONFLICT" in c and "SQ_LDS_IDX_ACTIVE" in c and c["SQ_LDS_IDX_ACTIVE"] > 0:
            lines.append(f"| {k} | LDS bank conflict cycles / LDS active cycles | "
                         f"{c['SQ_LDS_BANK_CONFLICT'] / c['SQ_LDS_IDX_ACTIVE']:.3f} |")
        if "SQ_WAVE_CYCLES" in c:
            for name in ("SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY"):
                if name in c:
                    lines.append(f"| {k} | {name} / SQ_WAVE_CYCLES | {100 * c[name] / c['SQ_WAVE_CYCLES']:.1f} % |")
    print("\n".join(lines))
    return 0


def measure_peaks(torch, stream) -> dict:
    """What this device sustains: a plain 256 MiB device-to-device copy
    (read + write bytes over time) and a loop of independent bf16 MFMAs on
    every SIMD (paper_2609_34325_amd/csrc/calibrate.hip)."""
    import ctypes
    peaks = {}
    nbytes = 256 * 2 ** 20
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    peaks["copy_GBs"] = 2 * nbytes * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    from paper_2609_34325_amd import build as pkg_build
    if os.path.exists(pkg_build.CALIB_LIB):
        lib = ctypes.CDLL(pkg_build.CALIB_LIB)
        lib.dora_calibrate_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        lib.dora_calibrate_mfma_bf16_flops.restype = ctypes.c_double
        lib.dora_calibrate_mfma_bf16_flops.argtypes = [ctypes.c_int, ctypes.c_int]
        blocks = 2 * torch.cuda.get_device_properties(0).multi_processor_count
        iters = 4096
        out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
        for _ in range(2):
            assert lib.dora_calibrate_mfma_bf16(blocks, iters, out.data_ptr(), stream.cuda_stream) == 0
        e0.record(stream)
        for _ in range(5):
            lib.dora_calibrate_mfma_bf16(blocks, iters, out.data_ptr(), stream.cuda_stream)
        e1.record(stream)
        torch.cuda.synchronize()
        flops = 5 * lib.dora_calibrate_mfma_bf16_flops(blocks, iters)
        peaks["mfma_bf16_TFLOPs"] = flops / (e0.elapsed_time(e1) * 1e-3) / 1e12
    return peaks


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def run_cpu_baseline(w: W.Workload, r: W.RoundInputs, repeats: int = 9, repeats_1: int = 3) -> dict:
    """The oracle as it stands, timed on this host's cores over the full batch:
    the median of `repeats` passes on all the process's cores and of
    `repeats_1` passes on one thread (about 8-12 s of CPU work at DeiT-B)."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    times = []
    for _ in range(repeats):
        t0 = time.perf_counter()
        idx, cu, packed, st = oracle.select_pack(r.scores, r.keep, r.tokens)
        oracle.varlen_attn(r.q, r.k, r.v, cu, w.dtype, threads=threads)
        times.append(time.perf_counter() - t0)
        assert st == 0
    t = statistics.median(times)
    times_1 = []
    for _ in range(repeats_1):
        t0 = time.perf_counter()
        idx, cu, packed, st = oracle.select_pack(r.scores, r.keep, r.tokens)
        oracle.varlen_attn(r.q, r.k, r.v, cu, w.dtype, threads=1)
        times_1.append(time.perf_counter() - t0)
    t1 = statistics.median(times_1)
    return {"value": r.total_keep / t, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "value_1_thread": r.total_keep / t1,
            "sample": f"full {w.name} batch (B={w.B}, sum keep={r.total_keep}), select+pack+attention, "
                      f"median of {repeats} passes on {threads} threads ({t:.3f} s each) and of "
                      f"{repeats_1} on one thread ({t1:.3f} s each), "
                      f"{repeats * t + repeats_1 * t1:.1f} s of CPU work in all, CPU: {cpu_model()}"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--repeats", type=int, default=5)
    ap.add_argument("--workload", default=W.HEADLINE, choices=sorted(W.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cold-sets", type=int, default=3,
                    help="also time the step rotating through this many buffer sets (cold MALL); <= 1: off")
    ap.add_argument("--no-peaks", action="store_true", help="skip measuring the copy and MFMA peaks")
    ap.add_argument("--no-actor", action="store_true", help="skip timing the actor decode (outside the step)")
    ap.add_argument("--no-pl", action="store_true", help="skip timing the Plackett-Luce draw (outside the step)")
    ap.add_argument("--no-lc1", action="store_true", help="skip timing the LC1 readout input (outside the step)")
    ap.add_argument("--no-flops", action="store_true", help="skip timing the trajectory FLOP count (outside the step)")
    ap.add_argument("--no-residual", action="store_true",
                    help="skip timing select/pack after the attention residual (outside the step)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before timing, run one plain device copy of MIB MiB (a reference dispatch "
                         "for scaling hardware byte counters)")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch (from rocprofv3 counters), if present")
    ap.add_argument("--summarize-pmc", metavar="DIR",
                    help="print matrix-unit / LDS counter summaries from rocprofv3 --pmc runs under DIR/*/")
    ap.add_argument("--summarize-profile", metavar="DIR",
                    help="no benchmark: summarise rocprofv3 output under DIR/{stats,fetch,write} "
                         "for --workload and update --traffic-json")
    args = ap.parse_args()
    if args.summarize_pmc:
        return summarize_pmc(args.summarize_pmc, args.workload)
    if args.summarize_profile:
        return summarize_profile(args.summarize_profile, args.workload, args.traffic_json,
                                 args.calibrate_copy or 256)

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path shards by image; see the design notes).", file=sys.stderr)
        return 2

    import torch
    import paper_2609_34325_amd as dora

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dora.load_library()
    torch.cuda.set_device(0)
    w = W.WORKLOADS[args.workload]
    r = W.generate(w)[0]
    print(f"[bench] {w.name}: B={w.B} N={w.N} H={w.H} C={w.C} {w.dtype} sum_keep={r.total_keep}",
          file=sys.stderr, flush=True)

    def dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    sk = r.total_keep
    max_seqlen = int(r.keep.max())
    stream = torch.cuda.current_stream()

    def buffer_set(src=None):
        """Inputs (copied from `src`, or uploaded) and outputs of one step."""
        b = {}
        if src is None:
            b["scores"], b["keep"], b["tokens"] = dev(r.scores), dev(r.keep), dev(r.tokens)
            b["q"], b["k"], b["v"] = dev(r.q), dev(r.k), dev(r.v)
        else:
            for name in ("scores", "keep", "tokens", "q", "k", "v"):
                b[name] = src[name].clone()
        b["idx"] = torch.empty(sk, dtype=torch.int32, device="cuda")
        b["cu"] = torch.empty(w.B + 1, dtype=torch.int32, device="cuda")
        b["packed"] = torch.empty((sk, w.C), dtype=b["tokens"].dtype, device="cuda")
        b["out"] = torch.empty_like(b["q"])
        b["ws"] = dora.new_workspace(w.B, w.H, max_seqlen)
        b["st"] = dora.new_status()
        return b

    def step(b, ev=None):
        if ev is not None:
            ev[0].record(stream)
        dora.dora_select_pack_plan(b["scores"], b["keep"], b["tokens"], w.H, max_seqlen, sk, b["ws"],
                                   idx_out=b["idx"], cu_out=b["cu"], packed_out=b["packed"], cap_rows=sk,
                                   dev_status=b["st"], stream=stream)
        if ev is not None:
            ev[1].record(stream)
        dora.dora_varlen_attn_execute(b["q"], b["k"], b["v"], b["cu"], max_seqlen, b["ws"], out=b["out"],
                                      dev_status=b["st"], stream=stream)
        if ev is not None:
            ev[2].record(stream)

    def timed(sets, tag):
        """Median over repeats of (step time, select/pack+plan time, attention
        time) in ms; step i uses sets[i % len(sets)].  Each repeat times K steps
        twice: once bare (events only at the two ends) and once with events
        around every kernel (per-kernel durations; an event between two kernels
        adds a few microseconds of dispatch latency to the interval, so these
        are upper bounds)."""
        for i in range(args.warmup):
            step(sets[i % len(sets)])
        torch.cuda.synchronize()
        reps = []
        for rep in range(args.repeats):
            t_start = torch.cuda.Event(enable_timing=True)
            t_end = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            t_start.record(stream)
            for i in range(args.steps):
                step(sets[i % len(sets)])
            t_end.record(stream)
            torch.cuda.synchronize()
            total_ms = t_start.elapsed_time(t_end)
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
            torch.cuda.synchronize()
            for i in range(args.steps):
                step(sets[i % len(sets)], evs[i])
            torch.cuda.synchronize()
            sel = np.mean([e[0].elapsed_time(e[1]) for e in evs])
            attn = np.mean([e[1].elapsed_time(e[2]) for e in evs])
            reps.append((total_ms / args.steps, sel, attn))
            print(f"[bench] {tag} repeat {rep}: {total_ms / args.steps * 1e3:.1f} us/step "
                  f"(per kernel with events: select_pack+plan {sel * 1e3:.1f}, "
                  f"attention {attn * 1e3:.1f})", file=sys.stderr, flush=True)
        for b in sets:
            assert int(b["st"].item()) == 0, f"device status {int(b['st'].item())}"
        return sorted(reps, key=lambda x: x[0])[len(reps) // 2]

    main_set = buffer_set()
    if args.calibrate_copy > 0:
        src = torch.ones(args.calibrate_copy * 2 ** 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Warm: the same buffers every step, as in deployment, where the producing
    # kernel has just written the inputs.
    ms_step, ms_sel, ms_attn = timed([main_set], "warm")
    # Cold: rotate through enough buffer sets that one rotation exceeds twice
    # the 256 MB MALL, so every step's inputs come from HBM.
    cold = None
    if args.cold_sets > 1:
        set_bytes = sum(t.numel() * t.element_size() for t in main_set.values())
        cold_sets = [main_set] + [buffer_set(main_set) for _ in range(args.cold_sets - 1)]
        c_step, c_sel, c_attn = timed(cold_sets, "cold")
        cold = {"sets": args.cold_sets, "bytes_per_set": set_bytes, "ms_per_step": c_step,
                "value": sk / (c_step * 1e-3),
                "us": {"select_pack_plan": c_sel * 1e3, "attention": c_attn * 1e3, "step": c_step * 1e3}}

    # Beside the path: deletion after the attention residual (the kept rows of
    # tokens + attention output) on the same batch, timed on its own, warm and,
    # with a second attention-output buffer per set, cold.
    residual = None
    if not args.no_residual:
        a_host = W.generate(w, parts=("keep", "attn_out"))[0].attn_out
        a_main = dev(a_host)

        def res_launch(b, a):
            dora.dora_select_pack_residual(b["scores"], b["keep"], b["tokens"], a, idx_out=b["idx"],
                                           cu_out=b["cu"], packed_out=b["packed"], cap_rows=sk,
                                           dev_status=b["st"], stream=stream)

        def res_timed(pairs, tag):
            for i in range(args.warmup):
                res_launch(*pairs[i % len(pairs)])
            reps = []
            for rep in range(args.repeats):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record(stream)
                for i in range(args.steps):
                    res_launch(*pairs[i % len(pairs)])
                e1.record(stream)
                torch.cuda.synchronize()
                reps.append(e0.elapsed_time(e1) / args.steps)
                print(f"[bench] residual {tag} repeat {rep}: {reps[-1] * 1e3:.1f} us/launch",
                      file=sys.stderr, flush=True)
            for b, _ in pairs:
                assert int(b["st"].item()) == 0, f"device status {int(b['st'].item())}"
            return sorted(reps)[len(reps) // 2]

        rb = residual_bytes(w, r.keep, r.n_in)
        ms_res = res_timed([(main_set, a_main)], "warm")
        residual = {"entry": "dora_select_pack_residual", "kernel": "select_pack_residual_kernel",
                    "bound": "hbm", "us": ms_res * 1e3, "achieved": rb / (ms_res * 1e-3) / 1e9,
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "algorithmic_bytes": rb,
                    "tokens_per_s": sk / (ms_res * 1e-3), "regime": "warm"}
        residual["frac"] = residual["achieved"] / HBM_PEAK_GBS
        if args.cold_sets > 1:
            pairs = [(main_set, a_main)] + [(b, a_main.clone()) for b in cold_sets[1:]]
            ms_c = res_timed(pairs, "cold")
            residual["cold"] = {"us": ms_c * 1e3, "achieved": rb / (ms_c * 1e-3) / 1e9,
                                "frac": rb / (ms_c * 1e-3) / 1e9 / HBM_PEAK_GBS}
            del pairs
        del a_main
    if args.cold_sets > 1:
        del cold_sets

    def time_calls(fn):
        """Median over repeats of the mean time of `steps` back-to-back calls
        of fn (after `warmup` calls), HIP events at the two ends, in ms."""
        for _ in range(args.warmup):
            fn()
        reps = []
        for _ in range(args.repeats):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(args.steps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            reps.append(e0.elapsed_time(e1) / args.steps)
        return sorted(reps)[len(reps) // 2]

    # Beside the path: the deterministic actor's decode that produces its
    # inputs (gate + compaction, then budget argmax, keep counts and
    # keep-scores), timed as a pair of launches.
    actor = None
    if not args.no_actor:
        M = W.budget_outputs(w)
        p_h, logits_h, removal_h = W.actor_outputs(w)
        p_d, logits_d, removal_d = dev(p_h), dev(logits_h), dev(removal_h)
        on_rank = torch.empty(w.B, dtype=torch.int32, device="cuda")
        on_list = torch.empty_like(on_rank)
        n_on = torch.empty(1, dtype=torch.int32, device="cuda")
        keep_d = torch.empty_like(on_rank)
        ks_d = torch.empty_like(removal_d)
        st_a = dora.new_status()

        def actor_pair():
            dora.dora_actor_gate(p_d, M, w.N, on_rank=on_rank, on_list=on_list, n_on=n_on, dev_status=st_a,
                                 stream=stream)
            dora.dora_actor_decode(logits_d, on_rank, w.N, removal_scores=removal_d, keep_out=keep_d,
                                   scores_out=ks_d, dev_status=st_a, stream=stream)

        ms_actor = time_calls(actor_pair)
        assert int(st_a.item()) == 0, f"device status {int(st_a.item())}"
        actor = {"entries": ["dora_actor_gate", "dora_actor_decode"], "bound": "latency",
                 "us_per_pair": ms_actor * 1e3, "gate_on": int(n_on.item()), "M": M,
                 "note": "two small launches back to back; the cost is launch and dependency latency"}
        print(f"[bench] actor decode: {ms_actor * 1e3:.1f} us per gate+decode pair, "
              f"{actor['gate_on']} of {w.B} gates open", file=sys.stderr, flush=True)

    # Beside the path: the LC1 readout input (LayerNorm + segmented mean over
    # the packed rows of the same batch), an HBM-bound segmented reduction.
    lc1 = None
    if not args.no_lc1:
        x_h, gamma_h, beta_h = W.readout_rows(w, r.keep)
        cu_h = np.concatenate([[0], np.cumsum(r.keep)]).astype(np.int32)
        x_d, cu_d, gamma_d, beta_d = dev(x_h), dev(cu_h), dev(gamma_h), dev(beta_h)
        out_d = torch.empty((w.B, 2 * w.C), dtype=torch.float32, device="cuda")
        st_l = dora.new_status()
        ws_l = dora.new_lc1_workspace(w.B, w.C)

        def lc1_call():
            dora.dora_lc1_readout(x_d, cu_d, gamma_d, beta_d, 1e-6, out=out_d, workspace=ws_l, dev_status=st_l,
                                  stream=stream)

        ms_lc1 = time_calls(lc1_call)
        assert int(st_l.item()) == 0, f"device status {int(st_l.item())}"
        lb = lc1_bytes(w, r.keep)
        lc1 = {"entry": "dora_lc1_readout", "kernel": "lc1_readout_kernel (+ lc1_combine_kernel when split)",
               "bound": "hbm", "us": ms_lc1 * 1e3,
               "achieved": lb / (ms_lc1 * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
               "frac": lb / (ms_lc1 * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": lb, "regime": "warm"}
        print(f"[bench] lc1 readout: {ms_lc1 * 1e3:.1f} us per launch ({lc1['achieved']:.0f} GB/s)",
              file=sys.stderr, flush=True)
        del x_d

    # Beside the path: FLOP accounting of the batch's realised trajectories
    # over a 12-block backbone (pruning at block 0 with this batch's keep
    # counts, then none): one small latency-bound launch.
    traj = None
    if not args.no_flops:
        L_blocks = 12
        T = np.vstack([np.full((1, w.B), w.N, np.int32), np.tile(r.keep.astype(np.int32), (L_blocks, 1))])
        T_d = dev(np.ascontiguousarray(T))
        f_d = torch.empty(w.B, dtype=torch.int64, device="cuda")
        tot_d = torch.empty(1, dtype=torch.int64, device="cuda")
        st_f = dora.new_status()

        def flops_call():
            dora.dora_trajectory_flops(T_d, w.C, w.N - 1, 16, flops_out=f_d, total_out=tot_d, dev_status=st_f,
                                       stream=stream)

        ms_fl = time_calls(flops_call)
        assert int(st_f.item()) == 0, f"device status {int(st_f.item())}"
        traj = {"entry": "dora_trajectory_flops", "kernel": "trajectory_flops_kernel", "bound": "latency",
                 "us": ms_fl * 1e3, "images": w.B, "blocks": L_blocks,
                 "gflops_per_image": int(tot_d.item()) / w.B / 1e9}
        print(f"[bench] trajectory flops: {ms_fl * 1e3:.1f} us per launch", file=sys.stderr, flush=True)

    # Beside the path: the training-time draw (Gumbel-top-k Plackett-Luce
    # deletion of n - keep tokens per image, with its ordered log-probability).
    pl = None
    if not args.no_pl:
        k_h = (r.n_in - r.keep).astype(np.int32)
        g_h = W.gumbel_noise(w)
        s_d, g_d, k_d = dev(r.scores), dev(g_h), dev(k_h)
        order = torch.empty(int(k_h.sum()) + 1, dtype=torch.int32, device="cuda")
        cu_o = torch.empty(w.B + 1, dtype=torch.int32, device="cuda")
        lp_d = torch.empty(w.B, dtype=torch.float32, device="cuda")
        st_p = dora.new_status()

        def pl_call():
            dora.dora_pl_sample(s_d, g_d, k_d, order_out=order, cu_order_out=cu_o, logprob_out=lp_d,
                                dev_status=st_p, stream=stream)

        ms_pl = time_calls(pl_call)
        assert int(st_p.item()) == 0, f"device status {int(st_p.item())}"
        pl = {"entry": "dora_pl_sample", "kernel": "pl_kernel", "bound": "latency", "us": ms_pl * 1e3,
              "draws": int(k_h.sum()), "images": w.B,
              "note": "one workgroup per image: LDS bitonic sort of the visual keys and a block scan"}
        print(f"[bench] pl sample: {ms_pl * 1e3:.1f} us per launch ({int(k_h.sum())} draws)",
              file=sys.stderr, flush=True)

    flops = attn_flops(w, r.keep)
    sp_bytes = select_pack_bytes(w, r.keep, r.n_in)
    a_bytes = attn_bytes(w, r.keep)
    attn_tflops = flops / (ms_attn * 1e-3) / 1e12
    sp_gbs = sp_bytes / (ms_sel * 1e-3) / 1e9
    peak = MFMA_PEAK_TFLOPS[w.dtype]

    traffic = load_traffic(args.traffic_json, w.name)

    # The attention roofline is the lower of the two ceilings at its
    # arithmetic intensity (flops per algorithmic byte): below the ridge point
    # (peak flops / peak bandwidth) the kernel is bound by HBM.
    intensity = flops / a_bytes
    attn_gbs = a_bytes / (ms_attn * 1e-3) / 1e9
    kname = "attn_fwd_bf16_kernel" if w.dtype == "bf16" else "attn_fwd_f32_kernel"
    common = {"kernel": kname, "traffic": traffic.get("attn"), "algorithmic_bytes": a_bytes, "flops": flops,
              "intensity_flop_per_byte": intensity, "ridge_flop_per_byte": peak * 1e3 / HBM_PEAK_GBS,
              "tflops": attn_tflops, "mfma_peak_tflops": peak, "mfma_frac": attn_tflops / peak}
    if intensity < peak * 1e3 / HBM_PEAK_GBS:
        attn_roofline = {"bound": "hbm", "achieved": attn_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": attn_gbs / HBM_PEAK_GBS, **common}
    else:
        attn_roofline = {"bound": "mfma", "achieved": attn_tflops, "peak": peak, "unit": "TFLOP/s",
                         "frac": attn_tflops / peak, **common}

    peaks = {} if args.no_peaks else measure_peaks(torch, stream)
    attn_roofline["attainable_tflops"] = min(peak, intensity * HBM_PEAK_GBS / 1e3)
    if "copy_GBs" in peaks:
        attn_roofline["frac_of_measured_copy"] = attn_gbs / peaks["copy_GBs"]
    if "mfma_bf16_TFLOPs" in peaks and w.dtype == "bf16":
        attn_roofline["frac_of_measured_mfma"] = attn_tflops / peaks["mfma_bf16_TFLOPs"]
    if cold is not None:
        c_attn, c_sel = cold["us"]["attention"] * 1e-6, cold["us"]["select_pack_plan"] * 1e-6
        cold["attn_GBs"] = a_bytes / c_attn / 1e9
        cold["attn_hbm_frac"] = cold["attn_GBs"] / HBM_PEAK_GBS
        cold["attn_tflops"] = flops / c_attn / 1e12
        cold["select_pack_GBs"] = sp_bytes / c_sel / 1e9
        cold["select_pack_hbm_frac"] = cold["select_pack_GBs"] / HBM_PEAK_GBS

    result = {
        "metric": METRIC,
        "value": sk / (ms_step * 1e-3),
        "unit": "packed tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "N": w.N, "H": w.H, "head_dim": W.HEAD_DIM, "C": w.C,
                   "sum_keep": sk, "sum_keep_sq": int(np.sum(r.keep.astype(np.int64) ** 2)),
                   "max_seqlen": max_seqlen},
        "roofline": attn_roofline,
        "roofline_select_pack": {"bound": "hbm", "kernel": "select_pack_kernel", "achieved": sp_gbs,
                                 "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": sp_gbs / HBM_PEAK_GBS,
                                 "traffic": traffic.get("select_pack"), "algorithmic_bytes": sp_bytes},
        "select_pack_tokens_per_s": sk / (ms_sel * 1e-3),
        "attn_tflops": attn_tflops,
        "us": {"select_pack_plan": ms_sel * 1e3, "attention": ms_attn * 1e3, "step": ms_step * 1e3},
        "repeats": args.repeats,
        "regime": "warm: the same input buffers every step",
        "cold": cold,
        "measured_peaks": peaks,
    }
    if "copy_GBs" in peaks:
        result["roofline_select_pack"]["frac_of_measured_copy"] = sp_gbs / peaks["copy_GBs"]
    if residual is not None:
        residual["traffic"] = traffic.get("residual")
        if "copy_GBs" in peaks:
            residual["frac_of_measured_copy"] = residual["achieved"] / peaks["copy_GBs"]
        result["residual_select_pack"] = residual
    if lc1 is not None:
        lc1["traffic"] = traffic.get("lc1")
        if "copy_GBs" in peaks:
            lc1["frac_of_measured_copy"] = lc1["achieved"] / peaks["copy_GBs"]
        result["lc1_readout"] = lc1
    if actor is not None:
        result["actor_decode"] = actor
    if pl is not None:
        result["pl_sample"] = pl
    if traj is not None:
        result["trajectory_flops"] = traj
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        result["cpu_baseline"] = run_cpu_baseline(w, r)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
