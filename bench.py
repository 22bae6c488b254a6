"""Benchmark of the DORA deployment hot path on one MI355X.

One step = one pass of the whole path over one batch:
    dora_select_pack_plan     (top-k with CLS pinned + cu_seqlens + packed
                               gather, and the attention work queue of the
                               packed layout, in one launch)
    dora_varlen_attn_execute  (varlen attention, bf16 MFMA)
on synthetic inputs already resident in HBM; a cascaded workload chains its
rounds inside one step (round r+1 reads round r's packed output and
cu_seqlens).  Prints one JSON line for the headline workload (DeiT-B), with a
record of its own for every other workload, each checked against the oracle
in the CPU-baseline leg.  Beside the step it also times, on the headline
batch, the adjacent entry points: dora_select_pack_residual (the kept rows of
tokens + attention output), the actor decode (dora_actor_gate +
dora_actor_decode), dora_lc1_readout, dora_trajectory_flops and
dora_pl_sample.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import collections
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
# Workloads with a record of their own next to the headline (the DINOv2 shape
# serves the LC1 readout only).
CONFIG_ORDER = ("deit_tiny_fp32", "deit_s_bf16", "deit_b_bf16", "vit_l_cascade_bf16", "vit_b384_skew_bf16")
BF16_MAX_ABS, BF16_MEAN_ABS, F32_MAX_ABS = 2e-2, 2e-3, 1e-5   # attention tolerances


def select_pack_bytes(w: W.Workload, keep: np.ndarray, n_in: np.ndarray, n_items: int, packed_in: bool) -> int:
    """Algorithmic HBM bytes of select/pack with its attention plan: read scores
    and keep (and cu_in for packed input), read and write each kept row once,
    write the kept indices, cu_seqlens, the plan's items (8 bytes each) and
    its 2 KB header."""
    sk = int(keep.sum())
    B = len(keep)
    cu_in = 4 * (B + 1) if packed_in else 0
    return 2 * sk * w.C * w.elt + 4 * (int(n_in.sum()) + sk + 2 * B + 1) + cu_in + 8 * n_items + 2048


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
    """4 H d sum(k^2): QK^T and PV of every (sequence, head)."""
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
                "scan": ("keep_scan_kernel",),
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


class PhaseLog:
    """Launch counts per kernel key for each timed phase, in launch order, so
    that a rocprofv3 kernel trace of the same run can be split by phase (one
    stream, phases separated by synchronisation)."""

    def __init__(self):
        self.phases = []   # [name, {key: count}]
        self.paused = False  # while a graph is captured (its launches run, and are counted, at replay)

    def start(self, name: str):
        self.phases.append([name, collections.Counter()])

    def count(self, *keys):
        if self.paused:
            return
        if not self.phases:
            self.start("setup")
        for k in keys:
            self.phases[-1][1][k] += 1

    def dump(self, path: str):
        with open(path, "w") as fh:
            json.dump([[n, dict(c)] for n, c in self.phases], fh, indent=0)


def split_by_phase(dispatches: dict, phase_log: list) -> dict:
    """dispatches: key -> durations (ns) in dispatch order.  Returns
    phase -> key -> durations."""
    pos = collections.defaultdict(int)
    out = collections.defaultdict(dict)
    for name, counts in phase_log:
        for k, n in counts.items():
            seq = dispatches.get(k, [])
            out[name][k] = seq[pos[k]:pos[k] + n]
            pos[k] += n
    return out


def summarize_profile(d: str, workload: str, traffic_json: str, calib_mib: int, phase_log: str = None) -> int:
    """Reads the rocprofv3 CSV output of three runs of this script under
    DIR/stats (--kernel-trace --stats), DIR/fetch (--pmc FETCH_SIZE) and
    DIR/write (--pmc WRITE_SIZE), each run with --calibrate-copy; scales the
    counters by what they read for the plain calibration copy; prints a
    markdown summary (with the kernel trace split by the bench's phases when
    a phase log is given) and stores the per-launch bytes in the traffic file."""
    import csv
    lines = []
    stats = os.path.join(d, "stats", "run_kernel_stats.csv")
    if os.path.exists(stats):
        lines += ["| Kernel | Calls | Average (ns) | Min (ns) | Max (ns) | Share |", "|---|---|---|---|---|---|"]
        for r in csv.DictReader(open(stats)):
            name = r["Name"].replace("dora::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
            lines.append(f"| {name} | {r['Calls']} | {float(r['AverageNs']):,.0f} | {int(r['MinNs']):,} | "
                         f"{int(r['MaxNs']):,} | {float(r['Percentage']):.1f} % |")
        lines.append("")
    trace = os.path.join(d, "stats", "run_kernel_trace.csv")
    if phase_log and os.path.exists(trace) and os.path.exists(phase_log):
        rows = sorted(csv.DictReader(open(trace)), key=lambda r: int(r["Dispatch_Id"]))
        disp = collections.defaultdict(list)
        for r in rows:
            k = _kernel_key(r["Kernel_Name"])
            if k is not None:
                disp[k].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        per = split_by_phase(disp, json.load(open(phase_log)))
        lines += ["Kernel trace split by the bench's phases (average duration per launch):", "",
                  "| Phase | Kernel | Launches | Average (ns) |", "|---|---|---|---|"]
        for name, ks in per.items():
            for k, v in sorted(ks.items()):
                if v:
                    lines.append(f"| {name} | {k} | {len(v)} | {sum(v) / len(v):,.0f} |")
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
    if measured:
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
    the launches after the first two.  Where a run left its phase log
    (DIR/<run>/phases.json, from --phase-log), the attention and select/pack
    counters are also given per timed phase: in the step, and alone (back to
    back on one buffer set, the MALL-resident regime)."""
    import csv
    w = W.WORKLOADS[workload]
    keep = W.generate(w, parts=("keep",))[0].keep
    alg = {"attn": attn_flops(w, keep)}
    per = collections.defaultdict(lambda: collections.defaultdict(lambda: collections.defaultdict(float)))
    dur = collections.defaultdict(dict)
    phase_of = {}  # (run, dispatch id) -> phase name
    for sub in sorted(os.listdir(d)):
        f = os.path.join(d, sub, "run_counter_collection.csv")
        if not os.path.exists(f):
            continue
        order = collections.defaultdict(set)  # kernel key -> dispatch ids of this run
        for r in csv.DictReader(open(f)):
            k = _kernel_key(r["Kernel_Name"])
            if k is None:
                continue
            disp = (sub, int(r["Dispatch_Id"]))
            per[k][r["Counter_Name"]][disp] += float(r["Counter_Value"])
            dur[k][disp] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
            order[k].add(disp[1])
        plog = os.path.join(d, sub, "phases.json")
        if os.path.exists(plog):
            seq = {k: sorted(v) for k, v in order.items()}
            for name, ids in split_by_phase(seq, json.load(open(plog))).items():
                for k, v in ids.items():
                    for i in v:
                        phase_of[(sub, i)] = name

    def mean(vals):
        vals = [vals[i] for i in sorted(vals)]
        vals = vals[2:] if len(vals) > 3 else vals
        return sum(vals) / len(vals) if vals else float("nan")

    def derived(k, c, t):
        out = []
        grbm = c.get("GRBM_GUI_ACTIVE")
        if grbm and "SQ_VALU_MFMA_BUSY_CYCLES" in c:
            util = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (grbm / N_XCD * N_SIMD)
            out.append((f"MFMA busy = MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / {N_XCD} x {N_SIMD} SIMDs)",
                        f"{100 * util:.1f} %"))
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in c and k in alg:
            ex = c["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
            out.append(("bf16 MFMA flops executed / algorithmic",
                        f"{ex / 1e9:,.2f} G / {alg[k] / 1e9:,.2f} G = {ex / alg[k]:.2f}"))
            out.append(("executed bf16 MFMA rate over the duration",
                        f"{ex / t / 1e12:,.0f} TFLOP/s ({100 * ex / t / 1e12 / MFMA_PEAK_TFLOPS['bf16']:.1f} % of peak)"))
        if "SQ_LDS_BANK_CONFLICT" in c and "SQ_LDS_IDX_ACTIVE" in c and c["SQ_LDS_IDX_ACTIVE"] > 0:
            out.append(("LDS bank conflict cycles / LDS active cycles",
                        f"{c['SQ_LDS_BANK_CONFLICT'] / c['SQ_LDS_IDX_ACTIVE']:.3f}"))
        if "SQ_WAVE_CYCLES" in c:
            for name in ("SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY"):
                if name in c:
                    out.append((f"{name} / SQ_WAVE_CYCLES", f"{100 * c[name] / c['SQ_WAVE_CYCLES']:.1f} %"))
        return out

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
        for name, val in derived(k, c, t):
            lines.append(f"| {k} | {name} | {val} |")
    if phase_of:
        # Per timed phase (warm-up phases left out), for the step kernels.
        lines += ["", "Per timed phase (averages over the phase's launches in every run that logged its phases):", "",
                  "| Kernel | Phase | Launches | Duration (us) | Derived |", "|---|---|---|---|---|"]
        for k in ("attn", "select_pack"):
            if k not in per:
                continue
            names = sorted({phase_of[dd] for dd in dur[k] if dd in phase_of and not phase_of[dd].endswith("warmup")})
            for ph in names:
                sel = lambda vals: {dd: v for dd, v in vals.items() if phase_of.get(dd) == ph}
                c = {name: (sum(sel(v).values()) / len(sel(v)) if sel(v) else float("nan")) for name, v in per[k].items()}
                dd_ph = sel(dur[k])
                t = sum(dd_ph.values()) / len(dd_ph)
                der = "; ".join(f"{n}: {v}" for n, v in derived(k, c, t))
                lines.append(f"| {k} | {ph} | {len(dd_ph)} | {t * 1e6:,.1f} | {der} |")
    print("\n".join(lines))
    return 0


def copy_fracs(achieved_gbs: float, peaks: dict) -> dict:
    """An HBM-bound kernel's rate as fractions of the measured copies:
    the runtime's copy (`frac_of_measured_copy`), the streaming kernel with
    plain stores and with write-through stores."""
    out = {}
    for key, name in (("copy_GBs", "frac_of_measured_copy"), ("copy_kernel_GBs", "frac_of_copy_kernel"),
                      ("copy_kernel_through_GBs", "frac_of_copy_kernel_through")):
        if key in peaks:
            out[name] = achieved_gbs / peaks[key]
    return out


def measure_peaks(torch, stream) -> dict:
    """What this device sustains: a 256 MiB device-to-device copy by the
    runtime (read + write bytes over time), the same copy by a streaming
    kernel with plain stores and with the library's write-through stores,
    and a loop of independent bf16 MFMAs on every SIMD
    (paper_2609_34325_amd/csrc/calibrate.hip)."""
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
        del out
        lib.dora_calibrate_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_void_p]
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        cblocks = 4 * torch.cuda.get_device_properties(0).multi_processor_count
        for through, key in ((0, "copy_kernel_GBs"), (1, "copy_kernel_through_GBs")):
            for _ in range(3):
                assert lib.dora_calibrate_copy(src.data_ptr(), dst.data_ptr(), nbytes, cblocks, through,
                                               stream.cuda_stream) == 0
            e0.record(stream)
            for _ in range(10):
                lib.dora_calibrate_copy(src.data_ptr(), dst.data_ptr(), nbytes, cblocks, through, stream.cuda_stream)
            e1.record(stream)
            torch.cuda.synchronize()
            peaks[key] = 2 * nbytes * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
        del src, dst
    return peaks


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def _median_rep(reps):
    return sorted(reps, key=lambda x: x[0] if isinstance(x, tuple) else x)[len(reps) // 2]


class ConfigRun:
    """Device buffers and launches of one workload's step (all its rounds)."""

    def __init__(self, w: W.Workload, torch, dora, stream, phases: PhaseLog):
        self.w, self.torch, self.dora, self.stream, self.phases = w, torch, dora, stream, phases
        self.rounds = W.generate(w)
        self.R = len(self.rounds)
        self.max_seqlen = [int(r.keep.max()) for r in self.rounds]
        self.sum_keep = [r.total_keep for r in self.rounds]
        self.sets = [self._buffers()]

    def dev(self, a):
        torch = self.torch
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    def _buffers(self, src=None):
        """Inputs (uploaded, or copied from the buffer set `src`) and outputs of
        every round of one step."""
        torch, dora, w = self.torch, self.dora, self.w
        rounds = []
        for i, r in enumerate(self.rounds):
            b = {}
            names = ("scores", "keep", "q", "k", "v") + (("tokens",) if i == 0 else ())
            for name in names:
                b[name] = src[i][name].clone() if src is not None else self.dev(getattr(r, name))
            sk = r.total_keep
            dt = rounds[0]["tokens"].dtype if i > 0 else b["tokens"].dtype
            b["idx"] = torch.empty(sk, dtype=torch.int32, device="cuda")
            b["cu"] = torch.empty(w.B + 1, dtype=torch.int32, device="cuda")
            b["packed"] = torch.empty((sk, w.C), dtype=dt, device="cuda")
            b["out"] = torch.empty_like(b["q"])
            b["ws"] = dora.new_workspace(w.B, w.H, self.max_seqlen[i])
            b["st"] = dora.new_status()
            rounds.append(b)
        return rounds

    def launches(self, bs):
        """The step's launches in order: (kernel key, round, callable)."""
        dora, w, stream = self.dora, self.w, self.stream
        out = []
        for i in range(self.R):
            b = bs[i]
            prev = bs[i - 1] if i > 0 else None
            sk, ms = self.sum_keep[i], self.max_seqlen[i]

            def sp(b=b, prev=prev, sk=sk, ms=ms):
                dora.dora_select_pack_plan(
                    b["scores"], b["keep"], b["tokens"] if prev is None else prev["packed"], w.H, ms, sk, b["ws"],
                    cu_in=None if prev is None else prev["cu"], N=None if prev is None else w.N,
                    idx_out=b["idx"], cu_out=b["cu"], packed_out=b["packed"], cap_rows=sk, dev_status=b["st"],
                    stream=stream)

            def at(b=b, ms=ms):
                dora.dora_varlen_attn_execute(b["q"], b["k"], b["v"], b["cu"], ms, b["ws"], out=b["out"],
                                              dev_status=b["st"], stream=stream)

            out += [("select_pack", i, sp), ("attn", i, at)]
        return out

    def step(self, bs, evs=None):
        ls = self.launches(bs)
        if evs is not None:
            evs[0].record(self.stream)
        for j, (key, _, fn) in enumerate(ls):
            fn()
            self.phases.count(key)
            if evs is not None:
                evs[j + 1].record(self.stream)

    def check_status(self, sets=None):
        for bs in sets or self.sets:
            for b in bs:
                st = int(b["st"].item())
                assert st == 0, f"{self.w.name}: device status {st}"

    def plan_items(self, i: int) -> tuple:
        """(items, queries per item) of round i's plan, read from the plan header."""
        hdr = self.sets[0][i]["ws"][:32].view(self.torch.int32).cpu().numpy()
        return int(hdr[2]), int(hdr[7])

    def host_outputs(self):
        torch = self.torch
        res = []
        for b in self.sets[0]:
            def bits(t):
                return t.view(torch.int16).cpu().numpy().view(np.uint16) if t.dtype == torch.bfloat16 \
                    else t.cpu().numpy()
            res.append({"idx": b["idx"].cpu().numpy(), "cu": b["cu"].cpu().numpy(),
                        "packed": bits(b["packed"]), "out": bits(b["out"])})
        return res


CAPTURE_FAILURES = []


def capture(torch, stream, body, phases=None):
    """body()'s launches (all on `stream`, a non-default stream) captured
    into a HIP graph, not run.  The entry points allocate nothing, set no
    memory and never synchronise, so a timed loop can be replayed as one
    graph: the host's per-call cost (the Python binding takes several
    microseconds a call) then no longer bounds short kernels."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    if phases is not None:
        phases.paused = True
    try:
        with torch.cuda.graph(g, stream=stream):
            body()
    except RuntimeError as e:  # the loop is then timed eagerly, and the line says so
        print(f"[bench] graph capture failed ({e}); timing eagerly", file=sys.stderr, flush=True)
        CAPTURE_FAILURES.append(str(e))
        torch.cuda.synchronize()
        return None
    finally:
        if phases is not None:
            phases.paused = False
    torch.cuda.synchronize()
    return g


def time_steps(run: ConfigRun, sets, args, tag: str):
    """Median over repeats of the step time (ms) and of each launch's duration
    (ms, HIP events around every kernel).  Step i uses sets[i % len(sets)].
    Each repeat times K steps twice: bare (events only at the two ends) and
    with events around every kernel (an event between two kernels adds a few
    microseconds of dispatch latency to the interval, so these are upper
    bounds)."""
    torch, stream, phases = run.torch, run.stream, run.phases
    phases.start(f"{run.w.name}:{tag}:warmup")
    for i in range(args.warmup):
        run.step(sets[i % len(sets)])
    torch.cuda.synchronize()
    n = 2 * run.R
    keys = [k for k, _, _ in run.launches(sets[0])]

    def steps():
        for i in range(args.steps):
            run.step(sets[i % len(sets)])

    g = None if args.eager else capture(torch, stream, steps, phases)
    if g is not None:
        g.replay()  # the graph's first replay, untimed
        for _ in range(args.steps):
            phases.count(*keys)
        torch.cuda.synchronize()
    reps = []
    for rep in range(args.repeats):
        phases.start(f"{run.w.name}:{tag}:bare")
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record(stream)
        if g is not None:
            g.replay()
            for _ in range(args.steps):
                phases.count(*keys)
        else:
            steps()
        t1.record(stream)
        torch.cuda.synchronize()
        step_ms = t0.elapsed_time(t1) / args.steps
        phases.start(f"{run.w.name}:{tag}:events")
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n + 1)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            run.step(sets[i % len(sets)], evs[i])
        torch.cuda.synchronize()
        per = [float(np.mean([e[j].elapsed_time(e[j + 1]) for e in evs])) for j in range(n)]
        reps.append((step_ms, per))
        print(f"[bench] {run.w.name} {tag} repeat {rep}: {step_ms * 1e3:.1f} us/step (per kernel with events: "
              + ", ".join(f"{k}{r} {p * 1e3:.1f}" for (k, r, _), p in zip(run.launches(sets[0]), per)) + ")",
              file=sys.stderr, flush=True)
    run.check_status(sets)
    return _median_rep(reps)


def time_calls(torch, stream, fn, args, phases=None, tag=None, keys=()):
    """Median over repeats of the mean time (ms) of `steps` back-to-back calls
    of fn (after `warmup` calls), HIP events at the two ends; the calls are
    replayed as one HIP graph unless --eager."""
    if phases is not None:
        phases.start(f"{tag}:warmup")
    for _ in range(args.warmup):
        fn()
        if phases is not None:
            phases.count(*keys)

    def calls():
        for _ in range(args.steps):
            fn()
            if phases is not None:
                phases.count(*keys)

    g = None if args.eager else capture(torch, stream, calls, phases)
    if g is not None:
        g.replay()  # untimed
        if phases is not None:
            for _ in range(args.steps):
                phases.count(*keys)
        torch.cuda.synchronize()
    reps = []
    for _ in range(args.repeats):
        if phases is not None:
            phases.start(f"{tag}:timed")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        if g is not None:
            g.replay()
            if phases is not None:
                for _ in range(args.steps):
                    phases.count(*keys)
        else:
            calls()
        e1.record(stream)
        torch.cuda.synchronize()
        reps.append(e0.elapsed_time(e1) / args.steps)
    return sorted(reps)[len(reps) // 2]


def bench_config(run: ConfigRun, args) -> dict:
    """Step timing (bare and per kernel), each kernel alone back to back on
    the same buffers, and the rates, for every round of one workload."""
    torch, stream, w = run.torch, run.stream, run.w
    step_ms, per = time_steps(run, run.sets, args, "warm")
    ls = run.launches(run.sets[0])
    alone = []
    for key, i, fn in ls:
        alone.append(time_calls(torch, stream, fn, args, run.phases, f"{w.name}:alone:{key}{i}", (key,)))
    run.check_status()
    peak = MFMA_PEAK_TFLOPS[w.dtype]
    rec = {"B": w.B, "N": w.N, "H": w.H, "C": w.C, "dtype": w.dtype, "rounds": run.R,
           "sum_keep": run.sum_keep, "max_seqlen": run.max_seqlen,
           "sum_keep_sq": [int(np.sum(r.keep.astype(np.int64) ** 2)) for r in run.rounds],
           "us_per_step": step_ms * 1e3, "packed_tokens_per_s": sum(run.sum_keep) / (step_ms * 1e-3),
           "select_pack": [], "attention": []}
    for i, r in enumerate(run.rounds):
        n_items, q_tile = run.plan_items(i)
        sp_b = select_pack_bytes(w, r.keep, r.n_in, n_items, packed_in=i > 0)
        sp_in, sp_al = per[2 * i], alone[2 * i]
        rec["select_pack"].append({
            "algorithmic_bytes": sp_b, "us_in_step_events": sp_in * 1e3, "us_alone": sp_al * 1e3,
            "GBs_alone": sp_b / (sp_al * 1e-3) / 1e9, "hbm_frac_alone": sp_b / (sp_al * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "GBs_in_step": sp_b / (sp_in * 1e-3) / 1e9,
            "tokens_per_s_alone": r.total_keep / (sp_al * 1e-3), "plan_items": n_items, "q_tile": q_tile})
        fl, ab = attn_flops(w, r.keep), attn_bytes(w, r.keep)
        at_in, at_al = per[2 * i + 1], alone[2 * i + 1]
        rec["attention"].append({
            "flops": fl, "algorithmic_bytes": ab, "us_in_step_events": at_in * 1e3, "us_alone": at_al * 1e3,
            "tflops_in_step": fl / (at_in * 1e-3) / 1e12, "mfma_frac_in_step": fl / (at_in * 1e-3) / 1e12 / peak,
            "tflops_alone": fl / (at_al * 1e-3) / 1e12, "mfma_frac_alone": fl / (at_al * 1e-3) / 1e12 / peak,
            "GBs_in_step": ab / (at_in * 1e-3) / 1e9, "GBs_alone": ab / (at_al * 1e-3) / 1e9,
            "attainable_tflops": min(peak, fl / ab * HBM_PEAK_GBS / 1e3)})
    print(f"[bench] {w.name}: {step_ms * 1e3:.1f} us/step; alone: "
          + ", ".join(f"{k}{i} {a * 1e3:.1f} us" for (k, i, _), a in zip(ls, alone)), file=sys.stderr, flush=True)
    return rec


def attn_errors(got_bits: np.ndarray, want: np.ndarray, dtype: str):
    got = (W.bf16_bits_to_f32(got_bits) if dtype == "bf16" else got_bits).astype(np.float64)
    d = np.abs(got - want)
    return float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0, bool(np.all(np.isfinite(got)))


def oracle_leg(run_rounds, gpu_out, w: W.Workload, passes: int, threads: int):
    """The oracle as it stands, on this host's cores, over the whole step
    (every round): select/pack and attention timed separately (median of
    `passes`), and its outputs compared with the GPU outputs of the timed
    step: idx, cu_seqlens and the packed rows bit for bit, attention within
    the stated tolerance over every element."""
    import oracle
    t_sp, t_at = [], []
    outs = None
    for p in range(passes):
        res = []
        tok, cu_prev = None, None
        a_sp = a_at = 0.0
        for i, r in enumerate(run_rounds):
            t0 = time.perf_counter()
            if i == 0:
                idx, cu, packed, st = oracle.select_pack(r.scores, r.keep, r.tokens)
            else:
                idx, cu, packed, st = oracle.select_pack(r.scores, r.keep, tok, cu_in=cu_prev, N=w.N)
            t1 = time.perf_counter()
            o = oracle.varlen_attn(r.q, r.k, r.v, cu, w.dtype, threads=threads)
            t2 = time.perf_counter()
            assert st == 0
            a_sp += t1 - t0
            a_at += t2 - t1
            res.append((idx, cu, packed, o))
            tok, cu_prev = packed, cu
        t_sp.append(a_sp)
        t_at.append(a_at)
        outs = res
    parity = {"ok": True, "rounds": []}
    for i, ((idx, cu, packed, o), g) in enumerate(zip(outs, gpu_out)):
        mx, mean, finite = attn_errors(g["out"], o, w.dtype)
        tol = (mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS) if w.dtype == "bf16" else mx <= F32_MAX_ABS
        rp = {"idx_bit_exact": bool(np.array_equal(g["idx"], idx)), "cu_bit_exact": bool(np.array_equal(g["cu"], cu)),
              "packed_bit_exact": bool(np.array_equal(g["packed"], packed)),
              "attn_max_abs": mx, "attn_mean_abs": mean, "attn_elements": int(o.size),
              "attn_within_tolerance": bool(tol and finite)}
        rp["ok"] = rp["idx_bit_exact"] and rp["cu_bit_exact"] and rp["packed_bit_exact"] and rp["attn_within_tolerance"]
        parity["ok"] = parity["ok"] and rp["ok"]
        parity["rounds"].append(rp)
    parity["tolerance"] = ({"attn_max_abs": BF16_MAX_ABS, "attn_mean_abs": BF16_MEAN_ABS} if w.dtype == "bf16"
                           else {"attn_max_abs": F32_MAX_ABS})
    sp, at = statistics.median(t_sp), statistics.median(t_at)
    sk = sum(r.total_keep for r in run_rounds)
    fl = sum(attn_flops(w, r.keep) for r in run_rounds)
    cpu = {"value": sk / (sp + at), "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "select_pack_s": sp, "select_pack_tokens_per_s": sk / sp, "attn_s": at, "attn_gflops": fl / at / 1e9,
           "passes": passes}
    return cpu, parity


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--repeats", type=int, default=5)
    ap.add_argument("--workload", default=W.HEADLINE, choices=sorted(W.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (CPU baseline and parity of the timed outputs)")
    ap.add_argument("--no-configs", action="store_true", help="time the headline workload only")
    ap.add_argument("--cold-sets", type=int, default=3,
                    help="also time the step rotating through this many buffer sets (cold MALL); <= 1: off")
    ap.add_argument("--no-peaks", action="store_true", help="skip measuring the copy and MFMA peaks")
    ap.add_argument("--no-adjacent", action="store_true",
                    help="skip the adjacent entry points (residual, actor, LC1, FLOPs, Plackett-Luce)")
    ap.add_argument("--eager", action="store_true",
                    help="time the loops as eager back-to-back launches instead of one HIP graph replay")
    ap.add_argument("--no-large-batch", action="store_true",
                    help="skip the select/pack runs at 8192 and 65536 images (their launches would mix "
                         "into the per-launch counter averages of the headline select/pack)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before timing, run one plain device copy of MIB MiB (a reference dispatch "
                         "for scaling hardware byte counters)")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch (from rocprofv3 counters), if present")
    ap.add_argument("--phase-log", metavar="FILE", help="write the launch counts of every timed phase here")
    ap.add_argument("--summarize-pmc", metavar="DIR",
                    help="print matrix-unit / LDS counter summaries from rocprofv3 --pmc runs under DIR/*/")
    ap.add_argument("--summarize-profile", metavar="DIR",
                    help="no benchmark: summarise rocprofv3 output under DIR/{stats,fetch,write} "
                         "for --workload and update --traffic-json (kernel trace split by --phase-log)")
    args = ap.parse_args()
    if args.summarize_pmc:
        return summarize_pmc(args.summarize_pmc, args.workload)
    if args.summarize_profile:
        return summarize_profile(args.summarize_profile, args.workload, args.traffic_json,
                                 args.calibrate_copy or 256, args.phase_log)

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path shards by image; see the design notes).", file=sys.stderr)
        return 2

    import torch
    import paper_2609_34325_amd as dora

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dora.load_library()
    torch.cuda.set_device(0)
    # A stream of its own (graph capture needs a non-default stream), current
    # for everything the bench does.
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    phases = PhaseLog()
    w = W.WORKLOADS[args.workload]
    head = ConfigRun(w, torch, dora, stream, phases)
    r = head.rounds[0]
    print(f"[bench] {w.name}: B={w.B} N={w.N} H={w.H} C={w.C} {w.dtype} sum_keep={r.total_keep}",
          file=sys.stderr, flush=True)
    sk = sum(head.sum_keep)
    if args.calibrate_copy > 0:
        src = torch.ones(args.calibrate_copy * 2 ** 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Warm: the same buffers every step, as in deployment, where the producing
    # kernel has just written the inputs; then each kernel alone, back to back
    # (attention alone: Q/K/V/O resident in the MALL).
    rec = bench_config(head, args)
    head_out = head.host_outputs()
    ms_step = rec["us_per_step"] * 1e-3
    sp0, at0 = rec["select_pack"][0], rec["attention"][0]

    # Cold: rotate through enough buffer sets that one rotation exceeds twice
    # the 256 MB MALL, so every step's inputs come from HBM.
    cold = None
    if args.cold_sets > 1 and head.R == 1:
        set_bytes = sum(t.numel() * t.element_size() for t in head.sets[0][0].values())
        cold_sets = [head.sets[0]] + [head._buffers(head.sets[0]) for _ in range(args.cold_sets - 1)]
        c_step, c_per = time_steps(head, cold_sets, args, "cold")
        c_sel, c_attn = c_per[0], c_per[1]
        cold = {"sets": args.cold_sets, "bytes_per_set": set_bytes, "ms_per_step": c_step,
                "value": sk / (c_step * 1e-3),
                "us": {"select_pack_plan": c_sel * 1e3, "attention": c_attn * 1e3, "step": c_step * 1e3},
                "attn_GBs": at0["algorithmic_bytes"] / (c_attn * 1e-3) / 1e9,
                "attn_tflops": at0["flops"] / (c_attn * 1e-3) / 1e12,
                "select_pack_GBs": sp0["algorithmic_bytes"] / (c_sel * 1e-3) / 1e9}
        cold["attn_mfma_frac"] = cold["attn_tflops"] / MFMA_PEAK_TFLOPS[w.dtype]
        cold["select_pack_hbm_frac"] = cold["select_pack_GBs"] / HBM_PEAK_GBS
        # The cold sets stay for the residual leg below.
    else:
        cold_sets = None

    extras = {} if args.no_adjacent else adjacent_legs(head, cold_sets, args, torch, dora, stream, phases)
    del cold_sets
    main_bufs = head.sets
    head.sets = None
    del main_bufs
    torch.cuda.empty_cache()

    # The other workloads, each with a record of its own.
    configs, runs = {}, {}
    if not args.no_configs:
        for name in CONFIG_ORDER:
            if name == w.name:
                continue
            cr = ConfigRun(W.WORKLOADS[name], torch, dora, stream, phases)
            configs[name] = bench_config(cr, args)
            runs[name] = (cr.rounds, cr.host_outputs())
            cr.sets = None
            del cr
            torch.cuda.empty_cache()

    peaks = {} if args.no_peaks else measure_peaks(torch, stream)
    traffic = load_traffic(args.traffic_json, w.name)
    peak = MFMA_PEAK_TFLOPS[w.dtype]

    # The dominant kernel (attention) on the matrix-unit roofline, at its
    # in-step duration; the HBM view and the MALL-resident timing beside it.
    fl, ab = at0["flops"], at0["algorithmic_bytes"]
    at_in = at0["us_in_step_events"] * 1e-6
    intensity = fl / ab
    roofline = {"bound": "mfma", "achieved": fl / at_in / 1e12, "peak": peak, "unit": "TFLOP/s",
                "frac": fl / at_in / 1e12 / peak,
                "kernel": "attn_fwd_bf16_kernel" if w.dtype == "bf16" else "attn_fwd_f32_kernel",
                "traffic": traffic.get("attn"), "flops": fl, "algorithmic_bytes": ab,
                "duration_us": at0["us_in_step_events"],
                "duration_source": "HIP events around the kernel inside the step (an upper bound: includes "
                                   "the dispatch gap after the preceding event)",
                "intensity_flop_per_byte": intensity, "ridge_flop_per_byte": peak * 1e3 / HBM_PEAK_GBS,
                "attainable_tflops": at0["attainable_tflops"],
                "frac_of_attainable": fl / at_in / 1e12 / at0["attainable_tflops"],
                "hbm_view": {"achieved": ab / at_in / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": ab / at_in / 1e9 / HBM_PEAK_GBS},
                "resident": {"regime": "attention alone, back to back on one Q/K/V/O set resident in the MALL",
                             "us": at0["us_alone"], "tflops": at0["tflops_alone"], "mfma_frac": at0["mfma_frac_alone"],
                             "GBs": at0["GBs_alone"]}}
    roofline["hbm_view"].update(copy_fracs(roofline["hbm_view"]["achieved"], peaks))
    if "mfma_bf16_TFLOPs" in peaks and w.dtype == "bf16":
        roofline["frac_of_measured_mfma"] = roofline["achieved"] / peaks["mfma_bf16_TFLOPs"]
    sp_b, sp_al = sp0["algorithmic_bytes"], sp0["us_alone"] * 1e-6
    roofline_sp = {"bound": "hbm", "kernel": "select_pack_kernel", "achieved": sp_b / sp_al / 1e9,
                   "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": sp_b / sp_al / 1e9 / HBM_PEAK_GBS,
                   "traffic": traffic.get("select_pack"), "algorithmic_bytes": sp_b, "duration_us": sp0["us_alone"],
                   "duration_source": "dora_select_pack_plan alone, back to back on the same buffers",
                   "in_step_events": {"us": sp0["us_in_step_events"], "GBs": sp0["GBs_in_step"],
                                      "frac": sp0["GBs_in_step"] / HBM_PEAK_GBS}}
    roofline_sp.update(copy_fracs(roofline_sp["achieved"], peaks))

    result = {
        "metric": METRIC,
        "value": sk / ms_step * 1e3,
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
                   "rounds": head.R, "sum_keep": rec["sum_keep"][0] if head.R == 1 else rec["sum_keep"],
                   "sum_keep_sq": rec["sum_keep_sq"][0] if head.R == 1 else rec["sum_keep_sq"],
                   "max_seqlen": rec["max_seqlen"][0] if head.R == 1 else rec["max_seqlen"]},
        "roofline": roofline,
        "roofline_select_pack": roofline_sp,
        "select_pack_tokens_per_s": sp0["tokens_per_s_alone"],
        "attn_tflops": roofline["achieved"],
        "us": {"select_pack_plan_in_step": sp0["us_in_step_events"], "attention_in_step": at0["us_in_step_events"],
               "select_pack_plan_alone": sp0["us_alone"], "attention_alone": at0["us_alone"],
               "step": ms_step * 1e3},
        "repeats": args.repeats,
        "regime": "warm: the same input buffers every step",
        "timing": ("eager back-to-back launches" if args.eager else
                   f"eager back-to-back launches where graph capture failed ({len(CAPTURE_FAILURES)} loops)"
                   if CAPTURE_FAILURES else
                   "the K timed steps (and each kernel's K calls alone) replayed as one HIP graph; in-step kernel "
                   "durations from an eager loop with HIP events around every kernel"),
        "cold": cold,
        "measured_peaks": peaks,
        "parity": None,
    }
    result.update(extras)
    for k in ("residual_select_pack", "lc1_readout"):
        if k in result:
            result[k]["traffic"] = traffic.get("residual" if k.startswith("residual") else "lc1")
            result[k].update(copy_fracs(result[k]["achieved"], peaks))

    if not args.no_cpu_baseline:
        threads = len(os.sched_getaffinity(0))
        print("[bench] oracle leg: CPU baseline and parity of the timed outputs", file=sys.stderr, flush=True)
        cpu, parity = oracle_leg(head.rounds, head_out, w, 5, threads)
        # one thread, for scale
        import oracle
        t1 = []
        for _ in range(2):
            t0 = time.perf_counter()
            idx, cu, _, _ = oracle.select_pack(r.scores, r.keep, r.tokens)
            oracle.varlen_attn(r.q, r.k, r.v, cu, w.dtype, threads=1)
            t1.append(time.perf_counter() - t0)
        cpu["value_1_thread"] = sk / statistics.median(t1)
        cpu["sample"] = (f"full {w.name} batch (B={w.B}, sum keep={sk}), select+pack+attention, median of 5 passes "
                         f"on {threads} threads ({cpu['select_pack_s'] + cpu['attn_s']:.3f} s each) and of 2 on one "
                         f"thread ({statistics.median(t1):.3f} s each); CPU: {cpu_model()}")
        result["cpu_baseline"] = cpu
        result["parity"] = parity
        for name, (rounds, outs) in runs.items():
            c, p = oracle_leg(rounds, outs, W.WORKLOADS[name], 3, threads)
            configs[name]["cpu_baseline"] = c
            configs[name]["parity"] = p
        print(f"[bench] parity: {w.name} {'ok' if parity['ok'] else 'FAILED'}; "
              + ", ".join(f"{n} {'ok' if c['parity']['ok'] else 'FAILED'}" for n, c in configs.items()),
              file=sys.stderr, flush=True)
    result["configs"] = configs
    if args.phase_log:
        phases.dump(args.phase_log)
    print(json.dumps(result), flush=True)
    return 0


def adjacent_legs(head: ConfigRun, cold_sets, args, torch, dora, stream, phases) -> dict:
    """The entry points beside the path, on the headline batch, each timed on
    its own (events at the two ends of back-to-back calls)."""
    w, r = head.w, head.rounds[0]
    b0 = head.sets[0][0]
    sk = r.total_keep
    out = {}

    # Deletion after the attention residual (the kept rows of tokens +
    # attention output), warm and, with a second attention-output buffer per
    # set, cold.
    a_main = head.dev(W.generate(w, parts=("keep", "attn_out"))[0].attn_out)

    def res_launch(b, a):
        dora.dora_select_pack_residual(b["scores"], b["keep"], b["tokens"], a, idx_out=b["idx"], cu_out=b["cu"],
                                       packed_out=b["packed"], cap_rows=sk, dev_status=b["st"], stream=stream)

    rb = residual_bytes(w, r.keep, r.n_in)
    ms_res = time_calls(torch, stream, lambda: res_launch(b0, a_main), args, phases, "residual:warm", ("residual",))
    res = {"entry": "dora_select_pack_residual", "kernel": "select_pack_residual_kernel", "bound": "hbm",
           "us": ms_res * 1e3, "achieved": rb / (ms_res * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "algorithmic_bytes": rb, "tokens_per_s": sk / (ms_res * 1e-3), "regime": "warm"}
    res["frac"] = res["achieved"] / HBM_PEAK_GBS
    if cold_sets is not None:
        pairs = [(cold_sets[0][0], a_main)] + [(s[0], a_main.clone()) for s in cold_sets[1:]]
        it = [0]

        def rot():
            b, a = pairs[it[0] % len(pairs)]
            it[0] += 1
            res_launch(b, a)

        ms_c = time_calls(torch, stream, rot, args, phases, "residual:cold", ("residual",))
        res["cold"] = {"us": ms_c * 1e3, "achieved": rb / (ms_c * 1e-3) / 1e9,
                       "frac": rb / (ms_c * 1e-3) / 1e9 / HBM_PEAK_GBS}
        del pairs
    head.check_status(cold_sets)
    out["residual_select_pack"] = res
    print(f"[bench] residual select/pack: {ms_res * 1e3:.1f} us warm", file=sys.stderr, flush=True)
    del a_main

    # The deterministic actor's decode that produces the path's inputs (gate +
    # compaction, then budget argmax, keep counts and keep-scores), timed as a
    # pair of launches.
    M = W.budget_outputs(w)
    p_h, logits_h, removal_h = W.actor_outputs(w)
    p_d, logits_d, removal_d = head.dev(p_h), head.dev(logits_h), head.dev(removal_h)
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

    ms_actor = time_calls(torch, stream, actor_pair, args, phases, "actor", ("actor", "actor"))
    assert int(st_a.item()) == 0, f"device status {int(st_a.item())}"
    out["actor_decode"] = {"entries": ["dora_actor_gate", "dora_actor_decode"], "bound": "latency",
                           "us_per_pair": ms_actor * 1e3, "gate_on": int(n_on.item()), "M": M,
                           "note": "two small launches back to back; the cost is launch and dependency latency"}
    print(f"[bench] actor decode: {ms_actor * 1e3:.1f} us per gate+decode pair", file=sys.stderr, flush=True)

    # The LC1 readout input (LayerNorm + segmented mean over the packed rows of
    # the same batch), an HBM-bound segmented reduction.
    x_h, gamma_h, beta_h = W.readout_rows(w, r.keep)
    cu_h = np.concatenate([[0], np.cumsum(r.keep)]).astype(np.int32)
    x_d, cu_d, gamma_d, beta_d = head.dev(x_h), head.dev(cu_h), head.dev(gamma_h), head.dev(beta_h)
    out_d = torch.empty((w.B, 2 * w.C), dtype=torch.float32, device="cuda")
    st_l = dora.new_status()
    ws_l = dora.new_lc1_workspace(w.B, w.C)

    def lc1_call():
        dora.dora_lc1_readout(x_d, cu_d, gamma_d, beta_d, 1e-6, out=out_d, workspace=ws_l, dev_status=st_l,
                              stream=stream)

    ms_lc1 = time_calls(torch, stream, lc1_call, args, phases, "lc1", ("lc1",))
    assert int(st_l.item()) == 0, f"device status {int(st_l.item())}"
    lb = lc1_bytes(w, r.keep)
    out["lc1_readout"] = {"entry": "dora_lc1_readout", "kernel": "lc1_readout_kernel (+ lc1_combine_kernel when split)",
                          "bound": "hbm", "us": ms_lc1 * 1e3, "achieved": lb / (ms_lc1 * 1e-3) / 1e9,
                          "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": lb / (ms_lc1 * 1e-3) / 1e9 / HBM_PEAK_GBS,
                          "algorithmic_bytes": lb, "regime": "warm"}
    print(f"[bench] lc1 readout: {ms_lc1 * 1e3:.1f} us per launch", file=sys.stderr, flush=True)
    del x_d

    # FLOP accounting of the batch's realised trajectories over a 12-block
    # backbone (pruning at block 0 with this batch's keep counts, then none).
    L_blocks = 12
    T = np.vstack([np.full((1, w.B), w.N, np.int32), np.tile(r.keep.astype(np.int32), (L_blocks, 1))])
    T_d = head.dev(np.ascontiguousarray(T))
    f_d = torch.empty(w.B, dtype=torch.int64, device="cuda")
    tot_d = torch.empty(1, dtype=torch.int64, device="cuda")
    st_f = dora.new_status()

    def flops_call():
        dora.dora_trajectory_flops(T_d, w.C, w.N - 1, 16, flops_out=f_d, total_out=tot_d, dev_status=st_f,
                                   stream=stream)

    ms_fl = time_calls(torch, stream, flops_call, args, phases, "flops", ("flops",))
    assert int(st_f.item()) == 0, f"device status {int(st_f.item())}"
    out["trajectory_flops"] = {"entry": "dora_trajectory_flops", "kernel": "trajectory_flops_kernel",
                               "bound": "latency", "us": ms_fl * 1e3, "images": w.B, "blocks": L_blocks,
                               "gflops_per_image": int(tot_d.item()) / w.B / 1e9}

    # The training-time draw (Gumbel-top-k Plackett-Luce deletion of n - keep
    # tokens per image, with its ordered log-probability).
    k_h = (r.n_in - r.keep).astype(np.int32)
    g_h = W.gumbel_noise(w)
    s_d, g_d, k_d = head.dev(r.scores), head.dev(g_h), head.dev(k_h)
    order = torch.empty(int(k_h.sum()) + 1, dtype=torch.int32, device="cuda")
    cu_o = torch.empty(w.B + 1, dtype=torch.int32, device="cuda")
    lp_d = torch.empty(w.B, dtype=torch.float32, device="cuda")
    st_p = dora.new_status()

    def pl_call():
        dora.dora_pl_sample(s_d, g_d, k_d, order_out=order, cu_order_out=cu_o, logprob_out=lp_d,
                            dev_status=st_p, stream=stream)

    ms_pl = time_calls(torch, stream, pl_call, args, phases, "pl", ("pl",))
    assert int(st_p.item()) == 0, f"device status {int(st_p.item())}"
    out["pl_sample"] = {"entry": "dora_pl_sample", "kernel": "pl_kernel", "bound": "latency", "us": ms_pl * 1e3,
                        "draws": int(k_h.sum()), "images": w.B,
                        "note": "one workgroup per image: bitonic sort of the visual keys (in registers up to 1024 words) and a block scan"}
    print(f"[bench] trajectory flops {ms_fl * 1e3:.1f} us, pl sample {ms_pl * 1e3:.1f} us",
          file=sys.stderr, flush=True)
    del s_d, g_d

    # Large batches: past 2048 images a block scan writes cu_seqlens before
    # the gather (DeiT-B's keep rule; scores and keep counts from the seeded
    # host streams, token rows filled on the device from a seeded generator).
    large = []
    for Bl, C in (() if args.no_large_batch else ((8192, 768), (65536, 192))):
        wl = W.Workload(f"{w.name}_B{Bl}", w.seed, Bl, w.N, C // W.HEAD_DIM, w.dtype, w.keep_rule)
        rl = W.generate(wl, parts=("keep", "scores"))[0]
        gen = torch.Generator(device="cuda")
        gen.manual_seed(wl.seed)
        tok = torch.randint(-2 ** 15, 2 ** 15, (Bl, w.N, C), dtype=torch.int16, device="cuda",
                            generator=gen).view(torch.bfloat16)
        sc, kp = head.dev(rl.scores), head.dev(rl.keep)
        skl = rl.total_keep
        idx_l = torch.empty(skl, dtype=torch.int32, device="cuda")
        cu_l = torch.empty(Bl + 1, dtype=torch.int32, device="cuda")
        pk_l = torch.empty((skl, C), dtype=torch.bfloat16, device="cuda")
        st_l2 = dora.new_status()

        def big_call():
            dora.dora_select_pack(sc, kp, tok, idx_out=idx_l, cu_out=cu_l, packed_out=pk_l, cap_rows=skl,
                                  dev_status=st_l2, stream=stream)

        ms_b = time_calls(torch, stream, big_call, args, phases, f"select_pack:B{Bl}", ("scan", "select_pack"))
        assert int(st_l2.item()) == 0, f"device status {int(st_l2.item())}"
        bl = 2 * skl * C * 2 + 4 * (Bl * w.N + skl + 2 * Bl + 1)
        large.append({"B": Bl, "N": w.N, "C": C, "sum_keep": skl, "us": ms_b * 1e3, "algorithmic_bytes": bl,
                      "GBs": bl / (ms_b * 1e-3) / 1e9, "hbm_frac": bl / (ms_b * 1e-3) / 1e9 / HBM_PEAK_GBS,
                      "tokens_per_s": skl / (ms_b * 1e-3)})
        print(f"[bench] select/pack B={Bl} C={C}: {ms_b * 1e3:.1f} us ({large[-1]['GBs']:.0f} GB/s)",
              file=sys.stderr, flush=True)
        del tok, pk_l, idx_l, sc, kp
        torch.cuda.empty_cache()
    out["large_batch_select_pack"] = {"entry": "dora_select_pack", "kernels": ["keep_scan_kernel", "select_pack_kernel"],
                                      "note": "past 2048 images one workgroup scans the keep counts first",
                                      "runs": large}
    return out


if __name__ == "__main__":
    sys.exit(main())
