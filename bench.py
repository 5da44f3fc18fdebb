"""Round-trip throughput of the constant-Q transform on one MI355X.

One step = analysis T (packed FFT, routed band inverse FFTs) followed by
synthesis S (band FFTs, owner overlap-add, packed inverse FFT) over one batch
of synthetic audio resident in HBM. Default workload: 128 signals of 88,200
samples at 22.05 kHz, 55 Hz..fs/2 at 36 bins per octave (the throughput
stress workload). Prints one JSON line. The default line also carries
`train_fwdbwd`: the other batched workload, the training front end (16
signals of 220,500 samples at 44.1 kHz, 40 Hz..fs/2 at 24 bins per octave),
timed as analysis T followed by its adjoint T^dagger, with its own roofline.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--batch B]
                  [--mode roundtrip|step]

--mode step times the differentiable round trip of the paper's second
experiment instead (eager: T, S, squared error against a target, and the
backward pass through the explicit adjoints). --mode fwdbwd times analysis
T followed by its adjoint T^dagger on a random cotangent (the training
front end). --workload long times the full-length round trip of the 60 s
signal and the sliced round trip (slices of 2^17, 50 % overlap), with the
peak workspace of each.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12          # MI355X HBM3E, bytes/s
METRIC = "CQT analysis+synthesis round-trip audio samples/s and % HBM peak; round-trip SNR dB"


# hipEventDisableSystemFence: timing-only events skip the system-scope cache
# writeback and invalidation at record, which would otherwise add to (and
# perturb) the bracketed kernel's measured time
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class HipEvents:
    """A few HIP events through the runtime's C API (timing only)."""

    def __init__(self, n):
        self.rt = ctypes.CDLL("libamdhip64.so")
        self.rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if self.rt.hipEventCreateWithFlags(ctypes.byref(e), HIP_EVENT_DISABLE_SYSTEM_FENCE) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.ev.append(e.value)

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.rt.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for e in self.ev:
            self.rt.hipEventDestroy(ctypes.c_void_p(e))


def strip_c_comments(text):
    """C/C++ source without its comments and with runs of whitespace
    collapsed, so that edits to comments or layout keep the same hash.
    String and character literals are kept as they are."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash():
    """Hash of the library's C++/HIP sources (kernels, launches and plan
    building), comments and whitespace excluded: stored counter summaries
    are reported only while it matches."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_29119_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if not f.endswith((".hip", ".hpp", ".cpp", ".h")):
            continue
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode() + b"\0" + strip_c_comments(fh.read()).encode())
    return h.hexdigest()[:16]


def profile_traffic(workload):
    """{stage: HBM bytes per launch} from the committed counter summary, if it
    was taken on the current kernel sources; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("source_hash") != kernel_source_hash():
        return None
    return {k: v.get("hbm_bytes_per_launch") for k, v in d.get("kernels", {}).items()}


def traffic_from_profiles(workload, kernel):
    """HBM bytes per launch of one kernel (see profile_traffic), or None."""
    t = profile_traffic(workload)
    return None if t is None else t.get(kernel)


def counted_step_bytes(workload, kernels):
    """Counted HBM bytes of one step: the sum over its launches, or None when
    the summary is stale or misses one of them."""
    t = profile_traffic(workload)
    if t is None or any(t.get(k) is None for k in kernels):
        return None
    return float(sum(t[k] for k in kernels))


def stage_elements(label):
    """{stage: elements one launch produces} of a profiled workload's step
    (host-only plans; no GPU needed): coefficients for the band kernels,
    packed-spectrum points for the FFT passes and the overlap-add pass,
    output samples for the sliced overlap-add. label is a workload name, or
    long_full / long_sliced for the two round trips of the long workload."""
    import workloads
    import paper_2609_29119_amd as nc
    w = workloads.WORKLOADS[label.split("_")[0]]
    if label == "long_sliced":
        plan = nc.Plan.sliced(w.fs, w.fmin, w.fmax, w.bins_per_octave, w.slice_len, 16, device=False)
        ops, b = (nc.OP_ANALYSE, nc.OP_SYNTHESISE), 16
    else:
        b = 1 if w.slice_len else w.batch
        plan = nc.Plan(*w.plan_args, batch=b, device=False)
        ops = (nc.OP_ANALYSE, nc.OP_ADJ_ANALYSIS) if w.name == "train" else (nc.OP_ANALYSE, nc.OP_SYNTHESISE)
    L, C = plan.info.packed_len, plan.n_coeffs
    out = {}
    for op in ops:
        for n, by in plan.stage_info(op):
            if n.startswith("band_analysis"):
                e = by / (8.0 * L / C + 8.0)         # (c_b / C) 8 L b + 8 c_b b
            elif n.startswith("band_synthesis"):
                e = by / 16.0                        # 16 c_b b
            elif n == "fft_inv_a_overlap_add":
                e = by / (8.0 * C / L + 8.0)         # (8 C + 8 L) b
            elif n == "sliced_overlap_add":
                e = by / 12.0                        # 6 N b bytes, N / 2 samples per slice
            else:
                e = by / 16.0                        # 16 L b
            out.setdefault(n, e)
    return out


def calib_copies(mb):
    """Device copies of mb MiB (none for 0): the counter runs read FETCH_SIZE
    and WRITE_SIZE on them to scale the kernels' counts to bytes."""
    if not mb:
        return
    import torch
    src = torch.empty(mb * 1024 * 1024 // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def make_plan(w, batch):
    import paper_2609_29119_amd as nc
    if w.layout == "table1":
        fs, N, specs = nc.table1_layout()
        return nc.Plan.from_bands(fs, N, specs, batch=batch)
    return nc.Plan(*w.plan_args, batch=batch)


def describe(w, b, N):
    if w.layout == "table1":
        return f"{w.name}: {b} x {N} samples @ {w.fs:g} Hz, Table 1 multi-resolution layout (154 bands)"
    return (f"{w.name}: {b} x {N} samples @ {w.fs:g} Hz, {w.fmin:g} Hz..fs/2, "
            f"{w.bins_per_octave} bins/oct")


def cpu_baseline(w, x, target_s=12.0, gpu_c=None, gpu_x=None, mode="direct"):
    """The fp64 oracle's round trip (analysis + synthesis) timed on a bounded
    sample of the workload: signal counts double until one run reaches the
    whole batch or target_s seconds; whole-batch passes then repeat until
    about target_s seconds of CPU work have been timed in total.

    With the GPU's coefficients and round-trip signals of the same inputs
    (gpu_c [b][C] complex, gpu_x [b][N]), the last untimed-over result also
    gives their relative L2 error against the oracle on the sampled signals,
    max over the signals.

    mode "direct" is the parity reference (a direct DFT per band); "fft"
    is the same definition with pocketfft per band."""
    import oracle
    from threadpoolctl import threadpool_info
    if w.layout == "table1":
        lay = oracle.build_band_layout(*oracle.table1_specs())
    else:
        lay = oracle.build_layout(*w.plan_args)
    k = 1
    while True:
        t0 = time.perf_counter()
        c_ref = oracle.analyse(lay, x[:k], mode=mode)
        x_ref = oracle.synthesise(lay, c_ref, mode=mode)
        dt = time.perf_counter() - t0
        if dt >= target_s or k >= x.shape[0]:
            break
        k = min(x.shape[0], max(2 * k, int(k * target_s / max(dt, 1e-3))))
    passes, total = 1, dt
    while total < target_s:
        t0 = time.perf_counter()
        c_ref = oracle.analyse(lay, x[:k], mode=mode)
        x_ref = oracle.synthesise(lay, c_ref, mode=mode)
        total += time.perf_counter() - t0
        passes += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    out = {"value": passes * k * w.n_samples / total, "unit": "samples/s", "cores": int(threads),
           "kind": "oracle",
           "sample": f"{passes} pass(es) over {k} of {x.shape[0]} signals, fp64 {mode} band DFTs, "
                     f"analysis+synthesis, {total:.1f} s",
           "host_cpus": len(os.sched_getaffinity(0))}
    if gpu_c is not None and gpu_x is not None:
        out["parity"] = {"signals": k,
                         "coeffs_rel_l2_max": float(oracle.rel_l2(gpu_c[:k], c_ref).max()),
                         "worst_band_rel_l2": float(oracle.band_rel_l2(gpu_c[:k], c_ref, lay.offsets()).max()),
                         "worst_band_max_err_over_rms": float(
                             oracle.band_max_err_over_rms(gpu_c[:k], c_ref, lay.offsets()).max()),
                         "roundtrip_rel_l2_max": float(oracle.rel_l2(gpu_x[:k], x_ref).max())}
    return out


# HIP kernel (rocprofv3 name) -> stage name reported by nsgcqt_stage_info
def stage_of_kernel(name):
    import re
    if re.search(r"\bk_ola\b", name):
        return "sliced_overlap_add"
    m = re.search(r"k_(fwd_a|inv_a|pass_b|band_analysis|band_synthesis|big_a|big_b)<(\d+), (\d+)(?:, (true|false))?>",
                  name)
    if not m:
        return None
    k, nt, ept, inv = m.groups()
    if k == "fwd_a":
        return "fft_fwd_a"
    if k == "inv_a":
        return "fft_inv_a_overlap_add"
    if k == "pass_b":
        return "fft_inv_b" if inv == "true" else "fft_fwd_b"
    if k in ("big_a", "big_b"):
        # one kernel per pass serves both directions
        return "huge_band_" + ("columns" if k == "big_a" else "rows")
    return f"{k}_{nt}x{ept}"


def summarize_profile(trace_dir, fetch_dir, write_dir, workload, command, calib_bytes):
    """Per-kernel durations (kernel trace) and HBM bytes (FETCH_SIZE /
    WRITE_SIZE, KiB per dispatch) scaled by the same counters read on a
    device copy of calib_bytes bytes. Writes profiles/ summaries."""
    import csv
    import glob
    import statistics

    def rows(d, suffix):
        f = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
        return list(csv.DictReader(open(f[0]))) if f else []

    stats = rows(trace_dir, "kernel_stats.csv")
    lines = [f"# Kernel trace: {workload} round trip", "", "Command:", "", "```", command["trace"], "```", "",
             "| kernel | stage | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|---|"]
    for r in stats:
        st = stage_of_kernel(r["Name"]) or "-"
        short = r["Name"].split("(")[0].replace("nsg::", "")
        lines.append(f"| `{short}` | {st} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    out = {"workload": workload, "source_hash": kernel_source_hash(), "commands": command, "kernels": {}}
    per = {}
    for d, cname in ((fetch_dir, "FETCH_SIZE"), (write_dir, "WRITE_SIZE")):
        for r in rows(d, "counter_collection.csv"):
            if r["Counter_Name"] != cname:
                continue
            per.setdefault(r["Kernel_Name"], {}).setdefault(cname, []).append(float(r["Counter_Value"]))
    if not per:
        # a kernel trace without counter runs
        os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
        with open(os.path.join(ROOT, "profiles", f"roundtrip_{workload}.md"), "w") as fh:
            fh.write("\n".join(lines) + "\n")
        print("\n".join(lines))
        return
    copy = [v for k, v in per.items() if "copy" in k.lower()]
    calib = None

    def top(vals):
        # the calibration copies are the largest copy dispatches of the run
        vals = [x for x in vals if x > 0]
        if not vals:
            return 0.0
        m = max(vals)
        return statistics.median([x for x in vals if x >= 0.9 * m])

    if copy and calib_bytes:
        f = top([x for c in copy for x in c.get("FETCH_SIZE", [])])
        w = top([x for c in copy for x in c.get("WRITE_SIZE", [])])
        calib = {"bytes": calib_bytes, "fetch_kib": f, "write_kib": w,
                 "fetch_factor": calib_bytes / 1024.0 / f if f else None,
                 "write_factor": calib_bytes / 1024.0 / w if w else None}
    out["copy_calibration"] = calib
    lines += ["", f"# HBM traffic per launch ({workload})", "", "Commands:", "", "```", command.get("fetch", ""),
              command.get("write", ""), "```", "",
              f"Copy calibration: {json.dumps(calib)}", "",
              "| stage | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes / launch (scaled) |", "|---|---|---|---|"]
    for k, c in per.items():
        st = stage_of_kernel(k)
        if not st:
            continue
        f = statistics.median(c.get("FETCH_SIZE", [float("nan")]))
        w = statistics.median(c.get("WRITE_SIZE", [float("nan")]))
        hb = None
        if calib and calib["fetch_factor"] and calib["write_factor"]:
            hb = f * 1024.0 * calib["fetch_factor"] + w * 1024.0 * calib["write_factor"]
        out["kernels"][st] = {"fetch_kib": f, "write_kib": w, "hbm_bytes_per_launch": hb}
        lines.append(f"| {st} | {f:.0f} | {w:.0f} | {hb if hb is None else f'{hb:.4g}'} |")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"traffic_{workload}.json"), "w") as fh:
        json.dump(out, fh, indent=1)
    with open(os.path.join(ROOT, "profiles", f"roundtrip_{workload}.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


# SQ counters summarised per kernel (one rocprofv3 --pmc run holds at most 8)
SQ_COUNTERS = ("SQ_WAVES", "SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_INSTS_SMEM", "SQ_INSTS_VMEM_RD",
               "SQ_INSTS_VMEM_WR", "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_ACTIVE_INST_VALU",
               "SQ_ACTIVE_INST_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_ANY", "SQ_INSTS_MFMA", "SQ_ACTIVE_INST_ANY",
               "SQ_INSTS_VALU_INT32", "SQ_INSTS_VALU_FMA_F32", "SQ_INSTS_VALU_MUL_F32", "SQ_INSTS_VALU_ADD_F32",
               "SQ_INSTS_VALU_CVT", "SQ_INSTS_BRANCH", "SQ_THREAD_CYCLES_VALU", "SQ_WAIT_INST_LDS")


def summarize_counters(sq_dirs, workload, command, elements):
    """Per-kernel SQ counters (median over the dispatches of each counter
    run) with per-wave and per-element figures (elements as in
    stage_elements). Writes profiles/counters_<workload>.json and .md."""
    import csv
    import glob
    import statistics
    per = {}
    for d in sq_dirs:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                st = stage_of_kernel(r["Kernel_Name"])
                if st and r["Counter_Name"] in SQ_COUNTERS:
                    per.setdefault(st, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    out = {"workload": workload, "source_hash": kernel_source_hash(), "commands": command, "kernels": {}}
    lines = [f"# SQ counters per kernel ({workload})", "", "Commands (one per counter run):", "", "```",
             *command.get("sq", []), "```", "",
             "Per wave: instructions issued; `wait %` = SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES; `valu %` = "
             "SQ_ACTIVE_INST_VALU / SQ_WAVE_CYCLES; `lanes` = SQ_THREAD_CYCLES_VALU / SQ_INSTS_VALU "
             "(active lanes per vector instruction). Per element (a coefficient for the band kernels, a "
             "packed-spectrum point for the FFT passes and the overlap-add pass): vector "
             "lane-instructions, split into int32, fp32 (add, mul, fma) and the rest.", "",
             "| stage | waves | VALU/wave | SALU/wave | LDS/wave | VMEM/wave | MFMA/wave | wait % | valu % | lanes "
             "| VALU lane-instr / element | int32 | fp32 | other |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for st, c in per.items():
        m = {k: statistics.median(v) for k, v in c.items()}
        wv = m.get("SQ_WAVES", 0.0)
        if not wv:
            continue
        k = {"waves": wv}
        for name in SQ_COUNTERS[1:]:
            if name in m:
                k[name] = m[name]
        out["kernels"][st] = k
        g = lambda n: m.get(n, float("nan"))   # noqa: E731
        elems = elements.get(st, float("nan"))
        valu = g("SQ_INSTS_VALU")
        i32, fp = g("SQ_INSTS_VALU_INT32"), g("SQ_INSTS_VALU_ADD_F32") + g("SQ_INSTS_VALU_MUL_F32") + g(
            "SQ_INSTS_VALU_FMA_F32")
        lanes = g("SQ_THREAD_CYCLES_VALU") / valu if valu else float("nan")
        k["valu_lane_instr_per_element"] = 64.0 * valu / elems
        k["active_lanes_per_valu_instr"] = lanes
        lines.append(
            f"| {st} | {wv:.0f} | {valu / wv:.0f} | {g('SQ_INSTS_SALU') / wv:.0f} | {g('SQ_INSTS_LDS') / wv:.0f} | "
            f"{(g('SQ_INSTS_VMEM_RD') + g('SQ_INSTS_VMEM_WR')) / wv:.0f} | {g('SQ_INSTS_MFMA') / wv:.1f} | "
            f"{100 * g('SQ_WAIT_INST_ANY') / g('SQ_WAVE_CYCLES'):.0f} | "
            f"{100 * g('SQ_ACTIVE_INST_VALU') / g('SQ_WAVE_CYCLES'):.0f} | {lanes:.0f} | "
            f"{64 * valu / elems:.0f} | {64 * i32 / elems:.0f} | {64 * fp / elems:.0f} | "
            f"{64 * (valu - i32 - fp) / elems:.0f} |")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"counters_{workload}.json"), "w") as fh:
        json.dump(out, fh, indent=1)
    with open(os.path.join(ROOT, "profiles", f"counters_{workload}.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def time_calls(plan, calls, K, W, use_ev=True):
    """Times a step made of library calls [(op, fn)] on the current stream:
    W untimed steps, then (with use_ev) a short pass with every kernel
    bracketed by HIP events through nsgcqt_set_stage_events, which gives the
    per-kernel table and names the dominant kernel, then K timed steps with
    only the dominant kernel bracketed, on the stream it is launched on.
    Returns the step time (max of the GPU clock and the host wall clock,
    ms), the allocator peak during the timed steps, the per-kernel table and
    the dominant kernel's average duration in the timed steps."""
    import torch
    infos = [plan.stage_info(op) for op, _ in calls]
    names = [n for st in infos for n, _ in st]
    algb = [b for st in infos for _, b in st]
    nev = [2 * len(st) for st in infos]          # a start and an end event per kernel

    armed = [True]      # whether the library may still hold stage events

    def step(evs=None):
        for i, (_, f) in enumerate(calls):
            e = None if evs is None else evs[i]
            if e is not None or armed[0]:
                plan.set_stage_events(e)
                armed[0] = e is not None
            f()
        if armed[0]:
            plan.set_stage_events(None)
            armed[0] = False

    for _ in range(W):
        step()
    torch.cuda.synchronize()
    stages, dom = [], None
    if use_ev:
        kc = min(K, 10)
        per = sum(nev)
        ev = HipEvents(kc * per)
        for i in range(kc):
            base, evs = i * per, []
            for n in nev:
                evs.append(ev.ev[base: base + n])
                base += n
            step(evs)
        torch.cuda.synchronize()
        dur = np.zeros(len(names))
        for i in range(kc):
            base = i * per
            for j in range(len(names)):
                dur[j] += ev.elapsed_ms(ev.ev[base + 2 * j], ev.ev[base + 2 * j + 1])
        dur /= kc
        ev.close()
        for n_, b_, d_ in zip(names, algb, dur):
            stages.append({"kernel": n_, "ms": round(float(d_), 5), "alg_bytes": b_,
                           "GBps": round(b_ / (d_ * 1e-3) / 1e9, 1)})
        dom = int(np.argmax(dur))
    evd = HipEvents(2 * K) if dom is not None else None

    # the timed steps' event arguments, built before the timed region: only
    # the call holding the dominant kernel brackets it, the others record none
    timed_evs = []
    if evd is not None:
        for i in range(K):
            j, evs = dom, []
            for n in nev:
                if 0 <= j < n // 2:
                    lst = [None] * (2 * j) + [evd.ev[2 * i], evd.ev[2 * i + 1]]
                    evs.append((ctypes.c_void_p * len(lst))(*lst))
                else:
                    evs.append(None)
                j -= n // 2
            timed_evs.append(evs)

    def timed_step(i):
        step(timed_evs[i] if timed_evs else None)

    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    mem0 = torch.cuda.memory_allocated()
    t0 = time.perf_counter()
    t_start.record()
    for i in range(K):
        timed_step(i)
    t_stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    alloc = torch.cuda.max_memory_allocated() - mem0
    ms = max(t_start.elapsed_time(t_stop), wall * 1e3) / K
    dom_ms = None
    if evd is not None:
        dom_ms = sum(evd.elapsed_ms(evd.ev[2 * i], evd.ev[2 * i + 1]) for i in range(K)) / K
        evd.close()
    return {"ms": ms, "alloc": alloc, "names": names, "algb": algb, "stages": stages, "dom": dom,
            "dom_ms": dom_ms}


def roofline(names, algb, dom, dom_ms, workload, traffic_ok):
    """The dominant kernel's algorithmic bytes over its measured duration
    against the HBM peak, with its counted traffic from the committed
    counter summary (None when stale or not for this batch)."""
    achieved = algb[dom] / (dom_ms * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": names[dom], "kernel_ms": round(dom_ms, 5),
            "achieved": round(achieved, 1), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": achieved / (HBM_PEAK / 1e9),
            "traffic": traffic_from_profiles(workload, names[dom]) if traffic_ok else None}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="stress")
    ap.add_argument("--batch", type=int, default=0, help="signals per step (default: the workload's)")
    ap.add_argument("--mode", choices=("roundtrip", "step", "fwdbwd"), default="roundtrip")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay timing")
    ap.add_argument("--no-train", action="store_true",
                    help="stress round trip only, without the training front end's T + T^dagger leg")
    ap.add_argument("--no-stage-events", action="store_true",
                    help="time the loop without per-kernel events (for profiler runs)")
    ap.add_argument("--copy-calib-mb", type=int, default=0,
                    help="after timing, run device copies of this many MiB (counter calibration)")
    ap.add_argument("--summarize-profile", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                    help="summarise rocprofv3 outputs into profiles/ and exit")
    ap.add_argument("--commands", default="{}", help="JSON of the profiler commands (for the summary)")
    ap.add_argument("--long-part", choices=("both", "full", "sliced"), default="both",
                    help="long workload: which round trip(s) to time")
    ap.add_argument("--summarize-counters", nargs="+", metavar="SQ_DIR",
                    help="summarise rocprofv3 SQ counter runs into profiles/ and exit")
    args = ap.parse_args()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.workload, json.loads(args.commands),
                           stage_elements(args.workload))
        return
    if args.summarize_profile:
        summarize_profile(*args.summarize_profile, args.workload, json.loads(args.commands),
                          args.copy_calib_mb * 1024 * 1024)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU; a batch shards across GPUs with no "
                          "communication, so --gpus must be 1"}))
        sys.exit(2)

    import torch
    import workloads
    import paper_2609_29119_amd as nc

    w = workloads.WORKLOADS[args.workload]
    if w.slice_len:
        return bench_long(args, w)
    b = args.batch or w.batch
    torch.cuda.init()
    plan = make_plan(w, b)
    x_np = workloads.signals(w, batch=b)
    x = torch.from_numpy(x_np).cuda()
    if args.mode == "step":
        return bench_step(args, w, plan, x)
    if args.mode == "fwdbwd":
        return bench_fwdbwd(args, w, plan, x)
    c = torch.empty((b, plan.n_coeffs), dtype=torch.complex64, device="cuda")
    xr = torch.empty_like(x)
    ws_a = plan.workspace(nc.OP_ANALYSE)
    ws_s = plan.workspace(nc.OP_SYNTHESISE)
    K, W = args.steps, args.warmup
    calls = [(nc.OP_ANALYSE, lambda: plan.analyse(x, out=c, ws=ws_a)),
             (nc.OP_SYNTHESISE, lambda: plan.synthesise(c, out=xr, ws=ws_s))]
    tm = time_calls(plan, calls, K, W, not args.no_stage_events)
    ms, alloc_steps = tm["ms"], tm["alloc"]
    names, algb, stages, dom, dom_ms = tm["names"], tm["algb"], tm["stages"], tm["dom"], tm["dom_ms"]

    def step():
        for _, f in calls:
            f()

    # the same step captured once into a HIP graph and replayed (the paper
    # times round trips under graph replay); the chain records no memsets
    graph_ms = None if args.no_graph else graph_replay_ms(step, K, W)

    calib_copies(args.copy_calib_mb)

    # accuracy of this run's round trip (GPU result against the input)
    xr_np = xr.cpu().numpy().astype(np.float64)
    x64 = x_np.astype(np.float64)
    snr = 10 * np.log10(np.sum(x64 ** 2, axis=1) / np.sum((x64 - xr_np) ** 2, axis=1))

    N, C = plan.n_samples, plan.n_coeffs
    b_alg = (24.0 * N + 16.0 * C) * b              # method's algorithmic bytes per round trip
    value = b * N / (ms * 1e-3)
    out = {
        "metric": METRIC, "value": value, "unit": "samples/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": describe(w, b, N) + ", analysis+synthesis round trip",
                   "batch": b, "n_samples": N, "n_bands": plan.n_bands, "n_coeffs": C},
        "pct_hbm_peak": 100.0 * b_alg / (ms * 1e-3) / HBM_PEAK,
        "alg_bytes_per_step": b_alg,
        # x and c only, without the packed spectrum staged between the passes
        "pct_hbm_peak_bmin": 100.0 * (8.0 * N + 16.0 * C) * b / (ms * 1e-3) / HBM_PEAK,
        "snr_db_min": float(snr.min()),
        "graph_replay_ms_per_step": graph_ms,
        "workspace_bytes_per_signal": max(plan.info.ws_analyse, plan.info.ws_synthesise) / b,
        # allocator peak above what was live before the timed steps (the
        # workspace and outputs are allocated beforehand)
        "alloc_during_steps_bytes": alloc_steps,
    }
    if dom is not None:
        out["roofline"] = roofline(names, algb, dom, dom_ms, w.name, b == w.batch)
        out["stages"] = stages
        counted = counted_step_bytes(w.name, names) if b == w.batch else None
        out["counted_bytes_per_step"] = counted
        out["pct_hbm_peak_counted"] = None if counted is None else 100.0 * counted / (ms * 1e-3) / HBM_PEAK
    if args.workload == "stress" and not args.batch and not args.no_train:
        # the other batched workload: the training front end's T + T^dagger
        wt = workloads.WORKLOADS["train"]
        pt = make_plan(wt, wt.batch)
        xt = torch.from_numpy(workloads.signals(wt)).cuda()
        out["train_fwdbwd"] = fwdbwd_result(wt, pt, xt, K, W, not args.no_stage_events, not args.no_graph)
        del pt, xt
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, x_np, gpu_c=c.cpu().numpy(), gpu_x=xr_np)
        # the same oracle with pocketfft band transforms: the fairer CPU figure
        out["cpu_baseline_fft"] = cpu_baseline(w, x_np, mode="fft")
    print(json.dumps(out), flush=True)


def bench_step(args, w, plan, x):
    """Eager differentiable round trip: xr = S T x, L = sum (xr - t)^2, and
    L.backward() through the explicit adjoints (T^dagger S^dagger)."""
    import torch
    import workloads
    from paper_2609_29119_amd import autograd as ag
    b, N = x.shape
    t = torch.from_numpy(workloads.white(w.cot_seed, b, N)).cuda()
    cqt = ag.CQT(plan)

    def step():
        xg = x.detach().requires_grad_()
        loss = ((cqt.inverse(cqt(xg)) - t) ** 2).sum()
        loss.backward()
        return xg.grad

    K, W = args.steps, args.warmup
    for _ in range(W):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        g = step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / K
    # the gradient is T^dagger S^dagger 2 (S T x - t) ~ 2 T^dagger S^dagger (x - t)
    out = {"metric": "CQT differentiable round-trip step (eager: T, S, squared error, backward through "
                     "the adjoints) audio samples/s",
           "value": b * N / (ms * 1e-3), "unit": "samples/s", "n_gpus": 1, "steps": K, "warmup": W,
           "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f32", "data": "synthetic",
           "config": {"workload": describe(w, b, N) + ", differentiable round-trip step",
                      "batch": b, "n_samples": N, "n_bands": plan.n_bands, "n_coeffs": plan.n_coeffs},
           "grad_finite": bool(torch.isfinite(g).all().item())}
    print(json.dumps(out), flush=True)



def _timed(fn, K, W):
    """Mean wall time per call of fn over K calls after W warm-up calls, with
    the device synchronised on both sides (ms)."""
    import torch
    for _ in range(W):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / K


def graph_replay_ms(step, K, W):
    """Mean time per replay of `step` captured once into a HIP graph (ms),
    after one eager run on a side stream and W untimed replays."""
    import torch
    cur = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(cur)
    with torch.cuda.stream(side):
        step()
    cur.wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(W):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        g.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / K
    del g
    return ms


def fwdbwd_result(w, plan, x, K, W, use_ev=True, graph=True):
    """Analysis T x, then T^dagger y for a fixed random coefficient cotangent
    y (the training front end's forward and backward): step time, rate,
    share of the HBM peak on the method's algorithmic bytes, the roofline
    of the dominant kernel, and the step's time under HIP-graph replay."""
    import torch
    import workloads
    import paper_2609_29119_amd as nc
    b, N = x.shape
    C = plan.n_coeffs
    y = torch.from_numpy(workloads.coeff_cotangent(w.cot_seed, b, C)).cuda()
    c = torch.empty((b, C), dtype=torch.complex64, device="cuda")
    g = torch.empty_like(x)
    ws_a, ws_t = plan.workspace(nc.OP_ANALYSE), plan.workspace(nc.OP_ADJ_ANALYSIS)
    calls = [(nc.OP_ANALYSE, lambda: plan.analyse(x, out=c, ws=ws_a)),
             (nc.OP_ADJ_ANALYSIS, lambda: plan.adjoint(nc.OP_ADJ_ANALYSIS, y, out=g, ws=ws_t))]
    tm = time_calls(plan, calls, K, W, use_ev)
    ms = tm["ms"]
    b_alg = (24.0 * N + 16.0 * C) * b      # T: 12N + 8C, T^dagger: 12N + 8C
    out = {"workload": describe(w, b, N) + ", analysis T then adjoint T^dagger",
           "ms_per_step": ms, "samples_per_s": b * N / (ms * 1e-3),
           "pct_hbm_peak": 100.0 * b_alg / (ms * 1e-3) / HBM_PEAK, "alg_bytes_per_step": b_alg,
           "workspace_bytes_per_signal": max(plan.info.ws_analyse, plan.info.ws_adjoint_analysis) / b}
    out["graph_replay_ms_per_step"] = graph_replay_ms(lambda: [f() for _, f in calls], K, W) if graph else None
    if tm["dom"] is not None:
        out["roofline"] = roofline(tm["names"], tm["algb"], tm["dom"], tm["dom_ms"], w.name, b == w.batch)
        out["stages"] = tm["stages"]
    return out


def bench_fwdbwd(args, w, plan, x):
    """The training front end's T + T^dagger as the headline of its own line."""
    b, N = x.shape
    r = fwdbwd_result(w, plan, x, args.steps, args.warmup, not args.no_stage_events, not args.no_graph)
    calib_copies(args.copy_calib_mb)
    out = {"metric": "CQT analysis forward + adjoint backward audio samples/s and % HBM peak",
           "value": r["samples_per_s"], "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": r["workload"], "batch": b, "n_samples": N, "n_bands": plan.n_bands,
                      "n_coeffs": plan.n_coeffs}, **{k: v for k, v in r.items() if k != "workload"}}
    print(json.dumps(out), flush=True)


def bench_long(args, w):
    """The 60 s signal: full-length round trip and sliced round trip, each
    with its per-kernel table and roofline (the sliced calls' kernels are
    those of one chunk of slices, timed on the first chunk), its plan's
    workspace and the device-memory high-water mark of the calls beyond
    their inputs and outputs. --long-part picks one of the two (profiler
    runs take each alone, so their counters are attributed to it)."""
    import torch
    import workloads
    import paper_2609_29119_amd as nc
    torch.cuda.init()
    x_np = workloads.signals(w)
    x = torch.from_numpy(x_np).cuda()
    N = w.n_samples
    K, W = args.steps, args.warmup
    use_ev = not args.no_stage_events
    res = {}

    def timing(plan, calls, label, b_alg):
        tm = time_calls(plan, calls, K, W, use_ev)
        r = {"ms_per_step": tm["ms"], "samples_per_s": N / (tm["ms"] * 1e-3),
             "alg_bytes_per_step": b_alg, "pct_hbm_peak": 100.0 * b_alg / (tm["ms"] * 1e-3) / HBM_PEAK,
             "alloc_peak_during_calls_bytes": int(tm["alloc"])}
        if tm["dom"] is not None:
            r["roofline"] = roofline(tm["names"], tm["algb"], tm["dom"], tm["dom_ms"], label, True)
            r["stages"] = tm["stages"]
        return r

    if args.long_part in ("both", "full"):
        # full length: one plan over all N samples
        plan = nc.Plan(*w.plan_args, batch=1)
        c = torch.empty((1, plan.n_coeffs), dtype=torch.complex64, device="cuda")
        xr = torch.empty_like(x)
        ws_a, ws_s = plan.workspace(nc.OP_ANALYSE), plan.workspace(nc.OP_SYNTHESISE)
        calls = [(nc.OP_ANALYSE, lambda: plan.analyse(x, out=c, ws=ws_a)),
                 (nc.OP_SYNTHESISE, lambda: plan.synthesise(c, out=xr, ws=ws_s))]
        r = timing(plan, calls, "long_full", 24.0 * N + 16.0 * plan.n_coeffs)
        e = (x_np[0].astype(np.float64) - xr.cpu().numpy()[0])
        r.update({"snr_db": float(10 * np.log10(np.sum(x_np.astype(np.float64) ** 2) / np.sum(e ** 2))),
                  "n_bands": plan.n_bands, "n_coeffs": plan.n_coeffs,
                  "workspace_bytes": max(plan.info.ws_analyse, plan.info.ws_synthesise),
                  "table_bytes": plan.info.table_bytes})
        res["full"] = r
        del plan, c, xr, ws_a, ws_s, calls
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    if args.long_part in ("both", "sliced"):
        # sliced: slices of slice_len, 50 % overlap, 16 slices per chunk
        sp = nc.Plan.sliced(w.fs, w.fmin, w.fmax, w.bins_per_octave, w.slice_len, 16)
        x1 = x[0].contiguous()
        J = sp.slice_count(N)
        cs = torch.empty((J, sp.n_coeffs), dtype=torch.complex64, device="cuda")
        xs = torch.empty_like(x1)
        wa, wsn = sp.workspace(nc.OP_ANALYSE), sp.workspace(nc.OP_SYNTHESISE)
        calls = [(nc.OP_ANALYSE, lambda: sp.sliced_analyse(x1, out=cs, ws=wa)),
                 (nc.OP_SYNTHESISE, lambda: sp.sliced_synthesise(cs, N, out=xs, ws=wsn))]
        # per slice the method's round-trip bytes at slice length
        r = timing(sp, calls, "long_sliced", J * (24.0 * w.slice_len + 16.0 * sp.n_coeffs))
        e = x_np[0].astype(np.float64) - xs.cpu().numpy()
        r.update({"snr_db": float(10 * np.log10(np.sum(x_np.astype(np.float64) ** 2) / np.sum(e ** 2))),
                  "slices": J, "slice_len": w.slice_len, "slices_per_chunk": 16,
                  "coeffs_per_slice": sp.n_coeffs,
                  "workspace_bytes": max(sp.info.ws_analyse, sp.info.ws_synthesise),
                  "table_bytes": sp.info.table_bytes})
        res["sliced"] = r
    calib_copies(args.copy_calib_mb)
    head = res.get("full") or res["sliced"]
    out = {"metric": "CQT analysis+synthesis round-trip audio samples/s (full-length and sliced); peak workspace",
           "value": head["samples_per_s"], "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": head["ms_per_step"], "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": f"{w.name}: 1 x {N} samples @ {w.fs:g} Hz, {w.fmin:g} Hz..fs/2, "
                                  f"{w.bins_per_octave} bins/oct, "
                                  + {"both": "full-length and sliced round trips", "full": "full-length round trip",
                                     "sliced": "sliced round trip"}[args.long_part]},
           **res}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
