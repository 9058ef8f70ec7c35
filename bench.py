#!/usr/bin/env python3
"""Benchmark of the MI355X batch-reduce GEMM TPP path.

Headline step: the transformer-encoder MLP block (8192 tokens, 1024 -> 4096 with fused bias +
GELU-tanh, then 4096 -> 1024 with fused bias), bf16 blocked 64x64 tiles, fp32 accumulation:
two batched BRGEMM launches (8192 instances x 16 pairs, then 2048 instances x 64 pairs).
``value`` is BRGEMM TFLOP/s over K timed steps (inputs resident in HBM, nothing between the
launches).  ``roofline`` takes the dominant launch's mean duration over K more steps with a
timing-only (fence-free) HIP event on its stream around each launch.  The same run also
times the other workloads (fp32 single BRGEMM, MLP fully-connected layer, 3x3 convolution with
batchnorm statistics via the Reduce TPP, gathered address-based BRGEMM, the Transform TPP's
transpose and VNNI formatting of a 64 MB tensor, the MLP block's backward pass, the sparse
embedding gather-reduce, and two TPP matrix equations) under ``per_config``,
and the CPU oracle on a bounded sample of the headline workload under ``cpu_baseline``.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

# MI355X published peaks (dense): bf16 MFMA, fp32 MFMA, HBM3E.
PEAK_BF16_TFLOPS = 2516.6
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--settle", type=float, default=3.0,
                    help="seconds of untimed headline steps before the counted warm-up, so that "
                         "the clock has settled under load when the timed steps start")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target wall time of the oracle CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-config", action="store_true")
    ap.add_argument("--traffic-run", action="store_true",
                    help="only launch the calibration copy and the calls of --workloads three "
                         "times each (for rocprofv3 --pmc counter passes), print nothing")
    ap.add_argument("--workloads", default="mlp_block,gathered",
                    help="comma-separated workloads of --traffic-run, in launch order (mlp_block, "
                         "gathered, mlp_fc, conv3x3, fp32_single, mlp_backward)")
    return ap.parse_args()


HERE = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(HERE, "profiles", "traffic_mlp_block_8192tok.txt")
TRAFFIC_GATHERED_FILE = os.path.join(HERE, "profiles", "traffic_gathered_4096x128.txt")
MFMA_FILE = os.path.join(HERE, "profiles", "mfma_mlp_block_8192tok.txt")
COPY_BYTES = 512 << 20   # calibration copy: 512 MiB read, 512 MiB written


def kernel_source_sha() -> str:
    """Hash of the sources that build and choose the BRGEMM kernels (the HBM-traffic counters
    below are valid for exactly these): the brgemm*.hip / brgemm*.h files, the shared internal
    header and the host API that picks the instance."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "paper_2104_05755_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")) and (name.startswith("brgemm") or
                                              name in ("internal.h", "tpp_api.hip")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def _profile_kv(path: str):
    """key = value lines of a committed counter summary, or None when it is missing or was taken
    on kernels other than the current sources."""
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    return kv if kv.get("kernel_source_sha") == kernel_source_sha() else None


def mfma_counters_from_profile(call_index: int, flops_per_launch: int):
    """The MFMA counters of call `call_index` from the committed counter summary: bf16 MFMA work
    (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512, which must equal the algorithmic FLOP), the MFMA busy
    share (SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE x 1024 SIMDs) and the shader clock during
    the launch (GRBM_GUI_ACTIVE over the launch's duration in the same run).  None when the
    summary is missing or the kernels changed since."""
    kv = _profile_kv(MFMA_FILE)
    if kv is None:
        return None
    try:
        mops = float(kv[f"call{call_index}_mfma_mops_bf16"])
        busy = float(kv[f"call{call_index}_mfma_busy_cycles"])
        gui = float(kv[f"call{call_index}_grbm_gui_active"])
        dur_ns = float(kv[f"call{call_index}_duration_ns"])
    except KeyError:
        return None
    out = {"mfma_flop": int(mops * 512), "mfma_flop_over_algorithmic": round(mops * 512 / flops_per_launch, 4),
           "mfma_busy": round(busy / (gui * 1024), 4), "sclk_mhz": round(gui / dur_ns * 1e3, 0),
           "source": os.path.relpath(MFMA_FILE, HERE)}
    for extra in ("tcc_hit", "tcc_miss"):
        if f"call{call_index}_{extra}" in kv:
            out[extra] = int(float(kv[f"call{call_index}_{extra}"]))
    if "tcc_hit" in out and "tcc_miss" in out:
        out["tcc_hit_rate"] = round(out["tcc_hit"] / max(1, out["tcc_hit"] + out["tcc_miss"]), 4)
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def traffic_from_profile(call_index: int, path: str = TRAFFIC_FILE):
    """HBM bytes per launch of call `call_index` from a committed rocprofv3 counter summary (the
    headline calls by default): FETCH_SIZE and WRITE_SIZE of the kernel, each scaled by what the
    same counter read for a copy of known size.  None when the summary is missing or the kernels
    changed since."""
    kv = _profile_kv(path)
    if kv is None:
        return None
    try:
        fetch = float(kv[f"call{call_index}_fetch_kib"]) * float(kv["fetch_scale"])
        write = float(kv[f"call{call_index}_write_kib"]) * float(kv["write_scale"])
    except KeyError:
        return None
    return int(round((fetch + write) * 1024))


def traffic_run(torch, tpp, torch_io, wk, stream, workloads):
    """Launch sequence for the counter passes: 3 copies of COPY_BYTES, then for each workload in
    order 3 launches of each of its calls (the gathered workload's pointer lists reach into pools
    about the size of the MALL)."""
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    make = {"mlp_block": wk.mlp_block, "gathered": wk.CONFIGS[5], "mlp_fc": wk.CONFIGS[2],
            "conv3x3": wk.CONFIGS[3], "fp32_single": wk.CONFIGS[1]}
    for name in workloads:
        if name == "mlp_backward":   # every step of the backward pass (forward with SAVE_PREACT first)
            wl = wk.mlp_backward()
            dev = torch_io.upload(wl)
            sts = [torch_io.prepare_step(st, dev) for st in wl.steps]
            torch.cuda.synchronize()
            for _ in range(3):
                for st in sts:
                    torch_io.launch_step(st, dev, stream)
            torch.cuda.synchronize()
            del dev, sts
            torch.cuda.empty_cache()
            continue
        wl = make[name]()
        dev = torch_io.upload(wl)
        dcs = [torch_io.prepare(c, dev) for c in wl.calls]
        torch.cuda.synchronize()
        for _ in range(3):
            for dc in dcs:
                torch_io.launch(dc, stream)
        torch.cuda.synchronize()
        del dev, dcs
        torch.cuda.empty_cache()


def array_bytes(a) -> int:
    return int(a.nbytes)


def alg_bytes(wl, call) -> int:
    """Compulsory HBM bytes of one call: its operand arrays once, C written (and read when
    beta != 0), bias, offset / pointer lists."""
    arrs = wl.arrays
    n = array_bytes(arrs[call.a]) + array_bytes(arrs[call.b])
    c_elems = call.G * call.m * call.n
    es_c = 4 if call.c_type == "f32" else 2
    n += c_elems * es_c * (2 if call.beta != 0.0 else 1)
    if call.bias:
        n += array_bytes(arrs[call.bias])
    if call.kind == "address":
        n += 16 * call.pairs + 8 * (call.G + 1)
    return n


def time_steps(fns, steps, warmup, torch):
    """Warm up, then time exactly `steps` steps (each fn once per step, in order) between two
    device synchronizations, with nothing else on the stream; returns elapsed seconds."""
    for _ in range(warmup):
        for f in fns:
            f()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        for f in fns:
            f()
    torch.cuda.synchronize()
    return time.perf_counter() - t0


class ClockSampler:
    """Samples the GPU's current GFX clock with `amd-smi metric -c` (a child process) from a thread
    while the headline steps run; `result()` gives the median over samples of the mean over the
    XCDs, in MHz, or None when the tool is missing or prints no clock."""

    def __init__(self):
        import threading
        self.samples, self.stop = [], threading.Event()
        self.thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        import re
        import subprocess
        while not self.stop.is_set():
            try:
                out = subprocess.run(["amd-smi", "metric", "-c", "-g", "0"], capture_output=True,
                                     text=True, timeout=10).stdout
            except (OSError, subprocess.SubprocessError):
                return
            # the GFX_i blocks' current clocks ("CLK: 2100 MHz" right after each "GFX_i:")
            clks = [int(m) for m in re.findall(r"GFX_\d+:\s*\n\s*CLK:\s*(\d+)\s*MHz", out)]
            if not clks:
                return
            self.samples.append(sum(clks) / len(clks))

    def __enter__(self):
        self.thread.start()
        return self

    def __exit__(self, *exc):
        # stop sampling without waiting for the last amd-smi call: a join here would leave the
        # GPU idle (and its clock dropping) right before the timed steps
        self.stop.set()

    def result(self):
        self.thread.join(timeout=15)
        if not self.samples:
            return None
        s = sorted(self.samples)
        return {"sclk_mhz_median": round(s[len(s) // 2], 0), "samples": len(s),
                "min": round(s[0], 0), "max": round(s[-1], 0),
                "how": "amd-smi metric -c during the untimed settle steps (mean of the XCDs' GFX clocks)"}


def settle(fns, seconds, torch):
    """Run whole steps, untimed, for about `seconds` (the clock ramps down under sustained MFMA
    load over the first second or so); returns the time spent."""
    if seconds <= 0:
        return 0.0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            for f in fns:
                f()
        torch.cuda.synchronize()
    return time.perf_counter() - t0


def time_bursts(fns, reps, torch):
    """Mean launch duration (ms) of each fn: `reps` back-to-back launches of it between two HIP
    events recorded on the launch stream (torch's current stream)."""
    out = []
    for f in fns:
        for _ in range(5):
            f()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            f()
        e1.record()
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) / reps)
    return out


class FenceFreeEvents:
    """Timing-only HIP events created with hipEventDisableSystemFence, from the HIP runtime that
    torch loaded (the library resolves to the same one).  With default flags every record is a
    system-scope release, i.e. an L2 writeback and invalidation between the kernels it separates:
    measured on MI355X as 8-17 us more per two-launch step and 0-5 us more per launch."""

    FLAGS = 0x20000000   # hipEventDisableSystemFence

    def __init__(self, torch):
        import ctypes
        torch.cuda.init()
        path = None
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    path = line.split()[-1]
                    break
        if path is None:
            raise RuntimeError("HIP runtime not found in the process")
        self.ct = ctypes
        self.hip = ctypes.CDLL(path)
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = self.ct.c_void_p()
        if self.hip.hipEventCreateWithFlags(self.ct.byref(e), self.FLAGS) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        return e

    def record(self, e, stream):
        if self.hip.hipEventRecord(e, self.ct.c_void_p(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, e0, e1) -> float:
        f = self.ct.c_float()
        if self.hip.hipEventElapsedTime(self.ct.byref(f), e0, e1) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(f.value)

    def destroy(self, e):
        self.hip.hipEventDestroy(e)


def time_cold(fn, reps, torch, stream):
    """Mean duration (ms) of fn with cold caches: before each launch a 512 MiB fill (more than the
    8 x 4 MB of L2 and the 256 MB MALL) evicts the inputs, then fence-free HIP events on the
    launch stream bracket the launch alone."""
    ev = FenceFreeEvents(torch)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    evs = [(ev.create(), ev.create()) for _ in range(reps)]
    torch.cuda.synchronize()
    for r in range(reps):
        flush.fill_(r & 0xFF)
        ev.record(evs[r][0], stream)
        fn()
        ev.record(evs[r][1], stream)
    torch.cuda.synchronize()
    ms = sum(ev.elapsed_ms(a, b) for a, b in evs) / reps
    for a, b in evs:
        ev.destroy(a)
        ev.destroy(b)
    del flush
    return ms


def time_in_steps(fns, steps, torch, stream, chunk=25, lead=3):
    """Mean duration (ms) of each fn as it runs inside the step: `steps` more steps with a
    fence-free HIP event on the launch stream before each launch and after the last one.  The
    steps go in chunks of `chunk`, each behind `lead` untimed steps and followed by a
    synchronisation: the host then stays ahead of the GPU while the timed steps run, so the
    events bracket launches and not host-side gaps (recording hundreds of events in one go can
    stall the host for milliseconds while the GPU drains its queue)."""
    ev = FenceFreeEvents(torch)
    evs = [[ev.create() for _ in range(len(fns) + 1)] for _ in range(min(chunk, steps))]
    sums = [0.0] * len(fns)
    done = 0
    torch.cuda.synchronize()
    while done < steps:
        n = min(chunk, steps - done)
        for _ in range(lead):
            for f in fns:
                f()
        for s in range(n):
            for i, f in enumerate(fns):
                ev.record(evs[s][i], stream)
                f()
            ev.record(evs[s][-1], stream)
        torch.cuda.synchronize()
        for s in range(n):
            for i in range(len(fns)):
                sums[i] += ev.elapsed_ms(evs[s][i], evs[s][i + 1])
        done += n
    for row in evs:
        for e in row:
            ev.destroy(e)
    return [x / steps for x in sums]


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2104_05755_amd as tpp
    from paper_2104_05755_amd import torch_io
    import workloads as wk

    torch.cuda.init()
    dev_name = torch.cuda.get_device_name(0)
    stream = tpp.current_stream()
    if args.traffic_run:
        traffic_run(torch, tpp, torch_io, wk, stream, [w for w in args.workloads.split(",") if w])
        return

    # ---------------- headline: transformer MLP block ----------------
    wl = wk.mlp_block()
    dev = torch_io.upload(wl)
    dcs = [torch_io.prepare(c, dev) for c in wl.calls]
    fns = [lambda dc=dc: torch_io.launch(dc, stream) for dc in dcs]
    with ClockSampler() as clock:
        settle_s = settle(fns, args.settle, torch)
    elapsed = time_steps(fns, args.steps, args.warmup, torch)
    per = time_in_steps(fns, args.steps, torch, stream)
    flops_step = wl.flops
    value = flops_step * args.steps / elapsed / 1e12
    kernel_names = [torch_io.describe(dc) for dc in dcs]
    # dominant kernel = the launch with the largest mean duration
    dom = int(np.argmax(per))
    dom_flops = wl.calls[dom].flops
    achieved = dom_flops / (per[dom] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic_from_profile(dom), "traffic_unit": "bytes per launch",
                "kernel": f"call {dom} ({'GEMM1 1024->4096 bias+GELU' if dom == 0 else 'GEMM2 4096->1024 bias'})",
                "launch_ms": round(per[dom], 4), "flops_per_launch": dom_flops,
                "kernel_instance": kernel_names[dom],
                "counters": mfma_counters_from_profile(dom, dom_flops),
                # the launches' in-step durations add up to about the step time of the
                # event-free steps (a value well above 1 would mean the events timed gaps)
                "launch_sum_over_step": round(sum(per) / (elapsed / args.steps * 1e3), 3)}
    result = {
        "metric": "BRGEMM TFLOP/s (bf16, fp32 acc) and % of MFMA peak per config",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "settle_s": round(settle_s, 2),
        "clock_under_load": clock.result(),
        "data": "synthetic (seeded numpy draws, bf16-rounded; no dataset, random-init weights)",
        "config": {"workload": "transformer MLP block as blocked BRGEMM: 8192 tokens, "
                               "1024->4096 (bias+GELU-tanh) -> 1024 (bias), bf16 64x64 blocks",
                   "tokens": 8192, "hidden": 1024, "intermediate": 4096,
                   "instances": [c.G for c in wl.calls], "pairs_per_instance": [c.count for c in wl.calls],
                   "flops_per_step": flops_step, "kernels": kernel_names,
                   "launch_ms": [round(x, 4) for x in per], "device": dev_name},
        "roofline": roofline,
    }
    del dev, dcs, fns
    torch.cuda.empty_cache()

    if not args.no_per_config:
        result["per_config"] = per_config(args, torch, tpp, torch_io, wk, np, stream)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = run_cpu_baseline(args.cpu_seconds, wl)
    print(json.dumps(result), flush=True)


def per_config(args, torch, tpp, torch_io, wk, np, stream):
    """Each of the other workloads: one launch per call (plus the reduce for the convolution),
    each timed over max(steps, 50) back-to-back launches after a warm-up (inputs warm in L2 and
    the MALL), and for the three small workloads also with cold caches (`cold_us`)."""
    out = {}
    steps = max(args.steps, 50)
    for cfg in (1, 2, 3, 5):
        wl = wk.CONFIGS[cfg]()
        dev = torch_io.upload(wl)
        dcs = [torch_io.prepare(c, dev) for c in wl.calls]
        fns = [lambda dc=dc: torch_io.launch(dc, stream) for dc in dcs]
        red = None
        if wl.reduce is not None:
            r = wl.reduce
            ox = torch.empty(r["m"], device="cuda")
            ox2 = torch.empty(r["m"], device="cuda")
            src = dev[r["src"]]
            flags = tpp.TPP_RED_BY_COLS | tpp.TPP_RED_X | tpp.TPP_RED_X2

            def red_fn(src=src, r=r, ox=ox, ox2=ox2, flags=flags):
                tpp.tpp_reduce(r["m"], r["n"], r["ld"], tpp.TPP_DT_BF16, src, tpp.TPP_RED_SUM,
                               flags, ox, ox2, stream)
            red = red_fn
            fns.append(red)
        time_steps(fns, min(steps, args.warmup), 0, torch)   # warm-up
        per = time_bursts(fns, steps, torch)
        call = wl.calls[0]
        ms = per[0]
        flops = call.flops
        tfl = flops / (ms * 1e-3) / 1e12
        byts = alg_bytes(wl, call)
        gbs = byts / (ms * 1e-3) / 1e9
        peak = PEAK_F32_TFLOPS if call.ab_type == "f32" else PEAK_BF16_TFLOPS
        entry = {"workload": wl.name, "kernel": torch_io.describe(dcs[0]),
                 "descriptor": tpp.tpp_brgemm_describe(dcs[0].handle),
                 "instances": call.G, "pairs": call.pairs, "launch_us": round(ms * 1e3, 2),
                 "tflops": round(tfl, 2), "mfma_frac": round(tfl / peak, 4),
                 "alg_bytes": byts, "hbm_gbs": round(gbs, 1),
                 "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
        if cfg == 5:
            # bytes past L2 per launch, from the counter passes (the gathered blocks come from
            # pools about the size of the MALL, so nearly every one misses L2)
            traffic = traffic_from_profile(0, TRAFFIC_GATHERED_FILE)
            entry["traffic"] = traffic
            if traffic is not None:
                entry["traffic_frac"] = round(traffic / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
        if cfg in (1, 2, 3):
            # the same launch with its inputs evicted from L2 and the MALL (from HBM)
            cold = time_cold(fns[0], 20, torch, stream)
            entry["cold_us"] = round(cold * 1e3, 2)
            entry["cold_hbm_frac"] = round(byts / (cold * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
        if red is not None:
            rb = wl.reduce["m"] * wl.reduce["n"] * 2 + 8 * wl.reduce["m"]
            entry["reduce"] = {"what": "per-channel sum and sum of squares of the conv output "
                                       "(Reduce TPP, by columns, bf16 in)",
                               "launch_us": round(per[1] * 1e3, 2), "alg_bytes": rb,
                               "hbm_gbs": round(rb / (per[1] * 1e-3) / 1e9, 1),
                               "hbm_frac": round(rb / (per[1] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
        out[str(cfg)] = entry
        del dev, dcs, fns
        torch.cuda.empty_cache()
    out.update(transform_entries(args, torch, tpp, stream))
    out["mlp_backward"] = backward_entry(args, torch, tpp, torch_io, wk, stream)
    out["embedding_bag"] = embedding_entry(args, torch, tpp, torch_io, wk, stream)
    out.update(equation_entries(args, torch, tpp, torch_io, wk, stream))
    return out


def equation_entries(args, torch, tpp, torch_io, wk, stream):
    """TPP matrix equations (Sec. 4): the paper's example tree on 4096 x 4096 fp32 tensors, a
    layer norm over 1024 features of 8192 tokens (Reduce TPP, then equations for the statistics
    and the normalization) and a softmax over 512 keys of 32768 columns (Reduce MAX, an exp
    equation, Reduce SUM, a scaling equation), each timed over max(steps, 50) back-to-back runs.
    HBM bound: the algorithmic bytes are every leaf tensor read once and the output written once
    (for the layer norm: X read twice, Y written once; for the softmax: X read twice, X' written
    once and read twice, Y written once)."""
    out = {}
    steps = max(args.steps, 50)
    for name, wl in (("equation_example", wk.equation_example()),
                     ("layernorm", wk.layernorm()), ("softmax", wk.softmax())):
        dev = torch_io.upload(wl)
        sts = [torch_io.prepare_step(st, dev) for st in wl.steps]
        fns = [lambda st=st: torch_io.launch_step(st, dev, stream) for st in sts]
        time_steps(fns, min(steps, args.warmup), 0, torch)   # warm-up
        elapsed = time_steps(fns, steps, 0, torch)
        ms = elapsed / steps * 1e3
        if name == "equation_example":
            st = wl.steps[0]
            byts = 6 * st.m * st.n * 4
            what = f"Tanh(T0) + (T1 x T2) / (T3 - T4), elementwise, {st.m} x {st.n} fp32"
        elif name == "layernorm":
            y = wl.steps[-1]
            byts = 2 * y.m * y.n * 2 + y.m * y.n * 2
            what = (f"layer norm over {y.m} features of {y.n} tokens, bf16 (Reduce, the rs "
                    f"equation, the normalize equation; mu a subtree of both)")
        else:
            y = wl.steps[-1]
            # X read twice (bf16), X' written once and read twice (fp32), Y written (bf16)
            byts = y.m * y.n * (2 * 2 + 3 * 4 + 2)
            what = (f"softmax over {y.m} keys of {y.n} columns, bf16 in and out, fp32 X' "
                    f"(Reduce MAX, exp equation, Reduce SUM, scaling equation)")
        gbs = byts / (ms * 1e-3) / 1e9
        out[name] = {"workload": what, "launch_us": round(ms * 1e3, 2), "launches": len(fns),
                     "alg_bytes": byts, "hbm_gbs": round(gbs, 1),
                     "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
        del dev, sts, fns
        torch.cuda.empty_cache()
    return out


def embedding_entry(args, torch, tpp, torch_io, wk, stream):
    """The sparse embedding gather-reduce (Alg. 5) on the DLRM-style lookup workload: one launch
    timed over max(steps, 50) back-to-back launches.  HBM bound: its algorithmic bytes are every
    listed row once per listing (the gather), the index and bag lists, and the output rows."""
    wl = wk.embedding_bag()
    dev = torch_io.upload(wl)
    st = wl.steps[0]
    pst = torch_io.prepare_step(st, dev)
    f = lambda: torch_io.launch_step(pst, dev, stream)
    time_steps([f], min(max(args.steps, 50), args.warmup), 0, torch)   # warm-up
    ms = time_bursts([f], max(args.steps, 50), torch)[0]
    n_bags = len(wl.arrays["begin"]) - 1
    lookups = int(wl.arrays["begin"][-1])
    es = 4 if st.w_type == "f32" else 2
    byts = lookups * st.E * es + 8 * lookups + 8 * (n_bags + 1) + n_bags * st.E * 4
    gbs = byts / (ms * 1e-3) / 1e9
    del dev, pst
    torch.cuda.empty_cache()
    return {"workload": f"{n_bags} bags of 1..64 lookups ({lookups} in all) into a {st.M} x "
                        f"{st.E} {st.w_type} table ({st.M * st.E * es / 1e6:.0f} MB), fp32 out",
            "launch_us": round(ms * 1e3, 2), "alg_bytes": byts, "hbm_gbs": round(gbs, 1),
            "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
            "lookups_per_s": round(lookups / (ms * 1e-3) / 1e9, 2), "lookups_unit": "G/s"}


def backward_entry(args, torch, tpp, torch_io, wk, stream):
    """The transformer MLP's backward pass at the headline size (see workloads.mlp_backward): the
    four gradient BRGEMMs (the weights read transposed by dZ and dX, the activations by dW2 and
    dW1, GELU_inv fused into dZ) and
    the bias-gradient reduces, timed as one step over K steps (nothing between the launches), and
    each launch's mean duration inside the step from fence-free events.  The forward call that
    keeps the pre-activation (GEMM1 + SAVE_PREACT) runs once before and is timed on its own."""
    wl = wk.mlp_backward()
    dev = torch_io.upload(wl)
    sts = [torch_io.prepare_step(st, dev) for st in wl.steps]
    fns = [lambda st=st: torch_io.launch_step(st, dev, stream) for st in sts]
    fwd, bwd = fns[0], fns[1:]
    steps = max(10, args.steps // 4)
    settle([fwd], 0.5, torch)
    ms_fwd = time_bursts([fwd], steps, torch)[0]
    elapsed = time_steps(bwd, steps, max(3, args.warmup // 10), torch)
    per = time_in_steps(bwd, steps, torch, stream)
    bw_calls = wl.calls[1:]
    bw_flops = sum(c.flops for c in bw_calls)
    launches = []
    names = {"dz": "dZ = (W2^T dY) * gelu'(Z)  [W2 read transposed, GELU_inv fused]",
             "dw2": "dW2 = sum_tokens dY H^T  [H read transposed]", "p2": "db2 (sum over token blocks)",
             "db2": "db2 (sum within a block)", "dx": "dX = W1^T dZ  [W1 read transposed]",
             "dw1": "dW1 = sum_tokens dZ X^T  [X read transposed]", "p1": "db1 (sum over token blocks)",
             "db1": "db1 (sum within a block)"}
    out_name = lambda st: (st.c if isinstance(st, wk.Call) else
                           st.dst if isinstance(st, wk.TransformStep) else st.dst_x)
    brgemm_ms = 0.0
    for i, (st, ms) in enumerate(zip(wl.steps[1:], per), start=1):
        e = {"what": names[out_name(st)], "launch_us": round(ms * 1e3, 2)}
        if isinstance(st, wk.Call):
            tfl = st.flops / (ms * 1e-3) / 1e12
            brgemm_ms += ms
            e.update(kernel=torch_io.describe(sts[i]), instances=st.G,
                     pairs=st.pairs, tflops=round(tfl, 1), mfma_frac=round(tfl / PEAK_BF16_TFLOPS, 4))
        elif isinstance(st, wk.TransformStep):
            byts = 2 * st.G * st.m * st.n * 2
            e.update(alg_bytes=byts, hbm_frac=round(byts / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4))
        else:
            es = 2 if st.in_type == "bf16" else 4
            byts = st.G * st.m * st.n * es
            e.update(alg_bytes=byts, hbm_frac=round(byts / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4))
        launches.append(e)
    out = {"workload": "backward of the transformer MLP block (8192 tokens, 1024 -> 4096 -> 1024, "
                       "bf16 64x64 blocks): dZ, dW2, db2, dX, dW1, db1",
           "ms_per_step": round(elapsed / steps * 1e3, 3),
           "brgemm_flops": bw_flops,
           "step_tflops": round(bw_flops / (elapsed / steps) / 1e12, 1),
           "brgemm_tflops": round(bw_flops / (brgemm_ms * 1e-3) / 1e12, 1),
           "launches": launches,
           "forward_save_preact": {
               "what": "GEMM1 1024->4096 bias+GELU keeping the pre-activation Z (aux store)",
               "kernel": torch_io.describe(sts[0]),
               "launch_us": round(ms_fwd * 1e3, 2),
               "tflops": round(wl.calls[0].flops / (ms_fwd * 1e-3) / 1e12, 1)}}
    del dev, sts, fns
    torch.cuda.empty_cache()
    return out


def transform_entries(args, torch, tpp, stream):
    """Transform TPP on the MLP block's hidden activations (8192 tokens x 4096 features, bf16,
    64 MB): its transpose and its VNNI formatting (alpha 2), each timed over max(steps, 50)
    back-to-back launches.  HBM bound: every entry is read once and written once."""
    m, n = 8192, 4096
    es = 2
    out = {}
    for name, kind, alpha in (("transform_transpose", tpp.TPP_TR_TRANSPOSE, 1),
                              ("transform_vnni", tpp.TPP_TR_VNNI, 2)):
        ld_out = n if kind == tpp.TPP_TR_TRANSPOSE else m * alpha
        groups = m if kind == tpp.TPP_TR_TRANSPOSE else n // alpha
        x = torch.randint(-32768, 32767, (m * n,), dtype=torch.int16, device="cuda")
        o = torch.empty(ld_out * groups, dtype=torch.int16, device="cuda")

        def f(kind=kind, alpha=alpha, ld_out=ld_out, x=x, o=o):
            tpp.tpp_transform(kind, m, n, m, ld_out, tpp.TPP_DT_BF16, alpha, x, o, stream)
        time_steps([f], min(max(args.steps, 50), args.warmup), 0, torch)   # warm-up
        ms = time_bursts([f], max(args.steps, 50), torch)[0]
        byts = 2 * m * n * es
        gbs = byts / (ms * 1e-3) / 1e9
        out[name] = {"workload": f"{name.split('_')[1]} of a {m} x {n} bf16 tensor (64 MB), "
                                 f"alpha {alpha}", "launch_us": round(ms * 1e3, 2),
                     "alg_bytes": byts, "hbm_gbs": round(gbs, 1),
                     "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}
        del x, o
        torch.cuda.empty_cache()
    return out


def run_cpu_baseline(seconds: float, wl):
    """Time the oracle (as it is) on growing samples of GEMM1 instances of the headline workload
    until the sample takes about `seconds`; report TFLOP/s on the threads it used."""
    import numpy as np
    import oracle
    sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "tests"))
    from helpers import run_oracle
    call = wl.calls[0]
    rng = np.random.default_rng(0)
    n = 16
    while True:
        sel = np.sort(rng.choice(call.G, size=min(n, call.G), replace=False))
        t0 = time.perf_counter()
        run_oracle(wl, 0, sel=sel)
        dt = time.perf_counter() - t0
        if dt >= seconds * 0.7 or n >= call.G:
            break
        n = min(call.G, max(2 * n, int(n * seconds / max(dt, 1e-3))))
    flops = 2 * call.m * call.n * call.k * call.count * len(sel)
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.max_threads(),
            "cpu_model": cpu_model(), "kind": "oracle",
            "sample": f"{len(sel)} of {call.G} GEMM1 instances (64x64 output block, 16 pairs of "
                      f"64x64x64) of the headline workload, fp64 loops, {dt:.1f} s"}


if __name__ == "__main__":
    main()
