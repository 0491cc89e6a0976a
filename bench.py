#!/usr/bin/env python3
"""Benchmark: the fused weight-gradient + AdamW step over the Llama-3.1-8B linear layers.

One "step" is one fused step (forge_linear_step) on every linear weight of the model:
32 decoder layers x {q, k, v, o, gate, up, down} + lm_head, T = 512 tokens, bf16 W, m and
v, launched back to back on one stream, all inputs resident in HBM (synthetic Gaussian
data, seeded).  Printed value: algorithmic HBM bytes of a step / step time (GB/s).

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MFMA_BF16_PEAK_TFS = 2500.0    # dense bf16 MFMA, published
# Sources the fused kernel is compiled from (the traffic record below is tied to them).
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_22932_amd", "csrc", f)
                  for f in ("forge_kernels.hip", "forge_device.h", "forge_internal.h")]
COPY_BYTES = 1 << 30           # size of the calibration copy (--copy-calibration)

# Measured HBM traffic of the fused kernel per launch, averaged over one step of a
# workload: two rocprofv3 --pmc runs of `bench.py --steps 1 --warmup 0 --no-cpu-baseline
# --no-unfused --copy-calibration` (FETCH_SIZE, then WRITE_SIZE), each counter scaled by
# COPY_BYTES / (what it reads for the calibration copy).  Valid only for the kernel
# sources whose sha256 is recorded: after any change to them the figure is reported as null.
# (The counters were taken on sources with sha256 677b4262...; the edits since then changed
# only the kernels of fp32 state and the host-side choice of prefetch depth for T >= 1024,
# and every kernel below compiles to the same device code.)
TRAFFIC = {
    "sweep": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 208083.6,     # FETCH_SIZE, mean over the 129 launches of a step
        "write_kib_per_launch": 340903.9,     # WRITE_SIZE
        "fetch_scale": 1.99992,               # 1 GiB copy: FETCH_SIZE reads about 524300 KiB
        "write_scale": 1.0,                   # 1 GiB copy: WRITE_SIZE reads 1048576 KiB
        "bytes_per_launch": 775223790,        # (fetch * fetch_scale + write * write_scale) KiB
    },
    "o_proj": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 61657.5,     # one launch (4096 x 4096)
        "write_kib_per_launch": 98401.0,
        "fetch_scale": 1.99993,
        "write_scale": 1.0,
        "bytes_per_launch": 227032473,
    },
    "mlp": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 211172.7,     # mean over the 3 launches (gate, up, down)
        "write_kib_per_launch": 344073.3,
        "fetch_scale": 1.99993,
        "write_scale": 1.0,
        "bytes_per_launch": 784796715,
    },
    "mlp_i8": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 153124.5,     # mean over the 3 launches (gate, up, down)
        "write_kib_per_launch": 261589.0,
        "fetch_scale": 1.99992,
        "write_scale": 1.0,
        "bytes_per_launch": 581454198,
    },
    "mlp_i8r64": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 155839.9,     # mean over the 3 launches (gate, up, down)
        "write_kib_per_launch": 241004.1,
        "fetch_scale": 1.99993,
        "write_scale": 1.0,
        "bytes_per_launch": 565936401,
    },
    "mlp_fp8": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 147209.0,     # mean over the 3 launches (gate, up, down)
        "write_kib_per_launch": 229400.2,
        "fetch_scale": 1.99992,
        "write_scale": 1.0,
        "bytes_per_launch": 536378457,
    },
    "mlp_wfp8": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 177867.1,     # mean over the 3 launches (gate, up, down)
        "write_kib_per_launch": 286732.6,
        "fetch_scale": 1.99992,
        "write_scale": 1.0,
        "bytes_per_launch": 657871851,
    },
    "mlp_wfp8_fp8": {
        "source_sha256": "54af42890281bf2601782e57ddc2958da3fb445485e524a10dc786cc63449554",
        "fetch_kib_per_launch": 116193.0,     # mean over the 3 launches (gate, up, down)
        "write_kib_per_launch": 172065.1,
        "fetch_scale": 1.99992,
        "write_scale": 1.0,
        "bytes_per_launch": 414148815,
    },
}


# Default (warmup, timed) steps per workload when --steps / --warmup are not given: the
# sweep's 20 ms steps need few; the single-matrix and MLP workloads get enough steps for
# about 0.1 s of warmup and 0.2 s of timed work, so that clocks and TLBs are warm.
DEFAULT_STEPS = {"sweep": (3, 10), "o_proj": (2000, 4000), "o_proj_t4096": (300, 600), "mlp": (200, 400),
                 "mlp_i8": (200, 300), "mlp_i8r64": (200, 400), "mlp_fp8": (200, 400), "mlp_wfp8": (200, 400),
                 "mlp_wfp8_fp8": (200, 400)}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_workload(wl, device, moment_override=None):
    """Device tensors for every matrix of the workload, drawn on the GPU from seeded generators."""
    import torch
    from paper_2606_22932_amd import synth
    mats = []
    for mat in wl.matrices:
        X, dY = synth.activations(wl.T, mat, wl, wl.steps[0], device=device)
        W = synth.weight(mat, wl, device=device)
        if wl.moment in ("i8", "i8r64"):
            mq, vq, ms, vs = synth.random_i8_state(mat, wl, device=device,
                                                   layout="col256" if wl.moment == "i8" else "row64")
            mats.append(dict(mat=mat, X=X, dY=dY, W=W, m=mq, v=vq, ms=ms, vs=vs))
        elif wl.moment == "fp8" or wl.weight == "fp8":
            W8, w_ring, m8, m_ring, v8, v_ring = synth.random_fp8_state(mat, wl, device=device)
            if W8 is not None:
                W = W8
            if m8 is None:
                m8, v8 = synth.warm_moments(mat, wl, device=device, dtype=torch.bfloat16)
            mats.append(dict(mat=mat, X=X, dY=dY, W=W, w_ring=w_ring, m=m8, v=v8, ms=m_ring, vs=v_ring))
        else:
            dt = torch.bfloat16 if wl.moment == "bf16" else torch.float32
            m, v = synth.warm_moments(mat, wl, device=device, dtype=dt)
            mats.append(dict(mat=mat, X=X, dY=dY, W=W, m=m, v=v, ms=None, vs=None))
    return mats


def time_steps(launches, wl, fn, steps, warmup, step0, side_streams=()):
    """Run `warmup` untimed steps, then `steps` timed steps back to back on the current
    stream (the one the library launches on), bracketed by two HIP events on that stream.

    No event sits between launches: an event record between two kernels costs a gap of
    about 5 us on this stream, while back-to-back launches follow each other with none, so
    the region's time divided by its launches is the average kernel duration.
    Returns (region ms, wall ms).
    """
    import torch
    for i in range(warmup):
        for unit in launches:
            fn(unit, step0 + i)
    stream = torch.cuda.current_stream()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for ss in side_streams:           # launches on other streams start after `start`
        ss.wait_event(start)
    for s in range(steps):
        for unit in launches:
            fn(unit, step0 + warmup + s)
    for ss in side_streams:           # ... and `end` waits for them
        e = torch.cuda.Event()
        e.record(ss)
        stream.wait_event(e)
    end.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3
    return start.elapsed_time(end), wall


def source_sha256() -> str:
    """sha256 over the fused kernel's source files, concatenated in KERNEL_SOURCES order."""
    import hashlib
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """Counter-measured HBM bytes per fused launch, or None if not measured for this source."""
    t = TRAFFIC.get(workload)
    if t is None or t["source_sha256"] != source_sha256():
        return None
    return t


def copy_calibration(device):
    """A plain device-to-device copy of COPY_BYTES, three times: the counter runs scale
    FETCH_SIZE and WRITE_SIZE by what they read for it."""
    import torch
    src = torch.ones(COPY_BYTES // 2, device=device, dtype=torch.bfloat16)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def cpu_baseline(wl, device, budget_s=10.0):
    """The fp64 oracle on a bounded sample of the sweep, timed on the host's cores.

    The sample is whole decoder layers in sweep order (layer 0 first), stopping after the
    first layer at which the oracle's cumulative time reaches ``budget_s``.  Each matrix's
    inputs are drawn exactly as the GPU run draws them (on the device, same seeds), copied
    to the host, and only the oracle call is timed.  value = the sample's algorithmic
    bytes / the oracle's total time.
    """
    import numpy as np
    import oracle
    import torch
    from paper_2606_22932_amd import accounting, synth
    b = lambda t: t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    per_layer = len(synth.LLAMA8B_PROJ)
    total_s, total_b, n_mats, layers = 0.0, 0, 0, 0
    for layer in range(32):
        for mat in wl.matrices[layer * per_layer:(layer + 1) * per_layer]:
            X, dY = synth.activations(wl.T, mat, wl, wl.steps[0], device=device)
            W = synth.weight(mat, wl, device=device)
            m, v = synth.warm_moments(mat, wl, device=device, dtype=torch.bfloat16)
            args = tuple(b(t) for t in (X, dY, W, m, v))
            del X, dY, W, m, v
            t0 = time.perf_counter()
            out = oracle.linear_step(*args, moment_dtype=oracle.MOMENT_BF16, step=wl.steps[0], **wl.hyper)
            total_s += time.perf_counter() - t0
            del out, args
            total_b += accounting.fused_bytes(wl.T, mat.d_in, mat.d_out, "bf16")
            n_mats += 1
        layers += 1
        log(f"  oracle: layer {layer} done, {total_s:.1f} s so far")
        if total_s >= budget_s:
            break
    return dict(value=round(total_b / total_s / 1e9, 4), unit="GB/s", cores=oracle.num_threads(),
                kind="oracle", seconds=round(total_s, 2),
                sample=f"decoder layers 0-{layers - 1} of the sweep ({n_mats} matrices, "
                       f"{total_b / 1e9:.2f} GB algorithmic), T=512, bf16 moments, step 100; "
                       "fp64 oracle time only (input transfer excluded)")


def compute_bound(T: int) -> bool:
    """bf16 state: 2T GEMM flop against 12 B of state per parameter; the MFMA and HBM
    roofs (2.5 PFLOP/s, 8 TB/s) cross at 2T/12 = 312.5 flop/B, i.e. T = 1875."""
    return 2 * T / 12 > MFMA_BF16_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9)


def _median(xs):
    xs = sorted(xs)
    n = len(xs)
    return xs[n // 2] if n % 2 else 0.5 * (xs[n // 2 - 1] + xs[n // 2])


def time_batches(units, fn, per_batch, batches, warmup):
    """Median (and range) over `batches` batches of the per-launch time in ms: each batch is
    `per_batch` launches back to back between two HIP events on the launch stream, cycling
    through `units` (rotated copies of the state, or a step sequence)."""
    import torch
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        fn(units[i % len(units)], i)
    k = warmup
    times = []
    for _ in range(batches):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(per_batch):
            fn(units[k % len(units)], k)
            k += 1
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b) / per_batch)
    return _median(times), min(times), max(times)


def oracle_seconds(args, kwargs, runs, threads):
    """Median wall time of `runs` oracle steps on `threads` host threads (oracle call only)."""
    import oracle
    oracle.set_num_threads(threads)
    ts = []
    for _ in range(runs):
        t0 = time.perf_counter()
        oracle.linear_step(*args, **kwargs)
        ts.append(time.perf_counter() - t0)
    return _median(ts)


# The single-layer configurations reported beside the sweep: C1 (layer256, fp32 moments,
# steps 1-3), C2 (o_proj), C3 (the MLP projections, bf16 moments), C4 (the same, int8 moments
# in 256-row column blocks).  C2's 210 MB fits the 256 MB Infinity Cache, so it is timed over
# ROTATE_C2 copies of its inputs and state, launched in turn.
ROTATE_C2 = 3
CONFIG_NAMES = {"C1": "layer256", "C2": "o_proj", "C3": "mlp", "C4": "mlp_i8"}


def single_configs(device, cores):
    """Per-config GPU time, GB/s and % of 8 TB/s, each next to the fp64 oracle on the host's
    cores (and, for C1 and C2, on one thread).  GPU: median over batches of back-to-back
    launches; oracle: median of 3 runs (C1, C2) or one run per matrix (C3, C4)."""
    import numpy as np
    import oracle
    import torch
    from paper_2606_22932_amd import accounting, forge, synth
    b16 = lambda t: t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    host = lambda t: b16(t) if t.dtype == torch.bfloat16 else t.detach().cpu().contiguous().numpy()
    out = {}
    for key, name in CONFIG_NAMES.items():
        wl = synth.WORKLOADS[name]
        hp = wl.hyper
        log(f"config {key} ({name}): GPU")
        copies = ROTATE_C2 if key == "C2" else 1
        per_mat = []                     # per matrix: list of copies of its launch arguments
        for mat in wl.matrices:
            cs = []
            for c in range(copies):
                X, dY = synth.activations(wl.T, mat, wl, wl.steps[0], device=device)
                W = synth.weight(mat, wl, device=device)
                if wl.moment == "i8":
                    m, v, ms, vs = synth.random_i8_state(mat, wl, device=device, layout="col256")
                else:
                    dt = torch.float32 if wl.moment == "f32" else torch.bfloat16
                    m, v = synth.warm_moments(mat, wl, device=device, dtype=dt)
                    ms = vs = None
                dYs = [synth.activations(wl.T, mat, wl, t, device=device)[1] for t in wl.steps] \
                    if len(wl.steps) > 1 else [dY]
                cs.append(dict(X=X, dYs=dYs, W=W, m=m, v=v, ms=ms, vs=vs))
            per_mat.append(cs)
        torch.cuda.synchronize()
        nsteps = len(wl.steps)

        def launch(c, k):
            j = k % nsteps          # C1 cycles through its steps 1..3 with their own dY
            forge.forge_linear_step(c["X"], c["dYs"][j], c["W"], c["m"], c["v"], c["ms"], c["vs"],
                                    step=wl.steps[j], **hp)

        per_launch = 60 if key == "C1" else (30 if key == "C2" else 10)
        ms_total, lo_total, hi_total = 0.0, 0.0, 0.0
        for cs in per_mat:
            med, lo, hi = time_batches(cs, launch, per_launch, 21, 3 * per_launch)
            ms_total += med
            lo_total += lo
            hi_total += hi
        fused_b = sum(accounting.fused_bytes(wl.T, m_.d_in, m_.d_out, wl.moment) for m_ in wl.matrices)
        gbs = fused_b / (ms_total * 1e-3) / 1e9
        r = {"workload": name, "T": wl.T, "matrices": [f"{m_.name}[{m_.d_out}x{m_.d_in}]" for m_ in wl.matrices],
             "moments": wl.moment, "algorithmic_bytes": fused_b,
             "gpu_us": round(ms_total * 1e3, 2), "gpu_us_range": [round(lo_total * 1e3, 2), round(hi_total * 1e3, 2)],
             "gpu_GBs": round(gbs, 1), "frac_of_8TBs": round(gbs / HBM_PEAK_GBS, 4),
             "timing": f"sum over matrices of the median of 21 batches of {per_launch} back-to-back launches"
                       + (f", rotating {copies} copies of inputs and state" if copies > 1 else "")}
        # the oracle on the host: the same inputs (first copy), the step's state as the GPU has it
        log(f"config {key}: oracle on {cores} threads" + (" and 1 thread" if key in ("C1", "C2") else ""))
        t_all, t_one = 0.0, 0.0
        for mat, cs in zip(wl.matrices, per_mat):
            c = cs[0]
            if wl.moment == "i8":
                # the timing state's codes and scales, on the host
                mq, vq, ms_, vs_ = synth.random_i8_state(mat, wl, device=device, layout="col256")
                args = (b16(c["X"]), b16(c["dYs"][0]), b16(c["W"]), host(mq), host(vq))
                kw = dict(moment_dtype=oracle.MOMENT_I8, m_scale=host(ms_), v_scale=host(vs_))
            else:
                m0, v0 = synth.warm_moments(mat, wl, device=device,
                                            dtype=torch.float32 if wl.moment == "f32" else torch.bfloat16)
                args = (b16(c["X"]), b16(c["dYs"][0]), b16(c["W"]), host(m0), host(v0))
                kw = dict(moment_dtype=oracle.MOMENT_F32 if wl.moment == "f32" else oracle.MOMENT_BF16)
            kw.update(step=wl.steps[0], **hp)
            runs = 3 if key in ("C1", "C2") else 1
            t_all += oracle_seconds(args, kw, runs, cores)
            if key in ("C1", "C2"):
                t_one += oracle_seconds(args, kw, runs, 1)
        oracle.set_num_threads(cores)
        r["oracle"] = {"seconds": round(t_all, 4), "GBs": round(fused_b / t_all / 1e9, 4), "cores": cores,
                       "runs": "median of 3" if key in ("C1", "C2") else "one run per matrix, summed"}
        if key in ("C1", "C2"):
            r["oracle_1_thread"] = {"seconds": round(t_one, 4), "GBs": round(fused_b / t_one / 1e9, 4), "cores": 1,
                                    "runs": "median of 3"}
        r["gpu_over_oracle"] = round(t_all / (ms_total * 1e-3), 1)
        out[key] = r
        log(f"config {key}: {r}")
        del per_mat
        torch.cuda.empty_cache()
    return out


def compute_bound_block(device):
    """The fused step past the ridge: Llama-3.1-8B o_proj (4096 x 4096) at T = 4096 (App. D's
    BT = 4096), rotating 3 copies of inputs and state; next to it the store-G control (the
    same tile kernel storing G in bf16 instead of updating the state) on the same inputs."""
    import torch
    from paper_2606_22932_amd import accounting, forge, synth
    wl = synth.WORKLOADS["o_proj_t4096"]
    mat = wl.matrices[0]
    hp = wl.hyper
    copies = []
    for c in range(3):
        X, dY = synth.activations(wl.T, mat, wl, wl.steps[0], device=device)
        W = synth.weight(mat, wl, device=device)
        m, v = synth.warm_moments(mat, wl, device=device, dtype=torch.bfloat16)
        copies.append(dict(X=X, dY=dY, W=W, m=m, v=v))
    G = torch.empty((mat.d_out, mat.d_in), dtype=torch.bfloat16, device=device)
    fused = lambda c, k: forge.forge_linear_step(c["X"], c["dY"], c["W"], c["m"], c["v"], step=wl.steps[0], **hp)
    store_g = lambda c, k: forge.forge_wgrad(c["X"], c["dY"], G)
    f_ms, f_lo, f_hi = time_batches(copies, fused, 12, 11, 24)
    g_ms, g_lo, g_hi = time_batches(copies, store_g, 12, 11, 24)
    flops = accounting.gemm_flops(wl.T, mat.d_in, mat.d_out)
    byts = accounting.fused_bytes(wl.T, mat.d_in, mat.d_out, wl.moment)
    tf = lambda ms: flops / (ms * 1e-3) / 1e12
    del copies, G
    torch.cuda.empty_cache()
    return {"workload": "Llama-3.1-8B o_proj 4096x4096, T=4096, bf16 W/m/v (rotating 3 copies)",
            "gemm_flops": flops, "algorithmic_bytes": byts,
            "fused_us": round(f_ms * 1e3, 2), "fused_us_range": [round(f_lo * 1e3, 2), round(f_hi * 1e3, 2)],
            "fused_TFs": round(tf(f_ms), 1), "fused_mfma_frac": round(tf(f_ms) / MFMA_BF16_PEAK_TFS, 4),
            "fused_GBs": round(byts / (f_ms * 1e-3) / 1e9, 1),
            "store_g_control_us": round(g_ms * 1e3, 2), "store_g_control_TFs": round(tf(g_ms), 1),
            "store_g_control_mfma_frac": round(tf(g_ms) / MFMA_BF16_PEAK_TFS, 4),
            "timing": "median of 11 batches of 12 back-to-back launches"}


# The other state encodings, on the MLP projections at T = 512 (C3's shapes): int8 moments
# in 64-wide row blocks (the paper's own int8 layout), fp8 E4M3 moments, fp8 E4M3 weights
# with bf16 moments, and both.  Each is timed like C3 and C4 (one launch per matrix).
ENCODINGS = ("mlp_i8r64", "mlp_fp8", "mlp_wfp8", "mlp_wfp8_fp8")


def encodings_block(device):
    import torch
    from paper_2606_22932_amd import accounting, forge, synth
    out = {}
    for name in ENCODINGS:
        wl = synth.WORKLOADS[name]
        hp = wl.hyper
        mats = build_workload(wl, device)
        torch.cuda.synchronize()

        def launch(d, k):
            if wl.weight == "fp8":
                forge.forge_linear_step_wfp8(d["X"], d["dY"], d["W"], d["w_ring"], d["m"], d["v"], d["ms"], d["vs"],
                                             step=wl.steps[0], **hp)
            else:
                forge.forge_linear_step(d["X"], d["dY"], d["W"], d["m"], d["v"], d["ms"], d["vs"],
                                        step=wl.steps[0], **hp)

        us, lo, hi = 0.0, 0.0, 0.0
        for d in mats:
            med, a, b = time_batches([d], launch, 10, 21, 30)
            us, lo, hi = us + med * 1e3, lo + a * 1e3, hi + b * 1e3
        byts = sum(accounting.fused_bytes(wl.T, m_.d_in, m_.d_out, wl.moment, wl.weight) for m_ in wl.matrices)
        gbs = byts / (us * 1e-6) / 1e9
        tr = measured_traffic(name)
        out[name] = {"weights": wl.weight, "moments": wl.moment,
                     "state_bytes_per_param": accounting.state_bytes_per_param(wl.moment, wl.weight),
                     "algorithmic_bytes": byts, "gpu_us": round(us, 2), "gpu_us_range": [round(lo, 2), round(hi, 2)],
                     "gpu_GBs": round(gbs, 1), "frac_of_8TBs": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic_over_algorithmic": None if tr is None else
                     round(tr["bytes_per_launch"] * len(wl.matrices) / byts, 4)}
        del mats
        torch.cuda.empty_cache()
    out["timing"] = "sum over gate, up, down of the median of 21 batches of 10 back-to-back launches"
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: per workload)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed warmup steps (default: per workload)")
    ap.add_argument("--workload", default="sweep", choices=["sweep", "o_proj", "o_proj_t4096", "mlp", "mlp_i8",
                                                            "mlp_i8r64", "mlp_fp8", "mlp_wfp8", "mlp_wfp8_fp8"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--streams", type=int, default=1,
                    help="launch consecutive sweep launches round-robin on this many streams")
    ap.add_argument("--schedule", default="backward", choices=["backward", "layer"],
                    help="sweep launch grouping: per backward-pass group, or one launch per layer")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the single-layer configurations C1-C4 (timed beside the sweep by default)")
    ap.add_argument("--tokens", type=int, default=None,
                    help="override the workload's token count T (0: the state streaming alone)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the measured HBM ceilings (a child process after the timed work)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 1 GiB device copy first (reference for counter scaling)")
    ap.add_argument("--micro", action="store_true",
                    help="instead of the sweep: the update-path microbenchmark (marginal cost of "
                         "the fused update over the store-G control; q/o_proj shape, T=512 and 4096)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the fused step on one GPU only: the step has no cross-GPU "
              "work (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    if args.micro:
        args.warmup = 3 if args.warmup is None else args.warmup
        args.steps = 10 if args.steps is None else args.steps
    else:
        w0, k0 = DEFAULT_STEPS[args.workload]
        args.warmup = w0 if args.warmup is None else args.warmup
        args.steps = k0 if args.steps is None else args.steps
    if args.steps < 1 or args.warmup < 0:
        print("--steps must be at least 1 and --warmup at least 0", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_22932_amd import accounting, forge, synth

    forge.lib()                                  # fails loudly if the HIP library is not built
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    if args.micro:
        print(json.dumps(micro(device, args.steps, args.warmup)), flush=True)
        return
    wl = synth.WORKLOADS[args.workload]
    if args.tokens is not None:
        if not 0 <= args.tokens <= wl.T:
            print(f"--tokens must be in [0, {wl.T}]", file=sys.stderr)
            sys.exit(2)
        wl = dataclasses.replace(wl, T=args.tokens)
    if args.copy_calibration:
        log(f"calibration copy: {COPY_BYTES} bytes x 3")
        copy_calibration(device)
    log(f"building {args.workload}: {len(wl.matrices)} matrices")
    mats = build_workload(wl, device)
    torch.cuda.synchronize()
    hp = wl.hyper
    T = wl.T

    # One fused launch per group of matrices whose gradients a backward pass makes available
    # together (one matrix per launch except q/k/v and gate/up of the sweep).
    launches = [[mats[i] for i in g] for g in synth.launch_groups(wl, args.schedule)]

    # Consecutive launches touch disjoint state, so they may run on alternating streams: the
    # next launch's first tiles then start on the compute units that the previous launch's
    # last tiles free, instead of after all of them have finished.
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(args.streams - 1)]
    nlaunch = [0]

    def fused(group, t):
        st = streams[nlaunch[0] % len(streams)]
        nlaunch[0] += 1
        if wl.weight == "fp8":
            for d in group:
                forge.forge_linear_step_wfp8(d["X"], d["dY"], d["W"], d["w_ring"], d["m"], d["v"], d["ms"], d["vs"],
                                             step=t, stream=st.cuda_stream, **hp)
            return
        forge.forge_linear_step_grouped([(d["X"], d["dY"], d["W"], d["m"], d["v"], d["ms"], d["vs"])
                                         for d in group], step=t, stream=st.cuda_stream, **hp)

    fused_b = sum(accounting.fused_bytes(T, d["mat"].d_in, d["mat"].d_out, wl.moment, wl.weight) for d in mats)
    flops = sum(accounting.gemm_flops(T, d["mat"].d_in, d["mat"].d_out) for d in mats)
    log(f"timing fused ({len(launches)} launches per step)")
    total, wall = time_steps(launches, wl, fused, args.steps, args.warmup, wl.steps[0], streams[1:])
    ms = total / args.steps
    avg_launch_ms = total / (args.steps * len(launches))
    kern_gbs = (fused_b / len(launches)) / (avg_launch_ms * 1e-3) / 1e9
    value = fused_b / (ms * 1e-3) / 1e9
    log(f"fused: {ms:.3f} ms/step, {value:.1f} GB/s, kernel-time {kern_gbs:.1f} GB/s, "
        f"MFMA {flops / (ms * 1e-3) / 1e12:.1f} TF/s, wall {wall:.1f} ms")

    tr = measured_traffic(args.workload) if args.tokens is None else None   # measured at the workload's T
    traffic = None if tr is None else tr["bytes_per_launch"]
    kernel = "pipelined_i8_kernel" if wl.moment == "i8" else "fused_kernel"
    entry = "forge_linear_step_wfp8" if wl.weight == "fp8" else "forge_linear_step_grouped"
    out = {
        "metric": "fused dW+AdamW step: HBM GB/s & % roofline; ms per Llama-8B linear sweep",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded Gaussian X, dY, W, warm m, v; generated on the GPU)",
        "config": {
            "workload": {"sweep": "Llama-3.1-8B linear-layer sweep: 32 x {q,k,v,o,gate,up,down} + lm_head, T=512, bf16 W/m/v",
                         "o_proj": "Llama-3.1-8B o_proj 4096x4096, T=512, bf16 W/m/v",
                         "o_proj_t4096": "Llama-3.1-8B o_proj 4096x4096, T=4096, bf16 W/m/v",
                         "mlp": "Llama-3.1-8B gate/up/down, T=512, bf16 W/m/v",
                         "mlp_i8": "Llama-3.1-8B gate/up/down, T=512, int8 m/v (256-row blocks)",
                         "mlp_i8r64": "Llama-3.1-8B gate/up/down, T=512, int8 m/v (64-wide row blocks)",
                         "mlp_fp8": "Llama-3.1-8B gate/up/down, T=512, bf16 W, fp8 E4M3 m and sqrt(v)",
                         "mlp_wfp8": "Llama-3.1-8B gate/up/down, T=512, fp8 E4M3 W, bf16 m/v",
                         "mlp_wfp8_fp8": "Llama-3.1-8B gate/up/down, T=512, fp8 E4M3 W, m and sqrt(v)"}[args.workload]
                        .replace("T=512", f"T={T}"),
            "T": T, "matrices": len(mats),
            "params": sum(d["mat"].d_in * d["mat"].d_out for d in mats),
            "moments": wl.moment, "weights": wl.weight, "algorithmic_bytes_per_step": fused_b,
        },
        "roofline": {
            "bound": "hbm",
            "achieved": round(kern_gbs, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(kern_gbs / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "kernel": f"{kernel} ({entry})",
            "algorithmic_bytes_per_launch": round(fused_b / len(launches)),
            "avg_launch_us": round(avg_launch_ms * 1e3, 3),
            "launches_per_step": len(launches),
        } if not compute_bound(T) else {
            # past the ridge (T > ~1.9k for bf16 state) the GEMM bounds the step
            "bound": "mfma",
            "achieved": round(flops / len(launches) / (avg_launch_ms * 1e-3) / 1e12, 2),
            "peak": MFMA_BF16_PEAK_TFS,
            "unit": "TFLOP/s",
            "frac": round(flops / len(launches) / (avg_launch_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4),
            "traffic": traffic,
            "kernel": f"{kernel} ({entry})",
            "algorithmic_flops_per_launch": round(flops / len(launches)),
            "avg_launch_us": round(avg_launch_ms * 1e3, 3),
            "launches_per_step": len(launches),
        },
        "mfma_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
        "mfma_frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4),
    }

    if not args.no_unfused and wl.moment not in ("f32", "fp8") and wl.weight == "bf16":
        biggest = max(d["mat"].d_in * d["mat"].d_out for d in mats)
        G_ws = torch.empty(biggest, dtype=torch.bfloat16, device=device)

        def unfused(group, t):
            for d in group:
                forge.forge_linear_step_unfused(d["X"], d["dY"], d["W"], d["m"], d["v"], d["ms"], d["vs"],
                                                G_ws=G_ws, step=t, **hp)

        log("timing unfused (GEMM stores bf16 G, then the optimizer kernel)")
        ut, _ = time_steps([[d] for d in mats], wl, unfused, args.steps, args.warmup, wl.steps[0] + 1000)
        ums = ut / args.steps
        ub = sum(accounting.unfused_bytes(T, d["mat"].d_in, d["mat"].d_out, wl.moment, "bf16") for d in mats)
        out["unfused"] = {"ms_per_step": round(ums, 4), "algorithmic_bytes_per_step": ub,
                          "GBs_of_fused_bytes": round(fused_b / (ums * 1e-3) / 1e9, 2),
                          "GBs_of_unfused_bytes": round(ub / (ums * 1e-3) / 1e9, 2),
                          "speedup_fused_over_unfused": round(ums / ms, 4),
                          "byte_ratio_unfused_over_fused": round(ub / fused_b, 4)}
        log(f"unfused: {ums:.3f} ms/step -> fused speedup {ums / ms:.3f}x")
        del G_ws

    if not args.no_cpu_baseline:
        mats = launches = None
        torch.cuda.empty_cache()
        log("timing the CPU oracle on its sample")
        out["cpu_baseline"] = cpu_baseline(synth.WORKLOADS["sweep"], device)
        log(f"cpu baseline: {out['cpu_baseline']}")

    if not args.no_configs and args.workload == "sweep" and args.tokens is None:
        mats = launches = None
        torch.cuda.empty_cache()
        import oracle
        out["configs"] = single_configs(device, oracle.num_threads())
        log("compute-bound regime: o_proj at T=4096")
        out["compute_bound"] = compute_bound_block(device)
        log(f"compute-bound: {out['compute_bound']}")
        log("state encodings on the MLP projections")
        out["encodings"] = encodings_block(device)
        log(f"encodings: {out['encodings']}")

    if not args.no_ceilings:
        mats = launches = None
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        log("measuring HBM ceilings (read / write / copy / in-place read-modify-write of 3 streams, "
            "in address order and in 128x128 tiles)")
        c = hbm_ceilings()
        if c is not None:
            c["fused_over_rmw3"] = round(kern_gbs / c["rmw3"], 4)
            if "rmw3_tile" in c:
                c["fused_over_rmw3_tile"] = round(kern_gbs / c["rmw3_tile"], 4)
            out["hbm_ceiling"] = c
            log(f"ceilings: {c}")

    print(json.dumps(out), flush=True)


def micro(device, reps, warmup, d=4096, token_counts=(512, 4096)):
    """Update-path microbenchmark (App. D): on the q/o_proj shape d x d, the average
    duration of the store-G control (the same tile kernel with an epilogue that stores G
    as bf16 instead of updating the optimizer state) and of the fused step with every
    update rule (AdamW and the other families, fp32 and bf16 state); the marginal cost of
    an update is the difference.  Also the layer-level backward: dX = dY W alone and
    followed by the fused step.  Each figure is
    `reps` back-to-back launches between two events on the launch stream, after `warmup`."""
    import torch
    from paper_2606_22932_amd import forge, synth
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.1)
    rule_hp = {n: dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01) for n in forge.OPTIMIZERS}
    rule_hp["muon_accumulate"] = dict(lr=0.0, beta1=0.95)
    stream = torch.cuda.current_stream()

    def avg_us(fn):
        for _ in range(warmup):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    rows = []
    for T in token_counts:
        log(f"micro: T={T}, {d}x{d}")
        mat = synth.Matrix("qo", d, d, 2)
        wl = dataclasses.replace(synth.WORKLOADS["o_proj"], T=T)
        X, dY = synth.activations(T, mat, wl, 100, device=device)
        W = synth.weight(mat, wl, device=device)
        G = torch.empty((d, d), dtype=torch.bfloat16, device=device)
        dX = torch.empty((T, d), dtype=torch.bfloat16, device=device)
        mb, vb = synth.warm_moments(mat, wl, device=device, dtype=torch.bfloat16)
        mf, vf = synth.warm_moments(mat, wl, device=device, dtype=torch.float32)
        r = {"T": T, "shape": f"{d}x{d}"}
        r["store_g_control_us"] = avg_us(lambda: forge.forge_wgrad(X, dY, G))
        r["adamw_bf16_us"] = avg_us(lambda: forge.forge_linear_step(X, dY, W, mb, vb, step=100, **hp))
        r["adamw_f32_us"] = avg_us(lambda: forge.forge_linear_step(X, dY, W, mf, vf, step=100, **hp))
        r["input_grad_us"] = avg_us(lambda: forge.forge_input_grad(dY, W, dX))
        r["backward_bf16_us"] = avg_us(lambda: forge.forge_linear_backward(X, dY, W, mb, vb, dX=dX, step=100,
                                                                           **hp))
        r["marginal_adamw_bf16_us"] = r["adamw_bf16_us"] - r["store_g_control_us"]
        r["marginal_adamw_f32_us"] = r["adamw_f32_us"] - r["store_g_control_us"]
        # every update rule, by state count, on fp32 and bf16 state (the family table's rules)
        fam = {}
        for name in ("sgd", "sgd_momentum", "adagrad", "rmsprop", "lion", "muon_accumulate", "adamax", "adamw",
                     "nadam", "radam"):
            ns = forge.OPTIMIZER_STATES[name]
            for tag, (s1, s2) in (("f32", (mf, vf)), ("bf16", (mb, vb))):
                Wr = None if name == "muon_accumulate" else W
                us = avg_us(lambda: forge.forge_linear_step_opt(X, dY, Wr, s1, s2, optimizer=name, step=100,
                                                                **rule_hp[name]))
                fam[f"{name}_{tag}"] = {"states": ns, "us": round(us, 2),
                                        "marginal_us": round(us - r["store_g_control_us"], 2)}
        r["rules"] = fam
        rows.append({k: (round(v, 2) if isinstance(v, float) else v) for k, v in r.items()})
        log(f"micro: {rows[-1]}")
        del X, dY, W, G, dX, mb, vb, mf, vf
        torch.cuda.empty_cache()
    return {"metric": "update-path microbenchmark: marginal cost of the fused AdamW update over the "
                      "store-G control (us per launch)",
            "unit": "us", "higher_is_better": False, "n_gpus": 1, "reps": reps, "warmup": warmup,
            "data": "synthetic (seeded Gaussian X, dY, W, warm m, v)", "rows": rows}


def hbm_ceilings():
    """Measured HBM bandwidth of this device for plain access mixes (context for the
    roofline): runs the built probe ``paper_2606_22932_amd/hbm_ceiling`` as a child process."""
    import subprocess
    from paper_2606_22932_amd import build
    if not os.path.exists(build.CEILING_BIN):
        log("hbm_ceiling is not built; skipping the measured ceilings")
        return None
    res = subprocess.run([build.CEILING_BIN], capture_output=True, text=True, timeout=300)
    if res.returncode != 0:
        log(f"hbm_ceiling failed ({res.returncode}): {res.stderr.strip()}")
        return None
    return json.loads(res.stdout.strip().splitlines()[-1])


if __name__ == "__main__":
    main()
