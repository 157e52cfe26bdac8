"""Benchmark of the TASQ masked-linear hot path on one MI355X.

One "step" is one full denoising schedule through ``tasq_run_schedule``:
28 PixArt-Sigma-shaped blocks (112 int8 linears: QKV 1152->3456, out
1152->1152, MLP 1152->4608 and 4608->1152, 2x4096 tokens each) over 20
denoising steps in 4 stages, every layer at b = table[l][stage], fp32
dequantised outputs.  Inputs are synthetic and already resident in HBM when
timing starts.

Prints one JSON line: whole-schedule int8 TOPS (2*M*N*K summed over every
GEMM of every denoising step, divided by wall time), the same schedule with a
static b = 8 table and with the per-layer maximum over stages, the dominant
kernel's roofline fraction, and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2608_03057_amd as T                      # noqa: E402
from paper_2608_03057_amd import inputs               # noqa: E402

METRIC = "int8 TOPS of masked GEMM + schedule wall-time vs static 8-bit, 1×MI355X"
PEAK_INT8_TOPS = 5000.0        # dense int8 MFMA, MI355X datasheet
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# Sources the grouped kernel of each weight layout is built from: recorded
# counter readings stay valid while none of these files changes.
KERNEL_SOURCES = {
    "k_masked_gemm_persistent": ["gemm_core.h", "gemm_pers.h", "tasq_internal.h",
                                 "tile_256x256_k128_w8_pf1.hip", "tasq_api.cpp"],
    "k_masked_gemm_grouped": ["gemm_core.h", "tasq_internal.h", "tile_256x256_k128_w8_pf1.hip",
                              "tasq_api.cpp"],
    "k_gemm_packed_persistent": ["gemm_core.h", "gemm_packed.h", "gemm_pers.h",
                                 "gemm_pers_packed.h", "tasq_internal.h",
                                 "ptile_256x256_k128_w8.hip", "tasq_api.cpp"],
}


def step_kernel(weights: str) -> str:
    """The kernel of one denoising step of the 28-block schedule: the
    persistent grouped launch of the weight layout."""
    return "k_gemm_packed_persistent" if weights == "packed" else "k_masked_gemm_persistent"


def kernel_source_sha256(kernel: str = "k_masked_gemm_persistent") -> str:
    """Hash of the HIP sources of one grouped kernel; ties recorded counter
    readings to the code."""
    h = hashlib.sha256()
    for name in sorted(KERNEL_SOURCES[kernel]):
        with open(os.path.join(ROOT, "paper_2608_03057_amd", "csrc", name), "rb") as fh:
            h.update(name.encode())
            h.update(fh.read())
    return h.hexdigest()


def _recorded(kernel: str, suffix: str):
    """A committed rocprofv3 record of the grouped kernel (JSON under
    profiles/), or None when the kernel's sources changed since it was
    taken."""
    try:
        with open(os.path.join(ROOT, "profiles", f"{kernel}_pixart28_{suffix}.json")) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != kernel_source_sha256(kernel):
        return None
    return rec


def recorded_traffic(kernel: str):
    """HBM bytes per grouped launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE readings (already scaled by the copy calibration), or None when
    the kernel sources changed since they were taken."""
    rec = _recorded(kernel, "traffic")
    if rec is None:
        return None
    return rec.get("fetch_bytes_per_launch", 0) + rec.get("write_bytes_per_launch", 0)


def recorded_counters(kernel: str):
    """Shader clock and matrix-pipe utilisation of the grouped launch under
    its own load, from the committed rocprofv3 counter readings
    (GRBM_GUI_ACTIVE per XCD over the dispatch time; SQ_VALU_MFMA_BUSY_CYCLES
    over GRBM_GUI_ACTIVE x 1024 SIMDs), per table; None when the kernel
    sources changed since they were taken."""
    rec = _recorded(kernel, "counters")
    if rec is None:
        return None
    return rec.get("per_table")


def build_workload(wl, device, packed=True):
    """Device tensors of every layer; X drawn on the GPU (integer recipe,
    identical to the CPU draw), W and sw on the CPU (fp64 Box-Muller).  With
    ``packed`` each layer keeps only its packed weight buffer (the one stored
    8-bit copy, in the matrix-instruction operand order)."""
    layers, keep = [], []
    for l, spec in enumerate(wl.layers):
        X = inputs.x_full(wl, l, device=device)
        W = inputs.w_full(wl, l).to(device)
        sw = inputs.sw_full(wl, l).to(device)
        y = torch.empty((spec.M, spec.N), dtype=torch.float32, device=device)
        if packed:
            P = T.pack_weights(W)
            torch.cuda.synchronize()
            del W
            keep.append((X, P, sw, y))
            layers.append(T.make_layer(X, None, wl.sx, sw, None, None, y, packed=P))
        else:
            keep.append((X, W, sw, y))
            layers.append(T.make_layer(X, W, wl.sx, sw, None, None, y))
    return layers, keep


def gemm_ops(wl):
    return sum(2.0 * s.M * s.N * s.K for s in wl.layers)


def gemm_bytes(wl):
    """Algorithmic HBM bytes of one denoising step: each layer reads X and W
    once and writes its fp32 output once."""
    return sum(float(s.M * s.K + s.N * s.K + 4 * s.M * s.N) for s in wl.layers)


def time_schedule(layers, table, wl, ws, steps, warmup):
    for _ in range(warmup):
        T.run_schedule(layers, table, wl.S, wl.T, 0, wl.T, workspace=ws)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        T.run_schedule(layers, table, wl.S, wl.T, 0, wl.T, workspace=ws)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def shard_shapes(wl, table, keep, full_ms, device, parts=8, steps=3, warmup=1):
    """The step on one GPU's share of a ``parts``-way split (shard 0), at its
    real shapes: the first M/parts token rows of every layer (W replicated),
    or its first N/parts output channels (W, sw and outputs split).  Neither
    split exchanges anything between GPUs, so a shard's step time is the
    split step's time.  The shard's operands are views of the full
    workload's device tensors (row-major weights); its outputs are fresh."""
    out = {"parts": parts}
    for axis, key in (("M", "token_split"), ("N", "channel_split")):
        swl = inputs.shard(wl, axis, parts)
        layers, ys = [], []
        for l, spec in enumerate(swl.layers):
            X, W, sw, _ = keep[l]
            if axis == "M":
                X = X[:spec.M]
            else:
                W, sw = W[:spec.N], sw[:spec.N]
            y = torch.empty((spec.M, spec.N), dtype=torch.float32, device=device)
            ys.append(y)
            layers.append(T.make_layer(X, W, swl.sx, sw, None, None, y))
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=device)
        ms = time_schedule(layers, table, swl, ws, steps, warmup)
        out[key] = {
            "shapes": sorted({(sp.M, sp.K, sp.N) for sp in swl.layers}),
            "ms_per_schedule": round(ms, 4),
            "ms_per_denoising_step": round(ms / swl.T, 4),
            "TOPS": round(gemm_ops(swl) * swl.T / (ms * 1e-3) / 1e12, 1),
            # the full step's time over `parts` against the shard's
            "split_efficiency": round(full_ms / parts / ms, 4),
        }
        del layers, ys, ws
        torch.cuda.empty_cache()
    return out


def measured_peaks(device, blocks=768, iters=40000, copy_reps=5):
    """What the GPU sustains, measured here rather than taken from the
    datasheet: the int8 matrix-instruction rate with no memory traffic
    (libtasq_probe.so, eight independent v_mfma_i32_32x32x32_i8 chains per
    wave, three workgroups of four waves per CU), the shader clock that rate
    implies (the datasheet 5.0 POP/s is reached at 2.4 GHz), and the
    bandwidth of a plain 1 GiB device-to-device copy (read + write bytes)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2608_03057_amd", "libtasq_probe.so")
    probe = ctypes.CDLL(path)
    probe.tasq_probe_mfma_peak.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                           ctypes.c_void_p]
    sink = torch.empty(blocks * 256, dtype=torch.int32, device=device)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def run(n):
        if probe.tasq_probe_mfma_peak(blocks, n, ctypes.c_void_p(sink.data_ptr()), stream):
            raise RuntimeError("tasq_probe_mfma_peak failed")

    run(100)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    run(iters)
    b.record()
    torch.cuda.synchronize()
    ops = blocks * 4 * iters * probe.tasq_probe_mfma_chains() * 2.0 * 32 * 32 * 32
    tops = ops / (a.elapsed_time(b) * 1e-3) / 1e12
    src = torch.empty(1 << 30, dtype=torch.uint8, device=device)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    a.record()
    for _ in range(copy_reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    copy = 2.0 * src.numel() * copy_reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    return {"mfma_int8_TOPS": round(tops, 1), "mfma_frac_of_datasheet": round(tops / PEAK_INT8_TOPS, 4),
            "implied_clock_GHz": round(2.4 * tops / PEAK_INT8_TOPS, 3),
            "copy_GBps": round(copy, 1), "copy_frac_of_datasheet": round(copy / PEAK_HBM_GBS, 4),
            "kernels": "k_mfma_peak (libtasq_probe.so); torch copy_ of 1 GiB"}


def time_launches(layers, table, wl, ws):
    """Duration of each grouped launch (one denoising step) of one whole
    schedule: the library records a HIP event pair on the launch stream
    around each step's launch (tasq_opts.step_events), so the per-call
    upload of the layer list is outside every pair.  Returns the mean over
    the schedule's steps, in ms."""
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * wl.T)]
    for e in evs:              # torch creates the event at its first record
        e.record()
    T.run_schedule(layers, table, wl.S, wl.T, 0, wl.T, workspace=ws, step_events=evs)
    torch.cuda.synchronize()
    return float(np.mean([evs[2 * i].elapsed_time(evs[2 * i + 1]) for i in range(wl.T)]))


def time_tables_interleaved(layers, tables, wl, ws, rounds=5):
    """Whole-schedule wall time of several tables on identical inputs, the
    tables taking turns round by round (so that a drift of the clock or the
    temperature over the run does not favour the table timed first).
    Returns per table the median, min and max ms over the rounds."""
    times = {name: [] for name in tables}
    ev = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    for name, tab in tables.items():
        T.run_schedule(layers, tab, wl.S, wl.T, 0, wl.T, workspace=ws)
    torch.cuda.synchronize()
    for _ in range(rounds):
        for name, tab in tables.items():
            a, b = ev(), ev()
            a.record()
            T.run_schedule(layers, tab, wl.S, wl.T, 0, wl.T, workspace=ws)
            b.record()
            torch.cuda.synchronize()
            times[name].append(a.elapsed_time(b))
    return {name: {"median": round(float(np.median(v)), 4), "min": round(min(v), 4),
                   "max": round(max(v), 4)} for name, v in times.items()}


def skinny_schedule(wl, table, keep, device, M=16, reps=3):
    """The same 112 layers at M tokens (weight-streaming regime): schedule
    wall time per denoising step with the weights read as int8 rows, as the
    packed buffer, or as the top b bit planes (each layer holding only that
    copy), and under the library's AUTO choice with all three copies given
    (the planes below b = 8, the packed copy at b = 8), at the TASQ table and
    at a static b = 8.  Reuses the weights already on the GPU."""
    layers = {"rows": [], "packed": [], "planes": [], "auto": []}
    hold = []
    for l, spec in enumerate(wl.layers):
        W = keep[l][1]
        if W.dim() == 1:           # packed-only run: no row-major copy to stream
            return None
        X = inputs.x_rows(wl, l, np.arange(M), device=device)
        sw = keep[l][2]
        y = torch.empty((M, spec.N), dtype=torch.float32, device=device)
        P = T.pack_weights(W)
        Q = T.pack_planes(W)
        hold += [X, y, P, Q]
        layers["rows"].append(T.make_layer(X, W, wl.sx, sw, None, None, y))
        layers["packed"].append(T.make_layer(X, None, wl.sx, sw, None, None, y, packed=P))
        layers["planes"].append(T.make_layer(X, None, wl.sx, sw, None, None, y, planes=Q))
        layers["auto"].append(T.make_layer(X, W, wl.sx, sw, None, None, y, packed=P, planes=Q))
    torch.cuda.synchronize()
    ws = torch.empty(T.schedule_workspace_bytes(layers["rows"]), dtype=torch.uint8, device=device)
    t8 = torch.full_like(table, 8)
    out = {}
    for name, ls in layers.items():
        for tname, tab in (("tasq", table), ("b8", t8)):
            T.run_schedule(ls, tab, wl.S, wl.T, 0, wl.T, workspace=ws)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                T.run_schedule(ls, tab, wl.S, wl.T, 0, wl.T, workspace=ws)
            b.record()
            torch.cuda.synchronize()
            out[f"{name}_{tname}"] = round(a.elapsed_time(b) / reps / wl.T, 4)
    wbytes = sum(float(s.N * s.K) for s in wl.layers)
    mean_b = float(table.float().mean())
    planes_b = wbytes * mean_b / 8.0
    return {"M": M, "ms_per_denoising_step": out,
            "weight_bytes_per_step": {"int8": wbytes, "planes_tasq": planes_b},
            "planes_tasq_GBps": round(planes_b / (out["planes_tasq"] * 1e-3) / 1e9, 1),
            "packed_GBps": round(wbytes / (out["packed_b8"] * 1e-3) / 1e9, 1),
            "planes_speedup_vs_b8": round(out["planes_b8"] / out["planes_tasq"], 3),
            "auto_tasq_vs_auto_b8": round(out["auto_b8"] / out["auto_tasq"], 3),
            "auto_tasq_vs_rows_b8": round(out["rows_b8"] / out["auto_tasq"], 3)}


def skinny_sweep(device, steps=64):
    """Single weight-streaming layers: M in {1, 16, 64} on the (K, N) pairs
    of the PixArt and SANA blocks, the weight read as int8 rows, as the packed
    buffer or as the top b planes.  Each figure is one tasq_run_schedule call
    over `steps` steps of the one layer (per-layer launches issued back to
    back from the library), timed with HIP events; returns one dict per
    (M, K, N) with microseconds per launch and weight bytes read per
    microsecond."""
    rows = []
    for l_cfg in (1, 2):
        wl = inputs.workload(l_cfg)
        for l, spec in enumerate(wl.layers):
            W = inputs.w_full(wl, l).to(device)
            sw = inputs.sw_full(wl, l).to(device)
            P, Q = T.pack_weights(W), T.pack_planes(W)
            for M in (1, 16, 64):
                X = inputs.x_rows(wl, l, np.arange(M), device=device)
                y = torch.empty((M, spec.N), dtype=torch.float32, device=device)
                srcs = {"rows": (T.make_layer(X, W, wl.sx, sw, None, None, y), T.VARIANT_AUTO),
                        "packed": (T.make_layer(X, None, wl.sx, sw, None, None, y, packed=P),
                                   T.VARIANT_AUTO),
                        "planes": (T.make_layer(X, None, wl.sx, sw, None, None, y, planes=Q),
                                   T.VARIANT_BITPLANE)}
                row = {"workload": wl.name, "layer": spec.name, "M": M, "K": spec.K, "N": spec.N}
                for name, (layer, variant) in srcs.items():
                    for bits in ((2, 4, 6, 8) if name == "planes" else (8,)):
                        tab = torch.full((1, 1), bits, dtype=torch.uint8)
                        T.run_schedule([layer], tab, 1, steps, 0, steps, variant=variant)
                        torch.cuda.synchronize()
                        a = torch.cuda.Event(enable_timing=True)
                        b_ = torch.cuda.Event(enable_timing=True)
                        a.record()
                        T.run_schedule([layer], tab, 1, steps, 0, steps, variant=variant)
                        b_.record()
                        torch.cuda.synchronize()
                        us = a.elapsed_time(b_) / steps * 1e3
                        wbytes = spec.N * spec.K * (bits / 8.0 if name == "planes" else 1.0)
                        row[f"{name}_b{bits}_us"] = round(us, 2)
                        row[f"{name}_b{bits}_GBps"] = round(wbytes / us / 1e3, 1)
                rows.append(row)
    return rows


def shape_sweep(device, reps=50, warmup=10):
    """Single layers of the four per-shape workloads (one 1152->1152 layer at
    256 tokens; the PixArt, SANA and SDXL-Turbo blocks, the latter with its
    3x3 conv), fp32 output, each timed alone: `warmup` launches, then `reps`
    launches each bracketed by HIP events on the launch stream, the Infinity
    Cache flushed before each (a 512 MB buffer written between launches,
    outside the events).  Per shape: median / p10 / p90 microseconds at b = 8
    and at the lowest b of the layer's table row, the roofline of the shape
    (2MNK ops against the dense int8 MFMA peak, M*K + N*K + 4*M*N bytes
    against HBM), the packed-weight kernel's median, the median under AUTO
    with both int8 copies given, and, as external context only, the vendor
    int8 GEMM (hipBLASLt through torch._int_mm, int32 output, b = 8)."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=device)
    ev = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731

    def timed(fn):
        for _ in range(warmup):
            fn()
        ts = []
        for _ in range(reps):
            flush.zero_()
            a, b = ev(), ev()
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        ts.sort()
        return ts[len(ts) // 2], ts[len(ts) // 10], ts[(9 * len(ts)) // 10]

    rows = []
    for cfg in range(4):
        wl = inputs.workload(cfg)
        table = inputs.b_table(wl)
        for l, spec in enumerate(wl.layers):
            conv = spec.kind == "conv3x3"
            X = inputs.x_full(wl, l, device=device)
            W = inputs.w_full(wl, l)
            if conv:
                W = W.reshape(spec.N, 3, 3, spec.C)
            W = W.to(device)
            sw = inputs.sw_full(wl, l).to(device)
            P = T.pack_weights(W)
            # the split-K room the library asks for, given to every layer kind alike
            wsb = T.workspace_bytes(spec.M, spec.N, spec.K)
            ws = torch.empty(wsb, dtype=torch.uint8, device=device) if wsb else None
            yb = torch.empty((spec.M, spec.N), dtype=torch.float32, device=device)
            if conv:
                yb = yb.reshape(spec.H, spec.Wd, spec.N)
            bmin = int(table[l].min())
            row = {"workload": wl.name, "layer": spec.name, "M": spec.M, "N": spec.N,
                   "K": spec.K, "kind": spec.kind, "b_low": bmin}
            for bits in (8, bmin):
                if conv:
                    f = lambda b=bits: T.masked_conv3x3(X, W, wl.sx, sw, b, want_acc=False, y=yb,
                                                        workspace=ws)
                    fp = lambda b=bits: T.masked_conv3x3(X, None, wl.sx, sw, b, packed=P,
                                                         want_acc=False, y=yb)
                    fa = lambda b=bits: T.masked_conv3x3(X, W, wl.sx, sw, b, packed=P,
                                                         want_acc=False, y=yb, workspace=ws)
                else:
                    f = lambda b=bits: T.masked_linear(X, W, wl.sx, sw, b, want_acc=False, y=yb,
                                                       workspace=ws)
                    fp = lambda b=bits: T.masked_linear(X, None, wl.sx, sw, b, packed=P,
                                                        want_acc=False, y=yb)
                    fa = lambda b=bits: T.masked_linear(X, W, wl.sx, sw, b, packed=P,
                                                        want_acc=False, y=yb, workspace=ws)
                med, p10, p90 = timed(f)
                row[f"b{bits}_us"] = {"median": round(med, 2), "p10": round(p10, 2),
                                      "p90": round(p90, 2)}
                row[f"b{bits}_packed_us_median"] = round(timed(fp)[0], 2)
                # AUTO with both int8 copies given (it picks one by shape)
                row[f"b{bits}_auto_us_median"] = round(timed(fa)[0], 2)
            ops = 2.0 * spec.M * spec.N * spec.K
            byts = float(spec.M * (spec.C if conv else spec.K) + spec.N * spec.K
                         + 4 * spec.M * spec.N)
            t_mfma, t_hbm = ops / (PEAK_INT8_TOPS * 1e12), byts / (PEAK_HBM_GBS * 1e9)
            med8 = row["b8_us"]["median"]
            row.update({"tops_b8": round(ops / (med8 * 1e-6) / 1e12, 1),
                        "bound": "mfma" if t_mfma > t_hbm else "hbm",
                        "roofline_us": round(max(t_mfma, t_hbm) * 1e6, 2),
                        "frac_b8": round(max(t_mfma, t_hbm) * 1e6 / med8, 3)})
            if not conv and hasattr(torch, "_int_mm"):
                try:
                    row["vendor_int8_int32out_us_median"] = round(
                        timed(lambda: torch._int_mm(X, W.t()))[0], 2)
                except RuntimeError:
                    row["vendor_int8_int32out_us_median"] = None
            rows.append(row)
            del X, W, P, ws
    return rows


def config_schedules(device, steps=5, warmup=2):
    """The schedules of the per-shape workloads (PixArt, SANA and SDXL-Turbo
    blocks with their tables): milliseconds per denoising step with one
    grouped launch per step and with per-layer launches."""
    rows = []
    for cfg in (1, 2, 3):
        wl = inputs.workload(cfg)
        table = inputs.b_table(wl)
        layers, keep = build_workload(wl, device, packed=False)
        ws = torch.empty(schedule_ws := T.schedule_workspace_bytes(layers), dtype=torch.uint8,
                         device=device)
        g = time_schedule(layers, table, wl, ws, steps, warmup) / wl.T
        p = time_schedule(layers, table, wl, None, steps, warmup) / wl.T
        ops = gemm_ops(wl)
        rows.append({"workload": wl.name, "schedule": {
            "grouped_ms_per_step": round(g, 4), "per_layer_ms_per_step": round(p, 4),
            "grouped_tops": round(ops / (g * 1e-3) / 1e12, 1),
            "per_layer_tops": round(ops / (p * 1e-3) / 1e12, 1),
            "workspace_bytes": schedule_ws}})
        del layers, keep, ws
    return rows


def act_schedule(wl, table, keep, ws, device, reps=2, rank=32):
    """The asymmetric-activation form of the same schedule: each layer's input
    arrives as fp32 (seeded normal draws with a few large channels), is
    quantized per tensor on the GPU, and the grouped launch dequantises with
    the zero-point term.  Per denoising step: one batched quantizer call over
    the 112 inputs, then one grouped launch.  Timed three ways: plain (with
    the same quantization as one call per tensor timed beside it), with a
    rank-`rank` 16-bit low-rank branch on every layer (SVDQuant-initialised
    models), where the quantizer also writes the down projection (one call
    per tensor) and the grouped launch adds the up projection, and with
    weight zero points (row sums of the codes).  Returns milliseconds per
    denoising step for the quantizer, the grouped launch and both, and the
    quantizer's HBM roofline (algorithmic bytes: 4 read + 1 written per
    element, plus 4 per element of the projection with the branch)."""
    xs, codes, Ts, plain, lowrank, wzero, hold = [], [], [], [], [], [], []
    rsums = []
    params = torch.empty((len(wl.layers), T.TASQ_ACT_PARAMS_FLOATS), dtype=torch.float32,
                         device=device)
    gen = torch.Generator(device=device)
    for l, spec in enumerate(wl.layers):
        X, W, sw, y = keep[l]
        if W.dim() == 1:           # packed-only run: no row-major copy for the channel sums
            return None
        gen.manual_seed(wl.seed * 1000 + l)
        x = torch.randn((spec.M, spec.K), generator=gen, device=device, dtype=torch.float32)
        x[:, ::61] *= 24.0
        down = (0.05 * torch.randn((rank, spec.K), generator=gen, device=device)).to(
            torch.bfloat16)
        up = (0.05 * torch.randn((spec.N, rank), generator=gen, device=device)).to(
            torch.bfloat16)
        q = torch.empty((spec.M, spec.K), dtype=torch.int8, device=device)
        Tl = torch.empty((spec.M, rank), dtype=torch.float32, device=device)
        cs = T.weight_colsums(W)
        zw = 128.0 + 8.0 * torch.randn(spec.N, generator=gen, device=device)
        rs = torch.empty(spec.M, dtype=torch.int32, device=device)
        rsums.append(rs)
        xs.append((x, down))
        codes.append(q)
        Ts.append(Tl)
        hold += [cs, up, zw]
        plain.append(T.make_layer(q, W, 0.0, sw, None, None, y, act=params[l], colsums=cs))
        lowrank.append(T.make_layer(q, W, 0.0, sw, None, None, y, act=params[l], colsums=cs,
                                    lowrank=(Tl, up)))
        wzero.append(T.make_layer(q, W, 0.0, sw, None, None, y, act=params[l], colsums=cs,
                                  wzero=(zw, rs)))
    torch.cuda.synchronize()

    xlist = [x for x, _ in xs]
    plist = [params[l] for l in range(len(xs))]

    def quantize_all(kind):
        if kind == "lowrank":
            for l, (x, down) in enumerate(xs):
                T.quantize_activations_lowrank(x, down, out=codes[l], params=params[l], T=Ts[l])
            return
        if kind == "single":
            for l, x in enumerate(xlist):
                T.quantize_activations(x, out=codes[l], params=params[l])
            return
        T.quantize_activations_batch(xlist, codes, plist)
        if kind == "wzero":
            for l in range(len(xs)):
                T.row_sums(codes[l], out=rsums[l])

    ev = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    elems = sum(float(s.M * s.K) for s in wl.layers)
    out = {}
    for name, layers, kind in (("plain", plain, "plain"), (f"lowrank_r{rank}", lowrank, "lowrank"),
                               ("zero_point_weights", wzero, "wzero")):
        with_lr = kind == "lowrank"
        quantize_all(kind)
        T.run_schedule(layers, table, wl.S, wl.T, 0, 1, workspace=ws)
        torch.cuda.synchronize()
        q_ms, g_ms = [], []
        a0, a1 = ev(), ev()
        a0.record()
        for _ in range(reps):
            for t in range(wl.T):
                e0, e1, e2 = ev(), ev(), ev()
                e0.record()
                quantize_all(kind)
                e1.record()
                T.run_schedule(layers, table, wl.S, wl.T, t, t + 1, workspace=ws)
                e2.record()
                q_ms.append((e0, e1))
                g_ms.append((e1, e2))
        a1.record()
        torch.cuda.synchronize()
        qm = float(np.mean([a.elapsed_time(b) for a, b in q_ms]))
        gm = float(np.mean([a.elapsed_time(b) for a, b in g_ms]))
        alg = 5.0 * elems + (4.0 * rank * sum(float(s.M) for s in wl.layers) if with_lr else 0)
        if kind == "wzero":            # the row sums read the codes once more
            alg += elems + 4.0 * sum(float(s.M) for s in wl.layers)
        ach = alg / (qm * 1e-3) / 1e9
        if kind == "plain":
            # the same quantization as one pair of launches per tensor
            quantize_all("single")
            torch.cuda.synchronize()
            s0, s1 = ev(), ev()
            s0.record()
            for _ in range(reps * 4):
                quantize_all("single")
            s1.record()
            torch.cuda.synchronize()
            single_ms = s0.elapsed_time(s1) / (reps * 4)
        out[name] = {
            "ms_per_denoising_step": round(a0.elapsed_time(a1) / reps / wl.T, 4),
            "quantize_ms": round(qm, 4), "grouped_launch_ms": round(gm, 4),
            "quantizer_roofline": {
                "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4), "algorithmic_bytes": alg,
                "kernels": {"plain": "k_act_batch (one launch per group of tensors, plus one)",
                            "lowrank": "k_lowrank_down<true>, k_act_quantize per layer",
                            "wzero": "k_act_batch, then k_row_sums per layer"}[kind]}}
        if kind == "plain":
            out[name]["quantize_ms_per_tensor_calls"] = round(single_ms, 4)
    return out


def weight_quantizer(wl, device, reps=3):
    """The offline step before the weight buffer exists: the per-channel
    weight quantizer over the fp32 weights of all 112 layers (seeded normal
    draws, per-channel spread), as one batched call (outputs allocated
    once) and as one call per layer.  Milliseconds per pass and its HBM
    roofline (algorithmic bytes: 4 read + 1 written per weight)."""
    gen = torch.Generator(device=device)
    Ws = []
    for l, spec in enumerate(wl.layers):
        gen.manual_seed(wl.seed * 7000 + l)
        Ws.append(0.03 * torch.randn((spec.N, spec.K), generator=gen, device=device))
    outs = T.quantize_weights_batch(Ws)
    torch.cuda.synchronize()
    ev = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731
    a, b = ev(), ev()
    a.record()
    for _ in range(reps):
        T.quantize_weights_batch(Ws, outs)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    # the same as one tasq_quantize_weights call per layer
    c, d = ev(), ev()
    c.record()
    for _ in range(reps):
        for W in Ws:
            T.quantize_weights(W)
    d.record()
    torch.cuda.synchronize()
    single_ms = c.elapsed_time(d) / reps
    elems = sum(float(s.N * s.K) for s in wl.layers)
    ach = 5.0 * elems / (ms * 1e-3) / 1e9
    return {"ms_all_layers": round(ms, 4), "ms_one_call_per_layer": round(single_ms, 4),
            "weights": elems,
            "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                         "algorithmic_bytes": 5.0 * elems,
                         "kernel": "k_weight_quantize_batch (one launch per 16 layers)"}}


def host_info():
    """Logical CPUs of this process and the CPU model (lscpu)."""
    import subprocess
    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    return {"nproc": len(os.sched_getaffinity(0)), "cpu_model": model}


def cpu_baseline(wl, table, run_s=3.0, runs=3):
    """The CPU oracle on a bounded sample: the first R rows of each of block
    0's four linears at its stage-0 b.  For one thread and for every thread
    the oracle uses (OpenMP over output rows), R is grown until one pass
    takes about run_s seconds; then `runs` passes are timed and the median
    taken.  Returns int8 TOPS (same op count convention); `value` is the
    all-thread median."""
    import oracle
    oracle.build(force=False)
    all_threads = oracle.num_threads()
    Ws = [inputs.w_full(wl, l) for l in range(4)]
    sws = [inputs.sw_full(wl, l) for l in range(4)]

    def one_pass(R):
        Xs = [inputs.x_rows(wl, l, np.arange(R)) for l in range(4)]
        ops, t0 = 0.0, time.perf_counter()
        for l in range(4):
            spec = wl.layers[l]
            oracle.masked_linear(Xs[l], Ws[l], wl.sx, sws[l], int(table[l][0]))
            ops += 2.0 * R * spec.N * spec.K
        return ops, time.perf_counter() - t0

    out = {}
    for name, threads in (("single_thread", 1), ("all_threads", all_threads)):
        oracle.set_num_threads(threads)
        R = 4
        while True:
            ops, dt = one_pass(R)
            if dt >= run_s / 2 or R >= 8192:
                break
            R = min(8192, int(R * max(2.0, run_s / max(dt, 1e-3))))
        tops = []
        for _ in range(runs):
            ops, dt = one_pass(R)
            tops.append(ops / dt / 1e12)
        out[name] = {"TOPS_median": float(np.median(tops)), "TOPS_runs": tops, "threads": threads,
                     "rows": R, "macs_per_run": ops / 2}
    oracle.set_num_threads(all_threads)
    info = host_info()
    allt = out["all_threads"]
    return dict(value=allt["TOPS_median"], unit="TOPS", cores=all_threads, kind="oracle",
                sample=f"rows 0..R-1 of block 0's four linears at the stage-0 b, median of "
                       f"{runs} runs per thread count (all threads: R = {allt['rows']}, "
                       f"{allt['macs_per_run']:.3g} MACs per run; one thread: R = "
                       f"{out['single_thread']['rows']})",
                single_thread_TOPS=out["single_thread"]["TOPS_median"],
                all_threads_TOPS=allt["TOPS_median"], runs=out, **info)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--tokens", type=int, default=None, help="override M (skinny sweeps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--rounds", type=int, default=5,
                    help="rounds of the interleaved TASQ / static-8 / static-max timing")
    ap.add_argument("--skinny-sweep", action="store_true",
                    help="only time single weight-streaming layers (M = 1, 16, 64) and print one "
                         "JSON line per layer shape")
    ap.add_argument("--shape-sweep", action="store_true",
                    help="only time the single layers of the four per-shape workloads (median / "
                         "p10 / p90 over 50 cache-flushed launches) and print one JSON line each")
    ap.add_argument("--skinny-only", action="store_true",
                    help="only time the 112-layer schedule at M = 16 (weight streaming) and print "
                         "its JSON")
    ap.add_argument("--no-skinny", action="store_true",
                    help="skip the extra weight-streaming (M=16) schedule measurement")
    ap.add_argument("--shard-shapes", action="store_true",
                    help="only the step at one GPU's share of the 8-way token and channel "
                         "splits (one JSON line)")
    ap.add_argument("--no-act", action="store_true",
                    help="skip the extra asymmetric-activation (fp32 input) measurement")
    ap.add_argument("--per-layer", action="store_true",
                    help="launch each layer separately instead of one grouped launch per step")
    ap.add_argument("--weights", choices=("packed", "rowmajor"), default="rowmajor",
                    help="weight buffer layout: packed (operand order, no LDS staging of "
                         "weights) or row-major [N][K] (weights staged through LDS)")
    ap.add_argument("--print-source-hash", action="store_true",
                    help="print the HIP source hash that recorded counter readings refer to "
                         "(of the grouped kernel of --weights)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only copy a 1 GiB buffer (reference for the FETCH_SIZE/WRITE_SIZE "
                         "counters) and exit")
    args = ap.parse_args()
    if args.print_source_hash:
        print(kernel_source_sha256(step_kernel(args.weights)))
        return
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel(), "reps": 3}), flush=True)
        return
    if args.shape_sweep:
        for row in shape_sweep("cuda"):
            print(json.dumps(row), flush=True)
        for row in config_schedules("cuda"):
            print(json.dumps(row), flush=True)
        return
    if args.shard_shapes:
        wl = inputs.workload(4)
        table = inputs.b_table(wl)
        log("building the full step and timing it")
        layers, keep = build_workload(wl, "cuda", packed=False)
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device="cuda")
        full_ms = time_schedule(layers, table, wl, ws, 3, 1)
        log("timing one GPU's share of the 8-way token and channel splits")
        row = {"workload": wl.name, "full_ms_per_schedule": round(full_ms, 4),
               "full_ms_per_denoising_step": round(full_ms / wl.T, 4)}
        row.update(shard_shapes(wl, table, keep, full_ms, "cuda"))
        print(json.dumps(row), flush=True)
        return
    if args.skinny_sweep:
        for row in skinny_sweep("cuda"):
            print(json.dumps(row), flush=True)
        return
    if args.skinny_only:
        wl = inputs.workload(4)
        keep = [(None, inputs.w_full(wl, l).to("cuda"), inputs.sw_full(wl, l).to("cuda"), None)
                for l in range(len(wl.layers))]
        print(json.dumps(skinny_schedule(wl, inputs.b_table(wl), keep, "cuda", M=args.tokens or 16)),
              flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus}); the path shards by "
              "rows or output channels with no exchange, see DESIGN.md", file=sys.stderr)
        sys.exit(2)
    dev = "cuda"
    wl = inputs.workload(4, M_override=args.tokens)
    table = inputs.b_table(wl)
    log(f"building {len(wl.layers)} layers, M={wl.layers[0].M}")
    layers, keep = build_workload(wl, dev, packed=args.weights == "packed")
    ws = None
    if not args.per_layer:
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=dev)
    t8 = torch.full_like(table, 8)
    tmax = table.max(dim=1, keepdim=True).values.expand_as(table).contiguous()
    torch.cuda.synchronize()

    log("timing schedules")
    ms = time_schedule(layers, table, wl, ws, args.steps, args.warmup)
    ops_step = gemm_ops(wl)
    total_ops = ops_step * wl.T
    value = total_ops / (ms * 1e-3) / 1e12

    roof = None
    kname = step_kernel(args.weights)
    launch_ms = launch_pairs_ms = None
    if ws is not None:
        # The timed region holds nothing but this kernel's launches (one per
        # denoising step, back to back, plus one upload of the layer list per
        # schedule call), so its average launch duration is the timed time
        # over the launches; event pairs around single launches (which add a
        # lone launch's dispatch latency) are reported beside it.
        launch_ms = ms / wl.T
        launch_pairs_ms = time_launches(layers, table, wl, ws)
    log("timing the TASQ, static b=8 and static max-over-stages tables in turn")
    inter = time_tables_interleaved(layers, {"tasq_table": table, "static_b8": t8,
                                             "static_max_over_stages": tmax}, wl, ws,
                                    rounds=args.rounds)
    if launch_ms is not None:
        t_mfma = ops_step / (PEAK_INT8_TOPS * 1e12)
        t_hbm = gemm_bytes(wl) / (PEAK_HBM_GBS * 1e9)
        if t_hbm >= t_mfma:
            ach = gemm_bytes(wl) / (launch_ms * 1e-3) / 1e9
            roof = dict(bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                        frac=round(ach / PEAK_HBM_GBS, 4), traffic=recorded_traffic(kname))
        else:
            ach = ops_step / (launch_ms * 1e-3) / 1e12
            roof = dict(bound="mfma", achieved=round(ach, 1), peak=PEAK_INT8_TOPS, unit="TOP/s",
                        frac=round(ach / PEAK_INT8_TOPS, 4), traffic=recorded_traffic(kname))
        roof["kernel"] = (f"{kname}_ds" if kname == "k_masked_gemm_persistent" else kname) + " (one launch = one denoising step, 112 GEMMs)"
        roof["launch_ms"] = round(launch_ms, 4)
        roof["launch_ms_event_pairs"] = round(launch_pairs_ms, 4)
        roof["mfma_frac"] = round(ops_step / (launch_ms * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4)
        roof["roofline_ms"] = round(max(t_mfma, t_hbm) * 1e3, 4)
        roof["algorithmic_bytes"] = gemm_bytes(wl)
        roof["algorithmic_ops"] = ops_step
        ctr = recorded_counters(kname)
        roof["clock_GHz_under_load"] = None if ctr is None else ctr["tasq_table"]["clock_GHz"]
        roof["mfma_busy_pct"] = None if ctr is None else ctr["tasq_table"]["mfma_busy_pct"]

    peaks = measured_peaks(dev)
    if roof is not None:
        # the same launch against what this GPU was measured to sustain
        if roof["bound"] == "hbm":
            roof["frac_of_measured_peak"] = round(roof["achieved"] / peaks["copy_GBps"], 4)
        else:
            roof["frac_of_measured_peak"] = round(roof["achieved"] / peaks["mfma_int8_TOPS"], 4)

    skinny = None
    if not args.no_skinny and not args.per_layer:
        log("timing the weight-streaming schedule at M=16")
        skinny = skinny_schedule(wl, table, keep, dev)

    act = wq = None
    if not args.no_act and not args.per_layer:
        log("timing the asymmetric-activation schedule")
        act = act_schedule(wl, table, keep, ws, dev)
        log("timing the weight quantizer")
        wq = weight_quantizer(wl, dev)

    # The paper's compute accounting of the same schedule next to the
    # measured wall-time ratios (table vs static 8-bit weights).
    cost = T.schedule_cost([(sp.M, sp.N, sp.K) for sp in wl.layers], table, wl.S, wl.T, 0,
                           wl.T, 8)
    accounting = {k: round(v, 4) if k not in ("macs", "bitops") else v for k, v in cost.items()}
    accounting["measured_ratio_vs_static_b8"] = round(
        inter["tasq_table"]["median"] / inter["static_b8"]["median"], 4)
    if skinny is not None:
        accounting["measured_ratio_vs_static_b8_m16_auto"] = round(
            skinny["ms_per_denoising_step"]["auto_tasq"] /
            skinny["ms_per_denoising_step"]["auto_b8"], 4)

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle sample")
        cpu = cpu_baseline(wl, table)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": len(wl.layers), "M": wl.layers[0].M,
                   "denoising_steps": wl.T, "stages": wl.S, "output": "fp32",
                   "launch": "per-layer" if args.per_layer else "grouped per denoising step",
                   "weights": args.weights},
        "schedule_ms": {"tasq_table": round(ms, 4),
                        "interleaved": inter,
                        "interleaved_rounds": args.rounds},
        "margin_vs_static_b8": round(
            1.0 - inter["tasq_table"]["median"] / inter["static_b8"]["median"], 4),
        "margin_vs_static_max_over_stages": round(
            1.0 - inter["tasq_table"]["median"] / inter["static_max_over_stages"]["median"], 4),
        "mean_bits": round(float(table.float().mean()), 3),
        "accounting": accounting,
        "roofline": roof,
        "measured_peaks": peaks,
        "skinny_schedule": skinny,
        "asymmetric_activations": act,
        "weight_quantizer": wq,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
