"""Boundary semantics through the C ABI on the GPU: calls are asynchronous
and stream-ordered (a schedule returns to the host while earlier work on its
stream still runs, and its results are there once the stream is
synchronised); repeated grouped schedules write identical bits; and the
AUTO variant reads the weight copy its per-shape rule names (the top b bit
planes for weight streams of at most 64 tokens, the packed copy at b = 8,
the packed or row-major copy for large M).  To see which copy a call read,
the row-major, packed and bit-plane buffers passed together hold three
different weights, each with its own oracle result."""
import ctypes
import os
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_parity import DEV, check_outputs, f32, small_schedule_layers

pytestmark = pytest.mark.gpu
SX = f32(0.02)
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def busy_kernel():
    """A launcher of ~tens of milliseconds of matrix-instruction work on the
    current stream (the benchmark's peak probe, 768 workgroups)."""
    probe = ctypes.CDLL(os.path.join(ROOT, "paper_2608_03057_amd", "libtasq_probe.so"))
    probe.tasq_probe_mfma_peak.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                           ctypes.c_void_p]
    sink = torch.empty(768 * 256, dtype=torch.int32, device=DEV)

    def run(iters):
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        assert probe.tasq_probe_mfma_peak(768, iters, ctypes.c_void_p(sink.data_ptr()),
                                          stream) == 0
    return run, sink


def test_schedule_is_asynchronous_and_stream_ordered():
    busy, sink = busy_kernel()
    host, dev, rng = small_schedule_layers(31)
    S, Tn = 4, 20
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S)), dtype=torch.uint8)
    layers = [T.make_layer(d["X"], d["W"], SX, d["sw"], d.get("bias"), d["acc"], d["y"])
              for d in dev]
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    T.run_schedule(layers, table, S, Tn, 0, 1, workspace=ws)
    busy(100)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    busy(100000)
    b.record()
    torch.cuda.synchronize()
    busy_ms = a.elapsed_time(b)
    assert busy_ms > 20.0, f"busy kernel too short to test with ({busy_ms:.1f} ms)"
    for d in dev:
        d["acc"].fill_(12345)
        d["y"].fill_(-7.0)
    done = torch.cuda.Event()
    busy(100000)
    t0 = time.perf_counter()
    T.run_schedule(layers, table, S, Tn, 3, 11, workspace=ws)
    host_ms = (time.perf_counter() - t0) * 1e3
    done.record()
    pending = not done.query()
    torch.cuda.synchronize()
    assert host_ms < 0.25 * busy_ms, f"run_schedule held the host {host_ms:.2f} ms " \
                                     f"behind {busy_ms:.1f} ms of queued work"
    assert pending, "the schedule finished before the earlier work on its stream"
    ref = oracle.run_schedule(host, table.numpy(), S, Tn, 3, 11, SX)
    for h, d, (ra, ry, bb) in zip(host, dev, ref):
        check_outputs(d["acc"], d["y"], ra, ry, SX, h["sw"], h.get("bias"), f"b={bb}")
    del sink


def test_grouped_schedule_deterministic_over_100_runs():
    host, dev, rng = small_schedule_layers(32)
    S, Tn = 4, 20
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S)), dtype=torch.uint8)
    layers = [T.make_layer(d["X"], d["W"], SX, d["sw"], d.get("bias"), d["acc"], d["y"])
              for d in dev]
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    first = None
    for rep in range(100):
        T.run_schedule(layers, table, S, Tn, 5, 6, workspace=ws)
        got = [(d["acc"].clone(), d["y"].view(torch.int32).clone()) for d in dev]
        if first is None:
            first = got
        else:
            for (a0, y0), (a1, y1) in zip(first, got):
                assert torch.equal(a0, a1) and torch.equal(y0, y1), f"run {rep}"
    torch.cuda.synchronize()


def three_weights(seed, N, K):
    """Three different int8 weights of one shape and their scales."""
    Ws = [inputs.random_case(seed + i, 1, N, K)[1] for i in range(3)]
    sw = inputs.uniform_f32(seed, 3, torch.arange(N), 1e-3, 1e-2)
    return Ws, sw


@pytest.mark.parametrize("M", [1, 16, 64, 65, 8192])
def test_auto_picks_weight_copy_per_shape(M):
    N, K = 160, 384
    (W_rows, W_packed, W_planes), sw = three_weights(700 + M, N, K)
    X = inputs.random_case(710 + M, M, N, K)[0]
    Xd, swd = X.to(DEV), sw.to(DEV)
    rows_d = W_rows.to(DEV)
    packed_d = T.pack_weights(W_packed.to(DEV))
    planes_d = T.pack_planes(W_planes.to(DEV))
    skinny = M <= 64
    for b in (8, 5, 1):
        cases = [
            # (copies given, weight AUTO must read)
            (dict(W=rows_d, planes=planes_d), W_planes if skinny else W_rows),
            # rows and packed: a stream takes the packed copy; a layer of at
            # most 128 256x256 tiles (this one has 32 at M = 8192) the rows
            (dict(W=rows_d, planes=planes_d, packed=packed_d),
             (W_planes if b < 8 else W_packed) if skinny else W_rows),
            (dict(W=None, planes=planes_d), W_planes),
            (dict(W=None, planes=planes_d, packed=packed_d),
             W_planes if skinny and b < 8 else W_packed),
        ]
        for copies, want in cases:
            W = copies.pop("W")
            acc, y = T.masked_linear(Xd, W, SX, swd, b, **copies)
            torch.cuda.synchronize()
            ra, ry = oracle.masked_linear(X, want, SX, sw, b)
            check_outputs(acc, y, ra, ry, SX, sw, None,
                          f"M={M} b={b} copies={sorted(copies) + (['W'] if W is not None else [])}")


def test_auto_large_layer_reads_packed_copy():
    """A single layer of more than 128 256x256 tiles (4096 x 4352: 272) under
    AUTO with both int8 copies given reads the packed copy; the same weights
    in a grouped schedule read the rows (the persistent step).  Sampled rows
    against the oracle."""
    M, N, K = 4096, 4352, 256
    (W_rows, W_packed, _), sw = three_weights(760, N, K)
    X = inputs.random_case(761, M, N, K)[0]
    Xd, swd = X.to(DEV), sw.to(DEV)
    rows_d, packed_d = W_rows.to(DEV), T.pack_weights(W_packed.to(DEV))
    rows = slice(2000, 2064)
    acc, y = T.masked_linear(Xd, rows_d, SX, swd, 6, packed=packed_d)
    torch.cuda.synchronize()
    ra, ry = oracle.masked_linear(X[rows], W_packed, SX, sw, 6)
    check_outputs(acc[rows], y[rows], ra, ry, SX, sw, None, "single layer, AUTO, packed copy")
    acc.fill_(0)
    y.fill_(0)
    layer = T.make_layer(Xd, rows_d, SX, swd, None, acc, y, packed=packed_d)
    ws = torch.empty(T.schedule_workspace_bytes([layer]), dtype=torch.uint8, device=DEV)
    T.run_schedule([layer], torch.tensor([[6]], dtype=torch.uint8), 1, 1, 0, 1, workspace=ws)
    torch.cuda.synchronize()
    ra, ry = oracle.masked_linear(X[rows], W_rows, SX, sw, 6)
    check_outputs(acc[rows], y[rows], ra, ry, SX, sw, None, "schedule, AUTO, rows")


def test_auto_schedule_streams_planes():
    """A grouped weight-streaming schedule (every layer at 16 tokens) under
    AUTO with the row-major weight and its planes given reads the planes;
    with a static b = 8 table and packed copies as well it reads the packed
    copies."""
    shapes = [(16, 200, 1152), (16, 96, 640), (16, 33, 128)]
    S, Tn = 2, 4
    host, layers, keep = [], [], []
    for i, (M, N, K) in enumerate(shapes):
        (W_rows, W_packed, W_planes), sw = three_weights(720 + 10 * i, N, K)
        X = inputs.random_case(730 + i, M, N, K)[0]
        d = dict(X=X.to(DEV), W=W_rows.to(DEV), sw=sw.to(DEV),
                 P=T.pack_planes(W_planes.to(DEV)), Wp=T.pack_weights(W_packed.to(DEV)),
                 acc=torch.empty((M, N), dtype=torch.int32, device=DEV),
                 y=torch.empty((M, N), dtype=torch.float32, device=DEV))
        keep.append(d)
        host.append((X, W_rows, W_packed, W_planes, sw))
    for with_packed, tab in ((False, [[7, 3], [2, 8], [5, 8]]), (True, [[8, 8], [8, 8], [8, 8]])):
        table = torch.tensor(tab, dtype=torch.uint8)
        layers = [T.make_layer(d["X"], d["W"], SX, d["sw"], None, d["acc"], d["y"],
                               planes=d["P"], packed=d["Wp"] if with_packed else None)
                  for d in keep]
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
        T.run_schedule(layers, table, S, Tn, 0, Tn, workspace=ws)
        torch.cuda.synchronize()
        for i, (d, (X, W_rows, W_packed, W_planes, sw)) in enumerate(zip(keep, host)):
            b = int(table[i, S - 1])
            want = W_packed if with_packed else W_planes
            ra, ry = oracle.masked_linear(X, want, SX, sw, b)
            check_outputs(d["acc"], d["y"], ra, ry, SX, sw, None,
                          f"layer {i} packed={with_packed} b={b}")
