"""Config 4 at full size in the benchmark's own launch configuration: the
28-block PixArt-shaped stack (112 linears at M = 8192) through
tasq_run_schedule with a workspace, i.e. one persistent grouped launch per
denoising step, fp32 outputs only, inputs drawn exactly as bench.py draws
them.  After a step range every layer holds the output of the range's last
step, at that step's stage b; sampled outputs of every layer are checked
against the oracle entry by entry: fp32 within 1e-6 relative, and, in a
second pass with int32 outputs requested as well (the general epilogue of
the same launch), the int32 accumulators bit-exactly."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_parity import DEV, check_outputs, f32, sample_rows

pytestmark = pytest.mark.gpu


def check_layer(wl, l, W, sw, y, acc, b, rng, where):
    spec = wl.layers[l]
    sx = f32(wl.sx)
    rows = sample_rows(spec.M, rng, 3)
    cols = np.array(sorted(set(rng.integers(0, spec.N, 3).tolist() + [spec.N - 1])), np.int64)
    Xr = inputs.x_rows(wl, l, rows)
    rr = np.repeat(np.arange(len(rows)), spec.N)
    cc = np.tile(np.arange(spec.N), len(rows))
    ra, ry = oracle.masked_linear_entries(Xr, W, sx, sw, b, rr, cc)
    ti = torch.as_tensor(rows)
    check_outputs(None if acc is None else acc[ti], y[ti], ra.reshape(len(rows), spec.N),
                  ry.reshape(len(rows), spec.N), sx, sw, None, f"{where} rows")
    # every row of a few columns
    Xa = inputs.x_full(wl, l)
    tc = torch.as_tensor(cols)
    rr = np.repeat(np.arange(spec.M), len(cols))
    cc = np.tile(np.arange(len(cols)), spec.M)
    ra, ry = oracle.masked_linear_entries(Xa, W[tc], sx, sw[tc], b, rr, cc)
    check_outputs(None if acc is None else acc[:, tc], y[:, tc], ra.reshape(spec.M, len(cols)),
                  ry.reshape(spec.M, len(cols)), sx, sw[tc], None, f"{where} cols")


def test_config4_schedule_bench_launch_sampled():
    wl = inputs.workload(4)
    table = inputs.b_table(wl)
    L = len(wl.layers)
    Ws, sws, keep, ys, layers = [], [], [], [], []
    for l, spec in enumerate(wl.layers):
        X = inputs.x_full(wl, l, device=DEV)
        W = inputs.w_full(wl, l)
        sw = inputs.sw_full(wl, l)
        Wd, swd = W.to(DEV), sw.to(DEV)
        y = torch.full((spec.M, spec.N), -7.0, dtype=torch.float32, device=DEV)
        layers.append(T.make_layer(X, Wd, wl.sx, swd, None, None, y))
        keep.append((X, Wd, swd))
        Ws.append(W)
        sws.append(sw)
        ys.append(y)
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    rng = np.random.default_rng(44)
    # the benchmark's step: all 20 denoising steps
    T.run_schedule(layers, table, wl.S, wl.T, 0, wl.T, workspace=ws)
    torch.cuda.synchronize()
    stage = oracle.stage_of_step(wl.T - 1, wl.S, wl.T)
    for l in range(L):
        b = int(table[l, stage])
        check_layer(wl, l, Ws[l], sws[l], ys[l].cpu(), None, b, rng,
                    f"config 4 [0,{wl.T}) layer {l} b={b}")

    # one step of stage 1 with int32 outputs as well, every layer
    accs = []
    layers = []
    for l, spec in enumerate(wl.layers):
        acc = torch.full((spec.M, spec.N), 12345, dtype=torch.int32, device=DEV)
        accs.append(acc)
        X, Wd, swd = keep[l]
        layers.append(T.make_layer(X, Wd, wl.sx, swd, None, acc, ys[l]))
    t = 7
    T.run_schedule(layers, table, wl.S, wl.T, t, t + 1, workspace=ws)
    torch.cuda.synchronize()
    stage = oracle.stage_of_step(t, wl.S, wl.T)
    for l in range(0, L, 5):
        b = int(table[l, stage])
        check_layer(wl, l, Ws[l], sws[l], ys[l].cpu(), accs[l].cpu(), b, rng,
                    f"config 4 [{t},{t + 1}) layer {l} b={b} with int32")
