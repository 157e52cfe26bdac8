"""Full-size schedules through tasq_run_schedule with a workspace.

Config 4 at full size in the benchmark's own launch configuration: the
28-block PixArt-shaped stack (112 linears at M = 8192) through
tasq_run_schedule with a workspace, i.e. one persistent grouped launch per
denoising step, fp32 outputs only, inputs drawn exactly as bench.py draws
them.  After a step range every layer holds the output of the range's last
step, at that step's stage b; sampled outputs of every layer are checked
against the oracle entry by entry: fp32 within 1e-6 relative, and, in a
second pass with int32 outputs requested as well (the general epilogue of
the same launch), the int32 accumulators bit-exactly.  Configs 1-3 (one
DiT, one SANA and one UNet block with its 3x3 conv) likewise, sampled
outputs of every layer at the end of each stage."""
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


@pytest.fixture(scope="module")
def cfg4():
    """Config 4's 112 layers on the GPU, drawn as bench.py draws them."""
    wl = inputs.workload(4)
    table = inputs.b_table(wl)
    Ws, sws, keep = [], [], []
    for l, spec in enumerate(wl.layers):
        X = inputs.x_full(wl, l, device=DEV)
        W = inputs.w_full(wl, l)
        sw = inputs.sw_full(wl, l)
        keep.append((X, W.to(DEV), sw.to(DEV)))
        Ws.append(W)
        sws.append(sw)
    return wl, table, Ws, sws, keep


def test_config4_schedule_bench_launch_sampled(cfg4):
    wl, table, Ws, sws, keep = cfg4
    L = len(wl.layers)
    ys, layers = [], []
    for l, spec in enumerate(wl.layers):
        X, Wd, swd = keep[l]
        y = torch.full((spec.M, spec.N), -7.0, dtype=torch.float32, device=DEV)
        layers.append(T.make_layer(X, Wd, wl.sx, swd, None, None, y))
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


def test_config4_comparison_tables_and_packed_weights_sampled(cfg4):
    """The benchmark's comparison schedules at full size: the static b = 8
    table and the per-layer maximum over stages through the same grouped
    launch, and the TASQ table with every layer holding only its packed
    weight (bench.py --weights packed: the grouped packed-weight launch);
    sampled outputs of every seventh layer after the last step."""
    wl, table, Ws, sws, keep = cfg4
    L = len(wl.layers)
    t8 = torch.full_like(table, 8)
    tmax = table.max(dim=1, keepdim=True).values.expand_as(table).contiguous()
    ys = [torch.empty((s.M, s.N), dtype=torch.float32, device=DEV) for s in wl.layers]
    layers = [T.make_layer(keep[l][0], keep[l][1], wl.sx, keep[l][2], None, None, ys[l])
              for l in range(L)]
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    rng = np.random.default_rng(45)
    stage = oracle.stage_of_step(wl.T - 1, wl.S, wl.T)
    for name, tab in (("static b=8", t8), ("static max over stages", tmax)):
        for y in ys:
            y.fill_(-7.0)
        T.run_schedule(layers, tab, wl.S, wl.T, wl.T - 2, wl.T, workspace=ws)
        torch.cuda.synchronize()
        for l in range(0, L, 7):
            b = int(tab[l, stage])
            check_layer(wl, l, Ws[l], sws[l], ys[l].cpu(), None, b, rng,
                        f"config 4 {name} layer {l} b={b}")
    packs = [T.pack_weights(keep[l][1]) for l in range(L)]
    layers = [T.make_layer(keep[l][0], None, wl.sx, keep[l][2], None, None, ys[l],
                           packed=packs[l]) for l in range(L)]
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for y in ys:
        y.fill_(-7.0)
    T.run_schedule(layers, table, wl.S, wl.T, wl.T - 2, wl.T, workspace=ws)
    torch.cuda.synchronize()
    for l in range(3, L, 7):
        b = int(table[l, stage])
        check_layer(wl, l, Ws[l], sws[l], ys[l].cpu(), None, b, rng,
                    f"config 4 packed weights layer {l} b={b}")


@pytest.mark.parametrize("source", ["rows", "packed", "planes", "auto"])
def test_config4_weight_streaming_schedule_m16_sampled(cfg4, source):
    """The benchmark's weight-streaming schedule at full size: config 4's 112
    layers at 16 tokens (the first 16 activation rows, as bench.py draws
    them), one grouped weight-streaming launch per step, the weight read as
    int8 rows, as the packed copy, as the top b planes, or under AUTO with
    all three copies given (the planes below b = 8).  After steps 18-19 every
    layer holds the last step's output: all 16 rows of 40 sampled columns
    (and the last) per layer against the oracle, fp32 within 1e-6 relative
    and the int32 accumulators bit-exactly."""
    wl, table, Ws, sws, keep = cfg4
    L, M = len(wl.layers), 16
    rng = np.random.default_rng(61)
    hold, layers, outs = [], [], []
    for l, spec in enumerate(wl.layers):
        X = inputs.x_rows(wl, l, np.arange(M), device=DEV)
        W = keep[l][1]
        P = T.pack_weights(W) if source in ("packed", "auto") else None
        Q = T.pack_planes(W) if source in ("planes", "auto") else None
        y = torch.full((M, spec.N), -7.0, dtype=torch.float32, device=DEV)
        acc = torch.full((M, spec.N), 12345, dtype=torch.int32, device=DEV)
        Wuse = W if source in ("rows", "auto") else None
        layers.append(T.make_layer(X, Wuse, wl.sx, keep[l][2], None, acc, y, packed=P, planes=Q))
        hold += [X, P, Q]
        outs.append((acc, y))
    variant = T.VARIANT_BITPLANE if source == "planes" else T.VARIANT_AUTO
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    T.run_schedule(layers, table, wl.S, wl.T, wl.T - 2, wl.T, workspace=ws, variant=variant)
    torch.cuda.synchronize()
    stage = oracle.stage_of_step(wl.T - 1, wl.S, wl.T)
    sx = f32(wl.sx)
    for l, spec in enumerate(wl.layers):
        b = int(table[l, stage])
        cols = np.array(sorted(set(rng.integers(0, spec.N, 40).tolist() + [spec.N - 1])),
                        np.int64)
        Xr = inputs.x_rows(wl, l, np.arange(M))
        tc = torch.as_tensor(cols)
        rr = np.repeat(np.arange(M), len(cols))
        cc = np.tile(np.arange(len(cols)), M)
        ra, ry = oracle.masked_linear_entries(Xr, Ws[l][tc], sx, sws[l][tc], b, rr, cc)
        acc, y = outs[l]
        check_outputs(acc[:, tc].cpu(), y[:, tc].cpu(), ra.reshape(M, len(cols)),
                      ry.reshape(M, len(cols)), sx, sws[l][tc], None,
                      f"config 4 at 16 tokens, {source}, layer {l} b={b}")


@pytest.mark.parametrize("axis", ["M", "N"])
def test_config4_shard_schedules_sampled(cfg4, axis):
    """One GPU's share of an 8-way split of config 4 at its real shapes, as
    bench.py --shard-shapes times it: shard 0 of the token split (the first
    1024 rows of every layer) or of the channel split (the first N/8 output
    channels: 432, 144, 576, 144 per block), operands as views of the full
    device tensors, all 20 denoising steps through the bench's launch.
    Sampled outputs of the layers of blocks 0, 9, 18 and 27 against the
    oracle, fp32 within 1e-6 relative."""
    wl, table, Ws, sws, keep = cfg4
    swl = inputs.shard(wl, axis, 8)
    layers, ys = [], []
    for l, spec in enumerate(swl.layers):
        X, Wd, swd = keep[l]
        if axis == "M":
            X = X[:spec.M]
        else:
            Wd, swd = Wd[:spec.N], swd[:spec.N]
        y = torch.full((spec.M, spec.N), -7.0, dtype=torch.float32, device=DEV)
        layers.append(T.make_layer(X, Wd, swl.sx, swd, None, None, y))
        ys.append(y)
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    T.run_schedule(layers, table, swl.S, swl.T, 0, swl.T, workspace=ws)
    torch.cuda.synchronize()
    stage = oracle.stage_of_step(swl.T - 1, swl.S, swl.T)
    rng = np.random.default_rng(45)
    for blk in (0, 9, 18, 27):
        for l in range(4 * blk, 4 * blk + 4):
            spec = swl.layers[l]
            W = Ws[l] if axis == "M" else Ws[l][:spec.N]
            sw = sws[l] if axis == "M" else sws[l][:spec.N]
            check_layer(swl, l, W, sw, ys[l], None, int(table[l, stage]), rng,
                        f"config 4 shard 0 of 8 along {axis}, layer {l}")


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_block_schedules_full_size_sampled(cfg):
    """Configs 1-3 as full-size schedules through tasq_run_schedule with a
    workspace (the grouped per-step launch: persistent for the DiT blocks,
    one workgroup per tile for the UNet block with its 3x3 conv), every step
    range ending in each stage; sampled outputs of every layer (pixels x all
    channels for the conv) against the oracle, int32 bit-exact and fp32
    within 1e-6 relative."""
    wl = inputs.workload(cfg)
    table = inputs.b_table(wl)
    sx = f32(wl.sx)
    host, keep, layers = [], [], []
    for l, spec in enumerate(wl.layers):
        X = inputs.x_full(wl, l)
        W = inputs.w_full(wl, l)
        if spec.kind == "conv3x3":
            W = W.reshape(spec.N, 3, 3, spec.C)
            shape = (spec.H, spec.Wd, spec.N)
        else:
            shape = (spec.M, spec.N)
        sw = inputs.sw_full(wl, l)
        Xd, Wd, swd = X.to(DEV), W.to(DEV), sw.to(DEV)
        acc = torch.full(shape, 12345, dtype=torch.int32, device=DEV)
        y = torch.full(shape, -7.0, dtype=torch.float32, device=DEV)
        layers.append(T.make_layer(Xd, Wd, wl.sx, swd, None, acc, y))
        keep.append((Xd, Wd, swd))
        host.append((X, W, sw, acc, y))
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    rng = np.random.default_rng(50 + cfg)
    ends = sorted({max(t for t in range(wl.T) if oracle.stage_of_step(t, wl.S, wl.T) == s)
                   for s in range(wl.S)})
    for t1 in ends:
        t0 = max(0, t1 - 1)
        T.run_schedule(layers, table, wl.S, wl.T, t0, t1 + 1, workspace=ws)
        torch.cuda.synchronize()
        stage = oracle.stage_of_step(t1, wl.S, wl.T)
        for l, spec in enumerate(wl.layers):
            X, W, sw, acc, y = host[l]
            b = int(table[l, stage])
            where = f"config {cfg} [{t0},{t1 + 1}) {spec.name} b={b}"
            if spec.kind == "conv3x3":
                pix = sorted(set([0, spec.Wd - 1, spec.Wd, spec.H * spec.Wd - 1]
                                 + rng.integers(0, spec.H * spec.Wd, 6).tolist()))
                pp = np.repeat(np.array(pix), spec.N)
                cc = np.tile(np.arange(spec.N), len(pix))
                ra, ry = oracle.conv3x3_entries(X, W, sx, sw, b, pp, cc)
                ti = torch.as_tensor(pix)
                check_outputs(acc.reshape(-1, spec.N)[ti], y.reshape(-1, spec.N)[ti],
                              ra.reshape(len(pix), spec.N), ry.reshape(len(pix), spec.N), sx,
                              sw, None, where)
            else:
                rows = sample_rows(spec.M, rng, 4)
                rr = np.repeat(np.arange(len(rows)), spec.N)
                cc = np.tile(np.arange(spec.N), len(rows))
                ra, ry = oracle.masked_linear_entries(X[torch.as_tensor(rows)], W, sx, sw, b,
                                                      rr, cc)
                ti = torch.as_tensor(rows)
                check_outputs(acc[ti], y[ti], ra.reshape(len(rows), spec.N),
                              ry.reshape(len(rows), spec.N), sx, sw, None, where)
