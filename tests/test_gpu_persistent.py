"""The persistent form of the grouped step (one workgroup per compute unit
walking its XCD's run of tiles, the next tile's first loads issued before
the current tile's stores), forced through the library's tuning overrides
(tasq_opts.persistent = 2, persistent_wgs workgroups per XCD,
persistent_parties parts of each XCD's run walked side by side, tile),
against the oracle on ragged linear layers, symmetric and asymmetric codes,
with and without bias.  With one or three workgroups per XCD every
workgroup runs many tiles of several layers, so each tile boundary (a new
segment, a new b, a ragged edge) is crossed inside one workgroup.  Bars as
in the other GPU tests: int32 bit-exact, fp32 within 1e-6 relative."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_act import check_asym, quantize
from test_gpu_parity import DEV, check_outputs, f32

pytestmark = pytest.mark.gpu

SX = f32(0.02)
SHAPES = [(300, 200, 304), (40, 70, 128), (33, 65, 32), (520, 260, 1152), (130, 129, 640)]


def build(seed, asym_layers=()):
    host, layers, keep = [], [], []
    for i, (M, N, K) in enumerate(SHAPES):
        X, W, sw, bias = inputs.random_case(seed * 10 + i, M, N, K)
        h = dict(X=X, W=W, sw=sw, bias=bias if i % 2 == 0 else None, asym=i in asym_layers)
        Wd = W.to(DEV)
        acc = torch.full((M, N), 12345, dtype=torch.int32, device=DEV)
        y = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
        act = cs = None
        if h["asym"]:
            x = inputs.activations_f32(seed * 10 + 5 + i, torch.arange(M), K, "skewed")
            Xd, act, h["alpha"], h["z"], h["Q"] = quantize(x)
            cs = T.weight_colsums(Wd)
        else:
            Xd = X.to(DEV)
        swd = sw.to(DEV)
        bd = None if h["bias"] is None else h["bias"].to(DEV)
        layers.append(T.make_layer(Xd, Wd, SX, swd, bd, acc, y, act=act, colsums=cs))
        keep.append((Xd, Wd, swd, bd, act, cs))
        h["acc"], h["y"] = acc, y
        host.append(h)
    return host, layers, keep


def check_layer(h, b, where):
    if h["asym"]:
        ra, ry = oracle.masked_linear_asym(h["Q"], h["W"], h["alpha"], h["z"], h["sw"], b,
                                           h["bias"])
        check_asym(h["acc"], h["y"], ra, ry, h["alpha"], h["z"], h["sw"],
                   oracle.weight_colsums(h["W"])[b - 1], h["bias"], where)
    else:
        ra, ry = oracle.masked_linear(h["X"], h["W"], SX, h["sw"], b, h["bias"])
        check_outputs(h["acc"], h["y"], ra, ry, SX, h["sw"], h["bias"], where)


@pytest.mark.parametrize("tile,wgs,parties", [(0, 1, 1), (0, 3, 1), (0, 32, 1), (2, 1, 1),
                                              (3, 5, 1), (0, 4, 2), (0, 6, 3), (2, 32, 4)])
def test_persistent_schedule(tile, wgs, parties):
    tune = dict(persistent=2, persistent_wgs=wgs, persistent_parties=parties, tile=tile + 1)
    host, layers, keep = build(70 + tile, asym_layers=(1, 3))
    S, Tn = 4, 20
    rng = np.random.default_rng(71 + wgs)
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S)), dtype=torch.uint8)
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for (t0, t1) in [(0, 20), (0, 1), (6, 7), (12, 16)]:
        T.run_schedule(layers, table, S, Tn, t0, t1, workspace=ws, tune=tune)
        torch.cuda.synchronize()
        stage = oracle.stage_of_step(t1 - 1, S, Tn)
        for i, h in enumerate(host):
            b = int(table[i, stage])
            check_layer(h, b, f"tile {tile} wgs {wgs} parties {parties} [{t0},{t1}) layer {i} "
                              f"b={b}")


@pytest.mark.parametrize("tune", [dict(persistent=2, persistent_wgs=3, tile=1),
                                  dict(persistent=1), None])
def test_schedule_with_empty_and_k0_layers(tune):
    """Layers without a product inside a grouped schedule: one with outputs
    but K = 0 (with a non-null weight pointer, as a C-ABI caller may pass
    one) writes its bias and zero accumulators, layers with M = 0 or N = 0
    write nothing, and the layers around them match the oracle, through the
    persistent launch, the one-workgroup-per-tile grouped launch and AUTO."""
    dummy = torch.zeros(4096, dtype=torch.int8, device=DEV)          # never read
    shapes = [(300, 200, 304), (40, 70, 0), (0, 64, 128), (33, 0, 32), (300, 70, 0),
              (520, 260, 1152)]
    host, layers, keep = [], [], []
    for i, (M, N, K) in enumerate(shapes):
        X, W, sw, bias = inputs.random_case(300 + i, M, N, K)
        Xd, Wd, swd, bd = X.to(DEV), W.to(DEV), sw.to(DEV), bias.to(DEV)
        acc = torch.full((M, N), 12345, dtype=torch.int32, device=DEV)
        y = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
        ly = T.make_layer(Xd, Wd, SX, swd, bd, acc, y)
        if K == 0:
            ly.W = dummy.data_ptr()
        layers.append(ly)
        keep.append((Xd, Wd, swd, bd))
        host.append((X, W, sw, bias, acc, y))
    table = torch.tensor([[3, 8], [5, 1], [8, 8], [2, 4], [6, 2], [7, 6]], dtype=torch.uint8)
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    T.run_schedule(layers, table, 2, 4, 0, 4, workspace=ws, tune=tune)
    torch.cuda.synchronize()
    stage = oracle.stage_of_step(3, 2, 4)
    for i, (X, W, sw, bias, acc, y) in enumerate(host):
        b = int(table[i, stage])
        ra, ry = oracle.masked_linear(X, W, SX, sw, b, bias)
        check_outputs(acc, y, ra, ry, SX, sw, bias, f"layer {i} {tuple(X.shape)}x{W.shape[0]} "
                                                     f"b={b} tune={tune}")


def test_persistent_matches_grouped():
    """The persistent step (forced on) and the non-persistent grouped launch
    (forced off) write identical outputs at the 256x256 tile."""
    M, N, K = 2048, 2304, 256
    layers, outs, keep = [], [], []
    for i in range(3):
        X, W, sw, bias = inputs.random_case(90 + i, M, N, K)
        Xd, Wd, swd = X.to(DEV), W.to(DEV), sw.to(DEV)
        bd = bias.to(DEV) if i == 0 else None
        acc = torch.empty((M, N), dtype=torch.int32, device=DEV)
        y = torch.empty((M, N), dtype=torch.float32, device=DEV)
        layers.append(T.make_layer(Xd, Wd, SX, swd, bd, acc, y))
        outs.append((acc, y))
        keep.append((Xd, Wd, swd, bd))
    table = torch.tensor([[8, 5, 3, 1], [7, 6, 2, 4], [1, 2, 8, 6]], dtype=torch.uint8)
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    results = {}
    for mode in ("1", "0"):
        tune = dict(persistent=2 if mode == "1" else 1)
        for (t0, t1) in [(0, 1), (19, 20)]:
            for acc, y in outs:
                acc.fill_(12345)
                y.fill_(-7.0)
            T.run_schedule(layers, table, 4, 20, t0, t1, workspace=ws, tune=tune)
            torch.cuda.synchronize()
            results[(mode, t0)] = [(a.cpu().clone(), v.cpu().clone()) for a, v in outs]
    for t0 in (0, 19):
        for (a1, y1), (a0, y0) in zip(results[("1", t0)], results[("0", t0)]):
            assert torch.equal(a1, a0)
            assert torch.equal(y1, y0)
    # one sampled block of rows against the oracle
    X, W, sw, bias = inputs.random_case(90, M, N, K)
    rows = slice(1000, 1100)
    ra, ry = oracle.masked_linear(X[rows], W, SX, sw, 8, bias)
    check_outputs(results[("1", 0)][0][0][rows], results[("1", 0)][0][1][rows], ra, ry, SX, sw,
                  bias, "persistent 2048x2304x256 rows 1000..1099 b=8")


@pytest.mark.parametrize("wgs,parties", [(1, 1), (3, 1), (32, 1), (6, 3), (32, 4)])
def test_persistent_packed_schedule(wgs, parties):
    """The persistent step on packed weights (the weights streamed from the
    packed layout into registers, the activation K tiles requested three
    ahead across tile boundaries), forced with few workgroups per XCD so that
    every workgroup's request positions cross many tiles and layers."""
    tune = dict(persistent=2, persistent_wgs=wgs, persistent_parties=parties, packed_tile=1)
    host, layers, keep = build(170 + wgs, asym_layers=(1, 3))
    packed = []
    for h, ly in zip(host, layers):
        P = T.pack_weights(h["W"].to(DEV))
        packed.append(P)
        ly.W = None
        ly.W_packed = P.data_ptr()
    S, Tn = 4, 20
    rng = np.random.default_rng(171 + wgs)
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S)), dtype=torch.uint8)
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for (t0, t1) in [(0, 20), (0, 1), (6, 7), (12, 16)]:
        for h in host:
            h["acc"].fill_(12345)
            h["y"].fill_(-7.0)
        T.run_schedule(layers, table, S, Tn, t0, t1, workspace=ws, tune=tune)
        torch.cuda.synchronize()
        stage = oracle.stage_of_step(t1 - 1, S, Tn)
        for i, h in enumerate(host):
            b = int(table[i, stage])
            check_layer(h, b, f"packed wgs {wgs} parties {parties} [{t0},{t1}) layer {i} b={b}")
