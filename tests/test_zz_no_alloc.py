"""The allocation-free schedule entry point (tasq_run_schedule_noalloc)
against the workspace one (tasq_run_schedule) through the C ABI: the same
layers, table and step range give the same bits, on two calls in a row, the
second with fewer and smaller layers (the per-GPU scratch array keeps the
first call's contents, which the second must not read); a schedule whose
long-K conv runs unsplit here (split-K with a workspace) matches too; more
layers than the array holds is an error that enqueues nothing."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import _lib, inputs
from test_gpu_parity import DEV, check_outputs, f32, small_schedule_layers

pytestmark = pytest.mark.gpu
SX = f32(0.02)


def build(shapes, seed, dev_lists):
    host, dev = [], []
    for i, (M, N, K) in enumerate(shapes):
        X, W, sw, bias = inputs.random_case(seed * 10 + i, M, N, K)
        host.append(dict(X=X, W=W, sw=sw, bias=bias if i % 2 else None))
        d = dict(X=X.to(DEV), W=W.to(DEV), sw=sw.to(DEV),
                 bias=None if i % 2 == 0 else bias.to(DEV))
        for k in dev_lists:
            d[k] = (torch.full((M, N), 12345, dtype=torch.int32, device=DEV),
                    torch.full((M, N), -7.0, dtype=torch.float32, device=DEV))
        dev.append(d)
    return host, dev


def layers_of(dev, key):
    return [T.make_layer(d["X"], d["W"], SX, d["sw"], d["bias"], d[key][0], d[key][1])
            for d in dev]


@pytest.mark.parametrize("first,second", [
    ([(2048, 2304, 512), (300, 200, 304), (520, 260, 1152), (1024, 1152, 1152)],
     [(130, 129, 640), (40, 70, 128)]),
    ([(300, 200, 304), (33, 65, 300), (130, 129, 640)], [(40, 70, 128)]),
])
def test_noalloc_matches_workspace_schedule_twice(first, second):
    S, Tn = 4, 20
    for call, (shapes, seed) in enumerate(((first, 40), (second, 41))):
        host, dev = build(shapes, seed, ("ws", "na"))
        rng = np.random.default_rng(seed)
        table = torch.as_tensor(rng.integers(1, 9, size=(len(shapes), S)), dtype=torch.uint8)
        lw, ln = layers_of(dev, "ws"), layers_of(dev, "na")
        ws = torch.empty(T.schedule_workspace_bytes(lw), dtype=torch.uint8, device=DEV)
        for (t0, t1) in [(0, 20), (6, 7)]:
            T.run_schedule(lw, table, S, Tn, t0, t1, workspace=ws)
            T.run_schedule_noalloc(ln, table, S, Tn, t0, t1)
            torch.cuda.synchronize()
            for i, d in enumerate(dev):
                where = f"call {call} [{t0},{t1}) layer {i}"
                assert torch.equal(d["ws"][0], d["na"][0]), where
                assert torch.equal(d["ws"][1].view(torch.int32), d["na"][1].view(torch.int32)), where
            ref = oracle.run_schedule(host, table.numpy(), S, Tn, t0, t1, SX)
            for h, d, (ra, ry, b) in zip(host, dev, ref):
                check_outputs(d["na"][0], d["na"][1], ra, ry, SX, h["sw"], h.get("bias"),
                              f"call {call} [{t0},{t1}) b={b}")


def test_noalloc_small_schedule_with_conv():
    """Linear layers and a 3x3 conv (the helper's small block), grouped."""
    host, dev, rng = small_schedule_layers(44)
    S, Tn = 4, 20
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S)), dtype=torch.uint8)
    layers = [T.make_layer(d["X"], d["W"], SX, d["sw"], d.get("bias"), d["acc"], d["y"])
              for d in dev]
    T.run_schedule_noalloc(layers, table, S, Tn, 3, 11)
    torch.cuda.synchronize()
    ref = oracle.run_schedule(host, table.numpy(), S, Tn, 3, 11, SX)
    for h, d, (ra, ry, b) in zip(host, dev, ref):
        check_outputs(d["acc"], d["y"], ra, ry, SX, h["sw"], h.get("bias"), f"b={b}")


def test_noalloc_long_k_conv_runs_unsplit():
    """The SDXL-Turbo 3x3 conv (K = 11520 on 20 tiles), which a workspace
    schedule launches on its own with split-K, runs unsplit here: the same
    bits as the workspace schedule."""
    wl = inputs.workload(3)
    cs, ls = wl.layers[8], wl.layers[4]
    Xc = inputs.x_full(wl, 8).to(DEV)
    Wc = inputs.w_full(wl, 8).reshape(cs.N, 3, 3, cs.C).to(DEV)
    swc = inputs.sw_full(wl, 8).to(DEV)
    Xl, Wl, swl = (inputs.x_full(wl, 4).to(DEV), inputs.w_full(wl, 4).to(DEV),
                   inputs.sw_full(wl, 4).to(DEV))
    outs = {k: [torch.full((cs.H, cs.Wd, cs.N), 1, dtype=torch.int32, device=DEV),
                torch.full((cs.H, cs.Wd, cs.N), 1.0, dtype=torch.float32, device=DEV),
                torch.full((ls.M, ls.N), 1, dtype=torch.int32, device=DEV),
                torch.full((ls.M, ls.N), 1.0, dtype=torch.float32, device=DEV)]
            for k in ("ws", "na")}
    mk = lambda o: [T.make_layer(Xc, Wc, SX, swc, None, o[0], o[1]),   # noqa: E731
                    T.make_layer(Xl, Wl, SX, swl, None, o[2], o[3])]
    table = torch.tensor([[6, 5, 7, 8], [4, 8, 6, 5]], dtype=torch.uint8)
    lw = mk(outs["ws"])
    ws = torch.empty(T.schedule_workspace_bytes(lw), dtype=torch.uint8, device=DEV)
    T.run_schedule(lw, table, 4, 4, 0, 2, workspace=ws)
    T.run_schedule_noalloc(mk(outs["na"]), table, 4, 4, 0, 2)
    torch.cuda.synchronize()
    for a, b in zip(outs["ws"], outs["na"]):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_noalloc_rejects_too_many_layers_and_enqueues_nothing():
    host, dev = build([(40, 70, 128)], 45, ("na",))
    layer = layers_of(dev, "na")[0]
    L = _lib.TASQ_STATIC_MAX_LAYERS + 1
    table = torch.full((L, 1), 8, dtype=torch.uint8)
    with pytest.raises(T.TasqError) as e:
        T.run_schedule_noalloc([layer] * L, table, 1, 1, 0, 1)
    assert e.value.status == _lib.TASQ_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((dev[0]["na"][0] == 12345).all()) and bool((dev[0]["na"][1] == -7.0).all())


@pytest.mark.parametrize("packed", [False, True])
def test_noalloc_persistent_step_matches(packed):
    """The persistent grouped step (forced on, 3 workgroups per XCD so that
    each walks many tiles) through both entry points, on row-major and on
    packed weights: the same bits."""
    shapes = [(520, 260, 1152), (300, 200, 304), (1024, 1152, 1152)]
    host, dev = build(shapes, 47 + packed, ("ws", "na"))
    keep = []
    lw, ln = layers_of(dev, "ws"), layers_of(dev, "na")
    if packed:
        for d, a, b in zip(dev, lw, ln):
            P = T.pack_weights(d["W"])
            keep.append(P)
            for ly in (a, b):
                ly.W = None
                ly.W_packed = P.data_ptr()
    S, Tn = 4, 20
    table = torch.as_tensor(np.random.default_rng(48).integers(1, 9, size=(len(shapes), S)),
                            dtype=torch.uint8)
    tune = dict(persistent=2, persistent_wgs=3)
    ws = torch.empty(T.schedule_workspace_bytes(lw), dtype=torch.uint8, device=DEV)
    T.run_schedule(lw, table, S, Tn, 0, Tn, workspace=ws, tune=tune)
    T.run_schedule_noalloc(ln, table, S, Tn, 0, Tn, tune=tune)
    torch.cuda.synchronize()
    for i, d in enumerate(dev):
        assert torch.equal(d["ws"][0], d["na"][0]), f"packed={packed} layer {i}"
        assert torch.equal(d["ws"][1].view(torch.int32), d["na"][1].view(torch.int32)), i
    ref = oracle.run_schedule(host, table.numpy(), S, Tn, 0, Tn, SX)
    for h, d, (ra, ry, b) in zip(host, dev, ref):
        check_outputs(d["na"][0], d["na"][1], ra, ry, SX, h["sw"], h.get("bias"),
                      f"packed={packed} b={b}")
