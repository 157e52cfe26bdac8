"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bar (int32 accumulators): bit-exact.  Bar (fp32 dequantised output):
|y_gpu - y64| <= 1e-6 * (|acc * sx * sw[n]| + |bias[n]|), where y64 is the
oracle's fp64 value.  The kernel's fp32 result carries at most four roundings
(int32 -> fp32, sx*sw, the product, the bias add), about 2.4e-7 of that
magnitude, so 1e-6 is the stated maximum relative error with margin.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs

pytestmark = pytest.mark.gpu

DEV = "cuda"
RTOL = 1e-6


def f32(v):
    return float(np.float32(v))


def check_outputs(acc_gpu, y_gpu, acc_ref, y_ref, sx, sw, bias, where=""):
    acc_ref = np.asarray(acc_ref)
    if acc_gpu is not None:
        a = acc_gpu.cpu().numpy().reshape(acc_ref.shape)
        bad = np.argwhere(a != acc_ref)
        assert bad.size == 0, f"{where}: {len(bad)} int32 mismatches, first {bad[:3].tolist()}"
    if y_gpu is not None:
        y = y_gpu.cpu().numpy().astype(np.float64).reshape(acc_ref.shape)
        sw = np.asarray(sw, np.float64)
        bb = np.zeros_like(sw) if bias is None else np.asarray(bias, np.float64)
        mag = np.abs(acc_ref.astype(np.float64) * float(sx) * sw) + np.abs(bb)
        err = np.abs(y - np.asarray(y_ref))
        worst = float(np.max(err - RTOL * mag)) if err.size else -1.0
        assert worst <= 0.0, f"{where}: fp32 error above tolerance by {worst}"


def gpu_linear(X, W, sx, sw, b, bias=None, **kw):
    Xd = torch.as_tensor(X).to(DEV)
    Wd = None if W is None else torch.as_tensor(W).to(DEV)
    swd = torch.as_tensor(sw).to(DEV)
    bd = None if bias is None else torch.as_tensor(bias).to(DEV)
    acc, y = T.masked_linear(Xd, Wd, sx, swd, b, bd, **kw)
    torch.cuda.synchronize()
    return acc, y


# ------------------------------------------------------------------ config 0

@pytest.mark.parametrize("b", [8, 6, 4, 2])
def test_config0_single_layer(b):
    """1152 -> 1152 at 256 tokens, int32 and fp32 outputs, b in {8, 6, 4, 2}."""
    wl = inputs.workload(0)
    X, W, sw = inputs.x_full(wl, 0), inputs.w_full(wl, 0), inputs.sw_full(wl, 0)
    sx = f32(wl.sx)
    acc, y = gpu_linear(X, W, sx, sw, b)
    ra, ry = oracle.masked_linear(X, W, sx, sw, b)
    check_outputs(acc, y, ra, ry, sx, sw, None, f"cfg0 b={b}")


# ---------------------------------------------------------------- fuzz shapes

FUZZ = [(1, 1, 1), (3, 33, 31), (17, 1, 64), (255, 33, 5600 // 8), (1, 6720 // 10, 1153),
        (3, 17, 11520 // 16), (64, 64, 128), (65, 129, 257), (300, 520, 1040), (257, 129, 1000),
        (128, 256, 2240), (1, 300, 16)]


@pytest.mark.parametrize("case", range(len(FUZZ)))
def test_fuzz_shapes(case):
    M, N, K = FUZZ[case]
    X, W, sw, bias = inputs.random_case(100 + case, M, N, K)
    X[0, 0] = -128
    W[0, 0] = -128
    sx = f32(0.013)
    for b in ([8, 7, 5, 3, 1] if case % 2 else [6, 4, 2, 1, 8]):
        use_bias = bias if b % 2 else None
        acc, y = gpu_linear(X, W, sx, sw, b, use_bias)
        ra, ry = oracle.masked_linear(X, W, sx, sw, b, use_bias)
        check_outputs(acc, y, ra, ry, sx, sw, use_bias, f"fuzz {M}x{N}x{K} b={b}")


@pytest.mark.parametrize("M,N,K", [(3, 33, 131071), (3, 40, 131056), (70, 40, 131071),
                                   (70, 33, 131056)])
def test_max_k_extreme_values(M, N, K):
    """K at TASQ_MAX_K (and the largest multiple of 16 below it): rows of
    -128 against columns of -128 put acc at 128 * 128 * K, 16384 below
    2^31 at K = 131071, through the weight-streaming kernels (M = 3), the
    GEMM (M = 70), the packed buffer and the bit planes, at b = 8 and b = 1
    (where -128 is kept whole); other rows and columns are random."""
    X, W, sw, _ = inputs.random_case(1000 + M + N + K % 977, M, N, K)
    X[0, :] = -128
    W[0, :] = -128
    W[1, :] = 127
    sx = f32(1.0 / 65536)
    Wd = W.to(DEV)
    for b in (8, 1):
        ra, ry = oracle.masked_linear(X, W, sx, sw, b)
        assert ra[0, 0] == 128 * 128 * K
        acc, y = gpu_linear(X, W, sx, sw, b)
        check_outputs(acc, y, ra, ry, sx, sw, None, f"max K {M}x{N}x{K} b={b} rows")
        acc, y = gpu_linear(X, None, sx, sw, b, packed=T.pack_weights(Wd))
        check_outputs(acc, y, ra, ry, sx, sw, None, f"max K {M}x{N}x{K} b={b} packed")
        acc, y = gpu_linear(X, None, sx, sw, b, variant=T.VARIANT_BITPLANE,
                            planes=T.pack_planes(Wd))
        check_outputs(acc, y, ra, ry, sx, sw, None, f"max K {M}x{N}x{K} b={b} planes")


def test_output_modes():
    M, N, K = 70, 90, 300
    X, W, sw, bias = inputs.random_case(7, M, N, K)
    sx = f32(0.02)
    ra, ry = oracle.masked_linear(X, W, sx, sw, 5, bias)
    acc, y = gpu_linear(X, W, sx, sw, 5, bias, want_y=False)
    assert y is None
    check_outputs(acc, None, ra, ry, sx, sw, bias)
    acc, y = gpu_linear(X, W, sx, sw, 5, bias, want_acc=False)
    assert acc is None
    check_outputs(None, y, ra, ry, sx, sw, bias)


def test_k_zero_writes_bias():
    M, N = 5, 7
    X = torch.zeros((M, 0), dtype=torch.int8)
    W = torch.zeros((N, 0), dtype=torch.int8)
    sw = torch.full((N,), 0.5)
    bias = torch.arange(N, dtype=torch.float32)
    acc, y = gpu_linear(X, W, 1.0, sw, 3, bias)
    assert not acc.any()
    assert torch.equal(y.cpu(), bias.expand(M, N))


def test_inputs_untouched_and_deterministic():
    M, N, K = 513, 700, 1152
    X, W, sw, bias = inputs.random_case(9, M, N, K)
    Xd, Wd, swd = X.to(DEV), W.to(DEV), sw.to(DEV)
    x0, w0, s0 = Xd.clone(), Wd.clone(), swd.clone()
    first = None
    for _ in range(100):
        acc, y = T.masked_linear(Xd, Wd, 0.02, swd, 4)
        if first is None:
            first = (acc.clone(), y.clone())
        else:
            assert torch.equal(acc, first[0]) and torch.equal(y.view(torch.int32),
                                                              first[1].view(torch.int32))
    torch.cuda.synchronize()
    assert torch.equal(Xd, x0) and torch.equal(Wd, w0) and torch.equal(swd, s0)


def test_precision_switch_between_launches():
    """Alternating b on one stream changes nothing but b (no state carried)."""
    M, N, K = 200, 300, 640
    X, W, sw, _ = inputs.random_case(11, M, N, K)
    Xd, Wd, swd = X.to(DEV), W.to(DEV), sw.to(DEV)
    outs = {}
    for b in [8, 2, 7, 3, 6, 1, 5, 4, 8, 1]:
        acc, _ = T.masked_linear(Xd, Wd, 1.0, swd, b, want_y=False)
        outs.setdefault(b, []).append(acc)
    torch.cuda.synchronize()
    for b, lst in outs.items():
        ra, _ = oracle.masked_linear(X, W, 1.0, sw, b)
        for a in lst:
            assert np.array_equal(a.cpu().numpy(), ra)


# --------------------------------------------------- full-size, sampled rows

def sample_rows(M, rng, n=24):
    fixed = [0, 1, 31, 32, 63, 64, 127, 128, 255, 256, M - 1, M - 2]
    r = sorted(set([v for v in fixed if 0 <= v < M] + rng.integers(0, M, n).tolist()))
    return np.array(r, np.int64)


FULL = [(1, l) for l in range(4)] + [(2, l) for l in range(4)] + [(3, l) for l in range(8)]


@pytest.mark.parametrize("cfg,l", FULL)
def test_full_size_layers_sampled(cfg, l):
    """Every linear of configs 1-3 at full size, at each distinct b of its
    table row: sampled rows (all columns) and sampled columns (all rows)
    against the oracle, plus the linearity property over the whole output."""
    wl = inputs.workload(cfg)
    spec = wl.layers[l]
    rng = np.random.default_rng(cfg * 100 + l)
    X = inputs.x_full(wl, l)
    W = inputs.w_full(wl, l)
    sw = inputs.sw_full(wl, l)
    sx = f32(wl.sx)
    Xd, Wd, swd = X.to(DEV), W.to(DEV), sw.to(DEV)
    table = inputs.b_table(wl)
    bits = sorted(set(int(v) for v in table[l].tolist()))
    rows = sample_rows(spec.M, rng)
    cols = sample_rows(spec.N, rng, 8)
    Xr = X[torch.as_tensor(rows)]
    for b in bits:
        acc, y = T.masked_linear(Xd, Wd, sx, swd, b)
        torch.cuda.synchronize()
        # rows x all columns
        rr = np.repeat(np.arange(len(rows)), spec.N)
        cc = np.tile(np.arange(spec.N), len(rows))
        ra, ry = oracle.masked_linear_entries(Xr, W, sx, sw, b, rr, cc)
        check_outputs(acc[torch.as_tensor(rows)], y[torch.as_tensor(rows)],
                      ra.reshape(len(rows), spec.N), ry.reshape(len(rows), spec.N), sx, sw,
                      None, f"cfg{cfg} {spec.name} b={b} rows")
        # all rows x sampled columns
        Wc = W[torch.as_tensor(cols)]
        rr = np.repeat(np.arange(spec.M), len(cols))
        cc = np.tile(np.arange(len(cols)), spec.M)
        ra, ry = oracle.masked_linear_entries(X, Wc, sx, sw[torch.as_tensor(cols)], b, rr, cc)
        check_outputs(acc[:, torch.as_tensor(cols)], y[:, torch.as_tensor(cols)],
                      ra.reshape(spec.M, len(cols)), ry.reshape(spec.M, len(cols)), sx,
                      sw[torch.as_tensor(cols)], None, f"cfg{cfg} {spec.name} b={b} cols")
        # linearity over the whole output: acc(W_b) + acc(W - W_b) = acc(W)
        if b < 8:
            low = (Wd.to(torch.int32) & ((1 << (8 - b)) - 1)).to(torch.int8)
            a8, _ = T.masked_linear(Xd, Wd, sx, swd, 8, want_y=False)
            alow, _ = T.masked_linear(Xd, low, sx, swd, 8, want_y=False)
            torch.cuda.synchronize()
            assert torch.equal(acc + alow, a8), f"cfg{cfg} {spec.name} b={b} linearity"
        del acc, y


# ---------------------------------------------------------------- convolution

@pytest.mark.parametrize("H,Wd,C,N", [(5, 7, 32, 40), (4, 3, 3, 5), (1, 1, 16, 1), (9, 9, 48, 70)])
def test_conv_small(H, Wd, C, N):
    X, _, sw, bias = inputs.random_case(H * 1000 + C, H * Wd, N, C)
    X = X.reshape(H, Wd, C)
    Wt = inputs.random_case(N + 5, 1, N, 9 * C)[1].reshape(N, 3, 3, C)
    sx = f32(0.02)
    for b in (8, 5, 2):
        acc, y = T.masked_conv3x3(X.to(DEV), Wt.to(DEV), sx, sw.to(DEV), b, bias.to(DEV))
        torch.cuda.synchronize()
        ra, ry = oracle.conv3x3(X, Wt, sx, sw, b, bias)
        check_outputs(acc, y, ra, ry, sx, sw, bias, f"conv {H}x{Wd}x{C}->{N} b={b}")


def test_conv_full_size_sampled():
    """The 32x32x1280 -> 1280 3x3 conv of config 3 at every b of its table
    row, on sampled pixels (all borders, corners, interior) x all channels."""
    wl = inputs.workload(3)
    l = 8
    spec = wl.layers[l]
    X = inputs.x_full(wl, l)
    Wt = inputs.w_full(wl, l).reshape(spec.N, 3, 3, spec.C)
    sw = inputs.sw_full(wl, l)
    sx = f32(wl.sx)
    rng = np.random.default_rng(3)
    pix = sorted(set([0, 31, 32, 33, 63, 992, 1023, 31 * 32 + 5, 5 * 32]
                     + rng.integers(0, 1024, 10).tolist()))
    for b in sorted(set(int(v) for v in inputs.b_table(wl)[l].tolist())):
        acc, y = T.masked_conv3x3(X.to(DEV), Wt.to(DEV), sx, sw.to(DEV), b)
        torch.cuda.synchronize()
        pp = np.repeat(np.array(pix), spec.N)
        cc = np.tile(np.arange(spec.N), len(pix))
        ra, ry = oracle.conv3x3_entries(X, Wt, sx, sw, b, pp, cc)
        check_outputs(acc.reshape(-1, spec.N)[torch.as_tensor(pix)],
                      y.reshape(-1, spec.N)[torch.as_tensor(pix)],
                      ra.reshape(len(pix), spec.N), ry.reshape(len(pix), spec.N), sx, sw, None,
                      f"conv full b={b}")


# ----------------------------------------------------------------- bit planes

@pytest.mark.parametrize("N,K", [(1, 1), (5, 31), (7, 128), (33, 300), (1152, 1152)])
def test_pack_planes_bit_exact(N, K):
    W = inputs.random_case(N * 7 + K, 1, N, K)[1]
    W[0, 0] = -128
    planes = T.pack_planes(W.to(DEV))
    torch.cuda.synchronize()
    ref = oracle.pack_planes(W)
    assert np.array_equal(planes.cpu().numpy().view(np.uint32), ref)


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (16, 1152, 1152), (3, 70, 300), (64, 640, 2560),
                                   (130, 200, 640)])
def test_bitplane_variant(M, N, K):
    X, W, sw, bias = inputs.random_case(M + N + K, M, N, K)
    X[0, 0] = -128
    W[0, 0] = -128
    planes = T.pack_planes(W.to(DEV))
    sx = f32(0.02)
    for b in range(1, 9):
        acc, y = gpu_linear(X, None, sx, sw, b, bias if b % 2 else None,
                            variant=T.VARIANT_BITPLANE, planes=planes)
        ra, ry = oracle.masked_linear(X, W, sx, sw, b, bias if b % 2 else None)
        check_outputs(acc, y, ra, ry, sx, sw, bias if b % 2 else None,
                      f"bitplane {M}x{N}x{K} b={b}")


# ---------------------------------------------------- skinny (M <= 64) paths

SKINNY = [(1, 37, 1152), (5, 300, 1040), (16, 1152, 144), (32, 33, 16), (33, 257, 1152),
          (64, 130, 528), (16, 4608, 1152)]


@pytest.mark.parametrize("case", range(len(SKINNY)))
@pytest.mark.parametrize("source", ["rows", "packed", "planes"])
def test_skinny_weight_streaming(case, source):
    """M <= 64 runs the weight-streaming kernels (int8 rows, the packed
    buffer, or the top b bit planes), with and without an int32 output."""
    M, N, K = SKINNY[case]
    X, W, sw, bias = inputs.random_case(300 + case, M, N, K)
    X[0, 0] = -128
    W[0, 0] = -128
    Xd, Wd, swd, bd = X.to(DEV), W.to(DEV), sw.to(DEV), bias.to(DEV)
    if source == "planes":
        kw = dict(variant=T.VARIANT_BITPLANE, planes=T.pack_planes(Wd))
    elif source == "packed":
        kw = dict(packed=T.pack_weights(Wd))
    else:
        kw = {}
    Wuse = Wd if source == "rows" else None
    sx = f32(0.02)
    for b in range(1, 9):
        use_bias = bd if b % 3 == 0 else None
        ra, ry = oracle.masked_linear(X, W, sx, sw, b, bias if b % 3 == 0 else None)
        acc, y = T.masked_linear(Xd, Wuse, sx, swd, b, use_bias, **kw)
        torch.cuda.synchronize()
        check_outputs(acc, y, ra, ry, sx, sw, bias if b % 3 == 0 else None,
                      f"skinny {M}x{N}x{K} {source} b={b}")
        _, y2 = T.masked_linear(Xd, Wuse, sx, swd, b, use_bias, want_acc=False, **kw)
        torch.cuda.synchronize()
        check_outputs(None, y2, ra, ry, sx, sw, bias if b % 3 == 0 else None,
                      f"skinny y-only {M}x{N}x{K} {source} b={b}")


SKINNY_SCHEDULES = {
    # four 16-token tiles (largest M 64)
    "m64": [(16, 1152, 1152), (16, 3456, 1152), (64, 130, 528), (33, 257, 1152),
            (1, 37, 1152)],
    # one 16-token tile (largest M 16): ragged N, K = 1040 and 144 (a partial
    # last 128-wide block), a layer whose K blocks outnumber the waves
    "m16": [(16, 1152, 1152), (5, 300, 1040), (1, 37, 1152), (16, 1152, 4608),
            (9, 77, 144), (2, 3456, 1152)],
    # two tiles (largest M 32) and three (largest M 40)
    "m32": [(32, 300, 1040), (17, 1152, 1152), (1, 37, 144)],
    "m40": [(40, 130, 528), (16, 1152, 1152), (33, 77, 1040)],
}


@pytest.mark.parametrize("group", sorted(SKINNY_SCHEDULES))
@pytest.mark.parametrize("source", ["rows", "packed", "planes"])
def test_skinny_schedule_grouped(source, group):
    """A schedule of skinny layers (M <= 64) runs one weight-streaming launch
    per step; every step range matches the oracle's literal step loop."""
    shapes = SKINNY_SCHEDULES[group]
    host, dev = [], []
    for i, (M, N, K) in enumerate(shapes):
        X, W, sw, bias = inputs.random_case(700 + i, M, N, K)
        host.append(dict(X=X, W=W, sw=sw, bias=bias if i == 2 else None))
        d = dict(X=X.to(DEV), W=W.to(DEV), sw=sw.to(DEV),
                 bias=bias.to(DEV) if i == 2 else None)
        d["acc"] = torch.full((M, N), 12345, dtype=torch.int32, device=DEV)
        d["y"] = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
        dev.append(d)
    S, Tn = 4, 20
    rng = np.random.default_rng(17)
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S)), dtype=torch.uint8)
    sx = f32(0.02)
    variant = T.VARIANT_AUTO
    layers = []
    for d in dev:
        W = d["W"] if source == "rows" else None
        planes = T.pack_planes(d["W"]) if source == "planes" else None
        packed = T.pack_weights(d["W"]) if source == "packed" else None
        d["keep"] = (planes, packed)
        layers.append(T.make_layer(d["X"], W, sx, d["sw"], d["bias"], d["acc"], d["y"],
                                   planes=planes, packed=packed))
    if source == "planes":
        variant = T.VARIANT_BITPLANE
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for (t0, t1) in [(0, 20), (0, 1), (6, 7), (14, 20)]:
        T.run_schedule(layers, table, S, Tn, t0, t1, workspace=ws, variant=variant)
        torch.cuda.synchronize()
        ref = oracle.run_schedule(host, table.numpy(), S, Tn, t0, t1, sx)
        for h, d, (ra, ry, b) in zip(host, dev, ref):
            check_outputs(d["acc"], d["y"], ra, ry, sx, h["sw"], h.get("bias"),
                          f"skinny schedule {source} [{t0},{t1}) b={b}")


# ------------------------------------------------------------------- schedule

def small_schedule_layers(seed):
    rng = np.random.default_rng(seed)
    shapes = [(40, 70, 128), (33, 65, 300), (130, 129, 640)]
    host, dev = [], []
    for i, (M, N, K) in enumerate(shapes):
        X, W, sw, bias = inputs.random_case(seed * 10 + i, M, N, K)
        host.append(dict(X=X, W=W, sw=sw, bias=bias if i == 1 else None))
    Xc, _, swc, _ = inputs.random_case(seed * 10 + 9, 6 * 5, 24, 32)
    Wc = inputs.random_case(seed * 10 + 8, 1, 24, 9 * 32)[1].reshape(24, 3, 3, 32)
    host.append(dict(kind="conv3x3", X=Xc.reshape(6, 5, 32), W=Wc, sw=swc))
    for h in host:
        d = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in h.items()}
        if h.get("kind") == "conv3x3":
            shape = (6, 5, 24)
        else:
            shape = (h["X"].shape[0], h["W"].shape[0])
        d["acc"] = torch.full(shape, 12345, dtype=torch.int32, device=DEV)
        d["y"] = torch.full(shape, -7.0, dtype=torch.float32, device=DEV)
        dev.append(d)
    return host, dev, rng


@pytest.mark.parametrize("grouped", [False, True])
def test_schedule_matches_oracle(grouped):
    host, dev, rng = small_schedule_layers(3)
    S, Tn = 4, 20
    table = torch.as_tensor(rng.integers(2, 9, size=(len(host), S)), dtype=torch.uint8)
    sx = f32(0.02)
    layers = [T.make_layer(d["X"], d["W"], sx, d["sw"], d.get("bias"), d["acc"], d["y"])
              for d in dev]
    ws = None
    if grouped:
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for (t0, t1) in [(0, 20), (0, 1), (5, 6), (12, 13), (19, 20), (3, 11)]:
        T.run_schedule(layers, table, S, Tn, t0, t1, workspace=ws)
        torch.cuda.synchronize()
        ref = oracle.run_schedule(host, table.numpy(), S, Tn, t0, t1, sx)
        for h, d, (ra, ry, b) in zip(host, dev, ref):
            check_outputs(d["acc"], d["y"], ra, ry, sx, h["sw"], h.get("bias"),
                          f"schedule [{t0},{t1}) b={b} grouped={grouped}")


def test_schedule_error_enqueues_nothing():
    host, dev, rng = small_schedule_layers(4)
    S, Tn = 4, 20
    table = torch.full((len(host), S), 8, dtype=torch.uint8)
    table[len(host) - 1, 3] = 0
    layers = [T.make_layer(d["X"], d["W"], 0.02, d["sw"], None, d["acc"], d["y"]) for d in dev]
    with pytest.raises(T.TasqError):
        T.run_schedule(layers, table, S, Tn, 0, 1)
    torch.cuda.synchronize()
    for d in dev:
        assert bool((d["acc"] == 12345).all()) and bool((d["y"] == -7.0).all())


def test_schedule_constant8_equals_static():
    host, dev, rng = small_schedule_layers(5)
    S, Tn = 4, 20
    layers = [T.make_layer(d["X"], d["W"], 0.02, d["sw"], None, d["acc"], d["y"]) for d in dev]
    T.run_schedule(layers, torch.full((len(host), S), 8, dtype=torch.uint8), S, Tn, 0, Tn)
    torch.cuda.synchronize()
    for h, d in zip(host, dev):
        if h.get("kind") == "conv3x3":
            ra, _ = oracle.conv3x3(h["X"], h["W"], 0.02, h["sw"], 8)
        else:
            ra, _ = oracle.masked_linear(h["X"], h["W"], 0.02, h["sw"], 8)
        assert np.array_equal(d["acc"].cpu().numpy(), ra)
