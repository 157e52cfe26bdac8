"""GPU parity of the 16-bit low-rank branch (SVDQuant-initialised layers,
Sec. 4.1 setup): the down projection T = bf16(x) D^T, alone and fused with
the activation quantizer, and the up projection T U^T added to y by every
kernel family, against the oracle's fp64 branch.

Bar.  Codes, alpha, z and int32 accumulators: bit-exact.  The branch is
compared against its fp64 value lr64 with the bound derived from the
kernels' arithmetic, relative to S[m,n] = sum_j |U[n,j]| A[m,j],
A[m,j] = sum_k |bf16(x[m,k]) D[j,k]|:
  * T: fp32 MFMA accumulation, at most ceil(K/16) MFMAs per wave of 16
    products each, then a fixed-order sum of 8 wave partials:
    (ceil(K/16) + 24) u A[m,j], u = 2^-24;
  * T as two bfloat16 parts (exact truncation, then the remainder rounded):
    2^-16 |T|;
  * T U^T: 2 ceil(r/16) bfloat16 MFMAs of 16 products (weight-streaming
    kernels: r sequential fp32 FMAs), at most 70 u of the sum of |terms|;
  * one rounding adding the branch to the dequantised value.
  eps(K) = 2^-16 + (ceil(K/16) + 96) u, and
  |y_gpu - (y64 + lr64)| <= 1e-6 * (dequant magnitude) + eps(K) * S[m,n].
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_parity import DEV, sample_rows

pytestmark = pytest.mark.gpu

RTOL = 1e-6
U32 = 2.0 ** -24
SX = float(np.float32(0.02))


def eps_lr(K):
    return 2.0 ** -16 + (math.ceil(K / 16) + 96) * U32


def branch(seed, M, K, r, N, shape="outlier"):
    x = inputs.activations_f32(seed, np.arange(M), K, shape)
    D = inputs.bf16_bits(seed, 11, (r, K))
    U = inputs.bf16_bits(seed, 12, (N, r))
    return x, D, U


def lr_magnitude(x, D, U):
    xt = np.abs(oracle.bf16_value(oracle.bf16_round(x)))
    A = xt @ np.abs(oracle.bf16_value(D)).T
    return A, A @ np.abs(oracle.bf16_value(U)).T


def dev_bf16(bits):
    return bits.to(DEV).view(torch.bfloat16)


def check_T(T_gpu, x, D, where):
    no_up = np.zeros((1, D.shape[0]), np.uint16)
    T64, _ = oracle.lowrank(x, D, no_up)
    A, _ = lr_magnitude(x, D, no_up)
    K = x.shape[1]
    err = np.abs(T_gpu.cpu().numpy().astype(np.float64) - T64)
    worst = float(np.max(err - (math.ceil(K / 16) + 24) * U32 * A)) if err.size else -1.0
    assert worst <= 0.0, f"{where}: T error above bound by {worst}"


@pytest.mark.parametrize("M,K,r", [(1, 1152, 16), (33, 300, 32), (64, 1152, 32), (300, 4608, 32),
                                   (513, 1160, 16), (32, 8, 32), (7, 1, 16)])
def test_lowrank_down(M, K, r):
    x, D, _ = branch((M * 5 + K) % 30011, M, K, r, 1)
    Tg = T.lowrank_down(x.to(DEV), dev_bf16(D))
    torch.cuda.synchronize()
    check_T(Tg, x, D, f"down {M}x{K} r={r}")


def test_lowrank_down_k_zero_writes_zeros():
    x = torch.empty((5, 0), dtype=torch.float32, device=DEV)
    D = torch.empty((16, 0), dtype=torch.bfloat16, device=DEV)
    out = torch.full((5, 16), 3.0, device=DEV)
    T.lowrank_down(x, D, out=out)
    torch.cuda.synchronize()
    assert not out.any()


@pytest.mark.parametrize("M,K,r", [(1, 1152, 32), (40, 300, 16), (4096, 1152, 32),
                                   (2, 4 * 1024 + 3, 32)])
def test_quantize_lowrank_fused(M, K, r):
    """One read of x gives codes, alpha and z bit-exact, and T within bound."""
    x, D, _ = branch((M * 3 + K) % 30011, M, K, r, 1, "skewed")
    q, params, Tg = T.quantize_activations_lowrank(x.to(DEV), dev_bf16(D))
    torch.cuda.synchronize()
    alpha, z, Q = oracle.act_quant(x)
    p = params.cpu().numpy()
    assert np.float32(p[0]).tobytes() == np.float32(alpha).tobytes()
    assert np.float32(p[1]).tobytes() == np.float32(z).tobytes()
    assert np.array_equal((q.cpu().numpy().astype(np.int16) + 128).astype(np.uint8), Q)
    check_T(Tg, x, D, f"fused {M}x{K}")


def check_y(y_gpu, y_main, mag_main, lr64, S, K, where):
    y = y_gpu.cpu().numpy().astype(np.float64)
    err = np.abs(y - (y_main + lr64))
    worst = float(np.max(err - RTOL * mag_main - eps_lr(K) * S)) if err.size else -1.0
    assert worst <= 0.0, f"{where}: error above bound by {worst}"


LINEAR = [(1, 37, 1152), (16, 1152, 144), (33, 257, 304), (64, 130, 528), (65, 70, 128),
          (300, 129, 640), (513, 1152, 1152), (256, 512, 4608)]


@pytest.mark.parametrize("case", range(len(LINEAR)))
@pytest.mark.parametrize("source", ["rows", "packed", "planes"])
@pytest.mark.parametrize("asym", [False, True])
def test_linear_with_lowrank(case, source, asym):
    M, N, K = LINEAR[case]
    r = 32 if case % 2 else 16
    X, W, sw, bias = inputs.random_case(400 + case, M, N, K)
    x, D, U = branch(410 + case, M, K, r, N)
    Wd, swd, bd = W.to(DEV), sw.to(DEV), bias.to(DEV)
    if asym:
        q, params, Tg = T.quantize_activations_lowrank(x.to(DEV), dev_bf16(D))
        alpha, z, Q = oracle.act_quant(x)
        cs = T.weight_colsums(Wd)
        Xd = q
    else:
        Tg = T.lowrank_down(x.to(DEV), dev_bf16(D))
        Xd = X.to(DEV)
    Ud = dev_bf16(U)
    _, lr64 = oracle.lowrank(x, D, U)
    _, S = lr_magnitude(x, D, U)
    if source == "planes":
        kw = dict(variant=T.VARIANT_BITPLANE, planes=T.pack_planes(Wd))
    elif source == "packed":
        kw = dict(packed=T.pack_weights(Wd))
    else:
        kw = {}
    Wuse = Wd if source == "rows" else None
    for b in ([8, 5, 2] if case % 2 else [7, 4, 1]):
        use_bias = bias if b % 2 else None
        if asym:
            acc, y = T.masked_linear(Xd, Wuse, 0.0, swd, b, bd if b % 2 else None, act=params,
                                     colsums=cs, lowrank=(Tg, Ud), **kw)
            ra, ry = oracle.masked_linear_asym(Q, W, alpha, z, sw, b, use_bias)
            cs_b = oracle.weight_colsums(W)[b - 1].astype(np.float64)
            mag = np.abs(alpha * sw.numpy().astype(np.float64)) * (
                np.abs(ra.astype(np.float64)) + np.abs((128.0 - z) * cs_b))
        else:
            acc, y = T.masked_linear(Xd, Wuse, SX, swd, b, bd if b % 2 else None,
                                     lowrank=(Tg, Ud), **kw)
            ra, ry = oracle.masked_linear(X, W, SX, sw, b, use_bias)
            mag = np.abs(ra.astype(np.float64) * SX * sw.numpy().astype(np.float64))
        if use_bias is not None:
            mag = mag + np.abs(use_bias.numpy().astype(np.float64))
        torch.cuda.synchronize()
        assert np.array_equal(acc.cpu().numpy(), ra), f"acc {M}x{N}x{K} {source} b={b}"
        check_y(y, ry, mag, lr64, S, K, f"lowrank {M}x{N}x{K} {source} asym={asym} b={b}")


@pytest.mark.parametrize("cfg,l", [(1, 0), (1, 3), (2, 2)])
def test_lowrank_full_size_sampled(cfg, l):
    """A full-size layer with a rank-32 branch: sampled rows x all columns."""
    wl = inputs.workload(cfg)
    spec = wl.layers[l]
    rng = np.random.default_rng(cfg * 17 + l)
    X, W, sw = inputs.x_full(wl, l), inputs.w_full(wl, l), inputs.sw_full(wl, l)
    x, D, U = branch(wl.seed * 100 + l, spec.M, spec.K, 32, spec.N)
    Tg = T.lowrank_down(x.to(DEV), dev_bf16(D))
    rows = sample_rows(spec.M, rng)
    idx = torch.as_tensor(rows)
    xr = x[idx]
    rr = np.repeat(np.arange(len(rows)), spec.N)
    cc = np.tile(np.arange(spec.N), len(rows))
    lr64 = oracle.lowrank_entries(xr, D, U, rr, cc).reshape(len(rows), spec.N)
    _, S = lr_magnitude(xr, D, U)
    Xd, Wd, swd, Ud = X.to(DEV), W.to(DEV), sw.to(DEV), dev_bf16(U)
    for b in sorted(set(int(v) for v in inputs.b_table(wl)[l].tolist()))[:2]:
        acc, y = T.masked_linear(Xd, Wd, SX, swd, b, lowrank=(Tg, Ud))
        torch.cuda.synchronize()
        ra, ry = oracle.masked_linear_entries(X[idx], W, SX, sw, b, rr, cc)
        ra = ra.reshape(len(rows), spec.N)
        assert np.array_equal(acc[idx].cpu().numpy(), ra)
        mag = np.abs(ra.astype(np.float64) * SX * sw.numpy().astype(np.float64))
        check_y(y[idx], ry.reshape(len(rows), spec.N), mag, lr64, S, spec.K,
                f"lowrank cfg{cfg} {spec.name} b={b}")
        del acc, y


@pytest.mark.parametrize("mode", ["per_layer", "grouped", "persistent", "skinny", "packed"])
def test_lowrank_schedule(mode):
    """Schedules mixing layers with and without a branch (and asymmetric
    codes): every step range leaves each layer at its last step's b."""
    if mode == "skinny":
        shapes = [(16, 1152, 1152), (64, 130, 528), (33, 257, 304)]
    else:
        shapes = [(40, 70, 128), (130, 129, 640), (300, 65, 304)]
    S_, Tn = 4, 20
    rng = np.random.default_rng(43)
    table = torch.as_tensor(rng.integers(1, 9, size=(len(shapes), S_)), dtype=torch.uint8)
    host, layers, keep = [], [], []
    for i, (M, N, K) in enumerate(shapes):
        X, W, sw, _ = inputs.random_case(970 + i, M, N, K)
        x, D, U = branch(980 + i, M, K, 32 if i != 2 else 16, N)
        Wd, swd = W.to(DEV), sw.to(DEV)
        acc = torch.full((M, N), 12345, dtype=torch.int32, device=DEV)
        y = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
        h = dict(X=X, W=W, sw=sw, x=x, D=D, U=U, acc=acc, y=y, asym=(i == 1), lr=(i != 0))
        act = cs = None
        if h["asym"]:
            q, act, Tg = T.quantize_activations_lowrank(x.to(DEV), dev_bf16(D))
            h["alpha"], h["z"], h["Q"] = oracle.act_quant(x)
            cs = T.weight_colsums(Wd)
            Xd = q
        else:
            Tg = T.lowrank_down(x.to(DEV), dev_bf16(D))
            Xd = X.to(DEV)
        Ud = dev_bf16(U)
        packed = T.pack_weights(Wd) if mode == "packed" else None
        L = T.make_layer(Xd, None if packed is not None else Wd, SX, swd, None, acc, y,
                         packed=packed, act=act, colsums=cs,
                         lowrank=(Tg, Ud) if h["lr"] else None)
        keep.append((Xd, Wd, swd, packed, act, cs, Tg, Ud, L))
        host.append(h)
        layers.append(L)
    ws = None
    if mode != "per_layer":
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for (t0, t1) in [(0, 20), (0, 1), (6, 7), (14, 20)]:
        # persistent: the one-workgroup-per-CU step with its epilogue operands
        # staged in the weight stages (forced on, 256x256 tiles)
        tune = dict(persistent=2, tile=1) if mode == "persistent" else None
        T.run_schedule(layers, table, S_, Tn, t0, t1, workspace=ws, tune=tune)
        torch.cuda.synchronize()
        stage = oracle.stage_of_step(t1 - 1, S_, Tn)
        for i, h in enumerate(host):
            b = int(table[i, stage])
            if h["asym"]:
                ra, ry = oracle.masked_linear_asym(h["Q"], h["W"], h["alpha"], h["z"], h["sw"], b)
                cs_b = oracle.weight_colsums(h["W"])[b - 1].astype(np.float64)
                mag = np.abs(h["alpha"] * h["sw"].numpy().astype(np.float64)) * (
                    np.abs(ra.astype(np.float64)) + np.abs((128.0 - h["z"]) * cs_b))
            else:
                ra, ry = oracle.masked_linear(h["X"], h["W"], SX, h["sw"], b)
                mag = np.abs(ra.astype(np.float64) * SX * h["sw"].numpy().astype(np.float64))
            assert np.array_equal(h["acc"].cpu().numpy(), ra), f"{mode} layer {i} b={b}"
            if h["lr"]:
                _, lr64 = oracle.lowrank(h["x"], h["D"], h["U"])
                _, S = lr_magnitude(h["x"], h["D"], h["U"])
            else:
                lr64, S = 0.0, 0.0
            check_y(h["y"], ry, mag, lr64, S, h["X"].shape[1],
                    f"{mode} [{t0},{t1}) layer {i} b={b}")
