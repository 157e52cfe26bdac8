"""Every tile configuration, forced through the library's tuning overrides
(tasq_opts.tile for the staged kernels, packed_tile for the packed-weight ones),
against the oracle: a ragged linear layer with bias, the same layer with
every optional epilogue term at once (asymmetric codes, low-rank branch,
weight zero points: the LDS staging those terms use is sized per tile), a
3x3 conv, and a grouped schedule.  Bars as in the other GPU tests."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_parity import DEV, check_outputs, f32, small_schedule_layers
from test_gpu_lowrank import branch, dev_bf16, eps_lr, lr_magnitude

pytestmark = pytest.mark.gpu

STAGED, PACKED = 6, 7          # tile configurations of each kind
SX = f32(0.02)


def layer_case(seed, M=300, N=200, K=304):
    X, _, _, bias = inputs.random_case(seed, M, N, K)
    W = inputs.random_case(seed + 1, 1, N, K)[1]
    sw = inputs.uniform_f32(seed, 3, torch.arange(N), 1e-3, 1e-2)
    return X, W, sw, bias


def run_layer(X, W, sw, bias, b, packed, tune, **kw):
    Wd = W.to(DEV)
    wkw = dict(packed=T.pack_weights(Wd)) if packed else {}
    return T.masked_linear(X.to(DEV) if X.device.type == "cpu" else X, None if packed else Wd,
                           SX, sw.to(DEV), b, None if bias is None else bias.to(DEV), **wkw,
                           tune=tune, **kw)


@pytest.mark.parametrize("kind,tile", [("staged", t) for t in range(STAGED)] +
                         [("packed", t) for t in range(PACKED)])
def test_forced_tile(kind, tile):
    packed = kind == "packed"
    tune = {"packed_tile" if packed else "tile": tile + 1}
    where = f"{kind} tile {tile}"
    # plain layer, ragged in M, N and K
    X, W, sw, bias = layer_case(600 + tile)
    for b in (8, 5, 1):
        acc, y = run_layer(X, W, sw, bias, b, packed, tune)
        torch.cuda.synchronize()
        ra, ry = oracle.masked_linear(X, W, SX, sw, b, bias)
        check_outputs(acc, y, ra, ry, SX, sw, bias, f"{where} b={b}")

    # every optional epilogue term at once
    M, N, K = 300, 200, 304
    Wf = inputs.weights_f32(610 + tile, N, K)
    Qd, alpha, zwd, swd = T.quantize_weights(Wf.to(DEV))
    rQ, _, zw, rsw = oracle.weight_quant(Wf)
    Wc = (rQ.astype(np.int16) - 128).astype(np.int8)
    x, D, U = branch(620 + tile, M, K, 32, N)
    q, params, Tg = T.quantize_activations_lowrank(x.to(DEV), dev_bf16(D))
    ax, zx, Qx = oracle.act_quant(x)
    Xc = (Qx.astype(np.int16) - 128).astype(np.int8)
    rs = T.row_sums(q)
    cs = T.weight_colsums(Qd)
    wkw = dict(packed=T.pack_weights(Qd)) if packed else {}
    acc, y = T.masked_linear(q, None if packed else Qd, 0.0, swd, 6, act=params, colsums=cs,
                             lowrank=(Tg, dev_bf16(U)), wzero=(zwd, rs), tune=tune, **wkw)
    torch.cuda.synchronize()
    ra, ry = oracle.layer_dequant(Xc, Wc, rsw, 6, act=(ax, zx), zw=zw)
    _, lr64 = oracle.lowrank(x, D, U)
    _, S = lr_magnitude(x, D, U)
    assert np.array_equal(acc.cpu().numpy(), ra), where
    R = oracle.row_sums(Xc) + K * (128.0 - zx)
    corr = (128.0 - zx) * oracle.weight_colsums(Wc)[5].astype(np.float64)
    scale = ax * rsw.astype(np.float64)
    mag = np.abs(scale) * (np.abs(ra.astype(np.float64)) + np.abs(corr)
                           + np.abs((128.0 - zw.astype(np.float64)) * R[:, None]))
    err = np.abs(y.cpu().numpy().astype(np.float64) - (ry + lr64))
    worst = float(np.max(err - 1e-6 * mag - eps_lr(K) * S))
    assert worst <= 0.0, f"{where} extras: error above bound by {worst}"

    # 3x3 conv (NHWC), ragged channel counts
    H, Wd_, C, Nc = 9, 9, 48, 70
    Xi, _, swc, biasc = inputs.random_case(630 + tile, H * Wd_, Nc, C)
    Xi = Xi.reshape(H, Wd_, C)
    Wt = inputs.random_case(631 + tile, 1, Nc, 9 * C)[1].reshape(Nc, 3, 3, C)
    ckw = dict(packed=T.pack_weights(Wt.to(DEV))) if packed else {}
    acc, y = T.masked_conv3x3(Xi.to(DEV), None if packed else Wt.to(DEV), SX, swc.to(DEV), 4,
                              biasc.to(DEV), tune=tune, **ckw)
    torch.cuda.synchronize()
    ra, ry = oracle.conv3x3(Xi, Wt, SX, swc, 4, biasc)
    check_outputs(acc, y, ra, ry, SX, swc, biasc, f"{where} conv")

    # grouped schedule
    host, dev, rng = small_schedule_layers(11 + tile)
    S_, Tn = 4, 20
    table = torch.as_tensor(rng.integers(1, 9, size=(len(host), S_)), dtype=torch.uint8)
    packs = [T.pack_weights(h["W"].to(DEV)) if packed else None for h in host]
    layers = [T.make_layer(d["X"], None if packed else d["W"], SX, d["sw"], d.get("bias"),
                           d["acc"], d["y"], packed=p) for d, p in zip(dev, packs)]
    ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    T.run_schedule(layers, table, S_, Tn, 3, 11, workspace=ws, tune=tune)
    torch.cuda.synchronize()
    ref = oracle.run_schedule(host, table.numpy(), S_, Tn, 3, 11, SX)
    for h, d, (ra, ry, b) in zip(host, dev, ref):
        check_outputs(d["acc"], d["y"], ra, ry, SX, h["sw"], h.get("bias"),
                      f"{where} schedule b={b}")
