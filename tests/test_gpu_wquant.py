"""GPU parity of the offline weight quantizer (App. A.1.1) and of the layer
on its zero-pointed codes: codes, alpha, z and sw bit-exact against the
oracle (both decide in IEEE single precision), activation row sums
bit-exact, and the layer y = sum_k x_hat sw (W_b + 128 - z_w) through every
kernel family and schedule mode against the oracle's fp64 definition.

Bar (fp32 output): |y_gpu - y64| <= 1e-6 * (|scale| (|acc| + |corr| +
|(128 - z_w) R[m]|) + |bias|) + 1e-12 sum_k |x_hat w_hat_b|, scale = sx sw
(or alpha_x sw), corr the activation zero-point term, R[m] the row's
activation sum; the last term covers the oracle's own fp64 summation (it
adds the K terms of the definition one by one, so a cancelling sum need
not come out exactly zero).  The kernel adds
fl(fl((128 - z_w) scale) R) to the dequantised value: a few roundings
relative to those terms, well inside 1e-6.  With a low-rank branch the
bound of test_gpu_lowrank is added.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_parity import DEV, sample_rows
from test_gpu_lowrank import branch, dev_bf16, eps_lr, lr_magnitude

pytestmark = pytest.mark.gpu

RTOL = 1e-6
SX = float(np.float32(0.02))


def quantize_w(Wf):
    Q, alpha, z, sw = T.quantize_weights(Wf.to(DEV))
    torch.cuda.synchronize()
    rQ, ra, rz, rsw = oracle.weight_quant(Wf)
    got = (Q.cpu().numpy().astype(np.int16) + 128).astype(np.uint8).reshape(rQ.shape)
    bad = np.argwhere(got != rQ)
    assert bad.size == 0, f"{len(bad)} code mismatches, first {bad[:3].tolist()}"
    for name, g, r in (("alpha", alpha, ra), ("z", z, rz), ("sw", sw, rsw)):
        assert np.array_equal(g.cpu().numpy().view(np.uint32), r.view(np.uint32)), name
    return Q, sw, z, (rQ.astype(np.int16) - 128).astype(np.int8), rsw, rz


@pytest.mark.parametrize("N,K", [(1, 1), (5, 31), (64, 128), (1152, 1152), (70, 9 * 48),
                                 (3, 70000), (4608, 1152)])
def test_weight_quantizer_bit_exact(N, K):
    quantize_w(inputs.weights_f32((N * 7 + K) % 30011, N, K))


def test_weight_quantizer_special_rows():
    rows = [np.full(9, 0.25), np.linspace(-1, 1, 9), np.array([0, 0, 0, 0, 0, 0, 0, 0, 1.0]),
            np.array([-3.0, 5.0, 1.0, 1.0, -3.0, 2.5, 0.125, 4.0, 4.99])]
    quantize_w(torch.as_tensor(np.stack(rows).astype(np.float32)))
    # a view that is not 16-byte aligned takes the element-wise path
    Wf = inputs.weights_f32(5, 6, 65)
    flat = Wf.reshape(-1).to(DEV)
    view = flat[1:1 + 6 * 64].reshape(6, 64)
    Q, alpha, z, sw = T.quantize_weights(view)
    torch.cuda.synchronize()
    rQ = oracle.weight_quant(view.cpu())[0]
    assert np.array_equal((Q.cpu().numpy().astype(np.int16) + 128).astype(np.uint8), rQ)


def test_weight_quantizer_batch_matches_single():
    """The batched quantizer over 35 weights (three launches of up to 16;
    ragged K, K not a multiple of 4, a 4-byte-aligned view, an empty weight)
    gives each weight's single-call codes, alpha, z and sw bit for bit, and
    the oracle's on a sample."""
    shapes = [(1, 1), (5, 31), (64, 128), (1152, 1152), (70, 9 * 48), (3, 7000), (0, 16),
              (4608, 1152), (33, 65), (257, 640)] * 3 + [(9, 10), (2, 2), (1152, 4608), (7, 3),
                                                          (16, 1)]
    Ws = [inputs.weights_f32((i * 131 + N * 7 + K) % 30011, N, K).to(DEV)
          for i, (N, K) in enumerate(shapes)]
    flat = inputs.weights_f32(5, 6, 65).reshape(-1).to(DEV)
    Ws[8] = flat[1:1 + 6 * 64].reshape(6, 64)          # not 16-byte aligned: element-wise path
    got = T.quantize_weights_batch(Ws)
    torch.cuda.synchronize()
    assert len(got) == len(Ws)
    for i, (W, g) in enumerate(zip(Ws, got)):
        ref = T.quantize_weights(W)
        torch.cuda.synchronize()
        assert torch.equal(g[0], ref[0]), f"codes of weight {i} {tuple(W.shape)}"
        for name, a, r in zip(("alpha", "z", "sw"), g[1:], ref[1:]):
            assert torch.equal(a.view(torch.int32), r.view(torch.int32)), f"{name} of weight {i}"
    for i in (1, 8, 9, 33):
        rQ, ra, rz, rsw = oracle.weight_quant(Ws[i].cpu())
        Q = (got[i][0].cpu().numpy().astype(np.int16) + 128).astype(np.uint8).reshape(rQ.shape)
        assert np.array_equal(Q, rQ), f"oracle codes of weight {i}"
        assert np.array_equal(got[i][1].cpu().numpy().view(np.uint32), ra.view(np.uint32))


@pytest.mark.parametrize("M,K", [(1, 1), (7, 13), (300, 1152), (5, 4099)])
def test_row_sums_bit_exact(M, K):
    X = inputs.random_case(M + K, M, 1, K)[0]
    got = T.row_sums(X.to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy(), oracle.row_sums(X))


def term_abs(Xc, Wc, sw, b, sx=0.0, act=None, zw=None):
    """sum_k |x_hat| |w_hat_b| per output: the oracle's own fp64 summation
    error is below 1e-12 of it (it sums those terms in fp64)."""
    Xc = np.asarray(Xc).astype(np.float64)
    xh = np.abs(sx * Xc) if act is None else np.abs(act[0] * (Xc + 128.0 - act[1]))
    Wb = oracle.mask(np.asarray(Wc), b).astype(np.float64)
    if zw is not None:
        Wb = Wb + 128.0 - np.asarray(zw, np.float64)[:, None]
    return (xh @ np.abs(Wb).T) * np.abs(np.asarray(sw, np.float64))


def check_y(y_gpu, ry, mag, where, extra=0.0):
    y = y_gpu.cpu().numpy().astype(np.float64)
    err = np.abs(y - ry)
    worst = float(np.max(err - RTOL * mag - extra)) if err.size else -1.0
    assert worst <= 0.0, f"{where}: error above bound by {worst}"


def magnitude(acc, scale, zw, R, corr=0.0, bias=None):
    m = np.abs(scale) * (np.abs(acc.astype(np.float64)) + np.abs(corr)
                         + np.abs((128.0 - zw.astype(np.float64)) * R[:, None]))
    return m if bias is None else m + np.abs(np.asarray(bias, np.float64))


LINEAR = [(1, 37, 1152), (16, 1152, 144), (33, 257, 304), (64, 130, 528), (65, 70, 128),
          (300, 129, 640), (513, 1152, 1152)]


@pytest.mark.parametrize("case", range(len(LINEAR)))
@pytest.mark.parametrize("source", ["rows", "packed", "planes"])
@pytest.mark.parametrize("act", ["sym", "asym", "asym_lowrank"])
def test_layer_on_quantized_weights(case, source, act):
    M, N, K = LINEAR[case]
    Wf = inputs.weights_f32(500 + case, N, K)
    Qd, swd, zwd, Wc, sw, zw = quantize_w(Wf)
    X, _, _, bias = inputs.random_case(510 + case, M, N, K)
    lr = None
    extra = 0.0
    if act == "sym":
        Xd = X.to(DEV)
        Xc = X.numpy()
        actp = None
    else:
        x = inputs.activations_f32(520 + case, np.arange(M), K, "skewed")
        if act == "asym_lowrank":
            _, D, U = branch(530 + case, M, K, 32, N)
            Xd, params, Tg = T.quantize_activations_lowrank(x.to(DEV), dev_bf16(D))
            lr = (Tg, dev_bf16(U))
            _, lr64 = oracle.lowrank(x, D, U)
            _, S = lr_magnitude(x, D, U)
            extra = eps_lr(K) * S
        else:
            Xd, params = T.quantize_activations(x.to(DEV))
        alpha, z, Qx = oracle.act_quant(x)
        Xc = (Qx.astype(np.int16) - 128).astype(np.int8)
        actp = (alpha, z)
    rs = T.row_sums(Xd)
    if source == "planes":
        kw = dict(variant=T.VARIANT_BITPLANE, planes=T.pack_planes(Qd))
    elif source == "packed":
        kw = dict(packed=T.pack_weights(Qd))
    else:
        kw = {}
    Wuse = Qd if source == "rows" else None
    R = oracle.row_sums(Xc).astype(np.float64)
    for b in ([8, 5, 2] if case % 2 else [7, 4, 1]):
        use_bias = bias if b % 3 == 1 else None
        bd = None if use_bias is None else use_bias.to(DEV)
        if actp is None:
            acc, y = T.masked_linear(Xd, Wuse, SX, swd, b, bd, wzero=(zwd, rs), **kw)
            scale = SX * sw.astype(np.float64)
            corr = 0.0
        else:
            acc, y = T.masked_linear(Xd, Wuse, 0.0, swd, b, bd, act=params,
                                     colsums=T.weight_colsums(Qd), wzero=(zwd, rs), lowrank=lr,
                                     **kw)
            scale = actp[0] * sw.astype(np.float64)
            corr = (128.0 - actp[1]) * oracle.weight_colsums(Wc)[b - 1].astype(np.float64)
            R = oracle.row_sums(Xc) + K * (128.0 - actp[1])
        torch.cuda.synchronize()
        ra, ry = oracle.layer_dequant(Xc, Wc, sw, b, sx=SX, act=actp, zw=zw, bias=use_bias)
        if lr is not None:
            ry = ry + lr64
        assert np.array_equal(acc.cpu().numpy(), ra), f"acc {M}x{N}x{K} {source} {act} b={b}"
        check_y(y, ry, magnitude(ra, scale, zw, R, corr, use_bias),
                f"wquant {M}x{N}x{K} {source} {act} b={b}",
                extra + 1e-12 * term_abs(Xc, Wc, sw, b, SX, actp, zw))


@pytest.mark.parametrize("cfg,l", [(1, 0), (1, 3), (2, 1)])
def test_quantized_weights_full_size_sampled(cfg, l):
    """A full-size layer quantized from real-valued weights; symmetric int8
    activations; sampled rows x all columns."""
    wl = inputs.workload(cfg)
    spec = wl.layers[l]
    rng = np.random.default_rng(cfg * 19 + l)
    Wf = inputs.weights_f32(wl.seed * 50 + l, spec.N, spec.K)
    Qd, swd, zwd, Wc, sw, zw = quantize_w(Wf)
    X = inputs.x_full(wl, l)
    Xd = X.to(DEV)
    rs = T.row_sums(Xd)
    rows = sample_rows(spec.M, rng)
    idx = torch.as_tensor(rows)
    rr = np.repeat(np.arange(len(rows)), spec.N)
    cc = np.tile(np.arange(spec.N), len(rows))
    R = oracle.row_sums(X[idx]).astype(np.float64)
    for b in sorted(set(int(v) for v in inputs.b_table(wl)[l].tolist()))[:2]:
        acc, y = T.masked_linear(Xd, Qd, SX, swd, b, wzero=(zwd, rs))
        torch.cuda.synchronize()
        ra, ry = oracle.layer_dequant_entries(X[idx], Wc, sw, b, rr, cc, sx=SX, zw=zw)
        ra = ra.reshape(len(rows), spec.N)
        assert np.array_equal(acc[idx].cpu().numpy(), ra)
        check_y(y[idx], ry.reshape(len(rows), spec.N),
                magnitude(ra, SX * sw.astype(np.float64), zw, R), f"cfg{cfg} {spec.name} b={b}",
                1e-12 * term_abs(X[idx].numpy(), Wc, sw, b, SX, None, zw))
        del acc, y


@pytest.mark.parametrize("mode", ["per_layer", "grouped", "persistent", "skinny", "packed"])
def test_quantized_weights_schedule(mode):
    if mode == "skinny":
        shapes = [(16, 1152, 1152), (64, 130, 528), (33, 257, 304)]
    else:
        shapes = [(40, 70, 128), (130, 129, 640), (300, 65, 304)]
    S_, Tn = 4, 20
    rng = np.random.default_rng(47)
    table = torch.as_tensor(rng.integers(1, 9, size=(len(shapes), S_)), dtype=torch.uint8)
    host, layers, keep = [], [], []
    for i, (M, N, K) in enumerate(shapes):
        X = inputs.random_case(990 + i, M, N, K)[0]
        Wq = i != 1                    # layer 1 keeps zero points 0
        if Wq:
            Qd, swd, zwd, Wc, sw, zw = quantize_w(inputs.weights_f32(995 + i, N, K))
        else:
            _, Wc, swt, _ = inputs.random_case(995 + i, M, N, K)
            Qd, swd, sw, zw, zwd = Wc.to(DEV), swt.to(DEV), swt.numpy(), None, None
            Wc = Wc.numpy()
        Xd = X.to(DEV)
        rs = T.row_sums(Xd)
        acc = torch.full((M, N), 12345, dtype=torch.int32, device=DEV)
        y = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
        packed = T.pack_weights(Qd) if mode == "packed" else None
        L = T.make_layer(Xd, None if packed is not None else Qd, SX, swd, None, acc, y,
                         packed=packed, wzero=(zwd, rs) if Wq else None)
        keep.append((Xd, Qd, swd, zwd, rs, packed, L))
        host.append(dict(X=X.numpy(), W=Wc, sw=sw, zw=zw, acc=acc, y=y))
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
            ra, ry = oracle.layer_dequant(h["X"], h["W"], h["sw"], b, sx=SX, zw=h["zw"])
            assert np.array_equal(h["acc"].cpu().numpy(), ra), f"{mode} layer {i} b={b}"
            zw = h["zw"] if h["zw"] is not None else np.full(h["W"].shape[0], 128.0, np.float32)
            check_y(h["y"], ry, magnitude(ra, SX * np.asarray(h["sw"], np.float64), zw,
                                          oracle.row_sums(h["X"]).astype(np.float64)),
                    f"{mode} [{t0},{t1}) layer {i} b={b}",
                    1e-12 * term_abs(h["X"], h["W"], h["sw"], b, SX, None, h["zw"]))
