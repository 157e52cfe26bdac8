"""GPU parity of the asymmetric activation path (App. A.1.2): the quantizer
(codes, alpha and z bit-exact against the oracle, both deciding in IEEE
single precision), the masked-weight channel sums (bit-exact), and the masked
layer on asymmetric codes through every kernel family, against the oracle's
fp64 sum of alpha (Q - z) sw W_b.

Bar (fp32 output): |y_gpu - y64| <= 1e-6 * (|alpha sw[n]| (|acc| +
|(128 - z) colsum_b[n]|) + |bias[n]|).  The kernel forms
((float)acc + (128 - z) * colsum) * (alpha * sw) + bias: six roundings of at
most 2^-24 each, relative to those terms, about 3.6e-7 of the bound's
magnitude, so 1e-6 holds with margin whatever the cancellation between the
accumulator and the zero-point term."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import inputs
from test_gpu_parity import DEV, sample_rows

pytestmark = pytest.mark.gpu

RTOL = 1e-6
SX = float(np.float32(0.02))


def quantize(x):
    """GPU codes and params of fp32 x, checked bit-exact against the oracle."""
    q, params = T.quantize_activations(x.to(DEV))
    torch.cuda.synchronize()
    alpha, z, Q = oracle.act_quant(x)
    p = params.cpu().numpy()
    assert np.float32(p[0]).tobytes() == np.float32(alpha).tobytes(), (p[0], alpha)
    assert np.float32(p[1]).tobytes() == np.float32(z).tobytes(), (p[1], z)
    got = (q.cpu().numpy().astype(np.int16) + 128).astype(np.uint8)
    bad = np.argwhere(got != Q.reshape(got.shape))
    assert bad.size == 0, f"{len(bad)} code mismatches, first {bad[:3].tolist()}"
    return q, params, alpha, z, Q


def check_asym(acc_gpu, y_gpu, acc_ref, y_ref, alpha, z, sw, colsum, bias, where=""):
    acc_ref = np.asarray(acc_ref)
    if acc_gpu is not None:
        a = acc_gpu.cpu().numpy().reshape(acc_ref.shape)
        bad = np.argwhere(a != acc_ref)
        assert bad.size == 0, f"{where}: {len(bad)} int32 mismatches, first {bad[:3].tolist()}"
    if y_gpu is not None:
        y = y_gpu.cpu().numpy().astype(np.float64).reshape(acc_ref.shape)
        sc = np.abs(float(alpha) * np.asarray(sw, np.float64))
        zc = np.abs((128.0 - float(z)) * np.asarray(colsum, np.float64))
        bb = 0.0 if bias is None else np.abs(np.asarray(bias, np.float64))
        mag = sc * (np.abs(acc_ref.astype(np.float64)) + zc) + bb
        err = np.abs(y - np.asarray(y_ref))
        worst = float(np.max(err - RTOL * mag)) if err.size else -1.0
        assert worst <= 0.0, f"{where}: fp32 error above tolerance by {worst}"


# ----------------------------------------------------------------- quantizer

@pytest.mark.parametrize("M,K", [(1, 1), (1, 3), (7, 13), (5, 1001), (256, 1152),
                                 (4096, 1152), (1, 4 * 1024 * 1024 + 3)])
@pytest.mark.parametrize("shape", ["outlier", "skewed"])
def test_quantizer_bit_exact(M, K, shape):
    x = inputs.activations_f32((M * 7 + K) % 30011, torch.arange(M), K, shape)
    quantize(x)


def test_quantizer_special_inputs():
    # constant tensors, one-sided ranges, exact grid points and their midpoints
    cases = [torch.full((3, 5), 2.5), torch.full((1, 8), -0.75), torch.zeros(2, 9),
             torch.linspace(0.0, 255.0, 256).reshape(16, 16),
             torch.linspace(-1.0, 3.0, 1021).reshape(1, 1021),
             torch.tensor([[1.0, 2.0, 3.0], [4.0, 5.0, 1e-30]]),
             torch.tensor([[100.0, 100.5, 101.0]]),
             -torch.arange(1, 300, dtype=torch.float32).reshape(1, 299)]
    for x in cases:
        quantize(x.to(torch.float32).contiguous())


def test_quantizer_unaligned_and_repeated():
    """A view starting 4 bytes into its storage takes the element-wise path;
    a second call with a smaller tensor reuses the params buffer."""
    x = inputs.activations_f32(9, torch.arange(33), 257, "skewed")
    flat = x.reshape(-1).to(DEV)
    params = torch.empty(T.TASQ_ACT_PARAMS_FLOATS, dtype=torch.float32, device=DEV)
    for off, n in [(1, flat.numel() - 1), (3, 1000), (0, 17)]:
        view = flat[off:off + n]
        q = torch.empty(n + 1, dtype=torch.int8, device=DEV)[1:]
        T.quantize_activations(view, out=q, params=params)
        torch.cuda.synchronize()
        alpha, z, Q = oracle.act_quant(view.cpu())
        assert params[0].item() == alpha and params[1].item() == z
        assert np.array_equal((q.cpu().numpy().astype(np.int16) + 128).astype(np.uint8), Q)


def check_codes_vs_oracle(x_cpu, q, params, where):
    alpha, z, Q = oracle.act_quant(x_cpu)
    p = params.cpu().numpy()
    assert np.float32(p[0]).tobytes() == np.float32(alpha).tobytes(), (where, p[0], alpha)
    assert np.float32(p[1]).tobytes() == np.float32(z).tobytes(), (where, p[1], z)
    got = (q.cpu().numpy().astype(np.int16) + 128).astype(np.uint8).reshape(-1)
    bad = np.argwhere(got != Q.reshape(-1))
    assert bad.size == 0, f"{where}: {len(bad)} code mismatches, first {bad[:3].tolist()}"


def test_quantizer_batch_matches_single_and_oracle():
    """The batched quantizer over 22 tensors (three groups of launches):
    ragged shapes, an unaligned view (element-wise path), empty tensors in
    the list and one tensor of more than a million elements; every tensor's
    codes, alpha and z against the oracle and bit-identical to the
    single-tensor call."""
    shapes = [(1, 1), (7, 13), (33, 257), (5, 1001), (256, 1152), (1, 3), (64, 64), (0, 5),
              (3, 0), (129, 577), (2, 2), (300, 70), (1, 4099), (17, 17), (900, 1152), (8, 8),
              (1000, 1030), (4, 4), (11, 1), (1, 11), (45, 45)]
    xs_cpu, xs = [], []
    for i, (M, K) in enumerate(shapes):
        x = inputs.activations_f32(500 + i, torch.arange(M), K, "skewed" if i % 2 else "outlier")
        xs_cpu.append(x)
        xs.append(x.to(DEV))
    flat = inputs.activations_f32(77, torch.arange(9), 333, "skewed").reshape(-1).to(DEV)
    xs_cpu.append(flat[1:].cpu())
    xs.append(flat[1:])                  # 4 bytes into its storage: element-wise path
    outs, params = T.quantize_activations_batch(xs)
    torch.cuda.synchronize()
    for i, (x, q, p) in enumerate(zip(xs, outs, params)):
        if x.numel() == 0:
            continue
        q1, p1 = T.quantize_activations(x)
        torch.cuda.synchronize()
        assert torch.equal(q, q1), f"tensor {i}: codes differ from the single call"
        assert torch.equal(p[:2], p1[:2]), f"tensor {i}: params differ from the single call"
        check_codes_vs_oracle(xs_cpu[i], q, p, f"tensor {i} {tuple(x.shape)}")


def test_quantizer_batch_full_size_step():
    """The inputs of one block of the 28-block schedule (M = 8192; K = 1152,
    1152, 1152, 4608) in one batched call, twice in a row into the same
    buffers: every tensor against the oracle and bit-identical to the single
    call."""
    Ks = [1152, 1152, 1152, 4608]
    xs = [inputs.activations_f32(900 + i, torch.arange(8192), K, "skewed") for i, K in enumerate(Ks)]
    xd = [x.to(DEV) for x in xs]
    outs = [torch.empty(x.shape, dtype=torch.int8, device=DEV) for x in xs]
    params = [torch.empty(T.TASQ_ACT_PARAMS_FLOATS, dtype=torch.float32, device=DEV)
              for _ in xs]
    for rep in range(2):
        T.quantize_activations_batch(xd, outs, params)
        torch.cuda.synchronize()
        for i, x in enumerate(xd):
            q1, p1 = T.quantize_activations(x)
            torch.cuda.synchronize()
            assert torch.equal(outs[i], q1), f"rep {rep} tensor {i}"
            assert torch.equal(params[i][:2], p1[:2]), f"rep {rep} tensor {i}"
            if rep == 0:
                check_codes_vs_oracle(xs[i], outs[i], params[i], f"tensor {i} K={Ks[i]}")


# -------------------------------------------------------------- channel sums

@pytest.mark.parametrize("N,K", [(1, 1), (5, 31), (64, 128), (1152, 1152), (70, 9 * 48),
                                 (3, 70000)])
def test_weight_colsums_bit_exact(N, K):
    W = inputs.random_case((N * 3 + K) % 30011, 1, N, K)[1]
    W[0, 0] = -128
    W[-1, -1] = 127
    c = T.weight_colsums(W.to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(c.cpu().numpy(), oracle.weight_colsums(W))


# ------------------------------------------------------- layer on the codes

def weight_source(Wd, source):
    if source == "planes":
        return None, dict(variant=T.VARIANT_BITPLANE, planes=T.pack_planes(Wd))
    if source == "packed":
        return None, dict(packed=T.pack_weights(Wd))
    return Wd, {}


ASYM = [(1, 37, 1152), (16, 1152, 144), (33, 257, 300), (64, 130, 528), (65, 70, 128),
        (300, 129, 640), (513, 1152, 1152)]


@pytest.mark.parametrize("case", range(len(ASYM)))
@pytest.mark.parametrize("source", ["rows", "packed", "planes"])
def test_asym_linear_matches_oracle(case, source):
    M, N, K = ASYM[case]
    _, W, sw, bias = inputs.random_case(900 + case, M, N, K)
    W[0, 0] = -128
    x = inputs.activations_f32(910 + case, torch.arange(M), K,
                               "skewed" if case % 2 else "outlier")
    q, params, alpha, z, Q = quantize(x)
    Wd, swd, bd = W.to(DEV), sw.to(DEV), bias.to(DEV)
    cs = T.weight_colsums(Wd)
    Wuse, kw = weight_source(Wd, source)
    for b in range(1, 9):
        use_bias = bias if b % 2 else None
        acc, y = T.masked_linear(q, Wuse, 0.0, swd, b, bd if b % 2 else None, act=params,
                                 colsums=cs, **kw)
        torch.cuda.synchronize()
        ra, ry = oracle.masked_linear_asym(Q, W, alpha, z, sw, b, use_bias)
        check_asym(acc, y, ra, ry, alpha, z, sw, oracle.weight_colsums(W)[b - 1], use_bias,
                   f"asym {M}x{N}x{K} {source} b={b}")


@pytest.mark.parametrize("cfg,l", [(1, 0), (1, 3), (2, 3), (3, 7)])
def test_asym_full_size_sampled(cfg, l):
    """Full-size layers on real-valued activations: the quantizer over the
    whole tensor bit-exact, then sampled rows x all columns of the layer."""
    wl = inputs.workload(cfg)
    spec = wl.layers[l]
    rng = np.random.default_rng(cfg * 13 + l)
    x = inputs.activations_f32(wl.seed + l, torch.arange(spec.M), spec.K, "outlier")
    q, params, alpha, z, Q = quantize(x)
    W, sw = inputs.w_full(wl, l), inputs.sw_full(wl, l)
    Wd, swd = W.to(DEV), sw.to(DEV)
    cs = T.weight_colsums(Wd)
    rows = sample_rows(spec.M, rng)
    rr = np.repeat(np.arange(len(rows)), spec.N)
    cc = np.tile(np.arange(spec.N), len(rows))
    csh = oracle.weight_colsums(W)
    for b in sorted(set(int(v) for v in inputs.b_table(wl)[l].tolist())):
        acc, y = T.masked_linear(q, Wd, 0.0, swd, b, act=params, colsums=cs)
        torch.cuda.synchronize()
        ra, ry = oracle.masked_linear_asym_entries(Q[rows], W, alpha, z, sw, b, rr, cc)
        idx = torch.as_tensor(rows)
        check_asym(acc[idx], y[idx], ra.reshape(len(rows), spec.N),
                   ry.reshape(len(rows), spec.N), alpha, z, sw, csh[b - 1], None,
                   f"asym cfg{cfg} {spec.name} b={b}")
        del acc, y


@pytest.mark.parametrize("mode", ["per_layer", "grouped", "skinny", "packed"])
def test_asym_schedule(mode):
    """A schedule mixing asymmetric and symmetric layers: every step range
    leaves each layer's output at the b of its last step's stage."""
    if mode == "skinny":
        shapes = [(16, 1152, 1152), (64, 130, 528), (33, 257, 304)]
    else:
        shapes = [(40, 70, 128), (130, 129, 640), (300, 65, 300)]
    S, Tn = 4, 20
    rng = np.random.default_rng(41)
    table = torch.as_tensor(rng.integers(1, 9, size=(len(shapes), S)), dtype=torch.uint8)
    host, layers, keep = [], [], []
    for i, (M, N, K) in enumerate(shapes):
        X, W, sw, bias = inputs.random_case(950 + i, M, N, K)
        asym = i != 1
        h = dict(X=X, W=W, sw=sw, bias=bias if i == 2 else None, asym=asym)
        Wd = W.to(DEV)
        acc = torch.full((M, N), 12345, dtype=torch.int32, device=DEV)
        y = torch.full((M, N), -7.0, dtype=torch.float32, device=DEV)
        act = cs = None
        if asym:
            x = inputs.activations_f32(960 + i, torch.arange(M), K, "skewed")
            q, act, h["alpha"], h["z"], h["Q"] = quantize(x)
            cs = T.weight_colsums(Wd)
            Xd = q
        else:
            Xd = X.to(DEV)
        packed = T.pack_weights(Wd) if mode == "packed" else None
        # the layer struct holds raw pointers: keep every device tensor alive
        swd = sw.to(DEV)
        bd = None if h["bias"] is None else h["bias"].to(DEV)
        L = T.make_layer(Xd, None if packed is not None else Wd, SX, swd, bd, acc, y,
                         packed=packed, act=act, colsums=cs)
        keep.append((Xd, Wd, swd, bd, packed, act, cs, L))
        h["acc"], h["y"] = acc, y
        host.append(h)
        layers.append(L)
    ws = None
    if mode != "per_layer":
        ws = torch.empty(T.schedule_workspace_bytes(layers), dtype=torch.uint8, device=DEV)
    for (t0, t1) in [(0, 20), (0, 1), (6, 7), (14, 20)]:
        T.run_schedule(layers, table, S, Tn, t0, t1, workspace=ws)
        torch.cuda.synchronize()
        stage = oracle.stage_of_step(t1 - 1, S, Tn)
        for i, h in enumerate(host):
            b = int(table[i, stage])
            if h["asym"]:
                ra, ry = oracle.masked_linear_asym(h["Q"], h["W"], h["alpha"], h["z"], h["sw"],
                                                   b, h["bias"])
                check_asym(h["acc"], h["y"], ra, ry, h["alpha"], h["z"], h["sw"],
                           oracle.weight_colsums(h["W"])[b - 1], h["bias"],
                           f"{mode} [{t0},{t1}) layer {i} b={b}")
            else:
                ra, ry = oracle.masked_linear(h["X"], h["W"], SX, h["sw"], b, h["bias"])
                assert np.array_equal(h["acc"].cpu().numpy(), ra)
                y = h["y"].cpu().numpy().astype(np.float64)
                mag = np.abs(ra * SX * h["sw"].numpy().astype(np.float64))
                assert np.all(np.abs(y - ry) <= RTOL * mag + 1e-30)
