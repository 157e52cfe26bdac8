"""Seeded synthetic inputs for the masked-linear workloads.

This module only draws numbers and fixes shapes; it holds none of the
method's arithmetic (no masking, no products, no dequantisation), so that
both the HIP path and the CPU oracle can consume the same arrays without
sharing any computation.

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), used counter-style: element ``i`` of
tensor ``tid`` under seed ``seed`` is ``splitmix64(seed*2^48 + tid*2^32 + i)``.
Counter-based draws let any single row be regenerated without the rest of the
tensor, which the full-size sampled parity checks rely on.  The same integer
recipe runs on CPU or GPU tensors and gives identical integers on both
(int64 arithmetic wraps modulo 2^64 on both).

Workload shapes stand in for the paper's three backbones (Sec. 4.1: PixArt-
Sigma and SANA at 20 steps in four stages, SDXL-Turbo at four steps with one
stage per step); the models, weights and prompt sets are not used.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import torch

_GOLDEN = -7046029254386353131      # 0x9E3779B97F4A7C15 as int64
_MIX1 = -4658895280553007687        # 0xBF58476D1CE4E5B9
_MIX2 = -7723592293110705685        # 0x94D049BB133111EB


def _lsr(x: torch.Tensor, s: int) -> torch.Tensor:
    """Logical right shift of int64 bit patterns."""
    return (x >> s) & ((1 << (64 - s)) - 1)


def splitmix64(counter: torch.Tensor) -> torch.Tensor:
    """SplitMix64 output for each int64 counter (bit pattern of a uint64)."""
    z = counter + _GOLDEN
    z = (z ^ _lsr(z, 30)) * _MIX1
    z = (z ^ _lsr(z, 27)) * _MIX2
    return z ^ _lsr(z, 31)


def _counters(seed: int, tid: int, idx: torch.Tensor) -> torch.Tensor:
    if not (0 <= seed < 2 ** 15 and 0 <= tid < 2 ** 16):
        raise ValueError("seed must be < 2^15 and tensor id < 2^16")
    return idx + ((seed << 48) | (tid << 32))


def raw(seed: int, tid: int, idx: torch.Tensor) -> torch.Tensor:
    """Raw 64-bit draws (as int64) for the element indices ``idx``."""
    return splitmix64(_counters(seed, tid, idx.to(torch.int64)))


def uniform_int(seed, tid, idx, lo, hi, dtype=torch.int8):
    """Integers uniform on [lo, hi] from the top 53 bits of each draw."""
    u = _lsr(raw(seed, tid, idx), 11)                      # 53-bit value
    span = hi - lo + 1
    if span >= 1 << 10:
        raise ValueError("span too wide for the exact 53x10-bit product")
    return (lo + _lsr(u * span, 53)).to(dtype)


def uniform_f32(seed, tid, idx, lo, hi):
    """fp32 uniform on [lo, hi) from the top 24 bits of each draw."""
    u = _lsr(raw(seed, tid, idx), 40).to(torch.float64) * (2.0 ** -24)
    return (lo + (hi - lo) * u).to(torch.float32)


def normal_int8(seed, tid, idx, sigma=32.0):
    """clip(rint(sigma * z), -127, 127) with z ~ N(0,1) by Box-Muller in fp64.

    Always evaluated on the CPU so that log/cos rounding cannot differ
    between devices; callers move the result where they need it.
    """
    idx = idx.to(torch.int64).cpu()
    u1 = _lsr(raw(seed, tid, 2 * idx), 11).to(torch.float64) * (2.0 ** -53)
    u2 = _lsr(raw(seed, tid, 2 * idx + 1), 11).to(torch.float64) * (2.0 ** -53)
    z = torch.sqrt(-2.0 * torch.log1p(-u1)) * torch.cos(2.0 * math.pi * u2)
    return torch.clamp(torch.round(sigma * z), -127, 127).to(torch.int8)


def normal_f32(seed, tid, idx):
    """fp32 N(0, 1) draws by Box-Muller in fp64 on the CPU (as normal_int8)."""
    idx = idx.to(torch.int64).cpu()
    u1 = _lsr(raw(seed, tid, 2 * idx), 11).to(torch.float64) * (2.0 ** -53)
    u2 = _lsr(raw(seed, tid, 2 * idx + 1), 11).to(torch.float64) * (2.0 ** -53)
    z = torch.sqrt(-2.0 * torch.log1p(-u1)) * torch.cos(2.0 * math.pi * u2)
    return z.to(torch.float32)


def _grid(rows: Sequence[int] | torch.Tensor, ncols: int, device) -> torch.Tensor:
    r = torch.as_tensor(rows, dtype=torch.int64, device=device).reshape(-1, 1)
    c = torch.arange(ncols, dtype=torch.int64, device=device).reshape(1, -1)
    return r * ncols + c


def _draw_rows(rows, ncols: int, device, dtype, fn) -> torch.Tensor:
    """[len(rows) x ncols] array whose element (i, j) is fn(rows[i]*ncols + j),
    evaluated a few thousand rows at a time so temporaries stay small."""
    rows = torch.as_tensor(rows, dtype=torch.int64).reshape(-1)
    out = torch.empty((rows.numel(), ncols), dtype=dtype, device=device)
    if rows.numel() == 0 or ncols == 0:
        return out
    budget = (1 << 16) if torch.device(device).type == "cpu" else (1 << 24)
    step = max(1, budget // ncols)
    for i in range(0, rows.numel(), step):
        r = rows[i:i + step].to(device)
        out[i:i + step] = fn(_grid(r, ncols, device))
    return out


# ---------------------------------------------------------------- workloads

@dataclasses.dataclass(frozen=True)
class LayerSpec:
    """One quantized layer: X int8 [M x K], W int8 [N x K] (out x in).

    ``kind`` is "linear" or "conv3x3" (NHWC H x Wd x C input, stride 1, pad 1,
    W laid out [N][3][3][C], so K = 9*C and M = H*Wd)."""
    name: str
    M: int
    K: int
    N: int
    kind: str = "linear"
    H: int = 0
    Wd: int = 0
    C: int = 0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    layers: List[LayerSpec]
    S: int                 # number of denoising stages
    T: int                 # number of denoising steps
    b_lo: int              # b table drawn uniformly from [b_lo, b_hi]
    b_hi: int
    sx: float = 0.02
    bits: Optional[Sequence[int]] = None   # fixed b sweep for the single layer


def _dit_block(M, hidden, mlp, prefix=""):
    return [LayerSpec(prefix + "qkv", M, hidden, 3 * hidden),
            LayerSpec(prefix + "out", M, hidden, hidden),
            LayerSpec(prefix + "mlp_up", M, hidden, mlp),
            LayerSpec(prefix + "mlp_down", M, mlp, hidden)]


def workload(i: int, M_override: Optional[int] = None) -> Workload:
    """The five synthetic workloads.

    0: one 1152->1152 layer at 256 tokens, b in {8,6,4,2}.
    1: PixArt-Sigma-shaped DiT block, 1024px: 2x4096 tokens, hidden 1152.
    2: SANA-1.6B-shaped block: 4x1024 tokens, hidden 2240, GLU FFN.
    3: SDXL-Turbo-shaped UNet linears at 512px (64x64x640 and 32x32x1280)
       plus one 3x3 conv 1280->1280 at 32x32 as an implicit GEMM.
    4: 28 PixArt-Sigma-shaped blocks (112 layers), 20 steps, 4 stages.
    ``M_override`` replaces the token count (skinny-M sweeps).
    """
    def m(v):
        return v if M_override is None else M_override
    if i == 0:
        return Workload("single_1152", 0, [LayerSpec("linear", m(256), 1152, 1152)],
                        S=1, T=1, b_lo=8, b_hi=8, bits=(8, 6, 4, 2))
    if i == 1:
        return Workload("pixart_block", 1, _dit_block(m(8192), 1152, 4608),
                        S=1, T=1, b_lo=3, b_hi=8)
    if i == 2:
        M = m(4096)
        return Workload("sana_block", 2,
                        [LayerSpec("qkv", M, 2240, 6720), LayerSpec("out", M, 2240, 2240),
                         LayerSpec("glu_up", M, 2240, 11200),
                         LayerSpec("glu_down", M, 5600, 2240)],
                        S=4, T=20, b_lo=2, b_hi=8)
    if i == 3:
        MA, MB = m(4096), m(1024)
        layers = []
        for tag, M, C in (("A_", MA, 640), ("B_", MB, 1280)):
            layers += [LayerSpec(tag + "qkv", M, C, 3 * C), LayerSpec(tag + "proj", M, C, C),
                       LayerSpec(tag + "geglu_up", M, C, 8 * C),
                       LayerSpec(tag + "ff_down", M, 4 * C, C)]
        layers.append(LayerSpec("conv3x3", 32 * 32, 9 * 1280, 1280, kind="conv3x3",
                                H=32, Wd=32, C=1280))
        return Workload("sdxl_turbo_unet", 3, layers, S=4, T=4, b_lo=4, b_hi=8)
    if i == 4:
        layers = []
        for blk in range(28):
            layers += _dit_block(m(8192), 1152, 4608, prefix=f"blk{blk}_")
        return Workload("pixart_28block_schedule", 4, layers, S=4, T=20, b_lo=2, b_hi=8)
    raise ValueError(f"no workload {i}")


def shard(wl: Workload, axis: str, parts: int) -> Workload:
    """Shard 0 of a ``parts``-way split of every layer of ``wl``.

    ``axis`` "M" keeps the first ceil(M / parts) token rows (X and the
    outputs split, W replicated); "N" keeps the first ceil(N / parts) output
    channels (W, sw and the outputs split, X replicated).  Neither split
    needs an exchange between shards, and b stays per layer.  The seed is
    kept, and every draw is counter-based, so the shard's tensors are
    exactly those rows or channels of the full workload's tensors.
    Convolutions are not split."""
    if axis not in ("M", "N") or parts < 1:
        raise ValueError("axis is 'M' or 'N', parts >= 1")
    layers = []
    for spec in wl.layers:
        if spec.kind != "linear":
            raise ValueError("only linear layers are split")
        if axis == "M":
            layers.append(dataclasses.replace(spec, M=-(-spec.M // parts)))
        else:
            layers.append(dataclasses.replace(spec, N=-(-spec.N // parts)))
    return dataclasses.replace(wl, name=f"{wl.name}_{axis}{parts}", layers=layers)


# tensor ids within a workload's seed
def tid_x(l): return 2 * l
def tid_w(l): return 2 * l + 1
def tid_sw(l): return 1000 + l
def tid_bias(l): return 2000 + l
TID_TABLE = 999


def x_rows(wl: Workload, l: int, rows, device="cpu") -> torch.Tensor:
    """Rows of X_l (int8 [len(rows) x K]); uniform on [-127, 127].

    For a conv layer X is the NHWC image flattened to [H*Wd x C] and the
    rows are pixels."""
    spec = wl.layers[l]
    width = spec.C if spec.kind == "conv3x3" else spec.K
    return _draw_rows(rows, width, device, torch.int8,
                      lambda idx: uniform_int(wl.seed, tid_x(l), idx, -127, 127))


def x_full(wl: Workload, l: int, device="cpu") -> torch.Tensor:
    spec = wl.layers[l]
    rows = spec.H * spec.Wd if spec.kind == "conv3x3" else spec.M
    out = x_rows(wl, l, torch.arange(rows), device)
    if spec.kind == "conv3x3":
        return out.reshape(spec.H, spec.Wd, spec.C)
    return out


def w_rows(wl: Workload, l: int, rows) -> torch.Tensor:
    """Rows (output channels) of W_l, int8 [len(rows) x K] on the CPU."""
    spec = wl.layers[l]
    return _draw_rows(rows, spec.K, "cpu", torch.int8,
                      lambda idx: normal_int8(wl.seed, tid_w(l), idx))


def w_full(wl: Workload, l: int) -> torch.Tensor:
    spec = wl.layers[l]
    return w_rows(wl, l, torch.arange(spec.N))


def sw_full(wl: Workload, l: int) -> torch.Tensor:
    """Per-output-channel weight scales, fp32 uniform on [1e-3, 1e-2)."""
    spec = wl.layers[l]
    return uniform_f32(wl.seed, tid_sw(l), torch.arange(spec.N), 1e-3, 1e-2)


def bias_full(wl: Workload, l: int) -> torch.Tensor:
    """Optional bias, fp32 uniform on [-1, 1); the workloads run without it."""
    spec = wl.layers[l]
    return uniform_f32(wl.seed, tid_bias(l), torch.arange(spec.N), -1.0, 1.0)


def b_table(wl: Workload) -> torch.Tensor:
    """uint8 [L x S] table of effective weight bits, uniform on [b_lo, b_hi]."""
    L = len(wl.layers)
    idx = torch.arange(L * wl.S, dtype=torch.int64)
    return uniform_int(wl.seed, TID_TABLE, idx, wl.b_lo, wl.b_hi,
                       dtype=torch.uint8).reshape(L, wl.S)


def activations_f32(seed: int, rows, K: int, shape: str = "outlier") -> torch.Tensor:
    """Rows of a real-valued activation matrix, fp32 [len(rows) x K] on the
    CPU, for the activation quantizer.

    "outlier": N(0, 1) with every 61st channel scaled by 24 (the few large
    channels of transformer activations).  "skewed": 0.5 z^2 - 0.17 with
    z ~ N(0, 1), a one-sided tail above a small negative floor, like the
    input of an MLP's second projection, the case an asymmetric range fits
    better than a symmetric one."""
    z = _draw_rows(rows, K, "cpu", torch.float32, lambda idx: normal_f32(seed, 5, idx))
    if shape == "outlier":
        gain = torch.ones(K, dtype=torch.float32)
        gain[::61] = 24.0
        return z * gain
    if shape == "skewed":
        return 0.5 * z * z - 0.17
    raise ValueError(shape)


def weights_f32(seed: int, N: int, K: int) -> torch.Tensor:
    """fp32 [N x K] real-valued weights for the weight quantizer: N(0, 1)
    scaled per output channel by sigma_n ~ U[0.01, 0.05) and shifted by
    mu_n ~ U[-0.005, 0.005) (channels of different spread and a small
    offset, so that per-channel zero points differ from the centre)."""
    z = _draw_rows(torch.arange(N), K, "cpu", torch.float32, lambda idx: normal_f32(seed, 6, idx))
    sigma = uniform_f32(seed, 7, torch.arange(N), 0.01, 0.05).reshape(N, 1)
    mu = uniform_f32(seed, 8, torch.arange(N), -0.005, 0.005).reshape(N, 1)
    return z * sigma + mu


def bf16_bits(seed: int, tid: int, shape, emin: int = -9, emax: int = -3) -> torch.Tensor:
    """int16 [shape] bit patterns of random bfloat16 values: a uniform sign,
    a uniform exponent in [emin, emax] and a uniform 7-bit mantissa, i.e.
    +-(1 + m/128) 2^e (the weights of a low-rank branch).  Drawn as integer
    fields, so no rounding is involved."""
    n = math.prod(shape)
    idx = torch.arange(n, dtype=torch.int64)
    sign = uniform_int(seed, tid, 3 * idx, 0, 1, dtype=torch.int32)
    expo = uniform_int(seed, tid, 3 * idx + 1, emin + 127, emax + 127, dtype=torch.int32)
    mant = uniform_int(seed, tid, 3 * idx + 2, 0, 127, dtype=torch.int32)
    bits = (sign << 15) | (expo << 7) | mant
    return torch.where(bits >= 32768, bits - 65536, bits).to(torch.int16).reshape(shape)


def random_case(seed: int, M: int, N: int, K: int, device="cpu"):
    """Free-form fuzz case: X, W uniform over the whole int8 range [-128, 127]
    (so both operands reach -128), sw uniform on [1e-3, 1e-2)."""
    X = _draw_rows(torch.arange(M), K, device, torch.int8,
                   lambda idx: uniform_int(seed, 1, idx, -128, 127))
    W = _draw_rows(torch.arange(N), K, device, torch.int8,
                   lambda idx: uniform_int(seed, 2, idx, -128, 127))
    sw = uniform_f32(seed, 3, torch.arange(N), 1e-3, 1e-2)
    bias = uniform_f32(seed, 4, torch.arange(N), -1.0, 1.0)
    return X, W, sw, bias
