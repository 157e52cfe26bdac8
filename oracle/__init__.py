"""CPU oracle for the TASQ masked quantized linear layer.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
CPU-baseline leg of the benchmark, never by the product path.  It shares no
code with the HIP library (``paper_2608_03057_amd``) and imports nothing from
it; the two meet only in the seeded inputs the tests hand to both.

The arithmetic lives in ``tasq_oracle.c`` (plain C, int64 accumulation, fp64
dequantisation).  This module loads it with ctypes and adds the schedule
(Sec. 3.2 contiguous stages, Sec. 4.1 step/stage counts), which only loops
over the C definition, and the 16-bit low-rank branch in numpy fp64 (its
products of bfloat16 values are exact in fp64).  ``brute.py`` is a second,
pure-Python route for tiny shapes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tasq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EBITS, EOVERFLOW, EDIM = 0, 1, 2, 3


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP over output rows)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Werror", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        L.oracle_num_threads.restype = ctypes.c_int
        L.oracle_set_num_threads.argtypes = [ctypes.c_int]
        L.oracle_set_num_threads.restype = None
        L.oracle_mask.argtypes = [p, i64, ctypes.c_int, p]
        L.oracle_stage_of_step.argtypes = [ctypes.c_int] * 3
        L.oracle_masked_linear.argtypes = [p, p, ctypes.c_double, p, p, i64, i64, i64,
                                           ctypes.c_int, p, p]
        L.oracle_masked_linear_entries.argtypes = [p, p, ctypes.c_double, p, p, i64,
                                                   ctypes.c_int, p, p, i64, p, p]
        L.oracle_conv3x3.argtypes = [p, p, ctypes.c_double, p, p, i64, i64, i64, i64,
                                     ctypes.c_int, p, p]
        L.oracle_conv3x3_entries.argtypes = [p, p, ctypes.c_double, p, p, i64, i64, i64,
                                             ctypes.c_int, p, p, i64, p, p]
        L.oracle_pack_planes.argtypes = [p, i64, i64, p]
        L.oracle_pack_weights.argtypes = [p, i64, i64, p]
        L.oracle_act_quant.argtypes = [p, i64, p, p, p]
        L.oracle_weight_colsums.argtypes = [p, i64, i64, p]
        L.oracle_masked_linear_asym.argtypes = [p, p, ctypes.c_double, ctypes.c_double, p, p,
                                                i64, i64, i64, ctypes.c_int, p, p]
        L.oracle_masked_linear_asym_entries.argtypes = [p, p, ctypes.c_double, ctypes.c_double,
                                                        p, p, i64, ctypes.c_int, p, p, i64, p, p]
        L.oracle_weight_quant.argtypes = [p, i64, i64, ctypes.c_int, p, p, p, p]
        d = ctypes.c_double
        L.oracle_layer_dequant.argtypes = [p, ctypes.c_int, d, d, d, p, p, p, p, i64, i64, i64,
                                           ctypes.c_int, p, p]
        L.oracle_layer_dequant_entries.argtypes = [p, ctypes.c_int, d, d, d, p, p, p, p, i64,
                                                   ctypes.c_int, p, p, i64, p, p]
        _lib = L
    return _lib


def _np(a, dtype):
    """Contiguous numpy view of a numpy array or CPU torch tensor."""
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data


def num_threads() -> int:
    return lib().oracle_num_threads()


def set_num_threads(n: int) -> None:
    """OpenMP threads of the oracle's following calls."""
    lib().oracle_set_num_threads(int(n))


def mask(W, b: int) -> np.ndarray:
    """2^k * floor(W / 2^k), k = 8 - b (App. G.2 Eq. hw_rightshift, masked form)."""
    W = _np(W, np.int8)
    out = np.empty_like(W)
    rc = lib().oracle_mask(_ptr(W), W.size, b, _ptr(out))
    if rc != OK:
        raise ValueError(f"oracle_mask: b={b} outside [1, 8]")
    return out


def stage_of_step(t: int, S: int, T: int) -> int:
    """Stage of denoising step t: floor(t*S/T), step 0 the noisiest."""
    s = lib().oracle_stage_of_step(t, S, T)
    if s < 0:
        raise ValueError(f"bad (t, S, T) = {(t, S, T)}")
    return s


def masked_linear(X, W, sx: float, sw, b: int, bias=None):
    """(acc int32 [M x N], y fp64 [M x N]) of the masked quantized linear."""
    X = _np(X, np.int8)
    W = _np(W, np.int8)
    sw = _np(sw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    M, K = X.shape
    N, K2 = W.shape
    assert K == K2 and sw.shape == (N,)
    acc = np.empty((M, N), np.int32)
    y = np.empty((M, N), np.float64)
    rc = lib().oracle_masked_linear(_ptr(X), _ptr(W), float(sx), _ptr(sw), _ptr(bias),
                                    M, N, K, b, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_masked_linear rc={rc}")
    return acc, y


def masked_linear_entries(X, W, sx, sw, b, rows, cols, bias=None):
    """The (rows[i], cols[i]) outputs only, each computed as one dot product.

    ``X`` is addressed by ``rows`` and ``W`` by ``cols`` (row n of W is output
    channel n), so callers may pass just the rows of X and W they sample,
    with ``rows``/``cols`` indexing those arrays, and ``sw``/``bias`` indexed
    likewise."""
    X = _np(X, np.int8)
    W = _np(W, np.int8)
    sw = _np(sw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    rows = _np(rows, np.int64)
    cols = _np(cols, np.int64)
    K = X.shape[1]
    assert W.shape[1] == K and rows.shape == cols.shape
    assert rows.size == 0 or (0 <= rows.min() and rows.max() < X.shape[0])
    assert cols.size == 0 or (0 <= cols.min() and cols.max() < W.shape[0])
    acc = np.empty(rows.size, np.int32)
    y = np.empty(rows.size, np.float64)
    rc = lib().oracle_masked_linear_entries(_ptr(X), _ptr(W), float(sx), _ptr(sw),
                                            _ptr(bias), K, b, _ptr(rows), _ptr(cols),
                                            rows.size, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_masked_linear_entries rc={rc}")
    return acc, y


def conv3x3(X, Wt, sx: float, sw, b: int, bias=None):
    """Direct 3x3 / stride 1 / pad 1 NHWC convolution with the masked weight.

    X int8 [H x Wd x Ci], Wt int8 [Co x 3 x 3 x Ci]; returns acc int32 and
    y fp64, both [H x Wd x Co]."""
    X = _np(X, np.int8)
    Wt = _np(Wt, np.int8)
    sw = _np(sw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    H, Wd, Ci = X.shape
    Co = Wt.shape[0]
    assert Wt.shape == (Co, 3, 3, Ci) and sw.shape == (Co,)
    acc = np.empty((H, Wd, Co), np.int32)
    y = np.empty((H, Wd, Co), np.float64)
    rc = lib().oracle_conv3x3(_ptr(X), _ptr(Wt), float(sx), _ptr(sw), _ptr(bias),
                              H, Wd, Ci, Co, b, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_conv3x3 rc={rc}")
    return acc, y


def conv3x3_entries(X, Wt, sx, sw, b, pix, cols, bias=None):
    """Outputs (pix[i] = h*Wd + w, cols[i]) of the masked 3x3 convolution,
    each computed as its own convolution sum."""
    X = _np(X, np.int8)
    Wt = _np(Wt, np.int8)
    sw = _np(sw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    pix = _np(pix, np.int64)
    cols = _np(cols, np.int64)
    H, Wd, Ci = X.shape
    Co = Wt.shape[0]
    assert Wt.shape == (Co, 3, 3, Ci) and pix.shape == cols.shape
    assert pix.size == 0 or (0 <= pix.min() and pix.max() < H * Wd)
    assert cols.size == 0 or (0 <= cols.min() and cols.max() < Co)
    acc = np.empty(pix.size, np.int32)
    y = np.empty(pix.size, np.float64)
    rc = lib().oracle_conv3x3_entries(_ptr(X), _ptr(Wt), float(sx), _ptr(sw), _ptr(bias), H, Wd,
                                      Ci, b, _ptr(pix), _ptr(cols), pix.size, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_conv3x3_entries rc={rc}")
    return acc, y


def pack_planes(W) -> np.ndarray:
    """uint32 [ceil(N/32), 8, ceil(K/128), 16, 4, 2] bit planes: index
    (nb, q, kb, r, w, f) is word w of channel n = 32*nb + 16*f + r in block kb
    of plane p = 7 - q (most significant first).  Element j of a row,
    e = j % 128, with s = e // 32, h = (e % 32) // 16, i = (e % 16) // 4,
    c = e % 4, lands in word 2*h + s // 2 of block j // 128 at bit
    (8*c + 4*(s % 2) + i + p) % 32."""
    W = _np(W, np.int8)
    N, K = W.shape
    NB, KB = (N + 31) // 32, (K + 127) // 128
    planes = np.empty((NB, 8, KB, 16, 4, 2), np.uint32)
    lib().oracle_pack_planes(_ptr(W), N, K, _ptr(planes))
    return planes


def pack_weights(W) -> np.ndarray:
    """Flat int8 buffer of W [N, K] in the int8 matrix-instruction operand
    order: W[n][k] at byte ((n//32 * KS + k//32) * 64 + n%32 + 32*((k%32)//16)) * 16
    + k%16, KS = 4*ceil(K/128), zeros elsewhere."""
    W = _np(W, np.int8)
    N, K = W.shape
    out = np.empty(32 * ((N + 31) // 32) * 128 * ((K + 127) // 128), np.int8)
    lib().oracle_pack_weights(_ptr(W), N, K, _ptr(out))
    return out


def act_quant(x):
    """(alpha, z, Q uint8 of x's shape): the per-tensor asymmetric 8-bit
    activation quantizer of App. A.1.2, decided in IEEE single precision."""
    x = _np(x, np.float32)
    q = np.empty(x.shape, np.uint8)
    a = np.empty(1, np.float32)
    z = np.empty(1, np.float32)
    rc = lib().oracle_act_quant(_ptr(x), x.size, _ptr(a), _ptr(z), _ptr(q))
    if rc != OK:
        raise ValueError(f"oracle_act_quant rc={rc}")
    return float(a[0]), float(z[0]), q


def weight_colsums(W) -> np.ndarray:
    """int32 [8 x N]: row b-1 holds sum_k W_b[n][k] for every output channel."""
    W = _np(W, np.int8)
    N = W.shape[0]
    K = W.size // N if N else 0
    out = np.empty((8, N), np.int32)
    rc = lib().oracle_weight_colsums(_ptr(W), N, K, _ptr(out))
    if rc != OK:
        raise ValueError(f"oracle_weight_colsums rc={rc}")
    return out


def masked_linear_asym(Q, W, alpha: float, z: float, sw, b: int, bias=None):
    """(acc int32 [M x N] of the signed codes Q - 128, y fp64 [M x N] of
    sum_k alpha (Q - z) sw W_b) for asymmetric activation codes Q."""
    Q = _np(Q, np.uint8)
    W = _np(W, np.int8)
    sw = _np(sw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    M, K = Q.shape
    N, K2 = W.shape
    assert K == K2 and sw.shape == (N,)
    acc = np.empty((M, N), np.int32)
    y = np.empty((M, N), np.float64)
    rc = lib().oracle_masked_linear_asym(_ptr(Q), _ptr(W), float(alpha), float(z), _ptr(sw),
                                         _ptr(bias), M, N, K, b, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_masked_linear_asym rc={rc}")
    return acc, y


def masked_linear_asym_entries(Q, W, alpha, z, sw, b, rows, cols, bias=None):
    """The (rows[i], cols[i]) outputs of masked_linear_asym, one dot product
    each (rows index Q, cols index W, sw and bias)."""
    Q = _np(Q, np.uint8)
    W = _np(W, np.int8)
    sw = _np(sw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    rows = _np(rows, np.int64)
    cols = _np(cols, np.int64)
    K = Q.shape[1]
    assert W.shape[1] == K and rows.shape == cols.shape
    acc = np.empty(rows.size, np.int32)
    y = np.empty(rows.size, np.float64)
    rc = lib().oracle_masked_linear_asym_entries(_ptr(Q), _ptr(W), float(alpha), float(z),
                                                 _ptr(sw), _ptr(bias), K, b, _ptr(rows),
                                                 _ptr(cols), rows.size, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_masked_linear_asym_entries rc={rc}")
    return acc, y


# ------------------------------------------------------ weight quantizer


def weight_quant(W, nbits: int = 8):
    """(Q uint8 [N x K], alpha [N], z [N], sw [N]) of fp32 W [N x K]: the
    per-channel n-bit weight quantizer of App. A.1.1 (floor, 2^n grid, real
    zero point), sw = alpha 2^n / (2^n - 1) the dequantisation factor."""
    W = _np(W, np.float32)
    N = W.shape[0]
    K = W.size // N if N else 0
    Q = np.empty((N, K), np.uint8)
    alpha = np.empty(N, np.float32)
    z = np.empty(N, np.float32)
    sw = np.empty(N, np.float32)
    rc = lib().oracle_weight_quant(_ptr(W), N, K, nbits, _ptr(Q), _ptr(alpha), _ptr(z), _ptr(sw))
    if rc != OK:
        raise ValueError(f"oracle_weight_quant rc={rc}")
    return Q, alpha, z, sw


def row_sums(X) -> np.ndarray:
    """int64 [M]: sum_k X[m][k] of int8 codes (the weight zero point's term)."""
    return np.asarray(X).astype(np.int64).reshape(np.asarray(X).shape[0], -1).sum(axis=1)


def _layer_args(act, sx):
    if act is None:
        return 0, float(sx), 0.0, 0.0
    ax, zx = act
    return 1, 0.0, float(ax), float(zx)


def layer_dequant(X, W, sw, b: int, sx: float = 0.0, act=None, zw=None, bias=None):
    """(acc int32, y fp64) of sum_k x_hat w_hat_b (+ bias): x_hat = sx X, or
    alpha (X + 128 - z) with act = (alpha, z); w_hat_b = sw W_b, or
    sw (W_b + 128 - zw[n]) with per-channel zero points zw."""
    X = _np(X, np.int8)
    W = _np(W, np.int8)
    sw = _np(sw, np.float32)
    zw = None if zw is None else _np(zw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    M, K = X.shape
    N = W.shape[0]
    acc = np.empty((M, N), np.int32)
    y = np.empty((M, N), np.float64)
    asym, sxv, ax, zx = _layer_args(act, sx)
    rc = lib().oracle_layer_dequant(_ptr(X), asym, sxv, ax, zx, _ptr(W), _ptr(sw), _ptr(zw),
                                    _ptr(bias), M, N, K, b, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_layer_dequant rc={rc}")
    return acc, y


def layer_dequant_entries(X, W, sw, b, rows, cols, sx=0.0, act=None, zw=None, bias=None):
    """The (rows[i], cols[i]) outputs of layer_dequant."""
    X = _np(X, np.int8)
    W = _np(W, np.int8)
    sw = _np(sw, np.float32)
    zw = None if zw is None else _np(zw, np.float32)
    bias = None if bias is None else _np(bias, np.float32)
    rows = _np(rows, np.int64)
    cols = _np(cols, np.int64)
    K = X.shape[1]
    acc = np.empty(rows.size, np.int32)
    y = np.empty(rows.size, np.float64)
    asym, sxv, ax, zx = _layer_args(act, sx)
    rc = lib().oracle_layer_dequant_entries(_ptr(X), asym, sxv, ax, zx, _ptr(W), _ptr(sw),
                                            _ptr(zw), _ptr(bias), K, b, _ptr(rows), _ptr(cols),
                                            rows.size, _ptr(acc), _ptr(y))
    if rc == EOVERFLOW:
        raise OverflowError("accumulator outside int32")
    if rc != OK:
        raise ValueError(f"oracle_layer_dequant_entries rc={rc}")
    return acc, y


# --------------------------------------------------- 16-bit low-rank branch
#
# The SVDQuant-initialised models carry a frozen 16-bit low-rank branch beside
# the quantized layer (Sec. 4.1 setup: rank 16 at the 6-bit setting, rank 32
# at 4 bits; App. training details).  Its output is added to the dequantised
# GEMM:  y = dequant(X W_b^T) + (x~ D^T) U^T,  with D [r x K] the down and
# U [N x r] the up projection held in bfloat16, and x~ the activation rounded
# to bfloat16 (the branch runs in 16 bits).  The oracle evaluates the branch
# in fp64 from those 16-bit values; every product of two bfloat16 values is
# exact in fp64.


def bf16_value(bits) -> np.ndarray:
    """fp64 values of bfloat16 bit patterns (the upper half of an IEEE
    single with the same bits)."""
    bits = np.asarray(bits).astype(np.uint16).astype(np.uint32)
    return (bits << np.uint32(16)).view(np.float32).astype(np.float64)


def bf16_round(x) -> np.ndarray:
    """bfloat16 bit patterns of fp32 values, rounded to nearest with ties to
    even: the nearest multiple of the bfloat16 spacing at x's binade (2^(e-8)
    for x = m 2^e, 1/2 <= |m| < 1, and 2^-133 below the normal range)."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    _, e = np.frexp(x)
    spacing = np.ldexp(1.0, np.maximum(e - 8, -133))
    v = np.rint(x / spacing) * spacing                      # exact in fp64
    return (v.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def lowrank(x, down, up):
    """(T fp64 [M x r], lr fp64 [M x N]) of the low-rank branch:
    T = x~ D^T, lr = T U^T, with x~ = bf16_round(x) and D, U given as
    bfloat16 bit patterns ([r x K] and [N x r])."""
    xt = bf16_value(bf16_round(x))
    D = bf16_value(down)
    U = bf16_value(up)
    assert xt.shape[1] == D.shape[1] and U.shape[1] == D.shape[0]
    T = xt @ D.T
    return T, T @ U.T


def lowrank_entries(x_rows, down, up, rows, cols) -> np.ndarray:
    """lr[rows[i], cols[i]] where ``rows`` index x_rows (the branch of a few
    activation rows, e.g. sampled from a full-size layer)."""
    T, _ = lowrank(x_rows, down, up[:1])
    U = bf16_value(up)
    rows = np.asarray(rows, np.int64)
    cols = np.asarray(cols, np.int64)
    return np.einsum("ij,ij->i", T[rows], U[cols])


def run_schedule(layers, table, S: int, T: int, t_begin: int, t_end: int, sx: float):
    """Buffers left by running denoising steps t_begin..t_end-1 of a schedule.

    ``layers`` is a list of dicts with keys X, W, sw, bias (optional) and
    kind ("linear" or "conv3x3").  Each step t computes every layer at
    b = table[l][stage(t)] and overwrites that layer's output buffers
    (Sec. 3.2: one mask per layer and stage).  Returns, per layer, the last
    (acc, y, b) written, or None if the range is empty (buffers untouched).
    Literal loop over steps: meant for small shapes.
    """
    if not (0 <= t_begin <= t_end <= T):
        raise ValueError("bad step range")
    out = [None] * len(layers)
    for t in range(t_begin, t_end):
        s = stage_of_step(t, S, T)
        for l, layer in enumerate(layers):
            b = int(table[l][s])
            if layer.get("kind", "linear") == "conv3x3":
                acc, y = conv3x3(layer["X"], layer["W"], sx, layer["sw"], b,
                                 layer.get("bias"))
            else:
                acc, y = masked_linear(layer["X"], layer["W"], sx, layer["sw"], b,
                                       layer.get("bias"))
            out[l] = (acc, y, b)
    return out


# ------------------------------------------------ BitOPs and cycle accounting
#
# Sec. 4 reports Eff. W-bit (average operating weight precision) and Rel.
# BitOPs (compute normalised to static W8A8) per schedule; Sec. 3.3 / 4.3
# measure the bit-serial engine, whose cycles grow with the product of
# weight and activation planes L R with no cost for switching precision
# (Tab. measured: 528 cycles for four W1A4 tiles, i.e. 33 cycles per plane
# pair per tile), and give per-tile totals for three dataflows at R = 4
# (Tab. codesign), each linear in L.

TPE_CYCLES_PER_PLANE_PAIR = 33
# (slope, intercept) of total cycles per tile at R = 4 (Tab. codesign).
TPE_TILE_LAW_R4 = {"naive": (4560, 173), "weight_stationary": (2850, 173),
                   "activation_stationary": (570, 2603)}


def tpe_cycles_measured(tile_bits, R: int = 4) -> int:
    """Cycles of tiles run at weight precisions tile_bits and R activation
    planes under the measured law (no switching overhead)."""
    return sum(TPE_CYCLES_PER_PLANE_PAIR * int(L) * R for L in tile_bits)


def tpe_tile_cycles(dataflow: str, L: int) -> int:
    slope, icpt = TPE_TILE_LAW_R4[dataflow]
    return slope * L + icpt


def fetch_planes(dataflow: str, L: int, R: int) -> int:
    """Bit planes fetched per tile (Tab. codesign model column)."""
    return {"naive": 2 * L * R, "weight_stationary": L + L * R,
            "activation_stationary": L + R}[dataflow]


def schedule_cost(macs_per_layer, table, S: int, T: int, t_begin: int, t_end: int,
                  act_bits: int) -> dict:
    """Accounting of steps t_begin..t_end-1 of a schedule, summed over every
    (layer, step) GEMM with b = table[l][stage(t)]:
      macs, b_eff = sum MACs b / macs (MAC-weighted), b_mean = plain mean of
      b over (layer, step), bitops = sum MACs b a, rel_bitops = bitops /
      (64 macs), rel_cycles_measured = sum MACs b a / sum MACs 8 a (the
      measured law), rel_cycles_as_a4 = sum MACs (570 b + 2603) / sum MACs
      (570*8 + 2603) (activation-stationary tile law at R = 4)."""
    macs = bw = bitops = c_as = c_as8 = 0
    bsum = count = 0
    for t in range(t_begin, t_end):
        s = stage_of_step(t, S, T)
        for l, mac in enumerate(macs_per_layer):
            b = int(table[l][s])
            macs += mac
            bw += mac * b
            bitops += mac * b * act_bits
            c_as += mac * tpe_tile_cycles("activation_stationary", b)
            c_as8 += mac * tpe_tile_cycles("activation_stationary", 8)
            bsum += b
            count += 1
    if count == 0:
        return dict(macs=0.0, b_eff=0.0, b_mean=0.0, bitops=0.0, rel_bitops=0.0,
                    rel_cycles_measured=0.0, rel_cycles_as_a4=0.0)
    return dict(macs=float(macs), b_eff=bw / macs if macs else 0.0, b_mean=bsum / count,
                bitops=float(bitops), rel_bitops=bitops / (64 * macs) if macs else 0.0,
                rel_cycles_measured=bitops / (8 * act_bits * macs) if macs else 0.0,
                rel_cycles_as_a4=c_as / c_as8 if macs else 0.0)
