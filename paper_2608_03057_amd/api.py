"""Torch-facing wrappers of the C ABI (argument marshalling only).

Each wrapper checks that tensors are on the GPU with the dtype and shape the
C ABI documents, passes ``data_ptr()`` and the current HIP stream, and
raises ``TasqError`` on a non-zero status.  The work is enqueued on the
current stream and is asynchronous like any other GPU op.
"""
from __future__ import annotations

import ctypes
from typing import List, Optional, Sequence

import torch

from . import _lib
from ._lib import Layer, Opts, check


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _need(t: Optional[torch.Tensor], dtype, shape, name):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _opts(variant, planes, workspace, split_k, packed=None, act=None, colsums=None,
          lowrank=None, wzero=None, tune=None) -> Opts:
    """``tune``: dict of tasq_opts tuning overrides (tile, packed_tile,
    persistent, persistent_wgs, persistent_parties; values as the header
    documents them, 0 = the library's choice)."""
    o = Opts()
    for k, v in (tune or {}).items():
        if k not in _lib.TUNING_FIELDS:
            raise ValueError(f"unknown tuning field {k}")
        setattr(o, k, int(v))
    o.variant = variant
    o.split_k = split_k
    o.W_planes = _ptr(planes)
    o.workspace = _ptr(workspace)
    o.workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    o.W_packed = _ptr(packed)
    o.act_params = _ptr(act)
    o.colsums = _ptr(colsums)
    if lowrank is not None:
        o.lowrank_T, o.lowrank_up, o.lowrank_rank = _lowrank_fields(lowrank)
    if wzero is not None:
        o.w_zero, o.x_rowsums = _ptr(wzero[0]), _ptr(wzero[1])
    return o


def _lowrank_fields(lowrank):
    """(T, up) of a low-rank branch -> the three struct fields."""
    T, up = lowrank
    if up.dtype not in (torch.bfloat16, torch.int16):
        raise ValueError("lowrank up projection must be bfloat16 (or its int16 bit patterns)")
    _need(T, torch.float32, (T.shape[0], up.shape[1]), "lowrank T")
    return _ptr(T), _ptr(up), int(up.shape[1])


def status_string(status: int) -> str:
    return _lib.status_string(status)


def stage_of_step(t: int, S: int, T: int) -> int:
    """floor(t*S/T) via the library; raises on a bad (t, S, T)."""
    s = _lib.lib().tasq_stage_of_step(t, S, T)
    if s < 0:
        raise _lib.TasqError(s, "tasq_stage_of_step")
    return s


def planes_bytes(N: int, K: int) -> int:
    return _lib.lib().tasq_planes_bytes(N, K)


def workspace_bytes(M: int, N: int, K: int) -> int:
    return _lib.lib().tasq_workspace_bytes(M, N, K)


def pack_planes(W: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """uint32 planes (as int32 storage) of int8 W [N, K], shaped
    [ceil(N/32), 8, ceil(K/128), 16, 4, 2]: (32-channel block, plane, K block,
    channel within a half, word, half), the layout of tasq_pack_planes."""
    N, K = W.shape
    _need(W, torch.int8, (N, K), "W")
    shape = ((N + 31) // 32, 8, (K + 127) // 128, 16, 4, 2)
    if out is None:
        out = torch.empty(shape, dtype=torch.int32, device=W.device)
    _need(out, torch.int32, shape, "planes")
    check(_lib.lib().tasq_pack_planes(_ptr(W), N, K, _ptr(out), _stream()), "tasq_pack_planes")
    return out


def packed_weight_bytes(N: int, K: int) -> int:
    return _lib.lib().tasq_packed_weight_bytes(N, K)


def pack_weights(W: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int8 W [N, K] (or conv W [N, 3, 3, C]) in the MFMA operand order,
    a flat int8 buffer of packed_weight_bytes(N, K) bytes."""
    N = W.shape[0]
    K = W.numel() // N if N else 0
    _need(W, torch.int8, tuple(W.shape), "W")
    nbytes = packed_weight_bytes(N, K)
    if out is None:
        out = torch.empty(nbytes, dtype=torch.int8, device=W.device)
    _need(out, torch.int8, (nbytes,), "packed")
    check(_lib.lib().tasq_pack_weights(_ptr(W), N, K, _ptr(out), _stream()), "tasq_pack_weights")
    return out


def quantize_activations(x: torch.Tensor, out: Optional[torch.Tensor] = None,
                         params: Optional[torch.Tensor] = None):
    """(int8 codes Q - 128 of x's shape, fp32 [TASQ_ACT_PARAMS_FLOATS] params
    with alpha at 0 and z at 1) of fp32 activations x, per tensor (App. A.1.2)."""
    M = x.shape[0] if x.dim() else 1
    K = x.numel() // M if M else 0
    _need(x, torch.float32, tuple(x.shape), "x")
    if out is None:
        out = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    if params is None:
        params = torch.empty(_lib.TASQ_ACT_PARAMS_FLOATS, dtype=torch.float32, device=x.device)
    _need(out, torch.int8, tuple(x.shape), "out")
    _need(params, torch.float32, (_lib.TASQ_ACT_PARAMS_FLOATS,), "params")
    check(_lib.lib().tasq_quantize_activations(_ptr(x), M, K, _ptr(out), _ptr(params), _stream()),
          "tasq_quantize_activations")
    return out, params


def quantize_activations_batch(xs, outs=None, params=None):
    """quantize_activations over a list of fp32 tensors in few launches
    (App. A.1.2): returns the lists of codes and params, each entry equal to
    what quantize_activations gives for that tensor.  Every tensor needs its
    own params buffer."""
    xs = list(xs)
    n = len(xs)
    outs = list(outs) if outs is not None else [None] * n
    params = list(params) if params is not None else [None] * n
    if len(outs) != n or len(params) != n:
        raise ValueError("xs, outs and params differ in length")
    jobs = (_lib.ActJob * max(n, 1))()
    for j, x in enumerate(xs):
        M = x.shape[0] if x.dim() else 1
        K = x.numel() // M if M else 0
        _need(x, torch.float32, tuple(x.shape), "x")
        if outs[j] is None:
            outs[j] = torch.empty(x.shape, dtype=torch.int8, device=x.device)
        if params[j] is None:
            params[j] = torch.empty(_lib.TASQ_ACT_PARAMS_FLOATS, dtype=torch.float32,
                                    device=x.device)
        _need(outs[j], torch.int8, tuple(x.shape), "out")
        _need(params[j], torch.float32, (_lib.TASQ_ACT_PARAMS_FLOATS,), "params")
        jobs[j] = _lib.ActJob(_ptr(x), M, K, _ptr(outs[j]), _ptr(params[j]))
    check(_lib.lib().tasq_quantize_activations_batch(jobs, n, _stream()),
          "tasq_quantize_activations_batch")
    return outs, params


def quantize_weights(W: torch.Tensor):
    """(codes int8 [N, ...], alpha, z, sw fp32 [N]) of fp32 weights W
    [N, ...]: the per-channel 8-bit quantizer of App. A.1.1; z is the
    w_zero and sw the sw of masked_linear."""
    N = W.shape[0]
    K = W.numel() // N if N else 0
    _need(W, torch.float32, tuple(W.shape), "W")
    Q = torch.empty(W.shape, dtype=torch.int8, device=W.device)
    alpha, z, sw = (torch.empty(N, dtype=torch.float32, device=W.device) for _ in range(3))
    check(_lib.lib().tasq_quantize_weights(_ptr(W), N, K, _ptr(Q), _ptr(alpha), _ptr(z),
                                           _ptr(sw), _stream()), "tasq_quantize_weights")
    return Q, alpha, z, sw


def quantize_weights_batch(Ws, outs=None):
    """quantize_weights over a list of fp32 weights in one launch per 16
    (App. A.1.1): returns one (codes, alpha, z, sw) tuple per weight, each
    equal to what quantize_weights gives for it.  ``outs``: such tuples to
    write into (allocated here when None)."""
    Ws = list(Ws)
    n = len(Ws)
    jobs = (_lib.WeightJob * max(n, 1))()
    if outs is None:
        outs = [None] * n
    outs = list(outs)
    if len(outs) != n:
        raise ValueError("Ws and outs differ in length")
    for j, W in enumerate(Ws):
        N = W.shape[0]
        K = W.numel() // N if N else 0
        _need(W, torch.float32, tuple(W.shape), "W")
        if outs[j] is None:
            outs[j] = (torch.empty(W.shape, dtype=torch.int8, device=W.device),
                       *(torch.empty(N, dtype=torch.float32, device=W.device) for _ in range(3)))
        Q, alpha, z, sw = outs[j]
        _need(Q, torch.int8, tuple(W.shape), "codes")
        for t, name in ((alpha, "alpha"), (z, "z"), (sw, "sw")):
            _need(t, torch.float32, (N,), name)
        jobs[j] = _lib.WeightJob(_ptr(W), N, K, _ptr(Q), _ptr(alpha), _ptr(z), _ptr(sw))
    check(_lib.lib().tasq_quantize_weights_batch(jobs, n, _stream()),
          "tasq_quantize_weights_batch")
    return outs


def row_sums(X: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int32 [M]: sum_k X[m, k] of int8 codes X [M, K]."""
    M = X.shape[0]
    K = X.numel() // M if M else 0
    _need(X, torch.int8, tuple(X.shape), "X")
    if out is None:
        out = torch.empty(M, dtype=torch.int32, device=X.device)
    _need(out, torch.int32, (M,), "out")
    check(_lib.lib().tasq_row_sums(_ptr(X), M, K, _ptr(out), _stream()), "tasq_row_sums")
    return out


def lowrank_down(x: torch.Tensor, down: torch.Tensor, out: Optional[torch.Tensor] = None):
    """T = bf16(x) down^T, fp32 [M, r], of fp32 x [M, K] and a bfloat16 (or
    int16 bit-pattern) down projection [r, K]."""
    M, K = x.shape
    r = down.shape[0]
    _need(x, torch.float32, (M, K), "x")
    if down.dtype not in (torch.bfloat16, torch.int16) or tuple(down.shape) != (r, K):
        raise ValueError("down must be bfloat16 [r, K]")
    if out is None:
        out = torch.empty((M, r), dtype=torch.float32, device=x.device)
    _need(out, torch.float32, (M, r), "out")
    check(_lib.lib().tasq_lowrank_down(_ptr(x), M, K, _ptr(down), r, _ptr(out), _stream()),
          "tasq_lowrank_down")
    return out


def quantize_activations_lowrank(x: torch.Tensor, down: torch.Tensor,
                                 out: Optional[torch.Tensor] = None,
                                 params: Optional[torch.Tensor] = None,
                                 T: Optional[torch.Tensor] = None):
    """(codes, params, T): quantize_activations and lowrank_down of x in one
    read of x."""
    M, K = x.shape
    r = down.shape[0]
    _need(x, torch.float32, (M, K), "x")
    if down.dtype not in (torch.bfloat16, torch.int16) or tuple(down.shape) != (r, K):
        raise ValueError("down must be bfloat16 [r, K]")
    if out is None:
        out = torch.empty((M, K), dtype=torch.int8, device=x.device)
    if params is None:
        params = torch.empty(_lib.TASQ_ACT_PARAMS_FLOATS, dtype=torch.float32, device=x.device)
    if T is None:
        T = torch.empty((M, r), dtype=torch.float32, device=x.device)
    _need(out, torch.int8, (M, K), "out")
    _need(params, torch.float32, (_lib.TASQ_ACT_PARAMS_FLOATS,), "params")
    _need(T, torch.float32, (M, r), "T")
    check(_lib.lib().tasq_quantize_activations_lowrank(_ptr(x), M, K, _ptr(out), _ptr(params),
                                                       _ptr(down), r, _ptr(T), _stream()),
          "tasq_quantize_activations_lowrank")
    return out, params, T


def weight_colsums(W: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """int32 [8, N]: row b-1 holds sum_k W_b[n][k] of int8 W [N, ...]."""
    N = W.shape[0]
    K = W.numel() // N if N else 0
    _need(W, torch.int8, tuple(W.shape), "W")
    if out is None:
        out = torch.empty((8, N), dtype=torch.int32, device=W.device)
    _need(out, torch.int32, (8, N), "colsums")
    check(_lib.lib().tasq_weight_colsums(_ptr(W), N, K, _ptr(out), _stream()),
          "tasq_weight_colsums")
    return out


def masked_linear(X: torch.Tensor, W: Optional[torch.Tensor], sx: float, sw: torch.Tensor,
                  b: int, bias: Optional[torch.Tensor] = None, *, want_acc: bool = True,
                  want_y: bool = True, acc: Optional[torch.Tensor] = None,
                  y: Optional[torch.Tensor] = None, variant: int = _lib.VARIANT_AUTO,
                  planes: Optional[torch.Tensor] = None, packed: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None, split_k: int = 0,
                  act: Optional[torch.Tensor] = None, colsums: Optional[torch.Tensor] = None,
                  lowrank=None, wzero=None, tune: Optional[dict] = None):
    """(acc int32 [M, N] or None, y fp32 [M, N] or None) of the masked layer.
    ``workspace`` (uint8, at least workspace_bytes(M, N, K) bytes) lets the
    library cut a long K into ranges (split_k); none is allocated here.
    With ``act`` (params of quantize_activations) and ``colsums`` X holds
    asymmetric activation codes and sx is ignored.  ``lowrank`` = (T, up)
    adds the low-rank branch T up^T to y (T from lowrank_down, up bfloat16
    [N, r]).  ``wzero`` = (z_w fp32 [N], row sums int32 [M]) takes W as
    zero-pointed codes (quantize_weights)."""
    M, K = X.shape
    N = sw.shape[0]
    _need(X, torch.int8, (M, K), "X")
    _need(W, torch.int8, (N, K), "W")
    _need(packed, torch.int8, (packed_weight_bytes(N, K),), "packed")
    _need(sw, torch.float32, (N,), "sw")
    _need(bias, torch.float32, (N,), "bias")
    if want_acc and acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=X.device)
    if want_y and y is None:
        y = torch.empty((M, N), dtype=torch.float32, device=X.device)
    _need(acc, torch.int32, (M, N), "acc")
    _need(y, torch.float32, (M, N), "y")
    _need(colsums, torch.int32, (8, N), "colsums")
    o = _opts(variant, planes, workspace, split_k, packed, act, colsums, lowrank, wzero, tune)
    rc = _lib.lib().tasq_masked_linear(_ptr(X), _ptr(W), float(sx), _ptr(sw), _ptr(bias), M, N,
                                       K, int(b), _ptr(acc), _ptr(y), ctypes.byref(o), _stream())
    check(rc, "tasq_masked_linear")
    return acc, y


def masked_conv3x3(X: torch.Tensor, W: Optional[torch.Tensor], sx: float, sw: torch.Tensor,
                   b: int, bias: Optional[torch.Tensor] = None, *, want_acc: bool = True,
                   want_y: bool = True, acc=None, y=None, workspace=None, split_k: int = 0,
                   packed: Optional[torch.Tensor] = None, variant: int = _lib.VARIANT_AUTO,
                   tune: Optional[dict] = None):
    """3x3 / pad 1 conv, X NHWC [H, Wd, C], W [N, 3, 3, C] -> [H, Wd, N].
    ``workspace`` as in masked_linear (with M = H*Wd, K = 9*C)."""
    H, Wd, C = X.shape
    N = sw.shape[0]
    _need(X, torch.int8, (H, Wd, C), "X")
    _need(W, torch.int8, (N, 3, 3, C), "W")
    _need(packed, torch.int8, (packed_weight_bytes(N, 9 * C),), "packed")
    _need(sw, torch.float32, (N,), "sw")
    _need(bias, torch.float32, (N,), "bias")
    if want_acc and acc is None:
        acc = torch.empty((H, Wd, N), dtype=torch.int32, device=X.device)
    if want_y and y is None:
        y = torch.empty((H, Wd, N), dtype=torch.float32, device=X.device)
    _need(acc, torch.int32, (H, Wd, N), "acc")
    _need(y, torch.float32, (H, Wd, N), "y")
    o = _opts(variant, None, workspace, split_k, packed, tune=tune)
    rc = _lib.lib().tasq_masked_conv3x3(_ptr(X), _ptr(W), float(sx), _ptr(sw), _ptr(bias), H, Wd,
                                        C, N, int(b), _ptr(acc), _ptr(y), ctypes.byref(o),
                                        _stream())
    check(rc, "tasq_masked_conv3x3")
    return acc, y


def make_layer(X, W, sx, sw, bias=None, acc=None, y=None, planes=None, kind=None,
               packed=None, act=None, colsums=None, lowrank=None, wzero=None) -> Layer:
    """A tasq_layer for run_schedule; tensors must stay alive while in use."""
    L = Layer()
    if kind is None:
        kind = _lib.KIND_CONV3X3 if X.dim() == 3 else _lib.KIND_LINEAR
    L.kind = kind
    if kind == _lib.KIND_CONV3X3:
        H, Wd, C = X.shape
        L.H, L.Wd, L.C = H, Wd, C
        L.M, L.K = H * Wd, 9 * C
    else:
        L.M, L.K = X.shape
    L.N = sw.shape[0]
    L.sx = float(sx)
    L.X, L.W, L.W_planes = _ptr(X), _ptr(W), _ptr(planes)
    L.sw, L.bias, L.acc, L.y = _ptr(sw), _ptr(bias), _ptr(acc), _ptr(y)
    L.W_packed = _ptr(packed)
    L.act_params = _ptr(act)
    L.colsums = _ptr(colsums)
    if lowrank is not None:
        L.lowrank_T, L.lowrank_up, L.lowrank_rank = _lowrank_fields(lowrank)
    if wzero is not None:
        L.w_zero, L.x_rowsums = _ptr(wzero[0]), _ptr(wzero[1])
    return L


def _layer_array(layers: Sequence[Layer]):
    arr = (Layer * len(layers))(*layers)
    return arr


def schedule_workspace_bytes(layers: Sequence[Layer]) -> int:
    arr = _layer_array(layers)
    return _lib.lib().tasq_schedule_workspace_bytes(arr, len(layers))


def schedule_cost(layers, table, S: int, T: int, t_begin: int, t_end: int,
                  act_bits: int = 8) -> dict:
    """Compute accounting of a schedule (tasq_schedule_cost): ``layers`` are
    Layer structs or (M, N, K) shapes, ``table`` a uint8 [L, S] host array.
    Host only."""
    structs = []
    for ly in layers:
        if isinstance(ly, Layer):
            structs.append(ly)
        else:
            st = Layer()
            st.kind = _lib.KIND_LINEAR
            st.M, st.N, st.K = (int(v) for v in ly)
            structs.append(st)
    table = torch.as_tensor(table).to(torch.uint8).contiguous().cpu()
    L = len(structs)
    if tuple(table.shape) != (L, S):
        raise ValueError(f"table must be [{L}, {S}]")
    arr = _layer_array(structs)
    out = _lib.Cost()
    check(_lib.lib().tasq_schedule_cost(arr, L, table.data_ptr(), S, T, t_begin, t_end,
                                        act_bits, ctypes.byref(out)), "tasq_schedule_cost")
    return {name: getattr(out, name) for name, _ in _lib.Cost._fields_}


def run_schedule(layers: Sequence[Layer], table: torch.Tensor, S: int, T: int, t_begin: int,
                 t_end: int, *, workspace: Optional[torch.Tensor] = None,
                 variant: int = _lib.VARIANT_AUTO, split_k: int = 0,
                 tune: Optional[dict] = None, step_events=None) -> None:
    """Runs steps t_begin..t_end-1; ``table`` is a host uint8 [L, S] tensor.
    ``step_events``: 2 * (t_end - t_begin) torch.cuda.Event objects, each
    recorded once already (torch creates the event at its first record); the
    library records pair i around the launches of step t_begin + i."""
    table = table.to(torch.uint8).contiguous().cpu()
    L = len(layers)
    if tuple(table.shape) != (L, S):
        raise ValueError(f"table must be [{L}, {S}]")
    arr = _layer_array(layers)
    o = _opts(variant, None, workspace, split_k, tune=tune)
    if step_events is not None:
        if len(step_events) != 2 * (t_end - t_begin):
            raise ValueError("step_events needs 2 * (t_end - t_begin) events")
        handles = [int(e.cuda_event) for e in step_events]
        if not all(handles):
            raise ValueError("record each step event once before passing it")
        evarr = (ctypes.c_void_p * len(handles))(*handles)
        o.step_events = ctypes.cast(evarr, ctypes.POINTER(ctypes.c_void_p))
    rc = _lib.lib().tasq_run_schedule(arr, L, table.data_ptr(), S, T, t_begin, t_end,
                                      ctypes.byref(o), _stream())
    check(rc, "tasq_run_schedule")


def run_schedule_noalloc(layers: Sequence[Layer], table: torch.Tensor, S: int, T: int,
                         t_begin: int, t_end: int, *, variant: int = _lib.VARIANT_AUTO,
                         tune: Optional[dict] = None) -> None:
    """run_schedule with the layer list in the library's per-GPU scratch array
    (tasq_run_schedule_noalloc): no workspace, nothing allocated."""
    table = table.to(torch.uint8).contiguous().cpu()
    L = len(layers)
    if tuple(table.shape) != (L, S):
        raise ValueError(f"table must be [{L}, {S}]")
    arr = _layer_array(layers)
    o = _opts(variant, None, None, 0, tune=tune)
    rc = _lib.lib().tasq_run_schedule_noalloc(arr, L, table.data_ptr(), S, T, t_begin, t_end,
                                              ctypes.byref(o), _stream())
    check(rc, "tasq_run_schedule_noalloc")
