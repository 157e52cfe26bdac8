"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/tasq.h declares, and rejects every bad argument before touching a
device (the pointers below are never dereferenced: each call fails
validation, or is an empty problem that enqueues nothing)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT, read_golden
from paper_2608_03057_amd import _lib
from paper_2608_03057_amd._lib import Layer, Opts

L = _lib.lib()
FAKE = 0x10000          # 256-byte aligned, never dereferenced


def header_symbols():
    text = open(os.path.join(ROOT, "include", "tasq.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tasq_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    syms = header_symbols()
    assert set(syms) == set(_lib.EXPORTS)
    for s in syms:
        assert hasattr(L, s), s


def test_status_strings():
    for code in range(0, -11, -1):
        s = _lib.status_string(code)
        assert s and s != "unknown status"
    assert _lib.status_string(-99) == "unknown status"


def test_stage_of_step_golden():
    for row in read_golden("stage_map.txt"):
        T, S, stages = row[0], row[1], row[2:]
        assert [L.tasq_stage_of_step(t, S, T) for t in range(T)] == stages


@pytest.mark.parametrize("t,S,T", [(-1, 4, 20), (20, 4, 20), (0, 0, 20), (0, 5, 4), (0, 1, 0)])
def test_stage_of_step_range(t, S, T):
    assert L.tasq_stage_of_step(t, S, T) == _lib.TASQ_ERR_RANGE


def test_planes_bytes():
    # 8 planes x 32 * ceil(N/32) channels x ceil(K/128) blocks x 16 bytes
    assert L.tasq_planes_bytes(1152, 1152) == 8 * 9 * 1152 * 16
    assert L.tasq_planes_bytes(3, 1) == 8 * 1 * 32 * 16
    assert L.tasq_planes_bytes(3, 129) == 8 * 2 * 32 * 16
    assert L.tasq_planes_bytes(33, 128) == 8 * 1 * 64 * 16
    assert L.tasq_planes_bytes(0, 128) == 0 and L.tasq_planes_bytes(5, 0) == 0


def lin(**kw):
    a = dict(X=FAKE, W=FAKE, sx=0.02, sw=FAKE, bias=None, M=4, N=4, K=32, b=8, acc=FAKE,
             y=FAKE, opts=None)
    a.update(kw)
    o = a["opts"]
    return L.tasq_masked_linear(a["X"], a["W"], a["sx"], a["sw"], a["bias"], a["M"], a["N"],
                                a["K"], a["b"], a["acc"], a["y"],
                                ctypes.byref(o) if o is not None else None, None)


def opts(**kw):
    o = Opts()
    for k, v in kw.items():
        setattr(o, k, v)
    return o


@pytest.mark.parametrize("kw,code", [
    (dict(X=None), _lib.TASQ_ERR_NULL),
    (dict(W=None), _lib.TASQ_ERR_NULL),
    (dict(sw=None), _lib.TASQ_ERR_NULL),
    (dict(acc=None, y=None), _lib.TASQ_ERR_NULL),
    (dict(M=-1), _lib.TASQ_ERR_DIM),
    (dict(N=-5), _lib.TASQ_ERR_DIM),
    (dict(K=-1), _lib.TASQ_ERR_DIM),
    (dict(b=0), _lib.TASQ_ERR_BITS),
    (dict(b=9), _lib.TASQ_ERR_BITS),
    (dict(b=-3), _lib.TASQ_ERR_BITS),
    (dict(K=131072), _lib.TASQ_ERR_OVERFLOW),
    (dict(opts=opts(variant=7)), _lib.TASQ_ERR_KIND),
    (dict(opts=opts(variant=_lib.VARIANT_BITPLANE)), _lib.TASQ_ERR_LAYOUT),
    (dict(W=None, opts=opts(variant=_lib.VARIANT_MASKED_I8)), _lib.TASQ_ERR_NULL),
    (dict(opts=opts(workspace=FAKE + 8, workspace_bytes=1024)), _lib.TASQ_ERR_ALIGN),
    (dict(opts=opts(split_k=-2)), _lib.TASQ_ERR_RANGE),
    (dict(opts=opts(variant=_lib.VARIANT_PACKED)), _lib.TASQ_ERR_LAYOUT),
    (dict(opts=opts(W_packed=FAKE + 4)), _lib.TASQ_ERR_ALIGN),
    (dict(W=None, opts=opts(variant=_lib.VARIANT_MASKED_I8, W_packed=FAKE)), _lib.TASQ_ERR_NULL),
    (dict(W=None, b=0, opts=opts(W_packed=FAKE)), _lib.TASQ_ERR_BITS),
    (dict(opts=opts(act_params=FAKE)), _lib.TASQ_ERR_NULL),
    (dict(opts=opts(act_params=FAKE + 2, colsums=FAKE)), _lib.TASQ_ERR_ALIGN),
    (dict(opts=opts(act_params=FAKE, colsums=FAKE + 1)), _lib.TASQ_ERR_ALIGN),
    (dict(opts=opts(lowrank_T=FAKE, lowrank_rank=16)), _lib.TASQ_ERR_NULL),
    (dict(opts=opts(lowrank_T=FAKE, lowrank_up=FAKE, lowrank_rank=24)), _lib.TASQ_ERR_DIM),
    (dict(opts=opts(lowrank_T=FAKE, lowrank_up=FAKE, lowrank_rank=0)), _lib.TASQ_ERR_DIM),
    (dict(opts=opts(lowrank_T=FAKE + 4, lowrank_up=FAKE, lowrank_rank=16)), _lib.TASQ_ERR_ALIGN),
    (dict(opts=opts(lowrank_T=FAKE, lowrank_up=FAKE + 8, lowrank_rank=32)), _lib.TASQ_ERR_ALIGN),
    (dict(opts=opts(w_zero=FAKE)), _lib.TASQ_ERR_NULL),
    (dict(opts=opts(w_zero=FAKE + 2, x_rowsums=FAKE)), _lib.TASQ_ERR_ALIGN),
    (dict(opts=opts(w_zero=FAKE, x_rowsums=FAKE + 1)), _lib.TASQ_ERR_ALIGN),
])
def test_masked_linear_rejects(kw, code):
    assert lin(**kw) == code


@pytest.mark.parametrize("kw", [dict(M=0), dict(N=0), dict(M=0, N=0, K=0)])
def test_masked_linear_empty_is_noop(kw):
    assert lin(**kw) == _lib.TASQ_OK


def test_bitplane_variant_accepts_missing_w_only_with_planes():
    o = opts(variant=_lib.VARIANT_BITPLANE, W_planes=FAKE)
    assert lin(W=None, M=0, opts=o) == _lib.TASQ_OK
    assert lin(W=None, b=0, opts=o) == _lib.TASQ_ERR_BITS


def test_packed_variant_accepts_missing_w_only_with_packed():
    for v in (_lib.VARIANT_AUTO, _lib.VARIANT_PACKED):
        assert lin(W=None, M=0, opts=opts(variant=v, W_packed=FAKE)) == _lib.TASQ_OK
    assert lin(W=None, M=0, opts=opts(variant=_lib.VARIANT_PACKED)) == _lib.TASQ_ERR_LAYOUT


def test_workspace_bytes_split_k():
    """Workspace of the split-K choice: only for K >= 8192 with at most 64
    tiles of 256x256; s ranges of at least 1024 of K, as many as fill the 256
    CUs once, rounded to 128-wide chunks (the SDXL-Turbo conv: 11 ranges
    asked, chunks of 1152, 10 used)."""
    assert L.tasq_workspace_bytes(1024, 1280, 11520) == 10 * 1024 * 1280 * 4
    assert L.tasq_workspace_bytes(256, 256, 16384) == 16 * 256 * 256 * 4
    assert L.tasq_workspace_bytes(1024, 1280, 5120) == 0       # K too short
    assert L.tasq_workspace_bytes(8192, 3456, 1152) == 0      # enough tiles
    assert L.tasq_workspace_bytes(1024, 1280, 1280) == 0      # K too short
    assert L.tasq_workspace_bytes(0, 1280, 5120) == 0


def test_forced_split_without_workspace_rejected():
    assert lin(M=300, N=64, K=512, opts=opts(split_k=4)) == _lib.TASQ_ERR_WORKSPACE
    assert lin(M=300, N=64, K=512, opts=opts(split_k=4, workspace=FAKE,
                                              workspace_bytes=1024)) == _lib.TASQ_ERR_WORKSPACE


def test_packed_weight_bytes():
    assert L.tasq_packed_weight_bytes(1152, 1152) == 1152 * 1152
    assert L.tasq_packed_weight_bytes(33, 129) == 64 * 256
    assert L.tasq_packed_weight_bytes(1, 1) == 32 * 128
    assert L.tasq_packed_weight_bytes(0, 5) == 0


def test_pack_weights_rejects():
    assert L.tasq_pack_weights(None, 4, 4, FAKE, None) == _lib.TASQ_ERR_NULL
    assert L.tasq_pack_weights(FAKE, 4, 4, None, None) == _lib.TASQ_ERR_NULL
    assert L.tasq_pack_weights(FAKE, -1, 4, FAKE, None) == _lib.TASQ_ERR_DIM
    assert L.tasq_pack_weights(FAKE, 4, 131072, FAKE, None) == _lib.TASQ_ERR_OVERFLOW
    assert L.tasq_pack_weights(FAKE, 4, 4, FAKE + 8, None) == _lib.TASQ_ERR_ALIGN
    assert L.tasq_pack_weights(FAKE, 0, 4, FAKE, None) == _lib.TASQ_OK


def test_quantize_activations_rejects():
    q = L.tasq_quantize_activations
    assert q(None, 4, 4, FAKE, FAKE, None) == _lib.TASQ_ERR_NULL
    assert q(FAKE, 4, 4, None, FAKE, None) == _lib.TASQ_ERR_NULL
    assert q(FAKE, 4, 4, FAKE, None, None) == _lib.TASQ_ERR_NULL
    assert q(FAKE, -1, 4, FAKE, FAKE, None) == _lib.TASQ_ERR_DIM
    assert q(FAKE, 4, -2, FAKE, FAKE, None) == _lib.TASQ_ERR_DIM
    assert q(FAKE + 2, 4, 4, FAKE, FAKE, None) == _lib.TASQ_ERR_ALIGN
    assert q(FAKE, 4, 4, FAKE, FAKE + 1, None) == _lib.TASQ_ERR_ALIGN
    assert q(None, 0, 4, None, None, None) == _lib.TASQ_OK          # empty: nothing enqueued


def test_quantize_activations_batch_rejects():
    """Every job is validated before anything is enqueued; a bad job anywhere
    in the list fails the whole call."""
    f = L.tasq_quantize_activations_batch

    def jobs(*js):
        arr = (_lib.ActJob * len(js))()
        for i, j in enumerate(js):
            arr[i] = _lib.ActJob(*j)
        return arr
    good = (FAKE, 4, 4, FAKE, FAKE)
    other = (FAKE, 4, 4, FAKE, FAKE + 4096)
    assert f(None, 0, None) == _lib.TASQ_OK                           # nothing to do
    assert f(None, 2, None) == _lib.TASQ_ERR_NULL
    assert f(jobs(good), -1, None) == _lib.TASQ_ERR_RANGE
    assert f(jobs(good, (None, 4, 4, FAKE, FAKE + 8192)), 2, None) == _lib.TASQ_ERR_NULL
    assert f(jobs(good, (FAKE, 4, 4, None, FAKE + 8192)), 2, None) == _lib.TASQ_ERR_NULL
    assert f(jobs(good, (FAKE, 4, 4, FAKE, None)), 2, None) == _lib.TASQ_ERR_NULL
    assert f(jobs(good, (FAKE, -1, 4, FAKE, FAKE + 8192)), 2, None) == _lib.TASQ_ERR_DIM
    assert f(jobs(good, (FAKE, 4, -3, FAKE, FAKE + 8192)), 2, None) == _lib.TASQ_ERR_DIM
    assert f(jobs(good, (FAKE + 2, 4, 4, FAKE, FAKE + 8192)), 2, None) == _lib.TASQ_ERR_ALIGN
    assert f(jobs(good, (FAKE, 4, 4, FAKE, FAKE + 8194)), 2, None) == _lib.TASQ_ERR_ALIGN
    # two jobs sharing one act_params buffer
    assert f(jobs(good, other, (FAKE, 8, 8, FAKE, FAKE)), 3, None) == _lib.TASQ_ERR_RANGE
    # empty jobs are skipped, whatever their pointers
    assert f(jobs((None, 0, 4, None, None), (None, 5, 0, None, None)), 2, None) == _lib.TASQ_OK


def test_quantize_weights_batch_rejects():
    """Every weight job is validated before anything is enqueued, as the
    single call validates its arguments; a bad job anywhere fails the call."""
    f = L.tasq_quantize_weights_batch

    def jobs(*js):
        arr = (_lib.WeightJob * len(js))()
        for i, j in enumerate(js):
            arr[i] = _lib.WeightJob(*j)
        return arr
    good = (FAKE, 4, 8, FAKE, FAKE, FAKE, FAKE)

    def job(**kw):
        names = ["W", "N", "K", "W_out", "alpha_out", "z_out", "sw_out"]
        v = dict(zip(names, (FAKE, 4, 8, FAKE, FAKE + 8192, FAKE, FAKE)))
        v.update(kw)
        return tuple(v[n] for n in names)
    assert f(None, 0, None) == _lib.TASQ_OK                           # nothing to do
    assert f(None, 2, None) == _lib.TASQ_ERR_NULL
    assert f(jobs(good), -1, None) == _lib.TASQ_ERR_RANGE
    for name in ("W", "W_out", "alpha_out", "z_out", "sw_out"):
        assert f(jobs(good, job(**{name: None})), 2, None) == _lib.TASQ_ERR_NULL, name
    assert f(jobs(good, job(N=-1)), 2, None) == _lib.TASQ_ERR_DIM
    assert f(jobs(good, job(K=-3)), 2, None) == _lib.TASQ_ERR_DIM
    assert f(jobs(good, job(K=0)), 2, None) == _lib.TASQ_ERR_DIM     # N > 0 with K == 0
    assert f(jobs(good, job(K=_lib.TASQ_MAX_K + 1)), 2, None) == _lib.TASQ_ERR_OVERFLOW
    for name in ("W", "alpha_out", "z_out", "sw_out"):
        bad = job(**{name: FAKE + 8192 + 2})
        assert f(jobs(good, bad), 2, None) == _lib.TASQ_ERR_ALIGN, name
    # two jobs sharing one alpha_out buffer
    assert f(jobs(good, job(alpha_out=FAKE)), 2, None) == _lib.TASQ_ERR_RANGE
    # empty jobs are skipped, whatever their pointers
    assert f(jobs((None, 0, 4, None, None, None, None), (None, 0, 0, None, None, None, None)),
             2, None) == _lib.TASQ_OK


def test_lowrank_down_rejects():
    f = L.tasq_lowrank_down
    assert f(FAKE, 4, 4, FAKE, 24, FAKE, None) == _lib.TASQ_ERR_DIM
    assert f(FAKE, 4, 4, FAKE, 64, FAKE, None) == _lib.TASQ_ERR_DIM
    assert f(FAKE, -1, 4, FAKE, 16, FAKE, None) == _lib.TASQ_ERR_DIM
    assert f(None, 4, 4, FAKE, 16, FAKE, None) == _lib.TASQ_ERR_NULL
    assert f(FAKE, 4, 4, None, 16, FAKE, None) == _lib.TASQ_ERR_NULL
    assert f(FAKE, 4, 4, FAKE, 16, None, None) == _lib.TASQ_ERR_NULL
    assert f(FAKE + 2, 4, 4, FAKE, 16, FAKE, None) == _lib.TASQ_ERR_ALIGN
    assert f(FAKE, 4, 4, FAKE + 1, 16, FAKE, None) == _lib.TASQ_ERR_ALIGN
    assert f(FAKE, 1 << 24, 4, FAKE, 32, FAKE, None) == _lib.TASQ_ERR_DIM   # M*r*4 >= 2^31
    assert f(None, 0, 4, None, 16, None, None) == _lib.TASQ_OK
    g = L.tasq_quantize_activations_lowrank
    assert g(FAKE, 4, 4, None, FAKE, FAKE, 16, FAKE, None) == _lib.TASQ_ERR_NULL
    assert g(FAKE, 4, 4, FAKE, None, FAKE, 16, FAKE, None) == _lib.TASQ_ERR_NULL
    assert g(FAKE, 4, 4, FAKE, FAKE + 2, FAKE, 16, FAKE, None) == _lib.TASQ_ERR_ALIGN
    assert g(FAKE, 4, 4, FAKE, FAKE, FAKE, 48, FAKE, None) == _lib.TASQ_ERR_DIM
    assert g(None, 0, 4, None, None, None, 32, None, None) == _lib.TASQ_OK


def test_quantize_weights_and_row_sums_reject():
    q = L.tasq_quantize_weights
    assert q(None, 4, 4, FAKE, FAKE, FAKE, FAKE, None) == _lib.TASQ_ERR_NULL
    assert q(FAKE, 4, 4, FAKE, FAKE, None, FAKE, None) == _lib.TASQ_ERR_NULL
    assert q(FAKE, 4, 0, FAKE, FAKE, FAKE, FAKE, None) == _lib.TASQ_ERR_DIM
    assert q(FAKE, -1, 4, FAKE, FAKE, FAKE, FAKE, None) == _lib.TASQ_ERR_DIM
    assert q(FAKE, 4, 131072, FAKE, FAKE, FAKE, FAKE, None) == _lib.TASQ_ERR_OVERFLOW
    assert q(FAKE + 2, 4, 4, FAKE, FAKE, FAKE, FAKE, None) == _lib.TASQ_ERR_ALIGN
    assert q(FAKE, 4, 4, FAKE, FAKE, FAKE, FAKE + 1, None) == _lib.TASQ_ERR_ALIGN
    assert q(None, 0, 4, None, None, None, None, None) == _lib.TASQ_OK
    r = L.tasq_row_sums
    assert r(None, 4, 4, FAKE, None) == _lib.TASQ_ERR_NULL
    assert r(FAKE, 4, 4, None, None) == _lib.TASQ_ERR_NULL
    assert r(FAKE, -1, 4, FAKE, None) == _lib.TASQ_ERR_DIM
    assert r(FAKE, 4, 131072, FAKE, None) == _lib.TASQ_ERR_OVERFLOW
    assert r(FAKE, 4, 4, FAKE + 2, None) == _lib.TASQ_ERR_ALIGN
    assert r(None, 0, 4, None, None) == _lib.TASQ_OK


def test_weight_colsums_rejects():
    c = L.tasq_weight_colsums
    assert c(None, 4, 4, FAKE, None) == _lib.TASQ_ERR_NULL
    assert c(FAKE, 4, 4, None, None) == _lib.TASQ_ERR_NULL
    assert c(FAKE, -1, 4, FAKE, None) == _lib.TASQ_ERR_DIM
    assert c(FAKE, 4, 131072, FAKE, None) == _lib.TASQ_ERR_OVERFLOW
    assert c(FAKE, 0, 4, None, None) == _lib.TASQ_OK


def test_schedule_asymmetric_layer_needs_colsums():
    tbl = [8, 7, 6, 5, 4, 3, 2, 1]
    conv = layer(kind=_lib.KIND_CONV3X3, H=2, Wd=2, C=16, M=4, K=144, act_params=FAKE,
                 colsums=FAKE)
    assert sched([layer(), conv], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_LAYOUT
    conv_lr = layer(kind=_lib.KIND_CONV3X3, H=2, Wd=2, C=16, M=4, K=144, lowrank_T=FAKE,
                    lowrank_up=FAKE, lowrank_rank=16)
    assert sched([layer(), conv_lr], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_LAYOUT
    assert sched([layer(lowrank_T=FAKE, lowrank_up=FAKE, lowrank_rank=32)] * 2, tbl, 4, 20,
                 0, 0) == _lib.TASQ_OK
    conv_wz = layer(kind=_lib.KIND_CONV3X3, H=2, Wd=2, C=16, M=4, K=144, w_zero=FAKE,
                    x_rowsums=FAKE)
    assert sched([layer(), conv_wz], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_LAYOUT
    assert sched([layer(w_zero=FAKE)], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_NULL
    assert sched([layer(), layer(act_params=FAKE)], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_NULL
    assert sched([layer(act_params=FAKE, colsums=FAKE + 2), layer()], tbl, 4, 20, 0, 1) \
        == _lib.TASQ_ERR_ALIGN
    assert sched([layer(act_params=FAKE, colsums=FAKE)] * 2, tbl, 4, 20, 0, 0) == _lib.TASQ_OK


def test_conv_rejects():
    def conv(**kw):
        a = dict(X=FAKE, W=FAKE, sx=1.0, sw=FAKE, bias=None, H=4, Wd=4, C=16, N=8, b=8,
                 acc=FAKE, y=FAKE)
        a.update(kw)
        return L.tasq_masked_conv3x3(a["X"], a["W"], a["sx"], a["sw"], a["bias"], a["H"],
                                     a["Wd"], a["C"], a["N"], a["b"], a["acc"], a["y"], None,
                                     None)
    assert conv(X=None) == _lib.TASQ_ERR_NULL
    assert conv(H=-1) == _lib.TASQ_ERR_DIM
    assert conv(b=0) == _lib.TASQ_ERR_BITS
    assert conv(C=14564) == _lib.TASQ_ERR_OVERFLOW          # 9 * C > 131071
    assert conv(H=0) == _lib.TASQ_OK
    assert conv(acc=None, y=None) == _lib.TASQ_ERR_NULL


def test_pack_planes_rejects():
    assert L.tasq_pack_planes(None, 4, 4, FAKE, None) == _lib.TASQ_ERR_NULL
    assert L.tasq_pack_planes(FAKE, 4, 4, None, None) == _lib.TASQ_ERR_NULL
    assert L.tasq_pack_planes(FAKE, -1, 4, FAKE, None) == _lib.TASQ_ERR_DIM
    assert L.tasq_pack_planes(FAKE, 0, 4, FAKE, None) == _lib.TASQ_OK


def layer(**kw):
    a = Layer()
    a.kind, a.M, a.N, a.K = _lib.KIND_LINEAR, 4, 4, 32
    a.sx = 0.02
    a.X = a.W = a.sw = a.acc = a.y = FAKE
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def sched(layers, table, S, T, t0, t1, o=None):
    arr = (Layer * len(layers))(*layers)
    tab = (ctypes.c_uint8 * max(1, len(table)))(*table)
    return L.tasq_run_schedule(arr, len(layers), tab, S, T, t0, t1,
                               ctypes.byref(o) if o is not None else None, None)


def test_schedule_rejects_before_launching():
    good = [layer(), layer()]
    tbl = [8, 7, 6, 5, 4, 3, 2, 1]
    assert sched(good, tbl, 4, 20, 0, 0) == _lib.TASQ_OK              # empty step range
    assert sched([], [], 4, 20, 0, 20) == _lib.TASQ_OK                 # no layers
    assert sched(good, tbl, 0, 20, 0, 20) == _lib.TASQ_ERR_RANGE
    assert sched(good, tbl, 5, 4, 0, 4) == _lib.TASQ_ERR_RANGE
    assert sched(good, tbl, 4, 20, 3, 2) == _lib.TASQ_ERR_RANGE
    assert sched(good, tbl, 4, 20, 0, 21) == _lib.TASQ_ERR_RANGE
    assert sched(good, tbl, 4, 20, -1, 2) == _lib.TASQ_ERR_RANGE
    # one bad table entry anywhere fails the whole call, whatever the range
    assert sched(good, [8, 7, 6, 5, 4, 3, 2, 0], 4, 20, 0, 1) == _lib.TASQ_ERR_BITS
    assert sched(good, [8, 7, 6, 5, 4, 9, 2, 1], 4, 20, 0, 1) == _lib.TASQ_ERR_BITS
    # a bad layer anywhere fails the whole call
    assert sched([layer(), layer(X=None)], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_NULL
    assert sched([layer(), layer(K=200000)], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_OVERFLOW
    assert sched([layer(kind=5), layer()], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_KIND
    bad_conv = layer(kind=_lib.KIND_CONV3X3, H=2, Wd=2, C=16, M=5, K=144)
    assert sched([bad_conv, layer()], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_DIM
    assert sched(good, tbl, 4, 20, 0, 1, opts(workspace=FAKE + 16, workspace_bytes=1 << 20)) \
        == _lib.TASQ_ERR_ALIGN
    # a layer without its row-major weight needs a packed copy
    assert sched([layer(), layer(W=None)], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_NULL
    assert sched([layer(), layer(W_packed=FAKE + 2)], tbl, 4, 20, 0, 1) == _lib.TASQ_ERR_ALIGN
    assert sched([layer(W=None, W_packed=FAKE)] * 2, tbl, 4, 20, 0, 0) == _lib.TASQ_OK
    assert L.tasq_run_schedule(None, 2, None, 4, 20, 0, 1, None, None) == _lib.TASQ_ERR_NULL
    assert L.tasq_run_schedule(None, -1, None, 4, 20, 0, 1, None, None) == _lib.TASQ_ERR_RANGE


def test_schedule_workspace_bytes_grows_with_layers():
    a = L.tasq_schedule_workspace_bytes((Layer * 1)(layer()), 1)
    b = L.tasq_schedule_workspace_bytes((Layer * 112)(*[layer()] * 112), 112)
    assert 0 < a <= b and a % 256 == 0 and b % 256 == 0


def test_schedule_workspace_bytes_holds_split_partials():
    """A schedule with a layer that split-K would cut (the UNet block's 3x3
    conv: K = 11520 on 20 tiles of 256x256) reserves that layer's int32
    partials after the layer list and the bit table; the 28-block DiT
    schedule (K <= 4608) reserves none."""
    lin = layer(M=4096, N=1920, K=640)
    conv = layer(kind=_lib.KIND_CONV3X3, H=32, Wd=32, C=1280, M=1024, N=1280, K=11520)
    base = L.tasq_schedule_workspace_bytes((Layer * 2)(lin, lin), 2)
    with_conv = L.tasq_schedule_workspace_bytes((Layer * 2)(lin, conv), 2)
    assert with_conv == base + L.tasq_workspace_bytes(1024, 1280, 11520)
    assert L.tasq_workspace_bytes(1024, 1280, 11520) == 10 * 1024 * 1280 * 4
    dit = [layer(M=8192, N=n, K=k) for k, n in [(1152, 3456), (1152, 1152), (1152, 4608),
                                                (4608, 1152)]] * 28
    assert L.tasq_schedule_workspace_bytes((Layer * 112)(*dit), 112) == \
        L.tasq_schedule_workspace_bytes((Layer * 112)(*[layer()] * 112), 112)


def test_probe_library_exports_its_header_and_stays_out_of_the_abi():
    """The benchmark's measurement probe is a library of its own: it exports
    what include/tasq_probe.h declares, libtasq.so exports none of it, and
    its argument checks fail before any launch."""
    text = open(os.path.join(ROOT, "include", "tasq_probe.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    syms = sorted(set(re.findall(r"\b(tasq_\w+)\s*\(", text)))
    assert syms == ["tasq_probe_mfma_chains", "tasq_probe_mfma_peak"]
    probe = ctypes.CDLL(os.path.join(ROOT, "paper_2608_03057_amd", "libtasq_probe.so"))
    for s in syms:
        assert hasattr(probe, s), s
        assert s not in _lib.EXPORTS and not hasattr(L, s), s
    probe.tasq_probe_mfma_peak.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                           ctypes.c_void_p]
    assert probe.tasq_probe_mfma_peak(0, 10, FAKE, None) == -1
    assert probe.tasq_probe_mfma_peak(4, 0, FAKE, None) == -1
    assert probe.tasq_probe_mfma_peak(4, 10, None, None) == -1
    assert probe.tasq_probe_mfma_chains() == 8


def test_struct_layouts_match_header(tmp_path):
    """The ctypes structs mirror tasq_opts and tasq_layer field by field: a C
    program compiled against include/tasq.h prints each field's offset and
    the struct sizes."""
    structs = {"tasq_opts": Opts, "tasq_layer": Layer, "tasq_act_job": _lib.ActJob,
               "tasq_weight_job": _lib.WeightJob}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "tasq.h"', "int main(void){"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    import subprocess
    subprocess.check_call(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src),
                           "-o", str(exe)])
    got = subprocess.check_output([str(exe)]).decode().split("\n")
    for line in filter(None, got):
        cname, field, val = line.split()
        py = structs[cname]
        want = ctypes.sizeof(py) if field == "size" else getattr(py, field).offset
        assert int(val) == want, (cname, field, int(val), want)


@pytest.mark.parametrize("kw", [dict(tile=-1), dict(tile=_lib.TILE_COUNT + 1),
                                dict(packed_tile=_lib.PTILE_COUNT + 1), dict(persistent=3),
                                dict(persistent=-1), dict(persistent_wgs=1025),
                                dict(persistent_parties=-2)])
def test_tuning_overrides_out_of_range(kw):
    assert lin(opts=opts(**kw)) == _lib.TASQ_ERR_RANGE
    assert sched([layer()], [8, 7, 6, 5], 4, 20, 0, 0, opts(**kw)) == _lib.TASQ_ERR_RANGE


def test_tuning_overrides_in_range_pass_validation():
    for kw in (dict(tile=_lib.TILE_COUNT), dict(packed_tile=1), dict(persistent=2),
               dict(persistent_wgs=1024, persistent_parties=4)):
        assert lin(M=0, opts=opts(**kw)) == _lib.TASQ_OK
        assert sched([layer()], [8, 7, 6, 5], 4, 20, 0, 0, opts(**kw)) == _lib.TASQ_OK


def test_schedule_ignores_split_k():
    """split_k is a single-call control: a schedule validates with any
    non-negative value (a long-K layer it launches on its own takes the
    automatic split), and rejects a negative one like every call."""
    tbl = [8, 7, 6, 5, 4, 3, 2, 1]
    conv = layer(kind=_lib.KIND_CONV3X3, H=32, Wd=32, C=1280, M=1024, N=1280, K=11520)
    for sk in (1, 2, 7, 16, 1000):
        assert sched([layer(), conv], tbl, 4, 20, 0, 0, opts(split_k=sk)) == _lib.TASQ_OK
    assert sched([layer(), conv], tbl, 4, 20, 0, 0, opts(split_k=-1)) == _lib.TASQ_ERR_RANGE


def test_auto_reads_planes_when_no_other_copy():
    """Under AUTO a linear layer may carry only the bit planes; a conv may
    not (the bit-plane kernels are linear-only)."""
    o = opts(W_planes=FAKE)
    assert lin(W=None, M=0, opts=o) == _lib.TASQ_OK
    assert lin(W=None, b=0, opts=o) == _lib.TASQ_ERR_BITS
    assert sched([layer(W=None, W_planes=FAKE)] * 2, [8, 7, 6, 5, 4, 3, 2, 1], 4, 20, 0, 0) \
        == _lib.TASQ_OK
    conv = layer(kind=_lib.KIND_CONV3X3, H=2, Wd=2, C=16, M=4, K=144, W=None, W_planes=FAKE)
    assert sched([conv], [8, 7, 6, 5], 4, 20, 0, 0) == _lib.TASQ_ERR_NULL
    assert lin(W=None, M=0, opts=opts(variant=_lib.VARIANT_MASKED_I8, W_planes=FAKE)) \
        == _lib.TASQ_ERR_NULL


def test_noalloc_schedule_rejects_before_touching_a_device():
    """tasq_run_schedule_noalloc validates like tasq_run_schedule and rejects
    more layers than its scratch array holds, before any HIP call."""
    def na(layers, table, S, T, t0, t1):
        arr = (Layer * len(layers))(*layers)
        tab = (ctypes.c_uint8 * max(1, len(table)))(*table)
        return L.tasq_run_schedule_noalloc(arr, len(layers), tab, S, T, t0, t1, None, None)
    L_max = _lib.TASQ_STATIC_MAX_LAYERS
    assert na([layer()] * (L_max + 1), [8] * (L_max + 1), 1, 1, 0, 1) == _lib.TASQ_ERR_WORKSPACE
    assert na([layer()] * 2, [8, 7, 6, 5, 4, 3, 2, 0], 4, 20, 0, 1) == _lib.TASQ_ERR_BITS
    assert na([layer()] * 2, [8] * 8, 4, 20, 3, 2) == _lib.TASQ_ERR_RANGE
    assert na([layer()] * 2, [8] * 8, 4, 20, 5, 5) == _lib.TASQ_OK
    assert _lib.TASQ_STATIC_SCRATCH_BYTES == 376832
