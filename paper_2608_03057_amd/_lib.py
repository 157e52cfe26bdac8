"""ctypes binding of libtasq.so (the C ABI in include/tasq.h).

Argument marshalling only: every step of the masked linear runs in the HIP
kernels behind the C ABI.  The library must have been built
(``python -m paper_2608_03057_amd.build`` or ``__graft_entry__.build()``);
there is no fallback, and a missing library raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtasq.so")

TASQ_OK = 0
TASQ_ERR_NULL = -1
TASQ_ERR_DIM = -2
TASQ_ERR_BITS = -3
TASQ_ERR_OVERFLOW = -4
TASQ_ERR_RANGE = -5
TASQ_ERR_LAYOUT = -6
TASQ_ERR_WORKSPACE = -7
TASQ_ERR_HIP = -8
TASQ_ERR_KIND = -9
TASQ_ERR_ALIGN = -10
TASQ_MAX_K = 131071
TASQ_ACT_PARAMS_FLOATS = 1028
TASQ_STATIC_MAX_LAYERS = 256
TASQ_STATIC_SCRATCH_BYTES = 376832

VARIANT_AUTO = 0
VARIANT_MASKED_I8 = 1
VARIANT_BITPLANE = 2
VARIANT_PACKED = 3

KIND_LINEAR = 0
KIND_CONV3X3 = 1

# Every exported symbol the header declares.
EXPORTS = (
    "tasq_masked_linear", "tasq_masked_conv3x3", "tasq_pack_planes", "tasq_planes_bytes",
    "tasq_pack_weights", "tasq_packed_weight_bytes", "tasq_quantize_activations",
    "tasq_quantize_activations_batch", "tasq_quantize_weights_batch",
    "tasq_weight_colsums", "tasq_lowrank_down", "tasq_quantize_activations_lowrank",
    "tasq_quantize_weights", "tasq_row_sums", "tasq_schedule_cost",
    "tasq_stage_of_step", "tasq_run_schedule", "tasq_run_schedule_noalloc",
    "tasq_workspace_bytes", "tasq_schedule_workspace_bytes", "tasq_status_string",
)


class Opts(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int32), ("split_k", ctypes.c_int32),
                ("W_planes", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t), ("W_packed", ctypes.c_void_p),
                ("act_params", ctypes.c_void_p), ("colsums", ctypes.c_void_p),
                ("lowrank_T", ctypes.c_void_p), ("lowrank_up", ctypes.c_void_p),
                ("lowrank_rank", ctypes.c_int32), ("w_zero", ctypes.c_void_p),
                ("x_rowsums", ctypes.c_void_p), ("tile", ctypes.c_int32),
                ("packed_tile", ctypes.c_int32), ("persistent", ctypes.c_int32),
                ("persistent_wgs", ctypes.c_int32), ("persistent_parties", ctypes.c_int32),
                ("step_events", ctypes.POINTER(ctypes.c_void_p))]


# Tuning overrides of tasq_opts (sweeps and tests): staged and packed tile ids.
TILE_COUNT = 6
PTILE_COUNT = 7
TUNING_FIELDS = ("tile", "packed_tile", "persistent", "persistent_wgs", "persistent_parties")


class Cost(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("macs", "b_eff", "b_mean", "bitops", "rel_bitops",
                                               "rel_cycles_measured", "rel_cycles_as_a4")]


class Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("M", ctypes.c_int32), ("N", ctypes.c_int32),
                ("K", ctypes.c_int32), ("H", ctypes.c_int32), ("Wd", ctypes.c_int32),
                ("C", ctypes.c_int32), ("sx", ctypes.c_float),
                ("X", ctypes.c_void_p), ("W", ctypes.c_void_p), ("W_planes", ctypes.c_void_p),
                ("sw", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("acc", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("W_packed", ctypes.c_void_p),
                ("act_params", ctypes.c_void_p), ("colsums", ctypes.c_void_p),
                ("lowrank_T", ctypes.c_void_p), ("lowrank_up", ctypes.c_void_p),
                ("lowrank_rank", ctypes.c_int32), ("w_zero", ctypes.c_void_p),
                ("x_rowsums", ctypes.c_void_p)]


class ActJob(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("M", ctypes.c_int32), ("K", ctypes.c_int32),
                ("X_out", ctypes.c_void_p), ("act_params", ctypes.c_void_p)]


class WeightJob(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("N", ctypes.c_int32), ("K", ctypes.c_int32),
                ("W_out", ctypes.c_void_p), ("alpha_out", ctypes.c_void_p),
                ("z_out", ctypes.c_void_p), ("sw_out", ctypes.c_void_p)]


class TasqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2608_03057_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
        L.tasq_masked_linear.argtypes = [vp, vp, f32, vp, vp, i32, i32, i32, i32, vp, vp,
                                         ctypes.POINTER(Opts), vp]
        L.tasq_masked_linear.restype = i32
        L.tasq_masked_conv3x3.argtypes = [vp, vp, f32, vp, vp, i32, i32, i32, i32, i32, vp, vp,
                                          ctypes.POINTER(Opts), vp]
        L.tasq_masked_conv3x3.restype = i32
        L.tasq_pack_planes.argtypes = [vp, i32, i32, vp, vp]
        L.tasq_pack_planes.restype = i32
        L.tasq_planes_bytes.argtypes = [i32, i32]
        L.tasq_planes_bytes.restype = ctypes.c_size_t
        L.tasq_pack_weights.argtypes = [vp, i32, i32, vp, vp]
        L.tasq_pack_weights.restype = i32
        L.tasq_packed_weight_bytes.argtypes = [i32, i32]
        L.tasq_packed_weight_bytes.restype = ctypes.c_size_t
        L.tasq_quantize_activations.argtypes = [vp, i32, i32, vp, vp, vp]
        L.tasq_quantize_activations.restype = i32
        L.tasq_quantize_activations_batch.argtypes = [ctypes.POINTER(ActJob), i32, vp]
        L.tasq_quantize_activations_batch.restype = i32
        L.tasq_quantize_weights_batch.argtypes = [ctypes.POINTER(WeightJob), i32, vp]
        L.tasq_quantize_weights_batch.restype = i32
        L.tasq_weight_colsums.argtypes = [vp, i32, i32, vp, vp]
        L.tasq_weight_colsums.restype = i32
        L.tasq_schedule_cost.argtypes = [vp, i32, vp, i32, i32, i32, i32, i32, vp]
        L.tasq_schedule_cost.restype = i32
        L.tasq_quantize_weights.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp]
        L.tasq_quantize_weights.restype = i32
        L.tasq_row_sums.argtypes = [vp, i32, i32, vp, vp]
        L.tasq_row_sums.restype = i32
        L.tasq_lowrank_down.argtypes = [vp, i32, i32, vp, i32, vp, vp]
        L.tasq_lowrank_down.restype = i32
        L.tasq_quantize_activations_lowrank.argtypes = [vp, i32, i32, vp, vp, vp, i32, vp, vp]
        L.tasq_quantize_activations_lowrank.restype = i32
        L.tasq_stage_of_step.argtypes = [i32, i32, i32]
        L.tasq_stage_of_step.restype = i32
        L.tasq_run_schedule.argtypes = [ctypes.POINTER(Layer), i32, vp, i32, i32, i32, i32,
                                        ctypes.POINTER(Opts), vp]
        L.tasq_run_schedule.restype = i32
        L.tasq_run_schedule_noalloc.argtypes = L.tasq_run_schedule.argtypes
        L.tasq_run_schedule_noalloc.restype = i32
        L.tasq_workspace_bytes.argtypes = [i32, i32, i32]
        L.tasq_workspace_bytes.restype = ctypes.c_size_t
        L.tasq_schedule_workspace_bytes.argtypes = [ctypes.POINTER(Layer), i32]
        L.tasq_schedule_workspace_bytes.restype = ctypes.c_size_t
        L.tasq_status_string.argtypes = [i32]
        L.tasq_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().tasq_status_string(status).decode()


def check(status: int, where: str) -> None:
    if status != TASQ_OK:
        raise TasqError(status, where)
