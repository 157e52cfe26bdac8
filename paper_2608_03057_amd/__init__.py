"""TASQ masked quantized linear layer on MI355X (gfx950).

Python face of the C ABI in ``include/tasq.h``: torch tensors in, device
pointers and the current HIP stream out to ``libtasq.so``.  Nothing here
computes; every operation is one call into the library.
"""
from __future__ import annotations

from .api import (  # noqa: F401
    masked_linear, masked_conv3x3, pack_planes, planes_bytes, pack_weights, packed_weight_bytes,
    quantize_activations, quantize_activations_batch, quantize_activations_lowrank,
    lowrank_down, weight_colsums,
    quantize_weights, quantize_weights_batch, row_sums, schedule_cost,
    stage_of_step, run_schedule, run_schedule_noalloc, schedule_workspace_bytes,
    workspace_bytes, make_layer, status_string,
)
from ._lib import (  # noqa: F401
    TasqError, VARIANT_AUTO, VARIANT_MASKED_I8, VARIANT_BITPLANE, VARIANT_PACKED, KIND_LINEAR,
    KIND_CONV3X3, TASQ_ACT_PARAMS_FLOATS,
)
