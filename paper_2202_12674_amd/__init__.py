"""MI355X-native LS-SVM training hot path (PLSSVM, arXiv 2202.12674).

The reduced LS-SVM system of Sec. II-F is solved by conjugate gradients
(Sec. III-B) with the implicit reduced-matrix product of Eq. (16) on the
gfx950 matrix cores. The public entry points wrap the C ABI of
include/lssvm.h; PyTorch supplies device memory and streams only.
"""
from ._binding import (F32, F64, LINEAR, POLY, RBF, LssvmError, TrainResult,  # noqa: F401
                       alloc_workspace, cg_step, cg_step_noalloc, host_contexts, last_error, lib,
                       matvec, mfma_peak, predict, predict_workspace_bytes, tile_plan, train,
                       workspace_bytes)
from .build import LIB_PATH  # noqa: F401

__all__ = ["train", "predict", "matvec", "cg_step", "cg_step_noalloc", "mfma_peak",
           "workspace_bytes", "predict_workspace_bytes", "alloc_workspace", "host_contexts",
           "tile_plan",
           "LssvmError", "TrainResult", "lib", "last_error"]
