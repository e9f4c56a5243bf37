"""K-Forcing batched joint next-k-token decode on MI355X (gfx950).

The compute path lives in libkforcing.so (hand-written HIP kernels behind the
C ABI of include/kforcing.h).  This package is its thin Python binding:
argument marshalling only.  PyTorch supplies device memory and the stream.
"""
from .binding import (  # noqa: F401
    KF_BF16, KF_EHIP, KF_ECTX, KF_EINVAL, KF_ENOMEM, KF_ESTATE, KF_FLAG_DEBUG_LOGITS, KF_FP32,
    KF_KC_NAMES, KF_MASK_DOUBLE, KF_MASK_SINGLE, KF_OK, KfConfig, KfError, KForcing, lib,
    lib_path, training_attention, training_attention_shapes,
)
