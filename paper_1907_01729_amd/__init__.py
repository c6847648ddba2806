"""Batched log-domain Sinkhorn on MI355X (gfx950): Python binding of the C ABI.

Viehmann, "Implementation of batched Sinkhorn iterations for
entropy-regularized Wasserstein loss" (arXiv:1907.01729).

Every step of the computation runs in the HIP library ``libsinkhorn_hip.so``
(see ``include/sinkhorn.h``); this package only marshals arguments: it checks
tensor shapes, allocates outputs and the workspace with PyTorch on the GPU and
passes raw device pointers and the current HIP stream.  There is no CPU
fallback -- without the built library every call raises.
"""
from ._binding import (  # noqa: F401
    NOALLOC_SCRATCH_BYTES,
    SinkhornError,
    library_path,
    load_library,
    sinkhorn_backward,
    sinkhorn_backward_points,
    sinkhorn_backward_sharp,
    sinkhorn_forward,
    sinkhorn_forward_noalloc,
    sinkhorn_forward_points,
    sinkhorn_forward_select,
    sinkhorn_points_workspace_bytes,
    sinkhorn_regime,
    sinkhorn_describe,
    sinkhorn_sharp_workspace_bytes,
    sinkhorn_status_string,
    sinkhorn_workspace_bytes,
)
from .loss import SinkhornLoss, SinkhornPointsLoss, sinkhorn_loss, sinkhorn_loss_points  # noqa: F401

__all__ = [
    "NOALLOC_SCRATCH_BYTES",
    "SinkhornError",
    "SinkhornLoss",
    "SinkhornPointsLoss",
    "library_path",
    "load_library",
    "sinkhorn_backward",
    "sinkhorn_backward_points",
    "sinkhorn_backward_sharp",
    "sinkhorn_forward",
    "sinkhorn_forward_noalloc",
    "sinkhorn_forward_points",
    "sinkhorn_forward_select",
    "sinkhorn_loss",
    "sinkhorn_loss_points",
    "sinkhorn_points_workspace_bytes",
    "sinkhorn_regime",
    "sinkhorn_describe",
    "sinkhorn_sharp_workspace_bytes",
    "sinkhorn_status_string",
    "sinkhorn_workspace_bytes",
]
