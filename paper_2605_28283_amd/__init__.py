"""PrunePath sparse-FFN forward for MI355X (gfx950).

The computation runs in the HIP library libprunepath.so (C ABI in
include/prunepath.h); this package is its thin Python binding plus the seeded
synthetic-input generators (``workloads``).
"""
from ._lib import (EXPORTED, PP_AGG_SIGMOID, PP_AGG_SUM, PP_EHIP, PP_EINVAL, PP_ENOMEM,  # noqa: F401
                   PP_ENOTCONVERGED, prunepath_balanced_kmeans, prunepath_kmeans_workspace,
                   PP_EUNSUPPORTED, PP_KERNEL_COUNT, PP_KERNEL_DISPATCH, PP_KERNEL_DOWN,
                   PP_KERNEL_GATEUP, PP_KERNEL_ROUTE, PP_OK, PP_SELECT_LTE, PP_SELECT_NUCLEUS,
                   PP_SELECT_STRICT, PP_SELECT_TOPK, PrunePathError, load, prunepath_create,
                   prunepath_create_mlp,
                   prunepath_destroy, prunepath_ffn_decode, prunepath_ffn_prefill,
                   prunepath_profile_begin, prunepath_profile_end, prunepath_residual_rmsnorm,
                   prunepath_route, prunepath_router_loss, prunepath_router_loss_noalloc,
                   prunepath_router_loss_workspace,
                   prunepath_status_string)
