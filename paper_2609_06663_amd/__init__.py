"""ECOKV prefill-time KV-cache eviction pass on AMD MI355X (gfx950).

The product is ``libecokv.so`` (C ABI in ``include/ecokv.h``); ``ecokv`` is
its thin Python binding.  ``pipeline`` strings the three calls together for
torch tensors.
"""
from .ecokv import (  # noqa: F401
    BF16, F32, PER_HEAD, LAYER_FLAT, HEAD_BUDGETS, IMP_ATTN, IMP_ATTN_VNORM, NORM_MINMAX, NORM_WINSOR, NORM_MAD,
    RED_EUCLID, RED_STD, CENTROID_ALL, CENTROID_PREFIX, NSTATS, STAT, EcoKVError, Params, Shape,
    ecokv_compact, ecokv_decode, ecokv_decode_workspace_size, ecokv_default_params, ecokv_index_count, ecokv_index_count_mode, ecokv_last_error,
    ecokv_prefill_workspace_size, ecokv_prefill_write, ecokv_pyramid_budgets, ecokv_score, ecokv_score_noalloc, ecokv_score_pre, ecokv_score_v, ecokv_select, ecokv_select_workspace_size, ecokv_stage_times, ecokv_workspace_size,
    ecokv_workspace_status, OK, EINVAL, EWORKSPACE, EUNSUPPORTED, EHIP, ETIMEOUT,
)
