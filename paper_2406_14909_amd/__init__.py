"""MI355X (gfx950) Mixture-of-Attention-Spans attention: HIP kernels behind a C ABI.

The binding lives in :mod:`paper_2406_14909_amd.moa`; the library is built by
:mod:`paper_2406_14909_amd.build`.
"""
from .moa import (MOA_BAND_BLOCK, MOA_BLOCK_BAND, MOA_SPAN_INCLUDES_SINKS, MoaError, Plan,
                  load_library, moa_decode, moa_decode_ragged, moa_influence, moa_rule_loss,
                  moa_decode_workspace_bytes, moa_kv_append, moa_kv_append_ragged, moa_plan,
                  moa_prefill, new_cache, new_workspace)

__all__ = [
    "MOA_BAND_BLOCK", "MOA_BLOCK_BAND", "MOA_SPAN_INCLUDES_SINKS", "MoaError", "Plan", "load_library", "moa_decode", "moa_decode_ragged", "moa_influence", "moa_rule_loss",
    "moa_decode_workspace_bytes", "moa_kv_append", "moa_kv_append_ragged", "moa_plan",
    "moa_prefill", "new_cache", "new_workspace",
]
