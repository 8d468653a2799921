"""Row-typed associative-algebra projections (Y = X *_q W) on MI355X.

The computation lives in ``libstarq.so`` (hand-written gfx950 HIP kernels
behind the C ABI of ``include/star_proj.h``); ``binding`` is its thin ctypes
binding.  The binding is loaded on first use of any entry point and raises
ImportError if the library has not been built
(``python -m paper_2609_32814_amd.build``); there is no fallback path.
"""

_EXPORTS = (
    "LIB_PATH", "Algebra", "StarError",
    "star_count_macs", "star_count_products", "star_decode", "star_ffn_bwd", "star_ffn_fwd",
    "star_plan_bytes", "star_proj_bwd_data", "star_proj_bwd_data_planned",
    "star_proj_bwd_weight", "star_proj_bwd_weight_planned", "star_proj_fwd",
    "star_proj_fwd_planned", "star_status_string", "star_type_plan", "star_validate_types",
    "star_workspace_bytes", "star_swiglu_fwd", "star_swiglu_bwd", "star_add", "star_swiglu_ffn_fwd",
    "star_swiglu_ffn_bwd", "star_decode_gated", "star_decode_status", "star_decode_noalloc",
    "AttnShape", "star_attn_fwd", "star_attn_decode", "star_attn_decode_workspace_bytes",
    "star_set_fwd_tiles", "star_swiglu_merged_fwd", "star_swiglu_up_fwd_planned", "pack_gate_up",
)

__all__ = list(_EXPORTS)


def __getattr__(name):
    if name in _EXPORTS:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
