"""MonarchAttention forward pass (and its gradient) on MI355X (gfx950): HIP kernels behind a C ABI.

The C ABI is declared in include/monarch_attn.h; this package is its thin
Python binding (ctypes, with torch used only for device memory and streams).
If libmonarch_attn.so has not been built, importing the package still works
(so that ``paper_2505_18698_amd.build`` can run) but every binding attribute
raises the ImportError: there is no fallback path.
"""
try:
    from ._binding import (  # noqa: F401
        EXPORTS,
        KIND_NAMES,
        LIB,
        LIB_PATH,
        MAX_T_16BIT,
        MAX_T_16BIT_BWD,
        NOALLOC_SCRATCH_BYTES,
        MA_BF16,
        MA_EHIP,
        MA_EINVAL,
        MA_ENOMEM,
        MA_EUNSUPPORTED,
        MA_F16,
        MA_F32,
        MA_OK,
        PATH_AUTO,
        PATH_HALF_STEPS,
        PATH_FUSED,
        PATH_GROUPED,
        MonarchAttnError,
        dtype_code,
        fused_applies,
        grouped_applies,
        monarch_attention,
        monarch_attention_autograd,
        monarch_attn_bwd,
        monarch_attn_bwd_varlen,
        monarch_attn_bwd_check,
        monarch_attn_bwd_workspace_bytes,
        monarch_attn_build_id,
        monarch_attn_check,
        monarch_attn_fwd,
        monarch_attn_fwd_noalloc,
        monarch_attn_fwd_objective,
        monarch_attn_fwd_prepad,
        monarch_attn_fwd_varlen,
        monarch_attn_exact_fwd,
        monarch_attn_fwd_raw,
        monarch_attn_last_error,
        monarch_attn_release_workspace,
        monarch_attn_set_path,
        monarch_attn_timing_enable,
        monarch_attn_timing_read,
        monarch_attn_workspace_bytes,
    )
except ImportError as _err:  # library not built
    _missing = _err

    def __getattr__(name):
        if name.startswith("__"):
            raise AttributeError(name)
        raise ImportError(str(_missing))
