"""Flash Swin attention (and HRSAM's Cycle-scan) for AMD MI355X (gfx950).

The compute lives in the HIP library ``libfla_swin.so`` built from ``csrc/``; this
package only marshals arguments to its C ABI (see ``binding``).  Importing the package
does not load the library; the first call does, and fails loudly if it is missing.
"""
from .binding import (  # noqa: F401
    FLA_PAD_MASK,
    FLA_PAD_KVTOKEN,
    FlaError,
    fla_swin_attn_fwd,
    fla_swin_attn_fwd_f32,
    fla_status_string,
    fla_swin_attn_work,
    fla_swin_attn_ms_fwd,
    fla_swin_attn_ms_fwd_f32,
    fla_swin_attn_ms_work,
    fla_swin_attn_fwd_lse,
    fla_swin_attn_ms_fwd_lse,
    fla_swin_attn_bwd_workspace,
    fla_swin_attn_bwd,
    fla_swin_attn_ms_bwd,
    fla_swin_attn_bwd_work,
    swin_attn,
    swin_attn_ms,
    swin_attn_fwd_train,
    fla_swin_attn_rope_fwd,
    fla_swin_attn_rope_fwd_lse,
    fla_swin_attn_rope_bwd,
    swin_attn_rope,
    swin_attn_bwd,
    swin_attn_rope_fwd_train,
    swin_attn_rope_bwd,
    swin_attention,
    fla_cycle_scan,
    fla_cycle_scan_workspace,
    fla_cycle_scan_work,
    cycle_scan,
    library_path,
    load_library,
)
