"""Plain fp64 CPU oracle for Flash Swin attention (HRSAM, arXiv 2407.02109, Sec. 3.3-3.4, App. A-B).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import this package.
The GPU library never imports it and shares no code, table or helper with it.

Every function here is a slow, obviously-correct restatement of the paper's
definitions in float64 NumPy; see ``swin_oracle`` for the four single-grid forms,
``multiscale`` for the multi-scale (several grids in one sequence) forms of App. C and
``backward`` for the gradients (dq, dk, dv) and the log-sum-exp a training forward keeps,
``rope`` for 2-D rotary position embedding of q and k ahead of the attention, and
``cycle_scan`` for the Cycle-scan module's selective state-space scan (Sec. 3.5).
"""
from .swin_oracle import (  # noqa: F401
    PAD_MASK,
    PAD_KVTOKEN,
    swin_attention_textbook,
    swin_attention_canvas,
    swin_attention_fla,
    swin_attention_bruteforce,
    swin_attention_at,
    fla_shift_window_indices,
    fla_kv_padding_indices,
    window_sizes,
    work_counts,
)
from .backward import (  # noqa: F401
    swin_attention_bwd,
    swin_attention_lse,
    swin_attention_ms_bwd,
    swin_attention_ms_lse,
)
from .rope import (  # noqa: F401
    apply_rope,
    rope_angles,
    swin_attention_rope,
    swin_attention_rope_at,
    swin_attention_rope_bwd,
    swin_attention_rope_lse,
)
from .multiscale import (  # noqa: F401
    grid_offsets,
    ms_kv_padding_indices,
    ms_shift_window_indices,
    ms_work_counts,
    swin_attention_ms,
    swin_attention_ms_at,
    swin_attention_ms_fla,
)
from . import cycle_scan  # noqa: F401  (the module: cycle_scan.cycle_scan, .selective_scan, .zoh)
