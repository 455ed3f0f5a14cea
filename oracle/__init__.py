"""fp64 CPU oracle for MSSA (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU library never imports it, and it imports
nothing from the library.
"""
from .mssa_oracle import (  # noqa: F401
    KIND_HIST, KIND_SINK, KIND_WIN, algorithmic_flops, attention,
    brute_force_attention, context, context_rows, frame_tokens, grid,
    mssa_attention, num_hist_tokens, num_sink_tokens, num_window_tokens,
    pool_frame, pooled_kv, query_groups, resample_mode, scales_in_use, softmax_scale, tables,
    window_frames,
)
from .mssa_backward import attention_backward, mssa_backward, pool_frame_adjoint  # noqa: F401,E402
from .mssa_tiers import patch_embed, patch_unembed, patchify, qkv_project, unpatchify  # noqa: F401,E402
