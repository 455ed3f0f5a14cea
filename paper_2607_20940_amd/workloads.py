"""The synthetic MSSA workloads (plain data).

Each entry holds a plan descriptor (the fields of ``mssa_plan_desc``), the
input dtype, the seed and the amplitude of the Gaussian inputs.  Shapes
follow Wan2.1-style DiT layers: the paper's model is Wan2.1-T2V-1.3B at
832x480 (a 30x52 latent token grid), with T = 5 window states of 3 latent
frames (Sec. 5.1) and the schedule (p, p, 2p, 2p, 2p) (Sec. 4.1).
"""

import math

_AMP = 1.0 / math.sqrt(128.0)

WORKLOADS = {
    # 1 head x 64, 8x8 grid, 1 sink frame, no history, 2 states of 1 frame.
    "tiny_f32": dict(
        desc=dict(num_states=2, scales=[1, 2], grid_h=8, grid_w=8, frames_per_state=1,
                  sink_frames=1, hist_frames=0, num_heads=1, head_dim=64),
        dtype="f32", seed=0, amplitude=1.0),
    # Wan-1.3B-shaped layer: 12 x 128, 30x52 grid, 3 sink, 6 history, 5 x 3 window.
    "wan13b_layer": dict(
        desc=dict(num_states=5, scales=[1, 1, 2, 2, 2], grid_h=30, grid_w=52,
                  frames_per_state=3, sink_frames=3, hist_frames=6, num_heads=12,
                  head_dim=128),
        dtype="bf16", seed=1, amplitude=_AMP),
    # Long history (21 frames) and a three-level schedule with ragged 4x pooling.
    "wan13b_longhist": dict(
        desc=dict(num_states=5, scales=[1, 1, 2, 2, 4], grid_h=30, grid_w=52,
                  frames_per_state=3, sink_frames=3, hist_frames=21, num_heads=12,
                  head_dim=128),
        dtype="bf16", seed=2, amplitude=_AMP),
    # Wan-14B-shaped 720p layer: 40 x 128, 45x80 grid (ragged at 2x and 4x).
    "wan14b_720p": dict(
        desc=dict(num_states=5, scales=[1, 1, 2, 2, 4], grid_h=45, grid_w=80,
                  frames_per_state=3, sink_frames=3, hist_frames=9, num_heads=40,
                  head_dim=128),
        dtype="bf16", seed=3, amplitude=_AMP),
}

# Steady-state streaming: 30 stacked layers of the Wan-1.3B shape over 64
# rolling passes.  Each pass moves the emitted head state (3 native frames)
# into a history FIFO capped at 21 frames (starting from 6 frames), and a
# fresh N(0,1) window enters.  Seeds: the window Q/K/V of pass p are drawn,
# layer by layer (q, k, v each), from one generator seeded seed_base + p;
# the sink and initial history of layer L from a generator seeded
# init_seed_base + L.
STREAMING = dict(
    layer=WORKLOADS["wan13b_layer"]["desc"], layers=30, passes=64,
    hist_start_frames=6, hist_cap_frames=21, dtype="bf16", seed_base=4,
    init_seed_base=4_001_000, amplitude=1.0)


def input_shapes(desc, n_q, n_sink, n_hist):
    """Shapes of the seven inputs given token counts (from a plan)."""
    nh, d = int(desc["num_heads"]), int(desc["head_dim"])
    return {
        "q_win": (n_q, nh, d), "k_win": (n_q, nh, d), "v_win": (n_q, nh, d),
        "k_sink": (n_sink, nh, d), "v_sink": (n_sink, nh, d),
        "k_hist": (n_hist, nh, d), "v_hist": (n_hist, nh, d),
    }
