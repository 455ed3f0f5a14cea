"""Wrong readings of Eq. 4 (Sec. 4.1), for the negative controls.

A perturbed copy of the oracle's context construction: each mutation is a
plausible mistake in reading the method or in implementing it, planted here
on the CPU so that the tests can show the parity tolerances reject it.  The
mutants use the oracle's own grids, window layout, pooling and attention
wherever the mistake does not touch them.

  dropped_sink    the sink frames left out of every context
  pooled_sink     the sink resampled to the query scale like history
  pad_count_mean  a ragged block's mean divided by f*f instead of the
                  number of cells it holds
  floor_grid      pooled frames on the floor grid (the partial blocks at a
                  ragged edge dropped)
  upsampled_keys  window frames coarser than the query repeated up to the
                  query's grid instead of kept at their own scale
  causal_window   a query state attends only to window states up to its own
"""

import numpy as np

import oracle

MUTATIONS = ("dropped_sink", "pooled_sink", "pad_count_mean", "floor_grid", "upsampled_keys",
             "causal_window")


def _pool(x, gh, gw, f, mutation):
    """oracle.pool_frame (block mean) with the pooling mistakes."""
    if f == 1 or mutation not in ("pad_count_mean", "floor_grid"):
        return oracle.pool_frame(x, gh, gw, f)
    x = np.asarray(x, dtype=np.float64)
    img = x.reshape(gh, gw, *x.shape[1:])
    if mutation == "floor_grid":
        oh, ow = gh // f, gw // f
    else:
        oh, ow = -(-gh // f), -(-gw // f)
    out = np.zeros((oh, ow) + x.shape[1:], dtype=np.float64)
    for Y in range(oh):
        for X in range(ow):
            block = img[f * Y: f * Y + f, f * X: f * X + f]
            out[Y, X] = block.reshape(-1, *x.shape[1:]).sum(axis=0) / (f * f)
    return out.reshape(oh * ow, *x.shape[1:])


def _upsample(x, gh, gw, r, ogh, ogw):
    """Nearest repeat of a frame on grid (gh, gw) by r, cropped to (ogh, ogw)."""
    img = np.asarray(x, dtype=np.float64).reshape(gh, gw, *x.shape[1:])
    up = np.repeat(np.repeat(img, r, axis=0), r, axis=1)[:ogh, :ogw]
    return up.reshape(ogh * ogw, *x.shape[1:])


def context(desc, s, q_state, x_sink, x_hist, x_win, mutation):
    """K (or V) context of queries at scale s in window state q_state (0-based)
    under `mutation`."""
    parts = []
    n1 = oracle.frame_tokens(desc, 1)
    gh1, gw1 = oracle.grid(desc, 1)
    for f in range(int(desc["sink_frames"])):
        sink = np.asarray(x_sink[f * n1: (f + 1) * n1], dtype=np.float64)
        if mutation == "dropped_sink":
            continue
        parts.append(_pool(sink, gh1, gw1, s, None) if mutation == "pooled_sink" else sink)
    for f in range(int(desc["hist_frames"])):
        parts.append(_pool(x_hist[f * n1: (f + 1) * n1], gh1, gw1, s, mutation))
    for (w, b, p, first, n) in oracle.window_frames(desc):
        if mutation == "causal_window" and b > q_state:
            continue
        gh, gw = oracle.grid(desc, p)
        x = x_win[first: first + n]
        if p >= s:
            if mutation == "upsampled_keys" and p > s:
                parts.append(_upsample(x, gh, gw, p // s, *oracle.grid(desc, s)))
            else:
                parts.append(np.asarray(x, dtype=np.float64))
        else:
            parts.append(_pool(x, gh, gw, s // p, mutation))
    return np.concatenate(parts, axis=0)


def attention(desc, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, rows, mutation):
    """MSSA output [len(rows), heads, head_dim] of the sampled query rows
    under `mutation`, float64."""
    nh, d = int(desc["num_heads"]), int(desc["head_dim"])
    scale = oracle.softmax_scale(desc)
    rows = np.asarray(rows)
    state_of = np.empty(oracle.num_window_tokens(desc), dtype=np.int64)
    scale_of = np.empty_like(state_of)
    for (_, b, p, first, n) in oracle.window_frames(desc):
        state_of[first: first + n] = b
        scale_of[first: first + n] = p
    out = np.empty((len(rows), nh, d), dtype=np.float64)
    keys = sorted({(int(scale_of[r]), int(state_of[r]) if mutation == "causal_window" else -1) for r in rows})
    for (s, qs) in keys:
        sel = np.nonzero((scale_of[rows] == s) & ((state_of[rows] == qs) if qs >= 0 else True))[0]
        for h in range(nh):
            def hd(x):
                return np.zeros((0, d)) if x is None else np.asarray(x[:, h], dtype=np.float64)
            kc = context(desc, s, qs, hd(k_sink), hd(k_hist), hd(k_win), mutation)
            vc = context(desc, s, qs, hd(v_sink), hd(v_hist), hd(v_win), mutation)
            out[sel, h] = oracle.attention(np.asarray(q_win[rows[sel], h], dtype=np.float64), kc, vc, scale)
    return out
