"""fp64 CPU oracle for Multi-Scale Self-Attention (MSSA) over a Multi-Scale
Patchification (MSP) rolling window.

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that the
GPU library is checked against.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the library itself never does, and
this module imports nothing from the library.  It shares no code, tables or
constants with the HIP path.

What is computed (Ms. Forcing, Sec. 4.1):

* MSP token grids (Eq. 3): a latent frame of H x W native tokens tokenized at
  patch scale s (a multiple of the native patch) has a ceil(H/s) x ceil(W/s)
  grid.  Eq. 3 writes HW/p_l^2, which is the divisible case; the ceil grid is
  the reading used when s does not divide H or W.
* The rolling window (Sec. 3.1, Eq. 2) holds T states; state l (1-based) has
  patch scale p_l, nondecreasing in l, and F latent frames.  Window tokens are
  ordered by (state, frame, row, col); queries of one scale form a contiguous
  group because the schedule is nondecreasing.
* MSSA context (Eq. 4): queries at scale s attend to
  [sink at native density || every visible non-sink frame resampled with
  stride max(1, s / p_b)].  The sink is never resampled (Sec. 4.1).  The
  visible set is every history frame and every window state, the query's own
  state included: the window attends bidirectionally (Sec. 3.1) and MSSA keeps
  the original attention mask (Fig. 3 caption).  A frame coarser than the
  query keeps its own scale (stride is at least 1, never an upsampling).
* "Subsample" is read as a 2-D spatial average pool over each f x f block of
  the frame's own grid, f = max(1, s / p_b), averaging only the cells that
  exist on a ragged edge (Sec. 3.2 uses the 2 x 2 block mean as the
  coarse-token proxy).  The literal strided reading of Eq. 4 (and of the
  stride-2 probe of Sec. 3.2) is the variant resample="stride": each f x f
  block is represented by its first (top-left) cell, i.e. rows and columns
  0, f, 2f, ... of the frame's grid, which on a ragged grid also gives the
  ceil(gh/f) x ceil(gw/f) grid.
* Attention: softmax(scale * q k^T) v over the whole context, per head, no
  mask inside the context, no bias for pooled tokens.

Nothing here is blocked, fused or reordered beyond these definitions.  All
arithmetic is float64 on the exact input values the GPU receives.

A descriptor is a mapping with the keys
    num_states, scales, grid_h, grid_w, frames_per_state, sink_frames,
    hist_frames, num_heads, head_dim, softmax_scale (optional, <= 0 or absent
    means 1/sqrt(head_dim)), resample (optional, "mean" (default) or
    "stride").
Tensors are token-major arrays [tokens, heads, head_dim].
"""

import math

import numpy as np

# Kind codes of context segment rows.
KIND_SINK = 0
KIND_HIST = 1
KIND_WIN = 2


def _ceil_div(a, b):
    return -(-a // b)


def _scales(desc):
    return [int(s) for s in desc["scales"][: int(desc["num_states"])]]


def resample_mode(desc):
    """How a frame is brought to a coarser scale: "mean" (block average) or
    "stride" (first cell of each block)."""
    m = desc.get("resample", "mean")
    if m not in ("mean", "stride"):
        raise ValueError("resample must be 'mean' or 'stride'")
    return m


def softmax_scale(desc):
    s = float(desc.get("softmax_scale", 0.0) or 0.0)
    return s if s > 0.0 else 1.0 / math.sqrt(int(desc["head_dim"]))


def grid(desc, s):
    """Token grid of one latent frame patchified at scale s (Eq. 3, ceil)."""
    return _ceil_div(int(desc["grid_h"]), s), _ceil_div(int(desc["grid_w"]), s)


def frame_tokens(desc, s):
    gh, gw = grid(desc, s)
    return gh * gw


def scales_in_use(desc):
    """Native scale plus every scale of the schedule, ascending."""
    return sorted(set([1] + _scales(desc)))


def window_frames(desc):
    """Window latent frames in token order: list of (frame index w, state
    index b (0-based), scale p_b, first token, token count)."""
    out = []
    first = 0
    F = int(desc["frames_per_state"])
    for b, p in enumerate(_scales(desc)):
        for f in range(F):
            n = frame_tokens(desc, p)
            out.append((b * F + f, b, p, first, n))
            first += n
    return out


def num_window_tokens(desc):
    return sum(w[4] for w in window_frames(desc))


def num_sink_tokens(desc):
    return int(desc["sink_frames"]) * frame_tokens(desc, 1)


def num_hist_tokens(desc):
    return int(desc["hist_frames"]) * frame_tokens(desc, 1)


def query_groups(desc):
    """(scale, q_begin, q_end) for each distinct query scale, in token order."""
    groups = []
    for (_, _, p, first, n) in window_frames(desc):
        if groups and groups[-1][0] == p:
            groups[-1][2] = first + n
        else:
            groups.append([p, first, first + n])
    return [tuple(g) for g in groups]


def context_rows(desc, s):
    """Eq. 4 for queries at scale s: one row per context frame, in the order
    sink, history (oldest first), window (state 1..T, frame order).

    Row = (kind, frame, src_scale, eff_scale, factor, n_tok)."""
    rows = []
    for f in range(int(desc["sink_frames"])):
        rows.append((KIND_SINK, f, 1, 1, 1, frame_tokens(desc, 1)))
    for f in range(int(desc["hist_frames"])):
        rows.append((KIND_HIST, f, 1, s, s, frame_tokens(desc, s)))
    for (w, _, p, _, _) in window_frames(desc):
        eff = max(s, p)
        rows.append((KIND_WIN, w, p, eff, max(1, s // p), frame_tokens(desc, eff)))
    return rows


def tables(desc):
    """The static plan as integer tables.

    GRID rows  [scale, gh, gw, tok] for every scale in use;
    QGRP rows  [q_scale, q_begin, q_end, n_kv];
    SEG rows   [q_scale, kind, frame, src_scale, eff_scale, factor, n_tok,
                kv_begin] (kv_begin is the running token offset within the
                query scale's context);
    TOTAL      [n_q, pairs_per_head] where pairs = sum over groups of
               (q_end - q_begin) * n_kv.
    """
    GRID = [[s, *grid(desc, s), frame_tokens(desc, s)] for s in scales_in_use(desc)]
    QGRP, SEG = [], []
    pairs = 0
    for (s, qb, qe) in query_groups(desc):
        kv = 0
        for (kind, frame, src, eff, fac, n) in context_rows(desc, s):
            SEG.append([s, kind, frame, src, eff, fac, n, kv])
            kv += n
        QGRP.append([s, qb, qe, kv])
        pairs += (qe - qb) * kv
    TOTAL = [num_window_tokens(desc), pairs]
    return {
        "GRID": np.array(GRID, dtype=np.int64).reshape(-1, 4),
        "QGRP": np.array(QGRP, dtype=np.int64).reshape(-1, 4),
        "SEG": np.array(SEG, dtype=np.int64).reshape(-1, 8),
        "TOTAL": np.array(TOTAL, dtype=np.int64),
    }


def pool_frame(x, gh, gw, f, mode="mean"):
    """Resample one frame's tokens x [gh*gw, ...] over f x f blocks of its
    grid.  mode "mean": block average, a block on a ragged edge averaging only
    the cells it holds.  mode "stride": the block's first cell (grid row f*Y,
    column f*X), which always exists."""
    x = np.asarray(x, dtype=np.float64)
    if f == 1:
        return x.copy()
    img = x.reshape(gh, gw, *x.shape[1:])
    oh, ow = _ceil_div(gh, f), _ceil_div(gw, f)
    out = np.empty((oh, ow) + x.shape[1:], dtype=np.float64)
    for Y in range(oh):
        for X in range(ow):
            if mode == "stride":
                out[Y, X] = img[f * Y, f * X]
            else:
                block = img[f * Y: f * Y + f, f * X: f * X + f]
                out[Y, X] = block.reshape(-1, *x.shape[1:]).mean(axis=0)
    return out.reshape(oh * ow, *x.shape[1:])


def hist_frame(desc, x_hist, f):
    n = frame_tokens(desc, 1)
    return x_hist[f * n: (f + 1) * n]


def context(desc, s, x_sink, x_hist, x_win):
    """Concatenated K (or V) context for queries at scale s, float64, in
    the canonical row order of context_rows()."""
    parts = []
    mode = resample_mode(desc)
    n1 = frame_tokens(desc, 1)
    gh1, gw1 = grid(desc, 1)
    wf = {w: (p, first, n) for (w, _, p, first, n) in window_frames(desc)}
    for (kind, frame, src, eff, fac, n) in context_rows(desc, s):
        if kind == KIND_SINK:
            parts.append(np.asarray(x_sink[frame * n1: (frame + 1) * n1], dtype=np.float64))
        elif kind == KIND_HIST:
            parts.append(pool_frame(hist_frame(desc, x_hist, frame), gh1, gw1, fac, mode))
        else:
            p, first, nsrc = wf[frame]
            gh, gw = grid(desc, p)
            parts.append(pool_frame(x_win[first: first + nsrc], gh, gw, fac, mode))
    return np.concatenate(parts, axis=0)


def attention(q, k, v, scale, chunk=1024):
    """softmax(scale q k^T) v for one head, max-subtracted, float64.
    q [nq, d], k/v [nkv, d].  Queries are processed in chunks only to bound
    memory; rows are independent."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    out = np.empty((q.shape[0], v.shape[1]), dtype=np.float64)
    for i in range(0, q.shape[0], chunk):
        z = scale * (q[i: i + chunk] @ k.T)
        z -= z.max(axis=1, keepdims=True)
        w = np.exp(z)
        w /= w.sum(axis=1, keepdims=True)
        out[i: i + chunk] = w @ v
    return out


def pooled_kv(desc, x_hist, x_win):
    """Every pooled frame MSSA needs, keyed (kind, frame, eff_scale) ->
    float64 tokens: history frames and window frames resampled to each query
    scale coarser than their own."""
    out = {}
    mode = resample_mode(desc)
    n1 = frame_tokens(desc, 1)
    gh1, gw1 = grid(desc, 1)
    for (s, _, _) in query_groups(desc):
        for (kind, frame, src, eff, fac, n) in context_rows(desc, s):
            if fac == 1 or kind == KIND_SINK:
                continue
            if kind == KIND_HIST:
                out[(kind, frame, eff)] = pool_frame(
                    x_hist[frame * n1: (frame + 1) * n1], gh1, gw1, fac, mode)
            else:
                p, first, nsrc = {w: (p, f0, nn) for (w, _, p, f0, nn) in window_frames(desc)}[frame]
                gh, gw = grid(desc, p)
                out[(kind, frame, eff)] = pool_frame(x_win[first: first + nsrc], gh, gw, fac, mode)
    return out


def mssa_attention(desc, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win,
                   heads=None, q_index=None):
    """MSSA output [n_q, heads, head_dim] in float64 (Eq. 4 context, softmax
    attention per head and query scale).

    heads   optional list of head indices to compute (others are NaN);
    q_index optional sorted array of query token indices to compute (others
            are NaN) -- used to check sampled outputs of large problems.
    """
    nh = int(desc["num_heads"])
    d = int(desc["head_dim"])
    nq = num_window_tokens(desc)
    scale = softmax_scale(desc)
    heads = list(range(nh)) if heads is None else list(heads)
    out = np.full((nq, nh, d), np.nan, dtype=np.float64)
    want = np.ones(nq, dtype=bool)
    if q_index is not None:
        want[:] = False
        want[np.asarray(q_index, dtype=np.int64)] = True
    for (s, qb, qe) in query_groups(desc):
        rows = np.nonzero(want[qb:qe])[0] + qb
        if rows.size == 0:
            continue
        for h in heads:
            kc = context(desc, s, _head(k_sink, h), _head(k_hist, h), _head(k_win, h))
            vc = context(desc, s, _head(v_sink, h), _head(v_hist, h), _head(v_win, h))
            out[rows, h] = attention(np.asarray(q_win[rows, h], dtype=np.float64), kc, vc, scale)
    return out


def _head(x, h):
    if x is None:
        return np.zeros((0, 1))
    return np.asarray(x[:, h], dtype=np.float64)


def brute_force_attention(desc, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win):
    """Per-token re-derivation of MSSA for tiny problems, written
    independently of the vectorised path above: each query token builds its
    own context one key at a time from explicit per-cell sums, then takes
    an exp-normalised weighted sum.  Pure Python loops; float64."""
    T = int(desc["num_states"])
    sched = [int(x) for x in desc["scales"][:T]]
    H, W = int(desc["grid_h"]), int(desc["grid_w"])
    F = int(desc["frames_per_state"])
    S = int(desc["sink_frames"])
    Hh = int(desc["hist_frames"])
    nh, d = int(desc["num_heads"]), int(desc["head_dim"])
    sc = softmax_scale(desc)
    pick_first = resample_mode(desc) == "stride"

    def cells(s):
        return (H + s - 1) // s, (W + s - 1) // s

    # Where each window frame's tokens live, in token order.
    win_start = []
    pos = 0
    for b in range(T):
        gh, gw = cells(sched[b])
        for f in range(F):
            win_start.append((b, pos))
            pos += gh * gw
    n_q = pos

    def avg(src, base, src_gh, src_gw, f, Y, X, h):
        acc = [0.0] * d
        cnt = 0
        for dy in range(f):
            for dx in range(f):
                r, c = f * Y + dy, f * X + dx
                if pick_first and (dy or dx):
                    continue
                if r < src_gh and c < src_gw:
                    t = base + r * src_gw + c
                    for j in range(d):
                        acc[j] += float(src[t, h, j])
                    cnt += 1
        return [a / cnt for a in acc]

    out = np.zeros((n_q, nh, d), dtype=np.float64)
    for qi in range(n_q):
        # which state does this query token belong to?
        b_q = max(i for i, (b, st) in enumerate(win_start) if st <= qi)
        s = sched[win_start[b_q][0]]
        for h in range(nh):
            keys, vals = [], []
            n1 = H * W
            for f in range(S):
                for t in range(n1):
                    keys.append([float(x) for x in k_sink[f * n1 + t, h]])
                    vals.append([float(x) for x in v_sink[f * n1 + t, h]])
            gh, gw = cells(s)
            for f in range(Hh):
                for Y in range(gh):
                    for X in range(gw):
                        keys.append(avg(k_hist, f * n1, H, W, s, Y, X, h))
                        vals.append(avg(v_hist, f * n1, H, W, s, Y, X, h))
            for (b, st) in win_start:
                pb = sched[b]
                f = max(1, s // pb)
                sgh, sgw = cells(pb)
                ogh, ogw = (sgh + f - 1) // f, (sgw + f - 1) // f
                for Y in range(ogh):
                    for X in range(ogw):
                        keys.append(avg(k_win, st, sgh, sgw, f, Y, X, h))
                        vals.append(avg(v_win, st, sgh, sgw, f, Y, X, h))
            q = [float(x) for x in q_win[qi, h]]
            logits = [sc * sum(q[j] * kk[j] for j in range(d)) for kk in keys]
            mx = max(logits)
            e = [math.exp(z - mx) for z in logits]
            tot = sum(e)
            for j in range(d):
                out[qi, h, j] = sum(e[t] * vals[t][j] for t in range(len(vals))) / tot
    return out


def algorithmic_flops(desc):
    """4 * head_dim * heads * sum over query scales of n_q * n_kv: the
    multiply-adds of q k^T and p v that MSSA performs, at 2 flops each."""
    t = tables(desc)
    return 4 * int(desc["head_dim"]) * int(desc["num_heads"]) * int(t["TOTAL"][1])
