"""fp64 CPU oracle for the gradients of Multi-Scale Self-Attention (MSSA).

TEST INFRASTRUCTURE ONLY.  Like the forward oracle, this module is the slow,
plain reference that the GPU library is checked against; only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it.
It shares no code with the HIP path.

What is differentiated is exactly the forward of the forward oracle (Sec. 4.1,
Eq. 4): for every head and query scale s,
    out = softmax(scale * q k_s^T) v_s,
where the context k_s / v_s concatenates the native sink, every history frame
resampled to s and every window frame resampled to max(s, own scale).  The
paper trains through these windows (Sec. 3.1 and Alg. 1 update the DiT by
gradient descent on the rolling window), so the backward is the chain rule
applied to that definition:

* per head and query scale, with P the softmax weights and dO the incoming
  gradient of the output,
      dV_s = P^T dO
      dP   = dO V_s^T
      dZ   = P * (dP - rowsum(P * dP))     (softmax Jacobian, row by row)
      dQ   = scale dZ K_s,   dK_s = scale dZ^T Q;
* every context row goes back to the frame it was made from: sink rows and
  native rows unchanged, resampled rows through the adjoint of the
  resampling (the block mean hands g / c to each of its c cells; the strided
  pick hands g to the block's first cell);
* a source token that appears in the contexts of several query scales sums
  its gradients over them.

Nothing is blocked, fused or reordered beyond these definitions; queries
are processed in chunks only to bound memory.  All arithmetic is float64.
"""

import numpy as np

from . import mssa_oracle as fwd


def attention_backward(q, k, v, d_out, scale, chunk=1024):
    """Gradients (dq, dk, dv) of out = softmax(scale q k^T) v for one head,
    given d_out = dL/d(out).  q, d_out [nq, d]; k, v [nkv, d]; float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    d_out = np.asarray(d_out, dtype=np.float64)
    dq = np.empty_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for i in range(0, q.shape[0], chunk):
        z = scale * (q[i: i + chunk] @ k.T)
        z -= z.max(axis=1, keepdims=True)
        p = np.exp(z)
        p /= p.sum(axis=1, keepdims=True)
        do = d_out[i: i + chunk]
        dv += p.T @ do
        dp = do @ v.T
        dz = p * (dp - (p * dp).sum(axis=1, keepdims=True))
        dq[i: i + chunk] = scale * (dz @ k)
        dk += scale * (dz.T @ q[i: i + chunk])
    return dq, dk, dv


def pool_frame_adjoint(g, gh, gw, f, mode="mean"):
    """Adjoint of the forward oracle's pool_frame: the gradient with respect to
    a frame's tokens [gh*gw, ...] given the gradient g of its resampled
    tokens [ceil(gh/f)*ceil(gw/f), ...]."""
    g = np.asarray(g, dtype=np.float64)
    if f == 1:
        return g.copy()
    oh, ow = -(-gh // f), -(-gw // f)
    gi = g.reshape(oh, ow, *g.shape[1:])
    out = np.zeros((gh, gw) + g.shape[1:], dtype=np.float64)
    for Y in range(oh):
        for X in range(ow):
            if mode == "stride":
                out[f * Y, f * X] += gi[Y, X]
            else:
                block = out[f * Y: f * Y + f, f * X: f * X + f]
                block += gi[Y, X] / (block.shape[0] * block.shape[1])
    return out.reshape(gh * gw, *g.shape[1:])


def _context_adjoint(desc, s, g_ctx, n_sink, n_hist, n_win):
    """Send the gradient of the context of query scale s (rows in the order
    of context_rows) back to the sink, history and window tokens."""
    mode = fwd.resample_mode(desc)
    n1 = fwd.frame_tokens(desc, 1)
    gh1, gw1 = fwd.grid(desc, 1)
    wf = {w: (p, first, n) for (w, _, p, first, n) in fwd.window_frames(desc)}
    tail = g_ctx.shape[1:]
    g_sink = np.zeros((n_sink,) + tail)
    g_hist = np.zeros((n_hist,) + tail)
    g_win = np.zeros((n_win,) + tail)
    pos = 0
    for (kind, frame, src, eff, fac, n) in fwd.context_rows(desc, s):
        g = g_ctx[pos: pos + n]
        pos += n
        if kind == fwd.KIND_SINK:
            g_sink[frame * n1: (frame + 1) * n1] += g
        elif kind == fwd.KIND_HIST:
            g_hist[frame * n1: (frame + 1) * n1] += pool_frame_adjoint(g, gh1, gw1, fac, mode)
        else:
            p, first, nsrc = wf[frame]
            gh, gw = fwd.grid(desc, p)
            g_win[first: first + nsrc] += pool_frame_adjoint(g, gh, gw, fac, mode)
    assert pos == g_ctx.shape[0]
    return g_sink, g_hist, g_win


def mssa_backward(desc, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, d_out, heads=None):
    """Gradients of MSSA with respect to all seven inputs, float64, as a dict
    with keys dq_win, dk_sink, dv_sink, dk_hist, dv_hist, dk_win, dv_win
    (each shaped like its input; heads not listed in `heads` are NaN)."""
    nh = int(desc["num_heads"])
    d = int(desc["head_dim"])
    scale = fwd.softmax_scale(desc)
    nq = fwd.num_window_tokens(desc)
    ns = fwd.num_sink_tokens(desc)
    nhst = fwd.num_hist_tokens(desc)
    heads = list(range(nh)) if heads is None else list(heads)
    out = {}
    for name, n in (("dq_win", nq), ("dk_win", nq), ("dv_win", nq), ("dk_sink", ns), ("dv_sink", ns),
                    ("dk_hist", nhst), ("dv_hist", nhst)):
        a = np.full((n, nh, d), np.nan, dtype=np.float64)
        a[:, heads] = 0.0
        out[name] = a
    for h in heads:
        ks, vs = fwd._head(k_sink, h), fwd._head(v_sink, h)
        kh, vh = fwd._head(k_hist, h), fwd._head(v_hist, h)
        kw, vw = fwd._head(k_win, h), fwd._head(v_win, h)
        for (s, qb, qe) in fwd.query_groups(desc):
            kc = fwd.context(desc, s, ks, kh, kw)
            vc = fwd.context(desc, s, vs, vh, vw)
            dq, dkc, dvc = attention_backward(np.asarray(q_win[qb:qe, h], dtype=np.float64), kc, vc,
                                              np.asarray(d_out[qb:qe, h], dtype=np.float64), scale)
            out["dq_win"][qb:qe, h] = dq
            for which, g_ctx in (("k", dkc), ("v", dvc)):
                g_sink, g_hist, g_win = _context_adjoint(desc, s, g_ctx, ns, nhst, nq)
                out["d" + which + "_sink"][:, h] += g_sink
                out["d" + which + "_hist"][:, h] += g_hist
                out["d" + which + "_win"][:, h] += g_win
    return out
