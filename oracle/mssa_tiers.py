"""fp64 CPU oracle for the steps on either side of MSSA: Multi-Scale
Patchification (MSP) tier patch embedding / de-embedding and the QKV
projection that feeds the attention.

TEST INFRASTRUCTURE ONLY (see the package docstring): imported by the test
suite, the smoke check and the benchmark's CPU-baseline leg, never by the
library, and sharing no code with it.

What is computed (Ms. Forcing, Sec. 4.1, Multi-Scale Patchification):

* Window state l is tokenized with patch size p * p_l (p: the native patch
  in latent pixels, p_l: the state's scale).  A tier's patch embedding maps
  each non-overlapping (p p_l) x (p p_l) patch of every latent channel to
  one token of the model width: tokens = patches @ W_l^T + b_l, the patch
  flattened in (channel, row, column) order, which is a 2-D convolution with
  kernel = stride = p p_l.  Every tier has its own embedding and
  de-embedding (Sec. 4.1); the backbone is shared.
* The token grid of a latent frame is ceil(H/(p p_l)) x ceil(W/(p p_l)) (the
  ceil reading of Eq. 3, as for the attention); a patch that runs past the
  frame's bottom or right edge sees zeros there.
* The de-embedding maps each token back to its patch (tokens @ W_out^T +
  b_out, unflattened in the same order) and keeps the pixels inside the
  frame.
* The attention's q, k, v are x @ W_qkv^T + b_qkv split into three blocks of
  the model width, each viewed as [tokens, heads, head_dim].

Latent frames are arrays [frames, channels, H, W]; window frames are in
window order (state, frame), states at their own scales.
"""

import numpy as np

from . import mssa_oracle as fwd


def patchify(frame, P):
    """One latent frame [C, H, W] -> patches [ceil(H/P) * ceil(W/P), C*P*P]
    (row-major patch grid, features in (channel, row, column) order, zeros
    past the frame's edge)."""
    frame = np.asarray(frame, dtype=np.float64)
    C, H, W = frame.shape
    gh, gw = -(-H // P), -(-W // P)
    out = np.zeros((gh * gw, C * P * P), dtype=np.float64)
    for Y in range(gh):
        for X in range(gw):
            patch = np.zeros((C, P, P), dtype=np.float64)
            block = frame[:, Y * P: Y * P + P, X * P: X * P + P]
            patch[:, : block.shape[1], : block.shape[2]] = block
            out[Y * gw + X] = patch.reshape(-1)
    return out


def unpatchify(patches, P, C, H, W):
    """Inverse of patchify: patches [ceil(H/P) * ceil(W/P), C*P*P] -> frame
    [C, H, W], pixels past the frame's edge dropped."""
    patches = np.asarray(patches, dtype=np.float64)
    gh, gw = -(-H // P), -(-W // P)
    full = np.zeros((C, gh * P, gw * P), dtype=np.float64)
    for Y in range(gh):
        for X in range(gw):
            full[:, Y * P: Y * P + P, X * P: X * P + P] = patches[Y * gw + X].reshape(C, P, P)
    return full[:, :H, :W]


def _window_scales(desc):
    """Scale of every window frame, in window order."""
    return [p for (_, _, p, _, _) in fwd.window_frames(desc)]


def patch_embed(desc, patch, latent, w_embed, b_embed):
    """Window latent frames [T*F, C, H, W] (H = grid_h * patch) -> tokens
    [n_q, hidden] in the attention's window token order.  w_embed / b_embed
    map each scale s of the schedule to its tier's [hidden, C*(patch*s)^2]
    weights and [hidden] bias."""
    out = []
    for f, s in enumerate(_window_scales(desc)):
        P = patch * s
        out.append(patchify(latent[f], P) @ np.asarray(w_embed[s], dtype=np.float64).T
                   + np.asarray(b_embed[s], dtype=np.float64))
    return np.concatenate(out, axis=0)


def patch_unembed(desc, patch, channels, tokens, w_out, b_out):
    """Tokens [n_q, hidden] -> window latent frames [T*F, C, H, W]; w_out /
    b_out map each scale s to its tier's [C*(patch*s)^2, hidden] weights and
    [C*(patch*s)^2] bias."""
    H, W = int(desc["grid_h"]) * patch, int(desc["grid_w"]) * patch
    frames = []
    for (w, _, s, first, n) in fwd.window_frames(desc):
        P = patch * s
        pt = np.asarray(tokens[first: first + n], dtype=np.float64) @ np.asarray(w_out[s], dtype=np.float64).T \
            + np.asarray(b_out[s], dtype=np.float64)
        frames.append(unpatchify(pt, P, channels, H, W))
    return np.stack(frames)


def qkv_project(x, w_qkv, b_qkv, num_heads):
    """x [n, hidden] -> (q, k, v), each [n, heads, hidden / heads]."""
    y = np.asarray(x, dtype=np.float64) @ np.asarray(w_qkv, dtype=np.float64).T + np.asarray(b_qkv, dtype=np.float64)
    n, three_h = y.shape
    hidden = three_h // 3
    return tuple(y[:, i * hidden: (i + 1) * hidden].reshape(n, num_heads, hidden // num_heads) for i in range(3))
