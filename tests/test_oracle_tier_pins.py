"""Pins of the tier patch embedding / de-embedding and QKV projection oracle
(no GPU): torch's 2-D convolution and transposed convolution with kernel =
stride = patch (float64), the exact patchify/unpatchify round trip, Eq. 3's
token counts and torch's linear layer.  A transposed weight, a wrong
feature order, a missing edge pad or a swapped q/k/v block fails one."""

import numpy as np
import pytest
import torch

import oracle


def _desc(scales, H, W, F=1):
    return dict(num_states=len(scales), scales=list(scales), grid_h=H, grid_w=W, frames_per_state=F,
                sink_frames=0, hist_frames=0, num_heads=2, head_dim=8)


@pytest.mark.parametrize("C,H,W,P", [(3, 8, 12, 2), (4, 10, 13, 4), (2, 7, 9, 8), (16, 12, 20, 4)])
def test_patch_embed_is_strided_convolution(C, H, W, P):
    rng = np.random.default_rng(P + H)
    hidden = 5
    x = rng.standard_normal((C, H, W))
    w = rng.standard_normal((hidden, C * P * P))
    b = rng.standard_normal(hidden)
    tok = oracle.patchify(x, P) @ w.T + b
    ph, pw = -H % P, -W % P
    xt = torch.nn.functional.pad(torch.tensor(x)[None], (0, pw, 0, ph))
    ref = torch.nn.functional.conv2d(xt, torch.tensor(w).reshape(hidden, C, P, P), torch.tensor(b), stride=P)
    assert np.allclose(tok, ref[0].permute(1, 2, 0).reshape(-1, hidden).numpy(), atol=1e-12)


@pytest.mark.parametrize("C,H,W,P", [(3, 8, 12, 2), (4, 10, 13, 4), (2, 7, 9, 8)])
def test_patch_unembed_is_transposed_convolution(C, H, W, P):
    rng = np.random.default_rng(P * W)
    hidden = 6
    gh, gw = -(-H // P), -(-W // P)
    tok = rng.standard_normal((gh * gw, hidden))
    w = rng.standard_normal((C * P * P, hidden))
    b = rng.standard_normal(C * P * P)
    got = oracle.unpatchify(tok @ w.T + b, P, C, H, W)
    # conv_transpose2d weight [in=hidden, out=C, P, P]; the per-pixel bias
    # of the de-embedding is a per-(channel, row, column) constant added after
    wt = torch.tensor(w.T).reshape(hidden, C, P, P)
    y = torch.nn.functional.conv_transpose2d(torch.tensor(tok).T.reshape(1, hidden, gh, gw), wt, stride=P)[0]
    y = y + torch.tensor(b).reshape(C, P, P).repeat(1, gh, gw)
    assert np.allclose(got, y[:, :H, :W].numpy(), atol=1e-12)


@pytest.mark.parametrize("C,H,W,P", [(3, 8, 12, 2), (2, 7, 9, 4), (1, 5, 5, 8)])
def test_patchify_round_trip(C, H, W, P):
    x = np.random.default_rng(1).standard_normal((C, H, W))
    assert np.array_equal(oracle.unpatchify(oracle.patchify(x, P), P, C, H, W), x)


def test_window_token_counts_follow_eq3():
    """(p, p, 2p, 2p, 2p) on the 30 x 52 native grid: 1560 tokens per native
    frame, 390 per coarse frame, 12870 in the window, 0.55 of the native
    count (Eq. 3); the embedding emits the attention's window tokens."""
    desc = _desc([1, 1, 2, 2, 2], 30, 52, F=3)
    patch, C = 2, 1
    lat = np.zeros((15, C, 60, 104))
    w = {s: np.zeros((4, C * (patch * s) ** 2)) for s in (1, 2)}
    b = {s: np.zeros(4) for s in (1, 2)}
    tok = oracle.patch_embed(desc, patch, lat, w, b)
    assert tok.shape == (12870, 4) == (oracle.num_window_tokens(desc), 4)
    assert tok.shape[0] / (15 * 1560) == pytest.approx(0.55)


def test_window_embed_uses_each_states_tier():
    """Frame f of state l is embedded with its own scale's weights and lands
    at the attention's token offset of that frame."""
    desc = _desc([1, 2, 4], 5, 7, F=2)
    patch, C, hidden = 2, 3, 4
    rng = np.random.default_rng(3)
    lat = rng.standard_normal((6, C, 10, 14))
    w = {s: rng.standard_normal((hidden, C * (patch * s) ** 2)) for s in (1, 2, 4)}
    b = {s: rng.standard_normal(hidden) for s in (1, 2, 4)}
    tok = oracle.patch_embed(desc, patch, lat, w, b)
    for (wi, _, s, first, n) in oracle.window_frames(desc):
        want = oracle.patchify(lat[wi], patch * s) @ w[s].T + b[s]
        assert np.array_equal(tok[first: first + n], want)
    out = oracle.patch_unembed(desc, patch, C, tok,
                               {s: rng.standard_normal((C * (patch * s) ** 2, hidden)) for s in (1, 2, 4)},
                               {s: np.zeros(C * (patch * s) ** 2) for s in (1, 2, 4)})
    assert out.shape == (6, C, 10, 14)


def test_qkv_projection_is_linear():
    rng = np.random.default_rng(4)
    n, heads, d = 7, 3, 4
    x = rng.standard_normal((n, heads * d))
    w = rng.standard_normal((3 * heads * d, heads * d))
    b = rng.standard_normal(3 * heads * d)
    q, k, v = oracle.qkv_project(x, w, b, heads)
    ref = torch.nn.functional.linear(torch.tensor(x), torch.tensor(w), torch.tensor(b)).numpy()
    assert np.allclose(np.concatenate([q, k, v], axis=1).reshape(n, 3, heads * d),
                       ref.reshape(n, 3, heads * d), atol=1e-12)
    assert np.allclose(k.reshape(n, -1), ref[:, heads * d: 2 * heads * d], atol=1e-12)
