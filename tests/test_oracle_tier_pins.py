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


def _conv_embed_frame(frame, w, b, P):
    """torch's strided convolution of one latent frame [C, H, W] (zero pad to
    a multiple of P), kernel = stride = P: tokens [gh * gw, hidden]."""
    C, H, W = frame.shape
    xt = torch.nn.functional.pad(torch.tensor(frame)[None], (0, -W % P, 0, -H % P))
    y = torch.nn.functional.conv2d(xt, torch.tensor(w).reshape(w.shape[0], C, P, P), torch.tensor(b), stride=P)
    return y[0].permute(1, 2, 0).reshape(-1, w.shape[0]).numpy()


def _conv_unembed_frame(tok, w, b, P, C, H, W):
    """torch's transposed convolution of one frame's tokens, cropped to the
    frame: [C, H, W]."""
    gh, gw = -(-H // P), -(-W // P)
    hidden = tok.shape[1]
    wt = torch.tensor(w.T).reshape(hidden, C, P, P)
    y = torch.nn.functional.conv_transpose2d(torch.tensor(tok).T.reshape(1, hidden, gh, gw), wt, stride=P)[0]
    y = y + torch.tensor(b).reshape(C, P, P).repeat(1, gh, gw)
    return y[:, :H, :W].numpy()


# Window of three states at scales 1, 2, 4 (two latent frames each) on a 5 x 7
# patch grid with patch 2: the token grids are 5 x 7, 3 x 4 and 2 x 2 (Eq. 3,
# ceil), so state l's frames hold 35, 12 and 4 tokens.  Offsets of every
# window frame in token order, written out by hand from those counts:
# state 1 frames at 0 and 35, state 2 at 70 and 82, state 3 at 94 and 98.
_TIER_DESC = _desc([1, 2, 4], 5, 7, F=2)
_TIER_LAYOUT = [  # (window frame, scale, first token, tokens)
    (0, 1, 0, 35), (1, 1, 35, 35), (2, 2, 70, 12), (3, 2, 82, 12), (4, 4, 94, 4), (5, 4, 98, 4)]
_TIER_NQ = 102


def _tier_inputs(seed):
    patch, C, hidden = 2, 3, 4
    rng = np.random.default_rng(seed)
    lat = rng.standard_normal((6, C, 10, 14))
    w = {s: rng.standard_normal((hidden, C * (patch * s) ** 2)) for s in (1, 2, 4)}
    b = {s: rng.standard_normal(hidden) for s in (1, 2, 4)}
    wo = {s: rng.standard_normal((C * (patch * s) ** 2, hidden)) for s in (1, 2, 4)}
    bo = {s: rng.standard_normal(C * (patch * s) ** 2) for s in (1, 2, 4)}
    return patch, C, hidden, lat, w, b, wo, bo


def _expected_embed(patch, lat, w, b):
    """Window tokens built frame by frame with torch's convolution and each
    state's own tier weights, placed at the hand-written offsets."""
    out = np.full((_TIER_NQ, next(iter(w.values())).shape[0]), np.nan)
    for (f, s, first, n) in _TIER_LAYOUT:
        tok = _conv_embed_frame(lat[f], w[s], b[s], patch * s)
        assert tok.shape[0] == n
        out[first: first + n] = tok
    return out


def _expected_unembed(patch, C, tokens, wo, bo):
    frames = np.full((6, C, 10, 14), np.nan)
    for (f, s, first, n) in _TIER_LAYOUT:
        frames[f] = _conv_unembed_frame(tokens[first: first + n], wo[s], bo[s], patch * s, C, 10, 14)
    return frames


def test_window_layout_is_eq3_by_hand():
    """The hand-written layout is the attention's window token order."""
    assert oracle.num_window_tokens(_TIER_DESC) == _TIER_NQ
    assert [(w, p, first, n) for (w, _, p, first, n) in oracle.window_frames(_TIER_DESC)] == _TIER_LAYOUT


def test_window_embed_uses_each_states_tier():
    """Frame f of state l is embedded with its own tier's weights (torch's
    convolution with kernel = stride = patch * p_l) and lands at the token
    offset Eq. 3's counts give."""
    patch, C, hidden, lat, w, b, _, _ = _tier_inputs(3)
    tok = oracle.patch_embed(_TIER_DESC, patch, lat, w, b)
    assert np.allclose(tok, _expected_embed(patch, lat, w, b), atol=1e-12)


def test_window_unembed_uses_each_states_tier():
    """De-embedding: frame f of state l comes from its own tokens through its
    tier's transposed convolution, cropped to the frame."""
    patch, C, hidden, lat, w, b, wo, bo = _tier_inputs(4)
    tokens = np.random.default_rng(5).standard_normal((_TIER_NQ, hidden))
    got = oracle.patch_unembed(_TIER_DESC, patch, C, tokens, wo, bo)
    assert np.allclose(got, _expected_unembed(patch, C, tokens, wo, bo), atol=1e-12)


def _embed_mutant(desc, patch, latent, w, b, slip):
    """oracle.patch_embed with a planted mistake: "frames" embeds the two
    frames of every state in swapped order; "tier" embeds every state with
    weights of its tier's shape that are not its tier's (the tier's rows
    reversed)."""
    out = []
    for (f, _, s, _, _) in oracle.window_frames(desc):
        src = f ^ 1 if slip == "frames" else f
        ws = w[s][::-1] if slip == "tier" else w[s]
        bs = b[s][::-1] if slip == "tier" else b[s]
        out.append(oracle.patchify(latent[src], patch * s) @ ws.T + bs)
    return np.concatenate(out, axis=0)


def _unembed_mutant(desc, patch, C, tokens, wo, bo, slip):
    """oracle.patch_unembed with the same planted mistakes."""
    H, W = int(desc["grid_h"]) * patch, int(desc["grid_w"]) * patch
    frames = [None] * len(oracle.window_frames(desc))
    for (f, _, s, first, n) in oracle.window_frames(desc):
        ws = wo[s][:, ::-1] if slip == "tier" else wo[s]
        pt = tokens[first: first + n] @ ws.T + bo[s]
        frames[f ^ 1 if slip == "frames" else f] = oracle.unpatchify(pt, patch * s, C, H, W)
    return np.stack(frames)


@pytest.mark.parametrize("slip", ["frames", "tier"])
def test_tier_pins_reject_planted_mistakes(slip):
    """The two pins above have teeth: copies of the oracle functions that
    embed a state's frames in the wrong order, or with weights that are not
    the state's tier's, fail them; unmutated copies pass."""
    patch, C, hidden, lat, w, b, wo, bo = _tier_inputs(6)
    tokens = np.random.default_rng(7).standard_normal((_TIER_NQ, hidden))
    want = _expected_embed(patch, lat, w, b)
    want_un = _expected_unembed(patch, C, tokens, wo, bo)
    assert np.allclose(_embed_mutant(_TIER_DESC, patch, lat, w, b, None), want, atol=1e-12)
    assert np.allclose(_unembed_mutant(_TIER_DESC, patch, C, tokens, wo, bo, None), want_un, atol=1e-12)
    assert not np.allclose(_embed_mutant(_TIER_DESC, patch, lat, w, b, slip), want, atol=1e-6)
    assert not np.allclose(_unembed_mutant(_TIER_DESC, patch, C, tokens, wo, bo, slip), want_un, atol=1e-6)


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
