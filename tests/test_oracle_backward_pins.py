"""Pins of the fp64 backward oracle against what the mathematics fixes (no
GPU): the derivative definition (central differences of the pinned forward
oracle), torch's autograd of plain softmax attention when every scale is
native, the adjoint identity of resampling, and the two sum rules of
softmax attention.  A dropped 1/c, a wrong sign in the softmax Jacobian, a
transposed product or a missing query scale fails one of them."""

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle

NAMES = ("q_win", "k_sink", "v_sink", "k_hist", "v_hist", "k_win", "v_win")


def _desc(T, scales, H, W, F=1, S=1, Hh=1, nh=1, d=4, **kw):
    return dict(num_states=T, scales=list(scales), grid_h=H, grid_w=W, frames_per_state=F,
                sink_frames=S, hist_frames=Hh, num_heads=nh, head_dim=d, **kw)


def _inputs(desc, seed):
    rng = np.random.default_rng(seed)
    nh, d = desc["num_heads"], desc["head_dim"]
    n = dict(q_win=oracle.num_window_tokens(desc), k_win=oracle.num_window_tokens(desc),
             v_win=oracle.num_window_tokens(desc), k_sink=oracle.num_sink_tokens(desc),
             v_sink=oracle.num_sink_tokens(desc), k_hist=oracle.num_hist_tokens(desc),
             v_hist=oracle.num_hist_tokens(desc))
    x = {k: rng.standard_normal((n[k], nh, d)) for k in NAMES}
    dout = rng.standard_normal((n["q_win"], nh, d))
    return x, dout


def _fwd(desc, x):
    return oracle.mssa_attention(desc, *(x[k] for k in NAMES))


def _bwd(desc, x, dout):
    return oracle.mssa_backward(desc, *(x[k] for k in NAMES), dout)


CASES = [
    _desc(3, [1, 2, 4], 5, 7, F=2, S=1, Hh=2, nh=2, d=3),                    # ragged at 2x and 4x
    _desc(3, [1, 2, 4], 5, 7, F=2, S=1, Hh=2, nh=2, d=3, resample="stride"),
    _desc(2, [2, 2], 6, 4, F=1, S=2, Hh=1, nh=1, d=4),                       # no native query scale
    _desc(4, [1, 1, 2, 2], 4, 6, F=1, S=0, Hh=0, nh=1, d=5),                 # no sink, no history
]


@pytest.mark.parametrize("desc", CASES, ids=["mean_ragged", "stride_ragged", "all_coarse", "window_only"])
def test_backward_equals_directional_derivative(desc):
    """For a random direction u of every input, <grad, u> equals the central
    difference (L(x + e u) - L(x - e u)) / 2e of L = <dout, out>."""
    x, dout = _inputs(desc, 1)
    g = _bwd(desc, x, dout)
    rng = np.random.default_rng(2)
    for name in NAMES:
        if x[name].size == 0:
            continue
        u = rng.standard_normal(x[name].shape)
        eps = 1e-5
        xp, xm = dict(x), dict(x)
        xp[name] = x[name] + eps * u
        xm[name] = x[name] - eps * u
        fd = (np.sum(dout * _fwd(desc, xp)) - np.sum(dout * _fwd(desc, xm))) / (2 * eps)
        an = np.sum(g["d" + name] * u)
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (name, fd, an)


def test_backward_single_entries_by_finite_differences():
    """Entry by entry on one history token that is pooled twice (into the
    2x and the 4x contexts) and one coarse window token."""
    desc = CASES[0]
    x, dout = _inputs(desc, 3)
    g = _bwd(desc, x, dout)
    eps = 1e-6
    for name, idx in (("k_hist", (12, 1, 2)), ("v_hist", (34, 0, 0)), ("k_win", (75, 1, 1)),
                      ("k_sink", (0, 0, 2)), ("q_win", (80, 1, 0))):
        if idx[0] >= x[name].shape[0]:
            idx = (x[name].shape[0] - 1,) + idx[1:]
        xp, xm = dict(x), dict(x)
        xp[name] = x[name].copy()
        xm[name] = x[name].copy()
        xp[name][idx] += eps
        xm[name][idx] -= eps
        fd = (np.sum(dout * _fwd(desc, xp)) - np.sum(dout * _fwd(desc, xm))) / (2 * eps)
        assert abs(fd - g["d" + name][idx]) <= 1e-7, (name, idx, fd, g["d" + name][idx])


def test_all_native_backward_is_torch_autograd():
    """With every scale 1, MSSA is softmax attention over [sink | history |
    window]; its gradients are torch's autograd of SDPA (float64)."""
    desc = _desc(3, [1, 1, 1], 4, 5, F=2, S=1, Hh=2, nh=2, d=8)
    x, dout = _inputs(desc, 4)
    g = _bwd(desc, x, dout)
    t = {k: torch.tensor(x[k], requires_grad=True) for k in NAMES}
    kc = torch.cat([t["k_sink"], t["k_hist"], t["k_win"]]).permute(1, 0, 2)
    vc = torch.cat([t["v_sink"], t["v_hist"], t["v_win"]]).permute(1, 0, 2)
    o = torch.nn.functional.scaled_dot_product_attention(t["q_win"].permute(1, 0, 2), kc, vc)
    o.backward(torch.tensor(dout).permute(1, 0, 2))
    for k in NAMES:
        assert np.allclose(g["d" + k], t[k].grad.numpy(), atol=1e-12, rtol=0), k


@settings(max_examples=40, deadline=None)
@given(gh=st.integers(1, 9), gw=st.integers(1, 9), f=st.sampled_from([1, 2, 4]),
       mode=st.sampled_from(["mean", "stride"]), seed=st.integers(0, 1000))
def test_resample_adjoint_identity(gh, gw, f, mode, seed):
    """<pool(x), y> == <x, pool_adjoint(y)> for every grid, ragged included."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((gh * gw, 2))
    y = rng.standard_normal((-(-gh // f) * -(-gw // f), 2))
    lhs = np.sum(oracle.pool_frame(x, gh, gw, f, mode) * y)
    rhs = np.sum(x * oracle.pool_frame_adjoint(y, gh, gw, f, mode))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


@pytest.mark.parametrize("desc", CASES[:3], ids=["mean", "stride", "all_coarse"])
def test_backward_sum_rules(desc):
    """Softmax weights sum to one and their Jacobian rows sum to zero, and
    resampling adjoints keep the total: summed over every source token,
    dV equals the sum of dout over all queries and dK is zero."""
    x, dout = _inputs(desc, 5)
    g = _bwd(desc, x, dout)
    dv = sum(g[k].sum(axis=0) for k in ("dv_sink", "dv_hist", "dv_win"))
    dk = sum(g[k].sum(axis=0) for k in ("dk_sink", "dk_hist", "dk_win"))
    assert np.allclose(dv, dout.sum(axis=0), atol=1e-12)
    assert np.abs(dk).max() <= 1e-12


def test_backward_heads_subset_and_nan():
    desc = CASES[0]
    x, dout = _inputs(desc, 6)
    full = _bwd(desc, x, dout)
    part = oracle.mssa_backward(desc, *(x[k] for k in NAMES), dout, heads=[1])
    for k in full:
        assert np.array_equal(part[k][:, 1], full[k][:, 1])
        assert np.isnan(part[k][:, 0]).all()
