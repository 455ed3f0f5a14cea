"""Pins of the fp64 oracle against what the paper and the mathematics fix
(no GPU).  Each test would fail for a plausible slip in the oracle: a dropped
or pooled sink, a wrong visible set, an upsampled key, a count-including-pad
mean, a wrong softmax scale or a transposed operand."""

import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle
from paper_2607_20940_amd.workloads import WORKLOADS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            vals[parts[0]] = [float(x) for x in parts[1:3] if _isnum(x)]
    return vals


def _isnum(x):
    try:
        float(x)
        return True
    except ValueError:
        return False


def _desc(T, scales, H, W, F=1, S=1, Hh=1, nh=1, d=4):
    return dict(num_states=T, scales=list(scales), grid_h=H, grid_w=W, frames_per_state=F,
                sink_frames=S, hist_frames=Hh, num_heads=nh, head_dim=d)


def _rand_inputs(desc, seed):
    rng = np.random.default_rng(seed)
    nh, d = desc["num_heads"], desc["head_dim"]
    nq = oracle.num_window_tokens(desc)
    ns = oracle.num_sink_tokens(desc)
    nhst = oracle.num_hist_tokens(desc)
    g = lambda n: rng.standard_normal((n, nh, d))  # noqa: E731
    return dict(q_win=g(nq), k_win=g(nq), v_win=g(nq), k_sink=g(ns), v_sink=g(ns),
                k_hist=g(nhst), v_hist=g(nhst))


def _run(desc, x, **kw):
    return oracle.mssa_attention(desc, x["q_win"], x["k_sink"], x["v_sink"], x["k_hist"],
                                 x["v_hist"], x["k_win"], x["v_win"], **kw)


# ---------------------------------------------------------------- Eq. 3


def test_eq3_token_fraction_paper_schedule():
    """(p,p,2p,2p,2p) keeps 0.55 of the window tokens: a 45 % reduction
    (Sec. 4.1, Eq. 3).  Counted from the oracle's grids on a divisible grid."""
    g = _golden("paper_values.txt")
    desc = _desc(5, [1, 1, 2, 2, 2], 8, 12, F=3)
    n_msp = oracle.num_window_tokens(desc)
    n_rf = 5 * 3 * 8 * 12
    assert n_msp / n_rf == pytest.approx(g["rho_tok"][0], abs=1e-15)
    assert round(100 * (1 - n_msp / n_rf)) == g["token_reduction_pct"][0]


def test_eq3_counts_wan13b_workload():
    g = _golden("workload_counts.txt")
    desc = WORKLOADS["wan13b_layer"]["desc"]
    assert oracle.frame_tokens(desc, 1) == g["native_frame_tokens"][0]
    assert oracle.frame_tokens(desc, 2) == g["coarse2_frame_tokens"][0]
    assert oracle.num_window_tokens(desc) == g["active_query_tokens"][0]
    assert 5 * 3 * oracle.frame_tokens(desc, 1) == g["native_query_tokens"][0]


# ---------------------------------------------------------------- Eq. 5


def _pairs_without_mssa(desc):
    """Query-key pairs of MSP alone: every query sees every context frame at
    the frame's own MSP scale (no resampling)."""
    n1 = oracle.frame_tokens(desc, 1)
    ctx = desc["sink_frames"] * n1 + desc["hist_frames"] * n1
    ctx += sum(w[4] for w in oracle.window_frames(desc))
    return oracle.num_window_tokens(desc) * ctx


def test_eq5_reduction_paper_layout():
    """1 sink + 1 history + 5 window frames under (p,p,2p,2p,2p) gives a
    12.9 % cut of dot products (Sec. 4.1 after Eq. 5).  The oracle's pair
    count on an 8x8 grid gives exactly 27/209."""
    g = _golden("paper_values.txt")
    desc = _desc(5, [1, 1, 2, 2, 2], 8, 8, F=1, S=1, Hh=1)
    pairs = int(oracle.tables(desc)["TOTAL"][1])
    r = 1.0 - pairs / _pairs_without_mssa(desc)
    assert r == pytest.approx(27 / 209, abs=1e-15)
    assert 100 * r == pytest.approx(g["r_mssa_pct"][0], abs=g["r_mssa_pct"][1])


def test_eq5_closed_form_matches_counts_on_divisible_grids():
    """Eq. 5 in eta/stride form equals the oracle's token-pair ratio for any
    schedule on grids that every scale divides."""
    for sched in ([1, 1, 2, 2, 2], [1, 2, 4], [1, 1, 1, 4], [2, 2, 4, 8], [1]):
        T = len(sched)
        desc = _desc(T, sched, 16, 32, F=1, S=1, Hh=2)
        eta = [1.0 / p ** 2 for p in sched]
        vis = [(1.0, 1)] * 2 + [(eta[b], sched[b]) for b in range(T)]  # history + window
        num = den = 0.0
        for a in range(T):
            num += eta[a] * (1 + sum(e / max(1, sched[a] // p) ** 2 for e, p in vis))
            den += eta[a] * (1 + sum(e for e, _ in vis))
        pairs = int(oracle.tables(desc)["TOTAL"][1])
        assert 1 - pairs / _pairs_without_mssa(desc) == pytest.approx(1 - num / den, abs=1e-14)


def test_eq5_rejects_other_visible_sets():
    """The printed 12.9 % singles out the bidirectional visible set with
    history; causal or exclude-self masks give other values."""
    sched = [1, 1, 2, 2, 2]
    eta = [1.0 / p ** 2 for p in sched]

    def r(visible):
        num = den = 0.0
        for a in range(5):
            vis = [(1.0, 1)] + [(eta[b], sched[b]) for b in visible(a)]
            num += eta[a] * (1 + sum(e / max(1, sched[a] // p) ** 2 for e, p in vis))
            den += eta[a] * (1 + sum(e for e, _ in vis))
        return 100 * (1 - num / den)

    assert r(lambda a: range(5)) == pytest.approx(12.9, abs=0.05)
    assert abs(r(lambda a: [b for b in range(5) if b != a]) - 12.9) > 1
    assert abs(r(lambda a: range(a + 1)) - 12.9) > 1


# ---------------------------------------------------------------- tables


def test_tables_wan13b_context_sizes():
    desc = WORKLOADS["wan13b_layer"]["desc"]
    t = oracle.tables(desc)
    assert t["QGRP"].tolist() == [[1, 0, 9360, 26910], [2, 9360, 12870, 12870]]
    seg = t["SEG"]
    # the sink is never resampled, at any query scale
    sink = seg[seg[:, 1] == oracle.KIND_SINK]
    assert (sink[:, 4] == 1).all() and (sink[:, 5] == 1).all()
    # no key is denser than... coarser keys keep their own scale
    win = seg[seg[:, 1] == oracle.KIND_WIN]
    assert (win[:, 4] == np.maximum(win[:, 0], win[:, 3])).all()


def test_tables_wan13b_seg_rows_by_hand():
    """Every SEG row of the Wan-1.3B-shaped layer written out by hand from
    Eq. 3 and Eq. 4: 1560 tokens per native frame (30 x 52), 390 per frame at
    scale 2 (15 x 26); context order sink (3 frames, native), history (6
    frames, pooled by the query scale), window frames 0..14 (states 1-2 native,
    states 3-5 at scale 2), kv_begin the running token offset."""
    t = oracle.tables(WORKLOADS["wan13b_layer"]["desc"])
    # (q_scale, kind, frame, src_scale, eff_scale, factor, n_tok, kv_begin)
    s1 = ([(1, 0, f, 1, 1, 1, 1560, 1560 * f) for f in range(3)]
          + [(1, 1, f, 1, 1, 1, 1560, 4680 + 1560 * f) for f in range(6)]
          + [(1, 2, w, 1, 1, 1, 1560, 14040 + 1560 * w) for w in range(6)]
          + [(1, 2, w, 2, 2, 1, 390, 23400 + 390 * (w - 6)) for w in range(6, 15)])
    s2 = ([(2, 0, f, 1, 1, 1, 1560, 1560 * f) for f in range(3)]
          + [(2, 1, f, 1, 2, 2, 390, 4680 + 390 * f) for f in range(6)]
          + [(2, 2, w, 1, 2, 2, 390, 7020 + 390 * w) for w in range(6)]
          + [(2, 2, w, 2, 2, 1, 390, 9360 + 390 * (w - 6)) for w in range(6, 15)])
    assert [tuple(r) for r in t["SEG"].tolist()] == s1 + s2
    # last row ends at n_kv: 23400 + 9 * 390 = 26910 and 9360 + 9 * 390 = 12870
    assert t["QGRP"][:, 3].tolist() == [23400 + 9 * 390, 9360 + 9 * 390]


def test_ragged_grid_uses_ceil():
    desc = WORKLOADS["wan13b_longhist"]["desc"]
    assert oracle.grid(desc, 4) == (8, 13)
    assert oracle.num_window_tokens(desc) == 9360 + 2340 + 312
    desc3 = WORKLOADS["wan14b_720p"]["desc"]
    assert oracle.grid(desc3, 2) == (23, 40) and oracle.grid(desc3, 4) == (12, 20)


# ---------------------------------------------------------------- pooling


@settings(max_examples=60, deadline=None)
@given(gh=st.integers(1, 9), gw=st.integers(1, 9), f=st.sampled_from([1, 2, 4, 8]),
       c=st.sampled_from([0.75, -3.5, 1.0]))
def test_pool_constant_field_is_identity(gh, gw, f, c):
    x = np.full((gh * gw, 2, 3), c)
    y = oracle.pool_frame(x, gh, gw, f)
    assert y.shape == (-(-gh // f) * -(-gw // f), 2, 3)
    assert np.array_equal(y, np.full_like(y, c))


@settings(max_examples=40, deadline=None)
@given(gh=st.integers(1, 9), gw=st.integers(1, 9), f=st.sampled_from([2, 4]),
       seed=st.integers(0, 1000))
def test_pool_is_affine_and_preserves_mass(gh, gw, f, seed):
    """mean(a x + b) = a mean(x) + b, and each output times its cell count
    sums back to the input total."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((gh * gw, 1, 2))
    y = oracle.pool_frame(x, gh, gw, f)
    assert np.allclose(oracle.pool_frame(3 * x - 2, gh, gw, f), 3 * y - 2, atol=1e-13)
    oh, ow = -(-gh // f), -(-gw // f)
    cnt = np.array([min(f, gh - f * Y) * min(f, gw - f * X) for Y in range(oh) for X in range(ow)])
    assert np.allclose((y * cnt[:, None, None]).sum(0), x.sum(0), atol=1e-12)


def test_two_stage_pool_equals_direct_when_divisible():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((8 * 12, 1, 3))
    two = oracle.pool_frame(oracle.pool_frame(x, 8, 12, 2), 4, 6, 2)
    assert np.allclose(two, oracle.pool_frame(x, 8, 12, 4), atol=1e-14)


# ------------------------------------------------- strided-subsample variant


@settings(max_examples=60, deadline=None)
@given(gh=st.integers(1, 11), gw=st.integers(1, 11), f=st.sampled_from([1, 2, 4, 8]),
       seed=st.integers(0, 1000))
def test_stride_pool_is_grid_slicing(gh, gw, f, seed):
    """Stride f keeps grid rows and columns 0, f, 2f, ...: numpy's img[::f, ::f]."""
    x = np.random.default_rng(seed).standard_normal((gh * gw, 2, 3))
    y = oracle.pool_frame(x, gh, gw, f, "stride")
    ref = x.reshape(gh, gw, 2, 3)[::f, ::f].reshape(-1, 2, 3)
    assert np.array_equal(y, ref)


def test_stride_two_stage_equals_direct_on_every_grid():
    """Two stride-2 steps are one stride-4 step on any grid, ragged 3 mod 4
    included (where the block mean's two-stage route differs)."""
    rng = np.random.default_rng(8)
    for gh, gw in [(8, 12), (7, 11), (3, 5), (15, 26)]:
        x = rng.standard_normal((gh * gw, 1, 2))
        one = oracle.pool_frame(oracle.pool_frame(x, gh, gw, 2, "stride"), -(-gh // 2), -(-gw // 2), 2, "stride")
        assert np.array_equal(one, oracle.pool_frame(x, gh, gw, 4, "stride"))
    x = rng.standard_normal((7 * 11, 1, 2))
    two = oracle.pool_frame(oracle.pool_frame(x, 7, 11, 2), 4, 6, 2)
    assert not np.allclose(two, oracle.pool_frame(x, 7, 11, 4))


@settings(max_examples=30, deadline=None)
@given(gh=st.integers(1, 9), gw=st.integers(1, 9), f=st.sampled_from([2, 4]), seed=st.integers(0, 1000))
def test_stride_equals_mean_on_block_constant_fields(gh, gw, f, seed):
    """A field constant on every f x f block (ragged edge blocks included)
    has its block mean equal to its first cell."""
    oh, ow = -(-gh // f), -(-gw // f)
    c = np.random.default_rng(seed).standard_normal((oh, ow, 1, 2))
    x = np.repeat(np.repeat(c, f, axis=0), f, axis=1)[:gh, :gw].reshape(gh * gw, 1, 2)
    assert np.allclose(oracle.pool_frame(x, gh, gw, f, "stride"), oracle.pool_frame(x, gh, gw, f), atol=1e-14)


def test_stride_variant_keeps_tables_and_changes_outputs():
    """Eq. 5 counts only tokens, so both readings of Subsample give the same
    plan; the outputs differ once a frame is resampled."""
    desc = _desc(3, [1, 2, 4], 6, 9, F=2, S=1, Hh=2, nh=1, d=8)
    sdesc = dict(desc, resample="stride")
    a, b = oracle.tables(desc), oracle.tables(sdesc)
    for k in a:
        assert np.array_equal(a[k], b[k])
    x = _rand_inputs(desc, 6)
    assert not np.allclose(_run(desc, x), _run(sdesc, x))
    with pytest.raises(ValueError):
        oracle.resample_mode(dict(desc, resample="max"))


@settings(max_examples=10, deadline=None)
@given(H=st.integers(1, 7), W=st.integers(1, 7),
       sched=st.lists(st.sampled_from([1, 2, 4]), min_size=1, max_size=3).map(sorted),
       F=st.integers(1, 2), S=st.integers(0, 1), Hh=st.integers(0, 2),
       seed=st.integers(0, 10000))
def test_stride_matches_brute_force_tiny(H, W, sched, F, S, Hh, seed):
    desc = dict(_desc(len(sched), sched, H, W, F=F, S=S, Hh=Hh, nh=2, d=3), resample="stride")
    x = _rand_inputs(desc, seed)
    a = _run(desc, x)
    b = oracle.brute_force_attention(desc, x["q_win"], x["k_sink"], x["v_sink"], x["k_hist"],
                                     x["v_hist"], x["k_win"], x["v_win"])
    assert np.allclose(a, b, atol=1e-12, rtol=0)


# ---------------------------------------------------------------- attention


def test_all_native_scales_is_full_attention():
    """With every scale 1, MSSA is plain softmax attention over
    [sink | history | window] (checked against torch's SDPA in float64)."""
    desc = _desc(3, [1, 1, 1], 5, 7, F=2, S=1, Hh=2, nh=2, d=16)
    x = _rand_inputs(desc, 0)
    out = _run(desc, x)
    k = np.concatenate([x["k_sink"], x["k_hist"], x["k_win"]])
    v = np.concatenate([x["v_sink"], x["v_hist"], x["v_win"]])
    tq = torch.from_numpy(x["q_win"]).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        tq, torch.from_numpy(k).permute(1, 0, 2), torch.from_numpy(v).permute(1, 0, 2))
    assert np.allclose(out, ref.permute(1, 0, 2).numpy(), atol=1e-12, rtol=0)


def test_softmax_rows_sum_to_one():
    desc = _desc(3, [1, 2, 4], 6, 9, F=2, S=1, Hh=1, nh=2, d=8)
    x = _rand_inputs(desc, 1)
    for k in ("v_sink", "v_hist", "v_win"):
        x[k] = np.ones_like(x[k])
    out = _run(desc, x)
    assert np.abs(out - 1).max() <= 1e-12
    # a constant value vector comes out unchanged
    c = np.arange(8, dtype=np.float64)
    for k in ("v_sink", "v_hist", "v_win"):
        x[k] = np.broadcast_to(c, x[k].shape).copy()
    assert np.abs(_run(desc, x) - c).max() <= 1e-12


def test_invariances():
    desc = _desc(2, [1, 2], 4, 6, F=1, S=1, Hh=1, nh=1, d=8)
    x = _rand_inputs(desc, 2)
    base = _run(desc, x)
    # shifting every key by one vector leaves each query's softmax unchanged
    y = dict(x)
    shift = np.random.default_rng(9).standard_normal(8)
    for k in ("k_sink", "k_hist", "k_win"):
        y[k] = x[k] + shift
    assert np.allclose(_run(desc, y), base, atol=1e-12)
    # linear in V
    z = dict(x)
    for k in ("v_sink", "v_hist", "v_win"):
        z[k] = 2 * x[k] + 1
    assert np.allclose(_run(desc, z), 2 * base + 1, atol=1e-12)
    # key order inside a context does not matter
    q = x["q_win"][:, 0]
    kc = oracle.context(desc, 2, x["k_sink"][:, 0], x["k_hist"][:, 0], x["k_win"][:, 0])
    vc = oracle.context(desc, 2, x["v_sink"][:, 0], x["v_hist"][:, 0], x["v_win"][:, 0])
    perm = np.random.default_rng(3).permutation(kc.shape[0])
    a = oracle.attention(q, kc, vc, 0.3)
    b = oracle.attention(q, kc[perm], vc[perm], 0.3)
    assert np.allclose(a, b, atol=1e-13)
    # a single key returns its value
    assert np.allclose(oracle.attention(q, kc[:1], vc[:1], 0.3), np.broadcast_to(vc[0], q.shape))


def test_softmax_scale_default_and_override():
    desc = _desc(1, [1], 2, 2, S=1, Hh=0, d=16)
    assert oracle.softmax_scale(desc) == 0.25
    desc["softmax_scale"] = 0.5
    assert oracle.softmax_scale(desc) == 0.5


@settings(max_examples=12, deadline=None)
@given(H=st.integers(1, 7), W=st.integers(1, 7),
       sched=st.lists(st.sampled_from([1, 2, 4]), min_size=1, max_size=3).map(sorted),
       F=st.integers(1, 2), S=st.integers(0, 1), Hh=st.integers(0, 2),
       seed=st.integers(0, 10000))
def test_matches_brute_force_tiny(H, W, sched, F, S, Hh, seed):
    desc = _desc(len(sched), sched, H, W, F=F, S=S, Hh=Hh, nh=2, d=3)
    x = _rand_inputs(desc, seed)
    a = _run(desc, x)
    b = oracle.brute_force_attention(desc, x["q_win"], x["k_sink"], x["v_sink"], x["k_hist"],
                                     x["v_hist"], x["k_win"], x["v_win"])
    assert np.allclose(a, b, atol=1e-12, rtol=0)


def test_matches_brute_force_ragged_mod4():
    """Grids with a side of 3 mod 4 (where a two-stage 2x2 route would
    differ from direct 4x4 pooling)."""
    desc = _desc(3, [1, 2, 4], 7, 11, F=1, S=1, Hh=1, nh=1, d=4)
    x = _rand_inputs(desc, 11)
    a = _run(desc, x)
    b = oracle.brute_force_attention(desc, x["q_win"], x["k_sink"], x["v_sink"], x["k_hist"],
                                     x["v_hist"], x["k_win"], x["v_win"])
    assert np.allclose(a, b, atol=1e-12, rtol=0)


def test_sampled_queries_equal_full_run():
    desc = _desc(3, [1, 2, 2], 6, 8, F=2, S=1, Hh=2, nh=3, d=8)
    x = _rand_inputs(desc, 4)
    full = _run(desc, x)
    idx = np.array([0, 5, 47, 48, 60, oracle.num_window_tokens(desc) - 1])
    part = _run(desc, x, q_index=idx, heads=[1, 2])
    assert np.allclose(part[idx][:, 1:], full[idx][:, 1:], atol=1e-14, rtol=0)
    assert np.isnan(part[1]).all()


def test_algorithmic_flops_wan13b():
    desc = WORKLOADS["wan13b_layer"]["desc"]
    assert oracle.algorithmic_flops(desc) == 4 * 128 * 12 * (9360 * 26910 + 3510 * 12870)
    assert math.isclose(oracle.algorithmic_flops(desc), 1.8251e12, rel_tol=1e-4)
