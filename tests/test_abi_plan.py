"""C-ABI checks that need no GPU: the library loads and exports every
declared symbol, the scheduler's tables equal the oracle's bit for bit, and
invalid calls are rejected before anything is enqueued."""

import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from paper_2607_20940_amd import mssa
from paper_2607_20940_amd.workloads import STREAMING, WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "libmssa.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mssa_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert set(names) == set(mssa.EXPORTS)
    for name in names:
        assert hasattr(mssa.lib, name), name


def _plan(desc, **kw):
    d = dict(desc)
    d.update(kw)
    return mssa.mssa_plan_create(d)


def _assert_tables_equal(desc):
    got = _plan(desc).tables()
    want = oracle.tables(desc)
    for key in ("GRID", "QGRP", "SEG", "TOTAL"):
        assert np.array_equal(got[key], want[key]), key


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_tables_bit_exact_workloads(name):
    _assert_tables_equal(WORKLOADS[name]["desc"])


@pytest.mark.parametrize("hist", [6, 9, 12, 15, 18, 21])
def test_tables_bit_exact_streaming_history_lengths(hist):
    _assert_tables_equal(dict(STREAMING["layer"], hist_frames=hist))


@settings(max_examples=150, deadline=None)
@given(H=st.integers(1, 70), W=st.integers(1, 90),
       sched=st.lists(st.sampled_from([1, 2, 4, 8, 16]), min_size=1, max_size=8).map(sorted),
       F=st.integers(1, 4), S=st.integers(0, 4), Hh=st.integers(0, 25),
       nh=st.integers(1, 48), d=st.sampled_from([64, 128]))
def test_tables_bit_exact_fuzz(H, W, sched, F, S, Hh, nh, d):
    desc = dict(num_states=len(sched), scales=sched, grid_h=H, grid_w=W, frames_per_state=F,
                sink_frames=S, hist_frames=Hh, num_heads=nh, head_dim=d)
    _assert_tables_equal(desc)


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_info_matches_oracle(name):
    w = WORKLOADS[name]
    desc = dict(w["desc"], dtype=w["dtype"])
    info = _plan(desc).info()
    assert info["n_q"] == oracle.num_window_tokens(desc)
    assert info["n_sink_tok"] == oracle.num_sink_tokens(desc)
    assert info["n_hist_tok"] == oracle.num_hist_tokens(desc)
    assert info["flops_alg"] == oracle.algorithmic_flops(desc)
    groups = oracle.tables(desc)["QGRP"]
    assert info["group_scale"] == groups[:, 0].tolist()
    assert info["n_kv"] == groups[:, 3].tolist()
    # pooled tokens per scale: everything in the context that is resampled
    for g, s in enumerate(info["group_scale"]):
        rows = [r for r in oracle.context_rows(desc, s) if r[4] > 1 and r[0] != oracle.KIND_SINK]
        assert info["pooled_tokens"][g] == sum(r[5] for r in rows)


def test_pool_bytes_wan13b():
    desc = WORKLOADS["wan13b_layer"]["desc"]
    info = _plan(desc).info()
    ld = 12 * 128 * 2
    read = 9360 + 2 * 3 * 1560          # 6 history frames + window states 1-2
    write = 6 * 390 + 6 * 390            # both pooled to 15x26
    assert info["pool_bytes_alg"] == 2 * (read + write) * ld


@pytest.mark.parametrize("bad, status", [
    (dict(num_states=0), mssa.MSSA_ERR_INVALID_ARG),
    (dict(num_states=9), mssa.MSSA_ERR_INVALID_ARG),
    (dict(scales=[1, 1, 3, 3, 3]), mssa.MSSA_ERR_UNSUPPORTED),
    (dict(scales=[2, 1, 2, 2, 2]), mssa.MSSA_ERR_UNSUPPORTED),
    (dict(scales=[1, 1, 2, 2, 128]), mssa.MSSA_ERR_UNSUPPORTED),
    (dict(head_dim=96), mssa.MSSA_ERR_UNSUPPORTED),
    (dict(grid_h=0), mssa.MSSA_ERR_INVALID_ARG),
    (dict(frames_per_state=0), mssa.MSSA_ERR_INVALID_ARG),
    (dict(sink_frames=-1), mssa.MSSA_ERR_INVALID_ARG),
    (dict(num_heads=0), mssa.MSSA_ERR_INVALID_ARG),
    (dict(dtype=7), mssa.MSSA_ERR_INVALID_ARG),
    (dict(softmax_scale=float("nan")), mssa.MSSA_ERR_INVALID_ARG),
    (dict(grid_h=40000, grid_w=40000, hist_frames=4), mssa.MSSA_ERR_UNSUPPORTED),
])
def test_invalid_descriptors(bad, status):
    with pytest.raises(mssa.MssaError) as e:
        _plan(WORKLOADS["wan13b_layer"]["desc"], **bad)
    assert e.value.status == status
    assert mssa.lib.mssa_last_error().decode()


def test_calls_rejected_before_launch():
    """Every failure below is detected on the host; no kernel is enqueued
    (no GPU is touched: all pointers are fake, misaligned or NULL)."""
    plan = _plan(WORKLOADS["wan13b_layer"]["desc"])
    info = plan.info()
    fake = 1 << 20  # 256-byte aligned, never dereferenced
    ws = info["workspace_bytes"]
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_kv(plan, fake, fake, fake, fake, fake, ws - 1, stream=0)
    assert e.value.status == mssa.MSSA_ERR_WORKSPACE
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_kv(plan, None, fake, fake, fake, fake, ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_kv(plan, fake, fake, fake, fake, fake + 16, ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward(plan, fake, fake, fake, fake, fake, fake, fake, fake, fake,
                          workspace_bytes=0, stream=0)
    assert e.value.status == mssa.MSSA_ERR_WORKSPACE
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward(plan, fake, None, fake, fake, fake, fake, fake, fake, fake,
                          workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward(plan, fake + 8, fake, fake, fake, fake, fake, fake, fake, fake + 4096,
                          workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward(plan, fake, fake, fake, fake, fake, fake, fake, fake, fake,
                          workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG  # out aliases q_win
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_plan_query(mssa.Plan(None, {}))
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG


def test_table_buffer_too_small():
    import ctypes
    plan = _plan(WORKLOADS["tiny_f32"]["desc"])
    need = ctypes.c_int64()
    buf = (ctypes.c_int64 * 4)()
    st_ = mssa.lib.mssa_plan_tables(plan.handle, buf, 4, ctypes.byref(need))
    assert st_ == mssa.MSSA_ERR_INVALID_ARG and need.value > 4


RING = mssa.MSSA_PLAN_POOLED_HIST_RING


@pytest.mark.parametrize("name", ["wan13b_layer", "wan13b_longhist", "wan14b_720p"])
def test_pooled_hist_ring_plan_same_context(name):
    """A plan whose pooled history lives in the caller's rings has the same
    context tables (the same Eq. 4 construction) and pools only window
    frames: its workspace and pool traffic drop by the history's share."""
    desc = WORKLOADS[name]["desc"]
    plain, ring = _plan(desc), _plan(desc, flags=RING)
    a, b = plain.tables(), ring.tables()
    for key in ("GRID", "QGRP", "SEG", "TOTAL"):
        assert np.array_equal(a[key], b[key]), key
    ia, ib = plain.info(), ring.info()
    assert ib["flops_alg"] == ia["flops_alg"]
    nh, d = desc["num_heads"], desc["head_dim"]
    tok1 = desc["grid_h"] * desc["grid_w"]
    ld_bytes = nh * d * 2
    hist_pooled = 0
    for s in ia["group_scale"]:
        if s > 1:
            hist_pooled += desc["hist_frames"] * (-(-desc["grid_h"] // s)) * (-(-desc["grid_w"] // s))
    assert ia["pool_bytes_alg"] - ib["pool_bytes_alg"] == 2 * (desc["hist_frames"] * tok1 + hist_pooled) * ld_bytes
    for g, s in enumerate(ia["group_scale"]):
        hp = desc["hist_frames"] * (-(-desc["grid_h"] // s)) * (-(-desc["grid_w"] // s)) if s > 1 else 0
        assert ib["pooled_tokens"][g] == ia["pooled_tokens"][g] - hp
    assert ib["workspace_bytes"] < ia["workspace_bytes"]


@pytest.mark.parametrize("name", ["tiny_f32", "wan13b_layer", "wan13b_longhist", "wan14b_720p"])
def test_strided_plan_same_tables(name):
    """The strided-subsample plan builds the same Eq. 4 context (tables,
    workspace, FLOP) as the block-mean plan, equal to the oracle's tables for
    resample="stride"; its pool reads one source token per pooled token."""
    desc = WORKLOADS[name]["desc"]
    mean, stride = _plan(desc), _plan(desc, resample="stride")
    a, b = mean.tables(), stride.tables()
    want = oracle.tables(dict(desc, resample="stride"))
    for key in ("GRID", "QGRP", "SEG", "TOTAL"):
        assert np.array_equal(a[key], b[key]), key
        assert np.array_equal(b[key].reshape(want[key].shape), want[key]), key
    ia, ib = mean.info(), stride.info()
    for key in ("flops_alg", "workspace_bytes", "pooled_tokens", "n_kv"):
        assert ia[key] == ib[key], key
    row = desc["num_heads"] * desc["head_dim"] * 2  # bf16 plan
    assert ib["pool_bytes_alg"] == 2 * 2 * sum(ib["pooled_tokens"]) * row
    with pytest.raises(ValueError):
        _plan(desc, resample="max")


def test_pooled_hist_ring_calls_checked():
    """Ring entry points refuse plans without the flag and the plain ones
    refuse ring plans, before anything is enqueued; unknown flags are
    rejected at plan creation."""
    desc = WORKLOADS["wan13b_layer"]["desc"]
    with pytest.raises(mssa.MssaError) as e:
        _plan(desc, flags=16)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    plain, ring = _plan(desc), _plan(desc, flags=RING)
    fake = 1 << 20
    ws = ring.info()["workspace_bytes"]
    pools = [None, fake]  # group 0 is scale 1, group 1 scale 2
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward(ring, fake, fake, fake, fake, fake, fake, fake, fake, fake + 4096,
                          workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward_ring(plain, fake, fake, fake, fake, fake, pools, pools, fake, fake, fake,
                               fake + 4096, workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_forward_ring(ring, fake, fake, fake, fake, fake, [None, None], pools, fake, fake, fake,
                               fake + 4096, workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_hist_append_ring(plain, fake, fake, fake, fake, fake, pools, pools, mssa.Ring(21),
                                   workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_hist_append_ring(ring, fake, fake, fake, fake, fake, [None, None], pools,
                                   mssa.Ring(21), workspace_bytes=ws, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_hist_ring(plain, fake, fake, pools, pools, stream=0)
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_hist_ring(ring, fake, fake, [None, None], pools, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG


def test_backward_calls_checked():
    """Bad calls are rejected before anything is enqueued."""
    desc = dict(num_states=2, scales=[1, 2], grid_h=12, grid_w=8, frames_per_state=2, sink_frames=0,
                hist_frames=2, num_heads=2, head_dim=128)
    plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    fake = 1 << 20
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_backward(plan, fake, None, None, fake, fake, fake, fake, fake, fake, fake, fake,
                           fake + 4096, None, None, fake + 8192, fake + 8192, fake + 8192, fake + 8192,
                           workspace_bytes=16, stream=0)
    assert e.value.status == mssa.MSSA_ERR_WORKSPACE
    wsz = mssa.mssa_backward_workspace_size(plan)
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_backward(plan, fake, None, None, fake, fake, fake, fake, fake, fake, fake, fake,
                           fake, None, None, fake + 8192, fake + 8192, fake + 8192, fake + 8192,
                           workspace_bytes=wsz, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG  # dq aliases q


def test_tier_calls_checked():
    """Tier entry points validate before enqueuing anything."""
    desc = dict(num_states=2, scales=[1, 2], grid_h=6, grid_w=8, frames_per_state=1, sink_frames=1,
                hist_frames=0, num_heads=2, head_dim=64)
    plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    tier = mssa.tier_desc(16, 2, 128)
    need = mssa.mssa_tier_workspace_size(plan, tier)
    # patch rows of both tiers: 48 tokens x 64 features + 12 tokens x 256 features, bf16
    assert need == (48 * 64 * 2 + 255) // 256 * 256 + (12 * 256 * 2 + 255) // 256 * 256
    f32 = mssa.mssa_plan_create(dict(desc, dtype="f32"))
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_tier_workspace_size(f32, tier)
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_tier_workspace_size(plan, mssa.tier_desc(16, 2, 100))
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_tier_workspace_size(plan, mssa.tier_desc(1, 1, 64))  # C p^2 = 1
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    fake = 1 << 20
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_patch_embed(plan, tier, fake, [fake, fake], [fake, fake], fake, fake, workspace_bytes=16, stream=0)
    assert e.value.status == mssa.MSSA_ERR_WORKSPACE
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_qkv_project(10, 128, fake, fake, fake, fake, fake + 4096, fake + 8192, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG  # q aliases x
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_qkv_project(10, 12, fake, fake, fake, fake + 4096, fake + 8192, fake + 12288, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_qkv_project_scaled(10, 128, fake, fake, fake, float("nan"), fake + 4096, fake + 8192,
                                     fake + 12288, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG


def _context_runs(seg_rows):
    """Token counts of a context's runs: maximal stretches of consecutive SEG
    rows read from one buffer, i.e. of one class among sink frames, native
    history frames, resampled frames (history or window, which share one
    pooled block) and native window frames."""
    runs, last = [], None
    for _, kind, _, _, _, factor, n_tok, _ in seg_rows:
        cls = "sink" if kind == 0 else ("pooled" if factor > 1 else ("hist" if kind == 1 else "win"))
        if cls == last:
            runs[-1] += int(n_tok)
        else:
            runs.append(int(n_tok))
        last = cls
    return runs


def test_backward_workspace_layout():
    """The backward workspace is the forward's, then rowsum(dO * O) and lse in
    log2 units ([heads, n_q] fp32 each), then fp32 K and V context gradients
    per query group, then (bf16 plans) per group the dS tiles: 4 KB each, per
    head, 32-query block (an even count) and 64-key stage of the context's
    runs; every region 256-byte aligned."""
    def a256(x):
        return (x + 255) // 256 * 256

    for d in (128, 64):
        for dtype in ("bf16", "f32"):
            desc = dict(num_states=4, scales=[1, 1, 2, 4], grid_h=10, grid_w=13, frames_per_state=2,
                        sink_frames=1, hist_frames=3, num_heads=3, head_dim=d)
            plan = mssa.mssa_plan_create(dict(desc, dtype=dtype))
            info = plan.info()
            nh, nq = desc["num_heads"], info["n_q"]
            want = a256(info["workspace_bytes"]) + 2 * a256(nh * nq * 4)
            want += sum(2 * a256(n_kv * nh * d * 4)
                        for n_kv in info["n_kv"][: info["n_groups"]])
            if dtype == "bf16":
                want += _ds_bytes(plan, nh)
            assert mssa.mssa_backward_workspace_size(plan) == want


def _ds_bytes(plan, nh):
    """dS tile bytes of a bf16 plan: per group, per head of a chunk, 32-query
    block (an even count) and 64-key stage of the context's runs, 4 KB; a
    chunk is as many whole heads as fit in 8 GiB, at least one."""
    t = mssa.mssa_plan_tables(plan)
    per_group = []
    for scale, q0, q1, n_kv in t["QGRP"]:
        runs = _context_runs([r for r in t["SEG"] if r[0] == scale])
        assert sum(runs) == n_kv
        stages = sum(-(-n // 64) for n in runs)
        qblocks = 2 * -(-(q1 - q0) // 64)
        per_group.append(qblocks * stages * 4096)
    heads = max(1, min(nh, (8 << 30) // sum(per_group)))
    return sum((heads * b + 255) // 256 * 256 for b in per_group)


def test_backward_workspace_chunks_heads():
    """At the three layer workloads the dS tiles of whole heads fit in 8 GiB:
    all 12 heads of the 1.3B-shaped layer, 8 of the 21-frame history, 2 of the
    14B-shaped 720p layer's 40."""
    from paper_2607_20940_amd.workloads import WORKLOADS
    for name, heads in (("wan13b_layer", 12), ("wan13b_longhist", 8), ("wan14b_720p", 2)):
        desc = WORKLOADS[name]["desc"]
        plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
        info = plan.info()
        nh, nq, d = desc["num_heads"], info["n_q"], desc["head_dim"]
        base = (info["workspace_bytes"] + 255) // 256 * 256 + 2 * ((nh * nq * 4 + 255) // 256 * 256)
        base += sum(2 * ((n_kv * nh * d * 4 + 255) // 256 * 256) for n_kv in info["n_kv"][: info["n_groups"]])
        ds = mssa.mssa_backward_workspace_size(plan) - base
        assert ds == _ds_bytes(plan, nh)
        t = mssa.mssa_plan_tables(plan)
        per_head = sum(2 * -(-(q1 - q0) // 64) * sum(-(-n // 64) for n in _context_runs([r for r in t["SEG"] if r[0] == s]))
                       * 4096 for s, q0, q1, _ in t["QGRP"])
        assert heads * per_head <= ds < (heads + 1) * per_head and heads * per_head <= 8 << 30


HEAD = mssa.MSSA_PLAN_HEAD_IN_RING


def test_head_in_ring_plan_rules():
    """The copy-free cache roll needs pooled rings, a native head state and
    bf16; its plan keeps the Eq. 4 tables and FLOP, and its pool reads state
    1 once and writes it pooled to every coarser scale."""
    desc = STREAMING["layer"]
    for bad in (dict(flags=HEAD), dict(flags=RING | HEAD, scales=[2, 2, 2, 4, 4]),
                dict(flags=RING | HEAD, dtype="f32")):
        with pytest.raises(mssa.MssaError) as e:
            _plan(dict(desc, hist_frames=6), **bad)
        assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    ring, head = _plan(dict(desc, hist_frames=21), flags=RING), _plan(dict(desc, hist_frames=21), flags=RING | HEAD)
    a, b = ring.tables(), head.tables()
    for key in ("GRID", "QGRP", "SEG", "TOTAL"):
        assert np.array_equal(a[key], b[key]), key
    ia, ib = ring.info(), head.info()
    assert ia["flops_alg"] == ib["flops_alg"]
    # state 1 (3 native frames) leaves the workspace's pooled block
    assert ib["pooled_tokens"][1] == ia["pooled_tokens"][1] - 3 * 390
    # pool traffic: the same, state 1 now pooled into the rings (read 3 x 1560,
    # write 3 x 390 tokens, K and V)
    assert ib["pool_bytes_alg"] == ia["pool_bytes_alg"]


def test_head_ring_roll_and_state_checks():
    """The roll is host-only arithmetic on (count, spare); ring states that
    break the rules are rejected before anything is enqueued."""
    desc = dict(STREAMING["layer"], dtype="bf16")
    plans = {h: _plan(dict(desc, hist_frames=h), flags=RING | HEAD) for h in range(0, 22, 3)}
    r = mssa.HeadRing(24, count=6)
    seen = []
    for _ in range(12):
        mssa.mssa_head_ring_roll(plans[r.count], r)
        seen.append((r.count, r.spare))
    assert seen == [(9, 9), (12, 12), (15, 15), (18, 18), (21, 21), (21, 0), (21, 3), (21, 6), (21, 9),
                    (21, 12), (21, 15), (21, 18)]
    fake = 1 << 20
    pools = [None, fake]
    for frames, count, spare in ((23, 6, 6), (24, 6, 7), (24, 6, 24), (24, 9, 6), (3, 0, 0)):
        with pytest.raises(mssa.MssaError) as e:
            mssa.mssa_forward_head_ring(plans[6], fake, fake, fake, fake, fake, pools, pools, fake, fake, fake,
                                        fake + 4096, mssa.HeadRing(frames, count, spare), workspace_bytes=1 << 30,
                                        stream=0)
        assert e.value.status == mssa.MSSA_ERR_INVALID_ARG, (frames, count, spare)
        with pytest.raises(mssa.MssaError) as e:
            mssa.mssa_head_ring_roll(plans[6], mssa.HeadRing(frames, count, spare))
        assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_kv_head_ring(_plan(dict(desc, hist_frames=6), flags=RING), fake, fake, fake, fake, pools,
                                    pools, fake, mssa.HeadRing(24, 6), workspace_bytes=1 << 30, stream=0)
    assert e.value.status == mssa.MSSA_ERR_UNSUPPORTED
    with pytest.raises(mssa.MssaError) as e:
        mssa.mssa_pool_kv_head_ring(plans[6], fake, fake, fake, fake, [None, None], pools, fake,
                                    mssa.HeadRing(24, 6), workspace_bytes=1 << 30, stream=0)
    assert e.value.status == mssa.MSSA_ERR_INVALID_ARG
