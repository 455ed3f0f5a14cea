"""The entry point that allocates nothing (mssa_attention_noalloc) against
mssa_pool_kv + mssa_forward on a caller workspace: bitwise the same output,
on two calls in a row (the second with a smaller plan, so the library's
scratch holds the first call's bytes), and a host-side rejection of a plan
whose workspace exceeds the scratch."""

import numpy as np
import pytest
import torch

from paper_2607_20940_amd import mssa
from paper_2607_20940_amd.workloads import WORKLOADS

from gpu_common import GpuRun, assert_close

pytestmark = pytest.mark.gpu

AMP = 1.0 / np.sqrt(128.0)
SMALL = dict(num_states=4, scales=[1, 1, 2, 4], grid_h=10, grid_w=13, frames_per_state=2, sink_frames=1,
             hist_frames=3, num_heads=3, head_dim=128)


def _noalloc(r):
    d = r.d
    out = torch.full_like(r.out, float("nan"))
    mssa.mssa_attention_noalloc(r.plan, d["q_win"], d["k_sink"], d["v_sink"], d["k_hist"], d["v_hist"],
                                d["k_win"], d["v_win"], out)
    torch.cuda.synchronize()
    return out


def test_noalloc_equals_workspace_path_twice():
    w = WORKLOADS["wan13b_layer"]
    big = GpuRun(w["desc"], w["dtype"], w["seed"], w["amplitude"])
    small = GpuRun(SMALL, "bf16", 7, AMP)
    assert big.info["workspace_bytes"] <= mssa.MSSA_NOALLOC_SCRATCH_BYTES
    for label, r in (("wan13b_layer", big), ("small", small)):
        print(f"[noalloc] {label}", flush=True)
        want = r.run().clone()
        got = _noalloc(r)
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), label
        if label == "small":
            assert_close(r.output(), r.oracle(), "bf16", label)
    # and once more on the first plan, after the smaller one
    got = _noalloc(big)
    assert torch.equal(got.view(torch.int16), big.run().view(torch.int16))


def test_noalloc_q_prescaled():
    """A plan with pre-scaled queries (the layout bench.py times) through the
    no-alloc entry point: bitwise the workspace path's output, which meets
    the oracle on the unscaled queries."""
    w = WORKLOADS["wan13b_layer"]
    r = GpuRun(dict(w["desc"], q_prescaled=True), w["dtype"], w["seed"], w["amplitude"])
    small = GpuRun(dict(SMALL, q_prescaled=True), "bf16", 8, 1.0)
    for label, run in (("wan13b_layer", r), ("small", small)):
        print(f"[noalloc] pre-scaled {label}", flush=True)
        want = run.run().clone()
        got = _noalloc(run)
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), label
    assert_close(small.output(), small.oracle(), "bf16", "small pre-scaled")


def test_noalloc_rejects_plans_beyond_the_scratch():
    w = WORKLOADS["wan14b_720p"]
    plan = mssa.mssa_plan_create(dict(w["desc"], dtype=w["dtype"]))
    assert plan.info()["workspace_bytes"] > mssa.MSSA_NOALLOC_SCRATCH_BYTES
    t = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(mssa.MssaError, match="MSSA_ERR_WORKSPACE"):
        mssa.mssa_attention_noalloc(plan, t, t, t, t, t, t, t, t)
    # a pooled-ring plan is refused before anything is enqueued
    ring = mssa.mssa_plan_create(dict(SMALL, dtype="bf16", flags=mssa.MSSA_PLAN_POOLED_HIST_RING))
    with pytest.raises(mssa.MssaError, match="MSSA_ERR_UNSUPPORTED"):
        mssa.mssa_attention_noalloc(ring, t, t, t, t, t, t, t, t)
