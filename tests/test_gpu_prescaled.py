"""Queries supplied pre-scaled by softmax_scale * log2(e)
(MSSA_PLAN_Q_PRESCALED): the same Eq. 4 attention as the plain path, so the
HIP output is compared with the fp64 oracle fed the unscaled queries
q = q' / (softmax_scale log2 e), at the tolerances of the plain path, on
ragged shapes, split items, logits from tiny to 16x spread, full-size
sampled rows, and the backward (dq' = dq / (softmax_scale log2 e))."""

import numpy as np
import pytest

from gpu_common import GpuRun, assert_close, assert_close_by_group
from test_gpu_parity import AMP, SMALL, _groups, _sample_rows
from paper_2607_20940_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def _check(desc, dtype, seed, amp, label, attention_blocks=0):
    desc = dict(desc, q_prescaled=True)
    print(f"[prescaled] {label} desc={desc} dtype={dtype} seed={seed}", flush=True)
    r = GpuRun(desc, dtype, seed, amp, attention_blocks=attention_blocks)
    r.run()
    e = assert_close(r.output(), r.oracle(), dtype, label)
    print(f"[prescaled] {label} ok {e}", flush=True)
    return r


@pytest.mark.parametrize("name", ["ragged_3level_d128", "ragged_3level_d64", "paper_schedule_small",
                                  "no_history", "tiny_runs", "eight_states"])
def test_prescaled_small(name):
    desc, seed = SMALL[name]
    _check(desc, "bf16", seed + 500, AMP, name)


@pytest.mark.parametrize("mult", [1.0, 4.0, 16.0])
def test_prescaled_large_logits(mult):
    """Unit-variance inputs with softmax_scale = mult / sqrt(d): the first
    tile's max path and the lazy rescale run often; no accuracy is lost
    against the plain path's bound."""
    desc, seed = SMALL["ragged_3level_d128"]
    desc = dict(desc, softmax_scale=mult / np.sqrt(128.0))
    _check(desc, "bf16", seed + 600, 1.0, f"logits_x{mult:g}")


def test_prescaled_very_negative_logits():
    """Every query's scores far below zero (q' = -|q'| against positive keys
    would underflow exp2 without a max): the first tile of each piece must
    still set the running max."""
    desc, seed = SMALL["paper_schedule_small"]
    desc = dict(desc, softmax_scale=64.0 / np.sqrt(128.0))
    r = GpuRun(dict(desc, q_prescaled=True), "bf16", seed + 700, 1.0)
    from paper_2607_20940_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits
    import torch
    for k in ("k_sink", "k_hist", "k_win"):
        if r.x[k] is not None:
            r.x[k] = f32_to_bf16_bits(np.abs(bf16_bits_to_f32(r.x[k])) + 0.5)
    r.x["q_win"] = f32_to_bf16_bits(-np.abs(bf16_bits_to_f32(r.x["q_win"])) - 0.5)
    from gpu_common import to_device
    r.d = {k: to_device(v, "bf16") for k, v in r.x.items()}
    r.out = torch.empty_like(r.d["q_win"])
    r.run()
    ref = r.oracle()
    assert assert_close(r.output(), ref, "bf16", "very_negative")


@pytest.mark.parametrize("ranges", [2, 7, 1000])
def test_prescaled_split_items(ranges):
    """Items split over many persistent blocks: the partial records carry the
    running max of the pre-scaled path and merge in the combine kernel."""
    desc, seed = SMALL["ragged_3level_d128"]
    _check(desc, "bf16", seed + 800, 1.0, f"ranges{ranges}", attention_blocks=ranges)


def test_prescaled_f32():
    """fp32 plans accept the flag (the correctness path takes the base-2
    logits as they come)."""
    desc, seed = SMALL["ragged_3level_d128"]
    _check(desc, "f32", seed + 900, 1.0, "f32")


@pytest.mark.parametrize("name", ["wan13b_layer", "wan13b_longhist", "wan14b_720p"])
def test_prescaled_full_size_sampled(name):
    """The layer workloads at full size with pre-scaled queries (the layout
    bench.py times): sampled rows of three heads against the oracle."""
    w = WORKLOADS[name]
    desc = dict(w["desc"], q_prescaled=True)
    print(f"[prescaled] full-size {name}", flush=True)
    r = GpuRun(desc, w["dtype"], w["seed"] + 1000, w["amplitude"])
    r.run()
    rng = np.random.default_rng(321)
    rows = _sample_rows(r.info, rng)
    nh = w["desc"]["num_heads"]
    heads = sorted({0, nh - 1, int(rng.integers(0, nh))})
    ref = r.oracle(heads=heads, q_index=rows)[rows]
    got = r.output()[rows][:, heads]
    e = assert_close_by_group(got, ref, rows, _groups(r.info), w["dtype"], name + "_prescaled")
    print(f"[prescaled] full-size {name} rows={len(rows)} heads={heads} {e}", flush=True)


def test_prescaled_matches_plain_within_rounding():
    """The plain and pre-scaled paths on the same unscaled queries differ only
    by the rounding of q' (one bf16 rounding of scale log2(e) q, applied here
    on the host): both meet the oracle, and their outputs stay close."""
    desc, seed = SMALL["ragged_3level_d128"]
    plain = GpuRun(desc, "bf16", seed + 1100, AMP)
    plain.run()
    pre = _check(desc, "bf16", seed + 1100, AMP, "same_draws")
    d = np.abs(plain.output() - pre.output()).max()
    assert d <= 2e-2, d
