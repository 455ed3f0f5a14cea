"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20940_amd.inputs import make_inputs, to_f64
from paper_2607_20940_amd.workloads import WORKLOADS, input_shapes

from gpu_common import GpuRun, assert_close, assert_close_by_group, errors
from tolerances import sample_rows

pytestmark = pytest.mark.gpu

AMP = 1.0 / np.sqrt(128.0)


def _desc(T, scales, H, W, F=1, S=1, Hh=1, nh=1, d=128):
    return dict(num_states=T, scales=list(scales), grid_h=H, grid_w=W, frames_per_state=F,
                sink_frames=S, hist_frames=Hh, num_heads=nh, head_dim=d)


def _full_check(desc, dtype, seed, amp, label, attention_blocks=0):
    print(f"[parity] {label} desc={desc} dtype={dtype} seed={seed}", flush=True)
    r = GpuRun(desc, dtype, seed, amp, attention_blocks=attention_blocks)
    r.run()
    e = assert_close(r.output(), r.oracle(), dtype, label)
    print(f"[parity] {label} ok {e}", flush=True)
    return r


# ------------------------------------------------------------------ fp32


def test_tiny_f32_workload():
    w = WORKLOADS["tiny_f32"]
    _full_check(w["desc"], "f32", w["seed"], w["amplitude"], "tiny_f32")


def test_f32_head_dim_128_ragged():
    _full_check(_desc(3, [1, 2, 4], 7, 11, F=2, S=1, Hh=2, nh=2, d=128), "f32", 21, 1.0, "f32_d128")


# ------------------------------------------------------------------ bf16, full outputs

SMALL = {
    # several 256-query tiles, 64-key tiles and ragged tails at every level
    "ragged_3level_d128": (_desc(4, [1, 1, 2, 4], 10, 13, F=2, S=1, Hh=3, nh=3, d=128), 7),
    "ragged_3level_d64": (_desc(4, [1, 1, 2, 4], 10, 13, F=2, S=1, Hh=3, nh=3, d=64), 8),
    "paper_schedule_small": (_desc(5, [1, 1, 2, 2, 2], 6, 10, F=3, S=1, Hh=2, nh=2, d=128), 9),
    "no_history": (_desc(3, [1, 2, 2], 9, 9, F=2, S=2, Hh=0, nh=2, d=128), 10),
    "no_sink": (_desc(2, [1, 2], 12, 8, F=2, S=0, Hh=2, nh=2, d=128), 11),
    "single_state_native": (_desc(1, [1], 11, 17, F=3, S=1, Hh=1, nh=2, d=128), 12),
    "all_coarse_equal": (_desc(3, [2, 2, 2], 9, 14, F=1, S=1, Hh=2, nh=1, d=128), 13),
    "tiny_runs": (_desc(3, [1, 2, 4], 2, 3, F=1, S=1, Hh=1, nh=1, d=128), 14),
    "eight_states": (_desc(8, [1, 1, 2, 2, 4, 4, 8, 8], 16, 16, F=1, S=1, Hh=1, nh=1, d=64), 15),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_bf16_small_full(name):
    desc, seed = SMALL[name]
    _full_check(desc, "bf16", seed, AMP, name)


@pytest.mark.parametrize("name", ["ragged_3level_d128", "paper_schedule_small"])
def test_bf16_stress_unit_logits(name):
    """N(0,1) inputs: logits with unit spread, so the softmax is far from
    uniform and the online rescaling is exercised."""
    desc, seed = SMALL[name]
    _full_check(desc, "bf16", seed + 100, 1.0, name + "_stress")


@pytest.mark.parametrize("mult", [4.0, 16.0])
def test_bf16_large_logits(mult):
    """N(0,1) inputs with softmax_scale = mult / sqrt(d): logits spread
    ~mult, most of the weight on a few keys."""
    desc, seed = SMALL["ragged_3level_d128"]
    desc = dict(desc, softmax_scale=mult / np.sqrt(128.0))
    _full_check(desc, "bf16", seed + 200, 1.0, f"large_logits_x{mult:g}")


@pytest.mark.parametrize("ranges", [1, 2, 3, 7, 97, 1000])
@pytest.mark.parametrize("name", ["ragged_3level_d128", "ragged_3level_d64", "tiny_runs"])
def test_bf16_forced_tile_ranges(name, ranges):
    """Items split across 1..many persistent attention blocks (tile ranges;
    partial records merged by the combine kernel) give the same result."""
    desc, seed = SMALL[name]
    _full_check(desc, "bf16", seed + 300, 1.0, f"{name}_ranges{ranges}", attention_blocks=ranges)


def test_zero_output_fails_guard():
    """The comparison rejects an all-zero output."""
    desc, seed = SMALL["paper_schedule_small"]
    r = GpuRun(desc, "bf16", seed, AMP)
    ref = r.oracle()
    with pytest.raises(AssertionError):
        assert_close(np.zeros_like(ref), ref, "bf16")


def test_deterministic():
    desc, seed = SMALL["ragged_3level_d128"]
    r = GpuRun(desc, "bf16", seed, AMP)
    a = r.run().clone()
    b = r.run(torch.empty_like(a))
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_deterministic_full_size():
    """Bitwise-equal outputs over three passes of the 21-frame-history layer
    in the benchmark's launch configuration (persistent schedule, split
    items merged in range order)."""
    w = WORKLOADS["wan13b_longhist"]
    print("[parity] full-size determinism", flush=True)
    r = GpuRun(w["desc"], w["dtype"], w["seed"], w["amplitude"])
    a = r.run().clone()
    for _ in range(2):
        b = r.run(torch.empty_like(a))
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


# ------------------------------------------------------------------ pooling


def _check_pool(r, label):
    """Pooled workspace vs the oracle's fp64 means rounded to bf16."""
    x = r.oracle_inputs()
    want = oracle.pooled_kv(r.desc, x["k_hist"], x["k_win"])
    want_v = oracle.pooled_kv(r.desc, x["v_hist"], x["v_win"])
    info = r.info
    n_ulp_diff = 0
    total = 0
    for g, s in enumerate(info["group_scale"]):
        if info["pooled_tokens"][g] == 0:
            continue
        rows = [row for row in oracle.context_rows(r.desc, s)
                if row[0] != oracle.KIND_SINK and row[4] > 1]
        for which, ref_map in (("k", want), ("v", want_v)):
            got = r.pooled(g, which)
            ref = np.concatenate([ref_map[(row[0], row[1], row[3])] for row in rows])
            assert got.shape == ref.shape
            ref_b = to_f64(_round_bf16(ref), "bf16") if r.dtype == "bf16" else ref
            diff = np.abs(got - ref_b)
            if r.dtype == "bf16":
                ulp = np.abs(ref_b) * 2.0 ** -7 + 1e-30
                assert (diff <= ulp).all(), f"{label}: pooled {which} off by more than 1 bf16 ulp"
                n_ulp_diff += int((diff > 0).sum())
                total += diff.size
            else:
                assert diff.max() <= 1e-6 * max(1.0, np.abs(ref).max())
    if total:
        assert n_ulp_diff <= 1e-4 * total, f"{label}: {n_ulp_diff}/{total} pooled values differ"


def _round_bf16(x64):
    from paper_2607_20940_amd.inputs import f32_to_bf16_bits
    # exact RNE to bf16 from float64: via float32 is exact enough except on
    # float32 ties, which the 1-ulp bound covers
    return f32_to_bf16_bits(x64.astype(np.float32))


@pytest.mark.parametrize("name", ["ragged_3level_d128", "ragged_3level_d64", "eight_states", "all_coarse_equal"])
def test_pool_small(name):
    """Pooled K/V: frames pooled by 2 and by 4 in one pass (the 3-level
    schedules, at both head dims), factor 2 alone, and factor 8 (generic)."""
    desc, seed = SMALL[name]
    r = GpuRun(desc, "bf16", seed, 1.0)
    r.run()
    _check_pool(r, name)


def test_pool_two_levels_sides_3_mod_4():
    """Both grid sides 3 mod 4: the last 4 x 4 block of every row and column
    holds a whole 2 x 2 cell and a 1-wide one."""
    desc = _desc(3, [1, 2, 4], 7, 11, F=2, S=1, Hh=2, nh=2, d=128)
    r = GpuRun(desc, "bf16", 31, 1.0)
    r.run()
    _check_pool(r, "pool_7x11")
    e = assert_close(r.output(), r.oracle(), "bf16", "pool_7x11_attention")
    print(f"[parity] pool_7x11 attention ok {e}", flush=True)


def test_pool_f32():
    r = GpuRun(_desc(3, [1, 2, 4], 7, 11, F=2, S=1, Hh=2, nh=2, d=64), "f32", 5, 1.0)
    r.run()
    _check_pool(r, "pool_f32")


# ------------------------------------------------------------------ full-size workloads


def _groups(info):
    return list(zip(info["group_scale"], info["q_begin"], info["q_end"]))


def _sample_rows(info, rng, n_random=48):
    return sample_rows(_groups(info), info["n_q"], rng, n_random)


@pytest.mark.parametrize("name", ["wan13b_layer", "wan13b_longhist", "wan14b_720p"])
def test_full_size_sampled(name):
    w = WORKLOADS[name]
    print(f"[parity] full-size {name}", flush=True)
    r = GpuRun(w["desc"], w["dtype"], w["seed"], w["amplitude"])
    r.run()
    rng = np.random.default_rng(123)
    rows = _sample_rows(r.info, rng)
    nh = w["desc"]["num_heads"]
    heads = sorted({0, nh - 1, int(rng.integers(0, nh))})
    ref = r.oracle(heads=heads, q_index=rows)[rows]
    got = r.output()[rows][:, heads]
    e = assert_close_by_group(got, ref, rows, _groups(r.info), w["dtype"], name)
    print(f"[parity] {name} rows={len(rows)} heads={heads} {e}", flush=True)
    # On these N(0,1)/sqrt(128) inputs an all-zero output meets the absolute
    # bounds; the relative guard is what rejects it.
    z = errors(np.zeros_like(ref), ref)
    assert z["max_abs"] <= 2e-2 and z["mean_abs"] <= 2e-3
    with pytest.raises(AssertionError):
        assert_close(np.zeros_like(ref), ref, w["dtype"])
    if name == "wan13b_layer":
        _check_pool(r, name)


# ------------------------------------------------------------------ strided-subsample variant


def _check_pool_exact(r, label):
    """Strided pooled blocks are copies of source tokens: bit-equal to the
    oracle's picks of the same input values."""
    x = r.oracle_inputs()
    want = {"k": oracle.pooled_kv(r.desc, x["k_hist"], x["k_win"]),
            "v": oracle.pooled_kv(r.desc, x["v_hist"], x["v_win"])}
    n = 0
    for g, s in enumerate(r.info["group_scale"]):
        if r.info["pooled_tokens"][g] == 0:
            continue
        rows = [row for row in oracle.context_rows(r.desc, s) if row[0] != oracle.KIND_SINK and row[4] > 1]
        for which in ("k", "v"):
            ref = np.concatenate([want[which][(row[0], row[1], row[3])] for row in rows])
            got = r.pooled(g, which)
            assert got.shape == ref.shape
            assert np.array_equal(got, ref), f"{label}: strided pooled {which} of group {g} differs"
            n += got.size
    assert n > 0
    print(f"[parity] {label} strided pool bit-exact over {n} values", flush=True)


@pytest.mark.parametrize("name", ["ragged_3level_d128", "ragged_3level_d64", "paper_schedule_small",
                                  "eight_states", "tiny_runs"])
def test_stride_small_full(name):
    desc, seed = SMALL[name]
    r = _full_check(dict(desc, resample="stride"), "bf16", seed, AMP, f"stride_{name}")
    _check_pool_exact(r, f"stride_{name}")


def test_stride_f32():
    r = _full_check(dict(_desc(3, [1, 2, 4], 7, 11, F=2, S=1, Hh=2, nh=2, d=64), resample="stride"),
                    "f32", 22, 1.0, "stride_f32")
    _check_pool_exact(r, "stride_f32")


def test_stride_full_size_sampled():
    """Long history with ragged 4x resampling (30x52 -> 8x13), strided."""
    w = WORKLOADS["wan13b_longhist"]
    desc = dict(w["desc"], resample="stride")
    r = GpuRun(desc, w["dtype"], w["seed"], w["amplitude"])
    r.run()
    rng = np.random.default_rng(321)
    rows = _sample_rows(r.info, rng)
    heads = [0, 5, 11]
    ref = r.oracle(heads=heads, q_index=rows)[rows]
    e = assert_close(r.output()[rows][:, heads], ref, w["dtype"], "stride_wan13b_longhist")
    print(f"[parity] stride wan13b_longhist rows={len(rows)} {e}", flush=True)
    _check_pool_exact(r, "stride_wan13b_longhist")
    # the variant is not the block mean: the outputs differ measurably
    m = dict(w["desc"])
    rm = GpuRun(m, w["dtype"], w["seed"], w["amplitude"])
    rm.run()
    assert not np.array_equal(rm.output()[rows], r.output()[rows])
