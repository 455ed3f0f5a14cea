"""Seeded random plan descriptors: forward and backward of the HIP path
against the fp64 oracle over the whole output, on shapes the fixed cases do
not spell out (any nondecreasing power-of-two schedule up to 8 states,
ragged grids from 1 x 1, with and without sink or history, one to three
heads, both head dims, block-mean and strided resampling, bf16 and fp32).
The descriptors come from a fixed generator seed, so every run checks the
same cases; each prints its descriptor before it runs."""

import numpy as np
import pytest

from gpu_common import GpuRun, assert_close
from test_gpu_backward import _check as bwd_check

pytestmark = pytest.mark.gpu


def _random_desc(rng):
    T = int(rng.integers(1, 9))
    scales = sorted(int(2 ** rng.integers(0, 4)) for _ in range(T))
    desc = dict(num_states=T, scales=scales, grid_h=int(rng.integers(1, 17)),
                grid_w=int(rng.integers(1, 17)), frames_per_state=int(rng.integers(1, 3)),
                sink_frames=int(rng.integers(0, 3)), hist_frames=int(rng.integers(0, 4)),
                num_heads=int(rng.integers(1, 4)), head_dim=int(rng.choice([64, 128])))
    if rng.random() < 0.3:
        desc["resample"] = "stride"
    return desc


def _cases(seed, n):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        desc = _random_desc(rng)
        dtype = "f32" if rng.random() < 0.25 else "bf16"
        out.append((i, desc, dtype, int(rng.integers(0, 2**31))))
    return out


FWD_CASES = _cases(2026, 64)
BWD_CASES = _cases(4242, 20)


def _id(case):
    i, d, dtype, _ = case
    return (f"{i}-{dtype}-T{d['num_states']}-{''.join(map(str, d['scales']))}-{d['grid_h']}x{d['grid_w']}"
            f"-d{d['head_dim']}{'-stride' if d.get('resample') == 'stride' else ''}")


@pytest.mark.parametrize("case", FWD_CASES, ids=_id)
def test_forward_random_descriptor(case):
    i, desc, dtype, seed = case
    amp = 1.0 if dtype == "f32" else 1.0 / np.sqrt(128.0)
    print(f"[fuzz] forward {_id(case)} desc={desc} seed={seed}", flush=True)
    r = GpuRun(desc, dtype, seed, amp)
    r.run()
    e = assert_close(r.output(), r.oracle(), dtype, _id(case))
    print(f"[fuzz] ok {e}", flush=True)


@pytest.mark.parametrize("case", BWD_CASES, ids=_id)
def test_backward_random_descriptor(case):
    i, desc, dtype, seed = case
    amp = 1.0 if dtype == "f32" else 1.0 / np.sqrt(128.0)
    bwd_check(desc, dtype, seed, amp, f"fuzz {_id(case)}")


QPRE_FWD_CASES = _cases(7777, 24)
QPRE_BWD_CASES = _cases(8888, 8)


@pytest.mark.parametrize("case", QPRE_FWD_CASES, ids=_id)
def test_forward_random_descriptor_q_prescaled(case):
    """The same generator with queries pre-scaled by softmax_scale * log2(e)
    (MSSA_PLAN_Q_PRESCALED) at unit amplitude, so that the first-tile max
    path and the lazy rescale run often; the oracle reads the unscaled
    queries."""
    i, desc, dtype, seed = case
    desc = dict(desc, q_prescaled=True)
    print(f"[fuzz] forward pre-scaled {_id(case)} desc={desc} seed={seed}", flush=True)
    r = GpuRun(desc, dtype, seed, 1.0)
    r.run()
    e = assert_close(r.output(), r.oracle(), dtype, _id(case))
    print(f"[fuzz] ok {e}", flush=True)


@pytest.mark.parametrize("case", QPRE_BWD_CASES, ids=_id)
def test_backward_random_descriptor_q_prescaled(case):
    i, desc, dtype, seed = case
    bwd_check(dict(desc, q_prescaled=True), dtype, seed, 1.0, f"fuzz pre-scaled {_id(case)}")
