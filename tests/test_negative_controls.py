"""Negative controls (no GPU): the tolerances the parity tests apply reject
every plausible wrong reading of Eq. 4 (Sec. 4.1) at the real shapes and
amplitudes of the full-size layer workloads, on the same kind of sampled
rows the full-size GPU checks compare.

Each wrong reading is computed by a perturbed copy of the oracle
(tests/oracle_mutants.py) on the same inputs as the correct oracle.  With
N(0,1)/sqrt(128) inputs the logits are tiny and the softmax nearly uniform,
so the absolute bounds alone accept almost anything (an all-zero output
passes them); the relative guard, applied to all sampled rows and to each
query scale's rows on its own, is what must reject the mutants.  Inputs
carry three heads (the workload's per-head statistics, a third of the
cost of one full head set); token counts and amplitudes are the workload's.
"""

import numpy as np
import pytest

import oracle
from paper_2607_20940_amd.inputs import make_inputs, to_f64
from paper_2607_20940_amd.workloads import WORKLOADS, input_shapes

import oracle_mutants
from tolerances import assert_close, assert_close_by_group, sample_rows

HEADS = 3


def _case(name):
    w = WORKLOADS[name]
    desc = dict(w["desc"], num_heads=HEADS)
    shapes = input_shapes(desc, oracle.num_window_tokens(desc), oracle.num_sink_tokens(desc),
                          oracle.num_hist_tokens(desc))
    x = {k: to_f64(v, w["dtype"]) for k, v in make_inputs(shapes, w["seed"], w["amplitude"], w["dtype"]).items()}
    groups = oracle.query_groups(desc)
    rows = sample_rows(groups, oracle.num_window_tokens(desc), np.random.default_rng(123))
    args = (x["q_win"], x["k_sink"], x["v_sink"], x["k_hist"], x["v_hist"], x["k_win"], x["v_win"])
    ref = oracle.mssa_attention(desc, *args, q_index=rows)[rows]
    return desc, w["dtype"], groups, rows, args, ref


_CACHE = {}


def _cached(name):
    if name not in _CACHE:
        _CACHE[name] = _case(name)
    return _CACHE[name]


def _ragged(desc):
    """True if some pooled grid is ragged (a scale that does not divide the
    native grid is in use)."""
    H, W = int(desc["grid_h"]), int(desc["grid_w"])
    return any(H % s or W % s for s in oracle.scales_in_use(desc))


@pytest.mark.parametrize("mutation", oracle_mutants.MUTATIONS)
@pytest.mark.parametrize("name", ["wan13b_layer", "wan13b_longhist", "wan14b_720p"])
def test_tolerance_rejects_wrong_reading(name, mutation):
    desc, dtype, groups, rows, args, ref = _cached(name)
    if mutation in ("pad_count_mean", "floor_grid") and not _ragged(desc):
        pytest.skip("every pooled grid divides the native grid: this reading equals the correct one")
    if mutation == "upsampled_keys" and len(groups) == 1:
        pytest.skip("a single query scale has no coarser keys")
    got = oracle_mutants.attention(desc, *args, rows, mutation)
    assert np.isfinite(got).all()
    # the mutant really computes something else
    assert not np.allclose(got, ref, rtol=0, atol=1e-12)
    with pytest.raises(AssertionError):
        assert_close_by_group(got, ref, rows, groups, dtype, f"{name}/{mutation}")


@pytest.mark.parametrize("name", ["wan13b_layer", "wan13b_longhist", "wan14b_720p"])
def test_unmutated_copy_passes(name):
    """The perturbed copy with no mutation is the oracle."""
    desc, dtype, groups, rows, args, ref = _cached(name)
    got = oracle_mutants.attention(desc, *args, rows, None)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-15)
    assert_close_by_group(got, ref, rows, groups, dtype, name)


def test_zero_output_passes_absolute_bounds_only():
    """Why the relative guard exists: on these inputs an all-zero output
    meets the absolute bounds, and only the guard rejects it."""
    desc, dtype, groups, rows, args, ref = _cached("wan13b_layer")
    z = np.zeros_like(ref)
    err = np.abs(z - ref)
    assert err.max() <= 2e-2 and err.mean() <= 2e-3
    with pytest.raises(AssertionError):
        assert_close(z, ref, dtype)
