"""Output comparison used by every parity test: the workload's absolute
bounds plus a relative guard, so that a near-zero output cannot pass on the
tiny-amplitude inputs.  No GPU needed."""

import numpy as np

# Tolerances (max-abs / mean-abs for bf16 and fp32 outputs), plus the
# relative guard (rms error against the reference rms, max error against the
# reference's largest magnitude).
TOL = {
    "f32": dict(max_abs=1e-5, mean_abs=1e-6, rel_rms=1e-5, rel_max=1e-4),
    "bf16": dict(max_abs=2e-2, mean_abs=2e-3, rel_rms=1e-2, rel_max=5e-2),
}


def errors(got, ref):
    err = np.abs(got - ref)
    return dict(max_abs=float(err.max()), mean_abs=float(err.mean()),
                rel_rms=float(np.sqrt((err ** 2).mean()) / max(np.sqrt((ref ** 2).mean()), 1e-300)),
                rel_max=float(err.max() / max(np.abs(ref).max(), 1e-300)))


def assert_close(got, ref, dtype, label=""):
    assert np.isfinite(got).all(), f"{label}: non-finite output"
    assert np.abs(ref).max() > 0, f"{label}: degenerate reference"
    e = errors(got, ref)
    tol = TOL[dtype]
    bad = {k: (e[k], tol[k]) for k in tol if not e[k] <= tol[k]}
    assert not bad, f"{label}: errors above tolerance {bad}"
    return e


def assert_close_by_group(got, ref, rows, q_groups, dtype, label=""):
    """assert_close over all sampled rows, then over the rows of each query
    scale on its own (a mistake that touches one scale's queries is not
    diluted by the others).  rows: the sampled query indices (got and ref
    are indexed like rows); q_groups: (scale, q_begin, q_end) per group."""
    out = {"all": assert_close(got, ref, dtype, label)}
    rows = np.asarray(rows)
    for (s, qb, qe) in q_groups:
        sel = (rows >= qb) & (rows < qe)
        if sel.any():
            out[s] = assert_close(got[sel], ref[sel], dtype, f"{label} scale {s}")
    return out


def sample_rows(q_groups, n_q, rng, n_random=48):
    """Query rows the sampled full-size checks compare: the first rows of
    every query group and of its first 32-row and 128-row blocks, its last
    rows, and n_random rows drawn from rng.  q_groups: (scale, q_begin,
    q_end) per group."""
    rows = set()
    for (_, qb, qe) in q_groups:
        for off in (0, 1, 31, 32, 127, 128):
            if qb + off < qe:
                rows.add(qb + off)
        for off in (1, 2, 33):
            if qe - off >= qb:
                rows.add(qe - off)
    rows.update(rng.integers(0, n_q, n_random).tolist())
    return np.array(sorted(rows))
