"""GPU parity of the MSP tier steps (patch embedding, de-embedding, QKV
projection) through the C ABI against the fp64 tier oracle.

Tolerances: each output is an fp32 sum of exact bf16 products rounded once
to bf16 (relative error <= 2^-8 per element; measured rms 1.7e-3), so the bound is 4e-3 of the
reference rms and 8e-3 of its max.  With identity weights (hidden = C P^2)
every step is a pure gather or scatter of bf16 values and must be exact."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20940_amd import mssa
from paper_2607_20940_amd.inputs import bf16_bits_to_f32, f32_to_bf16_bits

from gpu_common import errors

pytestmark = pytest.mark.gpu


def _desc(scales, H, W, F=1, nh=1, d=64):
    return dict(num_states=len(scales), scales=list(scales), grid_h=H, grid_w=W, frames_per_state=F,
                sink_frames=0, hist_frames=0, num_heads=nh, head_dim=d)


def _bf16(rng, shape, scale=1.0):
    """Seeded draw rounded to bf16: (device tensor, float64 values)."""
    bits = f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))
    t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
    return t, bf16_bits_to_f32(bits).astype(np.float64)


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _close(got, ref, label):
    e = errors(got, ref)
    assert np.isfinite(got).all(), label
    assert e["rel_rms"] <= 4e-3 and e["rel_max"] <= 8e-3, (label, e)
    print(f"[tiers] {label} {e}", flush=True)


def _weights(rng, plan, desc, C, patch, hidden, out=False):
    info = plan.info()
    w, b, wd, bd = [], [], {}, {}
    for s in info["group_scale"]:
        kp = C * (patch * s) ** 2
        shape = (kp, hidden) if out else (hidden, kp)
        wt, wv = _bf16(rng, shape, 1.0 / np.sqrt(shape[1]))
        bt, bv = _bf16(rng, (shape[0],), 0.1)
        w.append(wt)
        b.append(bt)
        wd[s], bd[s] = wv, bv
    return w, b, wd, bd


CASES = {
    "ragged_3tier": (_desc([1, 2, 4], 5, 7, F=2), 16, 2, 128, 1),
    "paper_schedule_small": (_desc([1, 1, 2, 2, 2], 6, 10, F=3), 16, 2, 256, 2),
    "odd_channels": (_desc([1, 2], 9, 4, F=1), 2, 2, 64, 3),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_patch_embed_and_unembed(name):
    desc, C, patch, hidden, seed = CASES[name]
    rng = np.random.default_rng(seed)
    plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    tier = mssa.tier_desc(C, patch, hidden)
    nq = plan.info()["n_q"]
    T, F = desc["num_states"], desc["frames_per_state"]
    H, W = desc["grid_h"] * patch, desc["grid_w"] * patch
    ws = torch.empty(max(256, mssa.mssa_tier_workspace_size(plan, tier)), dtype=torch.uint8, device="cuda")
    lat, lat64 = _bf16(rng, (T * F, C, H, W))
    w, b, wd, bd = _weights(rng, plan, desc, C, patch, hidden)
    tok = torch.empty((nq, hidden), dtype=torch.bfloat16, device="cuda")
    mssa.mssa_patch_embed(plan, tier, lat, w, b, ws, tok)
    torch.cuda.synchronize()
    _close(_f64(tok), oracle.patch_embed(desc, patch, lat64, wd, bd), name + " embed")

    t_in, t64 = _bf16(rng, (nq, hidden))
    wo, bo, wod, bod = _weights(rng, plan, desc, C, patch, hidden, out=True)
    out = torch.full((T * F, C, H, W), float("nan"), dtype=torch.bfloat16, device="cuda")
    mssa.mssa_patch_unembed(plan, tier, t_in, wo, bo, ws, out)
    torch.cuda.synchronize()
    _close(_f64(out), oracle.patch_unembed(desc, patch, C, t64, wod, bod), name + " unembed")


@pytest.mark.parametrize("H,W", [(6, 10), (5, 7)])
def test_identity_tiers_are_exact(H, W):
    """hidden = C P^2 and W = I, b = 0: embedding is the patch gather and
    de-embedding its inverse, bit for bit (ragged edges: zeros in, dropped out)."""
    C, patch, s = 16, 2, 2
    desc = _desc([s, s], H, W, F=2)
    kp = C * (patch * s) ** 2
    plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    tier = mssa.tier_desc(C, patch, kp)
    rng = np.random.default_rng(5)
    lat, lat64 = _bf16(rng, (4, C, H * patch, W * patch))
    eye = [torch.eye(kp, dtype=torch.bfloat16, device="cuda")]
    zero = [torch.zeros(kp, dtype=torch.bfloat16, device="cuda")]
    ws = torch.empty(mssa.mssa_tier_workspace_size(plan, tier), dtype=torch.uint8, device="cuda")
    nq = plan.info()["n_q"]
    tok = torch.empty((nq, kp), dtype=torch.bfloat16, device="cuda")
    mssa.mssa_patch_embed(plan, tier, lat, eye, zero, ws, tok)
    back = torch.empty_like(lat)
    mssa.mssa_patch_unembed(plan, tier, tok, eye, zero, ws, back)
    torch.cuda.synchronize()
    want = np.concatenate([oracle.patchify(lat64[f], patch * s) for f in range(4)])
    assert np.array_equal(_f64(tok), want)
    assert torch.equal(back.view(torch.int16), lat.view(torch.int16))


@pytest.mark.parametrize("n,heads,d", [(77, 2, 64), (300, 3, 128), (1, 1, 64)])
def test_qkv_projection_small(n, heads, d):
    rng = np.random.default_rng(n)
    hidden = heads * d
    x, x64 = _bf16(rng, (n, hidden))
    w, w64 = _bf16(rng, (3 * hidden, hidden), 1.0 / np.sqrt(hidden))
    b, b64 = _bf16(rng, (3 * hidden,), 0.1)
    q, k, v = (torch.empty((n, heads, d), dtype=torch.bfloat16, device="cuda") for _ in range(3))
    mssa.mssa_qkv_project(n, hidden, x, w, b, q, k, v)
    torch.cuda.synchronize()
    for got, ref, nm in zip((q, k, v), oracle.qkv_project(x64, w64, b64, heads), "qkv"):
        _close(_f64(got), ref, f"qkv n={n} {nm}")


LOG2E = 1.4426950408889634


# (n, heads, d): the register-staged GEMM (K = 72, not a multiple of 64), the
# 128 x 128 direct-transfer GEMM, and the 256 x 256 GEMM (1.3B window width)
@pytest.mark.parametrize("n,heads,d", [(50, 1, 72), (300, 3, 128), (12870, 12, 128)])
def test_qkv_projection_scaled(n, heads, d):
    """mssa_qkv_project_scaled with q_scale = softmax_scale log2(e): q is the
    oracle's projection times the factor (taken on the fp32 sum, rounded
    once), k and v are bit for bit those of mssa_qkv_project."""
    rng = np.random.default_rng(n + 1)
    hidden = heads * d
    c = LOG2E / np.sqrt(d)
    x, x64 = _bf16(rng, (n, hidden))
    w, w64 = _bf16(rng, (3 * hidden, hidden), 1.0 / np.sqrt(hidden))
    b, b64 = _bf16(rng, (3 * hidden,), 0.1)
    out = [torch.empty((n, heads, d), dtype=torch.bfloat16, device="cuda") for _ in range(6)]
    mssa.mssa_qkv_project(n, hidden, x, w, b, *out[:3])
    mssa.mssa_qkv_project_scaled(n, hidden, x, w, b, c, *out[3:])
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(min(n, 64)), rng.integers(0, n, 64), [n - 1]]))
    ref = oracle.qkv_project(x64[rows], w64, b64, heads)
    _close(_f64(out[3])[rows], ref[0] * np.float32(c), f"scaled q n={n}")
    for i in (1, 2):
        assert torch.equal(out[3 + i].view(torch.int16), out[i].view(torch.int16)), "k / v changed"


def test_qkv_scaled_feeds_prescaled_attention():
    """The library's own pipeline for MSSA_PLAN_Q_PRESCALED: tokens -> scaled
    QKV projection -> pool + attention with pre-scaled queries, against the
    oracle on the projected (unscaled) queries and the same K / V, and close
    to the plain pipeline's output."""
    desc = dict(_desc([1, 1, 2, 2, 2], 10, 13, F=2, nh=2, d=128), sink_frames=1, hist_frames=2)
    plain = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    pre = mssa.mssa_plan_create(dict(desc, dtype="bf16", q_prescaled=True))
    info = plain.info()
    nq, hidden, d = info["n_q"], 256, 128
    c = LOG2E / np.sqrt(d)
    rng = np.random.default_rng(17)
    x, _ = _bf16(rng, (nq, hidden))
    w, _ = _bf16(rng, (3 * hidden, hidden), 1.0 / np.sqrt(hidden))
    b, _ = _bf16(rng, (3 * hidden,), 0.1)
    shapes = {k: (n, 2, d) for k, n in (("k_sink", info["n_sink_tok"]), ("v_sink", info["n_sink_tok"]),
                                          ("k_hist", info["n_hist_tok"]), ("v_hist", info["n_hist_tok"]))}
    ctx = {k: _bf16(rng, s)[0] if s[0] else None for k, s in shapes.items()}
    outs = {}
    for name, plan, scaled in (("plain", plain, False), ("pre", pre, True)):
        q, k, v = (torch.empty((nq, 2, d), dtype=torch.bfloat16, device="cuda") for _ in range(3))
        if scaled:
            mssa.mssa_qkv_project_scaled(nq, hidden, x, w, b, c, q, k, v)
        else:
            mssa.mssa_qkv_project(nq, hidden, x, w, b, q, k, v)
        ws = torch.empty(max(256, plan.info()["workspace_bytes"]), dtype=torch.uint8, device="cuda")
        o = torch.empty_like(q)
        mssa.mssa_pool_kv(plan, ctx["k_hist"], ctx["v_hist"], k, v, ws)
        mssa.mssa_forward(plan, q, ctx["k_sink"], ctx["v_sink"], ctx["k_hist"], ctx["v_hist"], k, v, ws, o)
        torch.cuda.synchronize()
        f = {kk: (None if t is None else _f64(t)) for kk, t in ctx.items()}
        qf = _f64(q) / (c if scaled else 1.0)
        ref = oracle.mssa_attention(desc, qf, f["k_sink"], f["v_sink"], f["k_hist"], f["v_hist"], _f64(k), _f64(v))
        got = _f64(o)
        e = errors(got, ref)
        assert np.isfinite(got).all() and e["max_abs"] <= 2e-2 and e["mean_abs"] <= 2e-3 and e["rel_rms"] <= 1e-2, (name, e)
        print(f"[tiers] pipeline {name} {e}", flush=True)
        outs[name] = got
    assert np.abs(outs["pre"] - outs["plain"]).max() <= 2e-2


def test_tiers_wan13b_layer_shapes():
    """The 1.3B-shaped window (30 x 52 tokens of 2 x 2 patches over 16 latent
    channels, schedule (p, p, 2p, 2p, 2p), width 1536 = 12 x 128): every
    embedded token, the de-embedded latent, and sampled rows of q, k, v."""
    desc = _desc([1, 1, 2, 2, 2], 30, 52, F=3, nh=12, d=128)
    C, patch, hidden = 16, 2, 1536
    rng = np.random.default_rng(11)
    plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    tier = mssa.tier_desc(C, patch, hidden)
    nq = plan.info()["n_q"]
    ws = torch.empty(mssa.mssa_tier_workspace_size(plan, tier), dtype=torch.uint8, device="cuda")
    lat, lat64 = _bf16(rng, (15, C, 60, 104))
    w, b, wd, bd = _weights(rng, plan, desc, C, patch, hidden)
    tok = torch.empty((nq, hidden), dtype=torch.bfloat16, device="cuda")
    mssa.mssa_patch_embed(plan, tier, lat, w, b, ws, tok)
    wq, wq64 = _bf16(rng, (3 * hidden, hidden), 1.0 / np.sqrt(hidden))
    bq, bq64 = _bf16(rng, (3 * hidden,), 0.1)
    q, k, v = (torch.empty((nq, 12, 128), dtype=torch.bfloat16, device="cuda") for _ in range(3))
    x, x64 = _bf16(rng, (nq, hidden))
    mssa.mssa_qkv_project(nq, hidden, x, wq, bq, q, k, v)
    wo, bo, wod, bod = _weights(rng, plan, desc, C, patch, hidden, out=True)
    out = torch.empty_like(lat)
    mssa.mssa_patch_unembed(plan, tier, x, wo, bo, ws, out)
    torch.cuda.synchronize()
    _close(_f64(tok), oracle.patch_embed(desc, patch, lat64, wd, bd), "wan13b embed")
    _close(_f64(out), oracle.patch_unembed(desc, patch, C, x64, wod, bod), "wan13b unembed")
    for got, ref, nm in zip((q, k, v), oracle.qkv_project(x64, wq64, bq64, 12), "qkv"):
        _close(_f64(got), ref, f"wan13b {nm}")


def test_qkv_projection_large_ragged():
    """The 256 x 256-tile product with both edges ragged: 4452 tokens (17
    full row tiles and 100 rows) and 3 x 1344 = 4032 features (15 full
    feature tiles and 192 features), every output against the oracle."""
    n, heads, d = 4452, 21, 64
    rng = np.random.default_rng(41)
    hidden = heads * d
    x, x64 = _bf16(rng, (n, hidden))
    w, w64 = _bf16(rng, (3 * hidden, hidden), 1.0 / np.sqrt(hidden))
    b, b64 = _bf16(rng, (3 * hidden,), 0.1)
    q, k, v = (torch.empty((n, heads, d), dtype=torch.bfloat16, device="cuda") for _ in range(3))
    mssa.mssa_qkv_project(n, hidden, x, w, b, q, k, v)
    torch.cuda.synchronize()
    for got, ref, nm in zip((q, k, v), oracle.qkv_project(x64, w64, b64, heads), "qkv"):
        _close(_f64(got), ref, f"qkv ragged {nm}")
