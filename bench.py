"""Benchmark of the MSSA hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--resample mean|stride]

One step is one rolling pass of one layer: mssa_pool_kv (K/V resampling)
followed by mssa_forward (multi-scale attention) over inputs already resident
in HBM.  Input sets are rotated between steps (distinct device copies) so
that the pool kernel reads from HBM rather than from the 256 MB last-level
cache.  Kernel durations come from HIP events recorded around each launch on
the stream the kernels run on.

Prints one JSON line: effective TFLOP/s (algorithmic FLOP / pass time), ms per
pass, the roofline of the attention kernel and the fp64 CPU oracle timed on a
bounded sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA: 256 CU x 4096 flop/clk x 2.4 GHz
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0
LOG2E = 1.4426950408889634


def q_factor(desc, args):
    """Factor on the query draws: softmax_scale * log2(e) for the pre-scaled
    query layout (MSSA_PLAN_Q_PRESCALED: the producer folds the score scale
    into its epilogue, and the values are drawn at that amplitude and rounded
    once), 1 for the plain layout."""
    if getattr(args, "q_layout", "plain") != "prescaled":
        return 1.0
    s = float(desc.get("softmax_scale", 0.0) or 0.0)
    return (s if s > 0.0 else 1.0 / np.sqrt(float(desc["head_dim"]))) * LOG2E


Q_LAYOUT_NOTE = {"prescaled": "queries pre-scaled by softmax_scale*log2(e) (MSSA_PLAN_Q_PRESCALED)",
                 "plain": "plain queries (the kernel applies softmax_scale)"}
METRIC = "MSSA effective TFLOP/s + ms per rolling pass; % of bf16 MFMA peak (1 GPU)"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "mssa_fwd_traffic_{workload}.txt")
FWD_SOURCE = os.path.join(ROOT, "paper_2607_20940_amd", "csrc", "attention_fwd.hip")
POOL_SOURCE = os.path.join(ROOT, "paper_2607_20940_amd", "csrc", "pool_kv.hip")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class ClockSampler:
    """The GPU's current shader and memory clocks, sampled from a host thread
    while named sections of the benchmark run: the starred lines of the amdgpu
    driver's pp_dpm_sclk and pp_dpm_mclk ("S: <MHz> *" is the current level).
    The sustained shader clock under a long MFMA load is set by power, not by
    the 2.4 GHz peak the roofline's peak assumes, so the % of peak depends on
    it."""

    def __init__(self, period_s=0.01, kind="sclk"):
        import glob
        import threading

        paths = sorted(glob.glob(f"/sys/class/drm/card*/device/pp_dpm_{kind}"))
        self.path = paths[0] if paths else None
        self.kind = kind
        self.period = period_s
        self.samples = {}
        self.current = None
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._loop, daemon=True)

    def _read(self):
        try:
            with open(self.path) as f:
                for line in f:
                    if line.rstrip().endswith("*"):
                        return float(line.split(":", 1)[1].strip().split("M")[0])
        except (OSError, ValueError, IndexError):
            return None
        return None

    def _loop(self):
        while not self._stop.is_set():
            name = self.current
            if name is not None:
                mhz = self._read()
                if mhz is not None:
                    self.samples.setdefault(name, []).append(mhz)
            self._stop.wait(self.period)

    def start(self):
        if self.path:
            self._thread.start()

    def stop(self):
        self._stop.set()
        if self._thread.is_alive():
            self._thread.join()

    def section(self, name):
        import contextlib

        @contextlib.contextmanager
        def cm():
            self.current = name
            try:
                yield
            finally:
                self.current = None
        return cm()

    def summary(self):
        if not self.path:
            return {"source": None, "note": f"no pp_dpm_{self.kind} readable on this host"}
        out = {"source": self.path, "period_ms": self.period * 1e3}
        for name, v in self.samples.items():
            a = np.array(v)
            out[name] = {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
                         "p90": float(np.percentile(a, 90)), "samples": int(a.size)}
        return out


class Clocks:
    """Shader and memory clocks sampled together (see ClockSampler)."""

    def __init__(self):
        self.samplers = [ClockSampler(kind="sclk"), ClockSampler(kind="mclk")]

    def start(self):
        for c in self.samplers:
            c.start()

    def stop(self):
        for c in self.samplers:
            c.stop()

    def section(self, name):
        import contextlib

        stack = contextlib.ExitStack()
        for c in self.samplers:
            stack.enter_context(c.section(name))
        return stack

    def summary(self):
        return {f"{c.kind}_mhz": c.summary() for c in self.samplers}


def kernel_source_hash(path=None):
    with open(path or FWD_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def read_traffic(workload, kernel="forward"):
    """HBM bytes per launch of the attention call (kernel="forward") or of
    mssa_pool_kv (kernel="pool") from the committed counter summary, if it
    was taken on the current source of that kernel (else None)."""
    path = TRAFFIC_FILE.format(workload=workload)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if kernel == "pool":
        key_hash, key_bytes, src = "pool_source_sha256_16", "pool_hbm_bytes_per_launch", POOL_SOURCE
    else:
        key_hash, key_bytes, src = "kernel_source_sha256_16", "hbm_bytes_per_launch", FWD_SOURCE
    if vals.get(key_hash) != kernel_source_hash(src):
        return None
    try:
        return float(vals[key_bytes])
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, x, info, budget_s, qf=1.0):
    """Time the fp64 oracle (as it stands) on the host: whole heads of the
    workload (pool + attention for every query), one at a time, until the
    time budget is used.  Returns the oracle's effective TFLOP/s and its
    outputs {head: [n_q, head_dim] float64}."""
    import oracle
    from paper_2607_20940_amd.inputs import to_f64

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = os.cpu_count() or 1
    desc = dict(w["desc"])
    nh = desc["num_heads"]
    flops_per_head = info["flops_alg"] / nh
    done, t_total = 0, 0.0
    refs = {}
    for h in range(nh):
        xh = {k: (None if v is None else to_f64(v[:, [h]], w["dtype"])) for k, v in x.items()}
        xh["q_win"] = xh["q_win"] / qf  # the oracle takes the unscaled queries
        d1 = dict(desc, num_heads=1)
        t0 = time.perf_counter()
        o = oracle.mssa_attention(d1, xh["q_win"], xh["k_sink"], xh["v_sink"], xh["k_hist"],
                                  xh["v_hist"], xh["k_win"], xh["v_win"])
        t_total += time.perf_counter() - t0
        refs[h] = o[:, 0]
        done += 1
        log(f"cpu oracle head {h}: {t_total:.1f} s cumulative")
        if t_total >= budget_s:
            break
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {
        "value": flops_per_head * done / t_total / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "cpu_model": cpu_model,
        "nproc": os.cpu_count(),
        "sample": f"{done} of {nh} heads of {w['name']} (pool + attention, all {info['n_q']} queries), "
                  f"fp64 numpy, {t_total:.1f} s",
        "ms_per_pass_extrapolated": 1e3 * t_total / done * nh,
    }, refs


# Parity bounds of the workload (bf16 outputs): absolute max / mean error,
# plus the relative guard (rms error against the reference rms, max error
# against the reference's largest magnitude) that rejects near-zero outputs.
PARITY_TOL = {"max_abs": 2e-2, "mean_abs": 2e-3, "rel_rms": 1e-2, "rel_max": 5e-2}


def parity_vs_oracle(out, refs, w):
    """Every element of the GPU output of the heads the oracle computed
    against the oracle's float64 output."""
    import torch

    from paper_2607_20940_amd.inputs import to_f64

    heads = sorted(refs)
    got = to_f64(out[:, heads].contiguous().view(torch.int16).cpu().numpy().view(np.uint16), "bf16")
    ref = np.stack([refs[h] for h in heads], axis=1)
    err = np.abs(got - ref)
    e = {"max_abs": float(err.max()), "mean_abs": float(err.mean()),
         "rel_rms": float(np.sqrt((err ** 2).mean()) / np.sqrt((ref ** 2).mean())),
         "rel_max": float(err.max() / np.abs(ref).max())}
    return {**{k: float(f"{v:.4g}") for k, v in e.items()},
            "within_tolerance": bool(np.isfinite(got).all() and all(e[k] <= PARITY_TOL[k] for k in PARITY_TOL)),
            "tolerance": PARITY_TOL, "heads": f"{len(heads)} of {w['desc']['num_heads']}",
            "elements": int(got.size), "against": "fp64 oracle, every query row"}


def bench_streaming(args):
    """Steady-state streaming: stacked layers over rolling passes (pool +
    forward + history append per layer and pass); window inputs of a pass
    are generated on the device before that pass is timed.  Returns the
    result line."""
    import torch

    from paper_2607_20940_amd.streaming import StreamingMSSA, init_inputs, window_inputs, window_inputs_head_ring
    from paper_2607_20940_amd.workloads import STREAMING

    w = STREAMING
    layers = args.layers or w["layers"]
    passes = args.passes or w["passes"]
    desc = w["layer"]
    F = desc["frames_per_state"]
    head_in_ring = getattr(args, "head_in_ring", False)
    qf = q_factor(desc, args)
    st = StreamingMSSA(desc, layers, w["hist_cap_frames"], dtype=w["dtype"], pooled_ring=args.pooled_ring,
                       head_in_ring=head_in_ring, q_prescaled=qf != 1.0)
    init_shapes = st.shapes(w["hist_start_frames"])
    for L in range(layers):
        x = init_inputs(w, L, init_shapes)
        st.init_layer(L, x["k_sink"], x["v_sink"], x["k_hist"], x["v_hist"])
    win_shapes = st.shapes(0)
    outs = [torch.empty(win_shapes["q_win"], dtype=torch.bfloat16, device="cuda") for _ in range(layers)]
    stream = torch.cuda.current_stream()
    pass_ms, pass_flops = [], []
    bufs = st.window_buffers() if args.graph else None
    kinds = []
    for p in range(passes):
        # window inputs of the pass (state 1 written into the ring's spare
        # slots by its producer when the roll moves no data)
        wins = (window_inputs_head_ring(w, p, st, q_scale=qf) if head_in_ring
                else window_inputs(w, p, layers, win_shapes, q_scale=qf))
        flops = sum(st.plan(st.ring[L].count).info()["flops_alg"] for L in range(layers))
        if args.graph:
            for L in range(layers):
                for k in ("q_win", "k_win", "v_win"):
                    bufs[L][k].copy_(wins[L][k])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        if args.graph:
            kinds.append(st.graph_pass())
        else:
            for L in range(layers):
                st.layer_pass(L, wins[L]["q_win"], wins[L]["k_win"], wins[L]["v_win"], outs[L])
        e1.record(stream)
        torch.cuda.synchronize()
        pass_ms.append(e0.elapsed_time(e1))
        pass_flops.append(flops)
        if p % 8 == 0 or p == passes - 1:
            log(f"pass {p}: {pass_ms[-1]:.2f} ms, history {st.ring[0].count} frames")
    steady = list(range(min(5, passes - 1), passes))
    if args.graph:
        # graph capture runs on the host while the GPU waits; steady state is
        # the replay-only passes (one capture per ring head position)
        steady = [i for i in steady if kinds[i] == "replayed"] or steady
    tot_ms = sum(pass_ms)
    st_ms = sum(pass_ms[i] for i in steady)
    result = {
        "metric": "MSSA attention ms per emitted latent frame (stacked layers, rolling passes)",
        "value": round(st_ms / (len(steady) * F), 4),
        "unit": "ms/frame",
        "n_gpus": 1,
        "steps": passes,
        "warmup": 0,
        "ms_per_step": round(tot_ms / passes, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w["dtype"],
        "data": "synthetic",
        "config": {"workload": "streaming_wan13b", "layers": layers, "passes": passes,
                   "hist_frames": f"{w['hist_start_frames']}->{w['hist_cap_frames']} FIFO",
                   "frames_per_state": F,
                   "history_pooling": "pooled_ring" if st.pooled_ring else "per_pass",
                   "cache_roll": "in place (head state written into the ring)" if head_in_ring else "device copies",
                   "launch": "hip_graph_per_pass" if args.graph else "eager",
                   "q_layout": Q_LAYOUT_NOTE[getattr(args, "q_layout", "plain")]},
        "all_passes_ms_per_frame": round(tot_ms / (passes * F), 4),
        "steady_state_passes": [steady[0], steady[-1]],
        "steady_state_pass_count": len(steady),
        "effective_tflops_steady": round(sum(pass_flops[i] for i in steady) / (st_ms * 1e-3) / 1e12, 2),
    }
    return result


def bench_training(args):
    """One training step of one layer's MSSA: mssa_pool_kv, mssa_forward_lse
    and mssa_backward (all seven input gradients) on one workspace.  The
    backward's algorithmic work is 2.5x the forward's (the products
    P^T dO, dO V^T, dS K and dS^T Q besides Q K^T), the usual count; the dQ
    kernel's recomputation of Q K^T and dO V^T is overhead, not work."""
    import torch

    from paper_2607_20940_amd import mssa
    from paper_2607_20940_amd.inputs import make_grad_output, make_inputs
    from paper_2607_20940_amd.workloads import WORKLOADS, input_shapes

    w = dict(WORKLOADS[args.workload], name=args.workload)
    desc, dtype = w["desc"], w["dtype"]
    qf = q_factor(desc, args)
    plan = mssa.mssa_plan_create(dict(desc, dtype=dtype, q_prescaled=qf != 1.0))
    info = plan.info()
    shapes = input_shapes(desc, info["n_q"], info["n_sink_tok"], info["n_hist_tok"])
    x = make_inputs(shapes, w["seed"], w["amplitude"], dtype,
                    q_amplitude=w["amplitude"] * qf if qf != 1.0 else None)
    go = make_grad_output(shapes["q_win"], w["seed"] + 7919, 1.0, dtype)

    def dev(a):
        if a is None:
            return None
        if dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    d = {k: dev(v) for k, v in x.items()}
    g_out = dev(go)
    ws = torch.empty(mssa.mssa_backward_workspace_size(plan), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(d["q_win"])
    lse = torch.empty(desc["num_heads"] * info["n_q"], dtype=torch.float32, device="cuda")
    grads = {k: (None if v is None else torch.empty_like(v)) for k, v in d.items()}
    names = ("q_win", "k_sink", "v_sink", "k_hist", "v_hist", "k_win", "v_win")
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        mssa.mssa_pool_kv(plan, d["k_hist"], d["v_hist"], d["k_win"], d["v_win"], ws)
        mssa.mssa_forward_lse(plan, d["q_win"], d["k_sink"], d["v_sink"], d["k_hist"], d["v_hist"],
                              d["k_win"], d["v_win"], ws, out, lse)
        if ev is not None:
            ev[1].record(stream)
        mssa.mssa_backward(plan, *(d[k] for k in names), out, lse, g_out, ws, *(grads[k] for k in names))
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for e in evs:
        step(e)
    torch.cuda.synchronize()
    fwd_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    bwd_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    step_ms = fwd_ms + bwd_ms
    F = info["flops_alg"]
    result = {
        "metric": "MSSA training step (pool + forward + backward) effective TFLOP/s (1 GPU)",
        "value": round(3.5 * F / (step_ms.mean() * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(float(step_ms.mean()), 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic",
        "config": {"workload": args.workload, "flops_alg_forward": F, "flops_alg_backward": 2.5 * F,
                   "q_layout": Q_LAYOUT_NOTE[getattr(args, "q_layout", "plain")]},
        "forward_pool_ms": round(float(fwd_ms.mean()), 4),
        "backward_ms": round(float(bwd_ms.mean()), 4),
        "backward_ms_p10_p90": [round(float(np.percentile(bwd_ms, 10)), 4),
                                round(float(np.percentile(bwd_ms, 90)), 4)],
        "backward_tflops": round(2.5 * F / (bwd_ms.mean() * 1e-3) / 1e12, 2),
        "backward_pct_of_bf16_peak": round(100 * 2.5 * F / (bwd_ms.mean() * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
    }
    return result


def bench_tiers(args):
    """The steps on either side of the attention for the 1.3B-shaped window
    (16 latent channels, patch 2, width 1536 = 12 x 128): tier patch
    embedding, QKV projection and de-embedding, synthetic weights."""
    import torch

    from paper_2607_20940_amd import mssa
    from paper_2607_20940_amd.workloads import WORKLOADS

    desc = WORKLOADS["wan13b_layer"]["desc"]
    C, patch = 16, 2
    hidden = desc["num_heads"] * desc["head_dim"]
    plan = mssa.mssa_plan_create(dict(desc, dtype="bf16"))
    info = plan.info()
    nq = info["n_q"]
    tier = mssa.tier_desc(C, patch, hidden)
    gen = torch.Generator(device="cuda").manual_seed(7)
    rnd = lambda *s: (torch.randn(*s, generator=gen, device="cuda") * 0.05).to(torch.bfloat16)  # noqa: E731
    frames = desc["num_states"] * desc["frames_per_state"]
    lat = rnd(frames, C, desc["grid_h"] * patch, desc["grid_w"] * patch)
    kps = [C * (patch * s) ** 2 for s in info["group_scale"]]
    w_in = [rnd(hidden, kp) for kp in kps]
    b_in = [rnd(hidden) for _ in kps]
    w_out = [rnd(kp, hidden) for kp in kps]
    b_out = [rnd(kp) for kp in kps]
    w_qkv, b_qkv = rnd(3 * hidden, hidden), rnd(3 * hidden)
    ws = torch.empty(mssa.mssa_tier_workspace_size(plan, tier), dtype=torch.uint8, device="cuda")
    tok = torch.empty((nq, hidden), dtype=torch.bfloat16, device="cuda")
    q, k, v = (torch.empty_like(tok) for _ in range(3))
    out = torch.empty_like(lat)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        mssa.mssa_patch_embed(plan, tier, lat, w_in, b_in, ws, tok)
        if ev is not None:
            ev[1].record(stream)
        mssa.mssa_qkv_project(nq, hidden, tok, w_qkv, b_qkv, q, k, v)
        if ev is not None:
            ev[2].record(stream)
        mssa.mssa_patch_unembed(plan, tier, q, w_out, b_out, ws, out)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for e in evs:
        step(e)
    torch.cuda.synchronize()
    t = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(3)] for e in evs]).mean(axis=0)
    qkv_flops = 2.0 * nq * hidden * 3 * hidden
    emb_flops = sum(2.0 * (g1 - g0) * hidden * kp for g0, g1, kp in zip(info["q_begin"], info["q_end"], kps))
    result = {
        "metric": "MSP tier steps around MSSA: patch embedding, QKV projection, de-embedding (1 GPU)",
        "value": round(qkv_flops / (t[1] * 1e-3) / 1e12, 2), "unit": "TFLOP/s (QKV projection)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(float(t.sum()), 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "wan13b_layer tiers", "latent_channels": C, "patch": patch, "hidden": hidden,
                   "n_q": nq},
        "patch_embed_ms": round(float(t[0]), 4), "qkv_ms": round(float(t[1]), 4),
        "patch_unembed_ms": round(float(t[2]), 4),
        "qkv_pct_of_bf16_peak": round(100 * qkv_flops / (t[1] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "embed_unembed_tflops": round(2 * emb_flops / ((t[0] + t[2]) * 1e-3) / 1e12, 2),
    }
    # The same projection at the Wan-14B-shaped 720p window (width 40 x 128):
    # enough output tiles that the last round of blocks is a small share.
    d14 = WORKLOADS["wan14b_720p"]["desc"]
    n14 = mssa.mssa_plan_create(dict(d14, dtype="bf16")).info()["n_q"]
    h14 = d14["num_heads"] * d14["head_dim"]
    x14, w14, b14 = rnd(n14, h14), rnd(3 * h14, h14), rnd(3 * h14)
    o14 = [torch.empty((n14, h14), dtype=torch.bfloat16, device="cuda") for _ in range(3)]
    for _ in range(max(args.warmup, 2)):
        mssa.mssa_qkv_project(n14, h14, x14, w14, b14, *o14)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = max(args.steps // 4, 3)
    e0.record(stream)
    for _ in range(reps):
        mssa.mssa_qkv_project(n14, h14, x14, w14, b14, *o14)
    e1.record(stream)
    torch.cuda.synchronize()
    ms14 = e0.elapsed_time(e1) / reps
    f14 = 2.0 * n14 * h14 * 3 * h14
    result["qkv_wan14b_720p"] = {"m_n_k": [n14, 3 * h14, h14], "ms": round(ms14, 4),
                                 "tflops": round(f14 / (ms14 * 1e-3) / 1e12, 2),
                                 "pct_of_bf16_peak": round(100 * f14 / (ms14 * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2)}
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="wan13b_layer")
    ap.add_argument("--input-sets", type=int, default=4,
                    help="distinct device copies of the inputs rotated between steps")
    ap.add_argument("--cpu-budget", type=float, default=30.0,
                    help="seconds of oracle time (whole heads; the 1.3B-shaped layer needs ~11 s for all)")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the named layer workload (skip the other layers, streaming and training)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layers", type=int, default=0, help="streaming: layers (default 30)")
    ap.add_argument("--passes", type=int, default=0, help="streaming: rolling passes (default 64)")
    ap.add_argument("--tiers", action="store_true",
                    help="time the tier patch embedding, QKV projection and de-embedding instead")
    ap.add_argument("--training", action="store_true",
                    help="time pool + forward (with lse) + backward of one layer instead")
    ap.add_argument("--graph", action="store_true",
                    help="streaming: replay each full pass as one HIP graph (static window buffers)")
    ap.add_argument("--pooled-ring", action="store_true",
                    help="streaming: keep pooled history rings instead of re-pooling history each pass")
    ap.add_argument("--head-in-ring", action="store_true",
                    help="streaming: pooled rings with window state 1 written into the rings' spare slots "
                         "(the cache roll copies nothing)")
    ap.add_argument("--resample", choices=("mean", "stride"), default="mean",
                    help="K/V resampling of the layer workloads: block mean (default) or the "
                         "strided pick of each block's first cell (both timed the same way)")
    ap.add_argument("--q-layout", choices=("prescaled", "plain"), default="prescaled",
                    help="queries handed over pre-scaled by softmax_scale*log2(e) (the producer folds the "
                         "score scale into its epilogue; MSSA_PLAN_Q_PRESCALED, default) or plain")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="only run a plain device copy of this many MiB (5 times), the reference "
                         "for scaling HBM byte counters")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only: MSSA here is a single-GPU kernel path with no "
              f"collectives (asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    if args.workload == "streaming":
        print(json.dumps(bench_streaming(args)), flush=True)
        return
    if args.training:
        print(json.dumps(bench_training(args)), flush=True)
        return
    if args.tiers:
        bench_tiers(args)
        return
    if args.copy_calibration_mb:
        import torch
        n = args.copy_calibration_mb * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n * 4, "copies": 5}), flush=True)
        return

    clock = Clocks()
    clock.start()
    result, out0, x, w, info = bench_layer(args, args.workload, host_inputs=True, clock=clock)
    if not args.no_cpu_baseline:
        base, ref = cpu_baseline(w, x, info, args.cpu_budget, qf=q_factor(w["desc"], args))
        result["cpu_baseline"] = base
        result["parity"] = parity_vs_oracle(out0, ref, w)
        log(f"parity against the oracle: {result['parity']}")
    if args.workload == "wan13b_layer" and args.resample == "mean" and not args.no_extras:
        # the same layer with the other query layout, the other layer
        # workloads, the stacked-layer streaming workload and the training
        # step, each timed the same way on this GPU
        oargs = argparse.Namespace(**vars(args))
        oargs.q_layout = "plain" if args.q_layout == "prescaled" else "prescaled"
        r, _, _, _, _ = bench_layer(oargs, args.workload, host_inputs=False, clock=clock,
                                    section=args.workload + "_" + oargs.q_layout)
        result[oargs.q_layout + "_q"] = {
            "q_layout": Q_LAYOUT_NOTE[oargs.q_layout],
            **{k: r[k] for k in ("ms_per_step", "value", "pct_of_bf16_peak", "forward_ms", "forward_ms_median",
                                 "forward_ms_p10_p90")},
            "forward_frac_of_bf16_peak": r["roofline"]["frac"]}
        result["other_layers"] = {}
        for name in ("wan13b_longhist", "wan14b_720p"):
            r, _, _, _, _ = bench_layer(args, name, host_inputs=False, clock=clock)
            result["other_layers"][name] = {
                k: r[k] for k in ("ms_per_step", "value", "pct_of_bf16_peak", "forward_ms", "forward_ms_median",
                                  "forward_ms_p10_p90", "pool_ms")}
            result["other_layers"][name]["forward_frac_of_bf16_peak"] = r["roofline"]["frac"]
            result["other_layers"][name]["pool_gbps"] = r["pool"]["achieved"]
            result["other_layers"][name]["config"] = r["config"]
        for key, head in (("streaming", True), ("streaming_copy_roll", False)):
            sargs = argparse.Namespace(**vars(args))
            sargs.pooled_ring, sargs.head_in_ring, sargs.graph = True, head, False
            with clock.section(key):
                s_res = bench_streaming(sargs)
            result[key] = {k: s_res[k] for k in ("value", "unit", "all_passes_ms_per_frame", "steady_state_passes",
                                                 "effective_tflops_steady", "config")}
        targs = argparse.Namespace(**vars(args))
        targs.workload = "wan13b_layer"
        with clock.section("training"):
            t_res = bench_training(targs)
        result["training"] = {k: t_res[k] for k in ("ms_per_step", "forward_pool_ms", "backward_ms", "backward_ms_p10_p90",
                                                    "backward_tflops", "backward_pct_of_bf16_peak", "value", "unit")}
    clock.stop()
    result.update(clock.summary())
    print(json.dumps(result), flush=True)


def bench_layer(args, workload, host_inputs, clock, section=None):
    """Time K passes (mssa_pool_kv + mssa_forward) of one layer workload.
    host_inputs: the seeded host inputs the oracle also reads (returned);
    else device-drawn inputs of the same distribution.  Returns (result
    line, output of input set 0, host inputs or None, workload, plan info)."""
    import torch

    from paper_2607_20940_amd import mssa
    from paper_2607_20940_amd.inputs import make_inputs, make_inputs_device
    from paper_2607_20940_amd.workloads import WORKLOADS, input_shapes

    w = dict(WORKLOADS[workload], name=workload)
    if args.resample != "mean":
        w["desc"] = dict(w["desc"], resample=args.resample)
    desc = w["desc"]
    dtype = w["dtype"]
    qf = q_factor(desc, args)
    qa = w["amplitude"] * qf if qf != 1.0 else None
    plan = mssa.mssa_plan_create(dict(desc, dtype=dtype, q_prescaled=qf != 1.0))
    info = plan.info()
    shapes = input_shapes(desc, info["n_q"], info["n_sink_tok"], info["n_hist_tok"])
    log(f"workload {workload}: n_q={info['n_q']} n_kv={info['n_kv']} flops={info['flops_alg']:.4e}")
    t0 = time.perf_counter()

    def dev(a):
        if a is None:
            return None
        if dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    if host_inputs:
        x = make_inputs(shapes, w["seed"], w["amplitude"], dtype, q_amplitude=qa)
        base = {k: dev(v) for k, v in x.items()}
    else:
        x = None
        base = make_inputs_device(shapes, w["seed"], w["amplitude"], dtype, q_amplitude=qa)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")
    sets = [base] + [{k: (None if v is None else v.clone()) for k, v in base.items()}
                     for _ in range(args.input_sets - 1)]
    ws = [torch.empty(max(256, info["workspace_bytes"]), dtype=torch.uint8, device="cuda")
          for _ in sets]
    outs = [torch.empty_like(base["q_win"]) for _ in sets]
    stream = torch.cuda.current_stream()

    def step(i, ev=None):
        s = sets[i % len(sets)]
        if ev is not None:
            ev[0].record(stream)
        mssa.mssa_pool_kv(plan, s["k_hist"], s["v_hist"], s["k_win"], s["v_win"], ws[i % len(sets)])
        if ev is not None:
            ev[1].record(stream)
        mssa.mssa_forward(plan, s["q_win"], s["k_sink"], s["v_sink"], s["k_hist"], s["v_hist"],
                          s["k_win"], s["v_win"], ws[i % len(sets)], outs[i % len(sets)])
        if ev is not None:
            ev[2].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps done")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with clock.section(section or workload):
        start.record(stream)
        for i in range(args.steps):
            step(i, evs[i])
        end.record(stream)
        torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    pool_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    fwd_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    ms_per_step = total_ms / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.4f} ms/pass, forward mean {fwd_ms.mean():.4f} ms, "
        f"pool mean {pool_ms.mean():.4f} ms")

    flops = info["flops_alg"]
    value = flops / (ms_per_step * 1e-3) / 1e12
    fwd_tflops = flops / (fwd_ms.mean() * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS
    pool_gbps = info["pool_bytes_alg"] / (pool_ms.mean() * 1e-3) / 1e9 if pool_ms.mean() > 0 else None

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {
            "workload": workload,
            "heads": desc["num_heads"], "head_dim": desc["head_dim"],
            "grid": f"{desc['grid_h']}x{desc['grid_w']}", "schedule": desc["scales"],
            "sink_frames": desc["sink_frames"], "hist_frames": desc["hist_frames"],
            "states": desc["num_states"], "frames_per_state": desc["frames_per_state"],
            "n_q": info["n_q"], "n_kv": info["n_kv"], "flops_alg": flops,
            "input_sets_rotated": len(sets), "resample": args.resample,
            "inputs": "seeded host draws" if host_inputs else "device draws",
            "q_layout": Q_LAYOUT_NOTE[getattr(args, "q_layout", "plain")],
        },
        "pct_of_bf16_peak": round(100 * value / PEAK_BF16_TFLOPS, 2),
        "forward_ms": round(float(fwd_ms.mean()), 4),
        "forward_ms_median": round(float(np.median(fwd_ms)), 4),
        "forward_ms_p10_p90": [round(float(np.percentile(fwd_ms, 10)), 4),
                               round(float(np.percentile(fwd_ms, 90)), 4)],
        "pool_ms": round(float(pool_ms.mean()), 4),
        "pool": {"bound": "hbm", "achieved": None if pool_gbps is None else round(pool_gbps, 1),
                 "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                 "frac": None if pool_gbps is None else round(pool_gbps / PEAK_HBM_GBPS, 4),
                 "bytes_alg": info["pool_bytes_alg"], "traffic": read_traffic(workload, "pool")},
        "roofline": {"kernel": "mssa_forward (fwd_bf16_kernel + combine_kernel)" if dtype == "bf16" else "mssa_forward (fwd_f32_kernel)",
                     "bound": "mfma", "achieved": round(fwd_tflops, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(fwd_tflops / peak, 4),
                     "traffic": read_traffic(workload)},
    }
    out0 = outs[0]
    del sets, ws
    return result, out0, x, w, info


if __name__ == "__main__":
    main()
