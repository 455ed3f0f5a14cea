"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare with the fp64 oracle."""

import numpy as np
import torch

import oracle
from paper_2607_20940_amd import mssa
from paper_2607_20940_amd.inputs import make_inputs, to_f64
from paper_2607_20940_amd.workloads import input_shapes

from tolerances import TOL, assert_close, assert_close_by_group, errors  # noqa: F401


def to_device(x, dtype):
    if x is None:
        return None
    if dtype == "bf16":
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(x).cuda()


def from_device(t, dtype):
    if dtype == "bf16":
        return to_f64(t.view(torch.int16).cpu().numpy().view(np.uint16), "bf16")
    return t.cpu().numpy().astype(np.float64)


LOG2E = 1.4426950408889634


def q_prescale(desc):
    """The factor softmax_scale * log2(e) that a MSSA_PLAN_Q_PRESCALED plan
    expects on the queries (float64)."""
    return oracle.softmax_scale(desc) * LOG2E


class GpuRun:
    """Plan + seeded inputs + one pool_kv/forward pass on cuda:0.  With
    desc["q_prescaled"] the queries are drawn at amplitude * softmax_scale *
    log2(e) (rounded once) and the oracle gets them divided by that factor."""

    def __init__(self, desc, dtype, seed, amplitude, inputs=None, attention_blocks=0):
        self.desc = dict(desc)
        self.dtype = dtype
        if attention_blocks:
            self.plan = mssa.mssa_plan_create_ex(dict(desc, dtype=dtype), attention_blocks)
        else:
            self.plan = mssa.mssa_plan_create(dict(desc, dtype=dtype))
        self.info = self.plan.info()
        shapes = input_shapes(desc, self.info["n_q"], self.info["n_sink_tok"], self.info["n_hist_tok"])
        qa = amplitude * q_prescale(desc) if desc.get("q_prescaled") else None
        self.x = inputs if inputs is not None else make_inputs(shapes, seed, amplitude, dtype, q_amplitude=qa)
        self.d = {k: to_device(v, dtype) for k, v in self.x.items()}
        self.ws = torch.empty(max(256, self.info["workspace_bytes"]), dtype=torch.uint8, device="cuda")
        self.out = torch.empty_like(self.d["q_win"])

    def run(self, out=None):
        d = self.d
        out = self.out if out is None else out
        mssa.mssa_pool_kv(self.plan, d["k_hist"], d["v_hist"], d["k_win"], d["v_win"], self.ws)
        mssa.mssa_forward(self.plan, d["q_win"], d["k_sink"], d["v_sink"], d["k_hist"], d["v_hist"],
                          d["k_win"], d["v_win"], self.ws, out)
        torch.cuda.synchronize()
        return out

    def output(self):
        return from_device(self.out, self.dtype)

    def pooled(self, g, which):
        """Pooled K ('k') or V ('v') block of group g from the workspace, as
        float64 [tokens, heads, head_dim]."""
        info = self.info
        n = info["pooled_tokens"][g]
        nh, hd = self.desc["num_heads"], self.desc["head_dim"]
        eb = 2 if self.dtype == "bf16" else 4
        off = info["pooled_k_offset" if which == "k" else "pooled_v_offset"][g]
        raw = self.ws[off: off + n * nh * hd * eb].cpu().numpy()
        if self.dtype == "bf16":
            return to_f64(raw.view(np.uint16).reshape(n, nh, hd), "bf16")
        return raw.view(np.float32).reshape(n, nh, hd).astype(np.float64)

    def oracle_inputs(self, heads=None):
        """Inputs widened to float64, optionally restricted to some heads."""
        out = {}
        for k, v in self.x.items():
            if v is None:
                out[k] = None
                continue
            v = v if heads is None else v[:, heads]
            out[k] = to_f64(v, self.dtype)
        if self.desc.get("q_prescaled"):
            out["q_win"] = out["q_win"] / q_prescale(self.desc)
        return out

    def oracle(self, heads=None, q_index=None):
        x = self.oracle_inputs(heads)
        desc = dict(self.desc)
        if heads is not None:
            desc["num_heads"] = len(heads)
        return oracle.mssa_attention(desc, x["q_win"], x["k_sink"], x["v_sink"], x["k_hist"],
                                     x["v_hist"], x["k_win"], x["v_win"], q_index=q_index)
