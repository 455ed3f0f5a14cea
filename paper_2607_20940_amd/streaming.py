"""Rolling-window streaming of stacked MSSA layers (Ms. Forcing, Sec. 3.1
Eq. 2 and Alg. 1's per-pass KV-cache update) driven through the C ABI.

Each layer keeps its sink K/V and a history ring of native frames.  A layer
pass is: mssa_pool_kv (history and fine window frames resampled), then
mssa_forward, then mssa_hist_append (the head state's native frames become
the newest history frames, FIFO-capped).  The ring's valid frames are always
slots [0, count), read as a plan whose hist_frames equals count; one plan per
history length is kept.

With pooled_ring=True each layer also keeps, for every coarser query scale,
a ring of the history already pooled to that scale: mssa_pool_kv then pools
only window frames, mssa_forward_ring reads those rings, and
mssa_hist_append_ring moves the head state's pooled frames (computed by this
pass's mssa_pool_kv) into them, so history is never pooled again.  The
pooled rings hold exactly the bytes re-pooling would give; outputs agree
with the plain path up to the attention kernel's rounding (key tiles fall
differently around the separate pooled-history run).

With head_in_ring=True (pooled rings too) the cache roll moves no data: the
native and pooled rings have cap + F slots, window state 1 of a pass is
written by its producer straight into the F spare slots of the native ring
(head_slots()), mssa_pool_kv_head_ring pools it into the same slots of the
pooled rings, mssa_forward_head_ring reads history and state 1 from the
rings and the rest of the window from k_win / v_win (states 2..T only), and
mssa_head_ring_roll advances the ring state on the host.

graph_pass() runs a whole pass (every layer) over static window buffers as
one HIP graph: once every ring is full the plan no longer changes and the
ring head cycles through cap / gcd(cap, F) positions, so one graph per head
position is captured on first use and replayed after (the library enqueues
only kernels and device-to-device copies, and allocates nothing).  While the
rings fill, passes run eagerly.

This module only sequences library calls and owns device buffers (torch
allocations); all arithmetic runs in the library.
"""

from . import mssa
from .workloads import input_shapes


class StreamingMSSA:
    def __init__(self, layer_desc, layers, hist_cap_frames, dtype="bf16", device="cuda", pooled_ring=False,
                 head_in_ring=False, q_prescaled=False):
        import torch

        self.head_in_ring = bool(head_in_ring)
        self.pooled_ring = bool(pooled_ring) or self.head_in_ring
        flags = mssa.MSSA_PLAN_POOLED_HIST_RING if self.pooled_ring else 0
        if self.head_in_ring:
            flags |= mssa.MSSA_PLAN_HEAD_IN_RING
        self.desc = dict(layer_desc, flags=flags, q_prescaled=bool(q_prescaled))
        self.layers = int(layers)
        self.cap = int(hist_cap_frames)
        self.dtype = dtype
        self.device = device
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self._plans = {}
        base = self.plan(0)
        info = base.info()
        self.n_q = info["n_q"]
        self.tok1 = int(layer_desc["grid_h"]) * int(layer_desc["grid_w"])
        nh, d = int(layer_desc["num_heads"]), int(layer_desc["head_dim"])
        ws = max(self.plan(h).info()["workspace_bytes"] for h in range(self.cap + 1))
        self.workspace = torch.empty(max(256, ws), dtype=torch.uint8, device=device)
        self.F = int(layer_desc["frames_per_state"])
        # ring slots: the history cap, plus the spare slots of window state 1
        self.slots = self.cap + (self.F if self.head_in_ring else 0)
        shape = (self.slots * self.tok1, nh, d)
        self.k_ring = [torch.zeros(shape, dtype=self.tdtype, device=device) for _ in range(self.layers)]
        self.v_ring = [torch.zeros(shape, dtype=self.tdtype, device=device) for _ in range(self.layers)]
        self.ring = [mssa.HeadRing(self.slots) if self.head_in_ring else mssa.Ring(self.cap)
                     for _ in range(self.layers)]
        self.k_sink = [None] * self.layers
        self.v_sink = [None] * self.layers
        self._win = None
        self._graphs = {}
        # Pooled-history rings [layer][group] (None for groups at scale 1).
        self.k_pool = [[None] * info["n_groups"] for _ in range(self.layers)]
        self.v_pool = [[None] * info["n_groups"] for _ in range(self.layers)]
        if self.pooled_ring:
            gh, gw = int(layer_desc["grid_h"]), int(layer_desc["grid_w"])
            for g, sc in enumerate(info["group_scale"]):
                if sc == 1:
                    continue
                tok_s = -(-gh // sc) * -(-gw // sc)
                pshape = (self.slots * tok_s, nh, d)
                for layer in range(self.layers):
                    self.k_pool[layer][g] = torch.zeros(pshape, dtype=self.tdtype, device=device)
                    self.v_pool[layer][g] = torch.zeros(pshape, dtype=self.tdtype, device=device)

    def plan(self, hist_frames):
        if hist_frames not in self._plans:
            self._plans[hist_frames] = mssa.mssa_plan_create(
                dict(self.desc, hist_frames=hist_frames, dtype=self.dtype))
        return self._plans[hist_frames]

    def shapes(self, hist_frames):
        info = self.plan(hist_frames).info()
        return input_shapes(self.desc, info["n_q"], info["n_sink_tok"], info["n_hist_tok"])

    def init_layer(self, layer, k_sink, v_sink, k_hist, v_hist):
        """Sink K/V and the initial history (oldest first) of one layer."""
        self.k_sink[layer], self.v_sink[layer] = k_sink, v_sink
        n = 0 if k_hist is None else k_hist.shape[0] // self.tok1
        if n > self.cap:
            raise ValueError("initial history longer than the ring")
        if n:
            self.k_ring[layer][: n * self.tok1].copy_(k_hist)
            self.v_ring[layer][: n * self.tok1].copy_(v_hist)
        self.ring[layer] = mssa.HeadRing(self.slots, count=n) if self.head_in_ring else mssa.Ring(self.cap, count=n)
        if self.pooled_ring and n:
            mssa.mssa_pool_hist_ring(self.plan(n), self.k_ring[layer], self.v_ring[layer],
                                     self.k_pool[layer], self.v_pool[layer])

    def head_slots(self, layer):
        """(k, v) views of the native ring's spare slots, where the producer
        of window state 1's K/V writes them before the pass (head_in_ring)."""
        r = self.ring[layer]
        a, b = r.spare * self.tok1, (r.spare + self.F) * self.tok1
        return self.k_ring[layer][a:b], self.v_ring[layer][a:b]

    def window_buffers(self):
        """Static per-layer window buffers {q_win, k_win, v_win, out} that
        graph_pass() reads and writes."""
        import torch

        if self._win is None:
            sh = self.shapes(0)
            rest = (sh["k_win"][0] - (self.F * self.tok1 if self.head_in_ring else 0),) + tuple(sh["k_win"][1:])
            self._win = [{k: torch.zeros(sh["q_win"] if k in ("q_win", "out") else rest, dtype=self.tdtype,
                                         device=self.device)
                          for k in ("q_win", "k_win", "v_win", "out")} for _ in range(self.layers)]
        return self._win

    def graph_pass(self):
        """One pass of every layer over window_buffers(): eager until every
        ring is full, then the captured graph of the current head position.
        Returns "eager", "captured" (recorded, then replayed) or "replayed"."""
        import torch

        bufs = self.window_buffers()

        def run_all():
            for L in range(self.layers):
                b = bufs[L]
                self.layer_pass(L, b["q_win"], b["k_win"], b["v_win"], b["out"])

        heads = {r.spare if self.head_in_ring else r.head for r in self.ring}
        if any(r.count != self.cap for r in self.ring) or len(heads) != 1:
            run_all()
            return "eager"
        h = heads.pop()
        g = self._graphs.get(h)
        if g is None:
            # Capturing records the pass without running it and advances the
            # host-side ring state as the pass would; the replay runs it.
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run_all()
            self._graphs[h] = g
            g.replay()
            return "captured"
        g.replay()
        for r in self.ring:  # a full ring overwrites its F oldest slots
            if self.head_in_ring:
                r.spare = (r.spare + self.F) % self.slots
            else:
                r.head = (r.head + self.F) % self.cap
        return "replayed"

    def layer_pass(self, layer, q_win, k_win, v_win, out, stream=None):
        """One layer's pass.  head_in_ring: k_win / v_win hold window states
        2..T only (state 1 is already in head_slots(layer))."""
        ring = self.ring[layer]
        plan = self.plan(ring.count)
        if self.head_in_ring:
            mssa.mssa_pool_kv_head_ring(plan, self.k_ring[layer], self.v_ring[layer], k_win, v_win, self.k_pool[layer],
                                        self.v_pool[layer], self.workspace, ring, stream=stream)
            mssa.mssa_forward_head_ring(plan, q_win, self.k_sink[layer], self.v_sink[layer], self.k_ring[layer],
                                        self.v_ring[layer], self.k_pool[layer], self.v_pool[layer], k_win, v_win,
                                        self.workspace, out, ring, stream=stream)
            mssa.mssa_head_ring_roll(plan, ring)
            return
        nh = ring.count * self.tok1
        kh = self.k_ring[layer][:nh] if nh else None
        vh = self.v_ring[layer][:nh] if nh else None
        mssa.mssa_pool_kv(plan, kh, vh, k_win, v_win, self.workspace, stream=stream)
        if self.pooled_ring:
            mssa.mssa_forward_ring(plan, q_win, self.k_sink[layer], self.v_sink[layer], kh, vh,
                                   self.k_pool[layer], self.v_pool[layer], k_win, v_win, self.workspace,
                                   out, stream=stream)
            mssa.mssa_hist_append_ring(plan, k_win, v_win, self.workspace, self.k_ring[layer],
                                       self.v_ring[layer], self.k_pool[layer], self.v_pool[layer], ring,
                                       stream=stream)
        else:
            mssa.mssa_forward(plan, q_win, self.k_sink[layer], self.v_sink[layer], kh, vh, k_win, v_win,
                              self.workspace, out, stream=stream)
            mssa.mssa_hist_append(plan, k_win, v_win, self.k_ring[layer], self.v_ring[layer], ring,
                                  stream=stream)


def init_inputs(stream_w, layer, shapes, device="cuda"):
    """Sink and initial history of one layer (seeded init_seed_base + layer)."""
    from .inputs import make_inputs_device

    return make_inputs_device(shapes, stream_w["init_seed_base"] + layer, stream_w["amplitude"],
                              stream_w["dtype"], names=("k_sink", "v_sink", "k_hist", "v_hist"),
                              device=device)


def window_inputs_head_ring(stream_w, pass_index, st, device="cuda", q_scale=1.0):
    """Window Q/K/V of every layer for one pass of a head_in_ring driver: one
    generator seeded seed_base + pass_index draws, layer by layer, q, then
    K of state 1 (written into the layer's spare ring slots, as its producer
    would), K of states 2..T, V of state 1 (ring) and V of states 2..T.
    q_scale multiplies the query draws before rounding (pre-scaled queries).
    Returns per layer {q_win, k_win, v_win} with k_win / v_win the states
    2..T only."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(int(stream_w["seed_base"] + pass_index))
    tdt = torch.bfloat16 if stream_w["dtype"] == "bf16" else torch.float32
    amp = stream_w["amplitude"]
    shapes = st.shapes(0)
    n_head = st.F * st.tok1
    out = []
    for layer in range(st.layers):
        kh, vh = st.head_slots(layer)
        rest = (shapes["k_win"][0] - n_head,) + tuple(shapes["k_win"][1:])
        t = {"q_win": (torch.randn(shapes["q_win"], generator=gen, device=device) * (amp * q_scale)).to(tdt)}
        kh.copy_((torch.randn(kh.shape, generator=gen, device=device) * amp).to(tdt))
        t["k_win"] = (torch.randn(rest, generator=gen, device=device) * amp).to(tdt)
        vh.copy_((torch.randn(vh.shape, generator=gen, device=device) * amp).to(tdt))
        t["v_win"] = (torch.randn(rest, generator=gen, device=device) * amp).to(tdt)
        out.append(t)
    return out


def window_inputs(stream_w, pass_index, layers, shapes, device="cuda", q_scale=1.0):
    """Window Q/K/V of every layer for one pass: one generator seeded
    seed_base + pass_index draws q, k, v of layer 0, then layer 1, ...
    (q_scale multiplies the query draws before rounding)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(int(stream_w["seed_base"] + pass_index))
    tdt = torch.bfloat16 if stream_w["dtype"] == "bf16" else torch.float32
    out = []
    for _ in range(layers):
        t = {}
        for name in ("q_win", "k_win", "v_win"):
            x = torch.randn(shapes[name], generator=gen, device=device, dtype=torch.float32)
            t[name] = (x * (stream_w["amplitude"] * (q_scale if name == "q_win" else 1.0))).to(tdt)
        out.append(t)
    return out
