"""GPU parity of the rolling-window streaming path (pool + forward + history
append per layer and pass) against the fp64 oracle.  The oracle's history is
rebuilt on the host from the generated inputs (the emitted head-state frames
of earlier passes, oldest first, FIFO-capped); nothing is read back from the
library's ring."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_20940_amd.streaming import StreamingMSSA, init_inputs, window_inputs
from paper_2607_20940_amd.workloads import STREAMING

from gpu_common import assert_close

pytestmark = pytest.mark.gpu


def _f64(t):
    return None if t is None else t.float().cpu().numpy().astype(np.float64)


def _run(stream_w, layers, passes, check):
    desc = stream_w["layer"]
    F = desc["frames_per_state"]
    st = StreamingMSSA(desc, layers, stream_w["hist_cap_frames"], dtype=stream_w["dtype"])
    tok1 = st.tok1
    hist = {}
    init_shapes = st.shapes(stream_w["hist_start_frames"])
    for L in range(layers):
        x = init_inputs(stream_w, L, init_shapes)
        st.init_layer(L, x["k_sink"], x["v_sink"], x["k_hist"], x["v_hist"])
        kh, vh = _f64(x["k_hist"]), _f64(x["v_hist"])
        n0 = stream_w["hist_start_frames"]
        hist[L] = dict(sink=(_f64(x["k_sink"]), _f64(x["v_sink"])),
                       k=[kh[i * tok1:(i + 1) * tok1] for i in range(n0)],
                       v=[vh[i * tok1:(i + 1) * tok1] for i in range(n0)])
    win_shapes = st.shapes(0)
    checked = 0
    for p in range(passes):
        wins = window_inputs(stream_w, p, layers, win_shapes)
        for L in range(layers):
            w = wins[L]
            out = torch.empty_like(w["q_win"])
            st.layer_pass(L, w["q_win"], w["k_win"], w["v_win"], out)
            h = hist[L]
            if check(p, L):
                torch.cuda.synchronize()
                print(f"[stream] pass {p} layer {L} hist_frames {len(h['k'])}", flush=True)
                d = dict(desc, hist_frames=len(h["k"]))
                got = out.float().cpu().numpy().astype(np.float64)
                ks = np.concatenate(h["k"]) if h["k"] else None
                vs = np.concatenate(h["v"]) if h["v"] else None
                kw, vw, qw = _f64(w["k_win"]), _f64(w["v_win"]), _f64(w["q_win"])
                rows, heads = check(p, L)
                if heads is not None:
                    d["num_heads"] = len(heads)
                    sel = lambda a: None if a is None else a[:, heads]  # noqa: E731
                else:
                    sel = lambda a: a  # noqa: E731
                ref = oracle.mssa_attention(d, sel(qw), sel(h["sink"][0]), sel(h["sink"][1]), sel(ks),
                                            sel(vs), sel(kw), sel(vw), q_index=rows)
                if rows is not None:
                    ref, got = ref[rows], got[rows]
                if heads is not None:
                    got = got[:, heads]
                e = assert_close(got, ref, stream_w["dtype"], f"pass {p} layer {L}")
                print(f"[stream] ok {e}", flush=True)
                checked += 1
            # the emitted head state's native frames become the newest history
            kw, vw = _f64(w["k_win"]), _f64(w["v_win"])
            for f in range(F):
                h["k"].append(kw[f * tok1:(f + 1) * tok1])
                h["v"].append(vw[f * tok1:(f + 1) * tok1])
            del h["k"][:-stream_w["hist_cap_frames"]]
            del h["v"][:-stream_w["hist_cap_frames"]]
    torch.cuda.synchronize()
    return st, checked


def test_streaming_small_every_output():
    """Small layers through the fill and several wrap-arounds of the ring."""
    w = dict(STREAMING, layer=dict(num_states=3, scales=[1, 1, 2], grid_h=6, grid_w=8,
                                   frames_per_state=2, sink_frames=1, hist_frames=0,
                                   num_heads=2, head_dim=128),
             hist_start_frames=2, hist_cap_frames=6, seed_base=40, init_seed_base=7000)
    st, n = _run(w, layers=2, passes=7, check=lambda p, L: (None, None))
    assert n == 14
    assert [r.count for r in st.ring] == [6, 6]
    # 2 + 7 * 2 = 16 frames appended into 6 slots: head advanced by 10 mod 6
    assert [r.head for r in st.ring] == [4, 4]


def test_streaming_wan13b_shape_sampled():
    """The streaming workload's layer shape (history 6 -> 21 frames, FIFO),
    two layers over eight passes, sampled rows and heads."""
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([[0, 9359, 9360, 12869], rng.integers(0, 12870, 40)]))

    def check(p, L):
        return (rows, [0, 11]) if (p in (0, 5, 7) and L == 1) else None

    st, n = _run(STREAMING, layers=2, passes=8, check=check)
    assert n == 3
    assert st.ring[0].count == 21 and st.ring[0].head == 9  # 6 + 8*3 = 30 frames -> 9 evicted
