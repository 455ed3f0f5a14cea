"""ctypes binding of libmssa (include/libmssa.h): argument marshalling only.

Every step of the path runs in the library's HIP kernels; this module turns
tensors into device pointers and the current torch stream into a hipStream_t.
Importing it loads ``libmssa.so`` from this package directory and raises
ImportError if it has not been built (``python -m paper_2607_20940_amd.build``).
There is no fallback implementation.
"""

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmssa.so")

MSSA_MAX_STATES = 8
MSSA_OK, MSSA_ERR_INVALID_ARG, MSSA_ERR_UNSUPPORTED = 0, 1, 2
MSSA_ERR_WORKSPACE, MSSA_ERR_DEVICE, MSSA_ERR_NO_MEMORY = 3, 4, 5
MSSA_BF16, MSSA_F32 = 0, 1
MSSA_PLAN_POOLED_HIST_RING = 1
MSSA_PLAN_STRIDED_SUBSAMPLE = 2
MSSA_PLAN_HEAD_IN_RING = 4
MSSA_PLAN_Q_PRESCALED = 8

# Every symbol include/libmssa.h declares.
EXPORTS = ("mssa_plan_create", "mssa_plan_create_ex", "mssa_plan_destroy", "mssa_plan_query", "mssa_plan_tables",
           "mssa_pool_kv", "mssa_forward", "mssa_hist_append", "mssa_pool_hist_ring",
           "mssa_forward_ring", "mssa_hist_append_ring", "mssa_forward_lse", "mssa_backward_workspace_size",
           "mssa_backward", "mssa_tier_workspace_size", "mssa_patch_embed", "mssa_patch_unembed",
           "mssa_qkv_project", "mssa_qkv_project_scaled", "mssa_attention_noalloc", "mssa_pool_kv_head_ring", "mssa_forward_head_ring",
           "mssa_head_ring_roll", "mssa_status_string", "mssa_last_error")

MSSA_NOALLOC_SCRATCH_BYTES = 256 << 20


class mssa_tier_desc(ctypes.Structure):
    _fields_ = [("latent_channels", ctypes.c_int32), ("patch", ctypes.c_int32), ("hidden", ctypes.c_int32)]


class mssa_plan_desc(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("scales", ctypes.c_int32 * MSSA_MAX_STATES),
                ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
                ("frames_per_state", ctypes.c_int32), ("sink_frames", ctypes.c_int32),
                ("hist_frames", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("flags", ctypes.c_int32)]


_I32S = ctypes.c_int32 * MSSA_MAX_STATES
_I64S = ctypes.c_int64 * MSSA_MAX_STATES


class mssa_plan_info(ctypes.Structure):
    _fields_ = [("n_q", ctypes.c_int64), ("n_sink_tok", ctypes.c_int64),
                ("n_hist_tok", ctypes.c_int64), ("workspace_bytes", ctypes.c_int64),
                ("pairs_per_head", ctypes.c_int64), ("flops_alg", ctypes.c_int64),
                ("pool_bytes_alg", ctypes.c_int64), ("n_groups", ctypes.c_int32),
                ("group_scale", _I32S), ("q_begin", _I32S), ("q_end", _I32S),
                ("n_kv", _I64S), ("pooled_k_offset", _I64S), ("pooled_v_offset", _I64S),
                ("pooled_tokens", _I64S)]


def _load():
    # torch ships its own HIP runtime with the same soname as ROCm's
    # (libamdhip64.so.7).  Loading torch first makes libmssa bind to that one
    # runtime; a second runtime in the process would see no device.
    import torch  # noqa: F401

    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2607_20940_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, V, I64 = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64
    lib.mssa_plan_create.argtypes = [ctypes.POINTER(mssa_plan_desc), ctypes.POINTER(P)]
    lib.mssa_plan_create_ex.argtypes = [ctypes.POINTER(mssa_plan_desc), ctypes.c_int32, ctypes.POINTER(P)]
    lib.mssa_plan_destroy.argtypes = [P]
    lib.mssa_plan_destroy.restype = None
    lib.mssa_plan_query.argtypes = [P, ctypes.POINTER(mssa_plan_info)]
    lib.mssa_plan_tables.argtypes = [P, ctypes.POINTER(I64), I64, ctypes.POINTER(I64)]
    lib.mssa_pool_kv.argtypes = [P, V, V, V, V, V, I64, V]
    lib.mssa_forward.argtypes = [P, V, V, V, V, V, V, V, V, I64, V, V]
    lib.mssa_hist_append.argtypes = [P, V, V, V, V, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                     ctypes.POINTER(ctypes.c_int32), V]
    PP = ctypes.POINTER(ctypes.c_void_p)
    lib.mssa_pool_hist_ring.argtypes = [P, V, V, PP, PP, V]
    lib.mssa_forward_ring.argtypes = [P, V, V, V, V, V, PP, PP, V, V, V, I64, V, V]
    lib.mssa_hist_append_ring.argtypes = [P, V, V, V, I64, V, V, PP, PP, ctypes.c_int32,
                                          ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32), V]
    lib.mssa_forward_lse.argtypes = [P, V, V, V, V, V, V, V, V, I64, V, V, V]
    lib.mssa_attention_noalloc.argtypes = [P, V, V, V, V, V, V, V, V, V]
    I32 = ctypes.c_int32
    lib.mssa_pool_kv_head_ring.argtypes = [P, V, V, V, V, PP, PP, V, I64, I32, I32, I32, V]
    lib.mssa_forward_head_ring.argtypes = [P, V, V, V, V, V, PP, PP, V, V, V, I64, V, I32, I32, I32, V]
    lib.mssa_head_ring_roll.argtypes = [P, I32, ctypes.POINTER(I32), ctypes.POINTER(I32)]
    lib.mssa_backward_workspace_size.argtypes = [P, ctypes.POINTER(I64)]
    lib.mssa_backward.argtypes = [P, V, V, V, V, V, V, V, V, V, V, V, I64, V, V, V, V, V, V, V, V]
    TD = ctypes.POINTER(mssa_tier_desc)
    lib.mssa_tier_workspace_size.argtypes = [P, TD, ctypes.POINTER(I64)]
    lib.mssa_patch_embed.argtypes = [P, TD, V, PP, PP, V, I64, V, V]
    lib.mssa_patch_unembed.argtypes = [P, TD, V, PP, PP, V, I64, V, V]
    lib.mssa_qkv_project.argtypes = [I64, ctypes.c_int32, V, V, V, V, V, V, V]
    lib.mssa_qkv_project_scaled.argtypes = [I64, ctypes.c_int32, V, V, V, ctypes.c_float, V, V, V, V]
    lib.mssa_status_string.argtypes = [ctypes.c_int]
    lib.mssa_status_string.restype = ctypes.c_char_p
    lib.mssa_last_error.argtypes = []
    lib.mssa_last_error.restype = ctypes.c_char_p
    for name in ("mssa_plan_create", "mssa_plan_create_ex", "mssa_plan_query", "mssa_plan_tables", "mssa_pool_kv",
                 "mssa_forward", "mssa_hist_append", "mssa_pool_hist_ring", "mssa_forward_ring",
                 "mssa_hist_append_ring"):
        getattr(lib, name).restype = ctypes.c_int
    runtimes = _loaded_hip_runtimes()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes are loaded ({sorted(runtimes)}); libmssa would not see "
                          "the device torch uses")
    return lib


def _loaded_hip_runtimes():
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


lib = _load()


class MssaError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        name = lib.mssa_status_string(status).decode()
        detail = lib.mssa_last_error().decode()
        super().__init__(f"{where}: {name}: {detail}")


def _check(status, where):
    if status != MSSA_OK:
        raise MssaError(status, where)


def _ptr(x):
    """Device pointer of a tensor (or an int address); None -> NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _nbytes(x):
    if x is None:
        return 0
    return x.numel() * x.element_size()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


class Plan:
    """Owning handle of an mssa_plan (released when garbage collected)."""

    def __init__(self, handle, desc):
        self._h = handle
        self.desc = dict(desc)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        # at interpreter exit the module globals may already be gone
        if h and lib is not None:
            lib.mssa_plan_destroy(h)

    def info(self):
        return mssa_plan_query(self)

    def tables(self):
        return mssa_plan_tables(self)


def make_desc(desc):
    """dict (oracle-style keys, plus optional dtype 'bf16'/'f32') -> struct."""
    d = mssa_plan_desc()
    d.num_states = int(desc["num_states"])
    sc = list(desc["scales"])[:MSSA_MAX_STATES]
    for i, s in enumerate(sc):
        d.scales[i] = int(s)
    d.grid_h, d.grid_w = int(desc["grid_h"]), int(desc["grid_w"])
    d.frames_per_state = int(desc["frames_per_state"])
    d.sink_frames, d.hist_frames = int(desc["sink_frames"]), int(desc["hist_frames"])
    d.num_heads, d.head_dim = int(desc["num_heads"]), int(desc["head_dim"])
    dt = desc.get("dtype", "bf16")
    d.dtype = MSSA_BF16 if dt in ("bf16", MSSA_BF16) else MSSA_F32 if dt in ("f32", MSSA_F32) else int(dt)
    d.softmax_scale = float(desc.get("softmax_scale", 0.0) or 0.0)
    d.flags = int(desc.get("flags", 0) or 0)
    resample = desc.get("resample", "mean")
    if resample not in ("mean", "stride"):
        raise ValueError("resample must be 'mean' or 'stride'")
    if resample == "stride":
        d.flags |= MSSA_PLAN_STRIDED_SUBSAMPLE
    if desc.get("q_prescaled"):
        d.flags |= MSSA_PLAN_Q_PRESCALED
    return d


def mssa_plan_create(desc):
    h = ctypes.c_void_p()
    d = make_desc(desc)
    _check(lib.mssa_plan_create(ctypes.byref(d), ctypes.byref(h)), "mssa_plan_create")
    return Plan(h.value, desc)


def mssa_plan_create_ex(desc, attention_blocks):
    h = ctypes.c_void_p()
    d = make_desc(desc)
    _check(lib.mssa_plan_create_ex(ctypes.byref(d), int(attention_blocks), ctypes.byref(h)), "mssa_plan_create_ex")
    return Plan(h.value, desc)


def mssa_plan_query(plan):
    info = mssa_plan_info()
    _check(lib.mssa_plan_query(plan.handle, ctypes.byref(info)), "mssa_plan_query")
    G = info.n_groups
    return dict(
        n_q=info.n_q, n_sink_tok=info.n_sink_tok, n_hist_tok=info.n_hist_tok,
        workspace_bytes=info.workspace_bytes, pairs_per_head=info.pairs_per_head,
        flops_alg=info.flops_alg, pool_bytes_alg=info.pool_bytes_alg, n_groups=G,
        group_scale=list(info.group_scale[:G]), q_begin=list(info.q_begin[:G]),
        q_end=list(info.q_end[:G]), n_kv=list(info.n_kv[:G]),
        pooled_k_offset=list(info.pooled_k_offset[:G]),
        pooled_v_offset=list(info.pooled_v_offset[:G]),
        pooled_tokens=list(info.pooled_tokens[:G]))


def mssa_plan_tables(plan):
    need = ctypes.c_int64()
    lib.mssa_plan_tables(plan.handle, None, 0, ctypes.byref(need))
    buf = (ctypes.c_int64 * need.value)()
    _check(lib.mssa_plan_tables(plan.handle, buf, need.value, ctypes.byref(need)), "mssa_plan_tables")
    t = np.frombuffer(buf, dtype=np.int64).copy()
    ng, nq, ns = int(t[0]), int(t[1]), int(t[2])
    o = 3
    GRID = t[o: o + 4 * ng].reshape(ng, 4)
    o += 4 * ng
    QGRP = t[o: o + 4 * nq].reshape(nq, 4)
    o += 4 * nq
    SEG = t[o: o + 8 * ns].reshape(ns, 8)
    o += 8 * ns
    return {"GRID": GRID, "QGRP": QGRP, "SEG": SEG, "TOTAL": t[o: o + 2]}


def mssa_pool_kv(plan, k_hist, v_hist, k_win, v_win, workspace, workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_pool_kv(plan.handle, _ptr(k_hist), _ptr(v_hist), _ptr(k_win), _ptr(v_win),
                            _ptr(workspace), wb, _stream(stream)), "mssa_pool_kv")


def mssa_forward(plan, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, workspace, out,
                 workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_forward(plan.handle, _ptr(q_win), _ptr(k_sink), _ptr(v_sink), _ptr(k_hist),
                            _ptr(v_hist), _ptr(k_win), _ptr(v_win), _ptr(workspace), wb,
                            _ptr(out), _stream(stream)), "mssa_forward")


def mssa_forward_lse(plan, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, workspace, out, lse,
                     workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_forward_lse(plan.handle, _ptr(q_win), _ptr(k_sink), _ptr(v_sink), _ptr(k_hist),
                                _ptr(v_hist), _ptr(k_win), _ptr(v_win), _ptr(workspace), wb,
                                _ptr(out), _ptr(lse), _stream(stream)), "mssa_forward_lse")


def mssa_attention_noalloc(plan, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, out, stream=None):
    _check(lib.mssa_attention_noalloc(plan.handle, _ptr(q_win), _ptr(k_sink), _ptr(v_sink), _ptr(k_hist),
                                      _ptr(v_hist), _ptr(k_win), _ptr(v_win), _ptr(out), _stream(stream)),
           "mssa_attention_noalloc")


def mssa_backward_workspace_size(plan):
    n = ctypes.c_int64()
    _check(lib.mssa_backward_workspace_size(plan.handle, ctypes.byref(n)), "mssa_backward_workspace_size")
    return n.value


def mssa_backward(plan, q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, out, lse, d_out, workspace,
                  dq_win, dk_sink, dv_sink, dk_hist, dv_hist, dk_win, dv_win, workspace_bytes=None,
                  stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_backward(plan.handle, _ptr(q_win), _ptr(k_sink), _ptr(v_sink), _ptr(k_hist),
                             _ptr(v_hist), _ptr(k_win), _ptr(v_win), _ptr(out), _ptr(lse), _ptr(d_out),
                             _ptr(workspace), wb, _ptr(dq_win), _ptr(dk_sink), _ptr(dv_sink),
                             _ptr(dk_hist), _ptr(dv_hist), _ptr(dk_win), _ptr(dv_win), _stream(stream)),
           "mssa_backward")


def tier_desc(latent_channels, patch, hidden):
    return mssa_tier_desc(int(latent_channels), int(patch), int(hidden))


def mssa_tier_workspace_size(plan, tier):
    n = ctypes.c_int64()
    _check(lib.mssa_tier_workspace_size(plan.handle, ctypes.byref(tier), ctypes.byref(n)),
           "mssa_tier_workspace_size")
    return n.value


def mssa_patch_embed(plan, tier, latent, w_embed, b_embed, workspace, tokens, workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_patch_embed(plan.handle, ctypes.byref(tier), _ptr(latent), _ptr_array(w_embed),
                                _ptr_array(b_embed), _ptr(workspace), wb, _ptr(tokens), _stream(stream)),
           "mssa_patch_embed")


def mssa_patch_unembed(plan, tier, tokens, w_out, b_out, workspace, latent, workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_patch_unembed(plan.handle, ctypes.byref(tier), _ptr(tokens), _ptr_array(w_out),
                                  _ptr_array(b_out), _ptr(workspace), wb, _ptr(latent), _stream(stream)),
           "mssa_patch_unembed")


def mssa_qkv_project(n_tokens, hidden, x, w_qkv, b_qkv, q, k, v, stream=None):
    _check(lib.mssa_qkv_project(int(n_tokens), int(hidden), _ptr(x), _ptr(w_qkv), _ptr(b_qkv), _ptr(q), _ptr(k),
                                _ptr(v), _stream(stream)), "mssa_qkv_project")


def mssa_qkv_project_scaled(n_tokens, hidden, x, w_qkv, b_qkv, q_scale, q, k, v, stream=None):
    _check(lib.mssa_qkv_project_scaled(int(n_tokens), int(hidden), _ptr(x), _ptr(w_qkv), _ptr(b_qkv),
                                       float(q_scale), _ptr(q), _ptr(k), _ptr(v), _stream(stream)),
           "mssa_qkv_project_scaled")


class HeadRing:
    """Host-side state of the rings of a MSSA_PLAN_HEAD_IN_RING plan: slots
    (ring_frames), history frames (count) and the first spare slot (spare),
    where window state 1 of the current pass lives."""

    def __init__(self, frames, count=0, spare=None):
        self.frames = int(frames)
        self.count = int(count)
        self.spare = int(count if spare is None else spare)


def mssa_pool_kv_head_ring(plan, k_ring, v_ring, k_win, v_win, k_ring_pooled, v_ring_pooled, workspace, ring,
                           workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_pool_kv_head_ring(plan.handle, _ptr(k_ring), _ptr(v_ring), _ptr(k_win), _ptr(v_win),
                                      _ptr_array(k_ring_pooled), _ptr_array(v_ring_pooled), _ptr(workspace), wb,
                                      ring.frames, ring.count, ring.spare, _stream(stream)),
           "mssa_pool_kv_head_ring")


def mssa_forward_head_ring(plan, q_win, k_sink, v_sink, k_ring, v_ring, k_ring_pooled, v_ring_pooled, k_win, v_win,
                           workspace, out, ring, workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_forward_head_ring(plan.handle, _ptr(q_win), _ptr(k_sink), _ptr(v_sink), _ptr(k_ring),
                                      _ptr(v_ring), _ptr_array(k_ring_pooled), _ptr_array(v_ring_pooled),
                                      _ptr(k_win), _ptr(v_win), _ptr(workspace), wb, _ptr(out), ring.frames,
                                      ring.count, ring.spare, _stream(stream)),
           "mssa_forward_head_ring")


def mssa_head_ring_roll(plan, ring):
    count = ctypes.c_int32(ring.count)
    spare = ctypes.c_int32(ring.spare)
    _check(lib.mssa_head_ring_roll(plan.handle, ring.frames, ctypes.byref(count), ctypes.byref(spare)),
           "mssa_head_ring_roll")
    ring.count, ring.spare = count.value, spare.value


class Ring:
    """Host-side head/count of a history ring used with mssa_hist_append."""

    def __init__(self, cap_frames, count=0, head=0):
        self.cap = int(cap_frames)
        self.count = int(count)
        self.head = int(head)


def mssa_hist_append(plan, k_win, v_win, k_ring, v_ring, ring, stream=None):
    head = ctypes.c_int32(ring.head)
    count = ctypes.c_int32(ring.count)
    _check(lib.mssa_hist_append(plan.handle, _ptr(k_win), _ptr(v_win), _ptr(k_ring), _ptr(v_ring),
                                ring.cap, ctypes.byref(head), ctypes.byref(count), _stream(stream)),
           "mssa_hist_append")
    ring.head, ring.count = head.value, count.value


def _ptr_array(xs):
    """Per-group pointer array (None entries -> NULL)."""
    arr = (ctypes.c_void_p * max(1, len(xs)))()
    for i, x in enumerate(xs):
        arr[i] = _ptr(x)
    return arr


def mssa_pool_hist_ring(plan, k_ring, v_ring, k_ring_pooled, v_ring_pooled, stream=None):
    _check(lib.mssa_pool_hist_ring(plan.handle, _ptr(k_ring), _ptr(v_ring), _ptr_array(k_ring_pooled),
                                   _ptr_array(v_ring_pooled), _stream(stream)), "mssa_pool_hist_ring")


def mssa_forward_ring(plan, q_win, k_sink, v_sink, k_hist, v_hist, k_hist_pooled, v_hist_pooled, k_win,
                      v_win, workspace, out, workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    _check(lib.mssa_forward_ring(plan.handle, _ptr(q_win), _ptr(k_sink), _ptr(v_sink), _ptr(k_hist),
                                 _ptr(v_hist), _ptr_array(k_hist_pooled), _ptr_array(v_hist_pooled),
                                 _ptr(k_win), _ptr(v_win), _ptr(workspace), wb, _ptr(out),
                                 _stream(stream)), "mssa_forward_ring")


def mssa_hist_append_ring(plan, k_win, v_win, workspace, k_ring, v_ring, k_ring_pooled, v_ring_pooled, ring,
                          workspace_bytes=None, stream=None):
    wb = _nbytes(workspace) if workspace_bytes is None else int(workspace_bytes)
    head = ctypes.c_int32(ring.head)
    count = ctypes.c_int32(ring.count)
    _check(lib.mssa_hist_append_ring(plan.handle, _ptr(k_win), _ptr(v_win), _ptr(workspace), wb,
                                     _ptr(k_ring), _ptr(v_ring), _ptr_array(k_ring_pooled),
                                     _ptr_array(v_ring_pooled), ring.cap, ctypes.byref(head),
                                     ctypes.byref(count), _stream(stream)), "mssa_hist_append_ring")
    ring.head, ring.count = head.value, count.value
