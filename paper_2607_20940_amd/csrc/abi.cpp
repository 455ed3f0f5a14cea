// C ABI of libmssa (declared in include/libmssa.h).  Validates every call
// before enqueuing work, turns the immutable plan into kernel arguments, and
// keeps C++ exceptions on this side of the boundary.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <memory>
#include <new>
#include <string>
#include <vector>

#include "../../include/libmssa.h"
#include "kernels.hpp"
#include "noalloc.hpp"
#include "plan.hpp"

struct mssa_plan_s {
  mssa::Plan p;
};

namespace {

// Message of the last failure on this thread.  A fixed buffer: recording a
// failure never allocates, so it cannot throw.
thread_local char g_last_error[512] = "";

mssa_status fail(mssa_status s, const char* msg) noexcept {
  std::snprintf(g_last_error, sizeof g_last_error, "%s", msg);
  return s;
}

mssa_status fail(mssa_status s, const char* what, const char* detail) noexcept {
  std::snprintf(g_last_error, sizeof g_last_error, "%s: %s", what, detail);
  return s;
}

// Body of an entry point: no C++ exception leaves the library.  A failed
// host allocation is MSSA_ERR_NO_MEMORY, anything else MSSA_ERR_INVALID_ARG.
template <class Body>
mssa_status guarded(const char* where, Body&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(MSSA_ERR_NO_MEMORY, where, "host allocation failed");
  } catch (...) {
    return fail(MSSA_ERR_INVALID_ARG, where, "unexpected internal error");
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Attention blocks resident at once on the current device (CUs x blocks per
// CU), or 0 when there is no usable device (the plan then assumes 512).
int resident_attention_blocks(int head_dim) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  const int per_cu = mssa::forward_blocks_per_cu(head_dim);
  return per_cu > 0 ? cus * per_cu : 0;
}

mssa_status check_device(hipError_t e, const char* what) {
  if (e == hipSuccess) return MSSA_OK;
  return fail(MSSA_ERR_DEVICE, what, hipGetErrorString(e));
}

// Launch pool jobs (source and destination pointers filled in), at most
// kMaxPoolJobs per launch.
mssa_status launch_pool_jobs(const mssa::Plan& p, std::vector<mssa::PoolJobArgs>& jobs, void* stream) {
  // Jobs that pool the same source frames by 2 and by 4 (block mean) become
  // one two-level job, so those frames are read once for both scales.
  for (mssa::PoolJobArgs& A : jobs) A.levels = 1;
  if (!p.strided) {
    std::vector<bool> gone(jobs.size(), false);
    for (size_t i = 0; i < jobs.size(); ++i) {
      mssa::PoolJobArgs& A = jobs[i];
      if (gone[i] || A.factor != 2) continue;
      for (size_t k = 0; k < jobs.size(); ++k) {
        const mssa::PoolJobArgs& B = jobs[k];
        if (k == i || gone[k] || B.factor != 4 || B.src_k != A.src_k || B.src_v != A.src_v ||
            B.src_gh != A.src_gh || B.src_gw != A.src_gw || B.n_frames != A.n_frames)
          continue;
        A.levels = 2;
        A.dst2_k = B.dst_k;
        A.dst2_v = B.dst_v;
        A.dst2_gh = B.dst_gh;
        A.dst2_gw = B.dst_gw;
        gone[k] = true;
        break;
      }
    }
    size_t w = 0;
    for (size_t i = 0; i < jobs.size(); ++i)
      if (!gone[i]) jobs[w++] = jobs[i];
    jobs.resize(w);
  }
  mssa::PoolArgs a{};
  a.ld = p.ld;
  a.chunks_per_tok = static_cast<int32_t>(p.ld * p.elem_bytes / 16);
  a.pick_first = p.strided ? 1 : 0;
  size_t j0 = 0;
  while (j0 < jobs.size()) {
    const size_t nj = std::min<size_t>(mssa::kMaxPoolJobs, jobs.size() - j0);
    int64_t blocks = 0;
    for (size_t i = 0; i < nj; ++i) {
      mssa::PoolJobArgs& A = a.jobs[i];
      A = jobs[j0 + i];
      A.block_begin = static_cast<int32_t>(blocks);
      const int64_t cells = A.levels == 2 ? static_cast<int64_t>(A.dst2_gh) * A.dst2_gw
                                          : static_cast<int64_t>(A.dst_gh) * A.dst_gw;
      const int64_t work = static_cast<int64_t>(A.n_frames) * cells * a.chunks_per_tok;
      blocks += (work + mssa::kPoolThreads - 1) / mssa::kPoolThreads;
    }
    if (blocks > 0x7fffffff) return fail(MSSA_ERR_UNSUPPORTED, "pool grid too large");
    a.n_jobs = static_cast<int32_t>(nj);
    const mssa_status s = check_device(
        mssa::launch_pool(a, static_cast<int>(blocks), p.desc.dtype == MSSA_BF16, static_cast<hipStream_t>(stream)),
        "pool kernel launch");
    if (s != MSSA_OK) return s;
    j0 += nj;
  }
  return MSSA_OK;
}

// Argument checks of mssa_pool_kv (nothing is enqueued).
mssa_status pool_check(const mssa::Plan& p, const void* k_hist, const void* v_hist, const void* k_win,
                       const void* v_win, const void* workspace, int64_t workspace_bytes) {
  if (p.pool_jobs.empty()) return MSSA_OK;
  if (!k_win || !v_win) return fail(MSSA_ERR_INVALID_ARG, "k_win and v_win must be non-null");
  bool reads_hist = false;
  for (const mssa::PoolJob& J : p.pool_jobs) reads_hist |= J.buffer == mssa::kBufHist;
  if (reads_hist && (!k_hist || !v_hist))
    return fail(MSSA_ERR_INVALID_ARG, "k_hist and v_hist must be non-null when history is pooled");
  if (!workspace || workspace_bytes < p.workspace_bytes)
    return fail(MSSA_ERR_WORKSPACE, "workspace smaller than mssa_plan_info.workspace_bytes");
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
    return fail(MSSA_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (!aligned16(k_win) || !aligned16(v_win) || (k_hist && !aligned16(k_hist)) || (v_hist && !aligned16(v_hist)))
    return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  return MSSA_OK;
}

// The pool jobs of a checked mssa_pool_kv call, enqueued on `stream`.
mssa_status pool_launch(const mssa::Plan& p, const void* k_hist, const void* v_hist, const void* k_win,
                        const void* v_win, void* workspace, void* stream) {
  if (p.pool_jobs.empty()) return MSSA_OK;
  const int64_t row_bytes = p.ld * p.elem_bytes;
  auto* ws = static_cast<char*>(workspace);
  std::vector<mssa::PoolJobArgs> jobs;
  for (const mssa::PoolJob& J : p.pool_jobs) {
    mssa::PoolJobArgs A{};
    const char* sk = static_cast<const char*>(J.buffer == mssa::kBufHist ? k_hist : k_win);
    const char* sv = static_cast<const char*>(J.buffer == mssa::kBufHist ? v_hist : v_win);
    A.src_k = sk + J.src_tok * row_bytes;
    A.src_v = sv + J.src_tok * row_bytes;
    A.dst_k = ws + p.pooled_k_off[J.group] + J.dst_tok * row_bytes;
    A.dst_v = ws + p.pooled_v_off[J.group] + J.dst_tok * row_bytes;
    A.src_gh = J.src_gh;
    A.src_gw = J.src_gw;
    A.dst_gh = J.dst_gh;
    A.dst_gw = J.dst_gw;
    A.factor = J.factor;
    A.n_frames = J.n_frames;
    jobs.push_back(A);
  }
  return launch_pool_jobs(p, jobs, stream);
}

// Ring slots (FIFO once full) that F appended frames take, with the head and
// count after them; false for an inconsistent head / count.
bool ring_slots(int32_t cap, int32_t F, int32_t* head, int32_t* count, std::vector<int32_t>& slots) {
  const int32_t h0 = *head, c0 = *count;
  if (c0 < 0 || c0 > cap || h0 < 0 || h0 >= cap || (h0 != 0 && c0 != cap)) return false;
  int32_t h = h0, c = c0;
  slots.clear();
  for (int32_t f = 0; f < F; ++f) {
    if (c < cap) {
      slots.push_back(c++);
    } else {
      slots.push_back(h);
      h = (h + 1) % cap;
    }
  }
  *head = h;
  *count = c;
  return true;
}

// Token count of one frame at scale s.
int64_t frame_tokens(const mssa::Plan& p, int32_t s) {
  const int64_t gh = (p.desc.grid_h + s - 1) / s, gw = (p.desc.grid_w + s - 1) / s;
  return gh * gw;
}

// Validation and slot assignment shared by both appends; enqueues the native
// frame copies.  On success *ring_head / *ring_count are advanced and slots
// holds the ring slot of each appended frame.
mssa_status append_native(const mssa::Plan& p, const void* k_win, const void* v_win, void* k_ring, void* v_ring,
                          int32_t ring_cap_frames, int32_t* ring_head, int32_t* ring_count,
                          std::vector<int32_t>& slots, void* stream) {
  if (!k_win || !v_win || !k_ring || !v_ring || !ring_head || !ring_count)
    return fail(MSSA_ERR_INVALID_ARG, "null argument");
  const int32_t F = p.desc.frames_per_state;
  if (p.desc.scales[0] != 1)
    return fail(MSSA_ERR_UNSUPPORTED, "the emitted head state must be at native scale (scales[0] == 1)");
  if (ring_cap_frames < F) return fail(MSSA_ERR_UNSUPPORTED, "ring_cap_frames < frames_per_state");
  int32_t head = *ring_head, count = *ring_count;
  if (!ring_slots(ring_cap_frames, F, &head, &count, slots))
    return fail(MSSA_ERR_INVALID_ARG, "inconsistent ring_head / ring_count");
  const size_t frame_bytes = static_cast<size_t>(p.tok1 * p.ld * p.elem_bytes);
  const char* kw = static_cast<const char*>(k_win);
  const char* vw = static_cast<const char*>(v_win);
  char* kr = static_cast<char*>(k_ring);
  char* vr = static_cast<char*>(v_ring);
  const size_t ring_bytes = frame_bytes * ring_cap_frames;
  const size_t win_bytes = frame_bytes * F;
  auto overlap = [](const char* x, size_t nx, const char* y, size_t ny) { return x < y + ny && y < x + nx; };
  if (overlap(kr, ring_bytes, kw, win_bytes) || overlap(kr, ring_bytes, vw, win_bytes) ||
      overlap(vr, ring_bytes, kw, win_bytes) || overlap(vr, ring_bytes, vw, win_bytes) ||
      overlap(kr, ring_bytes, vr, ring_bytes))
    return fail(MSSA_ERR_INVALID_ARG, "ring buffers overlap each other or the window");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  for (int32_t f = 0; f < F; ++f) {
    const size_t slot = static_cast<size_t>(slots[f]);
    mssa_status s = check_device(hipMemcpyAsync(kr + slot * frame_bytes, kw + f * frame_bytes, frame_bytes,
                                                hipMemcpyDeviceToDevice, st), "history append (K)");
    if (s != MSSA_OK) return s;
    s = check_device(hipMemcpyAsync(vr + slot * frame_bytes, vw + f * frame_bytes, frame_bytes,
                                    hipMemcpyDeviceToDevice, st), "history append (V)");
    if (s != MSSA_OK) return s;
  }
  *ring_head = head;
  *ring_count = count;
  return MSSA_OK;
}

// mssa_forward / mssa_forward_ring: validate, pack the kernel arguments and
// launch.  k_hist_pooled / v_hist_pooled (ring plans only) give each group's
// pooled-history ring.
// Device addresses of the first token (head 0) of run R of group g, K and V.
struct KvSources {
  const void *k_sink, *v_sink, *k_hist, *v_hist;
  const void* const* k_hist_pooled;
  const void* const* v_hist_pooled;
  const void *k_win, *v_win;
  const char* ws;
};

void run_pointers(const mssa::Plan& p, int g, const mssa::Run& R, const KvSources& s, const void** kp,
                  const void** vp) {
  const int64_t row_bytes = p.ld * p.elem_bytes;
  const char *kb = nullptr, *vb = nullptr;
  switch (R.buffer) {
    case mssa::kBufSink: kb = static_cast<const char*>(s.k_sink); vb = static_cast<const char*>(s.v_sink); break;
    case mssa::kBufHist: kb = static_cast<const char*>(s.k_hist); vb = static_cast<const char*>(s.v_hist); break;
    case mssa::kBufWin: kb = static_cast<const char*>(s.k_win); vb = static_cast<const char*>(s.v_win); break;
    case mssa::kBufHistPooled:
      kb = static_cast<const char*>(s.k_hist_pooled[g]);
      vb = static_cast<const char*>(s.v_hist_pooled[g]);
      break;
    default: kb = s.ws + p.pooled_k_off[g]; vb = s.ws + p.pooled_v_off[g]; break;
  }
  *kp = kb + R.tok_offset * row_bytes;
  *vp = vb + R.tok_offset * row_bytes;
}

// Argument checks of forward_impl (nothing is enqueued).
mssa_status forward_check(const mssa::Plan& p, const void* q_win, const void* k_sink, const void* v_sink,
                          const void* k_hist, const void* v_hist, const void* const* k_hist_pooled,
                          const void* const* v_hist_pooled, const void* k_win, const void* v_win,
                          const void* workspace, int64_t workspace_bytes, const void* out, const float* lse) {
  if (!q_win || !k_win || !v_win || !out)
    return fail(MSSA_ERR_INVALID_ARG, "q_win, k_win, v_win and out must be non-null");
  if (p.n_sink_tok > 0 && (!k_sink || !v_sink))
    return fail(MSSA_ERR_INVALID_ARG, "k_sink and v_sink must be non-null when sink_frames > 0");
  if (p.n_hist_tok > 0 && (!k_hist || !v_hist))
    return fail(MSSA_ERR_INVALID_ARG, "k_hist and v_hist must be non-null when hist_frames > 0");
  if (p.workspace_bytes > 0 && (!workspace || workspace_bytes < p.workspace_bytes))
    return fail(MSSA_ERR_WORKSPACE, "workspace smaller than mssa_plan_info.workspace_bytes");
  for (const void* t : {q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, out})
    if (t && !aligned16(t)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
  if (out == q_win || out == k_win || out == v_win)
    return fail(MSSA_ERR_INVALID_ARG, "out must not alias an input");
  if (lse && !aligned16(lse)) return fail(MSSA_ERR_INVALID_ARG, "lse must be 16-byte aligned");
  if (p.hist_ring && p.n_hist_tok > 0) {
    if (!k_hist_pooled || !v_hist_pooled)
      return fail(MSSA_ERR_INVALID_ARG, "k_hist_pooled and v_hist_pooled must be non-null");
    for (size_t g = 0; g < p.groups.size(); ++g) {
      if (p.groups[g].scale == 1) continue;
      const void* kp = k_hist_pooled[g];
      const void* vp = v_hist_pooled[g];
      if (!kp || !vp) return fail(MSSA_ERR_INVALID_ARG, "null pooled-history ring for a coarse query scale");
      if (!aligned16(kp) || !aligned16(vp)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    }
  }
  return MSSA_OK;
}

// A context run as device addresses (head 0, channel 0 of its first token).
struct PtrRun {
  const void* k;
  const void* v;
  int64_t n_tok;
};
using GroupRuns = std::vector<std::vector<PtrRun>>;

// Appends a run, merged with the previous one when it continues it in memory.
void push_run(std::vector<PtrRun>& rs, const void* k, const void* v, int64_t n_tok, int64_t row_bytes) {
  if (n_tok <= 0) return;
  if (!rs.empty()) {
    PtrRun& b = rs.back();
    if (static_cast<const char*>(b.k) + b.n_tok * row_bytes == k &&
        static_cast<const char*>(b.v) + b.n_tok * row_bytes == v) {
      b.n_tok += n_tok;
      return;
    }
  }
  rs.push_back({k, v, n_tok});
}

GroupRuns plan_runs(const mssa::Plan& p, const KvSources& src) {
  GroupRuns out(p.groups.size());
  for (size_t g = 0; g < p.groups.size(); ++g)
    for (const mssa::Run& R : p.runs[g]) {
      PtrRun r{nullptr, nullptr, R.n_tok};
      run_pointers(p, static_cast<int>(g), R, src, &r.k, &r.v);
      out[g].push_back(r);
    }
  return out;
}

// The kernels' two score factors: `scale` turns q k^T into natural-log
// logits (the fp32 paths and the gradients), `scale_log2e` into base-2 ones
// (the bf16 softmax).  For queries supplied pre-scaled by
// softmax_scale * log2(e), q' k^T already is the base-2 logit: the factors
// become ln 2 and 1.
void set_score_scales(const mssa::Plan& p, float& scale, float& scale_log2e) {
  if (p.q_prescaled) {
    scale = 0.69314718055994531f;
    scale_log2e = 1.0f;
  } else {
    scale = p.softmax_scale;
    scale_log2e = p.softmax_scale * 1.4426950408889634f;
  }
}

// Enqueues the attention kernels over the given runs and schedule.
mssa_status forward_launch(const mssa::Plan& p, const GroupRuns& runs, const mssa::Schedule& sc, const void* q_win,
                           const void* workspace, void* out, float* lse, void* stream) {
  const bool bf16 = p.desc.dtype == MSSA_BF16;
  const int bm = bf16 ? mssa::kFwdBM : mssa::kFwdF32BM;
  mssa::FwdArgs a{};
  a.q = q_win;
  a.out = out;
  a.lse = lse;
  a.n_q = static_cast<int32_t>(p.n_q);
  a.ld = p.ld;
  a.num_heads = p.desc.num_heads;
  set_score_scales(p, a.scale, a.scale_log2e);
  a.q_prescaled = p.q_prescaled ? 1 : 0;
  a.n_ranges = p.n_ranges;
  a.total_tiles = sc.total_tiles;
  a.tail_begin = sc.tail_begin;
  a.dp_rounds = sc.dp_rounds;
  const char* ws = static_cast<const char*>(workspace);
  a.partial = p.partial_bytes > 0 ? reinterpret_cast<float*>(const_cast<char*>(ws) + p.partial_off) : nullptr;
  a.range_table = p.partial_bytes > 0 ? reinterpret_cast<int64_t*>(const_cast<char*>(ws) + p.range_table_off) : nullptr;
  int64_t blocks = 0;
  int gi = 0;
  for (int g : p.order) {
    const mssa::QGroup& Q = p.groups[g];
    mssa::FwdGroupArgs& A = a.groups[gi++];
    A.q_begin = Q.q_begin;
    A.q_end = Q.q_end;
    A.n_qtiles = (Q.q_end - Q.q_begin + bm - 1) / bm;
    A.block_begin = static_cast<int32_t>(blocks);
    A.tiles_per_item = sc.tiles_per_item[g];
    A.tile_begin = sc.tile_begin[g];
    if (runs[g].size() > static_cast<size_t>(mssa::kMaxRuns))
      return fail(MSSA_ERR_UNSUPPORTED, "too many context runs for one query scale");
    A.n_runs = static_cast<int32_t>(runs[g].size());
    for (size_t r = 0; r < runs[g].size(); ++r) {
      A.runs[r].k = runs[g][r].k;
      A.runs[r].v = runs[g][r].v;
      A.runs[r].n_tok = static_cast<int32_t>(runs[g][r].n_tok);
    }
    blocks += static_cast<int64_t>(A.n_qtiles) * p.desc.num_heads;
  }
  if (blocks > 0x7fffffff) return fail(MSSA_ERR_UNSUPPORTED, "attention grid too large");
  a.n_groups = gi;
  a.n_blocks = static_cast<int32_t>(blocks);
  return check_device(mssa::launch_forward(a, p.desc.head_dim, bf16, static_cast<hipStream_t>(stream)),
                      "attention kernel launch");
}

mssa_status forward_impl(const mssa::Plan& p, const void* q_win, const void* k_sink, const void* v_sink,
                         const void* k_hist, const void* v_hist, const void* const* k_hist_pooled,
                         const void* const* v_hist_pooled, const void* k_win, const void* v_win,
                         const void* workspace, int64_t workspace_bytes, void* out, float* lse, void* stream) {
  const mssa_status chk = forward_check(p, q_win, k_sink, v_sink, k_hist, v_hist, k_hist_pooled, v_hist_pooled,
                                        k_win, v_win, workspace, workspace_bytes, out, lse);
  if (chk != MSSA_OK) return chk;
  const KvSources src{k_sink, v_sink, k_hist, v_hist, k_hist_pooled, v_hist_pooled,
                      k_win, v_win, static_cast<const char*>(workspace)};
  return forward_launch(p, plan_runs(p, src), p.sched, q_win, workspace, out, lse, stream);
}

// ---------------------------------------------------------------- head state in the ring

// Ring state rules of MSSA_PLAN_HEAD_IN_RING plans.
mssa_status head_ring_check(const mssa::Plan& p, int32_t ring_frames, int32_t count, int32_t spare) {
  if (!p.head_ring) return fail(MSSA_ERR_UNSUPPORTED, "plan lacks MSSA_PLAN_HEAD_IN_RING");
  const int32_t F = p.desc.frames_per_state;
  if (ring_frames < 2 * F || ring_frames % F != 0)
    return fail(MSSA_ERR_INVALID_ARG, "ring_frames must be a multiple of frames_per_state, at least two of them");
  if (spare < 0 || spare >= ring_frames || spare % F != 0)
    return fail(MSSA_ERR_INVALID_ARG, "ring_spare must be a multiple of frames_per_state below ring_frames");
  if (count != p.desc.hist_frames || count > ring_frames - F)
    return fail(MSSA_ERR_INVALID_ARG, "ring_count must equal hist_frames and not exceed ring_frames - F");
  return MSSA_OK;
}

// Context runs of every group: sink | history and window state 1 in the
// group's ring, slots spare - count .. spare + F - 1 (mod ring_frames; two
// runs if they wrap) | the rest of the window as placed by the plan.
GroupRuns head_ring_runs(const mssa::Plan& p, const void* k_sink, const void* v_sink, const void* k_ring,
                         const void* v_ring, const void* const* k_pool, const void* const* v_pool, const void* k_win,
                         const void* v_win, const char* ws, int32_t N, int32_t count, int32_t spare) {
  const int64_t rb = p.ld * p.elem_bytes;
  const int32_t F = p.desc.frames_per_state;
  GroupRuns out(p.groups.size());
  for (size_t g = 0; g < p.groups.size(); ++g) {
    const int32_t sc = p.groups[g].scale;
    std::vector<PtrRun>& rs = out[g];
    bool ring_done = false;
    for (const mssa::SegRow& r : p.segs) {
      if (r.q_scale != sc) continue;
      if (r.kind == mssa::kSink) {
        push_run(rs, static_cast<const char*>(k_sink) + r.tok_offset * rb,
                 static_cast<const char*>(v_sink) + r.tok_offset * rb, r.n_tok, rb);
      } else if (r.kind == mssa::kHist || r.buffer == mssa::kBufRingHead) {
        if (ring_done) continue;
        ring_done = true;
        const char* kb = static_cast<const char*>(sc == 1 ? k_ring : k_pool[g]);
        const char* vb = static_cast<const char*>(sc == 1 ? v_ring : v_pool[g]);
        const int64_t slot_tok = r.n_tok;  // a history frame and a state-1 frame at this scale
        const int32_t a = ((spare - count) % N + N) % N, b = spare + F;
        if (a < b) {
          push_run(rs, kb + a * slot_tok * rb, vb + a * slot_tok * rb, int64_t{b - a} * slot_tok, rb);
        } else {
          push_run(rs, kb + a * slot_tok * rb, vb + a * slot_tok * rb, int64_t{N - a} * slot_tok, rb);
          push_run(rs, kb, vb, int64_t{b} * slot_tok, rb);
        }
      } else if (r.buffer == mssa::kBufPooled) {
        push_run(rs, ws + p.pooled_k_off[g] + r.tok_offset * rb, ws + p.pooled_v_off[g] + r.tok_offset * rb,
                 r.n_tok, rb);
      } else {
        push_run(rs, static_cast<const char*>(k_win) + r.tok_offset * rb,
                 static_cast<const char*>(v_win) + r.tok_offset * rb, r.n_tok, rb);
      }
    }
  }
  return out;
}

}  // namespace

extern "C" {

mssa_status mssa_plan_create_ex(const mssa_plan_desc* desc, int32_t attention_blocks, mssa_plan* out) {
  return guarded("mssa_plan_create_ex", [&]() -> mssa_status {
    if (!desc || !out) return fail(MSSA_ERR_INVALID_ARG, "desc and out must be non-null");
    if (attention_blocks < 0) return fail(MSSA_ERR_INVALID_ARG, "attention_blocks must be >= 0");
    std::unique_ptr<mssa_plan_s> h(new mssa_plan_s);
    std::string err;
    const mssa_status s = mssa::build_plan(*desc, resident_attention_blocks(desc->head_dim), attention_blocks,
                                           h->p, err);
    if (s != MSSA_OK) return fail(s, err.c_str());
    *out = h.release();
    return MSSA_OK;
  });
}

mssa_status mssa_plan_create(const mssa_plan_desc* desc, mssa_plan* out) {
  return mssa_plan_create_ex(desc, 0, out);
}

void mssa_plan_destroy(mssa_plan plan) { delete plan; }

mssa_status mssa_plan_query(mssa_plan plan, mssa_plan_info* info) {
  return guarded("mssa_plan_query", [&]() -> mssa_status {
    if (!plan || !info) return fail(MSSA_ERR_INVALID_ARG, "plan and info must be non-null");
    const mssa::Plan& p = plan->p;
    std::memset(info, 0, sizeof(*info));
    info->n_q = p.n_q;
    info->n_sink_tok = p.n_sink_tok;
    info->n_hist_tok = p.n_hist_tok;
    info->workspace_bytes = p.workspace_bytes;
    info->pairs_per_head = p.pairs_per_head;
    info->flops_alg = 4 * static_cast<int64_t>(p.desc.head_dim) * p.desc.num_heads * p.pairs_per_head;
    info->pool_bytes_alg = p.pool_bytes_alg;
    info->n_groups = static_cast<int32_t>(p.groups.size());
    for (size_t g = 0; g < p.groups.size(); ++g) {
      info->group_scale[g] = p.groups[g].scale;
      info->q_begin[g] = p.groups[g].q_begin;
      info->q_end[g] = p.groups[g].q_end;
      info->n_kv[g] = p.groups[g].n_kv;
      info->pooled_k_offset[g] = p.pooled_k_off[g];
      info->pooled_v_offset[g] = p.pooled_v_off[g];
      info->pooled_tokens[g] = p.pooled_tokens[g];
    }
    return MSSA_OK;
  });
}

mssa_status mssa_plan_tables(mssa_plan plan, int64_t* dst, int64_t cap, int64_t* needed) {
  return guarded("mssa_plan_tables", [&]() -> mssa_status {
    if (!plan || !needed) return fail(MSSA_ERR_INVALID_ARG, "plan and needed must be non-null");
    const std::vector<int64_t> t = mssa::export_tables(plan->p);
    *needed = static_cast<int64_t>(t.size());
    if (!dst || cap < *needed) return fail(MSSA_ERR_INVALID_ARG, "table buffer too small");
    std::memcpy(dst, t.data(), t.size() * sizeof(int64_t));
    return MSSA_OK;
  });
}

mssa_status mssa_pool_kv(mssa_plan plan, const void* k_hist, const void* v_hist, const void* k_win,
                         const void* v_win, void* workspace, int64_t workspace_bytes, void* stream) {
  return guarded("mssa_pool_kv", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa_status s = pool_check(plan->p, k_hist, v_hist, k_win, v_win, workspace, workspace_bytes);
    if (s != MSSA_OK) return s;
    return pool_launch(plan->p, k_hist, v_hist, k_win, v_win, workspace, stream);
  });
}

mssa_status mssa_forward(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                         const void* k_hist, const void* v_hist, const void* k_win, const void* v_win,
                         const void* workspace, int64_t workspace_bytes, void* out, void* stream) {
  return guarded("mssa_forward", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    if (plan->p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "plan has MSSA_PLAN_POOLED_HIST_RING: use mssa_forward_ring");
    return forward_impl(plan->p, q_win, k_sink, v_sink, k_hist, v_hist, nullptr, nullptr, k_win, v_win, workspace,
                        workspace_bytes, out, nullptr, stream);
  });
}

mssa_status mssa_forward_ring(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                              const void* k_hist, const void* v_hist, const void* const* k_hist_pooled,
                              const void* const* v_hist_pooled, const void* k_win, const void* v_win,
                              const void* workspace, int64_t workspace_bytes, void* out, void* stream) {
  return guarded("mssa_forward_ring", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    if (!plan->p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "plan lacks MSSA_PLAN_POOLED_HIST_RING: use mssa_forward");
    return forward_impl(plan->p, q_win, k_sink, v_sink, k_hist, v_hist, k_hist_pooled, v_hist_pooled, k_win, v_win,
                        workspace, workspace_bytes, out, nullptr, stream);
  });
}

mssa_status mssa_forward_lse(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                             const void* k_hist, const void* v_hist, const void* k_win, const void* v_win,
                             const void* workspace, int64_t workspace_bytes, void* out, float* lse, void* stream) {
  return guarded("mssa_forward_lse", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    if (plan->p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "mssa_forward_lse takes plans without MSSA_PLAN_POOLED_HIST_RING");
    if (!lse) return fail(MSSA_ERR_INVALID_ARG, "lse must be non-null");
    return forward_impl(plan->p, q_win, k_sink, v_sink, k_hist, v_hist, nullptr, nullptr, k_win, v_win, workspace,
                        workspace_bytes, out, lse, stream);
  });
}

mssa_status mssa_attention_noalloc(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                                   const void* k_hist, const void* v_hist, const void* k_win, const void* v_win,
                                   void* out, void* stream) {
  return guarded("mssa_attention_noalloc", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    if (p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "plan has MSSA_PLAN_POOLED_HIST_RING: use mssa_forward_ring");
    if (p.workspace_bytes > mssa::kScratchBytes)
      return fail(MSSA_ERR_WORKSPACE, "the plan's workspace_bytes exceed MSSA_NOALLOC_SCRATCH_BYTES");
    void* ws = nullptr;
    mssa_status s = check_device(mssa::scratch_address(&ws), "library scratch lookup");
    if (s != MSSA_OK) return s;
    const int64_t wsb = mssa::kScratchBytes;
    s = pool_check(p, k_hist, v_hist, k_win, v_win, ws, wsb);
    if (s != MSSA_OK) return s;
    s = forward_check(p, q_win, k_sink, v_sink, k_hist, v_hist, nullptr, nullptr, k_win, v_win, ws, wsb, out,
                      nullptr);
    if (s != MSSA_OK) return s;
    s = pool_launch(p, k_hist, v_hist, k_win, v_win, ws, stream);
    if (s != MSSA_OK) return s;
    return forward_impl(p, q_win, k_sink, v_sink, k_hist, v_hist, nullptr, nullptr, k_win, v_win, ws, wsb, out,
                        nullptr, stream);
  });
}

mssa_status mssa_backward_workspace_size(mssa_plan plan, int64_t* bytes) {
  return guarded("mssa_backward_workspace_size", [&]() -> mssa_status {
    if (!plan || !bytes) return fail(MSSA_ERR_INVALID_ARG, "plan and bytes must be non-null");
    *bytes = plan->p.bwd_workspace_bytes;
    return MSSA_OK;
  });
}

mssa_status mssa_backward(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                          const void* k_hist, const void* v_hist, const void* k_win, const void* v_win,
                          const void* out, const float* lse, const void* d_out, void* workspace,
                          int64_t workspace_bytes, void* dq_win, void* dk_sink, void* dv_sink, void* dk_hist,
                          void* dv_hist, void* dk_win, void* dv_win, void* stream) {
  return guarded("mssa_backward", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    if (p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "mssa_backward takes plans without MSSA_PLAN_POOLED_HIST_RING");
    if (!q_win || !k_win || !v_win || !out || !lse || !d_out || !dq_win || !dk_win || !dv_win)
      return fail(MSSA_ERR_INVALID_ARG, "window tensors, out, lse, d_out and their gradients must be non-null");
    if (p.n_sink_tok > 0 && (!k_sink || !v_sink || !dk_sink || !dv_sink))
      return fail(MSSA_ERR_INVALID_ARG, "sink tensors and their gradients must be non-null when sink_frames > 0");
    if (p.n_hist_tok > 0 && (!k_hist || !v_hist || !dk_hist || !dv_hist))
      return fail(MSSA_ERR_INVALID_ARG, "history tensors and their gradients must be non-null when hist_frames > 0");
    if (!workspace || workspace_bytes < p.bwd_workspace_bytes)
      return fail(MSSA_ERR_WORKSPACE, "workspace smaller than mssa_backward_workspace_size");
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
      return fail(MSSA_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    const void* ins[] = {q_win, k_sink, v_sink, k_hist, v_hist, k_win, v_win, out, lse, d_out};
    const void* grads[] = {dq_win, dk_sink, dv_sink, dk_hist, dv_hist, dk_win, dv_win};
    for (const void* t : ins)
      if (t && !aligned16(t)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    for (const void* t : grads) {
      if (!t) continue;
      if (!aligned16(t)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
      for (const void* u : ins)
        if (t == u) return fail(MSSA_ERR_INVALID_ARG, "gradients must not alias an input");
    }
    const int G = static_cast<int>(p.groups.size());
    if (G > mssa::kMaxGroups) return fail(MSSA_ERR_UNSUPPORTED, "too many query scales");
    if (p.scatter_jobs.size() > static_cast<size_t>(mssa::kMaxScatterJobs))
      return fail(MSSA_ERR_UNSUPPORTED, "too many source frame runs");

    const bool bf16 = p.desc.dtype == MSSA_BF16;
    const int hd = p.desc.head_dim, nh = p.desc.num_heads;
    auto hs = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    float* dsum = reinterpret_cast<float*>(ws + p.bwd_dsum_off);
    float* lse2 = reinterpret_cast<float*>(ws + p.bwd_lse2_off);

    mssa::DotArgs da{};
    da.out = out;
    da.d_out = d_out;
    da.dsum = dsum;
    da.lse = bf16 ? lse : nullptr;
    da.lse2 = lse2;
    da.ld = p.ld;
    da.n_q = static_cast<int32_t>(p.n_q);
    da.num_heads = nh;
    da.head_dim = hd;
    {
      float sc = 0.f, sc2 = 0.f;
      set_score_scales(p, sc, sc2);
      da.inv_scale = 1.0f / sc;
    }
    mssa_status s = check_device(mssa::launch_bwd_dot(da, bf16, hs), "backward rowsum launch");
    if (s != MSSA_OK) return s;

    mssa::BwdArgs a{};
    a.q = q_win;
    a.d_out = d_out;
    a.lse = lse;
    a.dsum = dsum;
    a.lse2 = lse2;
    a.dq = dq_win;
    a.ld = p.ld;
    a.n_q = static_cast<int32_t>(p.n_q);
    a.num_heads = nh;
    a.n_groups = G;
    set_score_scales(p, a.scale, a.scale_log2e);
    a.q_prescaled = p.q_prescaled ? 1 : 0;
    const int qb = bf16 ? mssa::kBwdQ : mssa::kBwdF32, kb = bf16 ? mssa::kBwdK : mssa::kBwdF32;
    const KvSources src{k_sink, v_sink, k_hist, v_hist, nullptr, nullptr, k_win, v_win, ws};
    int gi = 0;
    for (int g : p.order) {
      mssa::BwdGroupArgs& A = a.groups[gi++];
      const mssa::QGroup& Q = p.groups[g];
      A.q_begin = Q.q_begin;
      A.q_end = Q.q_end;
      A.n_kv = static_cast<int32_t>(Q.n_kv);
      if (p.runs[g].size() > static_cast<size_t>(mssa::kMaxRuns))
        return fail(MSSA_ERR_UNSUPPORTED, "too many context runs for one query scale");
      A.n_runs = static_cast<int32_t>(p.runs[g].size());
      for (size_t r = 0; r < p.runs[g].size(); ++r) {
        run_pointers(p, g, p.runs[g][r], src, &A.runs[r].k, &A.runs[r].v);
        A.runs[r].n_tok = static_cast<int32_t>(p.runs[g][r].n_tok);
      }
      A.dk_ctx = reinterpret_cast<float*>(ws + p.bwd_dk_off[g]);
      A.dv_ctx = reinterpret_cast<float*>(ws + p.bwd_dv_off[g]);
      A.ds = bf16 ? ws + p.bwd_ds_off[g] : nullptr;
      A.ds_stages = p.bwd_ds_stages[g];
      A.ds_qblocks = p.bwd_ds_qblocks[g];
      A.n_qblocks = (Q.q_end - Q.q_begin + qb - 1) / qb;
      A.n_kblocks = static_cast<int32_t>((Q.n_kv + kb - 1) / kb);
    }
    // bf16: heads in chunks of bwd_ds_heads, each chunk's dK/dV kernel
    // writing the dS tiles its dQ kernel reads; fp32: one launch of each.
    const int chunk = bf16 ? p.bwd_ds_heads : nh;
    for (int h0 = 0; h0 < nh; h0 += chunk) {
      a.head0 = h0;
      a.num_heads = std::min(chunk, nh - h0);
      int64_t dq_blocks = 0, kv_blocks = 0;
      for (int g = 0; g < G; ++g) {
        mssa::BwdGroupArgs& A = a.groups[g];
        A.dq_block_begin = static_cast<int32_t>(dq_blocks);
        A.kv_block_begin = static_cast<int32_t>(kv_blocks);
        dq_blocks += static_cast<int64_t>(A.n_qblocks) * a.num_heads;
        kv_blocks += static_cast<int64_t>(A.n_kblocks) * a.num_heads;
      }
      if (dq_blocks > 0x7fffffff || kv_blocks > 0x7fffffff)
        return fail(MSSA_ERR_UNSUPPORTED, "backward grid too large");
      s = check_device(mssa::launch_bwd(a, static_cast<int>(dq_blocks), static_cast<int>(kv_blocks), hd, bf16, hs),
                       "backward attention launch");
      if (s != MSSA_OK) return s;
    }

    mssa::ScatterArgs sa{};
    for (int g = 0; g < G; ++g) {
      sa.ctx_k[g] = reinterpret_cast<const float*>(ws + p.bwd_dk_off[g]);
      sa.ctx_v[g] = reinterpret_cast<const float*>(ws + p.bwd_dv_off[g]);
    }
    sa.ld = p.ld;
    sa.chunks_per_tok = static_cast<int32_t>(p.ld * p.elem_bytes / 16);
    sa.n_groups = G;
    sa.pick_first = p.strided ? 1 : 0;
    const int64_t row_bytes = p.ld * p.elem_bytes;
    int64_t blocks = 0;
    int nj = 0;
    for (const mssa::ScatterJob& J : p.scatter_jobs) {
      mssa::ScatterJobArgs& A = sa.jobs[nj++];
      char* dk = static_cast<char*>(J.buffer == mssa::kBufSink ? dk_sink : J.buffer == mssa::kBufHist ? dk_hist : dk_win);
      char* dv = static_cast<char*>(J.buffer == mssa::kBufSink ? dv_sink : J.buffer == mssa::kBufHist ? dv_hist : dv_win);
      A.dst_k = dk + J.src_tok * row_bytes;
      A.dst_v = dv + J.src_tok * row_bytes;
      A.n_frames = J.n_frames;
      A.gh = J.gh;
      A.gw = J.gw;
      A.block_begin = static_cast<int32_t>(blocks);
      for (int g = 0; g < G; ++g) {
        A.g[g].ctx_begin = J.ctx_begin[g];
        A.g[g].frame_stride = J.frame_stride[g];
        A.g[g].factor = J.factor[g];
      }
      const int64_t work = static_cast<int64_t>(J.n_frames) * J.gh * J.gw * sa.chunks_per_tok;
      blocks += (work + mssa::kPoolThreads - 1) / mssa::kPoolThreads;
    }
    sa.n_jobs = nj;
    if (blocks > 0x7fffffff) return fail(MSSA_ERR_UNSUPPORTED, "scatter grid too large");
    return check_device(mssa::launch_scatter(sa, static_cast<int>(blocks), bf16, hs), "backward scatter launch");
  });
}

// ---------------------------------------------------------------- MSP tiers

namespace {

// Per query group: first window frame, frame count, patch size and patch-row
// features, and the group's patch rows in the tier workspace.
struct TierGroup {
  int64_t frame0, n_frames;
  int32_t P, kp;
  int64_t rows_off;
  int64_t partial_off;  // fp32 partial tiles of a GEMM split over K (shared by the groups, used in turn)
};

mssa_status tier_layout(const mssa::Plan& p, const mssa_tier_desc* t, std::vector<TierGroup>& out, int64_t* bytes) {
  if (!t) return fail(MSSA_ERR_INVALID_ARG, "tier must be non-null");
  if (p.desc.dtype != MSSA_BF16) return fail(MSSA_ERR_UNSUPPORTED, "tier kernels take bf16 plans");
  if (t->latent_channels < 1 || t->patch < 1 || t->hidden < 8 || t->hidden % 8 != 0)
    return fail(MSSA_ERR_INVALID_ARG, "latent_channels and patch must be >= 1, hidden a positive multiple of 8");
  out.clear();
  int64_t off = 0, frame = 0;
  for (const mssa::QGroup& g : p.groups) {
    TierGroup tg{};
    tg.P = t->patch * g.scale;
    const int64_t kp = static_cast<int64_t>(t->latent_channels) * tg.P * tg.P;
    if (kp % 8 != 0 || kp > (1 << 20)) return fail(MSSA_ERR_UNSUPPORTED, "C * (patch * scale)^2 must be a multiple of 8");
    tg.kp = static_cast<int32_t>(kp);
    const int64_t tok = static_cast<int64_t>((p.desc.grid_h + g.scale - 1) / g.scale) *
                        ((p.desc.grid_w + g.scale - 1) / g.scale);
    tg.n_frames = (g.q_end - g.q_begin) / tok;
    tg.frame0 = frame;
    frame += tg.n_frames;
    tg.rows_off = off;
    off += (static_cast<int64_t>(g.q_end - g.q_begin) * kp * 2 + 255) / 256 * 256;
    out.push_back(tg);
  }
  // the embedding (K = C (p s)^2) and de-embedding (N = C (p s)^2) GEMMs of
  // every group may split over K into this region
  int64_t partial = 0;
  for (size_t i = 0; i < out.size(); ++i) {
    const int32_t m = p.groups[i].q_end - p.groups[i].q_begin;
    partial = std::max({partial, mssa::gemm_split_bytes(m, t->hidden, out[i].kp),
                        mssa::gemm_split_bytes(m, out[i].kp, t->hidden)});
  }
  for (TierGroup& tg : out) tg.partial_off = off;
  *bytes = off + (partial + 255) / 256 * 256;
  return MSSA_OK;
}

}  // namespace

mssa_status mssa_tier_workspace_size(mssa_plan plan, const mssa_tier_desc* tier, int64_t* bytes) {
  return guarded("mssa_tier_workspace_size", [&]() -> mssa_status {
    if (!plan || !bytes) return fail(MSSA_ERR_INVALID_ARG, "plan and bytes must be non-null");
    std::vector<TierGroup> tg;
    return tier_layout(plan->p, tier, tg, bytes);
  });
}

mssa_status mssa_patch_embed(mssa_plan plan, const mssa_tier_desc* tier, const void* latent,
                             const void* const* w_embed, const void* const* b_embed, void* workspace,
                             int64_t workspace_bytes, void* tokens, void* stream) {
  return guarded("mssa_patch_embed", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    std::vector<TierGroup> tg;
    int64_t need = 0;
    mssa_status s = tier_layout(p, tier, tg, &need);
    if (s != MSSA_OK) return s;
    if (!latent || !w_embed || !b_embed || !tokens) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    if (!workspace || workspace_bytes < need) return fail(MSSA_ERR_WORKSPACE, "workspace smaller than mssa_tier_workspace_size");
    if (!aligned16(latent) || !aligned16(tokens) || !aligned16(workspace))
      return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    for (size_t g = 0; g < tg.size(); ++g)
      if (!w_embed[g] || !b_embed[g] || !aligned16(w_embed[g])) return fail(MSSA_ERR_INVALID_ARG, "null or misaligned tier weights");
    auto hs = static_cast<hipStream_t>(stream);
    const int32_t H = p.desc.grid_h * tier->patch, W = p.desc.grid_w * tier->patch, hid = tier->hidden;
    for (size_t g = 0; g < tg.size(); ++g) {
      const TierGroup& t = tg[g];
      const mssa::QGroup& Q = p.groups[g];
      mssa::PatchArgs pa{};
      pa.latent = const_cast<void*>(latent);
      pa.rows = static_cast<char*>(workspace) + t.rows_off;
      pa.frame0 = t.frame0;
      pa.n_frames = t.n_frames;
      pa.C = tier->latent_channels;
      pa.H = H;
      pa.W = W;
      pa.P = t.P;
      pa.gh = (H + t.P - 1) / t.P;
      pa.gw = (W + t.P - 1) / t.P;
      s = check_device(mssa::launch_patchify(pa, hs), "patchify launch");
      if (s != MSSA_OK) return s;
      mssa::GemmArgs ga{};
      ga.y0_scale = 1.f;
      ga.x = pa.rows;
      ga.w = w_embed[g];
      ga.bias = b_embed[g];
      ga.y[0] = static_cast<char*>(tokens) + static_cast<int64_t>(Q.q_begin) * hid * 2;
      ga.M = Q.q_end - Q.q_begin;
      ga.N = hid;
      ga.K = t.kp;
      ga.split = hid;
      ga.ldx = t.kp;
      ga.ldy = hid;
      s = check_device(mssa::launch_gemm_split(ga, reinterpret_cast<float*>(static_cast<char*>(workspace) + t.partial_off), hs),
                       "patch embedding GEMM launch");
      if (s != MSSA_OK) return s;
    }
    return MSSA_OK;
  });
}

mssa_status mssa_patch_unembed(mssa_plan plan, const mssa_tier_desc* tier, const void* tokens,
                               const void* const* w_out, const void* const* b_out, void* workspace,
                               int64_t workspace_bytes, void* latent, void* stream) {
  return guarded("mssa_patch_unembed", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    std::vector<TierGroup> tg;
    int64_t need = 0;
    mssa_status s = tier_layout(p, tier, tg, &need);
    if (s != MSSA_OK) return s;
    if (!latent || !w_out || !b_out || !tokens) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    if (!workspace || workspace_bytes < need) return fail(MSSA_ERR_WORKSPACE, "workspace smaller than mssa_tier_workspace_size");
    if (!aligned16(latent) || !aligned16(tokens) || !aligned16(workspace))
      return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    for (size_t g = 0; g < tg.size(); ++g)
      if (!w_out[g] || !b_out[g] || !aligned16(w_out[g])) return fail(MSSA_ERR_INVALID_ARG, "null or misaligned tier weights");
    auto hs = static_cast<hipStream_t>(stream);
    const int32_t H = p.desc.grid_h * tier->patch, W = p.desc.grid_w * tier->patch, hid = tier->hidden;
    for (size_t g = 0; g < tg.size(); ++g) {
      const TierGroup& t = tg[g];
      const mssa::QGroup& Q = p.groups[g];
      mssa::GemmArgs ga{};
      ga.y0_scale = 1.f;
      ga.x = static_cast<const char*>(tokens) + static_cast<int64_t>(Q.q_begin) * hid * 2;
      ga.w = w_out[g];
      ga.bias = b_out[g];
      ga.y[0] = static_cast<char*>(workspace) + t.rows_off;
      ga.M = Q.q_end - Q.q_begin;
      ga.N = t.kp;
      ga.K = hid;
      ga.split = t.kp;
      ga.ldx = hid;
      ga.ldy = t.kp;
      s = check_device(mssa::launch_gemm_split(ga, reinterpret_cast<float*>(static_cast<char*>(workspace) + t.partial_off), hs),
                       "patch de-embedding GEMM launch");
      if (s != MSSA_OK) return s;
      mssa::PatchArgs pa{};
      pa.latent = latent;
      pa.rows = ga.y[0];
      pa.frame0 = t.frame0;
      pa.n_frames = t.n_frames;
      pa.C = tier->latent_channels;
      pa.H = H;
      pa.W = W;
      pa.P = t.P;
      pa.gh = (H + t.P - 1) / t.P;
      pa.gw = (W + t.P - 1) / t.P;
      s = check_device(mssa::launch_unpatchify(pa, hs), "unpatchify launch");
      if (s != MSSA_OK) return s;
    }
    return MSSA_OK;
  });
}

namespace {

mssa_status qkv_project(const char* who, int64_t n_tokens, int32_t hidden, const void* x, const void* w_qkv,
                        const void* b_qkv, float q_scale, void* q, void* k, void* v, void* stream) {
  return guarded(who, [&]() -> mssa_status {
    if (n_tokens < 0 || n_tokens > 0x7fffffff || hidden < 8 || hidden % 8 != 0 || hidden > (1 << 20))
      return fail(MSSA_ERR_INVALID_ARG, "n_tokens must fit int32 and hidden be a positive multiple of 8");
    if (!x || !w_qkv || !b_qkv || !q || !k || !v) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    if (!std::isfinite(q_scale)) return fail(MSSA_ERR_INVALID_ARG, "q_scale must be finite");
    for (const void* t : {x, w_qkv, static_cast<const void*>(q), static_cast<const void*>(k), static_cast<const void*>(v)})
      if (!aligned16(t)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    if (q == x || k == x || v == x) return fail(MSSA_ERR_INVALID_ARG, "outputs must not alias x");
    mssa::GemmArgs ga{};
    ga.x = x;
    ga.w = w_qkv;
    ga.bias = b_qkv;
    ga.y[0] = q;
    ga.y[1] = k;
    ga.y[2] = v;
    ga.M = static_cast<int32_t>(n_tokens);
    ga.N = 3 * hidden;
    ga.K = hidden;
    ga.split = hidden;
    ga.ldx = hidden;
    ga.ldy = hidden;
    ga.y0_scale = q_scale;
    return check_device(mssa::launch_gemm(ga, static_cast<hipStream_t>(stream)), "QKV GEMM launch");
  });
}

}  // namespace

mssa_status mssa_qkv_project(int64_t n_tokens, int32_t hidden, const void* x, const void* w_qkv, const void* b_qkv,
                             void* q, void* k, void* v, void* stream) {
  return qkv_project("mssa_qkv_project", n_tokens, hidden, x, w_qkv, b_qkv, 1.f, q, k, v, stream);
}

mssa_status mssa_qkv_project_scaled(int64_t n_tokens, int32_t hidden, const void* x, const void* w_qkv,
                                    const void* b_qkv, float q_scale, void* q, void* k, void* v, void* stream) {
  return qkv_project("mssa_qkv_project_scaled", n_tokens, hidden, x, w_qkv, b_qkv, q_scale, q, k, v, stream);
}

mssa_status mssa_hist_append(mssa_plan plan, const void* k_win, const void* v_win, void* k_ring, void* v_ring,
                             int32_t ring_cap_frames, int32_t* ring_head, int32_t* ring_count, void* stream) {
  return guarded("mssa_hist_append", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    std::vector<int32_t> slots;
    return append_native(plan->p, k_win, v_win, k_ring, v_ring, ring_cap_frames, ring_head, ring_count, slots,
                         stream);
  });
}

mssa_status mssa_hist_append_ring(mssa_plan plan, const void* k_win, const void* v_win, const void* workspace,
                                  int64_t workspace_bytes, void* k_ring, void* v_ring, void* const* k_ring_pooled,
                                  void* const* v_ring_pooled, int32_t ring_cap_frames, int32_t* ring_head,
                                  int32_t* ring_count, void* stream) {
  return guarded("mssa_hist_append_ring", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    const mssa::Plan& p = plan->p;
    if (!p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "plan lacks MSSA_PLAN_POOLED_HIST_RING: use mssa_hist_append");
    if (!k_ring_pooled || !v_ring_pooled) return fail(MSSA_ERR_INVALID_ARG, "null pooled ring array");
    bool coarse = false;
    for (size_t g = 0; g < p.groups.size(); ++g) {
      if (p.groups[g].scale == 1) continue;
      coarse = true;
      if (!k_ring_pooled[g] || !v_ring_pooled[g])
        return fail(MSSA_ERR_INVALID_ARG, "null pooled-history ring for a coarse query scale");
    }
    if (coarse && (!workspace || workspace_bytes < p.workspace_bytes))
      return fail(MSSA_ERR_WORKSPACE, "workspace smaller than mssa_plan_info.workspace_bytes");
    std::vector<int32_t> slots;
    const mssa_status s0 = append_native(p, k_win, v_win, k_ring, v_ring, ring_cap_frames, ring_head, ring_count,
                                         slots, stream);
    if (s0 != MSSA_OK) return s0;
    // The head state's frames pooled to each coarse scale: window frames
    // 0 .. F-1 of that group's context, which mssa_pool_kv wrote to the
    // group's pooled block.
    const int64_t row_bytes = p.ld * p.elem_bytes;
    const char* ws = static_cast<const char*>(workspace);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    for (size_t g = 0; g < p.groups.size(); ++g) {
      const int32_t sc = p.groups[g].scale;
      if (sc == 1) continue;
      const int64_t tok_s = frame_tokens(p, sc);
      const size_t fbytes = static_cast<size_t>(tok_s * row_bytes);
      for (const mssa::SegRow& r : p.segs) {
        if (r.q_scale != sc || r.kind != mssa::kWin || r.frame >= p.desc.frames_per_state) continue;
        if (r.buffer != mssa::kBufPooled || r.n_tok != tok_s)
          return fail(MSSA_ERR_UNSUPPORTED, "head frames are not pooled to a coarse scale in this plan");
        const size_t slot = static_cast<size_t>(slots[r.frame]);
        mssa_status s = check_device(
            hipMemcpyAsync(static_cast<char*>(k_ring_pooled[g]) + slot * fbytes,
                           ws + p.pooled_k_off[g] + r.tok_offset * row_bytes, fbytes, hipMemcpyDeviceToDevice, st),
            "pooled history append (K)");
        if (s != MSSA_OK) return s;
        s = check_device(
            hipMemcpyAsync(static_cast<char*>(v_ring_pooled[g]) + slot * fbytes,
                           ws + p.pooled_v_off[g] + r.tok_offset * row_bytes, fbytes, hipMemcpyDeviceToDevice, st),
            "pooled history append (V)");
        if (s != MSSA_OK) return s;
      }
    }
    return MSSA_OK;
  });
}

mssa_status mssa_pool_hist_ring(mssa_plan plan, const void* k_ring, const void* v_ring, void* const* k_ring_pooled,
                                void* const* v_ring_pooled, void* stream) {
  return guarded("mssa_pool_hist_ring", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    if (!p.hist_ring)
      return fail(MSSA_ERR_UNSUPPORTED, "plan lacks MSSA_PLAN_POOLED_HIST_RING");
    if (p.n_hist_tok == 0) return MSSA_OK;
    if (!k_ring || !v_ring || !k_ring_pooled || !v_ring_pooled) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    if (!aligned16(k_ring) || !aligned16(v_ring)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    std::vector<mssa::PoolJobArgs> jobs;
    for (size_t g = 0; g < p.groups.size(); ++g) {
      const int32_t sc = p.groups[g].scale;
      if (sc == 1) continue;
      if (!k_ring_pooled[g] || !v_ring_pooled[g])
        return fail(MSSA_ERR_INVALID_ARG, "null pooled-history ring for a coarse query scale");
      if (!aligned16(k_ring_pooled[g]) || !aligned16(v_ring_pooled[g]))
        return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
      mssa::PoolJobArgs A{};
      A.src_k = k_ring;
      A.src_v = v_ring;
      A.dst_k = k_ring_pooled[g];
      A.dst_v = v_ring_pooled[g];
      A.src_gh = p.desc.grid_h;
      A.src_gw = p.desc.grid_w;
      A.factor = sc;
      A.dst_gh = (p.desc.grid_h + sc - 1) / sc;
      A.dst_gw = (p.desc.grid_w + sc - 1) / sc;
      A.n_frames = p.desc.hist_frames;
      jobs.push_back(A);
    }
    return launch_pool_jobs(p, jobs, stream);
  });
}

mssa_status mssa_pool_kv_head_ring(mssa_plan plan, const void* k_ring, const void* v_ring, const void* k_win,
                                   const void* v_win, void* const* k_ring_pooled, void* const* v_ring_pooled,
                                   void* workspace, int64_t workspace_bytes, int32_t ring_frames,
                                   int32_t ring_count, int32_t ring_spare, void* stream) {
  return guarded("mssa_pool_kv_head_ring", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    mssa_status s = head_ring_check(p, ring_frames, ring_count, ring_spare);
    if (s != MSSA_OK) return s;
    if (!k_ring || !v_ring || !k_ring_pooled || !v_ring_pooled)
      return fail(MSSA_ERR_INVALID_ARG, "k_ring, v_ring and the pooled ring arrays must be non-null");
    if (!aligned16(k_ring) || !aligned16(v_ring)) return fail(MSSA_ERR_INVALID_ARG, "tensors must be 16-byte aligned");
    for (size_t g = 0; g < p.groups.size(); ++g) {
      if (p.groups[g].scale == 1) continue;
      if (!k_ring_pooled[g] || !v_ring_pooled[g] || !aligned16(k_ring_pooled[g]) || !aligned16(v_ring_pooled[g]))
        return fail(MSSA_ERR_INVALID_ARG, "null or misaligned pooled ring for a coarse query scale");
    }
    s = pool_check(p, nullptr, nullptr, k_win, v_win, workspace, workspace_bytes);
    if (s != MSSA_OK) return s;
    // the plan's jobs (window states 2..T into the workspace), then state 1
    // from the native ring's spare slots into every pooled ring's
    const int64_t rb = p.ld * p.elem_bytes;
    auto* ws = static_cast<char*>(workspace);
    std::vector<mssa::PoolJobArgs> jobs;
    for (const mssa::PoolJob& J : p.pool_jobs) {
      mssa::PoolJobArgs A{};
      A.src_k = static_cast<const char*>(k_win) + J.src_tok * rb;
      A.src_v = static_cast<const char*>(v_win) + J.src_tok * rb;
      A.dst_k = ws + p.pooled_k_off[J.group] + J.dst_tok * rb;
      A.dst_v = ws + p.pooled_v_off[J.group] + J.dst_tok * rb;
      A.src_gh = J.src_gh;
      A.src_gw = J.src_gw;
      A.dst_gh = J.dst_gh;
      A.dst_gw = J.dst_gw;
      A.factor = J.factor;
      A.n_frames = J.n_frames;
      jobs.push_back(A);
    }
    for (size_t g = 0; g < p.groups.size(); ++g) {
      const int32_t sc = p.groups[g].scale;
      if (sc == 1) continue;
      mssa::PoolJobArgs A{};
      const int64_t tok_s = frame_tokens(p, sc);
      A.src_k = static_cast<const char*>(k_ring) + int64_t{ring_spare} * p.tok1 * rb;
      A.src_v = static_cast<const char*>(v_ring) + int64_t{ring_spare} * p.tok1 * rb;
      A.dst_k = static_cast<char*>(k_ring_pooled[g]) + int64_t{ring_spare} * tok_s * rb;
      A.dst_v = static_cast<char*>(v_ring_pooled[g]) + int64_t{ring_spare} * tok_s * rb;
      A.src_gh = p.desc.grid_h;
      A.src_gw = p.desc.grid_w;
      A.factor = sc;
      A.dst_gh = (p.desc.grid_h + sc - 1) / sc;
      A.dst_gw = (p.desc.grid_w + sc - 1) / sc;
      A.n_frames = p.desc.frames_per_state;
      jobs.push_back(A);
    }
    if (jobs.empty()) return MSSA_OK;
    return launch_pool_jobs(p, jobs, stream);
  });
}

mssa_status mssa_forward_head_ring(mssa_plan plan, const void* q_win, const void* k_sink, const void* v_sink,
                                   const void* k_ring, const void* v_ring, const void* const* k_ring_pooled,
                                   const void* const* v_ring_pooled, const void* k_win, const void* v_win,
                                   const void* workspace, int64_t workspace_bytes, void* out, int32_t ring_frames,
                                   int32_t ring_count, int32_t ring_spare, void* stream) {
  return guarded("mssa_forward_head_ring", [&]() -> mssa_status {
    if (!plan) return fail(MSSA_ERR_INVALID_ARG, "plan must be non-null");
    const mssa::Plan& p = plan->p;
    mssa_status s = head_ring_check(p, ring_frames, ring_count, ring_spare);
    if (s != MSSA_OK) return s;
    if (!k_ring || !v_ring || !k_ring_pooled || !v_ring_pooled)
      return fail(MSSA_ERR_INVALID_ARG, "k_ring, v_ring and the pooled ring arrays must be non-null");
    for (size_t g = 0; g < p.groups.size(); ++g)
      if (p.groups[g].scale > 1 && (!k_ring_pooled[g] || !v_ring_pooled[g]))
        return fail(MSSA_ERR_INVALID_ARG, "null pooled ring for a coarse query scale");
    // state 2 onwards may be empty (a single state): k_win may then be null
    const bool rest = p.n_q > p.win_shift;
    s = forward_check(p, q_win, k_sink, v_sink, k_ring, v_ring, k_ring_pooled, v_ring_pooled,
                      rest ? k_win : k_ring, rest ? v_win : v_ring, workspace, workspace_bytes, out, nullptr);
    if (s != MSSA_OK) return s;
    const GroupRuns runs = head_ring_runs(p, k_sink, v_sink, k_ring, v_ring, k_ring_pooled, v_ring_pooled, k_win,
                                          v_win, static_cast<const char*>(workspace), ring_frames, ring_count,
                                          ring_spare);
    std::vector<std::vector<int64_t>> n_tok(runs.size());
    for (size_t g = 0; g < runs.size(); ++g)
      for (const PtrRun& r : runs[g]) n_tok[g].push_back(r.n_tok);
    return forward_launch(p, runs, mssa::make_schedule(p, n_tok), q_win, workspace, out, nullptr, stream);
  });
}

mssa_status mssa_head_ring_roll(mssa_plan plan, int32_t ring_frames, int32_t* ring_count, int32_t* ring_spare) {
  return guarded("mssa_head_ring_roll", [&]() -> mssa_status {
    if (!plan || !ring_count || !ring_spare) return fail(MSSA_ERR_INVALID_ARG, "null argument");
    const mssa::Plan& p = plan->p;
    const mssa_status s = head_ring_check(p, ring_frames, *ring_count, *ring_spare);
    if (s != MSSA_OK) return s;
    const int32_t F = p.desc.frames_per_state;
    *ring_count = std::min(*ring_count + F, ring_frames - F);
    *ring_spare = (*ring_spare + F) % ring_frames;
    return MSSA_OK;
  });
}

const char* mssa_status_string(mssa_status s) {
  switch (s) {
    case MSSA_OK: return "MSSA_OK";
    case MSSA_ERR_INVALID_ARG: return "MSSA_ERR_INVALID_ARG";
    case MSSA_ERR_UNSUPPORTED: return "MSSA_ERR_UNSUPPORTED";
    case MSSA_ERR_WORKSPACE: return "MSSA_ERR_WORKSPACE";
    case MSSA_ERR_DEVICE: return "MSSA_ERR_DEVICE";
    case MSSA_ERR_NO_MEMORY: return "MSSA_ERR_NO_MEMORY";
  }
  return "MSSA_ERR_UNKNOWN";
}

const char* mssa_last_error(void) { return g_last_error; }

}  // extern "C"
