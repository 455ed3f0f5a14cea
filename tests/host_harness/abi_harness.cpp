// Host harness of the scheduler and the C ABI, built without any GPU code
// (under AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitized.py).  The kernel launchers and the few HIP
// runtime calls the C ABI makes are replaced by stubs: a launcher stub checks
// that every address range the kernel would read or write, derived from its
// argument struct, lies inside a buffer the caller passed; a copy stub checks
// both ranges.  Device buffers are address ranges that are never
// dereferenced.
//
// The harness creates plans for the layer workloads, the streaming history
// lengths and 150 seeded random descriptors, calls every entry point on each
// (pool, forward, forward with lse, backward, cache roll, pooled rings, tier
// steps, QKV projection, the entry point without allocations), and checks
// that invalid descriptors and calls are rejected with the documented status.
// Exit status 0 iff every check passed.  With the argument "plant" every
// workspace is 256 bytes shorter than the size the harness passes, a mistake
// the range checks must report.
#include <hip/hip_runtime_api.h>

#include <cinttypes>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/libmssa.h"
#include "../../paper_2607_20940_amd/csrc/kernels.hpp"
#include "../../paper_2607_20940_amd/csrc/noalloc.hpp"

namespace {

int g_failures = 0;
int g_checks = 0;
bool g_plant = false;  // "plant": a workspace 256 bytes shorter than the size passed
std::string g_case;

void failure(const char* what) {
  ++g_failures;
  if (g_failures <= 40) std::fprintf(stderr, "FAIL [%s]: %s\n", g_case.c_str(), what);
}

// Fake device buffers: disjoint address ranges, 2^36 bytes apart.
struct Range {
  uintptr_t b, e;
};
std::vector<Range> g_bufs;
uintptr_t g_next = uintptr_t{1} << 44;

void* dev_alloc(int64_t bytes) {
  if (bytes <= 0) return nullptr;
  const uintptr_t b = g_next;
  g_next += uintptr_t{1} << 36;
  g_bufs.push_back({b, b + static_cast<uintptr_t>(bytes)});
  return reinterpret_cast<void*>(b);
}

// The library scratch of the entry point without allocations, at a fixed
// address of its own.
const uintptr_t kScratchBase = uintptr_t{1} << 46;

void dev_reset() {
  g_bufs.clear();
  g_next = uintptr_t{1} << 44;
  g_bufs.push_back({kScratchBase, kScratchBase + static_cast<uintptr_t>(mssa::kScratchBytes)});
}

// [p, p + bytes) inside one buffer?
void check_range(const void* p, int64_t bytes, const char* what) {
  ++g_checks;
  if (bytes <= 0) return;
  const uintptr_t b = reinterpret_cast<uintptr_t>(p);
  for (const Range& r : g_bufs)
    if (b >= r.b && b < r.e) {
      if (b + static_cast<uintptr_t>(bytes) > r.e) {
        char msg[256];
        std::snprintf(msg, sizeof msg, "%s: %" PRId64 " bytes from buffer offset %" PRIuPTR " overrun its %" PRIuPTR,
                      what, bytes, b - r.b, r.e - r.b);
        failure(msg);
      }
      return;
    }
  char msg[160];
  std::snprintf(msg, sizeof msg, "%s: address outside every buffer", what);
  failure(msg);
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace

// ------------------------------------------------------------ HIP runtime stubs
extern "C" {
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t attr, int) {
  *v = attr == hipDeviceAttributeMultiprocessorCount ? 256 : 0;
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stub"; }
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  check_range(dst, static_cast<int64_t>(n), "copy destination");
  check_range(src, static_cast<int64_t>(n), "copy source");
  return hipSuccess;
}
}

// ------------------------------------------------------------ launcher stubs
namespace mssa {

hipError_t scratch_address(void** out) {
  *out = reinterpret_cast<void*>(kScratchBase);
  return hipSuccess;
}

int forward_blocks_per_cu(int) { return 1; }

hipError_t launch_pool(const PoolArgs& a, int n_blocks, bool bf16, hipStream_t) {
  const int64_t rb = a.ld * (bf16 ? 2 : 4);
  if (a.chunks_per_tok * 16 != rb) failure("pool: chunks_per_tok");
  int64_t blocks = 0;
  for (int j = 0; j < a.n_jobs; ++j) {
    const PoolJobArgs& J = a.jobs[j];
    if (J.block_begin != blocks) failure("pool: block_begin");
    const int64_t src = int64_t{J.n_frames} * J.src_gh * J.src_gw * rb;
    check_range(J.src_k, src, "pool source K");
    check_range(J.src_v, src, "pool source V");
    check_range(J.dst_k, int64_t{J.n_frames} * J.dst_gh * J.dst_gw * rb, "pool destination K");
    check_range(J.dst_v, int64_t{J.n_frames} * J.dst_gh * J.dst_gw * rb, "pool destination V");
    if (J.dst_gh != ceil_div(J.src_gh, J.factor) || J.dst_gw != ceil_div(J.src_gw, J.factor))
      failure("pool: destination grid");
    int64_t cells = int64_t{J.dst_gh} * J.dst_gw;
    if (J.levels == 2) {
      check_range(J.dst2_k, int64_t{J.n_frames} * J.dst2_gh * J.dst2_gw * rb, "pool destination K (level 2)");
      check_range(J.dst2_v, int64_t{J.n_frames} * J.dst2_gh * J.dst2_gw * rb, "pool destination V (level 2)");
      if (J.dst2_gh != ceil_div(J.src_gh, 2 * J.factor) || J.dst2_gw != ceil_div(J.src_gw, 2 * J.factor))
        failure("pool: level-2 grid");
      cells = int64_t{J.dst2_gh} * J.dst2_gw;
    }
    blocks += ceil_div(int64_t{J.n_frames} * cells * a.chunks_per_tok, kPoolThreads);
  }
  if (blocks != n_blocks) failure("pool: grid size");
  return hipSuccess;
}

hipError_t launch_forward(const FwdArgs& a, int head_dim, bool bf16, hipStream_t) {
  const int64_t eb = bf16 ? 2 : 4, rb = a.ld * eb;
  if (a.ld != int64_t{a.num_heads} * head_dim) failure("forward: ld");
  check_range(a.q, a.n_q * rb, "forward q");
  check_range(a.out, a.n_q * rb, "forward out");
  if (a.lse) check_range(a.lse, int64_t{a.num_heads} * a.n_q * 4, "forward lse");
  const int bm = bf16 ? kFwdBM : kFwdF32BM;
  int64_t blocks = 0, tiles = 0;
  for (int g = 0; g < a.n_groups; ++g) {
    const FwdGroupArgs& G = a.groups[g];
    if (G.q_begin < 0 || G.q_end > a.n_q || G.q_begin >= G.q_end) failure("forward: query range");
    if (G.n_qtiles != ceil_div(G.q_end - G.q_begin, bm)) failure("forward: n_qtiles");
    if (G.block_begin != blocks) failure("forward: block_begin");
    int64_t t = 0;
    for (int r = 0; r < G.n_runs; ++r) {
      check_range(G.runs[r].k, int64_t{G.runs[r].n_tok} * rb, "forward K run");
      check_range(G.runs[r].v, int64_t{G.runs[r].n_tok} * rb, "forward V run");
      t += ceil_div(G.runs[r].n_tok, kFwdBN);
    }
    if (bf16 && (G.tiles_per_item != t || G.tile_begin != tiles)) failure("forward: tile counts");
    blocks += int64_t{G.n_qtiles} * a.num_heads;
    tiles += int64_t{G.n_qtiles} * a.num_heads * t;
  }
  if (blocks != a.n_blocks) failure("forward: n_blocks");
  if (bf16) {
    if (tiles != a.total_tiles) failure("forward: total_tiles");
    if (a.n_ranges > 1) {
      check_range(a.partial, 2 * int64_t{a.n_ranges} * partial_record_floats(head_dim) * 4, "forward partial records");
      check_range(a.range_table, (int64_t{a.n_ranges} + 1) * 8, "forward range table");
    }
    if (a.tail_begin < 0 || a.tail_begin > a.total_tiles) failure("forward: tail_begin");
  }
  return hipSuccess;
}

hipError_t launch_bwd_dot(const DotArgs& a, bool bf16, hipStream_t) {
  const int64_t rb = a.ld * (bf16 ? 2 : 4);
  check_range(a.out, a.n_q * rb, "rowsum out");
  check_range(a.d_out, a.n_q * rb, "rowsum d_out");
  check_range(a.dsum, int64_t{a.num_heads} * a.n_q * 4, "rowsum dsum");
  if (a.lse) {
    check_range(a.lse, int64_t{a.num_heads} * a.n_q * 4, "rowsum lse");
    check_range(a.lse2, int64_t{a.num_heads} * a.n_q * 4, "rowsum lse2");
  }
  return hipSuccess;
}

// Heads the backward launches of one call have covered so far, in order.
int64_t g_bwd_next_head = 0, g_bwd_heads = 0;

hipError_t launch_bwd(const BwdArgs& a, int dq_blocks, int kv_blocks, int head_dim, bool bf16, hipStream_t) {
  const int64_t rb = a.ld * (bf16 ? 2 : 4);
  if (head_dim <= 0 || a.ld % head_dim != 0) failure("backward: ld");
  const int64_t H = a.ld / head_dim;
  if (a.head0 == 0) g_bwd_next_head = 0;
  if (a.num_heads <= 0 || a.head0 != g_bwd_next_head || a.head0 + a.num_heads > H)
    failure("backward: launch heads");
  g_bwd_next_head = a.head0 + a.num_heads;
  g_bwd_heads = H;
  check_range(a.q, a.n_q * rb, "backward q");
  check_range(a.d_out, a.n_q * rb, "backward d_out");
  check_range(a.dq, a.n_q * rb, "backward dq");
  check_range(a.lse, H * a.n_q * 4, "backward lse");
  check_range(a.dsum, H * a.n_q * 4, "backward dsum");
  check_range(a.lse2, H * a.n_q * 4, "backward lse2");
  int64_t qblocks = 0, kblocks = 0;
  for (int g = 0; g < a.n_groups; ++g) {
    const BwdGroupArgs& G = a.groups[g];
    int64_t n = 0, stages = 0;
    for (int r = 0; r < G.n_runs; ++r) {
      check_range(G.runs[r].k, int64_t{G.runs[r].n_tok} * rb, "backward K run");
      check_range(G.runs[r].v, int64_t{G.runs[r].n_tok} * rb, "backward V run");
      n += G.runs[r].n_tok;
      stages += ceil_div(int64_t{G.runs[r].n_tok}, int64_t{kBwdKS});
    }
    if (n != G.n_kv) failure("backward: runs do not cover the context");
    check_range(G.dk_ctx, int64_t{G.n_kv} * a.ld * 4, "backward dK context");
    check_range(G.dv_ctx, int64_t{G.n_kv} * a.ld * 4, "backward dV context");
    if (G.dq_block_begin != qblocks || G.kv_block_begin != kblocks) failure("backward: block ranges");
    qblocks += int64_t{G.n_qblocks} * a.num_heads;
    kblocks += int64_t{G.n_kblocks} * a.num_heads;
    if (bf16) {
      // the dS tiles of every head of the launch, every 32-query block the
      // dK/dV kernel's 64-query stages write, every 64-key stage of the runs
      if (G.ds_stages != stages) failure("backward: dS stages");
      if (int64_t{G.ds_qblocks} < 2 * ceil_div(int64_t{G.q_end - G.q_begin}, int64_t{kBwdQS}) ||
          int64_t{G.n_qblocks} * kBwdQ > int64_t{G.ds_qblocks} * 32 + kBwdQ - 32)
        failure("backward: dS query blocks");
      check_range(G.ds, int64_t{a.num_heads} * G.ds_qblocks * G.ds_stages * kBwdKS * 32 * 2, "backward dS tiles");
    }
  }
  if (qblocks != dq_blocks || kblocks != kv_blocks) failure("backward: grid size");
  return hipSuccess;
}

hipError_t launch_scatter(const ScatterArgs& a, int n_blocks, bool bf16, hipStream_t) {
  if (g_bwd_next_head != g_bwd_heads) failure("backward: heads not covered before the scatter");
  const int64_t rb = a.ld * (bf16 ? 2 : 4);
  int64_t blocks = 0;
  for (int j = 0; j < a.n_jobs; ++j) {
    const ScatterJobArgs& J = a.jobs[j];
    if (J.block_begin != blocks) failure("scatter: block_begin");
    check_range(J.dst_k, int64_t{J.n_frames} * J.gh * J.gw * rb, "scatter dK");
    check_range(J.dst_v, int64_t{J.n_frames} * J.gh * J.gw * rb, "scatter dV");
    for (int g = 0; g < a.n_groups; ++g) {
      const ScatterGroupArgs& S = J.g[g];
      const int64_t rows = S.ctx_begin + int64_t{J.n_frames} * S.frame_stride;
      check_range(a.ctx_k[g] + S.ctx_begin * a.ld, (rows - S.ctx_begin) * a.ld * 4, "scatter context dK");
      check_range(a.ctx_v[g] + S.ctx_begin * a.ld, (rows - S.ctx_begin) * a.ld * 4, "scatter context dV");
    }
    blocks += ceil_div(int64_t{J.n_frames} * J.gh * J.gw * a.chunks_per_tok, kPoolThreads);
  }
  if (blocks != n_blocks) failure("scatter: grid size");
  return hipSuccess;
}

static void check_patch(const PatchArgs& a, const char* what) {
  check_range(static_cast<char*>(a.latent) + a.frame0 * a.C * a.H * a.W * 2, a.n_frames * a.C * a.H * a.W * 2, what);
  check_range(a.rows, a.n_frames * a.gh * a.gw * int64_t{a.C} * a.P * a.P * 2, what);
  if (a.gh != ceil_div(a.H, a.P) || a.gw != ceil_div(a.W, a.P)) failure("patch grid");
}

hipError_t launch_patchify(const PatchArgs& a, hipStream_t) {
  check_patch(a, "patchify");
  return hipSuccess;
}

hipError_t launch_unpatchify(const PatchArgs& a, hipStream_t) {
  check_patch(a, "unpatchify");
  return hipSuccess;
}

hipError_t launch_gemm(const GemmArgs& a, hipStream_t) {
  check_range(a.x, (int64_t{a.M} - 1) * a.ldx * 2 + int64_t{a.K} * 2, "gemm x");
  check_range(a.w, int64_t{a.N} * a.K * 2, "gemm w");
  check_range(a.bias, int64_t{a.N} * 2, "gemm bias");
  for (int j = 0; j * a.split < a.N; ++j)
    check_range(a.y[j], (int64_t{a.M} - 1) * a.ldy * 2 + int64_t{a.split} * 2, "gemm y");
  // only the QKV projection (three outputs) may scale its first output
  if (!std::isfinite(a.y0_scale) || (a.split == a.N && a.y0_scale != 1.f)) failure("gemm y0_scale");
  return hipSuccess;
}

hipError_t launch_gemm_split(const GemmArgs& a, float* partial, hipStream_t s) {
  const int64_t bytes = gemm_split_bytes(a.M, a.N, a.K);
  if (bytes > 0 && partial) check_range(partial, bytes, "gemm partial tiles");
  return launch_gemm(a, s);
}

}  // namespace mssa

// ------------------------------------------------------------ driving the entry points
namespace {

uint64_t g_rng = 0x9E3779B97F4A7C15ull;
uint32_t rnd(uint32_t n) {  // xorshift64*, uniform in [0, n)
  g_rng ^= g_rng >> 12;
  g_rng ^= g_rng << 25;
  g_rng ^= g_rng >> 27;
  return static_cast<uint32_t>((g_rng * 0x2545F4914F6CDD1Dull) >> 33) % n;
}

void expect(mssa_status got, mssa_status want, const char* what) {
  ++g_checks;
  if (got != want) {
    char msg[256];
    std::snprintf(msg, sizeof msg, "%s: status %s, expected %s (%s)", what, mssa_status_string(got),
                  mssa_status_string(want), mssa_last_error());
    failure(msg);
  }
}

mssa_plan_desc make_desc(int T, const int* scales, int H, int W, int F, int S, int Hh, int nh, int d, int dtype,
                         int flags) {
  mssa_plan_desc desc;
  std::memset(&desc, 0, sizeof desc);
  desc.num_states = T;
  for (int l = 0; l < T; ++l) desc.scales[l] = scales[l];
  desc.grid_h = H;
  desc.grid_w = W;
  desc.frames_per_state = F;
  desc.sink_frames = S;
  desc.hist_frames = Hh;
  desc.num_heads = nh;
  desc.head_dim = d;
  desc.dtype = dtype;
  desc.flags = flags;
  return desc;
}

// Every entry point on one descriptor, with buffers of exactly the sizes the
// header documents.
void exercise(const mssa_plan_desc& desc, int32_t attention_blocks) {
  dev_reset();
  mssa_plan plan = nullptr;
  expect(mssa_plan_create_ex(&desc, attention_blocks, &plan), MSSA_OK, "plan");
  if (!plan) return;
  mssa_plan_info info;
  expect(mssa_plan_query(plan, &info), MSSA_OK, "query");
  int64_t need = 0;
  mssa_plan_tables(plan, nullptr, 0, &need);
  std::vector<int64_t> tab(static_cast<size_t>(need));
  expect(mssa_plan_tables(plan, tab.data(), need, &need), MSSA_OK, "tables");
  {  // TOTAL pairs = sum over QGRP of queries x n_kv; QGRP equals the info
    const int64_t ng = tab[0], nq = tab[1], ns = tab[2];
    const int64_t* q = tab.data() + 3 + 4 * ng;
    int64_t pairs = 0;
    for (int64_t g = 0; g < nq; ++g) {
      pairs += (q[4 * g + 2] - q[4 * g + 1]) * q[4 * g + 3];
      if (q[4 * g + 3] != info.n_kv[g]) failure("QGRP n_kv differs from the plan info");
    }
    const int64_t* tot = tab.data() + 3 + 4 * ng + 4 * nq + 8 * ns;
    if (tot[1] != pairs || tot[0] != info.n_q) failure("TOTAL row");
    ++g_checks;
  }
  const bool ring = (desc.flags & MSSA_PLAN_POOLED_HIST_RING) != 0;
  const int64_t eb = desc.dtype == MSSA_BF16 ? 2 : 4, rb = int64_t{desc.num_heads} * desc.head_dim * eb;
  void* q = dev_alloc(info.n_q * rb);
  void* kw = dev_alloc(info.n_q * rb);
  void* vw = dev_alloc(info.n_q * rb);
  void* ks = dev_alloc(info.n_sink_tok * rb);
  void* vs = dev_alloc(info.n_sink_tok * rb);
  void* kh = dev_alloc(info.n_hist_tok * rb);
  void* vh = dev_alloc(info.n_hist_tok * rb);
  void* out = dev_alloc(info.n_q * rb);
  const int64_t wsb = info.workspace_bytes > 0 ? info.workspace_bytes : 256;
  void* ws = dev_alloc(g_plant && wsb > 256 ? wsb - 256 : wsb);
  expect(mssa_pool_kv(plan, kh, vh, kw, vw, ws, wsb, nullptr), MSSA_OK, "pool");
  const int32_t tok1 = desc.grid_h * desc.grid_w;
  if (!ring) {
    expect(mssa_forward(plan, q, ks, vs, kh, vh, kw, vw, ws, wsb, out, nullptr), MSSA_OK, "forward");
    if (info.workspace_bytes <= MSSA_NOALLOC_SCRATCH_BYTES)
      expect(mssa_attention_noalloc(plan, q, ks, vs, kh, vh, kw, vw, out, nullptr), MSSA_OK, "noalloc");
    else
      expect(mssa_attention_noalloc(plan, q, ks, vs, kh, vh, kw, vw, out, nullptr), MSSA_ERR_WORKSPACE, "noalloc");
    void* lse = dev_alloc(int64_t{desc.num_heads} * info.n_q * 4);
    expect(mssa_forward_lse(plan, q, ks, vs, kh, vh, kw, vw, ws, wsb, out, static_cast<float*>(lse), nullptr),
           MSSA_OK, "forward_lse");
    int64_t bws = 0;
    expect(mssa_backward_workspace_size(plan, &bws), MSSA_OK, "backward workspace size");
    void* bw = dev_alloc(bws);
    void* dout = dev_alloc(info.n_q * rb);
    void* dq = dev_alloc(info.n_q * rb);
    void* dks = dev_alloc(info.n_sink_tok * rb);
    void* dvs = dev_alloc(info.n_sink_tok * rb);
    void* dkh = dev_alloc(info.n_hist_tok * rb);
    void* dvh = dev_alloc(info.n_hist_tok * rb);
    void* dkw = dev_alloc(info.n_q * rb);
    void* dvw = dev_alloc(info.n_q * rb);
    expect(mssa_pool_kv(plan, kh, vh, kw, vw, bw, bws, nullptr), MSSA_OK, "pool (backward workspace)");
    expect(mssa_backward(plan, q, ks, vs, kh, vh, kw, vw, out, static_cast<float*>(lse), dout, bw, bws, dq, dks, dvs,
                         dkh, dvh, dkw, dvw, nullptr),
           MSSA_OK, "backward");
    if (desc.scales[0] == 1) {
      const int cap = desc.hist_frames + desc.frames_per_state + 1;
      void* kr = dev_alloc(int64_t{cap} * tok1 * rb);
      void* vr = dev_alloc(int64_t{cap} * tok1 * rb);
      int32_t head = 0, count = desc.hist_frames;
      for (int pass = 0; pass < 4; ++pass)
        expect(mssa_hist_append(plan, kw, vw, kr, vr, cap, &head, &count, nullptr), MSSA_OK, "hist_append");
    }
  } else if (desc.flags & MSSA_PLAN_HEAD_IN_RING) {
    // rings of N slots (a multiple of F, cap >= history); every spare position
    const int F = desc.frames_per_state;
    const int N = (static_cast<int>(ceil_div(desc.hist_frames, F)) + 2) * F;
    std::vector<void*> kp(MSSA_MAX_STATES, nullptr), vp(MSSA_MAX_STATES, nullptr);
    for (int g = 0; g < info.n_groups; ++g) {
      const int s = info.group_scale[g];
      if (s == 1) continue;
      const int64_t tok_s = ceil_div(desc.grid_h, s) * ceil_div(desc.grid_w, s);
      kp[g] = dev_alloc(N * tok_s * rb);
      vp[g] = dev_alloc(N * tok_s * rb);
    }
    void* kr = dev_alloc(int64_t{N} * tok1 * rb);
    void* vr = dev_alloc(int64_t{N} * tok1 * rb);
    const int64_t rest = info.n_q - int64_t{F} * tok1;
    void* kw2 = dev_alloc(rest * rb);
    void* vw2 = dev_alloc(rest * rb);
    for (int spare = 0; spare < N; spare += F) {
      expect(mssa_pool_kv_head_ring(plan, kr, vr, kw2, vw2, kp.data(), vp.data(), ws, wsb, N, desc.hist_frames, spare,
                                    nullptr),
             MSSA_OK, "pool_kv_head_ring");
      expect(mssa_forward_head_ring(plan, q, ks, vs, kr, vr, const_cast<const void* const*>(kp.data()),
                                    const_cast<const void* const*>(vp.data()), kw2, vw2, ws, wsb, out, N,
                                    desc.hist_frames, spare, nullptr),
             MSSA_OK, "forward_head_ring");
      int32_t c = desc.hist_frames, sp = spare;
      expect(mssa_head_ring_roll(plan, N, &c, &sp), MSSA_OK, "head_ring_roll");
      if (sp != (spare + F) % N || c != std::min(desc.hist_frames + F, N - F)) failure("head_ring_roll arithmetic");
    }
    expect(mssa_forward_head_ring(plan, q, ks, vs, kr, vr, const_cast<const void* const*>(kp.data()),
                                  const_cast<const void* const*>(vp.data()), kw2, vw2, ws, wsb, out, N,
                                  desc.hist_frames, 1, nullptr),
           F == 1 ? MSSA_OK : MSSA_ERR_INVALID_ARG, "forward_head_ring at a misaligned spare slot");
  } else {
    std::vector<void*> kp(MSSA_MAX_STATES, nullptr), vp(MSSA_MAX_STATES, nullptr);
    const int cap = desc.hist_frames + desc.frames_per_state + 1;
    for (int g = 0; g < info.n_groups; ++g) {
      const int s = info.group_scale[g];
      if (s == 1) continue;
      const int64_t tok_s = ceil_div(desc.grid_h, s) * ceil_div(desc.grid_w, s);
      kp[g] = dev_alloc(cap * tok_s * rb);
      vp[g] = dev_alloc(cap * tok_s * rb);
    }
    void* kr = dev_alloc(int64_t{cap} * tok1 * rb);
    void* vr = dev_alloc(int64_t{cap} * tok1 * rb);
    expect(mssa_pool_hist_ring(plan, kr, vr, kp.data(), vp.data(), nullptr), MSSA_OK, "pool_hist_ring");
    expect(mssa_forward_ring(plan, q, ks, vs, desc.hist_frames ? kr : nullptr, desc.hist_frames ? vr : nullptr,
                             const_cast<const void* const*>(kp.data()), const_cast<const void* const*>(vp.data()), kw,
                             vw, ws, wsb, out, nullptr),
           MSSA_OK, "forward_ring");
    if (desc.scales[0] == 1) {
      int32_t head = 0, count = desc.hist_frames;
      for (int pass = 0; pass < 4; ++pass)
        expect(mssa_hist_append_ring(plan, kw, vw, ws, wsb, kr, vr, kp.data(), vp.data(), cap, &head, &count, nullptr),
               MSSA_OK, "hist_append_ring");
    }
  }
  if (desc.dtype == MSSA_BF16) {
    mssa_tier_desc tier{2, 2, desc.num_heads * desc.head_dim};
    int64_t tws = 0;
    expect(mssa_tier_workspace_size(plan, &tier, &tws), MSSA_OK, "tier workspace size");
    void* tw = dev_alloc(tws);
    const int64_t frames = int64_t{desc.num_states} * desc.frames_per_state;
    void* lat = dev_alloc(frames * tier.latent_channels * (desc.grid_h * 2) * (desc.grid_w * 2) * 2);
    void* tok = dev_alloc(info.n_q * tier.hidden * 2);
    std::vector<const void*> w(MSSA_MAX_STATES), b(MSSA_MAX_STATES);
    for (int g = 0; g < info.n_groups; ++g) {
      const int64_t kp = int64_t{tier.latent_channels} * (2 * info.group_scale[g]) * (2 * info.group_scale[g]);
      w[g] = dev_alloc(kp * tier.hidden * 2);
      b[g] = dev_alloc(std::max(kp, int64_t{tier.hidden}) * 2);
    }
    expect(mssa_patch_embed(plan, &tier, lat, w.data(), b.data(), tw, tws, tok, nullptr), MSSA_OK, "patch_embed");
    expect(mssa_patch_unembed(plan, &tier, tok, w.data(), b.data(), tw, tws, lat, nullptr), MSSA_OK, "patch_unembed");
    void* wq = dev_alloc(int64_t{3} * tier.hidden * tier.hidden * 2);
    void* bq = dev_alloc(int64_t{3} * tier.hidden * 2);
    void* o3[3] = {dev_alloc(info.n_q * tier.hidden * 2), dev_alloc(info.n_q * tier.hidden * 2),
                   dev_alloc(info.n_q * tier.hidden * 2)};
    expect(mssa_qkv_project(info.n_q, tier.hidden, tok, wq, bq, o3[0], o3[1], o3[2], nullptr), MSSA_OK, "qkv");
    expect(mssa_qkv_project_scaled(info.n_q, tier.hidden, tok, wq, bq, 0.1275f, o3[0], o3[1], o3[2], nullptr), MSSA_OK,
           "qkv scaled");
  }
  // rejected calls: nothing enqueued, the documented status
  expect(mssa_forward(plan, nullptr, ks, vs, kh, vh, kw, vw, ws, wsb, out, nullptr),
         ring ? MSSA_ERR_UNSUPPORTED : MSSA_ERR_INVALID_ARG, "forward without q");
  if (!ring && info.workspace_bytes > 0)
    expect(mssa_forward(plan, q, ks, vs, kh, vh, kw, vw, ws, info.workspace_bytes - 1, out, nullptr),
           MSSA_ERR_WORKSPACE, "forward with a small workspace");
  if (!ring)
    expect(mssa_forward(plan, q, ks, vs, kh, vh, kw, vw, ws, wsb, static_cast<char*>(out) + 2, nullptr),
           MSSA_ERR_INVALID_ARG, "forward with a misaligned output");
  mssa_plan_destroy(plan);
}

void invalid_descriptors() {
  g_case = "invalid descriptors";
  const int sc[8] = {1, 1, 2, 2, 2, 4, 4, 8};
  const mssa_plan_desc ok = make_desc(5, sc, 30, 52, 3, 3, 6, 12, 128, MSSA_BF16, 0);
  struct Case {
    const char* what;
    void (*edit)(mssa_plan_desc&);
    mssa_status want;
  };
  const Case cases[] = {
      {"num_states 0", [](mssa_plan_desc& d) { d.num_states = 0; }, MSSA_ERR_INVALID_ARG},
      {"num_states 9", [](mssa_plan_desc& d) { d.num_states = 9; }, MSSA_ERR_INVALID_ARG},
      {"grid 0", [](mssa_plan_desc& d) { d.grid_h = 0; }, MSSA_ERR_INVALID_ARG},
      {"grid huge", [](mssa_plan_desc& d) { d.grid_w = 1 << 20; }, MSSA_ERR_INVALID_ARG},
      {"frames 0", [](mssa_plan_desc& d) { d.frames_per_state = 0; }, MSSA_ERR_INVALID_ARG},
      {"sink < 0", [](mssa_plan_desc& d) { d.sink_frames = -1; }, MSSA_ERR_INVALID_ARG},
      {"hist < 0", [](mssa_plan_desc& d) { d.hist_frames = -1; }, MSSA_ERR_INVALID_ARG},
      {"heads 0", [](mssa_plan_desc& d) { d.num_heads = 0; }, MSSA_ERR_INVALID_ARG},
      {"dtype 7", [](mssa_plan_desc& d) { d.dtype = 7; }, MSSA_ERR_INVALID_ARG},
      {"scale inf", [](mssa_plan_desc& d) { d.softmax_scale = 1.0f / 0.0f; }, MSSA_ERR_INVALID_ARG},
      {"flags 16", [](mssa_plan_desc& d) { d.flags = 16; }, MSSA_ERR_INVALID_ARG},
      {"head in ring alone", [](mssa_plan_desc& d) { d.flags = MSSA_PLAN_HEAD_IN_RING; }, MSSA_ERR_UNSUPPORTED},
      {"scale 3", [](mssa_plan_desc& d) { d.scales[2] = 3; }, MSSA_ERR_UNSUPPORTED},
      {"scale 128", [](mssa_plan_desc& d) { d.scales[4] = 128; }, MSSA_ERR_UNSUPPORTED},
      {"decreasing", [](mssa_plan_desc& d) { d.scales[4] = 1; }, MSSA_ERR_UNSUPPORTED},
      {"head_dim 96", [](mssa_plan_desc& d) { d.head_dim = 96; }, MSSA_ERR_UNSUPPORTED},
      {"2^31 tokens", [](mssa_plan_desc& d) { d.grid_h = 65536; d.grid_w = 65536; d.hist_frames = 1; },
       MSSA_ERR_UNSUPPORTED},
  };
  for (const Case& c : cases) {
    mssa_plan_desc d = ok;
    c.edit(d);
    mssa_plan plan = nullptr;
    expect(mssa_plan_create(&d, &plan), c.want, c.what);
    if (plan) {
      failure("an invalid descriptor produced a plan");
      mssa_plan_destroy(plan);
    }
  }
  mssa_plan plan = nullptr;
  expect(mssa_plan_create(nullptr, &plan), MSSA_ERR_INVALID_ARG, "null desc");
  expect(mssa_plan_create(&ok, nullptr), MSSA_ERR_INVALID_ARG, "null out");
  expect(mssa_plan_create_ex(&ok, -1, &plan), MSSA_ERR_INVALID_ARG, "negative attention_blocks");
  expect(mssa_plan_query(nullptr, nullptr), MSSA_ERR_INVALID_ARG, "query without a plan");
  expect(mssa_pool_kv(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr), MSSA_ERR_INVALID_ARG,
         "pool without a plan");
  expect(mssa_attention_noalloc(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                nullptr),
         MSSA_ERR_INVALID_ARG, "noalloc without a plan");
  mssa_plan_destroy(nullptr);
  ++g_checks;
}

}  // namespace

int main(int argc, char** argv) {
  g_plant = argc > 1 && std::strcmp(argv[1], "plant") == 0;
  invalid_descriptors();
  // the layer workloads and the streaming history lengths
  const int s12[5] = {1, 1, 2, 2, 2}, s124[5] = {1, 1, 2, 2, 4}, t12[2] = {1, 2};
  std::vector<std::pair<std::string, mssa_plan_desc>> named = {
      {"tiny fp32", make_desc(2, t12, 8, 8, 1, 1, 0, 1, 64, MSSA_F32, 0)},
      {"1.3B layer", make_desc(5, s12, 30, 52, 3, 3, 6, 12, 128, MSSA_BF16, 0)},
      {"21-frame history", make_desc(5, s124, 30, 52, 3, 3, 21, 12, 128, MSSA_BF16, 0)},
      {"720p layer", make_desc(5, s124, 45, 80, 3, 3, 9, 40, 128, MSSA_BF16, 0)},
  };
  for (int h = 6; h <= 21; h += 3)
    named.push_back({"streaming history " + std::to_string(h), make_desc(5, s12, 30, 52, 3, 3, h, 12, 128, MSSA_BF16,
                                                                       MSSA_PLAN_POOLED_HIST_RING)});
  for (int h = 6; h <= 21; h += 3)
    named.push_back({"streaming head in ring " + std::to_string(h),
                     make_desc(5, s12, 30, 52, 3, 3, h, 12, 128, MSSA_BF16,
                               MSSA_PLAN_POOLED_HIST_RING | MSSA_PLAN_HEAD_IN_RING)});
  for (const auto& c : named) {
    g_case = c.first;
    exercise(c.second, 0);
  }
  g_case = "1.3B layer, 7 attention blocks";
  exercise(named[1].second, 7);
  g_case = "1.3B layer, 1000 attention blocks";
  exercise(named[1].second, 1000);
  // 150 seeded random descriptors (the ranges of the table fuzz test)
  const int pick[5] = {1, 2, 4, 8, 16};
  for (int i = 0; i < 150; ++i) {
    int T = 1 + static_cast<int>(rnd(8)), sc[8];
    for (int l = 0; l < T; ++l) sc[l] = pick[rnd(5)];
    std::sort(sc, sc + T);
    int flags = static_cast<int>(rnd(4));
    const bool bf = rnd(4) != 0;
    if ((flags & MSSA_PLAN_POOLED_HIST_RING) && sc[0] == 1 && bf && rnd(2)) flags |= MSSA_PLAN_HEAD_IN_RING;
    if (rnd(2)) flags |= MSSA_PLAN_Q_PRESCALED;
    const mssa_plan_desc d = make_desc(T, sc, 1 + static_cast<int>(rnd(70)), 1 + static_cast<int>(rnd(90)),
                                       1 + static_cast<int>(rnd(4)), static_cast<int>(rnd(5)),
                                       static_cast<int>(rnd(26)), 1 + static_cast<int>(rnd(48)),
                                       rnd(2) ? 128 : 64, bf ? MSSA_BF16 : MSSA_F32, flags);
    g_case = "random descriptor " + std::to_string(i) + " T=" + std::to_string(T) + " sc0=" + std::to_string(sc[0]) +
             " last=" + std::to_string(sc[T - 1]) + " H=" + std::to_string(d.grid_h) + " W=" + std::to_string(d.grid_w) +
             " F=" + std::to_string(d.frames_per_state) + " S=" + std::to_string(d.sink_frames) +
             " Hh=" + std::to_string(d.hist_frames) + " nh=" + std::to_string(d.num_heads) +
             " d=" + std::to_string(d.head_dim) + " dt=" + std::to_string(d.dtype) + " fl=" + std::to_string(flags);
    exercise(d, rnd(3) == 0 ? 1 + static_cast<int>(rnd(600)) : 0);
  }
  std::printf("%d checks, %d failures\n", g_checks, g_failures);
  return g_failures == 0 ? 0 : 1;
}
