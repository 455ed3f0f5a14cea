// Kernel-argument structs passed by value (kernarg segment) to the MSSA
// kernels.  Plain data; shared by the host launch code and the kernels.
#pragma once

#include <cstdint>

namespace mssa {

constexpr int kMaxGroups = 8;      // distinct query scales (<= num_states)
constexpr int kMaxRuns = 6;        // contiguous context runs per query scale
constexpr int kMaxPoolJobs = 16;   // pool jobs per launch

// Tile shapes of the bf16 attention kernel: 8 waves x 32 queries (two
// groups of four waves that alternate matrix-core and softmax phases), 64 keys.
constexpr int kFwdBM = 256;
constexpr int kFwdBN = 64;
constexpr int kFwdThreads = 512;
// Merge of split items: threads per block (one output float4 each).
constexpr int kCombineThreads = 256;
// fp32 attention kernel: one query per lane, one wave per block.
constexpr int kFwdF32BM = 64;

constexpr int kPoolThreads = 256;

struct FwdRunArgs {
  const void* k;   // first token of the run (head 0, channel 0)
  const void* v;
  int32_t n_tok;
  int32_t pad;
};

struct FwdGroupArgs {
  int32_t q_begin, q_end;   // query token range of this scale
  int32_t n_qtiles;         // ceil((q_end - q_begin) / BM)
  int32_t block_begin;      // first item (fp32 kernel: first block) of this group
  int32_t n_runs;
  int32_t tiles_per_item;   // bf16 kernel: sum over runs of ceil(n_tok / BN)
  int64_t tile_begin;       // bf16 kernel: first tile of this group in the linear tile space
  FwdRunArgs runs[kMaxRuns];
};

struct FwdArgs {
  const void* q;
  void* out;
  int64_t ld;               // elements between tokens: heads * head_dim
  int32_t n_groups;
  int32_t num_heads;
  int32_t n_blocks;
  float scale_log2e;        // softmax scale * log2(e)
  float scale;              // softmax scale
  int32_t n_ranges;         // bf16 kernel: persistent blocks
  int64_t total_tiles;      // bf16 kernel: tiles of all (group, head, query tile) items
  int64_t tail_begin;       // bf16 kernel: first tile after the whole-item rounds
  int32_t dp_rounds;        // bf16 kernel: rounds of whole items before the tail ranges
  int32_t pad2;
  float* partial;           // bf16 kernel: 2 * n_ranges partial records
  int64_t* range_table;     // bf16 kernel: first tile of each tail range (n_ranges + 1), written by the attention kernel
  float* lse;               // optional [heads, n_q]: log of the softmax denominator (natural log)
  int32_t n_q;
  int32_t q_prescaled;      // bf16 kernel: queries arrive multiplied by scale * log2(e)
  FwdGroupArgs groups[kMaxGroups];  // in launch order (longest context first)
};

// One partial record: unnormalised O [BM][D] (fp32), running max m [BM] and
// row sum l [BM] of one piece of an item that spans several tile ranges.
constexpr int64_t partial_record_floats(int head_dim) { return static_cast<int64_t>(kFwdBM) * (head_dim + 2); }

// ---------------------------------------------------------------- backward

// bf16 backward kernels: 8 waves, 32 queries (dQ kernel) or 32 keys (dK/dV
// kernel) per wave or wave pair; the other operands stream through LDS in
// stages.
constexpr int kBwdQ = 256;     // dQ kernel: queries per block (8 waves x 32)
constexpr int kBwdQThreads = 512;   // dQ kernel: 8 waves, two per SIMD
constexpr int kBwdKS = 64;     // dQ kernel: keys per LDS stage (and per dS tile)
constexpr int kBwdK = 128;     // dK/dV kernel: keys per block (4 wave pairs x 32)
constexpr int kBwdKVThreads = 512;  // dK/dV kernel: 8 waves, two per SIMD
constexpr int kBwdQS = 64;     // dK/dV kernel: queries per LDS stage
constexpr int64_t kBwdDsBudget = int64_t(8) << 30;  // bytes of dS tiles held at once (whole heads, at least one)
constexpr int kBwdF32 = 64;    // fp32 kernels: one query or key per lane
constexpr int kDotThreads = 256;
constexpr int kMaxScatterJobs = 10;

struct BwdGroupArgs {
  int32_t q_begin, q_end;     // query token range of this scale
  int32_t n_kv;               // context tokens
  int32_t n_runs;
  int32_t dq_block_begin;     // first block of the group in the dQ grid (head-major inside)
  int32_t kv_block_begin;     // first block of the group in the dK/dV grid
  int32_t n_qblocks;          // dQ blocks per head
  int32_t n_kblocks;          // dK/dV blocks per head
  FwdRunArgs runs[kMaxRuns];  // context runs (K, V source tokens), context order
  float* dk_ctx;              // [n_kv, heads * head_dim] fp32 context gradients
  float* dv_ctx;
  void* ds;                   // bf16: dS tiles [launch heads][ds_qblocks][ds_stages][64 keys][32 queries]
  int32_t ds_stages;          // 64-key stages of the runs (each run starts a stage)
  int32_t ds_qblocks;         // 32-query blocks (even)
};

struct BwdArgs {
  const void* q;
  const void* d_out;
  const float* lse;         // [heads, n_q] from the forward
  float* dsum;              // [heads, n_q]: -rowsum(d_out * out), written by dot_kernel
  float* lse2;              // [heads, n_q]: -lse / scale, in units of q k^T (bf16), written by dot_kernel
  void* dq;
  int64_t ld;               // elements between tokens: heads * head_dim
  int32_t n_q;
  int32_t num_heads;        // heads of this launch: head0 .. head0 + num_heads - 1
  int32_t head0;            // first head of this launch (the dS tiles hold these heads)
  int32_t n_groups;
  float scale;              // softmax scale
  float scale_log2e;
  int32_t q_prescaled;      // queries arrive multiplied by scale * log2(e)
  BwdGroupArgs groups[kMaxGroups];  // longest query range first
};
static_assert(sizeof(BwdArgs) <= 4096, "kernel argument block");

struct DotArgs {
  const void* out;
  const void* d_out;
  float* dsum;              // [heads, n_q]: -rowsum(d_out * out)
  const float* lse;         // [heads, n_q] natural log (bf16 plans; may be null)
  float* lse2;              // [heads, n_q] -lse / scale: minus the row max of q k^T (written when lse is set)
  int64_t ld;
  int32_t n_q;
  int32_t num_heads;
  int32_t head_dim;
  float inv_scale;          // 1 / the natural-log score factor
};

// One run of source frames (sink, history, or window frames of one scale)
// whose gradient gathers from every query scale's context gradient: frame f
// of the job sits in group g's context at token ctx_begin + f * frame_stride,
// resampled by factor.
struct ScatterGroupArgs {
  int64_t ctx_begin;
  int32_t frame_stride;
  int32_t factor;
};

struct ScatterJobArgs {
  void* dst_k;              // gradient of the job's first source token (head 0, channel 0)
  void* dst_v;
  int32_t n_frames;
  int32_t gh, gw;           // source grid
  int32_t block_begin;
  ScatterGroupArgs g[kMaxGroups];
};

struct ScatterArgs {
  const float* ctx_k[kMaxGroups];
  const float* ctx_v[kMaxGroups];
  int64_t ld;
  int32_t chunks_per_tok;   // output chunks per token: 8 elements (bf16) or 4 (fp32)
  int32_t n_jobs;
  int32_t n_groups;
  int32_t pick_first;       // strided resampling: only each block's first cell
  ScatterJobArgs jobs[kMaxScatterJobs];
};

// ---------------------------------------------------------------- MSP tiers

constexpr int kTierThreads = 256;
// Output tile (rows x features) and K stage of the 4-wave GEMM kernels.
constexpr int kGemmTile = 128, kGemmStage = 64;

// Patch rows of consecutive latent frames of one tier: frame frame0 + f of
// `latent` [frames, C, H, W] <-> rows [(f * gh + Y) * gw + X][C * P * P].
struct PatchArgs {
  void* latent;
  void* rows;
  int64_t frame0;
  int64_t n_frames;
  int32_t C, H, W, P;
  int32_t gh, gw;
};

// Y = X W^T + b: X [M, K] (row stride ldx), W [N, K] dense, b [N]; output
// feature j goes to y[j / split] at column j % split (row stride ldy).
struct GemmArgs {
  const void* x;
  const void* w;
  const void* bias;
  void* y[3];
  int32_t M, N, K;
  int32_t split;
  int64_t ldx, ldy;
  float* partial;     // k_splits > 1: fp32 partial tiles of every K slice (launch_gemm_split)
  int32_t k_splits;   // 0 or 1: the whole K in one block
  float y0_scale;     // factor on the outputs of y[0] (columns < split), applied to the fp32 sum before rounding
};

struct PoolJobArgs {
  const void* src_k;        // first source token of the job (head 0, ch 0)
  const void* src_v;
  void* dst_k;              // first destination token of the job (pooled by factor)
  void* dst_v;
  void* dst2_k;             // levels == 2: first destination token pooled by 2 * factor
  void* dst2_v;
  int32_t src_gh, src_gw;
  int32_t dst_gh, dst_gw;
  int32_t dst2_gh, dst2_gw;
  int32_t factor;
  int32_t levels;           // 1, or 2: the same source frames pooled by factor and by 2 * factor
  int32_t n_frames;
  int32_t block_begin;
};

struct PoolArgs {
  int64_t ld;               // elements between tokens
  int32_t chunks_per_tok;   // 16-byte chunks per token (all heads)
  int32_t n_jobs;
  int32_t pick_first;       // 1: copy each block's first cell (stride); 0: block mean
  int32_t pad;
  PoolJobArgs jobs[kMaxPoolJobs];
};

}  // namespace mssa
