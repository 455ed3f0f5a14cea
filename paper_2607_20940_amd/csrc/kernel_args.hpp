// Kernel-argument structs passed by value (kernarg segment) to the MSSA
// kernels.  Plain data; shared by the host launch code and the kernels.
#pragma once

#include <cstdint>

namespace mssa {

constexpr int kMaxGroups = 8;      // distinct query scales (<= num_states)
constexpr int kMaxRuns = 4;        // contiguous context runs per query scale
constexpr int kMaxPoolJobs = 16;   // pool jobs per launch

// Tile shapes of the bf16 attention kernel: 8 waves x 32 queries (two
// groups of four waves that alternate matrix-core and softmax phases), 64 keys.
constexpr int kFwdBM = 256;
constexpr int kFwdBN = 64;
constexpr int kFwdThreads = 512;
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
  FwdGroupArgs groups[kMaxGroups];  // in launch order (longest context first)
};

// One partial record: unnormalised O [BM][D] (fp32), running max m [BM] and
// row sum l [BM] of one piece of an item that spans several tile ranges.
constexpr int64_t partial_record_floats(int head_dim) { return static_cast<int64_t>(kFwdBM) * (head_dim + 2); }

struct PoolJobArgs {
  const void* src_k;        // first source token of the job (head 0, ch 0)
  const void* src_v;
  void* dst_k;              // first destination token of the job
  void* dst_v;
  int32_t src_gh, src_gw;
  int32_t dst_gh, dst_gw;
  int32_t factor;
  int32_t n_frames;
  int32_t block_begin;
  int32_t pad;
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
