// Static MSSA plan: MSP grids, query groups, Eq. 4 context tables, pool jobs
// and the kernel launch descriptions.  Host-only C++17; no HIP types, so the
// scheduler builds and runs without a GPU.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/libmssa.h"

namespace mssa {

enum Kind : int32_t { kSink = 0, kHist = 1, kWin = 2 };

// Where a run of context tokens lives.
// kBufHistPooled: the caller's pooled-history ring of the group (plans with
// MSSA_PLAN_POOLED_HIST_RING), frame f at token f * tok_s.
// kBufRingHead: a frame of window state 1 that lives in the ring's spare
// slots (plans with MSSA_PLAN_HEAD_IN_RING): the native ring for the native
// query scale, the group's pooled ring for a coarser one; frame f of the
// state in the f-th spare slot.
enum Buffer : int32_t {
  kBufSink = 0, kBufHist = 1, kBufWin = 2, kBufPooled = 3, kBufHistPooled = 4, kBufRingHead = 5
};

struct GridRow {
  int32_t scale, gh, gw, tok;
};

struct QGroup {
  int32_t scale, q_begin, q_end;
  int64_t n_kv;
};

struct SegRow {
  int32_t q_scale, kind, frame, src_scale, eff_scale, factor, n_tok;
  int64_t kv_begin;
  // placement used by the kernels (not exported)
  int32_t buffer;
  int64_t tok_offset;  // first token inside `buffer` (pooled: inside the group block)
};

// A maximal stretch of context tokens that is contiguous in one buffer.
struct Run {
  int32_t buffer;
  int64_t tok_offset;
  int64_t n_tok;
};

// One average-pool job: n_frames consecutive frames of grid (src_gh, src_gw)
// starting at src_tok of `buffer` (history or window) -> factor x factor
// pooled frames of grid (dst_gh, dst_gw) at dst_tok of group `group`'s
// pooled block.
struct PoolJob {
  int32_t group;
  int32_t buffer;
  int64_t src_tok;
  int32_t src_gh, src_gw;
  int32_t factor;
  int32_t n_frames;
  int32_t dst_gh, dst_gw;
  int64_t dst_tok;
};

// Source frames whose gradients gather from the context gradients of every
// query scale (the adjoint of building the contexts): sink frames, history
// frames, or consecutive window frames of one scale.
struct ScatterJob {
  int32_t buffer;                 // kBufSink, kBufHist or kBufWin
  int64_t src_tok;                // first token in that buffer
  int32_t n_frames, gh, gw;
  std::vector<int64_t> ctx_begin; // per group: context token of the job's first frame
  std::vector<int32_t> frame_stride, factor;  // per group
};

// Persistent attention schedule (bf16 forward): groups in launch order
// (longest context first), 64-key tiles per item of each group, first tile
// of each group in the linear tile space, whole-item rounds and the first
// tile of the tail ranges, for a fixed number of tile ranges (blocks).
struct Schedule {
  std::vector<int32_t> tiles_per_item;   // per group
  std::vector<int64_t> tile_begin;       // per group
  int64_t total_tiles = 0;
  int32_t dp_rounds = 0;    // rounds of whole items (one per block) before the tail
  int64_t tail_begin = 0;   // first tile of the tail ranges
};

struct Plan {
  mssa_plan_desc desc;
  bool hist_ring;  // MSSA_PLAN_POOLED_HIST_RING
  bool head_ring;  // MSSA_PLAN_HEAD_IN_RING: window state 1 read from the rings' spare slots
  int64_t win_shift;  // head_ring: window tokens before k_win / v_win (state 1's), else 0
  bool strided;    // MSSA_PLAN_STRIDED_SUBSAMPLE: first cell of each block
  bool q_prescaled;  // MSSA_PLAN_Q_PRESCALED: queries arrive multiplied by softmax_scale * log2(e)
  float softmax_scale;
  int64_t tok1;  // native tokens per frame
  int64_t n_q, n_sink_tok, n_hist_tok;
  int64_t ld;          // elements between consecutive tokens: heads * head_dim
  int64_t elem_bytes;  // 2 (bf16) or 4 (fp32)
  std::vector<GridRow> grids;
  std::vector<QGroup> groups;
  std::vector<SegRow> segs;             // all groups, context order
  std::vector<std::vector<Run>> runs;   // per group
  std::vector<PoolJob> pool_jobs;
  std::vector<int64_t> pooled_tokens;   // per group
  std::vector<int64_t> pooled_k_off, pooled_v_off;  // bytes, per group
  int64_t workspace_bytes;
  int64_t pairs_per_head;
  int64_t pool_bytes_alg;
  // Persistent attention schedule over the runs above (bf16): groups in
  // launch order and n_ranges tile ranges (one per block).
  std::vector<int> order;
  int32_t n_ranges;
  Schedule sched;
  int64_t partial_off, partial_bytes;    // partial records and the range table in the workspace
  int64_t range_table_off;               // n_ranges + 1 int64 first tiles of the tail ranges
  // Backward workspace: the forward's, then -rowsum(dO * O) [heads, n_q]
  // fp32, -lse / scale [heads, n_q] fp32, then per group the fp32 context
  // gradients of K and V, then (bf16) per group the dS tiles.
  int64_t bwd_dsum_off, bwd_lse2_off;
  std::vector<int64_t> bwd_dk_off, bwd_dv_off;  // bytes, per group
  // bf16 plans: per group dS = P * (dP - rowsum) in bf16, written by the
  // dK/dV kernel and read by the dQ kernel, in 4 KB tiles [head of the
  // chunk][32-query block][64-key stage of the context's runs][64 key
  // slots][32 queries], for bwd_ds_heads heads at a time.
  int32_t bwd_ds_heads = 0;             // heads per backward chunk
  std::vector<int64_t> bwd_ds_off;      // bytes, per group
  std::vector<int32_t> bwd_ds_stages;   // 64-key stages of the group's runs
  std::vector<int32_t> bwd_ds_qblocks;  // 32-query blocks, rounded up to an even count
  int64_t bwd_workspace_bytes;
  std::vector<ScatterJob> scatter_jobs;
};

// Validates `d` and fills `p`.  `slots` is the number of attention blocks
// the device keeps resident at once (<= 0: 512, two per CU of an MI355X);
// `attention_blocks` > 0 sets the number of persistent attention blocks
// (tile ranges) instead.  Returns MSSA_OK or an error status with a message
// in `err`.
mssa_status build_plan(const mssa_plan_desc& d, int slots, int attention_blocks, Plan& p, std::string& err);

// The attention schedule of plan p over per-group runs whose token counts
// are n_tok[g] (the plan's own runs, or runs placed at call time).
Schedule make_schedule(const Plan& p, const std::vector<std::vector<int64_t>>& n_tok);

// Flat int64 export of GRID / QGRP / SEG / TOTAL (layout in libmssa.h).
std::vector<int64_t> export_tables(const Plan& p);

}  // namespace mssa
