// Static MSSA plan (host).  Every table follows Sec. 4.1 of Ms. Forcing:
// MSP grids from Eq. 3 (ceil grid when a scale does not divide the native
// grid), query groups per distinct scale, and the Eq. 4 context of each
// query scale s:
//   sink frames        native, never resampled;
//   history frames     native, pooled by s;
//   window frame of b  at max(s, p_b), pooled by max(1, s / p_b);
// in the order sink, history (oldest first), window (state 1..T).
#include "plan.hpp"

#include "kernel_args.hpp"

#include <algorithm>
#include <cmath>
#include <limits>

namespace mssa {
namespace {

bool is_pow2(int32_t x) { return x > 0 && (x & (x - 1)) == 0; }

int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

}  // namespace

mssa_status build_plan(const mssa_plan_desc& d, int slots, int attention_blocks, Plan& p, std::string& err) {
  const int32_t T = d.num_states;
  if (T < 1 || T > MSSA_MAX_STATES) {
    err = "num_states must be in [1, " + std::to_string(MSSA_MAX_STATES) + "]";
    return MSSA_ERR_INVALID_ARG;
  }
  if (d.grid_h < 1 || d.grid_w < 1 || d.grid_h > 65536 || d.grid_w > 65536) {
    err = "grid_h and grid_w must be in [1, 65536]";
    return MSSA_ERR_INVALID_ARG;
  }
  if (d.frames_per_state < 1 || d.sink_frames < 0 || d.hist_frames < 0) {
    err = "frames_per_state must be >= 1, sink_frames and hist_frames >= 0";
    return MSSA_ERR_INVALID_ARG;
  }
  if (d.num_heads < 1) {
    err = "num_heads must be >= 1";
    return MSSA_ERR_INVALID_ARG;
  }
  if (d.dtype != MSSA_BF16 && d.dtype != MSSA_F32) {
    err = "dtype must be MSSA_BF16 or MSSA_F32";
    return MSSA_ERR_INVALID_ARG;
  }
  if (!std::isfinite(d.softmax_scale)) {
    err = "softmax_scale must be finite";
    return MSSA_ERR_INVALID_ARG;
  }
  if ((d.flags & ~(MSSA_PLAN_POOLED_HIST_RING | MSSA_PLAN_STRIDED_SUBSAMPLE | MSSA_PLAN_HEAD_IN_RING |
                   MSSA_PLAN_Q_PRESCALED)) != 0) {
    err = "unknown plan flags";
    return MSSA_ERR_INVALID_ARG;
  }
  for (int l = 0; l < T; ++l) {
    if (!is_pow2(d.scales[l]) || d.scales[l] > 64) {
      err = "scales must be powers of two in [1, 64]";
      return MSSA_ERR_UNSUPPORTED;
    }
    if (l > 0 && d.scales[l] < d.scales[l - 1]) {
      err = "scales must be nondecreasing (coarser patches for noisier states)";
      return MSSA_ERR_UNSUPPORTED;
    }
  }
  if (d.head_dim != 64 && d.head_dim != 128) {
    err = "head_dim must be 64 or 128";
    return MSSA_ERR_UNSUPPORTED;
  }
  if ((d.flags & MSSA_PLAN_HEAD_IN_RING) &&
      (!(d.flags & MSSA_PLAN_POOLED_HIST_RING) || d.scales[0] != 1 || d.dtype != MSSA_BF16)) {
    err = "MSSA_PLAN_HEAD_IN_RING needs MSSA_PLAN_POOLED_HIST_RING, a native head state (scales[0] == 1) and bf16";
    return MSSA_ERR_UNSUPPORTED;
  }

  p = Plan{};
  p.desc = d;
  p.hist_ring = (d.flags & MSSA_PLAN_POOLED_HIST_RING) != 0;
  p.head_ring = (d.flags & MSSA_PLAN_HEAD_IN_RING) != 0;
  p.strided = (d.flags & MSSA_PLAN_STRIDED_SUBSAMPLE) != 0;
  p.q_prescaled = (d.flags & MSSA_PLAN_Q_PRESCALED) != 0;
  p.softmax_scale = d.softmax_scale > 0.f ? d.softmax_scale
                                          : 1.0f / std::sqrt(static_cast<float>(d.head_dim));
  const int32_t F = d.frames_per_state;
  auto tok_at = [&](int32_t s) {
    return static_cast<int64_t>(ceil_div(d.grid_h, s)) * ceil_div(d.grid_w, s);
  };
  p.tok1 = tok_at(1);
  p.ld = static_cast<int64_t>(d.num_heads) * d.head_dim;
  p.elem_bytes = d.dtype == MSSA_BF16 ? 2 : 4;
  p.n_sink_tok = p.tok1 * d.sink_frames;
  p.n_hist_tok = p.tok1 * d.hist_frames;
  p.win_shift = p.head_ring ? p.tok1 * F : 0;

  // GRID: native scale plus every scheduled scale, ascending.
  std::vector<int32_t> sc{1};
  for (int l = 0; l < T; ++l) sc.push_back(d.scales[l]);
  std::sort(sc.begin(), sc.end());
  sc.erase(std::unique(sc.begin(), sc.end()), sc.end());
  for (int32_t s : sc)
    p.grids.push_back({s, ceil_div(d.grid_h, s), ceil_div(d.grid_w, s), static_cast<int32_t>(tok_at(s))});

  // Window frames in token order and the query groups (contiguous per scale
  // because the schedule is nondecreasing).
  struct WinFrame { int32_t w, p; int64_t first, n; };
  std::vector<WinFrame> wf;
  int64_t pos = 0;
  for (int l = 0; l < T; ++l)
    for (int f = 0; f < F; ++f) {
      const int64_t n = tok_at(d.scales[l]);
      wf.push_back({l * F + f, d.scales[l], pos, n});
      pos += n;
    }
  p.n_q = pos;
  for (const WinFrame& w : wf) {
    if (!p.groups.empty() && p.groups.back().scale == w.p)
      p.groups.back().q_end = static_cast<int32_t>(w.first + w.n);
    else
      p.groups.push_back({w.p, static_cast<int32_t>(w.first), static_cast<int32_t>(w.first + w.n), 0});
  }

  const int64_t kIdxMax = std::numeric_limits<int32_t>::max();
  if (p.n_q > kIdxMax || p.n_sink_tok > kIdxMax || p.n_hist_tok > kIdxMax) {
    err = "token counts exceed 32-bit indexing";
    return MSSA_ERR_UNSUPPORTED;
  }

  // SEG rows per group, their placement, runs and pool jobs.
  const int G = static_cast<int>(p.groups.size());
  p.runs.assign(G, {});
  p.pooled_tokens.assign(G, 0);
  p.pooled_k_off.assign(G, 0);
  p.pooled_v_off.assign(G, 0);
  p.pairs_per_head = 0;
  int64_t ws = 0;
  auto align256 = [](int64_t x) { return (x + 255) / 256 * 256; };
  std::vector<char> win_read(wf.size(), 0);
  bool hist_read = false;

  for (int g = 0; g < G; ++g) {
    QGroup& grp = p.groups[g];
    const int32_t s = grp.scale;
    int64_t kv = 0, pooled = 0;
    std::vector<SegRow> rows;
    for (int f = 0; f < d.sink_frames; ++f)
      rows.push_back({s, kSink, f, 1, 1, 1, static_cast<int32_t>(p.tok1), 0, kBufSink, f * p.tok1});
    for (int f = 0; f < d.hist_frames; ++f) {
      SegRow r{s, kHist, f, 1, s, s, static_cast<int32_t>(tok_at(s)), 0, kBufHist, f * p.tok1};
      if (s > 1 && p.hist_ring) {
        r.buffer = kBufHistPooled;
        r.tok_offset = f * r.n_tok;
      } else if (s > 1) {
        r.buffer = kBufPooled;
        r.tok_offset = pooled;
        pooled += r.n_tok;
        hist_read = true;
      }
      rows.push_back(r);
    }
    for (size_t i = 0; i < wf.size(); ++i) {
      const WinFrame& w = wf[i];
      const int32_t eff = std::max(s, w.p);
      const int32_t fac = std::max(1, s / w.p);
      SegRow r{s, kWin, w.w, w.p, eff, fac, static_cast<int32_t>(tok_at(eff)), 0, kBufWin, w.first - p.win_shift};
      if (p.head_ring && w.w < F) {
        // state 1 lives in the spare ring slots, pooled there by pool_kv
        r.buffer = kBufRingHead;
        r.tok_offset = w.w * r.n_tok;
      } else if (fac > 1) {
        r.buffer = kBufPooled;
        r.tok_offset = pooled;
        pooled += r.n_tok;
        win_read[i] = 1;
      }
      rows.push_back(r);
    }
    for (SegRow& r : rows) { r.kv_begin = kv; kv += r.n_tok; }
    if (kv > kIdxMax) {
      err = "context length exceeds 32-bit indexing";
      return MSSA_ERR_UNSUPPORTED;
    }
    grp.n_kv = kv;
    p.pairs_per_head += static_cast<int64_t>(grp.q_end - grp.q_begin) * kv;

    // Runs: merge rows that are contiguous in one buffer.
    for (const SegRow& r : rows) {
      std::vector<Run>& rs = p.runs[g];
      if (!rs.empty() && rs.back().buffer == r.buffer &&
          rs.back().tok_offset + rs.back().n_tok == r.tok_offset)
        rs.back().n_tok += r.n_tok;
      else
        rs.push_back({r.buffer, r.tok_offset, r.n_tok});
    }

    // Pool jobs: merge consecutive pooled rows of one source kind, source
    // scale and factor whose source and destination frames are contiguous.
    for (const SegRow& r : rows) {
      if (r.buffer != kBufPooled) continue;
      const int32_t src_buf = r.kind == kHist ? kBufHist : kBufWin;
      int64_t src_tok;
      int64_t src_n;
      if (r.kind == kHist) {
        src_tok = r.frame * p.tok1;
        src_n = p.tok1;
      } else {
        src_tok = wf[r.frame].first - p.win_shift;
        src_n = wf[r.frame].n;
      }
      const int32_t sgh = ceil_div(d.grid_h, r.src_scale), sgw = ceil_div(d.grid_w, r.src_scale);
      if (!p.pool_jobs.empty()) {
        PoolJob& j = p.pool_jobs.back();
        const int64_t jsrc_n = static_cast<int64_t>(j.src_gh) * j.src_gw;
        const int64_t jdst_n = static_cast<int64_t>(j.dst_gh) * j.dst_gw;
        if (j.group == g && j.buffer == src_buf && j.factor == r.factor && j.src_gh == sgh &&
            j.src_gw == sgw && j.src_tok + j.n_frames * jsrc_n == src_tok &&
            j.dst_tok + j.n_frames * jdst_n == r.tok_offset) {
          j.n_frames += 1;
          continue;
        }
      }
      (void)src_n;
      p.pool_jobs.push_back({g, src_buf, src_tok, sgh, sgw, r.factor, 1,
                             ceil_div(sgh, r.factor), ceil_div(sgw, r.factor), r.tok_offset});
    }

    p.pooled_tokens[g] = pooled;
    if (pooled > 0) {
      const int64_t bytes = align256(pooled * p.ld * p.elem_bytes);
      p.pooled_k_off[g] = ws;
      ws += bytes;
      p.pooled_v_off[g] = ws;
      ws += bytes;
    }
    for (SegRow& r : rows) p.segs.push_back(r);
  }
  // Persistent attention schedule: items (group, head, query tile) in launch
  // order, each a sequence of 64-key tiles over the group's runs.
  for (int g = 0; g < G; ++g) p.order.push_back(g);
  std::stable_sort(p.order.begin(), p.order.end(),
                   [&](int x, int y) { return p.groups[x].n_kv > p.groups[y].n_kv; });
  std::vector<std::vector<int64_t>> run_tok(G);
  int64_t n_items = 0;
  for (int g = 0; g < G; ++g) {
    for (const Run& r : p.runs[g]) run_tok[g].push_back(r.n_tok);
    n_items += static_cast<int64_t>((p.groups[g].q_end - p.groups[g].q_begin + kFwdBM - 1) / kFwdBM) * d.num_heads;
  }
  p.n_ranges = 1;
  const int64_t total = make_schedule(p, run_tok).total_tiles;
  if (slots <= 0) slots = 512;
  int64_t ranges = attention_blocks > 0 ? attention_blocks : std::min<int64_t>(slots, n_items);
  ranges = std::max<int64_t>(1, std::min<int64_t>(ranges, total));
  p.n_ranges = static_cast<int32_t>(ranges);
  p.sched = make_schedule(p, run_tok);
  p.partial_off = 0;
  p.partial_bytes = 0;
  p.range_table_off = 0;
  if (d.dtype == MSSA_BF16 && p.n_ranges > 1) {
    const int64_t rec_bytes = align256(2 * static_cast<int64_t>(p.n_ranges) * partial_record_floats(d.head_dim) * 4);
    p.partial_off = ws;
    p.range_table_off = ws + rec_bytes;
    p.partial_bytes = rec_bytes + align256((static_cast<int64_t>(p.n_ranges) + 1) * 8);
    ws += p.partial_bytes;
  }
  p.workspace_bytes = ws;

  // Backward workspace and the scatter of context gradients to the sources.
  ws = align256(ws);
  p.bwd_dsum_off = ws;
  ws += align256(static_cast<int64_t>(d.num_heads) * p.n_q * 4);
  p.bwd_lse2_off = ws;
  ws += align256(static_cast<int64_t>(d.num_heads) * p.n_q * 4);
  p.bwd_dk_off.assign(G, 0);
  p.bwd_dv_off.assign(G, 0);
  for (int g = 0; g < G; ++g) {
    const int64_t bytes = align256(p.groups[g].n_kv * p.ld * 4);
    p.bwd_dk_off[g] = ws;
    ws += bytes;
    p.bwd_dv_off[g] = ws;
    ws += bytes;
  }
  p.bwd_ds_off.assign(G, 0);
  p.bwd_ds_stages.assign(G, 0);
  p.bwd_ds_qblocks.assign(G, 0);
  p.bwd_ds_heads = d.num_heads;
  if (d.dtype == MSSA_BF16) {
    int64_t per_head = 0;
    for (int g = 0; g < G; ++g) {
      int64_t stages = 0;
      for (const Run& r : p.runs[g]) stages += (r.n_tok + kBwdKS - 1) / kBwdKS;
      const int64_t nq = p.groups[g].q_end - p.groups[g].q_begin;
      const int64_t qblocks = 2 * ((nq + kBwdQS - 1) / kBwdQS);
      // the dK/dV kernel addresses a stage's two 32-query blocks of tiles
      // with 32-bit offsets
      if (stages * 2 * kBwdKS * 64 > 0xffffffffLL || qblocks > 0x7fffffff) {
        err = "backward dS buffer too large";
        return MSSA_ERR_UNSUPPORTED;
      }
      p.bwd_ds_stages[g] = static_cast<int32_t>(stages);
      p.bwd_ds_qblocks[g] = static_cast<int32_t>(qblocks);
      per_head += qblocks * stages * kBwdKS * 32 * 2;
    }
    // whole heads per chunk within the budget, at least one
    p.bwd_ds_heads = static_cast<int32_t>(
        std::max<int64_t>(1, std::min<int64_t>(d.num_heads, kBwdDsBudget / std::max<int64_t>(1, per_head))));
    for (int g = 0; g < G; ++g) {
      p.bwd_ds_off[g] = ws;
      ws += align256(static_cast<int64_t>(p.bwd_ds_heads) * p.bwd_ds_qblocks[g] * p.bwd_ds_stages[g] * kBwdKS * 32 * 2);
    }
  }
  p.bwd_workspace_bytes = ws;
  auto seg_of = [&](int g, int32_t kind, int32_t frame) -> const SegRow& {
    for (const SegRow& r : p.segs)
      if (r.q_scale == p.groups[g].scale && r.kind == kind && r.frame == frame) return r;
    return p.segs.front();  // unreachable: every source frame is in every context
  };
  bool scatter_ok = true;
  auto add_job = [&](int32_t buffer, int32_t kind, int32_t frame0, int64_t src_tok, int32_t n_frames,
                     int32_t src_scale) {
    ScatterJob j;
    j.buffer = buffer;
    j.src_tok = src_tok;
    j.n_frames = n_frames;
    j.gh = ceil_div(d.grid_h, src_scale);
    j.gw = ceil_div(d.grid_w, src_scale);
    for (int g = 0; g < G; ++g) {
      const SegRow& r = seg_of(g, kind, frame0);
      j.ctx_begin.push_back(r.kv_begin);
      j.frame_stride.push_back(r.n_tok);
      j.factor.push_back(r.factor);
      // a resampled frame has ceil(gh / f) x ceil(gw / f) tokens, and the
      // job's frames lie inside the context
      scatter_ok &= r.kind == kind && r.frame == frame0 &&
                    static_cast<int64_t>(ceil_div(j.gh, r.factor)) * ceil_div(j.gw, r.factor) == r.n_tok &&
                    r.kv_begin + static_cast<int64_t>(n_frames) * r.n_tok <= p.groups[g].n_kv;
    }
    p.scatter_jobs.push_back(j);
  };
  if (d.sink_frames > 0) add_job(kBufSink, kSink, 0, 0, d.sink_frames, 1);
  if (d.hist_frames > 0) add_job(kBufHist, kHist, 0, 0, d.hist_frames, 1);
  for (size_t i = 0; i < wf.size();) {
    size_t e = i;
    while (e < wf.size() && wf[e].p == wf[i].p) ++e;
    add_job(kBufWin, kWin, wf[i].w, wf[i].first, static_cast<int32_t>(e - i), wf[i].p);
    i = e;
  }
  if (!scatter_ok) {
    err = "internal: inconsistent gradient scatter tables";
    return MSSA_ERR_UNSUPPORTED;
  }

  // Algorithmic pool traffic, K and V: block mean, each pooled source frame
  // read once and each pooled frame written once; stride, each pooled token
  // reads the one source token it copies.
  int64_t write_tok = 0;
  for (int64_t t : p.pooled_tokens) write_tok += t;
  int64_t read_tok = hist_read ? p.n_hist_tok : 0;
  for (size_t i = 0; i < wf.size(); ++i)
    if (win_read[i]) read_tok += wf[i].n;
  if (p.head_ring) {
    // state 1's frames, read once from the ring and written pooled to every
    // coarser query scale's ring
    bool any = false;
    for (const QGroup& g : p.groups)
      if (g.scale > 1) {
        write_tok += F * tok_at(g.scale);
        any = true;
      }
    if (any) read_tok += F * p.tok1;
  }
  if (p.strided) read_tok = write_tok;
  p.pool_bytes_alg = 2 * (read_tok + write_tok) * p.ld * p.elem_bytes;
  return MSSA_OK;
}

Schedule make_schedule(const Plan& p, const std::vector<std::vector<int64_t>>& n_tok) {
  const int G = static_cast<int>(p.groups.size());
  Schedule sc;
  sc.tiles_per_item.assign(G, 0);
  sc.tile_begin.assign(G, 0);
  int64_t n_items = 0, t_max = 0;
  std::vector<int64_t> item_first(G, 0);
  for (int g : p.order) {
    int64_t tiles = 0;
    for (int64_t n : n_tok[g]) tiles += (n + kFwdBN - 1) / kFwdBN;
    sc.tiles_per_item[g] = static_cast<int32_t>(tiles);
    sc.tile_begin[g] = sc.total_tiles;
    item_first[g] = n_items;
    const int64_t items =
        static_cast<int64_t>((p.groups[g].q_end - p.groups[g].q_begin + kFwdBM - 1) / kFwdBM) * p.desc.num_heads;
    n_items += items;
    sc.total_tiles += items * tiles;
    t_max = std::max(t_max, tiles);
  }
  const int64_t ranges = p.n_ranges;
  // Whole-item rounds: as many as fit without any block exceeding its even
  // share total_tiles / ranges; the rest is split into per-block tail ranges
  // sized to make every block's total equal.
  sc.dp_rounds = static_cast<int32_t>(
      std::min<int64_t>(n_items / ranges, (sc.total_tiles / ranges) / std::max<int64_t>(1, t_max)));
  const int64_t i = static_cast<int64_t>(sc.dp_rounds) * ranges;  // first tail item
  int gl = p.order.front();
  for (int g : p.order)
    if (i >= item_first[g]) gl = g;
  sc.tail_begin = sc.tile_begin[gl] + (i - item_first[gl]) * sc.tiles_per_item[gl];
  return sc;
}

std::vector<int64_t> export_tables(const Plan& p) {
  std::vector<int64_t> t;
  t.push_back(static_cast<int64_t>(p.grids.size()));
  t.push_back(static_cast<int64_t>(p.groups.size()));
  t.push_back(static_cast<int64_t>(p.segs.size()));
  for (const GridRow& g : p.grids) t.insert(t.end(), {g.scale, g.gh, g.gw, g.tok});
  for (const QGroup& g : p.groups) t.insert(t.end(), {g.scale, g.q_begin, g.q_end, g.n_kv});
  for (const SegRow& r : p.segs)
    t.insert(t.end(), {r.q_scale, r.kind, r.frame, r.src_scale, r.eff_scale, r.factor, r.n_tok, r.kv_begin});
  t.push_back(p.n_q);
  t.push_back(p.pairs_per_head);
  return t;
}


// K slices of a narrow GEMM (launch_gemm_split): enough blocks for two per
// CU at most, each slice at least three stages; 1 when the output tiles alone
// fill 256 CUs or K does not split into such slices.
int gemm_k_splits(int32_t M, int32_t N, int32_t K) {
  if (M <= 0 || N <= 0 || K % kGemmStage != 0) return 1;
  const int64_t tiles = static_cast<int64_t>((M + kGemmTile - 1) / kGemmTile) * ((N + kGemmTile - 1) / kGemmTile);
  if (tiles >= 256) return 1;
  const int stages = K / kGemmStage;
  int best = 1;
  for (int s = 2; s <= stages; ++s)
    if (stages % s == 0 && stages / s >= 3 && tiles * s <= 512) best = s;
  return best;
}

int64_t gemm_split_bytes(int32_t M, int32_t N, int32_t K) {
  const int s = gemm_k_splits(M, N, K);
  if (s <= 1) return 0;
  const int64_t tiles = static_cast<int64_t>((M + kGemmTile - 1) / kGemmTile) * ((N + kGemmTile - 1) / kGemmTile);
  return s * tiles * kGemmTile * kGemmTile * 4;
}

}  // namespace mssa
