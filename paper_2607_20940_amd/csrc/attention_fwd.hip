// Multi-scale self-attention forward (Ms. Forcing, Sec. 4.1, Eq. 4): for
// every head and query scale, softmax(scale q k^T) v over the concatenated
// context runs of that scale (sink | history at the query scale | window at
// max(query scale, own scale)).
//
// bf16 path (gfx950 matrix cores).  A persistent block of 8 waves attends
// 256 queries of one (query scale, head) at a time; each wave owns 32
// queries.  The block walks the scale's runs in 64-key tiles staged through
// LDS.  Per tile and wave:
//   S^T = K Q^T   with v_mfma_f32_32x32x16_bf16 (A = K rows from LDS,
//                 B = the wave's Q fragment held in registers), so each lane
//                 holds 16 keys of ONE query: the softmax row reductions are
//                 in-lane plus one exchange between the two half-waves;
//   online softmax in fp32 in the exp2 domain (scale * log2 e folded into
//                 one FMA per score; for queries supplied pre-scaled by
//                 scale * log2 e the running max enters the MFMA as its
//                 accumulator input instead, and a score needs nothing but
//                 its exponential);
//   O^T += V^T P^T with the same MFMA: the exponentiated scores are already
//                 laid out as the B operand (their key order defines the
//                 contraction order), and V^T comes from row-major V in LDS
//                 through the gfx950 transposing LDS read ds_read_b64_tr_b16.
// The two halves of the block alternate matrix-core and softmax phases so
// that every SIMD always has one wave feeding its matrix core.
// Keys past the end of a run are zero-filled in LDS and masked to -inf.
//
// fp32 path: one lane per query, plain fp32 FMA dot products and an online
// softmax with expf; used for fp32 plans (correctness path).
//
// Optionally (a.lse non-null) every path also writes, per head and query, the
// natural log of the softmax denominator, log sum_j exp(scale q k_j): the
// statistic the backward pass recomputes the probabilities from.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.hpp"
#include "lds_stage.hpp"

namespace mssa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;


// Logical block -> (group, head, query tile).  Groups are stored longest
// context first; inside a group consecutive blocks share a head.
struct Work {
  int g, head, tile;
};

__device__ inline Work decode(const FwdArgs& a, int L) {
  int g = 0;
  while (g + 1 < a.n_groups && L >= a.groups[g + 1].block_begin) ++g;
  const int idx = L - a.groups[g].block_begin;
  const int nt = a.groups[g].n_qtiles;
  return {g, idx / nt, idx % nt};
}

// Lazy rescaling threshold (log2 units): the running max used for the
// exponentials is raised only when a tile's max exceeds it by more than this,
// so exponentials stay <= 2^8 and most tiles skip the O rescale.  The final
// O / l is unchanged; only rounding differs.
constexpr float kRescaleLog2 = 8.0f;
constexpr float kRescaleSum = 256.0f;  // 2^kRescaleLog2
constexpr float kLn2 = 0.6931471805599453f;

// ---------------------------------------------------------------------------
// Persistent schedule.  An item is one (query scale, head, 256-query tile); its
// context is tiles_per_item 64-key tiles.  Items are numbered group by group
// (longest context first), head-major, and laid out in a linear tile space of
// total_tiles tiles.  Each of the n_ranges blocks first attends dp_rounds
// whole items (item r * n_ranges + rho in round r), in lockstep with the
// blocks of its XCD, which work on neighbouring query tiles of the same head
// and so share K/V in L2.  The remaining items (from tail_begin) are cut into
// one contiguous tail range per block, sized so that every block's total is
// total_tiles / n_ranges.  A tail range may begin or end inside an item: that
// piece writes a partial record (O unnormalised, running max, row sum) and
// combine_kernel merges the pieces of each split item in range order.  Record
// of the piece of an item inside tail range j: 2j if the item began at or
// before the range start (the range's first piece), else 2j + 1.

// First tile of item i (i may be the total item count).
__device__ inline int64_t item_tile(const FwdArgs& a, int64_t i) {
  int g = 0;
  while (g + 1 < a.n_groups && i >= a.groups[g + 1].block_begin) ++g;
  return a.groups[g].tile_begin + (i - a.groups[g].block_begin) * a.groups[g].tiles_per_item;
}

// Start of tail range rho: tail_begin + rho * total / n_ranges minus the
// tiles that the ranges before it spent on whole-item rounds.
__device__ inline int64_t range_begin(const FwdArgs& a, int rho) {
  const int B = a.n_ranges;
  int64_t dp = 0;
  for (int r = 0; r < a.dp_rounds; ++r)
    dp += item_tile(a, static_cast<int64_t>(r) * B + rho) - item_tile(a, static_cast<int64_t>(r) * B);
  return a.tail_begin + static_cast<int64_t>(rho) * a.total_tiles / B - dp;
}

// Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous eighth of the range indices so that its L2 serves few heads.
__device__ inline int range_of_block(int b, int B) {
  const int q = B / 8, r = B % 8, x = b % 8, j = b / 8;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

struct Loc {
  int g, item, k;      // group, item within the group, tile within the item
  int64_t item_begin;  // linear tile of the item's first tile
};

__device__ inline Loc locate(const FwdArgs& a, int64_t t) {
  int g = 0;
  while (g + 1 < a.n_groups && t >= a.groups[g + 1].tile_begin) ++g;
  const FwdGroupArgs& G = a.groups[g];
  const int64_t rel = t - G.tile_begin;
  const int item = static_cast<int>(rel / G.tiles_per_item);
  const int k = static_cast<int>(rel - static_cast<int64_t>(item) * G.tiles_per_item);
  return {g, item, k, G.tile_begin + static_cast<int64_t>(item) * G.tiles_per_item};
}

template <int D>
struct FwdTile {
  static constexpr int BM = kFwdBM, BN = kFwdBN;
  static constexpr int KS = D / 16;    // 16-wide k-steps of q k^T
  static constexpr int DB = D / 32;    // 32-row blocks of O^T
  // K and V tiles: 256-byte rows (the channels of one head, zero past D) in
  // the XOR-swizzled layout of lds_stage.hpp, so that the K row reads and
  // the transposing V reads are both conflict-free; filled by direct
  // global -> LDS transfers of 1 KB (four rows) per wave instruction.
  static constexpr int KT = BN * 128, VT = BN * 128;  // elements per LDS tile
  static constexpr int NDMA = BN * 256 / 1024 / 4;    // transfers per wave of a group, per tile
  static constexpr int kLead = 4;                     // operands read ahead of their MFMA
  static constexpr int LDS_BYTES = 2 * (2 * KT + 2 * VT);
  static_assert(NDMA == 4, "transfer addressing assumes 16 rows per wave");
};

__device__ inline float halfwave_max(float v) { return fmaxf(v, other_half(v)); }

__device__ inline float halfwave_sum(float v) { return v + other_half(v); }

// One piece: tiles [k, k + nt) of item `item` of group G, by the whole block.
// Writes the final output if the piece is the whole item, else partial
// record `rec`.
//
// The 8 waves form two groups of 4 (waves w and w + 4 share a SIMD); group 0
// owns queries 0..127 of the item's tile, group 1 queries 128..255.  Phases
// are separated by block barriers; in phase 2j group 0 runs its matrix-core
// step M(j) = {O += P_{j-1} V_{j-1}; S_j = K_j Q^T} while group 1 runs its
// softmax step on S_{j-1}, and in phase 2j + 1 the roles swap.  Each SIMD
// thus has one wave issuing MFMAs while the other issues VALU work.
//
// Tile traffic is by direct transfers, issued by the group in its softmax
// phase so that the matrix-core phases hold no transfer instructions: at the
// start of phase 2j group 1 issues V_j and at the start of phase 2j + 1 group
// 0 issues K_{j+1}, each waited for at the end of the same phase.  The first
// kLead operands of a matrix-core step (V^T of the previous tile) are read
// from LDS at the end of the wave's softmax phase, before the barrier, so
// the step starts with its operands in registers.  K_{j+1} goes to the
// buffer of K_{j-1} (last read in phase 2j - 1), V_j to that of V_{j-2}
// (last read in phase 2j - 1, prefetched in phase 2j - 2 at the latest).
//
// kQS: the queries arrive multiplied by scale * log2 e (MSSA_PLAN_Q_PRESCALED).
template <int D, bool kQS>
__device__ __forceinline__ void attend_piece(const FwdArgs& a, const FwdGroupArgs& G, int item, int k,
                                             int nt, bool whole, int rec, char* lds) {
  using P = FwdTile<D>;
  constexpr int BM = P::BM, BN = P::BN, KS = P::KS, DB = P::DB, NDMA = P::NDMA, kLead = P::kLead;
  constexpr int KT = P::KT, VT = P::VT;

  const int head = item / G.n_qtiles;
  const int qtile = item - head * G.n_qtiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // Wave-uniform values go through readfirstlane so that branches on them are
  // scalar branches: MFMA instructions ignore EXEC, so a lane-masked branch
  // around the matrix-core step would still run its MFMAs.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;  // 0: matrix core in even phases; 1: in odd phases
  const int n = lane & 31;    // query column of this lane
  const int hh = lane >> 5;   // half-wave
  const int q_row = G.q_begin + qtile * BM + wave * 32 + n;
  const bool q_ok = q_row < G.q_end;
  const int64_t ld = a.ld;
  const int64_t hoff = static_cast<int64_t>(head) * D;
  const uint32_t row_bytes = static_cast<uint32_t>(ld) * 2;
  const float c = a.scale_log2e;

  bf16x8 qf[KS];
  {
    const __bf16* qp = static_cast<const __bf16*>(a.q) + static_cast<int64_t>(q_ok ? q_row : G.q_begin) * ld +
                       hoff + hh * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 v = *reinterpret_cast<const bf16x8*>(qp + ks * 16);
      if (!q_ok) v = bf16x8{};
      qf[ks] = v;
    }
  }

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16{};
  float m_run = -INFINITY;  // running max in the exp2 domain (shared by both half-waves)
  float l_part = 0.f;       // this lane's share of the row sum
  // kQS only.  Accumulator input of the first MFMA of every S chain: -m_c in
  // all 16 elements (a lane's 16 elements all belong to its query), with
  // m_c = m_run once the first tile has set it and 0 before, so S arrives as
  // S - m_c.  The first tile's row sum is seeded with +inf (lbias), which
  // sends that tile through the max path whatever the size of its scores.
  f32x16 cneg = f32x16{};
  float lbias = INFINITY;
  f32x16 s[BN / 32];
  bf16x8 pb[BN / 32][2];
  bf16x8 ring[kLead];       // LDS operands of the matrix-core step, kLead ahead

  // Operand addresses in the swizzled tiles (elements).  K row reads: row
  // 32 kb + n, columns 16 ks + 8 hh, at 32 kb * 128 + (k_rd ^ 16 ks).
  // Transposing V reads: rows R + t_row (+ 8 for the upper half), columns
  // 32 db + t_col with R a multiple of 16, at R * 128 + v_rd[db][half]: the
  // swizzle of a row depends only on its index mod 16.
  const int k_rd = swz256(n, hh * 8);
  const int t_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int t_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int v_rd[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int h = 0; h < 2; ++h) v_rd[db][h] = swz256(t_row + 8 * h, db * 32 + t_col);
  __bf16* const Klds = reinterpret_cast<__bf16*>(lds);
  __bf16* const Vlds = Klds + 2 * KT;

  // This wave's tile transfers: transfer i fills LDS bytes
  // ((wave & 3) * NDMA + i) * 1024 + 16 lane, i.e. row (wave & 3) * 16 + 4 i +
  // lane / 16, physical chunk lane % 16, whose logical chunk is
  // lane % 16 ^ 4 (lane / 16) ^ i (the swizzle of rows 4 i .. 4 i + 3 mod 16).
  // The lane's global offset is then t_off ^ 16 i plus the scalar 4 i rows
  // (row_bytes is a multiple of 128, so the chunk bits do not carry).
  const int t_lc = (lane & 15) ^ ((lane >> 4) << 2);
  const uint32_t t_off = ((wave & 3) * 16 + (lane >> 4)) * row_bytes + t_lc * 16;

  // Tile streams over the item's context runs.  A stream points at its
  // current tile (head offset applied) and counts the tokens of the run from
  // there on, so stepping to the next tile is a pointer add and a subtract;
  // only a step past the end of a run (a few times per item) reads the run
  // table again, skipping empty runs.
  struct Stream {
    const __bf16* p;  // first token of the current tile
    int left;         // tokens of the current run from p on (> 0 while live)
    int r;            // current run
  };
  const int64_t tile_step = static_cast<int64_t>(BN) * ld;
  auto run_base = [&](bool is_v, int r) {
    return static_cast<const __bf16*>(is_v ? G.runs[r].v : G.runs[r].k) + hoff;
  };
  auto stream_at = [&](bool is_v, int j) {  // j: tile index within the item
    int r = 0;
    while (j >= (G.runs[r].n_tok + BN - 1) / BN) {
      j -= (G.runs[r].n_tok + BN - 1) / BN;
      ++r;
    }
    return Stream{run_base(is_v, r) + j * tile_step, G.runs[r].n_tok - j * BN, r};
  };
  auto step = [&](bool is_v, Stream& st) {
    st.left -= BN;
    st.p += tile_step;
    if (st.left <= 0) {
      do {
        ++st.r;
      } while (st.r < G.n_runs && G.runs[st.r].n_tok == 0);
      if (st.r < G.n_runs) {
        st.p = run_base(is_v, st.r);
        st.left = G.runs[st.r].n_tok;
      }
    }
  };

  // Direct transfers of the stream's current tile into K (is_v false) or V
  // buffer buf.  Waited for (vmcnt) before the barrier that publishes it.
  // Chunks past D (head_dim 64) point past the range and arrive as zeros.
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));
  auto issue = [&](const Stream& st, bool is_v, int buf) {
    const uint32_t base = lds0 + (is_v ? 2 * KT * 2 : 0) + buf * KT * 2 + (wave & 3) * NDMA * 1024;
    if (st.left >= BN) {
      // A whole tile: every row lies inside the run, so the 4 i rows of
      // transfer i ride in the scalar offset.
      const i32x4 rs = rsrc_of(st.p, static_cast<uint32_t>(BN - 1) * row_bytes + D * 2);
#pragma unroll
      for (int i = 0; i < NDMA; ++i) {
        const uint32_t vo = (D / 8 >= 16 || (t_lc ^ i) < D / 8) ? (t_off ^ (i * 16)) : kPastEnd;
        dma16_soff(rs, vo, i * 4 * row_bytes, __builtin_amdgcn_readfirstlane(base + i * 1024));
      }
    } else {
      // The run's last, partial tile: the whole row is in the lane's offset,
      // which the buffer range check covers (the scalar offset is not
      // checked), so rows past the run's end arrive as zeros and no byte
      // past the run is read.
      const i32x4 rs = rsrc_of(st.p, static_cast<uint32_t>(st.left - 1) * row_bytes + D * 2);
#pragma unroll
      for (int i = 0; i < NDMA; ++i) {
        const uint32_t vo = (D / 8 >= 16 || (t_lc ^ i) < D / 8) ? (t_off ^ (i * 16)) + i * 4 * row_bytes
                                                                : kPastEnd;
        dma16(rs, vo, __builtin_amdgcn_readfirstlane(base + i * 1024));
      }
    }
  };

  // Operands of a matrix-core step, in MFMA order: with pv_c the V^T
  // operands of O += P V (key block kb, 16-key half cc, column block db;
  // two transposing reads each), then with s_c the K operands of S = K Q^T
  // (k-step ks, key block kb; one row read each).
  auto operand = [&](auto pv_c, int i, int vb, int kb_) -> bf16x8 {
    constexpr int NPV = decltype(pv_c)::value ? 2 * (BN / 32) * DB : 0;
    if (i < NPV) {
      const int st = i / DB, db = i % DB, kb = st >> 1, cc = st & 1;
      const __bf16* vrow = Vlds + vb * VT + (kb * 32 + cc * 16) * 128;
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vrow + v_rd[db][0]));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vrow + v_rd[db][1]));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
    const int j = i - NPV, ks = j / (BN / 32), kb = j % (BN / 32);
    return *reinterpret_cast<const bf16x8*>(Klds + kb_ * KT + kb * 32 * 128 + (k_rd ^ (ks * 16)));
  };
  // The first kLead operands of a step into the ring (a step has at least
  // kLead operands: 2 (BN / 32) DB V^T operands, or KS (BN / 32) K operands).
  auto prefill = [&](auto pv_c, int vb, int kb_) {
    constexpr int N = (decltype(pv_c)::value ? 2 * (BN / 32) * DB : KS * (BN / 32));
    static_assert(N >= kLead, "ring longer than a step");
#pragma unroll
    for (int i = 0; i < kLead; ++i)
      if (i < N) ring[i] = operand(pv_c, i, vb, kb_);
  };

  // Matrix-core step: O += P V from V buffer vb (if pv_c), then S = K Q^T from
  // K buffer kb_ (if s_c), as one stream of MFMAs whose LDS operands run
  // kLead operands ahead in the register ring (filled before the step).
  // Scheduling group barriers fix the interleave: the compiler would
  // otherwise hoist every read to the top (more registers) or sink each next
  // to its MFMA (no overlap).
  auto mstep = [&](auto pv_c, auto s_c, int vb, int kb_) {
    constexpr bool kPV = decltype(pv_c)::value, kS = decltype(s_c)::value;
    constexpr int NPV = kPV ? 2 * (BN / 32) * DB : 0;  // (key block, 16-key half, d block)
    constexpr int NS = kS ? KS * (BN / 32) : 0;        // (d slice, key block)
    constexpr int N = NPV + NS;
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const bf16x8 av = ring[i % kLead];
      if (i < NPV) {
        const int st = i / DB, db = i % DB, kb = st >> 1, cc = st & 1;
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[kb][cc], o[db], 0, 0, 0);
      } else {
        const int j = i - NPV, ks = j / (BN / 32), kb = j % (BN / 32);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qf[ks], ks == 0 ? (kQS ? cneg : f32x16{}) : s[kb],
                                                         0, 0, 0);
      }
      if (i + kLead < N) ring[i % kLead] = operand(pv_c, i + kLead, vb, kb_);
    }
    // A V operand is two LDS reads, a K operand one.
    auto read_group = [&](int i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (i < NPV) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    };
#pragma unroll
    for (int i = 0; i < N; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i + kLead < N) read_group(i + kLead);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // Softmax step on S (keys >= nvalid of this tile masked): P = exp2(S c - m)
  // (kQS: exp2(S), m already subtracted by the MFMA) packed to bf16 as the B
  // operand of the next P V, with m the running max.  Lazy rescaling without
  // a per-tile max: P is first computed against the current m; if every
  // lane's sum over its 32 keys stays <= 2^kRescaleLog2, so does every P and
  // nothing else is needed.  Otherwise (the first tile, where m is -inf, or
  // scores well above m) the tile max is taken, m is raised if the max
  // exceeds it by more than kRescaleLog2 (O and l scaled down), and P is
  // recomputed (kQS: the new -m also goes into the accumulator input of the
  // next S).  Either way P <= 2^kRescaleLog2.
  auto sstep = [&](int nvalid) {
    if (nvalid < BN) {
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kb * 32 + 8 * (e >> 2) + 4 * hh + (e & 3);
          if (key >= nvalid) s[kb][e] = -INFINITY;
        }
    }
    // Row sum in fp32 VALU adds (four independent partial sums): the bf16 dot
    // instruction would wait on the matrix core that the other wave of this
    // SIMD keeps busy.
    // Exponent of a score: S c + off (plain), S (kQS, first pass) or S + off
    // (kQS, after the max path moved m); bias seeds the row sum.
    auto exps = [&](auto shift_c, float off, float bias) {
      constexpr bool kShift = decltype(shift_c)::value;
      auto arg = [&](float x) { return kQS ? (kShift ? x + off : x) : __builtin_fmaf(x, c, off); };
      float ls[4] = {bias, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(arg(s[kb][e]));
          const float p1 = __builtin_amdgcn_exp2f(arg(s[kb][e + 1]));
          ls[(e >> 1) & 3] += p0 + p1;
          pb[kb][e >> 3][e & 7] = static_cast<__bf16>(p0);
          pb[kb][e >> 3][(e & 7) + 1] = static_cast<__bf16>(p1);
        }
      return (ls[0] + ls[1]) + (ls[2] + ls[3]);
    };
    float lt = kQS ? exps(std::false_type{}, 0.f, lbias) : exps(std::false_type{}, -m_run, 0.f);
    if (__any(!(lt <= kRescaleSum))) {  // also true for inf / NaN sums
      float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
      for (int e = 2; e < 16; e += 2) mx = fmaxf(fmaxf(mx, s[0][e]), s[0][e + 1]);
#pragma unroll
      for (int kb = 1; kb < BN / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 16; e += 2) mx = fmaxf(fmaxf(mx, s[kb][e]), s[kb][e + 1]);
      const float m_c = kQS ? -cneg[0] : 0.f;  // kQS: what the MFMA subtracted
      const float mt = kQS ? halfwave_max(mx) + m_c : halfwave_max(mx) * c;
      if (__any(mt > m_run + kRescaleLog2)) {
        const float m_new = fmaxf(m_run, mt);
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_part *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= alpha;
      }
      if constexpr (kQS) {
        lt = exps(std::true_type{}, m_c - m_run, 0.f);
#pragma unroll
        for (int e = 0; e < 16; ++e) cneg[e] = -m_run;
        lbias = 0.f;
      } else {
        lt = exps(std::false_type{}, -m_run, 0.f);
      }
    }
    l_part += lt;
    // P and the row sum are pure register values, so the compiler is free to
    // sink their exponentials past the phase barrier into the next
    // matrix-core step, which would load that step with this one's VALU work.
    // Empty asm with read-write register operands pins them here.
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
      for (int h = 0; h < 2; ++h) asm volatile("" : "+v"(pb[kb][h]));
    asm volatile("" : "+v"(l_part));
  };

  Stream ts = stream_at(grp != 0, k);  // group 0: K tiles, group 1: V tiles
  Stream ss = stream_at(false, k);     // tile lengths for the softmax masks
  if (grp == 0) issue(ts, false, 0);
  wait_vmcnt<0>();
  __syncthreads();
  // Transfer of tile t (if it exists) of the group's tensor into buffer
  // t & 1 = buf: K_t for group 0, V_t for group 1.
  auto transfer = [&](int t, int buf) {
    if (t < nt) {
      if (t > 0 || grp == 0) step(grp != 0, ts);
      issue(ts, grp != 0, buf);
    }
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  // Matrix-core step with high issue priority, softmax with normal priority.
  auto mphase = [&](auto pv_c, auto s_c, int vb, int kb_) {
    __builtin_amdgcn_s_setprio(2);
    mstep(pv_c, s_c, vb, kb_);
    __builtin_amdgcn_s_setprio(0);
  };
  auto soft = [&]() {
    sstep(min(ss.left, BN));
    step(false, ss);
  };
  // The tile loops are unrolled by two so that every LDS buffer index is a
  // compile-time constant (par = j & 1) and operand addresses are immediates.
  if (grp == 0) {
    // phase 2j: M(j); phase 2j + 1: K_{j+1} issued, softmax(j), then the
    // first operands of M(j + 1) (V_j, published at the end of phase 2j).
    prefill(F_{}, 0, 0);
    mphase(F_{}, T_{}, 0, 0);
    __syncthreads();
    transfer(1, 1);
    soft();
    prefill(T_{}, 0, 1);
    wait_vmcnt<0>();
    __syncthreads();
    auto iter = [&](int j, auto par) {
      constexpr int p = decltype(par)::value;
      mphase(T_{}, T_{}, p ^ 1, p);
      __syncthreads();
      transfer(j + 1, p ^ 1);
      soft();
      prefill(T_{}, p, p ^ 1);
      wait_vmcnt<0>();
      __syncthreads();
    };
    int j = 1;
    for (; j + 1 < nt; j += 2) {
      iter(j, I1{});
      iter(j + 1, I0{});
    }
    if (j < nt) iter(j, I1{});
    if (nt & 1)
      mphase(T_{}, F_{}, 0, 1);
    else
      mphase(T_{}, F_{}, 1, 0);
    __syncthreads();
    __syncthreads();
  } else {
    // phase 2j: V_j issued, softmax(j - 1), wait for V_j, the first operands
    // of M(j) (V_{j-1}); phase 2j + 1: M(j).
    transfer(0, 0);
    prefill(F_{}, 0, 0);
    wait_vmcnt<0>();
    __syncthreads();
    mphase(F_{}, T_{}, 0, 0);
    __syncthreads();
    auto iter = [&](int j, auto par) {
      constexpr int p = decltype(par)::value;
      transfer(j, p);
      soft();
      prefill(T_{}, p ^ 1, p);
      wait_vmcnt<0>();
      __syncthreads();
      mphase(T_{}, T_{}, p ^ 1, p);
      __syncthreads();
    };
    int j = 1;
    for (; j + 1 < nt; j += 2) {
      iter(j, I1{});
      iter(j + 1, I0{});
    }
    if (j < nt) iter(j, I1{});
    soft();
    if (nt & 1) {
      prefill(T_{}, 0, 0);
      __syncthreads();
      mphase(T_{}, F_{}, 0, 1);
    } else {
      prefill(T_{}, 1, 0);
      __syncthreads();
      mphase(T_{}, F_{}, 1, 0);
    }
    __syncthreads();
  }

  const float l_tot = halfwave_sum(l_part);
  if (whole) {
    if (a.lse && q_ok && hh == 0)
      a.lse[static_cast<int64_t>(head) * a.n_q + q_row] = (m_run + log2f(l_tot)) * kLn2;
    if (q_ok) {
      const float inv = 1.0f / l_tot;
      __bf16* op = static_cast<__bf16*>(a.out) + static_cast<int64_t>(q_row) * ld + hoff + 4 * hh;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          bf16x4 v;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = static_cast<__bf16>(o[db][4 * jj + i] * inv);
          *reinterpret_cast<bf16x4*>(op + db * 32 + 8 * jj) = v;
        }
    }
  } else {
    float* ro = a.partial + static_cast<int64_t>(rec) * partial_record_floats(D);
    const int ql = wave * 32 + n;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = o[db][4 * jj + i];
        *reinterpret_cast<f32x4*>(ro + ql * D + db * 32 + 8 * jj + 4 * hh) = v;
      }
    if (hh == 0) {
      ro[BM * D + ql] = m_run;
      ro[BM * D + BM + ql] = l_tot;
    }
  }
}

template <int D, bool kQS>
__global__ __launch_bounds__(kFwdThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void fwd_bf16_kernel(FwdArgs a) {
  using P = FwdTile<D>;
  // [K buf0 | K buf1 | V buf0 | V buf1], 64 rows of 256 bytes each
  __shared__ __attribute__((aligned(16))) char lds[P::LDS_BYTES];
  const int rho = range_of_block(blockIdx.x, a.n_ranges);
  const int64_t S = range_begin(a, rho), E = range_begin(a, rho + 1);
  // The merge of split items reads the tail ranges from this table.
  if (a.range_table && threadIdx.x == 0) {
    a.range_table[rho] = S;
    if (rho == a.n_ranges - 1) a.range_table[rho + 1] = E;
  }
  // Whole items of the aligned rounds, then the pieces of the tail range;
  // one call site keeps a single copy of the attention loop.
  int round = 0;
  int64_t t = S;
  while (true) {
    int g, item, k, nt, rec;
    bool whole;
    if (round < a.dp_rounds) {
      const int64_t i = static_cast<int64_t>(round) * a.n_ranges + rho;
      g = 0;
      while (g + 1 < a.n_groups && i >= a.groups[g + 1].block_begin) ++g;
      item = static_cast<int>(i - a.groups[g].block_begin);
      k = 0;
      nt = a.groups[g].tiles_per_item;
      whole = true;
      rec = 0;
      ++round;
    } else if (t < E) {
      const Loc L = locate(a, t);
      const int64_t piece_end = min(E, L.item_begin + a.groups[L.g].tiles_per_item);
      g = L.g;
      item = L.item;
      k = L.k;
      nt = static_cast<int>(piece_end - t);
      whole = L.k == 0 && nt == a.groups[g].tiles_per_item;
      rec = t == S ? 2 * rho : 2 * rho + 1;
      t = piece_end;
    } else {
      break;
    }
    attend_piece<D, kQS>(a, a.groups[g], item, k, nt, whole, rec, lds);
  }
}

// Merge the pieces of items split across ranges.  Block (j, y) looks at tail
// range j: if the range ends inside an item whose first tile it holds, it
// combines queries [y QS, (y + 1) QS) of all of that item's pieces (ranges
// j .. j1) in range order.  Range bounds come from the table the attention
// kernel wrote.  Each thread owns one float4 of the output and loads it from
// up to kMaxMerge pieces at once (an item of the tail may be cut into many
// short pieces), then merges them in order.
template <int D>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(FwdArgs a) {
  constexpr int BM = kFwdBM, QS = kCombineThreads * 4 / D, kMaxMerge = 8;
  const int64_t* tab = a.range_table;
  const int j = blockIdx.x;
  const int64_t S = tab[j], E = tab[j + 1];
  if (S == E || E >= a.total_tiles) return;  // empty range, or nothing after it
  const Loc L = locate(a, E);
  if (L.k == 0) return;                      // the range ends at an item boundary
  const int64_t T = L.item_begin;
  if (S > T) return;                         // the item's first piece is in an earlier range
  const FwdGroupArgs& G = a.groups[L.g];
  const int64_t Tend = T + G.tiles_per_item;
  // Last range holding a piece of the item: the table is nondecreasing.
  int j1 = j;
  for (int w = j + 1; w < a.n_ranges; w += kCombineThreads) {
    const int jt = w + static_cast<int>(threadIdx.x);
    const int cnt = __syncthreads_count(jt < a.n_ranges && tab[jt] < Tend);
    j1 += cnt;
    if (cnt < kCombineThreads) break;
  }
  const int head = L.item / G.n_qtiles;
  const int qtile = L.item - head * G.n_qtiles;
  const int64_t rec_len = partial_record_floats(D);
  const int ql = blockIdx.y * QS + static_cast<int>(threadIdx.x) / (D / 4), d4 = threadIdx.x % (D / 4);
  // Pieces are merged in range order with a running max, like the online
  // softmax itself.
  f32x4 acc = f32x4{};
  float m = -INFINITY, l = 0.f;
  for (int base = j; base <= j1; base += kMaxMerge) {
    f32x4 ov[kMaxMerge];
    float mv[kMaxMerge], lv[kMaxMerge];
    bool have[kMaxMerge];
#pragma unroll
    for (int i = 0; i < kMaxMerge; ++i) {
      const int jj = base + i;
      have[i] = jj <= j1 && tab[jj] < tab[jj + 1];  // ranges inside the span may be empty
      if (have[i]) {
        const float* ro = a.partial + (jj > j || S == T ? 2 * jj : 2 * jj + 1) * rec_len;
        ov[i] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(ro + ql * D + 4 * d4));
        mv[i] = ro[BM * D + ql];
        lv[i] = ro[BM * D + BM + ql];
      }
    }
#pragma unroll
    for (int i = 0; i < kMaxMerge; ++i) {
      if (!have[i]) continue;
      const float mn = fmaxf(m, mv[i]);
      const float so = __builtin_amdgcn_exp2f(m - mn), sj = __builtin_amdgcn_exp2f(mv[i] - mn);
      acc = acc * so + sj * ov[i];
      l = l * so + sj * lv[i];
      m = mn;
    }
  }
  const int q_row = G.q_begin + qtile * BM + ql;
  if (q_row >= G.q_end) return;
  const float inv = 1.0f / l;
  if (a.lse && d4 == 0) a.lse[static_cast<int64_t>(head) * a.n_q + q_row] = (m + log2f(l)) * kLn2;
  bf16x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = static_cast<__bf16>(acc[i] * inv);
  *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(a.out) + static_cast<int64_t>(q_row) * a.ld +
                             static_cast<int64_t>(head) * D + 4 * d4) = v;
}

template <int D>
__global__ __launch_bounds__(kFwdF32BM) void fwd_f32_kernel(FwdArgs a) {
  const Work w = decode(a, blockIdx.x);
  const FwdGroupArgs& G = a.groups[w.g];
  const int q_row = G.q_begin + w.tile * kFwdF32BM + threadIdx.x;
  if (q_row >= G.q_end) return;
  const int64_t ld = a.ld;
  const int64_t hoff = static_cast<int64_t>(w.head) * D;
  const float* qp = static_cast<const float*>(a.q) + static_cast<int64_t>(q_row) * ld + hoff;
  float q[D], o[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = qp[d];
    o[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int r = 0; r < G.n_runs; ++r) {
    const float* Kg = static_cast<const float*>(G.runs[r].k) + hoff;
    const float* Vg = static_cast<const float*>(G.runs[r].v) + hoff;
    for (int j = 0; j < G.runs[r].n_tok; ++j) {
      const float* kp = Kg + static_cast<int64_t>(j) * ld;
      const float* vp = Vg + static_cast<int64_t>(j) * ld;
      float dot = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) dot = __builtin_fmaf(q[d], kp[d], dot);
      const float z = dot * a.scale;
      if (z > m) {
        const float alpha = expf(m - z);
        l *= alpha;
#pragma unroll
        for (int d = 0; d < D; ++d) o[d] *= alpha;
        m = z;
      }
      const float p = expf(z - m);
      l += p;
#pragma unroll
      for (int d = 0; d < D; ++d) o[d] = __builtin_fmaf(p, vp[d], o[d]);
    }
  }
  float* op = static_cast<float*>(a.out) + static_cast<int64_t>(q_row) * ld + hoff;
#pragma unroll
  for (int d = 0; d < D; ++d) op[d] = o[d] / l;
  if (a.lse) a.lse[static_cast<int64_t>(w.head) * a.n_q + q_row] = m + logf(l);
}

}  // namespace

hipError_t launch_forward(const FwdArgs& a, int head_dim, bool bf16, hipStream_t stream) {
  if (bf16) {
    if (a.n_ranges <= 0) return hipSuccess;
    if (head_dim == 128 && a.q_prescaled)
      hipLaunchKernelGGL((fwd_bf16_kernel<128, true>), dim3(a.n_ranges), dim3(kFwdThreads), 0, stream, a);
    else if (head_dim == 128)
      hipLaunchKernelGGL((fwd_bf16_kernel<128, false>), dim3(a.n_ranges), dim3(kFwdThreads), 0, stream, a);
    else if (a.q_prescaled)
      hipLaunchKernelGGL((fwd_bf16_kernel<64, true>), dim3(a.n_ranges), dim3(kFwdThreads), 0, stream, a);
    else
      hipLaunchKernelGGL((fwd_bf16_kernel<64, false>), dim3(a.n_ranges), dim3(kFwdThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.n_ranges < 2) return e;
    if (head_dim == 128)
      hipLaunchKernelGGL(combine_kernel<128>, dim3(a.n_ranges - 1, kFwdBM * 128 / 4 / kCombineThreads), dim3(kCombineThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(combine_kernel<64>, dim3(a.n_ranges - 1, kFwdBM * 64 / 4 / kCombineThreads), dim3(kCombineThreads), 0, stream, a);
    return hipGetLastError();
  }
  if (a.n_blocks <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(fwd_f32_kernel<128>, dim3(a.n_blocks), dim3(kFwdF32BM), 0, stream, a);
  else
    hipLaunchKernelGGL(fwd_f32_kernel<64>, dim3(a.n_blocks), dim3(kFwdF32BM), 0, stream, a);
  return hipGetLastError();
}

int forward_blocks_per_cu(int head_dim) {
  int n = 0;
  const hipError_t e = head_dim == 128
      ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fwd_bf16_kernel<128, false>, kFwdThreads, 0)
      : hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fwd_bf16_kernel<64, false>, kFwdThreads, 0);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return n;
}

}  // namespace mssa
