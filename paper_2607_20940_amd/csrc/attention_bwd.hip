// Multi-scale self-attention backward: the chain rule through Eq. 4 of Ms.
// Forcing (Sec. 4.1), whose rolling-window training (Sec. 3.1, Alg. 1)
// differentiates the attention of every window state.  For each head and
// query scale s, with P = softmax(scale q k_s^T) over the context of s and dO
// the gradient of the output:
//   dV_s = P^T dO,  dS = P * (dO V_s^T - rowsum(dO * O)),
//   dQ = scale dS K_s,  dK_s = scale dS^T Q.
// The statistics come from the forward: the log of each row's softmax
// denominator (lse), and rowsum(dO * O) (dot_kernel, which stores both
// negated in the units the kernels use).  Context gradients are kept per
// query scale in fp32; scatter_kernel then sums, for every sink, history and
// window token, the gradients of the context rows made from it (the adjoint
// of the resampling: the block mean hands g / c to each of its c cells, the
// strided pick g to the block's first cell).  Fixed summation orders and no
// atomics: the result is the same bits on every run.
//
// bf16 path (gfx950 matrix cores, v_mfma_f32_32x32x16_bf16, fp32
// accumulation), five products in two kernels so that no gradient needs
// atomics:
//   dkdv_kernel  pairs of waves sharing a SIMD (two waves per SIMD, 8 per
//                block); a pair owns 32 context keys and walks the scale's
//                queries in 64-query stages: wave A S = Q K^T, P (lane =
//                key) and dV^T += dO^T P; wave B, one stage later, dP = dO
//                V^T, dS = P (dP - rowsum), dK^T += Q^T dS, with dO^T, Q^T
//                from transposing reads, and dS (bf16, the value its own
//                product uses) to a tile in HBM.  Strict ping-pong: in each
//                of a stage's two barrier-separated phases one wave of the
//                pair issues only MFMAs and the other only VALU work.  Each
//                wave holds one operand fragment and one accumulator, which
//                is what lets two waves share a SIMD.
//   dq_kernel    dQ^T += K^T dS^T over the context, 32 queries per wave, K
//                rows and the wave's dS tiles streamed through LDS and read
//                transposed; it reads each dS element once from HBM instead
//                of recomputing S and dP.
// One XOR-swizzled copy of each staged K / Q / dO tile serves both read
// patterns without bank conflicts; stages arrive by direct global -> LDS
// transfers (no staging registers).  Rows past the end of a context or query
// range are zero-filled and add nothing to any gradient.
//
// fp32 path (correctness path for fp32 plans): one lane per query (dQ) or
// per context key (dK, dV), plain fp32 arithmetic with expf.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "lds_stage.hpp"

namespace mssa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous eighth of the logical blocks so that its L2 serves few heads.
__device__ inline int xcd_remap(int b, int n) {
  const int q = n / 8, r = n % 8, x = b % 8, j = b / 8;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// Context token j of group G -> its K (or V) row, head 0; nullptr past the end.
template <typename T>
__device__ inline const T* ctx_row(const BwdGroupArgs& G, int j, bool v, int64_t ld) {
  if (j >= G.n_kv) return nullptr;
  int r = 0;
  while (r + 1 < G.n_runs && j >= G.runs[r].n_tok) {
    j -= G.runs[r].n_tok;
    ++r;
  }
  return static_cast<const T*>(v ? G.runs[r].v : G.runs[r].k) + static_cast<int64_t>(j) * ld;
}

// Operand shapes of both bf16 kernels: a 32-row block is read as the A
// operand of a 32x32x16 MFMA (lane n takes row n and the 8 columns of its
// half-wave), or, through the transposing read, as X^T[d][row] of a 32-wide d
// block and 16 rows in the row order in which a 32x32 accumulator's lane holds
// its 16 values, so that the accumulator packed to bf16 is the matching B
// operand.
template <int D>
struct Lay {
  static constexpr int KS = D / 16, DB = D / 32;
};

// ------------------------------------------------------------------ rowsum(dO * O)

// One row (query, head) per group of L = head_dim * sizeof(T) / 16 lanes (8,
// 16 or 32; rows are contiguous, so a wave reads 1-2 KB in one piece), each
// lane 16 bytes of O and dO; the group's partial sums meet by lane
// exchanges in a fixed order.
template <typename T>
__global__ __launch_bounds__(kDotThreads) void dot_kernel(DotArgs a) {
  constexpr int N = 16 / sizeof(T);
  typedef T vecT __attribute__((ext_vector_type(N)));
  const int L = a.head_dim / N;
  const int64_t gt = static_cast<int64_t>(blockIdx.x) * kDotThreads + threadIdx.x;
  const int64_t r = gt / L, rows = static_cast<int64_t>(a.n_q) * a.num_heads;
  const int c = static_cast<int>(gt % L);
  float acc = 0.f;
  if (r < rows) {
    // rows are contiguous: row r = (query r / heads, head r % heads) at r * head_dim
    const int64_t off = r * a.head_dim + c * N;
    const vecT ov = *reinterpret_cast<const vecT*>(static_cast<const T*>(a.out) + off);
    const vecT gv = *reinterpret_cast<const vecT*>(static_cast<const T*>(a.d_out) + off);
#pragma unroll
    for (int e = 0; e < N; ++e) acc = __builtin_fmaf(static_cast<float>(ov[e]), static_cast<float>(gv[e]), acc);
  }
  for (int m = L >> 1; m >= 1; m >>= 1) acc += __shfl_xor(acc, m);
  if (r < rows && c == 0) {
    const int q = static_cast<int>(r / a.num_heads), h = static_cast<int>(r % a.num_heads);
    // Both statistics are stored negated, as the dK/dV kernel's accumulator
    // inputs: -rowsum, and -lse / scale (the row's log-sum-exp in units of the
    // unscaled scores q k^T).
    a.dsum[static_cast<int64_t>(h) * a.n_q + q] = -acc;
    if (a.lse) a.lse2[static_cast<int64_t>(h) * a.n_q + q] = -a.lse[static_cast<int64_t>(h) * a.n_q + q] * a.inv_scale;
  }
}

// ------------------------------------------------------------------ bf16 kernels

// Stage rows: one copy per tensor in the 256-byte swizzled layout of
// lds_stage.hpp (row reads and transposing reads both conflict-free), filled
// by direct transfers.
__device__ inline int swz(int row, int col) { return swz256(row, col); }

// ------------------------------------------------------------------ bf16: dQ

// dQ = scale dS K, from the dS tiles the dK/dV kernel wrote.  A block owns
// 256 queries, eight waves of 32 (two per SIMD).  The context streams through
// LDS in 64-key stages inside one run at a time, cut as the tiles were: the
// stage's K rows (one swizzled copy for the block) and each wave's own 4 KB
// dS tile arrive by direct transfers into three stage buffers (the one read
// and two in flight: the tiles come from HBM once, and HBM latency needs that
// depth).  Rows past a run's end arrive as zeros in both, so they add
// nothing.  Each wave accumulates dQ^T += K^T dS^T with both operands from
// transposing reads: K^T from the K rows, dS^T from the tile's 64-byte rows
// (keys) of 32 query positions, which become the accumulator's columns.
// Position p of a tile row holds query 8 ((p % 16) / 4) + 4 (p / 16) + p % 4
// of the 32-query block: the order in which the dK/dV kernel's lanes hold
// them.
template <int D>
__global__ __launch_bounds__(kBwdQThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dq_kernel(BwdArgs a) {
  constexpr int DB = Lay<D>::DB;
  constexpr int BN = kBwdKS;                       // keys per stage
  constexpr int NW = kBwdQThreads / 64;            // waves of 32 queries
  constexpr int KT = BN * 256;                     // bytes of the stage's K rows (256-byte swizzled rows)
  constexpr int DT = BN * 64;                      // bytes of one wave's dS tile
  // The tile's LDS footprint: its second half sits 128 bytes further on, so
  // that the two halves' rows a transposing read takes together fall in
  // different banks.
  constexpr int DTL = DT + 128;
  constexpr int STB = KT + NW * DTL;
  constexpr int NK = KT / 1024 / NW;               // 1 KB K transfers per wave and stage
  constexpr int NDS = DT / 1024;                   // 1 KB dS transfers per wave and stage
  static_assert(NK * 1024 * NW == KT && NW * 32 == kBwdQ && BN % 32 == 0 && NDS % 2 == 0, "stage shape");
  __shared__ __attribute__((aligned(16))) char lds[3 * STB];

  int n_blocks = 0;
  for (int g = 0; g < a.n_groups; ++g) n_blocks += a.groups[g].n_qblocks * a.num_heads;
  const int b = xcd_remap(blockIdx.x, n_blocks);
  int g = 0;
  while (g + 1 < a.n_groups && b >= a.groups[g + 1].dq_block_begin) ++g;
  const BwdGroupArgs& G = a.groups[g];
  const int idx = b - G.dq_block_begin;
  const int hl = idx / G.n_qblocks, qt = idx % G.n_qblocks;  // head of the launch
  const int head = a.head0 + hl;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, hh = lane >> 5;
  const int qb = qt * NW + wave;                   // the wave's 32-query block of the group
  const bool wave_ok = G.q_begin + qb * 32 < G.q_end;
  const int q_row = G.q_begin + qb * 32 + 8 * ((n & 15) >> 2) + 4 * (n >> 4) + (n & 3);
  const int64_t ld = a.ld, hoff = static_cast<int64_t>(head) * D;

  f32x16 acc[DB];  // dQ^T: lane n holds tile position n's query
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};

  const int nr = G.n_runs;
  int nst = 0;
  for (int r = 0; r < nr; ++r) nst += (G.runs[r].n_tok + BN - 1) / BN;
  struct Stream {
    const __bf16* k;
    int left;  // tokens of the current run from k on
    int r;
  };
  const int64_t tile_step = static_cast<int64_t>(BN) * ld;
  auto seek = [&](Stream& s, int r) {
    while (r < nr && G.runs[r].n_tok == 0) ++r;
    s.r = r;
    if (r < nr) {
      s.k = static_cast<const __bf16*>(G.runs[r].k) + hoff;
      s.left = G.runs[r].n_tok;
    }
  };
  auto step = [&](Stream& s) {
    s.left -= BN;
    s.k += tile_step;
    if (s.left <= 0) seek(s, s.r + 1);
  };

  // Per-lane global offsets of this wave's K transfers (the same every
  // stage): transfer t = wave NK + i covers bytes 1024 t of the K rows,
  // logical chunk of the fixed LDS slot, zero past D.  The dS tile is copied
  // as it lies, 1 KB per transfer, non-temporal (each element is read once;
  // -1 % against plain loads, K rows keep their L2 lines).
  const uint32_t row_bytes = static_cast<uint32_t>(ld) * 2;
  uint32_t voff[NK];
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    const int p = (wave * NK + i) * 1024 + 16 * lane;
    const int row = p >> 8, phys = (p >> 4) & 15;
    const int lc = unswz256(row, phys);
    voff[i] = lc < D / 8 ? row * row_bytes + lc * 16 : kPastEnd;
  }
  const __bf16* const ds_wave = static_cast<const __bf16*>(G.ds) +
      (static_cast<int64_t>(hl) * G.ds_qblocks + (wave_ok ? qb : 0)) * G.ds_stages * (BN * 32);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));
  auto issue = [&](const Stream& s, int st, int buf) {
    const int nv = min(s.left, BN);
    const i32x4 rk = rsrc_of(s.k, static_cast<uint32_t>(nv - 1) * row_bytes + D * 2);
    const uint32_t base = lds0 + buf * STB;
#pragma unroll
    for (int i = 0; i < NK; ++i) dma16(rk, voff[i], __builtin_amdgcn_readfirstlane(base + (wave * NK + i) * 1024));
    if (wave_ok) {
      // the tile's two halves (positions 16 hh + 8 j + e of every slot, j = 0, 1)
      // each hold 32 bytes per slot; slots past the run's end read as zeros
      const __bf16* tile = ds_wave + static_cast<int64_t>(st) * (BN * 32);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const i32x4 rd = rsrc_of(tile + j * (BN * 16), static_cast<uint32_t>(nv) * 32);
#pragma unroll
        for (int i = 0; i < NDS / 2; ++i)
          dma16_nt(rd, i * 1024 + 16 * lane,
                   __builtin_amdgcn_readfirstlane(base + KT + wave * DTL + j * (DT / 2 + 128) + i * 1024));
      }
    }
  };
  // all of this wave's transfers but the last stage's
  auto wait_but_one = [&]() {
    if (wave_ok)
      wait_vmcnt<NK + NDS>();
    else
      wait_vmcnt<NK>();
  };
  // Transposing reads: rows R + t_lane (+ 8 for the upper half), R a
  // multiple of 16; K at columns 32 db + t_col (swizzled rows), dS at t_col.
  const int t_lane = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int t_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int k_rd[DB][2], d_rd[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    d_rd[h] = ((t_col >> 3) & 1) * (BN * 16 + 64) + (t_lane + 8 * h) * 16 + (t_col >> 4) * 8 + (t_col & 7);
#pragma unroll
    for (int db = 0; db < DB; ++db) k_rd[db][h] = swz(t_lane + 8 * h, db * 32 + t_col);
  }
  auto tr = [](const __bf16* p0, int o0, int o1) {
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0 + o0));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0 + o1));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto stage = [&](int buf) {
    const __bf16* Ks = reinterpret_cast<const __bf16*>(lds + buf * STB);
    const __bf16* Ds = reinterpret_cast<const __bf16*>(lds + buf * STB + KT + wave * DTL);
#pragma unroll
    for (int rb = 0; rb < BN / 16; ++rb) {
      const bf16x8 dst = tr(Ds + rb * 16 * 16, d_rd[0], d_rd[1]);
#pragma unroll
      for (int db = 0; db < DB; ++db)
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr(Ks + rb * 16 * 128, k_rd[db][0], k_rd[db][1]), dst,
                                                          acc[db], 0, 0, 0);
    }
  };

  Stream ls;
  seek(ls, 0);
  if (nst > 0) issue(ls, 0, 0);
  if (nst > 1) {
    step(ls);
    issue(ls, 1, 1);
    wait_but_one();
  } else {
    wait_vmcnt<0>();
  }
  __syncthreads();
  for (int it = 0; it < nst; ++it) {
    if (it + 2 < nst) {
      step(ls);
      issue(ls, it + 2, (it + 2) % 3);
    }
    if (wave_ok) stage(it % 3);
    if (it + 2 < nst)
      wait_but_one();
    else
      wait_vmcnt<0>();
    __syncthreads();
  }

  if (wave_ok && q_row < G.q_end) {
    __bf16* op = static_cast<__bf16*>(a.dq) + static_cast<int64_t>(q_row) * ld + hoff + 4 * hh;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        bf16x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = static_cast<__bf16>(acc[db][4 * jj + i] * a.scale);
        *reinterpret_cast<bf16x4*>(op + db * 32 + 8 * jj) = v;
      }
  }
}

// ------------------------------------------------------------------ bf16: dK, dV

// dK/dV: a block owns 128 context keys, four pairs of waves of 32 keys each;
// the waves of a pair share a SIMD.  Wave A (waves 0-3) holds the keys' K
// fragment and dV accumulator, wave B (waves 4-7) their V fragment and dK
// accumulator.  Queries stream in 64-query stages t, each taking two phases
// separated by block barriers, in which one wave of the pair runs MFMAs while
// the other runs VALU work:
//   phase 2t:     A  dV^T += dO_{t-1}^T P_{t-1}, then S_t = Q_t K^T
//                 B  dS_{t-1} = P_{t-1} (dP_{t-1} - rowsum_{t-1})
//   phase 2t + 1: A  P_t = exp2(S_t c - lse_t), to registers and to LDS for B
//                 B  dK^T += Q_{t-1}^T dS_{t-1}, then dP_t = dO_t V^T
// Stage t's Q, dO and row statistics live in LDS buffer t % 4 and are read
// in phases 2t .. 2t + 3.  A issues stage t + 2 (direct transfers, the
// statistics included) at the start of its VALU phase 2t + 1 into buffer
// (t + 2) % 4, whose stage t - 2 was last read in phase 2t - 1, and waits
// for stage t + 1 at the end of that phase (the transfer instructions cost
// less there than at the end of the matrix-core phase: -2 %).  B also stores dS_{t-1}
// to HBM in phase 2t and never waits for memory: a wave's wait for its
// transfers would also wait for its earlier stores to complete.  P_t is
// written in phase 2t + 1 and read in 2t + 2; one block per pair suffices.
// The matrix-core step is one code site for both roles, so that the register
// allocation holds one set of accumulators, S/dP and P/dS registers.  Its row
// product starts from an accumulator loaded with the stage's negated row
// statistics (-lse / scale for A, -rowsum for B), so that S arrives as
// S - lse / scale (P = exp2(c S'); kQS, queries pre-scaled: c = 1 and
// P = exp2(S')) and dP as dP - rowsum (dS = P dP').
template <int D, bool kQS>
__global__ __launch_bounds__(kBwdKVThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void dkdv_kernel(BwdArgs a) {
  using L = Lay<D>;
  constexpr int KS = L::KS, DB = L::DB;
  constexpr int BQ = kBwdQS, NQB = BQ / 32;             // queries per stage, 32-query blocks
  constexpr int QT = BQ * 128 * 2;                      // bytes of one swizzled tile (256-byte rows)
  constexpr int STB = 2 * QT + 8 * BQ;                  // Q | dO | -lse / scale | -rowsum (fp32)
  constexpr int NDMA = 2 * QT / 1024 / 4;               // 1 KB transfers per B wave and stage (Q and dO)
  constexpr int PXB = NQB * 2 * 64 * 16;                // bytes of one pair's P block
  constexpr int kLead = 4;                              // LDS operands read ahead of their MFMA
  static_assert(NDMA * 1024 * 4 == 2 * QT && BQ % 32 == 0, "stage shape");
  constexpr int NBUF = 4;                               // stage buffers
  __shared__ __attribute__((aligned(16))) char lds[NBUF * STB + 4 * PXB];

  int n_blocks = 0;
  for (int g = 0; g < a.n_groups; ++g) n_blocks += a.groups[g].n_kblocks * a.num_heads;
  const int b = xcd_remap(blockIdx.x, n_blocks);
  int g = 0;
  while (g + 1 < a.n_groups && b >= a.groups[g + 1].kv_block_begin) ++g;
  const BwdGroupArgs& G = a.groups[g];
  const int idx = b - G.kv_block_begin;
  const int hl = idx / G.n_kblocks, kt = idx % G.n_kblocks;  // head of the launch
  const int head = a.head0 + hl;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pair = wave & 3, role = wave >> 2;  // role 0 (A): S, P, dV; role 1 (B): dP, dS, dK
  const int n = lane & 31, hh = lane >> 5;
  const int key = kt * kBwdK + pair * 32 + n;
  const bool k_ok = key < G.n_kv;
  const int64_t ld = a.ld, hoff = static_cast<int64_t>(head) * D;
  const float c = a.scale_log2e;

  // Where B stores its key's dS: byte offset, in the tiles of a 32-query
  // block, of the key's 64-key stage (its run's stages, as the dQ kernel
  // walks them), slot and the lane's 8 queries of each tile half (16 hh,
  // 16 hh + 8 .. of the row's 32 positions); the same offset every stage.
  // Keys past the context point past the range: the range check drops
  // their stores, so the store needs no branch.
  uint32_t ds_voff = kPastEnd;
  if (role != 0 && k_ok) {
    int j = key, st = 0, r = 0;
    while (r + 1 < G.n_runs && j >= G.runs[r].n_tok) {
      st += (G.runs[r].n_tok + kBwdKS - 1) / kBwdKS;
      j -= G.runs[r].n_tok;
      ++r;
    }
    ds_voff = static_cast<uint32_t>((st + j / kBwdKS) * (kBwdKS * 64) + (j % kBwdKS) * 32 + 16 * hh);
  }
  const uint32_t ds_qbytes = static_cast<uint32_t>(G.ds_stages) * (kBwdKS * 64);  // one 32-query block's tiles
  const __bf16* const ds_head =
      static_cast<const __bf16*>(G.ds) + static_cast<int64_t>(hl) * G.ds_qblocks * G.ds_stages * (kBwdKS * 32);

  // B operand of the wave's row product: this lane's key (K for A, V for B),
  // 8 channels of its half-wave per k step.
  bf16x8 xf[KS];
  {
    const __bf16* xp = ctx_row<__bf16>(G, key, role != 0, ld);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      xf[ks] = xp ? *reinterpret_cast<const bf16x8*>(xp + hoff + hh * 8 + ks * 16) : bf16x8{};
  }
  // The fragment loads complete before the first transfer: the compiler does
  // not count the transfers, so a later partial wait would leave it a full
  // wait before the first use of the fragment in every stage.
  wait_vmcnt<0>();
  f32x16 acc[DB];  // dV^T (A) or dK^T (B)
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16{};
  f32x16 s[NQB];       // S_t (A) or dP_t (B); zero before the first stage
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) s[qb] = f32x16{};
  bf16x8 w[NQB][2];    // P_t (A) or dS_{t-1} (B), packed as the B operand of the accumulating product
#pragma unroll
  for (int qb = 0; qb < NQB; ++qb) w[qb][0] = w[qb][1] = bf16x8{};

  // Per-lane global offsets of the A waves' transfers (the same every
  // stage): transfer t = wave NDMA + i covers bytes 1024 (t % (QT / 1024))
  // of the Q tile (t < QT / 1024) or of the dO tile; logical chunk of the
  // fixed LDS slot, zero past D.
  const uint32_t row_bytes = static_cast<uint32_t>(ld) * 2;
  uint32_t voff[NDMA];
#pragma unroll
  for (int i = 0; i < NDMA; ++i) {
    const int t = (wave & 3) * NDMA + i;
    const int p = (t % (QT / 1024)) * 1024 + 16 * lane;
    const int row = p >> 8, phys = (p >> 4) & 15;
    const int lc = unswz256(row, phys);
    voff[i] = lc < D / 8 ? row * row_bytes + lc * 16 : kPastEnd;
  }
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));
  // Stage queries [q0, q0 + BQ) into LDS buffer buf (A waves), all by
  // direct transfers: the Q (waves 0, 1) or dO (waves 2, 3) tile rows, and
  // the stage's negated statistics -lse / scale (wave 0) and -rowsum (wave
  // 1), one dword per lane.  Queries past the end arrive as zero rows with
  // zero statistics: their P = exp2(0) = 1 meets zero dO rows (no dV
  // contribution) and dS = 1 (0 - 0) = 0.  Loop-invariant values are kept in registers.
  static_assert(2 * NDMA * 1024 == QT && BQ == 64, "two A waves per tile, one statistic per lane");
  const int q_begin = G.q_begin, q_end = G.q_end;
  const __bf16* const x_head = static_cast<const __bf16*>((wave & 3) < 2 ? a.q : a.d_out) + hoff;
  const bool stat_wave = wave == 0 || wave == 1;
  const float* const s_head = (wave == 0 ? a.lse2 : a.dsum) + static_cast<int64_t>(head) * a.n_q;
  auto issue = [&](int q0, int buf) {
    const int nv = min(BQ, q_end - q0);
    const uint32_t bytes = static_cast<uint32_t>(nv - 1) * row_bytes + D * 2;
    const i32x4 rs = rsrc_of(x_head + static_cast<int64_t>(q0) * ld, bytes);
    const uint32_t base = lds0 + buf * STB;
#pragma unroll
    for (int i = 0; i < NDMA; ++i)
      dma16(rs, voff[i], __builtin_amdgcn_readfirstlane(base + ((wave & 3) * NDMA + i) * 1024));
    if (stat_wave)
      dma4(rsrc_of(s_head + q0, static_cast<uint32_t>(nv) * 4), 4 * lane,
           __builtin_amdgcn_readfirstlane(base + 2 * QT + wave * BQ * 4));
  };
  // Operand offsets in the swizzled tiles (elements), as in the dQ kernel.
  const int r_rd = swz(n, hh * 8);
  const int t_lane = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int t_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int t_rd[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int h = 0; h < 2; ++h) t_rd[db][h] = swz(t_lane + 8 * h, db * 32 + t_col);
  bf16x8* const pex = reinterpret_cast<bf16x8*>(lds + NBUF * STB + pair * PXB) + lane;
  auto tile = [&](int buf, int which) {  // 0: Q, 1: dO
    return reinterpret_cast<const __bf16*>(lds + buf * STB + which * QT);
  };

  // Matrix-core step of a phase: the accumulating product of the previous
  // stage (if acc_c: A^T rows of Ys, the wave's w as B operand), then the row
  // product of the current stage (if row_c: rows of Xs times the wave's
  // fragment, starting from the statistics at Cs), as one stream of MFMAs
  // whose LDS operands run kLead ahead.
  auto mstep = [&](auto acc_c, auto row_c, const __bf16* Ys, const __bf16* Xs, const float* Cs) {
    constexpr bool kA = decltype(acc_c)::value, kR = decltype(row_c)::value;
    constexpr int NA = kA ? NQB * 2 * DB : 0;  // (32-row block, 16-row half, column block)
    constexpr int NR = kR ? NQB * KS : 0;      // (32-row block, k step)
    constexpr int N = NA + NR;
    if constexpr (kR) {
#pragma unroll
      for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 c4 = *reinterpret_cast<const f32x4*>(Cs + qb * 32 + 8 * j + 4 * hh);
#pragma unroll
          for (int i = 0; i < 4; ++i) s[qb][4 * j + i] = c4[i];
        }
    }
    auto operand = [&](int i) -> bf16x8 {
      if (i < NA) {
        const int qb = i / (2 * DB), cc = (i / DB) & 1, db = i % DB;
        const __bf16* r0 = Ys + (qb * 32 + cc * 16) * 128;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(r0 + t_rd[db][0]));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(r0 + t_rd[db][1]));
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
      const int j = i - NA, qb = j / KS, ks = j % KS;
      return *reinterpret_cast<const bf16x8*>(Xs + qb * 32 * 128 + (r_rd ^ (ks * 16)));
    };
    bf16x8 ring[kLead];
#pragma unroll
    for (int i = 0; i < kLead; ++i)
      if (i < N) ring[i] = operand(i);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const bf16x8 av = ring[i % kLead];
      if (i < NA) {
        const int qb = i / (2 * DB), cc = (i / DB) & 1, db = i % DB;
        acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, w[qb][cc], acc[db], 0, 0, 0);
      } else {
        const int j = i - NA, qb = j / KS, ks = j % KS;
        s[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, xf[ks], s[qb], 0, 0, 0);
      }
      if (i + kLead < N) ring[i % kLead] = operand(i + kLead);
    }
    auto read_group = [&](int i) {  // an A^T operand is two LDS reads, a row operand one
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (i < NA) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    };
    if (kR) __builtin_amdgcn_sched_group_barrier(0x100, 4 * NQB, 0);  // the statistics
#pragma unroll
    for (int i = 0; i < (N < kLead ? N : kLead); ++i) read_group(i);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i + kLead < N) read_group(i + kLead);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Element e of a 32x32 accumulator in this layout holds query
  // qb*32 + 8(e/4) + 4hh + e%4 of the lane's key.
  // A: P_t = exp2(S'_t c) (S' = S - lse / scale) into w and into the pair's
  // LDS block.
  auto softmax_a = [&]() {
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        w[qb][e >> 3][e & 7] = static_cast<__bf16>(__builtin_amdgcn_exp2f(kQS ? s[qb][e] : s[qb][e] * c));
      pex[(qb * 2) * 64] = w[qb][0];
      pex[(qb * 2 + 1) * 64] = w[qb][1];
    }
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
      for (int h = 0; h < 2; ++h) asm volatile("" : "+v"(w[qb][h]));
  };
  // B: dS = P dP' (dP' = dP - rowsum) of stage ts into w, and to the dS
  // tiles of the stage's 32-query blocks 2 ts + qb for the dQ kernel.  Stage
  // -1 (the first phase) computes exact zeros from the zeroed P block and
  // dP registers, and its buffer range is empty, so nothing is stored.
  auto softmax_b = [&](int ts) {
    const i32x4 rd = rsrc_of(ds_head + static_cast<int64_t>(NQB * max(ts, 0)) * G.ds_stages * (kBwdKS * 32),
                             ts >= 0 ? NQB * ds_qbytes : 0u);
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb) {
      const bf16x8 p0 = pex[(qb * 2) * 64], p1 = pex[(qb * 2 + 1) * 64];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = static_cast<float>((e < 8 ? p0 : p1)[e & 7]);
        w[qb][e >> 3][e & 7] = static_cast<__bf16>(p * s[qb][e]);
      }
      bstore16_nt<0>(__builtin_bit_cast(i32x4, w[qb][0]), rd, ds_voff, qb * ds_qbytes);
      bstore16_nt<kBwdKS * 32>(__builtin_bit_cast(i32x4, w[qb][1]), rd, ds_voff, qb * ds_qbytes);
    }
#pragma unroll
    for (int qb = 0; qb < NQB; ++qb)
#pragma unroll
      for (int h = 0; h < 2; ++h) asm volatile("" : "+v"(w[qb][h]));
  };

  // One matrix-core step for every stage and both roles (one instantiation
  // keeps the register allocation tight): in the first stage the
  // accumulating product multiplies the zeroed buffer of stage -1 by w = 0,
  // adding exact zeros; in the stage after the last, the row product's
  // result is never used.  A issues stage t + 2 at the start of its VALU
  // phase 2t + 1, into the buffer of stage t - 2 (last read in phase 2t - 1),
  // and ends that phase once stage t + 1 has arrived.
  using T_ = std::true_type;
  const int nst = (q_end - q_begin + BQ - 1) / BQ;
  {
    bf16x8* z = reinterpret_cast<bf16x8*>(lds + (NBUF - 1) * STB);
#pragma unroll
    for (int i = 0; i < 2 * QT / 16 / kBwdKVThreads; ++i) z[tid + i * kBwdKVThreads] = bf16x8{};
    bf16x8* zp = reinterpret_cast<bf16x8*>(lds + NBUF * STB);  // the P exchange blocks
    static_assert(4 * PXB % (16 * kBwdKVThreads) == 0, "P blocks zeroed whole");
#pragma unroll
    for (int i = 0; i < 4 * PXB / 16 / kBwdKVThreads; ++i) zp[tid + i * kBwdKVThreads] = bf16x8{};
  }
  // this wave's transfers of one stage (the stage issued last may stay in flight)
  auto wait_all_but_last = [&]() {
    if (stat_wave)
      wait_vmcnt<NDMA + 1>();
    else
      wait_vmcnt<NDMA>();
  };
  if (role == 0) {
    issue(q_begin, 0);
    if (nst > 1) {
      issue(q_begin + BQ, 1);
      wait_all_but_last();
    } else {
      wait_vmcnt<0>();
    }
  }
  __syncthreads();
  // Phase ph = 2t + r: role r runs the matrix-core step of stage t, the
  // other role its VALU work.
  for (int ph = 0; ph < 2 * nst + 2; ++ph) {
    const int t = ph >> 1, cur = t % NBUF, prev = (t + NBUF - 1) % NBUF;  // buffers of stages t, t - 1
    if ((ph & 1) == role) {
      __builtin_amdgcn_s_setprio(2);
      mstep(T_{}, T_{}, tile(prev, 1 - role), tile(cur, role),
            reinterpret_cast<const float*>(lds + cur * STB + 2 * QT) + role * BQ);
      __builtin_amdgcn_s_setprio(0);
    } else if (role == 0) {
      if (t + 2 < nst) issue(q_begin + (t + 2) * BQ, (t + 2) % NBUF);
      if (t < nst) softmax_a();
      if (t + 2 < nst)
        wait_all_but_last();
      else
        wait_vmcnt<0>();
    } else {
      softmax_b(t - 1);
    }
    __syncthreads();
  }

  if (k_ok) {
    float* dst = role == 0 ? G.dv_ctx : G.dk_ctx;
    const float sc = role == 0 ? 1.f : a.scale;
    const int64_t off = static_cast<int64_t>(key) * ld + hoff + 4 * hh;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        f32x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = acc[db][4 * jj + i] * sc;
        *reinterpret_cast<f32x4*>(dst + off + db * 32 + 8 * jj) = v;
      }
  }
}

// ------------------------------------------------------------------ fp32 path

template <int D>
__global__ __launch_bounds__(kBwdF32) void dq_f32_kernel(BwdArgs a) {
  int g = 0;
  while (g + 1 < a.n_groups && static_cast<int>(blockIdx.x) >= a.groups[g + 1].dq_block_begin) ++g;
  const BwdGroupArgs& G = a.groups[g];
  const int idx = blockIdx.x - G.dq_block_begin;
  const int head = idx / G.n_qblocks, qt = idx % G.n_qblocks;
  const int q_row = G.q_begin + qt * kBwdF32 + threadIdx.x;
  if (q_row >= G.q_end) return;
  const int64_t ld = a.ld, hoff = static_cast<int64_t>(head) * D;
  const float* qp = static_cast<const float*>(a.q) + static_cast<int64_t>(q_row) * ld + hoff;
  const float* gp = static_cast<const float*>(a.d_out) + static_cast<int64_t>(q_row) * ld + hoff;
  const int64_t stat = static_cast<int64_t>(head) * a.n_q + q_row;
  const float lse = a.lse[stat], dsum = -a.dsum[stat];
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;
  for (int j = 0; j < G.n_kv; ++j) {
    const float* kp = ctx_row<float>(G, j, false, ld) + hoff;
    const float* vp = ctx_row<float>(G, j, true, ld) + hoff;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      s = __builtin_fmaf(qp[d], kp[d], s);
      dp = __builtin_fmaf(gp[d], vp[d], dp);
    }
    const float ds = expf(s * a.scale - lse) * (dp - dsum);
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] = __builtin_fmaf(ds, kp[d], acc[d]);
  }
  float* op = static_cast<float*>(a.dq) + static_cast<int64_t>(q_row) * ld + hoff;
#pragma unroll
  for (int d = 0; d < D; ++d) op[d] = acc[d] * a.scale;
}

template <int D>
__global__ __launch_bounds__(kBwdF32) void dkdv_f32_kernel(BwdArgs a) {
  int g = 0;
  while (g + 1 < a.n_groups && static_cast<int>(blockIdx.x) >= a.groups[g + 1].kv_block_begin) ++g;
  const BwdGroupArgs& G = a.groups[g];
  const int idx = blockIdx.x - G.kv_block_begin;
  const int head = idx / G.n_kblocks, kt = idx % G.n_kblocks;
  const int key = kt * kBwdF32 + threadIdx.x;
  if (key >= G.n_kv) return;
  const int64_t ld = a.ld, hoff = static_cast<int64_t>(head) * D;
  const float* kp = ctx_row<float>(G, key, false, ld) + hoff;
  const float* vp = ctx_row<float>(G, key, true, ld) + hoff;
  float dk[D], dv[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    dk[d] = 0.f;
    dv[d] = 0.f;
  }
  for (int q = G.q_begin; q < G.q_end; ++q) {
    const float* qp = static_cast<const float*>(a.q) + static_cast<int64_t>(q) * ld + hoff;
    const float* gp = static_cast<const float*>(a.d_out) + static_cast<int64_t>(q) * ld + hoff;
    const int64_t stat = static_cast<int64_t>(head) * a.n_q + q;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      s = __builtin_fmaf(qp[d], kp[d], s);
      dp = __builtin_fmaf(gp[d], vp[d], dp);
    }
    const float p = expf(s * a.scale - a.lse[stat]);
    const float ds = p * (dp + a.dsum[stat]);
#pragma unroll
    for (int d = 0; d < D; ++d) {
      dv[d] = __builtin_fmaf(p, gp[d], dv[d]);
      dk[d] = __builtin_fmaf(ds, qp[d], dk[d]);
    }
  }
  float* dkp = G.dk_ctx + static_cast<int64_t>(key) * ld + hoff;
  float* dvp = G.dv_ctx + static_cast<int64_t>(key) * ld + hoff;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    dkp[d] = dk[d] * a.scale;
    dvp[d] = dv[d];
  }
}

// ------------------------------------------------------------------ scatter to the sources

// One thread per 16-byte output chunk of a source token; it adds, in group
// order, the context gradient of the row each group made from this token.
template <typename T>
__global__ __launch_bounds__(kPoolThreads) void scatter_kernel(ScatterArgs a) {
  constexpr int N = 16 / sizeof(T);
  typedef T vecT __attribute__((ext_vector_type(N)));
  const int b = blockIdx.x;
  int jn = 0;
  while (jn + 1 < a.n_jobs && b >= a.jobs[jn + 1].block_begin) ++jn;
  const ScatterJobArgs& J = a.jobs[jn];
  const int64_t cpt = a.chunks_per_tok;
  const int64_t ftok = static_cast<int64_t>(J.gh) * J.gw;
  const int64_t idx = static_cast<int64_t>(b - J.block_begin) * kPoolThreads + threadIdx.x;
  if (idx >= J.n_frames * ftok * cpt) return;
  const int64_t chunk = idx % cpt;
  const int64_t t = idx / cpt;
  const int x = static_cast<int>(t % J.gw);
  const int y = static_cast<int>((t / J.gw) % J.gh);
  const int64_t fr = t / ftok;
  const bool is_v = blockIdx.y != 0;
  float acc[N];
#pragma unroll
  for (int e = 0; e < N; ++e) acc[e] = 0.f;
  for (int g = 0; g < a.n_groups; ++g) {
    const ScatterGroupArgs& S = J.g[g];
    const int f = S.factor;
    if (a.pick_first && f > 1 && ((y % f) != 0 || (x % f) != 0)) continue;
    const int Y = y / f, X = x / f;
    const int ow = (J.gw + f - 1) / f;
    const float cnt = a.pick_first ? 1.f : static_cast<float>(min(f, J.gh - f * Y) * min(f, J.gw - f * X));
    const float* src = (is_v ? a.ctx_v[g] : a.ctx_k[g]) +
                       (S.ctx_begin + fr * S.frame_stride + static_cast<int64_t>(Y) * ow + X) * a.ld + chunk * N;
#pragma unroll
    for (int e = 0; e < N; e += 4) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(src + e);
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[e + i] += v[i] / cnt;
    }
  }
  vecT o;
#pragma unroll
  for (int e = 0; e < N; ++e) o[e] = static_cast<T>(acc[e]);
  T* dst = static_cast<T*>(is_v ? J.dst_v : J.dst_k);
  *reinterpret_cast<vecT*>(dst + (fr * ftok + static_cast<int64_t>(y) * J.gw + x) * a.ld + chunk * N) = o;
}

}  // namespace

hipError_t launch_bwd_dot(const DotArgs& a, bool bf16, hipStream_t stream) {
  const int64_t rows = static_cast<int64_t>(a.n_q) * a.num_heads;
  if (rows == 0) return hipSuccess;
  if (a.ld != static_cast<int64_t>(a.num_heads) * a.head_dim) return hipErrorInvalidValue;
  const int64_t threads = rows * (a.head_dim * (bf16 ? 2 : 4) / 16);
  if ((threads + kDotThreads - 1) / kDotThreads > 0x7fffffff) return hipErrorInvalidValue;
  const int blocks = static_cast<int>((threads + kDotThreads - 1) / kDotThreads);
  if (bf16)
    hipLaunchKernelGGL(dot_kernel<__bf16>, dim3(blocks), dim3(kDotThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(dot_kernel<float>, dim3(blocks), dim3(kDotThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdArgs& a, int dq_blocks, int kv_blocks, int head_dim, bool bf16,
                      hipStream_t stream) {
  // dK/dV first: for bf16 plans it writes the dS tiles the dQ kernel reads.
  if (kv_blocks > 0) {
    if (bf16) {
      if (head_dim == 128 && a.q_prescaled)
        hipLaunchKernelGGL((dkdv_kernel<128, true>), dim3(kv_blocks), dim3(kBwdKVThreads), 0, stream, a);
      else if (head_dim == 128)
        hipLaunchKernelGGL((dkdv_kernel<128, false>), dim3(kv_blocks), dim3(kBwdKVThreads), 0, stream, a);
      else if (a.q_prescaled)
        hipLaunchKernelGGL((dkdv_kernel<64, true>), dim3(kv_blocks), dim3(kBwdKVThreads), 0, stream, a);
      else
        hipLaunchKernelGGL((dkdv_kernel<64, false>), dim3(kv_blocks), dim3(kBwdKVThreads), 0, stream, a);
    } else {
      if (head_dim == 128)
        hipLaunchKernelGGL(dkdv_f32_kernel<128>, dim3(kv_blocks), dim3(kBwdF32), 0, stream, a);
      else
        hipLaunchKernelGGL(dkdv_f32_kernel<64>, dim3(kv_blocks), dim3(kBwdF32), 0, stream, a);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (dq_blocks > 0) {
    if (bf16) {
      if (head_dim == 128)
        hipLaunchKernelGGL(dq_kernel<128>, dim3(dq_blocks), dim3(kBwdQThreads), 0, stream, a);
      else
        hipLaunchKernelGGL(dq_kernel<64>, dim3(dq_blocks), dim3(kBwdQThreads), 0, stream, a);
    } else {
      if (head_dim == 128)
        hipLaunchKernelGGL(dq_f32_kernel<128>, dim3(dq_blocks), dim3(kBwdF32), 0, stream, a);
      else
        hipLaunchKernelGGL(dq_f32_kernel<64>, dim3(dq_blocks), dim3(kBwdF32), 0, stream, a);
    }
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t launch_scatter(const ScatterArgs& a, int n_blocks, bool bf16, hipStream_t stream) {
  if (n_blocks <= 0) return hipSuccess;
  const dim3 grid(n_blocks, 2), block(kPoolThreads);
  if (bf16)
    hipLaunchKernelGGL(scatter_kernel<__bf16>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(scatter_kernel<float>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace mssa
