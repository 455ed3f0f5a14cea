// Multi-Scale Patchification tiers (Ms. Forcing, Sec. 4.1): the steps on
// either side of the attention.  Window state l is tokenized with patch
// p * p_l by its tier's own patch embedding, a strided 2-D convolution
// (each patch of every latent channel, flattened in (channel, row, column)
// order, times the tier's weights, plus bias); the de-embedding maps tokens
// back to pixels; the attention's q, k, v are one linear projection of the
// tokens.  Patches past a ragged frame edge see zeros; de-embedded pixels
// past it are dropped.
//
// Kernels:
//   patchify_kernel    latent [frames, C, H, W] -> the patch rows of one
//                      query group [tokens, C*P*P] (HBM-bound gather);
//   gemm_kernel        Y[M, N] = X[M, K] W[N, K]^T + b on the matrix cores
//                      (bf16 in, fp32 accumulation, bf16 out), 128 x 128
//                      tiles in 32-deep stages double-buffered in LDS; the
//                      output columns may be split over up to three tensors
//                      (q | k | v); gemm_dma_kernel is the same product for
//                      K a multiple of 64 with 64-deep stages filled by
//                      direct global -> LDS transfers; gemm256_kernel the
//                      same in 256 x 256 tiles (K a multiple of 64, at least
//                      256 rows and features);
//   unpatchify_kernel  patch rows [tokens, C*P*P] -> latent pixels.
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "lds_stage.hpp"

namespace mssa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// One thread per 8-feature chunk of one patch row: feature k = (c, dy, dx) of
// patch (Y, X) of frame f reads pixel (c, Y*P + dy, X*P + dx), zero past the
// frame's edge.
__global__ __launch_bounds__(kTierThreads) void patchify_kernel(PatchArgs a) {
  const int kp = a.C * a.P * a.P;
  const int cpr = kp / 8;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kTierThreads + threadIdx.x;
  const int64_t gtok = static_cast<int64_t>(a.gh) * a.gw;
  if (idx >= a.n_frames * gtok * cpr) return;
  const int chunk = static_cast<int>(idx % cpr);
  const int64_t t = idx / cpr;
  const int X = static_cast<int>(t % a.gw);
  const int Y = static_cast<int>((t / a.gw) % a.gh);
  const int64_t f = t / gtok;
  const __bf16* src = static_cast<const __bf16*>(a.latent) + (a.frame0 + f) * a.C * a.H * a.W;
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int k = chunk * 8 + e;
    const int c = k / (a.P * a.P), r = k % (a.P * a.P);
    const int y = Y * a.P + r / a.P, x = X * a.P + r % a.P;
    v[e] = (y < a.H && x < a.W) ? src[(static_cast<int64_t>(c) * a.H + y) * a.W + x] : static_cast<__bf16>(0.f);
  }
  *reinterpret_cast<bf16x8*>(static_cast<__bf16*>(a.rows) + t * kp + chunk * 8) = v;
}

// One thread per pixel: pixel (c, y, x) of frame f comes from feature
// (c, y % P, x % P) of patch (y / P, x / P).
__global__ __launch_bounds__(kTierThreads) void unpatchify_kernel(PatchArgs a) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kTierThreads + threadIdx.x;
  const int64_t fpix = static_cast<int64_t>(a.C) * a.H * a.W;
  if (idx >= a.n_frames * fpix) return;
  const int x = static_cast<int>(idx % a.W);
  const int y = static_cast<int>((idx / a.W) % a.H);
  const int c = static_cast<int>((idx / (static_cast<int64_t>(a.W) * a.H)) % a.C);
  const int64_t f = idx / fpix;
  const int kp = a.C * a.P * a.P;
  const int64_t tok = (f * a.gh + y / a.P) * a.gw + x / a.P;
  const int k = (c * a.P + y % a.P) * a.P + x % a.P;
  static_cast<__bf16*>(a.latent)[(a.frame0 + f) * fpix + (static_cast<int64_t>(c) * a.H + y) * a.W + x] =
      static_cast<const __bf16*>(a.rows)[tok * kp + k];
}

// Y = X W^T + b.  A block owns a 128 x 128 output tile (128 rows of X, 128
// output features); its 4 waves own 64 x 64 quarters as 2 x 2 matrix-core
// tiles.  The MFMA computes the transposed tile (A = W rows, B = X rows) so
// that a lane holds one output row and 16 features in runs of 4 (8-byte
// stores).  K advances in 32-deep stages; the next stage's global loads are
// in flight during the current stage's MFMAs.  Rows and features past the
// matrix edges load as zeros and are not stored.
constexpr int kGM = kGemmTile, kGN = kGemmTile, kGK = 32, kGStr = kGK + 8;  // LDS row stride: conflict-free 16-byte reads

__global__ __launch_bounds__(kTierThreads) void gemm_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) __bf16 lds[2][2][kGM * kGStr];  // [stage][X | W]
  const int tiles_m = (a.M + kGM - 1) / kGM;
  const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int n32 = lane & 31, hh = lane >> 5;
  const __bf16* X = static_cast<const __bf16*>(a.x);
  const __bf16* W = static_cast<const __bf16*>(a.w);

  // Stage loads: 128 rows x 4 chunks of 16 bytes per matrix, 2 chunks per thread.
  const int lr = tid >> 2, lc = (tid & 3) * 8;
  bf16x8 px[2], pw[2];
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = lr + i * 64;
      const int64_t xm = static_cast<int64_t>(tm) * kGM + r, wn_ = static_cast<int64_t>(tn) * kGN + r;
      const bool kok = k0 + lc < a.K;
      px[i] = (kok && xm < a.M) ? *reinterpret_cast<const bf16x8*>(X + xm * a.ldx + k0 + lc) : bf16x8{};
      pw[i] = (kok && wn_ < a.N) ? *reinterpret_cast<const bf16x8*>(W + wn_ * a.K + k0 + lc) : bf16x8{};
    }
  };
  auto store = [&](int s) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = lr + i * 64;
      *reinterpret_cast<bf16x8*>(&lds[s][0][r * kGStr + lc]) = px[i];
      *reinterpret_cast<bf16x8*>(&lds[s][1][r * kGStr + lc]) = pw[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = f32x16{};

  const int nst = (a.K + kGK - 1) / kGK;
  load(0);
  store(0);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) load((st + 1) * kGK);
    const __bf16* Xs = lds[st & 1][0];
    const __bf16* Ws = lds[st & 1][1];
#pragma unroll
    for (int ks = 0; ks < kGK / 16; ++ks) {
      bf16x8 xb[2], wa[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        xb[j] = *reinterpret_cast<const bf16x8*>(Xs + (wm * 64 + j * 32 + n32) * kGStr + ks * 16 + hh * 8);
        wa[j] = *reinterpret_cast<const bf16x8*>(Ws + (wn * 64 + j * 32 + n32) * kGStr + ks * 16 + hh * 8);
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[cb], xb[rb], acc[rb][cb], 0, 0, 0);
    }
    if (st + 1 < nst) store((st + 1) & 1);
    __syncthreads();
  }

  // acc[rb][cb] element e: row (wm*64 + rb*32 + n32), feature
  // (wn*64 + cb*32 + 8(e/4) + 4hh + e%4) of the tile.
  const __bf16* B = static_cast<const __bf16*>(a.bias);
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int64_t row = static_cast<int64_t>(tm) * kGM + wm * 64 + rb * 32 + n32;
    if (row >= a.M) continue;
#pragma unroll
    for (int cb = 0; cb < 2; ++cb)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int col = tn * kGN + wn * 64 + cb * 32 + 8 * jj + 4 * hh;
        if (col >= a.N) continue;
        const int part = col / a.split, pc = col % a.split;  // 4 features never straddle a split (split % 4 == 0)
        const float sc = part == 0 ? a.y0_scale : 1.f;
        bf16x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          v[i] = static_cast<__bf16>((acc[rb][cb][4 * jj + i] + static_cast<float>(B[col + i])) * sc);
        *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(a.y[part]) + row * a.ldy + pc) = v;
      }
  }
}

// The same product for K a multiple of 64: 64-deep stages of 128-byte rows in
// the swizzled layout of lds_stage.hpp, filled by direct global -> LDS
// transfers (no staging registers), 64 KB of LDS so that two blocks share a
// CU (two waves per SIMD); 16 MFMAs per wave between barriers.
constexpr int kG2K = kGemmStage, kG2Tile = kGM * kG2K * 2;  // bytes of one 128 x 64 operand tile

__global__ __launch_bounds__(kTierThreads, 2) void gemm_dma_kernel(GemmArgs a) {
  constexpr int NDMA = kG2Tile / 1024 / (kTierThreads / 64);
  static_assert(NDMA * 1024 * (kTierThreads / 64) == kG2Tile, "tile must split into 1 KB transfers per wave");
  __shared__ __attribute__((aligned(16))) char lds[2][2][kG2Tile];  // [stage][X | W]
  const int tiles_m = (a.M + kGM - 1) / kGM, tiles = tiles_m * ((a.N + kGN - 1) / kGN);
  // k_splits > 1: block b takes K slice b / tiles of output tile b % tiles
  const int ks_n = a.k_splits > 1 ? a.k_splits : 1;
  const int tile = blockIdx.x % tiles, slice = blockIdx.x / tiles;
  const int tm = tile % tiles_m, tn = tile / tiles_m;
  const int k_len = a.K / ks_n, k_begin = slice * k_len;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int n32 = lane & 31, hh = lane >> 5;

  // Per-lane offsets of this wave's transfers inside a stage (row p / 128 of
  // the tile, logical chunk of the physical slot): the same for every stage
  // of both operands up to the row stride.
  const uint32_t xrb = static_cast<uint32_t>(a.ldx) * 2, wrb = static_cast<uint32_t>(a.K) * 2;
  uint32_t xo[NDMA], wo[NDMA];
#pragma unroll
  for (int i = 0; i < NDMA; ++i) {
    const int p = (wave * NDMA + i) * 1024 + 16 * lane;
    const int row = p >> 7, lc = unswz128(row, (p >> 4) & 7);
    xo[i] = row * xrb + lc * 16;
    wo[i] = row * wrb + lc * 16;
  }
  const int mrows = min(kGM, a.M - tm * kGM), nrows = min(kGN, a.N - tn * kGN);
  const __bf16* X = static_cast<const __bf16*>(a.x) + static_cast<int64_t>(tm) * kGM * a.ldx + k_begin;
  const __bf16* W = static_cast<const __bf16*>(a.w) + static_cast<int64_t>(tn) * kGN * a.K + k_begin;
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&lds[0][0][0]));
  auto issue = [&](int k0, int s) {
    // rows past the matrix edge fall past the range: zeros
    const i32x4 rx = rsrc_of(X + k0, static_cast<uint32_t>(mrows - 1) * xrb + kG2K * 2);
    const i32x4 rw = rsrc_of(W + k0, static_cast<uint32_t>(nrows - 1) * wrb + kG2K * 2);
    const uint32_t base = lds0 + s * 2 * kG2Tile;
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const uint32_t dst = __builtin_amdgcn_readfirstlane(base + (wave * NDMA + i) * 1024);
      dma16(rx, xo[i], dst);
      dma16(rw, wo[i], dst + kG2Tile);
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = f32x16{};

  const int nst = k_len / kG2K;
  issue(0, 0);
  wait_vmcnt<0>();
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) issue((st + 1) * kG2K, (st + 1) & 1);
    const __bf16* Xs = reinterpret_cast<const __bf16*>(lds[st & 1][0]);
    const __bf16* Ws = reinterpret_cast<const __bf16*>(lds[st & 1][1]);
#pragma unroll
    for (int ks = 0; ks < kG2K / 16; ++ks) {
      bf16x8 xb[2], wa[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        xb[j] = *reinterpret_cast<const bf16x8*>(Xs + swz128(wm * 64 + j * 32 + n32, ks * 16 + hh * 8));
        wa[j] = *reinterpret_cast<const bf16x8*>(Ws + swz128(wn * 64 + j * 32 + n32, ks * 16 + hh * 8));
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb)
          acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa[cb], xb[rb], acc[rb][cb], 0, 0, 0);
    }
    wait_vmcnt<0>();
    __syncthreads();
  }

  if (ks_n > 1) {
    // A K slice's fp32 partial tile, in the lanes' own order: each store of a
    // wave is 1 KB contiguous.  gemm_reduce_kernel sums the slices.
    f32x4* P = reinterpret_cast<f32x4*>(a.partial) + ((static_cast<int64_t>(slice) * tiles + tile) * 4 + wave) * 1024 + lane;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int cb = 0; cb < 2; ++cb)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          f32x4 v;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = acc[rb][cb][4 * jj + i];
          P[((rb * 2 + cb) * 4 + jj) * 64] = v;
        }
    return;
  }
  // Epilogue through LDS (the stage buffers are free after the last barrier):
  // each wave writes its outputs plus bias, rounded to bf16, into a
  // row-major 128 x 128 tile (rows padded to 272 bytes: the 8-byte writes of
  // 16 consecutive rows hit distinct banks), then every thread stores 16-byte
  // pieces of whole rows, 16 threads per 256-byte row, coalesced.
  constexpr int kEStr = kGN + 8;
  static_assert(kGM * kEStr * 2 <= 2 * 2 * kG2Tile, "epilogue tile fits the stage buffers");
  __bf16* E = reinterpret_cast<__bf16*>(&lds[0][0][0]);
  const __bf16* B = static_cast<const __bf16*>(a.bias);
#pragma unroll
  for (int cb = 0; cb < 2; ++cb)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int ct = wn * 64 + cb * 32 + 8 * jj + 4 * hh;
      const int col = tn * kGN + ct;
      const bf16x4 bv = col < a.N ? *reinterpret_cast<const bf16x4*>(B + col) : bf16x4{};
      const float sc = col < a.split ? a.y0_scale : 1.f;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        bf16x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          v[i] = static_cast<__bf16>((acc[rb][cb][4 * jj + i] + static_cast<float>(bv[i])) * sc);
        *reinterpret_cast<bf16x4*>(E + (wm * 64 + rb * 32 + n32) * kEStr + ct) = v;
      }
    }
  __syncthreads();
#pragma unroll
  for (int p = 0; p < kGM * kGN / 8 / kTierThreads; ++p) {
    const int c = p * kTierThreads + tid, rt = c / (kGN / 8), ch = c % (kGN / 8);
    const int64_t row = static_cast<int64_t>(tm) * kGM + rt;
    const int col = tn * kGN + ch * 8;
    if (row < a.M && col < a.N) {
      const int part = col / a.split, pc = col % a.split;  // 8 features never straddle a split (split % 8 == 0)
      *reinterpret_cast<bf16x8*>(static_cast<__bf16*>(a.y[part]) + row * a.ldy + pc) =
          *reinterpret_cast<const bf16x8*>(E + rt * kEStr + ch * 8);
    }
  }
}

// Sum of the K slices' partial tiles of gemm_dma_kernel, slice 0 first, plus
// the bias, rounded to bf16: one thread per 4 output features of one row,
// reading the partials in the order they were written (coalesced).
__global__ __launch_bounds__(kTierThreads) void gemm_reduce_kernel(GemmArgs a) {
  const int tiles_m = (a.M + kGM - 1) / kGM, tiles = tiles_m * ((a.N + kGN - 1) / kGN);
  const int64_t u = static_cast<int64_t>(blockIdx.x) * kTierThreads + threadIdx.x;
  const int64_t per_slice = static_cast<int64_t>(tiles) * 4 * 1024;
  if (u >= per_slice) return;
  const int lane = static_cast<int>(u % 64), jj = static_cast<int>((u / 64) % 4), cb = static_cast<int>((u / 256) % 2);
  const int rb = static_cast<int>((u / 512) % 2), wave = static_cast<int>((u / 1024) % 4);
  const int tile = static_cast<int>(u / 4096);
  const int tm = tile % tiles_m, tn = tile / tiles_m;
  const int wm = wave & 1, wn = wave >> 1, n32 = lane & 31, hh = lane >> 5;
  const int64_t row = static_cast<int64_t>(tm) * kGM + wm * 64 + rb * 32 + n32;
  const int col = tn * kGN + wn * 64 + cb * 32 + 8 * jj + 4 * hh;
  if (row >= a.M || col >= a.N) return;
  const f32x4* P = reinterpret_cast<const f32x4*>(a.partial) + u;
  f32x4 s = P[0];
  for (int k = 1; k < a.k_splits; ++k) s += P[k * per_slice];
  const __bf16* B = static_cast<const __bf16*>(a.bias) + col;
  const int part = col / a.split, pc = col % a.split;
  const float sc = part == 0 ? a.y0_scale : 1.f;
  bf16x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = static_cast<__bf16>((s[i] + static_cast<float>(B[i])) * sc);
  *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(a.y[part]) + row * a.ldy + pc) = v;
}

// The same product for K a multiple of 64 and at least 256 rows and output
// features, in 256 x 256 output tiles: the operand bytes each tile streams
// from L2 per multiply-add are half those of a 128 x 128 tile.  A block of 8
// waves (two per SIMD) owns the tile; wave w owns rows 128 (w & 1) .. +127
// and features 64 (w >> 1) .. +63 as 4 x 2 matrix-core tiles (A = W rows,
// B = X rows).  K streams in 64-deep stages of 128-byte rows (whole cache
// lines; the swizzle of lds_stage.hpp's 128-byte rows) through two LDS
// buffers, each stage filled by direct global -> LDS transfers issued while
// the previous one is multiplied; one barrier per stage.  Tiles are taken in
// panels of four feature tiles, each XCD a contiguous run of them, so that
// the blocks of an XCD share operand rows in its L2.  The outputs leave
// through LDS as whole-row 16-byte stores, as in gemm_dma_kernel.
constexpr int kBM = 256, kBN = 256, kBK = 64, kBStages = 2, kBThreads = 512, kBPanel = 4;
constexpr int kBTile = kBM * kBK * 2;  // bytes of one operand tile of a stage

// kScale: y[0]'s outputs multiplied by y0_scale (an instance of its own, so
// that the unscaled product keeps its register allocation).
template <bool kScale>
__global__ __launch_bounds__(kBThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm256_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[kBStages][2][kBTile];  // [stage][X | W]
  const int tiles_m = (a.M + kBM - 1) / kBM, tiles_n = (a.N + kBN - 1) / kBN, T = tiles_m * tiles_n;
  // blockIdx -> tile: blocks are dispatched round-robin over the 8 XCDs
  const int b = blockIdx.x, q8 = T / 8, r8 = T % 8, x8 = b % 8, j8 = b / 8;
  const int t = (x8 < r8 ? x8 * (q8 + 1) : r8 * (q8 + 1) + (x8 - r8) * q8) + j8;
  const int panel = t / (tiles_m * kBPanel), pw = min(kBPanel, tiles_n - panel * kBPanel);
  const int ip = t - panel * tiles_m * kBPanel;
  const int tm = ip / pw, tn = panel * kBPanel + ip % pw;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int n32 = lane & 31, hh = lane >> 5;

  // This wave's transfers of a stage: 1 KB (8 rows of 128 bytes) each, rows
  // 8 (4 wave + i) + lane / 8, physical chunk lane % 8 holding logical chunk
  // unswz128(row, lane % 8).  Rows past the matrix edge fall past the range:
  // zeros.
  const uint32_t xrb = static_cast<uint32_t>(a.ldx) * 2, wrb = static_cast<uint32_t>(a.K) * 2;
  uint32_t xo[4], wo[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = (wave * 4 + i) * 8 + (lane >> 3), lc = unswz128(row, lane & 7);
    xo[i] = row * xrb + lc * 16;
    wo[i] = row * wrb + lc * 16;
  }
  const int mrows = min(kBM, a.M - tm * kBM), nrows = min(kBN, a.N - tn * kBN);
  const __bf16* X = static_cast<const __bf16*>(a.x) + static_cast<int64_t>(tm) * kBM * a.ldx;
  const __bf16* W = static_cast<const __bf16*>(a.w) + static_cast<int64_t>(tn) * kBN * a.K;
  const uint32_t xbytes = static_cast<uint32_t>(mrows - 1) * xrb + kBK * 2;
  const uint32_t wbytes = static_cast<uint32_t>(nrows - 1) * wrb + kBK * 2;
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&lds[0][0][0]));
  auto issue = [&](int st) {
    const i32x4 rx = rsrc_of(X + st * kBK, xbytes), rw = rsrc_of(W + st * kBK, wbytes);
    const uint32_t base = lds0 + (st % kBStages) * 2 * kBTile + wave * 4096;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dma16(rx, xo[i], __builtin_amdgcn_readfirstlane(base + i * 1024));
      dma16(rw, wo[i], __builtin_amdgcn_readfirstlane(base + kBTile + i * 1024));
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = f32x16{};

  // The bias of this lane's 32 output features, loaded before the loop.
  bf16x4 bias[2][4];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int col = tn * kBN + wn * 64 + nb * 32 + 8 * jj + 4 * hh;
      bias[nb][jj] = col < a.N ? *reinterpret_cast<const bf16x4*>(static_cast<const __bf16*>(a.bias) + col) : bf16x4{};
    }

  // Operand reads: row (block base + n32), columns 16 ks + 8 hh; the swizzle
  // of a row depends only on n32 (block bases are multiples of 32).
  int rd[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) rd[ks] = (swz128(n32, ks * 16 + hh * 8)) * 2;

  const int nst = a.K / kBK;
  issue(0);
  for (int st = 0; st < nst; ++st) {
    wait_vmcnt<0>();
    __syncthreads();
    if (st + 1 < nst) issue(st + 1);
    const char* Xs = lds[st % kBStages][0];
    const char* Ws = lds[st % kBStages][1];
    // Operands of k step ks in register set ks & 1: the reads of step ks + 1
    // run between the MFMAs of step ks.
    bf16x8 op[2][6];  // [set][W nb 0..1, X mb 0..3]
    auto rd_op = [&](int ks, int j) -> bf16x8 {
      return j < 2 ? *reinterpret_cast<const bf16x8*>(Ws + (wn * 64 + j * 32) * 128 + rd[ks])
                   : *reinterpret_cast<const bf16x8*>(Xs + (wm * 128 + (j - 2) * 32) * 128 + rd[ks]);
    };
#pragma unroll
    for (int j = 0; j < 6; ++j) op[0][j] = rd_op(0, j);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int c = ks & 1;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int mb = i >> 1, nb = i & 1;
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[c][nb], op[c][2 + mb], acc[mb][nb], 0, 0, 0);
        if (ks + 1 < kBK / 16 && i < 6) op[c ^ 1][i] = rd_op(ks + 1, i);
      }
    }
#pragma unroll
    for (int j = 0; j < 6; ++j) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (ks + 1 < kBK / 16 && i < 6) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    __builtin_amdgcn_sched_barrier(0);
  }

  // Epilogue through LDS in two halves of 128 rows (a padded 128 x 256 bf16
  // half tile is 67.6 KB of the 128 KB of stage buffers): the waves owning
  // the half write their outputs plus bias, then all threads store whole-row
  // 16-byte pieces, 32 threads per 512-byte row.
  constexpr int kEStr = kBN + 8;
  static_assert(128 * kEStr * 2 <= static_cast<int>(sizeof(lds)), "half tile fits the stage buffers");
  __bf16* E = reinterpret_cast<__bf16*>(&lds[0][0][0]);
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    __syncthreads();  // the stage buffers (half 0) or the previous half are free
    if (wm == half) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            bf16x4 v;
            if constexpr (kScale) {
              // y0_scale for the features of y[0], else 1
              const float sc = tn * kBN + wn * 64 + nb * 32 + 8 * jj + 4 * hh < a.split ? a.y0_scale : 1.f;
#pragma unroll
              for (int i = 0; i < 4; ++i)
                v[i] = static_cast<__bf16>((acc[mb][nb][4 * jj + i] + static_cast<float>(bias[nb][jj][i])) * sc);
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i)
                v[i] = static_cast<__bf16>(acc[mb][nb][4 * jj + i] + static_cast<float>(bias[nb][jj][i]));
            }
            *reinterpret_cast<bf16x4*>(E + (mb * 32 + n32) * kEStr + wn * 64 + nb * 32 + 8 * jj + 4 * hh) = v;
          }
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < 128 * kBN / 8 / kBThreads; ++p) {
      const int c = p * kBThreads + tid, rt = c / (kBN / 8), ch = c % (kBN / 8);
      const int64_t row = static_cast<int64_t>(tm) * kBM + half * 128 + rt;
      const int col = tn * kBN + ch * 8;
      if (row < a.M && col < a.N) {
        const int part = col / a.split, pc = col % a.split;  // 8 features never straddle a split (split % 8 == 0)
        *reinterpret_cast<bf16x8*>(static_cast<__bf16*>(a.y[part]) + row * a.ldy + pc) =
            *reinterpret_cast<const bf16x8*>(E + rt * kEStr + ch * 8);
      }
    }
  }
}

}  // namespace

hipError_t launch_patchify(const PatchArgs& a, hipStream_t stream) {
  const int64_t work = a.n_frames * a.gh * a.gw * (a.C * a.P * a.P / 8);
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(patchify_kernel, dim3(static_cast<uint32_t>((work + kTierThreads - 1) / kTierThreads)),
                     dim3(kTierThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_unpatchify(const PatchArgs& a, hipStream_t stream) {
  const int64_t work = a.n_frames * a.C * a.H * a.W;
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(unpatchify_kernel, dim3(static_cast<uint32_t>((work + kTierThreads - 1) / kTierThreads)),
                     dim3(kTierThreads), 0, stream, a);
  return hipGetLastError();
}

namespace {

// gemm_dma_kernel stores 16-byte pieces of output rows and reads the bias in
// 8-byte pieces.
bool dma_epilogue_ok(const GemmArgs& a) {
  bool ok = a.K % kG2K == 0 && a.N % 8 == 0 && a.split % 8 == 0 && a.ldy % 8 == 0 &&
            (reinterpret_cast<uintptr_t>(a.bias) & 7) == 0;
  for (int i = 0; i < 3; ++i) ok = ok && (reinterpret_cast<uintptr_t>(a.y[i]) & 15) == 0;
  return ok;
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, hipStream_t stream) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  const int64_t tiles = static_cast<int64_t>((a.M + kBM - 1) / kBM) * ((a.N + kBN - 1) / kBN);
  // enough tiles to fill the CUs; the bias read in 8-byte pieces
  if (a.K % kBK == 0 && a.N >= kBN && a.M >= kBM && tiles >= 256 && dma_epilogue_ok(a)) {
    if (a.y0_scale != 1.f)
      hipLaunchKernelGGL(gemm256_kernel<true>, dim3(static_cast<uint32_t>(tiles)), dim3(kBThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(gemm256_kernel<false>, dim3(static_cast<uint32_t>(tiles)), dim3(kBThreads), 0, stream, a);
    return hipGetLastError();
  }
  const int64_t blocks = static_cast<int64_t>((a.M + kGM - 1) / kGM) * ((a.N + kGN - 1) / kGN);
  if (dma_epilogue_ok(a)) {
    GemmArgs b = a;
    b.k_splits = 1;
    hipLaunchKernelGGL(gemm_dma_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTierThreads), 0, stream, b);
  } else {
    hipLaunchKernelGGL(gemm_kernel, dim3(static_cast<uint32_t>(blocks)), dim3(kTierThreads), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_split(const GemmArgs& a, float* partial, hipStream_t stream) {
  const int s = gemm_k_splits(a.M, a.N, a.K);
  if (s <= 1 || !partial || !dma_epilogue_ok(a)) return launch_gemm(a, stream);
  GemmArgs b = a;
  b.partial = partial;
  b.k_splits = s;
  const int64_t tiles = static_cast<int64_t>((a.M + kGM - 1) / kGM) * ((a.N + kGN - 1) / kGN);
  hipLaunchKernelGGL(gemm_dma_kernel, dim3(static_cast<uint32_t>(tiles * s)), dim3(kTierThreads), 0, stream, b);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t units = tiles * 4 * 1024;
  hipLaunchKernelGGL(gemm_reduce_kernel, dim3(static_cast<uint32_t>((units + kTierThreads - 1) / kTierThreads)),
                     dim3(kTierThreads), 0, stream, b);
  return hipGetLastError();
}

}  // namespace mssa
