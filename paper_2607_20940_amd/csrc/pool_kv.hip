// K/V resampling for MSSA (Ms. Forcing, Sec. 4.1, Eq. 4 "Subsample", read
// as a 2-D average pool; Sec. 3.2 uses the 2 x 2 block mean as the coarse
// token).  Each output cell averages the cells of its f x f block that exist
// on the source frame's grid, per head and channel, for K and V alike.  The
// strided variant (Eq. 4 read literally; the stride-2 probe of Sec. 3.2)
// copies the block's first cell instead: the same loop over a 1 x 1 block,
// whose sum divided by 1 is the source value exactly.
//
// HBM-bound: every source byte is read once and every pooled byte written
// once (frames pooled both by 2 and by 4 are read once for both).  One thread
// produces one 16-byte chunk of one pooled token (of the coarser level when
// two are fused); consecutive threads cover consecutive chunks of a token, so
// a wave reads and writes whole contiguous token rows (heads * head_dim
// elements) and every access is a coalesced 128-bit load or store.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace mssa {
namespace {

template <typename T>
struct Vec;
template <>
struct Vec<__bf16> {
  static constexpr int N = 8;  // elements per 16-byte chunk
};
template <>
struct Vec<float> {
  static constexpr int N = 4;
};

// One 16-byte chunk of one output cell pooled by a compile-time factor F from
// an F x F source block (all F * F loads issued before any is summed; cells
// past a ragged edge are skipped).  With kTwo the cell is one of the coarser
// level (factor F = 2 f, f = F / 2) and the four f x f quadrants of the block
// are also written as the cells of the finer level that exist: the same
// source bytes serve both levels, read once.
template <typename T, int F, bool kTwo>
__device__ __forceinline__ void pool_cell(const PoolArgs& a, const PoolJobArgs& J, int64_t idx, bool is_v) {
  constexpr int N = Vec<T>::N, H = F / 2;
  typedef T vecT __attribute__((ext_vector_type(N)));
  const int64_t cpt = a.chunks_per_tok;
  const int gh = kTwo ? J.dst2_gh : J.dst_gh, gw = kTwo ? J.dst2_gw : J.dst_gw;
  const int64_t chunk = idx % cpt;
  const int64_t t = idx / cpt;
  const int X = static_cast<int>(t % gw);
  const int64_t t2 = t / gw;
  const int Y = static_cast<int>(t2 % gh);
  const int64_t fr = t2 / gh;
  const T* src = static_cast<const T*>(is_v ? J.src_v : J.src_k);
  const int rows = min(F, J.src_gh - F * Y), cols = min(F, J.src_gw - F * X);
  const T* base = src + (fr * J.src_gh * J.src_gw + static_cast<int64_t>(F * Y) * J.src_gw + F * X) * a.ld + chunk * N;
  vecT v[F][F];
#pragma unroll
  for (int dy = 0; dy < F; ++dy)
#pragma unroll
    for (int dx = 0; dx < F; ++dx)
      v[dy][dx] = dy < rows && dx < cols
                      ? *reinterpret_cast<const vecT*>(base + (static_cast<int64_t>(dy) * J.src_gw + dx) * a.ld)
                      : vecT{};
  if constexpr (!kTwo) {
    float acc[N];
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = 0.f;
#pragma unroll
    for (int dy = 0; dy < F; ++dy)
#pragma unroll
      for (int dx = 0; dx < F; ++dx)
#pragma unroll
        for (int e = 0; e < N; ++e) acc[e] += static_cast<float>(v[dy][dx][e]);
    const float cnt = static_cast<float>(rows * cols);
    vecT o;
#pragma unroll
    for (int e = 0; e < N; ++e) o[e] = static_cast<T>(acc[e] / cnt);
    T* dst = static_cast<T*>(is_v ? J.dst_v : J.dst_k);
    *reinterpret_cast<vecT*>(dst + (fr * gh * gw + static_cast<int64_t>(Y) * gw + X) * a.ld + chunk * N) = o;
  } else {
    T* dst = static_cast<T*>(is_v ? J.dst_v : J.dst_k);
    T* dst2 = static_cast<T*>(is_v ? J.dst2_v : J.dst2_k);
    float tot[N];
#pragma unroll
    for (int e = 0; e < N; ++e) tot[e] = 0.f;
#pragma unroll
    for (int qa = 0; qa < 2; ++qa)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        float acc[N];
#pragma unroll
        for (int e = 0; e < N; ++e) acc[e] = 0.f;
#pragma unroll
        for (int dy = 0; dy < H; ++dy)
#pragma unroll
          for (int dx = 0; dx < H; ++dx)
#pragma unroll
            for (int e = 0; e < N; ++e) acc[e] += static_cast<float>(v[qa * H + dy][qb * H + dx][e]);
#pragma unroll
        for (int e = 0; e < N; ++e) tot[e] += acc[e];
        // the finer cell exists iff its first source row and column do
        if (qa * H < rows && qb * H < cols) {
          const float cnt = static_cast<float>(min(H, rows - qa * H) * min(H, cols - qb * H));
          vecT o;
#pragma unroll
          for (int e = 0; e < N; ++e) o[e] = static_cast<T>(acc[e] / cnt);
          const int64_t cell = (fr * J.dst_gh + 2 * Y + qa) * J.dst_gw + 2 * X + qb;
          *reinterpret_cast<vecT*>(dst + cell * a.ld + chunk * N) = o;
        }
      }
    const float cnt = static_cast<float>(rows * cols);
    vecT o;
#pragma unroll
    for (int e = 0; e < N; ++e) o[e] = static_cast<T>(tot[e] / cnt);
    *reinterpret_cast<vecT*>(dst2 + (fr * gh * gw + static_cast<int64_t>(Y) * gw + X) * a.ld + chunk * N) = o;
  }
}

// Any factor (a runtime loop), and the strided variant.
template <typename T>
__device__ __forceinline__ void pool_cell_any(const PoolArgs& a, const PoolJobArgs& J, int64_t idx, bool is_v) {
  constexpr int N = Vec<T>::N;
  typedef T vecT __attribute__((ext_vector_type(N)));
  const int64_t cpt = a.chunks_per_tok;
  const int64_t dst_tok = static_cast<int64_t>(J.dst_gh) * J.dst_gw;
  const int64_t chunk = idx % cpt;
  const int64_t t = idx / cpt;
  const int X = static_cast<int>(t % J.dst_gw);
  const int64_t t2 = t / J.dst_gw;
  const int Y = static_cast<int>(t2 % J.dst_gh);
  const int64_t fr = t2 / J.dst_gh;

  const T* src = static_cast<const T*>(is_v ? J.src_v : J.src_k);
  T* dst = static_cast<T*>(is_v ? J.dst_v : J.dst_k);
  const int f = J.factor;
  const int rows = a.pick_first ? 1 : min(f, J.src_gh - f * Y);
  const int cols = a.pick_first ? 1 : min(f, J.src_gw - f * X);
  const T* base = src + (fr * J.src_gh * J.src_gw + static_cast<int64_t>(f * Y) * J.src_gw + f * X) * a.ld +
                  chunk * N;
  float acc[N];
#pragma unroll
  for (int e = 0; e < N; ++e) acc[e] = 0.f;
  for (int dy = 0; dy < rows; ++dy) {
    const T* row = base + static_cast<int64_t>(dy) * J.src_gw * a.ld;
    for (int dx = 0; dx < cols; ++dx) {
      const vecT v = *reinterpret_cast<const vecT*>(row + dx * a.ld);
#pragma unroll
      for (int e = 0; e < N; ++e) acc[e] += static_cast<float>(v[e]);
    }
  }
  const float cnt = static_cast<float>(rows * cols);
  vecT o;
#pragma unroll
  for (int e = 0; e < N; ++e) o[e] = static_cast<T>(acc[e] / cnt);
  *reinterpret_cast<vecT*>(dst + (fr * dst_tok + static_cast<int64_t>(Y) * J.dst_gw + X) * a.ld + chunk * N) = o;
}

// Blocks of consecutive output chunks of one job; y = 0 pools K, y = 1 pools V.
template <typename T>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(PoolArgs a) {
  const int b = blockIdx.x;
  int j = 0;
  while (j + 1 < a.n_jobs && b >= a.jobs[j + 1].block_begin) ++j;
  const PoolJobArgs& J = a.jobs[j];
  const int gh = J.levels == 2 ? J.dst2_gh : J.dst_gh, gw = J.levels == 2 ? J.dst2_gw : J.dst_gw;
  const int64_t total = J.n_frames * static_cast<int64_t>(gh) * gw * a.chunks_per_tok;
  const int64_t idx = static_cast<int64_t>(b - J.block_begin) * kPoolThreads + threadIdx.x;
  if (idx >= total) return;
  const bool is_v = blockIdx.y != 0;
  if (J.levels == 2) {
    pool_cell<T, 4, true>(a, J, idx, is_v);  // factors 2 and 4 (the only fused pair)
  } else if (!a.pick_first && J.factor == 2) {
    pool_cell<T, 2, false>(a, J, idx, is_v);
  } else if (!a.pick_first && J.factor == 4) {
    pool_cell<T, 4, false>(a, J, idx, is_v);
  } else {
    pool_cell_any<T>(a, J, idx, is_v);
  }
}

}  // namespace

hipError_t launch_pool(const PoolArgs& a, int n_blocks, bool bf16, hipStream_t stream) {
  if (n_blocks <= 0) return hipSuccess;
  const dim3 grid(n_blocks, 2), block(kPoolThreads);
  if (bf16)
    hipLaunchKernelGGL(pool_kernel<__bf16>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(pool_kernel<float>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace mssa
