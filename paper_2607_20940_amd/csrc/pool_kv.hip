// K/V resampling for MSSA (Ms. Forcing, Sec. 4.1, Eq. 4 "Subsample", read
// as a 2-D average pool; Sec. 3.2 uses the 2 x 2 block mean as the coarse
// token).  Each output cell averages the cells of its f x f block that exist
// on the source frame's grid, per head and channel, for K and V alike.  The
// strided variant (Eq. 4 read literally; the stride-2 probe of Sec. 3.2)
// copies the block's first cell instead: the same loop over a 1 x 1 block,
// whose sum divided by 1 is the source value exactly.
//
// HBM-bound: every source byte is read once per output scale and every
// pooled byte written once.  One thread produces one 16-byte chunk of one
// pooled token; consecutive threads cover consecutive chunks of a token, so a
// wave reads and writes whole contiguous token rows (heads * head_dim
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

template <typename T>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(PoolArgs a) {
  constexpr int N = Vec<T>::N;
  typedef T vecT __attribute__((ext_vector_type(N)));
  const int b = blockIdx.x;
  int j = 0;
  while (j + 1 < a.n_jobs && b >= a.jobs[j + 1].block_begin) ++j;
  const PoolJobArgs& J = a.jobs[j];
  const int64_t cpt = a.chunks_per_tok;
  const int64_t dst_tok = static_cast<int64_t>(J.dst_gh) * J.dst_gw;
  const int64_t total = J.n_frames * dst_tok * cpt;
  const int64_t idx = static_cast<int64_t>(b - J.block_begin) * kPoolThreads + threadIdx.x;
  if (idx >= total) return;
  const int64_t chunk = idx % cpt;
  const int64_t t = idx / cpt;
  const int X = static_cast<int>(t % J.dst_gw);
  const int64_t t2 = t / J.dst_gw;
  const int Y = static_cast<int>(t2 % J.dst_gh);
  const int64_t fr = t2 / J.dst_gh;

  const T* src = static_cast<const T*>(blockIdx.y == 0 ? J.src_k : J.src_v);
  T* dst = static_cast<T*>(blockIdx.y == 0 ? J.dst_k : J.dst_v);
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
