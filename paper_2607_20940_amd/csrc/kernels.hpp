// Host-side launchers of the MSSA HIP kernels (defined in the .hip files).
#pragma once

#include <hip/hip_runtime_api.h>

#include "kernel_args.hpp"

namespace mssa {

// Average-pool jobs; grid = (n_blocks, 2): y = 0 pools K, y = 1 pools V.
hipError_t launch_pool(const PoolArgs& a, int n_blocks, bool bf16, hipStream_t stream);

// Attention forward over the groups of `a`.  bf16: a.n_ranges persistent
// blocks followed by the combine of split items; fp32: a.n_blocks blocks.
hipError_t launch_forward(const FwdArgs& a, int head_dim, bool bf16, hipStream_t stream);

// Backward: rowsum(d_out * out) per head and query.
hipError_t launch_bwd_dot(const DotArgs& a, bool bf16, hipStream_t stream);

// Backward: dQ kernel (dq_blocks blocks), then dK/dV context gradients
// (kv_blocks blocks).
hipError_t launch_bwd(const BwdArgs& a, int dq_blocks, int kv_blocks, int head_dim, bool bf16,
                      hipStream_t stream);

// Backward: context gradients to the sink, history and window tokens; grid
// (n_blocks, 2): y = 0 for K, y = 1 for V.
hipError_t launch_scatter(const ScatterArgs& a, int n_blocks, bool bf16, hipStream_t stream);

// MSP tiers: patch rows of latent frames, the inverse, and Y = X W^T + b.
hipError_t launch_patchify(const PatchArgs& a, hipStream_t stream);
hipError_t launch_unpatchify(const PatchArgs& a, hipStream_t stream);
hipError_t launch_gemm(const GemmArgs& a, hipStream_t stream);

// The same product with K split over several blocks per output tile when the
// output alone has too few tiles to fill the GPU (narrow outputs with a long
// K, such as the patch de-embedding): fp32 partial tiles into `partial`
// (gemm_split_bytes bytes, 256-byte aligned), then their sum in a fixed order
// plus the bias.  With gemm_split_bytes == 0 this is launch_gemm and partial
// may be null.
// (Host code in plan.cpp: the rule is part of the static launch plan.)
int gemm_k_splits(int32_t M, int32_t N, int32_t K);
int64_t gemm_split_bytes(int32_t M, int32_t N, int32_t K);
hipError_t launch_gemm_split(const GemmArgs& a, float* partial, hipStream_t stream);

// Resident blocks per CU of the bf16 attention kernel (0 if unknown).
int forward_blocks_per_cu(int head_dim);

}  // namespace mssa
