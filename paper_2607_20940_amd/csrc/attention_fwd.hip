// Multi-scale self-attention forward (Ms. Forcing, Sec. 4.1, Eq. 4): for
// every head and query scale, softmax(scale q k^T) v over the concatenated
// context runs of that scale (sink | history at the query scale | window at
// max(query scale, own scale)).
//
// bf16 path (gfx950 matrix cores).  One block = 4 waves = 128 queries of one
// (query scale, head); each wave owns 32 queries.  The block walks the
// scale's runs in 64-key tiles staged through LDS.  Per tile and wave:
//   S^T = K Q^T   with v_mfma_f32_32x32x16_bf16 (A = K rows from LDS,
//                 B = the wave's Q fragment held in registers), so each lane
//                 holds 16 keys of ONE query: the softmax row reductions are
//                 in-lane plus one exchange between the two half-waves;
//   online softmax in fp32 in the exp2 domain (scale * log2 e folded into
//                 one FMA per score);
//   O^T += V^T P^T with the same MFMA: the exponentiated scores are already
//                 laid out as the B operand (their key order defines the
//                 contraction order), and V^T comes from row-major V in LDS
//                 through the gfx950 transposing LDS read ds_read_b64_tr_b16.
// Keys past the end of a run are zero-filled in LDS and masked to -inf.
//
// fp32 path: one lane per query, plain fp32 FMA dot products and an online
// softmax with expf; used for fp32 plans (correctness path).
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.hpp"

namespace mssa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

__device__ constexpr bf16x2 kOnes2 = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};

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

// Buffer resource (gfx9 layout) over `bytes` bytes from `base`: loads past
// the end return zeros, which is how ragged K/V tiles are zero-filled without
// per-element selects.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

template <int D>
__global__ __launch_bounds__(kFwdThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void fwd_bf16_kernel(FwdArgs a) {
  constexpr int BM = kFwdBM, BN = kFwdBN;
  constexpr int KS = D / 16;    // 16-wide k-steps of q k^T
  constexpr int DB = D / 32;    // 32-row blocks of O^T
  constexpr int CPR = D / 8;    // 16-byte chunks per K/V row
  constexpr int RPL = kFwdThreads / CPR;  // rows covered by one pass of the block
  constexpr int KSTR = D + 8;   // K row stride: 16 consecutive rows hit disjoint banks (b128 reads)
  constexpr int VSTR = D + 32;  // V row stride: the 4x16 transposing reads of 32 lanes hit disjoint banks
  constexpr int NLD = BN / RPL; // 16-byte chunks per thread per tile and tensor
  constexpr int KT = BN * KSTR, VT = BN * VSTR;  // elements per LDS tile
  static_assert(NLD * RPL == BN, "tile load must divide evenly");
  // [K buf0 | K buf1 | V buf0 | V buf1]; every offset fits a ds instruction's immediate.
  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * KT + 2 * VT];

  const Work w = decode(a, blockIdx.x);
  const FwdGroupArgs& G = a.groups[w.g];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;   // query column of this lane
  const int hh = lane >> 5;  // half-wave
  const int q_row = G.q_begin + w.tile * BM + wave * 32 + n;
  const bool q_ok = q_row < G.q_end;
  const int64_t ld = a.ld;
  const int64_t hoff = static_cast<int64_t>(w.head) * D;
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

  // Per-thread constants of the tile copy: global byte offset inside a tile
  // and LDS element offset of chunk 0 (chunk i adds i * RPL rows).
  const int ld_row = tid / CPR, ld_col = (tid % CPR) * 8;
  const uint32_t g_off = ld_row * row_bytes + ld_col * 2;
  const int k_st = ld_row * KSTR + ld_col;
  const int v_st = ld_row * VSTR + ld_col;
  // Transposing-read offset of this lane inside a 16-key slab of V.
  const int gq = lane >> 4;
  const int v_rd = (4 * (gq >> 1) + ((lane & 15) >> 2)) * VSTR + 16 * (gq & 1) + 4 * (lane & 3);
  const int k_rd = n * KSTR + hh * 8;

  bf16x8 pk[NLD], pv[NLD];
  // Issue the loads of the tile starting at token t0 of run r (zero past the run's end).
  auto issue = [&](int r, int t0) {
    const int nv = min(G.runs[r].n_tok - t0, BN);
    const uint32_t bytes = static_cast<uint32_t>(nv - 1) * row_bytes + D * 2;
    const int64_t base = static_cast<int64_t>(t0) * ld + hoff;
    const auto rk = make_rsrc(static_cast<const __bf16*>(G.runs[r].k) + base, bytes);
    const auto rv = make_rsrc(static_cast<const __bf16*>(G.runs[r].v) + base, bytes);
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const uint32_t off = g_off + i * RPL * row_bytes;
      pk[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0));
      pv[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, 0));
    }
  };
  auto commit = [&](auto bufc) {
    constexpr int buf = decltype(bufc)::value;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      *reinterpret_cast<bf16x8*>(&lds[buf * KT + k_st + i * RPL * KSTR]) = pk[i];
      *reinterpret_cast<bf16x8*>(&lds[2 * KT + buf * VT + v_st + i * RPL * VSTR]) = pv[i];
    }
  };

  // One 64-key tile from LDS buffer `buf`: S^T = K Q^T, online softmax, O^T += V^T P^T.
  auto compute = [&](auto bufc, int nvalid) {
    constexpr int buf = decltype(bufc)::value;
    const __bf16* Kb = lds + buf * KT;
    const __bf16* Vb = lds + 2 * KT + buf * VT;
    f32x16 s[BN / 32];
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb) {
      const bf16x8 ka0 = *reinterpret_cast<const bf16x8*>(Kb + k_rd + kb * 32 * KSTR);
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka0, qf[0], f32x16{}, 0, 0, 0);
#pragma unroll
      for (int ks = 1; ks < KS; ++ks) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(Kb + k_rd + kb * 32 * KSTR + ks * 16);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[ks], s[kb], 0, 0, 0);
      }
    }
    if (nvalid < BN) {
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kb * 32 + 8 * (e >> 2) + 4 * hh + (e & 3);
          if (key >= nvalid) s[kb][e] = -INFINITY;
        }
    }
    float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
    for (int e = 2; e < 16; e += 2) mx = fmaxf(fmaxf(mx, s[0][e]), s[0][e + 1]);
#pragma unroll
    for (int kb = 1; kb < BN / 32; ++kb)
#pragma unroll
      for (int e = 0; e < 16; e += 2) mx = fmaxf(fmaxf(mx, s[kb][e]), s[kb][e + 1]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mt = mx * c;
    if (__any(mt > m_run + kRescaleLog2)) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= alpha;
    }
    const float mneg = -m_run;
    bf16x8 pb[BN / 32][2];
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
      for (int e = 0; e < 16; e += 2) {
        bf16x2 pair;
        pair[0] = static_cast<__bf16>(__builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][e], c, mneg)));
        pair[1] = static_cast<__bf16>(__builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][e + 1], c, mneg)));
        l_part = __builtin_amdgcn_fdot2_f32_bf16(pair, kOnes2, l_part, false);
        pb[kb][e >> 3][e & 7] = pair[0];
        pb[kb][e >> 3][(e & 7) + 1] = pair[1];
      }
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
      for (int cc = 0; cc < 2; ++cc) {
        const __bf16* vrow = Vb + v_rd + (kb * 32 + cc * 16) * VSTR;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vrow + db * 32));
          const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vrow + 8 * VSTR + db * 32));
          const bf16x8 va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kb][cc], o[db], 0, 0, 0);
        }
      }
  };

  // Walk the runs tile by tile; the loop body is unrolled over the two LDS
  // buffers so that every LDS address is a per-thread constant plus an
  // immediate.
  int r = 0, t0 = 0;
  while (r < G.n_runs && G.runs[r].n_tok == 0) ++r;
  auto advance = [&](int& rr, int& tt) {
    tt += BN;
    if (tt >= G.runs[rr].n_tok) {
      tt = 0;
      ++rr;
      while (rr < G.n_runs && G.runs[rr].n_tok == 0) ++rr;
    }
  };
  if (r < G.n_runs) {
    issue(r, 0);
    commit(std::integral_constant<int, 0>{});
  }
  __syncthreads();
  auto step = [&](auto bufc) -> bool {
    constexpr int buf = decltype(bufc)::value;
    const int nvalid = min(BN, G.runs[r].n_tok - t0);
    int rn = r, tn = t0;
    advance(rn, tn);
    const bool has_next = rn < G.n_runs;
    if (has_next) issue(rn, tn);
    compute(bufc, nvalid);
    if (has_next) commit(std::integral_constant<int, buf ^ 1>{});
    __syncthreads();
    r = rn;
    t0 = tn;
    return has_next;
  };
  if (r < G.n_runs) {
    while (step(std::integral_constant<int, 0>{}) && step(std::integral_constant<int, 1>{})) {
    }
  }

  const float l_tot = l_part + __shfl_xor(l_part, 32);
  const float inv = 1.0f / l_tot;
  if (q_ok) {
    __bf16* op = static_cast<__bf16*>(a.out) + static_cast<int64_t>(q_row) * ld + hoff + 4 * hh;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        bf16x4 v;
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = static_cast<__bf16>(o[db][4 * j + i] * inv);
        *reinterpret_cast<bf16x4*>(op + db * 32 + 8 * j) = v;
      }
  }
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
}

}  // namespace

hipError_t launch_forward(const FwdArgs& a, int head_dim, bool bf16, hipStream_t stream) {
  if (a.n_blocks <= 0) return hipSuccess;
  if (bf16) {
    if (head_dim == 128)
      hipLaunchKernelGGL(fwd_bf16_kernel<128>, dim3(a.n_blocks), dim3(kFwdThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(fwd_bf16_kernel<64>, dim3(a.n_blocks), dim3(kFwdThreads), 0, stream, a);
  } else {
    if (head_dim == 128)
      hipLaunchKernelGGL(fwd_f32_kernel<128>, dim3(a.n_blocks), dim3(kFwdF32BM), 0, stream, a);
    else
      hipLaunchKernelGGL(fwd_f32_kernel<64>, dim3(a.n_blocks), dim3(kFwdF32BM), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace mssa
