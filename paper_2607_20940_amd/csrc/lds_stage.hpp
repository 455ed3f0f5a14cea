// Device helpers for LDS stages filled by direct global -> LDS transfers and
// read through XOR-swizzled rows (gfx950), and the half-wave exchange of the
// attention kernels.  Included by the HIP kernels only.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace mssa {

typedef int i32x4 __attribute__((ext_vector_type(4)));

// 256-byte rows (128 bf16): 16-byte chunk c of row r is stored at chunk
// c ^ f(r & 15), f(r) = ((r & 3) << 2) | (r >> 2).  Sixteen consecutive rows
// read at one column (16-byte row reads: the A operand of a 32x32x16 MFMA)
// hit 16 distinct bank groups, and so do the 4 rows x 4 chunks of a
// ds_read_b64_tr_b16 (the transposed A operand), so one copy serves both.
// Returns the element offset of (row, col).
__device__ inline int swz256(int row, int col) {
  const int r = row & 15;
  return row * 128 + ((((col >> 3) ^ (((r & 3) << 2) | (r >> 2)))) << 3) + (col & 7);
}

// The logical 16-byte chunk stored at physical chunk `phys` of 256-byte row `row`.
__device__ inline int unswz256(int row, int phys) {
  const int r = row & 15;
  return phys ^ (((r & 3) << 2) | (r >> 2));
}

// 128-byte rows (64 bf16), row reads only: chunk c of row r at c ^ ((r >> 1) & 7);
// sixteen consecutive rows read at one column hit distinct bank groups.
__device__ inline int swz128(int row, int col) {
  return row * 64 + ((((col >> 3) ^ ((row >> 1) & 7))) << 3) + (col & 7);
}

__device__ inline int unswz128(int row, int phys) { return phys ^ ((row >> 1) & 7); }

// Direct global -> LDS load (buffer_load_dwordx4 ... lds): lane i's 16 bytes
// at buffer offset voff land at LDS byte address lds_addr + 16 i (lds_addr
// wave-uniform); offsets past the buffer's range write zeros.  Counted by
// vmcnt; issued from inline asm so the compiler does not make every later
// LDS read wait for it (kernels wait before the barrier that publishes the
// stage).  m0 is set here and not used otherwise.
__device__ inline void dma16(i32x4 rsrc, uint32_t voff, uint32_t lds_addr) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(lds_addr), "v"(voff), "s"(rsrc) : "memory", "m0");
#pragma clang diagnostic pop
}

// As dma16 for data read once (nt: streamed past the caches' normal
// retention, so it does not displace operands that are read again).
__device__ inline void dma16_nt(i32x4 rsrc, uint32_t voff, uint32_t lds_addr) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
               :: "s"(lds_addr), "v"(voff), "s"(rsrc) : "memory", "m0");
#pragma clang diagnostic pop
}

// As dma16 for 4 bytes per lane (buffer_load_dword ... lds): lane i's dword
// at buffer offset voff lands at LDS byte address lds_addr + 4 i.
__device__ inline void dma4(i32x4 rsrc, uint32_t voff, uint32_t lds_addr) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :: "s"(lds_addr), "v"(voff), "s"(rsrc) : "memory", "m0");
#pragma clang diagnostic pop
}

// As dma16, with a scalar byte offset soff added to the lane's offset.
__device__ inline void dma16_soff(i32x4 rsrc, uint32_t voff, uint32_t soff, uint32_t lds_addr) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds_addr), "v"(voff), "s"(rsrc), "s"(soff) : "memory", "m0");
#pragma clang diagnostic pop
}

// Store of lane i's 16 bytes at buffer offset voff + soff + IMM
// (buffer_store_dwordx4, non-temporal: data that another kernel reads once);
// lanes whose offset is past the buffer's range store nothing.
template <int IMM>
__device__ inline void bstore16_nt(i32x4 data, i32x4 rsrc, uint32_t voff, uint32_t soff) {
  asm volatile("buffer_store_dwordx4 %0, %1, %2, %3 offen offset:%4 nt"
               :: "v"(data), "v"(voff), "s"(rsrc), "s"(soff), "n"(IMM) : "memory");
}

// s_waitcnt vmcnt(N) alone (gfx9 encoding: expcnt and lgkmcnt at their maxima).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Raw buffer resource (gfx9 layout) over `bytes` bytes from `base`, in SGPRs.
__device__ inline i32x4 rsrc_of(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(static_cast<int>(b & 0xffffffffu));
  r[1] = __builtin_amdgcn_readfirstlane(static_cast<int>((b >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
  r[3] = 0x00020000;
  return r;
}

// Byte offset past any buffer this library builds: a transfer lane pointed
// here writes zeros (no 32-bit wrap of offset + 16).
constexpr uint32_t kPastEnd = 0x7ffffff0u;

// Value of lane l ^ 32.  v_permlane32_swap exchanges the upper half of its
// first operand with the lower half of its second; whether the compiler gives
// the two operands one register or two, lane l < 32 finds lane l + 32 in the
// second result and lane l >= 32 finds lane l - 32 in the first.
__device__ inline float other_half(float v) {
  const int b = __builtin_bit_cast(int, v);
  const auto sw = __builtin_amdgcn_permlane32_swap(b, b, false, false);
  return __builtin_bit_cast(float, (threadIdx.x & 32) ? sw[0] : sw[1]);
}

}  // namespace mssa
