// Device helpers shared by the two dX kernels (tgemm_bwd_dx.hip: two
// bfloat16 passes; tgemm_bwd_dx_f16.hip: one float16 pass): direct-to-LDS
// loads issued from inline assembly, the stage barrier that counts them, and
// the LDS layouts of the dY stage and of the decoded weight plane.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace tmk {

typedef __attribute__((ext_vector_type(4))) short dx_s16x4;
typedef __attribute__((address_space(3))) dx_s16x4 dx_lds_s16x4;
typedef __attribute__((ext_vector_type(2))) short dx_s16x2;

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// lane i: 16 bytes at base + voff -> LDS lds_base + 16 i (lds_base wave-uniform)
__device__ __forceinline__ void dx_dma16(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
// lane i: 4 bytes at base + voff -> LDS lds_base + 4 i
__device__ __forceinline__ void dx_dma4(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int kVm>
__device__ __forceinline__ void dx_stage_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(kVm) : "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <int I, int N, typename F>
__device__ __forceinline__ void dx_static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    dx_static_for<I + 1, N>(f);
  }
}

// byte offset of (weight row r, column c) inside a plane, c % 4 == 0.  The
// 32-byte units of row r are XOR-permuted by f = (r%4) ^ 2 (r%4), which is
// distinct modulo 4 and in its two upper bits over any four consecutive rows:
// the four rows of a transpose read land in distinct 32-byte bank groups, and
// so do the two column groups (units u and u + 1) read in the same cycle.
__device__ __forceinline__ uint32_t dx_poff(int r, int c) {
  const int f = (r & 3) ^ ((r & 3) << 1);
  return (uint32_t)(r * 512 + 32 * ((c >> 4) ^ f) + 2 * (c & 15));
}

// byte offset of 16-byte unit u (columns 8u .. 8u+7) of dY row r in a stage;
// the XOR ((r/2) % 4) ^ ((r/8) % 2) spreads any 8 (and any 16) consecutive
// rows over distinct 16-byte bank groups
__device__ __forceinline__ uint32_t dx_yoff(int r, int u) {
  return (uint32_t)(r * 64 + 16 * (u ^ ((r >> 1) & 3) ^ ((r >> 3) & 1)));
}

// 0xFFFF in each 16-bit half whose bit 15 is set
__device__ __forceinline__ uint32_t dx_halfmask(uint32_t y) {
  const dx_s16x2 v = __builtin_bit_cast(dx_s16x2, y) >> (short)15;
  return __builtin_bit_cast(uint32_t, v);
}

}  // namespace tmk
