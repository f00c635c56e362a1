// LDS-DMA helpers of the bf16 attention kernels (internal, not part of the C ABI): loads that
// travel global -> LDS without registers, their waits and barriers, transposed LDS reads and
// cross-half wave reductions.
#pragma once

#include "attn_common.h"

namespace nexus {

typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ bf16x8 tr_read_pair(const char *lo, const char *hi) {
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)lo);
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)hi);
  const u32x2 ua = __builtin_bit_cast(u32x2, a);
  const u32x2 ub = __builtin_bit_cast(u32x2, b);
  return __builtin_bit_cast(bf16x8, u32x4{ua[0], ua[1], ub[0], ub[1]});
}

// LDS DMA (global_load_lds_dwordx4: each lane's 16 bytes land at M0 + OFF + 16 * lane) issued
// from inline assembly, so that the compiler neither tracks these loads nor inserts its own
// vmcnt waits for them (it cannot tell ring stages apart and would wait for every load in
// flight before each LDS read).  The kernel orders them itself with wait_vm() + tile_barrier().
// The s_nop covers the one wait state an M0 write needs before an LDS DMA.
template <int OFF>
__device__ __forceinline__ void dma_s(uint32_t lds, const char *sbase, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 offset:%3"
               :: "s"(lds), "v"(voff), "s"(sbase), "i"(OFF) : "memory");
}
__device__ __forceinline__ void dma_v(uint32_t lds, const char *src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(lds), "v"(src) : "memory");
}
// s_waitcnt vmcnt(N) with lgkmcnt and expcnt unconstrained (gfx9 encoding: vmcnt[3:0],
// expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] in bits 15:14)
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
// Workgroup barrier ordering LDS only: unlike __syncthreads it does not wait for the LDS DMA
// loads still in flight for later ring stages.
__device__ __forceinline__ void tile_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// max over the two 32-lane halves of the wave (lanes i and i ^ 32), without an LDS round trip
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

}  // namespace nexus
