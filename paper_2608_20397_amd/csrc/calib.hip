// Measurement helpers (not part of the splice path): the ceilings a kernel on this GPU can
// reach, measured on the box so that roofline fractions can be quoted against them as well as
// against the published peaks.
//   * calib_copy_kernel: a plain device copy in 16-byte non-temporal chunks, one workgroup per
//     16 KiB, four loads per thread before their stores (the HBM ceiling of a read + write
//     stream);
//   * calib_mfma_kernel: v_mfma_f32_32x32x16_bf16 back to back on four independent accumulators
//     per wave, two waves per SIMD (the dense bf16 matrix ceiling at the clock the chip holds
//     under that load);
//   * calib_lds_dma_kernel: streams a buffer into LDS with global_load_lds_dwordx4, the load of
//     the attention kernels' K/V tiles, 16 KiB per workgroup and round: the bytes it reads are
//     known, so the memory counters' reading of such loads can be scaled against it.
#include "attn_dma.h"
#include "nexus.h"

namespace nexus {

constexpr int kCopyChunks = 4;   // 16-byte chunks per thread, all loads before the stores

__global__ __launch_bounds__(256) void calib_copy_kernel(const u32x4 *__restrict__ src,
                                                         u32x4 *__restrict__ dst, uint64_t n) {
  const uint64_t i0 = (uint64_t)blockIdx.x * (256 * kCopyChunks) + threadIdx.x;
  u32x4 v[kCopyChunks];
#pragma unroll
  for (int u = 0; u < kCopyChunks; ++u)
    if (i0 + 256 * u < n) v[u] = ld_stream(src + i0 + 256 * u);
#pragma unroll
  for (int u = 0; u < kCopyChunks; ++u)
    if (i0 + 256 * u < n) st_stream(v[u], dst + i0 + 256 * u);
}

constexpr int kCalibChains = 4;

__global__ __launch_bounds__(256) void calib_mfma_kernel(int iters, float *sink) {
  // operands from the thread index, so that nothing folds at compile time
  const float x = (float)(threadIdx.x & 7) * 0.125f;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(x + e);
    b[e] = (__bf16)(x - e);
  }
  f32x16 acc[kCalibChains];
#pragma unroll
  for (int c = 0; c < kCalibChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < kCalibChains; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kCalibChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  // written only for an impossible sum, which the compiler cannot rule out
  if (s == -1.0e30f) sink[blockIdx.x] = s;
}

constexpr uint32_t kDmaChunk = 16384;   // bytes per workgroup and round

__global__ __launch_bounds__(256) void calib_lds_dma_kernel(const char *__restrict__ src,
                                                            uint64_t n_chunks) {
  __shared__ __align__(1024) char buf[kDmaChunk];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const uint32_t dst = (uint32_t)(uintptr_t)buf + wave * 4096;
  const uint32_t voff = (uint32_t)lane * 16;
  for (uint64_t c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    const char *p = src + c * kDmaChunk + wave * 4096;
    dma_s<0>(dst, p, voff);
    dma_s<1024>(dst, p, voff);
    dma_s<2048>(dst, p, voff);
    dma_s<3072>(dst, p, voff);
    wait_vm<0>();
    tile_barrier();   // the buffer is refilled next round
  }
}

}  // namespace nexus

using namespace nexus;

extern "C" {

nexus_status nexus_calib_copy(const void *src, void *dst, size_t bytes, void *stream) {
  if (!src || !dst || bytes == 0 || bytes % 16) return NEXUS_EINVAL;
  if (((uintptr_t)src | (uintptr_t)dst) & 15) return NEXUS_EINVAL;
  const uint64_t n = bytes / 16;
  const uint64_t blocks = (n + 256 * kCopyChunks - 1) / (256 * kCopyChunks);
  if (blocks >= (1ull << 31)) return NEXUS_EINVAL;
  hipLaunchKernelGGL(calib_copy_kernel, dim3((uint32_t)blocks), dim3(256), 0, (hipStream_t)stream,
                     (const u32x4 *)src, (u32x4 *)dst, n);
  return hipGetLastError() == hipSuccess ? NEXUS_OK : NEXUS_EHIP;
}

nexus_status nexus_calib_mfma_bf16(int32_t iters, float *sink, double *flops, void *stream) {
  if (iters <= 0 || !sink || !flops) return NEXUS_EINVAL;
  const uint32_t blocks = 256 * 2;   // 8 waves per CU: two per SIMD
  hipLaunchKernelGGL(calib_mfma_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters,
                     sink);
  *flops = (double)blocks * 4 /* waves */ * iters * kCalibChains * (2.0 * 32 * 32 * 16);
  return hipGetLastError() == hipSuccess ? NEXUS_OK : NEXUS_EHIP;
}

nexus_status nexus_calib_lds_dma(const void *src, size_t bytes, void *stream) {
  if (!src || bytes == 0 || bytes % kDmaChunk || ((uintptr_t)src & 15)) return NEXUS_EINVAL;
  const uint64_t chunks = bytes / kDmaChunk;
  const uint32_t blocks = (uint32_t)(chunks < 2048 ? chunks : 2048);
  hipLaunchKernelGGL(calib_lds_dma_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream,
                     (const char *)src, chunks);
  return hipGetLastError() == hipSuccess ? NEXUS_OK : NEXUS_EHIP;
}

}  // extern "C"
