// Splice of a compiled KV block into a paged KV cache (Sec. VI-A; transposed V per Sec. VI-B).
//
// Pure data movement, bit-exact.  Block rows [l][j][h][:] are contiguous; cache rows
// [l][page][h][slot][:] are contiguous, so the row-major kernel streams 16-byte chunks in the
// block's own order (coalesced reads) and writes whole rows (256 B for bf16, head_dim 128),
// both with non-temporal accesses (config 3, 48 layers, steady state: 70.6 -> 64.6 us).
// The transposed-V kernel stages a 64-token x head_dim tile in LDS and writes it back
// token-innermost, so both the row reads and the column writes stay coalesced.
#include "device_common.h"
#include "launch.h"

namespace nexus {

constexpr int kSpliceItemsPerThread = 1;

// Row-major splice of K and V (blockIdx.z: 0 = K, 1 = V; z = 1 is skipped for a transposed V).
// Work item = one 16-byte chunk; a layer's items are ordered (token j, head h, chunk c).
__global__ __launch_bounds__(256) void splice_rows_kernel(
    const u32x4 *__restrict__ bk, const u32x4 *__restrict__ bv, u32x4 *__restrict__ ck,
    u32x4 *__restrict__ cv, const int32_t *__restrict__ map, int64_t offset,
    uint32_t items_per_layer, uint32_t chunks_per_row, uint32_t chunk_shift, FastDiv div_heads,
    uint32_t n_heads, uint32_t n_phys_pages, uint32_t n_tokens) {
  const uint32_t layer = blockIdx.y;
  const u32x4 *src = blockIdx.z == 0 ? bk : bv;
  u32x4 *dst = blockIdx.z == 0 ? ck : cv;
  const uint64_t src_layer = (uint64_t)layer * items_per_layer;
  const uint64_t dst_layer = (uint64_t)layer * n_phys_pages * n_heads * kPage * chunks_per_row;
  // items per thread and loop pass: one item per thread, many workgroups (config 3, 48 layers:
  // 66.0 us against 69.2 us with four items per thread and a quarter of the workgroups)
  constexpr int kUnroll = kSpliceItemsPerThread;
  const uint32_t stride = gridDim.x * blockDim.x;
  uint32_t idx = blockIdx.x * blockDim.x + threadIdx.x;
  for (; idx < items_per_layer; idx += kUnroll * stride) {
    u32x4 v[kUnroll];
    uint64_t daddr[kUnroll];
    bool ok[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t i = idx + u * stride;
      ok[u] = i < items_per_layer;
      const uint32_t ii = ok[u] ? i : idx;
      const uint32_t row = ii >> chunk_shift;          // j * H + h
      const uint32_t c = ii & (chunks_per_row - 1);
      const uint32_t j = fdiv(row, div_heads);
      const uint32_t h = row - j * n_heads;
      const int64_t t = offset + j;
      const uint32_t page = (uint32_t)map[t >> kPageShift];
      const uint32_t slot = (uint32_t)(t & (kPage - 1));
      daddr[u] = dst_layer + (((uint64_t)page * n_heads + h) * kPage + slot) * chunks_per_row + c;
      v[u] = ld_stream(src + src_layer + ii);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
      if (ok[u]) st_stream(v[u], dst + daddr[u]);
  }
  (void)n_tokens;
}

// Transposed-V splice.  One workgroup = (layer, head, 64-token window aligned to logical
// pages).  Block V rows for the window are read into LDS, then every head_dim row of the
// cache receives the window's tokens as 8-token (16-byte) column pieces.  Only tokens inside
// [offset, offset + n_tokens) are written.  Element type is 16-bit (bf16) or 32-bit (f32).
template <typename T>
__global__ __launch_bounds__(256) void splice_vt_kernel(
    const T *__restrict__ bv, T *__restrict__ cvt, const int32_t *__restrict__ map,
    int64_t offset, int32_t n_tokens, int32_t n_heads, int32_t head_dim, int32_t n_phys_pages,
    int64_t first_window_start) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  T *tile = reinterpret_cast<T *>(smem_raw);  // [64][head_dim + pad]
  const int pad = 16 / (int)sizeof(T);
  const int ld = head_dim + pad;
  const int layer = blockIdx.z;
  const int h = blockIdx.y;
  const int64_t w0 = first_window_start + (int64_t)blockIdx.x * 64;  // logical, page aligned
  // stage: tokens t in [w0, w0 + 64) that belong to the block
  const int epc = 16 / (int)sizeof(T);           // elements per 16-byte chunk
  const int cpr = head_dim / epc;                // chunks per row
  for (int u = threadIdx.x; u < 64 * cpr; u += blockDim.x) {
    const int tt = u / cpr, c = u - tt * cpr;
    const int64_t t = w0 + tt;
    if (t < offset || t >= offset + n_tokens) continue;
    const int64_t j = t - offset;
    const uint4 val = *reinterpret_cast<const uint4 *>(
        bv + (((int64_t)layer * n_tokens + j) * n_heads + h) * head_dim + (int64_t)c * epc);
    *reinterpret_cast<uint4 *>(tile + tt * ld + c * epc) = val;
  }
  __syncthreads();
  // write: for each d, 8 groups of 8 tokens
  const int64_t n_cols = (int64_t)n_phys_pages * kPage;
  T *base = cvt + ((int64_t)layer * n_heads + h) * head_dim * n_cols;
  for (int u = threadIdx.x; u < head_dim * 8; u += blockDim.x) {
    const int d = u >> 3, grp = u & 7;
    const int64_t t0 = w0 + grp * 8;
    if (t0 + 8 <= offset || t0 >= offset + n_tokens) continue;  // no block token in this group
    const int64_t page = map[t0 >> kPageShift];
    T *dst = base + (int64_t)d * n_cols + page * kPage + (t0 & (kPage - 1));
    const T *col = tile + (grp * 8) * ld + d;
    if (t0 >= offset && t0 + 8 <= offset + n_tokens) {
      if (sizeof(T) == 2) {
        uint4 w;
        w.x = (uint32_t)col[0 * ld] | ((uint32_t)col[1 * ld] << 16);
        w.y = (uint32_t)col[2 * ld] | ((uint32_t)col[3 * ld] << 16);
        w.z = (uint32_t)col[4 * ld] | ((uint32_t)col[5 * ld] << 16);
        w.w = (uint32_t)col[6 * ld] | ((uint32_t)col[7 * ld] << 16);
        *reinterpret_cast<uint4 *>(dst) = w;
      } else {
        uint4 w0v, w1v;
        w0v.x = col[0 * ld]; w0v.y = col[1 * ld]; w0v.z = col[2 * ld]; w0v.w = col[3 * ld];
        w1v.x = col[4 * ld]; w1v.y = col[5 * ld]; w1v.z = col[6 * ld]; w1v.w = col[7 * ld];
        reinterpret_cast<uint4 *>(dst)[0] = w0v;
        reinterpret_cast<uint4 *>(dst)[1] = w1v;
      }
    } else {
      for (int e = 0; e < 8; ++e) {
        const int64_t t = t0 + e;
        if (t >= offset && t < offset + n_tokens) dst[e] = col[e * ld];
      }
    }
  }
}

hipError_t launch_splice(const SpliceLaunch &p, hipStream_t stream) {
  const uint32_t esize = p.dtype_bytes;
  const uint32_t chunks_per_row = (uint32_t)p.head_dim * esize / 16;
  uint32_t shift = 0;
  while ((1u << shift) < chunks_per_row) ++shift;
  const uint64_t items = (uint64_t)p.n_tokens * p.n_heads * chunks_per_row;
  const int n_kv = p.v_transposed ? 1 : 2;
  if (!p.v_only) {
    const uint32_t threads = 256;
    uint64_t want = (items + threads * kSpliceItemsPerThread - 1) / (threads * kSpliceItemsPerThread);
    const uint32_t blocks = (uint32_t)(want < 1 ? 1 : (want > 65535 ? 65535 : want));
    dim3 grid(blocks, p.n_layers, n_kv);
    hipLaunchKernelGGL(splice_rows_kernel, grid, dim3(threads), 0, stream,
                       (const u32x4 *)p.block_k, (const u32x4 *)p.block_v, (u32x4 *)p.cache_k,
                       (u32x4 *)p.cache_v, p.map, p.offset, (uint32_t)items, chunks_per_row, shift,
                       make_fastdiv(p.n_heads), (uint32_t)p.n_heads, (uint32_t)p.n_phys_pages,
                       (uint32_t)p.n_tokens);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (p.v_transposed) {
    const int64_t w_first = (p.offset / 64) * 64;
    const int64_t w_last = (p.offset + p.n_tokens - 1) / 64;
    const uint32_t n_windows = (uint32_t)(w_last - p.offset / 64 + 1);
    dim3 grid(n_windows, p.n_heads, p.n_layers);
    const int pad = 16 / (int)esize;
    const size_t smem = (size_t)64 * (p.head_dim + pad) * esize;
    if (esize == 2)
      hipLaunchKernelGGL(splice_vt_kernel<uint16_t>, grid, dim3(256), smem, stream,
                         (const uint16_t *)p.block_v, (uint16_t *)p.cache_v, p.map, p.offset,
                         p.n_tokens, p.n_heads, p.head_dim, p.n_phys_pages, w_first);
    else
      hipLaunchKernelGGL(splice_vt_kernel<uint32_t>, grid, dim3(256), smem, stream,
                         (const uint32_t *)p.block_v, (uint32_t *)p.cache_v, p.map, p.offset,
                         p.n_tokens, p.n_heads, p.head_dim, p.n_phys_pages, w_first);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace nexus
