// Warm-prefix reuse on the paged cache (the exact-token prefix arena of Sec. VI-D): copying the
// K/V of a token range from one sequence's pages to another's, and sharing a prefix by page
// reference with only its partial last page copied.  Pure data movement, bit-exact, HBM-bound.
//
// One workgroup per (logical page of the range, layer, head).  A page-head block of K (and of a
// row-major V) is 16 rows of head_dim contiguous elements, so the slots [s0, s1) of one head
// are one contiguous run of (s1 - s0) * head_dim elements, copied in 16-byte chunks.  A
// transposed V holds each (head, feature) row token-innermost: the run is (s1 - s0) elements
// per row, copied as 16-byte chunks when the page is whole and element by element otherwise.
// Each thread issues the loads of up to kBatch chunks before their stores.
#include "device_common.h"
#include "launch_decode.h"

namespace nexus {

namespace {

constexpr int kBatch = 4;   // chunks whose loads are in flight together, per thread

template <typename T>
__global__ __launch_bounds__(256) void kv_copy_kernel(KvCopyLaunch p, int64_t first_page) {
  // prefix sharing: logical pages [0, share_n_full) of the destination take the source's
  // physical pages (the pages copied below are never among them)
  if (p.share_map != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0)
    for (int i = threadIdx.x; i < p.share_n_full; i += 256) p.share_map[i] = p.src_map[i];
  const int64_t lp = first_page + blockIdx.x;              // logical page
  const int layer = blockIdx.y, h = blockIdx.z;
  const int64_t t_lo = max(p.t0, lp * kPage);
  const int64_t t_hi = min(p.t0 + p.n_tokens, lp * kPage + kPage);
  const int s0 = (int)(t_lo - lp * kPage), s1 = (int)(t_hi - lp * kPage);
  if (s1 <= s0) return;                                     // no token of the range here
  const uint32_t src = (uint32_t)p.src_map[lp];
  const uint32_t dst = (uint32_t)p.dst_map[lp];
  if (src == dst) return;                                   // shared page: nothing to move
  const int H = p.n_kv_heads, D = p.head_dim;
  const size_t layer_elems = (size_t)p.n_phys_pages * H * kPage * D;
  constexpr int E = 16 / sizeof(T);                         // elements per 16-byte chunk
  // K and a row-major V of head h: (s1 - s0) * D contiguous elements each
  const int run = (s1 - s0) * D / E;                        // chunks per head
  const int n_kv = p.v_transposed ? 1 : 2;
  const size_t so0 = (((size_t)src * H + h) * kPage + s0) * D;
  const size_t do0 = (((size_t)dst * H + h) * kPage + s0) * D;
  T *const base_k = reinterpret_cast<T *>(p.cache_k) + (size_t)layer * layer_elems;
  T *const base_v = reinterpret_cast<T *>(p.cache_v) + (size_t)layer * layer_elems;
  for (int it0 = threadIdx.x; it0 < n_kv * run; it0 += 256 * kBatch) {
    u32x4 v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int it = min(it0 + 256 * u, n_kv * run - 1);
      const int kv = it >= run, c = it - kv * run;
      v[u] = *reinterpret_cast<const u32x4 *>((kv ? base_v : base_k) + so0 + (size_t)c * E);
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int it = it0 + 256 * u;
      if (it >= n_kv * run) break;
      const int kv = it >= run, c = it - kv * run;
      *reinterpret_cast<u32x4 *>((kv ? base_v : base_k) + do0 + (size_t)c * E) = v[u];
    }
  }
  if (!p.v_transposed) return;
  // transposed V: row (h, d) holds token column page * 16 + slot
  const size_t n_cols = (size_t)p.n_phys_pages * kPage;
  T *const vt = reinterpret_cast<T *>(p.cache_v) + (size_t)layer * layer_elems +
                (size_t)h * D * n_cols;
  if (s0 == 0 && s1 == kPage) {
    constexpr int CPR = kPage / E;                          // chunks per page row: 2 (bf16), 4 (f32)
    for (int it = threadIdx.x; it < D * CPR; it += 256) {
      const int d = it / CPR, c = it - d * CPR;
      const size_t ro = (size_t)d * n_cols;
      *reinterpret_cast<u32x4 *>(vt + ro + (size_t)dst * kPage + c * E) =
          *reinterpret_cast<const u32x4 *>(vt + ro + (size_t)src * kPage + c * E);
    }
  } else {
    const int w = s1 - s0;
    for (int it = threadIdx.x; it < D * w; it += 256) {
      const int d = it / w, e = it - d * w;
      const size_t ro = (size_t)d * n_cols;
      vt[ro + (size_t)dst * kPage + s0 + e] = vt[ro + (size_t)src * kPage + s0 + e];
    }
  }
}

}  // namespace

hipError_t launch_kv_copy(const KvCopyLaunch &p, hipStream_t stream) {
  // pages [first, last] of the range; with no token to copy, one workgroup still writes the
  // shared map entries
  const int64_t first = p.t0 / kPage;
  const int64_t last = p.n_tokens > 0 ? (p.t0 + p.n_tokens - 1) / kPage : first;
  const dim3 grid((unsigned)(last - first + 1), p.n_tokens > 0 ? p.n_layers : 1,
                  p.n_tokens > 0 ? p.n_kv_heads : 1);
  if (p.dtype_bytes == 2)
    hipLaunchKernelGGL(kv_copy_kernel<uint16_t>, grid, dim3(256), 0, stream, p, first);
  else
    hipLaunchKernelGGL(kv_copy_kernel<uint32_t>, grid, dim3(256), 0, stream, p, first);
  return hipGetLastError();
}

}  // namespace nexus
