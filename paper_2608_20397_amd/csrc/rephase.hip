// Re-anchoring of rotary keys (Sec. III-B): every key pair i of the selected rows is rotated
// by delta * theta_i, theta_i = base^(-2i/D), delta = splice position - compile anchor
// (the inverse of the drift of eq. (drift)).  In place; V is never touched.
//
// HBM-bound: the D/2 angles are formed in fp64 (reduced modulo 2*pi in fp64), their cosine and
// sine kept as fp32 head + tail pairs (c = c_hi + c_lo to about 2^-48) in LDS: for head_dim <= 256
// formed on the host and passed with the launch (HOST_TAB), otherwise by each workgroup;
// each thread owns a fixed group of feature pairs, holds their cos/sin in registers and streams
// rows with 16-byte non-temporal loads and stores.  The rotation x c - y s is evaluated in fp32
// with the product y s_hi split exactly by an FMA (Dekker's two-product) and the tail terms
// added separately, so the fp32 result is within about 2^-23 relative of the exact rotation
// even when the two products cancel; it is then rounded to the storage type (nearest-even).
#include "launch.h"
#include "rope_math.h"

namespace nexus {

// NEOX: thread chunk c owns pairs [N c, N c + N): elements [N c, +N) and [D/2 + N c, +N).
// INTERLEAVED: thread chunk c owns elements [2 N c, 2 N c + 2 N) = pairs [N c, N c + N).
//
// Rows are taken in memory order: a contiguous block row by row; a paged range page block by page
// block, (layer, page of the range, head, slot), so a workgroup's rows are whole 16-row page-head
// blocks and the slots of a partial first or last page that hold no token of the range are
// skipped.  A workgroup covers kBatch passes of 256 / tpr rows; its loads are issued before the
// angle table is formed, so the fp64 angles are computed while they are in flight.
template <typename T, bool INTERLEAVED, bool HOST_TAB>
__global__ __launch_bounds__(256) void rephase_kernel(
    T *__restrict__ k, const int32_t *__restrict__ map, int64_t offset, int64_t first_page,
    uint32_t n_rows, uint32_t tpr_shift, FastDiv div_heads, FastDiv div_pages, uint32_t n_heads,
    uint32_t n_range_pages, uint32_t n_tokens, uint32_t n_phys_pages, int32_t head_dim,
    int64_t delta, double base, const RopeTab tab) {
  constexpr int N = Pack<T>::N;
  constexpr int kBatch = 2;
  __shared__ float cs_tab[4][kMaxPairs];   // cos head, cos tail, sin head, sin tail
  const uint32_t c = threadIdx.x & ((1u << tpr_shift) - 1);
  const uint32_t rpp = blockDim.x >> tpr_shift;          // rows per pass
  const uint32_t sub = threadIdx.x >> tpr_shift;
  const uint32_t per_wg = kBatch * rpp;
  // key row r, or nullptr when r holds no token of the range
  auto row_ptr = [&](uint32_t r) -> T * {
    if (r >= n_rows) return nullptr;
    if (map == nullptr) return k + (uint64_t)r * head_dim;
    const uint32_t slot = r & (kPage - 1);
    const uint32_t lph = r >> kPageShift;                  // (layer, range page, head)
    const uint32_t lp = fdiv(lph, div_heads);
    const uint32_t h = lph - lp * n_heads;
    const uint32_t l = fdiv(lp, div_pages);
    const uint32_t p = lp - l * n_range_pages;
    const int64_t t = (first_page + p) * kPage + slot;
    if (t < offset || t >= offset + (int64_t)n_tokens) return nullptr;
    const uint64_t page = (uint32_t)map[first_page + p];
    return k + ((((uint64_t)l * n_phys_pages + page) * n_heads + h) * kPage + slot) * head_dim;
  };
  const uint32_t ea = INTERLEAVED ? 2 * N * c : N * c;                 // first element of each load
  const uint32_t eb = INTERLEAVED ? 2 * N * c + N : head_dim / 2 + N * c;
  T *rows[kBatch];
  u32x4 va[kBatch], vb[kBatch];
  // rows without a token load from row 0 (always valid) and are not stored
  auto issue = [&](uint32_t rb) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      rows[u] = row_ptr(rb + u * rpp);
      const T *src = rows[u] != nullptr ? rows[u] : k;
      va[u] = ld_stream(reinterpret_cast<const u32x4 *>(src + ea));
      vb[u] = ld_stream(reinterpret_cast<const u32x4 *>(src + eb));
    }
  };
  const uint32_t stride = gridDim.x * per_wg;
  uint32_t wb = blockIdx.x * per_wg;
  issue(wb + sub);
  for (int i = threadIdx.x; i < head_dim / 2; i += blockDim.x) {
    if constexpr (HOST_TAB) {
#pragma unroll
      for (int q = 0; q < 4; ++q) cs_tab[q][i] = tab.v[q][i];
    } else {
      pair_cs(delta, base, i, head_dim, cs_tab[0][i], cs_tab[1][i], cs_tab[2][i], cs_tab[3][i]);
    }
  }
  // LDS-only barrier: the row loads above stay in flight
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  float ch[N], cl[N], sh[N], sl[N];
#pragma unroll
  for (int e = 0; e < N; ++e) {
    ch[e] = cs_tab[0][N * c + e];
    cl[e] = cs_tab[1][N * c + e];
    sh[e] = cs_tab[2][N * c + e];
    sl[e] = cs_tab[3][N * c + e];
  }
  while (wb < n_rows) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (rows[u] == nullptr) continue;
      float x[2 * N], a[N], b[N];
      Pack<T>::unpack(va[u], x);
      Pack<T>::unpack(vb[u], x + N);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        a[e] = INTERLEAVED ? x[2 * e] : x[e];
        b[e] = INTERLEAVED ? x[2 * e + 1] : x[N + e];
      }
      rotate<N>(a, b, ch, cl, sh, sl);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        if (INTERLEAVED) {
          x[2 * e] = a[e];
          x[2 * e + 1] = b[e];
        } else {
          x[e] = a[e];
          x[N + e] = b[e];
        }
      }
      st_stream(Pack<T>::pack(x), reinterpret_cast<u32x4 *>(rows[u] + ea));
      st_stream(Pack<T>::pack(x + N), reinterpret_cast<u32x4 *>(rows[u] + eb));
    }
    wb += stride;
    if (wb < n_rows) issue(wb + sub);
  }
}

hipError_t launch_rephase(const RephaseLaunch &p, hipStream_t stream) {
  const int n_per16 = 16 / p.dtype_bytes;                // pairs per thread
  const uint32_t tpr = (uint32_t)(p.head_dim / 2 / n_per16);
  uint32_t shift = 0;
  while ((1u << shift) < tpr) ++shift;
  // rows: a contiguous block's rows, or every slot of the pages the paged range touches
  int64_t first_page = 0, n_pp = 1;
  uint64_t rows;
  if (p.map == nullptr) {
    rows = (uint64_t)p.n_layers * p.n_tokens * p.n_heads;
  } else {
    first_page = p.offset / kPage;
    n_pp = (p.offset + p.n_tokens - 1) / kPage - first_page + 1;
    rows = (uint64_t)p.n_layers * n_pp * p.n_heads * kPage;
  }
  if (rows >= (1ull << 32)) return hipErrorInvalidValue;
  // two passes of rows per workgroup, at most 4096 workgroups (measured best after a splice of
  // config 3: about 3% faster than 768 workgroups of 16 rows per thread)
  const uint64_t per_wg = 2 * (256u >> shift);
  uint64_t blocks = (rows + per_wg - 1) / per_wg;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  const FastDiv dh = make_fastdiv((uint32_t)p.n_heads);
  const FastDiv dp = make_fastdiv((uint32_t)n_pp);
  const bool host_tab = p.head_dim / 2 <= kTabPairs;
  RopeTab tab{};
  if (host_tab) rope_tab_host(p.delta, p.rope_base, p.head_dim, tab);
#define NEXUS_REPHASE(T, IL, HT)                                                                  \
  hipLaunchKernelGGL((rephase_kernel<T, IL, HT>), dim3((uint32_t)blocks), dim3(256), 0, stream,  \
                     (T *)p.k, p.map, p.offset, first_page, (uint32_t)rows, shift, dh, dp,        \
                     (uint32_t)p.n_heads, (uint32_t)n_pp, (uint32_t)p.n_tokens,                   \
                     (uint32_t)p.n_phys_pages, p.head_dim, p.delta, p.rope_base, tab)
#define NEXUS_REPHASE_T(T, IL)                                                                    \
  do {                                                                                            \
    if (host_tab) NEXUS_REPHASE(T, IL, true);                                                     \
    else NEXUS_REPHASE(T, IL, false);                                                             \
  } while (0)
  if (p.dtype_bytes == 2) {
    if (p.interleaved) NEXUS_REPHASE_T(uint16_t, true);
    else NEXUS_REPHASE_T(uint16_t, false);
  } else {
    if (p.interleaved) NEXUS_REPHASE_T(uint32_t, true);
    else NEXUS_REPHASE_T(uint32_t, false);
  }
#undef NEXUS_REPHASE_T
#undef NEXUS_REPHASE
  return hipGetLastError();
}

}  // namespace nexus
