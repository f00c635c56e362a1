// Re-anchoring of rotary keys (Sec. III-B): every key pair i of the selected rows is rotated
// by delta * theta_i, theta_i = base^(-2i/D), delta = splice position - compile anchor
// (the inverse of the drift of eq. (drift)).  In place; V is never touched.
//
// HBM-bound: each workgroup forms the D/2 angles once in fp64 (reduced modulo 2*pi in fp64) and
// keeps their cosine and sine in LDS as fp32 head + tail pairs (c = c_hi + c_lo to about 2^-48);
// each thread owns a fixed group of feature pairs, holds their cos/sin in registers and streams
// rows with 16-byte loads and stores.  The rotation x c - y s is evaluated in fp32 with the
// product y s_hi split exactly by an FMA (Dekker's two-product) and the tail terms added
// separately, so the fp32 result is within about 2^-23 relative of the exact rotation even
// when the two products cancel; it is then rounded to the storage type (nearest-even).
#include "launch.h"
#include "rope_math.h"

namespace nexus {

// NEOX: thread chunk c owns pairs [N c, N c + N): elements [N c, +N) and [D/2 + N c, +N).
// INTERLEAVED: thread chunk c owns elements [2 N c, 2 N c + 2 N) = pairs [N c, N c + N).
template <typename T, bool INTERLEAVED>
__global__ __launch_bounds__(256) void rephase_kernel(
    T *__restrict__ k, const int32_t *__restrict__ map, int64_t offset, uint32_t n_rows,
    uint32_t tpr_shift, FastDiv div_heads, FastDiv div_layer_rows, uint32_t n_heads,
    uint32_t n_tokens, uint32_t n_phys_pages, int32_t head_dim, int64_t delta, double base) {
  constexpr int N = Pack<T>::N;
  __shared__ float cs_tab[4][kMaxPairs];   // cos head, cos tail, sin head, sin tail
  for (int i = threadIdx.x; i < head_dim / 2; i += blockDim.x)
    pair_cs(delta, base, i, head_dim, cs_tab[0][i], cs_tab[1][i], cs_tab[2][i], cs_tab[3][i]);
  __syncthreads();

  const uint32_t tpr = 1u << tpr_shift;  // threads per row
  const uint32_t gtid = blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t c = gtid & (tpr - 1);
  const uint32_t row_step = (gridDim.x * blockDim.x) >> tpr_shift;
  float ch[N], cl[N], sh[N], sl[N];
#pragma unroll
  for (int e = 0; e < N; ++e) {
    ch[e] = cs_tab[0][N * c + e];
    cl[e] = cs_tab[1][N * c + e];
    sh[e] = cs_tab[2][N * c + e];
    sl[e] = cs_tab[3][N * c + e];
  }

  // rows in batches of kBatch: all loads of a batch are in flight before any rotation
  constexpr int kBatch = 4;
  auto row_ptr = [&](uint32_t r) -> T * {
    if (map == nullptr) return k + (uint64_t)r * head_dim;
    const uint32_t l = fdiv(r, div_layer_rows);
    const uint32_t rem = r - l * n_tokens * n_heads;
    const uint32_t j = fdiv(rem, div_heads);
    const uint32_t h = rem - j * n_heads;
    const int64_t t = offset + j;
    const uint64_t page = (uint32_t)map[t >> kPageShift];
    return k + ((((uint64_t)l * n_phys_pages + page) * n_heads + h) * kPage +
                (uint64_t)(t & (kPage - 1))) * head_dim;
  };
  for (uint32_t r0 = gtid >> tpr_shift; r0 < n_rows; r0 += kBatch * row_step) {
    u32x4 *pa[kBatch], *pb[kBatch];
    u32x4 va[kBatch], vb[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const uint32_t r = r0 + u * row_step;
      T *row = row_ptr(r < n_rows ? r : r0);
      if constexpr (INTERLEAVED) {
        pa[u] = reinterpret_cast<u32x4 *>(row + 2 * N * c);
        pb[u] = pa[u] + 1;
      } else {
        pa[u] = reinterpret_cast<u32x4 *>(row + N * c);
        pb[u] = reinterpret_cast<u32x4 *>(row + head_dim / 2 + N * c);
      }
      va[u] = *pa[u];
      vb[u] = *pb[u];
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (r0 + u * row_step >= n_rows) continue;
      float x[2 * N], a[N], b[N];
      Pack<T>::unpack(va[u], x);
      Pack<T>::unpack(vb[u], x + N);
      if constexpr (INTERLEAVED) {
#pragma unroll
        for (int e = 0; e < N; ++e) {
          a[e] = x[2 * e];
          b[e] = x[2 * e + 1];
        }
      } else {
#pragma unroll
        for (int e = 0; e < N; ++e) {
          a[e] = x[e];
          b[e] = x[N + e];
        }
      }
      rotate<N>(a, b, ch, cl, sh, sl);
      if constexpr (INTERLEAVED) {
#pragma unroll
        for (int e = 0; e < N; ++e) {
          x[2 * e] = a[e];
          x[2 * e + 1] = b[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < N; ++e) {
          x[e] = a[e];
          x[N + e] = b[e];
        }
      }
      *pa[u] = Pack<T>::pack(x);
      *pb[u] = Pack<T>::pack(x + N);
    }
  }
}

hipError_t launch_rephase(const RephaseLaunch &p, hipStream_t stream) {
  const int n_per16 = 16 / p.dtype_bytes;                // pairs per thread
  const uint32_t tpr = (uint32_t)(p.head_dim / 2 / n_per16);
  uint32_t shift = 0;
  while ((1u << shift) < tpr) ++shift;
  const uint64_t rows = (uint64_t)p.n_layers * p.n_tokens * p.n_heads;
  const uint64_t threads_needed = rows << shift;
  // about 16 rows per thread, at most 2048 workgroups: the per-workgroup angle table is cheap
  uint64_t blocks = (threads_needed + 256 * 16 - 1) / (256 * 16);
  if (blocks < 1) blocks = 1;
  if (blocks > 2048) blocks = 2048;
  const FastDiv dh = make_fastdiv((uint32_t)p.n_heads);
  const FastDiv dl = make_fastdiv((uint32_t)(p.n_tokens * p.n_heads));
  if (p.dtype_bytes == 2) {
    if (p.interleaved)
      hipLaunchKernelGGL((rephase_kernel<uint16_t, true>), dim3((uint32_t)blocks), dim3(256), 0,
                         stream, (uint16_t *)p.k, p.map, p.offset, (uint32_t)rows, shift, dh, dl,
                         (uint32_t)p.n_heads, (uint32_t)p.n_tokens, (uint32_t)p.n_phys_pages,
                         p.head_dim, p.delta, p.rope_base);
    else
      hipLaunchKernelGGL((rephase_kernel<uint16_t, false>), dim3((uint32_t)blocks), dim3(256), 0,
                         stream, (uint16_t *)p.k, p.map, p.offset, (uint32_t)rows, shift, dh, dl,
                         (uint32_t)p.n_heads, (uint32_t)p.n_tokens, (uint32_t)p.n_phys_pages,
                         p.head_dim, p.delta, p.rope_base);
  } else {
    if (p.interleaved)
      hipLaunchKernelGGL((rephase_kernel<uint32_t, true>), dim3((uint32_t)blocks), dim3(256), 0,
                         stream, (uint32_t *)p.k, p.map, p.offset, (uint32_t)rows, shift, dh, dl,
                         (uint32_t)p.n_heads, (uint32_t)p.n_tokens, (uint32_t)p.n_phys_pages,
                         p.head_dim, p.delta, p.rope_base);
    else
      hipLaunchKernelGGL((rephase_kernel<uint32_t, false>), dim3((uint32_t)blocks), dim3(256), 0,
                         stream, (uint32_t *)p.k, p.map, p.offset, (uint32_t)rows, shift, dh, dl,
                         (uint32_t)p.n_heads, (uint32_t)p.n_tokens, (uint32_t)p.n_phys_pages,
                         p.head_dim, p.delta, p.rope_base);
  }
  return hipGetLastError();
}

}  // namespace nexus
