// fp32 causal grouped-query suffix attention (Sec. III-A) for f32 caches.
//
// A small-shape kernel with fp32 arithmetic throughout: one workgroup per (query, query head),
// keys streamed in chunks of 256 with an online softmax; each thread scores one key of the
// chunk, the workgroup reduces max and sum, and thread d accumulates output feature d.
#include "device_common.h"
#include "launch.h"

namespace nexus {

namespace {

__device__ __forceinline__ float block_reduce_max(float v, float *red) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) r = fmaxf(r, red[i]);
  return r;
}

__device__ __forceinline__ float block_reduce_sum(float v, float *red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float r = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) r += red[i];
  return r;
}

}  // namespace

struct F32SeqTable {
  AttnSeq seq[64];
  int32_t row_begin[65];  // prefix sum of len
};

__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float *__restrict__ q, float *__restrict__ out, const float *__restrict__ kc,
    const float *__restrict__ vc, const int32_t *__restrict__ map, int32_t layer,
    int32_t n_phys_pages, int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim, int v_t,
    float scale, float softcap, F32SeqTable tab, int32_t n_seqs) {
  __shared__ float qs[256];
  __shared__ float ps[256];
  __shared__ float red[8];
  const int row = blockIdx.x;  // over all sequences' queries
  int b = 0;
  while (b + 1 < n_seqs && row >= tab.row_begin[b + 1]) ++b;
  const int i = row - tab.row_begin[b];
  const AttnSeq sq = tab.seq[b];
  const int qrow = sq.q_start + i;
  const int h = blockIdx.y;
  const int g = h / (n_q_heads / n_kv_heads);
  const int64_t pos = sq.n_past + i;
  const int64_t n_keys = pos + 1;
  const int tid = threadIdx.x;
  if (tid < head_dim) qs[tid] = q[((int64_t)qrow * n_q_heads + h) * head_dim + tid];
  __syncthreads();

  const int64_t n_cols = (int64_t)n_phys_pages * kPage;
  const float *kl = kc + (int64_t)layer * n_phys_pages * n_kv_heads * kPage * head_dim;
  const float *vl = vc + (int64_t)layer * n_phys_pages * n_kv_heads * kPage * head_dim;
  float m = -INFINITY, l = 0.f, acc = 0.f;
  for (int64_t base = 0; base < n_keys; base += 256) {
    const int64_t t = base + tid;
    float s = -INFINITY;
    if (t < n_keys) {
      const int64_t page = map[t >> kPageShift];
      const float *kr = kl + ((page * n_kv_heads + g) * kPage + (t & (kPage - 1))) * head_dim;
      float dot = 0.f;
      for (int d = 0; d < head_dim; ++d) dot = fmaf(qs[d], kr[d], dot);
      s = dot * scale;
      if (softcap > 0.f) s = softcap * tanhf(s / softcap);
    }
    const float m_tile = block_reduce_max(s, red);
    const float m_new = fmaxf(m, m_tile);
    const float p = (t < n_keys) ? __expf(s - m_new) : 0.f;
    const float alpha = (m == -INFINITY) ? 0.f : __expf(m - m_new);
    ps[tid] = p;
    const float psum = block_reduce_sum(p, red);   // its barriers also publish ps[]
    l = l * alpha + psum;
    if (tid < head_dim) {
      acc *= alpha;
      const int n = (int)((n_keys - base) < 256 ? (n_keys - base) : 256);
      for (int u = 0; u < n; ++u) {
        const int64_t tt = base + u;
        const int64_t page = map[tt >> kPageShift];
        float vv;
        if (v_t)
          vv = vl[((int64_t)g * head_dim + tid) * n_cols + page * kPage + (tt & (kPage - 1))];
        else
          vv = vl[((page * n_kv_heads + g) * kPage + (tt & (kPage - 1))) * head_dim + tid];
        acc = fmaf(ps[u], vv, acc);
      }
    }
    m = m_new;
    __syncthreads();
  }
  if (tid < head_dim) out[((int64_t)qrow * n_q_heads + h) * head_dim + tid] = acc / l;
}

hipError_t launch_attention_f32(const AttnLaunch &p, hipStream_t stream) {
  F32SeqTable tab{};
  int32_t rows = 0;
  for (int b = 0; b < p.n_seqs; ++b) {
    tab.seq[b] = p.seqs[b];
    tab.row_begin[b] = rows;
    rows += p.seqs[b].len;
  }
  tab.row_begin[p.n_seqs] = rows;
  dim3 grid(rows, p.n_q_heads);
  hipLaunchKernelGGL(attn_f32_kernel, grid, dim3(256), 0, stream, (const float *)p.q,
                     (float *)p.out, (const float *)p.cache_k, (const float *)p.cache_v, p.map,
                     p.layer, p.n_phys_pages, p.n_kv_heads, p.n_q_heads, p.head_dim,
                     p.v_transposed ? 1 : 0, p.scale, p.softcap, tab, p.n_seqs);
  return hipGetLastError();
}

}  // namespace nexus
