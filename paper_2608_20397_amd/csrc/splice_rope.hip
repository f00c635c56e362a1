// Keys rotated on their way into the paged cache, in one pass over the source rows:
//   * splice + re-anchor (Sec. III-B with Sec. VI-A): block key token j, compiled at anchor m0,
//     is rotated by (dst - m0) * theta_i and written to logical slot offset + j; its value row
//     is copied.  Same arithmetic as rephase_kernel, so the cache ends bit-identical to a
//     splice followed by an in-place re-anchor, while the block's keys are read once and every
//     cache element is written once;
//   * rope-append (the redecode writes of Sec. VI-A): freshly computed, un-rotated key token j
//     is rotated to its absolute position pos0 + j (RoPE, Sec. III-B) and written with its value
//     row to logical slot offset + j.
// A workgroup covers kTileTokens tokens of one layer, all heads: its source rows are one
// contiguous run of the block.  Each thread issues the loads of its first kBatch items, then the
// workgroup puts the cosine and sine of every (token, pair) angle it needs in LDS as fp32 head +
// tail pairs while those loads are in flight: with one rotation for every token, the host's
// table of the launch (the one the re-anchor uses, so both give the same bits), per token formed
// in fp64 by the workgroup; then the threads rotate and write their items.
// HBM-bound.
#include "launch.h"
#include "rope_math.h"

namespace nexus {

namespace {

// 4 tokens per workgroup and one item per thread at a time: with 8 KV heads of 128 bf16 features
// a workgroup's items are one per thread (config 3, 48 layers: one-pass splice + re-anchor 76 us
// and rope-append 81 us, against 80 and 87 us with 8 tokens and two items per thread, and 84
// and 91 us with 8 tokens x 16 layers per workgroup)
constexpr int kTileTokens = 4;        // tokens per workgroup
constexpr int kMaxPairsTab = kTabPairs;   // head_dim <= 256
constexpr int kBatch = 1;             // items per thread whose loads are in flight together
constexpr int kOccCapFloats = 9500;   // LDS reserve: 40 KB per workgroup with the table, 4 per CU

}  // namespace

// Thread item = (chunk c of a row, row), rows in source order (token t of the tile, head h).
// NEOX: chunk c covers pairs [N c, N c + N): elements [N c, +N) and [D/2 + N c, +N).
// INTERLEAVED: elements [2 N c, 2 N c + 2 N) = pairs [N c, N c + N).
template <typename T, bool INTERLEAVED, bool PER_TOKEN>
__global__ __launch_bounds__(256) void rope_splice_kernel(
    const T *__restrict__ src_k, const T *__restrict__ src_v, T *__restrict__ ck,
    T *__restrict__ cv, const int32_t *__restrict__ map, int64_t offset, int32_t n_layers,
    int32_t n_tokens, int32_t n_heads, FastDiv div_heads, int32_t head_dim, uint32_t tpr_shift,
    int32_t n_phys_pages, int64_t angle0, double base, const RopeTab tab) {
  constexpr int N = Pack<T>::N;
  __shared__ float cs_tab[4][PER_TOKEN ? kTileTokens : 1][kMaxPairsTab];
  // With the host's table the single-rotation instance needs 62 registers, so 8 of its
  // workgroups would share a CU; at 8 it ran 3% slower than at the 4 its fp64 angle code allowed
  // (config 3 shapes, 48 layers: 5.88 against 6.05 TB/s).  It reserves LDS so that 4 fit.
  __shared__ float occ_cap[PER_TOKEN ? 1 : kOccCapFloats];
  if (threadIdx.x >= blockDim.x) occ_cap[0] = 0.f;   // keeps the reservation
  const int j0 = blockIdx.x * kTileTokens;
  const int l = blockIdx.y;
  const int n_tok = min(kTileTokens, n_tokens - j0);
  const int n_pairs = head_dim / 2;
  const uint32_t items = (uint32_t)(n_tok * n_heads) << tpr_shift;
  const uint32_t tpr_mask = (1u << tpr_shift) - 1;
  const int64_t src0 = ((int64_t)l * n_tokens + j0) * n_heads * head_dim;   // the tile's rows

  struct Item {
    u32x4 ka, kb, va, vb;
    int64_t drow;
    int t, c;
  };
  // loads of item it (clamped to the last item: always a valid row)
  auto load = [&](uint32_t it_raw, Item &x) {
    const uint32_t it = it_raw < items ? it_raw : items - 1;
    const int c = it & tpr_mask;
    const uint32_t r = it >> tpr_shift;                    // t * n_heads + h
    const int t = fdiv(r, div_heads);
    const int h = r - t * n_heads;
    const int64_t srow = src0 + (int64_t)r * head_dim;
    const int64_t tok = offset + j0 + t;
    const int64_t page = (uint32_t)map[tok >> kPageShift];
    x.drow = ((((int64_t)l * n_phys_pages + page) * n_heads + h) * kPage + (tok & (kPage - 1))) *
             head_dim;
    x.t = t;
    x.c = c;
    const int ea = INTERLEAVED ? 2 * N * c : N * c;             // first element of each load
    const int eb = INTERLEAVED ? 2 * N * c + N : n_pairs + N * c;
    x.ka = ld_stream(reinterpret_cast<const u32x4 *>(src_k + srow + ea));
    x.kb = ld_stream(reinterpret_cast<const u32x4 *>(src_k + srow + eb));
    if (src_v != nullptr) {
      x.va = ld_stream(reinterpret_cast<const u32x4 *>(src_v + srow + ea));
      x.vb = ld_stream(reinterpret_cast<const u32x4 *>(src_v + srow + eb));
    }
  };
  Item cur[kBatch];
#pragma unroll
  for (int u = 0; u < kBatch; ++u) load(threadIdx.x + u * blockDim.x, cur[u]);

  if constexpr (PER_TOKEN) {
    // token j0 + t sits at angle0 + j0 + t
    for (int x = threadIdx.x; x < n_tok * n_pairs; x += blockDim.x) {
      const int t = x / n_pairs, i = x - t * n_pairs;
      pair_cs(angle0 + j0 + t, base, i, head_dim, cs_tab[0][t][i], cs_tab[1][t][i],
              cs_tab[2][t][i], cs_tab[3][t][i]);
    }
  } else {
    // every token turns by angle0
    for (int i = threadIdx.x; i < n_pairs; i += blockDim.x) {
#pragma unroll
      for (int q = 0; q < 4; ++q) cs_tab[q][0][i] = tab.v[q][i];
    }
  }
  // LDS-only barrier: the item loads above stay in flight
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");

  for (uint32_t it0 = threadIdx.x; it0 < items; it0 += kBatch * blockDim.x) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (it0 + u * blockDim.x >= items) continue;
      const Item &x0 = cur[u];
      const int c = x0.c;
      const int tt = PER_TOKEN ? x0.t : 0;
      const int ea = INTERLEAVED ? 2 * N * c : N * c;
      const int eb = INTERLEAVED ? 2 * N * c + N : n_pairs + N * c;
      float x[2 * N], a[N], b[N];
      Pack<T>::unpack(x0.ka, x);
      Pack<T>::unpack(x0.kb, x + N);
#pragma unroll
      for (int e = 0; e < N; ++e) {
        a[e] = INTERLEAVED ? x[2 * e] : x[e];
        b[e] = INTERLEAVED ? x[2 * e + 1] : x[N + e];
      }
      float ch[N], cl[N], sh[N], sl[N];
#pragma unroll
      for (int e = 0; e < N; ++e) {
        ch[e] = cs_tab[0][tt][N * c + e];
        cl[e] = cs_tab[1][tt][N * c + e];
        sh[e] = cs_tab[2][tt][N * c + e];
        sl[e] = cs_tab[3][tt][N * c + e];
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
      st_stream(Pack<T>::pack(x), reinterpret_cast<u32x4 *>(ck + x0.drow + ea));
      st_stream(Pack<T>::pack(x + N), reinterpret_cast<u32x4 *>(ck + x0.drow + eb));
      if (src_v != nullptr) {
        st_stream(x0.va, reinterpret_cast<u32x4 *>(cv + x0.drow + ea));
        st_stream(x0.vb, reinterpret_cast<u32x4 *>(cv + x0.drow + eb));
      }
    }
    if (it0 + kBatch * blockDim.x < items) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) load(it0 + (kBatch + u) * blockDim.x, cur[u]);
    }
  }
  (void)n_layers;
}

hipError_t launch_rope_splice(const RopeSpliceLaunch &p, hipStream_t stream) {
  // V of a transposed cache goes through the splice kernel's transposing path
  const bool v_rows = !p.v_transposed;
  const dim3 grid((p.n_tokens + kTileTokens - 1) / kTileTokens, p.n_layers);
  const uint32_t tpr = (uint32_t)(p.head_dim / 2 / (16 / p.dtype_bytes));
  uint32_t shift = 0;
  while ((1u << shift) < tpr) ++shift;
  const FastDiv dh = make_fastdiv((uint32_t)p.n_heads);
  RopeTab tab{};
  if (!p.per_token) rope_tab_host(p.angle0, p.rope_base, p.head_dim, tab);
#define NEXUS_ROPE_SPLICE(T, IL, PT)                                                              \
  hipLaunchKernelGGL((rope_splice_kernel<T, IL, PT>), grid, dim3(256), 0, stream,                \
                     (const T *)p.src_k, v_rows ? (const T *)p.src_v : nullptr, (T *)p.cache_k,  \
                     v_rows ? (T *)p.cache_v : nullptr, p.map, p.offset, p.n_layers, p.n_tokens, \
                     p.n_heads, dh, p.head_dim, shift, p.n_phys_pages, p.angle0, p.rope_base, tab)
  if (p.dtype_bytes == 2) {
    if (p.per_token) {
      if (p.interleaved) NEXUS_ROPE_SPLICE(uint16_t, true, true);
      else NEXUS_ROPE_SPLICE(uint16_t, false, true);
    } else {
      if (p.interleaved) NEXUS_ROPE_SPLICE(uint16_t, true, false);
      else NEXUS_ROPE_SPLICE(uint16_t, false, false);
    }
  } else {
    if (p.per_token) {
      if (p.interleaved) NEXUS_ROPE_SPLICE(uint32_t, true, true);
      else NEXUS_ROPE_SPLICE(uint32_t, false, true);
    } else {
      if (p.interleaved) NEXUS_ROPE_SPLICE(uint32_t, true, false);
      else NEXUS_ROPE_SPLICE(uint32_t, false, false);
    }
  }
#undef NEXUS_ROPE_SPLICE
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || v_rows) return e;
  SpliceLaunch s{};
  s.block_k = p.src_k;
  s.block_v = p.src_v;
  s.cache_k = p.cache_k;
  s.cache_v = p.cache_v;
  s.map = p.map;
  s.offset = p.offset;
  s.n_layers = p.n_layers;
  s.n_tokens = p.n_tokens;
  s.n_heads = p.n_heads;
  s.head_dim = p.head_dim;
  s.n_phys_pages = p.n_phys_pages;
  s.dtype_bytes = p.dtype_bytes;
  s.v_transposed = true;
  s.v_only = true;
  return launch_splice(s, stream);
}

}  // namespace nexus
