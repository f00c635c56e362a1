// Semantic Lookaside Buffer scan on MI355X (Sec. V-A): INT8 tool embeddings scanned with integer
// dot products against INT8 query embeddings, the best tools per query kept, and the margin gate
// (auto-route when the top-two score margin exceeds tau, else escalate).
//
// Score of tool t for query q: (float(dot_int32(T_t, Q_q)) * s_t) * s_q in fp32, each product
// rounded to nearest-even; the integer dot is exact and, with |dot| <= 127^2 * 1024 < 2^24,
// exactly representable in fp32.
//
// Scan kernel: a workgroup takes a block of 64 queries and a range of tools.  The query block
// sits in LDS; each of the 4 waves takes a 16-query sub-block and 16-tool tiles of the range and
// computes
// S^T = T.Q^T on v_mfma_i32_16x16x64_i8 (tool rows straight from global memory in the A-operand
// layout, B operands from LDS), loading the next tile while it computes the current one.  Lane l
// then holds tools 4 (l / 16) .. +3 of the tile for query column l % 16 and folds them into its
// own sorted list of the best KT (higher score first, lower index first among equal scores: both
// orders are carried by one 64-bit key, so the list update is a branch-free max/min pass).  With
// a full query block each wave owns one 16-query sub-block, so a query's 4 lists meet in one
// wave and are merged by lane exchanges; smaller blocks share sub-blocks among waves and merge
// those lists through LDS.  With one tool range the
// result is final (top-k, margin, gate); otherwise each range's best 8 go to the workspace and a
// second kernel merges them the same way.
#include "device_common.h"
#include "launch_slb.h"

namespace nexus {

namespace {

typedef __attribute__((ext_vector_type(4))) int i32x4;

constexpr int kTop = 8;          // candidates kept per (lane, query) and per range
constexpr int kWaves = 4;
constexpr int kSubBlocks = 4;    // 16-query sub-blocks per workgroup (64 queries)

// A candidate (score, tool index) is one 64-bit key whose unsigned order is the ranking order:
// the fp32 score mapped to an order-preserving 32-bit pattern in the high half, the complement
// of the index in the low half (so the lower index wins between equal scores); 0 = no tool.
__device__ __forceinline__ uint64_t cand_key(float score, int idx) {
  const uint32_t u = __float_as_uint(score);
  const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)ord << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)idx);
}
__device__ __forceinline__ int cand_idx(uint64_t k) {
  return k == 0 ? -1 : (int)(0xFFFFFFFFu - (uint32_t)k);
}
__device__ __forceinline__ float cand_score(uint64_t k) {
  if (k == 0) return -INFINITY;
  const uint32_t ord = (uint32_t)(k >> 32);
  return __uint_as_float((ord & 0x80000000u) ? (ord & 0x7FFFFFFFu) : ~ord);
}

// Insert x into the descending list b: a max/min pass carries x down to its place and drops the
// smallest.  Skipped by the whole wave when no lane's x beats its list's last entry.
template <int KT>
__device__ __forceinline__ void insert(uint64_t (&b)[KT], uint64_t x) {
  if (!__builtin_amdgcn_ballot_w64(x > b[KT - 1])) return;
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    const bool gt = x > b[j];
    const uint64_t hi = gt ? x : b[j];
    x = gt ? b[j] : x;
    b[j] = hi;
  }
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int off) {
  const uint32_t lo = __shfl_xor((uint32_t)v, off);
  const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), off);
  return ((uint64_t)hi << 32) | lo;
}

// The best KT of n candidate keys, selected by one wave: every lane sorts its
// share, then KT rounds take the wave-wide largest head (keys are distinct, so exactly one lane
// advances).
template <int KT>
__device__ __forceinline__ void wave_select(const uint64_t *c, int n, int lane,
                                            uint64_t (&out)[KT]) {
  uint64_t b[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) b[j] = 0;
  for (int i = lane; i < n; i += 64) insert<KT>(b, c[i]);
  int head = 0;
#pragma unroll
  for (int r = 0; r < KT; ++r) {
    uint64_t h = 0;
#pragma unroll
    for (int j = 0; j < KT; ++j) h = j == head ? b[j] : h;
    uint64_t w = h;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const uint64_t o = shfl_xor_u64(w, off);
      w = o > w ? o : w;
    }
    out[r] = w;
    if (w != 0 && h == w) ++head;
  }
}

struct SlbArgs {
  const int8_t *tools;
  const float *tool_scale;
  const int8_t *queries;
  const float *query_scale;
  int32_t n_tools, n_queries, dim, k;
  int32_t n_ranges, range_tools;     // tools per range (a multiple of 64)
  float tau;
  int32_t *top_idx;
  float *top_score;
  float *margin;
  int32_t *route;
  uint64_t *part;                     // [n_queries][n_ranges][KT] candidate keys
};

// Final outputs of one query from its sorted best keys (lane 0 writes).
template <int KT>
__device__ __forceinline__ void write_final(const SlbArgs &a, int q, const uint64_t (&b)[KT],
                                            int lane) {
  if (lane != 0) return;
#pragma unroll
  for (int j = 0; j < KT; ++j)
    if (j < a.k) {
      a.top_idx[(size_t)q * a.k + j] = cand_idx(b[j]);
      a.top_score[(size_t)q * a.k + j] = cand_score(b[j]);
    }
  // fewer than two tools: nothing to confuse the best one with
  const float m = b[1] == 0 ? INFINITY : cand_score(b[0]) - cand_score(b[1]);
  a.margin[q] = m;
  a.route[q] = m > a.tau ? 1 : 0;
}

// Merge the partner lane's sorted list into this lane's (both lanes end with the best KT of the
// union, the same list).
template <int KT>
__device__ __forceinline__ void merge_lanes(uint64_t (&b)[KT], int off) {
  uint64_t o[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) o[j] = shfl_xor_u64(b[j], off);
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    uint64_t x = o[j];
#pragma unroll
    for (int m = 0; m < KT; ++m) {
      const bool gt = x > b[m];
      const uint64_t hi = gt ? x : b[m];
      x = gt ? b[m] : x;
      b[m] = hi;
    }
  }
}

// MAXS: 64-byte steps of dim at most (dim <= 64 MAXS); KT: candidates kept, >= max(k, 2);
// SPW: 16-query sub-blocks per wave.
//   SPW = 1: wave w works on sub-block w % nsb (nsb = sub-blocks holding queries) and on every
//     (4 / nsb)-th tile of the range: a tile load feeds one MFMA chain, and with a full block each
//     wave owns its queries outright (small batches, few tiles per query block);
//   SPW = 4: every wave works on all sub-blocks and on every 4th tile: a tile load feeds four
//     MFMA chains (large batches, where the tool rows would otherwise be re-read four times).
template <int MAXS, int KT, int SPW>
__global__ __launch_bounds__(256) void slb_scan_kernel(SlbArgs a) {
  constexpr int QB = 16 * kSubBlocks;
  extern __shared__ __align__(16) unsigned char smem[];
  int8_t *qs = reinterpret_cast<int8_t *>(smem);                       // [QB][dim]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qn = lane & 15, grp = lane >> 4;
  const int q0 = blockIdx.y * QB;
  const int range = blockIdx.x;
  const int t_begin = range * a.range_tools;
  const int t_end = min(t_begin + a.range_tools, a.n_tools);
  const int dim = a.dim, steps = dim / 64;
  const int nsb = min(kSubBlocks, (a.n_queries - q0 + 15) / 16);     // sub-blocks with queries
  const int slot = SPW == 1 ? wave / nsb : wave;                       // rank among its waves
  const int n_slots = SPW == 1 ? (kWaves - 1 - wave % nsb) / nsb + 1 : kWaves;
  const int n_lists = SPW == 1 ? 1 : nsb;                              // sub-blocks of this wave
  auto sub_block = [&](int s) { return SPW == 1 ? wave % nsb : s; };

  // stage the query block (rows past n_queries are zero)
  for (int c = tid; c < QB * (dim / 16); c += 256) {
    const int r = c / (dim / 16), off = (c - r * (dim / 16)) * 16;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (q0 + r < a.n_queries)
      v = *reinterpret_cast<const u32x4 *>(a.queries + (size_t)(q0 + r) * dim + off);
    *reinterpret_cast<u32x4 *>(qs + r * dim + off) = v;
  }
  float sq[SPW];
#pragma unroll
  for (int s = 0; s < SPW; ++s) {
    const int q = q0 + 16 * sub_block(s) + qn;
    sq[s] = q < a.n_queries ? a.query_scale[q] : 0.f;
  }
  __syncthreads();

  uint64_t best[SPW][KT];
  uint64_t floor_key[SPW];   // a lower bound of the KT-th best key of each query column
#pragma unroll
  for (int s = 0; s < SPW; ++s) {
    floor_key[s] = 0;
#pragma unroll
    for (int j = 0; j < KT; ++j) best[s][j] = 0;
  }

  struct Tile {
    i32x4 a[MAXS];
    float st[4];
  };
  // Every call issues the same loads (rows and steps past the end re-read valid ones), so the
  // wait before a tile's use leaves the next tile's loads in flight.
  auto load_tile = [&](int t0, Tile &tl) {
    const int8_t *trow = a.tools + (size_t)min(t0 + qn, a.n_tools - 1) * dim + 16 * grp;
#pragma unroll
    for (int st = 0; st < MAXS; ++st)
      tl.a[st] = *reinterpret_cast<const i32x4 *>(trow + 64 * min(st, steps - 1));
#pragma unroll
    for (int i = 0; i < 4; ++i) tl.st[i] = a.tool_scale[min(t0 + 4 * grp + i, a.n_tools - 1)];
  };
  auto compute_tile = [&](int t0, const Tile &tl) {
    i32x4 acc[SPW];
#pragma unroll
    for (int s = 0; s < SPW; ++s) acc[s] = i32x4{0, 0, 0, 0};
#pragma unroll
    for (int st = 0; st < MAXS; ++st) {
      if (st < steps) {
#pragma unroll
        for (int s = 0; s < SPW; ++s) {
          if (s < n_lists) {
            const i32x4 bv = *reinterpret_cast<const i32x4 *>(
                qs + (16 * sub_block(s) + qn) * dim + 64 * st + 16 * grp);
            acc[s] = __builtin_amdgcn_mfma_i32_16x16x64_i8(tl.a[st], bv, acc[s], 0, 0, 0);
          }
        }
      }
    }
    // lane: tools t0 + 4 grp + i for query column qn.  A candidate that does not beat the
    // column's floor (the best KT-th entry among the column's 4 lanes, so at most the column's
    // KT-th best) cannot be among its best KT and is dropped.
#pragma unroll
    for (int s = 0; s < SPW; ++s) {
      if (s < n_lists) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = t0 + 4 * grp + i;
          const float score = ((float)acc[s][i] * tl.st[i]) * sq[s];
          const uint64_t key = t < t_end ? cand_key(score, t) : 0;
          insert<KT>(best[s], key > floor_key[s] ? key : 0);
        }
        uint64_t f = best[s][KT - 1];
        uint64_t o = shfl_xor_u64(f, 16);
        f = o > f ? o : f;
        o = shfl_xor_u64(f, 32);
        floor_key[s] = o > f ? o : f;
      }
    }
  };

  // this wave's 16-tool tiles: t_begin + 16 (slot + n_slots j)
  {
    const int stride = 16 * n_slots;
    Tile b0, b1;
    int t0 = t_begin + 16 * slot;
    if (t0 < t_end) {
      load_tile(t0, b0);
      for (;;) {
        load_tile(t0 + stride, b1);
        compute_tile(t0, b0);
        t0 += stride;
        if (t0 >= t_end) break;
        load_tile(t0 + stride, b0);
        compute_tile(t0, b1);
        t0 += stride;
        if (t0 >= t_end) break;
      }
    }
  }

  // each column's 4 lists inside the wave, then the sub-block's other waves through LDS
#pragma unroll
  for (int s = 0; s < SPW; ++s) {
    if (s < n_lists) {
      merge_lanes<KT>(best[s], 16);
      merge_lanes<KT>(best[s], 32);
    }
  }
  __syncthreads();                                                     // query block no longer read
  uint64_t *cl = reinterpret_cast<uint64_t *>(smem);                   // [wave][SPW][16][KT]
  if (slot > 0 && grp == 0)
#pragma unroll
    for (int s = 0; s < SPW; ++s)
      if (s < n_lists)
#pragma unroll
        for (int j = 0; j < KT; ++j) cl[((wave * SPW + s) * 16 + qn) * KT + j] = best[s][j];
  __syncthreads();
  if (slot > 0 || grp != 0) return;
#pragma unroll
  for (int s = 0; s < SPW; ++s) {
    if (s >= n_lists) break;
    const int q = q0 + 16 * sub_block(s) + qn;
    if (q >= a.n_queries) continue;
    // the other waves on this sub-block: SPW = 1, waves wave + nsb, ...; SPW = 4, waves 1 .. 3
    for (int w = SPW == 1 ? wave + nsb : 1; w < kWaves; w += SPW == 1 ? nsb : 1)
#pragma unroll
      for (int j = 0; j < KT; ++j) {
        uint64_t x = cl[((w * SPW + s) * 16 + qn) * KT + j];
#pragma unroll
        for (int m = 0; m < KT; ++m) {
          const bool gt = x > best[s][m];
          const uint64_t hi = gt ? x : best[s][m];
          x = gt ? best[s][m] : x;
          best[s][m] = hi;
        }
      }
    if (a.n_ranges == 1) {
#pragma unroll
      for (int j = 0; j < KT; ++j)
        if (j < a.k) {
          a.top_idx[(size_t)q * a.k + j] = cand_idx(best[s][j]);
          a.top_score[(size_t)q * a.k + j] = cand_score(best[s][j]);
        }
      const float m =
          best[s][1] == 0 ? INFINITY : cand_score(best[s][0]) - cand_score(best[s][1]);
      a.margin[q] = m;
      a.route[q] = m > a.tau ? 1 : 0;
    } else {
      const size_t o = ((size_t)q * a.n_ranges + range) * KT;
#pragma unroll
      for (int j = 0; j < KT; ++j) a.part[o + j] = best[s][j];
    }
  }
}

// One wave per query: the best KT of the ranges' lists, then the gate.
template <int KT>
__global__ __launch_bounds__(64) void slb_merge_kernel(SlbArgs a) {
  const int q = blockIdx.x, lane = threadIdx.x;
  uint64_t f[KT];
  wave_select<KT>(a.part + (size_t)q * a.n_ranges * KT, a.n_ranges * KT, lane, f);
  write_final<KT>(a, q, f, lane);
}

// Symmetric per-row INT8 quantisation: one wave per row; scale = max |x| / 127, code =
// x / scale rounded to nearest-even (IEEE fp32 division), |code| <= 127; a zero row gets scale 0.
__global__ __launch_bounds__(256) void slb_quantize_kernel(const float *x, int32_t n, int32_t dim,
                                                           int8_t *q, float *scale) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const float *xr = x + (size_t)row * dim;
  float m = 0.f;
  for (int j = lane; j < dim; j += 64) m = fmaxf(m, fabsf(xr[j]));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  const float s = m / 127.0f;
  if (lane == 0) scale[row] = s;
  int8_t *qr = q + (size_t)row * dim;
  for (int j = lane; j < dim; j += 64) {
    float c = s > 0.f ? rintf(xr[j] / s) : 0.f;
    c = fminf(fmaxf(c, -127.f), 127.f);
    qr[j] = (int8_t)(int)c;
  }
}

}  // namespace

void slb_geometry(int32_t n_tools, int32_t n_queries, int32_t dim, int32_t &n_ranges,
                  int32_t &range_tools) {
  (void)dim;
  const int qb = 16 * kSubBlocks;
  const int64_t q_blocks = ((int64_t)n_queries + qb - 1) / qb;
  const int64_t tiles = ((int64_t)n_tools + 63) / 64;                 // 64-tool units
  // about 1024 workgroups, at least 256 tools per range, at most 256 ranges (the merge reads
  // 8 candidates of each)
  int64_t nr = (1024 + q_blocks - 1) / q_blocks;
  const int64_t max_nr = (tiles + 3) / 4;
  if (nr > max_nr) nr = max_nr;
  if (nr > 256) nr = 256;
  if (nr < 1) nr = 1;
  const int64_t per = (tiles + nr - 1) / nr;
  range_tools = (int32_t)(per * 64);
  n_ranges = (int32_t)((n_tools + range_tools - 1) / range_tools);
}

size_t slb_workspace_bytes(int32_t n_tools, int32_t n_queries, int32_t dim) {
  int32_t nr, rt;
  slb_geometry(n_tools, n_queries, dim, nr, rt);
  if (nr <= 1) return 0;
  return (size_t)n_queries * nr * kTop * sizeof(uint64_t);
}

hipError_t launch_slb_quantize(const float *x, int32_t n, int32_t dim, int8_t *q, float *scale,
                               hipStream_t stream) {
  hipLaunchKernelGGL(slb_quantize_kernel, dim3((n + 3) / 4), dim3(256), 0, stream, x, n, dim, q,
                     scale);
  return hipGetLastError();
}

hipError_t launch_slb_scan(const SlbLaunch &p, hipStream_t stream) {
  SlbArgs a{};
  a.tools = p.tools;
  a.tool_scale = p.tool_scale;
  a.queries = p.queries;
  a.query_scale = p.query_scale;
  a.n_tools = p.n_tools;
  a.n_queries = p.n_queries;
  a.dim = p.dim;
  a.k = p.k;
  a.tau = p.tau;
  a.top_idx = p.top_idx;
  a.top_score = p.top_score;
  a.margin = p.margin;
  a.route = p.route;
  slb_geometry(p.n_tools, p.n_queries, p.dim, a.n_ranges, a.range_tools);
  if (a.n_ranges > 1) a.part = reinterpret_cast<uint64_t *>(p.workspace);
  const int qb = 16 * kSubBlocks;
  const dim3 grid(a.n_ranges, (p.n_queries + qb - 1) / qb);
  const size_t stage = (size_t)qb * p.dim;
  const size_t merge = (size_t)kWaves * kSubBlocks * 16 * kTop * 8;
  const size_t lds = stage > merge ? stage : merge;
  const int steps = p.dim / 64;
  const int kt = p.k <= 2 ? 2 : p.k <= 4 ? 4 : 8;
  // up to 8 query blocks: each wave owns a sub-block; more: the waves share tool tiles (measured:
  // 256 queries x 65536 tools 128 us against 156 us; 4096 queries 964 us against 1402 us)
  const bool shared = p.n_queries > 8 * qb;
#define NEXUS_SLB(S_, K_)                                                                     \
  do {                                                                                        \
    if (shared) hipLaunchKernelGGL((slb_scan_kernel<S_, K_, 4>), grid, dim3(256), lds, stream, a); \
    else hipLaunchKernelGGL((slb_scan_kernel<S_, K_, 1>), grid, dim3(256), lds, stream, a);        \
  } while (0)
#define NEXUS_SLB_S(K_)                      \
  do {                                       \
    if (steps <= 4) NEXUS_SLB(4, K_);        \
    else if (steps <= 8) NEXUS_SLB(8, K_);   \
    else if (steps <= 12) NEXUS_SLB(12, K_); \
    else NEXUS_SLB(16, K_);                  \
  } while (0)
  if (kt == 2) NEXUS_SLB_S(2);
  else if (kt == 4) NEXUS_SLB_S(4);
  else NEXUS_SLB_S(8);
#undef NEXUS_SLB_S
#undef NEXUS_SLB
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_ranges <= 1) return e;
  if (kt == 2) hipLaunchKernelGGL(slb_merge_kernel<2>, dim3(p.n_queries), dim3(64), 0, stream, a);
  else if (kt == 4) hipLaunchKernelGGL(slb_merge_kernel<4>, dim3(p.n_queries), dim3(64), 0, stream, a);
  else hipLaunchKernelGGL(slb_merge_kernel<8>, dim3(p.n_queries), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace nexus
