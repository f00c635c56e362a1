// Semantic Lookaside Buffer scan on MI355X (Sec. V-A): INT8 tool embeddings scanned with integer
// dot products against INT8 query embeddings, the best tools per query kept, and the margin gate
// (auto-route when the top-two score margin exceeds tau, else escalate).
//
// Score of tool t for query q: (float(dot_int32(T_t, Q_q)) * s_t) * s_q in fp32, each product
// rounded to nearest-even; the integer dot is exact and, with |dot| <= 127^2 * 1024 < 2^24,
// exactly representable in fp32.
//
// Scan kernel: a workgroup takes a block of 64 queries and a range of tools.  The query block
// sits in LDS; each of the 4 waves takes 16-tool tiles of the range in turn and computes
// S^T = T.Q^T on v_mfma_i32_16x16x64_i8 (tool rows straight from global memory in the A-operand
// layout, one MFMA chain per 16-query sub-block, B operands from LDS), loading the next tile
// while it computes the current one.  Lane l
// then holds tools 4 (l / 16) .. +3 of the tile for query column l % 16 of each sub-block and
// folds them into its own sorted list of the best 8 (higher score first, lower index first among
// equal scores; a lane sees its tools in increasing index order, so a strict comparison keeps the
// earlier of equal scores).  The 16 lists of every query (4 lane groups x 4 waves) are merged
// through LDS by one wave per query: 8 rounds of a wave-wide arg-max.  With one tool range the
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

// (score, index) order: a before b when a.score > b.score, or equal scores and a.idx < b.idx;
// index -1 (no tool) is last.
__device__ __forceinline__ bool better(float sa, int ia, float sb, int ib) {
  if (ib < 0) return ia >= 0;
  if (ia < 0) return false;
  return sa > sb || (sa == sb && ia < ib);
}

// Insert (s, i) into the sorted list (best first) if it beats the last entry.
__device__ __forceinline__ void insert(float (&bs)[kTop], int (&bi)[kTop], float s, int i) {
  if (!better(s, i, bs[kTop - 1], bi[kTop - 1])) return;
#pragma unroll
  for (int j = kTop - 1; j > 0; --j) {
    const bool shift = better(s, i, bs[j - 1], bi[j - 1]);
    const bool here = !shift && better(s, i, bs[j], bi[j]);
    const float ns = shift ? bs[j - 1] : (here ? s : bs[j]);
    const int ni = shift ? bi[j - 1] : (here ? i : bi[j]);
    bs[j] = ns;
    bi[j] = ni;
  }
  if (better(s, i, bs[0], bi[0])) {
    bs[0] = s;
    bi[0] = i;
  }
}

// Wave-wide best of one (score, index) per lane; every lane gets the winner.
__device__ __forceinline__ void wave_best(float &s, int &i) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float os = __shfl_xor(s, off);
    const int oi = __shfl_xor(i, off);
    if (better(os, oi, s, i)) {
      s = os;
      i = oi;
    }
  }
}

// The best kTop of n candidates (cs, ci) (n <= 64 * kTop), selected by one wave: every lane
// holds up to kTop candidates as a sorted list; kTop rounds take the wave-wide best head.
__device__ __forceinline__ void wave_select(const float *cs, const int *ci, int n, int lane,
                                            float (&out_s)[kTop], int (&out_i)[kTop]) {
  float bs[kTop];
  int bi[kTop];
#pragma unroll
  for (int j = 0; j < kTop; ++j) {
    bs[j] = -INFINITY;
    bi[j] = -1;
  }
  for (int c = lane; c < n; c += 64) insert(bs, bi, cs[c], ci[c]);
  int head = 0;
#pragma unroll
  for (int r = 0; r < kTop; ++r) {
    float hs = -INFINITY;
    int hi = -1;
#pragma unroll
    for (int j = 0; j < kTop; ++j)
      if (j == head) {
        hs = bs[j];
        hi = bi[j];
      }
    float ws = hs;
    int wi = hi;
    wave_best(ws, wi);
    out_s[r] = ws;
    out_i[r] = wi;
    if (wi >= 0 && hi == wi) ++head;   // indices are distinct: only the winner's lane advances
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
  float *part_s;                      // [n_queries][n_ranges][kTop]
  int32_t *part_i;
};

// Final outputs of one query from its sorted best list (lane 0 writes).
__device__ __forceinline__ void write_final(const SlbArgs &a, int q, const float (&s)[kTop],
                                            const int (&i)[kTop], int lane) {
  if (lane != 0) return;
#pragma unroll
  for (int j = 0; j < kTop; ++j)
    if (j < a.k) {
      a.top_idx[(size_t)q * a.k + j] = i[j];
      a.top_score[(size_t)q * a.k + j] = s[j];
    }
  // fewer than two tools: nothing to confuse the best one with
  const float m = i[1] < 0 ? INFINITY : s[0] - s[1];
  a.margin[q] = m;
  a.route[q] = m > a.tau ? 1 : 0;
}

template <int MAXS>   // 64-byte steps of dim at most (dim <= 64 * MAXS)
__global__ __launch_bounds__(256) void slb_scan_kernel(SlbArgs a) {
  constexpr int NSB = kSubBlocks;
  constexpr int QB = 16 * NSB;
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

  // stage the query block (rows past n_queries are zero)
  for (int c = tid; c < QB * (dim / 16); c += 256) {
    const int r = c / (dim / 16), off = (c - r * (dim / 16)) * 16;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (q0 + r < a.n_queries)
      v = *reinterpret_cast<const u32x4 *>(a.queries + (size_t)(q0 + r) * dim + off);
    *reinterpret_cast<u32x4 *>(qs + r * dim + off) = v;
  }
  float sq[NSB];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    const int q = q0 + 16 * sb + qn;
    sq[sb] = q < a.n_queries ? a.query_scale[q] : 0.f;
  }
  __syncthreads();

  float bs[NSB][kTop];
  int bi[NSB][kTop];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
    for (int j = 0; j < kTop; ++j) {
      bs[sb][j] = -INFINITY;
      bi[sb][j] = -1;
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
    for (int s = 0; s < MAXS; ++s)
      tl.a[s] = *reinterpret_cast<const i32x4 *>(trow + 64 * min(s, steps - 1));
#pragma unroll
    for (int i = 0; i < 4; ++i) tl.st[i] = a.tool_scale[min(t0 + 4 * grp + i, a.n_tools - 1)];
  };
  auto compute_tile = [&](int t0, const Tile &tl) {
    i32x4 acc[NSB];
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb) acc[sb] = i32x4{0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < MAXS; ++s) {
      if (s < steps) {
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb) {
          const i32x4 bv =
              *reinterpret_cast<const i32x4 *>(qs + (16 * sb + qn) * dim + 64 * s + 16 * grp);
          acc[sb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(tl.a[s], bv, acc[sb], 0, 0, 0);
        }
      }
    }
    // lane: tools t0 + 4 grp + i, query column qn of each sub-block
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = t0 + 4 * grp + i;
      if (t < t_end) {
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb)
          insert(bs[sb], bi[sb], ((float)acc[sb][i] * tl.st[i]) * sq[sb], t);
      }
    }
  };

  // this wave's 16-tool tiles of the range: t_begin + 16 wave + 64 j
  {
    Tile b0, b1;
    int t0 = t_begin + 16 * wave;
    if (t0 < t_end) {
      load_tile(t0, b0);
      for (;;) {
        load_tile(t0 + 16 * kWaves, b1);
        compute_tile(t0, b0);
        t0 += 16 * kWaves;
        if (t0 >= t_end) break;
        load_tile(t0 + 16 * kWaves, b0);
        compute_tile(t0, b1);
        t0 += 16 * kWaves;
        if (t0 >= t_end) break;
      }
    }
  }

  // merge the 16 lists of each query (4 lane groups x 4 waves) through LDS
  __syncthreads();                                                     // query block no longer read
  float *cs = reinterpret_cast<float *>(smem);                         // [QB][16][kTop]
  int *ci = reinterpret_cast<int *>(smem + QB * 16 * kTop * 4);
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
    for (int j = 0; j < kTop; ++j) {
      const int slot = ((16 * sb + qn) * 16 + wave * 4 + grp) * kTop + j;
      cs[slot] = bs[sb][j];
      ci[slot] = bi[sb][j];
    }
  __syncthreads();
  for (int ql = wave; ql < QB; ql += kWaves) {
    const int q = q0 + ql;
    if (q >= a.n_queries) break;
    float fs[kTop];
    int fi[kTop];
    wave_select(cs + ql * 16 * kTop, ci + ql * 16 * kTop, 16 * kTop, lane, fs, fi);
    if (a.n_ranges == 1) {
      write_final(a, q, fs, fi, lane);
    } else if (lane == 0) {
      const size_t o = ((size_t)q * a.n_ranges + range) * kTop;
#pragma unroll
      for (int j = 0; j < kTop; ++j) {
        a.part_s[o + j] = fs[j];
        a.part_i[o + j] = fi[j];
      }
    }
  }
}

// One wave per query: the best kTop of the ranges' lists, then the gate.
__global__ __launch_bounds__(64) void slb_merge_kernel(SlbArgs a) {
  const int q = blockIdx.x, lane = threadIdx.x;
  const size_t o = (size_t)q * a.n_ranges * kTop;
  float fs[kTop];
  int fi[kTop];
  wave_select(a.part_s + o, a.part_i + o, a.n_ranges * kTop, lane, fs, fi);
  write_final(a, q, fs, fi, lane);
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
  const int qb = 16 * kSubBlocks;
  const int64_t q_blocks = ((int64_t)n_queries + qb - 1) / qb;
  const int64_t tiles = ((int64_t)n_tools + 63) / 64;                 // 64-tool units
  // about 512 workgroups, at least 1024 tools per range, at most 64 ranges (merge width)
  int64_t nr = (512 + q_blocks - 1) / q_blocks;
  const int64_t max_nr = (tiles + 15) / 16;
  if (nr > max_nr) nr = max_nr;
  if (nr > 64) nr = 64;
  if (nr < 1) nr = 1;
  const int64_t per = (tiles + nr - 1) / nr;
  range_tools = (int32_t)(per * 64);
  n_ranges = (int32_t)((n_tools + range_tools - 1) / range_tools);
}

size_t slb_workspace_bytes(int32_t n_tools, int32_t n_queries, int32_t dim) {
  int32_t nr, rt;
  slb_geometry(n_tools, n_queries, dim, nr, rt);
  if (nr <= 1) return 0;
  return (size_t)n_queries * nr * kTop * (sizeof(float) + sizeof(int32_t));
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
  if (a.n_ranges > 1) {
    a.part_s = reinterpret_cast<float *>(p.workspace);
    a.part_i = reinterpret_cast<int32_t *>(a.part_s + (size_t)p.n_queries * a.n_ranges * kTop);
  }
  const int qb = 16 * kSubBlocks;
  const dim3 grid(a.n_ranges, (p.n_queries + qb - 1) / qb);
  const size_t stage = (size_t)qb * p.dim;
  const size_t merge = (size_t)qb * 16 * kTop * 8;
  const size_t lds = stage > merge ? stage : merge;
  const int steps = p.dim / 64;
  if (steps <= 4) hipLaunchKernelGGL(slb_scan_kernel<4>, grid, dim3(256), lds, stream, a);
  else if (steps <= 8) hipLaunchKernelGGL(slb_scan_kernel<8>, grid, dim3(256), lds, stream, a);
  else if (steps <= 12) hipLaunchKernelGGL(slb_scan_kernel<12>, grid, dim3(256), lds, stream, a);
  else hipLaunchKernelGGL(slb_scan_kernel<16>, grid, dim3(256), lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_ranges <= 1) return e;
  hipLaunchKernelGGL(slb_merge_kernel, dim3(p.n_queries), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace nexus
