// Semantic Lookaside Buffer scan on MI355X (Sec. V-A): INT8 tool embeddings scanned with integer
// dot products against INT8 query embeddings, the best tools per query kept, and the margin gate
// (auto-route when the top-two score margin exceeds tau, else escalate).
//
// Score of tool t for query q: (float(dot_int32(T_t, Q_q)) * s_t) * s_q in fp32, each product
// rounded to nearest-even; the integer dot is exact and, with |dot| <= 127^2 * 1024 < 2^24,
// exactly representable in fp32.
//
// Both scan kernels compute S^T = T.Q^T on v_mfma_i32_16x16x64_i8 (tool rows straight from
// global memory into the A-operand registers, the query block staged in LDS as the B operands),
// loading ahead while they compute.  Lane l then holds tools 4 (l / 16) .. +3 of a 16-tool tile
// for query column l % 16 and folds them into its own sorted list of the best KT (higher score
// first, lower index first among equal scores: both orders are carried by one 64-bit key, so
// the list update is a branch-free max/min pass).  A column's 4 lane lists are merged by lane
// exchanges and the 4 waves' lists through LDS.  With one tool range the result is final
// (top-k, margin, gate); otherwise each range's best 8 go to the workspace and a second kernel
// merges them the same way.
//
// * Up to 16 queries (the single-query lookup of a user turn): one 16-query block; the waves
//   take the range's 16-tool tiles in turn, each tile one MFMA chain.  HBM-bound for one query.
// * More queries: a workgroup holds 64 queries and its 4 waves take 64-tool blocks of the range
//   in turn; for one block a wave keeps 16 MFMA chains (4 tool tiles x 4 query sub-blocks) and
//   walks the dimension two 64-byte steps at a time, holding those steps of its 64 tool rows in
//   registers (the next two in flight), so every B operand read from LDS feeds four MFMAs and
//   every tool row is read once per workgroup.
#include "device_common.h"
#include "launch_slb.h"

namespace nexus {

namespace {

typedef __attribute__((ext_vector_type(4))) int i32x4;

constexpr int kTop = 8;          // candidates kept per (lane, query) and per range
constexpr int kWaves = 4;
constexpr int kSubBlocks = 4;    // 16-query sub-blocks per workgroup (64 queries)
// LDS row padding of the staged query block: dim is a multiple of 64 bytes, so unpadded rows
// start on the same bank and the 16 rows an MFMA B operand reads would all hit the same 4 banks
constexpr int kQPad = 16;

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

// A lower bound of the KT-th best key of a query column whose candidates are spread over 4 lane
// lists (lanes l, l ^ 16, l ^ 32, l ^ 48), each sorted descending: the largest of the lanes'
// KT-th entries, and the smallest of the lanes' (KT/4)-th entries (every lane then holds at least
// KT/4 keys at or above it, KT in all).  The second is the tight one while the lists are short
// of candidates of their own: after the first tile or block it sits near the column's KT-th best.
template <int KT>
__device__ __forceinline__ uint64_t column_floor(const uint64_t (&b)[KT]) {
  uint64_t f = b[KT - 1];
  uint64_t g = b[KT >= 4 ? KT / 4 - 1 : 0];
  uint64_t o = shfl_xor_u64(f, 16);
  f = o > f ? o : f;
  o = shfl_xor_u64(f, 32);
  f = o > f ? o : f;
  o = shfl_xor_u64(g, 16);
  g = o < g ? o : g;
  o = shfl_xor_u64(g, 32);
  g = o < g ? o : g;
  return f > g ? f : g;
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

// Small batches (at most 16 queries: one 16-query block, the single-query lookup of a user turn).
// MAXS: 64-byte steps of dim at most (dim <= 64 MAXS); KT: candidates kept, >= max(k, 2).  The
// query block sits in LDS; wave w takes the range's 16-tool tiles w, w + 4, ..., loading each
// tile's rows straight into the A-operand registers (the next tile in flight) and running one
// MFMA chain per tile; the 4 waves' lists of a query meet in LDS.
template <int MAXS, int KT>
__global__ __launch_bounds__(256) void slb_scan_kernel(SlbArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  int8_t *qs = reinterpret_cast<int8_t *>(smem);                       // [16][dim + kQPad]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qn = lane & 15, grp = lane >> 4;
  const int range = blockIdx.x;
  const int t_begin = range * a.range_tools;
  const int t_end = min(t_begin + a.range_tools, a.n_tools);
  const int dim = a.dim, steps = dim / 64, ld = dim + kQPad;

  // stage the query block (rows past n_queries are zero)
  for (int c = tid; c < 16 * (dim / 16); c += 256) {
    const int r = c / (dim / 16), off = (c - r * (dim / 16)) * 16;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (r < a.n_queries) v = *reinterpret_cast<const u32x4 *>(a.queries + (size_t)r * dim + off);
    *reinterpret_cast<u32x4 *>(qs + r * ld + off) = v;
  }
  const float sq = qn < a.n_queries ? a.query_scale[qn] : 0.f;
  __syncthreads();

  uint64_t best[KT];
  uint64_t floor_key = 0;   // a lower bound of the KT-th best key of this lane's query column
#pragma unroll
  for (int j = 0; j < KT; ++j) best[j] = 0;

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
    i32x4 acc = i32x4{0, 0, 0, 0};
#pragma unroll
    for (int st = 0; st < MAXS; ++st) {
      if (st < steps) {
        const i32x4 bv = *reinterpret_cast<const i32x4 *>(qs + qn * ld + 64 * st + 16 * grp);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(tl.a[st], bv, acc, 0, 0, 0);
      }
    }
    // lane: tools t0 + 4 grp + i for query column qn.  A candidate that does not beat the
    // column's floor (at most the column's KT-th best) cannot be among its best KT and is
    // dropped.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = t0 + 4 * grp + i;
      const float score = ((float)acc[i] * tl.st[i]) * sq;
      const uint64_t key = t < t_end ? cand_key(score, t) : 0;
      insert<KT>(best, key > floor_key ? key : 0);
    }
    floor_key = column_floor<KT>(best);
  };

  // this wave's 16-tool tiles: t_begin + 16 (wave + 4 j)
  {
    const int stride = 16 * kWaves;
    Tile b0, b1;
    int t0 = t_begin + 16 * wave;
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

  // each column's 4 lists inside the wave, then the other waves' lists through LDS
  merge_lanes<KT>(best, 16);
  merge_lanes<KT>(best, 32);
  __syncthreads();                                                     // query block no longer read
  uint64_t *cl = reinterpret_cast<uint64_t *>(smem);                   // [wave][16][KT]
  if (wave > 0 && grp == 0)
#pragma unroll
    for (int j = 0; j < KT; ++j) cl[(wave * 16 + qn) * KT + j] = best[j];
  __syncthreads();
  if (wave > 0 || grp != 0 || qn >= a.n_queries) return;
  const int q = qn;
  for (int w = 1; w < kWaves; ++w)
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      uint64_t x = cl[(w * 16 + qn) * KT + j];
#pragma unroll
      for (int m = 0; m < KT; ++m) {
        const bool gt = x > best[m];
        const uint64_t hi = gt ? x : best[m];
        x = gt ? best[m] : x;
        best[m] = hi;
      }
    }
  if (a.n_ranges == 1) {
#pragma unroll
    for (int j = 0; j < KT; ++j)
      if (j < a.k) {
        a.top_idx[(size_t)q * a.k + j] = cand_idx(best[j]);
        a.top_score[(size_t)q * a.k + j] = cand_score(best[j]);
      }
    const float m = best[1] == 0 ? INFINITY : cand_score(best[0]) - cand_score(best[1]);
    a.margin[q] = m;
    a.route[q] = m > a.tau ? 1 : 0;
  } else {
    const size_t o = ((size_t)q * a.n_ranges + range) * KT;
#pragma unroll
    for (int j = 0; j < KT; ++j) a.part[o + j] = best[j];
  }
}

// Batched scan.  Range tool scales are staged in LDS next to the query block, so the candidate
// pass reads them without a global load.  Lane (qn, grp) loads, for tool tile i of a block,
// bytes 64 st + 16 grp of tool row 16 i + qn (the A operand of v_mfma_i32_16x16x64_i8) and reads
// bytes 64 st + 16 grp of query row 16 sb + qn from LDS (the B operand); its accumulator holds
// the scores of tools 16 i + 4 grp + r (r = 0..3) for query column 16 sb + qn.
template <int KT>
__global__ __launch_bounds__(256, 2) void slb_block_kernel(SlbArgs a) {
  constexpr int QB = 64, NT = 4, NSB = 4, CS = 2;   // queries, tool tiles, sub-blocks, steps
  extern __shared__ __align__(16) unsigned char smem[];
  const int dim = a.dim, steps = dim / 64, ld = dim + kQPad;
  int8_t *qs = reinterpret_cast<int8_t *>(smem);                         // [QB][ld]
  float *tsc = reinterpret_cast<float *>(smem + (size_t)QB * ld);        // [range_tools]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qn = lane & 15, grp = lane >> 4;
  const int q0 = blockIdx.y * QB;
  const int range = blockIdx.x;
  const int t_begin = range * a.range_tools;
  const int t_end = min(t_begin + a.range_tools, a.n_tools);

  for (int c = tid; c < QB * (dim / 16); c += 256) {
    const int r = c / (dim / 16), off = (c - r * (dim / 16)) * 16;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (q0 + r < a.n_queries)
      v = *reinterpret_cast<const u32x4 *>(a.queries + (size_t)(q0 + r) * dim + off);
    *reinterpret_cast<u32x4 *>(qs + r * ld + off) = v;
  }
  for (int i = tid; i < t_end - t_begin; i += 256) tsc[i] = a.tool_scale[t_begin + i];
  float sq[NSB];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    const int q = q0 + 16 * sb + qn;
    sq[sb] = q < a.n_queries ? a.query_scale[q] : 0.f;
  }
  __syncthreads();

  uint64_t best[NSB][KT];
  uint64_t floor_key[NSB];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    floor_key[sb] = 0;
#pragma unroll
    for (int j = 0; j < KT; ++j) best[sb][j] = 0;
  }

  // this wave's blocks: wave, wave + 4, ... of the range's 64-tool blocks; each is n_chunks
  // chunks of CS steps, walked as one sequence u = block * n_chunks + chunk
  const int n_blocks = (t_end - t_begin + 63) / 64;
  const int my_blocks = n_blocks > wave ? (n_blocks - wave + kWaves - 1) / kWaves : 0;
  const int n_chunks = (steps + CS - 1) / CS;
  const int total = my_blocks * n_chunks;
  struct Chunk {
    i32x4 a[NT][CS];
  };
  // Every call issues the same loads (past the sequence's end it re-reads the last chunk; rows
  // and steps past the registry's end re-read valid ones), so the wait before a chunk's use
  // leaves the next chunk's loads in flight.
  auto load_chunk = [&](int u, Chunk &ch) {
    const int uu = min(u, total - 1);
    const int j = uu / n_chunks, c = uu - j * n_chunks;
    const int t0 = t_begin + 64 * (wave + kWaves * j);
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      const int8_t *trow = a.tools + (size_t)min(t0 + 16 * i + qn, a.n_tools - 1) * dim + 16 * grp;
#pragma unroll
      for (int s2 = 0; s2 < CS; ++s2)
        ch.a[i][s2] = *reinterpret_cast<const i32x4 *>(trow + 64 * min(c * CS + s2, steps - 1));
    }
  };
  i32x4 acc[NT][NSB];
  auto step = [&](int u, const Chunk &ch) {
    const int j = u / n_chunks, c = u - j * n_chunks;
    if (c == 0) {
#pragma unroll
      for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb) acc[i][sb] = i32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int s2 = 0; s2 < CS; ++s2) {
      const int st = c * CS + s2;
      if (st < steps) {
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb) {
          const i32x4 bv =
              *reinterpret_cast<const i32x4 *>(qs + (16 * sb + qn) * ld + 64 * st + 16 * grp);
#pragma unroll
          for (int i = 0; i < NT; ++i)
            acc[i][sb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ch.a[i][s2], bv, acc[i][sb], 0, 0, 0);
        }
      }
    }
    if (c != n_chunks - 1) return;
    // the candidate pass runs at a raised wave priority, so that its list upkeep interleaves
    // with the other wave's MFMA chains (about 4% faster at 65536 tools x 256 queries)
    __builtin_amdgcn_s_setprio(2);
    // the block's 64 x 64 scores: a candidate that does not beat its column's floor (at most
    // the column's KT-th best) cannot be among the column's best KT and is dropped
    const int tb = 64 * (wave + kWaves * j);                   // block start within the range
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      const f32x4 sc = *reinterpret_cast<const f32x4 *>(tsc + tb + 16 * i + 4 * grp);
#pragma unroll
      for (int sb = 0; sb < NSB; ++sb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = t_begin + tb + 16 * i + 4 * grp + r;
          const float score = ((float)acc[i][sb][r] * sc[r]) * sq[sb];
          const uint64_t key = t < t_end ? cand_key(score, t) : 0;
          insert<KT>(best[sb], key > floor_key[sb] ? key : 0);
        }
      }
    }
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb) floor_key[sb] = column_floor<KT>(best[sb]);
    __builtin_amdgcn_s_setprio(0);
  };
  if (total > 0) {
    Chunk b0, b1;
    int u = 0;
    load_chunk(0, b0);
    for (;;) {
      load_chunk(u + 1, b1);
      step(u, b0);
      if (++u >= total) break;
      load_chunk(u + 1, b0);
      step(u, b1);
      if (++u >= total) break;
    }
  }

  // each column's 4 lists inside the wave, then the 4 waves' lists through LDS
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    merge_lanes<KT>(best[sb], 16);
    merge_lanes<KT>(best[sb], 32);
  }
  __syncthreads();                                        // query block and scales no longer read
  uint64_t *cl = reinterpret_cast<uint64_t *>(smem);      // [wave][NSB][16][KT]
  if (wave > 0 && grp == 0)
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
      for (int j = 0; j < KT; ++j) cl[((wave * NSB + sb) * 16 + qn) * KT + j] = best[sb][j];
  __syncthreads();
  if (wave > 0 || grp != 0) return;
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) {
    const int q = q0 + 16 * sb + qn;
    if (q >= a.n_queries) continue;
    for (int w = 1; w < kWaves; ++w)
#pragma unroll
      for (int j = 0; j < KT; ++j) {
        uint64_t x = cl[((w * NSB + sb) * 16 + qn) * KT + j];
#pragma unroll
        for (int m = 0; m < KT; ++m) {
          const bool gt = x > best[sb][m];
          const uint64_t hi = gt ? x : best[sb][m];
          x = gt ? best[sb][m] : x;
          best[sb][m] = hi;
        }
      }
    if (a.n_ranges == 1) {
#pragma unroll
      for (int j = 0; j < KT; ++j)
        if (j < a.k) {
          a.top_idx[(size_t)q * a.k + j] = cand_idx(best[sb][j]);
          a.top_score[(size_t)q * a.k + j] = cand_score(best[sb][j]);
        }
      const float m =
          best[sb][1] == 0 ? INFINITY : cand_score(best[sb][0]) - cand_score(best[sb][1]);
      a.margin[q] = m;
      a.route[q] = m > a.tau ? 1 : 0;
    } else {
      const size_t o = ((size_t)q * a.n_ranges + range) * KT;
#pragma unroll
      for (int j = 0; j < KT; ++j) a.part[o + j] = best[sb][j];
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

namespace {
// More queries than this take the batched kernel (from two 16-query sub-blocks on, a tool row
// read feeds more than one query column).
constexpr int kBlockMinQueries = 16;
constexpr int64_t kBlockWgs = 512;        // batched kernel: two resident workgroups per CU
constexpr int64_t kBlockMaxRange = 32;    // 64-tool blocks per range (its scales sit in LDS)

bool batched(int32_t n_queries) { return n_queries > kBlockMinQueries; }

size_t block_lds_bytes(int32_t dim, int32_t range_tools) {
  const size_t stage = (size_t)64 * (dim + kQPad) + (size_t)range_tools * sizeof(float);
  const size_t merge = (size_t)kWaves * kSubBlocks * 16 * kTop * 8;
  return stage > merge ? stage : merge;
}
}  // namespace

void slb_geometry(int32_t n_tools, int32_t n_queries, int32_t dim, int32_t &n_ranges,
                  int32_t &range_tools) {
  (void)dim;
  const int qb = 16 * kSubBlocks;
  if (batched(n_queries)) {
    // about kBlockWgs workgroups, 4 to kBlockMaxRange 64-tool blocks per range (at least one
    // block per wave)
    const int64_t q_blocks = ((int64_t)n_queries + qb - 1) / qb;
    const int64_t blocks = ((int64_t)n_tools + 63) / 64;
    int64_t per = (blocks * q_blocks + kBlockWgs - 1) / kBlockWgs;
    if (per < 4) per = 4;
    if (per > kBlockMaxRange) per = kBlockMaxRange;
    range_tools = (int32_t)(per * 64);
    n_ranges = (int32_t)(((int64_t)n_tools + range_tools - 1) / range_tools);
    return;
  }
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
  const int kt = p.k <= 2 ? 2 : p.k <= 4 ? 4 : 8;
  if (batched(p.n_queries)) {
    const size_t lds = block_lds_bytes(p.dim, a.range_tools);
    auto run = [&](auto kernel) -> hipError_t {
      if (lds > 65536) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 (int)lds);
        if (e != hipSuccess) return e;
      }
      hipLaunchKernelGGL(kernel, grid, dim3(256), lds, stream, a);
      return hipGetLastError();
    };
    hipError_t e = kt == 2 ? run(slb_block_kernel<2>)
                   : kt == 4 ? run(slb_block_kernel<4>)
                             : run(slb_block_kernel<8>);
    if (e != hipSuccess || a.n_ranges <= 1) return e;
    if (kt == 2) hipLaunchKernelGGL(slb_merge_kernel<2>, dim3(p.n_queries), dim3(64), 0, stream, a);
    else if (kt == 4) hipLaunchKernelGGL(slb_merge_kernel<4>, dim3(p.n_queries), dim3(64), 0, stream, a);
    else hipLaunchKernelGGL(slb_merge_kernel<8>, dim3(p.n_queries), dim3(64), 0, stream, a);
    return hipGetLastError();
  }
  // at most 16 queries: one query block
  const size_t stage = (size_t)16 * (p.dim + kQPad);
  const size_t merge = (size_t)kWaves * 16 * kTop * 8;
  const size_t lds = stage > merge ? stage : merge;
  const int steps = p.dim / 64;
#define NEXUS_SLB(S_, K_) \
  hipLaunchKernelGGL((slb_scan_kernel<S_, K_>), grid, dim3(256), lds, stream, a)
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
