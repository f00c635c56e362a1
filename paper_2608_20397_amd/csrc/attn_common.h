// Shared definitions of the bf16 suffix-attention kernels (internal, not part of the C ABI).
#pragma once

#include "device_common.h"

namespace nexus {

constexpr int kMaxSeqs = 32;
constexpr int kWaves = 4;   // wave tasks per workgroup of the 32-query kernels
constexpr int kWavesWide = 8;   // wave tasks per workgroup of the head_dim-256 transposed-V kernel
constexpr int kQB = 32;     // queries per wave task of the 32-query kernels
constexpr int kMaxSplitKeys = 32768;   // keys one workgroup covers at most (LDS page table)

struct SeqPlan {
  int32_t q_start;     // first row of q / out
  int32_t len;         // queries
  int64_t n_past;      // position of the first query
  int32_t row_begin;   // prefix sum of len over sequences (combine indexing)
  int32_t first_unit;  // first (task group, split) unit of this sequence
  int32_t n_tasks;     // group * ceil(len / queries per task)
  int32_t n_tg;        // task groups: ceil(n_tasks / tasks per workgroup)
  int32_t n_splits;
  int32_t split_keys;  // keys per split, a multiple of the key tile
  int32_t longest_first;  // dispatch task groups last-first (causal prefill: n_past < len)
  int64_t ws_off;      // byte offset of the fp16 partial rows of this sequence in the workspace
  int64_t ml_off;      // byte offset of their {m, l, l 2^e, 0} records (16-byte aligned)
  // Two split classes: the first n_tg_a task groups in dispatch order take n_splits splits of
  // split_keys keys, the others n_splits_b splits of split_keys_b (a finer cut that fills the
  // last round of workgroups).  One class: n_tg_a = all groups, class b equal to class a.
  int32_t n_tg_a;
  int32_t n_splits_b;
  int32_t split_keys_b;
  int32_t max_splits;  // partial slots per row in the workspace: max(n_splits, n_splits_b)
};

// Work of unit `u` (counted from the sequence's first unit): task group, split, its first key,
// the split length and the group's split count.
struct UnitWork {
  int tgrp, split, k_begin, split_keys, n_splits;
};
__host__ __device__ __forceinline__ UnitWork unit_work(const SeqPlan &sp, int u) {
  UnitWork w;
  const int ua = sp.n_tg_a * sp.n_splits;
  int di;   // dispatch index of the task group
  if (u < ua) {
    di = u / sp.n_splits;
    w.split = u - di * sp.n_splits;
    w.split_keys = sp.split_keys;
    w.n_splits = sp.n_splits;
  } else {
    const int ub = u - ua;
    const int dib = ub / sp.n_splits_b;
    di = sp.n_tg_a + dib;
    w.split = ub - dib * sp.n_splits_b;
    w.split_keys = sp.split_keys_b;
    w.n_splits = sp.n_splits_b;
  }
  // prefill-like sequences take their task groups in reverse: later queries see more keys, so
  // the longest workgroups are dispatched first and the launch does not end on them
  w.tgrp = sp.longest_first ? sp.n_tg - 1 - di : di;
  w.k_begin = w.split * w.split_keys;
  return w;
}
// Split count of task group `tgrp`.
__host__ __device__ __forceinline__ int group_splits(const SeqPlan &sp, int tgrp) {
  const int di = sp.longest_first ? sp.n_tg - 1 - tgrp : tgrp;
  return di < sp.n_tg_a ? sp.n_splits : sp.n_splits_b;
}

// Several sequences share the cache prefix (blocks spliced into one context): their units are
// taken key range by key range, so that the workgroups resident together read the same keys.
// Split r of every sequence covers keys [r * split_keys, (r + 1) * split_keys) (one split
// length for all); range r holds, for each sequence with more than r splits (a prefix of the
// sequences ordered by decreasing key count), all its task groups.
constexpr int kMaxRanges = 64;

struct AttnPlan {
  SeqPlan seq[kMaxSeqs];
  int32_t n_seqs;
  int32_t qpw;                                // queries per wave task
  int32_t waves;                              // wave tasks per workgroup
  int32_t units_per_head;
  int32_t total_rows;
  int32_t any_split;
  size_t ws_bytes;
  int32_t range_major;                        // 0: units sequence by sequence (first_unit,
                                              // sequences in the order of `order`)
  int32_t n_ranges;
  int32_t range_first_unit[kMaxRanges + 1];   // first unit of each key range
  int32_t order[kMaxSeqs];                    // range-major: sequences by decreasing key
                                              // count; else the dispatch order
  int32_t tg_prefix[kMaxSeqs + 1];            // task groups of order[0 .. i - 1]
};

// Sequence and work of unit `unit` of a launch (one KV head's units).
struct UnitLoc {
  int seq;
  UnitWork w;
};
__host__ __device__ __forceinline__ UnitLoc locate_unit(const AttnPlan &plan, int unit) {
  UnitLoc loc;
  if (!plan.range_major) {
    // sequences in dispatch order (plan.order): their first units increase along it
    int i = 0;
    while (i + 1 < plan.n_seqs && unit >= plan.seq[plan.order[i + 1]].first_unit) ++i;
    const int b = plan.order[i];
    loc.seq = b;
    loc.w = unit_work(plan.seq[b], unit - plan.seq[b].first_unit);
    return loc;
  }
  int lo = 0, hi = plan.n_ranges;             // range_first_unit[lo] <= unit < [hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (unit >= plan.range_first_unit[mid]) lo = mid;
    else hi = mid;
  }
  const int local = unit - plan.range_first_unit[lo];
  int i0 = 0, i1 = plan.n_seqs;               // tg_prefix[i0] <= local < tg_prefix[i1]
  while (i1 - i0 > 1) {
    const int mid = (i0 + i1) >> 1;
    if (local >= plan.tg_prefix[mid]) i0 = mid;
    else i1 = mid;
  }
  const int b = plan.order[i0];
  const int di = local - plan.tg_prefix[i0];
  loc.seq = b;
  loc.w.tgrp = plan.seq[b].longest_first ? plan.seq[b].n_tg - 1 - di : di;
  loc.w.split = lo;
  loc.w.split_keys = plan.seq[b].split_keys;
  loc.w.n_splits = plan.seq[b].n_splits;
  loc.w.k_begin = lo * plan.seq[b].split_keys;
  return loc;
}

struct AttnArgs {
  const uint16_t *q;
  uint16_t *out;
  const uint16_t *kc;   // layer base of the K cache
  const uint16_t *vc;   // layer base of the V cache
  const int32_t *map;
  char *ws;             // split partials: fp16 rows at SeqPlan::ws_off, records at ml_off
  int32_t n_q_heads, n_kv_heads, group, n_phys_pages;
  float scale_log2;     // scale * log2(e)
  float cap_in;         // scale / softcap
  float cap_out;        // softcap * log2(e)
  float cap_k;          // 2 * scale * log2(e) / softcap
};

__device__ __forceinline__ float tanh_fast(float x) {
  // tanh x = 1 - 2 / (e^{2x} + 1); exp2 overflow to +inf gives 1, underflow to 0 gives -1.
  const float e = fast_exp2(x * 2.8853900817779268f);  // 2 / ln 2
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(e + 1.0f);
}

// The soft cap through r = 1 / (2^(s cap_k) + 1): tanh(s scale / cap) = 1 - 2 r, so the capped
// score in log2 units is cap_out (1 - 2 r), decreasing in r (2^.. overflowing to +inf gives
// r = 0, the cap itself; underflowing to 0 gives r = 1).
__device__ __forceinline__ float cap_r(float s, float cap_k) {
  return __builtin_amdgcn_rcpf(fast_exp2(s * cap_k) + 1.0f);
}

// Split-K partial of one output row (query, head) of the bf16 kernels, from the lane pair
// (j, j + 32) that holds the row: its O / l as fp16, scaled by 2^-e so that the row's largest
// magnitude lies in [2^14, 2^15), and the record {m, l, l 2^e, 0} that the combine weighs it
// with.  fp16 keeps 11 significant bits over the scaled range (the final output is bf16, 8
// bits); the power-of-two scale keeps any finite V in range and costs no rounding.
// part_scale: the factor that maps O to the stored values, and l 2^e in `c`.  Every lane of the
// wave calls it (cross-lane maximum); `amax` is the lane's largest |O| over its features.
__device__ __forceinline__ float part_scale(float amax, float l_tot, float &c) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(amax), __float_as_uint(amax),
                                                  false, false);
  amax = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  const float rmax = amax * inv;
  int e = 0;
  if (rmax > 0.f && rmax <= 3.0e38f)
    e = min(max((int)((__float_as_uint(rmax) >> 23) & 0xff) - 127 - 14, -100), 100);
  c = l_tot * __uint_as_float((uint32_t)(127 + e) << 23);
  return inv * __uint_as_float((uint32_t)(127 - e) << 23);
}
template <int NDB>
__device__ __forceinline__ float row_amax(const f32x16 (&o)[NDB]) {
  float m = 0.f;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) m = fmaxf(m, fabsf(o[db][v]));
  return m;
}
// Stores the lane's features of the row: feature 32 db + 8 gq + 4 hh + i holds o[db][4 gq + i]
// (the 32x32 MFMA accumulator layout of O^T), and the record from lane half 0.
template <int NDB, int D>
__device__ __forceinline__ void store_partial(const f32x16 (&o)[NDB], float sc, float m_ref,
                                              float l_tot, float c, int hh, char *ws,
                                              const SeqPlan &sp, int64_t prow) {
  uint16_t *op = reinterpret_cast<uint16_t *>(ws + sp.ws_off) + prow * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int d0 = 32 * db + 8 * gq + 4 * hh;
      *reinterpret_cast<u32x2 *>(op + d0) =
          u32x2{pack_f16x2(o[db][4 * gq + 0] * sc, o[db][4 * gq + 1] * sc),
                pack_f16x2(o[db][4 * gq + 2] * sc, o[db][4 * gq + 3] * sc)};
    }
  if (hh == 0)
    *reinterpret_cast<f32x4 *>(ws + sp.ml_off + prow * 16) = f32x4{m_ref, l_tot, c, 0.f};
}

// key index within a 16-key group -> its position in the V^T tile (swap bits 2 and 3)
__device__ __forceinline__ int vt_pos(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

// V^T tile row swizzle: 16-byte chunk c of feature row d lives at chunk c ^ vt_swz(d).  Distinct
// for 8 consecutive rows (conflict-free operand reads) and for rows 8 apart (tile writes).
template <int VSW>
__device__ __forceinline__ int vt_swz(int d) {
  return (d ^ (d >> 3)) & VSW;
}


}  // namespace nexus
