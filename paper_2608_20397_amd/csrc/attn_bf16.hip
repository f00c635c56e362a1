// bf16 causal grouped-query suffix attention on gfx950 MFMA (Sec. III-A; the re-decoded suffix
// of Sec. VI-A; optional tanh soft-cap and transposed V cache per Sec. VI-B).
//
// Work decomposition
//   A workgroup (4 waves) serves one KV head.  Each wave owns a "task": one query head of the
//   KV head's group and 32 consecutive queries.  Tasks are ordered query-major, so the 4 waves of
//   a workgroup need nearly the same key range; the workgroup stages every key tile once in LDS
//   and all 4 waves read it (the GQA group shares its K/V).  The key axis may be split over
//   several workgroups; a fixed-order combine kernel then merges the partials (m, l and O / l
//   as a scaled fp16 row, store_partial).
//   blockIdx.x % n_kv_heads selects the KV head, so on the 8-XCD MI355X every workgroup of one
//   KV head lands on the same XCD and its K/V tiles are shared through that XCD's L2.
//
// Per 64-key tile and wave (head_dim 128)
//   S^T (keys x queries) = K . Q^T   with v_mfma_f32_32x32x16_bf16: A = K rows from LDS,
//                                    B = Q held in registers for the whole kernel.
//   Each lane then holds 32 scores of one query: the online softmax (log2 domain, fp32) needs
//   one cross-lane max (lanes l and l^32 share a query) and no other shuffle.
//   O^T (d x queries) += V^T . P^T  with the same MFMA: B = P^T straight from the score
//                                    registers (bf16), A = V^T rows from LDS.
//   The MFMA output layout puts keys {4h..4h+3, 8+4h..8+4h+3} of each 16-key step in lane half
//   h, so the V^T tile stores each 16-key group with key bits 2 and 3 swapped: every A-operand
//   read is then one 16-byte LDS read.  K rows and V^T rows are XOR-swizzled in 16-byte
//   chunks to keep those reads free of bank conflicts.
#include "attn_common.h"
#include "launch.h"

#include <stdlib.h>

#include <algorithm>
#include <vector>

namespace nexus {

template <int D, int KT, bool VT, bool CAP>
__global__ __launch_bounds__(256, (D >= 256 ? 1 : 2)) void attn_bf16_kernel(const AttnArgs a,
                                                                             const AttnPlan plan) {
  constexpr int KCH = D / 8;                        // 16-byte chunks per K row
  constexpr int KSW = (KCH < 16 ? KCH : 16) - 1;    // K row swizzle mask
  constexpr int VCH = KT / 8;                       // 16-byte chunks per V^T row
  constexpr int VSW = VCH - 1;
  constexpr int NKB = KT / 32;                      // 32-key score blocks per tile
  constexpr int NDB = D / 32;                       // 32-row blocks of O^T
  constexpr int NS = D / 16;                        // k-steps of Q K^T
  constexpr int TPG = KT / kPage;                   // pages per tile
  constexpr float kSlack = 8.0f;                    // lazy rescale: p <= 2^8 between rescales
  __shared__ __align__(16) uint16_t Ks[2][KT * D];
  __shared__ __align__(16) uint16_t Vs[2][D * KT];
  __shared__ __align__(16) int32_t pg[kMaxSplitKeys / kPage + 8];  // pages of this workgroup

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int j = lane & 31, hh = lane >> 5;
  const int kvh = blockIdx.x % a.n_kv_heads;
  const UnitLoc loc = locate_unit(plan, blockIdx.x / a.n_kv_heads);
  const int b = loc.seq;
  const UnitWork uw = loc.w;
  const SeqPlan sp = plan.seq[b];
  const int tgrp = uw.tgrp, split = uw.split;
  const int G = a.group;

  const int task = tgrp * kWaves + wave;
  const bool active = task < sp.n_tasks;
  const int qb = task / G;
  const int g = task - qb * G;
  const int q0 = qb * kQB;
  const int qhead = kvh * G + g;
  const int last_task = min(tgrp * kWaves + kWaves - 1, sp.n_tasks - 1);
  const int last_q = min((last_task / G + 1) * kQB, sp.len);
  // positions fit in int32 and element offsets within a layer in uint32 (host-checked)
  const int wg_keys = (int)sp.n_past + last_q;
  const int k_begin = uw.k_begin;
  const int k_end = min(k_begin + uw.split_keys, wg_keys);
  const int wave_keys = active ? (int)sp.n_past + min(q0 + kQB, sp.len) : 0;
  const int qpos0 = (int)sp.n_past + q0;  // position of this wave's query 0
  const int n_tiles = k_end > k_begin ? (k_end - k_begin + KT - 1) / KT : 0;

  // physical page of every logical page this workgroup reads
  const int pg0 = k_begin >> kPageShift;
  if (n_tiles > 0) {
    const int n_pg = ((k_end - 1) >> kPageShift) - pg0 + 1;
    for (int i = tid; i < n_pg; i += 256) pg[i] = a.map[pg0 + i];
  }

  // Q of this wave as B operands: lane (hh, j) holds Q[q0 + j][16 s + 8 hh .. + 7].
  bf16x8 qreg[NS];
  if (active) {
    const int qi = min(q0 + j, sp.len - 1);
    const uint16_t *qrow = a.q + ((int64_t)(sp.q_start + qi) * a.n_q_heads + qhead) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qreg[s] = *reinterpret_cast<const bf16x8 *>(qrow + 16 * s + 8 * hh);
  }

  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float m_ref = -INFINITY;   // reference max (log2 units) shared by l and o
  float l = 0.f;             // this lane's share of the row sum (its key half)

  const uint32_t pstride = (uint32_t)a.n_kv_heads * kPage * D;   // one physical page, all heads
  const uint16_t *kbase = a.kc + (int64_t)kvh * kPage * D;
  const uint16_t *vbase = a.vc + (int64_t)kvh * kPage * D;
  const uint32_t n_cols = (uint32_t)a.n_phys_pages * kPage;        // transposed V row length
  const uint16_t *vtbase = a.vc + (int64_t)kvh * D * n_cols;

  // ---- per-thread staging assignment (invariant over tiles)
  constexpr int K_ITEMS = KT * KCH / 256;                   // 16-byte K chunks per thread
  constexpr int V_ITEMS_RM = (KT / 4) * (D / 8);            // (4-token, 8-dim) groups
  constexpr int V_PER_T_RM = (V_ITEMS_RM + 255) / 256;
  constexpr int V_ITEMS_T = D * (KT / 8);                   // (dim, 8-token) groups
  constexpr int V_PER_T_T = V_ITEMS_T / 256;
  static_assert(K_ITEMS >= 1 && KT * KCH % 256 == 0, "tile too small");
  static_assert(V_PER_T_RM == 1 || VT, "one V group per thread");
  // staging registers of the tiles on their way to LDS: with head_dim 256 (one workgroup per
  // CU, registers to spare) two tiles are in flight, else one
  constexpr int NPRE = D >= 256 ? 2 : 1;
  constexpr int VN = VT ? V_PER_T_T : 4;
  struct Stage {
    u32x4 k[K_ITEMS];
    u32x4 v[VN];
  };
  Stage stg[NPRE];

  // K: thread owns chunk kc of keys kkey[i]
  const int kc = tid % KCH;
  // V row-major: 4 tokens (4 vg4 .. 4 vg4 + 3) x 8 dims (8 vdc ..)
  const int vg4 = tid / (D / 8), vdc = tid % (D / 8);
  constexpr bool kAllOwnV = VT || V_ITEMS_RM >= 256;
  const bool v_owner = kAllOwnV || tid < V_ITEMS_RM;

  __syncthreads();   // pg[] visible

  // Tokens past the split end are clamped to the last valid key k_end - 1: real cache data, so
  // their K/V are finite; their scores are masked and their weights are exactly 0.  Global
  // addresses are a uniform base plus a 32-bit unsigned byte offset.
  const char *kbytes = reinterpret_cast<const char *>(kbase);
  const char *vbytes = reinterpret_cast<const char *>(VT ? vtbase : vbase);
  auto load_tile = [&](int it, Stage &sg) {
    const int kt = k_begin + it * KT;
    const int tl = k_end - 1;
#pragma unroll
    for (int i = 0; i < K_ITEMS; ++i) {
      const int key = (tid + 256 * i) / KCH;
      const uint32_t t = (uint32_t)min(kt + key, tl);
      const uint32_t page = (uint32_t)pg[(t >> kPageShift) - pg0];
      const uint32_t off = (__umul24(page, pstride) + (t & (kPage - 1)) * D + kc * 8) * 2u;
      sg.k[i] = *reinterpret_cast<const u32x4 *>(kbytes + off);
    }
    if constexpr (!VT) {
      if (kAllOwnV || v_owner) {
        const uint32_t t0 = (uint32_t)min(kt + 4 * vg4, tl);
        const uint32_t page = (uint32_t)pg[(t0 >> kPageShift) - pg0];
        const uint32_t base = __umul24(page, pstride) + vdc * 8;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t t = (uint32_t)min(kt + 4 * vg4 + e, tl);
          sg.v[e] = *reinterpret_cast<const u32x4 *>(vbytes + (base + (t & (kPage - 1)) * D) * 2u);
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < V_PER_T_T; ++i) {
        const int u = tid + 256 * i;
        const int d = u / (KT / 8), grp = u % (KT / 8);
        const int t0 = min(kt + 8 * grp, tl & ~7);   // 8-token group holding key t0
        const uint32_t page = (uint32_t)pg[(t0 >> kPageShift) - pg0];
        u32x4 val = *reinterpret_cast<const u32x4 *>(
            vbytes + ((uint32_t)d * n_cols + page * kPage + (uint32_t)(t0 & (kPage - 1))) * 2u);
        if (kt + 8 * grp + 8 > k_end) {
          // group crosses or lies past the split end: keep keys <= tl, zero the rest (slots
          // past the end of the written cache may hold anything)
          const int nvalid = max(0, min(8, k_end - (kt + 8 * grp)));
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e >= nvalid) val[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
        }
        sg.v[i] = val;
      }
    }
  };

  auto store_tile = [&](int buf, const Stage &sg) {
    uint16_t *ks = Ks[buf];
    uint16_t *vs = Vs[buf];
#pragma unroll
    for (int i = 0; i < K_ITEMS; ++i) {
      const int key = (tid + 256 * i) / KCH;
      *reinterpret_cast<u32x4 *>(ks + key * D + ((kc ^ (key & KSW)) * 8)) = sg.k[i];
    }
    if constexpr (!VT) {
      if (kAllOwnV || v_owner) {
        const int pos = (4 * vg4 & ~15) | vt_pos(4 * vg4 & 15);   // 4-aligned
        const int cc = pos >> 3, half = (pos >> 2) & 1;
#pragma unroll
        for (int dd = 0; dd < 8; ++dd) {
          const int wi = dd >> 1;
          // gather feature dd of the 4 tokens: low or high halves of word wi
          const uint32_t sel = (dd & 1) ? 0x07060302u : 0x05040100u;
          const uint32_t lo = __builtin_amdgcn_perm(sg.v[1][wi], sg.v[0][wi], sel);
          const uint32_t hi = __builtin_amdgcn_perm(sg.v[3][wi], sg.v[2][wi], sel);
          const int d = 8 * vdc + dd;
          *reinterpret_cast<u32x2 *>(vs + d * KT + ((cc ^ vt_swz<VSW>(d)) * 8) + half * 4) =
              u32x2{lo, hi};
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < V_PER_T_T; ++i) {
        const int u = tid + 256 * i;
        const int d = u / (KT / 8), grp = u % (KT / 8);
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int k4 = 8 * grp + 4 * hf;
          const int pos = (k4 & ~15) | vt_pos(k4 & 15);
          const int cc = pos >> 3, half = (pos >> 2) & 1;
          const u32x2 piece = hf ? u32x2{sg.v[i][2], sg.v[i][3]} : u32x2{sg.v[i][0], sg.v[i][1]};
          *reinterpret_cast<u32x2 *>(vs + d * KT + ((cc ^ vt_swz<VSW>(d)) * 8) + half * 4) = piece;
        }
      }
    }
  };

  const float c_scale = CAP ? 1.0f : a.scale_log2;   // raw score -> log2 units
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  // ---- pipeline: tile t is in LDS buffer t & 1 while tiles t + 1 .. t + NPRE wait in
  // registers; tile j is staged in stg[j % NPRE]
  if (n_tiles > 0) {
    load_tile(0, stg[0]);
    store_tile(0, stg[0]);
#pragma unroll
    for (int j = 1; j <= NPRE; ++j)
      if (j < n_tiles) load_tile(j, stg[j % NPRE]);
  }
  __syncthreads();
  auto step = [&](int it, Stage &nxt) {
    const int kt = k_begin + it * KT;
    const uint16_t *ks = Ks[it & 1];
    const uint16_t *vs = Vs[it & 1];
    if (active && kt < wave_keys) {
      // ---- S^T = K . Q^T
      f32x16 sacc[NKB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[kb][v] = 0.f;
        const int key = 32 * kb + j;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          const bf16x8 ka =
              *reinterpret_cast<const bf16x8 *>(ks + key * D + (((2 * s + hh) ^ (key & KSW)) * 8));
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[s], sacc[kb], 0, 0, 0);
        }
      }
      if constexpr (CAP) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) sacc[kb][v] = a.cap_out * tanh_fast(sacc[kb][v] * a.cap_in);
      }
      // ---- causal / tail mask on tiles that cross this wave's diagonal or the split end
      if ((kt + KT > k_end) || (kt + KT - 1 > qpos0)) {
        const int lim = min(qpos0 + j, k_end - 1) - kt - 4 * hh;   // last visible key - base
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (32 * kb + 8 * (v >> 2) + (v & 3) > lim) sacc[kb][v] = -INFINITY;
      }
      // ---- online softmax (log2 units), lazily rescaled
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[kb][v]);
      mt = fmaxf(mt, __shfl_xor(mt, 32)) * c_scale;
      if (__builtin_amdgcn_ballot_w64(mt > m_ref + kSlack) != 0) {
        const float m_new = fmaxf(m_ref, mt);
        const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_ref - m_new);
        l *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
        m_ref = m_new;
      }
      const float nm = (m_ref == -INFINITY) ? 0.f : -m_ref;
      bf16x8 pb[NKB][2];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          uint32_t w[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = fast_exp2(fmaf(sacc[kb][8 * hf + 2 * e], c_scale, nm));
            const float p1 = fast_exp2(fmaf(sacc[kb][8 * hf + 2 * e + 1], c_scale, nm));
            w[e] = pack_bf16x2(p0, p1);
            l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, l, false);
          }
          pb[kb][hf] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
        }

      // ---- O^T += V^T . P^T
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int ks2 = 2 * kb + hf;
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const int d = 32 * db + j;
            const bf16x8 va = *reinterpret_cast<const bf16x8 *>(
                vs + d * KT + (((2 * ks2 + hh) ^ vt_swz<VSW>(d)) * 8));
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kb][hf], o[db], 0, 0, 0);
          }
        }
    }
    // tile it + 1 leaves its registers for LDS, which then take tile it + 1 + NPRE
    if (it + 1 < n_tiles) store_tile((it + 1) & 1, nxt);
    if (it + 1 + NPRE < n_tiles) load_tile(it + 1 + NPRE, nxt);
    __syncthreads();
  };
  if constexpr (NPRE == 1) {
    for (int it = 0; it < n_tiles; ++it) step(it, stg[0]);
  } else {
    for (int it = 0; it < n_tiles; it += 2) {
      step(it, stg[1]);
      if (it + 1 < n_tiles) step(it + 1, stg[NPRE - 2]);
    }
  }

  // ---- epilogue
  const float l_tot = l + __shfl_xor(l, 32);
  float part_c = 0.f, part_sc = 0.f;
  if (uw.n_splits > 1) part_sc = part_scale(row_amax(o), l_tot, part_c);
  if (!active || q0 + j >= sp.len) return;
  const int row = q0 + j;  // within the sequence
  if (uw.n_splits == 1) {
    const float inv = 1.0f / l_tot;
    uint16_t *orow = a.out + ((int64_t)(sp.q_start + row) * a.n_q_heads + qhead) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * db + 8 * gq + 4 * hh;
        const uint32_t lo = pack_bf16x2(o[db][4 * gq + 0] * inv, o[db][4 * gq + 1] * inv);
        const uint32_t hi = pack_bf16x2(o[db][4 * gq + 2] * inv, o[db][4 * gq + 3] * inv);
        *reinterpret_cast<uint2 *>(orow + d0) = make_uint2(lo, hi);
      }
  } else {
    const int64_t prow = ((int64_t)split * sp.len + row) * a.n_q_heads + qhead;
    store_partial<NDB, D>(o, part_sc, m_ref, l_tot, part_c, hh, a.ws, sp, prow);
  }
}

// Fixed-order merge of the split partials (fp16 rows P_s = O_s / (l_s 2^e_s), records
// {m_s, l_s, c_s = l_s 2^e_s}): M = max m_s, w_s = 2^(m_s - M),
// out = sum_s w_s c_s P_s / sum_s w_s l_s.  One thread per 16 output features (two 16-byte
// partial loads per split), which puts config 3's merge in one round of resident workgroups.
constexpr int kCombinePre = 8;   // splits whose partials the combine loads up front

template <int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(const AttnArgs a, const AttnPlan plan) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  constexpr int Q8 = D / 8, Q16 = D / 16;
  const int64_t total = (int64_t)plan.total_rows * a.n_q_heads * Q16;
  if (gid >= total) return;
  const int d8 = 2 * (int)(gid % Q16);
  const int64_t rh = gid / Q16;
  const int head = (int)(rh % a.n_q_heads);
  const int rowg = (int)(rh / a.n_q_heads);
  int b = 0;
  while (b + 1 < plan.n_seqs && rowg >= plan.seq[b + 1].row_begin) ++b;
  const SeqPlan sp = plan.seq[b];
  const int row = rowg - sp.row_begin;
  // the split count of this row's task group (task order: query block major, head minor)
  const int n_splits = group_splits(sp, ((row / plan.qpw) * a.group + head % a.group) / plan.waves);
  if (n_splits == 1) return;
  const int64_t pstep = (int64_t)sp.len * a.n_q_heads;         // partial rows per split
  const int64_t prow0 = (int64_t)row * a.n_q_heads + head;
  const f32x4 *rec = reinterpret_cast<const f32x4 *>(a.ws + sp.ml_off);
  const u32x4 *part = reinterpret_cast<const u32x4 *>(a.ws + sp.ws_off) + d8;
  float mmax = -INFINITY;
  float lsum = 0.f;
  float acc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;
  auto add = [&](const f32x4 &ml, const u32x4 &ov, const u32x4 &ov2) {
    const float w = (ml[0] == -INFINITY) ? 0.f : fast_exp2(ml[0] - mmax);
    lsum += w * ml[1];
    const float wc = w * ml[2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x2 f = unpack_f16x2(ov[i]);
      acc[2 * i] += wc * f[0];
      acc[2 * i + 1] += wc * f[1];
      const f32x2 g = unpack_f16x2(ov2[i]);
      acc[8 + 2 * i] += wc * g[0];
      acc[8 + 2 * i + 1] += wc * g[1];
    }
  };
  if (n_splits <= kCombinePre) {
    // every split's record and row loaded up front, then merged in split order: one round
    // trip instead of one per split
    f32x4 ml[kCombinePre];
    u32x4 ov[kCombinePre], ov2[kCombinePre];
#pragma unroll
    for (int s = 0; s < kCombinePre; ++s) {
      if (s < n_splits) {
        const int64_t prow = s * pstep + prow0;
        ml[s] = rec[prow];
        ov[s] = part[prow * Q8];
        ov2[s] = part[prow * Q8 + 1];
      }
    }
#pragma unroll
    for (int s = 0; s < kCombinePre; ++s)
      if (s < n_splits) mmax = fmaxf(mmax, ml[s][0]);
#pragma unroll
    for (int s = 0; s < kCombinePre; ++s) {
      if (s >= n_splits) break;
      add(ml[s], ov[s], ov2[s]);
    }
  } else {
    for (int s = 0; s < n_splits; ++s) mmax = fmaxf(mmax, rec[s * pstep + prow0][0]);
    for (int s = 0; s < n_splits; ++s) {
      const int64_t prow = s * pstep + prow0;
      add(rec[prow], part[prow * Q8], part[prow * Q8 + 1]);
    }
  }
  const float inv = 1.0f / lsum;
  uint16_t *orow = a.out + ((int64_t)(sp.q_start + row) * a.n_q_heads + head) * D + 8 * d8;
  *reinterpret_cast<u32x4 *>(orow) =
      u32x4{pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv),
            pack_bf16x2(acc[4] * inv, acc[5] * inv), pack_bf16x2(acc[6] * inv, acc[7] * inv)};
  *reinterpret_cast<u32x4 *>(orow + 8) =
      u32x4{pack_bf16x2(acc[8] * inv, acc[9] * inv), pack_bf16x2(acc[10] * inv, acc[11] * inv),
            pack_bf16x2(acc[12] * inv, acc[13] * inv), pack_bf16x2(acc[14] * inv, acc[15] * inv)};
}

namespace {

int key_tile_for(int head_dim) { return head_dim >= 256 ? 32 : 64; }

// Geometry of the kernel that serves a launch: queries per wave task, key tile, how many of its
// workgroups are resident per CU, wave tasks per workgroup, and the plan's time per key of one
// workgroup (us, measured).
struct KernelShape {
  int qpw, key_tile, wgs_per_cu, waves;
  double us_per_key;
};

KernelShape kernel_shape(const AttnLaunch &p) {
  if (p.head_dim == 128 && !p.v_transposed) return {kQB, 64, 2, kWaves, 0.03};   // LDS DMA
  if (p.head_dim == 256 && p.v_transposed) return {kQB, 32, 1, kWavesWide, 0.04};   // LDS DMA
  return {kQB, key_tile_for(p.head_dim), p.head_dim >= 256 ? 1 : 2, kWaves,
          0.03 * p.head_dim / 128.0};
}

constexpr int kCUs = 256;

// Deterministic plan of an attention launch: task groups, key splits and workspace offsets.
// The same arguments always give the same plan (the workspace query relies on it).
// The split length is chosen to minimise an estimate of the launch time: the critical path over
// the resident workgroup slots (the longest piece of work, the total work spread over the slots,
// and the rounds that the near-full-length pieces need: uniform suffix shapes are decided by the
// the latter, causal prefills by the former two) at the kernel's measured time per key of one
// workgroup (KernelShape), plus, when keys are split, the combine: writing and reading the
// partials (priced as fp32 rows, split_cost_bytes) at about 4 TB/s and one more launch.  A piece's work is its keys plus a fixed 128 for
// its prologue and epilogue.
bool make_plan(const AttnLaunch &p, AttnPlan &plan) {
  if (p.n_seqs < 1 || p.n_seqs > kMaxSeqs) return false;
  const int G = p.n_q_heads / p.n_kv_heads;
  const KernelShape ks = kernel_shape(p);
  const int KT = ks.key_tile;
  const int64_t slots = (int64_t)kCUs * ks.wgs_per_cu;
  constexpr int64_t kPieceOverhead = 128;
  // shortest split in general, and in a launch whose pieces all fit the resident workgroup slots
  // at once (a few hundred queries: latency-bound, where shorter pieces shorten the critical
  // path; measured on the shallow depths of the depth-adaptive sweep, e.g. 90 queries at 742:
  // 22.8 -> 19.1 us, and on a single layer of 192 queries over 2560 keys: 34.1 -> 32.4 us)
  constexpr int64_t kMinSplitKeys = 512, kMinSplitKeysSmall = 256;
  plan = AttnPlan{};
  plan.n_seqs = p.n_seqs;
  plan.qpw = ks.qpw;
  plan.waves = ks.waves;
  int64_t max_keys = 0;
  for (int b = 0; b < p.n_seqs; ++b)
    max_keys = std::max<int64_t>(max_keys, p.seqs[b].n_past + p.seqs[b].len);
  auto n_tasks_of = [&](const AttnSeq &s) { return G * ((s.len + ks.qpw - 1) / ks.qpw); };
  // split length of a sequence for a global candidate: equal key counts rounded to the tile
  auto seq_split = [&](int64_t keys, int64_t sk) {
    int64_t ns = (keys + sk - 1) / sk;
    if (ns < 1) ns = 1;
    int64_t skb = (keys + ns - 1) / ns;
    return (skb + KT - 1) / KT * KT;
  };
  // keys of each task group (nondecreasing in the group index), once per sequence
  std::vector<std::vector<int64_t>> tg_keys(p.n_seqs);
  std::vector<double> seq_keys(p.n_seqs, 0.0);
  for (int b = 0; b < p.n_seqs; ++b) {
    const AttnSeq &s = p.seqs[b];
    const int n_tasks = n_tasks_of(s);
    const int n_tg = (n_tasks + ks.waves - 1) / ks.waves;
    tg_keys[b].resize(n_tg);
    for (int tg = 0; tg < n_tg; ++tg) {
      const int last_task = std::min(tg * ks.waves + ks.waves - 1, n_tasks - 1);
      tg_keys[b][tg] = s.n_past + std::min((last_task / G + 1) * ks.qpw, s.len);
      seq_keys[b] += (double)tg_keys[b][tg];
    }
  }
  // several suffix-like sequences (blocks spliced into one context, each re-decoding a suffix
  // over the shared prefix): one split length for all, units range by range (AttnPlan); the
  // split count candidates below keep the ranges within kMaxRanges.  A launch that also holds a
  // causal prefill (n_past < len) plans sequence by sequence instead, each with its own split,
  // so the prefill keeps its longest-first order (the depth-adaptive sweep's one-launch form,
  // context rows + redecoded rows: 1.06 -> 1.10x the full prefill at n_past 256, 0.94 -> 0.96x
  // at 16384).
  bool any_prefill = false;
  for (int b = 0; b < p.n_seqs; ++b) any_prefill |= p.seqs[b].n_past < p.seqs[b].len;
  // (beyond kMaxRanges splits of the longest length, i.e. over 2^21 keys, sequence by sequence)
  const bool range_major = p.n_seqs > 1 && !any_prefill &&
                           max_keys <= (int64_t)kMaxRanges * kMaxSplitKeys;
  int64_t best_sk = kMaxSplitKeys;
  double best_cost = 1e300;
  bool found = false;
  const double cap = p.ws_cap == SIZE_MAX ? 1e300 : (double)p.ws_cap;
  // workspace bytes of a sequence whose rows keep `n` partials each (none for one split): an
  // fp16 row and a 16-byte record per partial
  auto part_bytes = [&](const AttnSeq &s, int64_t n) {
    return n > 1 ? (double)n * s.len * p.n_q_heads * (2.0 * p.head_dim + 16.0) : 0.0;
  };
  // the split term of the cost: 8 (D + 2) bytes per partial row, i.e. its write and read as
  // fp32 O and (m, l).  The partials are stored at about half that (fp16 rows), but the term was
  // calibrated with these bytes, and it also stands for the per-unit costs of a split that the
  // estimate leaves out (more workgroups and prologues, empty units of causal groups): pricing
  // it at the stored bytes chose more splits and ran slower (one launch of a 2048-token prefill
  // and a 576-token suffix: 77 -> 121 us per layer; 123 queries at depth 512 with a 512-token
  // prefill: 25.6 -> 31.6 us), with configs 2 and 4 unchanged.
  auto split_cost_bytes = [&](const AttnSeq &s, int64_t n) {
    return n > 1 ? 8.0 * (double)n * s.len * p.n_q_heads * (p.head_dim + 2) : 0.0;
  };
  for (int ns = 1; ns <= kMaxRanges; ++ns) {
    int64_t sk = (max_keys + ns - 1) / ns;
    sk = (sk + KT - 1) / KT * KT;
    if (sk > kMaxSplitKeys) continue;
    if (sk < kMinSplitKeysSmall && ns > 1) break;
    int64_t max_splits = 1, n_full = 0, full_len = 0, max_piece = 0, n_pieces = 0;
    double total = 0.0, combine_bytes = 0.0, ws_need = 0.0;
    for (int b = 0; b < p.n_seqs; ++b) {
      const AttnSeq &s = p.seqs[b];
      const std::vector<int64_t> &wk = tg_keys[b];
      const int64_t keys = s.n_past + s.len;
      const int64_t skb = range_major ? sk : seq_split(keys, sk);
      const int64_t nsb = (keys + skb - 1) / skb;
      max_splits = std::max(max_splits, nsb);
      ws_need += part_bytes(s, nsb);
      if (nsb > 1)
        combine_bytes += split_cost_bytes(s, nsb) + 2.0 * s.len * p.n_q_heads * p.head_dim;
      // piece j of a task group is non-empty when its keys exceed j * skb, and counts as
      // full-length for the rounds when it holds at least half the split length.  Suffix-like
      // sequences (all task groups within 10% of the same keys) take the closed form.
      int64_t pieces = 0, full = 0;
      if (!wk.empty() && wk.front() * 10 >= wk.back() * 9) {
        const int64_t n_tg = (int64_t)wk.size();
        pieces = n_tg * nsb;
        full = n_tg * (nsb - 1) + (2 * (wk.back() - (nsb - 1) * skb) >= skb ? n_tg : 0);
        if (full > 0) full_len = std::max(full_len, skb);
      } else {
        for (int64_t jp = 0; jp < nsb; ++jp) {
          pieces += wk.end() - std::upper_bound(wk.begin(), wk.end(), jp * skb);
          const int64_t f =
              wk.end() - std::lower_bound(wk.begin(), wk.end(), jp * skb + (skb + 1) / 2);
          full += f;
          if (f > 0) full_len = std::max(full_len, skb);
        }
      }
      n_full += full * p.n_kv_heads;
      n_pieces += pieces * p.n_kv_heads;
      if (!wk.empty()) max_piece = std::max(max_piece, std::min(skb, wk.back()) + kPieceOverhead);
      total += (seq_keys[b] + (double)pieces * kPieceOverhead) * p.n_kv_heads;
    }
    if (sk < kMinSplitKeys && ns > 1 && n_pieces > slots) continue;
    if (ws_need > cap) continue;
    const double rounds_full = (double)((n_full + slots - 1) / slots);
    const double est = std::max({rounds_full * (double)(full_len + kPieceOverhead),
                                 (double)max_piece, total / (double)slots});
    const double cost = est * ks.us_per_key + (max_splits > 1 ? combine_bytes / 4.0e6 + 8.0 : 0.0);
    if (cost < best_cost - 1e-9) {
      best_cost = cost;
      best_sk = sk;
      found = true;
    }
  }
  // under a workspace cap every plan must fit it (without one the loop always finds a plan)
  if (!found && p.ws_cap != SIZE_MAX) return false;
  const int64_t split_keys = best_sk;

  // Two split classes (one suffix-like sequence): when the units of one split length leave the
  // last round of workgroup slots partly empty, the first n_a task groups keep a coarse split
  // that fills whole rounds and the remaining n_b groups take a finer split that fills one last
  // round, instead of a partial round of full-length units.  Same cost model; slots per KV head.
  int64_t two_n_a = -1, two_ns_a = 0, two_ns_b = 0;
  if (p.n_seqs == 1 && !tg_keys[0].empty() && tg_keys[0].front() * 10 >= tg_keys[0].back() * 9) {
    const AttnSeq &s = p.seqs[0];
    const int64_t keys = s.n_past + s.len;
    const int64_t n_tg = (int64_t)tg_keys[0].size();
    const int64_t slots_h = std::max<int64_t>(1, slots / p.n_kv_heads);
    const double rows_heads = (double)s.len * p.n_q_heads;
    auto split_len = [&](int64_t ns) { return seq_split(keys, (keys + ns - 1) / ns); };
    // split count of the cut that asks for `want` splits (as the plan below makes it)
    auto cut_count = [&](int64_t want) {
      const int64_t kk = ((keys + want - 1) / want + KT - 1) / KT * KT;
      return (keys + kk - 1) / kk;
    };
    for (int64_t ns_a = 1; ns_a <= 16; ++ns_a) {
      const int64_t la = split_len(ns_a);
      if (la > kMaxSplitKeys || (la < kMinSplitKeys && ns_a > 1)) continue;
      for (int64_t k = 1; k <= 4; ++k) {
        const int64_t n_a = std::min(n_tg, k * slots_h / ns_a);
        const int64_t n_b = n_tg - n_a;
        if (n_a < 1 || n_b < 1 || n_b > slots_h) continue;
        const int64_t ns_b = slots_h / n_b;
        const int64_t lb = split_len(ns_b);
        if (lb > kMaxSplitKeys || ns_b <= ns_a) continue;
        if (part_bytes(s, std::max(cut_count(ns_a), cut_count(ns_b))) > cap) continue;
        const int64_t rounds_a = (n_a * ns_a + slots_h - 1) / slots_h;
        const double est = (double)rounds_a * (la + kPieceOverhead) + (double)(lb + kPieceOverhead);
        const double comb = 8.0 * rows_heads * (p.head_dim + 2) *
                                (double)(n_a * ns_a + n_b * ns_b) / (double)n_tg +
                            2.0 * rows_heads * p.head_dim;
        const double cost = est * ks.us_per_key + comb / 4.0e6 + 8.0;
        if (cost < best_cost - 1e-9) {
          best_cost = cost;
          two_n_a = n_a;
          two_ns_a = ns_a;
          two_ns_b = ns_b;
        }
      }
    }
  }

  int32_t unit = 0, rows = 0;
  int64_t ws_bytes = 0;
  int32_t seq_units[kMaxSeqs];
  for (int b = 0; b < p.n_seqs; ++b) {
    const AttnSeq &s = p.seqs[b];
    SeqPlan &sp = plan.seq[b];
    sp.q_start = s.q_start;
    sp.len = s.len;
    sp.n_past = s.n_past;
    sp.row_begin = rows;
    sp.first_unit = unit;
    sp.n_tasks = G * ((s.len + ks.qpw - 1) / ks.qpw);
    const int n_tg = (sp.n_tasks + ks.waves - 1) / ks.waves;
    sp.n_tg = n_tg;
    const int64_t keys = s.n_past + s.len;
    int64_t ns = (keys + split_keys - 1) / split_keys;
    if (ns < 1) ns = 1;
    // balance the splits: equal key counts rounded to the tile (one sequence), or the launch's
    // common split length (several: aligned key ranges)
    int64_t sk = range_major ? split_keys : (keys + ns - 1) / ns;
    sk = (sk + KT - 1) / KT * KT;
    ns = (keys + sk - 1) / sk;
    sp.n_splits = (int32_t)ns;
    sp.split_keys = (int32_t)sk;
    sp.longest_first = s.n_past < s.len ? 1 : 0;
    sp.n_tg_a = n_tg;
    sp.n_splits_b = sp.n_splits;
    sp.split_keys_b = sp.split_keys;
    if (two_n_a > 0) {
      // the two-class cut replaces the single split (one sequence)
      auto cut = [&](int64_t want, int32_t &n_out, int32_t &k_out) {
        int64_t kk = (keys + want - 1) / want;
        kk = (kk + KT - 1) / KT * KT;
        k_out = (int32_t)kk;
        n_out = (int32_t)((keys + kk - 1) / kk);
      };
      cut(two_ns_a, sp.n_splits, sp.split_keys);
      cut(two_ns_b, sp.n_splits_b, sp.split_keys_b);
      sp.n_tg_a = (int32_t)two_n_a;
    }
    sp.max_splits = std::max(sp.n_splits, sp.n_splits_b);
    seq_units[b] = sp.n_tg_a * sp.n_splits + (n_tg - sp.n_tg_a) * sp.n_splits_b;
    unit += seq_units[b];
    rows += s.len;
    if (sp.max_splits > 1) {
      plan.any_split = 1;
      sp.ws_off = ws_bytes;
      ws_bytes += ((int64_t)sp.max_splits * s.len * p.n_q_heads * p.head_dim * 2 + 15) / 16 * 16;
      sp.ml_off = ws_bytes;
      ws_bytes += (int64_t)sp.max_splits * s.len * p.n_q_heads * 16;
    }
  }
  plan.units_per_head = unit;
  plan.total_rows = rows;
  plan.ws_bytes = (size_t)ws_bytes;
  if (!range_major) {
    // dispatch order: suffix-like sequences first (uniform units), then causal prefills, whose
    // longest-first order ends the launch on their short diagonal groups
    int n = 0;
    for (int pass = 0; pass < 2; ++pass)
      for (int b = 0; b < p.n_seqs; ++b)
        if ((p.seqs[b].n_past < p.seqs[b].len) == (pass == 1)) plan.order[n++] = b;
    int32_t u = 0;
    for (int i = 0; i < p.n_seqs; ++i) {
      plan.seq[plan.order[i]].first_unit = u;
      u += seq_units[plan.order[i]];
    }
  }
  if (range_major) {
    // sequences by decreasing split count (the sequences of range r are then a prefix), their
    // task-group prefix sums, and the first unit of each range
    plan.range_major = 1;
    for (int b = 0; b < p.n_seqs; ++b) plan.order[b] = b;
    std::stable_sort(plan.order, plan.order + p.n_seqs, [&](int x, int y) {
      return plan.seq[x].n_splits > plan.seq[y].n_splits;
    });
    plan.tg_prefix[0] = 0;
    for (int i = 0; i < p.n_seqs; ++i) {
      const SeqPlan &sp = plan.seq[plan.order[i]];
      plan.tg_prefix[i + 1] = plan.tg_prefix[i] + sp.n_tg;
    }
    plan.n_ranges = plan.seq[plan.order[0]].n_splits;
    if (plan.n_ranges > kMaxRanges) return false;
    plan.range_first_unit[0] = 0;
    for (int r = 0; r < plan.n_ranges; ++r) {
      int m = 0;
      while (m < p.n_seqs && plan.seq[plan.order[m]].n_splits > r) ++m;
      plan.range_first_unit[r + 1] = plan.range_first_unit[r] + plan.tg_prefix[m];
    }
    if (plan.range_first_unit[plan.n_ranges] != plan.units_per_head) return false;
  }
  return true;
}

template <int D, int KT, bool VT, bool CAP>
void launch_main(const AttnArgs &args, const AttnPlan &plan, int n_kv, hipStream_t stream) {
  hipLaunchKernelGGL((attn_bf16_kernel<D, KT, VT, CAP>), dim3(plan.units_per_head * n_kv),
                     dim3(256), 0, stream, args, plan);
}

template <int D, int KT>
void dispatch_main(const AttnArgs &args, const AttnPlan &plan, int n_kv, bool vt, bool cap,
                   hipStream_t stream) {
  if (vt) {
    if (cap) launch_main<D, KT, true, true>(args, plan, n_kv, stream);
    else launch_main<D, KT, true, false>(args, plan, n_kv, stream);
  } else {
    if (cap) launch_main<D, KT, false, true>(args, plan, n_kv, stream);
    else launch_main<D, KT, false, false>(args, plan, n_kv, stream);
  }
}

}  // namespace

hipError_t launch_attention_f32(const AttnLaunch &p, hipStream_t stream);
hipError_t launch_attn_d128_dma(const AttnArgs &args, const AttnPlan &plan, int n_kv, bool cap,
                                hipStream_t stream);
hipError_t launch_attn_d256_vt(const AttnArgs &args, const AttnPlan &plan, int n_kv, bool cap,
                               hipStream_t stream);

size_t attn_workspace_bytes(const AttnLaunch &p) {
  if (!p.is_bf16) return 0;
  AttnPlan plan;
  if (!make_plan(p, plan)) return (size_t)-1;
  return plan.ws_bytes;
}

hipError_t launch_attention(const AttnLaunch &p, hipStream_t stream) {
  if (!p.is_bf16) return launch_attention_f32(p, stream);
  AttnPlan plan;
  if (!make_plan(p, plan)) return hipErrorInvalidValue;
  if (plan.ws_bytes > p.workspace_bytes) return hipErrorInvalidValue;
  AttnArgs args;
  const int64_t layer_elems = (int64_t)p.n_phys_pages * p.n_kv_heads * kPage * p.head_dim;
  args.q = (const uint16_t *)p.q;
  args.out = (uint16_t *)p.out;
  args.kc = (const uint16_t *)p.cache_k + (int64_t)p.layer * layer_elems;
  args.vc = (const uint16_t *)p.cache_v + (int64_t)p.layer * layer_elems;
  args.map = p.map;
  args.ws = (char *)p.workspace;
  args.n_q_heads = p.n_q_heads;
  args.n_kv_heads = p.n_kv_heads;
  args.group = p.n_q_heads / p.n_kv_heads;
  args.n_phys_pages = p.n_phys_pages;
  const float log2e = 1.4426950408889634f;
  args.scale_log2 = p.scale * log2e;
  args.cap_in = p.softcap > 0.f ? p.scale / p.softcap : 0.f;
  args.cap_out = p.softcap * log2e;
  args.cap_k = p.softcap > 0.f ? 2.0f * p.scale * log2e / p.softcap : 0.f;
  const bool cap = p.softcap > 0.f;
  switch (p.head_dim) {
    case 64: dispatch_main<64, 64>(args, plan, p.n_kv_heads, p.v_transposed, cap, stream); break;
    case 128:
      if (!p.v_transposed) {
        const hipError_t e = launch_attn_d128_dma(args, plan, p.n_kv_heads, cap, stream);
        if (e != hipSuccess) return e;
      } else {
        dispatch_main<128, 64>(args, plan, p.n_kv_heads, p.v_transposed, cap, stream);
      }
      break;
    case 256:
      if (p.v_transposed) {
        const hipError_t e = launch_attn_d256_vt(args, plan, p.n_kv_heads, cap, stream);
        if (e != hipSuccess) return e;
      } else {
        dispatch_main<256, 32>(args, plan, p.n_kv_heads, p.v_transposed, cap, stream);
      }
      break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (plan.any_split) {
    const int64_t total = (int64_t)plan.total_rows * p.n_q_heads * (p.head_dim / 16);
    const uint32_t blocks = (uint32_t)((total + 255) / 256);
    switch (p.head_dim) {
      case 64: hipLaunchKernelGGL(attn_combine_kernel<64>, dim3(blocks), dim3(256), 0, stream, args, plan); break;
      case 128: hipLaunchKernelGGL(attn_combine_kernel<128>, dim3(blocks), dim3(256), 0, stream, args, plan); break;
      case 256: hipLaunchKernelGGL(attn_combine_kernel<256>, dim3(blocks), dim3(256), 0, stream, args, plan); break;
    }
    e = hipGetLastError();
  }
  return e;
}

}  // namespace nexus
