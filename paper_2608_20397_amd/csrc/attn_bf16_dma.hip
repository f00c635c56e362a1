// bf16 suffix attention, head_dim 128 with a row-major V cache: the variant that feeds LDS with
// gfx950's LDS DMA loads (Sec. III-A; the re-decoded suffix of Sec. VI-A).
//
// Same work decomposition and math as attn_bf16_kernel (one KV head per workgroup, 4 waves, each
// wave one query head x 32 queries, S^T = K.Q^T and O^T += V^T.P^T on 32x32x16 MFMA, online
// softmax in log2 units with a lazily moved reference, two workgroups per CU so that one
// workgroup's softmax overlaps the other's MFMA work), but:
//   * K and V tiles travel global -> LDS with global_load_lds_dwordx4: each lane's 16 bytes land
//     at base + 16 * lane, so the XOR swizzles below are produced by choosing each lane's source
//     chunk; no staging registers, no LDS write instructions.  The loads are issued from inline
//     assembly and ordered by explicit vmcnt waits and an LDS-only barrier: the compiler cannot
//     tell the buffers apart and would otherwise wait for every load in flight before each LDS
//     read, exposing the whole load latency every tile;
//   * a tile's 64 keys are 4 pages, one per wave, so the page address is wave-uniform;
//   * the PV A operand (8 keys of one feature) comes from the row-major V tile through two
//     ds_read_b64_tr_b16: in each 16-lane group, output lane i receives element i % 4 of the
//     8 bytes that source lane 4e + i / 4 points at, e = 0..3.  Source lane 4e + q points at
//     V[key_e][d0 + 4q], so output lane i receives V[key_0..3][d0 + i].  The keys each lane
//     needs follow the score layout of the S^T MFMA (keys 4h..4h+3 and 8+4h..8+4h+3 of a
//     16-key step for lane half h).
// LDS tiles: K row r (256 B) holds chunk c at c ^ (r & 15); V row r holds chunk c at
// c ^ 4 (r & 3).  Both keep the 16-byte K reads and the 8-byte transposed V reads of a wave free
// of bank conflicts.
#include "attn_common.h"
#include "attn_dma.h"
#include "launch.h"

#include <type_traits>

namespace nexus {

template <bool CAP>
__global__ __launch_bounds__(256, 2) void attn_bf16_d128_dma_kernel(const AttnArgs a,
                                                                    const AttnPlan plan) {
  constexpr int D = 128, KT = 64;
  constexpr int NKB = KT / 32, NDB = D / 32, NS = D / 16;
  constexpr int ROWB = D * 2;                 // bytes per K or V row
  constexpr int TILEB = KT * ROWB;            // bytes per K or V tile
  constexpr float kSlack = 8.0f;              // lazy rescale: p <= 2^8 between rescales
  constexpr int kPrioPV = 2;                  // wave priority of the PV phase
  __shared__ __align__(1024) char smem[2 * 2 * TILEB];   // K buffers 0, 1, V buffers 0, 1
  __shared__ __align__(16) int32_t pg[kMaxSplitKeys / kPage + 8];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
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
  const int wg_keys = (int)sp.n_past + last_q;
  const int k_begin = uw.k_begin;
  const int k_end = min(k_begin + uw.split_keys, wg_keys);
  const int qpos0 = (int)sp.n_past + q0;
  const int n_tiles = k_end > k_begin ? (k_end - k_begin + KT - 1) / KT : 0;

  const int pg0 = k_begin >> kPageShift;
  const int n_pg = n_tiles > 0 ? ((k_end - 1) >> kPageShift) - pg0 + 1 : 0;
  for (int i = tid; i < n_pg; i += 256) pg[i] = a.map[pg0 + i];

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
  float m_ref = -INFINITY;
  float l = 0.f;

  // ---- lane-invariant LDS read offsets
  uint32_t offk[NS];                          // S^T A operand: K row j, chunk 2s + hh
#pragma unroll
  for (int s = 0; s < NS; ++s) offk[s] = j * ROWB + (((2 * s + hh) ^ (j & 15)) * 16);
  uint32_t offv[NDB];                         // PV A operand: see the header comment
  {
    const int gg = lane >> 4, r = lane & 15, e = r >> 2, q = r & 3;
    const int h2 = gg >> 1, dh = gg & 1;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      offv[db] = (4 * h2 + e) * ROWB + 32 * dh + 8 * q + 64 * (db ^ e);
  }
  // ---- DMA: wave w fills tile rows 16 w .. 16 w + 15 (one page).  Instruction i covers rows
  // 4 i + r16; K chunk c of row r sits at c ^ (r & 15), V chunk c at c ^ 4 (r & 3).
  const int r16 = lane >> 4;
  const uint32_t kdo = r16 * ROWB + (((lane & 15) ^ r16) * 16);
  const uint32_t vdo = r16 * ROWB + (((lane & 15) ^ (4 * r16)) * 16);
  const uint32_t smem_base = (uint32_t)(uintptr_t)smem;
  const uint64_t pbytes = (uint64_t)a.n_kv_heads * kPage * ROWB;   // one physical page
  const char *kbytes = reinterpret_cast<const char *>(a.kc) + (uint64_t)kvh * kPage * ROWB;
  const char *vbytes = reinterpret_cast<const char *>(a.vc) + (uint64_t)kvh * kPage * ROWB;
  auto kbuf = [&](int i) { return smem + i * TILEB; };
  auto vbuf = [&](int i) { return smem + (2 + i) * TILEB; };

  // Q and the page table are waited for before any DMA is in flight: otherwise the compiler
  // waits for the Q loads at their first use inside the tile loop, with vmcnt values that count
  // the DMA loads too.
  wait_vm<0>();
  __syncthreads();   // pg[] visible

  // physical page of this wave's quarter of tile `it` (full tiles only)
  auto page_of = [&](int it) -> uint32_t {
    return (uint32_t)__builtin_amdgcn_readfirstlane(pg[it * (KT / kPage) + wave]);
  };
  // DMA of one K or V tile (`sel` 0 = K, 1 = V) of tile `it` into this wave's 4 KB quarter of the
  // buffer at `dstp`.  Full tiles use the wave-uniform page `page`.  The last, partial tile
  // clamps keys past the split end to the last valid key (finite data; their scores are
  // masked, so they get weight 0).
  auto dma_tile = [&](int it, int sel, char *dstp, uint32_t page) {
    const int kt = k_begin + it * KT;
    const char *src = sel ? vbytes : kbytes;
    const uint32_t dst = smem_base + (uint32_t)(dstp - smem) + wave * 4096;
    if (kt + KT <= k_end) {
      const char *ps = src + page * pbytes;
      if (sel) {
        dma_s<0>(dst, ps, vdo);
        dma_s<1024>(dst, ps, vdo);
        dma_s<2048>(dst, ps, vdo);
        dma_s<3072>(dst, ps, vdo);
      } else {
        dma_s<0>(dst, ps, kdo);
        dma_s<1024>(dst, ps, kdo ^ (1 << 6));
        dma_s<2048>(dst, ps, kdo ^ (2 << 6));
        dma_s<3072>(dst, ps, kdo ^ (3 << 6));
      }
    } else {
      const int tl = k_end - 1;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * wave + 4 * i + r16;
        const int t = min(kt + row, tl);
        const uint64_t pp = (uint32_t)pg[(t >> kPageShift) - pg0];
        const uint32_t tok = (uint32_t)(t & (kPage - 1)) * ROWB;
        const uint32_t c = sel ? ((lane & 15) ^ (4 * (row & 3))) : ((lane & 15) ^ (row & 15));
        dma_v(dst + i * 1024, src + pp * pbytes + tok + c * 16);
      }
    }
  };
  auto full = [&](int it) { return k_begin + it * KT + KT <= k_end; };

  const float c_scale = CAP ? 1.0f : a.scale_log2;
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  // S^T of one tile from K buffer `kl` (raw scores, or log2-scaled soft-capped ones)
  auto qk = [&](const char *kl, f32x16 *sacc) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[kb][v] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kl + kb * 32 * ROWB + offk[s]);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[s], sacc[kb], 0, 0, 0);
      }
  };

  // S(t) needs the causal / tail mask when its tile crosses this wave's diagonal or the split end
  auto needs_mask = [&](int t) {
    const int kt = k_begin + t * KT;
    return (kt + KT > k_end) || (kt + KT - 1 > qpos0);
  };
  // soft cap of S(t)
  auto cap = [&](f32x16 *sc) {
    if constexpr (CAP) {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) sc[kb][v] = a.cap_out * tanh_fast(sc[kb][v] * a.cap_in);
    }
  };
  // causal / tail mask of S(t) (tiles for which needs_mask(t))
  auto mask = [&](f32x16 *sc, int t) {
    const int lim = min(qpos0 + j, k_end - 1) - (k_begin + t * KT) - 4 * hh;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        if (32 * kb + 8 * (v >> 2) + (v & 3) > lim) sc[kb][v] = -INFINITY;
  };
  // row maximum of S(t) in log2 units
  auto row_max = [&](const f32x16 *sc) -> float {
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[kb][v]);
    return max_halves(mt) * c_scale;
  };
  // P of the 32 keys of a score block, as the B operands of two 16-key PV steps; adds their
  // sum to l (softmax_half: one of the two 16-key halves)
  auto softmax_block = [&](const f32x16 &sc, float nm, bf16x8 *pb) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = fast_exp2(fmaf(sc[8 * hf + 2 * e], c_scale, nm));
        const float p1 = fast_exp2(fmaf(sc[8 * hf + 2 * e + 1], c_scale, nm));
        w[e] = pack_bf16x2(p0, p1);
        l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, l, false);
      }
      pb[hf] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    }
  };
  auto softmax_half = [&](const f32x16 &sc, int hf, float nm, bf16x8 &pbo) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float p0 = fast_exp2(fmaf(sc[8 * hf + 2 * e], c_scale, nm));
      const float p1 = fast_exp2(fmaf(sc[8 * hf + 2 * e + 1], c_scale, nm));
      w[e] = pack_bf16x2(p0, p1);
      l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, l, false);
    }
    pbo = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
  };
  // O^T += V^T P^T over the 16 keys of step ks of the V tile at vl
  auto pv_step = [&](const char *vl, int ks, const bf16x8 &pbv) {
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const char *p = vl + ks * 16 * ROWB + offv[db];
      const bf16x8 va = tr_read_pair(p, p + 8 * ROWB);
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pbv, o[db], 0, 0, 0);
    }
  };

  // Pipeline, per iteration t: the DMA of K[t + 2] and V[t + 1] runs while the wave computes
  // S(t + 1) = K[t + 1] Q^T and O += V[t] P(t).  K buffers hold tiles t + 1 and t + 2, V
  // buffers tiles t and t + 1.  Pages: pk = page of tile t + 2 (K DMA), pgv = of tile t + 1.
  // Within the wave the matrix and vector work alternate: the S(t + 1) MFMAs run beside the
  // exponentials of S(t)'s first 48 keys, the PV MFMAs beside the exponentials of the last 16
  // and the soft cap and maximum of S(t + 1), which the next iteration's rescale needs.  The region has no branch, so the compiler's schedule can
  // follow the MFMA / LDS read / VALU pattern set below; the causal and tail masks, needed on
  // few tiles, are applied at the top of the next iteration.
  f32x16 sa[NKB], sb[NKB];
  uint32_t pgv = 0, pk = 0;
  if (n_tiles > 0) {
    const uint32_t p0 = full(0) ? page_of(0) : 0;
    dma_tile(0, 0, kbuf(0), p0);
    dma_tile(0, 1, vbuf(0), p0);
    if (n_tiles > 1) {
      pgv = full(1) ? page_of(1) : 0;
      dma_tile(1, 0, kbuf(1), pgv);
    }
    if (n_tiles > 2 && full(2)) pk = page_of(2);
  }
  wait_vm<0>();
  tile_barrier();
  float mt_cur = -INFINITY;                     // row maximum of S(t), log2 units
  if (active && n_tiles > 0) {
    qk(kbuf(0), sa);
    cap(sa);
    mt_cur = row_max(sa);        // unmasked: step 0 masks S(0) and takes its maximum again
  }
  tile_barrier();    // K buffer 0 is refilled in iteration 0

  auto step = [&](int t, auto parity, f32x16 *s_cur, f32x16 *s_nxt) {
    constexpr int P = decltype(parity)::value;     // t & 1
    if (t + 2 < n_tiles) dma_tile(t + 2, 0, kbuf(P), pk);
    if (t + 1 < n_tiles) dma_tile(t + 1, 1, vbuf(P ^ 1), pgv);
    if (active) {
      // the maximum of S(t) was taken before its mask: on the few tiles that need one, mask
      // and take it again
      if (needs_mask(t)) {
        mask(s_cur, t);
        mt_cur = row_max(s_cur);
      }
      if (__builtin_amdgcn_ballot_w64(mt_cur > m_ref + kSlack) != 0) {
        const float m_new = fmaxf(m_ref, mt_cur);
        const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_ref - m_new);
        l *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
        m_ref = m_new;
      }
      const float nm = (m_ref == -INFINITY) ? 0.f : -m_ref;
      const char *vl = vbuf(P);
      bf16x8 pb[4];
      qk(kbuf(P ^ 1), s_nxt);
      softmax_block(s_cur[0], nm, pb);
      softmax_half(s_cur[1], 0, nm, pb[2]);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
      }
      // O += V P and what follows run at a raised wave priority: of the two waves that share a
      // SIMD, the one in this phase issues first
      __builtin_amdgcn_s_setprio(kPrioPV);
      pv_step(vl, 0, pb[0]);
      pv_step(vl, 1, pb[1]);
      pv_step(vl, 2, pb[2]);
      softmax_half(s_cur[1], 1, nm, pb[3]);
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
#pragma unroll
      for (int i = 0; i < 12; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 1);
      }
      pv_step(vl, 3, pb[3]);
      cap(s_nxt);
      mt_cur = row_max(s_nxt);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 2);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 2);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    // pages for the next iteration's DMA (the LDS read overlaps the wait below)
    pgv = pk;
    if (t + 3 < n_tiles && full(t + 3)) pk = page_of(t + 3);
    // K[t + 2] and V[t + 1], issued above, are read in the next iteration
    wait_vm<0>();
    tile_barrier();
  };
  // Every iteration computes S(t + 1): on the last tile from a K buffer whose contents are
  // stale, a result never used.  A branch there would split the scheduled region, and peeling
  // the last tile off the loop made the register allocator spill.
  for (int t = 0; t < n_tiles; t += 2) {
    step(t, std::integral_constant<int, 0>{}, sa, sb);
    if (t + 1 < n_tiles) step(t + 1, std::integral_constant<int, 1>{}, sb, sa);
  }

  // ---- epilogue
  const float l_tot = sum_halves(l);
  float part_c = 0.f, part_sc = 0.f;
  if (uw.n_splits > 1) part_sc = part_scale(row_amax(o), l_tot, part_c);
  if (!active || q0 + j >= sp.len) return;
  const int row = q0 + j;
  if (uw.n_splits == 1) {
    const float inv = 1.0f / l_tot;
    uint16_t *orow = a.out + ((int64_t)(sp.q_start + row) * a.n_q_heads + qhead) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * db + 8 * gq + 4 * hh;
        *reinterpret_cast<u32x2 *>(orow + d0) =
            u32x2{pack_bf16x2(o[db][4 * gq + 0] * inv, o[db][4 * gq + 1] * inv),
                  pack_bf16x2(o[db][4 * gq + 2] * inv, o[db][4 * gq + 3] * inv)};
      }
  } else {
    const int64_t prow = ((int64_t)split * sp.len + row) * a.n_q_heads + qhead;
    store_partial<NDB, D>(o, part_sc, m_ref, l_tot, part_c, hh, a.ws, sp, prow);
  }
}

hipError_t launch_attn_d128_dma(const AttnArgs &args, const AttnPlan &plan, int n_kv, bool cap,
                                hipStream_t stream) {
  const dim3 grid(plan.units_per_head * n_kv);
  if (cap)
    hipLaunchKernelGGL(attn_bf16_d128_dma_kernel<true>, grid, dim3(256), 0, stream, args, plan);
  else
    hipLaunchKernelGGL(attn_bf16_d128_dma_kernel<false>, grid, dim3(256), 0, stream, args, plan);
  return hipGetLastError();
}

}  // namespace nexus
