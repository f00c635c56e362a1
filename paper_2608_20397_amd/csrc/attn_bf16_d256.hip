// bf16 suffix attention, head_dim 256 with a transposed (token-innermost) V cache: the layout and
// head size of the soft-capped model family of Sec. VI-B, fed by gfx950's LDS DMA loads
// (Sec. III-A; the re-decoded suffix of Sec. VI-A).
//
// Same work decomposition, math and split plan as the head_dim 128 DMA kernel (one KV head per
// workgroup, 4 waves of one query head x 32 queries, S^T = K.Q^T and O^T += V^T.P^T on
// 32x32x16 MFMA, online softmax in log2 units with a lazily moved reference, optional tanh
// soft-cap), with 32-key tiles and two workgroups per CU (two waves per SIMD: one workgroup's
// softmax runs beside the other's MFMAs; 64 KB of K/V buffers each).
//
// Key order.  The S^T MFMA leaves, for lane half h, tile rows {4h..4h+3, 8+4h..8+4h+3} of each
// 16-row group in a lane, while the PV B operand wants 8 consecutive keys per lane half.  The K
// tile is therefore DMA'd with its rows permuted: tile row r holds key r with bits 2 and 3
// swapped (within the row's page, so every wave's rows still come from one page).  The scores a
// lane holds are then keys 8h..8h+7 (+16) in order: P^T feeds the PV MFMA as computed, and the
// transposed V tile ([feature][key], 64 bytes per feature row) is DMA'd in natural key order,
// each lane's 16 bytes being 8 keys of one feature, read back with one ds_read_b128.
// LDS tiles: K rows go in pairs (one DMA instruction each), pair p at p * 1056 bytes (32 bytes of
// padding per pair), row r of the pair at + 512 r, its 16-byte chunk c at c ^ r; V^T row d
// (64 B) holds chunk c at c ^ ((d >> 2) & 3).  Both keep the 16-byte operand reads of a wave
// free of bank conflicts, and the K operand offsets of all 16 k-steps differ by constants.
//
// The last tile of a workgroup may reach past its last key: K rows there are clamped to the
// last key (finite, masked), and the V^T entries of those keys, which may hold anything, are
// set to zero in LDS once the tile has landed (their weights are zero, and 0 x NaN would not be).
#include "attn_common.h"
#include "attn_dma.h"
#include "launch.h"

#include <type_traits>

namespace nexus {

template <bool CAP>
__global__ __launch_bounds__(256, 2) void attn_bf16_d256_vt_kernel(const AttnArgs a,
                                                                   const AttnPlan plan) {
  constexpr int D = 256, KT = 32;
  constexpr int NS = D / 16;                  // k-steps of Q K^T
  constexpr int NDB = D / 32;                 // 32-row blocks of O^T
  constexpr int KROWB = D * 2;                // bytes per K row
  constexpr int VROWB = KT * 2;               // bytes per V^T tile row (one feature)
  constexpr int PAIRB = 2 * KROWB + 32;       // bytes per K row pair, padded
  constexpr int KTILEB = (KT / 2) * PAIRB;    // bytes per K tile
  constexpr int VTILEB = D * VROWB;           // bytes per V^T tile
  constexpr float kSlack = 8.0f;              // lazy rescale: p <= 2^8 between rescales
  constexpr int kPrioPV = 2;                  // wave priority of the PV phase
  __shared__ __align__(1024) char smem[2 * KTILEB + 2 * VTILEB];   // K 0, 1, V^T 0, 1
  __shared__ __align__(16) int32_t pg[kMaxSplitKeys / kPage + 8];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int j = lane & 31, hh = lane >> 5;
  const int kvh = blockIdx.x % a.n_kv_heads;
  const UnitLoc loc = locate_unit(plan, blockIdx.x / a.n_kv_heads);
  const SeqPlan sp = plan.seq[loc.seq];
  const UnitWork uw = loc.w;
  const int G = a.group;

  const int task = uw.tgrp * kWaves + wave;
  const bool active = task < sp.n_tasks;
  const int qb = task / G;
  const int g = task - qb * G;
  const int q0 = qb * kQB;
  const int qhead = kvh * G + g;
  const int last_task = min(uw.tgrp * kWaves + kWaves - 1, sp.n_tasks - 1);
  const int last_q = min((last_task / G + 1) * kQB, sp.len);
  const int wg_keys = (int)sp.n_past + last_q;
  const int k_begin = uw.k_begin;
  const int k_end = min(k_begin + uw.split_keys, wg_keys);
  const int wave_keys = active ? (int)sp.n_past + min(q0 + kQB, sp.len) : 0;
  const int qpos0 = (int)sp.n_past + q0;
  const int n_tiles = k_end > k_begin ? (k_end - k_begin + KT - 1) / KT : 0;

  const int pg0 = k_begin >> kPageShift;
  const int n_pg = n_tiles > 0 ? ((k_end - 1) >> kPageShift) - pg0 + 1 : 0;
  for (int i = tid; i < n_pg; i += 256) pg[i] = a.map[pg0 + i];

  // Q of this wave as B operands: lane (hh, j) holds Q[q0 + j][16 s + 8 hh .. + 7]
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

  // ---- lane-invariant LDS read offsets.  K: row j, chunk 2s + hh at (2s + hh) ^ (j & 1), i.e.
  // 32 s + 16 (hh ^ (j & 1)) into the row
  const uint32_t offk = (j >> 1) * PAIRB + (j & 1) * KROWB + 16 * (hh ^ (j & 1));
  // V^T: feature row 32 db + j, chunk 2 ks + hh at (2 ks + hh) ^ ((j >> 2) & 3)
  uint32_t offv[KT / 16];
#pragma unroll
  for (int ks = 0; ks < KT / 16; ++ks) offv[ks] = j * VROWB + (((2 * ks + hh) ^ ((j >> 2) & 3)) * 16);

  // ---- DMA.  K: wave w fills tile rows 8w .. 8w + 7 (keys of page w / 2), one row pair per
  // instruction; lane (h = lane / 32, slot = lane % 32) of instruction i fills row
  // r = 8w + 2i + h, position slot, with chunk slot ^ h of key perm(r), where
  // perm(r) & 15 = 8 (i / 2) + 4 (w & 1) + 2 (i & 1) + h.
  const int slot = lane & 31, h1 = lane >> 5;
  const uint32_t kdo = (uint32_t)(4 * (wave & 1) + h1) * KROWB + (uint32_t)((slot ^ h1) * 16);
  // V^T: wave w fills feature rows 64w .. 64w + 63, 16 per instruction; lane (r4 = lane / 4,
  // q = lane % 4) fills row 64w + 16i + r4, position q, with key chunk q ^ ((lane >> 4) & 3).
  const int vchunk = (lane & 3) ^ ((lane >> 4) & 3);
  const uint32_t n_cols = (uint32_t)a.n_phys_pages * kPage;        // V^T row length
  const uint32_t vrow0 = (uint32_t)(64 * wave + (lane >> 2)) * n_cols * 2u;
  const uint32_t vrow_step = 16u * n_cols * 2u;                    // 16 feature rows
  const uint32_t smem_base = (uint32_t)(uintptr_t)smem;
  const uint64_t pbytes = (uint64_t)a.n_kv_heads * kPage * KROWB;   // one physical K page
  const char *kbytes = reinterpret_cast<const char *>(a.kc) + (uint64_t)kvh * kPage * KROWB;
  const char *vtbytes = reinterpret_cast<const char *>(a.vc) + (uint64_t)kvh * D * n_cols * 2u;
  auto kbuf = [&](int i) { return smem + i * KTILEB; };
  auto vbuf = [&](int i) { return smem + 2 * KTILEB + i * VTILEB; };
  auto full = [&](int it) { return k_begin + it * KT + KT <= k_end; };

  // Q and the page table are waited for before any DMA is in flight (the compiler's own vmcnt
  // bookkeeping must never count DMA loads)
  wait_vm<0>();
  __syncthreads();   // pg[] visible

  auto dma_k = [&](int it, char *dstp) {
    const int kt = k_begin + it * KT;
    const uint32_t dst = smem_base + (uint32_t)(dstp - smem) + wave * 4 * PAIRB;
    if (full(it)) {
      const uint32_t page =
          (uint32_t)__builtin_amdgcn_readfirstlane(pg[it * (KT / kPage) + (wave >> 1)]);
      const char *ps = kbytes + page * pbytes;
      dma_s<0>(dst, ps, kdo);
      dma_s<0>(dst + PAIRB, ps + 2 * KROWB, kdo);
      dma_s<0>(dst + 2 * PAIRB, ps + 8 * KROWB, kdo);
      dma_s<0>(dst + 3 * PAIRB, ps + 10 * KROWB, kdo);
    } else {
      const int tl = k_end - 1;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 8 * wave + 2 * i + h1;
        const int key = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
        const int t = min(kt + key, tl);
        const uint64_t pp = (uint32_t)pg[(t >> kPageShift) - pg0];
        const uint32_t c = (uint32_t)(slot ^ h1);
        dma_v(dst + i * PAIRB, kbytes + pp * pbytes + (uint32_t)(t & (kPage - 1)) * KROWB + c * 16);
      }
    }
  };
  auto dma_vt = [&](int it, char *dstp) {
    const uint32_t dst = smem_base + (uint32_t)(dstp - smem) + wave * 64 * VROWB;
    // the page of this lane's 8 keys; past the last page (a partial last tile) the last page is
    // read and those keys are zeroed after arrival
    const int pi = min(it * (KT / kPage) + (vchunk >> 1), n_pg - 1);
    const uint32_t col = ((uint32_t)pg[pi] * kPage + 8u * (vchunk & 1)) * 2u;
    const uint32_t vo = vrow0 + col;
    dma_s<0>(dst, vtbytes, vo);
    dma_s<0>(dst + 1024, vtbytes, vo + vrow_step);
    dma_s<0>(dst + 2048, vtbytes, vo + 2 * vrow_step);
    dma_s<0>(dst + 3072, vtbytes, vo + 3 * vrow_step);
  };
  // zero the V^T entries of keys past k_end in a landed partial tile (thread = feature row)
  auto fix_vt = [&](int it, char *vl) {
    const int nvalid = k_end - (k_begin + it * KT);
    const int d = tid;
    uint16_t *row = reinterpret_cast<uint16_t *>(vl + d * VROWB);
    for (int k = nvalid; k < KT; ++k)
      row[8 * ((k >> 3) ^ ((d >> 2) & 3)) + (k & 7)] = 0;
  };

  const float c_scale = a.scale_log2;   // raw score -> log2 units (no cap)
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  if (n_tiles > 0) {
    dma_k(0, kbuf(0));
    dma_vt(0, vbuf(0));
  }
  wait_vm<0>();
  tile_barrier();
  if (n_tiles > 0 && !full(0)) {
    fix_vt(0, vbuf(0));
    tile_barrier();
  }

  auto step = [&](int t, auto parity) {
    constexpr int P = decltype(parity)::value;     // t & 1
    const int kt = k_begin + t * KT;
    if (t + 1 < n_tiles) {
      dma_k(t + 1, kbuf(P ^ 1));
      dma_vt(t + 1, vbuf(P ^ 1));
    }
    if (active && kt < wave_keys) {
      // ---- S^T = K . Q^T (tile rows in permuted key order)
      f32x16 sc;
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[v] = 0.f;
      const char *kl = kbuf(P);
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kl + offk + 32 * s);
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[s], sc, 0, 0, 0);
      }
      // soft cap: sc holds r = 1 / (2^(s cap_k) + 1), the capped score being cap_out (1 - 2 r)
      if constexpr (CAP) {
#pragma unroll
        for (int v = 0; v < 16; ++v) sc[v] = cap_r(sc[v], a.cap_k);
      }
      // ---- causal / tail mask: register v of lane half hh holds key kt + (v & 7) + 8 hh +
      // 16 (v >> 3); a masked score is -inf (r = +inf)
      constexpr float kMasked = CAP ? INFINITY : -INFINITY;
      if ((kt + KT > k_end) || (kt + KT - 1 > qpos0)) {
        const int lim = min(qpos0 + j, k_end - 1) - kt - 8 * hh;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if ((v & 7) + 16 * (v >> 3) > lim) sc[v] = kMasked;
      }
      // ---- online softmax (log2 units), lazily rescaled
      float mt;
      if constexpr (CAP) {
        float rmin = INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) rmin = fminf(rmin, sc[v]);
        rmin = -max_halves(-rmin);
        mt = fmaf(rmin, -2.0f * a.cap_out, a.cap_out);    // -inf when every key is masked
      } else {
        mt = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[v]);
        mt = max_halves(mt) * c_scale;
      }
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
      // p = 2^(score - m_ref): fma(s, scale, -m_ref), or with the cap fma(r, -2 cap_out,
      // cap_out - m_ref)
      const float pa = CAP ? -2.0f * a.cap_out : c_scale;
      const float pc = CAP ? a.cap_out + nm : nm;
      bf16x8 pb[KT / 16];
#pragma unroll
      for (int ks = 0; ks < KT / 16; ++ks) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = fast_exp2(fmaf(sc[8 * ks + 2 * e], pa, pc));
          const float p1 = fast_exp2(fmaf(sc[8 * ks + 2 * e + 1], pa, pc));
          w[e] = pack_bf16x2(p0, p1);
          l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, l, false);
        }
        pb[ks] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
      }
      // ---- O^T += V^T . P^T, at a raised wave priority: of the two waves sharing a SIMD, the
      // one in this phase issues first
      __builtin_amdgcn_s_setprio(kPrioPV);
      const char *vl = vbuf(P);
#pragma unroll
      for (int ks = 0; ks < KT / 16; ++ks)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8 va =
              *reinterpret_cast<const bf16x8 *>(vl + offv[ks] + db * 32 * VROWB);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[ks], o[db], 0, 0, 0);
        }
      __builtin_amdgcn_s_setprio(0);
    }
    // tile t + 1, issued above, is read in the next step
    wait_vm<0>();
    tile_barrier();
    if (t + 1 < n_tiles && !full(t + 1)) {
      fix_vt(t + 1, vbuf(P ^ 1));
      tile_barrier();
    }
  };
  for (int t = 0; t < n_tiles; t += 2) {
    step(t, std::integral_constant<int, 0>{});
    if (t + 1 < n_tiles) step(t + 1, std::integral_constant<int, 1>{});
  }

  // ---- epilogue
  const float l_tot = sum_halves(l);
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
    const int64_t prow = ((int64_t)uw.split * sp.len + row) * a.n_q_heads + qhead;
    float *op = a.ws + sp.ws_off + prow * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * db + 8 * gq + 4 * hh;
        *reinterpret_cast<f32x4 *>(op + d0) =
            f32x4{o[db][4 * gq + 0], o[db][4 * gq + 1], o[db][4 * gq + 2], o[db][4 * gq + 3]};
      }
    if (hh == 0) *reinterpret_cast<f32x2 *>(a.ws + sp.ml_off + prow * 2) = f32x2{m_ref, l_tot};
  }
}

hipError_t launch_attn_d256_vt(const AttnArgs &args, const AttnPlan &plan, int n_kv, bool cap,
                               hipStream_t stream) {
  const dim3 grid(plan.units_per_head * n_kv);
  if (cap)
    hipLaunchKernelGGL(attn_bf16_d256_vt_kernel<true>, grid, dim3(256), 0, stream, args, plan);
  else
    hipLaunchKernelGGL(attn_bf16_d256_vt_kernel<false>, grid, dim3(256), 0, stream, args, plan);
  return hipGetLastError();
}

}  // namespace nexus
