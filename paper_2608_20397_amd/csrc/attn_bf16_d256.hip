// bf16 suffix attention, head_dim 256 with a transposed (token-innermost) V cache: the layout and
// head size of the soft-capped model family of Sec. VI-B, fed by gfx950's LDS DMA loads
// (Sec. III-A; the re-decoded suffix of Sec. VI-A).
//
// Same math and split plan as the head_dim 128 DMA kernel (S^T = K.Q^T and O^T += V^T.P^T on
// 32x32x16 MFMA, online softmax in log2 units with a lazily moved reference, optional tanh
// soft-cap), with 32-key tiles and one workgroup of 8 wave tasks (query head x 32 queries) per
// CU, two waves per SIMD, all eight fed from one K / V^T ring (each tile crosses L2 -> LDS once
// per 256 query rows).
//
// Schedule.  Per tile t a wave computes S(t + 1) = K(t + 1) Q^T beside the exponentials of S(t),
// then O += V(t) P(t) beside the soft cap of S(t + 1) (with the cap a score costs three
// transcendentals).  Each of the two phases is written as 16 chunks of one MFMA, its operand
// reads two MFMAs ahead (three rotating registers) and a few vector instructions, with the chunk
// order pinned by sched_barrier: left to the compiler, the phases either ran their matrix and
// vector work one after the other or, under register pressure, single-buffered the operand reads
// and waited out every LDS read.  The cap is split in two stages so that both phases carry about
// as much vector work as matrix work.  Registers: O^T takes 128 and S(t), S(t + 1) 32 of the 256
// a wave has at two waves per SIMD, so Q keeps k-steps 0..5 (features 0..95) in registers and
// 6..15 in LDS (10 KB per wave, read as MFMA operands beside the K tile).
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
__global__ __launch_bounds__(64 * kWavesWide, 1) void attn_bf16_d256_vt_kernel(
    const AttnArgs a, const AttnPlan plan) {
  constexpr int W = kWavesWide;               // wave tasks (and waves) per workgroup
  constexpr int D = 256, KT = 32;
  constexpr int NS = D / 16;                  // k-steps of Q K^T
  constexpr int NSR = 6;                      // k-steps whose Q operand stays in registers
  constexpr int NDB = D / 32;                 // 32-row blocks of O^T
  constexpr int KROWB = D * 2;                // bytes per K row
  constexpr int VROWB = KT * 2;               // bytes per V^T tile row (one feature)
  constexpr int PAIRB = 2 * KROWB + 32;       // bytes per K row pair, padded
  constexpr int KTILEB = (KT / 2) * PAIRB;    // bytes per K tile
  constexpr int VTILEB = D * VROWB;           // bytes per V^T tile
  constexpr int NB = 2;                       // ring depth (K and V^T)
  constexpr int V0 = NB * KTILEB;             // V^T ring base
  constexpr int QL0 = V0 + NB * VTILEB;       // upper Q halves, (NS - NSR) KB per wave
  constexpr int QLB = (NS - NSR) * 1024;
  constexpr float kSlack = 8.0f;              // lazy rescale: p <= 2^8 between rescales
  __shared__ __align__(1024) char smem[QL0 + W * QLB];
  __shared__ __align__(16) int32_t pg[kMaxSplitKeys / kPage + 8];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int j = lane & 31, hh = lane >> 5;
  const int kvh = blockIdx.x % a.n_kv_heads;
  const UnitLoc loc = locate_unit(plan, blockIdx.x / a.n_kv_heads);
  const SeqPlan sp = plan.seq[loc.seq];
  const UnitWork uw = loc.w;
  const int G = a.group;

  const int task = uw.tgrp * W + wave;
  const bool active = task < sp.n_tasks;
  const int qb = task / G;
  const int g = task - qb * G;
  const int q0 = qb * kQB;
  const int qhead = kvh * G + g;
  const int last_task = min(uw.tgrp * W + W - 1, sp.n_tasks - 1);
  const int last_q = min((last_task / G + 1) * kQB, sp.len);
  const int wg_keys = (int)sp.n_past + last_q;
  const int k_begin = uw.k_begin;
  const int k_end = min(k_begin + uw.split_keys, wg_keys);
  const int qpos0 = (int)sp.n_past + q0;
  const int n_tiles = k_end > k_begin ? (k_end - k_begin + KT - 1) / KT : 0;

  const int pg0 = k_begin >> kPageShift;
  const int n_pg = n_tiles > 0 ? ((k_end - 1) >> kPageShift) - pg0 + 1 : 0;
  for (int i = tid; i < n_pg; i += 64 * W) pg[i] = a.map[pg0 + i];

  // Q of this wave as B operands: lane (hh, j) holds Q[q0 + j][16 s + 8 hh .. + 7]; k-steps
  // s < NSR in registers, the others in LDS at QL0 + wave * QLB + (s - NSR) * 1024 + 16 lane
  // (loaded once the first tiles' DMA is in flight, so that the two latencies overlap)
  bf16x8 qreg[NSR];
  const uint32_t qlds_off = QL0 + wave * QLB + 16 * lane;
  // (the LDS offsets live in registers, hidden from the compiler, so that buffer and block
  // offsets fit the 16-bit immediate of the LDS reads)
  uint32_t oq = qlds_off;
  asm volatile("" : "+v"(oq));

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
  for (int ks = 0; ks < KT / 16; ++ks) {
    offv[ks] = V0 + j * VROWB + (((2 * ks + hh) ^ ((j >> 2) & 3)) * 16);
    asm volatile("" : "+v"(offv[ks]));
  }

  // ---- DMA.  K: wave w fills tile rows 4w .. 4w + 3 (two row pairs of page w / 4), one pair per
  // instruction; lane (h = lane / 32, slot = lane % 32) of instruction i fills row r = 4w + 2i + h,
  // position slot, with chunk slot ^ h of key perm(r), whose place in the page is
  // 8 (w & 1) + 4 ((w >> 1) & 1) + 2i + h.
  const int slot = lane & 31, h1 = lane >> 5;
  const uint32_t kdo = (uint32_t)h1 * KROWB + (uint32_t)((slot ^ h1) * 16);
  const uint32_t kkey0 = 8u * (wave & 1) + 4u * ((wave >> 1) & 1);
  // V^T: wave w fills feature rows 32w .. 32w + 31, 16 per instruction; lane (r4 = lane / 4,
  // q = lane % 4) fills row 32w + 16i + r4, position q, with key chunk q ^ ((lane >> 4) & 3).
  const int vchunk = (lane & 3) ^ ((lane >> 4) & 3);
  const uint32_t n_cols = (uint32_t)a.n_phys_pages * kPage;        // V^T row length
  const uint32_t vrow0 = (uint32_t)(32 * wave + (lane >> 2)) * n_cols * 2u;
  const uint32_t vrow_step = 16u * n_cols * 2u;                    // 16 feature rows
  const uint32_t smem_base = (uint32_t)(uintptr_t)smem;
  const uint64_t pbytes = (uint64_t)a.n_kv_heads * kPage * KROWB;   // one physical K page
  const char *kbytes = reinterpret_cast<const char *>(a.kc) + (uint64_t)kvh * kPage * KROWB;
  const char *vtbytes = reinterpret_cast<const char *>(a.vc) + (uint64_t)kvh * D * n_cols * 2u;
  auto kbuf = [&](int i) { return smem + i * KTILEB; };
  auto vbuf = [&](int i) { return smem + V0 + i * VTILEB; };
  // V^T buffer i as the operand reads see it (their offsets carry the ring base)
  auto vrd = [&](int i) { return smem + i * VTILEB; };
  auto full = [&](int it) { return k_begin + it * KT + KT <= k_end; };

  // the page table is waited for before any DMA is in flight (the compiler's own vmcnt
  // bookkeeping must never count DMA loads)
  wait_vm<0>();
  __syncthreads();   // pg[] visible

  // page numbers of a tile's DMA, read from the LDS page table a step before they are used
  auto k_page = [&](int it) { return pg[max(min(it * (KT / kPage) + (wave >> 2), n_pg - 1), 0)]; };
  auto v_page = [&](int it) { return pg[max(min(it * (KT / kPage) + (vchunk >> 1), n_pg - 1), 0)]; };
  auto dma_k = [&](int it, char *dstp, int kpage) {
    const int kt = k_begin + it * KT;
    const uint32_t dst = smem_base + (uint32_t)(dstp - smem) + wave * 2 * PAIRB;
    if (full(it)) {
      const uint32_t page = (uint32_t)__builtin_amdgcn_readfirstlane(kpage);
      const char *ps = kbytes + page * pbytes + kkey0 * KROWB;
      dma_s<0>(dst, ps, kdo);
      dma_s<0>(dst + PAIRB, ps + 2 * KROWB, kdo);
    } else {
      const int tl = k_end - 1;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r = 4 * wave + 2 * i + h1;
        const int key = (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
        const int t = min(kt + key, tl);
        const uint64_t pp = (uint32_t)pg[(t >> kPageShift) - pg0];
        const uint32_t c = (uint32_t)(slot ^ h1);
        dma_v(dst + i * PAIRB, kbytes + pp * pbytes + (uint32_t)(t & (kPage - 1)) * KROWB + c * 16);
      }
    }
  };
  auto dma_vt = [&](char *dstp, int vpage) {
    const uint32_t dst = smem_base + (uint32_t)(dstp - smem) + wave * 32 * VROWB;
    // vpage: the page of this lane's 8 keys; past the last page (a partial last tile) the last
    // page is read and those keys are zeroed after arrival
    const uint32_t col = ((uint32_t)vpage * kPage + 8u * (vchunk & 1)) * 2u;
    const uint32_t vo = vrow0 + col;
    dma_s<0>(dst, vtbytes, vo);
    dma_s<0>(dst + 1024, vtbytes, vo + vrow_step);
  };
  // zero the V^T entries of keys past k_end in a landed partial tile: lanes 0..31 of wave w take
  // the feature rows 32w .. 32w + 31 that this wave loaded
  auto fix_vt = [&](int it, char *vl) {
    if (lane >= 32) return;
    const int nvalid = k_end - (k_begin + it * KT);
    const int d = 32 * wave + lane;
    uint16_t *row = reinterpret_cast<uint16_t *>(vl + d * VROWB);
    for (int k = nvalid; k < KT; ++k)
      row[8 * ((k >> 3) ^ ((d >> 2) & 3)) + (k & 7)] = 0;
  };

  const float c_scale = a.scale_log2;   // raw score -> log2 units (no cap)
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
  constexpr float kMasked = CAP ? INFINITY : -INFINITY;   // a masked score (r = +inf with the cap)

  // S^T of one tile (rows in permuted key order) from the K buffer at `kl`
  auto qk = [&](const char *kl, f32x16 &sc) __attribute__((always_inline)) {
#pragma unroll
    for (int v = 0; v < 16; ++v) sc[v] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(kl + offk + 32 * s);
      const bf16x8 qs = s < NSR ? qreg[s < NSR ? s : 0]
                                : *reinterpret_cast<const bf16x8 *>(smem + oq + (s - NSR) * 1024);
      sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qs, sc, 0, 0, 0);
    }
  };
  // Soft cap in two stages.  The capped score is cap_out (1 - 2 r) with r = 1 / e,
  // e = 2^(s cap_k) + 1 (e overflowing to +inf gives the cap itself, e = 1 its negative).  The
  // first stage, beside the PV MFMAs, leaves e in registers 8..15 and r in 0..7; the second,
  // beside the next tile's score MFMAs, takes the reciprocals of 8..15.  A masked score is
  // r = +inf (registers 0..7) or e = 0 (8..15).
  auto cap = [&](f32x16 &sc) __attribute__((always_inline)) {
    if constexpr (CAP) {
#pragma unroll
      for (int v = 0; v < 16; ++v) sc[v] = fast_exp2(sc[v] * a.cap_k) + 1.0f;
#pragma unroll
      for (int v = 0; v < 8; ++v) sc[v] = __builtin_amdgcn_rcpf(sc[v]);
    }
  };
  // causal / tail mask of tile t: register v of lane half hh holds key kt + (v & 7) + 8 hh +
  // 16 (v >> 3)
  auto needs_mask = [&](int t) {
    const int kt = k_begin + t * KT;
    return (kt + KT > k_end) || (kt + KT - 1 > qpos0);
  };
  auto mask = [&](f32x16 &sc, int t) __attribute__((always_inline)) {
    const int lim = min(qpos0 + j, k_end - 1) - (k_begin + t * KT) - 8 * hh;
#pragma unroll
    for (int v = 0; v < 16; ++v)
      if ((v & 7) + 16 * (v >> 3) > lim) sc[v] = (CAP && v >= 8) ? 0.f : kMasked;
  };
  // row maximum in log2 units (-inf when every key is masked; with the cap, of scores after its
  // first stage), in two steps: the lane's own registers, then across the two lane halves (a
  // cross-lane operation, kept out of the pinned regions)
  auto row_max_lane = [&](const f32x16 &sc) __attribute__((always_inline)) -> float {
    if constexpr (CAP) {
      // largest score = smallest r = 1 / largest e
      float rmin = INFINITY, emax = 0.f;
#pragma unroll
      for (int v = 0; v < 8; ++v) rmin = fminf(rmin, sc[v]);
#pragma unroll
      for (int v = 8; v < 16; ++v) emax = fmaxf(emax, sc[v]);
      return fmaxf(emax, __builtin_amdgcn_rcpf(rmin));
    } else {
      float mt = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[v]);
      return mt;
    }
  };
  auto row_max_finish = [&](float x) __attribute__((always_inline)) -> float {
    if constexpr (CAP)
      return fmaf(__builtin_amdgcn_rcpf(max_halves(x)), -2.0f * a.cap_out, a.cap_out);
    else
      return max_halves(x) * c_scale;
  };
  auto row_max = [&](const f32x16 &sc) __attribute__((always_inline)) -> float {
    return row_max_finish(row_max_lane(sc));
  };
  // S^T of the K tile at `kl` into sn, beside P = 2^(score - m_ref) of the scores in sc (after
  // the second cap stage), packed to bf16 into pb and summed into l: p = 2^fma(s, scale, -m_ref),
  // or with the cap 2^fma(r, -2 cap_out, cap_out - m_ref).  Chunk i issues the operand
  // reads of k-step i + 2 (three rotating registers each), MFMA i, the reciprocal of score
  // register 8 + i (i < 8, with the cap) and the exponential of score register i, its order
  // pinned by sched_barrier
  auto qk_exp = [&](const char *kl, f32x16 &sn, f32x16 &sc, float nm, bf16x8 *pb)
      __attribute__((always_inline)) {
    const float pa = CAP ? -2.0f * a.cap_out : c_scale;
    const float pc = CAP ? a.cap_out + nm : nm;
    auto kread = [&](int k) { return *reinterpret_cast<const bf16x8 *>(kl + offk + 32 * k); };
    auto qread = [&](int k) {
      return *reinterpret_cast<const bf16x8 *>(smem + oq + (k - NSR) * 1024);
    };
    bf16x8 kb[3], qb[3];
    kb[0] = kread(0);
    kb[1] = kread(1);
    if (0 >= NSR) qb[0] = qread(0);
    if (1 >= NSR) qb[1] = qread(1);
#pragma unroll
    for (int v = 0; v < 16; ++v) sn[v] = 0.f;
    uint32_t w[8];
    float p_even = 0.f;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      if (i + 2 < NS) {
        kb[(i + 2) % 3] = kread(i + 2);
        if (i + 2 >= NSR) qb[(i + 2) % 3] = qread(i + 2);
      }
      sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[i % 3], i < NSR ? qreg[i < NSR ? i : 0]
                                                                  : qb[i % 3], sn, 0, 0, 0);
      if constexpr (CAP) {
        if (i < 8) sc[8 + i] = __builtin_amdgcn_rcpf(sc[8 + i]);
      }
      const float p = fast_exp2(fmaf(sc[i], pa, pc));
      if (i & 1) {
        w[i >> 1] = pack_bf16x2(p_even, p);
        l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[i >> 1]), ones, l, false);
      } else {
        p_even = p;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    pb[0] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    pb[1] = __builtin_bit_cast(bf16x8, u32x4{w[4], w[5], w[6], w[7]});
  };
  // O^T += V^T P^T over the V^T tile at `vl`, beside the first cap stage of sn
  auto pv_cap = [&](const char *vl, const bf16x8 *pb, f32x16 &sn) __attribute__((always_inline)) {
    constexpr int NM = NDB * (KT / 16);
    auto vread = [&](int i) {
      return *reinterpret_cast<const bf16x8 *>(vl + offv[i / NDB] + (i % NDB) * 32 * VROWB);
    };
    bf16x8 vb[3];
    vb[0] = vread(0);
    vb[1] = vread(1);
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      if (i + 2 < NM) vb[(i + 2) % 3] = vread(i + 2);
      o[i % NDB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vb[i % 3], pb[i / NDB], o[i % NDB],
                                                           0, 0, 0);
      if constexpr (CAP) {
        sn[i] = fast_exp2(sn[i] * a.cap_k) + 1.0f;
        if (i < 8) sn[i] = __builtin_amdgcn_rcpf(sn[i]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  const int T = n_tiles;
  if (T > 0) {
    dma_k(0, kbuf(0), k_page(0));
    dma_vt(vbuf(0), v_page(0));
  }
  if (T > 1) dma_k(1, kbuf(1), k_page(1));
  int kp_next = k_page(2), vp_next = v_page(1);   // pages of K(t + 2) and V^T(t + 1), t = 0
  // Q, behind the DMA: the compiler's waits for these loads count only loads issued after
  // them, and the DMA loads, issued earlier, complete first
  if (active) {
    const int qi = min(q0 + j, sp.len - 1);
    const uint16_t *qrow = a.q + ((int64_t)(sp.q_start + qi) * a.n_q_heads + qhead) * D;
#pragma unroll
    for (int s = 0; s < NSR; ++s)
      qreg[s] = *reinterpret_cast<const bf16x8 *>(qrow + 16 * s + 8 * hh);
#pragma unroll
    for (int s = NSR; s < NS; ++s)
      *reinterpret_cast<bf16x8 *>(smem + qlds_off + (s - NSR) * 1024) =
          *reinterpret_cast<const bf16x8 *>(qrow + 16 * s + 8 * hh);
  }
  wait_vm<0>();
  if (T == 1 && !full(0)) fix_vt(0, vbuf(0));
  tile_barrier();

  // Pipeline, per iteration t: S(t + 1) = K(t + 1) Q^T beside the exponentials of S(t), then
  // O += V(t) P(t) beside the soft cap of S(t + 1), whose maximum the next iteration's rescale
  // needs.  The pinned regions have no branch; the causal and tail masks, needed on few tiles,
  // are applied at the top of the next iteration.
  f32x16 sa, sb;
  float mt_cur = -INFINITY;                     // row maximum of S(t), log2 units
  if (active && T > 0) {
    qk(kbuf(0), sa);
    cap(sa);
    mt_cur = row_max(sa);        // unmasked: iteration 0 masks S(0) and takes its maximum again
  }
  tile_barrier();                // every wave has read K(0): its buffer may be refilled

  auto step = [&](int t, auto par, f32x16 &s_cur, f32x16 &s_nxt) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;     // t % NB
    constexpr int P1 = (P + 1) % NB;
    // K(t + 2) into the buffer of K(t) (read in iteration t - 1), V^T(t + 1) into that of
    // V^T(t - 1) (iteration t - 1)
    if (t + 2 < T) dma_k(t + 2, kbuf(P), kp_next);
    if (t + 1 < T) dma_vt(vbuf(P1), vp_next);
    kp_next = k_page(t + 3);
    vp_next = v_page(t + 2);
    if (active) {
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
      bf16x8 pb[KT / 16];
      // S(t + 1) (on the last tile from a stale K buffer: a result never used) beside the
      // second cap stage and the exponentials of S(t), in 16 pinned chunks
      qk_exp(kbuf(P1), s_nxt, s_cur, nm, pb);
      // O += V P beside the first cap stage of S(t + 1), in 16 chunks whose order is pinned
      // (sched_barrier): chunk i issues the V^T operand read of MFMA i + 2 (three rotating
      // operand registers), MFMA i (ks = i / 8, db = i % 8) and the cap of score register i
      pv_cap(vrd(P), pb, s_nxt);
      mt_cur = row_max(s_nxt);
    }
    wait_vm<0>();
    // a partial last tile: zero its V^T entries past k_end in the feature rows this wave loaded
    if (t + 1 == T - 1 && !full(T - 1)) fix_vt(T - 1, vbuf(P1));
    tile_barrier();
  };
  for (int t = 0; t < T; t += 2) {
    step(t, std::integral_constant<int, 0>{}, sa, sb);
    if (t + 1 < T) step(t + 1, std::integral_constant<int, 1>{}, sb, sa);
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
    const int64_t prow = ((int64_t)uw.split * sp.len + row) * a.n_q_heads + qhead;
    store_partial<NDB, D>(o, part_sc, m_ref, l_tot, part_c, hh, a.ws, sp, prow);
  }
}

hipError_t launch_attn_d256_vt(const AttnArgs &args, const AttnPlan &plan, int n_kv, bool cap,
                               hipStream_t stream) {
  const dim3 grid(plan.units_per_head * n_kv);
  const dim3 block(64 * kWavesWide);
  if (cap)
    hipLaunchKernelGGL(attn_bf16_d256_vt_kernel<true>, grid, block, 0, stream, args, plan);
  else
    hipLaunchKernelGGL(attn_bf16_d256_vt_kernel<false>, grid, block, 0, stream, args, plan);
  return hipGetLastError();
}

}  // namespace nexus
