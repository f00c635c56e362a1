// bf16 suffix attention, head_dim 128 with a row-major V cache: the variant that feeds LDS with
// gfx950's LDS DMA loads (Sec. III-A; the re-decoded suffix of Sec. VI-A).
//
// Same math as attn_bf16_kernel (S^T = K.Q^T and O^T += V^T.P^T on 32x32x16 MFMA, online softmax
// in log2 units with a lazily moved reference), organised for one wave per SIMD:
//   * one KV head per workgroup, 4 waves; each wave owns one query head x 64 queries, held as two
//     32-query blocks, so every K or V operand read from LDS feeds two MFMAs' worth of queries
//     over a tile and the 512-register budget of a lone wave holds both blocks' O;
//   * K and V tiles (64 keys) travel global -> LDS with global_load_lds_dwordx4 through a
//     4-stage ring, three tiles ahead of the one being consumed: each lane's 16 bytes land at
//     base + 16 * lane, so the XOR swizzles below are produced by choosing each lane's source
//     chunk; no staging registers, no LDS write instructions;
//   * a tile's 64 keys are 4 pages, one per wave, so the page address is wave-uniform;
//   * per tile the wave runs S(block 0) on the MFMA pipe, then S(block 1) while the VALU turns
//     block 0's scores into probabilities, then O(block 0) while the VALU does block 1, then
//     O(block 1): the exponentials hide under MFMA work of the same wave;
//   * the PV A operand (8 keys of one feature) comes from the row-major V tile through two
//     ds_read_b64_tr_b16: in each 16-lane group, output lane i receives element i % 4 of the
//     8 bytes that source lane 4e + i / 4 points at, e = 0..3.  Source lane 4e + q points at
//     V[key_e][d0 + 4q], so output lane i receives V[key_0..3][d0 + i].  The keys each lane
//     needs follow the score layout of the S^T MFMA (keys 4h..4h+3 and 8+4h..8+4h+3 of a
//     16-key step for lane half h).
// LDS tiles: K row r (256 B) holds chunk c at c ^ (r & 15); V row r holds chunk c at
// c ^ 4 (r & 3).  Both keep the 16-byte K reads and the 8-byte transposed V reads of a wave free
// of bank conflicts.
// Built with the MFMA accumulators in VGPRs (-amdgpu-mfma-vgpr-form): with AGPR accumulators the
// register allocator shuttles O between the two files every tile.
#include "attn_common.h"
#include "launch.h"

namespace nexus {

namespace {

typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ bf16x8 tr_read_pair(const char *lo, const char *hi) {
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)lo);
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)hi);
  const u32x2 ua = __builtin_bit_cast(u32x2, a);
  const u32x2 ub = __builtin_bit_cast(u32x2, b);
  return __builtin_bit_cast(bf16x8, u32x4{ua[0], ua[1], ub[0], ub[1]});
}

// LDS DMA (global_load_lds_dwordx4: each lane's 16 bytes land at M0 + OFF + 16 * lane) issued
// from inline assembly, so that the compiler neither tracks these loads nor inserts its own
// vmcnt waits for them (it cannot tell ring stages apart and would wait for every load in
// flight before each LDS read).  The kernel orders them itself with wait_vm() + tile_barrier().
// The s_nop covers the one wait state an M0 write needs before an LDS DMA.
template <int OFF>
__device__ __forceinline__ void dma_s(uint32_t lds, const char *sbase, uint32_t voff) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 offset:%3"
               :: "s"(lds), "v"(voff), "s"(sbase), "i"(OFF) : "memory");
}
__device__ __forceinline__ void dma_v(uint32_t lds, const char *src) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(lds), "v"(src) : "memory");
}
// s_waitcnt vmcnt(N) with lgkmcnt and expcnt unconstrained (gfx9 encoding: vmcnt[3:0],
// expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] in bits 15:14)
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
// Workgroup barrier ordering LDS only: unlike __syncthreads it does not wait for the LDS DMA
// loads still in flight for later ring stages.
__device__ __forceinline__ void tile_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace

template <bool CAP>
__global__ __launch_bounds__(256, 1) void attn_bf16_d128_dma_kernel(const AttnArgs a,
                                                                    const AttnPlan plan) {
  constexpr int D = 128, KT = 64, QPW = kQPW_D128;
  constexpr int NQB = QPW / 32, NKB = KT / 32, NDB = D / 32, NS = D / 16, NKS = KT / 16;
  constexpr int ROWB = D * 2;                 // bytes per K or V row
  constexpr int TILEB = KT * ROWB;            // bytes per K or V tile
  constexpr int NSTAGE = 4;                   // LDS ring: tile t in stage t % 4, DMA distance 3
  constexpr int VM_TILE = 8;                  // DMA instructions per wave per tile
  constexpr float kSlack = 8.0f;              // lazy rescale: p <= 2^8 between rescales
  static_assert(NQB == 2 && NKB == 2, "the pipeline below is written for 2 x 2 blocks");
  __shared__ __align__(1024) char smem[NSTAGE * 2 * TILEB];   // [stage][K, V]
  __shared__ __align__(16) int32_t pg[kMaxSplitKeys / kPage + 8];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int j = lane & 31, hh = lane >> 5;
  const int kvh = blockIdx.x % a.n_kv_heads;
  int unit = blockIdx.x / a.n_kv_heads;
  int b = 0;
  while (b + 1 < plan.n_seqs && unit >= plan.seq[b + 1].first_unit) ++b;
  const SeqPlan sp = plan.seq[b];
  unit -= sp.first_unit;
  const int split = unit % sp.n_splits;
  const int tgrp = unit / sp.n_splits;
  const int G = a.group;

  // wave task: query head g of this KV head, queries q0 .. q0 + 63 (two 32-query blocks)
  const int task = tgrp * kWaves + wave;
  const bool active = task < sp.n_tasks;
  const int qb = task / G;
  const int g = task - qb * G;
  const int q0 = qb * QPW;
  const int qhead = kvh * G + g;
  const int last_task = min(tgrp * kWaves + kWaves - 1, sp.n_tasks - 1);
  const int last_q = min((last_task / G + 1) * QPW, sp.len);
  const int wg_keys = (int)sp.n_past + last_q;
  const int k_begin = split * sp.split_keys;
  const int k_end = min(k_begin + sp.split_keys, wg_keys);
  const int qpos0 = (int)sp.n_past + q0;
  const int n_tiles = k_end > k_begin ? (k_end - k_begin + KT - 1) / KT : 0;

  const int pg0 = k_begin >> kPageShift;
  const int n_pg = n_tiles > 0 ? ((k_end - 1) >> kPageShift) - pg0 + 1 : 0;
  for (int i = tid; i < n_pg; i += 256) pg[i] = a.map[pg0 + i];

  bf16x8 qreg[NQB][NS];
  if (active) {
#pragma unroll
    for (int qi = 0; qi < NQB; ++qi) {
      const int qr = min(q0 + 32 * qi + j, sp.len - 1);
      const uint16_t *qrow = a.q + ((int64_t)(sp.q_start + qr) * a.n_q_heads + qhead) * D;
#pragma unroll
      for (int s = 0; s < NS; ++s)
        qreg[qi][s] = *reinterpret_cast<const bf16x8 *>(qrow + 16 * s + 8 * hh);
    }
  }

  f32x16 o[NQB][NDB];
#pragma unroll
  for (int qi = 0; qi < NQB; ++qi)
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[qi][db][v] = 0.f;
  float m_ref[NQB], l[NQB];
#pragma unroll
  for (int qi = 0; qi < NQB; ++qi) {
    m_ref[qi] = -INFINITY;
    l[qi] = 0.f;
  }

  // ---- lane-invariant LDS read offsets
  uint32_t offk[NS];                          // S^T A operand: K row j, chunk 2s + hh
#pragma unroll
  for (int s = 0; s < NS; ++s) offk[s] = j * ROWB + (((2 * s + hh) ^ (j & 15)) * 16);
  uint32_t offv[NDB];                         // PV A operand (transposed reads)
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
  const uint64_t pbytes = (uint64_t)a.n_kv_heads * kPage * ROWB;
  const char *kbytes = reinterpret_cast<const char *>(a.kc) + (uint64_t)kvh * kPage * ROWB;
  const char *vbytes = reinterpret_cast<const char *>(a.vc) + (uint64_t)kvh * kPage * ROWB;
  const uint32_t smem_base = (uint32_t)(uintptr_t)smem;

  // DMA of tile `it` (K and V) into ring stage `st`: this wave's 4 KB quarter of each tile.
  // Full tiles: the wave's page is uniform.  The last, partial tile clamps keys past the split
  // end to the last valid key (finite data; masked scores give them weight 0).
  auto dma_tile = [&](int it, int st) {
    const int kt = k_begin + it * KT;
    const uint32_t kd = smem_base + st * 2 * TILEB + wave * 4096;
    const uint32_t vd = kd + TILEB;
    if (kt + KT <= k_end) {
      const uint32_t page =
          (uint32_t)__builtin_amdgcn_readfirstlane(pg[it * (KT / kPage) + wave]);
      const char *ks = kbytes + page * pbytes;
      const char *vs = vbytes + page * pbytes;
      dma_s<0>(kd, ks, kdo);
      dma_s<1024>(kd, ks, kdo ^ (1 << 6));
      dma_s<2048>(kd, ks, kdo ^ (2 << 6));
      dma_s<3072>(kd, ks, kdo ^ (3 << 6));
      dma_s<0>(vd, vs, vdo);
      dma_s<1024>(vd, vs, vdo);
      dma_s<2048>(vd, vs, vdo);
      dma_s<3072>(vd, vs, vdo);
    } else {
      const int tl = k_end - 1;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * wave + 4 * i + r16;
        const int t = min(kt + row, tl);
        const uint64_t page = (uint32_t)pg[(t >> kPageShift) - pg0];
        const uint32_t tok = (uint32_t)(t & (kPage - 1)) * ROWB;
        dma_v(kd + i * 1024, kbytes + page * pbytes + tok + ((lane & 15) ^ (row & 15)) * 16);
        dma_v(vd + i * 1024, vbytes + page * pbytes + tok + ((lane & 15) ^ (4 * (row & 3))) * 16);
      }
    }
  };

  const float c_scale = CAP ? 1.0f : a.scale_log2;
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  // S^T of query block qi for the K tile at kl: K operands stream from LDS
  auto qk = [&](const char *kl, int qi, f32x16 *sacc) {
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[kb][v] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      bf16x8 kop[NKB];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
        kop[kb] = *reinterpret_cast<const bf16x8 *>(kl + kb * 32 * ROWB + offk[s]);
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kb], qreg[qi][s], sacc[kb], 0, 0, 0);
    }
  };
  // soft-cap, causal / tail mask and running max of query block qi; moves the reference when
  // the tile max exceeds it by more than kSlack and returns the factor for O (1 when unmoved).
  // l is rescaled here; O later, by rescale_o, outside the MFMA/VALU overlap regions.
  auto prepare = [&](int kt, int qi, f32x16 *sacc, bool &moved) -> float {
    if constexpr (CAP) {
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) sacc[kb][v] = a.cap_out * tanh_fast(sacc[kb][v] * a.cap_in);
    }
    const int qpos = qpos0 + 32 * qi;
    if ((kt + KT > k_end) || (kt + KT - 1 > qpos)) {
      const int lim = min(qpos + j, k_end - 1) - kt - 4 * hh;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (32 * kb + 8 * (v >> 2) + (v & 3) > lim) sacc[kb][v] = -INFINITY;
    }
    float mt = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[kb][v]);
    mt = fmaxf(mt, __shfl_xor(mt, 32)) * c_scale;
    moved = __builtin_amdgcn_ballot_w64(mt > m_ref[qi] + kSlack) != 0;
    const float m_new = moved ? fmaxf(m_ref[qi], mt) : m_ref[qi];
    const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_ref[qi] - m_new);
    l[qi] *= alpha;
    m_ref[qi] = m_new;
    return alpha;
  };
  auto rescale_o = [&](int qi, bool moved, float alpha) {
    if (__builtin_expect(moved, 0)) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[qi][db][v] *= alpha;
    }
  };
  // P = 2^(s c - m) as bf16 B operands (16-key steps), row sums from the bf16 values
  auto probs = [&](int qi, const f32x16 *sacc, bf16x8 *pb) {
    const float nm = (m_ref[qi] == -INFINITY) ? 0.f : -m_ref[qi];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int kb = ks >> 1, hf = ks & 1;
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = fast_exp2(fmaf(sacc[kb][8 * hf + 2 * e], c_scale, nm));
        const float p1 = fast_exp2(fmaf(sacc[kb][8 * hf + 2 * e + 1], c_scale, nm));
        w[e] = pack_bf16x2(p0, p1);
        l[qi] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, l[qi], false);
      }
      pb[ks] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    }
  };
  // Keeps P where it is computed: without this the compiler sinks the exponentials past the
  // next branch to their MFMA users, out of the region where they overlap the MFMA pipe.
  auto pin = [&](bf16x8 *pb) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) asm volatile("" ::"v"(pb[ks]));
  };
  // O^T of query block qi += V^T P^T for the V tile at vl (transposed LDS reads)
  auto pv = [&](const char *vl, int qi, const bf16x8 *pb) {
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      bf16x8 vop[NDB];
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const char *p = vl + ks * 16 * ROWB + offv[db];
        vop[db] = tr_read_pair(p, p + 8 * ROWB);
      }
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        o[qi][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[db], pb[ks], o[qi][db], 0, 0, 0);
    }
  };

  // ---- prologue: tiles 0..2 in flight, tile 0 landed and visible.  Q and the page table are
  // waited for here, before any DMA is in flight: otherwise the compiler waits for the Q loads
  // at their first use inside the tile loop, with vmcnt values that count the DMA loads too.
  wait_vm<0>();
  __syncthreads();   // pg[] visible
  for (int i = 0; i < 3 && i < n_tiles; ++i) dma_tile(i, i);
  if (n_tiles >= 3) wait_vm<2 * VM_TILE>();
  else if (n_tiles == 2) wait_vm<VM_TILE>();
  else wait_vm<0>();
  tile_barrier();

  for (int t = 0; t < n_tiles; ++t) {
    const int kt = k_begin + t * KT;
    if (t + 3 < n_tiles) dma_tile(t + 3, (t + 3) & 3);
    if (active) {
      const char *kl = smem + (t & 3) * 2 * TILEB, *vl = kl + TILEB;
      f32x16 s0[NKB], s1[NKB];
      bf16x8 p0[NKS], p1[NKS];
      bool mv0, mv1;
      qk(kl, 0, s0);
      const float al0 = prepare(kt, 0, s0, mv0);
      qk(kl, 1, s1);            // MFMA pipe: S of block 1 ...
      probs(0, s0, p0);         // ... while the VALU turns block 0's scores into P
      pin(p0);
      const float al1 = prepare(kt, 1, s1, mv1);
      rescale_o(0, mv0, al0);
      pv(vl, 0, p0);            // MFMA pipe: O of block 0 ...
      probs(1, s1, p1);         // ... while the VALU computes block 1's P
      pin(p1);
      rescale_o(1, mv1, al1);
      pv(vl, 1, p1);
    }
    // the next iteration reads tile t + 1; tiles t + 2 and t + 3 may stay in flight
    if (t + 3 < n_tiles) wait_vm<2 * VM_TILE>();
    else if (t + 2 < n_tiles) wait_vm<VM_TILE>();
    else wait_vm<0>();
    tile_barrier();
  }

  // ---- epilogue
#pragma unroll
  for (int qi = 0; qi < NQB; ++qi) {
    const float l_tot = l[qi] + __shfl_xor(l[qi], 32);
    const int row = q0 + 32 * qi + j;
    if (!active || row >= sp.len) continue;
    if (sp.n_splits == 1) {
      const float inv = 1.0f / l_tot;
      uint16_t *orow = a.out + ((int64_t)(sp.q_start + row) * a.n_q_heads + qhead) * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const int d0 = 32 * db + 8 * gq + 4 * hh;
          *reinterpret_cast<u32x2 *>(orow + d0) =
              u32x2{pack_bf16x2(o[qi][db][4 * gq + 0] * inv, o[qi][db][4 * gq + 1] * inv),
                    pack_bf16x2(o[qi][db][4 * gq + 2] * inv, o[qi][db][4 * gq + 3] * inv)};
        }
    } else {
      const int64_t prow = ((int64_t)split * sp.len + row) * a.n_q_heads + qhead;
      float *op = a.ws + sp.ws_off + prow * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const int d0 = 32 * db + 8 * gq + 4 * hh;
          *reinterpret_cast<f32x4 *>(op + d0) = f32x4{o[qi][db][4 * gq + 0], o[qi][db][4 * gq + 1],
                                                     o[qi][db][4 * gq + 2], o[qi][db][4 * gq + 3]};
        }
      if (hh == 0)
        *reinterpret_cast<f32x2 *>(a.ws + sp.ml_off + prow * 2) = f32x2{m_ref[qi], l_tot};
    }
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
