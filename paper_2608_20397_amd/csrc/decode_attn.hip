// Decode-step attention over the paged cache: one new query token per sequence attends to every
// cached token of its own sequence (generation after the first token, over the spliced cache;
// scaled dot-product attention of Sec. III-A, soft-cap and transposed V of Sec. VI-B).
//
// Each sequence has its own page map and a device-resident length, so a decode loop can bump the
// lengths on the device and replay the same launch.  Keys are split into fixed runs of
// `split_pages` pages (flash-decoding); a workgroup handles one (sequence, KV head, query-head
// group of up to 16, split) and a second small kernel merges the splits.  The work is
// HBM-bound: each key and value row is read once per (sequence, KV head), shared by the G query
// heads of the group.
//
// bf16 (MFMA) kernel, per wave and 16-key page:
//   * S^T = K.Q^T on v_mfma_f32_16x16x32_bf16: lane l feeds key row l % 16, features
//     32 s + 8 (l / 16) .. +7 of step s straight from global memory (16 bytes); the query heads
//     of the group are the 16 columns (columns past G are zero).  Lane l then holds the scores
//     of keys 4 (l / 16) .. +3 for query column l % 16;
//   * online softmax in log2 units with a lazily moved reference (rescale only when a page's
//     maximum exceeds the reference by more than 8); P is rounded to bf16 and the row sums add
//     the rounded values;
//   * O^T += V^T.P^T on v_mfma_f32_16x16x16_bf16: the scores are already in the B-operand
//     layout.  A transposed V cache gives the A operand (4 consecutive keys of one feature)
//     directly from global memory; a row-major V page is staged in the wave's own LDS slot and
//     read back with ds_read_b64_tr_b16 (in each 16-lane group, output lane i receives element
//     i % 4 of the 8 bytes that source lane 4e + i / 4 points at).
// The 4 waves of a workgroup take the split's pages round-robin, prefetching the next page into
// registers while computing the current one, and merge their (m, l, O) through LDS at the end.
// Key rows past the sequence end are never used: the last page's loads re-read the last valid
// row (row-major) or are zeroed (transposed V), and their scores are -inf.
#include "attn_common.h"
#include "launch_decode.h"

namespace nexus {

namespace {

typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kDecWaves = 4;
constexpr float kDecSlack = 8.0f;   // log2 units the reference may lag behind the running max
constexpr int kMaxDecSplits = 1024; // splits per sequence at most (bounds the merge's loop)
constexpr int kMaxSplitPages = 2048;  // pages per split at most (page list in LDS)

struct DecodeArgs {
  const void *q;
  void *out;
  const void *kc;         // layer base of the K cache [NPP][Hkv][16][D]
  const void *vc;         // layer base of V: as K, or [Hkv][D][NPP * 16] when transposed
  const int32_t *maps;    // [n_seqs][map_stride]
  const int32_t *lens;    // [n_seqs]
  float *part;            // [n_seqs][Hq][max_splits][D] unnormalised split outputs
  float *part_ml;         // [n_seqs][Hq][max_splits][2] (reference m, row sum l)
  int32_t map_stride, max_len, n_q_heads, n_kv_heads, group, n_qgroups;
  int32_t split_pages, max_splits;
  uint32_t n_cols;        // transposed V: NPP * 16
  float scale_log2;       // scale * log2(e)
  float cap_in;           // scale / softcap
  float cap_out;          // softcap * log2(e)
};

__device__ __forceinline__ float max_x16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_x32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_x16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_x32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sequence length as the kernels read it: clamped to [0, max_len].
__device__ __forceinline__ int seq_len_of(const DecodeArgs &a, int b) {
  return min(max(a.lens[b], 0), a.max_len);
}

// 16-byte chunk c of row r of a staged V page lives at chunk c ^ vswz(r): the 16 rows of one
// transposed read (32 bytes each) and the 4 rows of one staging write cover distinct banks.
template <int D>
__device__ __forceinline__ int vswz(int r) {
  return D == 64 ? 2 * ((r >> 1) & 3) : 2 * (r & 7);
}

template <int D, bool VT, bool CAP>
__global__ __launch_bounds__(256) void decode_bf16_kernel(DecodeArgs a) {
  constexpr int NB = D == 256 ? 2 : 3;  // pages per wave in registers (1 computed, NB - 1 loading)
  constexpr int KS = D / 32;          // S^T MFMA steps
  constexpr int DT = D / 16;          // O^T tiles
  constexpr int ROWB = 2 * D;         // bytes per key row
  constexpr int VL = VT ? 1 : D / 32; // 16-byte V loads per lane per row-major page
  constexpr int MO_LD = D + 4;        // padded row of the merge buffer (floats)
  constexpr int STAGE_BYTES = kDecWaves * 16 * ROWB;
  constexpr int MERGE_BYTES = 2 * 16 * MO_LD * 4 + 2 * 2 * 16 * 4;
  constexpr int SMEM = STAGE_BYTES > MERGE_BYTES ? STAGE_BYTES : MERGE_BYTES;
  __shared__ __align__(16) char smem[SMEM];
  __shared__ int32_t pgs[kMaxSplitPages];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qn = lane & 15, grp = lane >> 4;
  const int b = blockIdx.z;
  const int qg = blockIdx.y % a.n_qgroups;
  const int h = blockIdx.y / a.n_qgroups;
  const int split = blockIdx.x;
  const int g_lo = qg * 16;
  const int g_cnt = min(16, a.group - g_lo);     // query heads of this workgroup
  const int hq0 = h * a.group + g_lo;            // first of them
  uint16_t *out = reinterpret_cast<uint16_t *>(a.out);

  const int len = seq_len_of(a, b);
  if (len == 0) {
    if (split == 0)
      for (int i = tid; i < g_cnt * D; i += 256)
        out[((size_t)b * a.n_q_heads + hq0) * D + i] = 0;
    return;
  }
  const int n_pages = (len + 15) >> 4;
  const int p_begin = split * a.split_pages;
  if (p_begin >= n_pages) return;
  const int p_end = min(p_begin + a.split_pages, n_pages);
  const int n_splits = (n_pages + a.split_pages - 1) / a.split_pages;

  // ---- queries: B operand of S^T = K.Q^T, column qn = query head hq0 + qn
  const bool q_ok = qn < g_cnt;
  u32x4 qreg[KS];
  {
    const uint16_t *qrow =
        reinterpret_cast<const uint16_t *>(a.q) + ((size_t)b * a.n_q_heads + hq0 + qn) * D;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qreg[s] = q_ok ? *reinterpret_cast<const u32x4 *>(qrow + 32 * s + 8 * grp)
                     : u32x4{0u, 0u, 0u, 0u};
  }

  // the split's physical pages, staged in LDS once
  const int n_sp = p_end - p_begin;
  {
    const int32_t *map = a.maps + (size_t)b * a.map_stride + p_begin;
    for (int i = tid; i < n_sp; i += 256) pgs[i] = map[i];
  }
  __syncthreads();
  const uint32_t page_elems = (uint32_t)a.n_kv_heads * 16u * D;
  const char *kbase = reinterpret_cast<const char *>(a.kc) + (size_t)h * 16 * ROWB;
  const char *vbase = VT ? reinterpret_cast<const char *>(a.vc) + (size_t)h * D * a.n_cols * 2
                         : reinterpret_cast<const char *>(a.vc) + (size_t)h * 16 * ROWB;
  char *vstage = smem + wave * 16 * ROWB;

  struct Page {
    u32x4 k[KS];
    u32x4 v[VT ? 1 : VL];
    u32x2 vt[VT ? DT : 1];
  };

  // p: logical page (keys 16 p ..), phys: its physical page.  Loads only; the last page's
  // masking happens in compute_page, so that no load result is needed here.
  auto load_page = [&](int p, uint32_t phys, Page &pg) {
    const int nvalid = min(16, len - 16 * p);
    const char *kp = kbase + (size_t)phys * page_elems * 2;
    const int krow = min(qn, nvalid - 1);
#pragma unroll
    for (int s = 0; s < KS; ++s)
      pg.k[s] = *reinterpret_cast<const u32x4 *>(kp + krow * ROWB + 64 * s + 16 * grp);
    if constexpr (!VT) {
      const char *vp = vbase + (size_t)phys * page_elems * 2;
#pragma unroll
      for (int j = 0; j < VL; ++j) {
        const int byte = 16 * lane + 1024 * j;
        const int row = min(byte / ROWB, nvalid - 1);
        pg.v[j] = *reinterpret_cast<const u32x4 *>(vp + row * ROWB + byte % ROWB);
      }
    } else {
      const char *vp = vbase + ((size_t)phys * 16 + 4 * grp) * 2;
#pragma unroll
      for (int t = 0; t < DT; ++t)
        pg.vt[t] = *reinterpret_cast<const u32x2 *>(vp + (size_t)(16 * t + qn) * a.n_cols * 2);
    }
  };

  f32x4 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_ref = -INFINITY;   // reference of query column qn (equal across the 4 lane groups)
  float lsum = 0.f;          // sum of this lane's rounded probabilities

  auto compute_page = [&](int p, const Page &pg) {
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KS; ++st)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, pg.k[st]),
                                                  __builtin_bit_cast(bf16x8, qreg[st]), s, 0, 0,
                                                  0);
    const int key0 = 16 * p + 4 * grp;
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float v = CAP ? a.cap_out * tanh_fast(s[i] * a.cap_in) : s[i] * a.scale_log2;
      x[i] = key0 + i < len ? v : -INFINITY;
    }
    float mx = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
    mx = max_x32(max_x16(mx));
    const bool need = mx > m_ref + kDecSlack;
    if (__builtin_amdgcn_ballot_w64(need)) {
      const float nm = need ? mx : m_ref;
      const float alpha = fast_exp2(m_ref - nm);
#pragma unroll
      for (int t = 0; t < DT; ++t) o[t] *= alpha;
      lsum *= alpha;
      m_ref = nm;
    }
    const uint32_t p01 = pack_bf16x2(fast_exp2(x[0] - m_ref), fast_exp2(x[1] - m_ref));
    const uint32_t p23 = pack_bf16x2(fast_exp2(x[2] - m_ref), fast_exp2(x[3] - m_ref));
    lsum += (__uint_as_float(p01 << 16) + __uint_as_float(p01 & 0xFFFF0000u)) +
            (__uint_as_float(p23 << 16) + __uint_as_float(p23 & 0xFFFF0000u));
    const s16x4 pb = __builtin_bit_cast(s16x4, u32x2{p01, p23});
    if constexpr (!VT) {
#pragma unroll
      for (int j = 0; j < VL; ++j) {
        const int byte = 16 * lane + 1024 * j;
        const int row = byte / ROWB, c = (byte % ROWB) >> 4;
        *reinterpret_cast<u32x4 *>(vstage + row * ROWB + 16 * (c ^ vswz<D>(row))) = pg.v[j];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int r = 4 * grp + (qn >> 2);
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const int c = 2 * t + ((qn & 3) >> 1);
        const char *src = vstage + r * ROWB + 16 * (c ^ vswz<D>(r)) + 8 * (qn & 1);
        const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)src);
        o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pb, o[t], 0, 0, 0);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    } else {
      // slots past the sequence end may hold anything: zero this lane's keys beyond it
      const int keep = len - key0;
      const uint32_t m0 = keep >= 2 ? 0xFFFFFFFFu : keep == 1 ? 0x0000FFFFu : 0u;
      const uint32_t m1 = keep >= 4 ? 0xFFFFFFFFu : keep == 3 ? 0x0000FFFFu : 0u;
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const u32x2 w = u32x2{pg.vt[t][0] & m0, pg.vt[t][1] & m1};
        o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, w), pb, o[t],
                                                         0, 0, 0);
      }
    }
  };

  // ---- this wave's pages p_begin + wave + 4 k, k = 0 .. n_mine - 1: a ring of NB register
  // buffers keeps NB - 1 pages in flight while one is computed.  Every step issues exactly one
  // page of loads (past the end it re-reads the wave's last page, unused), so the wait before
  // each computation leaves the younger pages in flight.
  {
    const int first = wave;
    const int n_mine = first < n_sp ? (n_sp - first + kDecWaves - 1) / kDecWaves : 0;
    if (n_mine > 0) {
      Page buf[NB];
      auto issue = [&](int k, Page &pg) {
        const int lp = first + kDecWaves * min(k, n_mine - 1);   // page within the split
        const uint32_t phys = (uint32_t)__builtin_amdgcn_readfirstlane(pgs[lp]);
        load_page(p_begin + lp, phys, pg);
      };
#pragma unroll
      for (int i = 0; i < NB - 1; ++i) issue(i, buf[i]);
      bool more = true;
      for (int k0 = 0; more; k0 += NB) {
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int k = k0 + j;
          if (k >= n_mine) {
            more = false;
            break;
          }
          issue(k + NB - 1, buf[(j + NB - 1) % NB]);
          compute_page(p_begin + first + kDecWaves * k, buf[j]);
        }
      }
    }
  }

  // ---- merge the 4 waves' (m, l, O^T) in registers, pairwise through LDS: waves 2 and 3 into
  // waves 0 and 1, then wave 1 into wave 0, which writes the result
  lsum = sum_x32(sum_x16(lsum));
  float *mo = reinterpret_cast<float *>(smem);   // [2 slots][16 columns][MO_LD]
  float *mml = mo + 2 * 16 * MO_LD;              // [2 slots][16 columns][m, l]
  auto store_state = [&](int slot) {
#pragma unroll
    for (int t = 0; t < DT; ++t)
      *reinterpret_cast<f32x4 *>(mo + (slot * 16 + qn) * MO_LD + 16 * t + 4 * grp) = o[t];
    if (grp == 0) {
      mml[2 * (slot * 16 + qn)] = m_ref;
      mml[2 * (slot * 16 + qn) + 1] = lsum;
    }
  };
  auto merge_state = [&](int slot) {
    const float mb = mml[2 * (slot * 16 + qn)];
    const float lb = mml[2 * (slot * 16 + qn) + 1];
    const float M = fmaxf(m_ref, mb);
    // a wave that saw no page has m = -inf and contributes nothing
    const float wa = m_ref > -INFINITY ? fast_exp2(m_ref - M) : 0.f;
    const float wb = mb > -INFINITY ? fast_exp2(mb - M) : 0.f;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const f32x4 ob =
          *reinterpret_cast<const f32x4 *>(mo + (slot * 16 + qn) * MO_LD + 16 * t + 4 * grp);
      o[t] = o[t] * wa + ob * wb;
    }
    lsum = lsum * wa + lb * wb;
    m_ref = M;
  };
  __syncthreads();   // the V staging slots are reused
  if (wave >= 2) store_state(wave - 2);
  __syncthreads();
  if (wave < 2) merge_state(wave);
  __syncthreads();
  if (wave == 1) store_state(0);
  __syncthreads();
  if (wave != 0) return;
  merge_state(0);
  if (!q_ok) return;
  const size_t row = (size_t)b * a.n_q_heads + hq0 + qn;
  if (n_splits == 1) {
    const float inv = 1.0f / lsum;
#pragma unroll
    for (int t = 0; t < DT; ++t)
      *reinterpret_cast<u32x2 *>(out + row * D + 16 * t + 4 * grp) =
          u32x2{pack_bf16x2(o[t][0] * inv, o[t][1] * inv),
                pack_bf16x2(o[t][2] * inv, o[t][3] * inv)};
  } else {
    const size_t slot = row * a.max_splits + split;
#pragma unroll
    for (int t = 0; t < DT; ++t)
      *reinterpret_cast<f32x4 *>(a.part + slot * D + 16 * t + 4 * grp) = o[t];
    if (grp == 0) {
      a.part_ml[2 * slot] = m_ref;
      a.part_ml[2 * slot + 1] = lsum;
    }
  }
}

// fp32 caches: one wave per (sequence, query head, split), VALU dot products.  Lane l holds key
// l % 16 of a page and a quarter of its features; the quarters are summed across lanes.
template <bool VT, bool CAP>
__global__ __launch_bounds__(64) void decode_f32_kernel(DecodeArgs a, int D) {
  const int lane = threadIdx.x;
  const int kq = lane & 15, quarter = lane >> 4;
  const int b = blockIdx.z, hq = blockIdx.y, split = blockIdx.x;
  const int h = hq / a.group;
  float *out = reinterpret_cast<float *>(a.out);
  const int len = seq_len_of(a, b);
  const size_t row = (size_t)b * a.n_q_heads + hq;
  if (len == 0) {
    if (split == 0)
      for (int d = lane; d < D; d += 64) out[row * D + d] = 0.f;
    return;
  }
  const int n_pages = (len + 15) >> 4;
  const int p_begin = split * a.split_pages;
  if (p_begin >= n_pages) return;
  const int p_end = min(p_begin + a.split_pages, n_pages);
  const int n_splits = (n_pages + a.split_pages - 1) / a.split_pages;
  const float *q = reinterpret_cast<const float *>(a.q) + row * D;
  const float *kc = reinterpret_cast<const float *>(a.kc);
  const float *vc = reinterpret_cast<const float *>(a.vc);
  const int32_t *map = a.maps + (size_t)b * a.map_stride;
  const int qd = D / 4;                       // features per quarter
  const int dpl = (D + 63) / 64;              // output features per lane (<= 4)
  float o[4] = {0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  for (int p = p_begin; p < p_end; ++p) {
    const uint32_t phys = (uint32_t)map[p];
    const int nvalid = min(16, len - 16 * p);
    const float *kr = kc + (((size_t)phys * a.n_kv_heads + h) * 16 + min(kq, nvalid - 1)) * D;
    float s = 0.f;
    for (int e = 0; e < qd; ++e) s = fmaf(q[quarter * qd + e], kr[quarter * qd + e], s);
    s = sum_x32(sum_x16(s));
    float x = CAP ? a.cap_out * tanh_fast(s * a.cap_in) : s * a.scale_log2;
    if (kq >= nvalid) x = -INFINITY;
    float mx = x;
    for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    const float nm = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - nm);
    m_run = nm;
    const float pk = fast_exp2(x - nm);        // lanes 0..15 hold the page's 16 probabilities
    float ps = pk;
    for (int off = 1; off < 16; off <<= 1) ps += __shfl_xor(ps, off);
    l_run = l_run * alpha + ps;
    for (int j = 0; j < dpl; ++j) o[j] *= alpha;
    for (int k = 0; k < nvalid; ++k) {
      const float pkk = __shfl(pk, k);
      for (int j = 0; j < dpl; ++j) {
        const int d = lane + 64 * j;
        if (d >= D) break;
        const float v = VT ? vc[((size_t)h * D + d) * a.n_cols + phys * 16 + k]
                           : vc[(((size_t)phys * a.n_kv_heads + h) * 16 + k) * D + d];
        o[j] = fmaf(pkk, v, o[j]);
      }
    }
  }
  const size_t slot = row * a.max_splits + split;
  for (int j = 0; j < dpl; ++j) {
    const int d = lane + 64 * j;
    if (d >= D) break;
    if (n_splits == 1) out[row * D + d] = o[j] / l_run;
    else a.part[slot * D + d] = o[j];
  }
  if (n_splits > 1 && lane == 0) {
    a.part_ml[2 * slot] = m_run;
    a.part_ml[2 * slot + 1] = l_run;
  }
}

// Merge of the splits of every (sequence, query head) that has more than one: one wave per
// (sequence, query head), lane l owning features l, l + 64, ...  The first kPre splits' outputs
// are loaded together with the (m, l) pairs, so that the round trips to memory overlap; the
// maximum and the weighted row sum are wave reductions and split s's weight is read from the
// lane that formed it.
template <bool BF16>
__global__ __launch_bounds__(64) void decode_combine_kernel(DecodeArgs a, int D) {
  constexpr int kPre = 16;          // splits whose outputs are loaded up front
  const int lane = threadIdx.x;
  const int hq = blockIdx.x, b = blockIdx.y;
  const int len = seq_len_of(a, b);
  const int n_pages = (len + 15) >> 4;
  const int ns = (n_pages + a.split_pages - 1) / a.split_pages;
  if (ns <= 1) return;
  const size_t row = (size_t)b * a.n_q_heads + hq;
  const float *ml = a.part_ml + 2 * row * a.max_splits;
  const float *po = a.part + row * a.max_splits * D;
  const int dpl = D > 64 ? D / 64 : 1;          // features per lane: 1, 2 or 4
  const bool dok = lane < D;
  float pre[kPre][4];
#pragma unroll
  for (int i = 0; i < kPre; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      pre[i][j] = (i < ns && j < dpl && dok) ? po[(size_t)i * D + lane + 64 * j] : 0.f;
  float m = -INFINITY;
  for (int s = lane; s < ns; s += 64) m = fmaxf(m, ml[2 * s]);
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  const float M = m;
  float lsum = 0.f;
  for (int s = lane; s < ns; s += 64) lsum += ml[2 * s + 1] * fast_exp2(ml[2 * s] - M);
  for (int off = 32; off > 0; off >>= 1) lsum += __shfl_xor(lsum, off);
  float o[4] = {0.f, 0.f, 0.f, 0.f};
  // lane k holds the weight of split 64 c + k of the current chunk c of 64 splits
  float wl = lane < ns ? fast_exp2(ml[2 * lane] - M) : 0.f;
  for (int s0 = 0; s0 < ns; s0 += kPre) {
    if (s0 > 0) {
      // the next kPre splits' outputs, all loads in flight together
#pragma unroll
      for (int i = 0; i < kPre; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          pre[i][j] = (s0 + i < ns && j < dpl && dok)
                          ? po[(size_t)(s0 + i) * D + lane + 64 * j] : 0.f;
      if ((s0 & 63) == 0) wl = s0 + lane < ns ? fast_exp2(ml[2 * (s0 + lane)] - M) : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      // splits past ns hold zeros
      const float w =
          __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), (s0 + i) & 63));
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] += pre[i][j] * w;
    }
  }
  if (!dok) return;
  const float inv = 1.0f / lsum;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j < dpl) {
      const float r = o[j] * inv;
      if (BF16) reinterpret_cast<uint16_t *>(a.out)[row * D + lane + 64 * j] =
          (uint16_t)(pack_bf16x2(r, 0.f) & 0xFFFFu);
      else reinterpret_cast<float *>(a.out)[row * D + lane + 64 * j] = r;
    }
  }
}

}  // namespace

int decode_split_pages(int32_t n_seqs, int32_t n_kv_heads, int32_t wgs_per_kv_head,
                       int32_t max_len) {
  // Measured on MI355X (256 CUs, two of these workgroups resident per CU): about 512
  // workgroups over the longest sequence, at least 32 pages (8 per wave) per split so that a
  // workgroup's set-up is amortised, and no partial second round of workgroups: between 256
  // and 512 workgroups, 256 is faster.
  constexpr int64_t kCUs = 256;
  constexpr int64_t kMinSplitPages = 32;
  const int64_t max_pages = ((int64_t)max_len + 15) / 16;
  if (max_pages <= 0) return 1;
  const int64_t pairs = (int64_t)n_seqs * n_kv_heads * wgs_per_kv_head;
  int64_t ns = (2 * kCUs + pairs - 1) / pairs;
  int64_t sp = (max_pages + ns - 1) / ns;
  if (sp < kMinSplitPages) sp = kMinSplitPages;
  ns = (max_pages + sp - 1) / sp;
  if (pairs * ns > kCUs && pairs * ns < 2 * kCUs && pairs <= kCUs) {
    ns = kCUs / pairs;
    sp = (max_pages + ns - 1) / ns;
  }
  // bounds of the page list in LDS and of the merge loop
  if (sp < (max_pages + kMaxDecSplits - 1) / kMaxDecSplits)
    sp = (max_pages + kMaxDecSplits - 1) / kMaxDecSplits;
  if (sp > kMaxSplitPages) sp = kMaxSplitPages;
  if (sp > max_pages) sp = max_pages;
  return (int)sp;
}

namespace {

// Splits of the launch: `sp` pages per split, `max_splits` over the longest sequence.
void decode_geometry(const DecodeLaunch &p, int &sp, int &max_splits) {
  const int group = p.n_q_heads / p.n_kv_heads;
  // bf16: one workgroup per 16 query heads of a group; f32: one wave per query head
  const int per_kv = p.is_bf16 ? (group + 15) / 16 : group;
  sp = decode_split_pages(p.n_seqs, p.n_kv_heads, per_kv, p.max_len);
  const int64_t max_pages = ((int64_t)p.max_len + 15) / 16;
  max_splits = (int)((max_pages + sp - 1) / sp);
  if (max_splits < 1) max_splits = 1;
}

}  // namespace

size_t decode_workspace_bytes(const DecodeLaunch &p) {
  int sp, max_splits;
  decode_geometry(p, sp, max_splits);
  if (max_splits <= 1) return 0;
  return (size_t)p.n_seqs * p.n_q_heads * max_splits * (p.head_dim + 2) * sizeof(float);
}

hipError_t launch_decode(const DecodeLaunch &p, hipStream_t stream) {
  const int group = p.n_q_heads / p.n_kv_heads;
  const int n_qgroups = (group + 15) / 16;
  int sp, max_splits;
  decode_geometry(p, sp, max_splits);
  DecodeArgs a{};
  const size_t esize = p.is_bf16 ? 2 : 4;
  const size_t layer_elems = (size_t)p.n_phys_pages * p.n_kv_heads * 16 * p.head_dim;
  a.q = p.q;
  a.out = p.out;
  a.kc = reinterpret_cast<const char *>(p.cache_k) + (size_t)p.layer * layer_elems * esize;
  a.vc = reinterpret_cast<const char *>(p.cache_v) + (size_t)p.layer * layer_elems * esize;
  a.maps = p.maps;
  a.lens = p.lens;
  float *ws = reinterpret_cast<float *>(p.workspace);
  const size_t part_elems = (size_t)p.n_seqs * p.n_q_heads * max_splits * p.head_dim;
  a.part = max_splits > 1 ? ws : nullptr;
  a.part_ml = max_splits > 1 ? ws + part_elems : nullptr;
  a.map_stride = p.map_stride;
  a.max_len = p.max_len;
  a.n_q_heads = p.n_q_heads;
  a.n_kv_heads = p.n_kv_heads;
  a.group = group;
  a.n_qgroups = n_qgroups;
  a.split_pages = sp;
  a.max_splits = max_splits;
  a.n_cols = (uint32_t)p.n_phys_pages * 16u;
  const float log2e = 1.4426950408889634f;
  a.scale_log2 = p.scale * log2e;
  a.cap_in = p.softcap > 0.f ? p.scale / p.softcap : 0.f;
  a.cap_out = p.softcap * log2e;
  const bool cap = p.softcap > 0.f;
  if (p.is_bf16) {
    const dim3 grid(max_splits, p.n_kv_heads * n_qgroups, p.n_seqs);
#define NEXUS_DEC(D_, VT_, CAP_) \
  hipLaunchKernelGGL((decode_bf16_kernel<D_, VT_, CAP_>), grid, dim3(256), 0, stream, a)
#define NEXUS_DEC_D(D_)                                             \
  do {                                                              \
    if (p.v_transposed) {                                           \
      if (cap) NEXUS_DEC(D_, true, true); else NEXUS_DEC(D_, true, false);   \
    } else {                                                        \
      if (cap) NEXUS_DEC(D_, false, true); else NEXUS_DEC(D_, false, false); \
    }                                                               \
  } while (0)
    if (p.head_dim == 64) NEXUS_DEC_D(64);
    else if (p.head_dim == 128) NEXUS_DEC_D(128);
    else NEXUS_DEC_D(256);
#undef NEXUS_DEC_D
#undef NEXUS_DEC
  } else {
    const dim3 grid(max_splits, p.n_q_heads, p.n_seqs);
    if (p.v_transposed) {
      if (cap) hipLaunchKernelGGL((decode_f32_kernel<true, true>), grid, dim3(64), 0, stream, a, p.head_dim);
      else hipLaunchKernelGGL((decode_f32_kernel<true, false>), grid, dim3(64), 0, stream, a, p.head_dim);
    } else {
      if (cap) hipLaunchKernelGGL((decode_f32_kernel<false, true>), grid, dim3(64), 0, stream, a, p.head_dim);
      else hipLaunchKernelGGL((decode_f32_kernel<false, false>), grid, dim3(64), 0, stream, a, p.head_dim);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || max_splits <= 1) return e;
  const dim3 cgrid(p.n_q_heads, p.n_seqs);
  if (p.is_bf16)
    hipLaunchKernelGGL((decode_combine_kernel<true>), cgrid, dim3(64), 0, stream, a, p.head_dim);
  else
    hipLaunchKernelGGL((decode_combine_kernel<false>), cgrid, dim3(64), 0, stream, a, p.head_dim);
  return hipGetLastError();
}

}  // namespace nexus
