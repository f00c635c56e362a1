// C-ABI entry points of libnexus: host-side validation (fail-closed: nothing is enqueued unless
// every check passes) and dispatch to the gfx950 kernels.  Stateless; allocates nothing.
#include "nexus.h"

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <mutex>
#include <vector>

#include "launch.h"
#include "launch_decode.h"
#include "launch_slb.h"

using namespace nexus;

namespace {

constexpr int kPageSize = 16;
constexpr int64_t kMaxElems32 = (int64_t)1 << 31;

int dtype_bytes(int32_t dt) { return dt == NEXUS_BF16 ? 2 : dt == NEXUS_F32 ? 4 : 0; }

bool valid_style(int32_t s) { return s == NEXUS_ROPE_NEOX || s == NEXUS_ROPE_INTERLEAVED; }
bool valid_layout(int32_t v) { return v == NEXUS_V_ROWMAJOR || v == NEXUS_V_TRANSPOSED; }

// rows of 16-byte chunks must tile head_dim, and pairs must tile whole 16-byte chunks
bool head_dim_ok(int32_t head_dim, int esize) {
  if (head_dim <= 0 || head_dim % 2) return false;
  const int per16 = 16 / esize;
  if (head_dim % (2 * per16)) return false;           // rephase: pairs per thread
  const int chunks = head_dim * esize / 16;
  if (chunks & (chunks - 1)) return false;            // splice: power-of-two chunks per row
  return head_dim <= 1024;
}

nexus_status check_block(const nexus_block *b) {
  if (!b || !b->k || !b->v) return NEXUS_EINVAL;
  if (b->n_layers <= 0 || b->n_tokens <= 0 || b->n_kv_heads <= 0 || b->head_dim <= 0)
    return NEXUS_EINVAL;
  const int es = dtype_bytes(b->dtype);
  if (!es) return NEXUS_EDTYPE;
  if (!valid_style(b->rope_style)) return NEXUS_EINVAL;
  if (!head_dim_ok(b->head_dim, es)) return NEXUS_ESHAPE;
  if (b->n_layers > 65535) return NEXUS_ESHAPE;
  if ((int64_t)b->n_tokens * b->n_kv_heads * b->head_dim >= kMaxElems32) return NEXUS_ESHAPE;
  if ((int64_t)b->n_layers * b->n_tokens * b->n_kv_heads >= kMaxElems32) return NEXUS_ESHAPE;
  if (!(b->rope_base > 1.0) || !isfinite(b->rope_base)) return NEXUS_EROPE;
  if (b->base_pos < 0) return NEXUS_ERANGE;
  return NEXUS_OK;
}

nexus_status check_cache(const nexus_kv_cache *c) {
  if (!c || !c->k || !c->v) return NEXUS_EINVAL;
  if (c->n_layers <= 0 || c->n_phys_pages <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0)
    return NEXUS_EINVAL;
  if (c->page_size != kPageSize) return NEXUS_ESHAPE;
  const int es = dtype_bytes(c->dtype);
  if (!es) return NEXUS_EDTYPE;
  if (!valid_layout(c->v_layout) || !valid_style(c->rope_style)) return NEXUS_EINVAL;
  if (!head_dim_ok(c->head_dim, es)) return NEXUS_ESHAPE;
  if (c->n_layers > 65535) return NEXUS_ESHAPE;
  // kernels address one layer of K or V with 32-bit element offsets
  if ((int64_t)c->n_phys_pages * kPageSize * c->n_kv_heads * c->head_dim >= kMaxElems32)
    return NEXUS_ESHAPE;
  if (!(c->rope_base > 1.0) || !isfinite(c->rope_base)) return NEXUS_EROPE;
  return NEXUS_OK;
}

nexus_status check_pt(const nexus_page_table *pt, const nexus_kv_cache *c) {
  if (!pt || !pt->map || pt->n_logical_pages <= 0) return NEXUS_EINVAL;
  if (pt->n_logical_pages > c->n_phys_pages) return NEXUS_ERANGE;
  return NEXUS_OK;
}

nexus_status from_hip(hipError_t e) { return e == hipSuccess ? NEXUS_OK : NEXUS_EHIP; }

hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Shared checks of the two attention entry points; fills `L` on success.
nexus_status prepare_attention(const void *q, int32_t n_q_heads, const nexus_kv_cache *cache,
                               const nexus_page_table *pt, int32_t layer, float softcap,
                               int32_t v_layout, float scale, void *out,
                               const AttnSeq *seqs, int32_t n_seqs, AttnLaunch &L) {
  nexus_status st = check_cache(cache);
  if (st) return st;
  if (!q || !out) return NEXUS_EINVAL;
  st = check_pt(pt, cache);
  if (st) return st;
  if (!valid_layout(v_layout)) return NEXUS_EINVAL;
  if (v_layout != cache->v_layout) return NEXUS_ELAYOUT;
  if (layer < 0 || layer >= cache->n_layers) return NEXUS_ERANGE;
  if (n_q_heads <= 0 || n_q_heads % cache->n_kv_heads) return NEXUS_ESHAPE;
  if (!(softcap >= 0.f) || !isfinite(softcap)) return NEXUS_EINVAL;
  if (!(scale >= 0.f) || !isfinite(scale)) return NEXUS_EINVAL;
  const bool bf16 = cache->dtype == NEXUS_BF16;
  if (bf16) {
    if (cache->head_dim != 64 && cache->head_dim != 128 && cache->head_dim != 256)
      return NEXUS_ESHAPE;
  } else if (cache->head_dim > 256) {
    return NEXUS_ESHAPE;
  }
  if (!seqs || n_seqs < 1 || n_seqs > 32) return NEXUS_EINVAL;
  const int64_t capacity = (int64_t)pt->n_logical_pages * kPageSize;
  int64_t rows = 0;
  for (int32_t b = 0; b < n_seqs; ++b) {
    const AttnSeq &s = seqs[b];
    if (s.len <= 0 || s.q_start < 0) return NEXUS_EINVAL;
    if (s.n_past < 0 || s.n_past + s.len > capacity) return NEXUS_ERANGE;
    rows += s.len;
    if ((int64_t)s.q_start + s.len > kMaxElems32 / 1024) return NEXUS_ERANGE;
  }
  if (rows * n_q_heads * cache->head_dim >= kMaxElems32) return NEXUS_ESHAPE;
  L = AttnLaunch{};
  L.q = q;
  L.out = out;
  L.cache_k = cache->k;
  L.cache_v = cache->v;
  L.map = pt->map;
  L.layer = layer;
  L.n_layers = cache->n_layers;
  L.n_phys_pages = cache->n_phys_pages;
  L.n_kv_heads = cache->n_kv_heads;
  L.n_q_heads = n_q_heads;
  L.head_dim = cache->head_dim;
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;
  L.is_bf16 = bf16;
  L.scale = scale > 0.f ? scale : 1.0f / sqrtf((float)cache->head_dim);
  L.softcap = softcap;
  L.n_seqs = n_seqs;
  L.seqs = seqs;
  return NEXUS_OK;
}

}  // namespace

extern "C" {

int32_t nexus_abi_version(void) { return NEXUS_ABI_VERSION; }

const char *nexus_status_str(int32_t s) {
  switch (s) {
    case NEXUS_OK: return "ok";
    case NEXUS_EINVAL: return "invalid argument (null pointer, bad size or enum)";
    case NEXUS_ESHAPE: return "shape mismatch or unsupported shape";
    case NEXUS_EDTYPE: return "element type mismatch or unsupported type";
    case NEXUS_EROPE: return "RoPE parameters or anchor differ from the block header";
    case NEXUS_ERANGE: return "token range or position outside the cache";
    case NEXUS_ELAYOUT: return "V layout differs from the cache layout";
    case NEXUS_EWORKSPACE: return "workspace missing or too small";
    case NEXUS_EHIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int64_t nexus_redecode_len(int64_t S, int64_t n_past, int32_t M, int32_t r_base_pct, int32_t K) {
  if (S < 0 || n_past < 0 || M <= 0 || r_base_pct < 0 || r_base_pct > 100 || K < 2) return -1;
  if (S > ((int64_t)1 << 40) || n_past > ((int64_t)1 << 40)) return -1;
  // R = r_base for n_past <= M, else r_base + (n_past - M)(100 - r_base) / (M (K - 1)),
  // clamped to 100.  With den = M (K - 1): S R / 100 = S (r_base den + (n_past - M)(100 - r_base))
  // / (100 den), and R >= 100 exactly when (n_past - M)(100 - r_base) >= (100 - r_base) den.
  if (n_past <= M) {
    return (S * r_base_pct + 99) / 100;
  }
  const int64_t den = (int64_t)M * (K - 1);
  const int64_t over = n_past - M;
  if (r_base_pct == 100 || over >= den) return S;   // clamped at 100%
  // 128-bit product to stay exact for large S
  const __int128 num = (__int128)S * ((__int128)r_base_pct * den + (__int128)over * (100 - r_base_pct));
  const __int128 d = (__int128)100 * den;
  const __int128 q = (num + d - 1) / d;
  return (int64_t)(q > S ? S : q);
}

nexus_status nexus_check_page_table(const int32_t *host_map, int32_t n_logical_pages,
                                    int32_t n_phys_pages) {
  if (!host_map || n_logical_pages <= 0 || n_phys_pages <= 0) return NEXUS_EINVAL;
  if (n_logical_pages > n_phys_pages) return NEXUS_ERANGE;
  std::vector<uint8_t> seen((size_t)n_phys_pages, 0);
  for (int32_t i = 0; i < n_logical_pages; ++i) {
    const int32_t p = host_map[i];
    if (p < 0 || p >= n_phys_pages || seen[(size_t)p]) return NEXUS_ERANGE;
    seen[(size_t)p] = 1;
  }
  return NEXUS_OK;
}

nexus_status nexus_rephase_k(nexus_block *block, int64_t src_pos, int64_t dst_pos,
                             double rope_base, void *stream) {
  nexus_status st = check_block(block);
  if (st) return st;
  if (src_pos < 0 || dst_pos < 0) return NEXUS_ERANGE;
  if (src_pos != block->base_pos || rope_base != block->rope_base) return NEXUS_EROPE;
  if (dst_pos == src_pos) return NEXUS_OK;
  RephaseLaunch L{};
  L.k = block->k;
  L.map = nullptr;
  L.offset = 0;
  L.n_layers = block->n_layers;
  L.n_tokens = block->n_tokens;
  L.n_heads = block->n_kv_heads;
  L.head_dim = block->head_dim;
  L.n_phys_pages = 0;
  L.dtype_bytes = dtype_bytes(block->dtype);
  L.interleaved = block->rope_style == NEXUS_ROPE_INTERLEAVED;
  L.delta = dst_pos - src_pos;
  L.rope_base = rope_base;
  st = from_hip(launch_rephase(L, as_stream(stream)));
  if (st == NEXUS_OK) block->base_pos = dst_pos;
  return st;
}

nexus_status nexus_rephase_k_paged(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                   int64_t offset, int32_t n_tokens, int64_t src_pos,
                                   int64_t dst_pos, double rope_base, void *stream) {
  nexus_status st = check_cache(cache);
  if (st) return st;
  st = check_pt(pt, cache);
  if (st) return st;
  if (n_tokens <= 0) return NEXUS_EINVAL;
  if (src_pos < 0 || dst_pos < 0 || offset < 0) return NEXUS_ERANGE;
  if (offset + n_tokens > (int64_t)pt->n_logical_pages * kPageSize) return NEXUS_ERANGE;
  if (rope_base != cache->rope_base) return NEXUS_EROPE;
  if ((int64_t)cache->n_layers * n_tokens * cache->n_kv_heads >= kMaxElems32) return NEXUS_ESHAPE;
  if (dst_pos == src_pos) return NEXUS_OK;
  RephaseLaunch L{};
  L.k = cache->k;
  L.map = pt->map;
  L.offset = offset;
  L.n_layers = cache->n_layers;
  L.n_tokens = n_tokens;
  L.n_heads = cache->n_kv_heads;
  L.head_dim = cache->head_dim;
  L.n_phys_pages = cache->n_phys_pages;
  L.dtype_bytes = dtype_bytes(cache->dtype);
  L.interleaved = cache->rope_style == NEXUS_ROPE_INTERLEAVED;
  L.delta = dst_pos - src_pos;
  L.rope_base = rope_base;
  return from_hip(launch_rephase(L, as_stream(stream)));
}

namespace {

// The fail-closed checks of a splice (the block header against the cache, Sec. VI-A).
nexus_status check_splice(const nexus_kv_cache *cache, const nexus_page_table *pt,
                          const nexus_block *block, int64_t offset) {
  nexus_status st = check_cache(cache);
  if (st) return st;
  st = check_block(block);
  if (st) return st;
  st = check_pt(pt, cache);
  if (st) return st;
  if (block->n_layers != cache->n_layers || block->n_kv_heads != cache->n_kv_heads ||
      block->head_dim != cache->head_dim)
    return NEXUS_ESHAPE;
  if (block->dtype != cache->dtype) return NEXUS_EDTYPE;
  if (block->rope_base != cache->rope_base || block->rope_style != cache->rope_style)
    return NEXUS_EROPE;
  if (offset < 0 || offset + block->n_tokens > (int64_t)pt->n_logical_pages * kPageSize)
    return NEXUS_ERANGE;
  const int es = dtype_bytes(cache->dtype);
  if (cache->v_layout == NEXUS_V_TRANSPOSED && (size_t)64 * (cache->head_dim + 16 / es) * es > 65536)
    return NEXUS_ESHAPE;
  return NEXUS_OK;
}

RopeSpliceLaunch rope_splice_launch(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                    const void *k, const void *v, int32_t n_tokens,
                                    int64_t offset) {
  RopeSpliceLaunch L{};
  L.src_k = k;
  L.src_v = v;
  L.cache_k = cache->k;
  L.cache_v = cache->v;
  L.map = pt->map;
  L.offset = offset;
  L.n_layers = cache->n_layers;
  L.n_tokens = n_tokens;
  L.n_heads = cache->n_kv_heads;
  L.head_dim = cache->head_dim;
  L.n_phys_pages = cache->n_phys_pages;
  L.dtype_bytes = dtype_bytes(cache->dtype);
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;
  L.interleaved = cache->rope_style == NEXUS_ROPE_INTERLEAVED;
  L.rope_base = cache->rope_base;
  return L;
}

}  // namespace

nexus_status nexus_splice_pages(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                const nexus_block *block, int64_t offset, void *stream) {
  const nexus_status st = check_splice(cache, pt, block, offset);
  if (st) return st;
  SpliceLaunch L{};
  L.block_k = block->k;
  L.block_v = block->v;
  L.cache_k = cache->k;
  L.cache_v = cache->v;
  L.map = pt->map;
  L.offset = offset;
  L.n_layers = cache->n_layers;
  L.n_tokens = block->n_tokens;
  L.n_heads = cache->n_kv_heads;
  L.head_dim = cache->head_dim;
  L.n_phys_pages = cache->n_phys_pages;
  L.dtype_bytes = dtype_bytes(cache->dtype);
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;
  return from_hip(launch_splice(L, as_stream(stream)));
}

nexus_status nexus_splice_rephase_pages(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                        const nexus_block *block, int64_t offset,
                                        int64_t dst_pos, void *stream) {
  const nexus_status st = check_splice(cache, pt, block, offset);
  if (st) return st;
  if (dst_pos < 0) return NEXUS_ERANGE;
  if (cache->head_dim > 256) return NEXUS_ESHAPE;
  if (dst_pos == block->base_pos) return nexus_splice_pages(cache, pt, block, offset, stream);
  RopeSpliceLaunch L = rope_splice_launch(cache, pt, block->k, block->v, block->n_tokens, offset);
  L.per_token = false;
  L.angle0 = dst_pos - block->base_pos;
  return from_hip(launch_rope_splice(L, as_stream(stream)));
}

nexus_status nexus_rope_append(const nexus_kv_cache *cache, const nexus_page_table *pt,
                               const void *k, const void *v, int32_t n_tokens, int64_t offset,
                               int64_t pos0, void *stream) {
  nexus_status st = check_cache(cache);
  if (st) return st;
  st = check_pt(pt, cache);
  if (st) return st;
  if (k == nullptr || v == nullptr || n_tokens <= 0) return NEXUS_EINVAL;
  if (offset < 0 || pos0 < 0 || offset + n_tokens > (int64_t)pt->n_logical_pages * kPageSize)
    return NEXUS_ERANGE;
  if (cache->head_dim > 256) return NEXUS_ESHAPE;
  if ((int64_t)n_tokens * cache->n_kv_heads * cache->head_dim >= kMaxElems32 ||
      (int64_t)cache->n_layers * n_tokens * cache->n_kv_heads >= kMaxElems32)
    return NEXUS_ESHAPE;
  const int es = dtype_bytes(cache->dtype);
  if (cache->v_layout == NEXUS_V_TRANSPOSED && (size_t)64 * (cache->head_dim + 16 / es) * es > 65536)
    return NEXUS_ESHAPE;
  RopeSpliceLaunch L = rope_splice_launch(cache, pt, k, v, n_tokens, offset);
  L.per_token = true;
  L.angle0 = pos0;
  return from_hip(launch_rope_splice(L, as_stream(stream)));
}

size_t nexus_suffix_attn_workspace(int32_t n_s, int32_t n_q_heads, const nexus_kv_cache *cache,
                                   int64_t n_past) {
  if (!cache || n_s <= 0 || n_q_heads <= 0 || n_past < 0 || cache->n_kv_heads <= 0 ||
      n_q_heads % cache->n_kv_heads)
    return SIZE_MAX;
  std::vector<AttnSeq> seqs{AttnSeq{0, n_s, n_past}};
  AttnLaunch L{};
  L.n_kv_heads = cache->n_kv_heads;
  L.n_q_heads = n_q_heads;
  L.head_dim = cache->head_dim;
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;   // the kernel (and plan) depend on it
  L.is_bf16 = cache->dtype == NEXUS_BF16;
  L.n_seqs = 1;
  L.seqs = seqs.data();
  return attn_workspace_bytes(L);
}

size_t nexus_suffix_attn_varlen_workspace(int32_t n_seqs, const int32_t *q_start,
                                          const int32_t *seq_len, const int64_t *seq_n_past,
                                          int32_t n_q_heads, const nexus_kv_cache *cache) {
  if (!cache || !q_start || !seq_len || !seq_n_past || n_seqs <= 0 || n_seqs > 32 ||
      n_q_heads <= 0 || cache->n_kv_heads <= 0 || n_q_heads % cache->n_kv_heads)
    return SIZE_MAX;
  std::vector<AttnSeq> seqs;
  for (int32_t b = 0; b < n_seqs; ++b) {
    if (seq_len[b] <= 0 || seq_n_past[b] < 0) return SIZE_MAX;
    seqs.push_back(AttnSeq{q_start[b], seq_len[b], seq_n_past[b]});
  }
  AttnLaunch L{};
  L.n_kv_heads = cache->n_kv_heads;
  L.n_q_heads = n_q_heads;
  L.head_dim = cache->head_dim;
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;
  L.is_bf16 = cache->dtype == NEXUS_BF16;
  L.n_seqs = n_seqs;
  L.seqs = seqs.data();
  return attn_workspace_bytes(L);
}

static nexus_status run_attention(AttnLaunch &L, void *workspace, size_t workspace_bytes,
                                  void *stream) {
  const size_t need = attn_workspace_bytes(L);
  if (need == SIZE_MAX) return NEXUS_EINVAL;
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return NEXUS_EWORKSPACE;
  L.workspace = workspace;
  L.workspace_bytes = workspace_bytes;
  return from_hip(launch_attention(L, as_stream(stream)));
}

nexus_status nexus_suffix_attn(const void *q, int32_t n_s, int32_t n_q_heads,
                               const nexus_kv_cache *cache, const nexus_page_table *pt,
                               int32_t layer, int64_t n_past, float softcap, int32_t v_layout,
                               float scale, void *out, void *workspace, size_t workspace_bytes,
                               void *stream) {
  if (n_s <= 0) return NEXUS_EINVAL;
  const AttnSeq seq{0, n_s, n_past};
  AttnLaunch L;
  nexus_status st = prepare_attention(q, n_q_heads, cache, pt, layer, softcap, v_layout, scale,
                                      out, &seq, 1, L);
  if (st) return st;
  return run_attention(L, workspace, workspace_bytes, stream);
}

}  // extern "C"

// ---- allocation-free suffix attention: the split partials live in a static device array.
// Each GPU the library runs on holds its own copy of `scratch` (NEXUS_NOALLOC_SCRATCH_BYTES)
// until the process ends.  In host code `scratch` names a host-side stand-in, never a device
// address: its device address is taken once per device with hipGetSymbolAddress and kept in
// scratch_ptr[], which is what the kernels receive.
static __device__ __align__(256) float scratch[NEXUS_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once known

// Device address of the current device's `scratch` (taken on the first call on that device,
// with that device current).  A non-null stream must belong to the current device.
nexus_status scratch_of_current_device(void *stream, void **ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return NEXUS_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return NEXUS_EINVAL;
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(as_stream(stream), &sdev) != hipSuccess) return NEXUS_EHIP;
    if (sdev != dev) return NEXUS_EINVAL;
  }
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return NEXUS_EHIP;
    scratch_ptr[dev] = p;
  }
  *ptr = scratch_ptr[dev];
  return NEXUS_OK;
}

}  // namespace

extern "C" {

nexus_status nexus_suffix_attn_noalloc(const void *q, int32_t n_s, int32_t n_q_heads,
                                       const nexus_kv_cache *cache, const nexus_page_table *pt,
                                       int32_t layer, int64_t n_past, float softcap,
                                       int32_t v_layout, float scale, void *out, void *stream) {
  if (n_s <= 0) return NEXUS_EINVAL;
  const AttnSeq seq{0, n_s, n_past};
  AttnLaunch L;
  nexus_status st = prepare_attention(q, n_q_heads, cache, pt, layer, softcap, v_layout, scale,
                                      out, &seq, 1, L);
  if (st) return st;
  // the plan of least estimated time among those whose partials fit the array: the plan of
  // nexus_suffix_attn whenever that one fits
  L.ws_cap = NEXUS_NOALLOC_SCRATCH_BYTES;
  const size_t need = attn_workspace_bytes(L);
  if (need == SIZE_MAX || need > NEXUS_NOALLOC_SCRATCH_BYTES) return NEXUS_EWORKSPACE;
  void *ws = nullptr;
  st = scratch_of_current_device(stream, &ws);
  if (st) return st;
  L.workspace = ws;
  L.workspace_bytes = NEXUS_NOALLOC_SCRATCH_BYTES;
  return from_hip(launch_attention(L, as_stream(stream)));
}

nexus_status nexus_suffix_attn_varlen(const void *q, int32_t n_seqs, const int32_t *q_start,
                                      const int32_t *seq_len, const int64_t *seq_n_past,
                                      int32_t n_q_heads, const nexus_kv_cache *cache,
                                      const nexus_page_table *pt, int32_t layer, float softcap,
                                      int32_t v_layout, float scale, void *out, void *workspace,
                                      size_t workspace_bytes, void *stream) {
  if (!q_start || !seq_len || !seq_n_past || n_seqs <= 0 || n_seqs > 32) return NEXUS_EINVAL;
  std::vector<AttnSeq> seqs;
  for (int32_t b = 0; b < n_seqs; ++b) seqs.push_back(AttnSeq{q_start[b], seq_len[b], seq_n_past[b]});
  AttnLaunch L;
  nexus_status st = prepare_attention(q, n_q_heads, cache, pt, layer, softcap, v_layout, scale,
                                      out, seqs.data(), (int32_t)seqs.size(), L);
  if (st) return st;
  return run_attention(L, workspace, workspace_bytes, stream);
}

namespace {

// Checks of the decode entry point; fills `L` (without the workspace) on success.
nexus_status prepare_decode(const void *q, int32_t n_seqs, int32_t n_q_heads,
                            const nexus_kv_cache *cache, const int32_t *maps, int32_t map_stride,
                            const int32_t *seq_len, int32_t max_seq_len, int32_t layer,
                            float softcap, int32_t v_layout, float scale, void *out,
                            DecodeLaunch &L) {
  nexus_status st = check_cache(cache);
  if (st) return st;
  if (!q || !out || !maps || !seq_len || n_seqs <= 0 || map_stride <= 0) return NEXUS_EINVAL;
  if (!valid_layout(v_layout)) return NEXUS_EINVAL;
  if (v_layout != cache->v_layout) return NEXUS_ELAYOUT;
  if (layer < 0 || layer >= cache->n_layers) return NEXUS_ERANGE;
  if (max_seq_len < 0 || (int64_t)map_stride * kPageSize < max_seq_len) return NEXUS_ERANGE;
  if (n_q_heads <= 0 || n_q_heads % cache->n_kv_heads) return NEXUS_ESHAPE;
  if (!(softcap >= 0.f) || !isfinite(softcap)) return NEXUS_EINVAL;
  if (!(scale >= 0.f) || !isfinite(scale)) return NEXUS_EINVAL;
  const bool bf16 = cache->dtype == NEXUS_BF16;
  if (bf16) {
    if (cache->head_dim != 64 && cache->head_dim != 128 && cache->head_dim != 256)
      return NEXUS_ESHAPE;
  } else if (cache->head_dim > 256) {
    return NEXUS_ESHAPE;
  }
  // grid limits and 32-bit row offsets of q / out / the page maps
  if (n_seqs > 65535 || n_q_heads > 65535) return NEXUS_ESHAPE;
  if ((int64_t)n_seqs * n_q_heads * cache->head_dim >= kMaxElems32) return NEXUS_ESHAPE;
  if ((int64_t)n_seqs * map_stride >= kMaxElems32) return NEXUS_ESHAPE;
  L = DecodeLaunch{};
  L.q = q;
  L.out = out;
  L.cache_k = cache->k;
  L.cache_v = cache->v;
  L.maps = maps;
  L.lens = seq_len;
  L.map_stride = map_stride;
  L.max_len = max_seq_len;
  L.layer = layer;
  L.n_phys_pages = cache->n_phys_pages;
  L.n_kv_heads = cache->n_kv_heads;
  L.n_q_heads = n_q_heads;
  L.head_dim = cache->head_dim;
  L.n_seqs = n_seqs;
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;
  L.is_bf16 = bf16;
  L.scale = scale > 0.f ? scale : 1.0f / sqrtf((float)cache->head_dim);
  L.softcap = softcap;
  return NEXUS_OK;
}

}  // namespace

size_t nexus_decode_attn_workspace(int32_t n_seqs, int32_t n_q_heads, const nexus_kv_cache *cache,
                                   int32_t max_seq_len) {
  if (!cache || n_seqs <= 0 || max_seq_len < 0 || n_q_heads <= 0 || cache->n_kv_heads <= 0 ||
      n_q_heads % cache->n_kv_heads || cache->head_dim <= 0)
    return SIZE_MAX;
  DecodeLaunch L{};
  L.n_seqs = n_seqs;
  L.n_q_heads = n_q_heads;
  L.n_kv_heads = cache->n_kv_heads;
  L.head_dim = cache->head_dim;
  L.max_len = max_seq_len;
  L.is_bf16 = cache->dtype == NEXUS_BF16;
  return decode_workspace_bytes(L);
}

nexus_status nexus_decode_attn(const void *q, int32_t n_seqs, int32_t n_q_heads,
                               const nexus_kv_cache *cache, const int32_t *maps,
                               int32_t map_stride, const int32_t *seq_len, int32_t max_seq_len,
                               int32_t layer, float softcap, int32_t v_layout, float scale,
                               void *out, void *workspace, size_t workspace_bytes,
                               void *stream) {
  DecodeLaunch L;
  nexus_status st = prepare_decode(q, n_seqs, n_q_heads, cache, maps, map_stride, seq_len,
                                   max_seq_len, layer, softcap, v_layout, scale, out, L);
  if (st) return st;
  const size_t need = decode_workspace_bytes(L);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return NEXUS_EWORKSPACE;
  L.workspace = workspace;
  return from_hip(launch_decode(L, as_stream(stream)));
}


namespace {

nexus_status prepare_kv_copy(const nexus_kv_cache *cache, const int32_t *src_map,
                             const int32_t *dst_map, int32_t n_map_pages, KvCopyLaunch &L) {
  nexus_status st = check_cache(cache);
  if (st) return st;
  if (!src_map || !dst_map || n_map_pages <= 0) return NEXUS_EINVAL;
  L = KvCopyLaunch{};
  L.cache_k = cache->k;
  L.cache_v = cache->v;
  L.src_map = src_map;
  L.dst_map = dst_map;
  L.n_layers = cache->n_layers;
  L.n_phys_pages = cache->n_phys_pages;
  L.n_kv_heads = cache->n_kv_heads;
  L.head_dim = cache->head_dim;
  L.dtype_bytes = dtype_bytes(cache->dtype);
  L.v_transposed = cache->v_layout == NEXUS_V_TRANSPOSED;
  return NEXUS_OK;
}

}  // namespace

nexus_status nexus_kv_copy_tokens(const nexus_kv_cache *cache, const int32_t *src_map,
                                  const int32_t *dst_map, int32_t n_map_pages, int64_t t0,
                                  int32_t n_tokens, void *stream) {
  KvCopyLaunch L;
  nexus_status st = prepare_kv_copy(cache, src_map, dst_map, n_map_pages, L);
  if (st) return st;
  if (n_tokens <= 0) return NEXUS_EINVAL;
  if (t0 < 0 || t0 + n_tokens > (int64_t)n_map_pages * kPageSize) return NEXUS_ERANGE;
  L.t0 = t0;
  L.n_tokens = n_tokens;
  return from_hip(launch_kv_copy(L, as_stream(stream)));
}

nexus_status nexus_kv_share_prefix(const nexus_kv_cache *cache, const int32_t *src_map,
                                   int32_t *dst_map, int32_t n_map_pages, int32_t n_tokens,
                                   void *stream) {
  KvCopyLaunch L;
  nexus_status st = prepare_kv_copy(cache, src_map, dst_map, n_map_pages, L);
  if (st) return st;
  if (n_tokens < 0 || n_tokens > (int64_t)n_map_pages * kPageSize) return NEXUS_ERANGE;
  if (n_tokens == 0) return NEXUS_OK;
  const int32_t n_full = n_tokens / kPageSize;
  L.share_map = dst_map;
  L.share_n_full = n_full;
  L.t0 = (int64_t)n_full * kPageSize;
  L.n_tokens = n_tokens - n_full * kPageSize;
  return from_hip(launch_kv_copy(L, as_stream(stream)));
}

nexus_status nexus_l0_longest_prefix(const int32_t *tokens, int32_t n_tokens,
                                     const int32_t *slot_tokens, const int32_t *slot_len,
                                     int32_t n_slots, int32_t slot_stride, int32_t *slot,
                                     int32_t *match_len) {
  if (!slot || !match_len) return NEXUS_EINVAL;
  *slot = -1;
  *match_len = 0;
  if (n_tokens < 0 || n_slots < 0 || slot_stride < 0) return NEXUS_EINVAL;
  if ((n_tokens > 0 && !tokens) || (n_slots > 0 && (!slot_tokens || !slot_len)))
    return NEXUS_EINVAL;
  for (int32_t s = 0; s < n_slots; ++s)
    if (slot_len[s] < 0 || slot_len[s] > slot_stride) return NEXUS_ERANGE;
  int32_t best = 0;
  for (int32_t s = 0; s < n_slots; ++s) {
    const int32_t *st = slot_tokens + (size_t)s * slot_stride;
    const int32_t lim = slot_len[s] < n_tokens ? slot_len[s] : n_tokens;
    if (lim <= best) continue;          // cannot beat the current match
    int32_t m = 0;
    while (m < lim && st[m] == tokens[m]) ++m;
    if (m > best) {
      best = m;
      *slot = s;
    }
  }
  *match_len = best;
  return NEXUS_OK;
}


nexus_status nexus_slb_quantize(const float *x, int32_t n, int32_t dim, int8_t *q, float *scale,
                                void *stream) {
  if (!x || !q || !scale || n <= 0 || dim <= 0) return NEXUS_EINVAL;
  if ((int64_t)n * dim >= kMaxElems32 * 2) return NEXUS_ESHAPE;
  return from_hip(launch_slb_quantize(x, n, dim, q, scale, as_stream(stream)));
}

namespace {

nexus_status check_slb(const void *tools, const float *tool_scale, int32_t n_tools,
                       const void *queries, const float *query_scale, int32_t n_queries,
                       int32_t dim, int32_t k, float tau) {
  if (!tools || !tool_scale || !queries || !query_scale) return NEXUS_EINVAL;
  if (n_tools <= 0 || n_queries <= 0 || k < 1 || k > 8) return NEXUS_EINVAL;
  if (!isfinite(tau)) return NEXUS_EINVAL;
  if (dim <= 0 || dim % 64 || dim > 1024) return NEXUS_ESHAPE;
  if ((int64_t)n_tools * dim >= ((int64_t)1 << 40)) return NEXUS_ESHAPE;
  if (n_queries > 65535 * 64) return NEXUS_ESHAPE;
  return NEXUS_OK;
}

}  // namespace

size_t nexus_slb_scan_workspace(int32_t n_tools, int32_t n_queries, int32_t dim, int32_t k) {
  if (n_tools <= 0 || n_queries <= 0 || k < 1 || k > 8 || dim <= 0 || dim % 64 || dim > 1024)
    return SIZE_MAX;
  return slb_workspace_bytes(n_tools, n_queries, dim);
}

nexus_status nexus_slb_scan(const int8_t *tools, const float *tool_scale, int32_t n_tools,
                            const int8_t *queries, const float *query_scale, int32_t n_queries,
                            int32_t dim, int32_t k, float tau, int32_t *top_idx,
                            float *top_score, float *margin, int32_t *route, void *workspace,
                            size_t workspace_bytes, void *stream) {
  nexus_status st = check_slb(tools, tool_scale, n_tools, queries, query_scale, n_queries, dim,
                              k, tau);
  if (st) return st;
  if (!top_idx || !top_score || !margin || !route) return NEXUS_EINVAL;
  const size_t need = slb_workspace_bytes(n_tools, n_queries, dim);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return NEXUS_EWORKSPACE;
  SlbLaunch L{};
  L.tools = tools;
  L.tool_scale = tool_scale;
  L.queries = queries;
  L.query_scale = query_scale;
  L.n_tools = n_tools;
  L.n_queries = n_queries;
  L.dim = dim;
  L.k = k;
  L.tau = tau;
  L.top_idx = top_idx;
  L.top_score = top_score;
  L.margin = margin;
  L.route = route;
  L.workspace = workspace;
  return from_hip(launch_slb_scan(L, as_stream(stream)));
}


}  // extern "C"
