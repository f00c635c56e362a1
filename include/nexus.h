/*
 * nexus.h - C ABI of the MI355X (gfx950) KV-block splice path.
 *
 * The path transplants a precompiled KV block (the keys and values of a tool schema, compiled
 * once at a RoPE anchor m0) into a live paged KV cache and repairs the seam, following
 * "Nexus: Depth-Adaptive KV-Cache Splicing" (arXiv 2608.20397):
 *
 *   1. nexus_splice_pages      write the block's K/V rows into the cache at a logical cursor
 *                              (Sec. VI-A; transposed-V caches per Sec. VI-B);
 *   2. nexus_rephase_k[_paged] re-anchor the block's rotary keys from m0 to the splice position,
 *                              the exact inverse of the phase drift of eq. (drift) (Sec. III-B);
 *   3. nexus_suffix_attn       causal grouped-query attention of the re-decoded suffix over the
 *                              spliced cache (Sec. III-A, Sec. III-C, Sec. VI-A), with optional
 *                              tanh logit soft-capping and a transposed V cache (Sec. VI-B);
 *   4. nexus_redecode_len      the redecode length ceil(S * R(n_past) / 100) of eq. (adaptive).
 *
 * Conventions shared by every call:
 *   - Memory: every tensor pointer is a DEVICE pointer unless the argument says "host".  The
 *     caller owns all memory; the library allocates nothing and keeps no state between calls.
 *   - Streams: `stream` is a hipStream_t passed as void* (NULL = the null stream).  A call
 *     validates its arguments on the host, enqueues its kernels on `stream` and returns without
 *     synchronizing.  Calls on one stream run in order; calls on different streams that touch
 *     the same memory race.
 *   - Errors: a status other than NEXUS_OK means nothing was enqueued and nothing was written,
 *     except NEXUS_EHIP (a HIP launch error; earlier kernels of the same call may have run).
 *     Faults inside a kernel surface at the caller's next synchronization.  Page-table entries
 *     live on the device and are not checked by the host: every entry of the logical pages a
 *     call touches must be in [0, n_phys_pages) (nexus_check_page_table checks a host copy).
 *   - Element types: bf16 (IEEE-754 binary32 truncated to its top 16 bits) and f32.
 *   - RoPE: pair i (0 <= i < D/2) of a token at position p is rotated by p * theta_i with
 *     theta_i = base^(-2i/D) (Sec. III-B).  NEOX pairs features (i, i + D/2); INTERLEAVED pairs
 *     (2i, 2i + 1).
 */
#ifndef NEXUS_H
#define NEXUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NEXUS_ABI_VERSION 1

typedef enum nexus_status {
  NEXUS_OK = 0,
  NEXUS_EINVAL = 1,      /* null pointer, non-positive size, unknown enum value              */
  NEXUS_ESHAPE = 2,      /* head counts, head_dim, layer or page size inconsistent/unsupported */
  NEXUS_EDTYPE = 3,      /* element type differs between operands or is unsupported          */
  NEXUS_EROPE = 4,       /* RoPE base / style / anchor differs from the block's header       */
  NEXUS_ERANGE = 5,      /* a token range or position lies outside the cache or is negative  */
  NEXUS_ELAYOUT = 6,     /* V layout argument differs from the cache's layout                */
  NEXUS_EWORKSPACE = 7,  /* workspace missing or smaller than nexus_suffix_attn_workspace()  */
  NEXUS_EHIP = 8         /* a HIP launch failed                                              */
} nexus_status;

typedef enum nexus_dtype { NEXUS_BF16 = 0, NEXUS_F32 = 1 } nexus_dtype;
typedef enum nexus_v_layout { NEXUS_V_ROWMAJOR = 0, NEXUS_V_TRANSPOSED = 1 } nexus_v_layout;
typedef enum nexus_rope_style { NEXUS_ROPE_NEOX = 0, NEXUS_ROPE_INTERLEAVED = 1 } nexus_rope_style;

/*
 * A compiled KV block resident in HBM: the device-side counterpart of the paper's compiled
 * tool block, whose header records the RoPE anchor and parameters (Sec. VI-A).
 *   k, v        [n_layers][n_tokens][n_kv_heads][head_dim], token-major, contiguous.
 *   base_pos    RoPE anchor of the keys currently stored in `k` (m0 when freshly compiled);
 *               nexus_rephase_k updates it.
 *   rope_base   b of theta_i = b^(-2i/D); rope_style as above.
 * head_dim is a power of two, 16..1024 for bf16 and 8..1024 for f32 (rows move as a power-of-two
 * number of 16-byte chunks); anything else is NEXUS_ESHAPE.  Caches take the same head_dim.
 */
typedef struct nexus_block {
  void *k;
  void *v;
  int32_t n_layers, n_tokens, n_kv_heads, head_dim;
  int32_t dtype;        /* nexus_dtype */
  int32_t rope_style;   /* nexus_rope_style */
  int64_t base_pos;
  double rope_base;
} nexus_block;

/*
 * A paged KV cache.  Logical token t lives in physical page map[t / page_size] at slot
 * t % page_size.
 *   k  [n_layers][n_phys_pages][n_kv_heads][page_size][head_dim]
 *   v  ROWMAJOR:   same layout as k
 *      TRANSPOSED: [n_layers][n_kv_heads][head_dim][n_phys_pages * page_size]; token t is
 *                  column map[t / page_size] * page_size + t % page_size (the token-innermost
 *                  V cache of soft-capped models, Sec. VI-B).  With an identity page table
 *                  this is exactly [kv_head][head_dim][seq].
 * page_size must be 16.
 */
typedef struct nexus_kv_cache {
  void *k;
  void *v;
  int32_t n_layers, n_phys_pages, page_size, n_kv_heads, head_dim;
  int32_t dtype;        /* nexus_dtype */
  int32_t v_layout;     /* nexus_v_layout */
  int32_t rope_style;   /* nexus_rope_style */
  double rope_base;
} nexus_kv_cache;

/* Logical -> physical page map, int32 on the device, n_logical_pages entries. */
typedef struct nexus_page_table {
  const int32_t *map;
  int32_t n_logical_pages;
} nexus_page_table;

/*
 * Re-anchor every key of a compiled block, in place (Sec. III-B, eq. drift).
 * Rotates each key pair i of every layer, token and head of block->k by
 * (dst_pos - src_pos) * theta_i; V is never touched.  The angle is formed and reduced modulo
 * 2*pi in fp64 and its cosine and sine taken in fp64 and held as fp32 head + tail pairs; the
 * rotation is evaluated in fp32 with compensated products (within about 2^-23 of the exact
 * rotation) and rounded to nearest-even back into the block.  dst_pos == src_pos enqueues
 * nothing, leaving the keys bit-identical.
 * Checks: src_pos == block->base_pos and rope_base == block->rope_base (else NEXUS_EROPE);
 * positions >= 0 (NEXUS_ERANGE).  On success block->base_pos (a host field) becomes dst_pos.
 */
nexus_status nexus_rephase_k(nexus_block *block, int64_t src_pos, int64_t dst_pos,
                             double rope_base, void *stream);

/*
 * Re-anchor in place the keys of logical tokens [offset, offset + n_tokens) of every layer and
 * KV head of a paged cache: the same rotation as nexus_rephase_k, applied where a block was
 * spliced.  Checks: rope_base == cache->rope_base (NEXUS_EROPE); 0 <= offset and
 * offset + n_tokens <= pt->n_logical_pages * page_size and pt->n_logical_pages <= n_phys_pages
 * (NEXUS_ERANGE); n_tokens > 0 (NEXUS_EINVAL).  dst_pos == src_pos enqueues nothing.
 */
nexus_status nexus_rephase_k_paged(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                   int64_t offset, int32_t n_tokens, int64_t src_pos,
                                   int64_t dst_pos, double rope_base, void *stream);

/*
 * Splice a block into the cache (Sec. VI-A, Fig. atb; transposed V per Sec. VI-B).
 * For every layer l, block token j and KV head h, logical slot offset + j of the cache receives
 * the block's K row (and V row, or V column when the cache is transposed), bit for bit.  No
 * other cache element is written.  Keys are copied as stored: re-anchor them with
 * nexus_rephase_k before, or nexus_rephase_k_paged after.
 * Checks (fail-closed, as the paper validates the block header before any splice): equal
 * n_layers, n_kv_heads, head_dim (NEXUS_ESHAPE) and dtype (NEXUS_EDTYPE); equal rope_base and
 * rope_style (NEXUS_EROPE); 0 <= offset, offset + n_tokens within the mapped logical pages
 * (NEXUS_ERANGE).
 */
nexus_status nexus_splice_pages(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                const nexus_block *block, int64_t offset, void *stream);

/*
 * Splice a block and re-anchor its keys in one pass (Sec. III-B with Sec. VI-A): the cache ends
 * bit-identical to nexus_splice_pages(cache, pt, block, offset) followed by
 * nexus_rephase_k_paged(cache, pt, offset, block->n_tokens, block->base_pos, dst_pos, ...),
 * while the block's keys are read once and each cache element is written once.  The block is
 * not modified (block->base_pos keeps its value).  Checks: those of nexus_splice_pages, plus
 * dst_pos >= 0 (NEXUS_ERANGE) and head_dim <= 256 (NEXUS_ESHAPE).  dst_pos == block->base_pos
 * is a plain splice.
 */
nexus_status nexus_splice_rephase_pages(const nexus_kv_cache *cache, const nexus_page_table *pt,
                                        const nexus_block *block, int64_t offset,
                                        int64_t dst_pos, void *stream);

/*
 * Append freshly computed tokens (the redecode writes of Sec. VI-A): k and v are
 * [cache->n_layers][n_tokens][cache->n_kv_heads][cache->head_dim] device arrays of the cache
 * dtype holding UN-rotated keys and values.  Key token j is rotated to absolute position
 * pos0 + j (RoPE with the cache's base and pairing, Sec. III-B; same arithmetic as
 * nexus_rephase_k) and written, with value token j, into logical slot offset + j of every layer
 * and KV head.  No other cache element is written; k and v are not modified.
 * Checks: k, v non-NULL and n_tokens > 0 (NEXUS_EINVAL); offset >= 0, pos0 >= 0 and
 * offset + n_tokens within the mapped logical pages (NEXUS_ERANGE); head_dim <= 256
 * (NEXUS_ESHAPE).
 */
nexus_status nexus_rope_append(const nexus_kv_cache *cache, const nexus_page_table *pt,
                               const void *k, const void *v, int32_t n_tokens, int64_t offset,
                               int64_t pos0, void *stream);

/*
 * Causal grouped-query attention of the re-decoded suffix (Sec. III-A; the suffix of Sec. VI-A).
 *   q        [n_s][n_q_heads][head_dim] of the cache dtype; query i sits at absolute position
 *            n_past + i and is already rotated.  Keys are read from layer `layer` of the cache
 *            through `pt`; the suffix's own keys must already be in the cache.
 *   n_past   cache tokens before the first suffix query.  Query i attends to keys
 *            0 .. n_past + i (inclusive).
 *   Query head h reads KV head h / (n_q_heads / n_kv_heads).
 *   scale    score scale; 0 selects 1/sqrt(head_dim).
 *   softcap  0 disables; otherwise score s becomes softcap * tanh(s / softcap) after scaling.
 *   v_layout must equal cache->v_layout (NEXUS_ELAYOUT).
 *   out      [n_s][n_q_heads][head_dim] of the cache dtype.
 *   workspace / workspace_bytes: device scratch of at least nexus_suffix_attn_workspace()
 *            bytes (may be NULL when that is 0).  Its contents on entry do not matter.
 * bf16 caches run on MFMA with fp32 accumulation and need head_dim in {64, 128, 256}; f32
 * caches run an fp32 kernel and need head_dim <= 256.
 */
nexus_status nexus_suffix_attn(const void *q, int32_t n_s, int32_t n_q_heads,
                               const nexus_kv_cache *cache, const nexus_page_table *pt,
                               int32_t layer, int64_t n_past, float softcap, int32_t v_layout,
                               float scale, void *out, void *workspace, size_t workspace_bytes,
                               void *stream);

/* Workspace bytes nexus_suffix_attn needs for these arguments (0 if none, SIZE_MAX if the
 * arguments are invalid). */
size_t nexus_suffix_attn_workspace(int32_t n_s, int32_t n_q_heads, const nexus_kv_cache *cache,
                                   int64_t n_past);

/*
 * nexus_suffix_attn for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same computation with no
 * workspace argument.  The split-K partials live in a static device array of
 * NEXUS_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds until the process ends.
 * The call allocates no device memory (its host-side plan uses a few small host buffers).
 *   - Plan: the key split of least estimated time among those whose partials fit the array;
 *     whenever the plan of nexus_suffix_attn fits (its workspace size <= the array), it is that
 *     plan and the output is bit-identical to nexus_suffix_attn's.
 *   - Limit: when no split fits (a suffix too long for the array), NEXUS_EWORKSPACE and nothing
 *     is enqueued.
 *   - Device: the array of the calling thread's current device is used; a non-null `stream`
 *     must belong to that device (else NEXUS_EINVAL).
 *   - Concurrency: every call on one GPU shares that GPU's array, which keeps the last call's
 *     contents (nothing in it needs to start at zero).  Calls that overlap on one GPU (other
 *     streams, other host threads) race on it: serialize them, e.g. on one stream.
 * Other arguments, layouts and errors as nexus_suffix_attn.
 */
#define NEXUS_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
nexus_status nexus_suffix_attn_noalloc(const void *q, int32_t n_s, int32_t n_q_heads,
                                       const nexus_kv_cache *cache, const nexus_page_table *pt,
                                       int32_t layer, int64_t n_past, float softcap,
                                       int32_t v_layout, float scale, void *out, void *stream);

/*
 * Several suffixes over one cache in one launch (many blocks spliced into one context, each
 * re-decoding its own tail).  Sequence b has seq_len[b] queries, rows q_start[b] ..
 * q_start[b] + seq_len[b] - 1 of q and out, at positions seq_n_past[b] + i.  seq_* are HOST
 * arrays of n_seqs entries (n_seqs <= 32); other arguments as nexus_suffix_attn.
 */
nexus_status nexus_suffix_attn_varlen(const void *q, int32_t n_seqs, const int32_t *q_start,
                                      const int32_t *seq_len, const int64_t *seq_n_past,
                                      int32_t n_q_heads, const nexus_kv_cache *cache,
                                      const nexus_page_table *pt, int32_t layer, float softcap,
                                      int32_t v_layout, float scale, void *out, void *workspace,
                                      size_t workspace_bytes, void *stream);

size_t nexus_suffix_attn_varlen_workspace(int32_t n_seqs, const int32_t *q_start,
                                          const int32_t *seq_len, const int64_t *seq_n_past,
                                          int32_t n_q_heads, const nexus_kv_cache *cache);

/*
 * Decode-step attention: one new query token per sequence over the paged cache (the token-by-
 * token generation that follows the spliced prefill; scaled dot-product attention of Sec. III-A,
 * soft-cap and transposed V per Sec. VI-B).  Each sequence has its own page map, and sequences
 * may share physical pages (a warm prefix).
 *   q           [n_seqs][n_q_heads][head_dim] of the cache dtype, already rotated; the query of
 *               sequence b sits at position seq_len[b] - 1 and its own key and value must
 *               already be in the cache (nexus_rope_append).
 *   maps        DEVICE int32 [n_seqs][map_stride]: logical page p of sequence b is physical page
 *               maps[b * map_stride + p].  Entries of pages below ceil(seq_len[b] / 16) must be
 *               in [0, n_phys_pages); they are not checked.
 *   seq_len     DEVICE int32 [n_seqs]: cached tokens of each sequence (the query attends to all
 *               of them).  Values are clamped to [0, max_seq_len]; a sequence of length 0 gets a
 *               zero output row.  Living on the device, the lengths can advance between replays
 *               of one captured launch.
 *   max_seq_len host upper bound of seq_len, 0 <= max_seq_len <= 16 * map_stride (NEXUS_ERANGE).
 *               It fixes the launch shape: keys are cut into splits of a fixed number of pages
 *               chosen from n_seqs, the head counts and max_seq_len, merged by a second kernel.
 *   layer, softcap, v_layout, scale: as nexus_suffix_attn (same checks, same head_dim limits).
 *   out         [n_seqs][n_q_heads][head_dim] of the cache dtype.
 *   workspace   at least nexus_decode_attn_workspace() bytes (NULL allowed when that is 0);
 *               contents on entry do not matter.
 * bf16 caches: each workgroup reads a KV head's keys and values once for up to 16 query heads
 * (MFMA, fp32 accumulation, probabilities rounded to bf16 as in nexus_suffix_attn).  f32 caches:
 * fp32 VALU kernel.
 */
nexus_status nexus_decode_attn(const void *q, int32_t n_seqs, int32_t n_q_heads,
                               const nexus_kv_cache *cache, const int32_t *maps,
                               int32_t map_stride, const int32_t *seq_len, int32_t max_seq_len,
                               int32_t layer, float softcap, int32_t v_layout, float scale,
                               void *out, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes nexus_decode_attn needs (0 if none, SIZE_MAX if the arguments are invalid). */
size_t nexus_decode_attn_workspace(int32_t n_seqs, int32_t n_q_heads, const nexus_kv_cache *cache,
                                   int32_t max_seq_len);

/*
 * Warm-prefix reuse on the paged cache (the exact-token prefix arena of Sec. VI-D, whose copy
 * within a pre-reserved arena becomes page-table work here).  Both calls take two DEVICE int32
 * page maps of one cache (n_map_pages entries each, logical page -> physical page) and move
 * every layer and KV head.  Entries of the pages a call touches must be in [0, n_phys_pages);
 * they are not checked.
 *
 * nexus_kv_copy_tokens: logical tokens [t0, t0 + n_tokens) of the destination receive the K
 * and V bits of the same logical tokens of the source; nothing else is written.  A logical page
 * that both maps send to the same physical page is skipped (it is already shared).  Checks:
 * n_tokens > 0 (NEXUS_EINVAL); 0 <= t0, t0 + n_tokens <= 16 * n_map_pages (NEXUS_ERANGE).
 *
 * nexus_kv_share_prefix: the first n_tokens tokens of the source become those of the
 * destination.  Whole pages are shared by reference: dst_map[p] = src_map[p] for
 * p < n_tokens / 16, written on the device.  The partial last page, if any, keeps the
 * destination's own physical page (dst_map[n_tokens / 16], which must differ from the
 * source's so that the destination can append after the prefix) and receives a copy of its
 * n_tokens % 16 slots.  One kernel launch; nothing is enqueued when n_tokens == 0.  The caller
 * owns page lifetimes (a shared page must outlive every map that names it).  Checks:
 * 0 <= n_tokens <= 16 * n_map_pages (NEXUS_ERANGE).
 */
nexus_status nexus_kv_copy_tokens(const nexus_kv_cache *cache, const int32_t *src_map,
                                  const int32_t *dst_map, int32_t n_map_pages, int64_t t0,
                                  int32_t n_tokens, void *stream);
nexus_status nexus_kv_share_prefix(const nexus_kv_cache *cache, const int32_t *src_map,
                                   int32_t *dst_map, int32_t n_map_pages, int32_t n_tokens,
                                   void *stream);

/*
 * Exact-token longest-common-prefix lookup over the slots of a warm-prefix arena (Sec. VI-D),
 * host only.  slot_tokens is a HOST [n_slots][slot_stride] array whose slot s holds slot_len[s]
 * tokens.  *slot receives the slot sharing the longest common prefix with tokens[0 .. n_tokens)
 * (the lowest index among equals; -1 when no slot shares a first token) and *match_len its
 * length.  Checks: non-negative sizes and non-NULL arrays where sizes are positive
 * (NEXUS_EINVAL); 0 <= slot_len[s] <= slot_stride (NEXUS_ERANGE).
 */
nexus_status nexus_l0_longest_prefix(const int32_t *tokens, int32_t n_tokens,
                                     const int32_t *slot_tokens, const int32_t *slot_len,
                                     int32_t n_slots, int32_t slot_stride, int32_t *slot,
                                     int32_t *match_len);

/*
 * Semantic Lookaside Buffer (Sec. V-A): tool embeddings INT8-quantised and scanned with integer
 * dot products; the top-two margin gate decides between auto-routing and escalation.
 *
 * nexus_slb_quantize: symmetric per-row INT8 codes of x [n][dim] (fp32, device):
 * scale[r] = max_j |x[r][j]| / 127 and q[r][j] = x[r][j] / scale[r] rounded to nearest-even
 * (IEEE fp32 division), so |q| <= 127; a row of zeros gets scale 0 and zero codes.  For the
 * registry (offline) and for each query embedding.  Checks: non-NULL, n > 0, dim > 0
 * (NEXUS_EINVAL).
 *
 * nexus_slb_scan: for every query q of queries [n_queries][dim] (int8, device, rows 16-byte
 * aligned) against tools [n_tools][dim] (int8, device), the score of tool t is
 * (float(dot(tools[t], queries[q])) * tool_scale[t]) * query_scale[q] in fp32, each product
 * rounded to nearest-even (the integer dot is exact).  Outputs per query, device arrays:
 *   top_idx [n_queries][k], top_score [n_queries][k]: the k best tools, higher score first and
 *     the lower index first among equal scores; index -1 and score -inf past n_tools;
 *   margin [n_queries]: top_score[0] - top_score[1] in fp32 (+inf when n_tools == 1);
 *   route [n_queries]: 1 when margin > tau (auto-route), else 0 (escalate to the reranker).
 *   The paper calibrates tau = 0.0136 (the 20th percentile of adversarial-pair margins).
 * workspace: nexus_slb_scan_workspace() bytes (NULL allowed when 0).  Checks: non-NULL arrays,
 * n_tools > 0, n_queries > 0, 1 <= k <= 8, finite tau (NEXUS_EINVAL); dim a multiple of 64 in
 * [64, 1024] (NEXUS_ESHAPE).  Up to 16 queries share one pass over the tool rows; larger batches
 * go in blocks of 64 queries on int8 MFMA, so a batch costs far less than its queries one by one.
 */
nexus_status nexus_slb_quantize(const float *x, int32_t n, int32_t dim, int8_t *q, float *scale,
                                void *stream);
nexus_status nexus_slb_scan(const int8_t *tools, const float *tool_scale, int32_t n_tools,
                            const int8_t *queries, const float *query_scale, int32_t n_queries,
                            int32_t dim, int32_t k, float tau, int32_t *top_idx,
                            float *top_score, float *margin, int32_t *route, void *workspace,
                            size_t workspace_bytes, void *stream);
/* Workspace bytes nexus_slb_scan needs (0 if none, SIZE_MAX if the arguments are invalid). */
size_t nexus_slb_scan_workspace(int32_t n_tools, int32_t n_queries, int32_t dim, int32_t k);

/*
 * Redecode length of eq. (adaptive): ceil(S * R(n_past) / 100) with R = r_base for n_past <= M
 * and R = r_base + (n_past - M) / (M (K - 1)) * (100 - r_base) above, clamped to 100 (Sec. III-C;
 * the suffix length of Sec. VI-A).  Exact integer arithmetic.  Host only; returns -1 unless
 * S >= 0, n_past >= 0, M > 0, 0 <= r_base_pct <= 100 and K >= 2.
 */
int64_t nexus_redecode_len(int64_t S, int64_t n_past, int32_t M, int32_t r_base_pct, int32_t K);

/* Host check of a host copy of a page map: entries in [0, n_phys_pages) and pairwise distinct.
 * Returns NEXUS_OK, NEXUS_EINVAL (null / bad sizes) or NEXUS_ERANGE. */
nexus_status nexus_check_page_table(const int32_t *host_map, int32_t n_logical_pages,
                                    int32_t n_phys_pages);

/*
 * Measurement helpers, not part of the splice path: the ceilings a kernel on this GPU reaches,
 * against which roofline fractions are also quoted.
 *   nexus_calib_copy       copies `bytes` (a multiple of 16; both pointers 16-byte aligned)
 *                          from src to dst on the device: the read + write HBM ceiling.
 *   nexus_calib_mfma_bf16  runs `iters` rounds of four independent 32x32x16 bf16 MFMAs on every
 *                          wave of 512 workgroups x 4 waves (two waves per SIMD); *flops (host)
 *                          receives the matrix FLOPs enqueued.  `sink` is a device array of 512
 *                          floats that the kernel never writes in practice.
 *   nexus_calib_lds_dma    reads `bytes` (a multiple of 16384; src 16-byte aligned) from src
 *                          into LDS with the LDS DMA loads the attention kernels use and writes
 *                          nothing: the reference against which the memory counters' reading of
 *                          those loads is scaled.
 * Each enqueues one kernel on `stream`; NEXUS_EINVAL on bad arguments.
 */
nexus_status nexus_calib_copy(const void *src, void *dst, size_t bytes, void *stream);
nexus_status nexus_calib_mfma_bf16(int32_t iters, float *sink, double *flops, void *stream);
nexus_status nexus_calib_lds_dma(const void *src, size_t bytes, void *stream);

/* Static text for a status code. */
const char *nexus_status_str(int32_t status);

/* NEXUS_ABI_VERSION of the built library. */
int32_t nexus_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* NEXUS_H */
