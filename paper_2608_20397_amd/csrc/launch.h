// Internal launch descriptors between the C-ABI layer (nexus_api.cpp) and the kernels.
// Every descriptor has been validated by the caller before a launch function sees it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nexus {

struct SpliceLaunch {
  const void *block_k, *block_v;   // [L][T][H][D]
  void *cache_k, *cache_v;         // [L][NPP][H][16][D]; V transposed: [L][H][D][NPP*16]
  const int32_t *map;
  int64_t offset;
  int32_t n_layers, n_tokens, n_heads, head_dim, n_phys_pages;
  int32_t dtype_bytes;             // 2 (bf16) or 4 (f32)
  bool v_transposed;
  bool v_only = false;             // skip the K rows (they are written elsewhere)
};
hipError_t launch_splice(const SpliceLaunch &p, hipStream_t stream);

// Keys rotated on the way into the pages: splice + re-anchor (angle0 = dst - src, the same
// rotation for every token) or rope-append (per_token: token j rotated to position angle0 + j).
struct RopeSpliceLaunch {
  const void *src_k, *src_v;       // [L][T][H][D]
  void *cache_k, *cache_v;         // as SpliceLaunch
  const int32_t *map;
  int64_t offset;
  int32_t n_layers, n_tokens, n_heads, head_dim, n_phys_pages;
  int32_t dtype_bytes;
  bool v_transposed, interleaved, per_token;
  int64_t angle0;
  double rope_base;
};
hipError_t launch_rope_splice(const RopeSpliceLaunch &p, hipStream_t stream);

struct RephaseLaunch {
  void *k;                 // block [L][T][H][D] (map == nullptr) or paged cache [L][NPP][H][16][D]
  const int32_t *map;      // nullptr: contiguous block rows
  int64_t offset;          // first logical token (paged) or 0
  int32_t n_layers, n_tokens, n_heads, head_dim, n_phys_pages;
  int32_t dtype_bytes;
  bool interleaved;
  int64_t delta;           // dst_pos - src_pos
  double rope_base;
};
hipError_t launch_rephase(const RephaseLaunch &p, hipStream_t stream);

// One suffix (sequence) of an attention launch.
struct AttnSeq {
  int32_t q_start;    // first row of q / out
  int32_t len;        // queries
  int64_t n_past;     // position of the first query
};

struct AttnLaunch {
  const void *q;
  void *out;
  const void *cache_k, *cache_v;
  const int32_t *map;
  int32_t layer, n_layers, n_phys_pages, n_kv_heads, n_q_heads, head_dim;
  bool v_transposed;
  bool is_bf16;
  float scale;        // resolved (never 0)
  float softcap;      // 0 = off
  int32_t n_seqs;
  const AttnSeq *seqs;  // host array
  void *workspace;
  size_t workspace_bytes;
  // Largest workspace the plan may use: the planner then only considers key splits whose
  // partials fit (SIZE_MAX: no limit, the plan of least estimated time).
  size_t ws_cap = SIZE_MAX;
};

// Workspace bytes an attention launch with these sequences needs.
size_t attn_workspace_bytes(const AttnLaunch &p);
hipError_t launch_attention(const AttnLaunch &p, hipStream_t stream);

}  // namespace nexus
