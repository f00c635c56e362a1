// Internal launch descriptors of the decode-step and warm-prefix kernels, between the C-ABI
// layer (nexus_api.cpp) and the kernels.  Every descriptor has been validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nexus {

// Decode-step attention: one query per sequence over its own page map.
struct DecodeLaunch {
  const void *q;
  void *out;
  const void *cache_k, *cache_v;
  const int32_t *maps;      // device [n_seqs][map_stride]
  const int32_t *lens;      // device [n_seqs]
  int32_t map_stride, max_len;
  int32_t layer, n_phys_pages, n_kv_heads, n_q_heads, head_dim, n_seqs;
  bool v_transposed;
  bool is_bf16;
  float scale;              // resolved (never 0)
  float softcap;            // 0 = off
  void *workspace;
};

// Pages per key split of a decode launch (fixed by the shape, not by the device lengths).
int decode_split_pages(int32_t n_seqs, int32_t n_kv_heads, int32_t wgs_per_kv_head,
                       int32_t max_len);
size_t decode_workspace_bytes(const DecodeLaunch &p);
hipError_t launch_decode(const DecodeLaunch &p, hipStream_t stream);

// Token-range copy between two page maps of one cache (all layers, K and V); optionally also
// writes the shared map entries of a prefix.
struct KvCopyLaunch {
  void *cache_k, *cache_v;
  const int32_t *src_map, *dst_map;   // device maps
  int64_t t0;                         // first logical token
  int32_t n_tokens;                   // tokens to copy (0: map entries only)
  int32_t n_layers, n_phys_pages, n_kv_heads, head_dim, dtype_bytes;
  bool v_transposed;
  int32_t *share_map;                 // nullptr, or dst map whose pages [0, share_n_full) ...
  int32_t share_n_full;               // ... take the source's physical pages
};
hipError_t launch_kv_copy(const KvCopyLaunch &p, hipStream_t stream);

}  // namespace nexus
