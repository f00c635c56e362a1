// Internal launch descriptors of the SLB (Semantic Lookaside Buffer) kernels, between the C-ABI
// layer (nexus_api.cpp) and the kernels.  Every descriptor has been validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace nexus {

struct SlbLaunch {
  const int8_t *tools;        // [n_tools][dim]
  const float *tool_scale;    // [n_tools]
  const int8_t *queries;      // [n_queries][dim]
  const float *query_scale;   // [n_queries]
  int32_t n_tools, n_queries, dim, k;
  float tau;
  int32_t *top_idx;           // [n_queries][k]
  float *top_score;           // [n_queries][k]
  float *margin;              // [n_queries]
  int32_t *route;             // [n_queries]
  void *workspace;
};

// Tool ranges of a scan (one workgroup column each) and the tools per range.
void slb_geometry(int32_t n_tools, int32_t n_queries, int32_t dim, int32_t &n_ranges,
                  int32_t &range_tools);
size_t slb_workspace_bytes(int32_t n_tools, int32_t n_queries, int32_t dim);
hipError_t launch_slb_scan(const SlbLaunch &p, hipStream_t stream);
hipError_t launch_slb_quantize(const float *x, int32_t n, int32_t dim, int8_t *q, float *scale,
                               hipStream_t stream);

}  // namespace nexus
