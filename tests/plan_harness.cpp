// Host-side harness for tests/test_plan_host.py: builds the attention plan of each launch read
// from stdin, with the library's own planner, and prints every unit's work as the kernels and the
// combine see it.  Compiled by the test with hipcc as host code (the kernel source is included
// for its planner; the launch functions it references are stubbed: nothing runs on a GPU).
//
// stdin, one launch per line:  n_q_heads n_kv_heads head_dim v_transposed ws_cap n_seqs
//                              len_0 n_past_0 ... len_{n-1} n_past_{n-1}
//   (ws_cap 0: no cap)
// stdout, per launch:  "plan ok|none units_per_head range_major qpw waves ws_bytes"
//   then per sequence: "seq b q_start len n_past n_tg n_tasks max_splits"
//   then per unit:     "unit u seq tgrp split k_begin split_keys n_splits group_splits"
//   then "end"
#include "attn_bf16.hip"

#include <cstdio>
#include <cstdlib>
#include <vector>

namespace nexus {
hipError_t launch_attention_f32(const AttnLaunch &, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_attn_d128_dma(const AttnArgs &, const AttnPlan &, int, bool, hipStream_t) {
  return hipErrorNotSupported;
}
hipError_t launch_attn_d256_vt(const AttnArgs &, const AttnPlan &, int, bool, hipStream_t) {
  return hipErrorNotSupported;
}
}  // namespace nexus

int main() {
  using namespace nexus;
  int hq, hkv, d, vt, n;
  long long cap;
  while (scanf("%d %d %d %d %lld %d", &hq, &hkv, &d, &vt, &cap, &n) == 6) {
    std::vector<AttnSeq> seqs(n);
    int q = 0;
    for (int b = 0; b < n; ++b) {
      long long np;
      if (scanf("%d %lld", &seqs[b].len, &np) != 2) return 1;
      seqs[b].n_past = np;
      seqs[b].q_start = q;
      q += seqs[b].len;
    }
    AttnLaunch p{};
    p.n_q_heads = hq;
    p.n_kv_heads = hkv;
    p.head_dim = d;
    p.v_transposed = vt != 0;
    p.is_bf16 = true;
    p.scale = 1.0f;
    p.n_seqs = n;
    p.seqs = seqs.data();
    p.ws_cap = cap > 0 ? (size_t)cap : SIZE_MAX;
    static AttnPlan plan;
    if (!make_plan(p, plan)) {
      printf("plan none\nend\n");
      continue;
    }
    printf("plan ok %d %d %d %d %zu\n", plan.units_per_head, plan.range_major, plan.qpw,
           plan.waves, plan.ws_bytes);
    for (int b = 0; b < n; ++b) {
      const SeqPlan &s = plan.seq[b];
      printf("seq %d %d %d %lld %d %d %d\n", b, s.q_start, s.len, (long long)s.n_past, s.n_tg,
             s.n_tasks, s.max_splits);
    }
    for (int u = 0; u < plan.units_per_head; ++u) {
      const UnitLoc l = locate_unit(plan, u);
      printf("unit %d %d %d %d %d %d %d %d\n", u, l.seq, l.w.tgrp, l.w.split, l.w.k_begin,
             l.w.split_keys, l.w.n_splits, group_splits(plan.seq[l.seq], l.w.tgrp));
    }
    printf("end\n");
    fflush(stdout);
  }
  return 0;
}
