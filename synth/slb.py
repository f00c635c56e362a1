"""Seeded synthetic registries and queries for the SLB scan (no arithmetic of the method).

The paper's tool vectors come from an embedding model over tool names and descriptions, which
is not available; unit-norm Gaussian vectors stand in.  Recipe: tool t is a N(0, I) draw of
dimension ``dim`` scaled to unit norm; query j mixes two tools, t_a + w t_b with w ~ U(0.9, 1.1),
plus N(0, noise^2 / dim) noise per feature, renormalised, so its best two tools are a and b and
the top-two margin spreads on both sides of the gate threshold (an adversarial pair in the
paper's sense).  fp32 values; quantisation is the method's (``nexus_slb_quantize`` /
``oracle.slb_quantize``).  Seeds: ``numpy.random.default_rng(SeedSequence([20397, 200 + case,
0, tag]))``.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import gen as G

TAG = dict(tools=30, targets=31, noise=32, rivals=33, weights=34)


@dataclass(frozen=True)
class SlbWorkload:
    case: int
    name: str
    n_tools: int
    n_queries: int
    dim: int
    noise: float
    k: int
    tau: float = 0.0136


def slb_workload(case: int) -> SlbWorkload:
    if case == 1:
        return SlbWorkload(1, "paper registry: 250 tools, one query", 250, 1, 768, 0.3, 3)
    if case == 2:
        return SlbWorkload(2, "250 tools, 64 queries", 250, 64, 768, 0.3, 3)
    if case == 3:
        return SlbWorkload(3, "65536 tools, 256 queries (serving batch)", 65536, 256, 768, 0.3, 8)
    if case == 4:
        return SlbWorkload(4, "ragged: 1 tool, 3 queries, dim 64", 1, 3, 64, 0.5, 2)
    if case == 5:
        return SlbWorkload(5, "ragged: 1000 tools, 100 queries, dim 1024", 1000, 100, 1024, 0.3, 8)
    if case == 6:
        return SlbWorkload(6, "5000 tools, 1 query, dim 384", 5000, 1, 384, 0.3, 1)
    raise ValueError(f"no slb case {case}")


def slb_inputs(case: int):
    """(tools fp32 [N][dim], queries fp32 [Q][dim], (a, b) tool pairs [Q][2])."""
    wl = slb_workload(case)
    r = G.rng(200 + case, 0, TAG["tools"])
    tools = r.standard_normal((wl.n_tools, wl.dim))
    tools /= np.linalg.norm(tools, axis=1, keepdims=True)
    a = G.rng(200 + case, 0, TAG["targets"]).integers(0, wl.n_tools, size=wl.n_queries)
    b = G.rng(200 + case, 0, TAG["rivals"]).integers(0, wl.n_tools, size=wl.n_queries)
    w = G.rng(200 + case, 0, TAG["weights"]).uniform(0.9, 1.1, size=wl.n_queries)
    noise = G.rng(200 + case, 0, TAG["noise"]).standard_normal((wl.n_queries, wl.dim))
    noise *= wl.noise / np.sqrt(wl.dim)
    q = tools[a] + w[:, None] * tools[b] + noise
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    return tools.astype(np.float32), q.astype(np.float32), np.stack([a, b], axis=1)
