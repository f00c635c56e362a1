"""Seeded synthetic decode batches: several sequences, each with its own page map over one shared
pool of physical pages, optionally sharing the physical pages of a common prefix (a warm
prefix reused across sequences).  No arithmetic of the method.

Recipe:
* Each sequence b has ``lens[b]`` cached tokens and one query (its newest token).
* The first ``shared_prefix // 16`` logical pages of every sequence map to the same physical
  pages; every other page of every sequence is private.  Physical pages are handed out from a
  seeded permutation of the pool (or in order when not shuffled).
* K, V and Q are N(0, std^2) draws cast to the storage type; pool pages that no sequence maps,
  and the slots past the end of each sequence's last page, hold a NaN sentinel, so any read of
  a key the query must not see shows up in the output.
* Host draws use ``numpy.random.default_rng(SeedSequence([20397, 100 + case, layer, tag]))``;
  large cases draw on the device with torch's generator (``synth.gen.device_normal``).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import PAGE
from . import gen as G

TAG = dict(q=20, k=21, v=22, perm=23, lens=24)


@dataclass(frozen=True)
class DecodeWorkload:
    case: int
    name: str
    dtype: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    lens: tuple              # cached tokens per sequence (the query's own token included)
    shared_prefix: int       # tokens whose pages every sequence shares (rounded down to pages)
    v_layout: str
    softcap: float
    shuffled: bool
    q_scale: float
    k_scale: float
    v_scale: float
    spare_pages: int = 3     # unmapped pool pages (NaN sentinel)

    @property
    def n_seqs(self) -> int:
        return len(self.lens)

    @property
    def max_len(self) -> int:
        return max(self.lens)

    @property
    def map_stride(self) -> int:
        return max(1, -(-self.max_len // PAGE))

    @property
    def shared_pages(self) -> int:
        return min(self.shared_prefix, min(self.lens)) // PAGE

    @property
    def n_phys_pages(self) -> int:
        private = sum(max(0, -(-n // PAGE) - self.shared_pages) for n in self.lens)
        return self.shared_pages + private + self.spare_pages


def _lens_mix(case: int, n: int, lo: int, hi: int) -> tuple:
    r = G.rng(100 + case, 0, TAG["lens"])
    return tuple(int(x) for x in r.integers(lo, hi + 1, size=n))


def decode_workload(case: int) -> DecodeWorkload:
    s = 128 ** -0.5
    if case == 1:
        return DecodeWorkload(1, "tiny fp32, mixed lengths", "f32", 1, 4, 1, 64,
                              lens=(225, 1, 17, 0, 40, 16, 600), shared_prefix=0,
                              v_layout="rowmajor", softcap=0.0, shuffled=False,
                              q_scale=1.0, k_scale=1.0, v_scale=1.0)
    if case == 2:
        return DecodeWorkload(2, "qwen2.5-14b heads, 8 sequences, shared 256-token prefix", "bf16",
                              1, 40, 8, 128, lens=(257, 271, 272, 273, 300, 1000, 2625, 4097),
                              shared_prefix=256, v_layout="rowmajor", softcap=0.0, shuffled=True,
                              q_scale=s, k_scale=s, v_scale=s)
    if case == 3:
        return DecodeWorkload(3, "qwen2.5-14b, one 17473-token sequence, 48 layers", "bf16", 48,
                              40, 8, 128, lens=(17473,), shared_prefix=0, v_layout="rowmajor",
                              softcap=0.0, shuffled=False, q_scale=s, k_scale=s, v_scale=s)
    if case == 4:
        return DecodeWorkload(4, "qwen2.5-14b, 32 sequences sharing a 16384-token prefix", "bf16",
                              1, 40, 8, 128, lens=_lens_mix(4, 32, 16385, 17473),
                              shared_prefix=16384, v_layout="rowmajor", softcap=0.0,
                              shuffled=True, q_scale=s, k_scale=s, v_scale=s)
    if case == 5:
        return DecodeWorkload(5, "gemma-2-style soft-capped, transposed V, head_dim 256", "bf16", 1,
                              16, 8, 256, lens=(1, 100, 4500, 9217), shared_prefix=0,
                              v_layout="transposed", softcap=50.0, shuffled=True,
                              q_scale=1.0, k_scale=3.0, v_scale=1.0)
    if case == 6:
        return DecodeWorkload(6, "head_dim 64, 32 query heads per KV head, lengths 0..700", "bf16",
                              1, 64, 2, 64, lens=(0, 1, 2, 15, 16, 17, 33, 700), shared_prefix=0,
                              v_layout="rowmajor", softcap=0.0, shuffled=True,
                              q_scale=1.0, k_scale=0.25, v_scale=1.0)
    if case == 7:
        return DecodeWorkload(7, "fp32, transposed V, soft-capped, shared prefix", "f32", 1, 6, 2,
                              32, lens=(48, 49, 80, 33), shared_prefix=32, v_layout="transposed",
                              softcap=20.0, shuffled=True, q_scale=1.0, k_scale=2.0, v_scale=1.0)
    raise ValueError(f"no decode case {case}")


def page_maps(wl: DecodeWorkload) -> np.ndarray:
    """int32 [n_seqs][map_stride]: shared prefix pages first, then private pages per sequence;
    entries past a sequence's last page are -1 (never read)."""
    order = (G.rng(100 + wl.case, 0, TAG["perm"]).permutation(wl.n_phys_pages) if wl.shuffled
             else np.arange(wl.n_phys_pages))
    order = order.astype(np.int32)
    maps = np.full((wl.n_seqs, wl.map_stride), -1, dtype=np.int32)
    nxt = wl.shared_pages
    for b, n in enumerate(wl.lens):
        npg = -(-n // PAGE)
        for p in range(npg):
            if p < wl.shared_pages:
                maps[b, p] = order[p]
            else:
                maps[b, p] = order[nxt]
                nxt += 1
    return maps


@dataclass
class DecodeHostCase:
    wl: DecodeWorkload
    maps: np.ndarray          # [n_seqs][map_stride] int32
    k: np.ndarray             # raw bits [L][NPP][H][16][D]
    v: np.ndarray             # raw bits, row-major as k or transposed [L][H][D][NPP * 16]
    q: np.ndarray             # raw bits [L][n_seqs][Hq][D] (one query batch per layer)


def written_slots(wl: DecodeWorkload, maps: np.ndarray) -> np.ndarray:
    """bool [NPP][16]: physical slots that hold a token of some sequence."""
    w = np.zeros((wl.n_phys_pages, PAGE), dtype=bool)
    for b, n in enumerate(wl.lens):
        for t in range(n):
            w[maps[b, t // PAGE], t % PAGE] = True
    return w


def decode_host_case(case: int, layers=None) -> DecodeHostCase:
    """Host draws of one decode case (all pool pages are drawn; unwritten slots get the NaN
    sentinel)."""
    return decode_host_case_wl(decode_workload(case), layers)


def decode_host_case_wl(wl: DecodeWorkload, layers=None) -> DecodeHostCase:
    """Host draws of any decode workload record (seeds from its ``case`` slot)."""
    case = wl.case
    layers = list(range(wl.n_layers)) if layers is None else list(layers)
    H, D, NPP = wl.n_kv_heads, wl.head_dim, wl.n_phys_pages
    maps = page_maps(wl)
    w = written_slots(wl, maps)
    sent = G.SENTINEL[wl.dtype]
    ks, vs, qs = [], [], []
    for l in layers:
        k = G.to_bits(G.normal(100 + case, l, TAG["k"], (NPP, H, PAGE, D), wl.k_scale), wl.dtype)
        v = G.to_bits(G.normal(100 + case, l, TAG["v"], (NPP, H, PAGE, D), wl.v_scale), wl.dtype)
        unwritten = np.broadcast_to(~w[:, None, :, None], k.shape)
        k[unwritten] = sent
        v[unwritten] = sent
        if wl.v_layout == "transposed":
            v = np.ascontiguousarray(v.transpose(1, 3, 0, 2).reshape(H, D, NPP * PAGE))
        ks.append(k)
        vs.append(v)
        qs.append(G.to_bits(G.normal(100 + case, l, TAG["q"], (wl.n_seqs, wl.n_q_heads, D),
                                     wl.q_scale), wl.dtype))
    return DecodeHostCase(wl, maps, np.stack(ks), np.stack(vs), np.stack(qs))
