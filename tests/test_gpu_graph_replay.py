"""The path captured in a HIP graph (as bench.py times it) gives the eager result bit for bit on
every replay: splice + re-anchor (one pass, or two calls), then the suffix attention with its key
splits and combine, at Qwen2.5-14B shapes (one suffix; four suffixes in one varlen launch over a
shuffled cache) and at head_dim 256 with a transposed V and the soft cap.  Between replays the
program does eager work of its own (restores the cache, poisons the output and the workspace)
and synchronises; each replay must rewrite all of it."""

import numpy as np
import pytest
import torch

from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

pytestmark = pytest.mark.gpu


def _capture(fn):
    fn()                                        # first call outside the capture (map check)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    return g


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _setup(tag, n_tok, H, Hq, D, vt, n_q, blk_len):
    npp = (n_tok + PAGE - 1) // PAGE + 3
    std = D ** -0.5
    k = G.device_normal(2, tag, 1, (1, npp, H, PAGE, D), std, "bf16", "cuda")
    vshape = (1, H, D, npp * PAGE) if vt else (1, npp, H, PAGE, D)
    v = G.device_normal(2, tag, 2, vshape, std, "bf16", "cuda")
    perm = np.random.default_rng([20397, 906, tag]).permutation(npp).astype(np.int32)
    pm = torch.from_numpy(perm[:(n_tok + PAGE - 1) // PAGE]).to("cuda")
    cache = N.PagedKVCache(k, v, pm, 1e6, N.V_TRANSPOSED if vt else N.V_ROWMAJOR)
    blk = N.Block(G.device_normal(2, tag, 3, (1, blk_len, H, D), std, "bf16", "cuda"),
                  G.device_normal(2, tag, 4, (1, blk_len, H, D), std, "bf16", "cuda"), 0, 1e6)
    q = G.device_normal(2, tag, 0, (n_q, Hq, D), std, "bf16", "cuda")
    return cache, blk, q


def _replays_match(fn, cache, out, ws):
    k0, v0 = cache.k.clone(), cache.v.clone()
    fn()                                        # eager reference
    torch.cuda.synchronize()
    ref = [_bits(x).clone() for x in (cache.k, cache.v, out)]
    cache.k.copy_(k0)
    cache.v.copy_(v0)
    g = _capture(fn)
    for rep in range(3):
        cache.k.copy_(k0)
        cache.v.copy_(v0)
        out.fill_(float("nan"))
        if ws is not None:
            ws.fill_(0xFF)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, x, r in zip(("cache k", "cache v", "out"), (cache.k, cache.v, out), ref):
            assert torch.equal(_bits(x), r), f"replay {rep}: {name} differs from the eager run"
        print(f"  replay {rep}: cache and output bit-identical to the eager run", flush=True)


def test_graph_one_pass_splice_and_attention_qwen14b():
    # one layer: a 512-token block spliced at 2048 with its keys re-anchored in the same pass,
    # then 192 queries at 2432 (the split plan and its combine)
    H, Hq, D = 8, 40, 128
    cache, blk, q = _setup(1, 2624, H, Hq, D, False, 192, 512)
    out = torch.empty_like(q)
    ws = torch.empty(max(N.suffix_attn_workspace_bytes(cache, 192, Hq, 2432), 16),
                     dtype=torch.uint8, device="cuda")

    def fn():
        N.splice_rephase_pages(cache, blk, 2048, 2048)
        N.suffix_attn(q, cache, 0, 2432, out=out, workspace=ws)

    _replays_match(fn, cache, out, ws)


def test_graph_two_call_splice_and_varlen_attention():
    # splice then re-anchor in place (two calls), then four suffixes over the shuffled cache in
    # one varlen launch (range by range)
    H, Hq, D = 8, 40, 128
    starts, lens, pasts = [0, 128, 256, 384], [128, 128, 128, 128], [900, 1700, 2500, 3300]
    cache, blk, q = _setup(2, 3428, H, Hq, D, False, 512, 384)
    out = torch.empty_like(q)
    ws = torch.empty(max(N.suffix_attn_varlen_workspace_bytes(cache, starts, lens, pasts, Hq), 16),
                     dtype=torch.uint8, device="cuda")

    def fn():
        N.splice_pages(cache, blk, 1000)
        N.rephase_k_paged(cache, 1000, 384, 0, 1000, 1e6)
        N.suffix_attn_varlen(q, starts, lens, pasts, cache, 0, out=out, workspace=ws)

    _replays_match(fn, cache, out, ws)


def test_graph_head_dim_256_transposed_softcap():
    # head_dim 256 with a transposed V and the soft cap: one-pass splice (V transposed on the
    # way in), then 256 queries at 2800
    H, Hq, D = 8, 16, 256
    cache, blk, q = _setup(3, 3056, H, Hq, D, True, 256, 512)
    out = torch.empty_like(q)
    ws = torch.empty(max(N.suffix_attn_workspace_bytes(cache, 256, Hq, 2800), 16),
                     dtype=torch.uint8, device="cuda")

    def fn():
        N.splice_rephase_pages(cache, blk, 2400, 2400)
        N.suffix_attn(q, cache, 0, 2800, 50.0, out=out, workspace=ws)

    _replays_match(fn, cache, out, ws)
