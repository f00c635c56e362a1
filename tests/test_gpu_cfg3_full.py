"""Config 3 at full size, bit level: every one of the 48 layers of the spliced, re-anchored cache
against the oracle (Sec. VI-A: rows written exactly; Sec. III-B: re-anchoring is the rotation by
the position difference).

The benchmarked workload (Qwen2.5-14B shapes, a 1024-token block compiled at 0 and spliced at
16384 into a 17472-token cache, 48 layers) is the only one whose re-anchor launch covers more key
rows (393,216) than one pass of its grid, so these tests are what reaches the kernels' grid-stride
continuation.  Inputs are device draws copied to the host before any kernel runs; the oracle
builds each layer from those host bits, and the comparison goes layer by layer to bound host
memory: values and every slot outside the block bit for bit (sentinels in unmapped pages
included), re-anchored keys within one bf16 step of the oracle's single rounding and at least
99.9% bit-equal.
"""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

from _pipeline import (check_keys, close_keys, device_case, empty_device_cache, gpu_build_cache,
                       host_subset, layer_of, oracle_cache, range_mask)

pytestmark = pytest.mark.gpu

EXTRA_PAGES = 3          # physical pages that no logical page maps to (they keep the sentinel)


def test_cfg3_splice_rephase_all_layers():
    """Splice + in-place re-anchor (two calls) and the one-pass splice + re-anchor of config 3:
    the two caches bit-identical, and each layer equal to the oracle's."""
    dc = device_case(3)
    hc = host_subset(dc, range(dc.wl.n_layers), with_q=False)    # before any kernel
    wl = hc.wl
    npp = wl.n_pages + EXTRA_PAGES
    print(f"cfg3 full: {wl.n_layers} layers, block {wl.block_len} at {wl.splice_pos[0]}, "
          f"{npp} physical pages", flush=True)
    two = gpu_build_cache(dc, n_phys_pages=npp)
    one = gpu_build_cache(dc, n_phys_pages=npp, fused=True)
    torch.cuda.synchronize()
    same_k = torch.equal(one.k.view(torch.int16), two.k.view(torch.int16))
    same_v = torch.equal(one.v.view(torch.int16), two.v.view(torch.int16))
    del one
    assert same_k, "one-pass K differs from splice + re-anchor"
    assert same_v, "one-pass V differs from splice + re-anchor"
    mask = range_mask(wl, 1, npp, hc.page_map)
    unmapped = sorted(set(range(npp)) - set(hc.page_map.tolist()))
    assert len(unmapped) == EXTRA_PAGES
    for layer in range(wl.n_layers):
        ck, cv = oracle_cache(layer_of(hc, layer), n_phys_pages=npp)
        gk = G.torch_to_bits(two.k[layer:layer + 1])
        gv = G.torch_to_bits(two.v[layer:layer + 1])
        assert np.array_equal(gv, cv), f"layer {layer}: V cache bits differ"
        check_keys(gk, ck, mask, "bf16", f"cfg3 layer {layer}")
        assert (gk[:, unmapped] == G.SENTINEL["bf16"]).all(), f"layer {layer}: unmapped page"


def test_cfg3_rephase_block_all_layers():
    """nexus_rephase_k on config 3's contiguous block (48 x 1024 x 8 key rows) from its anchor 0
    to 16384, against the oracle's rotation of the same bits; values untouched."""
    dc = device_case(3)
    wl = dc.wl
    k = dc.blk_k[0].clone()
    v = dc.blk_v[0]
    k_bits = G.torch_to_bits(k)
    v_bits = G.torch_to_bits(v)
    rows = k.shape[0] * k.shape[1] * k.shape[2]
    print(f"cfg3 block re-anchor: {rows} key rows", flush=True)
    assert rows > 4096 * 64           # more rows than one pass of the capped grid
    blk = N.Block(k, v, wl.anchor, wl.rope_base)
    dst = wl.splice_pos[0]
    N.rephase_k(blk, wl.anchor, dst, wl.rope_base)
    torch.cuda.synchronize()
    assert blk.base_pos == dst
    assert np.array_equal(G.torch_to_bits(v), v_bits), "values must not be rotated"
    for layer in range(wl.n_layers):
        ref = O.round_to_storage(
            O.rephase(O.storage_to_f64(k_bits[layer], "bf16"), wl.anchor, dst, wl.rope_base),
            "bf16")
        close_keys(G.torch_to_bits(k[layer]), ref, "bf16", f"block layer {layer}")


def test_cfg3_rope_append_all_layers():
    """nexus_rope_append of the 1088 redecoded tokens of config 3 (un-rotated K and V of all 48
    layers, device draws) at logical slots 16384 .. 17471, keys rotated to those positions: the
    oracle's RoPE at each position, one rounding; values and every other slot bit for bit."""
    wl = G.get_workload(3)
    L, H, D = wl.n_layers, wl.n_kv_heads, wl.head_dim
    T = wl.n_suffix
    off = wl.n_tokens - T
    std = wl.k_scale
    k_new = torch.stack([G.device_normal(3, l, 40, (T, H, D), std, "bf16", "cuda") for l in range(L)])
    v_new = torch.stack([G.device_normal(3, l, 41, (T, H, D), std, "bf16", "cuda") for l in range(L)])
    k_bits = G.torch_to_bits(k_new)
    v_bits = G.torch_to_bits(v_new)
    npp = wl.n_pages + EXTRA_PAGES
    pm = G.page_map(3, wl.n_pages, wl.shuffled_pages)
    print(f"cfg3 rope-append: {L} layers x {T} tokens at {off}", flush=True)
    cache = empty_device_cache(wl, L, npp, pm)
    N.rope_append(cache, k_new, v_new, off, off)
    torch.cuda.synchronize()
    assert np.array_equal(G.torch_to_bits(k_new), k_bits), "inputs must not be modified"
    kb1, vb1 = G.empty_cache_bits(wl, 1, npp)
    pos = off + np.arange(T)
    mask = np.zeros(kb1.shape, bool)
    for t in range(off, off + T):
        mask[:, pm[t // PAGE], :, t % PAGE, :] = True
    for layer in range(L):
        rot = O.round_to_storage(O.rope(O.storage_to_f64(k_bits[layer], "bf16"), pos,
                                        wl.rope_base), "bf16")
        ok, ov = O.splice_paged(kb1, vb1, pm, rot[None], v_bits[layer:layer + 1], off, PAGE)
        gk = G.torch_to_bits(cache.k[layer:layer + 1])
        gv = G.torch_to_bits(cache.v[layer:layer + 1])
        assert np.array_equal(gv, ov), f"layer {layer}: values must be copied bit for bit"
        check_keys(gk, ok, mask, "bf16", f"append layer {layer}")
