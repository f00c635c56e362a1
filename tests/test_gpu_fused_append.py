"""GPU parity of the one-pass splice + re-anchor and of rope-append against the oracle.

* nexus_splice_rephase_pages: the cache must be bit-identical to a splice followed by an
  in-place re-anchor (the same rotation arithmetic), and its keys within 1 bf16 ulp of the
  oracle's fp64 rotation (>= 99.9% exactly rounded) or 1e-5 for f32; values and every other
  element bit-exact; an anchored block (dst = anchor) is a plain bit copy.
* nexus_rope_append: un-rotated keys rotated to positions pos0 + j (the oracle's rope at those
  positions, one rounding) and values written bit for bit into logical slots offset + j; every
  other element keeps its bits.
"""

import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

from _pipeline import VL, check_keys, close_keys, gpu_build_cache, oracle_cache, range_mask

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [1, 2, 4, 5])
def test_fused_equals_splice_then_rephase_and_oracle(cfg):
    hc = G.host_case(cfg)
    wl = hc.wl
    npp = wl.n_pages + 3
    two = gpu_build_cache(hc, n_phys_pages=npp)
    one = gpu_build_cache(hc, n_phys_pages=npp, fused=True)
    torch.cuda.synchronize()
    k1, v1 = G.torch_to_bits(one.k), G.torch_to_bits(one.v)
    assert np.array_equal(k1, G.torch_to_bits(two.k)), "K differs from splice + re-anchor"
    assert np.array_equal(v1, G.torch_to_bits(two.v)), "V differs from splice + re-anchor"
    ck, cv = oracle_cache(hc, n_phys_pages=npp)
    assert np.array_equal(v1, cv)
    check_keys(k1, ck, range_mask(wl, 1, npp, hc.page_map), wl.dtype, f"cfg{cfg}")


def test_fused_anchored_block_is_a_bit_copy():
    hc = G.host_case(1)
    hc.wl = dataclasses.replace(hc.wl, anchor=128)
    cache = gpu_build_cache(hc, fused=True)
    torch.cuda.synchronize()
    ck, cv = oracle_cache(hc)
    assert np.array_equal(G.torch_to_bits(cache.k), ck)
    assert np.array_equal(G.torch_to_bits(cache.v), cv)


@pytest.mark.parametrize("v_layout", ["rowmajor", "transposed"])
@pytest.mark.parametrize("offset,T,anchor", [(0, 16, 0), (5, 1, 0), (7, 50, 3), (37, 200, 0),
                                             (1, 255, 11)])
def test_fused_unaligned_edges(v_layout, offset, T, anchor):
    wl = dataclasses.replace(G.get_workload(2), n_tokens=512, block_len=T, splice_pos=(offset,),
                             n_user=0, v_layout=v_layout, shuffled_pages=True, n_layers=2)
    rng = np.random.default_rng(offset * 1000 + T)
    blk_k = G.to_bits(rng.standard_normal((2, T, 8, 128)), "bf16")
    blk_v = G.to_bits(rng.standard_normal((2, T, 8, 128)), "bf16")
    npp = wl.n_pages + 4
    pm = rng.permutation(npp)[:wl.n_pages].astype(np.int32)
    kb, vb = G.empty_cache_bits(wl, 2, npp)
    cache = N.PagedKVCache(G.bits_to_torch(kb, "bf16", "cuda"), G.bits_to_torch(vb, "bf16", "cuda"),
                           torch.from_numpy(pm).cuda(), wl.rope_base, VL[v_layout])
    dst = offset + 4000
    N.splice_rephase_pages(cache, N.Block(G.bits_to_torch(blk_k, "bf16", "cuda"),
                                          G.bits_to_torch(blk_v, "bf16", "cuda"), anchor,
                                          wl.rope_base), offset, dst)
    torch.cuda.synchronize()
    ok, ov = O.splice_paged(kb, vb, pm, blk_k, blk_v, offset, PAGE, v_layout)
    ok = O.rephase_paged_bits(ok, "bf16", pm, PAGE, offset, T, anchor, dst, wl.rope_base)
    gk, gv = G.torch_to_bits(cache.k), G.torch_to_bits(cache.v)
    assert np.array_equal(gv, ov)
    check_keys(gk, ok, range_mask(wl, 2, npp, pm), "bf16", f"{v_layout} {offset} {T}")


@pytest.mark.parametrize("dtype,style,D,v_layout,base", [
    ("bf16", N.ROPE_NEOX, 128, "rowmajor", 1e6),
    ("bf16", N.ROPE_INTERLEAVED, 128, "rowmajor", 1e6),
    ("bf16", N.ROPE_NEOX, 256, "transposed", 1e4),
    ("bf16", N.ROPE_NEOX, 64, "transposed", 1e4),
    ("f32", N.ROPE_NEOX, 64, "rowmajor", 1e4),
    ("f32", N.ROPE_INTERLEAVED, 64, "transposed", 1e4)])
@pytest.mark.parametrize("offset,T,pos0", [(0, 1, 0), (13, 77, 13), (100, 200, 31744)])
def test_rope_append_matches_oracle_rope(dtype, style, D, v_layout, base, offset, T, pos0):
    L, H = 3, 2
    wl = dataclasses.replace(G.get_workload(2), n_tokens=320, n_kv_heads=H, head_dim=D,
                             dtype=dtype, v_layout=v_layout, rope_base=base)
    rng = np.random.default_rng(D * 7 + T + offset)
    k_bits = G.to_bits(rng.standard_normal((L, T, H, D)), dtype)
    v_bits = G.to_bits(rng.standard_normal((L, T, H, D)), dtype)
    npp = wl.n_pages + 2
    pm = rng.permutation(npp)[:wl.n_pages].astype(np.int32)
    kb, vb = G.empty_cache_bits(wl, L, npp)
    cache = N.PagedKVCache(G.bits_to_torch(kb, dtype, "cuda"), G.bits_to_torch(vb, dtype, "cuda"),
                           torch.from_numpy(pm).cuda(), base, VL[v_layout], style)
    k_dev = G.bits_to_torch(k_bits, dtype, "cuda")
    v_dev = G.bits_to_torch(v_bits, dtype, "cuda")
    N.rope_append(cache, k_dev, v_dev, offset, pos0)
    torch.cuda.synchronize()
    st = O.NEOX if style == N.ROPE_NEOX else O.INTERLEAVED
    pos = pos0 + np.arange(T)
    rot = np.stack([O.round_to_storage(O.rope(O.storage_to_f64(k_bits[l], dtype), pos, base, st),
                                       dtype) for l in range(L)])
    ok, ov = O.splice_paged(kb, vb, pm, rot, v_bits, offset, PAGE, v_layout)
    gk, gv = G.torch_to_bits(cache.k), G.torch_to_bits(cache.v)
    assert np.array_equal(gv, ov), "values must be copied bit for bit"
    untouched = np.ones(gk.shape, bool)
    for t in range(offset, offset + T):
        untouched[:, pm[t // PAGE], :, t % PAGE, :] = False
    assert np.array_equal(gk[untouched], ok[untouched]), "keys written outside the slots"
    close_keys(gk[~untouched], ok[~untouched], dtype, f"{dtype} {style} D{D}")
    assert np.array_equal(G.torch_to_bits(k_dev), k_bits)          # inputs are not modified


def test_rope_append_keys_at_their_positions():
    """The appended keys, read back through the logical view, are the oracle's RoPE of the
    un-rotated keys at positions 64 .. 111 (identity page table, 8 heads, 2 layers)."""
    rng = np.random.default_rng(5)
    L, T, H, D, base = 2, 48, 8, 128, 1e6
    pre = rng.standard_normal((L, T, H, D))
    pre_bits = G.to_bits(pre, "bf16")
    wl = dataclasses.replace(G.get_workload(2), n_tokens=256, n_layers=L)
    npp = wl.n_pages
    pm = np.arange(npp, dtype=np.int32)
    kb, vb = G.empty_cache_bits(wl, L, npp)
    a = N.PagedKVCache(G.bits_to_torch(kb, "bf16", "cuda"), G.bits_to_torch(vb, "bf16", "cuda"),
                       torch.from_numpy(pm).cuda(), base)
    N.rope_append(a, G.bits_to_torch(pre_bits, "bf16", "cuda"),
                  G.bits_to_torch(pre_bits, "bf16", "cuda"), 64, 64)
    torch.cuda.synchronize()
    lk, _ = O.gather_logical(G.torch_to_bits(a.k), G.torch_to_bits(a.v), pm, 112, PAGE)
    want = np.stack([O.round_to_storage(O.rope(O.storage_to_f64(pre_bits[l], "bf16"),
                                               64 + np.arange(T), base), "bf16") for l in range(L)])
    close_keys(lk[:, 64:112], want, "bf16", "append at 64")
