"""GPU parity of the warm-prefix page operations (Sec. VI-D on a paged cache) against the oracle:
token-range copies between two page maps and prefix sharing, bit for bit over the whole cache
and the destination map, for both V layouts and both element types, with ranges that start and
end inside pages, single tokens, whole pages and pages the two maps already share; then a
decode step over the shared prefix."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

pytestmark = pytest.mark.gpu

VL = {"rowmajor": N.V_ROWMAJOR, "transposed": N.V_TRANSPOSED}
BITS = {"bf16": np.uint16, "f32": np.uint32}


def _case(dtype, v_layout, L=3, npg=24, H=2, D=64, seed=0):
    rng = np.random.default_rng(seed)
    top = 1 << (16 if dtype == "bf16" else 32)
    ck = rng.integers(0, top, (L, npg, H, PAGE, D), dtype=np.uint64).astype(BITS[dtype])
    vs = (L, H, D, npg * PAGE) if v_layout == "transposed" else (L, npg, H, PAGE, D)
    cv = rng.integers(0, top, vs, dtype=np.uint64).astype(BITS[dtype])
    perm = rng.permutation(npg).astype(np.int32)
    src = perm[:8].copy()
    dst = perm[8:16].copy()
    dst[1] = src[1]                                  # logical page 1 already shared
    return ck, cv, src, dst


def _device(ck, cv, dtype, v_layout):
    # raw bits travel as integers; the library only moves bits
    idt = torch.int16 if dtype == "bf16" else torch.int32
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    k = torch.from_numpy(ck.view(np.int16 if dtype == "bf16" else np.int32)).cuda().view(tdt)
    v = torch.from_numpy(cv.view(np.int16 if dtype == "bf16" else np.int32)).cuda().view(tdt)
    cache = N.PagedKVCache(k, v, torch.zeros(1, dtype=torch.int32, device="cuda"), 1e4,
                           VL[v_layout])
    return cache, idt


def _host_bits(t, dtype):
    return G.torch_to_bits(t)


def test_share_with_partial_page_already_shared_is_a_no_op_copy():
    """A partial page that both maps already name is left as it is (the copy is skipped)."""
    ck, cv, src, dst = _case("bf16", "rowmajor", seed=3)
    cache, _ = _device(ck, cv, "bf16", "rowmajor")
    s_d, d_d = torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda()
    N.kv_share_prefix(cache, s_d, d_d, 20)          # logical page 1 is shared by construction
    torch.cuda.synchronize()
    assert np.array_equal(_host_bits(cache.k, "bf16"), ck)
    assert np.array_equal(d_d.cpu().numpy()[:1], src[:1])


@pytest.mark.parametrize("dtype,v_layout", [("bf16", "rowmajor"), ("bf16", "transposed"),
                                            ("f32", "rowmajor"), ("f32", "transposed")])
@pytest.mark.parametrize("t0,n", [(0, 128), (5, 60), (17, 1), (16, 16), (31, 2), (3, 110)])
def test_copy_tokens_bit_exact(dtype, v_layout, t0, n):
    ck, cv, src, dst = _case(dtype, v_layout, seed=t0 * 131 + n)
    cache, _ = _device(ck, cv, dtype, v_layout)
    s_d, d_d = torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda()
    N.kv_copy_tokens(cache, s_d, d_d, t0, n)
    torch.cuda.synchronize()
    rk, rv = O.copy_tokens(ck, cv, src, dst, t0, n, PAGE, v_layout)
    assert np.array_equal(_host_bits(cache.k, dtype), rk)
    assert np.array_equal(_host_bits(cache.v, dtype), rv)
    assert np.array_equal(d_d.cpu().numpy(), dst)


@pytest.mark.parametrize("dtype,v_layout", [("bf16", "rowmajor"), ("bf16", "transposed"),
                                            ("f32", "transposed")])
@pytest.mark.parametrize("n", [0, 1, 16, 37, 100, 128])
def test_share_prefix_bit_exact(dtype, v_layout, n):
    ck, cv, src, dst = _case(dtype, v_layout, seed=1000 + n)
    cache, _ = _device(ck, cv, dtype, v_layout)
    s_d, d_d = torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda()
    N.kv_share_prefix(cache, s_d, d_d, n)
    torch.cuda.synchronize()
    rk, rv, rmap = O.share_prefix(ck, cv, src, dst, n, PAGE, v_layout)
    assert np.array_equal(d_d.cpu().numpy(), rmap)
    assert np.array_equal(_host_bits(cache.k, dtype), rk)
    assert np.array_equal(_host_bits(cache.v, dtype), rv)


def test_decode_over_a_shared_prefix():
    """Sequence B takes A's first 300 tokens by sharing (18 pages aliased, 12 slots copied),
    then appends 45 tokens of its own; one decode step for both matches the oracle over the
    caches the oracle builds by the same steps."""
    rng = np.random.default_rng(7)
    H, Hq, D, npg = 2, 8, 128, 64
    ck = G.to_bits(rng.standard_normal((1, npg, H, PAGE, D)) * 0.3, "bf16")
    cv = G.to_bits(rng.standard_normal((1, npg, H, PAGE, D)), "bf16")
    perm = rng.permutation(npg).astype(np.int32)
    map_a, map_b = perm[:24].copy(), perm[24:48].copy()
    len_a, shared, len_b = 340, 300, 345
    cache, _ = _device(ck, cv, "bf16", "rowmajor")
    m = torch.from_numpy(np.stack([map_a, map_b])).cuda()
    N.kv_share_prefix(cache, m[0], m[1], shared)
    # B's own tokens 300 .. 344 (rows already in B's private pages: copy them from a fresh draw)
    own_k = G.to_bits(rng.standard_normal((1, len_b - shared, H, D)) * 0.3, "bf16")
    own_v = G.to_bits(rng.standard_normal((1, len_b - shared, H, D)), "bf16")
    blk = N.Block(G.bits_to_torch(own_k, "bf16", "cuda"), G.bits_to_torch(own_v, "bf16", "cuda"),
                  0, 1e4)
    cache_b = N.PagedKVCache(cache.k, cache.v, m[1].clone(), 1e4, N.V_ROWMAJOR)
    N.splice_pages(cache_b, blk, shared)
    q = G.to_bits(rng.standard_normal((2, Hq, D)), "bf16")
    lens = torch.tensor([len_a, len_b], dtype=torch.int32, device="cuda")
    out = N.decode_attn(G.bits_to_torch(q, "bf16", "cuda"), cache, m, lens, len_b, 0)
    torch.cuda.synchronize()
    # oracle: same steps on the host
    rk, rv, rmap_b = O.share_prefix(ck, cv, map_a, map_b, shared, PAGE)
    rk, rv = O.splice_paged(rk, rv, rmap_b, own_k, own_v, shared, PAGE)
    assert np.array_equal(m[1].cpu().numpy(), rmap_b)
    maps = np.stack([map_a, rmap_b])
    ref = O.decode_attention(O.bf16_bits_to_f64(q), O.bf16_bits_to_f64(rk[0]),
                             O.bf16_bits_to_f64(rv[0]), maps, (len_a, len_b), PAGE)
    got = out.float().cpu().double().numpy()
    err = np.abs(got - ref).max()
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    print(f"decode over shared prefix: max-abs {err:.3e} rel-RMS {rel:.3e}", flush=True)
    assert err <= 2e-2 and rel <= 5e-3
    # the shared part reads the same keys for both: attention of A and B over [0, 300) agree
    assert np.array_equal(O.gather_logical(rk, rv, map_a, shared, PAGE)[0],
                          O.gather_logical(rk, rv, rmap_b, shared, PAGE)[0])
