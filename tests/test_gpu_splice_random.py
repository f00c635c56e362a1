"""GPU parity of the splice, re-anchor and one-pass splice + re-anchor on seeded random
geometries against the oracle, over the whole cache: V bits equal, K bits equal outside the
re-anchored rows and within the re-anchor bound inside them (1 bf16 ulp, at least 99.9% exact;
1e-5 for f32), for random storage type, head_dim, KV heads, layers, context depth, block and
user lengths (page-unaligned), V layout and page shuffling, split and fused."""

import dataclasses

import numpy as np
import pytest
import torch

from synth import gen as G

from _pipeline import check_keys, custom_workload, gpu_build_cache, oracle_cache, range_mask

pytestmark = pytest.mark.gpu


def _draw(i: int):
    r = np.random.default_rng([20397, 970, i])
    f32 = i % 4 == 3
    d = int(r.choice([32, 64, 128])) if f32 else int(r.choice([64, 128, 256]))
    base = 1 if f32 else 2
    n_ctx = int(r.integers(0, 1200))
    block = int(r.integers(1, 300))
    n_user = int(r.integers(0, 40))
    wl = custom_workload(base, n_ctx, block, n_user, 1, head_dim=d,
                         n_kv_heads=int(r.choice([1, 2, 4, 8])),
                         v_layout=str(r.choice(["rowmajor", "transposed"])),
                         shuffled_pages=bool(r.integers(0, 2)))
    wl = dataclasses.replace(wl, n_layers=int(r.integers(1, 4)), n_q_heads=wl.n_kv_heads)
    return wl, bool(r.integers(0, 2))


CASES = [_draw(i) for i in range(16)]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_splice_rephase_parity(i):
    wl, fused = CASES[i]
    tag = (f"random splice {i}: {wl.dtype} D={wl.head_dim} H={wl.n_kv_heads} L={wl.n_layers} "
           f"ctx {wl.splice_pos[0]} block {wl.block_len} user {wl.n_user} {wl.v_layout} "
           f"shuffled {wl.shuffled_pages} fused {fused}")
    print(tag, flush=True)
    hc = G.host_case_wl(wl, 400 + i)
    npp = wl.n_pages + 2
    pm = hc.page_map
    cache = gpu_build_cache(hc, n_phys_pages=npp, fused=fused)
    torch.cuda.synchronize()
    ck, cv = oracle_cache(hc, n_phys_pages=npp)
    assert np.array_equal(G.torch_to_bits(cache.v), cv), tag
    check_keys(G.torch_to_bits(cache.k), ck, range_mask(wl, wl.n_layers, npp, pm), wl.dtype, tag)
