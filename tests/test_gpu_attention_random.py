"""GPU parity of the suffix attention on seeded random geometries against the fp64 oracle, every
query row and head compared: head_dim, GQA group, KV heads, context depth, block and user
lengths (page-unaligned splices), suffix length, V layout, soft-capping, page shuffling and
storage type drawn from a fixed-seed generator, so that shapes between the named configs and
edge cases (several tiles with ragged tails, short and long splits, one to many task groups)
are covered too.  Tolerances as the other attention tests."""

import numpy as np
import pytest

from synth import gen as G

from _pipeline import custom_workload
from test_gpu_attention import _run_full

pytestmark = pytest.mark.gpu


def _draw(i: int) -> dict:
    r = np.random.default_rng([20397, 900, i])
    f32 = i % 6 == 5
    if f32:
        base, d = 1, int(r.choice([32, 64, 128]))
        n_kv, g = int(r.choice([1, 2])), int(r.choice([1, 2, 4]))
    else:
        d = int(r.choice([64, 128, 128, 256]))
        base = 5 if d == 256 else 2
        n_kv = int(r.choice([1, 2, 4, 8]))
        g = int(r.choice([1, 2, 3, 5, 8]))
    n_ctx = int(r.integers(0, 2000))
    block = int(r.integers(1, 400))
    n_user = int(r.integers(0, 65))
    n_suffix = int(r.integers(1, block + n_user + 1))
    kw = dict(head_dim=d, n_kv_heads=n_kv, n_q_heads=g * n_kv,
              v_layout=str(r.choice(["rowmajor", "transposed"])),
              softcap=float(r.choice([0.0, 0.0, 30.0])),
              shuffled_pages=bool(r.integers(0, 2)))
    return dict(base=base, n_ctx=n_ctx, block=block, n_user=n_user, n_suffix=n_suffix, kw=kw)


CASES = [_draw(i) for i in range(18)]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_geometry_parity(i):
    c = CASES[i]
    wl = custom_workload(c["base"], c["n_ctx"], c["block"], c["n_user"], c["n_suffix"], **c["kw"])
    tag = (f"random {i}: {wl.dtype} D={wl.head_dim} Hkv={wl.n_kv_heads} Hq={wl.n_q_heads} "
           f"ctx {c['n_ctx']} block {c['block']} user {c['n_user']} suffix {c['n_suffix']} "
           f"{wl.v_layout} cap {wl.softcap} shuffled {wl.shuffled_pages}")
    print(tag, flush=True)
    hc = G.host_case_wl(wl, 300 + i)
    _run_full(hc, tag)


def _draw_d256(i: int) -> dict:
    """head_dim 256 with a transposed V (the soft-capped family's kernel): GQA groups 1..8, so
    that workgroups of 8 wave tasks hold several query blocks and heads or leave slots idle,
    contexts deep enough for several key splits, the cap on or off, ragged suffixes."""
    r = np.random.default_rng([20397, 901, i])
    n_kv = int(r.choice([1, 2, 4]))
    g = int(r.choice([1, 2, 3, 5, 8]))
    n_ctx = int(r.integers(0, 3000))
    block = int(r.integers(1, 300))
    n_user = int(r.integers(0, 65))
    n_suffix = int(r.integers(1, block + n_user + 1))
    kw = dict(head_dim=256, n_kv_heads=n_kv, n_q_heads=g * n_kv, v_layout="transposed",
              softcap=float(r.choice([0.0, 20.0, 50.0, 50.0])),
              shuffled_pages=bool(r.integers(0, 2)))
    return dict(base=5, n_ctx=n_ctx, block=block, n_user=n_user, n_suffix=n_suffix, kw=kw)


CASES_D256 = [_draw_d256(i) for i in range(10)]


@pytest.mark.parametrize("i", range(len(CASES_D256)))
def test_random_d256_transposed_parity(i):
    c = CASES_D256[i]
    wl = custom_workload(c["base"], c["n_ctx"], c["block"], c["n_user"], c["n_suffix"], **c["kw"])
    tag = (f"random D256 {i}: Hkv={wl.n_kv_heads} Hq={wl.n_q_heads} ctx {c['n_ctx']} "
           f"block {c['block']} user {c['n_user']} suffix {c['n_suffix']} cap {wl.softcap} "
           f"shuffled {wl.shuffled_pages}")
    print(tag, flush=True)
    hc = G.host_case_wl(wl, 400 + i)
    _run_full(hc, tag)
