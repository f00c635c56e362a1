"""GPU parity of the decode step on seeded random batches against the fp64 oracle: sequence
count and lengths (0, page edges, long), a shared prefix, head_dim, GQA group (1 to 32 query
heads per KV head), V layout, soft-capping, page shuffling and storage type drawn from a
fixed-seed generator.  Tolerances as the other decode tests."""

import dataclasses

import numpy as np
import pytest

from synth import decode as SD

from test_gpu_decode import _check, _oracle, _upload
from paper_2608_20397_amd import nexus as N

import torch

pytestmark = pytest.mark.gpu


def _draw(i: int) -> SD.DecodeWorkload:
    r = np.random.default_rng([20397, 950, i])
    f32 = i % 5 == 4
    d = int(r.choice([32, 64, 128])) if f32 else int(r.choice([64, 128, 128, 256]))
    n_kv = int(r.choice([1, 2, 4, 8]))
    g = int(r.choice([1, 2, 5, 8, 16, 32]))
    n_seqs = int(r.integers(1, 9))
    lens = [int(x) for x in r.integers(0, 3000, size=n_seqs)]
    for j in range(n_seqs):                     # some page-edge and tiny lengths
        if r.random() < 0.3:
            lens[j] = int(r.choice([0, 1, 15, 16, 17, 32, 33]))
    shared = int(r.choice([0, 0, 64, 300]))
    base = SD.decode_workload(1 if f32 else 2)
    return dataclasses.replace(
        base, case=1000 + i, name=f"random {i}", n_layers=1, n_q_heads=g * n_kv, n_kv_heads=n_kv,
        head_dim=d, lens=tuple(lens), shared_prefix=shared,
        v_layout=str(r.choice(["rowmajor", "transposed"])), softcap=float(r.choice([0.0, 30.0])),
        shuffled=bool(r.integers(0, 2)), q_scale=1.0, k_scale=d ** -0.5 * 2, v_scale=1.0)


CASES = [_draw(i) for i in range(15)]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_decode_parity(i):
    wl = CASES[i]
    print(f"random decode {i}: {wl.dtype} D={wl.head_dim} Hkv={wl.n_kv_heads} Hq={wl.n_q_heads} "
          f"lens {wl.lens} shared {wl.shared_prefix} {wl.v_layout} cap {wl.softcap}", flush=True)
    hc = SD.decode_host_case_wl(wl)
    cache, maps, lens, q = _upload(hc)
    out = N.decode_attn(q[0], cache, maps, lens, wl.max_len, 0, softcap=wl.softcap)
    torch.cuda.synchronize()
    got = out.float().cpu().double().numpy()
    _check(got, _oracle(hc, 0), wl.dtype, f"random decode {i}")
    for b, n in enumerate(wl.lens):
        if n == 0:
            assert np.array_equal(got[b], np.zeros_like(got[b])), b
