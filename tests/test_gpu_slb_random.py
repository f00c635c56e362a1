"""GPU parity of the SLB scan on seeded random registries against the oracle, bit for bit (top-k
indices and scores, margin, gate): random tool and query counts on both sides of the batched
kernel's threshold, dims (64-byte steps, odd and even counts), k, duplicated tools (ties) and
scales."""

import numpy as np
import pytest
import torch

from test_gpu_slb import _check_scan

pytestmark = pytest.mark.gpu


def _draw(i: int):
    r = np.random.default_rng([20397, 990, i])
    n_tools = int(r.choice([1, 7, 64, 65, 300, 1000, 5000, 20000]))
    n_q = int(r.choice([1, 2, 16, 17, 63, 64, 65, 130]))
    dim = 64 * int(r.integers(1, 17))
    k = int(r.integers(1, 9))
    return n_tools, n_q, dim, k, int(r.integers(0, 1 << 30))


CASES = [_draw(i) for i in range(14)]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_slb_parity(i):
    n_tools, n_q, dim, k, seed = CASES[i]
    rng = np.random.default_rng(seed)
    rtq = rng.integers(-127, 128, (n_tools, dim)).astype(np.int8)
    rts = rng.uniform(0.001, 0.01, n_tools).astype(np.float32)
    for _ in range(3):                           # duplicated tools: equal scores
        a, b = rng.integers(0, n_tools, 2)
        rtq[b], rts[b] = rtq[a], rts[a]
    rqq = rng.integers(-127, 128, (n_q, dim)).astype(np.int8)
    rqs = rng.uniform(0.001, 0.01, n_q).astype(np.float32)
    tq, ts = torch.from_numpy(rtq).cuda(), torch.from_numpy(rts).cuda()
    qq, qs = torch.from_numpy(rqq).cuda(), torch.from_numpy(rqs).cuda()
    _check_scan(tq, ts, qq, qs, k, float(rng.uniform(0.0, 0.05)), rtq, rts, rqq, rqs,
                f"random slb {i}: {n_tools} tools x {n_q} queries x {dim}, k {k}")
