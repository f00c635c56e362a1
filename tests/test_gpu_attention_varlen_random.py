"""GPU parity of one varlen attention launch on seeded random mixes of sequences over one cache
against the fp64 oracle, every row and head: causal prefills (n_past < queries, dispatched
longest first), re-decoded suffixes (a few hundred queries deep in the context) and single-query
tails, two to five of them per launch in random order, so that the plan takes its
sequence-by-sequence path with per-sequence key splits (or, when no prefill is present, its
range-by-range path) and the combine merges rows of sequences whose split counts differ.  Cache
pages shuffled; head_dim 64 / 128 with a row-major V, 256 with a transposed V and the soft cap.
Tolerances as the other attention tests."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

from _pipeline import BF16_MAX_ABS, BF16_REL_RMS, compare

pytestmark = pytest.mark.gpu


def _draw(i: int) -> dict:
    r = np.random.default_rng([20397, 902, i])
    d = int(r.choice([64, 128, 128, 256]))
    n_kv = int(r.choice([1, 2, 4]))
    g = int(r.choice([1, 2, 5]))
    n_tok = int(r.integers(600, 2600))
    seqs = []
    for _ in range(int(r.integers(2, 6))):
        kind = int(r.integers(0, 3))
        if kind == 0:                                  # causal prefill from a shallow start
            n_s = int(r.integers(100, min(900, n_tok) + 1))
            n_past = int(r.integers(0, n_s // 2 + 1))
        elif kind == 1:                                # re-decoded suffix deep in the context
            n_s = int(r.integers(20, 400))
            n_past = int(r.integers(n_s, n_tok - n_s + 1))
        else:                                          # one query at the end of its context
            n_s = 1
            n_past = int(r.integers(0, n_tok))
        n_past = min(n_past, n_tok - n_s)
        seqs.append((n_s, n_past))
    return dict(d=d, n_kv=n_kv, hq=g * n_kv, n_tok=n_tok, seqs=seqs,
                vt=d == 256, cap=50.0 if d == 256 else 0.0)


CASES = [_draw(i) for i in range(8)]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_varlen_mix_parity(i):
    c = CASES[i]
    d, H, Hq, n_tok = c["d"], c["n_kv"], c["hq"], c["n_tok"]
    lens = [s[0] for s in c["seqs"]]
    pasts = [s[1] for s in c["seqs"]]
    starts = list(np.cumsum([0] + lens[:-1]))
    tag = f"varlen {i}: D={d} Hkv={H} Hq={Hq} tokens {n_tok} seqs {list(zip(lens, pasts))}"
    print(tag, flush=True)
    npp = (n_tok + PAGE - 1) // PAGE + 3
    std = d ** -0.5
    k = G.device_normal(2, i, 1, (1, npp, H, PAGE, d), std * (3.0 if c["cap"] else 1.0), "bf16",
                        "cuda")
    vshape = (1, H, d, npp * PAGE) if c["vt"] else (1, npp, H, PAGE, d)
    v = G.device_normal(2, i, 2, vshape, std, "bf16", "cuda")
    perm = np.random.default_rng([20397, 903, i]).permutation(npp).astype(np.int32)
    pm = perm[:(n_tok + PAGE - 1) // PAGE]
    cache = N.PagedKVCache(k, v, torch.from_numpy(pm).to("cuda"), 1e4,
                           N.V_TRANSPOSED if c["vt"] else N.V_ROWMAJOR)
    q = G.device_normal(2, i, 0, (sum(lens), Hq, d), std, "bf16", "cuda")
    out = N.suffix_attn_varlen(q, starts, lens, pasts, cache, 0, c["cap"])
    torch.cuda.synchronize()
    lk, lv = O.gather_logical(G.torch_to_bits(k), G.torch_to_bits(v), pm, n_tok, PAGE,
                              O.TRANSPOSED if c["vt"] else O.ROWMAJOR)
    kk, vv = O.storage_to_f64(lk[0], "bf16"), O.storage_to_f64(lv[0], "bf16")
    qq = O.storage_to_f64(G.torch_to_bits(q), "bf16")
    got = O.bf16_bits_to_f64(G.torch_to_bits(out))
    for b, (q0, n_s, n_past) in enumerate(zip(starts, lens, pasts)):
        ref = O.suffix_attention(qq[q0:q0 + n_s], kk, vv, n_past, softcap=c["cap"])
        ma, rr = compare(got[q0:q0 + n_s], ref)
        print(f"  seq {b} ({n_s} queries at {n_past}): max-abs {ma:.3e} rel-RMS {rr:.3e}",
              flush=True)
        assert np.isfinite(got[q0:q0 + n_s]).all(), (tag, b)
        assert ma <= BF16_MAX_ABS and rr <= BF16_REL_RMS, (tag, b, ma, rr)
