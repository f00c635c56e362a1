"""GPU parity of the suffix attention at the limits of its plan, against the fp64 oracle:

* the most sequences one launch takes (32): all suffix-like (units taken key range by key
  range) and mixed with causal prefills (sequence by sequence), head_dim 128 and head_dim 256
  with a transposed V and the soft cap; every row of every sequence;
* the longest key range one workgroup covers (32768 keys, its LDS page table full): shapes
  whose plan gives some workgroups a single 32768-key split (the host planner test pins that
  these plans do); sampled rows at the start, middle and end of the suffix, two KV heads;
* a context longer than one workgroup may cover (70000 keys before 16 queries), so that every
  row merges dozens of splits; head_dim 64 (the generic kernel), 128 and 256 with transposed V
  and the soft cap; every row;
* two suffixes over more than 2^21 keys (past the range order), and the fp32 kernel at 32
  sequences and over a 70000-key context.

Tolerances as the other bf16 attention tests.
"""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

from _pipeline import BF16_MAX_ABS, BF16_REL_RMS, F32_TOL, compare

pytestmark = pytest.mark.gpu


def _cache(tag, n_tok, H, d, vt, k_mult=1.0, shuffle=True, dt="bf16"):
    npp = (n_tok + PAGE - 1) // PAGE + 2
    std = d ** -0.5
    k = G.device_normal(2, tag, 1, (1, npp, H, PAGE, d), std * k_mult, dt, "cuda")
    vshape = (1, H, d, npp * PAGE) if vt else (1, npp, H, PAGE, d)
    v = G.device_normal(2, tag, 2, vshape, std, dt, "cuda")
    perm = (np.random.default_rng([20397, 904, tag]).permutation(npp) if shuffle
            else np.arange(npp)).astype(np.int32)
    pm = perm[:(n_tok + PAGE - 1) // PAGE]
    cache = N.PagedKVCache(k, v, torch.from_numpy(pm).to("cuda"), 1e4,
                           N.V_TRANSPOSED if vt else N.V_ROWMAJOR)
    lk, lv = O.gather_logical(G.torch_to_bits(k), G.torch_to_bits(v), pm, n_tok, PAGE,
                              O.TRANSPOSED if vt else O.ROWMAJOR)
    return cache, O.storage_to_f64(lk[0], dt), O.storage_to_f64(lv[0], dt)


def _check(got, ref, what, dt="bf16"):
    ma, rr = compare(got, ref)
    print(f"  {what}: max-abs {ma:.3e} rel-RMS {rr:.3e}", flush=True)
    assert np.isfinite(got).all(), what
    if dt == "bf16":
        assert ma <= BF16_MAX_ABS and rr <= BF16_REL_RMS, (what, ma, rr)
    else:
        assert ma <= F32_TOL and rr <= F32_TOL, (what, ma, rr)


def _seqs32(r, n_tok, prefills):
    seqs = []
    for b in range(32):
        if prefills and b % 5 == 2:
            n = int(r.integers(40, 300))
            p = int(r.integers(0, n))
        elif b % 7 == 0:
            n, p = 1, int(r.integers(1, n_tok))
        else:
            n = int(r.integers(2, 90))
            p = int(r.integers(n, n_tok - n + 1))
        seqs.append((n, min(p, n_tok - n)))
    return seqs


@pytest.mark.parametrize("d,prefills", [(128, False), (128, True), (256, False), (256, True)])
def test_32_sequences_one_launch(d, prefills):
    tag = 10 + d // 128 + 2 * prefills
    vt, cap = d == 256, (50.0 if d == 256 else 0.0)
    H, Hq, n_tok = 2, 4, 2600
    seqs = _seqs32(np.random.default_rng([20397, 905, tag]), n_tok, prefills)
    lens = [s[0] for s in seqs]
    pasts = [s[1] for s in seqs]
    starts = [int(x) for x in np.cumsum([0] + lens[:-1])]
    print(f"32 sequences D={d} prefills={prefills}: {seqs}", flush=True)
    cache, kk, vv = _cache(tag, n_tok, H, d, vt, 3.0 if cap else 1.0)
    q = G.device_normal(2, tag, 0, (sum(lens), Hq, d), d ** -0.5, "bf16", "cuda")
    out = N.suffix_attn_varlen(q, starts, lens, pasts, cache, 0, cap)
    torch.cuda.synchronize()
    qq = O.storage_to_f64(G.torch_to_bits(q), "bf16")
    got = O.bf16_bits_to_f64(G.torch_to_bits(out))
    for b, (q0, n, p) in enumerate(zip(starts, lens, pasts)):
        ref = O.suffix_attention(qq[q0:q0 + n], kk, vv, p, softcap=cap)
        _check(got[q0:q0 + n], ref, f"seq {b} ({n} queries at {p})")


# (head_dim, transposed V, soft cap, H_q, H_kv, queries, n_past): plans with 32768-key splits
LONGEST_SPLIT = [(128, False, 0.0, 40, 8, 2048, 30720), (256, True, 50.0, 16, 8, 4096, 28672)]


@pytest.mark.parametrize("case", LONGEST_SPLIT)
def test_longest_split_sampled(case):
    d, vt, cap, Hq, H, n_s, n_past = case
    g = Hq // H
    n_tok = n_past + n_s
    print(f"longest split: D={d} Hq={Hq} Hkv={H} {n_s} queries at {n_past}", flush=True)
    cache, kk, vv = _cache(20 + d // 128, n_tok, H, d, vt, 3.0 if cap else 1.0)
    q = G.device_normal(2, 20 + d // 128, 0, (n_s, Hq, d), d ** -0.5, "bf16", "cuda")
    out = N.suffix_attn(q, cache, 0, n_past, cap)
    torch.cuda.synchronize()
    got = O.bf16_bits_to_f64(G.torch_to_bits(out))
    qq = O.storage_to_f64(G.torch_to_bits(q), "bf16")
    for kvh in (0, H - 1):
        for r0 in (0, n_s // 2 - 2, n_s - 4):
            rows = slice(r0, r0 + 4)
            heads = slice(kvh * g, (kvh + 1) * g)
            ref = O.suffix_attention(qq[rows, heads], kk[:, kvh:kvh + 1], vv[:, kvh:kvh + 1],
                                     n_past + r0, softcap=cap)
            _check(got[rows, heads], ref, f"kv head {kvh} rows {r0}..{r0 + 3}")


@pytest.mark.parametrize("d,vt,cap,Hq,H", [(64, False, 0.0, 8, 2), (128, False, 0.0, 8, 2),
                                           (256, True, 50.0, 4, 2)])
def test_context_beyond_one_split(d, vt, cap, Hq, H):
    n_s, n_past = 16, 70000
    tag = 30 + d // 64
    print(f"70000-key context: D={d} Hq={Hq} Hkv={H} vt={vt} cap={cap}", flush=True)
    cache, kk, vv = _cache(tag, n_past + n_s, H, d, vt, 3.0 if cap else 1.0)
    q = G.device_normal(2, tag, 0, (n_s, Hq, d), d ** -0.5, "bf16", "cuda")
    out = N.suffix_attn(q, cache, 0, n_past, cap)
    torch.cuda.synchronize()
    got = O.bf16_bits_to_f64(G.torch_to_bits(out))
    ref = O.suffix_attention(O.storage_to_f64(G.torch_to_bits(q), "bf16"), kk, vv, n_past,
                             softcap=cap)
    _check(got, ref, f"{n_s} queries over {n_past + n_s} keys")


# Soft cap of the head_dim-256 transposed-V kernel over logit spreads (q ~ N(0, 1),
# k ~ N(0, sd^2 / 256), so scale q.k ~ N(0, sd^2)) from barely bent by cap 50 to saturating it,
# and caps from 8 to 2000 (the capped score is cap (1 - 2 r) with r near 1/2, so the rounding
# of r weighs more as the cap grows).
@pytest.mark.parametrize("sd,cap", [(3.0, 50.0), (6.0, 50.0), (10.0, 50.0), (60.0, 50.0),
                                    (3.0, 8.0), (3.0, 300.0), (3.0, 2000.0)])
def test_softcap_logit_spread_and_cap(sd, cap):
    d, H, Hq, n_s, n_past = 256, 2, 4, 300, 2000
    tag = 40 + int(sd) + int(cap) % 97
    print(f"soft cap {cap}, logit std {sd}", flush=True)
    cache, kk, vv = _cache(tag, n_past + n_s, H, d, True, sd)
    q = G.device_normal(2, tag, 0, (n_s, Hq, d), 1.0, "bf16", "cuda")
    out = N.suffix_attn(q, cache, 0, n_past, cap)
    torch.cuda.synchronize()
    got = O.bf16_bits_to_f64(G.torch_to_bits(out))
    qq = O.storage_to_f64(G.torch_to_bits(q), "bf16")
    ref = O.suffix_attention(qq, kk, vv, n_past, softcap=cap)
    _check(got, ref, f"cap {cap} logit std {sd}")


# Two suffixes over a context of more than 2^21 keys (past the range order's 64 ranges of
# 32768 keys: the plan takes them sequence by sequence, each row merging over 64 splits), one KV
# head; every row.
@pytest.mark.parametrize("d", [64, 128])
def test_suffixes_beyond_the_range_order(d):
    n = 64 * 32768
    lens, pasts = [8, 8], [n + 100000, n + 50000]
    starts = [0, 8]
    n_tok = max(p + s for p, s in zip(pasts, lens))
    H, Hq = 1, 4
    tag = 60 + d // 64
    print(f"two suffixes over {n_tok} keys, D={d}", flush=True)
    cache, kk, vv = _cache(tag, n_tok, H, d, False)
    q = G.device_normal(2, tag, 0, (sum(lens), Hq, d), d ** -0.5, "bf16", "cuda")
    out = N.suffix_attn_varlen(q, starts, lens, pasts, cache, 0)
    torch.cuda.synchronize()
    qq = O.storage_to_f64(G.torch_to_bits(q), "bf16")
    got = O.bf16_bits_to_f64(G.torch_to_bits(out))
    for b, (q0, m, p) in enumerate(zip(starts, lens, pasts)):
        ref = O.suffix_attention(qq[q0:q0 + m], kk, vv, p)
        _check(got[q0:q0 + m], ref, f"seq {b} ({m} queries at {p})")


# fp32 caches (the fp32 kernel): 32 sequences in one launch (transposed V, soft cap, causal
# prefills among them) and 16 queries over a 70000-key context; every row, fp32 tolerance.
def test_f32_32_sequences_and_long_context():
    H, Hq, d, n_tok = 2, 4, 64, 2600
    seqs = _seqs32(np.random.default_rng([20397, 905, 70]), n_tok, True)
    lens = [x[0] for x in seqs]
    pasts = [x[1] for x in seqs]
    starts = [int(x) for x in np.cumsum([0] + lens[:-1])]
    print(f"f32: 32 sequences {seqs}", flush=True)
    cache, kk, vv = _cache(70, n_tok, H, d, True, dt="f32")
    q = G.device_normal(2, 70, 0, (sum(lens), Hq, d), d ** -0.5, "f32", "cuda")
    out = N.suffix_attn_varlen(q, starts, lens, pasts, cache, 0, 30.0)
    torch.cuda.synchronize()
    qq = O.storage_to_f64(G.torch_to_bits(q), "f32")
    got = O.storage_to_f64(G.torch_to_bits(out), "f32")
    for b, (q0, n, p) in enumerate(zip(starts, lens, pasts)):
        ref = O.suffix_attention(qq[q0:q0 + n], kk, vv, p, softcap=30.0)
        _check(got[q0:q0 + n], ref, f"f32 seq {b} ({n} queries at {p})", "f32")
    n_s, n_past, d, Hq = 16, 70000, 128, 8
    print("f32: 16 queries over a 70000-key context", flush=True)
    cache, kk, vv = _cache(71, n_past + n_s, H, d, False, dt="f32")
    q = G.device_normal(2, 71, 0, (n_s, Hq, d), d ** -0.5, "f32", "cuda")
    out = N.suffix_attn(q, cache, 0, n_past)
    torch.cuda.synchronize()
    ref = O.suffix_attention(O.storage_to_f64(G.torch_to_bits(q), "f32"), kk, vv, n_past)
    _check(O.storage_to_f64(G.torch_to_bits(out), "f32"), ref, "f32 long context", "f32")
