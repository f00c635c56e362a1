"""The depth-adaptive sweep's premise on the GPU: with position-independent pre-RoPE K/V, the
rows the splice path re-decodes equal the same rows of a full causal prefill over the spliced
cache (the 'R = 100% is a full prefill' identity, Sec. III-C, Table tab:perf), for the redecode
lengths eq. (adaptive) gives at K = 4 and 16.  Both GPU outputs are checked against each other
and sampled rows against the fp64 oracle; the context rows and the redecoded rows computed as two
sequences of one launch match the prefill's rows too."""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import gen as G

from _pipeline import BF16_MAX_ABS, BF16_REL_RMS, compare

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_past", [256, 512, 1024])
def test_redecoded_rows_equal_full_prefill_rows(n_past):
    Hq, H, D, S, u, base, cfg = 40, 8, 128, 512, 64, 1e6, 2
    std = 128 ** -0.5
    total = n_past + S + u
    npp = (total + PAGE - 1) // PAGE
    k = G.device_normal(cfg, n_past, G.TAG["k_ctx"], (1, npp, H, PAGE, D), std, "bf16", "cuda")
    v = G.device_normal(cfg, n_past, G.TAG["v_ctx"], (1, npp, H, PAGE, D), std, "bf16", "cuda")
    cache = N.PagedKVCache(k, v, torch.arange(npp, dtype=torch.int32, device="cuda"), base)
    bk = G.device_normal(cfg, n_past, G.TAG["k_blk"], (1, S, H, D), std, "bf16", "cuda")
    bv = G.device_normal(cfg, n_past, G.TAG["v_blk"], (1, S, H, D), std, "bf16", "cuda")
    N.splice_rephase_pages(cache, N.Block(bk, bv, 0, base), n_past, n_past)
    q = G.device_normal(cfg, n_past, G.TAG["q"], (total, Hq, D), std, "bf16", "cuda")
    full = N.suffix_attn(q, cache, 0, 0)
    torch.cuda.synchronize()
    full_bits = G.torch_to_bits(full)
    lk, lv = O.gather_logical(G.torch_to_bits(cache.k), G.torch_to_bits(cache.v),
                              np.arange(npp), total, PAGE)
    kk, vv = O.storage_to_f64(lk[0], "bf16"), O.storage_to_f64(lv[0], "bf16")
    qq = O.storage_to_f64(G.torch_to_bits(q), "bf16")
    for K in (4, 16):
        r = N.redecode_len(S, n_past, 256, 5, K)
        n_s = r + u
        suf = N.suffix_attn(q[total - n_s:].contiguous(), cache, 0, total - n_s)
        torch.cuda.synchronize()
        got = O.bf16_bits_to_f64(G.torch_to_bits(suf))
        ref_gpu = O.bf16_bits_to_f64(full_bits[total - n_s:])
        ma, rr = compare(got, ref_gpu)
        assert ma <= BF16_MAX_ABS and rr <= BF16_REL_RMS, (K, ma, rr)
        # the context rows and the redecoded rows as two sequences of one launch
        one = N.suffix_attn_varlen(torch.cat([q[:n_past], q[total - n_s:]]).contiguous(),
                                   [0, n_past], [n_past, n_s], [0, total - n_s], cache, 0)
        torch.cuda.synchronize()
        ob = O.bf16_bits_to_f64(G.torch_to_bits(one))
        for part, want in ((ob[:n_past], O.bf16_bits_to_f64(full_bits[:n_past])),
                           (ob[n_past:], ref_gpu)):
            ma, rr = compare(part, want)
            assert ma <= BF16_MAX_ABS and rr <= BF16_REL_RMS, ("one launch", K, ma, rr)
        # the first and last redecoded rows of KV head 3's query heads against the oracle
        rows = [0, n_s - 1]
        g0 = 3 * (Hq // H)
        for row in rows:
            w = O.suffix_attention(qq[total - n_s + row:total - n_s + row + 1, g0:g0 + Hq // H],
                                   kk[:, 3:4], vv[:, 3:4], total - n_s + row)
            ma, rr = compare(got[row:row + 1, g0:g0 + Hq // H], w)
            assert ma <= BF16_MAX_ABS and rr <= BF16_REL_RMS, (K, row, ma, rr)
