"""nexus_suffix_attn_noalloc (split partials in the library's static device array) against
nexus_suffix_attn (caller workspace), through the C ABI.

Calls in a row on one GPU share the array: a long suffix whose workspace plan does not fit the
array (Qwen2.5-14B shapes, 2048 queries at depth 16384: a capped plan, so within the bf16
attention tolerance of the workspace call), then a shorter one whose plan fits (192 queries at
2432: bit-identical), then head_dim 256 with a transposed V and a soft cap (256 queries at 1792:
bit-identical), and a suffix no plan fits into the array (refused, nothing written).  A split
partial takes 2 * head_dim + 16 bytes per row and head (fp16 row, fp32 record).
"""

import math

import pytest
import torch

from paper_2608_20397_amd import nexus as N
from synth import gen as G

pytestmark = pytest.mark.gpu

MAX_ABS, REL_RMS = 2e-2, 5e-3


def _case(seed, n_q, n_kv, D, n_past, n_s, v_layout=N.V_ROWMAJOR, k_std=None, base=1e6):
    n_tok = n_past + n_s
    npp = (n_tok + 15) // 16
    std = D ** -0.5
    k = G.device_normal(2, seed, 1, (1, npp, n_kv, 16, D), k_std or std, "bf16", "cuda")
    vshape = (1, n_kv, D, npp * 16) if v_layout == N.V_TRANSPOSED else (1, npp, n_kv, 16, D)
    v = G.device_normal(2, seed, 2, vshape, std, "bf16", "cuda")
    cache = N.PagedKVCache(k, v, torch.arange(npp, dtype=torch.int32, device="cuda"), base,
                           v_layout)
    q = G.device_normal(2, seed, 0, (n_s, n_q, D), std, "bf16", "cuda")
    return cache, q


def _rel(a, b):
    a, b = a.double(), b.double()
    return (a - b).abs().max().item(), ((a - b).norm() / b.norm()).item()


def test_noalloc_matches_workspace_call_twice_then_smaller():
    limit = 64 << 20
    # 1: Qwen2.5-14B attention shapes, 2048 queries at depth 16384; its workspace plan needs
    # more than the array holds
    cache, q = _case(70, 40, 8, 128, 16384, 2048)
    need = N.suffix_attn_workspace_bytes(cache, 2048, 40, 16384)
    assert need > limit
    ref = N.suffix_attn(q, cache, 0, 16384)
    got = torch.full_like(q, float("nan"))
    N.suffix_attn_noalloc(q, cache, 0, 16384, out=got)
    torch.cuda.synchronize()
    assert torch.isfinite(got.float()).all()
    ma, rr = _rel(got, ref)
    print(f"noalloc 2048 @ 16384 (capped plan): max-abs {ma:.3e} rel-RMS {rr:.3e}", flush=True)
    assert ma <= MAX_ABS and rr <= REL_RMS
    # 2: a smaller call right after: the plan fits, so the result is bit-identical
    cache2, q2 = _case(71, 40, 8, 128, 2432, 192)
    assert 0 < N.suffix_attn_workspace_bytes(cache2, 192, 40, 2432) <= limit
    ref2 = N.suffix_attn(q2, cache2, 0, 2432)
    got2 = torch.full_like(q2, float("nan"))
    N.suffix_attn_noalloc(q2, cache2, 0, 2432, out=got2)
    torch.cuda.synchronize()
    assert torch.equal(got2.view(torch.int16), ref2.view(torch.int16))
    # and the first call again, after the smaller one: still within tolerance, run to run equal
    again = torch.full_like(q, float("nan"))
    N.suffix_attn_noalloc(q, cache, 0, 16384, out=again)
    torch.cuda.synchronize()
    assert torch.equal(again.view(torch.int16), got.view(torch.int16))


def test_noalloc_head_dim_256_transposed_softcap_is_bit_identical():
    cache, q = _case(72, 16, 8, 256, 1792, 256, v_layout=N.V_TRANSPOSED, k_std=3.0, base=1e4)
    assert 0 < N.suffix_attn_workspace_bytes(cache, 256, 16, 1792) <= 64 << 20
    ref = N.suffix_attn(q, cache, 0, 1792, softcap=50.0)
    got = torch.full_like(q, float("nan"))
    N.suffix_attn_noalloc(q, cache, 0, 1792, softcap=50.0, out=got)
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16))


def test_noalloc_refuses_a_suffix_no_plan_fits():
    # 4096 queries x 40 heads over 36864 keys: at least two splits (a split covers <= 32768
    # keys), whose partials (2 x 4096 x 40 x (2 x 128 + 16) bytes) exceed the array
    cache, q = _case(73, 40, 8, 128, 32768, 4096)
    assert 2 * 4096 * 40 * (2 * 128 + 16) > 64 << 20
    out = torch.full_like(q, 7.0)
    with pytest.raises(N.NexusError) as e:
        N.suffix_attn_noalloc(q, cache, 0, 32768, out=out)
    assert e.value.status == N.EWORKSPACE
    torch.cuda.synchronize()
    assert (out.float() == 7.0).all()
    assert math.isfinite(float(N.suffix_attn(q[:64].contiguous(), cache, 0, 32768).float().sum()))
