"""Pins of the fp64 oracle against facts fixed outside it (CPU only).

Each test ties one oracle function to something other than its own formula: the values the
paper prints (Table tab:perf), library routines (torch SDPA, the Qwen2 rotary embedding and the
Gemma-2 eager soft-capped attention of ``transformers``, torch's bfloat16 conversion), closed
forms, or invariants of the mathematics.  A dropped term, a wrong sign or index or a transposed
operand in the oracle fails at least one of them.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


# ---------------------------------------------------------------- eq. (adaptive), Table tab:perf
def test_tab_perf_R_column():
    """Eq. (adaptive) must reproduce the printed R(%) column of Table tab:perf."""
    g = json.load(open(os.path.join(HERE, "golden", "tab_perf_R.json")))
    for row in g["rows"]:
        r = O.recompute_fraction(row["n_past"], g["M"], g["R_base"], row["K"])
        assert round(float(r), 1) == row["R_pct"], row


@pytest.mark.parametrize("K", [2, 3, 4, 8, 16])
def test_R_reaches_full_at_K_times_M(K):
    """Sec. III-C: K is the multiple of M at which recompute reaches 100%; below M it is R_base."""
    M = 256
    assert O.recompute_fraction(K * M, M, 5, K) == 100
    assert O.recompute_fraction(K * M - 1, M, 5, K) < 100
    assert O.recompute_fraction(K * M + 999, M, 5, K) == 100          # clamped
    assert O.recompute_fraction(M, M, 5, K) == 5
    assert O.recompute_fraction(0, M, 5, K) == 5
    prev = Fraction(0)
    for n in range(0, K * M + 64, 7):                                  # non-decreasing in depth
        r = O.recompute_fraction(n, M, 5, K)
        assert r >= prev
        prev = r


def test_redecode_len_values():
    """ceil(S * R / 100): R = 100 gives the whole block, R_base rounds the suffix up."""
    assert O.redecode_len(1024, 16384, 256, 5, 4) == 1024
    assert O.redecode_len(1024, 16384, 256, 5, 16) == 1024             # 16384 = 64 M >= 16 M
    assert O.redecode_len(64, 128, 256, 5, 4) == 4                     # 3.2 -> 4
    assert O.redecode_len(512, 512, 256, 5, 4) == 188                  # 512*110/300 = 187.7
    assert O.redecode_len(0, 5000, 256, 5, 4) == 0
    with pytest.raises(ValueError):
        O.recompute_fraction(300, 256, 5, 1)                           # K = 1 divides by zero


# ---------------------------------------------------------------- RoPE (Sec. III-B)
def test_rope_frequency_closed_form():
    for d, b in [(64, 1e4), (128, 1e6), (256, 1e4)]:
        th = O.rope_frequencies(d, b)
        assert th[0] == 1.0
        assert math.isclose(th[1], b ** (-2.0 / d), rel_tol=1e-15)
        assert math.isclose(th[-1] * b, b ** (2.0 / d), rel_tol=1e-13)   # theta_{d/2-1} = b^{-(d-2)/d}
        assert np.allclose(th[1:] / th[:-1], b ** (-2.0 / d), rtol=1e-13)  # geometric


def test_rope_matches_qwen2_rotary_embedding():
    """NEOX pairing, sign and frequencies equal transformers' Qwen2 RoPE (fp32 library)."""
    from transformers import Qwen2Config
    from transformers.models.qwen2.modeling_qwen2 import Qwen2RotaryEmbedding, apply_rotary_pos_emb
    d, base, T = 128, 1e6, 40
    cfg = Qwen2Config(hidden_size=40 * d, num_attention_heads=40, num_key_value_heads=8,
                      rope_theta=base, max_position_embeddings=4096)
    emb = Qwen2RotaryEmbedding(cfg)
    rng = np.random.default_rng(0)
    x = rng.standard_normal((T, 3, d))
    pos = np.arange(T) * 7 + 3
    xt = torch.tensor(x, dtype=torch.float32).permute(1, 0, 2)[None]        # [1, H, T, D]
    cos, sin = emb(xt, torch.tensor(pos)[None])
    ref, _ = apply_rotary_pos_emb(xt, xt, cos, sin)
    ref = ref[0].permute(1, 0, 2).double().numpy()
    got = O.rope(x, pos, base, O.NEOX)
    assert np.max(np.abs(got - ref)) < 2e-4                                # fp32 library, pos < 300


def test_rope_two_dim_is_complex_multiplication():
    """For d = 2 there is one pair with theta_0 = 1: RoPE is z * exp(i p)."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal((50, 2))
    pos = rng.integers(0, 40000, 50)
    z = (x[:, 0] + 1j * x[:, 1]) * np.exp(1j * pos.astype(np.float64))
    got = O.rope(x, pos, 1e4)
    assert np.allclose(got[:, 0], z.real, atol=1e-11) and np.allclose(got[:, 1], z.imag, atol=1e-11)


@settings(max_examples=25, deadline=None)
@given(m=st.integers(0, 20000), n=st.integers(0, 20000), c=st.integers(-5000, 5000),
       style=st.sampled_from([O.NEOX, O.INTERLEAVED]))
def test_rope_scores_depend_on_relative_position(m, n, c, style):
    """Sec. III-B: scores depend on the relative rotation: <R_m q, R_n k> = <R_{m+c} q, R_{n+c} k>."""
    if m + c < 0 or n + c < 0:
        return
    rng = np.random.default_rng(m * 7 + n)
    q, k = rng.standard_normal((2, 1, 64))
    a = O.rope(q, [m], 1e4, style) @ O.rope(k, [n], 1e4, style).T
    b = O.rope(q, [m + c], 1e4, style) @ O.rope(k, [n + c], 1e4, style).T
    assert abs(a - b).max() < 1e-9


def test_interleaved_is_neox_on_permuted_features():
    d = 16
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, d))
    perm = np.concatenate([np.arange(0, d, 2), np.arange(1, d, 2)])   # interleaved -> half split
    a = O.rope(x, np.arange(5) * 11, 1e4, O.INTERLEAVED)
    b = O.rope(x[:, perm], np.arange(5) * 11, 1e4, O.NEOX)
    assert np.allclose(a[:, perm], b, atol=1e-13)


# ---------------------------------------------------------------- re-anchoring (eq. drift)
@settings(max_examples=20, deadline=None)
@given(p1=st.integers(0, 32768), p2=st.integers(0, 32768), base=st.sampled_from([1e4, 1e6]),
       d=st.sampled_from([64, 128, 256]))
def test_rephase_composition(p1, p2, base, d):
    """Re-phasing a block compiled at p1 to p2 equals RoPE computed at p2 directly."""
    rng = np.random.default_rng(p1 ^ (p2 << 3))
    k = rng.standard_normal((9, 2, d))
    j = np.arange(9)
    got = O.rephase(O.rope(k, p1 + j, base), p1, p2, base)
    ref = O.rope(k, p2 + j, base)
    assert np.max(np.abs(got - ref)) < 1e-9


def test_rephase_inverse_norm_identity():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((33, 8, 128))
    a = O.rephase(k, 100, 16484, 1e6)
    back = O.rephase(a, 16484, 100, 1e6)
    assert np.max(np.abs(back - k)) < 1e-12
    half = 64
    n0 = k[..., :half] ** 2 + k[..., half:] ** 2
    n1 = a[..., :half] ** 2 + a[..., half:] ** 2
    assert np.max(np.abs(n0 - n1)) < 1e-12                       # per-pair norm preserved
    assert np.array_equal(O.rephase(k, 77, 77, 1e6), k)           # delta 0 is the identity
    assert not np.allclose(a, k)                                 # and delta != 0 is not


# ---------------------------------------------------------------- bfloat16 rounding
def test_bf16_rounding_matches_torch_on_fp32_values():
    rng = np.random.default_rng(4)
    x = np.concatenate([rng.standard_normal(200000) * 10.0 ** rng.integers(-30, 30, 200000),
                        [0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38, 1e-40, -1e-40, 6e-39]])
    x32 = x.astype(np.float32)
    # add exact ties: values halfway between bf16 neighbours
    ties = ((rng.integers(0, 1 << 16, 2000).astype(np.uint32) << 16) | 0x8000).view(np.float32)
    x32 = np.concatenate([x32, ties[np.isfinite(ties)]])
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = O.f64_to_bf16_bits(x32.astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_rounding_single_rounding_from_fp64():
    e = 2.0 ** -8
    assert O.bf16_bits_to_f64(O.f64_to_bf16_bits(np.array([1 + e]))) == 1.0            # tie -> even
    assert O.bf16_bits_to_f64(O.f64_to_bf16_bits(np.array([1 + 3 * e]))) == 1 + 4 * e  # tie -> even
    # just above a tie: fp64 -> bf16 directly rounds up; fp64 -> fp32 -> bf16 would round down
    assert O.bf16_bits_to_f64(O.f64_to_bf16_bits(np.array([1 + e + 2.0 ** -30]))) == 1 + 2 * e
    assert np.isinf(O.bf16_bits_to_f64(O.f64_to_bf16_bits(np.array([3.4e38])))).all()


# ---------------------------------------------------------------- splice and page addressing
def _rand_bits(rng, shape, dtype=np.uint16):
    return rng.integers(0, 0x7F00, shape).astype(dtype)


def _identity_logical(cache, v_layout, which):
    """Library reshape: an identity-mapped page cache is a plain reshaped logical tensor."""
    if which == "v" and v_layout == O.TRANSPOSED:
        return np.transpose(cache, (0, 3, 1, 2))                      # [L][H][D][N] -> [L][N][H][D]
    L, npg, H, P, D = cache.shape
    return np.transpose(cache, (0, 1, 3, 2, 4)).reshape(L, npg * P, H, D)


@pytest.mark.parametrize("v_layout", [O.ROWMAJOR, O.TRANSPOSED])
@pytest.mark.parametrize("offset", [0, 5, 16, 37])
def test_splice_places_rows_and_leaves_the_rest(v_layout, offset):
    rng = np.random.default_rng(offset)
    L, H, D, P, npg, T = 2, 3, 8, 16, 9, 50
    perm = rng.permutation(npg).astype(np.int32)
    ck = np.full((L, npg, H, P, D), 0x7FC1, np.uint16)
    cv = (np.full((L, H, D, npg * P), 0x7FC1, np.uint16) if v_layout == O.TRANSPOSED
          else ck.copy())
    bk, bv = _rand_bits(rng, (L, T, H, D)), _rand_bits(rng, (L, T, H, D))
    nk, nv = O.splice_paged(ck, cv, perm, bk, bv, offset, P, v_layout)
    # independent addressing: un-shuffle the pages with numpy, then reshape
    inv = np.argsort(perm)
    lk = _identity_logical(nk[:, perm], v_layout, "k")
    if v_layout == O.TRANSPOSED:
        cols = (perm[:, None] * P + np.arange(P)[None, :]).reshape(-1)
        lv = _identity_logical(nv[..., cols], v_layout, "v")
    else:
        lv = _identity_logical(nv[:, perm], v_layout, "v")
    assert np.array_equal(lk[:, offset:offset + T], bk)
    assert np.array_equal(lv[:, offset:offset + T], bv)
    mask = np.ones(npg * P, bool)
    mask[offset:offset + T] = False
    assert (lk[:, mask] == 0x7FC1).all() and (lv[:, mask] == 0x7FC1).all()
    assert inv.shape == perm.shape
    # gather_logical is the inverse addressing
    gk, gv = O.gather_logical(nk, nv, perm, npg * P, P, v_layout)
    assert np.array_equal(gk, lk) and np.array_equal(gv, lv)


def test_anchored_splice_is_bit_exact():
    """Sec. IV-A: an anchored splice (delta 0) is output-exact; the cache holds the block bits."""
    rng = np.random.default_rng(7)
    L, H, D, P, T, off = 1, 1, 64, 16, 64, 128
    ck = np.full((L, 14, H, P, D), 0x7FC00001, np.uint32)
    bk = rng.standard_normal((L, T, H, D)).astype(np.float32).view(np.uint32)
    nk, _ = O.splice_paged(ck, ck.copy(), np.arange(14, dtype=np.int32), bk, bk, off, P)
    kv = O.storage_to_f64(nk, "f32")
    same = O.rephase_paged(kv, np.arange(14), P, off, T, 128, 128, 1e4)
    assert np.array_equal(O.round_to_storage(same[:, 8:12], "f32"), nk[:, 8:12])


# ---------------------------------------------------------------- attention (Sec. III-A)
def _sdpa_reference(q, k, v, n_past, scale=None):
    """torch SDPA in fp64: explicit causal-offset mask, KV heads repeated G times."""
    n_s, hq, d = q.shape
    hk = k.shape[1]
    n = n_past + n_s
    qt = torch.tensor(q).permute(1, 0, 2)[None]
    kt = torch.tensor(k[:n]).permute(1, 0, 2).repeat_interleave(hq // hk, 0)[None]
    vt = torch.tensor(v[:n]).permute(1, 0, 2).repeat_interleave(hq // hk, 0)[None]
    mask = torch.arange(n)[None, :] <= (n_past + torch.arange(n_s))[:, None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    return o[0].permute(1, 0, 2).numpy()


@settings(max_examples=20, deadline=None)
@given(n_s=st.integers(1, 9), n_past=st.integers(0, 40), hk=st.sampled_from([1, 2, 3]),
       g=st.sampled_from([1, 2, 5]), d=st.sampled_from([4, 16]))
def test_attention_matches_torch_sdpa(n_s, n_past, hk, g, d):
    rng = np.random.default_rng(n_s * 1000 + n_past)
    q = rng.standard_normal((n_s, hk * g, d))
    k = rng.standard_normal((n_past + n_s + 3, hk, d))
    v = rng.standard_normal((n_past + n_s + 3, hk, d))
    got = O.suffix_attention(q, k, v, n_past)
    assert np.max(np.abs(got - _sdpa_reference(q, k, v, n_past))) < 1e-12


def test_softcap_matches_gemma2_eager_attention():
    """Scale first, then cap * tanh(s / cap): the Gemma-2 soft-cap of transformers."""
    from transformers.models.gemma2.modeling_gemma2 import eager_attention_forward

    class _M(torch.nn.Module):
        def __init__(self, g, d):
            super().__init__()
            self.num_key_value_groups, self.head_dim = g, d

    rng = np.random.default_rng(8)
    n_s, n_past, hk, g, d, cap = 6, 20, 2, 2, 32, 5.0
    q = rng.standard_normal((n_s, hk * g, d)) * 3
    k = rng.standard_normal((n_past + n_s, hk, d)) * 3
    v = rng.standard_normal((n_past + n_s, hk, d))
    n = n_past + n_s
    allowed = np.arange(n)[None, :] <= (n_past + np.arange(n_s))[:, None]
    add = torch.tensor(np.where(allowed, 0.0, -1e30))[None, None]
    ref, _ = eager_attention_forward(_M(g, d), torch.tensor(q).permute(1, 0, 2)[None],
                                     torch.tensor(k).permute(1, 0, 2)[None],
                                     torch.tensor(v).permute(1, 0, 2)[None], add,
                                     scaling=d ** -0.5, softcap=cap)
    ref = ref[0].double().numpy()                                     # [n_s][H_q][D]
    got = O.suffix_attention(q, k, v, n_past, softcap=cap)
    assert np.max(np.abs(got - ref)) < 2e-6                           # library softmax is fp32
    assert np.max(np.abs(got - O.suffix_attention(q, k, v, n_past))) > 1e-2  # the cap matters here


def test_softmax_rows_and_closed_forms():
    rng = np.random.default_rng(9)
    n_s, n_past, hk, g, d = 7, 30, 2, 3, 16
    q = rng.standard_normal((n_s, hk * g, d)) * 2
    k = rng.standard_normal((n_past + n_s, hk, d)) * 2
    v = rng.standard_normal((n_past + n_s, hk, d))
    out, p = O.suffix_attention(q, k, v, n_past, return_probs=True)
    assert np.max(np.abs(p.sum(-1) - 1)) < 1e-12 and (p >= 0).all()
    for i in range(n_s):                                            # causal: no future key
        assert (p[:, i, n_past + i + 1:] == 0).all() and (p[:, i, n_past + i] > 0).all()
    # identical keys -> uniform weights -> mean of the visible values
    kk = np.broadcast_to(k[:1], k.shape).copy()
    o2 = O.suffix_attention(q, kk, v, n_past)
    for i in range(n_s):
        mean = v[:n_past + i + 1].mean(axis=0)                      # [hk][d]
        assert np.allclose(o2[i], np.repeat(mean, g, axis=0), atol=1e-12)
    # a single visible key returns its value exactly
    o3 = O.suffix_attention(q[:1], k, v, 0)
    assert np.allclose(o3[0], np.repeat(v[0], g, axis=0), atol=1e-15)
    # a huge cap is no cap; a saturating cap flattens large same-sign scores
    assert np.max(np.abs(O.suffix_attention(q, k, v, n_past, softcap=1e9) - out)) < 1e-9
    kb = np.abs(k) + 50.0
    qb = np.abs(q) + 50.0
    o4 = O.suffix_attention(qb, kb, v, n_past, softcap=1.0)
    o5 = O.suffix_attention(qb, kk * 0 + 1.0, v, n_past)             # uniform reference
    assert np.max(np.abs(o4 - o5)) < 1e-6


# ---------------------------------------------------------------- the end-to-end equivalence
@pytest.mark.parametrize("v_layout", [O.ROWMAJOR, O.TRANSPOSED])
@pytest.mark.parametrize("softcap", [0.0, 4.0])
def test_full_prefill_equals_splice_plus_redecode(v_layout, softcap):
    """R = 100% is numerically a full prefill (Sec. III-C, Table tab:perf).

    Pre-RoPE K/V are position independent, so (A) rotating every token's key at its final
    position and attending over the whole sequence equals (B) compiling the block at m0,
    re-anchoring it to the splice position, splicing it into a shuffled paged cache and
    re-decoding the trailing suffix, for the suffix rows.
    """
    rng = np.random.default_rng(10)
    L, hk, g, d, P, base = 2, 2, 3, 16, 16, 1e4
    n_ctx, T, n_user, m0, n_red = 45, 40, 6, 7, 17
    n = n_ctx + T + n_user
    npg = -(-n // P) + 2
    k_pre = rng.standard_normal((L, n, hk, d))
    v_all = rng.standard_normal((L, n, hk, d))
    q_pre = rng.standard_normal((L, n, hk * g, d))
    pos = np.arange(n)
    perm = rng.permutation(npg).astype(np.int32)
    n_s = n_red + n_user
    first_q = n - n_s
    for layer in range(L):
        k_final = O.rope(k_pre[layer], pos, base)
        q_final = O.rope(q_pre[layer], pos, base)
        # (A) full causal prefill over the logical sequence
        full = O.suffix_attention(q_final, k_final, v_all[layer], 0, softcap=softcap)
        # (B) splice + re-anchor + redecode through the paged cache
        ck = np.zeros((1, npg, hk, P, d))
        cv = np.zeros((1, hk, d, npg * P)) if v_layout == O.TRANSPOSED else np.zeros_like(ck)
        ctx_k, ctx_v = k_final[None, :n_ctx], v_all[layer][None, :n_ctx]
        ck, cv = O.splice_paged(ck, cv, perm, ctx_k, ctx_v, 0, P, v_layout)
        blk_k = O.rope(k_pre[layer, n_ctx:n_ctx + T], m0 + np.arange(T), base)[None]
        ck, cv = O.splice_paged(ck, cv, perm, blk_k, v_all[layer][None, n_ctx:n_ctx + T],
                                n_ctx, P, v_layout)
        ck = O.rephase_paged(ck, perm, P, n_ctx, T, m0, n_ctx, base)
        ck, cv = O.splice_paged(ck, cv, perm, k_final[None, n_ctx + T:],
                                v_all[layer][None, n_ctx + T:], n_ctx + T, P, v_layout)
        lk, lv = O.gather_logical(ck, cv, perm, n, P, v_layout)
        red = O.suffix_attention(q_final[first_q:], lk[0], lv[0], first_q, softcap=softcap)
        assert np.max(np.abs(red - full[first_q:])) < 1e-10
        # the bare splice (no re-anchor) differs: the drift is real
        ck2 = np.zeros((1, npg, hk, P, d))
        ck2, _ = O.splice_paged(ck2, cv, perm, ctx_k, ctx_v, 0, P, v_layout)
        ck2, _ = O.splice_paged(ck2, cv, perm, blk_k, v_all[layer][None, n_ctx:n_ctx + T],
                                n_ctx, P, v_layout)
        ck2, _ = O.splice_paged(ck2, cv, perm, k_final[None, n_ctx + T:],
                                v_all[layer][None, n_ctx + T:], n_ctx + T, P, v_layout)
        lk2, _ = O.gather_logical(ck2, cv, perm, n, P, v_layout)
        bare = O.suffix_attention(q_final[first_q:], lk2[0], lv[0], first_q, softcap=softcap)
        assert np.max(np.abs(bare - full[first_q:])) > 1e-3


def test_layout_and_page_table_invariance():
    rng = np.random.default_rng(11)
    L, hk, d, P, npg, n = 1, 2, 8, 16, 6, 90
    k = _rand_bits(rng, (L, n, hk, d))
    v = _rand_bits(rng, (L, n, hk, d))
    res = []
    for v_layout in (O.ROWMAJOR, O.TRANSPOSED):
        for perm in (np.arange(npg, dtype=np.int32), rng.permutation(npg).astype(np.int32)):
            ck = np.zeros((L, npg, hk, P, d), np.uint16)
            cv = np.zeros((L, hk, d, npg * P), np.uint16) if v_layout == O.TRANSPOSED else ck.copy()
            ck, cv = O.splice_paged(ck, cv, perm, k, v, 0, P, v_layout)
            lk, lv = O.gather_logical(ck, cv, perm, n, P, v_layout)
            q = O.bf16_bits_to_f64(_rand_bits(np.random.default_rng(0), (10, 4, d)))
            res.append(O.suffix_attention(q, O.bf16_bits_to_f64(lk[0]), O.bf16_bits_to_f64(lv[0]), n - 10))
    for r in res[1:]:
        assert np.array_equal(r, res[0])


def test_rephase_paged_bits_rounds_only_the_range():
    """Bit-level re-anchor: the range equals the rounded fp64 rotation; all else keeps its bits."""
    rng = np.random.default_rng(12)
    L, npg, H, P, D = 2, 5, 2, 16, 32
    ck = np.full((L, npg, H, P, D), 0x7FC1, np.uint16)                # NaN sentinel
    perm = rng.permutation(npg).astype(np.int32)
    blk = O.f64_to_bf16_bits(rng.standard_normal((L, 30, H, D)))
    ck, _ = O.splice_paged(ck, ck.copy(), perm, blk, blk, 21, P)
    out = O.rephase_paged_bits(ck, "bf16", perm, P, 21, 30, 0, 999, 1e4)
    lk, _ = O.gather_logical(out, out, perm, npg * P, P)
    ref = O.f64_to_bf16_bits(O.rephase(O.bf16_bits_to_f64(blk), 0, 999, 1e4))
    assert np.array_equal(lk[:, 21:51], ref)
    l0, _ = O.gather_logical(ck, ck, perm, npg * P, P)
    assert np.array_equal(lk[:, :21], l0[:, :21]) and np.array_equal(lk[:, 51:], l0[:, 51:])
    assert np.array_equal(O.rephase_paged_bits(ck, "bf16", perm, P, 21, 30, 5, 5, 1e4), ck)


# ---------------------------------------------------------------- decode step (one query per sequence)
def _paged_values(rng, lens, hk, d, v_layout, shuffled=True, spare=2):
    """A paged value cache holding every sequence's tokens on private pages, NaN elsewhere, plus
    each sequence's logical K/V."""
    P = 16
    npg = [-(-n // P) for n in lens]
    n_phys = sum(npg) + spare
    order = rng.permutation(n_phys) if shuffled else np.arange(n_phys)
    maps = np.full((len(lens), max(1, max(npg))), -1, np.int64)
    ck = np.full((n_phys, hk, P, d), np.nan)
    cv = np.full((n_phys, hk, P, d), np.nan)
    logical = []
    nxt = 0
    for b, n in enumerate(lens):
        k = rng.standard_normal((n, hk, d))
        v = rng.standard_normal((n, hk, d))
        logical.append((k, v))
        for p in range(npg[b]):
            maps[b, p] = order[nxt]
            nxt += 1
        for t in range(n):
            ck[maps[b, t // P], :, t % P] = k[t]
            cv[maps[b, t // P], :, t % P] = v[t]
    if v_layout == O.TRANSPOSED:
        cv = np.ascontiguousarray(cv.transpose(1, 3, 0, 2).reshape(hk, d, n_phys * P))
    return ck, cv, maps, logical


@pytest.mark.parametrize("v_layout", [O.ROWMAJOR, O.TRANSPOSED])
def test_decode_matches_torch_sdpa_per_sequence(v_layout):
    """Each sequence's step equals torch SDPA (fp64, no mask) over its own logical keys, whatever
    page the keys sit on; NaN in every slot the query must not see changes nothing."""
    rng = np.random.default_rng(31)
    lens, hk, g, d = (1, 15, 16, 17, 40, 0), 2, 3, 16
    ck, cv, maps, logical = _paged_values(rng, lens, hk, d, v_layout)
    q = rng.standard_normal((len(lens), hk * g, d))
    got = O.decode_attention(q, ck, cv, maps, lens, 16, v_layout)
    for b, n in enumerate(lens):
        if n == 0:
            assert np.array_equal(got[b], np.zeros_like(got[b]))
            continue
        k, v = logical[b]
        qt = torch.tensor(q[b])[:, None, :]                                   # [Hq][1][D]
        kt = torch.tensor(k).permute(1, 0, 2).repeat_interleave(g, 0)         # [Hq][n][D]
        vt = torch.tensor(v).permute(1, 0, 2).repeat_interleave(g, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)[:, 0, :].numpy()
        assert np.max(np.abs(got[b] - ref)) < 1e-12, b


def test_decode_single_key_and_constant_values():
    """Closed forms: with one cached token the output is that token's value row; when every value
    row of a KV head is the same vector c, the output is c whatever the scores."""
    rng = np.random.default_rng(32)
    hk, g, d = 2, 2, 8
    ck, cv, maps, logical = _paged_values(rng, (1, 37), hk, d, O.ROWMAJOR)
    q = rng.standard_normal((2, hk * g, d))
    got = O.decode_attention(q, ck, cv, maps, (1, 37), 16)
    v0 = logical[0][1][0]                                                      # [hk][d]
    assert np.allclose(got[0], np.repeat(v0, g, axis=0), atol=1e-15)
    c = rng.standard_normal((hk, d))
    cv2 = np.where(np.isnan(cv), np.nan, 0.0) + c[None, :, None, :]
    got2 = O.decode_attention(q, ck, cv2, maps, (1, 37), 16, softcap=5.0)
    assert np.allclose(got2[1], np.repeat(c, g, axis=0), atol=1e-13)


def test_decode_shared_pages_and_softcap_limit():
    """Two sequences whose tokens are equal give equal outputs whether they share physical pages
    or not; a soft-cap far above every score changes the output by less than its O(s^3/cap^2)
    bound, and a small cap flattens the distribution toward the mean value row."""
    rng = np.random.default_rng(33)
    hk, g, d, P = 1, 4, 16, 16
    n = 50
    k = rng.standard_normal((n, hk, d))
    v = rng.standard_normal((n, hk, d))
    ck = np.full((9, hk, P, d), np.nan)
    cv = np.full((9, hk, P, d), np.nan)
    maps = np.array([[0, 1, 2, 3], [0, 1, 5, 6]])                               # shared 32-token prefix
    for t in range(n):
        for b in range(2):
            ck[maps[b, t // P], :, t % P] = k[t]
            cv[maps[b, t // P], :, t % P] = v[t]
    q1 = rng.standard_normal((1, hk * g, d))
    q = np.concatenate([q1, q1])
    got = O.decode_attention(q, ck, cv, maps, (n, n), P)
    assert np.array_equal(got[0], got[1])
    big = O.decode_attention(q, ck, cv, maps, (n, n), P, softcap=1e6)
    assert np.max(np.abs(big - got)) < 1e-9
    flat = O.decode_attention(q, ck, cv, maps, (n, n), P, softcap=1e-9)
    assert np.allclose(flat[0], np.repeat(v.mean(axis=0), g, axis=0), atol=1e-6)


# ---------------------------------------------------------------- warm-prefix reuse (Sec. VI-D)
@settings(max_examples=60, deadline=None)
@given(st.lists(st.lists(st.integers(0, 3), max_size=12), max_size=6),
       st.lists(st.integers(0, 3), max_size=12))
def test_longest_prefix_matches_commonprefix(slots, tokens):
    """Library routine: os.path.commonprefix over lists gives each slot's common prefix."""
    got = O.longest_prefix(tokens, slots)
    lens = [len(os.path.commonprefix([s, tokens])) for s in slots]
    best = max(lens, default=0)
    if best == 0:
        assert got == (-1, 0)
    else:
        assert got == (lens.index(best), best)


@pytest.mark.parametrize("v_layout", [O.ROWMAJOR, O.TRANSPOSED])
def test_copy_and_share_move_exactly_the_range(v_layout):
    """Copy: the destination's logical range reads back as the source's, every other bit
    unchanged, and a page both maps share is left alone.  Share: whole pages are aliased, the
    partial page is the destination's own and holds the source's slots, its later slots keep
    their bits."""
    rng = np.random.default_rng(41)
    L, npg, H, P, D = 2, 12, 2, 16, 8
    ck = rng.integers(0, 1 << 16, (L, npg, H, P, D), dtype=np.uint16)
    cv = (rng.integers(0, 1 << 16, (L, H, D, npg * P), dtype=np.uint16) if v_layout == O.TRANSPOSED
          else rng.integers(0, 1 << 16, (L, npg, H, P, D), dtype=np.uint16))
    src = np.array([3, 7, 1, 9, 4])
    dst = np.array([3, 2, 8, 0, 11])                         # logical page 0 is shared
    t0, n = 5, 60
    nk, nv = O.copy_tokens(ck, cv, src, dst, t0, n, P, v_layout)
    sk, sv = O.gather_logical(ck, cv, src, 5 * P, P, v_layout)
    dk, dv = O.gather_logical(nk, nv, dst, 5 * P, P, v_layout)
    assert np.array_equal(dk[:, t0:t0 + n], sk[:, t0:t0 + n])
    assert np.array_equal(dv[:, t0:t0 + n], sv[:, t0:t0 + n])
    ok, ov = O.gather_logical(ck, cv, dst, 5 * P, P, v_layout)
    for a, b in ((dk, ok), (dv, ov)):
        assert np.array_equal(a[:, t0 + n:], b[:, t0 + n:])
        assert np.array_equal(a[:, P:t0], b[:, P:t0]) if t0 > P else True
    untouched = np.setdiff1d(np.arange(npg), dst[1:])
    assert np.array_equal(nk[:, untouched], ck[:, untouched])
    # share 37 tokens: pages 0, 1 aliased, page 2 (physical 8) gets slots 0..4
    sk2, sv2, m2 = O.share_prefix(ck, cv, src, dst, 37, P, v_layout)
    assert list(m2) == [3, 7, 8, 0, 11]
    a_k, a_v = O.gather_logical(sk2, sv2, m2, 5 * P, P, v_layout)
    assert np.array_equal(a_k[:, :37], sk[:, :37]) and np.array_equal(a_v[:, :37], sv[:, :37])
    b_k, b_v = O.gather_logical(ck, cv, dst, 5 * P, P, v_layout)
    assert np.array_equal(a_k[:, 37:48], b_k[:, 37:48]) and np.array_equal(a_v[:, 37:48], b_v[:, 37:48])


# ---------------------------------------------------------------- SLB scan and gate (Sec. V-A)
def test_slb_quantize_bounds_and_extremes():
    """Codes lie in [-127, 127]; each row's largest magnitude maps to +-127; dequantised values
    are within half a step (plus fp32 rounding) of the input; a zero row stays zero."""
    rng = np.random.default_rng(51)
    x = rng.standard_normal((20, 96)).astype(np.float32) * rng.uniform(0.01, 10, (20, 1)).astype(np.float32)
    x[3] = 0
    q, s = O.slb_quantize(x)
    assert q.dtype == np.int8 and np.abs(q.astype(int)).max() <= 127
    for r in range(20):
        if r == 3:
            assert s[r] == 0 and not q[r].any()
            continue
        j = int(np.argmax(np.abs(x[r])))
        assert abs(int(q[r, j])) == 127 and np.sign(q[r, j]) == np.sign(x[r, j])
        err = np.abs(q[r].astype(np.float64) * s[r] - x[r])
        assert err.max() <= 0.5 * s[r] * (1 + 1e-5) + 1e-7


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 9), st.integers(1, 4), st.integers(1, 8), st.integers(0, 10**6))
def test_slb_scan_matches_brute_force(n_tools, n_q, k, seed):
    """Brute force on tiny inputs: every (query, tool) score from its definition, ranked by
    (-score, index) with Python's sort; duplicate tools exercise the tie order."""
    rng = np.random.default_rng(seed)
    dim = 8
    tq = rng.integers(-127, 128, (n_tools, dim)).astype(np.int8)
    if n_tools > 2:
        tq[2] = tq[0]                                       # a tie: tool 0 must rank first
    ts = rng.uniform(0.001, 0.02, n_tools).astype(np.float32)
    if n_tools > 2:
        ts[2] = ts[0]
    qq = rng.integers(-127, 128, (n_q, dim)).astype(np.int8)
    qs = rng.uniform(0.001, 0.02, n_q).astype(np.float32)
    tau = np.float32(rng.uniform(0, 0.05))
    idx, top, margin, route = O.slb_scan(tq, ts, qq, qs, k, float(tau))
    for q in range(n_q):
        sc = []
        for t in range(n_tools):
            d = sum(int(qq[q, e]) * int(tq[t, e]) for e in range(dim))
            sc.append(np.float32(np.float32(np.float32(d) * ts[t]) * qs[q]))
        order = sorted(range(n_tools), key=lambda t: (-sc[t], t))
        want = order[:k] + [-1] * (k - min(k, n_tools))
        assert list(idx[q]) == want
        if n_tools >= 2:
            assert margin[q] == np.float32(sc[order[0]] - sc[order[1]])
            assert route[q] == int(margin[q] > tau)
        else:
            assert np.isinf(margin[q]) and route[q] == 1


def test_slb_scan_is_cosine_ranking_on_unit_vectors():
    """On unit-norm vectors the INT8 score approximates the cosine similarity: the best tool is
    the fp64 cosine argmax when that argmax leads by more than the quantisation error."""
    rng = np.random.default_rng(52)
    t = rng.standard_normal((300, 768))
    t /= np.linalg.norm(t, axis=1, keepdims=True)
    q = t[[5, 77, 123]] + 0.2 * rng.standard_normal((3, 768)) / np.sqrt(768)
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    tq, ts = O.slb_quantize(t.astype(np.float32))
    qq, qs = O.slb_quantize(q.astype(np.float32))
    idx, top, margin, route = O.slb_scan(tq, ts, qq, qs, 2, 0.0136)
    cos = q @ t.T
    assert list(idx[:, 0]) == [5, 77, 123]
    assert np.allclose(top[:, 0], cos[np.arange(3), [5, 77, 123]], atol=2e-3)
    assert route.all()
