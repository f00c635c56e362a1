"""Plain fp64 CPU oracle for the KV-block splice path of *Nexus* (arXiv 2608.20397).

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct definition that the
GPU library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  The product library and its Python
binding never import, call or link it, and it imports nothing from them: the two sides share
only the seeded input generators in ``synth/``.

What it computes (paper sections cited per function):

* RoPE and its frequencies (Sec. III-B, the feature-pair rotation with theta_i = b^(-2i/d)).
* Re-anchoring a compiled key block from its compile anchor m0 to the splice position: the
  rotation by (n_past - m0) * theta_i that exactly undoes the phase drift of eq. (drift).
* Splicing a block's K/V rows into a paged KV cache at a logical cursor (Sec. VI-A), with a
  row-major or a transposed, token-innermost V cache (Sec. VI-B).
* Causal grouped-query scaled dot-product attention softmax(QK^T/sqrt(d))V (Sec. III-A) for the
  re-decoded suffix, with optional Gemma-2-style tanh logit soft-capping (Sec. VI-B names the
  soft-capped model family).  Full rows, two-pass softmax.
* The decode step that follows: one query per sequence over that sequence's own page map.
* The Semantic Lookaside Buffer scan (Sec. V-A): INT8 quantisation, integer dot products, the
  best tools per query and the top-two margin gate.
* Warm-prefix reuse (Sec. VI-D): exact-token longest-common-prefix match over arena slots, and
  copying or sharing a prefix's K/V between two page maps.
* The depth-adaptive recompute fraction R(n_past) of eq. (adaptive) and the redecode length
  ceil(S * R / 100) of Sec. VI-A, in exact rational arithmetic.
* Round-to-nearest-even from fp64 to bfloat16, used to round re-phased keys back to the
  storage type.

Every function here is pinned by a ``-m "not gpu"`` test against something other than itself
(values the paper prints, library routines, closed forms or invariants); see
``tests/test_oracle_pins.py``.  Parity is not pinned for the paper's D_KL / top-1 fidelity
numbers (they need model weights), which this oracle does not compute.
"""

from __future__ import annotations

import math
from fractions import Fraction

import numpy as np

NEOX = "neox"                # pair (i, i + d/2): the rotate-half convention of Qwen2 / Gemma-2
INTERLEAVED = "interleaved"  # pair (2i, 2i + 1)
ROWMAJOR = "rowmajor"        # V cache laid out like K: [L][phys_page][H_kv][P][D]
TRANSPOSED = "transposed"    # V cache token-innermost: [L][H_kv][D][phys_page * P + slot]


# --------------------------------------------------------------------------------------
# RoPE (Sec. III-B)
# --------------------------------------------------------------------------------------
def rope_frequencies(head_dim: int, base: float) -> np.ndarray:
    """theta_i = b^(-2i/d) for i = 0 .. d/2 - 1, in fp64 (Sec. III-B)."""
    if head_dim % 2:
        raise ValueError("head_dim must be even")
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * i / head_dim)


def _pairs(head_dim: int, style: str):
    half = head_dim // 2
    if style == NEOX:
        a = np.arange(half)
        return a, a + half
    if style == INTERLEAVED:
        a = 2 * np.arange(half)
        return a, a + 1
    raise ValueError(f"unknown rope style {style!r}")


def rotate_pairs(x: np.ndarray, angles: np.ndarray, style: str = NEOX) -> np.ndarray:
    """Rotate every feature pair (x_a, x_b) of the last axis by its angle.

    ``angles`` has shape ``x.shape[:-1] + (d/2,)`` or broadcasts to it.  The rotated pair is
    (x_a cos a - x_b sin a, x_a sin a + x_b cos a), the 2-D rotation RoPE applies (Sec. III-B).
    """
    x = np.asarray(x, dtype=np.float64)
    a_idx, b_idx = _pairs(x.shape[-1], style)
    xa = x[..., a_idx]
    xb = x[..., b_idx]
    c = np.cos(angles)
    s = np.sin(angles)
    out = np.empty(x.shape, dtype=np.float64)
    out[..., a_idx] = xa * c - xb * s
    out[..., b_idx] = xa * s + xb * c
    return out


def rope(x: np.ndarray, positions, base: float, style: str = NEOX) -> np.ndarray:
    """Apply RoPE to ``x`` of shape [T, ..., D] with one absolute position per row T.

    Pair i of the token at position p is rotated by p * theta_i (Sec. III-B).
    """
    x = np.asarray(x, dtype=np.float64)
    pos = np.asarray(positions, dtype=np.float64).reshape(-1)
    if pos.shape[0] != x.shape[0]:
        raise ValueError("one position per leading row")
    theta = rope_frequencies(x.shape[-1], base)
    ang = pos[:, None] * theta[None, :]                       # [T, D/2]
    ang = ang.reshape((x.shape[0],) + (1,) * (x.ndim - 2) + (theta.shape[0],))
    return rotate_pairs(x, ang, style)


def rephase(k: np.ndarray, src_pos: int, dst_pos: int, base: float,
            style: str = NEOX) -> np.ndarray:
    """Re-anchor keys compiled at anchor ``src_pos`` (m0) to the splice position ``dst_pos``.

    Eq. (drift) gives the phase a key compiled at m0 lacks when read at n_past:
    (n_past - m0) * theta_i.  Re-anchoring rotates every key pair of the block by exactly that
    angle (Sec. III-B), so every token of the block, whatever its index j, turns by the same
    (dst - src) * theta_i.  ``k`` has any shape [..., D]; V is never rotated.
    """
    k = np.asarray(k, dtype=np.float64)
    theta = rope_frequencies(k.shape[-1], base)
    delta = np.float64(int(dst_pos) - int(src_pos))
    return rotate_pairs(k, delta * theta, style)


# --------------------------------------------------------------------------------------
# bfloat16 storage rounding
# --------------------------------------------------------------------------------------
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (uint16) as fp64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to bfloat16 (8 significant bits) to nearest, ties to even.

    One rounding straight from the fp64 value: the value is scaled by a power of two so that
    the bfloat16 spacing of its binade becomes 1, rounded with ``np.rint`` (ties-to-even) and
    scaled back.  The spacing is 2^(e-8) for x = m * 2^e, 0.5 <= |m| < 1, and never below the
    subnormal spacing 2^-133.  Results beyond the largest finite bfloat16 become infinity.
    """
    x = np.asarray(x, dtype=np.float64)
    finite = np.isfinite(x)
    xf = np.where(finite, x, 0.0)
    _, e = np.frexp(xf)
    sp = np.maximum(e - 8, -133)
    q = np.rint(np.ldexp(xf, -sp))
    y = np.ldexp(q, sp)
    with np.errstate(over="ignore"):
        y32 = np.where(finite, y, x).astype(np.float32)
    return (y32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Raw storage bits of fp64 values: bf16 -> uint16 (RNE), f32 -> uint32 (RNE)."""
    if dtype == "bf16":
        return f64_to_bf16_bits(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32)
    raise ValueError(dtype)


def storage_to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of raw storage bits."""
    if dtype == "bf16":
        return bf16_bits_to_f64(bits)
    if dtype == "f32":
        return np.asarray(bits, dtype=np.uint32).view(np.float32).astype(np.float64)
    raise ValueError(dtype)


# --------------------------------------------------------------------------------------
# Paged KV cache: splice and logical view (Sec. VI-A, Sec. VI-B, Fig. atb)
# --------------------------------------------------------------------------------------
def splice_paged(cache_k: np.ndarray, cache_v: np.ndarray, page_map: np.ndarray,
                 block_k: np.ndarray, block_v: np.ndarray, offset: int, page_size: int,
                 v_layout: str = ROWMAJOR):
    """Write a block's K/V rows into the live cache at logical cursor ``offset``.

    Sec. VI-A: the splice writes the block's K/V rows into the live KV cells at the runtime
    cursor.  Here the live cache is paged: logical token t lives in physical page
    ``page_map[t // P]`` at slot ``t % P``.

    * ``cache_k``: [L][n_phys_pages][H_kv][P][D] raw bits (uint16 for bf16, uint32 for f32).
    * ``cache_v``: same as ``cache_k`` for a row-major V cache; for the transposed cache
      (Sec. VI-B, token-innermost) [L][H_kv][D][n_phys_pages * P], where token t is column
      ``page_map[t // P] * P + t % P``.
    * ``block_k`` / ``block_v``: [L][T][H_kv][D] raw bits, token-major.

    Pure data movement: returns new arrays in which block token j occupies logical slot
    ``offset + j`` and every other element keeps its bits.
    """
    ck = np.array(cache_k, copy=True)
    cv = np.array(cache_v, copy=True)
    n_tokens = block_k.shape[1]
    for j in range(n_tokens):
        t = offset + j
        page = int(page_map[t // page_size])
        slot = t % page_size
        ck[:, page, :, slot, :] = block_k[:, j, :, :]
        if v_layout == ROWMAJOR:
            cv[:, page, :, slot, :] = block_v[:, j, :, :]
        elif v_layout == TRANSPOSED:
            cv[:, :, :, page * page_size + slot] = block_v[:, j, :, :]
        else:
            raise ValueError(v_layout)
    return ck, cv


def gather_logical(cache_k: np.ndarray, cache_v: np.ndarray, page_map: np.ndarray,
                   n_tokens: int, page_size: int, v_layout: str = ROWMAJOR):
    """Logical [L][N][H_kv][D] views of the first ``n_tokens`` tokens of a paged cache.

    The inverse addressing of ``splice_paged``: logical token t is read from page
    ``page_map[t // P]``, slot ``t % P`` (or column ``page * P + slot`` of a transposed V).
    """
    ks, vs = [], []
    for t in range(n_tokens):
        page = int(page_map[t // page_size])
        slot = t % page_size
        ks.append(cache_k[:, page, :, slot, :])
        if v_layout == ROWMAJOR:
            vs.append(cache_v[:, page, :, slot, :])
        elif v_layout == TRANSPOSED:
            vs.append(cache_v[:, :, :, page * page_size + slot])
        else:
            raise ValueError(v_layout)
    return np.stack(ks, axis=1), np.stack(vs, axis=1)


def rephase_paged(cache_k_values: np.ndarray, page_map: np.ndarray, page_size: int,
                  offset: int, n_tokens: int, src_pos: int, dst_pos: int, base: float,
                  style: str = NEOX) -> np.ndarray:
    """Re-anchor, in the page view, the keys of logical tokens [offset, offset + n_tokens).

    ``cache_k_values`` is the fp64 value of a [L][n_phys_pages][H_kv][P][D] key cache.  Each
    key in the range is rotated by (dst_pos - src_pos) * theta_i (``rephase``); every other key
    is returned unchanged.  Splicing the raw block and then re-anchoring it in place is the same
    as re-anchoring the block first, since the splice only moves rows.
    """
    out = np.array(cache_k_values, dtype=np.float64, copy=True)
    for t in range(offset, offset + n_tokens):
        page = int(page_map[t // page_size])
        slot = t % page_size
        out[:, page, :, slot, :] = rephase(out[:, page, :, slot, :], src_pos, dst_pos, base, style)
    return out


def rephase_paged_bits(cache_k_bits: np.ndarray, dtype: str, page_map: np.ndarray,
                       page_size: int, offset: int, n_tokens: int, src_pos: int, dst_pos: int,
                       base: float, style: str = NEOX) -> np.ndarray:
    """``rephase_paged`` on raw storage bits: each re-anchored key row is rounded to nearest-even
    back into the storage type (the stored block is F16/bf16, Sec. VI-A); every other bit of the
    cache is returned unchanged."""
    out = np.array(cache_k_bits, copy=True)
    for t in range(offset, offset + n_tokens):
        page = int(page_map[t // page_size])
        slot = t % page_size
        rows = storage_to_f64(out[:, page, :, slot, :], dtype)
        out[:, page, :, slot, :] = round_to_storage(
            rephase(rows, src_pos, dst_pos, base, style), dtype)
    return out


# --------------------------------------------------------------------------------------
# Suffix-redecode attention (Sec. III-A; soft-cap per Sec. VI-B's soft-capped family)
# --------------------------------------------------------------------------------------
def suffix_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_past: int,
                     scale: float | None = None, softcap: float = 0.0,
                     return_probs: bool = False):
    """Causal grouped-query attention of the re-decoded suffix over the spliced cache.

    * ``q``: [n_s][H_q][D], query i sits at absolute position n_past + i (already rotated).
    * ``k``, ``v``: logical [N][H_kv][D] with N >= n_past + n_s.
    * Query head h reads KV head h // G with G = H_q / H_kv (contiguous groups).
    * Score s_t = scale * <q_i, k_t> with scale = 1/sqrt(D) unless given (Sec. III-A); if
      softcap > 0 the score becomes softcap * tanh(s_t / softcap) (scale first, then cap).
    * Query i sees keys t <= n_past + i (inclusive causal boundary).
    * Two-pass softmax over the full visible row, then o_i = sum_t p_t v_t.

    Returns [n_s][H_q][D] fp64 (and the [H_q][n_s][N] probabilities if ``return_probs``).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n_s, n_q_heads, d = q.shape
    n_kv_heads = k.shape[1]
    if n_q_heads % n_kv_heads:
        raise ValueError("n_q_heads must be a multiple of n_kv_heads")
    group = n_q_heads // n_kv_heads
    n_keys = n_past + n_s
    if k.shape[0] < n_keys or v.shape[0] < n_keys:
        raise ValueError("cache holds fewer tokens than n_past + n_s")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    visible = np.arange(n_keys)[None, :] <= (n_past + np.arange(n_s))[:, None]   # [n_s][N]
    out = np.zeros((n_s, n_q_heads, d), dtype=np.float64)
    probs = np.zeros((n_q_heads, n_s, n_keys), dtype=np.float64) if return_probs else None
    for h in range(n_q_heads):
        g = h // group
        s = scale * (q[:, h, :] @ k[:n_keys, g, :].T)                 # [n_s][N]
        if softcap > 0.0:
            s = softcap * np.tanh(s / softcap)
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        w = np.exp(s - m)                                            # masked -> exp(-inf) = 0
        p = w / w.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:n_keys, g, :]
        if return_probs:
            probs[h] = p
    return (out, probs) if return_probs else out


def decode_attention(q: np.ndarray, cache_k: np.ndarray, cache_v: np.ndarray,
                     page_maps: np.ndarray, seq_lens, page_size: int,
                     v_layout: str = ROWMAJOR, scale: float | None = None,
                     softcap: float = 0.0) -> np.ndarray:
    """One decode step per sequence over its own pages (Sec. III-A attention, one query).

    * ``q``: [B][H_q][D] values; the query of sequence b sits at position seq_lens[b] - 1.
    * ``cache_k`` / ``cache_v``: ONE layer of a paged cache as values, [n_phys_pages][H_kv][P][D]
      (V transposed: [H_kv][D][n_phys_pages * P]).
    * ``page_maps``: [B][stride], logical page p of sequence b -> physical page.

    The step is the suffix attention of a single query whose keys are the sequence's cached
    tokens 0 .. seq_lens[b] - 1, its own included: gather them through the sequence's map and
    call ``suffix_attention`` with n_past = seq_lens[b] - 1.  A sequence with no cached token
    gets a zero row.  Returns [B][H_q][D] fp64.
    """
    q = np.asarray(q, dtype=np.float64)
    out = np.zeros(q.shape, dtype=np.float64)
    for b, n in enumerate(seq_lens):
        n = int(n)
        if n == 0:
            continue
        k, v = gather_logical(cache_k[None], cache_v[None], page_maps[b], n, page_size, v_layout)
        out[b] = suffix_attention(q[b:b + 1], k[0], v[0], n - 1, scale, softcap)[0]
    return out


# --------------------------------------------------------------------------------------
# Warm-prefix reuse (Sec. VI-D): exact-token prefix match and KV copy / share on pages
# --------------------------------------------------------------------------------------
def longest_prefix(tokens, slots):
    """(slot, length): the slot whose token list shares the longest common prefix with
    ``tokens``, lowest index among equals; (-1, 0) when none shares a first token."""
    best, best_len = -1, 0
    for s, toks in enumerate(slots):
        n = 0
        while n < min(len(toks), len(tokens)) and toks[n] == tokens[n]:
            n += 1
        if n > best_len:
            best, best_len = s, n
    return best, best_len


def copy_tokens(cache_k: np.ndarray, cache_v: np.ndarray, src_map, dst_map, t0: int,
                n_tokens: int, page_size: int, v_layout: str = ROWMAJOR):
    """Every layer's K and V of logical tokens [t0, t0 + n_tokens) under ``dst_map`` become
    those under ``src_map``; all other bits are kept.  Raw-bit caches as ``splice_paged``."""
    ck = np.array(cache_k, copy=True)
    cv = np.array(cache_v, copy=True)
    for t in range(t0, t0 + n_tokens):
        ps, pd = int(src_map[t // page_size]), int(dst_map[t // page_size])
        slot = t % page_size
        ck[:, pd, :, slot, :] = cache_k[:, ps, :, slot, :]
        if v_layout == ROWMAJOR:
            cv[:, pd, :, slot, :] = cache_v[:, ps, :, slot, :]
        else:
            cv[:, :, :, pd * page_size + slot] = cache_v[:, :, :, ps * page_size + slot]
    return ck, cv


def share_prefix(cache_k: np.ndarray, cache_v: np.ndarray, src_map, dst_map, n_tokens: int,
                 page_size: int, v_layout: str = ROWMAJOR):
    """The destination's first n_tokens tokens become the source's: its whole pages take the
    source's physical pages, its partial last page (kept) receives a copy of the slots.
    Returns (cache_k, cache_v, new dst_map)."""
    n_full = n_tokens // page_size
    new_map = np.array(dst_map, copy=True)
    new_map[:n_full] = np.asarray(src_map)[:n_full]
    ck, cv = copy_tokens(cache_k, cache_v, src_map, new_map, n_full * page_size,
                         n_tokens - n_full * page_size, page_size, v_layout)
    return ck, cv, new_map


# --------------------------------------------------------------------------------------
# Semantic Lookaside Buffer (Sec. V-A): INT8 scan and top-two margin gate
# --------------------------------------------------------------------------------------
def slb_quantize(x: np.ndarray):
    """Symmetric per-row INT8 codes of fp32 rows: scale = max|x| / 127 and code =
    rint(x / scale) (fp32 division, ties to even), within [-127, 127]; a zero row gets scale 0
    and zero codes.  The INT8 tool and query vectors of Sec. V-A (its quantiser is not given;
    this is the reading)."""
    x = np.asarray(x, dtype=np.float32)
    scale = (np.max(np.abs(x), axis=1) / np.float32(127)).astype(np.float32)
    q = np.zeros(x.shape, dtype=np.int8)
    for r in range(x.shape[0]):
        if scale[r] > 0:
            q[r] = np.clip(np.rint(x[r] / scale[r]), -127, 127).astype(np.int8)
    return q, scale


def slb_scan(tools_q: np.ndarray, tool_scale: np.ndarray, queries_q: np.ndarray,
             query_scale: np.ndarray, k: int, tau: float):
    """Scan every tool for every query and gate on the top-two margin (Sec. V-A).

    Score = (float32(dot) * tool_scale) * query_scale, in fp32 with one rounding per product (the
    integer dot is exact).  The k best tools per query, higher score first and the lower index
    first among equal scores (index -1, score -inf past the registry); margin = s1 - s2 in fp32
    (+inf with a single tool); route = margin > tau (auto-route) else escalate to the reranker.
    Returns (top_idx [Q][k], top_score [Q][k], margin [Q], route [Q]).
    """
    dot = np.asarray(queries_q, dtype=np.int64) @ np.asarray(tools_q, dtype=np.int64).T
    score = (dot.astype(np.float32) * np.asarray(tool_scale, np.float32)[None, :]) \
        * np.asarray(query_scale, np.float32)[:, None]
    n_q, n_t = score.shape
    idx = np.full((n_q, k), -1, dtype=np.int32)
    top = np.full((n_q, k), -np.inf, dtype=np.float32)
    margin = np.zeros(n_q, dtype=np.float32)
    route = np.zeros(n_q, dtype=np.int32)
    for q in range(n_q):
        order = sorted(range(n_t), key=lambda t: (-float(score[q, t]), t))
        for j in range(min(k, n_t)):
            idx[q, j] = order[j]
            top[q, j] = score[q, order[j]]
        margin[q] = np.float32(np.inf) if n_t < 2 else \
            np.float32(score[q, order[0]] - score[q, order[1]])
        route[q] = 1 if margin[q] > np.float32(tau) else 0
    return idx, top, margin, route


# --------------------------------------------------------------------------------------
# Depth-adaptive recompute, eq. (adaptive), and the redecode length of Sec. VI-A
# --------------------------------------------------------------------------------------
def recompute_fraction(n_past: int, M: int = 256, r_base: int = 5, K: int = 4) -> Fraction:
    """R(n_past) in percent, as an exact rational (eq. adaptive), clamped to 100.

    R = R_base for n_past <= M; otherwise R_base + (n_past - M) / (M (K - 1)) * (100 - R_base).
    """
    if M <= 0 or K < 2 or not 0 <= r_base <= 100 or n_past < 0:
        raise ValueError("need M > 0, K >= 2, 0 <= r_base <= 100, n_past >= 0")
    if n_past <= M:
        return Fraction(r_base)
    r = Fraction(r_base) + Fraction(n_past - M, M * (K - 1)) * (100 - r_base)
    return min(r, Fraction(100))


def redecode_len(S: int, n_past: int, M: int = 256, r_base: int = 5, K: int = 4) -> int:
    """Number of trailing block tokens re-decoded: ceil(S * R(n_past) / 100) (Sec. VI-A)."""
    if S < 0:
        raise ValueError("S >= 0")
    return math.ceil(Fraction(S) * recompute_fraction(n_past, M, r_base, K) / 100)
