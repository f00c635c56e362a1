"""The five synthetic workloads of the splice path, as plain shape records.

Shapes follow the Qwen2.5-14B attention geometry (40 query heads, 8 KV heads, head_dim 128,
RoPE base 1e6, 48 layers) and a Gemma-2-style soft-capped geometry (16/8 heads, head_dim 256,
transposed V).  Nothing here computes any part of the method; it only names sizes and
positions.  Every config uses 16-token KV pages and blocks compiled at anchor m0 = 0.

Per block b the path is: splice the block's rows at ``splice_pos`` (logical cursor), re-anchor
its keys from ``anchor`` to ``splice_pos``, write the user-turn tokens after it, and run causal
attention for the ``n_suffix`` trailing queries, which start at ``attn_n_past``.
"""

from __future__ import annotations

from dataclasses import dataclass, field

PAGE = 16


@dataclass(frozen=True)
class Workload:
    cfg: int
    name: str
    dtype: str               # "bf16" or "f32" (storage and attention output)
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_base: float
    n_tokens: int            # logical cache capacity used (context + blocks + user tokens)
    block_len: int           # T, tokens per compiled block
    splice_pos: tuple        # logical cursor of each block (== its new position)
    anchor: int              # compile anchor m0 of every block
    n_user: int              # user-turn tokens written after the (single) block
    n_suffix: int            # queries per block re-decoded
    attn_n_past: tuple       # cache tokens before the first query of each block's suffix
    v_layout: str            # "rowmajor" or "transposed"
    shuffled_pages: bool
    softcap: float
    q_scale: float           # std of the seeded Q, K, V draws
    k_scale: float
    v_scale: float
    extra: dict = field(default_factory=dict)

    @property
    def n_pages(self) -> int:
        return -(-self.n_tokens // PAGE)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


def _cfg4_offsets(seed_draws):
    """Offsets o_b = r_b + 384 b with r the sorted draws: non-overlapping, unaligned blocks."""
    r = sorted(int(x) for x in seed_draws)
    return tuple(r[b] + 384 * b for b in range(16))


def workload(cfg: int, cfg4_draws=None) -> Workload:
    """Return config ``cfg`` (1..5).  Config 4 needs its 16 seeded offset draws."""
    s = 128 ** -0.5
    if cfg == 1:
        return Workload(1, "tiny fp32 bare splice", "f32", 1, 4, 1, 64, 1e4,
                        n_tokens=224, block_len=64, splice_pos=(128,), anchor=0, n_user=32,
                        n_suffix=32, attn_n_past=(192,), v_layout="rowmajor",
                        shuffled_pages=False, softcap=0.0, q_scale=1.0, k_scale=1.0, v_scale=1.0)
    if cfg == 2:
        return Workload(2, "qwen2.5-14b single layer, 2048-deep splice", "bf16", 1, 40, 8, 128,
                        1e6, n_tokens=2624, block_len=512, splice_pos=(2048,), anchor=0,
                        n_user=64, n_suffix=192, attn_n_past=(2432,), v_layout="rowmajor",
                        shuffled_pages=False, softcap=0.0, q_scale=s, k_scale=s, v_scale=s)
    if cfg == 3:
        return Workload(3, "qwen2.5-14b 48 layers, 16384-deep full repair", "bf16", 48, 40, 8,
                        128, 1e6, n_tokens=17472, block_len=1024, splice_pos=(16384,), anchor=0,
                        n_user=64, n_suffix=1088, attn_n_past=(16384,), v_layout="rowmajor",
                        shuffled_pages=False, softcap=0.0, q_scale=s, k_scale=s, v_scale=s)
    if cfg == 4:
        if cfg4_draws is None:
            raise ValueError("config 4 needs its offset draws (synth.gen.cfg4_draws)")
        offs = _cfg4_offsets(cfg4_draws)
        return Workload(4, "qwen2.5-14b single layer, 16 blocks in a shuffled 32k cache", "bf16",
                        1, 40, 8, 128, 1e6, n_tokens=32768, block_len=384, splice_pos=offs,
                        anchor=0, n_user=0, n_suffix=256,
                        attn_n_past=tuple(o + 128 for o in offs), v_layout="rowmajor",
                        shuffled_pages=True, softcap=0.0, q_scale=s, k_scale=s, v_scale=s)
    if cfg == 5:
        return Workload(5, "gemma-2-style soft-capped, transposed V", "bf16", 1, 16, 8, 256, 1e4,
                        n_tokens=9216, block_len=1024, splice_pos=(8192,), anchor=0, n_user=0,
                        n_suffix=512, attn_n_past=(8704,), v_layout="transposed",
                        shuffled_pages=False, softcap=50.0, q_scale=1.0, k_scale=3.0,
                        v_scale=1.0)
    raise ValueError(f"no config {cfg}")
