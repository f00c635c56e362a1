"""Seeded synthetic inputs shared by the GPU path's tests/bench and the oracle's tests.

This module holds no arithmetic of the method: it draws Gaussian tensors, casts them to the
storage type with the library's round-to-nearest-even, and produces page tables and offsets.

Recipe:
* Host draws: ``numpy.random.default_rng(SeedSequence([20397, cfg, layer, tag]))`` fp64
  N(0, 1) values times the config's std, cast fp64 -> fp32 -> storage type (bf16 by torch's
  RNE conversion).  Used wherever the oracle checks whole tensors.
* Device draws (large configs only): torch's Philox generator on the GPU seeded with the same
  (cfg, layer, tag) triple, fp32 N(0, 1) times the std, cast to the storage type.  A different
  stream from the host draws; the oracle sees device draws by copying them to the host.
* Q, context K and user K are drawn directly as *rotated* values: a rotation of an isotropic
  Gaussian pair is again an isotropic Gaussian pair, so drawing after RoPE has exactly the
  distribution of rotating a Gaussian draw.  Block K is likewise drawn as the block compiled at
  its anchor.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import PAGE, Workload, workload

SEED = 20397
TAG = dict(q=0, k_ctx=1, v_ctx=2, k_blk=3, v_blk=4, k_user=5, v_user=6, offsets=7, page_perm=8)

SENTINEL = {"bf16": np.uint16(0x7FC1), "f32": np.uint32(0x7FC00001)}
BITS_DTYPE = {"bf16": np.uint16, "f32": np.uint32}


def rng(cfg: int, layer: int, tag: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED, cfg, layer, tag]))


def normal(cfg: int, layer: int, tag: int, shape, std: float = 1.0) -> np.ndarray:
    """fp64 N(0, std^2) draws for one (config, layer, tag)."""
    return rng(cfg, layer, tag).standard_normal(shape) * std


def to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Cast fp64 draws to the storage type; returns raw bits (uint16 for bf16, uint32 for f32)."""
    x32 = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    if dtype == "f32":
        return x32.view(np.uint32)
    if dtype == "bf16":
        import torch
        t = torch.from_numpy(x32).to(torch.bfloat16)
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    raise ValueError(dtype)


def bits_to_torch(bits: np.ndarray, dtype: str, device="cpu"):
    """Wrap raw storage bits as a torch tensor of the storage type (no value change)."""
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.float32)).to(device)
    raise ValueError(dtype)


def torch_to_bits(t) -> np.ndarray:
    """Raw storage bits of a torch bf16 / f32 tensor, on the host."""
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    if t.dtype == torch.float32:
        return t.numpy().view(np.uint32).copy()
    raise ValueError(t.dtype)


def cfg4_draws() -> np.ndarray:
    """16 distinct draws from range(26625) = 0 .. 32768 - 16*384, the config-4 block offsets."""
    return rng(4, 0, TAG["offsets"]).choice(26625, size=16, replace=False)


def page_map(cfg: int, n_pages: int, shuffled: bool) -> np.ndarray:
    """Logical -> physical page map: identity or a seeded permutation (int32)."""
    if not shuffled:
        return np.arange(n_pages, dtype=np.int32)
    return rng(cfg, 0, TAG["page_perm"]).permutation(n_pages).astype(np.int32)


def get_workload(cfg: int) -> Workload:
    return workload(cfg, cfg4_draws() if cfg == 4 else None)


@dataclass
class HostCase:
    """Raw-bit host inputs of one config (all layers), from host draws.

    ``ctx_*`` cover logical tokens [0, n_ctx); ``blk_*[b]`` is block b compiled at the anchor;
    ``user_*`` cover the n_user tokens right after the (single) block; ``q`` holds every
    block's suffix queries back to back, block-major.
    """
    wl: Workload
    page_map: np.ndarray
    n_ctx: int
    ctx_k: np.ndarray
    ctx_v: np.ndarray
    blk_k: list
    blk_v: list
    user_k: np.ndarray
    user_v: np.ndarray
    q: np.ndarray


def host_case(cfg: int, layers=None) -> HostCase:
    """Draw one config's inputs on the host for the given layers (default: all)."""
    return host_case_wl(get_workload(cfg), cfg, layers)


def host_case_wl(wl: Workload, seed_cfg: int, layers=None) -> HostCase:
    """Draw inputs for any workload record; ``seed_cfg`` takes the config slot of the seed."""
    layers = list(range(wl.n_layers)) if layers is None else list(layers)
    H, D, Hq = wl.n_kv_heads, wl.head_dim, wl.n_q_heads
    n_blocks = len(wl.splice_pos)
    n_ctx = wl.n_tokens if n_blocks > 1 else wl.splice_pos[0]

    def draw(tag, shape, std, tag_offset=0):
        return np.stack([to_bits(normal(seed_cfg, l, tag + tag_offset, shape, std), wl.dtype)
                         for l in layers])

    ctx_k = draw(TAG["k_ctx"], (n_ctx, H, D), wl.k_scale)
    ctx_v = draw(TAG["v_ctx"], (n_ctx, H, D), wl.v_scale)
    # block b uses tags offset by 16*b so that every block is an independent draw
    blk_k = [draw(TAG["k_blk"], (wl.block_len, H, D), wl.k_scale, 16 * b) for b in range(n_blocks)]
    blk_v = [draw(TAG["v_blk"], (wl.block_len, H, D), wl.v_scale, 16 * b) for b in range(n_blocks)]
    user_k = draw(TAG["k_user"], (wl.n_user, H, D), wl.k_scale)
    user_v = draw(TAG["v_user"], (wl.n_user, H, D), wl.v_scale)
    q = draw(TAG["q"], (wl.n_suffix * n_blocks, Hq, D), wl.q_scale)
    pm = page_map(seed_cfg, wl.n_pages, wl.shuffled_pages)
    return HostCase(wl, pm, n_ctx, ctx_k, ctx_v, blk_k, blk_v, user_k, user_v, q)


def empty_cache_bits(wl: Workload, n_layers: int, n_phys_pages: int | None = None):
    """Sentinel-filled raw K and V caches for ``n_layers`` layers.

    K: [L][n_phys_pages][H_kv][P][D]; V: the same, or [L][H_kv][D][n_phys_pages * P] when
    transposed.
    """
    npp = wl.n_pages if n_phys_pages is None else n_phys_pages
    H, D = wl.n_kv_heads, wl.head_dim
    s = SENTINEL[wl.dtype]
    k = np.full((n_layers, npp, H, PAGE, D), s, dtype=BITS_DTYPE[wl.dtype])
    if wl.v_layout == "transposed":
        v = np.full((n_layers, H, D, npp * PAGE), s, dtype=BITS_DTYPE[wl.dtype])
    else:
        v = np.full((n_layers, npp, H, PAGE, D), s, dtype=BITS_DTYPE[wl.dtype])
    return k, v


def device_normal(cfg: int, layer: int, tag: int, shape, std: float, dtype: str, device):
    """Storage-type tensor of N(0, std^2) draws made on ``device`` by torch's generator."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((SEED * 1_000_003 + cfg * 10_007 + layer * 101 + tag) & 0x7FFFFFFFFFFFFFFF)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    x.mul_(std)
    return x.to(torch.bfloat16) if dtype == "bf16" else x
