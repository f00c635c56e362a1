"""ctypes binding of libnexus (include/nexus.h): argument marshalling only.

Every step of the path runs in the library's HIP kernels.  torch provides device memory and the
current stream; this module builds the C descriptors from tensors, calls the C entry points on
``torch.cuda.current_stream()`` and turns a non-zero status into :class:`NexusError`.  If the
shared library has not been built, :func:`lib` raises: there is no fallback.
"""

from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass, field

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnexus.so")

OK, EINVAL, ESHAPE, EDTYPE, EROPE, ERANGE, ELAYOUT, EWORKSPACE, EHIP = range(9)
BF16, F32 = 0, 1
V_ROWMAJOR, V_TRANSPOSED = 0, 1
ROPE_NEOX, ROPE_INTERLEAVED = 0, 1
PAGE = 16


class NexusError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        msg = lib().nexus_status_str(status).decode()
        super().__init__(f"{what}: status {status} ({msg})" if what else f"status {status} ({msg})")


class CBlock(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("n_layers", C.c_int32),
                ("n_tokens", C.c_int32), ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("dtype", C.c_int32), ("rope_style", C.c_int32), ("base_pos", C.c_int64),
                ("rope_base", C.c_double)]


class CKvCache(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("n_layers", C.c_int32),
                ("n_phys_pages", C.c_int32), ("page_size", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("dtype", C.c_int32), ("v_layout", C.c_int32),
                ("rope_style", C.c_int32), ("rope_base", C.c_double)]


class CPageTable(C.Structure):
    _fields_ = [("map", C.c_void_p), ("n_logical_pages", C.c_int32)]


_lib = None


def lib():
    """Load libnexus.so (built by ``paper_2608_20397_amd.build``); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_20397_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, f32, f64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_double, C.c_size_t
    pB, pC, pT = C.POINTER(CBlock), C.POINTER(CKvCache), C.POINTER(CPageTable)
    sigs = {
        "nexus_abi_version": (i32, []),
        "nexus_status_str": (C.c_char_p, [i32]),
        "nexus_redecode_len": (i64, [i64, i64, i32, i32, i32]),
        "nexus_check_page_table": (i32, [C.POINTER(C.c_int32), i32, i32]),
        "nexus_rephase_k": (i32, [pB, i64, i64, f64, vp]),
        "nexus_rephase_k_paged": (i32, [pC, pT, i64, i32, i64, i64, f64, vp]),
        "nexus_splice_pages": (i32, [pC, pT, pB, i64, vp]),
        "nexus_splice_rephase_pages": (i32, [pC, pT, pB, i64, i64, vp]),
        "nexus_rope_append": (i32, [pC, pT, vp, vp, i32, i64, i64, vp]),
        "nexus_suffix_attn": (i32, [vp, i32, i32, pC, pT, i32, i64, f32, i32, f32, vp, vp, sz, vp]),
        "nexus_suffix_attn_workspace": (sz, [i32, i32, pC, i64]),
        "nexus_suffix_attn_noalloc": (i32, [vp, i32, i32, pC, pT, i32, i64, f32, i32, f32, vp,
                                            vp]),
        "nexus_suffix_attn_varlen": (i32, [vp, i32, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                           C.POINTER(C.c_int64), i32, pC, pT, i32, f32, i32, f32,
                                           vp, vp, sz, vp]),
        "nexus_suffix_attn_varlen_workspace": (sz, [i32, C.POINTER(C.c_int32),
                                                    C.POINTER(C.c_int32), C.POINTER(C.c_int64),
                                                    i32, pC]),
        "nexus_decode_attn": (i32, [vp, i32, i32, pC, vp, i32, vp, i32, i32, f32, i32, f32, vp,
                                    vp, sz, vp]),
        "nexus_decode_attn_workspace": (sz, [i32, i32, pC, i32]),
        "nexus_kv_copy_tokens": (i32, [pC, vp, vp, i32, i64, i32, vp]),
        "nexus_kv_share_prefix": (i32, [pC, vp, vp, i32, i32, vp]),
        "nexus_l0_longest_prefix": (i32, [C.POINTER(C.c_int32), i32, C.POINTER(C.c_int32),
                                          C.POINTER(C.c_int32), i32, i32,
                                          C.POINTER(C.c_int32), C.POINTER(C.c_int32)]),
        "nexus_slb_quantize": (i32, [vp, i32, i32, vp, vp, vp]),
        "nexus_slb_scan": (i32, [vp, vp, i32, vp, vp, i32, i32, i32, f32, vp, vp, vp, vp, vp, sz,
                                 vp]),
        "nexus_slb_scan_workspace": (sz, [i32, i32, i32, i32]),
        "nexus_calib_copy": (i32, [vp, vp, sz, vp]),
        "nexus_calib_mfma_bf16": (i32, [i32, vp, C.POINTER(C.c_double), vp]),
        "nexus_calib_lds_dma": (i32, [vp, sz, vp]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int, what: str):
    if status != OK:
        raise NexusError(status, what)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise NexusError(EDTYPE, f"unsupported dtype {t.dtype}")


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


def _on_device(*named):
    """Every given (name, tensor) pair must be a device tensor, all on one device; returns that
    device.  The kernels dereference every pointer they get as a device address, so a host
    tensor must never reach them."""
    dev = None
    for name, t in named:
        if t is None:
            continue
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise NexusError(EINVAL, f"{name} must be a device tensor")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise NexusError(EINVAL, f"{name} is on {t.device}, the other operands on {dev}")
    return dev


@dataclass
class Block:
    """A compiled KV block in HBM: k, v [n_layers][n_tokens][n_kv_heads][head_dim]."""
    k: torch.Tensor
    v: torch.Tensor
    base_pos: int
    rope_base: float
    rope_style: int = ROPE_NEOX

    def c(self) -> CBlock:
        L, T, H, D = self.k.shape
        if tuple(self.v.shape) != (L, T, H, D) or not (self.k.is_contiguous() and self.v.is_contiguous()):
            raise NexusError(ESHAPE, "block k/v must be contiguous [L][T][H][D] of equal shape")
        _on_device(("block k", self.k), ("block v", self.v))
        return CBlock(self.k.data_ptr(), self.v.data_ptr(), L, T, H, D, _dtype_code(self.k),
                      self.rope_style, self.base_pos, self.rope_base)


@dataclass
class PagedKVCache:
    """k [L][n_phys_pages][H][16][D]; v the same or, transposed, [L][H][D][n_phys_pages*16];
    page_map int32 [n_logical_pages] on the device.

    The kernels read the page map's entries on the device without a host check, so the map is
    validated here (``nexus_check_page_table`` on a host copy: every entry a distinct physical
    page) the first time a call uses it and again whenever it has changed since (another tensor,
    or an in-place write that bumped its version counter)."""
    k: torch.Tensor
    v: torch.Tensor
    page_map: torch.Tensor
    rope_base: float
    v_layout: int = V_ROWMAJOR
    rope_style: int = ROPE_NEOX
    _map_checked: tuple | None = field(default=None, init=False, repr=False, compare=False)

    def c(self) -> CKvCache:
        L, npp, H, P, D = self.k.shape
        if P != PAGE or not (self.k.is_contiguous() and self.v.is_contiguous()):
            raise NexusError(ESHAPE, "cache k must be contiguous [L][pages][H][16][D]")
        _on_device(("cache k", self.k), ("cache v", self.v), ("page_map", self.page_map))
        want_v = (L, H, D, npp * P) if self.v_layout == V_TRANSPOSED else (L, npp, H, P, D)
        if tuple(self.v.shape) != want_v:
            raise NexusError(ESHAPE, f"cache v must be {want_v}, got {tuple(self.v.shape)}")
        if self.v.dtype != self.k.dtype:
            raise NexusError(EDTYPE, "cache k and v dtypes differ")
        return CKvCache(self.k.data_ptr(), self.v.data_ptr(), L, npp, P, H, D,
                        _dtype_code(self.k), self.v_layout, self.rope_style, self.rope_base)

    def pt(self) -> CPageTable:
        pm = self.page_map
        if pm.dtype != torch.int32 or pm.dim() != 1 or not pm.is_contiguous():
            raise NexusError(EINVAL, "page_map must be a contiguous int32 vector")
        _on_device(("cache k", self.k), ("page_map", pm))
        npp = self.k.shape[1]
        key = (pm.data_ptr(), pm._version, pm.numel(), npp)
        if self._map_checked != key:
            check_page_table(pm.cpu().numpy(), npp)      # raises NexusError(ERANGE)
            self._map_checked = key
        return CPageTable(pm.data_ptr(), pm.numel())

    @property
    def n_layers(self):
        return self.k.shape[0]


def splice_pages(cache: PagedKVCache, block: Block, offset: int):
    cc, pt, cb = cache.c(), cache.pt(), block.c()
    _on_device(("cache k", cache.k), ("block k", block.k))
    _check(lib().nexus_splice_pages(C.byref(cc), C.byref(pt), C.byref(cb), offset, _stream()),
           "nexus_splice_pages")


def splice_rephase_pages(cache: PagedKVCache, block: Block, offset: int, dst_pos: int):
    """Splice ``block`` at ``offset`` with its keys re-anchored from block.base_pos to
    ``dst_pos`` in the same pass (the block itself is left as it is)."""
    cc, pt, cb = cache.c(), cache.pt(), block.c()
    _on_device(("cache k", cache.k), ("block k", block.k))
    _check(lib().nexus_splice_rephase_pages(C.byref(cc), C.byref(pt), C.byref(cb), offset, dst_pos,
                                            _stream()), "nexus_splice_rephase_pages")


def rope_append(cache: PagedKVCache, k: torch.Tensor, v: torch.Tensor, offset: int, pos0: int):
    """Write un-rotated keys ``k`` (rotated here to positions pos0 + j) and values ``v``, both
    [L][T][H][D] of the cache dtype, into logical slots offset .. offset + T - 1."""
    cc, pt = cache.c(), cache.pt()
    L, T, H, D = k.shape
    if tuple(v.shape) != (L, T, H, D) or not (k.is_contiguous() and v.is_contiguous()):
        raise NexusError(ESHAPE, "k/v must be contiguous [L][T][H][D] of equal shape")
    _on_device(("cache k", cache.k), ("k", k), ("v", v))
    if (L, H, D) != (cc.n_layers, cc.n_kv_heads, cc.head_dim) or _dtype_code(k) != cc.dtype \
            or _dtype_code(v) != cc.dtype:
        raise NexusError(ESHAPE, "k/v must match the cache's layers, heads, head_dim and dtype")
    _check(lib().nexus_rope_append(C.byref(cc), C.byref(pt), _ptr(k), _ptr(v), T, offset, pos0,
                                   _stream()), "nexus_rope_append")


def rephase_k(block: Block, src_pos: int, dst_pos: int, rope_base: float):
    cb = block.c()
    _check(lib().nexus_rephase_k(C.byref(cb), src_pos, dst_pos, rope_base, _stream()),
           "nexus_rephase_k")
    block.base_pos = cb.base_pos


def rephase_k_paged(cache: PagedKVCache, offset: int, n_tokens: int, src_pos: int, dst_pos: int,
                    rope_base: float):
    cc, pt = cache.c(), cache.pt()
    _check(lib().nexus_rephase_k_paged(C.byref(cc), C.byref(pt), offset, n_tokens, src_pos,
                                       dst_pos, rope_base, _stream()), "nexus_rephase_k_paged")


def suffix_attn_workspace_bytes(cache: PagedKVCache, n_s: int, n_q_heads: int, n_past: int) -> int:
    cc = cache.c()
    n = lib().nexus_suffix_attn_workspace(n_s, n_q_heads, C.byref(cc), n_past)
    if n == (1 << 64) - 1:
        raise NexusError(EINVAL, "nexus_suffix_attn_workspace")
    return n


def _workspace(nbytes: int, device, workspace):
    if nbytes == 0:
        return None
    if workspace is not None:
        return workspace
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def suffix_attn(q: torch.Tensor, cache: PagedKVCache, layer: int, n_past: int,
                softcap: float = 0.0, v_layout: int | None = None, scale: float = 0.0,
                out: torch.Tensor | None = None, workspace: torch.Tensor | None = None):
    """q [n_s][n_q_heads][D] -> out [n_s][n_q_heads][D] (cache dtype)."""
    n_s, hq, _ = q.shape
    if not q.is_contiguous():
        raise NexusError(EINVAL, "q must be contiguous")
    if q.dtype != cache.k.dtype:
        raise NexusError(EDTYPE, "q dtype differs from the cache")
    if out is None:
        out = torch.empty_like(q)
    elif out.shape != q.shape or out.dtype != q.dtype or not out.is_contiguous():
        raise NexusError(EINVAL, "out must be contiguous, shaped and typed like q")
    cc, pt = cache.c(), cache.pt()
    _on_device(("cache k", cache.k), ("q", q), ("out", out), ("workspace", workspace))
    ws_bytes = lib().nexus_suffix_attn_workspace(n_s, hq, C.byref(cc), n_past)
    if ws_bytes == (1 << 64) - 1:
        raise NexusError(EINVAL, "nexus_suffix_attn_workspace")
    ws = _workspace(ws_bytes, q.device, workspace)
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().nexus_suffix_attn(_ptr(q), n_s, hq, C.byref(cc), C.byref(pt), layer, n_past,
                                   softcap, cache.v_layout if v_layout is None else v_layout,
                                   scale, _ptr(out), _ptr(ws), nbytes, _stream()),
           "nexus_suffix_attn")
    return out


def suffix_attn_noalloc(q: torch.Tensor, cache: PagedKVCache, layer: int, n_past: int,
                        softcap: float = 0.0, v_layout: int | None = None, scale: float = 0.0,
                        out: torch.Tensor | None = None):
    """suffix_attn without a workspace: the split partials live in the library's static device
    array (see nexus_suffix_attn_noalloc); with ``out`` given, nothing is allocated."""
    n_s, hq, _ = q.shape
    if not q.is_contiguous():
        raise NexusError(EINVAL, "q must be contiguous")
    if q.dtype != cache.k.dtype:
        raise NexusError(EDTYPE, "q dtype differs from the cache")
    if out is None:
        out = torch.empty_like(q)
    elif out.shape != q.shape or out.dtype != q.dtype or not out.is_contiguous():
        raise NexusError(EINVAL, "out must be contiguous, shaped and typed like q")
    cc, pt = cache.c(), cache.pt()
    _on_device(("cache k", cache.k), ("q", q), ("out", out))
    _check(lib().nexus_suffix_attn_noalloc(_ptr(q), n_s, hq, C.byref(cc), C.byref(pt), layer,
                                           n_past, softcap,
                                           cache.v_layout if v_layout is None else v_layout,
                                           scale, _ptr(out), _stream()),
           "nexus_suffix_attn_noalloc")
    return out


def suffix_attn_varlen_workspace_bytes(cache: PagedKVCache, q_start, seq_len, seq_n_past,
                                       n_q_heads: int) -> int:
    n = len(seq_len)
    cc = cache.c()
    nbytes = lib().nexus_suffix_attn_varlen_workspace(n, (C.c_int32 * n)(*q_start),
                                                      (C.c_int32 * n)(*seq_len),
                                                      (C.c_int64 * n)(*seq_n_past), n_q_heads,
                                                      C.byref(cc))
    if nbytes == (1 << 64) - 1:
        raise NexusError(EINVAL, "nexus_suffix_attn_varlen_workspace")
    return nbytes


def suffix_attn_varlen(q: torch.Tensor, q_start, seq_len, seq_n_past, cache: PagedKVCache,
                       layer: int, softcap: float = 0.0, v_layout: int | None = None,
                       scale: float = 0.0, out: torch.Tensor | None = None,
                       workspace: torch.Tensor | None = None):
    """Several suffixes in one launch: rows q_start[b] .. + seq_len[b] at positions
    seq_n_past[b] + i."""
    n = len(seq_len)
    qs = (C.c_int32 * n)(*q_start)
    ls = (C.c_int32 * n)(*seq_len)
    ps = (C.c_int64 * n)(*seq_n_past)
    _, hq, _ = q.shape
    if not q.is_contiguous():
        raise NexusError(EINVAL, "q must be contiguous")
    if q.dtype != cache.k.dtype:
        raise NexusError(EDTYPE, "q dtype differs from the cache")
    if out is None:
        out = torch.empty_like(q)
    elif out.shape != q.shape or out.dtype != q.dtype or not out.is_contiguous():
        raise NexusError(EINVAL, "out must be contiguous, shaped and typed like q")
    cc, pt = cache.c(), cache.pt()
    _on_device(("cache k", cache.k), ("q", q), ("out", out), ("workspace", workspace))
    ws_bytes = lib().nexus_suffix_attn_varlen_workspace(n, qs, ls, ps, hq, C.byref(cc))
    if ws_bytes == (1 << 64) - 1:
        raise NexusError(EINVAL, "nexus_suffix_attn_varlen_workspace")
    ws = _workspace(ws_bytes, q.device, workspace)
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().nexus_suffix_attn_varlen(_ptr(q), n, qs, ls, ps, hq, C.byref(cc), C.byref(pt),
                                          layer, softcap,
                                          cache.v_layout if v_layout is None else v_layout,
                                          scale, _ptr(out), _ptr(ws), nbytes, _stream()),
           "nexus_suffix_attn_varlen")
    return out


def decode_attn_workspace_bytes(cache: PagedKVCache, n_seqs: int, n_q_heads: int,
                                max_seq_len: int) -> int:
    cc = cache.c()
    n = lib().nexus_decode_attn_workspace(n_seqs, n_q_heads, C.byref(cc), max_seq_len)
    if n == (1 << 64) - 1:
        raise NexusError(EINVAL, "nexus_decode_attn_workspace")
    return n


def decode_attn(q: torch.Tensor, cache: PagedKVCache, maps: torch.Tensor, seq_len: torch.Tensor,
                max_seq_len: int, layer: int, softcap: float = 0.0, v_layout: int | None = None,
                scale: float = 0.0, out: torch.Tensor | None = None,
                workspace: torch.Tensor | None = None):
    """One query per sequence: q [n_seqs][n_q_heads][D] -> out (cache dtype).  ``maps`` is a
    device int32 [n_seqs][map_stride] tensor of per-sequence page maps and ``seq_len`` a device
    int32 [n_seqs] tensor (the cache's own page_map is not used)."""
    n, hq, _ = q.shape
    if not q.is_contiguous():
        raise NexusError(EINVAL, "q must be contiguous")
    if q.dtype != cache.k.dtype:
        raise NexusError(EDTYPE, "q dtype differs from the cache")
    if (maps.dtype != torch.int32 or maps.dim() != 2 or maps.shape[0] != n
            or not maps.is_contiguous() or maps.device != q.device):
        raise NexusError(EINVAL, "maps must be a contiguous int32 [n_seqs][stride] device tensor")
    if (seq_len.dtype != torch.int32 or tuple(seq_len.shape) != (n,)
            or not seq_len.is_contiguous() or seq_len.device != q.device):
        raise NexusError(EINVAL, "seq_len must be a contiguous int32 [n_seqs] device tensor")
    if out is None:
        out = torch.empty_like(q)
    elif out.shape != q.shape or out.dtype != q.dtype or not out.is_contiguous():
        raise NexusError(EINVAL, "out must be contiguous, shaped and typed like q")
    cc = cache.c()
    _on_device(("cache k", cache.k), ("q", q), ("maps", maps), ("seq_len", seq_len),
               ("out", out), ("workspace", workspace))
    ws_bytes = lib().nexus_decode_attn_workspace(n, hq, C.byref(cc), max_seq_len)
    if ws_bytes == (1 << 64) - 1:
        raise NexusError(EINVAL, "nexus_decode_attn_workspace")
    ws = _workspace(ws_bytes, q.device, workspace)
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().nexus_decode_attn(_ptr(q), n, hq, C.byref(cc), _ptr(maps), maps.shape[1],
                                   _ptr(seq_len), max_seq_len, layer, softcap,
                                   cache.v_layout if v_layout is None else v_layout, scale,
                                   _ptr(out), _ptr(ws), nbytes, _stream()),
           "nexus_decode_attn")
    return out


def _map_arg(m: torch.Tensor, what: str):
    if m.dtype != torch.int32 or m.dim() != 1 or not m.is_contiguous() or not m.is_cuda:
        raise NexusError(EINVAL, f"{what} must be a contiguous int32 device vector")
    return _ptr(m)


def kv_copy_tokens(cache: PagedKVCache, src_map: torch.Tensor, dst_map: torch.Tensor, t0: int,
                   n_tokens: int):
    """Copy logical tokens [t0, t0 + n_tokens) of every layer from the sequence mapped by
    ``src_map`` to the sequence mapped by ``dst_map`` (device int32 maps of equal length)."""
    if src_map.numel() != dst_map.numel():
        raise NexusError(EINVAL, "maps differ in length")
    cc = cache.c()
    _on_device(("cache k", cache.k), ("src_map", src_map), ("dst_map", dst_map))
    _check(lib().nexus_kv_copy_tokens(C.byref(cc), _map_arg(src_map, "src_map"),
                                      _map_arg(dst_map, "dst_map"), src_map.numel(), t0,
                                      n_tokens, _stream()), "nexus_kv_copy_tokens")


def kv_share_prefix(cache: PagedKVCache, src_map: torch.Tensor, dst_map: torch.Tensor,
                    n_tokens: int):
    """Share the first n_tokens tokens of the source with the destination: whole pages by
    reference (dst_map is updated on the device), the partial last page by copy."""
    if src_map.numel() != dst_map.numel():
        raise NexusError(EINVAL, "maps differ in length")
    cc = cache.c()
    _on_device(("cache k", cache.k), ("src_map", src_map), ("dst_map", dst_map))
    _check(lib().nexus_kv_share_prefix(C.byref(cc), _map_arg(src_map, "src_map"),
                                       _map_arg(dst_map, "dst_map"), src_map.numel(), n_tokens,
                                       _stream()), "nexus_kv_share_prefix")


def l0_longest_prefix(tokens, slots):
    """(slot, length) of the slot sharing the longest common prefix with ``tokens`` (host)."""
    import numpy as np
    t = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
    n_slots = len(slots)
    stride = max([len(x) for x in slots] + [1])
    arr = np.zeros((max(n_slots, 1), stride), dtype=np.int32)
    lens = np.zeros(max(n_slots, 1), dtype=np.int32)
    for i, x in enumerate(slots):
        arr[i, :len(x)] = x
        lens[i] = len(x)
    P = C.POINTER(C.c_int32)
    slot, mlen = C.c_int32(0), C.c_int32(0)
    _check(lib().nexus_l0_longest_prefix(t.ctypes.data_as(P), t.size, arr.ctypes.data_as(P),
                                         lens.ctypes.data_as(P), n_slots, stride, C.byref(slot),
                                         C.byref(mlen)), "nexus_l0_longest_prefix")
    return slot.value, mlen.value


def slb_quantize(x: torch.Tensor, out=None):
    """x [n][dim] fp32 (device) -> (int8 codes [n][dim], fp32 scales [n]); ``out`` may hold
    preallocated (codes, scales)."""
    if x.dtype != torch.float32 or x.dim() != 2 or not x.is_contiguous() or not x.is_cuda:
        raise NexusError(EINVAL, "x must be a contiguous fp32 [n][dim] device tensor")
    n, dim = x.shape
    if out is None:
        q = torch.empty((n, dim), dtype=torch.int8, device=x.device)
        s = torch.empty((n,), dtype=torch.float32, device=x.device)
    else:
        q, s = out
        if (q.dtype != torch.int8 or tuple(q.shape) != (n, dim) or not q.is_contiguous()
                or s.dtype != torch.float32 or s.numel() != n):
            raise NexusError(EINVAL, "out must be (int8 [n][dim], fp32 [n]) contiguous tensors")
    _on_device(("x", x), ("codes", q), ("scales", s))
    _check(lib().nexus_slb_quantize(_ptr(x), n, dim, _ptr(q), _ptr(s), _stream()),
           "nexus_slb_quantize")
    return q, s


def slb_scan(tools: torch.Tensor, tool_scale: torch.Tensor, queries: torch.Tensor,
             query_scale: torch.Tensor, k: int = 2, tau: float = 0.0136,
             workspace: torch.Tensor | None = None, out=None):
    """Top-k tools per query, the top-two margin and the gate (1 = auto-route).  Returns
    (top_idx [Q][k] int32, top_score [Q][k] fp32, margin [Q] fp32, route [Q] int32)."""
    for t, dt, nd in ((tools, torch.int8, 2), (queries, torch.int8, 2),
                      (tool_scale, torch.float32, 1), (query_scale, torch.float32, 1)):
        if t.dtype != dt or t.dim() != nd or not t.is_contiguous() or not t.is_cuda:
            raise NexusError(EINVAL, "slb_scan: bad operand dtype, shape or device")
    n_tools, dim = tools.shape
    n_q = queries.shape[0]
    if queries.shape[1] != dim or tool_scale.numel() != n_tools or query_scale.numel() != n_q:
        raise NexusError(ESHAPE, "slb_scan: operand shapes disagree")
    dev = _on_device(("tools", tools), ("tool_scale", tool_scale), ("queries", queries),
                     ("query_scale", query_scale), ("workspace", workspace))
    if out is not None:
        _on_device(("tools", tools), *[(f"out[{i}]", t) for i, t in enumerate(out)])
    if out is None:
        out = (torch.empty((n_q, k), dtype=torch.int32, device=dev),
               torch.empty((n_q, k), dtype=torch.float32, device=dev),
               torch.empty((n_q,), dtype=torch.float32, device=dev),
               torch.empty((n_q,), dtype=torch.int32, device=dev))
    ws_bytes = lib().nexus_slb_scan_workspace(n_tools, n_q, dim, k)
    if ws_bytes == (1 << 64) - 1:
        ws_bytes = 0             # invalid arguments: the call itself reports which check failed
    ws = _workspace(ws_bytes, dev, workspace)
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    idx, score, margin, route = out
    _check(lib().nexus_slb_scan(_ptr(tools), _ptr(tool_scale), n_tools, _ptr(queries),
                                _ptr(query_scale), n_q, dim, k, tau, _ptr(idx), _ptr(score),
                                _ptr(margin), _ptr(route), _ptr(ws), nbytes, _stream()),
           "nexus_slb_scan")
    return out


def redecode_len(S: int, n_past: int, M: int = 256, r_base_pct: int = 5, K: int = 4) -> int:
    r = lib().nexus_redecode_len(S, n_past, M, r_base_pct, K)
    if r < 0:
        raise NexusError(EINVAL, "nexus_redecode_len")
    return r


def check_page_table(host_map, n_phys_pages: int) -> None:
    import numpy as np
    a = np.ascontiguousarray(np.asarray(host_map, dtype=np.int32))
    _check(lib().nexus_check_page_table(a.ctypes.data_as(C.POINTER(C.c_int32)), a.size,
                                        n_phys_pages), "nexus_check_page_table")


def calib_copy(src: torch.Tensor, dst: torch.Tensor):
    """Device copy of src's bytes into dst (measurement helper: the HBM read + write ceiling)."""
    _on_device(("src", src), ("dst", dst))
    n = src.numel() * src.element_size()
    if not (src.is_contiguous() and dst.is_contiguous()) or dst.numel() * dst.element_size() < n:
        raise NexusError(EINVAL, "calib_copy: contiguous src, and dst at least as large")
    _check(lib().nexus_calib_copy(_ptr(src), _ptr(dst), n, _stream()), "nexus_calib_copy")


def calib_lds_dma(src: torch.Tensor):
    """Stream src's bytes into LDS with LDS DMA loads (measurement helper: the reference for the
    memory counters' reading of the attention kernels' loads)."""
    _on_device(("src", src))
    n = src.numel() * src.element_size()
    if not src.is_contiguous() or n == 0 or n % 16384:
        raise NexusError(EINVAL, "calib_lds_dma: contiguous src of a multiple of 16384 bytes")
    _check(lib().nexus_calib_lds_dma(_ptr(src), n, _stream()), "nexus_calib_lds_dma")


def calib_mfma_bf16(iters: int, sink: torch.Tensor) -> float:
    """Enqueue the bf16 MFMA ceiling kernel; returns the matrix FLOPs it performs."""
    _on_device(("sink", sink))
    if sink.dtype != torch.float32 or sink.numel() < 512:
        raise NexusError(EINVAL, "calib_mfma_bf16: sink must hold 512 fp32 values")
    fl = C.c_double(0.0)
    _check(lib().nexus_calib_mfma_bf16(iters, _ptr(sink), C.byref(fl), _stream()),
           "nexus_calib_mfma_bf16")
    return fl.value
