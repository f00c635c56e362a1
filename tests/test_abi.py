"""CPU tests of the C ABI: the library loads, exports every declared entry point, and its host
logic (redecode length, page-table check, fail-closed validation) behaves as declared.

Validation calls use tiny descriptors.  Without a GPU their pointers are placeholders that no
code path dereferences (every call here must fail validation or enqueue nothing); with a GPU
they are real device buffers of the described sizes, so nothing can fault either way.
"""

import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "nexus.h")).read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w \t\*]*?\b(nexus_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 10, names
    L = N.lib()
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", N.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (nexus_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    assert N.lib().nexus_abi_version() == 1


def test_redecode_len_matches_oracle_eq_adaptive():
    L = N.lib()
    for K in (2, 3, 4, 8, 16):
        for M in (1, 64, 256):
            for rb in (0, 5, 37, 100):
                for S in (0, 1, 63, 384, 512, 1024, 4097):
                    for n in (0, M - 1, M, M + 1, 300, 511, 512, 1024, 2048, 4 * M, 16384, 70001):
                        if n < 0:
                            continue
                        assert L.nexus_redecode_len(S, n, M, rb, K) == O.redecode_len(S, n, M, rb, K), \
                            (S, n, M, rb, K)
    for bad in [(-1, 0, 256, 5, 4), (10, -1, 256, 5, 4), (10, 0, 0, 5, 4), (10, 0, 256, 101, 4),
                (10, 0, 256, -1, 4), (10, 300, 256, 5, 1)]:
        assert L.nexus_redecode_len(*bad) == -1


def test_redecode_len_tab_perf_rows():
    """The suffix the orchestrator re-decodes for a 512-token block at the Table tab:perf depths."""
    got = [N.redecode_len(512, n, 256, 5, K) for K in (4, 16) for n in (256, 512, 1024, 2048)]
    assert got == [26, 188, 512, 512, 26, 59, 123, 253]   # 512 * 34/3 / 100 = 58.03 -> 59


def test_check_page_table():
    N.check_page_table(np.arange(10), 10)
    N.check_page_table(np.random.default_rng(0).permutation(12)[:10], 12)
    for bad, npp in [([0, 1, 1], 5), ([0, 5], 5), ([-1, 0], 5), ([0, 1, 2], 2)]:
        with pytest.raises(N.NexusError) as e:
            N.check_page_table(bad, npp)
        assert e.value.status == N.ERANGE


# ------------------------------------------------------------------ fail-closed validation
class _Bufs:
    """Placeholder addresses without a GPU; real device buffers with one."""

    def __init__(self):
        self.keep = []
        self.gpu = torch.cuda.is_available()

    def __call__(self, nbytes):
        if not self.gpu:
            return 0x10000 + 0x1000 * len(self.keep) + (self.keep.append(None) or 0)
        t = torch.zeros(max(nbytes, 16), dtype=torch.uint8, device="cuda")
        self.keep.append(t)
        return t.data_ptr()


def _setup(dtype=N.BF16, v_layout=N.V_ROWMAJOR, L=2, npp=6, H=2, D=64, T=20, base=1e4):
    buf = _Bufs()
    es = 2 if dtype == N.BF16 else 4
    cache = N.CKvCache(buf(L * npp * H * 16 * D * es), buf(L * npp * H * 16 * D * es), L, npp, 16,
                       H, D, dtype, v_layout, N.ROPE_NEOX, base)
    block = N.CBlock(buf(L * T * H * D * es), buf(L * T * H * D * es), L, T, H, D, dtype,
                     N.ROPE_NEOX, 0, base)
    pt = N.CPageTable(buf(npp * 4), npp)
    return buf, cache, block, pt


def test_splice_validation_fails_closed():
    L = N.lib()
    buf, cache, block, pt = _setup()
    s = C.c_void_p(0)
    assert L.nexus_splice_pages(None, C.byref(pt), C.byref(block), 0, s) == N.EINVAL
    bad = N.CBlock.from_buffer_copy(block); bad.rope_base = 1e6
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(bad), 0, s) == N.EROPE
    bad = N.CBlock.from_buffer_copy(block); bad.rope_style = N.ROPE_INTERLEAVED
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(bad), 0, s) == N.EROPE
    bad = N.CBlock.from_buffer_copy(block); bad.n_kv_heads = 1
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(bad), 0, s) == N.ESHAPE
    bad = N.CBlock.from_buffer_copy(block); bad.dtype = N.F32
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(bad), 0, s) == N.EDTYPE
    bad = N.CBlock.from_buffer_copy(block); bad.dtype = 7
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(bad), 0, s) == N.EDTYPE
    # 20 tokens at offset 77 end at 97 > 6 pages * 16 = 96
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(block), 77, s) == N.ERANGE
    assert L.nexus_splice_pages(C.byref(cache), C.byref(pt), C.byref(block), -1, s) == N.ERANGE
    big = N.CPageTable(pt.map, 7)                       # more logical than physical pages
    assert L.nexus_splice_pages(C.byref(cache), C.byref(big), C.byref(block), 0, s) == N.ERANGE
    bc = N.CKvCache.from_buffer_copy(cache); bc.page_size = 32
    assert L.nexus_splice_pages(C.byref(bc), C.byref(pt), C.byref(block), 0, s) == N.ESHAPE
    bc = N.CKvCache.from_buffer_copy(cache); bc.head_dim = 60; block2 = N.CBlock.from_buffer_copy(block); block2.head_dim = 60
    assert L.nexus_splice_pages(C.byref(bc), C.byref(pt), C.byref(block2), 0, s) == N.ESHAPE
    # head_dim must be a power of two: 96 and 48 pass the per-chunk divisibility checks
    for hd in (96, 48):
        bc = N.CKvCache.from_buffer_copy(cache); bc.head_dim = hd
        block2 = N.CBlock.from_buffer_copy(block); block2.head_dim = hd
        assert L.nexus_splice_pages(C.byref(bc), C.byref(pt), C.byref(block2), 0, s) == N.ESHAPE


def test_rephase_validation_and_identity():
    L = N.lib()
    buf, cache, block, pt = _setup()
    s = C.c_void_p(0)
    assert L.nexus_rephase_k(C.byref(block), 5, 9, 1e4, s) == N.EROPE        # anchor is 0
    assert L.nexus_rephase_k(C.byref(block), 0, 9, 1e6, s) == N.EROPE        # base mismatch
    assert L.nexus_rephase_k(C.byref(block), 0, -3, 1e4, s) == N.ERANGE
    assert block.base_pos == 0
    # delta 0: nothing is enqueued, the anchor stays
    assert L.nexus_rephase_k(C.byref(block), 0, 0, 1e4, s) == N.OK
    assert block.base_pos == 0
    assert L.nexus_rephase_k_paged(C.byref(cache), C.byref(pt), 0, 20, 7, 7, 1e4, s) == N.OK
    assert L.nexus_rephase_k_paged(C.byref(cache), C.byref(pt), 90, 20, 0, 7, 1e4, s) == N.ERANGE
    assert L.nexus_rephase_k_paged(C.byref(cache), C.byref(pt), 0, 0, 0, 7, 1e4, s) == N.EINVAL
    assert L.nexus_rephase_k_paged(C.byref(cache), C.byref(pt), 0, 20, 0, 7, 2e4, s) == N.EROPE


def test_fused_splice_and_rope_append_validation_fails_closed():
    L = N.lib()
    buf, cache, block, pt = _setup()
    s = C.c_void_p(0)
    f = L.nexus_splice_rephase_pages
    # the splice checks apply unchanged
    assert f(None, C.byref(pt), C.byref(block), 0, 5, s) == N.EINVAL
    bad = N.CBlock.from_buffer_copy(block); bad.rope_base = 1e6
    assert f(C.byref(cache), C.byref(pt), C.byref(bad), 0, 5, s) == N.EROPE
    bad = N.CBlock.from_buffer_copy(block); bad.n_kv_heads = 1
    assert f(C.byref(cache), C.byref(pt), C.byref(bad), 0, 5, s) == N.ESHAPE
    bad = N.CBlock.from_buffer_copy(block); bad.dtype = N.F32
    assert f(C.byref(cache), C.byref(pt), C.byref(bad), 0, 5, s) == N.EDTYPE
    assert f(C.byref(cache), C.byref(pt), C.byref(block), 77, 5, s) == N.ERANGE
    assert f(C.byref(cache), C.byref(pt), C.byref(block), 0, -1, s) == N.ERANGE
    buf2, big, bigblk, pt2 = _setup(D=512)
    assert f(C.byref(big), C.byref(pt2), C.byref(bigblk), 0, 5, s) == N.ESHAPE
    assert block.base_pos == 0                          # the block is never re-anchored
    g = L.nexus_rope_append
    k, v = buf(2 * 20 * 2 * 64 * 2), buf(2 * 20 * 2 * 64 * 2)
    assert g(None, C.byref(pt), k, v, 20, 0, 0, s) == N.EINVAL
    assert g(C.byref(cache), C.byref(pt), None, v, 20, 0, 0, s) == N.EINVAL
    assert g(C.byref(cache), C.byref(pt), k, None, 20, 0, 0, s) == N.EINVAL
    assert g(C.byref(cache), C.byref(pt), k, v, 0, 0, 0, s) == N.EINVAL
    assert g(C.byref(cache), C.byref(pt), k, v, 20, -1, 0, s) == N.ERANGE
    assert g(C.byref(cache), C.byref(pt), k, v, 20, 0, -1, s) == N.ERANGE
    assert g(C.byref(cache), C.byref(pt), k, v, 20, 77, 0, s) == N.ERANGE
    assert g(C.byref(big), C.byref(pt2), k, v, 20, 0, 0, s) == N.ESHAPE
    bc = N.CKvCache.from_buffer_copy(cache); bc.page_size = 32
    assert g(C.byref(bc), C.byref(pt), k, v, 20, 0, 0, s) == N.ESHAPE


def test_attention_validation_fails_closed():
    L = N.lib()
    buf, cache, block, pt = _setup(D=128)
    s = C.c_void_p(0)
    q, out = buf(8 * 4 * 128 * 2), buf(8 * 4 * 128 * 2)
    ok_args = lambda **kw: dict(dict(q=q, n_s=8, hq=4, layer=1, n_past=40, cap=0.0,
                                     vl=N.V_ROWMAJOR, scale=0.0, out=out), **kw)

    def call(a, ws=None, wsb=0, cc=cache, ptt=pt):
        return L.nexus_suffix_attn(a["q"], a["n_s"], a["hq"], C.byref(cc), C.byref(ptt),
                                   a["layer"], a["n_past"], a["cap"], a["vl"], a["scale"],
                                   a["out"], ws, wsb, s)

    assert call(ok_args(vl=N.V_TRANSPOSED)) == N.ELAYOUT
    assert call(ok_args(hq=3)) == N.ESHAPE                  # 3 % 2 kv heads
    assert call(ok_args(layer=2)) == N.ERANGE
    assert call(ok_args(n_past=90)) == N.ERANGE             # 90 + 8 > 96
    assert call(ok_args(n_past=-1)) == N.ERANGE
    assert call(ok_args(n_s=0)) == N.EINVAL
    assert call(ok_args(q=None)) == N.EINVAL
    assert call(ok_args(cap=-1.0)) == N.EINVAL
    assert call(ok_args(cap=float("nan"))) == N.EINVAL
    bc = N.CKvCache.from_buffer_copy(cache); bc.head_dim = 96
    assert call(ok_args(), cc=bc) == N.ESHAPE                # bf16 MFMA path: D in {64,128,256}
    need = L.nexus_suffix_attn_workspace(8, 4, C.byref(cache), 40)
    if need > 0:
        assert call(ok_args()) == N.EWORKSPACE
        assert call(ok_args(), ws=buf(need), wsb=need - 1) == N.EWORKSPACE
    assert L.nexus_suffix_attn_workspace(8, 3, C.byref(cache), 40) == (1 << 64) - 1


def test_varlen_validation():
    L = N.lib()
    buf, cache, block, pt = _setup(D=128)
    s = C.c_void_p(0)
    q = buf(64 * 4 * 128 * 2)
    n = 33
    a32 = (C.c_int32 * n)(*([0] * n))
    l32 = (C.c_int32 * n)(*([1] * n))
    p64 = (C.c_int64 * n)(*([0] * n))
    assert L.nexus_suffix_attn_varlen(q, n, a32, l32, p64, 4, C.byref(cache), C.byref(pt), 0, 0.0,
                                      0, 0.0, q, None, 0, s) == N.EINVAL          # > 32 sequences
    l2 = (C.c_int32 * 2)(4, 0)
    assert L.nexus_suffix_attn_varlen(q, 2, a32, l2, p64, 4, C.byref(cache), C.byref(pt), 0, 0.0,
                                      0, 0.0, q, None, 0, s) == N.EINVAL          # empty sequence
    p2 = (C.c_int64 * 2)(10, 95)
    l3 = (C.c_int32 * 2)(4, 4)
    assert L.nexus_suffix_attn_varlen(q, 2, a32, l3, p2, 4, C.byref(cache), C.byref(pt), 0, 0.0,
                                      0, 0.0, q, None, 0, s) == N.ERANGE          # 95 + 4 > 96


def test_decode_validation_fails_closed():
    L = N.lib()
    buf, cache, block, pt = _setup(D=128)
    s = C.c_void_p(0)
    q, out = buf(3 * 4 * 128 * 2), buf(3 * 4 * 128 * 2)
    maps, lens = buf(3 * 6 * 4), buf(3 * 4)
    ok_args = lambda **kw: dict(dict(q=q, n=3, hq=4, maps=maps, stride=6, lens=lens, max_len=96,
                                     layer=1, cap=0.0, vl=N.V_ROWMAJOR, scale=0.0, out=out), **kw)

    def call(a, ws=None, wsb=0, cc=cache):
        return L.nexus_decode_attn(a["q"], a["n"], a["hq"], C.byref(cc), a["maps"], a["stride"],
                                   a["lens"], a["max_len"], a["layer"], a["cap"], a["vl"],
                                   a["scale"], a["out"], ws, wsb, s)

    assert call(ok_args(vl=N.V_TRANSPOSED)) == N.ELAYOUT
    assert call(ok_args(vl=7)) == N.EINVAL
    assert call(ok_args(hq=3)) == N.ESHAPE                  # 3 % 2 kv heads
    assert call(ok_args(layer=2)) == N.ERANGE
    assert call(ok_args(layer=-1)) == N.ERANGE
    assert call(ok_args(max_len=97)) == N.ERANGE            # > 16 * stride
    assert call(ok_args(max_len=-1)) == N.ERANGE
    assert call(ok_args(n=0)) == N.EINVAL
    assert call(ok_args(stride=0)) == N.EINVAL
    assert call(ok_args(q=None)) == N.EINVAL
    assert call(ok_args(maps=None)) == N.EINVAL
    assert call(ok_args(lens=None)) == N.EINVAL
    assert call(ok_args(out=None)) == N.EINVAL
    assert call(ok_args(cap=-1.0)) == N.EINVAL
    assert call(ok_args(scale=float("inf"))) == N.EINVAL
    bc = N.CKvCache.from_buffer_copy(cache); bc.head_dim = 96
    assert call(ok_args(), cc=bc) == N.ESHAPE
    # a long bound needs a split workspace
    need = L.nexus_decode_attn_workspace(3, 4, C.byref(cache), 96 * 64)
    assert need > 0
    assert call(ok_args(stride=6 * 64, max_len=96 * 64)) == N.EWORKSPACE
    assert call(ok_args(stride=6 * 64, max_len=96 * 64), ws=buf(need), wsb=need - 1) == N.EWORKSPACE
    assert L.nexus_decode_attn_workspace(3, 3, C.byref(cache), 96) == (1 << 64) - 1
    assert L.nexus_decode_attn_workspace(0, 4, C.byref(cache), 96) == (1 << 64) - 1


def test_status_strings():
    L = N.lib()
    for st in range(9):
        assert len(L.nexus_status_str(st)) > 0
    assert L.nexus_status_str(99) == b"unknown status"


def test_l0_longest_prefix_matches_oracle():
    """Host logic of the warm-prefix arena lookup against the oracle's definition (32 slots)."""
    import oracle as O
    rng = np.random.default_rng(5)
    for trial in range(200):
        base = list(rng.integers(0, 3, size=int(rng.integers(0, 40))))
        slots = []
        for s in range(int(rng.integers(0, 33))):
            k = int(rng.integers(0, len(base) + 1))
            tail = list(rng.integers(0, 3, size=int(rng.integers(0, 10))))
            slots.append(base[:k] + tail)
        q = base[:int(rng.integers(0, len(base) + 1))] + list(rng.integers(0, 3, size=3))
        assert N.l0_longest_prefix(q, slots) == O.longest_prefix(q, slots), trial
    assert N.l0_longest_prefix([], [[1, 2]]) == (-1, 0)
    assert N.l0_longest_prefix([1, 2], []) == (-1, 0)


def test_kv_copy_and_share_validation_fails_closed():
    L = N.lib()
    buf, cache, block, pt = _setup(D=64)
    s = C.c_void_p(0)
    a, b = buf(8 * 4), buf(8 * 4)
    f = L.nexus_kv_copy_tokens
    assert f(None, a, b, 8, 0, 5, s) == N.EINVAL
    assert f(C.byref(cache), None, b, 8, 0, 5, s) == N.EINVAL
    assert f(C.byref(cache), a, None, 8, 0, 5, s) == N.EINVAL
    assert f(C.byref(cache), a, b, 0, 0, 5, s) == N.EINVAL
    assert f(C.byref(cache), a, b, 8, 0, 0, s) == N.EINVAL
    assert f(C.byref(cache), a, b, 8, -1, 5, s) == N.ERANGE
    assert f(C.byref(cache), a, b, 8, 120, 9, s) == N.ERANGE          # 129 > 128
    g = L.nexus_kv_share_prefix
    assert g(C.byref(cache), a, b, 8, -1, s) == N.ERANGE
    assert g(C.byref(cache), a, b, 8, 129, s) == N.ERANGE
    assert g(C.byref(cache), a, b, 8, 0, s) == N.OK                   # nothing to do
    bc = N.CKvCache.from_buffer_copy(cache); bc.page_size = 32
    assert g(C.byref(bc), a, b, 8, 5, s) == N.ESHAPE
    P = C.POINTER(C.c_int32)
    t = (C.c_int32 * 3)(1, 2, 3)
    sl = (C.c_int32 * 2)(1, 2)
    ln = (C.c_int32 * 1)(2)
    out_s, out_l = C.c_int32(7), C.c_int32(7)
    h = L.nexus_l0_longest_prefix
    assert h(t, 3, sl, ln, 1, 2, None, C.byref(out_l)) == N.EINVAL
    assert h(t, -1, sl, ln, 1, 2, C.byref(out_s), C.byref(out_l)) == N.EINVAL
    assert h(None, 3, sl, ln, 1, 2, C.byref(out_s), C.byref(out_l)) == N.EINVAL
    bad = (C.c_int32 * 1)(3)
    assert h(t, 3, sl, bad, 1, 2, C.byref(out_s), C.byref(out_l)) == N.ERANGE
    assert h(t, 3, sl, ln, 1, 2, C.byref(out_s), C.byref(out_l)) == N.OK
    assert (out_s.value, out_l.value) == (0, 2)


def test_slb_validation_fails_closed():
    L = N.lib()
    buf = _Bufs()
    s = C.c_void_p(0)
    t, ts, q, qs = buf(100 * 768), buf(400), buf(768), buf(4)
    o1, o2, o3, o4 = buf(64), buf(64), buf(4), buf(4)
    ok = dict(t=t, ts=ts, n=100, q=q, qs=qs, nq=1, dim=768, k=2, tau=0.0136)

    def call(ws=None, wsb=0, **kw):
        a = dict(ok, **kw)
        return L.nexus_slb_scan(a["t"], a["ts"], a["n"], a["q"], a["qs"], a["nq"], a["dim"], a["k"],
                                a["tau"], o1, o2, o3, o4, ws, wsb, s)

    assert call(t=None) == N.EINVAL
    assert call(qs=None) == N.EINVAL
    assert call(n=0) == N.EINVAL
    assert call(nq=0) == N.EINVAL
    assert call(k=0) == N.EINVAL
    assert call(k=9) == N.EINVAL
    assert call(tau=float("nan")) == N.EINVAL
    assert call(dim=100) == N.ESHAPE
    assert call(dim=2048) == N.ESHAPE
    need = L.nexus_slb_scan_workspace(100000, 256, 768, 8)
    assert need > 0
    assert call(n=100000, nq=256, k=8) == N.EWORKSPACE
    assert L.nexus_slb_scan_workspace(100, 1, 100, 2) == (1 << 64) - 1
    assert L.nexus_slb_scan_workspace(250, 1, 768, 2) == 0          # one range: no workspace
    assert L.nexus_slb_quantize(None, 1, 64, o1, o2, s) == N.EINVAL
    assert L.nexus_slb_quantize(t, 0, 64, o1, o2, s) == N.EINVAL


def test_binding_rejects_host_tensors():
    """Every tensor the binding hands to the library must live on the device: host tensors are
    refused with EINVAL before any call (no GPU is needed to check this)."""
    import torch
    k = torch.zeros(1, 2, 1, 16, 64, dtype=torch.bfloat16)
    cache = N.PagedKVCache(k, k.clone(), torch.arange(2, dtype=torch.int32), 1e4)
    with pytest.raises(N.NexusError) as e:
        cache.c()
    assert e.value.status == N.EINVAL
    with pytest.raises(N.NexusError) as e:
        cache.pt()
    assert e.value.status == N.EINVAL
    b = torch.zeros(1, 4, 1, 64, dtype=torch.bfloat16)
    with pytest.raises(N.NexusError) as e:
        N.Block(b, b.clone(), 0, 1e4).c()
    assert e.value.status == N.EINVAL
    with pytest.raises(N.NexusError) as e:
        N.slb_quantize(torch.zeros(2, 64))
    assert e.value.status == N.EINVAL
