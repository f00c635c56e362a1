#!/usr/bin/env python3
"""Throughput of the splice path on one MI355X.

One step is one pass of the whole path over one batch of synthetic input already resident in
HBM: splice the compiled block(s) into the paged cache (all layers), re-anchor their keys in
place (all layers), splice the user-turn tokens, then run the suffix-redecode attention of every
layer back to back.  Default workload: Qwen2.5-14B attention shapes, 48 layers, a 1024-token
block spliced at depth 16384 with a full (R = 100%) redecode of the block plus 64 user tokens
over a 17472-token cache.

Prints one JSON line.  ``value`` is the whole-step attention throughput (algorithmic attention
FLOPs per step / step time, TFLOP/s); ``roofline`` reports the attention kernel against the bf16
MFMA peak and ``roofline_hbm`` the splice and re-anchor kernels against HBM bandwidth (each
timed alone after a streaming pass that evicts the Infinity Cache; their in-step times beside),
all on algorithmic work (the bytes or FLOPs the operation itself defines) and also against the
copy and MFMA ceilings measured on the GPU (``measured_peaks``).  ``configs`` holds the same
figures for the other bf16 workloads (one layer of Qwen2.5-14B shapes at depth 2048; 16 blocks
spliced into a shuffled 32K cache; head_dim 256 with a transposed V and a soft cap).
``cpu_baseline`` times the fp64 oracle on a bounded sample of each workload on the host cores.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
HBM_PEAK_GBPS = 8000.0           # MI355X HBM3E
METRIC = "suffix-redecode attn TFLOP/s + re-phase/splice GB/s, % of MI355X roofline"

# Committed counter summaries of one attention call per config (rocprofv3 FETCH_SIZE /
# WRITE_SIZE scaled by reference kernels of known bytes, and the MFMA / VALU / LDS counters),
# valid only for the kernel sources they were taken on.
PROFILE_TAG = {3: "qwen14b", 4: "qwen14b_16blocks", 5: "softcap_d256"}
ATTN_SOURCES = ["attn_bf16_dma.hip", "attn_bf16_d256.hip", "attn_bf16.hip", "attn_common.h",
                "attn_dma.h", "device_common.h", "launch.h"]


def traffic_file(cfg: int) -> str:
    return os.path.join(ROOT, "profiles", f"hbm_traffic_attn_cfg{cfg}_{PROFILE_TAG.get(cfg, '')}.txt")


def mfma_file(cfg: int) -> str:
    return os.path.join(ROOT, "profiles", f"mfma_util_attn_cfg{cfg}_{PROFILE_TAG.get(cfg, '')}.txt")


def attn_sources_sha() -> str:
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_20397_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counter_summary(path: str, cfg: int):
    """Key/value lines of a committed counter summary, or None when it was taken on other
    attention kernel sources or another workload."""
    try:
        kv = {}
        with open(path) as fh:
            for line in fh:
                if line.startswith("#") or ":" not in line:
                    continue
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    except OSError:
        return None
    if kv.get("workload") != f"cfg{cfg}" or kv.get("kernel_sources_sha256") != attn_sources_sha():
        return None
    return kv


def measured_traffic(cfg: int):
    """Bytes per attention call (FETCH_SIZE + WRITE_SIZE, copy-scaled) from the committed
    counter summary, or None."""
    kv = counter_summary(traffic_file(cfg), cfg)
    try:
        return int(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def counters_from(cfg: int):
    """Where `traffic` and `mfma_busy` come from: the committed counter summaries and the hash
    of the attention sources they were taken on (which matches the sources this run built), or
    None when they are not for these sources."""
    files = [traffic_file(cfg), mfma_file(cfg)]
    if any(counter_summary(f, cfg) is None for f in files):
        return None
    return {"files": [os.path.relpath(f, ROOT) for f in files],
            "attention_sources_sha256": attn_sources_sha()}


def measured_mfma_busy(cfg: int):
    """Fraction of SIMD cycles with the MFMA pipe busy in the attention kernel
    (SQ_VALU_MFMA_BUSY_CYCLES over GRBM_GUI_ACTIVE x SIMDs) from the committed counter
    summary, or None."""
    kv = counter_summary(mfma_file(cfg), cfg)
    try:
        return float(kv["mfma_busy_frac"]) if kv else None
    except (KeyError, ValueError):
        return None


def attn_flops(wl) -> float:
    """4 D H_q sum_i (n_past + i + 1) per layer and block: QK^T and PV over unmasked pairs."""
    tot = 0
    for n_past in wl.attn_n_past:
        n = wl.n_suffix
        tot += 4 * wl.head_dim * wl.n_q_heads * (n * n_past + n * (n + 1) // 2)
    return float(tot)


def setup(cfg: int):
    import torch
    from paper_2608_20397_amd import nexus as N
    from synth import PAGE
    from synth import gen as G

    wl = G.get_workload(cfg)
    dev = "cuda"
    L, H, D, Hq, T = wl.n_layers, wl.n_kv_heads, wl.head_dim, wl.n_q_heads, wl.block_len
    nb = len(wl.splice_pos)
    n_ctx = wl.n_tokens if nb > 1 else wl.splice_pos[0]
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

    def dn(tag, shape, std, off=0):
        return torch.stack([G.device_normal(cfg, l, tag + off, shape, std, wl.dtype, dev)
                            for l in range(L)])

    TG = G.TAG
    vl = N.V_TRANSPOSED if wl.v_layout == "transposed" else N.V_ROWMAJOR
    npp = wl.n_pages
    k = torch.zeros((L, npp, H, PAGE, D), dtype=dt, device=dev)
    v = torch.zeros((L, H, D, npp * PAGE) if vl == N.V_TRANSPOSED else (L, npp, H, PAGE, D),
                    dtype=dt, device=dev)
    pm = torch.from_numpy(G.page_map(cfg, npp, wl.shuffled_pages)).to(dev)
    cache = N.PagedKVCache(k, v, pm, wl.rope_base, vl)
    ctx = N.Block(dn(TG["k_ctx"], (n_ctx, H, D), wl.k_scale), dn(TG["v_ctx"], (n_ctx, H, D), wl.v_scale),
                  0, wl.rope_base)
    N.splice_pages(cache, ctx, 0)                       # context: set-up, not timed
    blocks = [N.Block(dn(TG["k_blk"], (T, H, D), wl.k_scale, 16 * b),
                      dn(TG["v_blk"], (T, H, D), wl.v_scale, 16 * b), wl.anchor, wl.rope_base)
              for b in range(nb)]
    user = None
    if wl.n_user:
        u0 = wl.splice_pos[0] + T
        user = (N.Block(dn(TG["k_user"], (wl.n_user, H, D), wl.k_scale),
                        dn(TG["v_user"], (wl.n_user, H, D), wl.v_scale), u0, wl.rope_base), u0)
    q = dn(TG["q"], (wl.n_suffix * nb, Hq, D), wl.q_scale)
    out = torch.empty_like(q)
    if nb == 1:
        ws_bytes = N.suffix_attn_workspace_bytes(cache, wl.n_suffix, Hq, wl.attn_n_past[0])
    else:
        import ctypes as C
        n = nb
        ws_bytes = N.lib().nexus_suffix_attn_varlen_workspace(
            n, (C.c_int32 * n)(*[b * wl.n_suffix for b in range(n)]),
            (C.c_int32 * n)(*[wl.n_suffix] * n), (C.c_int64 * n)(*wl.attn_n_past), Hq,
            C.byref(cache.c()))
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
    del ctx
    torch.cuda.synchronize()
    return dict(wl=wl, cache=cache, blocks=blocks, user=user, q=q, out=out, ws=ws)


def run_step(S, events=None):
    """One pass of the path; ``events`` collects (kind, start, end) CUDA events per call."""
    import torch
    from paper_2608_20397_amd import nexus as N
    wl, cache = S["wl"], S["cache"]

    def timed(kind, fn):
        if events is None:
            fn()
            return
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        events.append((kind, a, b))

    for b, pos in enumerate(wl.splice_pos):
        blk = S["blocks"][b]
        timed("splice", lambda: N.splice_pages(cache, blk, pos))
        timed("rephase", lambda: N.rephase_k_paged(cache, pos, wl.block_len, wl.anchor, pos,
                                                   wl.rope_base))
    if S["user"] is not None:
        ub, u0 = S["user"]
        timed("splice_user", lambda: N.splice_pages(cache, ub, u0))
    nb = len(wl.splice_pos)
    for layer in range(wl.n_layers):
        if nb == 1:
            timed("attn", lambda: N.suffix_attn(S["q"][layer], cache, layer, wl.attn_n_past[0],
                                                wl.softcap, out=S["out"][layer],
                                                workspace=S["ws"]))
        else:
            timed("attn", lambda: N.suffix_attn_varlen(
                S["q"][layer], [b * wl.n_suffix for b in range(nb)], [wl.n_suffix] * nb,
                list(wl.attn_n_past), cache, layer, wl.softcap, out=S["out"][layer],
                workspace=S["ws"]))


def attn_calls(S):
    """The attention calls of one step, one closure per layer (the calls run_step times)."""
    from paper_2608_20397_amd import nexus as N
    wl, cache = S["wl"], S["cache"]
    nb = len(wl.splice_pos)
    if nb == 1:
        return [lambda layer=layer: N.suffix_attn(S["q"][layer], cache, layer, wl.attn_n_past[0],
                                                  wl.softcap, out=S["out"][layer],
                                                  workspace=S["ws"])
                for layer in range(wl.n_layers)]
    return [lambda layer=layer: N.suffix_attn_varlen(
        S["q"][layer], [b * wl.n_suffix for b in range(nb)], [wl.n_suffix] * nb,
        list(wl.attn_n_past), cache, layer, wl.softcap, out=S["out"][layer], workspace=S["ws"])
        for layer in range(wl.n_layers)]


def cpu_baseline(cfg: int, n_kv_sample: int, n_layers: int, n_blocks: int = 0):
    """The fp64 oracle on a bounded sample: the first ``n_layers`` layers' splice + re-anchor
    (all heads) and the attention of ``n_kv_sample`` KV heads' query groups of the first
    ``n_blocks`` blocks (0: all), scaled to the whole step."""
    import dataclasses

    from threadpoolctl import threadpool_info

    import oracle as O
    from synth import PAGE
    from synth import gen as G

    wl = G.get_workload(cfg)
    n_layers = max(1, min(n_layers, wl.n_layers))
    nb = len(wl.splice_pos)
    n_blocks = nb if n_blocks <= 0 else min(n_blocks, nb)
    t_splice = t_attn = 0.0
    G_ = wl.group
    for layer in range(n_layers):
        hc = G.host_case_wl(dataclasses.replace(wl, n_layers=1), cfg, layers=[layer])
        pm = hc.page_map
        ck, cv = G.empty_cache_bits(hc.wl, 1)
        ck, cv = O.splice_paged(ck, cv, pm, hc.ctx_k, hc.ctx_v, 0, PAGE, wl.v_layout)
        t0 = time.perf_counter()
        for b, pos in enumerate(wl.splice_pos):
            ck, cv = O.splice_paged(ck, cv, pm, hc.blk_k[b], hc.blk_v[b], pos, PAGE, wl.v_layout)
            ck = O.rephase_paged_bits(ck, wl.dtype, pm, PAGE, pos, wl.block_len, wl.anchor, pos,
                                      wl.rope_base)
        if wl.n_user:
            u0 = wl.splice_pos[0] + wl.block_len
            ck, cv = O.splice_paged(ck, cv, pm, hc.user_k, hc.user_v, u0, PAGE, wl.v_layout)
        t_splice += time.perf_counter() - t0
        t0 = time.perf_counter()
        n_keys = max(wl.attn_n_past) + wl.n_suffix
        lk, lv = O.gather_logical(ck, cv, pm, n_keys, PAGE, wl.v_layout)
        k = O.storage_to_f64(lk[0], wl.dtype)
        v = O.storage_to_f64(lv[0], wl.dtype)
        for b, n_past in enumerate(wl.attn_n_past[:n_blocks]):
            qb = O.storage_to_f64(hc.q[0, b * wl.n_suffix:(b + 1) * wl.n_suffix], wl.dtype)
            for g in range(n_kv_sample):
                O.suffix_attention(qb[:, g * G_:(g + 1) * G_], k[:, g:g + 1], v[:, g:g + 1],
                                   n_past, softcap=wl.softcap)
        t_attn += time.perf_counter() - t0
    step_s = (wl.n_layers / n_layers) * (
        t_splice + t_attn * (wl.n_kv_heads / n_kv_sample) * (nb / n_blocks))
    flops = attn_flops(wl) * wl.n_layers
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    blk = f" of the first {n_blocks} of {nb} blocks" if n_blocks < nb else ""
    return {
        "value": flops / step_s / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "host_cpu_count": os.cpu_count(),
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": (f"cfg{cfg} layers 0..{n_layers - 1}: splice + re-anchor of all "
                   f"{wl.n_kv_heads} KV heads ({t_splice:.2f} s) and attention of {n_kv_sample} "
                   f"of {wl.n_kv_heads} KV-head query groups{blk} ({t_attn:.2f} s), scaled "
                   f"x{wl.n_layers / n_layers:g} layers, x{wl.n_kv_heads / n_kv_sample:g} heads"
                   f"{f' and x{nb / n_blocks:g} blocks' if blk else ''} to one step; fp64 numpy, "
                   f"`cores` BLAS threads for the matmuls (of host_cpu_count), elementwise exp "
                   f"single-threaded"),
        "step_s_estimate": step_s,
    }


def time_rotating(fns, reps: int):
    """Mean ms per call of back-to-back calls cycling through ``fns``, callables that each touch
    their own buffers: with enough of them, every call reads data last touched several hundred
    MiB earlier (evicted from the 256 MB Infinity Cache) while earlier calls' writes drain to
    HBM, the steady state of a stream of such calls.  The calls of one cycle are captured in a
    HIP graph and replayed, so that host launch cost stays out of the figure."""
    import torch
    for f in fns:
        f()                                   # first calls (and binding checks) outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        with torch.cuda.graph(g, stream=st):
            for f in fns:
                f()
    torch.cuda.current_stream().wait_stream(st)
    g.replay()
    torch.cuda.synchronize()
    n = max(reps, 3)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(n):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (n * len(fns))


def time_back_to_back(fn, reps: int):
    """Mean ms of ``fn`` over back-to-back calls between two events (repeats re-read what the
    previous call left in the caches)."""
    return time_rotating([fn], reps)


def hbm_row(nbytes: float, ms: float, **extra):
    gbps = nbytes / (ms * 1e-3) / 1e9
    row = {"mean_launch_ms": ms, "bytes_per_launch": int(nbytes), "achieved_GBps": gbps,
           "frac": gbps / HBM_PEAK_GBPS}
    row.update(extra)
    return row


ROT_MIB = 1536      # bytes the copies of a rotation touch together, at least


def time_hbm_kernels(S, reps: int):
    """The HBM-bound kernels of a config timed alone in steady state: each cycles over copies of
    its operands (a block and a cache of the block's pages) that together touch at least
    1.5 GiB, so every call reads HBM.  Splice of the block, in-place re-anchor of its pages, the
    one-pass splice + re-anchor, and the rope-append of the suffix tokens.  GB/s on algorithmic
    bytes: read + write of the block's K and V (splice, one-pass), of its K (re-anchor), of the
    appended tokens' K and V (rope-append).  The copies hold only the pages the block covers,
    at the block's page alignment; the kernels' work does not depend on the other pages."""
    import torch
    from paper_2608_20397_amd import nexus as N
    from synth import PAGE
    wl = S["wl"]
    esize = 2 if wl.dtype == "bf16" else 4
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    L, H, D, T = wl.n_layers, wl.n_kv_heads, wl.head_dim, wl.block_len
    blk_bytes = L * T * H * D * esize
    pos = wl.splice_pos[0]
    off = pos % PAGE                                   # same alignment within a page
    npp = (off + max(T, wl.n_suffix) + PAGE - 1) // PAGE
    vt = wl.v_layout == "transposed"
    n_rot = max(3, -(-(ROT_MIB << 20) // (4 * blk_bytes)))

    def cache_copy(with_v=True):
        k = torch.zeros((L, npp, H, PAGE, D), dtype=dt, device="cuda")
        if with_v:
            v = torch.zeros((L, H, D, npp * PAGE) if vt else (L, npp, H, PAGE, D), dtype=dt,
                            device="cuda")
        else:
            v = shared_v
        return N.PagedKVCache(k, v, torch.arange(npp, dtype=torch.int32, device="cuda"),
                              wl.rope_base, N.V_TRANSPOSED if vt else N.V_ROWMAJOR)

    shared_v = None
    caches = [cache_copy() for _ in range(n_rot)]
    blocks = [N.Block(torch.randn((L, T, H, D), device="cuda").to(dt),
                      torch.randn((L, T, H, D), device="cuda").to(dt), 0, wl.rope_base)
              for _ in range(n_rot)]
    out = {}
    out["splice"] = hbm_row(4 * blk_bytes, time_rotating(
        [lambda c=c, b=b: N.splice_pages(c, b, off) for c, b in zip(caches, blocks)], reps),
        rotation=n_rot)
    # the re-anchor touches only K: twice as many copies for the same span; each call rotates
    # its copy's keys one position further (a rotation keeps their norms)
    n_k = 2 * n_rot
    shared_v = caches[0].v
    kcaches = caches + [cache_copy(with_v=False) for _ in range(n_k - n_rot)]
    out["rephase"] = hbm_row(2 * blk_bytes, time_rotating(
        [lambda c=c: N.rephase_k_paged(c, off, T, pos, pos + 1, wl.rope_base) for c in kcaches],
        reps), rotation=n_k)
    del kcaches
    out["splice_rephase_fused"] = hbm_row(4 * blk_bytes, time_rotating(
        [lambda c=c, b=b: N.splice_rephase_pages(c, b, off, pos) for c, b in zip(caches, blocks)],
        reps), rotation=n_rot)
    n_app = wl.n_suffix
    apps = [(torch.randn((L, n_app, H, D), device="cuda").to(dt),
             torch.randn((L, n_app, H, D), device="cuda").to(dt)) for _ in range(n_rot)]
    out["rope_append"] = hbm_row(4 * L * n_app * H * D * esize, time_rotating(
        [lambda c=c, kv=kv: N.rope_append(c, kv[0], kv[1], off, pos) for c, kv in zip(caches, apps)],
        reps), tokens=n_app, rotation=n_rot)
    del caches, blocks, apps
    torch.cuda.empty_cache()
    return out


def batched_splice_cfg2(reps: int):
    """Supplementary figure for config 2, whose single-layer splice (4 MiB) is far below the
    size a launch needs to approach the HBM roofline: the same block shape (512 tokens x 8 KV
    heads x 128, bf16, spliced at 2048) over all 48 layers in one call, as a real splice moves
    every layer; timed like the other HBM kernels (steady state over rotated copies)."""
    import dataclasses

    from synth import gen as G
    wl = dataclasses.replace(G.get_workload(2), n_layers=48)
    out = time_hbm_kernels({"wl": wl}, reps)
    out["label"] = "supplementary: config 2's block shape over 48 layers in one launch"
    return out


def measured_peaks():
    """The copy and bf16 MFMA ceilings measured on this GPU with the library's calibration
    kernels: a 1 GiB device copy (read + write bytes / time) and 2 waves per SIMD of
    back-to-back 32x32x16 bf16 MFMAs."""
    import torch
    from paper_2608_20397_amd import nexus as N
    n = 1 << 30
    src = torch.empty(n // 4, dtype=torch.int32, device="cuda").random_()
    dst = torch.empty_like(src)
    ms = time_back_to_back(lambda: N.calib_copy(src, dst), 10)
    sink = torch.zeros(512, dtype=torch.float32, device="cuda")
    fl = [0.0]

    def mfma():
        fl[0] = N.calib_mfma_bf16(20000, sink)
    ms_m = time_back_to_back(mfma, 5)
    del src, dst
    return {"copy_GBps": 2 * n / (ms * 1e-3) / 1e9, "copy_bytes": 2 * n,
            "mfma_bf16_TFLOPs": fl[0] / (ms_m * 1e-3) / 1e12,
            "how": "nexus_calib_copy of 1 GiB, back to back; nexus_calib_mfma_bf16 "
                   "(4 independent 32x32x16 bf16 MFMA chains per wave, 2 waves per SIMD)"}


def _graph_time(fn, reps: int, inner: int = 1):
    """Mean ms of ``fn``'s launches, captured ``inner`` times in one HIP graph and replayed (no
    host overhead; a graph launch's own cost is spread over ``inner`` calls)."""
    import torch
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        with torch.cuda.graph(g, stream=st):
            for _ in range(inner):
                fn()
    torch.cuda.current_stream().wait_stream(st)
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (reps * inner)


def time_decode(S, reps: int):
    """Decode step and warm-prefix reuse after the measured steps.

    * decode_b1: one query over the whole spliced cache of the step (all cache tokens, its own
      page map), every layer, captured in a HIP graph;
    * decode_b32: 32 sequences of the same depth on private pages (8 layers of synthetic K/V),
      the warm-prefix pool's width;
    * share_prefix: the first 16384 + 5 tokens (config 3; fewer in a smaller cache) of one of
      those sequences shared with another (1024 pages by reference, 5 slots of each of the 8
      layers copied), one launch;
    * copy_tokens: a 16384-token prefix (at most the cache) copied into a third sequence's pages
      (the copy the paper's arena performs), 8 layers.
    GB/s on algorithmic bytes: K and V of every attended key plus q and out (decode); read +
    write of the copied slots (share, copy)."""
    import torch
    from paper_2608_20397_amd import nexus as N
    wl, cache = S["wl"], S["cache"]
    L, H, D, Hq = wl.n_layers, wl.n_kv_heads, wl.head_dim, wl.n_q_heads
    es = 2 if wl.dtype == "bf16" else 4
    dev = cache.k.device
    n = wl.n_tokens
    out = {}

    def decode_case(cch, n_seqs, layers, maps, tag):
        lens = torch.full((n_seqs,), n, dtype=torch.int32, device=dev)
        q = torch.randn((layers, n_seqs, Hq, D), device=dev).to(cache.k.dtype)
        o = torch.empty_like(q[0])
        wsb = N.decode_attn_workspace_bytes(cch, n_seqs, Hq, n)
        ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)

        def fn():
            for l in range(layers):
                N.decode_attn(q[l], cch, maps, lens, n, l, softcap=wl.softcap, out=o, workspace=ws)
        ms = _graph_time(fn, max(reps, 3)) / layers
        nbytes = n_seqs * (2 * n * H * D * es + 2 * Hq * D * es)
        out[tag] = {"sequences": n_seqs, "tokens_each": n, "layers_timed": layers,
                    "mean_launch_ms": ms, "bytes_per_launch": nbytes,
                    "achieved_GBps": nbytes / (ms * 1e-3) / 1e9,
                    "frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}

    n_pages = -(-n // 16)
    decode_case(cache, 1, L, cache.page_map[:n_pages].reshape(1, n_pages).contiguous(),
                "decode_b1")
    B, L8 = 32, 8
    npp = B * n_pages
    k = torch.randn((L8, npp, H, 16, D), device=dev).to(cache.k.dtype)
    v = torch.randn((L8, npp, H, 16, D), device=dev).to(cache.k.dtype)
    c32 = N.PagedKVCache(k, v, torch.zeros(1, dtype=torch.int32, device=dev), wl.rope_base,
                         N.V_ROWMAJOR)
    maps = torch.arange(npp, dtype=torch.int32, device=dev).view(B, n_pages).contiguous()
    decode_case(c32, B, L8, maps, "decode_b32")
    # warm-prefix reuse between two sequences of the 32-sequence cache (disjoint pages)
    src, dst = maps[0].contiguous(), maps[1].contiguous()
    slot_bytes = 2 * L8 * H * D * es                      # K and V of one token, all layers
    n_share = min(16384, (n // 16 - 1) * 16) + 5       # whole pages + 5 slots, inside the cache
    # idempotent after its first run: 50 calls per graph
    ms = _graph_time(lambda: N.kv_share_prefix(c32, src, dst, n_share), max(reps, 3), inner=50)
    tail = n_share % 16
    out["share_prefix"] = {"tokens": n_share, "layers": L8, "pages_shared": n_share // 16,
                           "slots_copied": tail, "mean_launch_ms": ms,
                           "bytes_per_launch": 2 * tail * slot_bytes}
    n_copy = min(16384, n)
    dst2 = maps[2].contiguous()
    ms = _graph_time(lambda: N.kv_copy_tokens(c32, src, dst2, 0, n_copy), max(reps, 3))
    nbytes = 2 * n_copy * slot_bytes
    out["copy_tokens"] = {"tokens": n_copy, "layers": L8, "mean_launch_ms": ms,
                          "bytes_per_launch": nbytes, "achieved_GBps": nbytes / (ms * 1e-3) / 1e9,
                          "frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}
    del k, v, c32, maps
    return out


def time_slb(reps: int):
    """The SLB scan and margin gate (Sec. V-A) after the measured steps, each timed in a HIP
    graph: the paper's registry (250 tools, one query, the query's quantisation included), a
    1M-tool registry with one query (a pass over 768 MB of INT8 rows: GB/s against HBM) and a
    serving batch (65536 tools x 256 queries: int8 TOPS).  Every row keeps the top 3, the
    shortlist whose recall the paper reports (top-1 / top-3)."""
    import numpy as np
    import torch
    from paper_2608_20397_amd import nexus as N
    from synth import slb as SL
    dev = "cuda"
    out = {}

    def run(tq, ts, qq, qs, k, tag, extra=None, quantize=None):
        n, dim = tq.shape
        nq = qq.shape[0]
        res = (torch.empty((nq, k), dtype=torch.int32, device=dev),
               torch.empty((nq, k), device=dev), torch.empty(nq, device=dev),
               torch.empty(nq, dtype=torch.int32, device=dev))
        wsb = N.lib().nexus_slb_scan_workspace(n, nq, dim, k)
        ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)

        def fn():
            if quantize is not None:
                quantize()
            N.slb_scan(tq, ts, qq, qs, k, 0.0136, workspace=ws, out=res)
        inner = 20 if n * nq <= 1 << 22 else 3
        ms = _graph_time(fn, max(reps, 3), inner=inner)
        row = {"tools": n, "queries": nq, "dim": dim, "k": k, "mean_launch_ms": ms,
               "tool_bytes": n * dim, "achieved_GBps": n * dim / (ms * 1e-3) / 1e9,
               "int8_TOPS": 2.0 * n * nq * dim / (ms * 1e-3) / 1e12,
               "route_rate": float(res[3].float().mean().item())}
        row.update(extra or {})
        out[tag] = row

    # the paper's registry size, synthetic unit-norm vectors; the query quantised in the loop
    t, q, _ = SL.slb_inputs(1)
    tq, ts = N.slb_quantize(torch.from_numpy(t).to(dev))
    qf = torch.from_numpy(q).to(dev)
    qq = torch.empty((1, t.shape[1]), dtype=torch.int8, device=dev)
    qs = torch.empty(1, device=dev)

    def quant():
        N.slb_quantize(qf, out=(qq, qs))
    run(tq, ts, qq, qs, 3, "slb_n250_q1", {"includes": "query quantisation + scan + gate"},
        quantize=quant)
    g = torch.Generator(device=dev)
    g.manual_seed(20397)
    big = torch.randint(-127, 128, (1 << 20, 768), dtype=torch.int8, device=dev, generator=g)
    bs = torch.rand(1 << 20, device=dev, generator=g) * 0.01
    q1 = torch.randint(-127, 128, (1, 768), dtype=torch.int8, device=dev, generator=g)
    s1 = torch.rand(1, device=dev, generator=g) * 0.01
    run(big, bs, q1, s1, 3, "slb_n1m_q1")
    out["slb_n1m_q1"]["frac_hbm"] = out["slb_n1m_q1"]["achieved_GBps"] / HBM_PEAK_GBPS
    mid, ms_ = big[:65536], bs[:65536]
    qb = torch.randint(-127, 128, (256, 768), dtype=torch.int8, device=dev, generator=g)
    sb = torch.rand(256, device=dev, generator=g) * 0.01
    run(mid, ms_, qb, sb, 3, "slb_n65536_q256")
    out["slb_n65536_q256"]["frac_int8_mfma"] = out["slb_n65536_q256"]["int8_TOPS"] / 5000.0
    del big
    return out


SWEEP_DEPTHS = (256, 512, 1024, 2048, 4096, 16384)


def sweep(reps: int):
    """Depth-adaptive sweep (the shape of Table tab:perf without weights): attention time of a full
    prefill against the splice path, all 48 layers of Qwen2.5-14B attention shapes, a 512-token
    block and 64 user tokens at context depth n_past.  Prefill = causal attention of all
    n_past + 512 + 64 tokens.  Splice path = prefill of the n_past context tokens, the one-pass
    splice + re-anchor of the block (all layers) and the attention of the redecoded
    r = redecode_len(512, n_past, 256, 5, K) block tokens plus the user tokens over the whole
    cache, as two launches per layer (context, then suffix) or as one (the context rows and the
    redecoded rows as two sequences of one varlen launch, after the splice).  Each variant's
    48-layer call sequence is captured in a HIP graph and replayed, so host launch overhead does
    not enter the comparison."""
    import torch
    from paper_2608_20397_amd import nexus as N
    from synth import PAGE
    from synth import gen as G
    L, Hq, H, D, S, u, base, cfg = 48, 40, 8, 128, 512, 64, 1e6, 2
    M, r_base = 256, 5
    std = 128 ** -0.5

    def graph_ms(calls):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            calls()                                   # warm-up outside the capture
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            calls()
        g.replay()
        torch.cuda.synchronize()
        ts = []
        for _ in range(max(reps, 5)):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            g.replay()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        ts.sort()
        return ts[len(ts) // 2]

    rows = []
    for n_past in SWEEP_DEPTHS:
        total = n_past + S + u
        npp = (total + PAGE - 1) // PAGE
        k = G.device_normal(cfg, n_past, G.TAG["k_ctx"], (L, npp, H, PAGE, D), std, "bf16", "cuda")
        v = G.device_normal(cfg, n_past, G.TAG["v_ctx"], (L, npp, H, PAGE, D), std, "bf16", "cuda")
        cache = N.PagedKVCache(k, v, torch.arange(npp, dtype=torch.int32, device="cuda"), base)
        blk = N.Block(G.device_normal(cfg, n_past, G.TAG["k_blk"], (L, S, H, D), std, "bf16", "cuda"),
                      G.device_normal(cfg, n_past, G.TAG["v_blk"], (L, S, H, D), std, "bf16", "cuda"),
                      0, base)
        q = G.device_normal(cfg, n_past, G.TAG["q"], (L, total, Hq, D), std, "bf16", "cuda")

        def attn_calls(r0, r1, n0):
            qs = [q[l, r0:r1].contiguous() for l in range(L)]
            outs = [torch.empty_like(x) for x in qs]
            ws = torch.empty(max(N.suffix_attn_workspace_bytes(cache, r1 - r0, Hq, n0), 16),
                             dtype=torch.uint8, device="cuda")

            def run():
                for l in range(L):
                    N.suffix_attn(qs[l], cache, l, n0, 0.0, out=outs[l], workspace=ws)
            return run

        def one_launch_calls(n_s):
            starts, lens, pasts = [0, n_past], [n_past, n_s], [0, total - n_s]
            qs = [torch.cat([q[l, :n_past], q[l, total - n_s:]]).contiguous() for l in range(L)]
            outs = [torch.empty_like(x) for x in qs]
            ws = torch.empty(max(N.suffix_attn_varlen_workspace_bytes(cache, starts, lens, pasts,
                                                                      Hq), 16),
                             dtype=torch.uint8, device="cuda")

            def run():
                for l in range(L):
                    N.suffix_attn_varlen(qs[l], starts, lens, pasts, cache, l, out=outs[l],
                                         workspace=ws)
            return run

        def flops(r0, r1):
            # QK^T and PV over the unmasked pairs of queries r0 .. r1 - 1 (query i sees i + 1 keys)
            return 4 * D * Hq * ((r1 * (r1 + 1) - r0 * (r0 + 1)) // 2)

        prefill = attn_calls(0, total, 0)
        context = attn_calls(0, n_past, 0)
        t_prefill = graph_ms(prefill)
        t_splice = graph_ms(lambda: N.splice_rephase_pages(cache, blk, n_past, n_past))
        t_ctx = graph_ms(context)
        for K in (4, 16):
            r = N.redecode_len(S, n_past, M, r_base, K)
            n_s = r + u
            suffix = attn_calls(total - n_s, total, total - n_s)

            def path():
                context()
                N.splice_rephase_pages(cache, blk, n_past, n_past)
                suffix()
            t_suf = graph_ms(suffix)
            t_path = graph_ms(path)
            # the same splice path with the context rows and the redecoded rows of a layer in
            # one launch (two sequences of one varlen call), after the splice
            one = one_launch_calls(n_s)

            def path1():
                N.splice_rephase_pages(cache, blk, n_past, n_past)
                one()
            t_path1 = graph_ms(path1)
            R = r_base if n_past <= M else min(
                100.0, r_base + (n_past - M) * (100.0 - r_base) / (M * (K - 1)))
            rows.append({"K": K, "n_past": n_past, "R_pct": round(R, 1), "redecode": r,
                         "prefill_ms": t_prefill, "context_ms": t_ctx, "splice_ms": t_splice,
                         "suffix_ms": t_suf, "suffix_us_per_layer": 1e3 * t_suf / L,
                         "splice_path_ms": t_path, "speedup": t_prefill / t_path,
                         "splice_path_one_launch_ms": t_path1,
                         "speedup_one_launch": t_prefill / t_path1,
                         "query_tokens_ratio": total / (n_past + n_s),
                         "attn_flops_ratio": flops(0, total) / (flops(0, n_past) + flops(total - n_s, total))})
        del k, v, cache, blk, q
        torch.cuda.empty_cache()
    return rows


def run_config(cfg: int, steps: int, warmup: int):
    """Set up config ``cfg``, run ``warmup`` untimed steps and ``steps`` timed ones; returns the
    set-up state, the step time and the mean duration of each kind of call (HIP events on the
    launch stream)."""
    import torch
    S = setup(cfg)
    print(f"bench: cfg{cfg} {S['wl'].name}: setup done", file=sys.stderr, flush=True)
    for _ in range(warmup):
        run_step(S)
    torch.cuda.synchronize()
    events = []
    t0 = time.perf_counter()
    for _ in range(steps):
        run_step(S, events)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    dur = {}
    for kind, a, b in events:
        dur.setdefault(kind, []).append(a.elapsed_time(b))
    mean = {k: sum(v) / len(v) for k, v in dur.items()}
    print(f"bench: cfg{cfg}: {steps} steps, {ms:.3f} ms/step, mean call ms {mean}",
          file=sys.stderr, flush=True)
    return S, ms, mean


def config_summary(S, ms: float, mean: dict, hbm: dict, peaks: dict):
    """Per-config figures: attention against the bf16 MFMA peak, splice and re-anchor against
    HBM (inside the step, and timed alone after a cache-evicting pass)."""
    wl = S["wl"]
    esize = 2 if wl.dtype == "bf16" else 4
    blk_bytes = wl.n_layers * wl.block_len * wl.n_kv_heads * wl.head_dim * esize
    nb = len(wl.splice_pos)
    fl = attn_flops(wl)
    tf = fl / (mean["attn"] * 1e-3) / 1e12
    splice_b, rephase_b = 4 * blk_bytes, 2 * blk_bytes
    # the step's attention calls replayed back to back from a HIP graph: no host enqueue gaps
    # (which the per-call events of a short single-layer call include)
    alone_ms = time_rotating(attn_calls(S), max(3, 10 // wl.n_layers))
    tf_alone = fl / (alone_ms * 1e-3) / 1e12
    return {
        "workload": f"cfg{wl.cfg}: {wl.name}",
        "dtype": wl.dtype,
        "ms_per_step": ms,
        "step_attn_TFLOPs": fl * wl.n_layers / (ms * 1e-3) / 1e12,
        "attn": {"achieved_TFLOPs": tf, "frac": tf / MFMA_BF16_PEAK_TFLOPS,
                 "frac_of_measured_mfma": tf / peaks["mfma_bf16_TFLOPs"],
                 "mean_launch_ms": mean["attn"], "flops_per_launch": fl,
                 "traffic": measured_traffic(wl.cfg),
                 "mfma_busy": measured_mfma_busy(wl.cfg),
                 "counters_from": counters_from(wl.cfg),
                 "alone": {"mean_launch_ms": alone_ms, "achieved_TFLOPs": tf_alone,
                           "frac": tf_alone / MFMA_BF16_PEAK_TFLOPS,
                           "timing": "the step's attention calls back to back in a HIP graph "
                                     "(operands may stay in the Infinity Cache between calls "
                                     "of a one-layer config)"},
                 "launches_per_step": wl.n_layers,
                 "call": "nexus_suffix_attn" if nb == 1 else f"nexus_suffix_attn_varlen ({nb} "
                                                              f"suffixes)"},
        "splice_in_step": hbm_row(splice_b, mean["splice"],
                                  note="block read from HBM (the previous step's attention "
                                       "evicted it)"),
        "rephase_in_step": hbm_row(rephase_b, mean["rephase"],
                                   note="right after the splice: its keys may still be in the "
                                        "Infinity Cache"),
        "hbm_alone": hbm,
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, choices=[2, 3, 4, 5])
    ap.add_argument("--only", action="store_true",
                    help="measure --config alone (no other configs, next rows or baselines)")
    ap.add_argument("--step-only", action="store_true",
                    help="run the steps of --config and print their times only (no peaks, "
                         "kernels timed alone, next rows or baselines): the command the counter "
                         "passes profile")
    ap.add_argument("--hbm-only", action="store_true",
                    help="time only the HBM-bound kernels of --config (splice, re-anchor, "
                         "one-pass splice + re-anchor, rope-append) in steady state and print "
                         "them: the command their counter passes profile")
    ap.add_argument("--cpu-kv-sample", type=int, default=8,
                    help="KV heads per layer the oracle baseline computes (0 skips it)")
    ap.add_argument("--cpu-layers", type=int, default=3,
                    help="layers the oracle baseline computes")
    ap.add_argument("--sweep", action="store_true",
                    help="only run the depth-adaptive sweep (attention-only prefill vs splice "
                         "path over context depths, K = 4 and 16), print it as JSON, then exit")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only time a plain device copy of MIB MiB and a stream of the same "
                         "bytes into LDS through LDS DMA loads (HBM references and the scales "
                         "of the FETCH_SIZE / WRITE_SIZE counters), then exit")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: runs on one GPU only (the library has no multi-GPU path); use --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_20397_amd import nexus as N
    N.lib()   # fail loudly if the library is not built
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").random_(0, 255)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        a.record()
        for _ in range(reps):
            dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        # the same bytes streamed into LDS with the attention kernels' DMA loads
        for _ in range(3):
            N.calib_lds_dma(src)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            N.calib_lds_dma(src)
        b.record()
        torch.cuda.synchronize()
        ms_dma = a.elapsed_time(b) / reps
        print(json.dumps({"copy_mib": args.copy_calibration, "ms_per_copy": ms,
                          "GBps_read_plus_write": 2 * n / (ms * 1e-3) / 1e9,
                          "ms_per_lds_dma_read": ms_dma,
                          "GBps_lds_dma_read": n / (ms_dma * 1e-3) / 1e9}), flush=True)
        return
    if args.sweep:
        print(json.dumps({"sweep": sweep(args.steps), "unit": "ms for all 48 layers",
                          "shapes": "Qwen2.5-14B attention (40/8/128, theta 1e6), block 512, "
                                    "user 64, bf16, 48 layers, HIP-graph replay"}), flush=True)
        return
    if args.hbm_only:
        from synth import gen as G
        print(json.dumps({"config": args.config,
                          "hbm": time_hbm_kernels({"wl": G.get_workload(args.config)},
                                                  args.steps)}), flush=True)
        return
    if args.step_only:
        _, ms, mean = run_config(args.config, args.steps, args.warmup)
        print(json.dumps({"config": args.config, "ms_per_step": ms, "mean_call_ms": mean}),
              flush=True)
        return
    peaks = measured_peaks()
    S, ms, mean = run_config(args.config, args.steps, args.warmup)
    wl = S["wl"]
    hbm = time_hbm_kernels(S, args.steps)
    summ = config_summary(S, ms, mean, hbm, peaks)

    fl_layer = attn_flops(wl)
    step_flops = fl_layer * wl.n_layers
    attn_tflops = summ["attn"]["achieved_TFLOPs"]
    nb = len(wl.splice_pos)
    res = {
        "metric": METRIC,
        "value": step_flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) draws at Qwen2.5-14B attention shapes; no weights)",
        "config": {
            "workload": f"cfg{wl.cfg}: {wl.name}",
            "layers": wl.n_layers, "n_q_heads": wl.n_q_heads, "n_kv_heads": wl.n_kv_heads,
            "head_dim": wl.head_dim, "rope_base": wl.rope_base, "page_size": 16,
            "blocks": nb, "block_len": wl.block_len, "splice_pos": list(wl.splice_pos)[:4],
            "suffix_queries": wl.n_suffix, "attn_n_past": list(wl.attn_n_past)[:4],
            "cache_tokens": wl.n_tokens, "v_layout": wl.v_layout, "softcap": wl.softcap,
        },
        "roofline": {
            "bound": "mfma",
            "kernel": ("one nexus_suffix_attn call per layer: attn_bf16_d128_dma_kernel + "
                       "attn_combine_kernel (split-K combine)"),
            "achieved": attn_tflops,
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": attn_tflops / MFMA_BF16_PEAK_TFLOPS,
            "traffic": measured_traffic(wl.cfg),
            "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-scaled)",
            "mfma_busy": measured_mfma_busy(wl.cfg),
            "mfma_busy_unit": ("fraction of SIMD cycles with the MFMA pipe busy, attention kernel "
                               "(SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x SIMDs))"),
            "counters_from": counters_from(wl.cfg),
            "algorithmic_flops_per_launch": fl_layer,
            "mean_launch_ms": mean["attn"],
            "alone": summ["attn"]["alone"],
            "frac_of_measured_peak": attn_tflops / peaks["mfma_bf16_TFLOPs"],
        },
        "roofline_hbm": {
            "bound": "hbm",
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "splice": hbm["splice"],
            "rephase": hbm["rephase"],
            "frac": ((hbm["splice"]["bytes_per_launch"] + hbm["rephase"]["bytes_per_launch"])
                     / ((hbm["splice"]["mean_launch_ms"] + hbm["rephase"]["mean_launch_ms"]) * 1e-3)
                     / 1e9 / HBM_PEAK_GBPS),
            "timing": ("each kernel alone in steady state, cycling over copies of its operands "
                       "that together touch >= 1.5 GiB (reads come from HBM)"),
            "in_step": {"splice": summ["splice_in_step"], "rephase": summ["rephase_in_step"]},
            "frac_of_measured_copy": {
                k: hbm[k]["achieved_GBps"] / peaks["copy_GBps"]
                for k in ("splice", "rephase", "splice_rephase_fused", "rope_append")},
        },
        "measured_peaks": peaks,
    }
    res["next_rows"] = {"splice_rephase_fused": hbm["splice_rephase_fused"],
                        "rope_append": hbm["rope_append"]}
    res["next_rows"].update(time_decode(S, args.steps))
    res["next_rows"].update(time_slb(args.steps))
    del S
    torch.cuda.empty_cache()
    others = [] if args.only else [c for c in (2, 4, 5) if c != args.config]
    if others:
        res["configs"] = {}
    for cfg in others:
        S2, ms2, mean2 = run_config(cfg, args.steps, args.warmup)
        row = config_summary(S2, ms2, mean2, time_hbm_kernels(S2, args.steps), peaks)
        if cfg == 2:
            row["splice_48_layers_supplementary"] = batched_splice_cfg2(args.steps)
        res["configs"][f"cfg{cfg}"] = row
        del S2
        torch.cuda.empty_cache()
    try:
        res["git"] = subprocess.run(["git", "-C", ROOT, "rev-parse", "--short", "HEAD"],
                                    capture_output=True, text=True).stdout.strip() or None
    except Exception:
        res["git"] = None
    if args.cpu_kv_sample > 0:
        print("bench: timing the oracle baseline on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(args.config, min(args.cpu_kv_sample, wl.n_kv_heads),
                                           args.cpu_layers)
        # smaller samples of the other configs (same oracle, same scaling rule)
        samples = {2: (8, 1, 0), 4: (2, 1, 4), 5: (8, 1, 0)}
        for cfg in others:
            kv, nl, nbk = samples[cfg]
            res["configs"][f"cfg{cfg}"]["cpu_baseline"] = cpu_baseline(cfg, kv, nl, nbk)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
