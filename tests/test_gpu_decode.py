"""GPU parity of the decode step (one query per sequence over its own page map) against the fp64
oracle, on the seeded decode batches of ``synth.decode``: mixed lengths (0, 1, page edges, long),
shared prefix pages, shuffled pools, NaN in every slot a query must not see, row-major and
transposed V, soft-capping, head_dim 32..256, 1 to 32 query heads per KV head, bf16 and fp32.

Tolerances as the suffix attention: bf16 max-abs 2e-2 and rel-RMS 5e-3, fp32 1e-5.
"""

import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_20397_amd import nexus as N
from synth import PAGE
from synth import decode as SD
from synth import gen as G

from _pipeline import BF16_MAX_ABS, BF16_REL_RMS, F32_TOL, compare, to_f64

pytestmark = pytest.mark.gpu

VL = {"rowmajor": N.V_ROWMAJOR, "transposed": N.V_TRANSPOSED}


def _upload(hc, dev="cuda"):
    wl = hc.wl
    k = G.bits_to_torch(hc.k, wl.dtype, dev)
    v = G.bits_to_torch(hc.v, wl.dtype, dev)
    q = G.bits_to_torch(hc.q, wl.dtype, dev)
    # the cache's own page map is not used by the decode call
    cache = N.PagedKVCache(k, v, torch.zeros(1, dtype=torch.int32, device=dev), 1e4,
                           VL[wl.v_layout])
    maps = torch.from_numpy(hc.maps).to(dev)
    lens = torch.tensor(wl.lens, dtype=torch.int32, device=dev)
    return cache, maps, lens, q


def _oracle(hc, layer_idx, lens=None):
    wl = hc.wl
    lens = wl.lens if lens is None else lens
    k = O.storage_to_f64(hc.k[layer_idx], wl.dtype)
    v = O.storage_to_f64(hc.v[layer_idx], wl.dtype)
    q = O.storage_to_f64(hc.q[layer_idx], wl.dtype)
    return O.decode_attention(q, k, v, hc.maps, lens, PAGE, wl.v_layout, softcap=wl.softcap)


def _check(got, ref, dtype, tag):
    ma, rr = compare(got, ref)
    print(f"{tag}: max-abs {ma:.3e} rel-RMS {rr:.3e}", flush=True)
    assert np.isfinite(got).all(), tag
    if dtype == "bf16":
        assert ma <= BF16_MAX_ABS and rr <= BF16_REL_RMS, (tag, ma, rr)
    else:
        assert ma <= F32_TOL and rr <= F32_TOL, (tag, ma, rr)


@pytest.mark.parametrize("case", [1, 2, 5, 6, 7])
def test_decode_parity(case):
    hc = SD.decode_host_case(case)
    wl = hc.wl
    cache, maps, lens, q = _upload(hc)
    for layer in range(wl.n_layers):
        out = N.decode_attn(q[layer], cache, maps, lens, wl.max_len, layer, softcap=wl.softcap)
        torch.cuda.synchronize()
        got = to_f64(out)
        ref = _oracle(hc, layer)
        _check(got, ref, wl.dtype, f"decode case {case} layer {layer}")
        for b, n in enumerate(wl.lens):
            if n == 0:
                assert np.array_equal(got[b], np.zeros_like(got[b])), b


def test_decode_full_size_single_sequence():
    """The benchmark's decode step: one 17473-token sequence, Qwen2.5-14B heads, two layers of
    48 (all 40 query heads compared)."""
    hc = SD.decode_host_case(3, layers=[0, 47])
    wl = hc.wl
    cache, maps, lens, q = _upload(hc)
    for i in range(2):
        out = N.decode_attn(q[i], cache, maps, lens, wl.max_len, i)
        torch.cuda.synchronize()
        _check(to_f64(out), _oracle(hc, i), wl.dtype, f"decode case 3 sampled layer {i}")


def test_decode_32_sequences_shared_prefix():
    """32 sequences (the warm-prefix pool) sharing the physical pages of a 16384-token prefix."""
    hc = SD.decode_host_case(4)
    wl = hc.wl
    cache, maps, lens, q = _upload(hc)
    out = N.decode_attn(q[0], cache, maps, lens, wl.max_len, 0)
    torch.cuda.synchronize()
    _check(to_f64(out), _oracle(hc, 0), wl.dtype, "decode case 4")


def test_decode_device_lengths_graph_replay():
    """Lengths live on the device: one captured launch, replayed after the lengths change,
    matches the oracle at the new lengths on every replay; a re-run is bit-identical."""
    hc = SD.decode_host_case(2)
    wl = hc.wl
    cache, maps, lens, q = _upload(hc)
    short = tuple(max(1, n - 37 * (b + 1)) for b, n in enumerate(wl.lens))
    lens.copy_(torch.tensor(short, dtype=torch.int32))
    ws_bytes = N.decode_attn_workspace_bytes(cache, wl.n_seqs, wl.n_q_heads, wl.max_len)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(q[0])
    N.decode_attn(q[0], cache, maps, lens, wl.max_len, 0, out=out, workspace=ws)
    torch.cuda.synchronize()
    first = out.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            N.decode_attn(q[0], cache, maps, lens, wl.max_len, 0, out=out, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    ref_short = _oracle(hc, 0, short)
    ref_full = _oracle(hc, 0)
    for rep, (ln, ref) in enumerate([(short, ref_short), (wl.lens, ref_full), (short, ref_short)]):
        lens.copy_(torch.tensor(ln, dtype=torch.int32))
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _check(to_f64(out), ref, wl.dtype, f"graph replay {rep}")
        if ln == short:
            assert torch.equal(out.view(torch.int16), first.view(torch.int16))


def test_decode_lengths_above_bound_are_clamped():
    """A device length above max_seq_len is read as max_seq_len: keys past the bound are never
    touched (the oracle at the clamped lengths)."""
    hc = SD.decode_host_case(2)
    wl = hc.wl
    cache, maps, lens, q = _upload(hc)
    bound = 1000
    big = torch.tensor([n if n < bound else 4097 for n in wl.lens], dtype=torch.int32,
                       device="cuda")
    out = N.decode_attn(q[0], cache, maps, big, bound, 0)
    torch.cuda.synchronize()
    ref = _oracle(hc, 0, tuple(min(n, bound) for n in wl.lens))
    _check(to_f64(out), ref, wl.dtype, "clamped lengths")


def test_decode_rejects_bad_arguments():
    hc = SD.decode_host_case(6)
    wl = hc.wl
    cache, maps, lens, q = _upload(hc)
    with pytest.raises(N.NexusError) as e:
        N.decode_attn(q[0], cache, maps, lens, maps.shape[1] * PAGE + 1, 0)
    assert e.value.status == N.ERANGE
    with pytest.raises(N.NexusError) as e:
        N.decode_attn(q[0], cache, maps, lens, wl.max_len, 1)
    assert e.value.status == N.ERANGE
    with pytest.raises(N.NexusError) as e:
        N.decode_attn(q[0], cache, maps, lens, wl.max_len, 0, v_layout=N.V_TRANSPOSED)
    assert e.value.status == N.ELAYOUT
    with pytest.raises(N.NexusError) as e:
        N.decode_attn(q[0][:, :63], cache, maps, lens, wl.max_len, 0)
    assert e.value.status in (N.EINVAL, N.ESHAPE)
