"""CPU tests of the attention launch plan (the host planner of the bf16 suffix-attention path):
on seeded random varlen launches and on the bench workloads' shapes, every query block of every
head meets every key of its sequence exactly once across the launch's units, the split lengths
are key-tile multiples within the kernels' page-table limit, the per-group split counts agree
with what the kernels and the combine read back, prefills are dispatched longest first, the
range-by-range order keeps ranges together, the workspace size is the sum of the partial slots
and respects a cap, and the plan is deterministic.

The planner is the library's own code, built for the host by a small harness (plan_harness.cpp)
that prints each plan; nothing here runs on a GPU.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_20397_amd", "csrc")
MAX_SPLIT_KEYS = 32768
MAX_SEQS = 32


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("plan") / "plan_harness")
    subprocess.run([hipcc, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", CSRC,
                    os.path.join(ROOT, "tests", "plan_harness.cpp"), "-o", exe],
                   check=True, capture_output=True)
    return exe


def _plans(exe, launches):
    """Run the harness on launches (hq, hkv, d, vt, ws_cap, [(len, n_past), ...])."""
    lines = []
    for hq, hkv, d, vt, cap, seqs in launches:
        flat = " ".join(f"{n} {p}" for n, p in seqs)
        lines.append(f"{hq} {hkv} {d} {int(vt)} {cap} {len(seqs)} {flat}")
    out = subprocess.run([exe], input="\n".join(lines) + "\n", capture_output=True, text=True,
                         check=True).stdout.split("\n")
    plans, cur = [], None
    for ln in out:
        f = ln.split()
        if not f:
            continue
        if f[0] == "plan":
            cur = None if f[1] == "none" else dict(
                units=int(f[2]), range_major=int(f[3]), qpw=int(f[4]), waves=int(f[5]),
                ws=int(f[6]), seqs=[], unit=[])
        elif f[0] == "seq":
            cur["seqs"].append(dict(zip(("b", "q_start", "len", "n_past", "n_tg", "n_tasks",
                                         "max_splits"), map(int, f[1:]))))
        elif f[0] == "unit":
            cur["unit"].append(tuple(map(int, f[1:])))
        elif f[0] == "end":
            plans.append(cur)
    assert len(plans) == len(launches)
    return plans


def _key_tile(d):
    return 32 if d >= 256 else 64


def _check(launch, plan):
    hq, hkv, d, vt, cap, seqs = launch
    g = hq // hkv
    waves = 8 if (d == 256 and vt) else 4
    assert plan["qpw"] == 32 and plan["waves"] == waves
    assert plan["units"] == len(plan["unit"])
    kt = _key_tile(d)
    # per sequence: task groups and their split sets
    ws = 0
    for b, ((n, n_past), sp) in enumerate(zip(seqs, plan["seqs"])):
        assert (sp["len"], sp["n_past"]) == (n, n_past)
        assert sp["q_start"] == sum(x[0] for x in seqs[:b])
        assert sp["n_tasks"] == g * -(-n // 32)
        assert sp["n_tg"] == -(-sp["n_tasks"] // waves)
        if sp["max_splits"] > 1:
            ws += -(-sp["max_splits"] * n * hq * d * 2 // 16) * 16 + sp["max_splits"] * n * hq * 16
    assert plan["ws"] == ws, (plan["ws"], ws)
    if cap:
        assert plan["ws"] <= cap
    seen = {}
    for u, (uu, b, tg, split, k_begin, sk, ns, gs) in enumerate(plan["unit"]):
        assert uu == u
        sp = plan["seqs"][b]
        keys = seqs[b][1] + seqs[b][0]
        assert 0 <= tg < sp["n_tg"]
        assert ns == gs, "unit split count differs from the group's (combine reads the latter)"
        assert 1 <= ns <= sp["max_splits"]
        assert 0 <= split < ns and k_begin == split * sk
        assert sk % kt == 0 and 0 < sk <= MAX_SPLIT_KEYS
        # the group's splits cover the sequence's keys, none starts past them
        assert (ns - 1) * sk < keys <= ns * sk
        key = (b, tg)
        s = seen.setdefault(key, [ns, sk, set()])
        assert (s[0], s[1]) == (ns, sk), "one task group, two split lengths"
        assert split not in s[2], "split dispatched twice"
        s[2].add(split)
    for b, sp in enumerate(plan["seqs"]):
        for tg in range(sp["n_tg"]):
            ns, _, got = seen[(b, tg)]
            assert got == set(range(ns)), (b, tg, got)
    # dispatch order of each sequence's task groups: a causal prefill (n_past < len) last-first
    if not plan["range_major"]:
        for b, (n, n_past) in enumerate(seqs):
            tgs = [x[2] for x in plan["unit"] if x[1] == b]
            first = list(dict.fromkeys(tgs))
            assert first == (sorted(first, reverse=True) if n_past < n else sorted(first)), b
            # a sequence's units are contiguous
            idx = [x[0] for x in plan["unit"] if x[1] == b]
            assert idx == list(range(idx[0], idx[0] + len(idx)))
    else:
        assert len(seqs) > 1 and all(p >= n for n, p in seqs)
        # ranges contiguous and in order; one split length over the launch
        splits = [x[3] for x in plan["unit"]]
        assert splits == sorted(splits)
        assert len({x[5] for x in plan["unit"]}) == 1


def _random_launch(r):
    d = int(r.choice([64, 128, 128, 256]))
    vt = bool(d == 256 and r.random() < 0.7) or bool(d == 128 and r.random() < 0.15)
    hkv = int(r.choice([1, 2, 4, 8]))
    hq = hkv * int(r.choice([1, 2, 4, 5, 8]))
    n_seqs = int(r.choice([1, 1, 2, 3, 5, 8, 16, MAX_SEQS]))
    seqs = []
    for _ in range(n_seqs):
        kind = int(r.integers(0, 4))
        if kind == 0:                                   # causal prefill
            n = int(r.integers(1, 4097))
            p = int(r.integers(0, n))
        elif kind == 1:                                 # re-decoded suffix
            n = int(r.integers(1, 1537))
            p = int(r.integers(n, 40000))
        elif kind == 2:                                 # one query deep in its context
            n, p = 1, int(r.integers(0, 60000))
        else:                                           # a handful of queries
            n = int(r.integers(2, 65))
            p = int(r.integers(0, 20000))
        seqs.append((n, p))
    return (hq, hkv, d, vt, 0, seqs)


# the bench workloads' attention shapes (single-sequence, 16-block, soft-capped transposed V)
_CFG4_PASTS = [(256, 1000 + 1900 * b) for b in range(16)]
WORKLOADS = [
    (40, 8, 128, False, 0, [(192, 2432)]),
    (40, 8, 128, False, 0, [(1088, 16384)]),
    (40, 8, 128, False, 0, _CFG4_PASTS),
    (16, 8, 256, True, 0, [(512, 8704)]),
    (4, 1, 64, False, 0, [(32, 192)]),
    (40, 8, 128, False, 0, [(2048, 0), (576, 1472)]),   # one-launch prefill + suffix
]


def test_plan_invariants_workloads(harness):
    plans = _plans(harness, WORKLOADS)
    for launch, plan in zip(WORKLOADS, plans):
        assert plan is not None, launch
        _check(launch, plan)
    # 16 suffixes over one prefix take the range-by-range order
    assert plans[2]["range_major"] == 1
    # a 16384-deep suffix of 1088 queries splits its keys
    assert plans[1]["seqs"][0]["max_splits"] > 1


def test_plan_invariants_random(harness):
    r = np.random.default_rng([20397, 77])
    launches = [_random_launch(r) for _ in range(300)]
    # single deep suffixes: the shapes that take the two-class split
    for _ in range(100):
        hkv = int(r.choice([1, 2, 4, 8]))
        d = int(r.choice([64, 128, 256]))
        n = int(r.integers(32, 2049))
        launches.append((hkv * int(r.choice([1, 2, 5, 8])), hkv, d, d == 256, 0,
                         [(n, int(r.integers(n, 60000)))]))
    plans = _plans(harness, launches)
    for launch, plan in zip(launches, plans):
        assert plan is not None, launch
        _check(launch, plan)
    # the draws reach both orders and both split regimes
    assert any(p["range_major"] for p in plans) and any(not p["range_major"] for p in plans)
    assert any(p["ws"] > 0 for p in plans) and any(p["ws"] == 0 for p in plans)
    # deterministic: the same launches give the same plans
    assert _plans(harness, launches[:40]) == plans[:40]


def test_plan_workspace_cap(harness):
    """Under a cap every plan fits it, or there is none (never a plan that overruns)."""
    r = np.random.default_rng([20397, 78])
    base = [_random_launch(r) for _ in range(120)] + WORKLOADS
    free = _plans(harness, base)
    capped = []
    for (hq, hkv, d, vt, _, seqs), p in zip(base, free):
        if p["ws"] > 0:
            for frac in (0.5, 0.1, 0.001):
                capped.append((hq, hkv, d, vt, max(1, int(p["ws"] * frac)), seqs))
    assert len(capped) > 60
    n_none = 0
    for launch, plan in zip(capped, _plans(harness, capped)):
        if plan is None:
            n_none += 1
            continue
        _check(launch, plan)
    # over 32768 keys a launch must split, so the tightest caps leave some without a plan; the
    # others fall back to fewer splits (or none)
    assert 0 < n_none < len(capped)


def test_plan_of_the_limit_launches(harness):
    """The GPU limit tests reach what they are named for: a 32768-key split (the workgroup's
    full page table), dozens of splits per row over a 70000-key context, and 32 sequences in
    the range-by-range order (all suffix-like) or the sequence order (with prefills)."""
    from test_gpu_attention_limits import LONGEST_SPLIT, _seqs32
    longest = [(hq, hkv, d, vt, 0, [(n, p)]) for d, vt, _, hq, hkv, n, p in LONGEST_SPLIT]
    beyond = [(8, 2, 64, False, 0, [(16, 70000)]), (8, 2, 128, False, 0, [(16, 70000)]),
              (4, 2, 256, True, 0, [(16, 70000)])]
    many = []
    for d, prefills in [(128, False), (128, True), (256, False), (256, True)]:
        tag = 10 + d // 128 + 2 * prefills
        seqs = _seqs32(np.random.default_rng([20397, 905, tag]), 2600, prefills)
        many.append((4, 2, d, d == 256, 0, seqs))
    launches = longest + beyond + many
    plans = _plans(harness, launches)
    for launch, plan in zip(launches, plans):
        _check(launch, plan)
    for plan in plans[:len(longest)]:
        assert max(x[5] for x in plan["unit"]) == MAX_SPLIT_KEYS
    for plan in plans[len(longest):len(longest) + len(beyond)]:
        assert min(x[6] for x in plan["unit"]) >= 30
    assert [p["range_major"] for p in plans[-4:]] == [1, 0, 1, 0]


def test_plan_beyond_the_range_order(harness):
    """Suffixes over more keys than the range order's 64 ranges of 32768 keys take the sequence
    order (each sequence with its own splits) instead of failing; at that size they keep the
    range order."""
    n = 64 * MAX_SPLIT_KEYS
    launches = [(4, 1, 64, False, 0, [(8, n - 8), (8, n - 1000)]),
                (4, 1, 64, False, 0, [(8, n + 100000), (8, n + 50000)]),
                (8, 2, 128, False, 0, [(16, n + 20000), (1, 5000), (64, n)])]
    plans = _plans(harness, launches)
    for launch, plan in zip(launches, plans):
        assert plan is not None, launch
        _check(launch, plan)
    assert [p["range_major"] for p in plans] == [1, 0, 0]
    assert max(x[6] for x in plans[1]["unit"]) > 64
