"""The GPU segment scheduler against plain-loop CPU grouping: bit-exact groups, ranks, chunking,
work list and each branch's ordered partial-row list, and identical schedules on repeated
runs."""
import json
import os

import numpy as np
import pytest
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import graphattn as G
from paper_2606_18954_amd import workloads as W

from gpu_util import params_of, say

pytestmark = pytest.mark.gpu

ROWS_PER_BLOCK = 128


def cost_class(cost):
    """Half-octave bins of the per-item cost: 1 + 2 floor(log2 c) + (the bit below the leading
    one), capped at 31; 0 for no cost."""
    cost = int(cost)
    if cost == 0:
        return 0
    e = cost.bit_length() - 1
    m = (cost >> (e - 1)) & 1 if e > 0 else 0
    return min(31, 1 + 2 * e + m)


def chains(g):
    """Chains of path segments with identical branch sets: s links to s' when every branch
    through s continues with s' and |B(s)| = |B(s')|.  Returns the chains (lists of segments, in
    path order) ordered by their first segment's id."""
    S = g.num_segments
    cnt = [0] * S
    succ = [None] * S
    for b in range(g.num_branches):
        p = [int(x) for x in g.path_segs[g.path_offsets[b]:g.path_offsets[b + 1]]]
        for i, s in enumerate(p):
            cnt[s] += 1
            n = p[i + 1] if i + 1 < len(p) else -1
            succ[s] = n if succ[s] is None else (n if succ[s] == n else -1)
    link = {s: succ[s] for s in range(S)
            if cnt[s] and succ[s] is not None and succ[s] >= 0 and cnt[succ[s]] == cnt[s]}
    has_pred = set(link.values())
    out = []
    for s in range(S):
        if cnt[s] and s not in has_pred:
            c = [s]
            while c[-1] in link:
                c.append(link[c[-1]])
            out.append(c)
    return out


SORT_CAP = 8192     # chains the scheduler orders by cost; more keep their first-segment order


def expected_items(g, group, chunk_pages, cnt):
    """Work list: items grouped by chain, chains by descending cost class of the per-item cost
    (pages of the chain's longest chunk x (2 + row tiles); a chain's chunks split its pages as
    evenly as whole pages allow), ties by first segment (beyond SORT_CAP chains, in first-segment
    order); within a chain chunk-major.  An item names its chain by the chain's first segment."""
    def npg(s):
        return (int(g.seg_len[s]) + 15) // 16

    def cost(c):
        tiles = (min(cnt[c[0]] * group, ROWS_PER_BLOCK) + 15) // 16
        pages = sum(npg(s) for s in c)
        nch = (pages + chunk_pages - 1) // chunk_pages
        return -(-pages // nch) * (2 + tiles)

    order = chains(g)
    if len(order) <= SORT_CAP:
        order = sorted(order, key=lambda c: (-cost_class(cost(c)), c[0]))
    items = []
    for c in order:
        pages = sum(npg(s) for s in c)
        nch = (pages + chunk_pages - 1) // chunk_pages
        nrb = (cnt[c[0]] * group + ROWS_PER_BLOCK - 1) // ROWS_PER_BLOCK
        for ch in range(nch):
            for rb in range(nrb):
                items.append((c[0], ch, rb))
    return np.array(items, dtype=np.int32).reshape(-1, 3)


def expected_partials(g, chunk_pages, offs, ranks):
    """Each branch's partial rows as a plain loop builds them: chains numbered in the order of
    their first segments, prow(v) the running sum of chunks x |B| over them, and for every path
    entry that starts a chain, one row per chunk, prow(v) + c |B(v)| + rank, in path order."""
    ch = chains(g)
    cnt = np.diff(offs)
    head = {c[0]: i for i, c in enumerate(ch)}
    nch = [(sum((int(g.seg_len[s]) + 15) // 16 for s in c) + chunk_pages - 1) // chunk_pages
           for c in ch]
    prow = [0]
    for i, c in enumerate(ch):
        prow.append(prow[-1] + nch[i] * int(cnt[c[0]]))
    boff, parts = [0], []
    for b in range(g.num_branches):
        for e in range(int(g.path_offsets[b]), int(g.path_offsets[b + 1])):
            s = int(g.path_segs[e])
            if s in head:
                v = head[s]
                parts += [prow[v] + c * int(cnt[s]) + int(ranks[e]) for c in range(nch[v])]
        boff.append(len(parts))
    return np.array(boff, dtype=np.int64), np.array(parts, dtype=np.int32)


def check_schedule(wl):
    g = wl.graph
    say(f"[case] schedule of {wl.name}")
    hg = G.HostGraph.from_graph(g)
    with G.Plan(hg, params_of(wl)) as plan:
        plan.schedule()
        d = plan.debug_dump()
        info = plan.info()
        plan.schedule()                       # rescheduling gives the same bits
        d2 = plan.debug_dump()
    offs, ids = O.segment_groups(g.path_offsets, g.path_segs, g.num_segments)
    ranks = O.branch_slot_ranks(g.path_offsets, g.path_segs, g.num_segments)
    assert np.array_equal(d["group_offsets"], offs)
    assert np.array_equal(d["group_branches"], ids)
    assert np.array_equal(d["entry_ranks"], ranks)
    cnt = np.diff(offs)
    group = wl.num_q_heads // wl.num_kv_heads
    exp_items = expected_items(g, group, info.chunk_pages, cnt)
    assert np.array_equal(d["items"], exp_items)
    # Chunks of each chain at its first segment, 0 elsewhere.
    chunks = np.zeros(g.num_segments, dtype=np.int32)
    ch = chains(g)
    for c in ch:
        pages = sum((int(g.seg_len[s]) + 15) // 16 for s in c)
        chunks[c[0]] = (pages + info.chunk_pages - 1) // info.chunk_pages
    assert info.num_chains == len(ch)
    assert np.array_equal(d["segment_chunks"], chunks)
    assert info.num_partial_rows == int(sum(chunks[s] for s in g.path_segs))
    boff, parts = expected_partials(g, info.chunk_pages, offs, ranks)
    assert np.array_equal(d["branch_part_offsets"], boff)
    assert np.array_equal(d["branch_parts"], parts)
    for k in d:
        assert np.array_equal(d[k], d2[k]), k


def test_golden_small_dag():
    with open(os.path.join(os.path.dirname(__file__), "golden", "groups_small_dag.json")) as f:
        fx = json.load(f)
    lens = [40, 17, 5, 90, 16, 1]
    paths = [fx["path_segs"][a:b] for a, b in zip(fx["path_offsets"][:-1], fx["path_offsets"][1:])]
    g = W.assemble_graph(lens, paths, 1, 2)
    wl = W.make_workload("golden small DAG", g, 8, 2, 64, "f32", 1)
    hg = G.HostGraph.from_graph(g)
    with G.Plan(hg, params_of(wl)) as plan:
        plan.schedule()
        d = plan.debug_dump()
    assert d["group_offsets"].tolist() == fx["group_offsets"]
    assert d["group_branches"].tolist() == fx["group_branches"]
    assert d["entry_ranks"].tolist() == fx["entry_ranks"]


@pytest.mark.parametrize("name,kw", [("c1", {}), ("c2", {}), ("c3", {"prompts": 12}),
                                     ("c4", {"prompts": 3}), ("c5graph", {"prompts": 3})])
def test_config_schedules(name, kw):
    check_schedule(W.CONFIGS[name](**kw))


def test_random_graphs():
    rng = np.random.default_rng(42)
    for t in range(6):
        g = W.random_graph(rng, int(rng.integers(1, 60)), int(rng.integers(1, 200)), 300, 12,
                           seed=t)
        check_schedule(W.make_workload(f"random {t}", g, 28, 4, 64, "bf16", t))


def test_segment_shared_by_many_branches():
    n = 600
    lens = [64] + [5] * n
    paths = [[0, 1 + i] for i in range(n)]
    g = W.assemble_graph(lens, paths, 3)
    check_schedule(W.make_workload("600-way shared root", g, 28, 4, 64, "bf16", 3))


def test_large_graphs_use_the_multi_kernel_path():
    """Graphs beyond the single-workgroup limits (4096 segments, 8192 path entries, 4095
    branches) take the multi-kernel scheduler; its output must be the same function of the
    graph."""
    rng = np.random.default_rng(7)
    # > 4096 segments and branches
    g = W.random_graph(rng, 5000, 4500, 40, 3, seed=1)
    check_schedule(W.make_workload("5000-segment graph", g, 28, 4, 64, "bf16", 1))
    # > 8192 path entries with few segments
    lens = [int(x) for x in rng.integers(1, 50, size=64)]
    paths = [list(rng.choice(64, size=10, replace=False)) for _ in range(900)]
    g2 = W.assemble_graph(lens, paths, 3)
    assert g2.path_segs.shape[0] == 9000
    check_schedule(W.make_workload("9000-entry graph", g2, 8, 2, 64, "f32", 3))


@pytest.mark.parametrize("n", [6000, 9000])
def test_chains_past_the_counting_sort(n):
    """A root shared by n branches, each of which ends in a segment of its own (n + 1 chains):
    6,001 chains are ordered by the bitonic sort (more than the counting sort's 4,096), 9,001
    keep their first-segment order (more than the 8,192 the sort holds); every other output is
    as for smaller graphs, and sampled branches match the oracle."""
    from gpu_util import check_workload
    rng = np.random.default_rng(n)
    lens = [200] + [int(x) for x in rng.integers(1, 40, size=n)]
    paths = [[0, 1 + i] for i in range(n)]
    g = W.assemble_graph(lens, paths, 5)
    wl = W.make_workload(f"{n + 1}-chain graph", g, 8, 2, 64, "bf16", 5)
    assert len(chains(g)) == n + 1 > 4096
    check_schedule(wl)
    check_workload(wl, branches=[0, 1, n // 2, n - 2, n - 1], out_f32=True)
