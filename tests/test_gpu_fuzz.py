"""Property-based fuzzing of every entry point against the oracle (hypothesis, derandomised so
that a run is reproducible and the failing example is printed).

Attention: small random rollout DAGs (1-6 segments of 1-40 tokens, 1-8 branches over random
duplicate-free segment lists, D in {64, 128}, query heads per kv-head in {1, 4, 5, 7}, bf16 and
float32, random slack pages), decode and multi-query extend, to the parity bar (float32 output
requested: contexts of a few tokens).  State forests: random prompt shapes from chains to stars,
sometimes beyond the 256-state one-workgroup class path and the 512-state one-launch reward
path; classes and edge similarities (inputs kept 1e-3 from kappa), the graph suffix (bit-exact)
and the graph reward and advantages (to fp64 rounding) from random classes.  Plans taken
through random length updates (graphattn_plan_set_lengths) on the same small DAGs.
"""
import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import graphattn as G
from paper_2606_18954_amd import workloads as W

from gpu_util import compare, params_of, require_gpu, say

pytestmark = pytest.mark.gpu

FUZZ = settings(derandomize=True, deadline=None, database=None, print_blob=True,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])


# ---------------------------------------------------------------------------------------------
# Strategies
# ---------------------------------------------------------------------------------------------

@st.composite
def rollout_graphs(draw):
    S = draw(st.integers(1, 6))
    lens = draw(st.lists(st.integers(1, 40), min_size=S, max_size=S))
    B = draw(st.integers(1, 8))
    paths = [draw(st.lists(st.integers(0, S - 1), min_size=1, max_size=S, unique=True))
             for _ in range(B)]
    return lens, paths


heads = st.tuples(st.sampled_from([1, 4, 5, 7]), st.sampled_from([1, 2, 4]),
                  st.sampled_from([64, 128]), st.sampled_from(["bf16", "f32"]))


@st.composite
def forests(draw):
    """Prompts with root first and p(v) < v; a prompt's shape runs from a chain (window 1) to a
    star (window = its size)."""
    seed = draw(st.integers(0, 2 ** 31 - 1))
    sizes = draw(st.lists(st.sampled_from([1, 2, 3, 7, 20, 60, 130, 256, 257, 300, 513]),
                          min_size=1, max_size=4))
    if sum(sizes) > 900:
        sizes = sizes[:1]
    rng = np.random.default_rng(seed)
    parent = []
    for n in sizes:
        base = len(parent)
        window = int(rng.integers(1, n + 1))
        parent.append(-1)
        for v in range(1, n):
            parent.append(base + int(rng.integers(max(0, v - window), v)))
    return np.asarray(parent, dtype=np.int32), seed


def random_classes(parent, rng, n_links):
    """Random classes as the union-find of random pairs from one prompt that are not
    ancestor-related; each label is the smallest member (the form the class kernels write)."""
    N = len(parent)
    root = np.zeros(N, dtype=np.int64)
    for v in range(N):
        root[v] = v if parent[v] < 0 else root[parent[v]]

    def ancestors(v):
        out = set()
        while v >= 0:
            out.add(v)
            v = int(parent[v])
        return out

    lab = np.arange(N, dtype=np.int32)
    for _ in range(n_links):
        u, v = (int(x) for x in rng.integers(0, N, 2))
        if u == v or root[u] != root[v] or u in ancestors(v) or v in ancestors(u):
            continue
        a, b = sorted((int(lab[u]), int(lab[v])))
        lab[lab == b] = a
    return lab


# ---------------------------------------------------------------------------------------------
# Attention
# ---------------------------------------------------------------------------------------------

@settings(FUZZ, max_examples=40)
@given(g=rollout_graphs(), h=heads, slack=st.integers(0, 4), seed=st.integers(0, 2 ** 20))
def test_fuzz_decode(g, h, slack, seed):
    require_gpu()
    lens, paths = g
    group, Hkv, D, dtype = h
    graph = W.assemble_graph(lens, paths, seed, slack)
    wl = W.make_workload(f"fuzz decode {group * Hkv}/{Hkv}/{D} {dtype}", graph, group * Hkv, Hkv,
                         D, dtype, seed, poison=True)
    say(f"[case] {wl.name} lens={lens} paths={paths} slack={slack} seed={seed}")
    q, pool = wl.q.cuda(), wl.pool.cuda()
    out, lse = G.decode(q, pool, G.HostGraph.from_graph(graph), params_of(wl, out_f32=True))
    torch.cuda.synchronize()
    oo, ol = O.decode(wl.q_bits(), wl.pool_bits(), graph.seg_len, graph.seg_page_offsets,
                      graph.seg_pages, graph.path_offsets, graph.path_segs, wl.num_q_heads,
                      wl.num_kv_heads, D, dtype)
    compare(wl.name, out.double().cpu().numpy(), lse.double().cpu().numpy(), oo, ol)


@settings(FUZZ, max_examples=30)
@given(g=rollout_graphs(), h=heads, slack=st.integers(0, 3), seed=st.integers(0, 2 ** 20),
       data=st.data())
def test_fuzz_extend(g, h, slack, seed, data):
    require_gpu()
    lens, paths = g
    group, Hkv, D, dtype = h
    B = len(paths)
    step = data.draw(st.lists(st.integers(1, 40), min_size=B, max_size=B))
    counts = [data.draw(st.integers(1, n)) for n in step]
    use_plan = data.draw(st.booleans())
    lens, paths = W.with_new_steps(lens, paths, step)
    graph = W.assemble_graph(lens, paths, seed, slack)
    wl = W.make_extend_workload(f"fuzz extend {group * Hkv}/{Hkv}/{D} {dtype}", graph, counts,
                                group * Hkv, Hkv, D, dtype, seed, poison=True)
    say(f"[case] {wl.name} lens={lens} paths={paths} counts={counts} slack={slack} "
        f"seed={seed} plan={use_plan}")
    q, pool = wl.q.cuda(), wl.pool.cuda()
    hg = G.HostGraph.from_graph(graph)
    p = params_of(wl, out_f32=True)
    if use_plan:
        R = int(np.sum(counts))
        out = torch.empty((R, wl.num_q_heads, D), dtype=torch.float32, device="cuda")
        lse = torch.empty((R, wl.num_q_heads), dtype=torch.float32, device="cuda")
        with G.Plan(hg, p, query_counts=wl.query_counts) as pl:
            pl.schedule()
            pl.run(q, pool, out, lse)
            torch.cuda.synchronize()
    else:
        out, lse = G.extend(q, pool, hg, wl.query_counts, p)
        torch.cuda.synchronize()
    oo, ol = O.extend(wl.q_bits(), wl.pool_bits(), graph.seg_len, graph.seg_page_offsets,
                      graph.seg_pages, graph.path_offsets, graph.path_segs, wl.query_counts,
                      wl.num_q_heads, wl.num_kv_heads, D, dtype)
    compare(wl.name, out.double().cpu().numpy(), lse.double().cpu().numpy(), oo, ol)


# ---------------------------------------------------------------------------------------------
# State forests
# ---------------------------------------------------------------------------------------------

@settings(FUZZ, max_examples=25)
@given(f=forests(), dim=st.sampled_from([64, 128, 256]), share=st.sampled_from([0.5, 1.0, 3.0]),
       kappa=st.floats(0.3, 0.99))
def test_fuzz_classes_and_edge_similarities(f, dim, share, kappa):
    require_gpu()
    parent, seed = f
    N = len(parent)
    z = W.draw_state_embeddings(parent, dim, seed, share=share)
    zb = z.view(torch.int16).numpy().view(np.uint16)
    m = O.similarity_margin(zb, "bf16", parent, kappa)
    if m < 1e-3:                                   # the decision is within rounding of kappa
        kappa = min(0.999, kappa + 2e-3)
        m = O.similarity_margin(zb, "bf16", parent, kappa)
    say(f"[case] fuzz classes N={N} dim={dim} share={share} kappa={kappa:.4f} seed={seed} "
        f"margin={m:.2e}")
    if m < 1e-3:
        return
    ref = O.equivalence_classes(zb, "bf16", parent, kappa)
    with G.Forest(parent) as fo:
        es = torch.empty(N, dtype=torch.float32, device="cuda")
        lab = fo.classes(z.cuda(), kappa, edge_sim=es)
        torch.cuda.synchronize()
        assert np.array_equal(lab.cpu().numpy(), ref)
        got = es.cpu().numpy().astype(np.float64)
    for v in range(N):
        if parent[v] >= 0:
            assert abs(got[v] - O.cosine(zb, "bf16", int(parent[v]), v)) <= 3e-4, v


@settings(FUZZ, max_examples=25)
@given(f=forests(), links=st.integers(0, 400), w=st.sampled_from([0.0, 0.3, 1.0]),
       lam=st.sampled_from([0.0, 0.5, 2.0]))
def test_fuzz_suffix_and_advantages(f, links, w, lam):
    require_gpu()
    parent, seed = f
    N = len(parent)
    rng = np.random.default_rng(seed + 1)
    lab = random_classes(parent, rng, links)
    reward = W.state_rewards(parent, seed)
    sim = rng.uniform(-1.0, 1.0, N).astype(np.float32)
    say(f"[case] fuzz suffix/advantages N={N} links={links} "
        f"classes={len(set(lab.tolist()))} w={w} lam={lam} seed={seed}")
    ro, rs = O.graph_suffix(lab, parent)
    ref = O.graph_advantages(parent, lab, reward, sim.astype(np.float64), w, lam)
    with G.Forest(parent) as fo:
        lab_d = torch.from_numpy(lab).cuda()
        offs = torch.empty(N + 1, dtype=torch.int64, device="cuda")
        total = fo.suffix_total(lab_d, offs)
        states = torch.empty(max(1, total), dtype=torch.int32, device="cuda")
        assert fo.suffix(lab_d, offs, states) == total == len(rs)
        out = fo.advantages(lab_d, torch.from_numpy(reward).cuda(), torch.from_numpy(sim).cuda(),
                            w, lam)
        torch.cuda.synchronize()
        assert np.array_equal(offs.cpu().numpy(), ro)
        assert np.array_equal(states[:total].cpu().numpy(), rs)
        for k, g in [("S", "score"), ("r", "step_reward"), ("A_cor", "a_cor"),
                     ("A_eff", "a_eff"), ("A_dual", "a_dual")]:
            a, b = out[g].cpu().numpy(), ref[k]
            assert np.array_equal(np.isnan(a), np.isnan(b)), k
            mk = ~np.isnan(b)
            err = float(np.abs(a[mk] - b[mk]).max()) if mk.any() else 0.0
            assert err <= 1e-9 * max(1.0, float(np.abs(b[mk]).max()) if mk.any() else 1.0), \
                (k, err)


@settings(FUZZ, max_examples=20)
@given(g=rollout_graphs(), h=heads, seed=st.integers(0, 2 ** 20), data=st.data())
def test_fuzz_set_lengths(g, h, seed, data):
    """A plan created at random lengths within each segment's pages, then given three random
    sets of lengths (graphattn_plan_set_lengths), each scheduled, run and compared."""
    require_gpu()
    lens_max, paths = g
    group, Hkv, D, dtype = h
    graph = W.assemble_graph(lens_max, paths, seed, 1)
    wl = W.make_workload(f"fuzz lengths {group * Hkv}/{Hkv}/{D} {dtype}", graph, group * Hkv,
                         Hkv, D, dtype, seed, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    draws = [[data.draw(st.integers(1, m)) for m in lens_max] for _ in range(4)]
    B, Hq = graph.num_branches, wl.num_q_heads
    hg = G.HostGraph(draws[0], graph.seg_page_offsets, graph.seg_pages, graph.path_offsets,
                     graph.path_segs)
    with G.Plan(hg, params_of(wl, out_f32=True)) as plan:
        for i, lens in enumerate(draws):
            if i:
                plan.set_lengths(lens)
            say(f"[case] {wl.name} max={lens_max} lengths={lens} paths={paths} seed={seed}")
            out = torch.empty((B, Hq, D), dtype=torch.float32, device="cuda")
            lse = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
            plan.schedule()
            plan.run(q, pool, out, lse)
            torch.cuda.synchronize()
            oo, ol = O.decode(wl.q_bits(), wl.pool_bits(), np.asarray(lens, dtype=np.int32),
                              graph.seg_page_offsets, graph.seg_pages, graph.path_offsets,
                              graph.path_segs, Hq, Hkv, D, dtype)
            compare(wl.name, out.double().cpu().numpy(), lse.double().cpu().numpy(), oo, ol)
