"""Parity of multi-query attention (graphattn_extend, through the C ABI) and of the page-pool
writes (graphattn_kv_append / graphattn_kv_copy) with the fp64 CPU oracle on seeded inputs.

Attention bar as for decode: max |out - oracle| <= 1e-2, max |lse - oracle| <= 1e-3 (float32
output requested where contexts are a few tokens, so that the comparison measures the kernels
and not the final bf16 rounding).  Page writes are byte moves: bit-exact.
"""
import numpy as np
import pytest
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import graphattn as G
from paper_2606_18954_amd import workloads as W

from gpu_util import compare, params_of, require_gpu, say

pytestmark = pytest.mark.gpu


def _wl(lens, paths, counts, Hq, Hkv, D, dtype, seed, slack=3):
    g = W.assemble_graph(lens, paths, seed, slack)
    return W.make_extend_workload(f"extend {Hq}/{Hkv}/{D} {dtype} S={len(lens)} B={len(paths)} "
                                  f"R={int(np.sum(counts))}", g, counts, Hq, Hkv, D, dtype, seed,
                                  poison=True)


def gpu_extend(wl, out_f32=False, plan=False):
    require_gpu()
    q, pool = wl.q.cuda(), wl.pool.cuda()
    hg = G.HostGraph.from_graph(wl.graph)
    p = params_of(wl, out_f32=out_f32)
    if plan:
        R = int(wl.query_counts.sum())
        out = torch.empty((R, wl.num_q_heads, wl.head_dim),
                          dtype=torch.float32 if out_f32 else q.dtype, device="cuda")
        lse = torch.empty((R, wl.num_q_heads), dtype=torch.float32, device="cuda")
        with G.Plan(hg, p, query_counts=wl.query_counts) as pl:
            assert pl.info().num_query_rows == R
            assert pl.info().num_branches == wl.graph.num_branches
            pl.schedule()
            pl.run(q, pool, out, lse)
            torch.cuda.synchronize()
    else:
        out, lse = G.extend(q, pool, hg, wl.query_counts, p)
        torch.cuda.synchronize()
    return out.double().cpu().numpy(), lse.double().cpu().numpy()


def oracle_extend(wl, rows=None):
    g = wl.graph
    return O.extend(wl.q_bits(), wl.pool_bits(), g.seg_len, g.seg_page_offsets, g.seg_pages,
                    g.path_offsets, g.path_segs, wl.query_counts, wl.num_q_heads,
                    wl.num_kv_heads, wl.head_dim, wl.dtype, rows=rows)


def check(wl, rows=None, out_f32=True, plan=False):
    say(f"[case] {wl.name} rows={'all' if rows is None else len(rows)} plan={plan}")
    go, gl = gpu_extend(wl, out_f32=out_f32, plan=plan)
    oo, ol = oracle_extend(wl, rows)
    if rows is not None:
        go, gl = go[rows], gl[rows]
    return compare(wl.name, go, gl, oo, ol)


def _tree(rng, n_branches, max_step, max_new):
    lens = [int(rng.integers(1, 300))] + [int(rng.integers(1, max_step)) for _ in range(4)]
    paths = []
    for b in range(n_branches):
        paths.append([0] + ([1 + b % 2] if b % 3 else []) + ([3 + b % 2] if b % 4 == 1 else []))
    step = [int(rng.integers(1, max_new)) for _ in range(n_branches)]
    lens, paths = W.with_new_steps(lens, paths, step)
    counts = [int(rng.integers(1, n + 1)) for n in step]
    return lens, paths, counts


@pytest.mark.parametrize("Hq,Hkv,D,dtype", [(28, 4, 128, "bf16"), (8, 2, 64, "f32"),
                                            (40, 8, 128, "bf16"), (4, 4, 64, "bf16"),
                                            (6, 3, 64, "bf16"), (24, 6, 128, "bf16"),
                                            (8, 1, 64, "bf16")])
def test_extend_tree(Hq, Hkv, D, dtype):
    """Causal trees at several head shapes, so that the causal kernel's work streams (one per
    kv-head up to gcd(Hkv, 8)) run with 8, 4, 2 and 1 streams, the last with the rotated stage
    order of single-stream launches."""
    rng = np.random.default_rng(Hq + D)
    lens, paths, counts = _tree(rng, 7, 90, 70)
    wl = _wl(lens, paths, counts, Hq, Hkv, D, dtype, Hq + D)
    with G.Plan(G.HostGraph.from_graph(wl.graph), params_of(wl),
                query_counts=wl.query_counts) as pl:
        assert pl.info().work_streams == max(s for s in (8, 4, 2, 1) if Hkv % s == 0)
    check(wl)


def test_extend_prompt_prefill_spans_chunks():
    """A bare prompt prefilled in full: one causal segment of 700 tokens, cut into page chunks,
    so the rows of early queries see nothing of the later chunks (empty partials)."""
    for dtype, Hq, Hkv, D in [("bf16", 28, 4, 128), ("f32", 8, 2, 64)]:
        wl = _wl([700], [[0]], [700], Hq, Hkv, D, dtype, 31)
        hg = G.HostGraph.from_graph(wl.graph)
        with G.Plan(hg, params_of(wl), query_counts=wl.query_counts) as pl:
            assert pl.info().chunk_pages < 44            # several chunks of the 44 pages
        rows = list(range(0, 700, 7)) + [1, 2, 255, 256, 257, 511, 512, 513, 699]
        check(wl, rows=sorted(set(rows)))


def test_extend_partial_query_counts_and_chains():
    """The newest segment follows private segments (one chain with ragged pages) and only its
    last tokens are queries: the causal origin sits pages into the chain."""
    lens = [40, 17, 3, 33, 16, 21, 50, 9]
    paths = [[0, 1, 2, 3], [0, 4, 5], [0, 1, 6], [7]]
    counts = [20, 21, 1, 9]
    for dtype, Hq, Hkv, D in [("bf16", 28, 4, 128), ("f32", 8, 2, 64)]:
        check(_wl(lens, paths, counts, Hq, Hkv, D, dtype, 32))
        check(_wl(lens, paths, counts, Hq, Hkv, D, dtype, 33), plan=True)


def test_extend_one_query_is_decode():
    """One query per branch: extend runs the decode problem and must give the same bits."""
    rng = np.random.default_rng(5)
    lens, paths, _ = _tree(rng, 9, 200, 90)
    g = W.assemble_graph(lens, paths, 34, 2)
    wl = W.make_workload("decode twin", g, 28, 4, 128, "bf16", 34, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    hg = G.HostGraph.from_graph(g)
    od, ld = G.decode(q, pool, hg, params_of(wl))
    oe, le = G.extend(q, pool, hg, [1] * g.num_branches, params_of(wl))
    torch.cuda.synchronize()
    assert torch.equal(od.view(torch.int16), oe.view(torch.int16))
    assert torch.equal(ld, le)


def test_extend_many_rows_large_scheduler():
    """40 branches x 128 queries over a shared prompt: 5120 query rows (beyond the one-workgroup
    scheduler), the prompt's group of 35840 rows split into 280 row blocks; sampled rows."""
    lens = [900] + [128] * 40
    paths = [[0, 1 + b] for b in range(40)]
    wl = _wl(lens, paths, [128] * 40, 28, 4, 128, "bf16", 35)
    rows = sorted(set(np.random.default_rng(35).choice(5120, 120, replace=False).tolist()
                      + [0, 127, 128, 5119]))
    check(wl, rows=rows, out_f32=False, plan=True)


def test_extend_merged_dag_sampled():
    """The merged-DAG rollout with a 16-token step per branch (4 prompts), sampled rows."""
    wl = W.config3_extend(prompts=4, poison=True, slack_pages=7)
    R = int(wl.query_counts.sum())
    rows = sorted(np.random.default_rng(36).choice(R, 150, replace=False).tolist())
    check(wl, rows=rows, out_f32=False, plan=True)


def test_extend_full_size_sampled():
    """The 16-token extend of the full merged-DAG rollout (1024 branches, 16384 query rows) in
    the launch configuration the benchmark times; sampled rows."""
    wl = W.config3_extend()
    R = int(wl.query_counts.sum())
    rows = sorted(np.random.default_rng(37).choice(R, 48, replace=False).tolist())
    check(wl, rows=rows, out_f32=False, plan=True)


def test_extend_full_size_runs_are_bit_identical():
    """The full 16-token extend scheduled and run twice on one plan, and once more from a fresh
    plan with kernel timing on (the causal kernel and the merge launched with their dispatch-
    bound events): the work streams hand units to whichever workgroup claims them first (and
    workgroups whose stream is empty claim from the others), but every unit's partial depends
    only on the unit, so all three runs give the same bits."""
    require_gpu()
    wl = W.config3_extend()
    q, pool = wl.q.cuda(), wl.pool.cuda()
    hg = G.HostGraph.from_graph(wl.graph)
    p = params_of(wl)
    R = int(wl.query_counts.sum())
    say(f"[case] full-size extend determinism: R={R}")

    def run(pl):
        out = torch.empty((R, wl.num_q_heads, wl.head_dim), dtype=q.dtype, device="cuda")
        lse = torch.empty((R, wl.num_q_heads), dtype=torch.float32, device="cuda")
        pl.schedule()
        pl.run(q, pool, out, lse)
        torch.cuda.synchronize()
        return out.view(torch.int16).cpu(), lse.cpu()

    with G.Plan(hg, p, query_counts=wl.query_counts) as pl:
        o1, l1 = run(pl)
        o2, l2 = run(pl)
    with G.Plan(hg, p, query_counts=wl.query_counts) as pl:
        pl.profile(1)
        o3, l3 = run(pl)
        pr = pl.profile_read()
        assert (pr.schedules, pr.runs) == (1, 1) and pr.attn_ms > 0.0 and pr.merge_ms > 0.0
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert torch.equal(o1, o3) and torch.equal(l1, l3)


# ---------------------------------------------------------------------------------------------
# Page-pool writes
# ---------------------------------------------------------------------------------------------

def _pool_and_rows(Np, Hkv, D, dtype, n, seed):
    gen = torch.Generator().manual_seed(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    pool = torch.randn((Np, Hkv, 2, 16, D), generator=gen).to(tdt)
    k = torch.randn((n, Hkv, D), generator=gen).to(tdt)
    v = torch.randn((n, Hkv, D), generator=gen).to(tdt)
    return pool, k, v


def _raw(t):
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()


@pytest.mark.parametrize("Hkv,D,dtype", [(4, 128, "bf16"), (2, 64, "f32"), (8, 64, "bf16")])
def test_kv_append_bit_exact(Hkv, D, dtype):
    require_gpu()
    Np, n = 40, 300
    pool, k, v = _pool_and_rows(Np, Hkv, D, dtype, n, Hkv + D)
    rng = np.random.default_rng(Hkv + D)
    words = rng.choice(Np * 16, n, replace=False).astype(np.int32)
    words[[3, 77, 150]] = [-1, Np * 16, 2 ** 31 - 1]          # skipped
    say(f"[case] kv_append Hkv={Hkv} D={D} {dtype} n={n}")
    ref = O.kv_append(_raw(pool), _raw(k), _raw(v), words)
    p = G.make_params(Hkv, Hkv, D, Np, dtype)
    pg = pool.cuda()
    G.kv_append(pg, k.cuda(), v.cuda(), torch.from_numpy(words).cuda(), p)
    torch.cuda.synchronize()
    assert np.array_equal(_raw(pg.cpu()), ref)


@pytest.mark.parametrize("Hkv,D,dtype", [(4, 128, "bf16"), (2, 64, "f32")])
def test_kv_copy_bit_exact(Hkv, D, dtype):
    require_gpu()
    Np = 30
    pool, _, _ = _pool_and_rows(Np, Hkv, D, dtype, 1, 7 + D)
    rng = np.random.default_rng(D)
    perm = rng.permutation(Np * 16).astype(np.int32)
    src, dst = perm[:150].copy(), perm[150:300].copy()
    src[5], dst[9] = -3, Np * 16                               # pairs skipped
    say(f"[case] kv_copy Hkv={Hkv} D={D} {dtype}")
    ref = O.kv_copy(_raw(pool), src, dst)
    p = G.make_params(Hkv, Hkv, D, Np, dtype)
    pg = pool.cuda()
    G.kv_copy(pg, torch.from_numpy(src).cuda(), torch.from_numpy(dst).cuda(), p)
    torch.cuda.synchronize()
    assert np.array_equal(_raw(pg.cpu()), ref)


def test_append_then_extend():
    """A decode step's bookkeeping on the GPU: the new step's K/V are appended into fresh pages
    (into a pool whose free pages hold NaN), then extend attends over them; checked against the
    oracle run on the oracle's own append."""
    require_gpu()
    lens = [300, 45, 60]
    paths = [[0, 1], [0, 2]]
    new = [37, 16]
    lens2, paths2 = W.with_new_steps(lens, paths, new)
    g = W.assemble_graph(lens2, paths2, 38, 2)
    wl = W.make_extend_workload("append then extend", g, new, 28, 4, 128, "bf16", 38,
                                poison=True)
    gen = torch.Generator().manual_seed(38)
    kn = torch.randn((sum(new), 4, 128), generator=gen).to(torch.bfloat16)
    vn = torch.randn((sum(new), 4, 128), generator=gen).to(torch.bfloat16)
    words = []
    for s in (3, 4):
        off = int(g.seg_page_offsets[s])
        words += [int(g.seg_pages[off + t // 16]) * 16 + t % 16 for t in range(int(g.seg_len[s]))]
    words = np.array(words, dtype=np.int32)
    pool_ref = O.kv_append(wl.pool_bits(), _raw(kn), _raw(vn), words)
    p = params_of(wl)
    pg = wl.pool.cuda()
    G.kv_append(pg, kn.cuda(), vn.cuda(), torch.from_numpy(words).cuda(), p)
    out, lse = G.extend(wl.q.cuda(), pg, G.HostGraph.from_graph(g), new, p)
    torch.cuda.synchronize()
    oo, ol = O.extend(wl.q_bits(), pool_ref, g.seg_len, g.seg_page_offsets, g.seg_pages,
                      g.path_offsets, g.path_segs, new, 28, 4, 128, "bf16")
    compare("append then extend", out.double().cpu().numpy(), lse.double().cpu().numpy(), oo, ol)


def test_kv_append_replayed_from_a_graph():
    """Append calls captured in a HIP graph: each replay (after eager work that restores the
    pool) must store exactly what the eager call stores."""
    require_gpu()
    Np, n, Hkv, D = 24, 200, 4, 128
    pool, k, v = _pool_and_rows(Np, Hkv, D, "bf16", n, 41)
    words = np.random.default_rng(41).choice(Np * 16, n, replace=False).astype(np.int32)
    ref = O.kv_append(_raw(pool), _raw(k), _raw(v), words)
    p = G.make_params(Hkv, Hkv, D, Np, "bf16")
    pg, kg, vg = pool.cuda(), k.cuda(), v.cuda()
    wd = torch.from_numpy(words).cuda()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(graph, stream=side):
            G.kv_append(pg, kg, vg, wd, p)
    torch.cuda.current_stream().wait_stream(side)
    orig = pool.cuda()
    for rep in range(3):
        pg.copy_(orig)                       # eager work between replays
        torch.cuda.synchronize()
        assert not np.array_equal(_raw(pg.cpu()), ref)
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_raw(pg.cpu()), ref), rep
