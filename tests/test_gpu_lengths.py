"""Plans whose segments grow between steps (graphattn_plan_set_lengths: the chains are rebuilt
on the device from new lengths), through the C ABI, against the oracle on the same lengths.

Each graph is built at its final lengths, so every segment owns the pages it will grow into
(page contents past the final lengths are NaN); plans start at shorter lengths and are moved
step by step, across page boundaries and through segment chains.  Bar as for decode and extend
(max |out - oracle| <= 1e-2, max |lse - oracle| <= 1e-3, float32 output requested).
"""
import numpy as np
import pytest
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import graphattn as G
from paper_2606_18954_amd import workloads as W

from gpu_util import compare, params_of, require_gpu, say

pytestmark = pytest.mark.gpu


def _host(g, lens):
    return G.HostGraph(list(int(x) for x in lens), g.seg_page_offsets, g.seg_pages,
                       g.path_offsets, g.path_segs)


def _oracle_decode(wl, lens, pool_bits=None):
    g = wl.graph
    return O.decode(wl.q_bits(), wl.pool_bits() if pool_bits is None else pool_bits,
                    np.asarray(lens, dtype=np.int32), g.seg_page_offsets, g.seg_pages,
                    g.path_offsets, g.path_segs, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
                    wl.dtype)


def _run(plan, q, pool, B, Hq, D):
    out = torch.empty((B, Hq, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, Hq), dtype=torch.float32, device="cuda")
    plan.schedule()
    plan.run(q, pool, out, lse)
    torch.cuda.synchronize()
    return out, lse


def _newest(paths):
    return sorted({p[-1] for p in paths})


# Paths: a shared root, chains of private segments ending in the newest one (3 -> 4), and a
# branch whose newest segment is also its only one.
LENS_MAX = [70, 40, 33, 21, 45, 50, 38]
PATHS = [[0, 1], [0, 2], [0, 3, 4], [5], [0, 6]]


@pytest.mark.parametrize("Hq,Hkv,D,dtype", [(28, 4, 128, "bf16"), (8, 2, 64, "f32")])
def test_newest_segments_grow_across_pages(Hq, Hkv, D, dtype):
    require_gpu()
    g = W.assemble_graph(LENS_MAX, PATHS, 41, 3)
    wl = W.make_workload(f"growing {Hq}/{Hkv}/{D} {dtype}", g, Hq, Hkv, D, dtype, 41, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    newest = _newest(PATHS)
    K = 24                                           # 14..38 tokens: crosses 16 and 32
    lens = np.array(LENS_MAX, dtype=np.int32)
    lens[newest] -= K
    B = g.num_branches
    with G.Plan(_host(g, lens), params_of(wl, out_f32=True)) as plan:
        for k in range(K + 1):
            cur = lens.copy()
            cur[newest] += k
            if k:
                plan.set_lengths(cur)
            out, lse = _run(plan, q, pool, B, Hq, D)
            if k % 4 == 0 or k in (1, 2, 3, K):
                say(f"[case] {wl.name} step {k}: newest lengths {cur[newest].tolist()}")
                oo, ol = _oracle_decode(wl, cur)
                compare(f"{wl.name} step {k}", out.double().cpu().numpy(),
                        lse.double().cpu().numpy(), oo, ol)


def test_any_segment_may_change():
    """Shared and private segments grow and shrink at random within their pages."""
    require_gpu()
    g = W.assemble_graph(LENS_MAX, PATHS, 43, 2)
    wl = W.make_workload("changing 28/4/128 bf16", g, 28, 4, 128, "bf16", 43, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    rng = np.random.default_rng(43)
    B = g.num_branches
    lens = np.array(LENS_MAX, dtype=np.int32)
    with G.Plan(_host(g, lens // 2 + 1), params_of(wl, out_f32=True)) as plan:
        for it in range(6):
            cur = np.array([int(rng.integers(1, m + 1)) for m in LENS_MAX], dtype=np.int32)
            plan.set_lengths(cur)
            out, lse = _run(plan, q, pool, B, 28, 128)
            say(f"[case] random lengths {cur.tolist()}")
            oo, ol = _oracle_decode(wl, cur)
            compare(f"random lengths {it}", out.double().cpu().numpy(),
                    lse.double().cpu().numpy(), oo, ol)


def test_rejected_lengths_leave_the_plan_unchanged():
    require_gpu()
    g = W.assemble_graph(LENS_MAX, PATHS, 44, 2)
    wl = W.make_workload("rejected 8/2/64 f32", g, 8, 2, 64, "f32", 44, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    B = g.num_branches
    lens = np.array(LENS_MAX, dtype=np.int32) - 5
    with G.Plan(_host(g, lens), params_of(wl, out_f32=True)) as plan:
        o1, l1 = _run(plan, q, pool, B, 8, 64)
        over = lens.copy()
        over[2] = 16 * ((LENS_MAX[2] + 15) // 16) + 1          # one token past its pages
        with pytest.raises(G.GraphAttnError) as e:
            plan.set_lengths(over)
        assert e.value.status == G.GA_EINVAL and "owns only" in str(e.value)
        zero = lens.copy()
        zero[0] = 0
        with pytest.raises(G.GraphAttnError) as e:
            plan.set_lengths(zero)
        assert e.value.status == G.GA_EINVAL
        out = torch.empty_like(o1)
        lse = torch.empty_like(l1)
        plan.run(q, pool, out, lse)                            # the old schedule still holds
        torch.cuda.synchronize()
        assert torch.equal(out, o1) and torch.equal(lse, l1)
        plan.set_lengths(lens)                                 # accepted: the schedule is gone
        out.zero_()
        lse.zero_()
        plan.run(q, pool, out, lse)                            # ... and run schedules again
        torch.cuda.synchronize()
        assert torch.equal(out, o1) and torch.equal(lse, l1)   # same lengths, same bits
        o2, l2 = _run(plan, q, pool, B, 8, 64)
        assert torch.equal(o2, o1) and torch.equal(l2, l1)


@pytest.mark.parametrize("Hq,Hkv,D,dtype", [(28, 4, 128, "bf16"), (8, 2, 64, "f32")])
def test_extend_plan_grows_by_its_queries(Hq, Hkv, D, dtype):
    """A multi-query plan: every step appends n_b tokens to each newest segment and queries
    them (the same query rows, new positions)."""
    require_gpu()
    counts = [3, 5, 2, 4, 1]
    steps = 4
    lens_max = list(LENS_MAX)
    g = W.assemble_graph(lens_max, PATHS, 45, 2)
    wl = W.make_extend_workload(f"growing extend {Hq}/{Hkv}/{D} {dtype}", g, counts, Hq, Hkv,
                                D, dtype, 45, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    R = int(np.sum(counts))
    lens = np.array(lens_max, dtype=np.int32)
    for b, p in enumerate(PATHS):
        lens[p[-1]] -= steps * counts[b]
    with G.Plan(_host(g, lens), params_of(wl, out_f32=True), query_counts=counts) as plan:
        for k in range(steps + 1):
            cur = lens.copy()
            for b, p in enumerate(PATHS):
                cur[p[-1]] += k * counts[b]
            if k:
                plan.set_lengths(cur)
            out, lse = _run(plan, q, pool, R, Hq, D)
            oo, ol = O.extend(wl.q_bits(), wl.pool_bits(), cur, g.seg_page_offsets, g.seg_pages,
                              g.path_offsets, g.path_segs, counts, Hq, Hkv, D, dtype)
            say(f"[case] {wl.name} step {k}: newest lengths {[int(cur[p[-1]]) for p in PATHS]}")
            compare(f"{wl.name} step {k}", out.double().cpu().numpy(),
                    lse.double().cpu().numpy(), oo, ol)
        bad = cur.copy()
        bad[PATHS[1][-1]] = counts[1] - 1                      # fewer tokens than queries
        with pytest.raises(G.GraphAttnError) as e:
            plan.set_lengths(bad)
        assert e.value.status == G.GA_EINVAL and "query count" in str(e.value)


def test_decode_loop_append_grow_attend():
    """The decode loop: store each branch's new token in the slot after its newest segment
    (graphattn_kv_append), grow the segment, schedule, attend; 20 steps across page
    boundaries, each against the oracle on the pool as it then is."""
    require_gpu()
    Hq, Hkv, D = 28, 4, 128
    g = W.assemble_graph(LENS_MAX, PATHS, 46, 2)
    wl = W.make_workload("decode loop 28/4/128 bf16", g, Hq, Hkv, D, "bf16", 46, poison=True)
    q, pool = wl.q.cuda(), wl.pool.cuda()
    newest = _newest(PATHS)
    K = 20
    lens = np.array(LENS_MAX, dtype=np.int32)
    lens[newest] -= K
    # the tokens past the starting lengths are overwritten by the appends below
    B = g.num_branches
    gen = torch.Generator().manual_seed(46)
    p = params_of(wl, out_f32=True)
    with G.Plan(_host(g, lens), p) as plan:
        cur = lens.copy()
        for k in range(1, K + 1):
            words = []
            for s in newest:
                t = int(cur[s])                                # slot of the new token
                page = int(g.seg_pages[g.seg_page_offsets[s] + t // 16])
                words.append(page * 16 + t % 16)
            n = len(words)
            kn = torch.randn((n, Hkv, D), generator=gen).to(torch.bfloat16).cuda()
            vn = torch.randn((n, Hkv, D), generator=gen).to(torch.bfloat16).cuda()
            G.kv_append(pool, kn, vn, torch.tensor(words, dtype=torch.int32).cuda(), p)
            cur[newest] += 1
            plan.set_lengths(cur)
            out, lse = _run(plan, q, pool, B, Hq, D)
            if k % 5 == 0 or k == 1:
                say(f"[case] decode loop step {k}: newest lengths {cur[newest].tolist()}")
                pb = pool.cpu().view(torch.int16).numpy().view(np.uint16)
                oo, ol = _oracle_decode(wl, cur, pb)
                compare(f"decode loop step {k}", out.double().cpu().numpy(),
                        lse.double().cpu().numpy(), oo, ol)


def _reschedule_round_trip(wl, seed):
    g = wl.graph
    lens = np.asarray(g.seg_len, dtype=np.int32)
    rng = np.random.default_rng(seed)
    with G.Plan(_host(g, lens), params_of(wl)) as plan:
        plan.schedule()
        first = plan.debug_dump()
        for it in range(3):
            other = np.array([int(rng.integers(1, int(n) + 1)) for n in lens], dtype=np.int32)
            plan.set_lengths(other)
            plan.schedule()
            mid = plan.debug_dump()
            for k in ("group_offsets", "group_branches", "entry_ranks"):
                assert np.array_equal(mid[k], first[k]), (it, k)
            if it == 0:
                assert not np.array_equal(mid["branch_part_offsets"], first["branch_part_offsets"]) \
                    or not np.array_equal(mid["items"], first["items"])
            plan.set_lengths(lens)
            plan.schedule()
            again = plan.debug_dump()
            for k, v in first.items():
                assert v.shape == again[k].shape and np.array_equal(v, again[k]), (it, k)
    say(f"[case] {wl.name}: {len(first['items'])} items, rescheduled 3 times")


def test_rescheduled_plan_matches_its_first_schedule_bit_for_bit():
    """After the first schedule a plan keeps its groups (B(s), the group lists, the entry ranks:
    they follow the paths, which a plan never changes) and recomputes only what the lengths
    decide.  Moving to other lengths (which reorders the work list) and back must give exactly
    the first schedule's arrays, and the groups must not change in between: on the
    single-workgroup scheduler (a merged DAG) and on the multi-kernel one (more than 4096
    segments and branches)."""
    require_gpu()
    _reschedule_round_trip(W.config3_merged_dag(prompts=6), 47)
    rng = np.random.default_rng(7)
    g = W.random_graph(rng, 5000, 4500, 40, 3, seed=1)
    _reschedule_round_trip(W.make_workload("5000-segment graph", g, 28, 4, 64, "bf16", 1), 48)
