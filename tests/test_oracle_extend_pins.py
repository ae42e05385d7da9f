"""Pins of the oracle's extend (several causal queries per branch), K/V append and K/V copy.

Each check takes the oracle module, so the planted-mistake test at the bottom can swap a piece of
the oracle for a plausible wrong one (on the CPU) and confirm that some pin fails.
"""
import math

import numpy as np
import pytest
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import workloads as W


def _scatter(g, K, V, Hkv, D):
    """Write a contiguous K/V sequence into the graph's pages, segment after segment."""
    pool = np.full((g.num_pages, Hkv, 2, 16, D), np.nan, dtype=np.float32)
    t0 = 0
    for s in range(g.num_segments):
        for t in range(int(g.seg_len[s])):
            page = g.seg_pages[g.seg_page_offsets[s] + t // 16]
            pool[page, :, 0, t % 16] = K[t0 + t]
            pool[page, :, 1, t % 16] = V[t0 + t]
        t0 += int(g.seg_len[s])
    return pool


def _extend(mod, g, q, pool, counts, Hq, Hkv, D, dtype="f32"):
    return mod.extend(q, pool, g.seg_len, g.seg_page_offsets, g.seg_pages, g.path_offsets,
                      g.path_segs, counts, Hq, Hkv, D, dtype)


def _tree_with_private_leaves(rng, seed, n_branches=5):
    """A small tree: a root, two shared steps, and one private newest segment per branch."""
    lens = [int(rng.integers(1, 40)) for _ in range(3)]
    paths = []
    for b in range(n_branches):
        lens.append(int(rng.integers(1, 45)))
        paths.append([0, 1 + b % 2, len(lens) - 1] if b % 3 else [0, len(lens) - 1])
    return W.assemble_graph(lens, paths, seed, slack_pages=2)


def check_extend_is_causal_sdpa(mod, seed=21):
    """One branch: its queries are the last n rows of ordinary causal self-attention over the
    whole context (torch SDPA, float64, is_causal, GQA)."""
    rng = np.random.default_rng(seed)
    for Hq, Hkv, D in [(8, 2, 64), (28, 4, 128), (3, 3, 16)]:
        lens = [int(x) for x in rng.integers(1, 60, size=3)]
        g = W.assemble_graph(lens, [[0, 1, 2]], seed, slack_pages=2)
        L = sum(lens)
        K = rng.standard_normal((L, Hkv, D)).astype(np.float32)
        V = rng.standard_normal((L, Hkv, D)).astype(np.float32)
        pool = _scatter(g, K, V, Hkv, D)
        Qall = rng.standard_normal((L, Hq, D)).astype(np.float32)
        qt = torch.from_numpy(Qall).double().permute(1, 0, 2).unsqueeze(0)   # [1, Hq, L, D]
        Kt = torch.from_numpy(K).double().permute(1, 0, 2).unsqueeze(0)
        Vt = torch.from_numpy(V).double().permute(1, 0, 2).unsqueeze(0)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, is_causal=True,
                                                                enable_gqa=True)[0]
        ref = ref.permute(1, 0, 2).numpy()                                     # [L, Hq, D]
        Kx = Kt.repeat_interleave(Hq // Hkv, dim=1)
        z = (qt @ Kx.transpose(-1, -2))[0] / math.sqrt(D)                      # [Hq, L, L]
        z = z.masked_fill(torch.ones(L, L, dtype=torch.bool).triu(1), -math.inf)
        ref_lse = torch.logsumexp(z, dim=-1).T.numpy()                         # [L, Hq]
        for n in sorted({1, lens[2], max(1, lens[2] // 2)}):
            out, lse = _extend(mod, g, Qall[L - n:], pool, [n], Hq, Hkv, D)
            assert np.allclose(out, ref[L - n:], rtol=0, atol=1e-12), (Hq, n)
            assert np.allclose(lse, ref_lse[L - n:], rtol=0, atol=1e-12), (Hq, n)


def check_extend_brute_force(mod, seed=22):
    """Token-by-token walk of the page table with Python floats: query i of branch b sees every
    token of the earlier path segments and tokens 0 .. len - n + i of the last one."""
    rng = np.random.default_rng(seed)
    for trial in range(3):
        g = _tree_with_private_leaves(rng, seed + trial, n_branches=4)
        Hq, Hkv, D = 4, 2, 4
        counts = [int(rng.integers(1, g.seg_len[g.path(b)[-1]] + 1))
                  for b in range(g.num_branches)]
        _, pool = W.draw_data(g, Hq, Hkv, D, "f32", seed + trial)
        pool = pool.numpy() * 0.5
        q = rng.standard_normal((sum(counts), Hq, D)).astype(np.float32) * 0.5
        out, lse = _extend(mod, g, q, pool, counts, Hq, Hkv, D)
        scale = 1.0 / math.sqrt(D)
        row = 0
        for b in range(g.num_branches):
            path = g.path(b)
            last_len = int(g.seg_len[path[-1]])
            for i in range(counts[b]):
                for h in range(Hq):
                    kv = h // (Hq // Hkv)
                    ws, vs = [], []
                    for s in path:
                        n_tok = int(g.seg_len[s])
                        if s == path[-1]:
                            n_tok = last_len - counts[b] + i + 1
                        for t in range(n_tok):
                            page = int(g.seg_pages[g.seg_page_offsets[s] + t // 16])
                            k = [float(x) for x in pool[page, kv, 0, t % 16]]
                            z = scale * math.fsum(float(q[row, h, d]) * k[d] for d in range(D))
                            ws.append(math.exp(z))
                            vs.append([float(x) for x in pool[page, kv, 1, t % 16]])
                    tot = math.fsum(ws)
                    ref = [math.fsum(w * v[d] for w, v in zip(ws, vs)) / tot for d in range(D)]
                    assert np.allclose(out[row, h], ref, rtol=0, atol=1e-12), (b, i, h)
                    assert abs(lse[row, h] - math.log(tot)) < 1e-12
                row += 1


def check_extend_single_query_is_decode(mod, seed=23):
    """With one query per branch, the query is the context's last token and sees it all."""
    rng = np.random.default_rng(seed)
    g = _tree_with_private_leaves(rng, seed, n_branches=6)
    q, pool = W.draw_data(g, 8, 2, 64, "f32", seed)
    q, pool = q.numpy(), pool.numpy()
    out, lse = _extend(mod, g, q, pool, [1] * g.num_branches, 8, 2, 64)
    ref, ref_lse = mod.decode(q, pool, g.seg_len, g.seg_page_offsets, g.seg_pages,
                              g.path_offsets, g.path_segs, 8, 2, 64, "f32")
    assert np.allclose(out, ref, rtol=0, atol=1e-12)
    assert np.allclose(lse, ref_lse, rtol=0, atol=1e-12)


def check_append_then_read(mod, seed=24):
    """Appending a segment's tokens to its page slots and reading the segment back returns
    exactly the appended bits; every other slot keeps its bits; padding words are skipped."""
    rng = np.random.default_rng(seed)
    g = W.assemble_graph([37, 5, 16], [[0, 1], [0, 2]], seed, slack_pages=3)
    Hkv, D = 2, 8
    for dtype in ("f32", "bf16"):
        if dtype == "f32":
            pool = rng.standard_normal((g.num_pages, Hkv, 2, 16, D)).astype(np.float32)
            kn = rng.standard_normal((37, Hkv, D)).astype(np.float32)
            vn = rng.standard_normal((37, Hkv, D)).astype(np.float32)
        else:
            pool = rng.integers(0, 0x7F00, size=(g.num_pages, Hkv, 2, 16, D), dtype=np.uint16)
            kn = rng.integers(0, 0x7F00, size=(37, Hkv, D), dtype=np.uint16)
            vn = rng.integers(0, 0x7F00, size=(37, Hkv, D), dtype=np.uint16)
        off = int(g.seg_page_offsets[0])
        words = [int(g.seg_pages[off + t // 16]) * 16 + t % 16 for t in range(37)]
        pad = [-1, -16, g.num_pages * 16, 2 ** 31 - 1]
        at = sorted(rng.choice(38, size=len(pad), replace=False))
        words_p, kn_p, vn_p = list(words), list(kn), list(vn)
        for j, w in zip(at, pad):
            words_p.insert(j, w)
            kn_p.insert(j, kn[0] * 0 + 1)
            vn_p.insert(j, vn[0] * 0 + 1)
        new = mod.kv_append(pool, np.array(kn_p), np.array(vn_p), words_p)
        k, v = mod.segment_tokens(new, dtype, g.seg_len, g.seg_page_offsets, g.seg_pages, 0)
        assert np.array_equal(k, mod.to_f64(kn, dtype)) and np.array_equal(v, mod.to_f64(vn, dtype))
        flat_new = new.transpose(0, 3, 1, 2, 4).reshape(g.num_pages * 16, -1)
        flat_old = pool.transpose(0, 3, 1, 2, 4).reshape(g.num_pages * 16, -1)
        keep = np.setdiff1d(np.arange(g.num_pages * 16), words)
        assert np.array_equal(flat_new[keep], flat_old[keep])


def check_split_by_copy_keeps_attention(mod, seed=25):
    """Cutting a segment inside a page and moving the tail to a fresh page with kv_copy leaves
    every branch's decode result unchanged (attention over a partition of the same tokens)."""
    rng = np.random.default_rng(seed)
    for cut in (1, 7, 16, 23, 40):
        g = W.assemble_graph([20, 41], [[0, 1]], seed, slack_pages=6)
        Hq, Hkv, D = 4, 2, 16
        q, pool = W.draw_data(g, Hq, Hkv, D, "f32", seed)
        q, pool = q.numpy(), pool.numpy()
        ref, ref_lse = mod.decode(q, pool, g.seg_len, g.seg_page_offsets, g.seg_pages,
                                  g.path_offsets, g.path_segs, Hq, Hkv, D, "f32")
        used = set(int(p) for p in g.seg_pages)
        free = [p for p in range(g.num_pages) if p not in used]
        n2 = 41 - cut
        npg2 = (n2 + 15) // 16
        off = int(g.seg_page_offsets[1])
        src = [int(g.seg_pages[off + t // 16]) * 16 + t % 16 for t in range(cut, 41)]
        dst = [free[t // 16] * 16 + t % 16 for t in range(n2)]
        new = mod.kv_copy(pool, src, dst)
        seg_len = np.array([20, cut, n2], dtype=np.int32)
        pages = np.concatenate([g.seg_pages[:off + (cut + 15) // 16],
                                np.array(free[:npg2], dtype=np.int32)])
        offs = np.array([0, off, off + (cut + 15) // 16, len(pages)], dtype=np.int64)
        out, lse = mod.decode(q, new, seg_len, offs, pages, np.array([0, 3], dtype=np.int64),
                              np.array([0, 1, 2], dtype=np.int32), Hq, Hkv, D, "f32")
        assert np.allclose(out, ref, rtol=0, atol=1e-12) and np.allclose(lse, ref_lse, atol=1e-12)


PINS = [check_extend_is_causal_sdpa, check_extend_brute_force, check_extend_single_query_is_decode,
        check_append_then_read, check_split_by_copy_keeps_attention]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_extend_pin(pin):
    pin(O)


def test_oracle_rejects_bad_extend_and_copy_inputs():
    g = W.assemble_graph([5, 3], [[0, 1]], 1, slack_pages=1)
    q, pool = W.draw_data(g, 2, 1, 4, "f32", 1)
    with pytest.raises(ValueError):
        _extend(O, g, np.zeros((4, 2, 4), np.float32), pool.numpy(), [4], 2, 1, 4)
    with pytest.raises(ValueError):
        _extend(O, g, np.zeros((0, 2, 4), np.float32), pool.numpy(), [0], 2, 1, 4)
    with pytest.raises(ValueError):
        O.kv_copy(pool.numpy(), [0, 1], [1, 2])
    with pytest.raises(ValueError):
        O.kv_append(pool.numpy(), np.zeros((2, 1, 4)), np.zeros((2, 1, 4)), [3, 3])


ORIG_QCL = O.query_context_length
ORIG_APPEND = O.kv_append
ORIG_COPY = O.kv_copy


@pytest.mark.parametrize("name,attr,repl", [
    ("excludes_itself", "query_context_length", lambda L, n, i: ORIG_QCL(L, n, i) - 1),
    ("sees_one_ahead", "query_context_length", lambda L, n, i: min(L, ORIG_QCL(L, n, i) + 1)),
    ("reversed_queries", "query_context_length", lambda L, n, i: ORIG_QCL(L, n, n - 1 - i)),
    ("k_v_swapped", "kv_append", lambda p, k, v, w: ORIG_APPEND(p, v, k, w)),
    ("copy_reversed", "kv_copy", lambda p, s, d: ORIG_COPY(p, d, s)),
])
def test_planted_mistake_is_caught(monkeypatch, name, attr, repl):
    monkeypatch.setattr(O, attr, repl)
    caught = False
    for pin in PINS:
        try:
            pin(O)
        except (AssertionError, IndexError, ValueError):
            caught = True
            break
    assert caught, f"planted mistake {name} went unnoticed"
