"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each check is a plain function taking the oracle module, so the mutation tests at the bottom can
plant a plausible mistake in the oracle (on the CPU) and confirm that some pin fails.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")



def _decode(mod, g, q, pool, Hq, Hkv, D, dtype="f32", scale=None, branches=None):
    return mod.decode(q, pool, g.seg_len, g.seg_page_offsets, g.seg_pages, g.path_offsets,
                      g.path_segs, Hq, Hkv, D, dtype, scale=scale, branches=branches)


# ---------------------------------------------------------------------------------------------
# Pins
# ---------------------------------------------------------------------------------------------

def check_bf16_decoding(mod):
    known = {0x3F80: 1.0, 0xC000: -2.0, 0x3F81: 1.0078125, 0x0001: 2.0 ** -133,
             0x7F7F: 3.3895313892515355e38, 0x8000: -0.0, 0x4049: 3.140625}
    got = mod.bf16_bits_to_f64(np.array(list(known), dtype=np.uint16))
    assert np.array_equal(got, np.array(list(known.values())))
    bits = np.random.default_rng(0).integers(0, 2 ** 16, size=4096, dtype=np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]                      # finite values only
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mod.bf16_bits_to_f64(bits), ref)


def check_brute_force(mod, seed=11):
    """Token-by-token walk of the raw page table with Python floats and math.fsum."""
    rng = np.random.default_rng(seed)
    for trial in range(6):
        S = int(rng.integers(1, 5))
        g = W.random_graph(rng, S, int(rng.integers(1, 5)), 20, 4, slack_pages=2, seed=seed + trial)
        Hq, Hkv, D = 4, 2, 4
        q, pool = W.draw_data(g, Hq, Hkv, D, "f32", seed + trial)
        q, pool = q.numpy() * 0.5, pool.numpy() * 0.5
        out, lse = _decode(mod, g, q, pool, Hq, Hkv, D)
        scale = 1.0 / math.sqrt(D)
        for b in range(g.num_branches):
            for h in range(Hq):
                kv = h // (Hq // Hkv)
                ws, vs = [], []
                for s in g.path(b):
                    for t in range(int(g.seg_len[s])):
                        page = int(g.seg_pages[g.seg_page_offsets[s] + t // 16])
                        k = [float(x) for x in pool[page, kv, 0, t % 16]]
                        v = [float(x) for x in pool[page, kv, 1, t % 16]]
                        z = scale * math.fsum(float(q[b, h, d]) * k[d] for d in range(D))
                        ws.append(math.exp(z))
                        vs.append(v)
                tot = math.fsum(ws)
                ref = [math.fsum(w * v[d] for w, v in zip(ws, vs)) / tot for d in range(D)]
                assert np.allclose(out[b, h], ref, rtol=0, atol=1e-12)
                assert abs(lse[b, h] - math.log(tot)) < 1e-12


def _scatter_contiguous(g, K, V, Hkv, D, Np):
    """Test-side inverse of the page table: write a contiguous K/V sequence into pages."""
    pool = np.full((Np, Hkv, 2, 16, D), np.nan, dtype=np.float32)
    t0 = 0
    for s in range(g.num_segments):
        for t in range(int(g.seg_len[s])):
            page = g.seg_pages[g.seg_page_offsets[s] + t // 16]
            pool[page, :, 0, t % 16] = K[t0 + t]
            pool[page, :, 1, t % 16] = V[t0 + t]
        t0 += int(g.seg_len[s])
    return pool


def check_single_branch_sdpa(mod, seed=5):
    """A one-branch graph is ordinary attention: torch SDPA (float64, GQA) over the sequence."""
    rng = np.random.default_rng(seed)
    for Hq, Hkv, D in [(8, 2, 64), (28, 4, 128), (5, 5, 64), (40, 8, 128)]:
        lens = [int(x) for x in rng.integers(1, 70, size=4)]
        L = sum(lens)
        g = W.assemble_graph(lens, [list(range(4))], seed, slack_pages=3)
        K = rng.standard_normal((L, Hkv, D)).astype(np.float32)
        V = rng.standard_normal((L, Hkv, D)).astype(np.float32)
        q = rng.standard_normal((1, Hq, D)).astype(np.float32)
        pool = _scatter_contiguous(g, K, V, Hkv, D, g.num_pages)
        out, lse = _decode(mod, g, q, pool, Hq, Hkv, D)
        qt = torch.from_numpy(q).double().view(1, Hq, 1, D)
        Kt = torch.from_numpy(K).double().permute(1, 0, 2).unsqueeze(0)   # [1, Hkv, L, D]
        Vt = torch.from_numpy(V).double().permute(1, 0, 2).unsqueeze(0)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt, enable_gqa=True)
        assert np.allclose(out[0], ref.view(Hq, D).numpy(), rtol=0, atol=1e-12)
        Kx = Kt.repeat_interleave(Hq // Hkv, dim=1)                           # [1, Hq, L, D]
        z = (qt @ Kx.transpose(-1, -2)).view(Hq, L) / math.sqrt(D)
        assert np.allclose(lse[0], torch.logsumexp(z, dim=-1).numpy(), rtol=0, atol=1e-12)


def check_rows_sum_to_one(mod, seed=3):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((300, 4, 128)) * 3
    V = rng.standard_normal((300, 4, 128))
    q = rng.standard_normal((28, 128)) * 3
    out, lse, p = mod.attend(q, K, V, 1 / math.sqrt(128), return_probs=True)
    assert np.all(p >= 0)
    assert np.allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-12)
    for h in range(28):
        assert np.allclose(out[h], p[h] @ V[:, h // 7], rtol=0, atol=1e-12)


def _random_bracketing_merge(mod, parts, rng):
    parts = list(parts)
    while len(parts) > 1:
        i = int(rng.integers(len(parts) - 1))
        merged = mod.merge([parts[i], parts[i + 1]])
        parts[i:i + 2] = [merged]
    return parts[0]


def check_merge_associativity(mod, seed=9):
    """Attention over a context == LSE merge of attention over any split, in any bracketing."""
    rng = np.random.default_rng(seed)
    for trial in range(20):
        L = int(rng.integers(2, 400))
        Hq, Hkv, D = 8, 2, 16
        K = rng.standard_normal((L, Hkv, D)) * 2
        V = rng.standard_normal((L, Hkv, D))
        q = rng.standard_normal((Hq, D)) * 2
        scale = 1 / math.sqrt(D)
        o_ref, l_ref = mod.attend(q, K, V, scale)
        ncut = int(rng.integers(1, min(8, L)))
        cuts = np.sort(rng.choice(np.arange(1, L), size=ncut, replace=False))
        bounds = [0] + list(cuts) + [L]
        parts = [mod.attend(q, K[a:b], V[a:b], scale) for a, b in zip(bounds[:-1], bounds[1:])]
        order = rng.permutation(len(parts))
        parts = [parts[i] for i in order]
        o, l = _random_bracketing_merge(mod, parts, rng)
        assert np.allclose(o, o_ref, rtol=0, atol=1e-12)
        assert np.allclose(l, l_ref, rtol=0, atol=1e-12)
        one = mod.merge([parts[0]])
        assert np.allclose(one[0], parts[0][0], atol=1e-15) and np.allclose(one[1], parts[0][1])
        empty = (np.zeros_like(o_ref), np.full_like(l_ref, -np.inf))
        o2, l2 = mod.merge([(o_ref, l_ref), empty])
        assert np.allclose(o2, o_ref, atol=1e-15) and np.allclose(l2, l_ref, atol=1e-15)


def check_tag_closed_form(mod):
    """K = 0 makes every score 0: lse = ln L_b exactly, out = sum_s (len_s / L_b) * tag_s."""
    wl = W.config2_tree(prompts=2, kzero_tags=True, slack_pages=5, poison=True)
    g = wl.graph
    out, lse = _decode(mod, g, wl.q_bits(), wl.pool_bits(), 28, 4, 128, "bf16")
    for b in range(g.num_branches):
        Lb = g.path_tokens(b)
        exp = np.zeros(128)
        for s in g.path(b):
            exp[s % 128] += (1 + s // 128) * g.seg_len[s] / Lb
        assert np.allclose(lse[b], math.log(Lb), rtol=0, atol=1e-12)
        assert np.allclose(out[b], exp[None, :], rtol=0, atol=1e-12)


def check_single_token(mod, seed=2):
    """A one-token context: out = v, lse = scale * <q, k>."""
    rng = np.random.default_rng(seed)
    g = W.assemble_graph([1], [[0]], seed, slack_pages=1)
    Hq, Hkv, D = 6, 3, 64
    pool = rng.standard_normal((g.num_pages, Hkv, 2, 16, D)).astype(np.float32)
    q = rng.standard_normal((1, Hq, D)).astype(np.float32)
    out, lse = _decode(mod, g, q, pool, Hq, Hkv, D)
    p = g.seg_pages[0]
    for h in range(Hq):
        kv = h // 2
        assert np.allclose(out[0, h], pool[p, kv, 1, 0].astype(np.float64), rtol=0, atol=0)
        ref = np.dot(q[0, h].astype(np.float64), pool[p, kv, 0, 0].astype(np.float64)) / 8.0
        assert abs(lse[0, h] - ref) < 1e-12


def check_path_order_invariance(mod, seed=4):
    rng = np.random.default_rng(seed)
    g = W.random_graph(rng, 6, 5, 40, 6, slack_pages=2, seed=seed)
    q, pool = W.draw_data(g, 8, 2, 64, "f32", seed)
    q, pool = q.numpy(), pool.numpy()
    out, lse = _decode(mod, g, q, pool, 8, 2, 64)
    segs = g.path_segs.copy()
    for b in range(g.num_branches):
        a, e = g.path_offsets[b], g.path_offsets[b + 1]
        segs[a:e] = segs[a:e][::-1]
    out2, lse2 = mod.decode(q, pool, g.seg_len, g.seg_page_offsets, g.seg_pages, g.path_offsets,
                            segs, 8, 2, 64, "f32")
    assert np.allclose(out, out2, rtol=0, atol=1e-12) and np.allclose(lse, lse2, rtol=0, atol=1e-12)


def check_groups_fixture(mod):
    """Hand-derived grouping of a small DAG stored in tests/golden."""
    with open(os.path.join(GOLDEN, "groups_small_dag.json")) as f:
        fx = json.load(f)
    po = np.array(fx["path_offsets"], dtype=np.int64)
    ps = np.array(fx["path_segs"], dtype=np.int32)
    offs, ids = mod.segment_groups(po, ps, fx["num_segments"])
    assert offs.tolist() == fx["group_offsets"]
    assert ids.tolist() == fx["group_branches"]
    assert mod.branch_slot_ranks(po, ps, fx["num_segments"]).tolist() == fx["entry_ranks"]


PINS = [check_bf16_decoding, check_brute_force, check_single_branch_sdpa, check_rows_sum_to_one,
        check_merge_associativity, check_tag_closed_form, check_single_token,
        check_path_order_invariance, check_groups_fixture]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin):
    pin(O)


def test_config1_tiny_closed_forms():
    """The tiny graph: B(root) = all 4 branches, each child is private; K=0 gives lse = ln 320."""
    wl = W.config1_tiny(kzero_tags=True)
    g = wl.graph
    offs, ids = O.segment_groups(g.path_offsets, g.path_segs, g.num_segments)
    assert offs.tolist() == [0, 4, 5, 6, 7, 8] and ids.tolist() == [0, 1, 2, 3, 0, 1, 2, 3]
    out, lse = _decode(O, g, wl.q_bits(), wl.pool_bits(), 8, 2, 64, "f32")
    assert np.allclose(lse, math.log(320.0), rtol=0, atol=1e-12)
    for b in range(4):
        exp = np.zeros(64)
        exp[0] += 256 / 320
        exp[1 + b] += 64 / 320
        assert np.allclose(out[b], exp[None], rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------------------------
# Planted mistakes: each must be caught by at least one pin
# ---------------------------------------------------------------------------------------------

def _caught(pins):
    for pin in pins:
        try:
            pin(O)
        except (AssertionError, IndexError):
            return True
    return False


def _wrong_slot_segment_tokens(pool_raw, dtype, seg_len, seg_page_offsets, seg_pages, s):
    k, v = ORIG_SEGMENT_TOKENS(pool_raw, dtype, seg_len, seg_page_offsets, seg_pages, s)
    if k.shape[0] > 1:                       # token order shifted by one inside the segment
        k = np.roll(k, 1, axis=0)
    return k, v


def _dropped_last_token(pool_raw, dtype, seg_len, seg_page_offsets, seg_pages, s):
    k, v = ORIG_SEGMENT_TOKENS(pool_raw, dtype, seg_len, seg_page_offsets, seg_pages, s)
    if k.shape[0] > 1:
        return k[:-1], v[:-1]
    return k, v


def _lse_base2_attend(q, K, V, scale, return_probs=False):
    r = ORIG_ATTEND(q, K, V, scale, return_probs)
    return (r[0], r[1] / math.log(2)) + tuple(r[2:])


def _merge_without_weights(partials):
    os_ = np.stack([o for o, _ in partials])
    lses = np.stack([l for _, l in partials])
    M = lses.max(axis=0)
    return os_.mean(axis=0), M + np.log(np.exp(lses - M).sum(axis=0))


def _bf16_truncating(bits):
    x = ORIG_BF16(bits)
    return np.trunc(x * 64) / 64


ORIG_SEGMENT_TOKENS = O.segment_tokens
ORIG_ATTEND = O.attend
ORIG_BF16 = O.bf16_bits_to_f64


@pytest.mark.parametrize("name,attr,repl", [
    ("gqa_interleaved", "kv_head_of", lambda h, group: h % group),
    ("gqa_shifted", "kv_head_of", lambda h, group: max(0, h - 1) // group),
    ("slot_order", "segment_tokens", _wrong_slot_segment_tokens),
    ("dropped_token", "segment_tokens", _dropped_last_token),
    ("lse_base2", "attend", _lse_base2_attend),
    ("merge_unweighted", "merge", _merge_without_weights),
    ("bf16_lossy", "bf16_bits_to_f64", _bf16_truncating),
])
def test_planted_mistake_is_caught(monkeypatch, name, attr, repl):
    monkeypatch.setattr(O, attr, repl)
    assert _caught(PINS), f"planted mistake {name} went unnoticed"
