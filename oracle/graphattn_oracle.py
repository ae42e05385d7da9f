"""Plain fp64 CPU oracle for graph-segment decode attention.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT. Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module. It shares no code with the HIP path: it
decodes stored bf16 bits itself, walks the page table itself and computes attention from its
textbook definition, one branch at a time, in float64.

What it computes (the passages it follows):

* A rollout graph has reasoning steps as edges and the prompt as root v0; the generation context
  of a state u, prefix(u), is the ordered concatenation of the *edge* tokens on the path from v0
  to u (Sec. 3.2 "Graph Construction"; Alg. S.1, Stage 1, "sample continuations from
  pi_theta(. | prefix(u))"). Tree rollouts let siblings share their parent's prefix (Sec. 1) and
  merged states share the representative's successors (Sec. 3.2, graph suffix C_g). A decoding
  branch is therefore a list of segment ids, and its context is the concatenation of those
  segments' K/V tokens.
* Each active branch issues one decode query per q-head; the attention of that query over its
  context is the standard scaled dot-product softmax attention. The paper does not print the
  formula (it never mentions attention); the definition used is the textbook one: scores
  z_j = scale * <q, k_j>, p = softmax(z), out = sum_j p_j v_j, lse = ln sum_j exp(z_j).
* Grouped-query attention: q-head h reads kv-head floor(h / (Hq / Hkv)).

Readings where the paper is silent (each also listed in the design notes):
all tokens of every segment on the path are attended, including the branch's own leaf segment;
no causal mask (a single query at the end of the path); scale = 1/sqrt(D) unless given;
lse is the natural log; segment order along a path does not change the result.

Parity status: every function below is pinned by CPU tests against brute force, a library
routine on a special case, closed forms and invariants (softmax rows sum to 1, merge
associativity, the K=0 tag closed form, the single-token case).
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

PAGE_TOKENS = 16


# ----------------------------------------------------------------------------------------------
# Storage decoding
# ----------------------------------------------------------------------------------------------

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns: a bf16 is the upper half of an IEEE binary32."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def to_f64(raw: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits_to_f64(raw)
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def kv_head_of(h: int, group: int) -> int:
    """Grouped-query mapping: consecutive groups of q-heads share one kv-head."""
    return h // group


# ----------------------------------------------------------------------------------------------
# Context materialisation: prefix(u) as the ordered concatenation of segment tokens
# ----------------------------------------------------------------------------------------------

def segment_tokens(pool_raw: np.ndarray, dtype: str, seg_len: np.ndarray,
                   seg_page_offsets: np.ndarray, seg_pages: np.ndarray, s: int
                   ) -> Tuple[np.ndarray, np.ndarray]:
    """K and V of one segment (one edge of the rollout graph), as [len, Hkv, D] float64.

    Token t of segment s sits in page seg_pages[seg_page_offsets[s] + t // 16], slot t % 16;
    the pool is [num_pages][Hkv][2][16][D] with K at index 0 and V at index 1.
    """
    L = int(seg_len[s])
    off = int(seg_page_offsets[s])
    npg = (L + PAGE_TOKENS - 1) // PAGE_TOKENS
    pages = np.asarray(seg_pages[off:off + npg], dtype=np.int64)
    blk = pool_raw[pages]                          # [npg, Hkv, 2, 16, D]
    blk = np.moveaxis(blk, 3, 1)                   # [npg, 16, Hkv, 2, D]
    tok = blk.reshape(npg * PAGE_TOKENS, blk.shape[2], 2, blk.shape[4])[:L]
    tok = to_f64(tok, dtype)
    return tok[:, :, 0, :], tok[:, :, 1, :]


def branch_context(pool_raw: np.ndarray, dtype: str, seg_len, seg_page_offsets, seg_pages,
                   path: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """prefix(u): the branch's segments concatenated in path order -> K_b, V_b [L_b, Hkv, D]."""
    ks, vs = [], []
    for s in path:
        k, v = segment_tokens(pool_raw, dtype, seg_len, seg_page_offsets, seg_pages, int(s))
        ks.append(k)
        vs.append(v)
    return np.concatenate(ks, axis=0), np.concatenate(vs, axis=0)


# ----------------------------------------------------------------------------------------------
# Textbook attention
# ----------------------------------------------------------------------------------------------

def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float, return_probs: bool = False):
    """Softmax attention of one query per q-head over a context.

    q [Hq, D], K/V [L, Hkv, D] (float64). Returns out [Hq, D], lse [Hq] (natural log) and,
    optionally, the probabilities [Hq, L]. The max subtraction only rescales numerator and
    denominator by the same factor; it does not change the definition.
    """
    Hq, D = q.shape
    L, Hkv, _ = K.shape
    group = Hq // Hkv
    out = np.empty((Hq, D), dtype=np.float64)
    lse = np.empty(Hq, dtype=np.float64)
    probs = np.empty((Hq, L), dtype=np.float64) if return_probs else None
    for h in range(Hq):
        kv = kv_head_of(h, group)
        z = scale * (K[:, kv, :] @ q[h])          # [L]
        m = z.max()
        e = np.exp(z - m)
        l = e.sum()
        p = e / l
        out[h] = p @ V[:, kv, :]
        lse[h] = m + math.log(l)
        if return_probs:
            probs[h] = p
    if return_probs:
        return out, lse, probs
    return out, lse


def decode(q_raw: np.ndarray, pool_raw: np.ndarray, seg_len, seg_page_offsets, seg_pages,
           path_offsets, path_segs, num_q_heads: int, num_kv_heads: int, head_dim: int,
           dtype: str, scale: Optional[float] = None,
           branches: Optional[Iterable[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Decode attention of every (or the listed) branch over its ancestor segment chain.

    Returns out [n, Hq, D] and lse [n, Hq] in float64 for the n requested branches (all
    branches in order if ``branches`` is None).
    """
    if num_q_heads % num_kv_heads:
        raise ValueError("Hq must be a multiple of Hkv")
    if scale is None or scale == 0.0:
        scale = 1.0 / math.sqrt(head_dim)
    B = len(path_offsets) - 1
    ids = list(range(B)) if branches is None else [int(b) for b in branches]
    out = np.empty((len(ids), num_q_heads, head_dim), dtype=np.float64)
    lse = np.empty((len(ids), num_q_heads), dtype=np.float64)
    for i, b in enumerate(ids):
        path = path_segs[path_offsets[b]:path_offsets[b + 1]]
        K, V = branch_context(pool_raw, dtype, seg_len, seg_page_offsets, seg_pages, path)
        qb = to_f64(q_raw[b], dtype)
        out[i], lse[i] = attend(qb, K, V, scale)
    return out, lse


# ----------------------------------------------------------------------------------------------
# Log-sum-exp merge of partial results over disjoint pieces of one context
# ----------------------------------------------------------------------------------------------

def merge(partials: Sequence[Tuple[np.ndarray, np.ndarray]]) -> Tuple[np.ndarray, np.ndarray]:
    """Combine (o_i, lse_i) computed over disjoint token sets into the result over their union.

    With lse_i = ln sum_{j in piece i} exp(z_j) and o_i the normalised output of piece i:
    lse = ln sum_i exp(lse_i) and out = sum_i exp(lse_i - lse) o_i. Pieces with lse = -inf (no
    tokens) contribute nothing. Shapes: o_i [..., D], lse_i [...].
    """
    lses = np.stack([np.asarray(l, dtype=np.float64) for _, l in partials])   # [n, ...]
    os_ = np.stack([np.asarray(o, dtype=np.float64) for o, _ in partials])    # [n, ..., D]
    M = lses.max(axis=0)
    Msafe = np.where(np.isfinite(M), M, 0.0)
    w = np.exp(lses - Msafe)
    tot = w.sum(axis=0)
    lse = Msafe + np.log(tot)
    out = (w[..., None] * np.where(w[..., None] > 0, os_, 0.0)).sum(axis=0) / tot[..., None]
    return out, lse


# ----------------------------------------------------------------------------------------------
# Integer reference for the scheduler's grouping
# ----------------------------------------------------------------------------------------------

def segment_groups(path_offsets, path_segs, num_segments: int) -> Tuple[np.ndarray, np.ndarray]:
    """B(s) = the ascending ids of the branches whose path contains s, as CSR (offsets, ids).

    Plain loops over the definition: for each segment, scan every branch's path.
    """
    B = len(path_offsets) - 1
    members: List[List[int]] = [[] for _ in range(num_segments)]
    for b in range(B):
        for s in path_segs[path_offsets[b]:path_offsets[b + 1]]:
            members[int(s)].append(b)
    offs = np.zeros(num_segments + 1, dtype=np.int64)
    for s in range(num_segments):
        offs[s + 1] = offs[s] + len(members[s])
    ids = np.array([b for m in members for b in sorted(m)], dtype=np.int32)
    return offs, ids


def branch_slot_ranks(path_offsets, path_segs, num_segments: int) -> np.ndarray:
    """For every path entry (branch b, segment s), the position of b inside B(s)."""
    offs, ids = segment_groups(path_offsets, path_segs, num_segments)
    B = len(path_offsets) - 1
    ranks = np.empty(len(path_segs), dtype=np.int32)
    for b in range(B):
        for e in range(int(path_offsets[b]), int(path_offsets[b + 1])):
            s = int(path_segs[e])
            grp = list(ids[offs[s]:offs[s + 1]])
            ranks[e] = grp.index(b)
    return ranks
