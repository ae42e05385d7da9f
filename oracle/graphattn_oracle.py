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

* Equivalence detection (Sec. 3.2; Alg. S.1, Stage 1): states of one prompt's graph that are
  not ancestor and descendant are compared by the cosine of their embeddings; pairs at or above
  kappa are joined by union-find into classes Q(v); the graph suffix C_g(u) adds the direct
  successors of the other class members that lie deeper than u.
* Graph reward and dual-group advantage (Sec. 3.3-3.4; Alg. S.1, Stages 2-3): terminal
  outcomes summed over each state's subtree, pooled over its class with weight w, step rewards
  from score gains discounted by endpoint similarity, correctness z-scores within each source's
  group E_cor, efficiency z-scores of route lengths within each class, gated by the class's
  mean score and spread over the route's edges.
* Extend: the queries of a branch are the newest tokens of its last path segment, each
  attending causally (Alg. S.1, Stage 1: a continuation is predicted token by token from
  prefix(u)); append and copy store tokens into page slots and move them between slots.

Readings where the paper is silent (each also listed in the design notes):
all tokens of every segment on the path are attended, including the branch's own leaf segment;
no causal mask (a single query at the end of the path); scale = 1/sqrt(D) unless given;
lse is the natural log; segment order along a path does not change the result.
For extend: the query segment is the path's last entry, a query sees itself, and a query at
position P of that segment sees exactly its tokens 0 .. P. A slot word is page * 16 + slot.
For equivalence detection: ancestry is that of the generation tree (p(v)); a class is labelled
by its smallest state id; pairs of different prompts are never compared.
For the graph reward: S(v) is undefined (NaN) without evidence, and such edges sit out of their
group with advantage 0; an edge's correctness advantage is taken in its own source's group;
std is the population standard deviation and a zero spread gives 0; a_Q is the deepest proper
ancestor of every member; an edge on several efficiency routes receives the sum.

Parity status: every function below is pinned by CPU tests against brute force, a library
routine on a special case, closed forms and invariants (softmax rows sum to 1, merge
associativity, the K=0 tag closed form, the single-token case); extend against torch's causal
SDPA and a token-by-token walk, append by reading the stored segment back, copy by splitting a
segment inside a page without changing attention; equivalence classes against scipy's connected
components of an independently built link graph, threshold extremes and the ancestor rule;
the graph suffix against a hand-derived fixture and the no-merge identity; the graph reward and
advantages against a hand-derived fixture, the Monte Carlo rate (no merges, or w = 0), the
pooled rate at w = 1 and the z-score invariants of unshared groups.
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


# ----------------------------------------------------------------------------------------------
# Multi-query attention over a branch's newest segment ("extend")
# ----------------------------------------------------------------------------------------------

def query_context_length(context_tokens: int, n_queries: int, i: int) -> int:
    """Tokens seen by query i of a branch whose context (its whole path) has context_tokens
    tokens and whose newest segment, last in the path, holds its n_queries queries at the end:
    all but the segment's n_queries - 1 - i final tokens (the query sees itself)."""
    return context_tokens - (n_queries - 1 - i)


def extend(q_raw: np.ndarray, pool_raw: np.ndarray, seg_len, seg_page_offsets, seg_pages,
           path_offsets, path_segs, query_counts, num_q_heads: int, num_kv_heads: int,
           head_dim: int, dtype: str, scale: Optional[float] = None,
           rows: Optional[Iterable[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Several query tokens per branch, causal inside the branch's newest segment.

    Continuations are sampled from pi_theta(. | prefix(u)) (Alg. S.1, Stage 1): every token of a
    new step segment is predicted from the state's prefix plus the step's earlier tokens. Branch
    b's last path segment is that step; its queries are the last n_b = query_counts[b] tokens of
    it, so query i (0 <= i < n_b) sits at position P_i = len(last) - n_b + i of the segment and
    attends to every token of the other path segments and to tokens 0 .. P_i of the last one
    (itself included). With n_b = 1 the single query sees the whole context, which is decode.

    q_raw holds one row per query, [sum_b n_b][Hq][D], branch-major and ascending i within a
    branch. Returns out [n][Hq][D] and lse [n][Hq] (float64) for the n requested query rows
    (all rows if ``rows`` is None).
    """
    if num_q_heads % num_kv_heads:
        raise ValueError("Hq must be a multiple of Hkv")
    if scale is None or scale == 0.0:
        scale = 1.0 / math.sqrt(head_dim)
    B = len(path_offsets) - 1
    counts = [int(c) for c in query_counts]
    if len(counts) != B:
        raise ValueError("one query count per branch")
    row_branch: List[Tuple[int, int]] = []
    for b in range(B):
        last = int(path_segs[path_offsets[b + 1] - 1])
        if not 1 <= counts[b] <= int(seg_len[last]):
            raise ValueError(f"branch {b}: query count outside [1, len(last segment)]")
        row_branch += [(b, i) for i in range(counts[b])]
    ids = list(range(len(row_branch))) if rows is None else [int(r) for r in rows]
    out = np.empty((len(ids), num_q_heads, head_dim), dtype=np.float64)
    lse = np.empty((len(ids), num_q_heads), dtype=np.float64)
    ctx_cache = {}
    for k, r in enumerate(ids):
        b, i = row_branch[r]
        if b not in ctx_cache:
            path = path_segs[path_offsets[b]:path_offsets[b + 1]]
            ctx_cache = {b: branch_context(pool_raw, dtype, seg_len, seg_page_offsets,
                                           seg_pages, path)}
        K, V = ctx_cache[b]
        visible = query_context_length(K.shape[0], counts[b], i)
        qi = to_f64(q_raw[r], dtype)
        out[k], lse[k] = attend(qi, K[:visible], V[:visible], scale)
    return out, lse


# ----------------------------------------------------------------------------------------------
# Writing K/V into the page pool
# ----------------------------------------------------------------------------------------------

def _slot_ok(word: int, num_pages: int) -> bool:
    return 0 <= word < num_pages * PAGE_TOKENS


def kv_append(pool_raw: np.ndarray, k_new_raw: np.ndarray, v_new_raw: np.ndarray,
              slot_words) -> np.ndarray:
    """Store new tokens' K and V in the pool; returns the updated copy of the pool.

    Each decode step extends every active branch's leaf segment by the token it produced, and a
    state's continuation splits into new step segments (Alg. S.1, Stage 1); a token of a segment
    lives in one page slot. slot_words[j] = page * 16 + slot names token j's destination;
    k_new_raw / v_new_raw are [n][Hkv][D] raw storage values (bf16 bits or float32). Words
    outside [0, num_pages * 16) are skipped (a negative word pads a batch). Destinations must be
    distinct.
    """
    out = np.array(pool_raw, copy=True)
    seen = set()
    for j, w in enumerate(int(x) for x in slot_words):
        if not _slot_ok(w, pool_raw.shape[0]):
            continue
        if w in seen:
            raise ValueError("destination slots must be distinct")
        seen.add(w)
        page, slot = divmod(w, PAGE_TOKENS)
        out[page, :, 0, slot, :] = k_new_raw[j]
        out[page, :, 1, slot, :] = v_new_raw[j]
    return out


def kv_copy(pool_raw: np.ndarray, src_words, dst_words) -> np.ndarray:
    """Copy tokens between page slots (every kv-head, K and V); returns the updated pool.

    Needed where a generated run of tokens is cut into step segments inside a page (Alg. S.1,
    Stage 1, "split them into segment-level transitions"): a segment begins at slot 0 of its
    own page, so the tokens after the cut move to fresh pages; a fork that lets children keep
    writing into a shared, partly filled page copies that page the same way. Pairs with either
    word outside the pool are skipped; sources are read as they were before the call, and
    destinations must be distinct and disjoint from the sources.
    """
    out = np.array(pool_raw, copy=True)
    Np = pool_raw.shape[0]
    pairs = [(int(s), int(d)) for s, d in zip(src_words, dst_words)
             if _slot_ok(int(s), Np) and _slot_ok(int(d), Np)]
    dsts = [d for _, d in pairs]
    if len(set(dsts)) != len(dsts) or set(dsts) & {s for s, _ in pairs}:
        raise ValueError("destinations must be distinct and disjoint from the sources")
    for s, d in pairs:
        sp, ss = divmod(s, PAGE_TOKENS)
        dp, ds = divmod(d, PAGE_TOKENS)
        out[dp, :, :, ds, :] = pool_raw[sp, :, :, ss, :]
    return out


# ----------------------------------------------------------------------------------------------
# Equivalence detection over rollout states (graph construction)
# ----------------------------------------------------------------------------------------------

def state_depths(parent) -> np.ndarray:
    """Depth of every state in its prompt's generation tree (a prompt's root has depth 0)."""
    par = [int(x) for x in parent]
    depth = np.zeros(len(par), dtype=np.int64)
    for v, p in enumerate(par):
        depth[v] = 0 if p < 0 else depth[p] + 1
    return depth


def is_ancestor(parent, u: int, v: int) -> bool:
    """True when u lies on v's generation path (u == v counts): walk v's predecessors."""
    x = int(v)
    while x >= 0:
        if x == u:
            return True
        x = int(parent[x])
    return False


def prompts_of(parent) -> List[List[int]]:
    """The states of each prompt's graph (grouped by the root their generation path starts at),
    in ascending id order."""
    root = {}
    groups: dict = {}
    for v in range(len(parent)):
        x = v
        while int(parent[x]) >= 0:
            x = int(parent[x])
        root[v] = x
        groups.setdefault(x, []).append(v)
    return [groups[r] for r in sorted(groups)]


def compared_pairs(parent) -> List[Tuple[int, int]]:
    """The pairs the method compares (Sec. 3.2): two states of the same prompt's graph, neither
    an ancestor of the other (comparing a state with its own ancestors could close a cycle)."""
    out = []
    for ids in prompts_of(parent):
        for i, u in enumerate(ids):
            for v in ids[i + 1:]:
                if not is_ancestor(parent, u, v) and not is_ancestor(parent, v, u):
                    out.append((u, v))
    return out


def similarity_matrix(z_raw: np.ndarray, dtype: str, ids: Sequence[int]) -> np.ndarray:
    """sim(u, v) = z_u . z_v / (|z_u| |z_v|) for all u, v in ids, float64 on the stored values
    (one matrix product of the row-normalised embeddings)."""
    z = to_f64(z_raw[np.asarray(ids, dtype=np.int64)], dtype)
    zn = z / np.sqrt((z * z).sum(axis=1, keepdims=True))
    return zn @ zn.T


def cosine(z_raw: np.ndarray, dtype: str, u: int, v: int) -> float:
    """sim(u, v) of one pair."""
    return float(similarity_matrix(z_raw, dtype, [u, v])[0, 1])


def _compared_similarities(z_raw, dtype, parent):
    for ids in prompts_of(parent):
        pos = {v: i for i, v in enumerate(ids)}
        sim = similarity_matrix(z_raw, dtype, ids)
        for i, u in enumerate(ids):
            for v in ids[i + 1:]:
                if not is_ancestor(parent, u, v) and not is_ancestor(parent, v, u):
                    yield u, v, float(sim[i, pos[v]])


def equivalence_classes(z_raw: np.ndarray, dtype: str, parent, kappa: float) -> np.ndarray:
    """Class label of every state: the smallest state id of its equivalence class Q(v).

    Compared pairs with sim(u, v) >= kappa are linked by union-find (Sec. 3.2; Alg. S.1,
    Stage 1), so the classes are the connected components of those links. Plain union-find
    with the smaller root kept as the representative, so a root is its class's minimum.
    """
    N = len(parent)
    rep = list(range(N))

    def find(x):
        while rep[x] != x:
            x = rep[x]
        return x

    for u, v, sim in _compared_similarities(z_raw, dtype, parent):
        if sim >= kappa:
            ru, rv = find(u), find(v)
            if ru != rv:
                rep[max(ru, rv)] = min(ru, rv)
    return np.array([find(v) for v in range(N)], dtype=np.int32)


def similarity_margin(z_raw: np.ndarray, dtype: str, parent, kappa: float) -> float:
    """Smallest |sim(u, v) - kappa| over the compared pairs (inf if there are none): how far
    the inputs keep every decision from the threshold."""
    m = math.inf
    for _, _, sim in _compared_similarities(z_raw, dtype, parent):
        m = min(m, abs(sim - kappa))
    return m


def graph_suffix(labels, parent) -> Tuple[np.ndarray, np.ndarray]:
    """Graph suffix C_g(u) of every state as CSR (offsets [N+1], ascending state ids).

    C_g(u) = C(u) together with the direct successors of the other members of Q(u) (Sec. 3.2,
    the equation of the graph suffix); a shared successor must lie deeper than u, which keeps
    the graph acyclic (the virtual merge only adds edges that point deeper).
    """
    N = len(parent)
    depth = state_depths(parent)
    out: List[List[int]] = []
    for u in range(N):
        cu = []
        for c in range(N):
            p = int(parent[c])
            if p < 0:
                continue
            if p == u or (labels[p] == labels[u] and depth[c] > depth[u]):
                cu.append(c)
        out.append(cu)
    offs = np.zeros(N + 1, dtype=np.int64)
    for u in range(N):
        offs[u + 1] = offs[u] + len(out[u])
    return offs, np.array([c for cu in out for c in cu], dtype=np.int32)


# ----------------------------------------------------------------------------------------------
# Graph reward and the dual-group advantage
# ----------------------------------------------------------------------------------------------

def subtree_outcomes(parent, reward) -> Tuple[np.ndarray, np.ndarray]:
    """c_own(v) = sum of R(z) and t_own(v) = |Z(v)| over the terminal states z reachable from v
    through direct generation edges (v's own subtree, v included): Sec. 3.3. reward[v] is R(v)
    in {0, 1} for a terminal state and -1 for any other state. Plain bottom-up accumulation."""
    N = len(parent)
    c = np.zeros(N, dtype=np.int64)
    t = np.zeros(N, dtype=np.int64)
    for v in range(N):
        if reward[v] >= 0:
            x = v
            while x >= 0:                       # v is in the subtree of each of its ancestors
                c[x] += int(reward[v])
                t[x] += 1
                x = int(parent[x])
    return c, t


def node_scores(parent, labels, reward, w: float) -> np.ndarray:
    """S(v) = (c_own(v) + w sum_{q in Q(v), q != v} c_own(q)) /
              (t_own(v) + w sum_{q in Q(v), q != v} t_own(q))   (Sec. 3.3, the pooled score).
    Defined where the denominator is positive; NaN (no evidence) elsewhere."""
    c, t = subtree_outcomes(parent, reward)
    N = len(parent)
    S = np.full(N, np.nan)
    for v in range(N):
        # the partners' counts are integers: summed exactly, then weighted by w once, so two
        # states with the same counts get the same score whatever the order of the sum
        cq = sum(int(c[q]) for q in range(N) if q != v and labels[q] == labels[v])
        tq = sum(int(t[q]) for q in range(N) if q != v and labels[q] == labels[v])
        ts = float(t[v]) + w * float(tq)
        if ts > 0:
            S[v] = (float(c[v]) + w * float(cq)) / ts
    return S


def step_rewards(parent, S, edge_sim) -> np.ndarray:
    """r_step(p(v), v) = (S(v) - S(p(v))) (1 - max(0, sim(p(v), v))) for the direct edge into
    each non-root state v (Sec. 3.3); edge_sim[v] = sim(p(v), v). NaN for a root and where a
    score is undefined."""
    N = len(parent)
    r = np.full(N, np.nan)
    for v in range(N):
        p = int(parent[v])
        if p >= 0:
            r[v] = (S[v] - S[p]) * (1.0 - max(0.0, float(edge_sim[v])))
    return r


# A correctness group whose rewards spread by no more than this has no spread.  Scores lie in
# [0, 1] and |r_step| <= 2, so rewards that are equal by the definition differ by fp64 rounding
# (~1e-16) at most, while unequal ones differ by far more; a plain zero test would turn that
# rounding into z-scores of order one.
SPREAD_FLOOR = 1e-12


def _zscores(values: Sequence[float], floor: float = 0.0) -> List[float]:
    """(x - mean) / std over a group, population std; 0 for every member if std <= floor."""
    n = len(values)
    m = math.fsum(values) / n
    sd = math.sqrt(math.fsum((x - m) ** 2 for x in values) / n)
    return [0.0 if sd <= floor else (x - m) / sd for x in values]


def correctness_advantage(parent, labels, r) -> np.ndarray:
    """A_cor of the edge into every state (Sec. 3.4, the step correctness group).

    The group of source state u is E_cor(u) = {(p(v), v) : v in C_g(u)}; groups exist for
    |C_g(u)| > 1 (Alg. S.1, Stage 3). An edge's advantage is taken in the group of its own
    source p(v); edges with an undefined reward take no part and get 0, and so does every edge
    of a group whose spread is at most SPREAD_FLOOR (no spread).
    """
    offs, states = graph_suffix(labels, parent)
    N = len(parent)
    A = np.zeros(N)
    for v in range(N):
        u = int(parent[v])
        if u < 0 or np.isnan(r[v]):
            continue
        grp = [int(x) for x in states[offs[u]:offs[u + 1]]]
        if len(grp) <= 1:
            continue
        vals = [float(r[x]) for x in grp if not np.isnan(r[x])]
        z = _zscores(vals, SPREAD_FLOOR)
        A[v] = z[[x for x in grp if not np.isnan(r[x])].index(v)]
    return A


def class_anchor(parent, members: Sequence[int]) -> int:
    """a_Q: the deepest state that is a predecessor (a proper ancestor) of every member."""
    def chain(v):
        out = []
        x = int(parent[v])
        while x >= 0:
            out.append(x)
            x = int(parent[x])
        return out
    common = set(chain(members[0]))
    for v in members[1:]:
        common &= set(chain(v))
    depth = state_depths(parent)
    return max(common, key=lambda x: depth[x])


def efficiency_advantage(parent, labels, S) -> np.ndarray:
    """A_eff on the edge into every state (Sec. 3.4, the efficiency group).

    For each class Q with |Q| >= 2: a_Q = class_anchor, l_v = d(v) - d(a_Q), the gate
    S_bar = mean of the defined S over Q (0 if none), A_eff(v) = S_bar z(-l_v) over Q, and
    A_eff(v) is given to every direct edge on the route from a_Q to v; an edge on several such
    routes receives their sum.
    """
    N = len(parent)
    depth = state_depths(parent)
    E = np.zeros(N)
    classes: dict = {}
    for v in range(N):
        classes.setdefault(int(labels[v]), []).append(v)
    for members in classes.values():
        if len(members) < 2:
            continue
        a = class_anchor(parent, members)
        ell = [int(depth[v] - depth[a]) for v in members]
        defined = [float(S[v]) for v in members if not np.isnan(S[v])]
        gate = math.fsum(defined) / len(defined) if defined else 0.0
        z = _zscores([-float(x) for x in ell])
        for v, zv in zip(members, z):
            x = v
            while x != a:                        # edges (p(x), x) from a_Q down to v
                E[x] += gate * zv
                x = int(parent[x])
    return E


def graph_advantages(parent, labels, reward, edge_sim, w: float, lam: float) -> dict:
    """The graph reward and dual-group advantage of every state's incoming edge (Sec. 3.3-3.4;
    Alg. S.1, Stages 2-3): S, r_step, A_cor, A_eff and A_dual = A_cor + lam A_eff."""
    S = node_scores(parent, labels, reward, w)
    r = step_rewards(parent, S, edge_sim)
    A_cor = correctness_advantage(parent, labels, r)
    A_eff = efficiency_advantage(parent, labels, S)
    return {"S": S, "r": r, "A_cor": A_cor, "A_eff": A_eff, "A_dual": A_cor + lam * A_eff}
