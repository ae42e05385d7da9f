"""Seeded synthetic rollout graphs: the inputs of graph-segment decode attention.

This module only *draws inputs*. It holds no attention, softmax or merge arithmetic, so both the
HIP path and the CPU oracle can consume what it produces without sharing any of the method's code.

The rollout graph follows GraphPO's problem statement (Sec. 3.2, "Graph Construction", and
Alg. S.1 Stage 1): reasoning steps are edges whose generated tokens form a *segment*; the
generation context of a state is the ordered concatenation of the edge tokens on its path from
the prompt (the root). A decoding *branch* is therefore a list of segment ids, root first.
Siblings share their parent's prefix segments, and virtually merged states share the
representative's suffix segments (Sec. 3.2, graph suffix C_g).

Memory layout produced here (the library's contract):

* ``pool``  ``[num_pages][Hkv][2][16][D]`` -- index 0 of the third axis is K, 1 is V; token ``t``
  of segment ``s`` lives at page ``seg_pages[seg_page_offsets[s] + t // 16]``, slot ``t % 16``.
* ``q``     ``[B][Hq][D]`` -- one decode query per branch.
* ``seg_len`` int32 ``[S]``, ``seg_page_offsets`` int64 ``[S+1]``, ``seg_pages`` int32,
  ``path_offsets`` int64 ``[B+1]``, ``path_segs`` int32 ``[E]``.

Values are i.i.d. N(0,1) drawn in fp32 from a seeded ``torch.Generator`` (CPU) and rounded to
bf16 with round-to-nearest-even (fp32 workloads keep the fp32 draw). Structure comes from
``numpy.random.default_rng``. Page placement is a seeded permutation of the pool.
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

PAGE = 16
SEED_BASE = 260618954
# Pages drawn per chunk of the data RNG stream (part of the generator's definition: changing it
# changes the drawn values).
_DRAW_CHUNK_PAGES = 2048


@dataclasses.dataclass
class RolloutGraph:
    """Segment table + branch paths of one decode step (host arrays)."""

    seg_len: np.ndarray           # int32 [S]
    seg_page_offsets: np.ndarray  # int64 [S+1]
    seg_pages: np.ndarray         # int32 [sum of pages]
    path_offsets: np.ndarray      # int64 [B+1]
    path_segs: np.ndarray         # int32 [E]
    num_pages: int                # pool extent (referenced + free pages)
    info: Dict = dataclasses.field(default_factory=dict)

    @property
    def num_segments(self) -> int:
        return int(self.seg_len.shape[0])

    @property
    def num_branches(self) -> int:
        return int(self.path_offsets.shape[0] - 1)

    def path(self, b: int) -> np.ndarray:
        return self.path_segs[self.path_offsets[b]:self.path_offsets[b + 1]]

    def path_tokens(self, b: int) -> int:
        return int(self.seg_len[self.path(b)].sum())

    def unique_tokens(self) -> int:
        """Tokens of segments referenced by at least one branch."""
        used = np.zeros(self.num_segments, dtype=bool)
        used[self.path_segs] = True
        return int(self.seg_len[used].sum())

    def attended_tokens(self) -> int:
        return int(self.seg_len[self.path_segs].sum())


@dataclasses.dataclass
class Workload:
    name: str
    graph: RolloutGraph
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str                    # "bf16" or "f32"
    q: torch.Tensor               # CPU [B][Hq][D], torch.bfloat16 or torch.float32
    pool: torch.Tensor            # CPU [Np][Hkv][2][16][D]
    seed: int
    # Multi-query (extend) workloads: queries per branch; q then holds sum(query_counts) rows.
    query_counts: Optional[np.ndarray] = None

    @property
    def elt_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def unique_kv_bytes(self) -> int:
        return self.graph.unique_tokens() * 2 * self.num_kv_heads * self.head_dim * self.elt_bytes

    def pool_bits(self) -> np.ndarray:
        """The pool as raw storage: uint16 bf16 bit patterns, or float32 values."""
        if self.dtype == "bf16":
            return self.pool.view(torch.int16).numpy().view(np.uint16)
        return self.pool.numpy()

    def q_bits(self) -> np.ndarray:
        if self.dtype == "bf16":
            return self.q.view(torch.int16).numpy().view(np.uint16)
        return self.q.numpy()


# ----------------------------------------------------------------------------------------------
# Structure -> pages
# ----------------------------------------------------------------------------------------------

def assemble_graph(seg_lens: Sequence[int], paths: Sequence[Sequence[int]], seed: int,
                   slack_pages: int = 0, info: Optional[Dict] = None) -> RolloutGraph:
    """Give each segment its own whole pages and place all pages by a seeded permutation.

    Every segment starts at slot 0 of its first page; its last page may be partial and pages
    are never shared between segments. ``slack_pages`` extra free pages are added to the pool.
    """
    seg_len = np.asarray(seg_lens, dtype=np.int32)
    npg = (seg_len.astype(np.int64) + PAGE - 1) // PAGE
    seg_page_offsets = np.zeros(seg_len.shape[0] + 1, dtype=np.int64)
    np.cumsum(npg, out=seg_page_offsets[1:])
    used = int(seg_page_offsets[-1])
    num_pages = used + int(slack_pages)
    perm = np.random.default_rng(seed + 1000).permutation(num_pages)
    seg_pages = perm[:used].astype(np.int32)
    path_offsets = np.zeros(len(paths) + 1, dtype=np.int64)
    np.cumsum([len(p) for p in paths], out=path_offsets[1:])
    path_segs = (np.concatenate([np.asarray(p, dtype=np.int32) for p in paths])
                 if len(paths) else np.zeros(0, dtype=np.int32))
    return RolloutGraph(seg_len, seg_page_offsets, seg_pages, path_offsets, path_segs,
                        num_pages, dict(info or {}))


def _bf16_rne(x: torch.Tensor) -> torch.Tensor:
    return x.to(torch.bfloat16)


def _chunk_seed(seed: int, stream: int) -> int:
    """Independent 63-bit seed for one chunk of the data stream."""
    st = np.random.SeedSequence([int(seed), int(stream) + 1]).generate_state(1, np.uint64)[0]
    return int(st) & ((1 << 63) - 1)


def _randn(seed: int, stream: int, shape) -> torch.Tensor:
    gen = torch.Generator(device="cpu")
    gen.manual_seed(_chunk_seed(seed, stream))
    return torch.randn(shape, generator=gen, dtype=torch.float32)


def draw_data(graph: RolloutGraph, Hq: int, Hkv: int, D: int, dtype: str, seed: int,
              poison: bool = False, kzero_tags: bool = False):
    """Draw pool then q, i.i.d. N(0,1) in fp32, then round to ``dtype``.

    The pool is drawn in chunks of pages, chunk c from its own generator seeded by (seed, c), so
    chunks can be drawn in parallel and the values do not depend on the thread count; q comes
    from the stream after the last pool chunk.

    ``poison`` writes NaN into every free page and into the unused slots of each segment's last
    page (the contract says those contents are unspecified). ``kzero_tags`` sets K = 0 and
    writes a per-segment tag vector into V (token values of segment s are
    ``(1 + s // D) * e_{s mod D}``), which gives every branch a closed-form answer.
    """
    import concurrent.futures
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Np = graph.num_pages
    pool = torch.empty((Np, Hkv, 2, PAGE, D), dtype=tdt)
    starts = list(range(0, Np, _DRAW_CHUNK_PAGES))

    def one(ci):
        p0 = starts[ci]
        p1 = min(Np, p0 + _DRAW_CHUNK_PAGES)
        blk = _randn(seed, ci, (p1 - p0, Hkv, 2, PAGE, D))
        pool[p0:p1] = _bf16_rne(blk) if dtype == "bf16" else blk

    workers = max(1, min(16, os.cpu_count() or 1, len(starts)))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(one, range(len(starts))))
    B = graph.num_branches
    q = _randn(seed, len(starts), (B, Hq, D))
    q = _bf16_rne(q) if dtype == "bf16" else q
    S = graph.num_segments
    if kzero_tags:
        pool[:, :, 0] = 0
        for s in range(S):
            pages = graph.seg_pages[graph.seg_page_offsets[s]:graph.seg_page_offsets[s + 1]]
            tag = torch.zeros(D, dtype=torch.float32)
            tag[s % D] = 1.0 + (s // D)
            pool[torch.as_tensor(pages, dtype=torch.long), :, 1] = tag.to(tdt)
    if poison:
        used = np.zeros(Np, dtype=bool)
        used[graph.seg_pages] = True
        free = np.nonzero(~used)[0]
        if free.size:
            pool[torch.as_tensor(free, dtype=torch.long)] = float("nan")
        for s in range(S):
            L = int(graph.seg_len[s])
            if L % PAGE:
                last = int(graph.seg_pages[graph.seg_page_offsets[s + 1] - 1])
                pool[last, :, :, L % PAGE:, :] = float("nan")
    return q, pool


def make_workload(name: str, graph: RolloutGraph, Hq: int, Hkv: int, D: int, dtype: str,
                  seed: int, poison: bool = False, kzero_tags: bool = False) -> Workload:
    q, pool = draw_data(graph, Hq, Hkv, D, dtype, seed, poison=poison, kzero_tags=kzero_tags)
    return Workload(name, graph, Hq, Hkv, D, dtype, q, pool, seed)


# ----------------------------------------------------------------------------------------------
# The five rollout-graph configurations
# ----------------------------------------------------------------------------------------------

def _tree_segments(rng, schedule: Sequence[int], root_len: int, step_lo: int, step_hi: int):
    """A step tree with per-depth branching ``schedule`` (Table S1's T = {b_1..b_H}).

    Returns (lengths, paths) with segment 0 the root and the rest in BFS order.
    """
    lens = [int(root_len)]
    frontier = [(0, [0])]
    for b in schedule:
        nxt = []
        for node, path in frontier:
            for _ in range(b):
                sid = len(lens)
                lens.append(int(rng.integers(step_lo, step_hi + 1)))
                nxt.append((sid, path + [sid]))
        frontier = nxt
    return lens, [p for _, p in frontier]


def config1_tiny(slack_pages: int = 0, poison: bool = False, kzero_tags: bool = False,
                 seed: Optional[int] = None) -> Workload:
    """Tiny graph, fp32: a 256-token prompt and 4 child steps of 64 tokens; 8/2 heads, D=64."""
    seed = SEED_BASE + 1 if seed is None else seed
    lens = [256, 64, 64, 64, 64]
    paths = [[0, 1 + i] for i in range(4)]
    g = assemble_graph(lens, paths, seed, slack_pages, {"config": 1})
    return make_workload("tiny graph fp32 (8/2 heads, D=64, 4 branches)", g, 8, 2, 64, "f32",
                         seed, poison, kzero_tags)


def config2_tree(prompts: int = 16, slack_pages: int = 0, poison: bool = False,
                 kzero_tags: bool = False, seed: Optional[int] = None) -> Workload:
    """7B-shaped layer: 16 prompts, 512-token root, T={2,2,2}, steps U{128..384}; 28/4/128."""
    seed = SEED_BASE + 2 if seed is None else seed
    rng = np.random.default_rng(seed)
    lens: List[int] = []
    paths: List[List[int]] = []
    for _ in range(prompts):
        l, p = _tree_segments(rng, (2, 2, 2), 512, 128, 384)
        base = len(lens)
        lens += l
        paths += [[base + s for s in path] for path in p]
    g = assemble_graph(lens, paths, seed, slack_pages, {"config": 2, "prompts": prompts})
    return make_workload(f"7B-shaped tree layer (28/4/128, {prompts} prompts, T={{2,2,2}})", g,
                         28, 4, 128, "bf16", seed, poison, kzero_tags)


class _Node:
    __slots__ = ("depth", "children", "alive", "merged_into", "is_rep", "seg")

    def __init__(self, depth):
        self.depth = depth
        self.children: List["_Node"] = []
        self.alive = True
        self.merged_into: Optional["_Node"] = None
        self.is_rep = False
        self.seg = -1


def _kill(node: _Node):
    for c in node.children:
        c.alive = False
        _kill(c)


def merged_dag_prompt(rng, schedule=(2, 2, 2, 2, 1, 1), root_lo=512, root_hi=1024,
                      step_lo=64, step_hi=1024, merge_p=0.25):
    """One prompt of the merged-DAG rollout.

    A full tree with branching ``schedule`` is drawn; then nodes at depths 1..H-1 are visited in
    BFS order and each alive node that is neither merged nor a representative is, with
    probability ``merge_p``, virtually merged into a representative drawn uniformly from the
    other alive, unmerged nodes of the same depth (same depth: never an ancestor/descendant
    pair, Sec. 3.2). The merged node keeps its own segment, its descendants are never generated
    (their budget is saved), and branches reaching it continue along the representative's
    successors -- the shared suffix of the graph suffix C_g.

    Returns (segment lengths, paths, stats).
    """
    H = len(schedule)
    root = _Node(0)
    levels = [[root]]
    for b in schedule:
        nxt = []
        for u in levels[-1]:
            for _ in range(b):
                c = _Node(u.depth + 1)
                u.children.append(c)
                nxt.append(c)
        levels.append(nxt)
    merges = 0
    for d in range(1, H):
        for v in levels[d]:
            if not v.alive or v.merged_into is not None or v.is_rep:
                continue
            if rng.random() < merge_p:
                cands = [u for u in levels[d] if u is not v and u.alive and u.merged_into is None]
                if not cands:
                    continue
                r = cands[int(rng.integers(len(cands)))]
                v.merged_into = r
                r.is_rep = True
                _kill(v)
                merges += 1
    lens = [int(rng.integers(root_lo, root_hi + 1))]
    root.seg = 0
    for d in range(1, H + 1):
        for v in levels[d]:
            if v.alive:
                v.seg = len(lens)
                lens.append(int(rng.integers(step_lo, step_hi + 1)))
    paths = []
    nleaf = int(np.prod(schedule))
    for slot in range(nleaf):
        digits = []
        x = slot
        for b in reversed(schedule):
            digits.append(x % b)
            x //= b
        digits.reverse()
        cur = root
        path = [root.seg]
        for d in range(H):
            child = cur.children[digits[d]]
            path.append(child.seg)
            cur = child.merged_into if child.merged_into is not None else child
        paths.append(path)
    step_nodes = sum(1 for d in range(1, H + 1) for v in levels[d] if v.alive)
    merged_nodes = sum(1 for d in range(1, H + 1) for v in levels[d]
                       if v.alive and v.merged_into is not None)
    return lens, paths, {"merges": merges, "step_nodes": step_nodes, "merged_nodes": merged_nodes}


def _merged_dag_structure(prompts: int, seed: int, merge_p: float):
    rng = np.random.default_rng(seed)
    lens: List[int] = []
    paths: List[List[int]] = []
    step_nodes = merged = 0
    for _ in range(prompts):
        l, p, st = merged_dag_prompt(rng, merge_p=merge_p)
        base = len(lens)
        lens += l
        paths += [[base + s for s in path] for path in p]
        step_nodes += st["step_nodes"]
        merged += st["merged_nodes"]
    info = {"config": 3, "prompts": prompts, "merge_p": merge_p,
            "merged_fraction": merged / max(1, step_nodes)}
    return lens, paths, info


def config3_merged_dag(prompts: int = 64, slack_pages: int = 0, poison: bool = False,
                       kzero_tags: bool = False, seed: Optional[int] = None,
                       merge_p: float = 0.25) -> Workload:
    """Merged-DAG rollout, 7B shape: 64 prompts, root U{512..1024}, depth-6 graph with 16 leaves,
    steps U{64..1024}, per-node merge probability 0.25; 1024 branches of 7 segments."""
    seed = SEED_BASE + 3 if seed is None else seed
    lens, paths, info = _merged_dag_structure(prompts, seed, merge_p)
    g = assemble_graph(lens, paths, seed, slack_pages, info)
    return make_workload(f"merged-DAG rollout, 7B shape (28/4/128, {prompts} prompts, "
                         f"{len(paths)} branches)", g, 28, 4, 128, "bf16", seed, poison, kzero_tags)


def _fill(rng, total: int, lo: int, hi: int) -> List[int]:
    """Segments of length U{lo..hi} until ``total`` tokens, the last one clipped."""
    out = []
    rem = int(total)
    while rem > 0:
        n = min(int(rng.integers(lo, hi + 1)), rem)
        out.append(n)
        rem -= n
    return out


def config4_long(prompts: int = 32, branches_per_prompt: int = 8, path_tokens: int = 16384,
                 slack_pages: int = 0, poison: bool = False, kzero_tags: bool = False,
                 seed: Optional[int] = None) -> Workload:
    """Long-reasoning 32B shape (40/8/128): 32 prompts x 8 branches, every path 16384 tokens,
    shared prefix fraction rho ~ U[0.5, 0.9] per prompt (1024-token prompt + U{256..2048}
    steps), private suffixes of U{256..2048} steps; last segments clipped."""
    seed = SEED_BASE + 4 if seed is None else seed
    rng = np.random.default_rng(seed)
    lens: List[int] = []
    paths: List[List[int]] = []
    for _ in range(prompts):
        rho = float(rng.uniform(0.5, 0.9))
        shared = int(round(path_tokens * rho))
        pre = [1024] + _fill(rng, shared - 1024, 256, 2048)
        base = len(lens)
        lens += pre
        pre_ids = list(range(base, base + len(pre)))
        for _ in range(branches_per_prompt):
            priv = _fill(rng, path_tokens - shared, 256, 2048)
            b0 = len(lens)
            lens += priv
            paths.append(pre_ids + list(range(b0, b0 + len(priv))))
    g = assemble_graph(lens, paths, seed, slack_pages,
                       {"config": 4, "prompts": prompts, "path_tokens": path_tokens})
    return make_workload(f"long-reasoning 32B shape (40/8/128, {prompts}x{branches_per_prompt} "
                         f"branches, {path_tokens}-token paths)", g, 40, 8, 128, "bf16", seed,
                         poison, kzero_tags)


def config5_chain(paths_n: int = 256, path_tokens: int = 8192, slack_pages: int = 0,
                  poison: bool = False, kzero_tags: bool = False,
                  seed: Optional[int] = None) -> Workload:
    """Chain baseline, 7B shape: independent single-segment paths (flat paged decode)."""
    seed = SEED_BASE + 5 if seed is None else seed
    lens = [path_tokens] * paths_n
    paths = [[i] for i in range(paths_n)]
    g = assemble_graph(lens, paths, seed, slack_pages, {"config": "5-chain"})
    return make_workload(f"chain baseline, 7B shape ({paths_n} x {path_tokens} tokens)", g,
                         28, 4, 128, "bf16", seed, poison, kzero_tags)


def equal_budget_tree_prompt(rng, depth: int = 8, max_leaves: int = 16, root_len: int = 1024,
                             prompt_tokens: int = 65536):
    """One prompt of the equal-budget graph case: a depth-``depth`` step tree grown breadth
    first, each frontier node drawing b in {2,3} but capped so the prompt never exceeds
    ``max_leaves`` leaves; every step segment gets an equal share of the prompt's budget
    (remainder +1 in BFS order), so each prompt holds exactly ``prompt_tokens`` unique tokens."""
    parent = [-1]
    frontier = [0]
    for _ in range(depth):
        leaves = len(frontier)
        nxt = []
        for k, u in enumerate(frontier):
            b = int(rng.integers(2, 4))
            # leaves if u gets b children: already-expanded children + b + unexpanded rest
            room = max_leaves - (len(nxt) + (leaves - k - 1))
            b = max(1, min(b, room))
            for _ in range(b):
                parent.append(u)
                nxt.append(len(parent) - 1)
        frontier = nxt
    n_steps = len(parent) - 1
    budget = prompt_tokens - root_len
    base, rem = divmod(budget, n_steps)
    lens = [root_len] + [base + (1 if i < rem else 0) for i in range(n_steps)]
    paths = []
    for leaf in frontier:
        p = []
        u = leaf
        while u != -1:
            p.append(u)
            u = parent[u]
        paths.append(p[::-1])
    return lens, paths


def config5_graph(prompts: int = 32, slack_pages: int = 0, poison: bool = False,
                  kzero_tags: bool = False, seed: Optional[int] = None) -> Workload:
    """Graph case at the chain's token budget: 32 prompts of exactly 65536 unique tokens (1024
    root + equal-length steps), depth-8 trees with branching 2..3 capped at 16 leaves."""
    seed = SEED_BASE + 5 + 100 if seed is None else seed
    rng = np.random.default_rng(seed)
    lens: List[int] = []
    paths: List[List[int]] = []
    for _ in range(prompts):
        l, p = equal_budget_tree_prompt(rng)
        base = len(lens)
        lens += l
        paths += [[base + s for s in path] for path in p]
    g = assemble_graph(lens, paths, seed, slack_pages, {"config": "5-graph", "prompts": prompts})
    return make_workload(f"equal-budget graph, 7B shape ({prompts} prompts, {len(paths)} "
                         f"branches)", g, 28, 4, 128, "bf16", seed, poison, kzero_tags)


def with_new_steps(lens: Sequence[int], paths: Sequence[Sequence[int]],
                   step_lens: Sequence[int]):
    """Give every branch a new private segment (the step being extended) at the end of its
    path: branch b's new segment has step_lens[b] tokens."""
    lens = list(lens)
    out = []
    for p, n in zip(paths, step_lens):
        out.append(list(p) + [len(lens)])
        lens.append(int(n))
    return lens, out


def make_extend_workload(name: str, graph: RolloutGraph, query_counts: Sequence[int], Hq: int,
                         Hkv: int, D: int, dtype: str, seed: int,
                         poison: bool = False) -> Workload:
    """Pool as in draw_data; q [sum(query_counts)][Hq][D] from the data stream after the
    decode queries (i.i.d. N(0,1) rounded to dtype)."""
    _, pool = draw_data(graph, Hq, Hkv, D, dtype, seed, poison=poison)
    counts = np.asarray(query_counts, dtype=np.int32)
    nchunks = (graph.num_pages + _DRAW_CHUNK_PAGES - 1) // _DRAW_CHUNK_PAGES
    q = _randn(seed, nchunks + 1, (int(counts.sum()), Hq, D))
    q = _bf16_rne(q) if dtype == "bf16" else q
    return Workload(name, graph, Hq, Hkv, D, dtype, q, pool, seed, counts)


def config3_extend(prompts: int = 64, n_query: int = 16, slack_pages: int = 0,
                   poison: bool = False, seed: Optional[int] = None) -> Workload:
    """The merged-DAG rollout (7B shape) where every branch extends a new private step of
    n_query tokens, all of them queries (a multi-token step: drafted tokens checked at once)."""
    seed = SEED_BASE + 13 if seed is None else seed
    lens, paths, info = _merged_dag_structure(prompts, seed, 0.25)
    lens, paths = with_new_steps(lens, paths, [n_query] * len(paths))
    info.update({"config": "3-extend", "n_query": n_query})
    g = assemble_graph(lens, paths, seed, slack_pages, info)
    return make_extend_workload(f"merged-DAG rollout, 7B shape (28/4/128, {prompts} prompts, "
                                f"{len(paths)} branches), {n_query}-token extend", g,
                                [n_query] * len(paths), 28, 4, 128, "bf16", seed, poison)


# ----------------------------------------------------------------------------------------------
# Rollout states and their embeddings (equivalence detection)
# ----------------------------------------------------------------------------------------------

@dataclasses.dataclass
class StateWorkload:
    """States of a batch of prompts' rollout graphs: generation predecessors (each prompt's
    states consecutive, root first, p(v) < v) and one embedding per state."""
    name: str
    parent: np.ndarray            # int32 [N], -1 for a prompt's root
    z: torch.Tensor               # CPU [N][dim] bfloat16
    kappa: float
    seed: int

    def z_bits(self) -> np.ndarray:
        return self.z.view(torch.int16).numpy().view(np.uint16)


def state_forest(prompts: int, schedule: Sequence[int]) -> np.ndarray:
    """Full trees with the per-layer branching `schedule` (each state at depth h-1 samples
    schedule[h-1] continuations), numbered breadth first inside each prompt."""
    parent: List[int] = []
    for _ in range(prompts):
        root = len(parent)
        parent.append(-1)
        level = [root]
        for b in schedule:
            nxt = []
            for u in level:
                for _ in range(b):
                    nxt.append(len(parent))
                    parent.append(u)
            level = nxt
    return np.asarray(parent, dtype=np.int32)


def draw_state_embeddings(parent: np.ndarray, dim: int, seed: int, share: float = 3.0,
                          stay: float = 0.1, sigma: float = 0.2) -> torch.Tensor:
    """Clustered synthetic embeddings, bf16 [N][dim].

    Within a prompt, the n_h states of depth h >= 1 each draw a semantic centre from a pool of
    ceil(share * n_h) centres, except that with probability `stay` a state of depth >= 2 keeps
    its predecessor's centre (a step that does not change the summarised state); z_v is its
    centre plus sigma-scaled noise, all components N(0, 1).  States with one centre have
    cosine near 1 / (1 + sigma^2) (0.96 at sigma = 0.2), others near 0.
    """
    rng = np.random.default_rng(seed)
    N = len(parent)
    depth = np.zeros(N, dtype=np.int64)
    prompt = np.zeros(N, dtype=np.int64)
    for v in range(N):
        p = int(parent[v])
        depth[v] = 0 if p < 0 else depth[p] + 1
        prompt[v] = v if p < 0 else prompt[p]
    groups: Dict = {}
    for v in range(N):
        groups.setdefault((int(prompt[v]), int(depth[v])), []).append(v)
    center = np.zeros(N, dtype=np.int64)
    ncent = 0
    for (_, h), ids in groups.items():          # insertion order: by prompt, then depth
        if h == 0:
            center[ids[0]] = ncent
            ncent += 1
            continue
        pool = max(1, int(math.ceil(share * len(ids))))
        pick = rng.integers(0, pool, size=len(ids))
        keep = rng.random(len(ids)) < stay
        for u, k, kp in zip(ids, pick, keep):
            center[u] = center[parent[u]] if (kp and h > 1) else ncent + int(k)
        ncent += pool
    # Centres and noise in chunks of rows, chunk c from its own generator (seed, stream), so
    # the chunks are drawn in parallel and the values do not depend on the thread count.
    import concurrent.futures
    CH = 4096
    centres = torch.empty((ncent, dim), dtype=torch.float32)
    z = torch.empty((N, dim), dtype=torch.bfloat16)
    cidx = torch.from_numpy(center)

    def draw_centres(c):
        gen = torch.Generator(device="cpu")
        gen.manual_seed(_chunk_seed(seed, 2 * c))
        r0, r1 = c * CH, min(ncent, (c + 1) * CH)
        centres[r0:r1] = torch.randn((r1 - r0, dim), generator=gen, dtype=torch.float32)

    def draw_rows(c):
        gen = torch.Generator(device="cpu")
        gen.manual_seed(_chunk_seed(seed, 2 * c + 1))
        r0, r1 = c * CH, min(N, (c + 1) * CH)
        x = torch.randn((r1 - r0, dim), generator=gen, dtype=torch.float32).mul_(sigma)
        x += centres[cidx[r0:r1]]
        z[r0:r1] = _bf16_rne(x)

    workers = max(1, min(16, os.cpu_count() or 1))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(draw_centres, range((ncent + CH - 1) // CH)))
        list(ex.map(draw_rows, range((N + CH - 1) // CH)))
    return z


def state_rewards(parent: np.ndarray, seed: int, p_correct: float = 0.5,
                  p_stopped: float = 0.1) -> np.ndarray:
    """Verifier outcomes of a forest's terminal states: every leaf is terminal with R ~
    Bernoulli(p_correct), except that a fraction p_stopped of the leaves stopped early (no
    answer, -1); inner states are -1."""
    rng = np.random.default_rng(seed)
    N = len(parent)
    kids = np.bincount(parent[parent >= 0], minlength=N)
    r = np.where(kids == 0, (rng.random(N) < p_correct).astype(np.int32), -1).astype(np.int32)
    r[(kids == 0) & (rng.random(N) < p_stopped)] = -1
    return r


def equiv_batch(prompts: int = 512, schedule: Sequence[int] = (4, 5, 3, 2), dim: int = 4096,
                kappa: float = 0.92, seed: Optional[int] = None) -> StateWorkload:
    """One training batch's states: `prompts` rollout graphs with branching schedule T (205
    states per prompt at T = {4, 5, 3, 2}), embeddings of width `dim`, threshold kappa."""
    seed = SEED_BASE + 21 if seed is None else seed
    parent = state_forest(prompts, schedule)
    z = draw_state_embeddings(parent, dim, seed)
    return StateWorkload(f"rollout states ({prompts} prompts, T={tuple(schedule)}, "
                         f"{len(parent)} states, dim {dim})", parent, z, kappa, seed)


CONFIGS = {
    "c1": config1_tiny,
    "c2": config2_tree,
    "c3": config3_merged_dag,
    "c4": config4_long,
    "c5chain": config5_chain,
    "c5graph": config5_graph,
}


# ----------------------------------------------------------------------------------------------
# Small random graphs (fuzzing and edge cases)
# ----------------------------------------------------------------------------------------------

def random_graph(rng, n_segments: int, n_branches: int, max_len: int, max_path: int,
                 slack_pages: int = 0, seed: int = 0) -> RolloutGraph:
    """Random segment lengths in [1, max_len] and random duplicate-free paths."""
    lens = [int(rng.integers(1, max_len + 1)) for _ in range(n_segments)]
    paths = []
    for _ in range(n_branches):
        k = int(rng.integers(1, min(max_path, n_segments) + 1))
        paths.append([int(x) for x in rng.choice(n_segments, size=k, replace=False)])
    return assemble_graph(lens, paths, seed, slack_pages, {"random": True})


def sample_branches(graph: RolloutGraph, n: int, seed: int) -> np.ndarray:
    """A seeded sample of branch ids (sorted), for checking full-size runs row by row."""
    B = graph.num_branches
    if n >= B:
        return np.arange(B)
    return np.sort(np.random.default_rng(seed).choice(B, size=n, replace=False))
