"""Pins of the oracle's equivalence detection (cosine over compared pairs, union-find classes)
and graph suffix, against facts that do not come from the oracle itself.

Each check takes the oracle module, so the planted-mistake test at the bottom can swap a piece
of it for a plausible wrong one and confirm that some pin fails.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.sparse import coo_matrix
from scipy.sparse.csgraph import connected_components

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _euler(parent):
    """Entry / exit times of an explicit depth-first walk (the test's own ancestor test)."""
    N = len(parent)
    kids = [[] for _ in range(N)]
    for v, p in enumerate(parent):
        if p >= 0:
            kids[p].append(v)
    tin, tout, clock = [0] * N, [0] * N, 0
    for r in [v for v in range(N) if parent[v] < 0]:
        stack = [(r, 0)]
        while stack:
            v, i = stack.pop()
            if i == 0:
                tin[v] = clock
                clock += 1
            if i < len(kids[v]):
                stack.append((v, i + 1))
                stack.append((kids[v][i], 0))
            else:
                tout[v] = clock
    return np.array(tin), np.array(tout)


def _reference_labels(z_bits, parent, kappa):
    """Components (scipy) of the graph of compared pairs with cosine >= kappa, labelled by
    their smallest state id; cosines from one float64 matrix product."""
    z = torch.from_numpy(z_bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    zn = z / np.linalg.norm(z, axis=1, keepdims=True)
    sim = zn @ zn.T
    tin, tout = _euler(parent)
    root = np.array([v if parent[v] < 0 else -1 for v in range(len(parent))])
    for v in range(len(parent)):
        if root[v] < 0:
            root[v] = root[parent[v]]
    anc = (tin[:, None] <= tin[None, :]) & (tin[None, :] < tout[:, None])
    ok = (root[:, None] == root[None, :]) & ~anc & ~anc.T & (sim >= kappa)
    np.fill_diagonal(ok, False)
    n, comp = connected_components(coo_matrix(ok), directed=False)
    lab = np.empty(len(parent), dtype=np.int32)
    for c in range(n):
        ids = np.nonzero(comp == c)[0]
        lab[ids] = ids.min()
    return lab


def check_cosine_brute_force(mod, seed=51):
    rng = np.random.default_rng(seed)
    z = torch.from_numpy(rng.standard_normal((6, 40)).astype(np.float32)).to(torch.bfloat16)
    bits = z.view(torch.int16).numpy().view(np.uint16)
    vals = z.double().numpy()
    for u in range(6):
        for v in range(6):
            dot = math.fsum(float(a) * float(b) for a, b in zip(vals[u], vals[v]))
            nu = math.sqrt(math.fsum(float(a) ** 2 for a in vals[u]))
            nv = math.sqrt(math.fsum(float(b) ** 2 for b in vals[v]))
            assert abs(mod.cosine(bits, "bf16", u, v) - dot / (nu * nv)) < 1e-14


def check_classes_against_scipy(mod, seed=52):
    for trial, (prompts, sched, dim) in enumerate([(3, (4, 5, 3, 2), 128), (2, (3, 3, 3), 64),
                                                   (4, (2, 2, 2, 2), 96)]):
        wl = W.equiv_batch(prompts=prompts, schedule=sched, dim=dim, seed=seed + trial)
        for kappa in (0.92, 0.5, 0.97):
            lab = mod.equivalence_classes(wl.z_bits(), "bf16", wl.parent, kappa)
            ref = _reference_labels(wl.z_bits(), wl.parent, kappa)
            assert np.array_equal(lab, ref), (trial, kappa)


def check_threshold_extremes(mod, seed=53):
    """kappa above 1 links nothing; kappa below -1 links every compared pair: a prompt root
    stays alone (it is everyone's ancestor) and, with two or more subtrees under the root, all
    other states form one class; a chain-shaped prompt has no compared pairs at all."""
    parent = np.concatenate([W.state_forest(2, (2, 3)), W.state_forest(1, (1, 1, 1)) + 18])
    parent[18] = -1
    z = W.draw_state_embeddings(parent, 32, seed)
    bits = z.view(torch.int16).numpy().view(np.uint16)
    N = len(parent)
    assert np.array_equal(mod.equivalence_classes(bits, "bf16", parent, 1.5), np.arange(N))
    lab = mod.equivalence_classes(bits, "bf16", parent, -1.5)
    exp = np.arange(N)
    exp[1:9] = 1
    exp[10:18] = 10
    assert np.array_equal(lab, exp)


def check_ancestors_never_compared(mod):
    """Identical embeddings everywhere: a chain merges nothing, siblings merge."""
    chain = np.array([-1, 0, 1, 2, 3], dtype=np.int32)
    z = torch.ones((5, 16), dtype=torch.bfloat16)
    bits = z.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mod.equivalence_classes(bits, "bf16", chain, 0.9), np.arange(5))
    fork = np.array([-1, 0, 0, 1, 2], dtype=np.int32)
    assert mod.equivalence_classes(bits, "bf16", fork, 0.9).tolist() == [0, 1, 1, 1, 1]
    assert mod.compared_pairs(fork) == [(1, 2), (1, 4), (2, 3), (3, 4)]


def check_graph_suffix_fixture(mod):
    with open(os.path.join(GOLDEN, "graph_suffix_small.json")) as f:
        fx = json.load(f)
    offs, states = mod.graph_suffix(np.array(fx["labels"]), np.array(fx["parent"]))
    assert offs.tolist() == fx["offsets"] and states.tolist() == fx["states"]


def check_graph_suffix_without_merges(mod, seed=54):
    """With every state its own class, C_g(u) is exactly u's direct successors."""
    parent = W.state_forest(3, (3, 2, 2))
    offs, states = mod.graph_suffix(np.arange(len(parent)), parent)
    for u in range(len(parent)):
        assert states[offs[u]:offs[u + 1]].tolist() == [c for c in range(len(parent))
                                                        if parent[c] == u]


PINS = [check_cosine_brute_force, check_classes_against_scipy, check_threshold_extremes,
        check_ancestors_never_compared, check_graph_suffix_fixture,
        check_graph_suffix_without_merges]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_equiv_pin(pin):
    pin(O)


ORIG_CLASSES = O.equivalence_classes


def _largest(z, dt, par, k):
    """Classes labelled by their largest member instead of the smallest."""
    lab = ORIG_CLASSES(z, dt, par, k)
    big = {}
    for i, l in enumerate(lab):
        big[l] = max(big.get(l, i), i)
    return np.array([big[l] for l in lab], dtype=np.int32)


def _dot_only(z_raw, dtype, ids):
    z = O.to_f64(z_raw[np.asarray(ids, dtype=np.int64)], dtype)
    return z @ z.T


@pytest.mark.parametrize("name,attr,repl", [
    ("ancestors_compared", "is_ancestor", lambda parent, u, v: u == v),
    ("dot_not_cosine", "similarity_matrix", _dot_only),
    ("depth_as_id", "state_depths", lambda parent: np.arange(len(parent))),
    ("no_depth_rule", "state_depths", lambda parent: -np.arange(len(parent))),
    ("largest_label", "equivalence_classes", lambda z, dt, par, k: _largest(z, dt, par, k)),
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
