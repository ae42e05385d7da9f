"""Pins of the oracle's graph reward (node scores, step rewards) and dual-group advantage
against facts that do not come from the oracle itself: hand-derived fixtures (one with a_Q at
the root; two more with a_Q below it, routes shared by several members and classes, a shared
edge whose source's group differs from its class label's and a member of undefined score),
hand-derived anchors, the Monte Carlo rate the score reduces to without merges or with w = 0,
the pooled closed form at w = 1, and the z-score invariants of the correctness groups.
"""
import ast
import json
import math
import os

import numpy as np
import pytest

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fixture():
    with open(os.path.join(GOLDEN, "graph_reward_small.json")) as f:
        return json.load(f)


def _euler(parent):
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
    return tin, tout


def _random_rollout(seed, prompts=3, sched=(3, 3, 2), merge_every=5):
    rng = np.random.default_rng(seed)
    parent = W.state_forest(prompts, sched)
    N = len(parent)
    kids = np.bincount(parent[parent >= 0], minlength=N)
    reward = np.where(kids == 0, rng.integers(0, 2, N), -1)
    reward[rng.random(N) < 0.1] = -1                # some leaves stopped early
    labels = np.arange(N, dtype=np.int32)
    depth = O.state_depths(parent)
    roots = np.nonzero(parent < 0)[0].tolist() + [N]
    for a, b in zip(roots[:-1], roots[1:]):         # link a few same-depth states per prompt
        for v in range(a + 1, b, merge_every):
            same = [u for u in range(a + 1, b) if depth[u] == depth[v] and u != v]
            if same:
                u = int(rng.choice(same))
                lo, hi = min(labels[u], labels[v]), max(labels[u], labels[v])
                labels[labels == hi] = lo
    sim = rng.uniform(-0.3, 1.0, N)
    return parent, reward, labels, sim


def check_fixture(mod):
    fx = _fixture()
    res = mod.graph_advantages(np.array(fx["parent"]), np.array(fx["labels"]),
                               np.array(fx["reward"]), np.array(fx["edge_sim"]), fx["w"],
                               fx["lambda_eff"])
    for k in ["S", "r", "A_cor", "A_eff", "A_dual"]:
        exp = np.array([np.nan if x is None else x for x in fx[k]])
        assert np.allclose(res[k], exp, rtol=0, atol=1e-12, equal_nan=True), k


def check_monte_carlo_rate(mod, seed=61):
    """Without merges, and with merges at w = 0, S(v) is the share of correct terminal states
    in v's subtree (counted here with the test's own Euler intervals)."""
    parent, reward, labels, sim = _random_rollout(seed)
    tin, tout = _euler(parent)
    N = len(parent)
    for lab, w in [(np.arange(N), 0.7), (labels, 0.0)]:
        S = mod.node_scores(parent, lab, reward, w)
        for v in range(N):
            under = [z for z in range(N) if reward[z] >= 0 and tin[v] <= tin[z] < tout[v]]
            if under:
                assert abs(S[v] - sum(reward[z] for z in under) / len(under)) < 1e-15
            else:
                assert np.isnan(S[v])


def check_full_pooling(mod, seed=62):
    """At w = 1 every member of a class gets the class's pooled rate."""
    parent, reward, labels, sim = _random_rollout(seed)
    c, t = mod.subtree_outcomes(parent, reward)
    S = mod.node_scores(parent, labels, reward, 1.0)
    for lab in set(labels.tolist()):
        m = labels == lab
        if t[m].sum() > 0:
            assert np.allclose(S[m], c[m].sum() / t[m].sum(), rtol=0, atol=1e-15)


def check_step_reward_discount(mod):
    parent = np.array([-1, 0, 0, 0])
    S = np.array([0.5, 1.0, 0.0, 0.25])
    r = mod.step_rewards(parent, S, np.array([0.0, -0.4, 1.0, 0.5]))
    assert np.isnan(r[0]) and r[1] == 0.5 and r[2] == 0.0 and r[3] == -0.125


def check_correctness_groups(mod, seed=63):
    """In a group without shared successors (C_g(u) = C(u)), the advantages of u's edges are the
    z-scores of their rewards: mean 0 and population variance 1 (or all 0)."""
    parent, reward, labels, sim = _random_rollout(seed)
    N = len(parent)
    res = mod.graph_advantages(parent, np.arange(N), reward, sim, 0.7, 0.3)
    for u in range(N):
        kids = [v for v in range(N) if parent[v] == u and not np.isnan(res["r"][v])]
        if len(kids) < 2 or len([v for v in range(N) if parent[v] == u]) < 2:
            continue
        a = res["A_cor"][kids]
        assert abs(a.mean()) < 1e-12
        assert abs(np.mean(a * a) - 1) < 1e-12 or np.all(a == 0)
    assert np.all(res["A_eff"] == 0)                  # no class of two or more


def _routes_fixture():
    with open(os.path.join(GOLDEN, "graph_reward_routes.json")) as f:
        return json.load(f)["cases"]


def exact(expr: str) -> float:
    """Value of a fixture expression: numbers, + - * /, unary minus, sqrt(.) and nan."""
    def ev(n):
        if isinstance(n, ast.Expression):
            return ev(n.body)
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
            return float(n.value)
        if isinstance(n, ast.Name) and n.id == "nan":
            return math.nan
        if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
            return -ev(n.operand)
        if isinstance(n, ast.BinOp) and type(n.op) in _OPS:
            return _OPS[type(n.op)](ev(n.left), ev(n.right))
        if (isinstance(n, ast.Call) and isinstance(n.func, ast.Name) and n.func.id == "sqrt"
                and len(n.args) == 1):
            return math.sqrt(ev(n.args[0]))
        raise ValueError(f"unsupported expression {expr!r}")
    return ev(ast.parse(expr, mode="eval"))


_OPS = {ast.Add: lambda a, b: a + b, ast.Sub: lambda a, b: a - b,
        ast.Mult: lambda a, b: a * b, ast.Div: lambda a, b: a / b}


def check_route_fixture(mod):
    """Two hand-derived rollouts whose arithmetic is written out in the fixture: a class whose
    a_Q lies below the root, edges on the routes of two members and of two classes (summed),
    an edge whose source's correctness group differs from its class label's, and a class with
    a member of undefined score (the gate averages the defined ones)."""
    for fx in _routes_fixture():
        res = mod.graph_advantages(np.array(fx["parent"]), np.array(fx["labels"]),
                                   np.array(fx["reward"]), np.array(fx["edge_sim"]), fx["w"],
                                   fx["lambda_eff"])
        for k in ["S", "r", "A_cor", "A_eff", "A_dual"]:
            exp = np.array([exact(x) for x in fx[k]])
            assert np.allclose(res[k], exp, rtol=0, atol=1e-12, equal_nan=True), (fx["name"], k)


def check_anchors(mod):
    """a_Q, the deepest state that precedes every member (Sec. 3.4), on hand-derived classes;
    above a_Q the z-scores of a class sum to zero, so the advantages alone cannot pin it."""
    for fx in _routes_fixture():
        parent = np.array(fx["parent"])
        for a in fx["anchors"]:
            assert mod.class_anchor(parent, a["members"]) == a["a_Q"], (fx["name"], a)


PINS = [check_fixture, check_monte_carlo_rate, check_full_pooling, check_step_reward_discount,
        check_correctness_groups, check_route_fixture, check_anchors]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_reward_pin(pin):
    pin(O)


ORIG_SCORES = O.node_scores
ORIG_SUFFIX = O.graph_suffix
ORIG_EFF = O.efficiency_advantage
ORIG_COR = O.correctness_advantage


def _anchor_at_root(parent, members):
    x = int(members[0])
    while int(parent[x]) >= 0:
        x = int(parent[x])
    return x


def _efficiency_variant(parent, labels, S, last_write=False, nan_as_zero=False):
    """The oracle's efficiency advantage with one planted change."""
    depth = O.state_depths(parent)
    E = np.zeros(len(parent))
    classes = {}
    for v in range(len(parent)):
        classes.setdefault(int(labels[v]), []).append(v)
    for members in classes.values():
        if len(members) < 2:
            continue
        a = O.class_anchor(parent, members)
        if nan_as_zero:
            gate = sum(0.0 if np.isnan(S[v]) else float(S[v]) for v in members) / len(members)
        else:
            d = [float(S[v]) for v in members if not np.isnan(S[v])]
            gate = sum(d) / len(d) if d else 0.0
        z = O._zscores([-float(depth[v] - depth[a]) for v in members])
        for v, zv in zip(members, z):
            x = v
            while x != a:
                E[x] = gate * zv if last_write else E[x] + gate * zv
                x = int(parent[x])
    return E


def _cor_in_label_group(parent, labels, r):
    """A_cor of every edge taken in the group of its source's class label."""
    offs, states = O.graph_suffix(labels, parent)
    A = np.zeros(len(parent))
    for v in range(len(parent)):
        if parent[v] < 0 or np.isnan(r[v]):
            continue
        u = int(labels[int(parent[v])])
        grp = [int(x) for x in states[offs[u]:offs[u + 1]]]
        if v not in grp or len(grp) <= 1:
            continue
        ok = [x for x in grp if not np.isnan(r[x])]
        A[v] = O._zscores([float(r[x]) for x in ok], O.SPREAD_FLOOR)[ok.index(v)]
    return A


def _sample_std(values, floor=0.0):
    n = len(values)
    m = sum(values) / n
    sd = math.sqrt(sum((x - m) ** 2 for x in values) / max(1, n - 1))
    return [0.0 if sd <= floor else (x - m) / sd for x in values]


def _own_children_only(labels, parent):
    return ORIG_SUFFIX(np.arange(len(parent)), parent)


@pytest.mark.parametrize("name,attr,repl", [
    ("no_pooling", "node_scores", lambda p, l, r, w: ORIG_SCORES(p, l, r, 0.0)),
    ("sample_std", "_zscores", _sample_std),
    ("shared_successors_ignored", "graph_suffix", _own_children_only),
    ("similarity_not_clipped", "step_rewards",
     lambda parent, S, sim: np.array([np.nan if parent[v] < 0 else
                                      (S[v] - S[parent[v]]) * (1 - sim[v])
                                      for v in range(len(parent))])),
    ("gate_ignored", "efficiency_advantage",
     lambda parent, labels, S: ORIG_EFF(parent, labels, np.ones_like(S))),
    ("anchor_at_prompt_root", "class_anchor", _anchor_at_root),
    ("route_last_write", "efficiency_advantage",
     lambda parent, labels, S: _efficiency_variant(parent, labels, S, last_write=True)),
    ("gate_counts_undefined_as_zero", "efficiency_advantage",
     lambda parent, labels, S: _efficiency_variant(parent, labels, S, nan_as_zero=True)),
    ("cor_in_class_label_group", "correctness_advantage", _cor_in_label_group),
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


def test_equal_scores_are_bit_identical_and_give_no_spread():
    """States 4 and 11 (11 the only child of 4, one class) hold the same terminal evidence and
    the same partners, so S(4) = S(11) exactly (46/91 here) and r(11) = 0: the group of source 4
    then holds rewards that are all 0 by the definition and its z-scores are 0.  A sum of
    w c_own(q) taken in a different order for each state used to leave them one ulp apart and
    turn that ulp into A_cor(11) = -sqrt(3)."""
    parent = np.array([-1, 0, 1, 2, 3, 0, 5, 0, 3, 0, 2, 4, 6, 10, 6, 11, 15, 13, 14, 14],
                      dtype=np.int64)
    labels = np.array([0] + [1] * 17 + [18, 1])
    reward = np.array([-1, -1, -1, -1, -1, -1, -1, 0, 0, 0, -1, -1, 1, -1, -1, -1, 1, 0, 1, 0])
    S = O.node_scores(parent, labels, reward, 0.3)
    assert S[4] == S[11]
    c, t = O.subtree_outcomes(parent, reward)
    cq = int(c[labels == 1].sum()) - int(c[4])
    tq = int(t[labels == 1].sum()) - int(t[4])
    assert S[4] == pytest.approx((c[4] + 0.3 * cq) / (t[4] + 0.3 * tq), rel=1e-15)
    sim = np.linspace(-0.9, 0.9, len(parent))
    r = O.step_rewards(parent, S, sim)
    assert r[11] == 0.0
    A = O.correctness_advantage(parent, labels, r)
    offs, st = O.graph_suffix(labels, parent)
    grp = st[offs[4]:offs[5]].tolist()
    assert grp == [11, 15, 16, 17] and all(r[x] == 0.0 for x in grp)
    assert A[11] == 0.0


def test_spread_floor_keeps_real_spreads():
    """A real spread far below the scores' scale but above rounding still gives z-scores, and
    one within rounding gives none."""
    assert O._zscores([0.0, 1e-9], O.SPREAD_FLOOR) == pytest.approx([-1.0, 1.0])
    assert O._zscores([0.0, 0.0, 0.0, -1.1e-16], O.SPREAD_FLOOR) == [0.0] * 4
    assert O._zscores([0.0, 0.0, 0.0, -1.1e-16])[3] == pytest.approx(-math.sqrt(3))
