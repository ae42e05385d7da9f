"""Equivalence detection and the graph suffix on the GPU (through the C ABI) against the oracle.

Labels and suffix lists are integer results: bit-exact.  The cosine decision is taken in fp32
on the GPU and in float64 by the oracle, so every input here keeps all compared pairs at least
1e-3 from kappa (the kernel's error bound is 2.5e-4 at dim 4096); each test checks that margin
with the oracle before comparing.
"""
import numpy as np
import pytest
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import graphattn as G
from paper_2606_18954_amd import workloads as W

from gpu_util import require_gpu, say

pytestmark = pytest.mark.gpu
MARGIN = 1e-3


def gpu_labels(z, parent, kappa):
    require_gpu()
    lab = G.equivalence_classes(z.cuda(), G.HostForest(parent), kappa)
    torch.cuda.synchronize()
    return lab.cpu().numpy()


def check(wl, kappa=None):
    kappa = wl.kappa if kappa is None else kappa
    say(f"[case] {wl.name} kappa={kappa}")
    m = O.similarity_margin(wl.z_bits(), "bf16", wl.parent, kappa)
    assert m >= MARGIN, f"inputs within {m} of kappa"
    ref = O.equivalence_classes(wl.z_bits(), "bf16", wl.parent, kappa)
    got = gpu_labels(wl.z, wl.parent, kappa)
    merged = int((ref != np.arange(len(ref))).sum())
    say(f"[equiv] {wl.name}: {len(set(ref.tolist()))} classes, {merged} merged states, "
        f"margin {m:.4f}, equal={np.array_equal(got, ref)}")
    assert np.array_equal(got, ref)
    return got


@pytest.mark.parametrize("prompts,sched,dim", [(3, (4, 5, 3, 2), 256), (2, (4, 5, 3, 2), 4096),
                                               (4, (2, 2, 2, 2, 2), 128), (2, (6, 6, 8), 64),
                                               (5, (8, 8), 192)])
def test_classes_match_oracle(prompts, sched, dim):
    check(W.equiv_batch(prompts=prompts, schedule=sched, dim=dim, seed=prompts * 31 + dim))


def test_threshold_extremes_and_ancestor_rule():
    wl = W.equiv_batch(prompts=2, schedule=(3, 4), dim=64, seed=7)
    N = len(wl.parent)
    assert np.array_equal(gpu_labels(wl.z, wl.parent, 2.0), np.arange(N))
    lab = gpu_labels(wl.z, wl.parent, -2.0)
    assert np.array_equal(lab, O.equivalence_classes(wl.z_bits(), "bf16", wl.parent, -2.0))
    chain = np.array([-1, 0, 1, 2, 3, -1, 5, 5, 6, 7], dtype=np.int32)
    z = torch.ones((10, 64), dtype=torch.bfloat16)
    assert gpu_labels(z, chain, 0.9).tolist() == [0, 1, 2, 3, 4, 5, 6, 6, 6, 6]
    z[3] = 0                                          # a zero embedding is never linked
    zero = np.array([-1, 0, 0, 0, 0], dtype=np.int32)
    assert gpu_labels(z[:5], zero, 0.5).tolist() == [0, 1, 1, 3, 1]


def test_graph_suffix_matches_oracle():
    wl = W.equiv_batch(prompts=3, schedule=(4, 5, 3, 2), dim=256, seed=11)
    lab = check(wl)
    fo = G.HostForest(wl.parent)
    offs, states = G.graph_suffix(torch.from_numpy(lab).cuda(), fo)
    torch.cuda.synchronize()
    ro, rs = O.graph_suffix(lab, wl.parent)
    say(f"[suffix] {len(rs)} entries")
    assert np.array_equal(offs.cpu().numpy(), ro) and np.array_equal(states.cpu().numpy(), rs)
    # too small a buffer: GA_ERANGE, total reported, outputs untouched
    with pytest.raises(G.GraphAttnError) as e:
        G.graph_suffix(torch.from_numpy(lab).cuda(), fo, capacity=len(rs) - 1)
    assert e.value.status == G.GA_ERANGE


def test_graph_suffix_fixture_on_gpu():
    import json, os
    with open(os.path.join(os.path.dirname(__file__), "golden", "graph_suffix_small.json")) as f:
        fx = json.load(f)
    offs, states = G.graph_suffix(torch.tensor(fx["labels"], dtype=torch.int32).cuda(),
                                  G.HostForest(fx["parent"]))
    torch.cuda.synchronize()
    assert offs.cpu().tolist() == fx["offsets"] and states.cpu().tolist() == fx["states"]


def test_full_batch_sampled_prompts():
    """The benchmark's batch (512 prompts x 205 states, dim 4096): labels of sampled prompts
    against the oracle run on those prompts alone (classes never cross prompts)."""
    wl = W.equiv_batch()
    got = gpu_labels(wl.z, wl.parent, wl.kappa)
    per = 205
    for p in [0, 1, 137, 300, 511]:
        a, b = p * per, (p + 1) * per
        sub = wl.parent[a:b].copy()
        sub[1:] -= a
        zb = wl.z_bits()[a:b]
        assert O.similarity_margin(zb, "bf16", sub, wl.kappa) >= MARGIN
        ref = O.equivalence_classes(zb, "bf16", sub, wl.kappa) + a
        say(f"[equiv] prompt {p}: {len(set(ref.tolist()))} classes")
        assert np.array_equal(got[a:b], ref), p


def test_forest_plan_serves_several_thresholds():
    """One uploaded forest, classes at two thresholds and the suffix of each, against the
    one-shot calls and the oracle."""
    wl = W.equiv_batch(prompts=3, schedule=(4, 5, 3, 2), dim=512, seed=19)
    z = wl.z.cuda()
    with G.Forest(wl.parent) as f:
        for kappa in (0.92, 0.5):
            assert O.similarity_margin(wl.z_bits(), "bf16", wl.parent, kappa) >= MARGIN
            lab = f.classes(z, kappa)
            torch.cuda.synchronize()
            ref = O.equivalence_classes(wl.z_bits(), "bf16", wl.parent, kappa)
            assert np.array_equal(lab.cpu().numpy(), ref)
            ro, rs = O.graph_suffix(ref, wl.parent)
            offs = torch.empty(len(wl.parent) + 1, dtype=torch.int64, device="cuda")
            st = torch.empty(len(rs) + 5, dtype=torch.int32, device="cuda")
            n = f.suffix(lab, offs, st)
            torch.cuda.synchronize()
            assert n == len(rs)
            assert np.array_equal(offs.cpu().numpy(), ro)
            assert np.array_equal(st[:n].cpu().numpy(), rs)
