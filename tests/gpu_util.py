"""Helpers shared by the GPU tests: run the HIP path through the C ABI and the oracle on the
same seeded inputs, and compare."""
import math
import sys

import numpy as np
import torch

from oracle import graphattn_oracle as O
from paper_2606_18954_amd import graphattn as G

TOL_OUT = 1e-2   # max |out_gpu - out_oracle|, bf16 inputs, fp32 accumulation
TOL_LSE = 1e-3   # max |lse_gpu - lse_oracle|


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    G.load_library()


def params_of(wl, scale=0.0, out_f32=False):
    return G.make_params(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.graph.num_pages,
                         wl.dtype, scale, out_f32)


def to_device(wl):
    return wl.q.cuda(), wl.pool.cuda()


def gpu_decode(wl, q=None, pool=None, graph=None, out_f32=False):
    require_gpu()
    if q is None:
        q, pool = to_device(wl)
    hg = G.HostGraph.from_graph(wl.graph if graph is None else graph)
    out, lse = G.decode(q, pool, hg, params_of(wl, out_f32=out_f32))
    torch.cuda.synchronize()
    return out.double().cpu().numpy(), lse.double().cpu().numpy()


def oracle_decode(wl, branches=None, graph=None):
    g = wl.graph if graph is None else graph
    return O.decode(wl.q_bits(), wl.pool_bits(), g.seg_len, g.seg_page_offsets, g.seg_pages,
                    g.path_offsets, g.path_segs, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
                    wl.dtype, branches=branches)


def oracle_decode_all(wl, chunk=128):
    """The oracle over every branch, a chunk of branches at a time, with a progress line per
    chunk (the full-size configurations take tens of seconds)."""
    B = wl.graph.num_branches
    outs, lses = [], []
    for b0 in range(0, B, chunk):
        o, l = oracle_decode(wl, list(range(b0, min(B, b0 + chunk))))
        outs.append(o)
        lses.append(l)
        say(f"[oracle] {wl.name}: branches {b0}..{min(B, b0 + chunk) - 1} of {B}")
    return np.concatenate(outs), np.concatenate(lses)


def compare(tag, got_out, got_lse, ref_out, ref_lse, tol_out=TOL_OUT, tol_lse=TOL_LSE):
    assert got_out.shape == ref_out.shape and got_lse.shape == ref_lse.shape
    assert np.isfinite(got_out).all(), f"{tag}: non-finite output"
    assert np.isfinite(got_lse).all(), f"{tag}: non-finite lse"
    dout = float(np.abs(got_out - ref_out).max()) if got_out.size else 0.0
    dlse = float(np.abs(got_lse - ref_lse).max()) if got_lse.size else 0.0
    say(f"[parity] {tag}: max|dout|={dout:.3e} max|dlse|={dlse:.3e}")
    assert dout <= tol_out, f"{tag}: max|dout|={dout}"
    assert dlse <= tol_lse, f"{tag}: max|dlse|={dlse}"
    return dout, dlse


def check_workload(wl, branches=None, tol_out=TOL_OUT, tol_lse=TOL_LSE, out_f32=False):
    g = wl.graph
    say(f"[case] {wl.name}: B={g.num_branches} S={g.num_segments} pages={g.num_pages} "
        f"sampled={'all' if branches is None else len(branches)} out_f32={out_f32}")
    go, gl = gpu_decode(wl, out_f32=out_f32)
    oo, ol = oracle_decode(wl, branches)
    if branches is not None:
        go, gl = go[branches], gl[branches]
    return compare(wl.name, go, gl, oo, ol, tol_out, tol_lse)
