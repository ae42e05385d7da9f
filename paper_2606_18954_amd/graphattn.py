"""ctypes binding of libgraphattn.so (argument marshalling only).

Every step of the computation runs in the HIP library; this module only turns numpy index arrays
and torch device tensors into the C ABI's structs and pointers.  If the library is not built, or
the process has no GPU, the compute entry points raise instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgraphattn.so")

GA_OK, GA_EINVAL, GA_ERANGE, GA_ENOMEM, GA_EHIP, GA_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
GA_F32, GA_BF16 = 0, 1
STATUS_NAMES = {0: "GA_OK", -1: "GA_EINVAL", -2: "GA_ERANGE", -3: "GA_ENOMEM", -4: "GA_EHIP",
                -5: "GA_EUNSUPPORTED"}


class GraphAttnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class SegmentTable(ctypes.Structure):
    _fields_ = [("num_segments", ctypes.c_int32),
                ("seg_len", ctypes.POINTER(ctypes.c_int32)),
                ("seg_page_offsets", ctypes.POINTER(ctypes.c_int64)),
                ("seg_pages", ctypes.POINTER(ctypes.c_int32))]


class BranchPaths(ctypes.Structure):
    _fields_ = [("num_branches", ctypes.c_int32),
                ("path_offsets", ctypes.POINTER(ctypes.c_int64)),
                ("path_segs", ctypes.POINTER(ctypes.c_int32))]


class Params(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("out_f32", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("num_segments", ctypes.c_int32), ("num_branches", ctypes.c_int32),
                ("num_entries", ctypes.c_int32), ("chunk_pages", ctypes.c_int32),
                ("rows_per_block", ctypes.c_int32), ("num_items", ctypes.c_int64),
                ("num_partial_rows", ctypes.c_int64), ("num_chains", ctypes.c_int32),
                ("num_query_rows", ctypes.c_int32), ("workgroups_per_cu", ctypes.c_int32),
                ("work_streams", ctypes.c_int32)]


class StateForest(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("parent", ctypes.POINTER(ctypes.c_int32))]


class Advantages(ctypes.Structure):
    _fields_ = [("score", ctypes.c_void_p), ("step_reward", ctypes.c_void_p),
                ("a_cor", ctypes.c_void_p), ("a_eff", ctypes.c_void_p), ("a_dual", ctypes.c_void_p)]


class Profile(ctypes.Structure):
    _fields_ = [("schedules", ctypes.c_int32), ("runs", ctypes.c_int32),
                ("sched_ms", ctypes.c_double), ("attn_ms", ctypes.c_double),
                ("merge_ms", ctypes.c_double)]


_lib = None


def load_library() -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           f"`python -m paper_2606_18954_amd.build_lib` (there is no fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    P = ctypes.POINTER
    lib.graphattn_decode.argtypes = [vp, vp, P(SegmentTable), P(BranchPaths), vp, vp, P(Params), vp]
    lib.graphattn_decode.restype = ctypes.c_int
    lib.graphattn_decode_static.argtypes = lib.graphattn_decode.argtypes
    lib.graphattn_decode_static.restype = ctypes.c_int
    lib.graphattn_plan_create.argtypes = [P(SegmentTable), P(BranchPaths), P(Params), vp, P(vp)]
    lib.graphattn_plan_create.restype = ctypes.c_int
    lib.graphattn_extend.argtypes = [vp, vp, P(SegmentTable), P(BranchPaths), P(i32), vp, vp,
                                     P(Params), vp]
    lib.graphattn_extend.restype = ctypes.c_int
    lib.graphattn_plan_create_extend.argtypes = [P(SegmentTable), P(BranchPaths), P(i32),
                                                 P(Params), vp, P(vp)]
    lib.graphattn_plan_create_extend.restype = ctypes.c_int
    lib.graphattn_kv_append.argtypes = [vp, vp, vp, vp, i32, P(Params), vp]
    lib.graphattn_kv_append.restype = ctypes.c_int
    lib.graphattn_kv_copy.argtypes = [vp, vp, vp, i32, P(Params), vp]
    lib.graphattn_kv_copy.restype = ctypes.c_int
    lib.graphattn_equivalence_classes.argtypes = [vp, i32, i32, P(StateForest), ctypes.c_float,
                                                  vp, vp]
    lib.graphattn_equivalence_classes.restype = ctypes.c_int
    lib.graphattn_graph_suffix.argtypes = [vp, P(StateForest), vp, vp, i64, P(i64), vp]
    lib.graphattn_graph_suffix.restype = ctypes.c_int
    lib.graphattn_forest_create.argtypes = [P(StateForest), vp, P(vp)]
    lib.graphattn_forest_create.restype = ctypes.c_int
    lib.graphattn_forest_classes.argtypes = [vp, vp, i32, i32, ctypes.c_float, vp, vp, vp]
    lib.graphattn_forest_advantages.argtypes = [vp, vp, vp, vp, ctypes.c_double, ctypes.c_double,
                                                P(Advantages), vp]
    lib.graphattn_forest_advantages.restype = ctypes.c_int
    lib.graphattn_forest_classes.restype = ctypes.c_int
    lib.graphattn_forest_suffix.argtypes = [vp, vp, vp, vp, i64, P(i64), vp]
    lib.graphattn_forest_suffix.restype = ctypes.c_int
    lib.graphattn_forest_destroy.argtypes = [vp]
    lib.graphattn_forest_destroy.restype = None
    lib.graphattn_schedule.argtypes = [vp, vp]
    lib.graphattn_schedule.restype = ctypes.c_int
    lib.graphattn_plan_set_lengths.argtypes = [vp, P(i32), vp]
    lib.graphattn_plan_set_lengths.restype = ctypes.c_int
    lib.graphattn_run.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.graphattn_run.restype = ctypes.c_int
    lib.graphattn_plan_info.argtypes = [vp, P(PlanInfo)]
    lib.graphattn_plan_info.restype = ctypes.c_int
    lib.graphattn_plan_debug_dump.argtypes = [vp, vp, P(i64), P(i32), P(i32), P(i32), P(i32),
                                              P(i64), P(i32)]
    lib.graphattn_plan_debug_dump.restype = ctypes.c_int
    lib.graphattn_plan_profile.argtypes = [vp, i32]
    lib.graphattn_plan_profile.restype = ctypes.c_int
    lib.graphattn_plan_profile_read.argtypes = [vp, P(Profile)]
    lib.graphattn_plan_profile_read.restype = ctypes.c_int
    lib.graphattn_plan_destroy.argtypes = [vp]
    lib.graphattn_plan_destroy.restype = None
    lib.graphattn_last_error.argtypes = []
    lib.graphattn_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int):
    if status != GA_OK:
        msg = load_library().graphattn_last_error().decode(errors="replace")
        raise GraphAttnError(status, msg)


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class HostGraph:
    """The rollout graph's index arrays as the C structs (keeps the numpy arrays alive)."""

    def __init__(self, seg_len, seg_page_offsets, seg_pages, path_offsets, path_segs):
        self.seg_len = np.ascontiguousarray(seg_len, dtype=np.int32)
        self.seg_page_offsets = np.ascontiguousarray(seg_page_offsets, dtype=np.int64)
        self.seg_pages = np.ascontiguousarray(seg_pages, dtype=np.int32)
        self.path_offsets = np.ascontiguousarray(path_offsets, dtype=np.int64)
        self.path_segs = np.ascontiguousarray(path_segs, dtype=np.int32)
        self.st = SegmentTable(len(self.seg_len), _ptr(self.seg_len, ctypes.c_int32),
                               _ptr(self.seg_page_offsets, ctypes.c_int64),
                               _ptr(self.seg_pages, ctypes.c_int32))
        self.bp = BranchPaths(len(self.path_offsets) - 1, _ptr(self.path_offsets, ctypes.c_int64),
                              _ptr(self.path_segs, ctypes.c_int32))

    @classmethod
    def from_graph(cls, g) -> "HostGraph":
        return cls(g.seg_len, g.seg_page_offsets, g.seg_pages, g.path_offsets, g.path_segs)


def make_params(num_q_heads: int, num_kv_heads: int, head_dim: int, num_pages: int, dtype: str,
                softmax_scale: float = 0.0, out_f32: bool = False) -> Params:
    return Params(num_q_heads, num_kv_heads, head_dim, 16, num_pages,
                  GA_BF16 if dtype == "bf16" else GA_F32, softmax_scale, int(bool(out_f32)))


def _stream_handle(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _dev_ptr(t) -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise ValueError("tensors passed to the library must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return int(t.data_ptr())


def decode(q, pool, graph: HostGraph, params: Params, out=None, lse=None, stream=None):
    """graphattn_decode on torch tensors: returns (out [B, Hq, D], lse [B, Hq] float32)."""
    import torch
    lib = load_library()
    B = graph.bp.num_branches
    if out is None:
        odt = torch.float32 if params.out_f32 else q.dtype
        out = torch.empty((B, params.num_q_heads, params.head_dim), dtype=odt, device=q.device)
    if lse is None:
        lse = torch.empty((B, params.num_q_heads), dtype=torch.float32, device=q.device)
    _check(lib.graphattn_decode(_dev_ptr(q), _dev_ptr(pool), ctypes.byref(graph.st),
                                ctypes.byref(graph.bp), _dev_ptr(out), _dev_ptr(lse),
                                ctypes.byref(params), _stream_handle(stream)))
    return out, lse


def decode_static(q, pool, graph: HostGraph, params: Params, out, lse, stream=None):
    """graphattn_decode_static: graphattn_decode with its workspace in the library's static
    device array (no allocation; the caller passes out and lse)."""
    lib = load_library()
    _check(lib.graphattn_decode_static(_dev_ptr(q), _dev_ptr(pool), ctypes.byref(graph.st),
                                       ctypes.byref(graph.bp), _dev_ptr(out), _dev_ptr(lse),
                                       ctypes.byref(params), _stream_handle(stream)))
    return out, lse


def _counts(query_counts) -> np.ndarray:
    return np.ascontiguousarray(query_counts, dtype=np.int32)


def extend(q, pool, graph: HostGraph, query_counts, params: Params, out=None, lse=None,
           stream=None):
    """graphattn_extend on torch tensors: q [R, Hq, D] with R = sum(query_counts); returns
    (out [R, Hq, D], lse [R, Hq] float32)."""
    import torch
    lib = load_library()
    cnt = _counts(query_counts)
    if len(cnt) != graph.bp.num_branches:
        raise ValueError("one query count per branch")
    R = int(cnt.sum())
    if out is None:
        odt = torch.float32 if params.out_f32 else q.dtype
        out = torch.empty((R, params.num_q_heads, params.head_dim), dtype=odt, device=q.device)
    if lse is None:
        lse = torch.empty((R, params.num_q_heads), dtype=torch.float32, device=q.device)
    _check(lib.graphattn_extend(_dev_ptr(q), _dev_ptr(pool), ctypes.byref(graph.st),
                                ctypes.byref(graph.bp), _ptr(cnt, ctypes.c_int32), _dev_ptr(out),
                                _dev_ptr(lse), ctypes.byref(params), _stream_handle(stream)))
    return out, lse


def kv_append(pool, k_new, v_new, slot_words, params: Params, stream=None):
    """graphattn_kv_append: k_new / v_new [n, Hkv, D], slot_words int32 [n] (device)."""
    lib = load_library()
    n = int(slot_words.numel())
    if k_new.shape[0] != n or v_new.shape[0] != n:
        raise ValueError("one K row and one V row per slot word")
    _check(lib.graphattn_kv_append(_dev_ptr(pool), _dev_ptr(k_new), _dev_ptr(v_new),
                                   _dev_ptr(slot_words), n, ctypes.byref(params),
                                   _stream_handle(stream)))


def kv_copy(pool, src_words, dst_words, params: Params, stream=None):
    """graphattn_kv_copy: src_words / dst_words int32 [n] (device)."""
    lib = load_library()
    n = int(dst_words.numel())
    if src_words.numel() != n:
        raise ValueError("one source word per destination word")
    _check(lib.graphattn_kv_copy(_dev_ptr(pool), _dev_ptr(src_words), _dev_ptr(dst_words), n,
                                 ctypes.byref(params), _stream_handle(stream)))


class HostForest:
    """The states' generation predecessors as the C struct (keeps the array alive)."""

    def __init__(self, parent):
        self.parent = np.ascontiguousarray(parent, dtype=np.int32)
        self.c = StateForest(len(self.parent), _ptr(self.parent, ctypes.c_int32))


def equivalence_classes(z, forest: HostForest, kappa: float, labels=None, stream=None):
    """graphattn_equivalence_classes: z [N, dim] bf16 (device); returns labels int32 [N]."""
    import torch
    lib = load_library()
    N = forest.c.num_states
    if z.dim() != 2 or z.shape[0] != N:
        raise ValueError("one embedding row per state")
    if labels is None:
        labels = torch.empty(N, dtype=torch.int32, device=z.device)
    _check(lib.graphattn_equivalence_classes(_dev_ptr(z), int(z.shape[1]),
                                             GA_BF16 if z.dtype == torch.bfloat16 else GA_F32,
                                             ctypes.byref(forest.c), float(kappa),
                                             _dev_ptr(labels), _stream_handle(stream)))
    return labels


def graph_suffix(labels, forest: HostForest, capacity=None, stream=None):
    """graphattn_graph_suffix: returns (offsets int64 [N + 1], states int32 [total]) on the
    device; sized by a first call when capacity is not given."""
    import torch
    lib = load_library()
    N = forest.c.num_states
    total = ctypes.c_int64(0)
    offs = torch.empty(N + 1, dtype=torch.int64, device=labels.device)
    cap = int(capacity) if capacity is not None else 0
    states = torch.empty(max(cap, 1), dtype=torch.int32, device=labels.device)
    st = lib.graphattn_graph_suffix(_dev_ptr(labels), ctypes.byref(forest.c), _dev_ptr(offs),
                                    _dev_ptr(states), cap, ctypes.byref(total),
                                    _stream_handle(stream))
    if st == GA_ERANGE and capacity is None:
        cap = int(total.value)
        states = torch.empty(max(cap, 1), dtype=torch.int32, device=labels.device)
        st = lib.graphattn_graph_suffix(_dev_ptr(labels), ctypes.byref(forest.c), _dev_ptr(offs),
                                        _dev_ptr(states), cap, ctypes.byref(total),
                                        _stream_handle(stream))
    _check(st)
    return offs, states[:int(total.value)]


class Forest:
    """graphattn_forest_create / classes / suffix / destroy."""

    def __init__(self, parent, stream=None):
        self.lib = load_library()
        self.host = HostForest(parent)
        h = ctypes.c_void_p()
        _check(self.lib.graphattn_forest_create(ctypes.byref(self.host.c), _stream_handle(stream),
                                                ctypes.byref(h)))
        self.handle = h

    def classes(self, z, kappa: float, labels=None, edge_sim=None, stream=None):
        """Class labels; also sim(p(v), v) into edge_sim (float32 [N]) when it is given."""
        import torch
        N = self.host.c.num_states
        if labels is None:
            labels = torch.empty(N, dtype=torch.int32, device=z.device)
        _check(self.lib.graphattn_forest_classes(
            self.handle, _dev_ptr(z), int(z.shape[1]),
            GA_BF16 if z.dtype == torch.bfloat16 else GA_F32, float(kappa), _dev_ptr(labels),
            _dev_ptr(edge_sim), _stream_handle(stream)))
        return labels

    def advantages(self, labels, reward, edge_sim, w: float, lambda_eff: float, out=None,
                   stream=None):
        """Graph reward and dual-group advantage: dict of float64 [N] device tensors (score,
        step_reward, a_cor, a_eff, a_dual)."""
        import torch
        N = self.host.c.num_states
        if out is None:
            out = {k: torch.empty(N, dtype=torch.float64, device=labels.device)
                   for k in ("score", "step_reward", "a_cor", "a_eff", "a_dual")}
        adv = Advantages(*[_dev_ptr(out[k]) for k in ("score", "step_reward", "a_cor", "a_eff",
                                                      "a_dual")])
        _check(self.lib.graphattn_forest_advantages(
            self.handle, _dev_ptr(labels), _dev_ptr(reward), _dev_ptr(edge_sim), float(w),
            float(lambda_eff), ctypes.byref(adv), _stream_handle(stream)))
        return out

    def suffix(self, labels, offsets, states, stream=None) -> int:
        total = ctypes.c_int64(0)
        _check(self.lib.graphattn_forest_suffix(self.handle, _dev_ptr(labels), _dev_ptr(offsets),
                                                _dev_ptr(states), int(states.numel()),
                                                ctypes.byref(total), _stream_handle(stream)))
        return int(total.value)

    def suffix_total(self, labels, offsets, stream=None) -> int:
        """Entries the graph suffix needs (a call with no output buffer)."""
        total = ctypes.c_int64(0)
        st = self.lib.graphattn_forest_suffix(self.handle, _dev_ptr(labels), _dev_ptr(offsets),
                                              None, 0, ctypes.byref(total),
                                              _stream_handle(stream))
        if st not in (GA_OK, GA_ERANGE):
            _check(st)
        return int(total.value)

    def close(self):
        if self.handle:
            self.lib.graphattn_forest_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Plan:
    """graphattn_plan_create (or _create_extend with query_counts) / schedule / run /
    destroy."""

    def __init__(self, graph: HostGraph, params: Params, stream=None, query_counts=None):
        self.lib = load_library()
        self.graph = graph
        self.params = params
        h = ctypes.c_void_p()
        if query_counts is None:
            _check(self.lib.graphattn_plan_create(ctypes.byref(graph.st), ctypes.byref(graph.bp),
                                                  ctypes.byref(params), _stream_handle(stream),
                                                  ctypes.byref(h)))
        else:
            self.query_counts = _counts(query_counts)
            _check(self.lib.graphattn_plan_create_extend(
                ctypes.byref(graph.st), ctypes.byref(graph.bp),
                _ptr(self.query_counts, ctypes.c_int32), ctypes.byref(params),
                _stream_handle(stream), ctypes.byref(h)))
        self.handle = h

    def set_lengths(self, seg_len, stream=None):
        """New segment lengths (host int32 [num_segments]); schedule again before the next run."""
        import numpy as np
        a = np.ascontiguousarray(np.asarray(seg_len, dtype=np.int32))
        _check(self.lib.graphattn_plan_set_lengths(
            self.handle, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
            _stream_handle(stream)))

    def schedule(self, stream=None):
        """Run the GPU segment scheduler (run() also schedules a plan that has no schedule)."""
        _check(self.lib.graphattn_schedule(self.handle, _stream_handle(stream)))

    def run(self, q, pool, out, lse, stream=None):
        _check(self.lib.graphattn_run(self.handle, _dev_ptr(q), _dev_ptr(pool), _dev_ptr(out),
                                      _dev_ptr(lse), _stream_handle(stream)))

    def info(self) -> PlanInfo:
        inf = PlanInfo()
        _check(self.lib.graphattn_plan_info(self.handle, ctypes.byref(inf)))
        return inf

    def debug_dump(self, stream=None):
        """Device schedule as numpy arrays: group offsets/branches, entry ranks, items, chunks
        and each branch's partial-row list (CSR)."""
        inf = self.info()
        S, E, R = inf.num_segments, inf.num_entries, inf.num_query_rows
        goff = np.zeros(S + 1, dtype=np.int64)
        gbr = np.zeros(max(E, 1), dtype=np.int32)
        rk = np.zeros(max(E, 1), dtype=np.int32)
        nit = max(int(inf.num_items), 0)
        items = np.zeros(max(3 * nit, 3), dtype=np.int32)
        nch = np.zeros(max(S, 1), dtype=np.int32)
        boff = np.zeros(R + 1, dtype=np.int64)
        bpart = np.zeros(max(int(inf.num_partial_rows), 1), dtype=np.int32)
        _check(self.lib.graphattn_plan_debug_dump(
            self.handle, _stream_handle(stream), _ptr(goff, ctypes.c_int64),
            _ptr(gbr, ctypes.c_int32), _ptr(rk, ctypes.c_int32), _ptr(items, ctypes.c_int32),
            _ptr(nch, ctypes.c_int32), _ptr(boff, ctypes.c_int64), _ptr(bpart, ctypes.c_int32)))
        return {"group_offsets": goff, "group_branches": gbr[:E], "entry_ranks": rk[:E],
                "items": items[:3 * nit].reshape(nit, 3), "segment_chunks": nch[:S],
                "branch_part_offsets": boff, "branch_parts": bpart[:int(boff[-1])]}

    def profile(self, max_calls: int):
        """Record HIP-event kernel times for the next ``max_calls`` schedule/run calls."""
        _check(self.lib.graphattn_plan_profile(self.handle, int(max_calls)))

    def profile_read(self) -> Profile:
        pr = Profile()
        _check(self.lib.graphattn_plan_profile_read(self.handle, ctypes.byref(pr)))
        return pr

    def close(self):
        if self.handle:
            self.lib.graphattn_plan_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def validate_only(graph: HostGraph, params: Params, query_counts=None) -> int:
    """Run the library's host-side validation through graphattn_decode (graphattn_extend with
    query_counts) with NULL device buffers; used by CPU tests of the error paths.  Returns the
    status (only meaningful for invalid inputs, which are rejected before any HIP call)."""
    lib = load_library()
    if query_counts is None:
        return lib.graphattn_decode(None, None, ctypes.byref(graph.st), ctypes.byref(graph.bp),
                                    None, None, ctypes.byref(params), None)
    cnt = _counts(query_counts)
    return lib.graphattn_extend(None, None, ctypes.byref(graph.st), ctypes.byref(graph.bp),
                                _ptr(cnt, ctypes.c_int32) if len(cnt) else None, None, None,
                                ctypes.byref(params), None)


def last_error() -> str:
    return load_library().graphattn_last_error().decode(errors="replace")


def header_symbols() -> list:
    """Function names declared in include/graphattn.h."""
    import re
    hdr = os.path.join(os.path.dirname(_PKG), "include", "graphattn.h")
    text = open(hdr).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(graphattn_\w+)\s*\(", text)))
