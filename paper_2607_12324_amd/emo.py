"""Thin Python binding of the C ABI in include/emo.h (argument marshalling only).

Every computation runs in libemo.so (HIP kernels for gfx950).  PyTorch supplies device memory
and the stream: tensors are passed by data_ptr() and calls are enqueued on
torch.cuda.current_stream() unless a stream is given.  If the library is missing this module
raises at import time; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libemo.so")

OK = 0
STATUS_NAMES = {0: "EMO_OK", 1: "EMO_ERR_INVALID_ARGUMENT", 2: "EMO_ERR_CYCLE",
                3: "EMO_ERR_OUT_OF_MEMORY", 4: "EMO_ERR_DEVICE", 5: "EMO_ERR_UNSUPPORTED"}

ENTRY_POINTS = ("emo_load_graph", "emo_free_graph", "emo_graph_get_info",
                "emo_graph_set_kernel_mode", "emo_graph_topo_order",
                "emo_eval_policies", "emo_slack", "emo_select_policy", "emo_evaluate", "emo_evaluate_targets",
                "emo_select_from_results", "emo_select_from_results_noalloc", "emo_dp_search", "emo_eval_intervals",
                "emo_graph_set_timing_events", "emo_pack_kernels", "emo_contract_packs",
                "emo_pack_model",
                "emo_graph_specialized_source",
                "emo_graph_segmented_source", "emo_graph_cut_source", "emo_graph_interval_source",
                "emo_status_string",
                "emo_last_error")


class EmoError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class GraphInfo(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int32), ("num_edges", ctypes.c_int32),
                ("num_packs", ctypes.c_int32), ("num_levels", ctypes.c_int32),
                ("num_dynamic_nodes", ctypes.c_int32), ("num_dynamic_edges", ctypes.c_int32),
                ("eval_slots", ctypes.c_int32), ("max_depth", ctypes.c_int32),
                ("const_makespan", ctypes.c_float), ("device", ctypes.c_int32),
                ("pack_order_monotone", ctypes.c_int32), ("kernel_mode", ctypes.c_int32),
                ("specialized", ctypes.c_int32), ("compile_seconds", ctypes.c_float),
                ("last_kernels", ctypes.c_int32), ("chain_lanes", ctypes.c_int32),
                ("num_implied_edges", ctypes.c_int32), ("chain_window", ctypes.c_int32),
                ("cut_segments", ctypes.c_int32), ("chain_scan_window", ctypes.c_int32),
                ("chain_scan_full", ctypes.c_int32), ("hip_runtime_version", ctypes.c_int32),
                ("exact_time_sums", ctypes.c_int32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


KERNELS_AUTO, KERNELS_INTERPRETED, KERNELS_SPECIALIZED = 0, 1, 2


def _load_library():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                          "python -m paper_2607_12324_amd.build")
    # torch first: it carries its own HIP runtime, and libemo must bind to that same runtime
    # (loaded first, libemo would map the system's as a second runtime, which sees no device)
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    sig = {
        "emo_load_graph": [i32, i32, P, P, P, P, i32, i32, P, P, f32, i32, P],
        "emo_free_graph": [P],
        "emo_graph_get_info": [P, P],
        "emo_graph_set_kernel_mode": [P, i32],
        "emo_graph_topo_order": [P, P, P],
        "emo_eval_policies": [P, P, i64, P, P, P],
        "emo_slack": [P, P, i64, P, i32, P, P, P],
        "emo_select_policy": [P, P, i64, f32, P, P, P],
        "emo_evaluate": [P, P, i64, P, P, P, i32, f32, P, P, P],
        "emo_evaluate_targets": [P, P, i64, P, P, P, i32, i32, P, P, P, P],
        "emo_select_from_results": [P, P, i64, f32, P, P, P],
        "emo_select_from_results_noalloc": [P, P, i64, f32, P, P, P],
        "emo_dp_search": [P, f32, f32, P, i32, P, P, P],
        "emo_eval_intervals": [P, P, i64, i32, P, P, P, P, f32, P, P, P],
        "emo_graph_specialized_source": [P, P, P],
        "emo_graph_segmented_source": [P, P, P],
        "emo_graph_cut_source": [P, P, P],
        "emo_graph_interval_source": [P, P, P],
        "emo_graph_set_timing_events": [P, P, P],
        "emo_pack_kernels": [i32, i32, P, P, P, P, P, i32, i32, P, f32, P, P],
        "emo_pack_model": [i32, i32, P, i32, P, P, i32, P, P, P, P, i32],
        "emo_contract_packs": [i32, i32, P, P, P, P, i32, i32, P, P, P, i32, P, P, P, P, P, P,
                               P, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.emo_status_string.argtypes = [ctypes.c_int]
    lib.emo_status_string.restype = ctypes.c_char_p
    lib.emo_last_error.argtypes = []
    lib.emo_last_error.restype = ctypes.c_char_p
    return lib


lib = _load_library()


def _check(status: int):
    if status != OK:
        raise EmoError(status, lib.emo_last_error().decode())


def _np(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _nptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None and a.size else None


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dptr(t, dtype=None, numel=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


@dataclass
class Selection:
    index: int
    energy: float
    makespan: float
    num_feasible: int


def parse_selection(res) -> Selection:
    """Decode a 24-byte emo_selection held in a device int64 tensor of 3 elements."""
    raw = res.detach().cpu().numpy().view(np.uint8)
    idx = int(raw[0:8].view(np.int64)[0])
    e, t = raw[8:16].view(np.float32).tolist()
    n = int(raw[16:24].view(np.int64)[0])
    return Selection(idx, float(e), float(t), n)


class EmoGraph:
    """A graph loaded into libemo (emo_load_graph).  `device=-1` loads host-only."""

    def __init__(self, graph, device: int = 0, kernel_mode: int | None = None):
        self._h = ctypes.c_void_p()
        src = _np(graph.edge_src, np.int32)
        dst = _np(graph.edge_dst, np.int32)
        pack = _np(graph.node_pack, np.int32)
        dur = _np(graph.node_duration, np.float32)
        tt = _np(graph.pack_time, np.float32).reshape(-1)
        te = _np(graph.pack_energy, np.float32).reshape(-1)
        _check(lib.emo_load_graph(int(graph.num_nodes), int(src.size), _nptr(src), _nptr(dst),
                                  _nptr(pack), _nptr(dur), int(graph.num_packs),
                                  int(graph.num_levels), _nptr(tt), _nptr(te),
                                  float(graph.static_power), int(device), ctypes.byref(self._h)))
        self.num_nodes = int(graph.num_nodes)
        self.num_packs = int(graph.num_packs)
        self.num_levels = int(graph.num_levels)
        self.device = int(device)
        if kernel_mode is not None:
            self.set_kernel_mode(kernel_mode)

    def set_kernel_mode(self, mode: int):
        _check(lib.emo_graph_set_kernel_mode(self._h, int(mode)))

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib.emo_free_graph(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def info(self) -> dict:
        inf = GraphInfo()
        _check(lib.emo_graph_get_info(self._h, ctypes.byref(inf)))
        return inf.as_dict()

    def set_timing_events(self, begin=None, end=None):
        """Record torch.cuda.Event `begin`/`end` around the evaluating kernel of later calls
        (events that have been recorded once, so that they exist); None disables."""
        hb = ctypes.c_void_p(begin.cuda_event) if begin is not None else None
        he = ctypes.c_void_p(end.cuda_event) if end is not None else None
        _check(lib.emo_graph_set_timing_events(self._h, hb, he))

    def specialized_source(self) -> str:
        return self._source(lib.emo_graph_specialized_source)

    def segmented_source(self) -> str:
        return self._source(lib.emo_graph_segmented_source)

    def cut_source(self) -> str:
        return self._source(lib.emo_graph_cut_source)

    def interval_source(self) -> str:
        return self._source(lib.emo_graph_interval_source)

    def _source(self, fn) -> str:
        n = ctypes.c_int64(0)
        _check(fn(self._h, None, ctypes.byref(n)))
        buf = ctypes.create_string_buffer(n.value)
        _check(fn(self._h, buf, ctypes.byref(n)))
        return buf.value.decode()

    def topo_order(self):
        order = np.empty(self.num_nodes, dtype=np.int32)
        depth = np.empty(self.num_nodes, dtype=np.int32)
        _check(lib.emo_graph_topo_order(self._h, _nptr(order), _nptr(depth)))
        return order, depth

    def _levels(self, levels):
        import torch
        if levels.dim() != 2 or levels.shape[1] != self.num_packs:
            raise ValueError(f"levels must be [B, {self.num_packs}]")
        return _dptr(levels, torch.uint8, name="levels"), int(levels.shape[0])

    def eval_policies(self, levels, makespan=None, energy=None, stream=None):
        import torch
        lv, B = self._levels(levels)
        if makespan is None:
            makespan = torch.empty(B, dtype=torch.float32, device=levels.device)
        if energy is None:
            energy = torch.empty(B, dtype=torch.float32, device=levels.device)
        _check(lib.emo_eval_policies(self._h, lv, B, _dptr(makespan, torch.float32, B, "makespan"),
                                     _dptr(energy, torch.float32, B, "energy"), _stream(stream)))
        return makespan, energy

    def slack(self, levels, per_node: bool = False, out=None, makespan=None, energy=None,
              stream=None):
        import torch
        lv, B = self._levels(levels)
        cols = self.num_nodes if per_node else self.num_packs
        if out is None:
            out = torch.empty((B, cols), dtype=torch.float32, device=levels.device)
        _check(lib.emo_slack(self._h, lv, B, _dptr(out, torch.float32, B * cols, "slack"),
                             int(bool(per_node)), _dptr(makespan, torch.float32, B, "makespan"),
                             _dptr(energy, torch.float32, B, "energy"), _stream(stream)))
        return out

    def evaluate(self, levels, makespan=None, energy=None, slack=None, per_node: bool = False,
                 latency_target: float = 0.0, mask=None, result=None, stream=None):
        """One pass of the whole hot path (emo_evaluate); every output is optional."""
        import torch
        lv, B = self._levels(levels)
        cols = self.num_nodes if per_node else self.num_packs
        _check(lib.emo_evaluate(self._h, lv, B, _dptr(makespan, torch.float32, B, "makespan"),
                                _dptr(energy, torch.float32, B, "energy"),
                                _dptr(slack, torch.float32, B * cols, "slack"), int(bool(per_node)),
                                float(latency_target), _dptr(mask, torch.int32, (B + 31) // 32, "mask"),
                                _dptr(result, torch.int64, 3, "result"), _stream(stream)))
        return makespan, energy, slack, mask, result

    def evaluate_targets(self, levels, latency_targets, makespan=None, energy=None, slack=None,
                         per_node: bool = False, masks=None, results=None, stream=None):
        """emo_evaluate with several latency targets in one pass (emo_evaluate_targets).
        masks: None or a list of one int32 tensor (or None) per target; results: None or an
        int64 [n, 3] tensor (one emo_selection per target)."""
        import torch
        lv, B = self._levels(levels)
        cols = self.num_nodes if per_node else self.num_packs
        tg = np.ascontiguousarray(np.asarray(latency_targets, dtype=np.float32).reshape(-1))
        n = int(tg.size)
        mk = None
        if masks is not None:
            if len(masks) != n:
                raise ValueError(f"masks must hold {n} entries")
            mk = (ctypes.c_void_p * n)(*[_dptr(m, torch.int32, (B + 31) // 32, "mask") for m in masks])
        _check(lib.emo_evaluate_targets(self._h, lv, B, _dptr(makespan, torch.float32, B, "makespan"),
                                        _dptr(energy, torch.float32, B, "energy"),
                                        _dptr(slack, torch.float32, B * cols, "slack"),
                                        int(bool(per_node)), n, _nptr(tg) if n else None,
                                        ctypes.cast(mk, ctypes.c_void_p) if mk is not None else None,
                                        _dptr(results, torch.int64, 3 * n, "results"), _stream(stream)))
        return makespan, energy, slack, masks, results

    def select_policy(self, levels, latency_target: float, mask=None, result=None, stream=None,
                      want_mask: bool = True):
        import torch
        lv, B = self._levels(levels)
        if mask is None and want_mask:
            mask = torch.empty(max(1, (B + 31) // 32), dtype=torch.int32, device=levels.device)
        if result is None:
            result = torch.empty(3, dtype=torch.int64, device=levels.device)
        _check(lib.emo_select_policy(self._h, lv, B, float(latency_target),
                                     _dptr(mask, torch.int32, (B + 31) // 32, "mask"),
                                     _dptr(result, torch.int64, 3, "result"), _stream(stream)))
        return result, mask


    def eval_intervals(self, levels, change_points, idle_power, makespan=None, energy=None,
                       latency_target: float = 0.0, mask=None, result=None, stream=None):
        """Time-interval policies (emo_eval_intervals): levels [B, K] uint8 with K =
        len(change_points) + 1; idle_power has one value per level.  Returns (makespan, energy,
        mask, result); makespan and energy are allocated when not given."""
        import torch
        pts = _np(change_points, np.float32).reshape(-1)
        idle = _np(idle_power, np.float32).reshape(-1)
        K = int(pts.size) + 1
        if levels.dim() != 2 or levels.shape[1] != K:
            raise ValueError(f"levels must be [B, {K}] for {K - 1} change points")
        if idle.size != self.num_levels:
            raise ValueError(f"idle_power must hold {self.num_levels} values")
        B = int(levels.shape[0])
        if makespan is None:
            makespan = torch.empty(B, dtype=torch.float32, device=levels.device)
        if energy is None:
            energy = torch.empty(B, dtype=torch.float32, device=levels.device)
        _check(lib.emo_eval_intervals(self._h, _dptr(levels, torch.uint8, name="levels"), B, K,
                                      _nptr(pts) if pts.size else None, _nptr(idle),
                                      _dptr(makespan, torch.float32, B, "makespan"),
                                      _dptr(energy, torch.float32, B, "energy"), float(latency_target),
                                      _dptr(mask, torch.int32, (B + 31) // 32, "mask"),
                                      _dptr(result, torch.int64, 3, "result"), _stream(stream)))
        return makespan, energy, mask, result

    def dp_search(self, latency_target: float, quantum: float, pack_order=None,
                  max_states: int = 4096, best_levels=None, result=None, stream=None):
        """Policy search of Alg. 2 with one frequency interval per pack (emo_dp_search): returns
        the device tensors (levels [P] uint8, result [3] int64 as an emo_selection)."""
        import torch
        dev = f"cuda:{self.device}"
        if best_levels is None:
            best_levels = torch.empty(max(self.num_packs, 1), dtype=torch.uint8, device=dev)
        if result is None:
            result = torch.empty(3, dtype=torch.int64, device=dev)
        order = None if pack_order is None else _np(pack_order, np.int32)
        if order is not None and order.size != self.num_packs:
            raise ValueError(f"pack_order must hold {self.num_packs} pack ids")
        _check(lib.emo_dp_search(self._h, float(latency_target), float(quantum),
                                 None if order is None else _nptr(order), int(max_states),
                                 _dptr(best_levels, torch.uint8, self.num_packs, "best_levels"),
                                 _dptr(result, torch.int64, 3, "result"), _stream(stream)))
        return best_levels[: self.num_packs], result


def select_from_results(makespan, energy, latency_target: float, mask=None, result=None,
                        stream=None, want_mask: bool = True):
    import torch
    B = int(makespan.numel())
    if mask is None and want_mask:
        mask = torch.empty(max(1, (B + 31) // 32), dtype=torch.int32, device=makespan.device)
    if result is None:
        result = torch.empty(3, dtype=torch.int64, device=makespan.device)
    _check(lib.emo_select_from_results(_dptr(makespan, torch.float32, B, "makespan"),
                                       _dptr(energy, torch.float32, B, "energy"), B,
                                       float(latency_target),
                                       _dptr(mask, torch.int32, (B + 31) // 32, "mask"),
                                       _dptr(result, torch.int64, 3, "result"), _stream(stream)))
    return result, mask


def select_from_results_noalloc(makespan, energy, latency_target: float, mask, result,
                                stream=None):
    """emo_select_from_results_noalloc: the same selection with the library's static scratch;
    the caller passes every output (nothing is allocated here or in the library)."""
    import torch
    B = int(makespan.numel())
    _check(lib.emo_select_from_results_noalloc(
        _dptr(makespan, torch.float32, B, "makespan"), _dptr(energy, torch.float32, B, "energy"), B,
        float(latency_target), _dptr(mask, torch.int32, (B + 31) // 32, "mask"),
        _dptr(result, torch.int64, 3, "result"), _stream(stream)))
    return result, mask


def unpack_mask(mask, B: int) -> np.ndarray:
    """Feasibility bits (bit c % 32 of word c // 32) as a bool array of length B."""
    words = mask.detach().cpu().numpy().view(np.uint32)[: (B + 31) // 32]
    bits = np.unpackbits(words.view(np.uint8), bitorder="little")
    return bits[:B].astype(bool)


@dataclass
class PackedGraph:
    """A packed execution graph in the field layout of ``Graph`` (the loader's form)."""
    name: str
    num_nodes: int
    edge_src: np.ndarray
    edge_dst: np.ndarray
    node_pack: np.ndarray
    node_duration: np.ndarray
    num_packs: int
    num_levels: int
    pack_time: np.ndarray
    pack_energy: np.ndarray
    static_power: float
    packed_node: np.ndarray     # [V of the input] packed node standing for each input node

    @property
    def num_edges(self) -> int:
        return int(self.edge_src.shape[0])


def _graph_arrays(graph):
    return (_np(graph.edge_src, np.int32), _np(graph.edge_dst, np.int32),
            _np(graph.node_pack, np.int32), _np(graph.node_duration, np.float32),
            _np(graph.pack_time, np.float32).reshape(-1),
            _np(graph.pack_energy, np.float32).reshape(-1))


def pack_kernels(graph, node_stream, max_pack_duration: float):
    """Greedy dependency-aware packing (host pass): (group of each input pack, group count)."""
    src, dst, pk, dur, pt, _ = _graph_arrays(graph)
    stream = _np(node_stream, np.int32)
    if stream.shape[0] != int(graph.num_nodes):
        raise ValueError("node_stream needs one entry per node")
    group = np.empty(int(graph.num_packs), dtype=np.int32)
    n = ctypes.c_int32(0)
    _check(lib.emo_pack_kernels(int(graph.num_nodes), int(src.shape[0]), _nptr(src), _nptr(dst),
                                _nptr(pk), _nptr(dur), _nptr(stream), int(graph.num_packs),
                                int(graph.num_levels), _nptr(pt), float(max_pack_duration),
                                _nptr(group), ctypes.byref(n)))
    return group, int(n.value)


def contract_packs(graph, group, num_groups: int) -> PackedGraph:
    """The packed graph of a grouping of the input packs (host pass)."""
    src, dst, pk, dur, pt, pe = _graph_arrays(graph)
    V, E, F = int(graph.num_nodes), int(src.shape[0]), int(graph.num_levels)
    group = _np(group, np.int32)
    if group.shape[0] != int(graph.num_packs):
        raise ValueError("group needs one entry per pack")
    packed_node = np.empty(V, dtype=np.int32)
    node_pack = np.empty(V, dtype=np.int32)
    node_dur = np.empty(V, dtype=np.float32)
    psrc = np.empty(E, dtype=np.int32)
    pdst = np.empty(E, dtype=np.int32)
    gt = np.empty((int(num_groups), F), dtype=np.float32)
    ge = np.empty((int(num_groups), F), dtype=np.float32)
    counts = np.zeros(2, dtype=np.int32)
    _check(lib.emo_contract_packs(V, E, _nptr(src), _nptr(dst), _nptr(pk), _nptr(dur),
                                  int(graph.num_packs), F, _nptr(pt), _nptr(pe), _nptr(group),
                                  int(num_groups), _nptr(packed_node), _nptr(node_pack),
                                  _nptr(node_dur), _nptr(psrc), _nptr(pdst), _nptr(gt), _nptr(ge),
                                  _nptr(counts)))
    n, m = int(counts[0]), int(counts[1])
    return PackedGraph(name=f"{getattr(graph, 'name', 'graph')}-packed", num_nodes=n,
                       edge_src=psrc[:m].copy(), edge_dst=pdst[:m].copy(),
                       node_pack=node_pack[:n].copy(), node_duration=node_dur[:n].copy(),
                       num_packs=int(num_groups), num_levels=F, pack_time=gt, pack_energy=ge,
                       static_power=float(graph.static_power), packed_node=packed_node)


def pack_model(metric_matrix, bench_time, bench_energy, pack_metrics, num_threads: int = 0):
    """Microbenchmark pack model (host pass): weights [P, m] and tables [P, F] (Eq. 6-7)."""
    B = _np(metric_matrix, np.float32)
    bt = _np(bench_time, np.float32)
    be = _np(bench_energy, np.float32)
    b = _np(pack_metrics, np.float32)
    n, m = B.shape
    F = bt.shape[1]
    if bt.shape != (m, F) or be.shape != (m, F) or b.ndim != 2 or b.shape[1] != n:
        raise ValueError("pack_model: inconsistent shapes")
    P = b.shape[0]
    W = np.empty((P, m), dtype=np.float32)
    T = np.empty((P, F), dtype=np.float32)
    E = np.empty((P, F), dtype=np.float32)
    _check(lib.emo_pack_model(n, m, _nptr(B), F, _nptr(bt), _nptr(be), P, _nptr(b), _nptr(W),
                              _nptr(T), _nptr(E), int(num_threads)))
    return W, T, E
