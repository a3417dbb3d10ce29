"""CPU oracle for EMO's batched what-if policy evaluation -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this package.
The library under ``paper_2607_12324_amd`` never does: it shares no code with the oracle.

The arithmetic lives in ``emo_oracle.c`` (plain C, double precision), whose header lists the
paper passages each function follows.  This module compiles it with gcc and wraps it with
ctypes over numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "emo_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

OK, BAD_ARGUMENT, CYCLE, NO_MEMORY = 0, 1, 2, 3


class OracleError(RuntimeError):
    pass


def build(force: bool = False) -> str:
    """Compile the oracle shared library with gcc (OpenMP over independent candidates)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _bind(path):
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
    lib.oracle_topo_order.argtypes = [i32, i32, P, P, P, P]
    lib.oracle_topo_order.restype = i32
    lib.oracle_eval_batch.argtypes = [i32, i32, P, P, P, P, i32, i32, P, P, f64, P, i64, P, P, i32]
    lib.oracle_eval_batch.restype = i32
    lib.oracle_slack.argtypes = [i32, i32, P, P, P, P, i32, i32, P, P, f64, P, P, P, P, P, P, P]
    lib.oracle_slack.restype = i32
    lib.oracle_slack_batch.argtypes = [i32, i32, P, P, P, P, i32, i32, P, P, f64, P, i64, i32,
                                       P, P, P, i32]
    lib.oracle_slack_batch.restype = i32
    lib.oracle_select.argtypes = [P, P, i64, f64, P, P]
    lib.oracle_select.restype = i64
    return lib


def _load():
    global _lib
    if _lib is None:
        build()
        _lib = _bind(_LIB)
    return _lib


def use_library(path):
    """Point the wrappers at another build of the oracle source (used by the tests that plant
    mistakes in a copy of the oracle to show the pins catch them). Returns the previous one."""
    global _lib
    prev = _lib
    _lib = _bind(path) if isinstance(path, str) else path
    return prev


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc):
    if rc == CYCLE:
        raise OracleError("graph has a cycle")
    if rc != OK:
        raise OracleError(f"oracle error {rc}")


class _G:
    """Contiguous copies of a graph's arrays, kept alive for the C calls."""

    def __init__(self, g):
        self.V = int(g.num_nodes)
        self.src = _c(g.edge_src, np.int32)
        self.dst = _c(g.edge_dst, np.int32)
        self.E = int(self.src.shape[0])
        self.pack = _c(g.node_pack, np.int32)
        self.dur = _c(g.node_duration, np.float32)
        self.P = int(g.num_packs)
        self.F = int(g.num_levels)
        self.tt = _c(g.pack_time, np.float32).reshape(-1)
        self.te = _c(g.pack_energy, np.float32).reshape(-1)
        self.sp = float(np.float32(g.static_power))

    def args(self):
        return (self.V, self.E, _ptr(self.src), _ptr(self.dst), _ptr(self.pack), _ptr(self.dur),
                self.P, self.F, _ptr(self.tt), _ptr(self.te), self.sp)


def topo_order(num_nodes, edge_src, edge_dst):
    """Canonical topological order (sorted by depth, then id) and depths."""
    lib = _load()
    src = _c(edge_src, np.int32)
    dst = _c(edge_dst, np.int32)
    order = np.empty(num_nodes, dtype=np.int32)
    depth = np.empty(num_nodes, dtype=np.int32)
    _check(lib.oracle_topo_order(int(num_nodes), int(src.shape[0]), _ptr(src), _ptr(dst),
                                 _ptr(order), _ptr(depth)))
    return order, depth


def eval_batch(g, levels, nthreads: int = 1):
    """Makespan and energy (float64) of every row of `levels` ([B, P] uint8)."""
    lib = _load()
    G = _G(g)
    lv = _c(levels, np.uint8).reshape(-1, G.P) if G.P > 0 else np.zeros((len(levels), 0), np.uint8)
    B = int(lv.shape[0])
    T = np.empty(B, dtype=np.float64)
    E = np.empty(B, dtype=np.float64)
    _check(lib.oracle_eval_batch(*G.args(), _ptr(lv), B, _ptr(T), _ptr(E), int(nthreads)))
    return T, E


@dataclass
class SlackResult:
    makespan: float
    energy: float
    eft: np.ndarray          # [V] completion (earliest finish) times
    lft: np.ndarray          # [V] latest finish times
    slack: np.ndarray        # [V] total float
    critical_pred: np.ndarray  # [V] critical predecessor (Eq. 5), -1 for none


def slack(g, level_row) -> SlackResult:
    """Per-node forward/backward times and slack of one candidate."""
    lib = _load()
    G = _G(g)
    lv = _c(level_row, np.uint8).reshape(-1)
    if lv.shape[0] != G.P:
        raise OracleError("level row has the wrong length")
    V = G.V
    eft = np.empty(V); lft = np.empty(V); sl = np.empty(V)
    cp = np.empty(V, dtype=np.int32)
    T = ctypes.c_double(); E = ctypes.c_double()
    _check(lib.oracle_slack(*G.args(), _ptr(lv), _ptr(eft), _ptr(lft), _ptr(sl), _ptr(cp),
                            ctypes.byref(T), ctypes.byref(E)))
    return SlackResult(T.value, E.value, eft, lft, sl, cp)


def pack_slack(g, level_row) -> np.ndarray:
    """Slack of each pack, indexed by pack id ([P], float64)."""
    r = slack(g, level_row)
    out = np.full(int(g.num_packs), np.nan)
    pk = np.asarray(g.node_pack)
    m = pk >= 0
    out[pk[m]] = r.slack[m]
    return out


def slack_batch(g, levels, per_node: bool = False, nthreads: int = 1):
    """Makespan, energy ([B] float64) and slack of every row of `levels` ([B, P] uint8): [B, P]
    by pack id, or [B, V] by node id with per_node.  Rows with a level >= F are NaN."""
    lib = _load()
    G = _G(g)
    lv = _c(levels, np.uint8).reshape(-1, G.P) if G.P > 0 else np.zeros((len(levels), 0), np.uint8)
    B = int(lv.shape[0])
    T = np.empty(B, dtype=np.float64)
    E = np.empty(B, dtype=np.float64)
    S = np.empty((B, G.V if per_node else G.P), dtype=np.float64)
    _check(lib.oracle_slack_batch(*G.args(), _ptr(lv), B, int(bool(per_node)), _ptr(T), _ptr(E),
                                  _ptr(S), int(nthreads)))
    return T, E, S


def select(T, E, target):
    """(index or -1, feasible mask as bool [B], number feasible)."""
    lib = _load()
    T = _c(T, np.float64); E = _c(E, np.float64)
    B = int(T.shape[0])
    feas = np.empty(B, dtype=np.uint8)
    n = ctypes.c_int64()
    idx = lib.oracle_select(_ptr(T), _ptr(E), B, float(target), _ptr(feas), ctypes.byref(n))
    return int(idx), feas.astype(bool), int(n.value)
