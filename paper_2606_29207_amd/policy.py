"""ctypes binding of the scaling-policy entry points (include/kf_policy.h).

Argument marshalling only, over numpy host arrays: the policy itself
(Section 4.2, Algorithm 1, Eqs. (1) and (2)) runs in libkf.so.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np

from . import kf

SPAWN = 1
PUBLISH = 2

EXPORTS = ("kf_policy_token_bytes", "kf_policy_threshold", "kf_policy_layer_budget",
           "kf_policy_pipeline", "kf_policy_init", "kf_policy_monitor", "kf_policy_simulate",
           "kf_policy_build_routes")


class Params(ctypes.Structure):
    _fields_ = [("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("num_layers", ctypes.c_int32), ("elem_bytes", ctypes.c_int32),
                ("beta_mem", ctypes.c_double), ("beta_slo", ctypes.c_double),
                ("gamma", ctypes.c_double), ("t_a_max", ctypes.c_double),
                ("bw_hbm", ctypes.c_double), ("c_kv_cap", ctypes.c_double),
                ("t_step", ctypes.c_double), ("t_prewarm", ctypes.c_double)]


RANGE_DT = np.dtype([("seq", np.int32), ("node", np.int32), ("tok_begin", np.int64),
                     ("tok_end", np.int64)])
NODE_DT = np.dtype([("bytes", np.int64), ("live", np.int32), ("prewarm", np.int32),
                    ("prewarm_ready", np.int32), ("reserved", np.int32), ("tau_fill", np.float64)])
EVENT_DT = np.dtype([("step", np.int64), ("kind", np.int32), ("node", np.int32),
                     ("new_node", np.int32), ("count", np.int32)])
ROUTE_DT = np.dtype([(n, np.int32) for n in
                     ("seq", "part", "tok_begin", "tok_end", "page_base", "page_cap")])

_ready = False


def _lib():
    global _ready
    lib = kf.load()
    if not _ready:
        vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        pp = ctypes.POINTER(Params)
        sig = {
            "kf_policy_token_bytes": ([pp], i64),
            "kf_policy_threshold": ([pp, vp, vp, vp], ctypes.c_int),
            "kf_policy_layer_budget": ([dbl, dbl, i32, dbl, vp], ctypes.c_int),
            "kf_policy_pipeline": ([dbl, dbl, dbl, vp, vp], ctypes.c_int),
            "kf_policy_init": ([pp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp], ctypes.c_int),
            "kf_policy_monitor": ([pp, i64, i32, vp, vp, vp, vp, vp, i32, vp, vp, i32, vp, vp, i32],
                                  ctypes.c_int),
            "kf_policy_simulate": ([pp, vp, vp, i32, i64, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                    vp, vp, vp], ctypes.c_int),
            "kf_policy_build_routes": ([vp, i32, i32, vp, i32, vp, i32, vp, vp, vp, vp, i32, vp],
                                       ctypes.c_int),
        }
        for name, (args, res) in sig.items():
            f = getattr(lib, name)
            f.argtypes, f.restype = args, res
        _ready = True
    return lib


def _check(st: int, what: str):
    if st != 0:
        raise kf.KFError(f"{what}: {kf.status_str(st)} ({st})")


def _ptr(a: np.ndarray | None):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def params(**kw) -> Params:
    """Params from keyword arguments named as in kf_policy_params."""
    return Params(**kw)


def token_bytes(p: Params) -> int:
    v = _lib().kf_policy_token_bytes(ctypes.byref(p))
    if v < 0:
        raise kf.KFError("kf_policy_token_bytes: invalid parameters")
    return int(v)


def threshold(p: Params) -> tuple[float, float, float]:
    out = np.zeros(3, np.float64)
    _check(_lib().kf_policy_threshold(ctypes.byref(p), _ptr(out[0:]), _ptr(out[1:]), _ptr(out[2:])),
           "kf_policy_threshold")
    return float(out[0]), float(out[1]), float(out[2])


def layer_budget(t_slo, t_overhead, num_layers, t_w_stage) -> float | None:
    out = np.zeros(1, np.float64)
    st = _lib().kf_policy_layer_budget(t_slo, t_overhead, num_layers, t_w_stage, _ptr(out))
    if st == kf.ERR_INFEASIBLE:
        return None
    _check(st, "kf_policy_layer_budget")
    return float(out[0])


def pipeline(t_p, t_f, t_a) -> tuple[float, float]:
    out = np.zeros(2, np.float64)
    _check(_lib().kf_policy_pipeline(t_p, t_f, t_a, _ptr(out[0:]), _ptr(out[1:])),
           "kf_policy_pipeline")
    return float(out[0]), float(out[1])


@dataclass
class State:
    """Policy state in host arrays: nodes, ranges, tail (index into ranges per
    request), events; counts are the leading rows in use."""
    nodes: np.ndarray
    ranges: np.ndarray
    tail: np.ndarray
    events: np.ndarray
    num_nodes: int
    num_ranges: int
    num_events: int
    c_total: int = 0

    def live_ranges(self):
        return self.ranges[:self.num_ranges]


def init(p: Params, seq_lens, max_nodes=None, max_ranges=None, max_events=64) -> State:
    lens = np.ascontiguousarray(seq_lens, np.int64)
    B = len(lens)
    lib = _lib()
    c_total = np.zeros(1, np.int64)
    nn = np.zeros(1, np.int32)
    nr = np.zeros(1, np.int32)
    tail = np.zeros(max(B, 1), np.int32)
    if max_nodes is None or max_ranges is None:       # size query
        st = lib.kf_policy_init(ctypes.byref(p), _ptr(lens), B, 0, 0, _ptr(c_total), _ptr(nn),
                                None, None, _ptr(nr), _ptr(tail))
        if st not in (0, kf.ERR_CAPACITY):
            _check(st, "kf_policy_init")
        max_nodes = int(nn[0]) if max_nodes is None else max_nodes
        max_ranges = int(nr[0]) if max_ranges is None else max_ranges
    nodes = np.zeros(max(max_nodes, 1), NODE_DT)
    ranges = np.zeros(max(max_ranges, 1), RANGE_DT)
    _check(lib.kf_policy_init(ctypes.byref(p), _ptr(lens), B, max_nodes, max_ranges, _ptr(c_total),
                              _ptr(nn), _ptr(nodes), _ptr(ranges), _ptr(nr), _ptr(tail)),
           "kf_policy_init")
    return State(nodes, ranges, tail[:B], np.zeros(max(max_events, 1), EVENT_DT), int(nn[0]),
                 int(nr[0]), 0, int(c_total[0]))


def monitor(p: Params, step: int, state: State, active, seq_len) -> State:
    """One monitor pass; grows state's arrays in place (they must have room)."""
    act = np.ascontiguousarray(active, np.uint8)
    lens = np.ascontiguousarray(seq_len, np.int64)
    nn = np.array([state.num_nodes], np.int32)
    nr = np.array([state.num_ranges], np.int32)
    ne = np.array([state.num_events], np.int32)
    _check(_lib().kf_policy_monitor(ctypes.byref(p), step, len(act), _ptr(act), _ptr(lens),
                                    _ptr(state.tail), _ptr(state.nodes), _ptr(nn),
                                    len(state.nodes), _ptr(state.ranges), _ptr(nr),
                                    len(state.ranges), _ptr(state.events), _ptr(ne),
                                    len(state.events)), "kf_policy_monitor")
    state.num_nodes, state.num_ranges, state.num_events = int(nn[0]), int(nr[0]), int(ne[0])
    return state


def time_monitor(p: Params, state: State, active, seq_len, reps: int = 10000) -> float:
    """Seconds per kf_policy_monitor call on ``state`` (ctypes arguments built
    once; the state must already be in steady state: no node left to spawn
    or publish, so repeated passes only refresh the fill horizons)."""
    import time
    act = np.ascontiguousarray(active, np.uint8)
    lens = np.ascontiguousarray(seq_len, np.int64)
    nn = np.array([state.num_nodes], np.int32)
    nr = np.array([state.num_ranges], np.int32)
    ne = np.array([state.num_events], np.int32)
    f = _lib().kf_policy_monitor
    args = (ctypes.byref(p), 0, len(act), _ptr(act), _ptr(lens), _ptr(state.tail), _ptr(state.nodes),
            _ptr(nn), len(state.nodes), _ptr(state.ranges), _ptr(nr), len(state.ranges),
            _ptr(state.events), _ptr(ne), len(state.events))
    _check(f(*args), "kf_policy_monitor")
    before = (int(nn[0]), int(nr[0]), int(ne[0]))
    t0 = time.perf_counter()
    for _ in range(reps):
        f(*args)
    dt = (time.perf_counter() - t0) / reps
    if (int(nn[0]), int(nr[0]), int(ne[0])) != before:
        raise kf.KFError("time_monitor: the state changed while timing")
    return dt


@dataclass
class Simulation:
    state: State
    tails_per_step: np.ndarray     # [steps, B] node per append, -1 inactive
    seq_len: np.ndarray            # [B] final lengths
    max_node_bytes: int


def simulate(p: Params, seq_lens, gen_lens, steps: int, max_nodes=None, max_ranges=None,
             max_events=None) -> Simulation:
    """Sizes default to upper bounds: each step adds at most one node and
    two events per tail-holding node and one range per active request."""
    lens = np.ascontiguousarray(seq_lens, np.int64)
    gens = np.ascontiguousarray(gen_lens, np.int64)
    B = len(lens)
    if max_nodes is None or max_ranges is None or max_events is None:
        nn0, nr0 = np.zeros(1, np.int32), np.zeros(1, np.int32)
        c0, t0 = np.zeros(1, np.int64), np.zeros(max(B, 1), np.int32)
        st = _lib().kf_policy_init(ctypes.byref(p), _ptr(lens), B, 0, 0, _ptr(c0), _ptr(nn0),
                                   None, None, _ptr(nr0), _ptr(t0))
        if st not in (0, kf.ERR_CAPACITY):
            _check(st, "kf_policy_init")
        grow = int(min(int(np.count_nonzero(gens)), B) * steps)
        max_nodes = int(nn0[0]) + grow if max_nodes is None else max_nodes
        max_ranges = int(nr0[0]) + grow if max_ranges is None else max_ranges
        max_events = 2 * grow if max_events is None else max_events
    max_nodes, max_ranges, max_events = max(max_nodes, 1), max(max_ranges, 1), max(max_events, 1)
    nodes = np.zeros(max_nodes, NODE_DT)
    ranges = np.zeros(max_ranges, RANGE_DT)
    events = np.zeros(max_events, EVENT_DT)
    tail = np.zeros(max(B, 1), np.int32)
    tps = np.zeros((steps, max(B, 1)), np.int32)
    out_len = np.zeros(max(B, 1), np.int64)
    nn, nr, ne = (np.zeros(1, np.int32) for _ in range(3))
    peak = np.zeros(1, np.int64)
    _check(_lib().kf_policy_simulate(ctypes.byref(p), _ptr(lens), _ptr(gens), B, steps, max_nodes,
                                     max_ranges, max_events, _ptr(tps), _ptr(nodes), _ptr(nn),
                                     _ptr(ranges), _ptr(nr), _ptr(tail), _ptr(events), _ptr(ne),
                                     _ptr(out_len), _ptr(peak)), "kf_policy_simulate")
    st = State(nodes, ranges, tail[:B], events, int(nn[0]), int(nr[0]), int(ne[0]))
    return Simulation(st, tps[:, :B], out_len[:B], int(peak[0]))


@dataclass
class RouteTable:
    routes: np.ndarray             # [R, 6] int32 rows (seq, part, tok_begin, tok_end, page_base, page_cap)
    seq_route_begin: np.ndarray    # [B+1]
    range_to_route: np.ndarray     # [num ranges]
    page_ids: np.ndarray           # [pages]


def build_routes(ranges: np.ndarray, num_seqs: int, seq_len_now, page_size: int = kf.PAGE_SIZE,
                 free_pages=None) -> RouteTable:
    rg = np.ascontiguousarray(ranges, RANGE_DT)
    now = np.ascontiguousarray(seq_len_now, np.int64)
    R = len(rg)
    free = None if free_pages is None else np.ascontiguousarray(free_pages, np.int32)
    routes = np.zeros(max(R, 1), ROUTE_DT)
    srb = np.zeros(num_seqs + 1, np.int32)
    r2r = np.zeros(max(R, 1), np.int32)
    npg = np.zeros(1, np.int32)
    lib = _lib()
    args = lambda pids, cap: (_ptr(rg), R, num_seqs, _ptr(now), page_size, _ptr(free),
                              0 if free is None else len(free), _ptr(routes), _ptr(srb), _ptr(r2r),
                              _ptr(pids), cap, _ptr(npg))
    st = lib.kf_policy_build_routes(*args(None, 0))
    if st != kf.ERR_CAPACITY:
        _check(st, "kf_policy_build_routes")
    pids = np.zeros(max(int(npg[0]), 1), np.int32)
    _check(lib.kf_policy_build_routes(*args(pids, len(pids))), "kf_policy_build_routes")
    rows = routes[:R].view(np.int32).reshape(R, 6) if R else np.zeros((0, 6), np.int32)
    return RouteTable(rows.copy(), srb, r2r[:R].copy(), pids[:int(npg[0])].copy())
