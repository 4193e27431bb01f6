"""ctypes front end of the C oracle (test infrastructure only).

The C source (``aladdin_oracle.c``) holds all of the oracle's arithmetic; this
module only marshals numpy arrays.  It imports nothing from the GPU package
except the seeded workload generator.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "aladdin_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

ORA_OK, ORA_EINVAL, ORA_ENOMEM, ORA_EOVERFLOW, ORA_ECHECK = 0, -1, -2, -3, -4


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64 without contraction or fast-math)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
               "-shared", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, LIB)
    return LIB


class OraModel(ctypes.Structure):
    _fields_ = [("c1", ctypes.c_double), ("k1", ctypes.c_double), ("k1q", ctypes.c_double),
                ("c3", ctypes.c_double), ("c2", ctypes.c_double), ("k2", ctypes.c_double),
                ("ttft_slo", ctypes.c_double), ("decode_slo", ctypes.c_double),
                ("theta", ctypes.c_double), ("gamma_num", ctypes.c_int32),
                ("gamma_log2den", ctypes.c_int32)]


class OraScenario(ctypes.Structure):
    _fields_ = [("n_workers", ctypes.c_int32), ("gpus_per_worker", ctypes.c_int32),
                ("kv_capacity", ctypes.c_int64), ("model", OraModel)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        # ORACLE_LIB: a separately built copy of the oracle (the sanitizer test
        # builds one with AddressSanitizer and UBSan); otherwise build LIB here
        path = os.environ.get("ORACLE_LIB")
        if not path:
            build()
            path = LIB
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        L.ora_place.argtypes = [i32, P, P, P, P, P, P, ctypes.POINTER(OraModel), i32, P, P, i32, i32, i32,
                                i32, P, P, P, P, P, P, P, P, P, P, P, P, P]
        L.ora_place.restype = ctypes.c_int
        L.ora_place_hb.argtypes = [i32, P, P, P, P, P, P, ctypes.POINTER(OraModel), i32, P, P, P, i32,
                                   P, P, P, P, P, P, P, P, P, P, P, P, P]
        L.ora_place_hb.restype = ctypes.c_int
        L.ora_place_moves.argtypes = [i32, P, P, P, P, P, P, ctypes.POINTER(OraModel), i32, P, P, P, i32, P, P, P,
                                      P, P, P, P, P, P, P, P, P, P, P, P, P]
        L.ora_place_moves.restype = ctypes.c_int
        L.ora_place_grouped.argtypes = [i32, P, P, P, P, P, P, ctypes.POINTER(OraModel), i32, P, i32, P, P, i32,
                                        P, P, P, P, P, P, P, P, P, P, P, P, P]
        L.ora_place_grouped.restype = ctypes.c_int
        L.ora_route_groups.argtypes = [i32, P, i32, P]
        L.ora_route_groups.restype = ctypes.c_int
        L.ora_sweep.argtypes = [i32, P, P, i32, P, P, i32, P, P, P]
        L.ora_sweep.restype = ctypes.c_int
        L.ora_kv_peak.argtypes = [i64, P, P]
        L.ora_kv_peak.restype = i64
        L.ora_rb_sign.argtypes = [i64, i64, ctypes.POINTER(OraModel)]
        L.ora_rb_sign.restype = ctypes.c_int
        L.ora_rebalance.argtypes = [i32, ctypes.POINTER(OraModel), i32, P, P, P, P, P, i32, P, P, P, P, P, i32, P,
                                    P, P]
        L.ora_rebalance.restype = ctypes.c_int
        _lib = L
    return _lib


def to_model(m) -> OraModel:
    return OraModel(m.c1, m.k1, m.k1q, m.c3, m.c2, m.k2, m.ttft_slo, m.decode_slo, m.theta,
                    m.gamma_num, m.gamma_log2den)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


@dataclass
class PlaceResult:
    worker: np.ndarray          # int32 [Q]
    n_feasible: np.ndarray      # int32 [Q]
    near_tie: np.ndarray        # int32 [Q]
    kv_peak_chosen: np.ndarray  # int64 [Q]
    kv_excess_min: np.ndarray   # int64 [Q]
    ttft_chosen: np.ndarray     # float64 [Q]
    tdec_chosen: np.ndarray     # float64 [Q]
    B: np.ndarray               # int64 [W] final batch size
    sum_c: np.ndarray
    sum_r: np.ndarray
    peak: np.ndarray
    S1: np.ndarray
    S2: np.ndarray


def place(W, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated, model, q_l_in, q_l_pred,
          heartbeat_every=0, no_commit=False, check=False, n_threads=1, res_t_dec=None) -> PlaceResult:
    """res_t_dec: each resident's decode time so far in seconds; when given,
    constraint (d) is evaluated as well."""
    L = lib()
    Q = int(len(q_l_in))
    c64 = lambda a: np.ascontiguousarray(a, dtype=np.int64)
    c32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    M = c64(kv_capacity)
    off = c64(res_offsets) if res_offsets is not None else None
    rl, rp, rg = (c32(a) if a is not None else None for a in (res_l_in, res_l_pred, res_generated))
    td = np.ascontiguousarray(res_t_dec, dtype=np.float64) if res_t_dec is not None else None
    ql, qp = c32(q_l_in), c32(q_l_pred)
    out = PlaceResult(*(np.zeros(Q, t) for t in (np.int32, np.int32, np.int32, np.int64, np.int64,
                                                 np.float64, np.float64)),
                      *(np.zeros(W, np.int64) for _ in range(6)))
    m = to_model(model)
    rc = L.ora_place(W, _ptr(M), _ptr(off), _ptr(rl), _ptr(rp), _ptr(rg), _ptr(td), ctypes.byref(m), Q,
                     _ptr(ql), _ptr(qp), int(heartbeat_every), int(bool(no_commit)), int(bool(check)),
                     int(n_threads), _ptr(out.worker), _ptr(out.n_feasible), _ptr(out.near_tie),
                     _ptr(out.kv_peak_chosen), _ptr(out.kv_excess_min), _ptr(out.ttft_chosen),
                     _ptr(out.tdec_chosen), _ptr(out.B), _ptr(out.sum_c), _ptr(out.sum_r),
                     _ptr(out.peak), _ptr(out.S1), _ptr(out.S2))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_place failed with code %d" % rc)
    return out


def place_hb(W, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated, model, q_l_in, q_l_pred,
             hb_before, check=False, res_t_dec=None) -> PlaceResult:
    """As place, with hb_before[q] decode iterations (heartbeats) before query q."""
    L = lib()
    Q = int(len(q_l_in))
    c64 = lambda a: np.ascontiguousarray(a, dtype=np.int64)
    c32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    M = c64(kv_capacity)
    off = c64(res_offsets) if res_offsets is not None else None
    rl, rp, rg = (c32(a) if a is not None else None for a in (res_l_in, res_l_pred, res_generated))
    td = np.ascontiguousarray(res_t_dec, dtype=np.float64) if res_t_dec is not None else None
    ql, qp, hbb = c32(q_l_in), c32(q_l_pred), c32(hb_before)
    out = PlaceResult(*(np.zeros(Q, t) for t in (np.int32, np.int32, np.int32, np.int64, np.int64,
                                                 np.float64, np.float64)),
                      *(np.zeros(W, np.int64) for _ in range(6)))
    m = to_model(model)
    rc = L.ora_place_hb(W, _ptr(M), _ptr(off), _ptr(rl), _ptr(rp), _ptr(rg), _ptr(td), ctypes.byref(m), Q,
                        _ptr(ql), _ptr(qp), _ptr(hbb), int(bool(check)), _ptr(out.worker), _ptr(out.n_feasible),
                        _ptr(out.near_tie), _ptr(out.kv_peak_chosen), _ptr(out.kv_excess_min),
                        _ptr(out.ttft_chosen), _ptr(out.tdec_chosen), _ptr(out.B), _ptr(out.sum_c),
                        _ptr(out.sum_r), _ptr(out.peak), _ptr(out.S1), _ptr(out.S2))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_place_hb failed with code %d" % rc)
    return out


def place_moves(W, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated, model, q_l_in, q_l_pred,
                moves, hb_before=None, res_t_dec=None) -> PlaceResult:
    """As place_hb (hb_before None: no heartbeat), with moves = [(at, query, to)]:
    before query `at` the request of `query` (placed in the current window)
    moves to worker `to`."""
    L = lib()
    Q = int(len(q_l_in))
    c64 = lambda a: np.ascontiguousarray(a, dtype=np.int64)
    c32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    M = c64(kv_capacity)
    off = c64(res_offsets) if res_offsets is not None else None
    rl, rp, rg = (c32(a) if a is not None else None for a in (res_l_in, res_l_pred, res_generated))
    td = np.ascontiguousarray(res_t_dec, dtype=np.float64) if res_t_dec is not None else None
    ql, qp = c32(q_l_in), c32(q_l_pred)
    hbb = c32(hb_before) if hb_before is not None else None
    mv = np.asarray(moves, dtype=np.int32).reshape(-1, 3)
    at, qi, to = (np.ascontiguousarray(mv[:, k]) for k in range(3))
    out = PlaceResult(*(np.zeros(Q, t) for t in (np.int32, np.int32, np.int32, np.int64, np.int64,
                                                 np.float64, np.float64)),
                      *(np.zeros(W, np.int64) for _ in range(6)))
    m = to_model(model)
    rc = L.ora_place_moves(W, _ptr(M), _ptr(off), _ptr(rl), _ptr(rp), _ptr(rg), _ptr(td), ctypes.byref(m), Q,
                           _ptr(ql), _ptr(qp), _ptr(hbb), len(mv), _ptr(at), _ptr(qi), _ptr(to), _ptr(out.worker),
                           _ptr(out.n_feasible), _ptr(out.near_tie), _ptr(out.kv_peak_chosen),
                           _ptr(out.kv_excess_min), _ptr(out.ttft_chosen), _ptr(out.tdec_chosen), _ptr(out.B),
                           _ptr(out.sum_c), _ptr(out.sum_r), _ptr(out.peak), _ptr(out.S1), _ptr(out.S2))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_place_moves failed with code %d" % rc)
    return out


def route_groups(sizes, Q) -> np.ndarray:
    """App. A's router: the group of each of the first Q queries."""
    g = np.ascontiguousarray(sizes, dtype=np.int32)
    out = np.zeros(max(int(Q), 1), np.int32)
    rc = lib().ora_route_groups(len(g), _ptr(g), int(Q), _ptr(out))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_route_groups failed with code %d" % rc)
    return out[:int(Q)]


def place_grouped(W, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated, model, group_sizes, q_l_in,
                  q_l_pred, heartbeat_every=0, res_t_dec=None) -> PlaceResult:
    """Grouped placement (App. A): each query goes to the group the router
    picks and is placed among that group's workers; heartbeats every
    heartbeat_every queries of the whole stream."""
    L = lib()
    Q = int(len(q_l_in))
    c64 = lambda a: np.ascontiguousarray(a, dtype=np.int64)
    c32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    M = c64(kv_capacity)
    off = c64(res_offsets) if res_offsets is not None else None
    rl, rp, rg = (c32(a) if a is not None else None for a in (res_l_in, res_l_pred, res_generated))
    td = np.ascontiguousarray(res_t_dec, dtype=np.float64) if res_t_dec is not None else None
    ql, qp, gs = c32(q_l_in), c32(q_l_pred), c32(group_sizes)
    out = PlaceResult(*(np.zeros(Q, t) for t in (np.int32, np.int32, np.int32, np.int64, np.int64,
                                                 np.float64, np.float64)),
                      *(np.zeros(W, np.int64) for _ in range(6)))
    m = to_model(model)
    rc = L.ora_place_grouped(W, _ptr(M), _ptr(off), _ptr(rl), _ptr(rp), _ptr(rg), _ptr(td), ctypes.byref(m),
                             len(gs), _ptr(gs), Q, _ptr(ql), _ptr(qp), int(heartbeat_every), _ptr(out.worker),
                             _ptr(out.n_feasible), _ptr(out.near_tie), _ptr(out.kv_peak_chosen),
                             _ptr(out.kv_excess_min), _ptr(out.ttft_chosen), _ptr(out.tdec_chosen), _ptr(out.B),
                             _ptr(out.sum_c), _ptr(out.sum_r), _ptr(out.peak), _ptr(out.S1), _ptr(out.S2))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_place_grouped failed with code %d" % rc)
    return out


def place_trace(trace, q_slice=slice(None), **kw) -> PlaceResult:
    """Run the oracle on a workloads.Trace (optionally on a slice of its queries)."""
    return place(trace.n_workers, trace.kv_capacity, trace.res_offsets, trace.res_l_in,
                 trace.res_l_pred, trace.res_generated, trace.model, trace.q_l_in[q_slice],
                 trace.q_l_pred[q_slice], heartbeat_every=kw.pop("heartbeat_every", trace.heartbeat_every),
                 res_t_dec=kw.pop("res_t_dec", getattr(trace, "res_t_dec", None)), **kw)


def sweep(scenarios, q_l_in, q_l_pred, want_workers=False, n_threads=1, heartbeat_every=None):
    """heartbeat_every: None (no heartbeat), one period for every scenario, or one per scenario."""
    L = lib()
    S = len(scenarios)
    Q = int(len(q_l_in))
    arr = (OraScenario * max(S, 1))()
    for i, s in enumerate(scenarios):
        arr[i] = OraScenario(s.n_workers, s.gpus_per_worker, s.kv_capacity, to_model(s.model))
    rej = np.zeros(S, np.int32)
    first = np.zeros(S, np.int32)
    workers = np.zeros(S * Q, np.int32) if want_workers else None
    ql = np.ascontiguousarray(q_l_in, dtype=np.int32)
    qp = np.ascontiguousarray(q_l_pred, dtype=np.int32)
    H = None
    if heartbeat_every is not None:
        H = np.ascontiguousarray(np.broadcast_to(np.asarray(heartbeat_every, dtype=np.int32), (S,)))
    rc = L.ora_sweep(S, ctypes.cast(arr, ctypes.c_void_p), _ptr(H), Q, _ptr(ql), _ptr(qp), int(n_threads), _ptr(rej),
                     _ptr(first), _ptr(workers))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_sweep failed with code %d" % rc)
    return rej, first, (workers.reshape(S, Q) if want_workers else None)


def kv_peak(c, r) -> int:
    c = np.ascontiguousarray(c, dtype=np.int64)
    r = np.ascontiguousarray(r, dtype=np.int64)
    return int(lib().ora_kv_peak(len(c), _ptr(c), _ptr(r)))


def min_gpus(scenarios, rejected):
    """Smallest total GPU count (n_workers * gpus_per_worker) over scenarios with
    no rejection; ties go to the lowest scenario index.  Returns (gpus, index)
    or (None, -1) when every scenario rejects something."""
    best, idx = None, -1
    for i, (s, r) in enumerate(zip(scenarios, rejected)):
        if r == 0:
            g = s.n_workers * s.gpus_per_worker
            if best is None or g < best:
                best, idx = g, i
    return best, idx


@dataclass
class RebalanceResult:
    worker: np.ndarray      # int32 [n_new] worker of each new request after the moves
    le: np.ndarray          # int64 [W] output-length error per worker after the moves
    be: np.ndarray          # int64 [W] batch-size error per worker after the moves
    moves: np.ndarray       # int32 [n_moves, 2] (request, target worker) in the order applied
    obj_before: tuple       # sum over workers of |l^e + rho * b^e| before the moves, as (a, b) = a + rho * b
    obj_after: tuple


def rb_sign(a: int, b: int, model) -> int:
    """Exact sign of a + (c2 / k2) * b."""
    return int(lib().ora_rb_sign(int(a), int(b), ctypes.byref(to_model(model))))


def rebalance(W, model, old_worker, old_l_pred, old_l_out, old_l_real, old_l_repred, new_l_pred,
              new_worker) -> RebalanceResult:
    """Algorithm 2 on explicit arrays (the new requests' workers are not modified)."""
    L = lib()
    c32 = lambda a: np.ascontiguousarray(a, dtype=np.int32)
    ow, op, oo, orl, orp = (c32(a) for a in (old_worker, old_l_pred, old_l_out, old_l_real, old_l_repred))
    nlp = c32(new_l_pred)
    nw = np.array(new_worker, dtype=np.int32, copy=True)
    n_old, n_new = len(ow), len(nlp)
    le = np.zeros(W, np.int64)
    be = np.zeros(W, np.int64)
    cap = 4 * n_new + int(W)  # the oracle's own bound on the number of moves
    log = np.zeros(2 * max(cap, 1), np.int32)
    nm = ctypes.c_int32(0)
    ob = np.zeros(2, np.int64)
    oa = np.zeros(2, np.int64)
    m = to_model(model)
    rc = L.ora_rebalance(int(W), ctypes.byref(m), n_old, _ptr(ow), _ptr(op), _ptr(oo), _ptr(orl), _ptr(orp),
                         n_new, _ptr(nlp), _ptr(nw), _ptr(le), _ptr(be), ctypes.byref(nm), cap, _ptr(log),
                         _ptr(ob), _ptr(oa))
    if rc != ORA_OK:
        raise RuntimeError("oracle ora_rebalance failed with code %d" % rc)
    k = nm.value
    return RebalanceResult(nw, le, be, log[:2 * k].reshape(k, 2), (int(ob[0]), int(ob[1])),
                           (int(oa[0]), int(oa[1])))
