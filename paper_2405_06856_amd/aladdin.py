"""Python binding of libaladdin (argument marshalling only).

Every function named ``ald_*`` forwards to the C-ABI entry point of the same
name declared in ``include/aladdin.h``; device arrays are passed as torch CUDA
tensors (PyTorch supplies device memory and the stream, nothing else).  All
placement arithmetic runs in the HIP kernels of ``libaladdin.so``; there is no
CPU fallback, and importing this module fails when the library is missing.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
# torch first: it loads the HIP runtime it was built with, which the library
# then shares; loaded the other way round the process can hold two runtimes
import torch  # noqa: F401

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libaladdin.so")

ALD_OK, ALD_EINVAL, ALD_EHIP, ALD_ESLOTS, ALD_ESTATE, ALD_EOVERFLOW, ALD_ESPACE = 0, -1, -2, -3, -4, -5, -6
ALD_EINCOMPLETE, ALD_EBLOCKED = -7, -8

KERNEL_KINDS = {"build": 0, "eval": 1, "select": 2, "commit": 3, "rebalance": 4}


class AladdinError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (code %d)" % (msg, code))
        self.code = code


class Model(ctypes.Structure):
    _fields_ = [("c1", ctypes.c_double), ("k1", ctypes.c_double), ("k1q", ctypes.c_double),
                ("c3", ctypes.c_double), ("c2", ctypes.c_double), ("k2", ctypes.c_double),
                ("ttft_slo", ctypes.c_double), ("decode_slo", ctypes.c_double),
                ("theta", ctypes.c_double), ("gamma_num", ctypes.c_int32),
                ("gamma_log2den", ctypes.c_int32)]


class Scenario(ctypes.Structure):
    _fields_ = [("n_workers", ctypes.c_int32), ("gpus_per_worker", ctypes.c_int32),
                ("kv_capacity", ctypes.c_int64), ("model", Model)]


DIAG_DTYPE = np.dtype([("n_feasible", "<i4"), ("near_tie", "<i4"), ("kv_peak_chosen", "<i8"),
                       ("kv_excess_min", "<i8"), ("ttft_chosen", "<f8"), ("tdec_chosen", "<f8")])
assert DIAG_DTYPE.itemsize == 40

SYMBOLS = ("ald_create", "ald_destroy", "ald_set_workspace", "ald_workspace_needed", "ald_workspace_size",
           "ald_sweep_workspace_size", "ald_set_tile", "ald_load_workers", "ald_load_workers_history",
           "ald_place_stream", "ald_place_stream_async", "ald_place_resume", "ald_place_stream_hb",
           "ald_place_grouped", "ald_move_requests",
           "ald_sweep_scenarios", "ald_sweep_scenarios_hb", "ald_sweep_scenarios_async", "ald_rebalance",
           "ald_rebalance_noalloc",
           "ald_worker_summary", "ald_set_profiling", "ald_kernel_time", "ald_place_stats", "ald_last_error",
           "ald_strerror")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libaladdin.so is not built (run __graft_entry__.build()): %s" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "ald_create": ([ctypes.POINTER(P), ctypes.c_int, P], ctypes.c_int),
        "ald_destroy": ([P], ctypes.c_int),
        "ald_set_workspace": ([P, P, ctypes.c_size_t], ctypes.c_int),
        "ald_workspace_needed": ([P, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
        "ald_workspace_size": ([P, i32, i64, ctypes.POINTER(Model), i32, i32, i32, ctypes.POINTER(ctypes.c_size_t)],
                               ctypes.c_int),
        "ald_sweep_workspace_size": ([P, i32, P, i32, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
        "ald_set_tile": ([P, i32], ctypes.c_int),
        "ald_load_workers": ([P, i32, ctypes.POINTER(Model), P, P, P, P, P, i32], ctypes.c_int),
        "ald_load_workers_history": ([P, i32, ctypes.POINTER(Model), P, P, P, P, P, P, i32], ctypes.c_int),
        "ald_place_stream": ([P, i32, P, P, i32, P, P], ctypes.c_int),
        "ald_place_stream_async": ([P, i32, P, P, i32, i32, P, P, P], ctypes.c_int),
        "ald_place_resume": ([P], ctypes.c_int),
        "ald_place_grouped": ([P, i32, P, i32, P, P, i32, P, P], ctypes.c_int),
        "ald_place_stream_hb": ([P, i32, P, P, P, P, P], ctypes.c_int),
        "ald_move_requests": ([P, i32, P, P, P, P], ctypes.c_int),
        "ald_sweep_scenarios": ([P, i32, P, i32, P, P, P, P, P, P], ctypes.c_int),
        "ald_sweep_scenarios_hb": ([P, i32, P, P, i32, P, P, P, P, P, P], ctypes.c_int),
        "ald_sweep_scenarios_async": ([P, i32, P, P, i32, P, P, i32, P, P, P, P, P], ctypes.c_int),
        "ald_rebalance": ([P, i32, P, P, P, P, P, P, P, P, P, P, P, P, P, P, i32, P, P], ctypes.c_int),
        "ald_rebalance_noalloc": ([P, i32, P, P, P, P, P, P, P, P, P, P, P, P, P, P, i32, P, P], ctypes.c_int),
        "ald_worker_summary": ([P, P, P, P, P], ctypes.c_int),
        "ald_set_profiling": ([P, i32], ctypes.c_int),
        "ald_kernel_time": ([P, i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)], ctypes.c_int),
        "ald_place_stats": ([P, ctypes.POINTER(i64)], ctypes.c_int),
        "ald_last_error": ([P], ctypes.c_char_p),
        "ald_strerror": ([ctypes.c_int], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    return L


_L = _load()


def _check(h, rc: int):
    if rc != ALD_OK:
        msg = _L.ald_last_error(h).decode() if h else _L.ald_strerror(rc).decode()
        raise AladdinError(rc, msg)


def _dptr(t) -> Optional[int]:
    """Device pointer of a contiguous torch CUDA tensor (None passes NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device (CUDA/HIP) tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


# ----------------------------------------------------------------------------- C-ABI mirrors
def ald_create(device: int = 0, stream: Optional[int] = None) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    rc = _L.ald_create(ctypes.byref(h), int(device), stream)
    _check(None, rc)
    return h


def ald_destroy(h) -> None:
    _L.ald_destroy(h)


def ald_set_workspace(h, workspace, nbytes: Optional[int] = None) -> None:
    """workspace: a contiguous device tensor (its bytes are the workspace), or None."""
    if workspace is None:
        _check(h, _L.ald_set_workspace(h, None, 0))
        return
    n = workspace.numel() * workspace.element_size() if nbytes is None else int(nbytes)
    _check(h, _L.ald_set_workspace(h, _dptr(workspace), n))


def ald_workspace_needed(h) -> int:
    n = ctypes.c_size_t()
    _check(h, _L.ald_workspace_needed(h, ctypes.byref(n)))
    return n.value


def ald_workspace_size(h, W: int, n_resident: int, model: Model, slots_per_worker: int = 0, with_history: bool = False,
                       Q: int = 0) -> int:
    n = ctypes.c_size_t()
    _check(h, _L.ald_workspace_size(h, int(W), int(n_resident), ctypes.byref(model), int(slots_per_worker),
                                    int(bool(with_history)), int(Q), ctypes.byref(n)))
    return n.value


def ald_sweep_workspace_size(h, S: int, scen, Q: int) -> int:
    n = ctypes.c_size_t()
    _check(h, _L.ald_sweep_workspace_size(h, int(S), ctypes.cast(scen, ctypes.c_void_p), int(Q), ctypes.byref(n)))
    return n.value


def ald_set_tile(h, tile_queries: int) -> None:
    _check(h, _L.ald_set_tile(h, int(tile_queries)))


def ald_load_workers(h, W: int, model: Model, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated,
                     slots_per_worker: int = 0) -> None:
    _check(h, _L.ald_load_workers(h, int(W), ctypes.byref(model), _dptr(kv_capacity), _dptr(res_offsets),
                                  _dptr(res_l_in), _dptr(res_l_pred), _dptr(res_generated),
                                  int(slots_per_worker)))


def ald_load_workers_history(h, W: int, model: Model, kv_capacity, res_offsets, res_l_in, res_l_pred,
                             res_generated, res_t_dec, slots_per_worker: int = 0) -> None:
    _check(h, _L.ald_load_workers_history(h, int(W), ctypes.byref(model), _dptr(kv_capacity), _dptr(res_offsets),
                                          _dptr(res_l_in), _dptr(res_l_pred), _dptr(res_generated),
                                          _dptr(res_t_dec), int(slots_per_worker)))


def ald_place_stream(h, Q: int, q_l_in, q_l_pred, heartbeat_every: int, out_worker, out_diag=None) -> None:
    _check(h, _L.ald_place_stream(h, int(Q), _dptr(q_l_in), _dptr(q_l_pred), int(heartbeat_every),
                                  _dptr(out_worker), _dptr(out_diag)))


def ald_place_stream_async(h, Q: int, q_l_in, q_l_pred, heartbeat_every: int, spare_rounds: int, out_worker,
                           out_diag, status) -> None:
    """status: device int32 [1], written when the stream reaches the call."""
    _check(h, _L.ald_place_stream_async(h, int(Q), _dptr(q_l_in), _dptr(q_l_pred), int(heartbeat_every),
                                        int(spare_rounds), _dptr(out_worker), _dptr(out_diag), _dptr(status)))


def ald_place_resume(h) -> None:
    _check(h, _L.ald_place_resume(h))


def ald_place_stream_hb(h, Q: int, q_l_in, q_l_pred, hb_before, out_worker, out_diag=None) -> None:
    """hb_before: host array of Q heartbeat counts."""
    hb = np.ascontiguousarray(hb_before, dtype=np.int32)
    if hb.shape != (int(Q),):
        raise ValueError("hb_before must hold one count per query")
    _check(h, _L.ald_place_stream_hb(h, int(Q), _dptr(q_l_in), _dptr(q_l_pred), hb.ctypes.data_as(ctypes.c_void_p),
                                     _dptr(out_worker), _dptr(out_diag)))


def ald_move_requests(h, K: int, l_in, l_pred, from_worker, to_worker) -> None:
    """Host arrays of K moves."""
    a = [np.ascontiguousarray(x, dtype=np.int32) for x in (l_in, l_pred, from_worker, to_worker)]
    if any(x.shape != (int(K),) for x in a):
        raise ValueError("every move array must hold K entries")
    _check(h, _L.ald_move_requests(h, int(K), *[x.ctypes.data_as(ctypes.c_void_p) for x in a]))


def ald_place_grouped(h, G: int, group_workers, Q: int, q_l_in, q_l_pred, heartbeat_every: int, out_worker,
                      out_diag=None) -> None:
    """group_workers: host array of G group sizes."""
    gw = np.ascontiguousarray(group_workers, dtype=np.int32)
    if gw.shape != (G,):
        raise ValueError("group_workers must hold G sizes")
    _check(h, _L.ald_place_grouped(h, int(G), gw.ctypes.data_as(ctypes.c_void_p), int(Q), _dptr(q_l_in),
                                   _dptr(q_l_pred), int(heartbeat_every), _dptr(out_worker), _dptr(out_diag)))


def ald_sweep_scenarios(h, S: int, scen, Q: int, q_l_in, q_l_pred, out_rejected, out_first_reject,
                        out_worker=None, out_min_gpus=None) -> None:
    _check(h, _L.ald_sweep_scenarios(h, int(S), ctypes.cast(scen, ctypes.c_void_p), int(Q), _dptr(q_l_in),
                                     _dptr(q_l_pred), _dptr(out_rejected), _dptr(out_first_reject),
                                     _dptr(out_worker), _dptr(out_min_gpus)))


def ald_sweep_scenarios_async(h, S: int, scen, heartbeat_every, Q: int, q_l_in, q_l_pred, spare_rounds: int,
                              out_rejected, out_first_reject, out_worker, out_min_gpus, status) -> None:
    """heartbeat_every: None or a host array of S periods; status: device int32 [1]."""
    hb = None
    if heartbeat_every is not None:
        hb = np.ascontiguousarray(heartbeat_every, dtype=np.int32)
        if hb.shape != (int(S),):
            raise ValueError("heartbeat_every must hold one period per scenario")
    _check(h, _L.ald_sweep_scenarios_async(h, int(S), ctypes.cast(scen, ctypes.c_void_p),
                                           None if hb is None else hb.ctypes.data_as(ctypes.c_void_p), int(Q),
                                           _dptr(q_l_in), _dptr(q_l_pred), int(spare_rounds), _dptr(out_rejected),
                                           _dptr(out_first_reject), _dptr(out_worker), _dptr(out_min_gpus),
                                           _dptr(status)))


def ald_sweep_scenarios_hb(h, S: int, scen, heartbeat_every, Q: int, q_l_in, q_l_pred, out_rejected,
                           out_first_reject, out_worker=None, out_min_gpus=None) -> None:
    """heartbeat_every: host array of S periods."""
    hb = np.ascontiguousarray(heartbeat_every, dtype=np.int32)
    if hb.shape != (S,):
        raise ValueError("heartbeat_every must hold one period per scenario")
    _check(h, _L.ald_sweep_scenarios_hb(h, int(S), ctypes.cast(scen, ctypes.c_void_p),
                                        hb.ctypes.data_as(ctypes.c_void_p), int(Q), _dptr(q_l_in), _dptr(q_l_pred),
                                        _dptr(out_rejected), _dptr(out_first_reject), _dptr(out_worker),
                                        _dptr(out_min_gpus)))


def _rebalance_call(fn, h, P: int, n_workers, models, old_offsets, old_worker, old_l_pred, old_l_out, old_l_real,
                  old_l_repred, new_offsets, new_l_pred, new_worker, out_le=None, out_be=None, out_moves=None,
                  log_cap=0, out_log=None, out_obj=None) -> None:
    nw = np.ascontiguousarray(n_workers, dtype=np.int32)
    oo = np.ascontiguousarray(old_offsets, dtype=np.int64)
    no = np.ascontiguousarray(new_offsets, dtype=np.int64)
    _check(h, fn(h, int(P), nw.ctypes.data_as(ctypes.c_void_p), ctypes.cast(models, ctypes.c_void_p),
                               oo.ctypes.data_as(ctypes.c_void_p), _dptr(old_worker), _dptr(old_l_pred),
                               _dptr(old_l_out), _dptr(old_l_real), _dptr(old_l_repred),
                               no.ctypes.data_as(ctypes.c_void_p), _dptr(new_l_pred), _dptr(new_worker),
                               _dptr(out_le), _dptr(out_be), _dptr(out_moves), int(log_cap), _dptr(out_log),
                               _dptr(out_obj)))


def ald_rebalance(h, P: int, n_workers, models, old_offsets, old_worker, old_l_pred, old_l_out, old_l_real,
                  old_l_repred, new_offsets, new_l_pred, new_worker, out_le=None, out_be=None, out_moves=None,
                  log_cap=0, out_log=None, out_obj=None) -> None:
    """n_workers (int32), models (Model array) and the offsets (int64) are host
    arrays; everything else is a device tensor."""
    _rebalance_call(_L.ald_rebalance, h, P, n_workers, models, old_offsets, old_worker, old_l_pred, old_l_out,
                    old_l_real, old_l_repred, new_offsets, new_l_pred, new_worker, out_le, out_be, out_moves,
                    log_cap, out_log, out_obj)


def ald_rebalance_noalloc(h, P: int, n_workers, models, old_offsets, old_worker, old_l_pred, old_l_out,
                          old_l_real, old_l_repred, new_offsets, new_l_pred, new_worker, out_le, out_be,
                          out_moves=None, log_cap=0, out_log=None, out_obj=None) -> None:
    """As ald_rebalance, with the library's fixed device array instead of
    allocated tables (out_le and out_be required)."""
    _rebalance_call(_L.ald_rebalance_noalloc, h, P, n_workers, models, old_offsets, old_worker, old_l_pred,
                    old_l_out, old_l_real, old_l_repred, new_offsets, new_l_pred, new_worker, out_le, out_be,
                    out_moves, log_cap, out_log, out_obj)


def ald_worker_summary(h, B, sum_c, sum_r, peak) -> None:
    _check(h, _L.ald_worker_summary(h, _dptr(B), _dptr(sum_c), _dptr(sum_r), _dptr(peak)))


def ald_set_profiling(h, kinds: int) -> None:
    _check(h, _L.ald_set_profiling(h, int(kinds)))


def ald_kernel_time(h, kind: int):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(h, _L.ald_kernel_time(h, int(kind), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def ald_place_stats(h):
    out = (ctypes.c_int64 * 4)()
    _check(h, _L.ald_place_stats(h, out))
    return {"rounds": out[0], "cuts": out[1], "fallbacks": out[2], "stale_cuts": out[3]}


def ald_last_error(h) -> str:
    return _L.ald_last_error(h).decode()


def ald_strerror(code: int) -> str:
    return _L.ald_strerror(int(code)).decode()


# ----------------------------------------------------------------------------- convenience wrapper
def to_model(m) -> Model:
    return Model(m.c1, m.k1, m.k1q, m.c3, m.c2, m.k2, m.ttft_slo, m.decode_slo, m.theta, m.gamma_num,
                 m.gamma_log2den)


@dataclass
class Placement:
    worker: np.ndarray                 # int32 [Q]
    diag: Optional[np.ndarray] = None  # DIAG_DTYPE [Q]


class Evaluator:
    """A handle bound to one device and torch's current stream on it.  It owns
    the handle's workspace, a torch uint8 tensor that grows (by at least a
    quarter) whenever a call reports that it needs more."""

    def __init__(self, device: int = 0, tile: Optional[int] = None, workspace_bytes: int = 0):
        import torch
        self.torch = torch
        self.device = torch.device("cuda", device)
        self.stream = torch.cuda.current_stream(self.device)
        self.h = ald_create(device, self.stream.cuda_stream)
        if tile is not None:
            ald_set_tile(self.h, tile)
        self.W = 0
        self.ws = None
        self.ws_bytes = 0
        if workspace_bytes > 0:
            self.attach_workspace(workspace_bytes)

    def attach_workspace(self, nbytes: int) -> None:
        """Give the handle a workspace of at least nbytes (the loaded state moves along)."""
        nbytes = (int(nbytes) + (1 << 21) - 1) & ~((1 << 21) - 1)
        ws = self.torch.empty(nbytes, dtype=self.torch.uint8, device=self.device)
        ald_set_workspace(self.h, ws, nbytes)
        self.ws, self.ws_bytes = ws, nbytes

    def call(self, fn, *args, **kw):
        """fn(handle, ...), growing the workspace and calling again when it is too small."""
        while True:
            try:
                return fn(self.h, *args, **kw)
            except AladdinError as e:
                if e.code != ALD_ESPACE:
                    raise
                need = ald_workspace_needed(self.h)
                if need <= self.ws_bytes:
                    raise
                self.attach_workspace(max(need, self.ws_bytes + self.ws_bytes // 4))

    def close(self):
        if self.h is not None:
            ald_destroy(self.h)
            self.h = None
        self.ws = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _dev(self, a, dtype):
        t = self.torch
        return t.as_tensor(np.ascontiguousarray(a), dtype=dtype).to(self.device)

    def load(self, W, model, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated, slots_per_worker=0,
             res_t_dec=None):
        """res_t_dec: the residents' decode times so far (seconds); given, constraint
        (d) is checked for every later placement."""
        t = self.torch
        self._keep = [self._dev(kv_capacity, t.int64), self._dev(res_offsets, t.int64),
                      self._dev(res_l_in, t.int32), self._dev(res_l_pred, t.int32),
                      self._dev(res_generated, t.int32)]
        if res_t_dec is None:
            self.call(ald_load_workers, W, to_model(model), *self._keep, slots_per_worker=slots_per_worker)
        else:
            self._keep.append(self._dev(res_t_dec, t.float64))
            self.call(ald_load_workers_history, W, to_model(model), *self._keep, slots_per_worker=slots_per_worker)
        self.W = W

    def load_trace(self, trace, slots_per_worker=0):
        self.load(trace.n_workers, trace.model, trace.kv_capacity, trace.res_offsets, trace.res_l_in,
                  trace.res_l_pred, trace.res_generated, slots_per_worker,
                  res_t_dec=getattr(trace, "res_t_dec", None))

    def place_device(self, q_l_in, q_l_pred, heartbeat_every=0, diag=True, out=None, diag_out=None):
        """Device tensors in, device tensors out (no host copies).  `out` (int32
        [Q]) and `diag_out` (uint8 [Q * 40]) may be passed to reuse buffers."""
        t = self.torch
        Q = int(q_l_in.numel())
        if out is None:
            out = t.empty(Q, dtype=t.int32, device=self.device)
        elif out.dtype != t.int32 or out.numel() < Q:
            raise ValueError("out must be an int32 tensor of at least Q elements")
        d = None
        if diag:
            d = diag_out
            if d is None:
                d = t.empty(Q * DIAG_DTYPE.itemsize, dtype=t.uint8, device=self.device)
            elif d.dtype != t.uint8 or d.numel() < Q * DIAG_DTYPE.itemsize:
                raise ValueError("diag_out must be a uint8 tensor of at least Q * %d bytes" % DIAG_DTYPE.itemsize)
        self.call(ald_place_stream, Q, q_l_in, q_l_pred, heartbeat_every, out, d)
        return out, d

    def place_async(self, q_l_in, q_l_pred, heartbeat_every=0, diag=True, out=None, diag_out=None, status=None,
                    spare_rounds=0):
        """As place_device, returning once the work is enqueued: (out, diag,
        status), where status (int32 [1] on the device) reads ALD_OK once the
        stream has placed every query, ALD_EINCOMPLETE if the rounds ran out
        (resume() finishes the call) or ALD_EBLOCKED if an earlier call was
        unfinished (issue it again after resume())."""
        t = self.torch
        Q = int(q_l_in.numel())
        if out is None:
            out = t.empty(max(Q, 1), dtype=t.int32, device=self.device)
        elif out.dtype != t.int32 or out.numel() < Q:
            raise ValueError("out must be an int32 tensor of at least Q elements")
        d = None
        if diag:
            d = diag_out
            if d is None:
                d = t.empty(max(Q, 1) * DIAG_DTYPE.itemsize, dtype=t.uint8, device=self.device)
            elif d.dtype != t.uint8 or d.numel() < Q * DIAG_DTYPE.itemsize:
                raise ValueError("diag_out must be a uint8 tensor of at least Q * %d bytes" % DIAG_DTYPE.itemsize)
        if status is None:
            status = t.empty(1, dtype=t.int32, device=self.device)
        elif status.dtype != t.int32 or status.numel() < 1:
            raise ValueError("status must be an int32 tensor of at least one element")
        self.call(ald_place_stream_async, Q, q_l_in, q_l_pred, heartbeat_every, spare_rounds, out, d, status)
        return out[:Q], (None if d is None else d[:Q * DIAG_DTYPE.itemsize]), status

    def resume(self) -> None:
        """Finish an asynchronous placement that ran out of rounds (synchronously)."""
        ald_place_resume(self.h)

    def place(self, q_l_in, q_l_pred, heartbeat_every=0, diag=True, hb_before=None) -> Placement:
        """hb_before: decode iterations before each query (instead of a period)."""
        t = self.torch
        ql = self._dev(q_l_in, t.int32)
        qp = self._dev(q_l_pred, t.int32)
        if hb_before is None:
            out, d = self.place_device(ql, qp, heartbeat_every, diag)
        else:
            Q = int(ql.numel())
            out = t.empty(max(Q, 1), dtype=t.int32, device=self.device)
            d = t.empty(max(Q, 1) * DIAG_DTYPE.itemsize, dtype=t.uint8, device=self.device) if diag else None
            self.call(ald_place_stream_hb, Q, ql, qp, hb_before, out, d)
            out = out[:Q]
            d = None if d is None else d[:Q * DIAG_DTYPE.itemsize]
        res = Placement(worker=out.cpu().numpy())
        if d is not None:
            res.diag = d.cpu().numpy().view(DIAG_DTYPE)
        return res

    def move_requests(self, l_in, l_pred, from_worker, to_worker) -> None:
        """Move requests placed in the current heartbeat window between workers."""
        self.call(ald_move_requests, len(l_in), l_in, l_pred, from_worker, to_worker)

    def place_grouped(self, group_workers, q_l_in, q_l_pred, heartbeat_every=0, diag=True) -> Placement:
        """Grouped placement (App. A): the router gives group i the share
        N_i / N_w of the stream (every count within one query of its share) and
        each group places its queries on its own workers."""
        t = self.torch
        ql = self._dev(q_l_in, t.int32)
        qp = self._dev(q_l_pred, t.int32)
        Q = int(ql.numel())
        out = t.empty(max(Q, 1), dtype=t.int32, device=self.device)
        d = t.empty(max(Q, 1) * DIAG_DTYPE.itemsize, dtype=t.uint8, device=self.device) if diag else None
        self.call(ald_place_grouped, len(group_workers), group_workers, Q, ql, qp, heartbeat_every, out, d)
        res = Placement(worker=out[:Q].cpu().numpy())
        if diag:
            res.diag = d[:Q * DIAG_DTYPE.itemsize].cpu().numpy().view(DIAG_DTYPE)
        return res

    def summary(self):
        t = self.torch
        W = self.W
        B = t.empty(W, dtype=t.int32, device=self.device)
        sc = t.empty(W, dtype=t.int64, device=self.device)
        sr = t.empty(W, dtype=t.int64, device=self.device)
        pk = t.empty(W, dtype=t.int64, device=self.device)
        ald_worker_summary(self.h, B, sc, sr, pk)
        return {"B": B.cpu().numpy(), "sum_c": sc.cpu().numpy(), "sum_r": sr.cpu().numpy(),
                "peak": pk.cpu().numpy()}

    def sweep(self, scenarios, q_l_in, q_l_pred, want_workers=False, heartbeat_every=None, want_answer=False):
        """heartbeat_every: None (no heartbeat), one period for all scenarios, or
        one per scenario.  Returns (rejected, first rejected, workers or None),
        and with want_answer also the device's answer (fewest GPUs, scenario)."""
        t = self.torch
        S = len(scenarios)
        arr = (Scenario * S)()
        for i, s in enumerate(scenarios):
            arr[i] = Scenario(s.n_workers, s.gpus_per_worker, s.kv_capacity, to_model(s.model))
        ql = self._dev(q_l_in, t.int32)
        qp = self._dev(q_l_pred, t.int32)
        Q = int(ql.numel())
        rej = t.empty(S, dtype=t.int32, device=self.device)
        first = t.empty(S, dtype=t.int32, device=self.device)
        ow = t.empty(S * Q, dtype=t.int32, device=self.device) if want_workers else None
        best = t.empty(2, dtype=t.int64, device=self.device)
        if heartbeat_every is None:
            self.call(ald_sweep_scenarios, S, arr, Q, ql, qp, rej, first, ow, best)
        else:
            hb = np.broadcast_to(np.asarray(heartbeat_every, dtype=np.int32), (S,))
            self.call(ald_sweep_scenarios_hb, S, arr, hb, Q, ql, qp, rej, first, ow, best)
        out = (rej.cpu().numpy(), first.cpu().numpy(), ow.cpu().numpy().reshape(S, Q) if want_workers else None)
        if want_answer:
            b = best.cpu().numpy()
            out = out + ((None, -1) if b[0] < 0 else (int(b[0]), int(b[1])),)
        return out

    def sweep_async(self, scenarios, q_l_in, q_l_pred, want_workers=False, heartbeat_every=None, spare_rounds=0):
        """As sweep, with device query tensors, returning once the work is
        enqueued: device tensors (rejected, first rejected, workers or None,
        answer int64 [2], status int32 [1]); status reads ALD_OK once the
        stream has run the sweep, ALD_EINCOMPLETE if its rounds ran out."""
        t = self.torch
        S = len(scenarios)
        arr = (Scenario * S)()
        for i, s in enumerate(scenarios):
            arr[i] = Scenario(s.n_workers, s.gpus_per_worker, s.kv_capacity, to_model(s.model))
        Q = int(q_l_in.numel())
        rej = t.empty(S, dtype=t.int32, device=self.device)
        first = t.empty(S, dtype=t.int32, device=self.device)
        ow = t.empty(max(S * Q, 1), dtype=t.int32, device=self.device) if want_workers else None
        best = t.empty(2, dtype=t.int64, device=self.device)
        status = t.empty(1, dtype=t.int32, device=self.device)
        hb = None if heartbeat_every is None else np.broadcast_to(np.asarray(heartbeat_every, dtype=np.int32), (S,))
        self.call(ald_sweep_scenarios_async, S, arr, hb, Q, q_l_in, q_l_pred, spare_rounds, rej, first, ow, best,
                  status)
        return rej, first, ow, best, status

    def rebalance(self, batch, want_log=False):
        """Algorithm 2 on a workloads.RebalanceBatch; returns the new workers and
        per-problem results as numpy arrays (obj: [P, 4] pairs a + rho * b,
        before then after; log: per problem, its moves as (request, target))."""
        t = self.torch
        P = batch.P
        models = (Model * P)(*[to_model(m) for m in batch.models])
        d32 = lambda a: self._dev(a, t.int32)
        nw = d32(batch.new_worker)
        Wt = int(np.sum(batch.n_workers))
        le = t.empty(Wt, dtype=t.int64, device=self.device)
        be = t.empty(Wt, dtype=t.int64, device=self.device)
        mv = t.empty(P, dtype=t.int32, device=self.device)
        obj = t.empty(4 * P, dtype=t.int64, device=self.device)
        n_new = np.diff(batch.new_offsets)
        cap = int(4 * n_new.max() + int(np.max(batch.n_workers))) if want_log and P > 0 else 0
        log = t.empty(max(1, 2 * P * cap), dtype=t.int32, device=self.device) if want_log else None
        self.call(ald_rebalance, P, batch.n_workers, models, batch.old_offsets, d32(batch.old_worker),
                 d32(batch.old_l_pred), d32(batch.old_l_out), d32(batch.old_l_real), d32(batch.old_l_repred),
                 batch.new_offsets, d32(batch.new_l_pred), nw, le, be, mv, cap, log, obj)
        out = {"worker": nw.cpu().numpy(), "le": le.cpu().numpy(), "be": be.cpu().numpy(),
               "moves": mv.cpu().numpy(), "obj": obj.cpu().numpy().reshape(P, 4)}
        if want_log:
            lg = log.cpu().numpy()
            k = out["moves"]
            out["log"] = [lg[2 * p * cap:2 * p * cap + 2 * int(k[p])].reshape(-1, 2) for p in range(P)]
        return out

    def profiling(self, enable=True, kinds=None):
        """Time kernel kinds with HIP events: all of them, or the names in `kinds`."""
        if not enable:
            mask = 0
        elif kinds is None:
            mask = 31
        else:
            mask = 0
            for k in kinds:
                mask |= 1 << KERNEL_KINDS[k]
        ald_set_profiling(self.h, mask)

    def kernel_time(self, kind: str):
        return ald_kernel_time(self.h, KERNEL_KINDS[kind])

    def tile_stats(self):
        """How the last placement call split the arrival-order commit into tiles."""
        return ald_place_stats(self.h)


def smallest_feasible_cluster(scenarios, rejected):
    """The sweep's answer recomputed from its per-scenario rejections (a
    cross-check of the device's out_min_gpus): the scenario with no rejection
    and the fewest GPUs (n_workers * gpus_per_worker), lowest index on ties;
    returns (gpus, index) or (None, -1)."""
    best, idx = None, -1
    for i, s in enumerate(scenarios):
        if int(rejected[i]) != 0:
            continue
        g = s.n_workers * s.gpus_per_worker
        if best is None or g < best:
            best, idx = g, i
    return best, idx
