"""Seeded synthetic serving traces for the placement evaluator.

This module is the only code shared by the HIP path and the CPU oracle.  It
draws raw request descriptions (input length, predicted output length, tokens
generated so far) and builds latency-model coefficient sets.  It holds none of
the placement method's arithmetic: KV contexts, remaining lengths, peaks,
latencies and decisions are computed separately by each side.

The paper's workload is ShareGPT prompt lengths with model-generated output
lengths and Poisson arrivals (Evaluation, "Workload" paragraph); neither the
dataset nor the model outputs are available here, so clipped lognormal lengths
stand in for them, with the shapes listed in ``CONFIGS`` below.

Draw order for every trace (one ``numpy.random.default_rng(seed)`` each):
  1. resident input lengths      (worker-major, W*R values)
  2. resident predicted outputs  (W*R)
  3. resident generated-so-far   g ~ integers(0, l_pred), exclusive bound
  4. query input lengths         (Q)
  5. query predicted outputs     (Q)
  6. arrival process             (exponential inter-arrivals, thinned when the
                                  rate is time-varying); absent when no rate is
                                  given.
A length is ``clip(rint(lognormal(mu, sigma)), lo, hi)``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

__all__ = [
    "Model", "Trace", "Scenario", "SweepTrace", "CONFIGS", "make_config",
    "make_trace", "make_sweep", "BASE_MODEL", "scenario_index", "RebalanceBatch", "make_rebalance",
]


@dataclasses.dataclass(frozen=True)
class Model:
    """Latency/SLO model of one worker type (fp64 coefficients).

    Prefill iteration time (Eq. 2, plus a quadratic term the workloads add):
        T_p = (c1 + k1*S1) + k1q*S2,  S1 = sum l_in, S2 = sum l_in^2
    Decode iteration time (Eq. 3 written per batch):
        T_d = (c3 + c2*b) + k2*ctx
    ``ttft_slo`` is T_pre (Table 1), ``decode_slo`` the ATGT SLO T_dec (Sec. 2.2),
    ``theta`` the prediction-error knob of constraints (b)/(d) and
    gamma = gamma_num / 2**gamma_log2den the strictness knob of constraint (b).
    """
    c1: float
    k1: float
    k1q: float
    c3: float
    c2: float
    k2: float
    ttft_slo: float
    decode_slo: float
    theta: float = 1.0
    gamma_num: int = 1
    gamma_log2den: int = 1

    def scaled(self, factor: float) -> "Model":
        """All six latency coefficients multiplied by ``factor``."""
        return dataclasses.replace(
            self, c1=self.c1 * factor, k1=self.k1 * factor, k1q=self.k1q * factor,
            c3=self.c3 * factor, c2=self.c2 * factor, k2=self.k2 * factor)

    def per_gpu_scaled(self, gpus: int) -> "Model":
        """Compute (slope) terms divided by 0.8*gpus; intercepts c1, c3 kept.

        Follows the form of Eq. 5 (t = k4/N_g + c4): only the load-dependent
        part of an iteration shrinks with more GPUs per worker."""
        d = 0.8 * gpus
        return dataclasses.replace(self, k1=self.k1 / d, k1q=self.k1q / d,
                                   c2=self.c2 / d, k2=self.k2 / d)


# Coefficients stated for the tiny workload: T_p = 0.01 + 2e-5*sum(l_in) +
# 1e-9*sum(l_in^2), T_d = 0.008 + 1e-4*B + 2e-7*sum(KV); TTFT 1 s, decode 0.05 s.
BASE_MODEL = Model(c1=0.01, k1=2e-5, k1q=1e-9, c3=0.008, c2=1e-4, k2=2e-7,
                   ttft_slo=1.0, decode_slo=0.05)


@dataclasses.dataclass
class Trace:
    """One placement problem: W workers with residents, then Q queries."""
    name: str
    seed: int
    model: Model
    kv_capacity: np.ndarray        # int64 [W]
    res_offsets: np.ndarray        # int64 [W+1], CSR into the resident arrays
    res_l_in: np.ndarray           # int32 [n_res]
    res_l_pred: np.ndarray         # int32 [n_res]
    res_generated: np.ndarray      # int32 [n_res], 0 <= g < l_pred
    q_l_in: np.ndarray             # int32 [Q]
    q_l_pred: np.ndarray           # int32 [Q]
    arrivals: Optional[np.ndarray]  # float64 [Q] seconds, or None
    heartbeat_every: int = 0       # 0: the whole stream is one heartbeat
    res_t_dec: Optional[np.ndarray] = None  # float64 [n_res] decode time so far (s), or None

    @property
    def n_workers(self) -> int:
        return int(self.kv_capacity.shape[0])

    @property
    def n_queries(self) -> int:
        return int(self.q_l_in.shape[0])

    @property
    def n_resident(self) -> int:
        return int(self.res_l_in.shape[0])


@dataclasses.dataclass(frozen=True)
class Scenario:
    """One cluster configuration of a scaling sweep (workers start empty)."""
    n_workers: int
    gpus_per_worker: int
    kv_capacity: int
    model: Model


@dataclasses.dataclass
class SweepTrace:
    name: str
    seed: int
    scenarios: List[Scenario]
    q_l_in: np.ndarray
    q_l_pred: np.ndarray
    arrivals: Optional[np.ndarray]

    @property
    def n_queries(self) -> int:
        return int(self.q_l_in.shape[0])


def _lengths(rng: np.random.Generator, mu: float, sigma: float, lo: int, hi: int, n: int) -> np.ndarray:
    x = rng.lognormal(mu, sigma, n)
    return np.clip(np.rint(x), lo, hi).astype(np.int32)


def _poisson_arrivals(rng: np.random.Generator, n: int, rate: float) -> np.ndarray:
    return np.cumsum(rng.exponential(1.0 / rate, n))


def _thinned_arrivals(rng: np.random.Generator, n: int, base: float, depth: float, period: float) -> np.ndarray:
    """Non-homogeneous Poisson arrivals, rate base*(1 + depth*sin(2*pi*t/period)),
    by Lewis-Shedler thinning against the peak rate base*(1+depth)."""
    lam_max = base * (1.0 + depth)
    out = np.empty(n, dtype=np.float64)
    t = 0.0
    k = 0
    while k < n:
        m = 2 * (n - k) + 64
        gaps = rng.exponential(1.0 / lam_max, m)
        u = rng.random(m)
        for gap, uu in zip(gaps, u):
            t += gap
            lam = base * (1.0 + depth * math.sin(2.0 * math.pi * t / period))
            if uu * lam_max <= lam:
                out[k] = t
                k += 1
                if k == n:
                    break
    return out


def make_trace(name: str, seed: int, W: int, R: int, Q: int, kv_capacity: int, model: Model,
               in_dist=(5.5, 1.0, 16, 2048), out_dist=(5.0, 0.8, 8, 1024),
               rate: Optional[float] = None, diurnal: Optional[tuple] = None,
               heartbeat_every: int = 0, R_per_worker: Optional[np.ndarray] = None) -> Trace:
    """Generic trace builder.  ``R_per_worker`` (optional) gives ragged resident
    counts; otherwise every worker holds R residents."""
    rng = np.random.default_rng(seed)
    if R_per_worker is None:
        counts = np.full(W, R, dtype=np.int64)
    else:
        counts = np.asarray(R_per_worker, dtype=np.int64)
        assert counts.shape == (W,)
    n_res = int(counts.sum())
    offsets = np.zeros(W + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    res_l_in = _lengths(rng, *in_dist, n_res)
    res_l_pred = _lengths(rng, *out_dist, n_res)
    res_g = rng.integers(0, res_l_pred.astype(np.int64)).astype(np.int32) if n_res else np.zeros(0, np.int32)
    q_l_in = _lengths(rng, *in_dist, Q)
    q_l_pred = _lengths(rng, *out_dist, Q)
    arrivals = None
    if rate is not None:
        if diurnal is not None:
            arrivals = _thinned_arrivals(rng, Q, rate, diurnal[0], diurnal[1])
        else:
            arrivals = _poisson_arrivals(rng, Q, rate)
    return Trace(name=name, seed=seed, model=model,
                 kv_capacity=np.full(W, kv_capacity, dtype=np.int64),
                 res_offsets=offsets, res_l_in=res_l_in, res_l_pred=res_l_pred,
                 res_generated=res_g, q_l_in=q_l_in, q_l_pred=q_l_pred,
                 arrivals=arrivals, heartbeat_every=heartbeat_every)


def scenario_index(n_workers: int, gpus: int) -> int:
    """Canonical index of a sweep scenario: 4*(W/16 - 1) + log2(gpus)."""
    return 4 * (n_workers // 16 - 1) + int(round(math.log2(gpus)))


def make_sweep(name: str, seed: int, Q: int, worker_counts, gpu_counts, base_capacity: int,
               model: Model, in_dist, out_dist, rate: Optional[float]) -> SweepTrace:
    rng = np.random.default_rng(seed)
    # Same draw order as make_trace; scenarios start with no residents.
    q_l_in = _lengths(rng, *in_dist, Q)
    q_l_pred = _lengths(rng, *out_dist, Q)
    arrivals = _poisson_arrivals(rng, Q, rate) if rate is not None else None
    scen = []
    for W in worker_counts:
        for g in gpu_counts:
            scen.append(Scenario(n_workers=int(W), gpus_per_worker=int(g),
                                 kv_capacity=int(base_capacity * g), model=model.per_gpu_scaled(g)))
    return SweepTrace(name=name, seed=seed, scenarios=scen, q_l_in=q_l_in, q_l_pred=q_l_pred,
                      arrivals=arrivals)


SHORT_IN = (5.5, 1.0, 16, 2048)
SHORT_OUT = (5.0, 0.8, 8, 1024)
MID_IN = (6.5, 1.2, 16, 8192)
MID_OUT = (5.5, 1.0, 8, 2048)
LONG_IN = (8.0, 1.0, 256, 32768)
LONG_OUT = (6.0, 1.0, 16, 4096)

# The five workloads of the evaluator (name -> description).
CONFIGS = {
    "tiny": "W=8, M=16384, R=32, Q=256 @20/s, short lengths, base model",
    "medium": "W=64, M=65536, R=128, Q=4096 @200/s, short lengths, base model x0.7",
    "large": "W=512, M=262144, R=512, Q=65536 @2000/s +-50% diurnal (600 s), mid lengths",
    "sweep": "256 scenarios W in {16..1024 step 16} x gpus in {1,2,4,8}, empty start, "
             "Q=16384 @500/s mid lengths, M=65536*gpus, slopes / (0.8*gpus)",
    "long": "W=2048, M=1048576, R=1024, Q=131072, long lengths, heartbeat every 100, "
            "TTFT 4 s, decode 0.08 s",
    "rebalance": "Algorithm 2: 256 problems of W=128 workers x 64 ongoing requests and 1024 new ones, "
                 "mid output lengths, prediction error exp(0.5 N(0,1)), base model (rho = 500 tokens)",
}


def heartbeats_from_arrivals(arrivals: np.ndarray, period: float) -> np.ndarray:
    """Decode iterations (one per `period` seconds) that run before each query:
    the number of period boundaries crossed since the previous arrival (since
    time 0 for the first query)."""
    k = np.floor(np.asarray(arrivals, dtype=np.float64) / period).astype(np.int64)
    out = np.diff(np.concatenate([[0], k]))
    if (out < 0).any():
        raise ValueError("arrivals must not decrease")
    return out.astype(np.int32)


def with_decode_history(trace: Trace, seed: int, lo: float = 0.2, hi: float = 0.9) -> Trace:
    """A copy of `trace` whose residents carry a decode time so far: each one's
    g generated tokens took g * T_dec * f seconds, f uniform in [lo, hi) (seeded),
    so some residents are ahead of the per-token decode target and some behind."""
    rng = np.random.default_rng(seed)
    f = rng.uniform(lo, hi, trace.n_resident)
    t_dec = trace.res_generated.astype(np.float64) * trace.model.decode_slo * f
    return dataclasses.replace(trace, name=trace.name + "+history", res_t_dec=t_dec)


@dataclasses.dataclass
class RebalanceBatch:
    """P independent re-balancing problems (Algorithm 2): per problem, W workers
    with R ongoing requests each and n_new new requests of one heartbeat, in
    CSR form (worker indices local to the problem)."""
    name: str
    models: List[Model]
    n_workers: np.ndarray     # int32 [P]
    old_offsets: np.ndarray   # int64 [P+1]
    old_worker: np.ndarray    # int32 [n_old]
    old_l_pred: np.ndarray
    old_l_out: np.ndarray     # tokens generated so far
    old_l_real: np.ndarray    # real output length where it is known (finished), else max(l_out, l_pred)
    old_l_repred: np.ndarray  # re-prediction for a request decoding past its prediction
    new_offsets: np.ndarray   # int64 [P+1]
    new_l_pred: np.ndarray    # int32 [n_new]
    new_worker: np.ndarray    # int32 [n_new], -1 = not placed

    @property
    def P(self) -> int:
        return len(self.n_workers)

    def problem(self, p: int):
        """Problem p's arrays (views)."""
        o0, o1 = int(self.old_offsets[p]), int(self.old_offsets[p + 1])
        n0, n1 = int(self.new_offsets[p]), int(self.new_offsets[p + 1])
        return (int(self.n_workers[p]), self.models[p], self.old_worker[o0:o1], self.old_l_pred[o0:o1],
                self.old_l_out[o0:o1], self.old_l_real[o0:o1], self.old_l_repred[o0:o1],
                self.new_l_pred[n0:n1], self.new_worker[n0:n1])


def make_rebalance(name: str, seed: int, P: int, W, R, n_new, model: Model = None, out_dist=None,
                   sigma_err: float = 0.5, unplaced: float = 0.02) -> RebalanceBatch:
    """Synthetic prediction errors: a request's real output length is its
    predicted one times exp(sigma_err * N(0, 1)) (unbiased in the log, as the
    paper's predictor is unbiased), clipped to [1, 4 * the length range's top].
    Each ongoing request has run t ~ integers(0, max(l_pred, l_real) + 1)
    iterations: it generated l_out = min(t, l_real) tokens and has finished
    when t >= l_real; a finished request reports its real length, a running
    one max(l_out, l_pred) (its real length is not known yet).  The
    re-prediction is the mean real length given that it exceeds the
    prediction, l_pred * 2 exp(sigma^2 / 2) Phi(sigma), rounded.  New requests
    draw a predicted length and a worker uniformly, a fraction `unplaced` none.
    W, R, n_new: an int, or a per-problem sequence.
    Draw order: per problem, ongoing l_pred, error factors, progress t, then
    new l_pred, new workers, unplaced flags."""
    model = model or BASE_MODEL
    mu, sg, lo, hi = out_dist or MID_OUT
    rng = np.random.default_rng(seed)
    per = lambda v: [int(x) for x in (v if hasattr(v, "__len__") else [v] * P)]
    Ws, Rs, Ns = per(W), per(R), per(n_new)
    boost = 2.0 * math.exp(sigma_err * sigma_err / 2.0) * 0.5 * (1.0 + math.erf(sigma_err / math.sqrt(2.0)))
    cols = {k: [] for k in ("ow", "lp", "lo", "lr", "rp", "nl", "nw")}
    for p in range(P):
        n = Ws[p] * Rs[p]
        lp = _lengths(rng, mu, sg, lo, hi, n).astype(np.int64)
        real = np.clip(np.rint(lp * np.exp(sigma_err * rng.standard_normal(n))), 1, 4 * hi).astype(np.int64)
        t = rng.integers(0, np.maximum(lp, real) + 1)
        lout = np.minimum(t, real)
        rep_real = np.where(t >= real, real, np.maximum(lout, lp))
        cols["ow"].append(np.repeat(np.arange(Ws[p]), Rs[p]))
        cols["lp"].append(lp)
        cols["lo"].append(lout)
        cols["lr"].append(rep_real)
        cols["rp"].append(np.rint(lp * boost).astype(np.int64))
        cols["nl"].append(_lengths(rng, mu, sg, lo, hi, Ns[p]))
        w = rng.integers(0, Ws[p], Ns[p])
        cols["nw"].append(np.where(rng.random(Ns[p]) < unplaced, -1, w))
    cat = lambda k: np.concatenate(cols[k]).astype(np.int32) if cols[k] else np.zeros(0, np.int32)
    off = lambda ns: np.concatenate([[0], np.cumsum(ns)]).astype(np.int64)
    return RebalanceBatch(name, [model] * P, np.array(Ws, np.int32), off([w * r for w, r in zip(Ws, Rs)]),
                          cat("ow"), cat("lp"), cat("lo"), cat("lr"), cat("rp"), off(Ns), cat("nl"), cat("nw"))


def make_config(name: str):
    """Build one of the five named workloads (see ``CONFIGS``)."""
    if name == "tiny":
        return make_trace("tiny", 0, W=8, R=32, Q=256, kv_capacity=16384, model=BASE_MODEL,
                          in_dist=SHORT_IN, out_dist=SHORT_OUT, rate=20.0)
    if name == "medium":
        return make_trace("medium", 1, W=64, R=128, Q=4096, kv_capacity=65536,
                          model=BASE_MODEL.scaled(0.7), in_dist=SHORT_IN, out_dist=SHORT_OUT,
                          rate=200.0)
    if name == "large":
        return make_trace("large", 2, W=512, R=512, Q=65536, kv_capacity=262144, model=BASE_MODEL,
                          in_dist=MID_IN, out_dist=MID_OUT, rate=2000.0, diurnal=(0.5, 600.0))
    if name == "sweep":
        return make_sweep("sweep", 3, Q=16384, worker_counts=range(16, 1025, 16),
                          gpu_counts=(1, 2, 4, 8), base_capacity=65536, model=BASE_MODEL,
                          in_dist=MID_IN, out_dist=MID_OUT, rate=500.0)
    if name == "rebalance":
        return make_rebalance("rebalance", 5, P=256, W=128, R=64, n_new=1024)
    if name == "long":
        model = dataclasses.replace(BASE_MODEL, ttft_slo=4.0, decode_slo=0.08)
        return make_trace("long", 4, W=2048, R=1024, Q=131072, kv_capacity=1048576, model=model,
                          in_dist=LONG_IN, out_dist=LONG_OUT, rate=None, heartbeat_every=100)
    raise KeyError(name)
