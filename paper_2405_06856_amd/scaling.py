"""Worker-count prediction over arrival rates (Sec. 4.4, Eq. 7), on top of the
scaling sweep; the worker configuration (Sec. 4.1, Eq. 5-6) and the group
count of distributed scheduling (App. A, Eq. 8).

For an arrival rate r the sweep runs each cluster scenario with a heartbeat
after every H = r * T_dec processed queries: one heartbeat is one decode
iteration, which takes T_dec at the ATGT limit, so H queries arrive per
iteration (rates with r * T_dec < 1 are taken as one query per iteration).
The smallest cluster that places the whole stream without a rejection is the
worker count the rate needs.  Eq. 7 models that count as ceil(k5 * r + c5)
above a lower rate bound R; ``fit_eq7`` fits k5 and c5 by least squares.
Host arithmetic only: the placements come from the library's kernels.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Sequence

import numpy as np


def heartbeat_period(rate: float, decode_slo: float) -> int:
    """Queries per decode iteration at arrival rate `rate` (at least 1)."""
    return max(1, int(round(rate * decode_slo)))


@dataclass
class RatePoint:
    rate: float
    heartbeat_every: int
    workers: int          # smallest feasible worker count (None: no scenario feasible)
    gpus: int             # its total GPU count
    scenario: int         # its index in the sweep


def min_cluster_per_rate(ev, sweep, rates: Sequence[float], gpus_per_worker: int) -> List[RatePoint]:
    """For each rate, the fewest workers (of `gpus_per_worker` GPUs each: the
    worker configuration is fixed, Sec. 4.1) that place the sweep's stream with
    no rejection.  `ev` is an aladdin.Evaluator, `sweep` a workloads.SweepTrace."""
    idx = [i for i, s in enumerate(sweep.scenarios) if s.gpus_per_worker == gpus_per_worker]
    if not idx:
        raise ValueError("no scenario with %d GPUs per worker" % gpus_per_worker)
    scen = [sweep.scenarios[i] for i in idx]
    out = []
    for r in rates:
        H = heartbeat_period(r, scen[0].model.decode_slo)
        rej, _, _ = ev.sweep(scen, sweep.q_l_in, sweep.q_l_pred, heartbeat_every=H)
        ok = [k for k in range(len(scen)) if int(rej[k]) == 0]
        if ok:
            k = min(ok, key=lambda k: (scen[k].n_workers, k))
            out.append(RatePoint(float(r), H, scen[k].n_workers, scen[k].n_workers * gpus_per_worker, idx[k]))
        else:
            out.append(RatePoint(float(r), H, None, None, -1))
    return out


def fit_eq7(rates: Sequence[float], workers: Sequence[int]):
    """Least-squares k5, c5 of workers ~ k5 * rate + c5 (Eq. 7 before the ceiling)."""
    r = np.asarray(rates, dtype=np.float64)
    w = np.asarray(workers, dtype=np.float64)
    if r.size < 2 or np.ptp(r) == 0.0:
        raise ValueError("need at least two distinct rates")
    A = np.stack([r, np.ones_like(r)], axis=1)
    (k5, c5), *_ = np.linalg.lstsq(A, w, rcond=None)
    return float(k5), float(c5)


def predict_workers(k5: float, c5: float, rate: float) -> int:
    """Eq. 7: the smallest integer not below k5 * rate + c5."""
    return int(math.ceil(k5 * rate + c5))


# --------------------------------------------------------------------------- worker configuration
@dataclass
class WorkerConfig:
    gpus: int           # N_g
    kv_capacity: float  # M = N_g m_gpu - m_model
    iter_time: float    # t_compute + t_comm at the batch M / m_r
    batch_slo: int      # B: the largest batch meeting the ATGT SLO
    t_max: float        # Eq. 6, per GPU


def worker_throughput(n_gpus: int, m_gpu: float, m_model: float, m_r: float, k4: float, c4: float,
                      k_comm: float, decode_slo: float, c3: float, c2: float, k2: float, l_ave: float) -> WorkerConfig:
    """Eq. 6 for a tensor-parallel worker of n_gpus GPUs:
        T_max = min(M / (N_g m_r (t_compute + t_comm)), B / (N_g T_decode))
    with M = N_g m_gpu - m_model (Sec. 4.1), t_compute = k4 / N_g + c4 (Eq. 5),
    t_comm = k_comm (N_g - 1) / N_g (the all-reduce share the paper scales the
    communication time by), and B the largest batch whose decode iteration
    (Eq. 3 at average context l_ave) stays within T_decode:
    (k2 l_ave + c2) B + c3 <= T_decode.  Memory in any unit shared by m_gpu,
    m_model and m_r; a worker whose model does not fit has T_max = 0."""
    g = int(n_gpus)
    M = g * m_gpu - m_model
    t_iter = (k4 / g + c4) + k_comm * (g - 1) / g
    B = max(0, int(math.floor((decode_slo - c3) / (k2 * l_ave + c2))))
    if M <= 0:
        return WorkerConfig(g, M, t_iter, B, 0.0)
    t_max = min(M / (g * m_r * t_iter), B / (g * decode_slo))
    return WorkerConfig(g, M, t_iter, B, t_max)


def best_worker_config(candidates: Sequence[int], **kw) -> WorkerConfig:
    """The GPU count per worker with the largest per-GPU throughput (ties: fewer GPUs)."""
    best = None
    for g in sorted(candidates):
        w = worker_throughput(g, **kw)
        if best is None or w.t_max > best.t_max:
            best = w
    return best


# --------------------------------------------------------------------------- App. A group count
def group_count(rate: float, workers: int, err: float, rate_limit: float) -> int:
    """Eq. 8: N_group groups of rates r_i = rate / N_group with 1 / (2 err) <=
    (workers per group) and r_i <= r(T_s) = rate_limit (the rate one scheduler
    places within the scheduling latency limit).  The fewest groups meeting the
    rate limit, as long as every group keeps at least ceil(1 / (2 err))
    workers; None when both cannot hold."""
    if rate <= 0 or workers < 1 or not (0 < err) or rate_limit <= 0:
        raise ValueError("need rate > 0, workers >= 1, err > 0, rate_limit > 0")
    need = max(1, int(math.ceil(rate / rate_limit - 1e-12)))
    per_group = int(math.ceil(1.0 / (2.0 * err) - 1e-12))
    most = workers // per_group
    return need if need <= most else None
