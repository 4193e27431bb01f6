"""Worker-count prediction over arrival rates (Sec. 4.4, Eq. 7), on top of the
scaling sweep.

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
