"""Brute-force placement written straight from the paper's definitions.

Used only to pin the oracle on tiny inputs.  It is deliberately different in
form from the oracle:

* KV demand uses the explicit footprint vector of constraint (e) (Sec. 4.2):
  a request contributes [kv(l_in+g), kv(l_in+g+1), ..., kv(l_in+l_pred), 0, ...]
  from the current iteration on, with kv(x) = x (Eq. 1, h=1, j=0); the worker
  demand is the element-wise sum and must stay <= M at every element.
* The decode constraint (b) is checked in the division form of Eq. 4,
  sum(l_in + gamma*l_out) <= theta * (T_dec - c3 - c2*b) / k2, in exact
  rational arithmetic on the fp64 coefficient values.
* The TTFT constraint (c) is Eq. 2 (plus the quadratic term) in exact rationals.
* Algorithm 1's ranking uses capacity_norm = hypot(B, sum(D)) in fp64, sorted
  large to small with ties to the lower index, then the first feasible worker.
* A heartbeat drops the first element of every footprint vector (one decode
  iteration has run); empty vectors leave.  Heartbeats come after every H
  processed queries, or hb_before[q] of them before query q.
* Split-phase serving: a decode worker (infinite TTFT SLO) checks only (b) and (e).
* Constraint (d), with decode history: every request keeps its generated-token
  count g and decode time t_dec literally (exact rationals); a heartbeat's
  iteration time is Eq. 3, (c3 + c2*b) + k2*sum(context), over the batch before
  the iteration, and every request in the batch gains one token and that time.
  A request placed in the current heartbeat has not decoded yet and is not
  ongoing.  Prefill time (as in (c)) <= theta * min over ongoing (T_dec*g - t_dec).
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import List


class Req:
    __slots__ = ("l_in", "l_pred", "g", "new", "t_dec")

    def __init__(self, l_in, l_pred, g=0, new=False, t_dec=0.0):
        self.l_in, self.l_pred, self.g, self.new = int(l_in), int(l_pred), int(g), bool(new)
        self.t_dec = Fraction(t_dec)

    def footprint(self) -> List[int]:
        return [self.l_in + k for k in range(self.g, self.l_pred + 1)]


def demand_peak(vectors: List[List[int]]) -> int:
    K = max((len(v) for v in vectors), default=0)
    tot = [0] * K
    for v in vectors:
        for k, x in enumerate(v):
            tot[k] += x
    return max(tot, default=0)


class BruteWorker:
    def __init__(self, M, reqs=()):
        self.M = int(M)
        self.vecs = [r.footprint() for r in reqs]
        # per request: (context-now, remaining, l_in, is_new, generated, decode time)
        self.meta = [[r.l_in + r.g, r.l_pred - r.g, r.l_in, False, r.g, r.t_dec] for r in reqs]

    def heartbeat(self, model=None):
        F = Fraction
        t_iter = F(0)
        if model is not None and self.meta:
            b = len(self.meta)
            t_iter = F(model.c3) + F(model.c2) * b + F(model.k2) * sum(F(m[0]) for m in self.meta)
        keep_v, keep_m = [], []
        for v, m in zip(self.vecs, self.meta):
            v = v[1:]
            if v:
                keep_v.append(v)
                keep_m.append([m[0] + 1, m[1] - 1, m[2], False, m[4] + 1, m[5] + t_iter])
        self.vecs, self.meta = keep_v, keep_m

    def batch(self):
        return len(self.vecs)


def brute_place(workers: List[BruteWorker], model, queries, heartbeat_every=0, use_d=False, hb_before=None,
                moves=()):
    """Per query a dict: chosen worker (-1 = none), n_feasible, per-worker KV
    peaks and a flag telling whether any exact latency margin is so small that
    fp64 rounding could decide it (those queries are not comparable bit for bit)."""
    gamma = Fraction(model.gamma_num, 2 ** model.gamma_log2den)
    F = Fraction
    decode_only = math.isinf(model.ttft_slo)  # a decode worker of split-phase serving
    out = []
    since = 0
    placed = {}  # query -> worker, for the moves
    moves = sorted(moves, key=lambda m: m[0])

    def apply_moves(at):
        for m_at, j, y in moves:
            if m_at != at:
                continue
            x = placed[j]
            # the query's own request: new this window, nothing generated yet
            k = next(k for k, m in enumerate(workers[x].meta)
                     if m[3] and m[2] == queries[j][0] and m[1] == queries[j][1])
            workers[x].vecs.pop(k)
            workers[x].meta.pop(k)
            q = Req(queries[j][0], queries[j][1], 0, True)
            workers[y].vecs.append(q.footprint())
            workers[y].meta.append([q.l_in, q.l_pred, q.l_in, True, 0, Fraction(0)])
            placed[j] = y
            out[j]["worker"] = y

    for qi, (l_in, l_pred) in enumerate(queries):
        apply_moves(qi)
        for _ in range(hb_before[qi] if hb_before is not None else 0):
            for w in workers:
                w.heartbeat(model)
        q = Req(l_in, l_pred, 0, True)
        qv = q.footprint()
        feas, norms, peaks = [], [], []
        close = False
        for w in workers:
            b = w.batch() + 1
            peak = demand_peak(w.vecs + [qv])
            kv_ok = peak <= w.M
            # sum of (l_in + gamma * l_out) with l_out split into generated (counted
            # fully, it is already in the context) and remaining (weighted by gamma)
            sumD = sum(F(c) + gamma * F(r) for c, r, _, _, _, _ in w.meta) + F(l_in) + gamma * F(l_pred)
            ld = (F(model.decode_slo) - F(model.c3) - F(model.c2) * b) / F(model.k2)
            dec_ok = sumD <= F(model.theta) * ld
            lim = F(model.theta) * ld
            if abs(lim - sumD) <= F(1, 10 ** 9) * max(abs(lim), abs(sumD)):
                close = True
            if decode_only:
                # split-phase decode worker: the prefill ran elsewhere, only (b) and (e)
                feas.append(kv_ok and dec_ok)
                sumD_now = sum(F(c) + gamma * F(r) for c, r, _, _, _, _ in w.meta)
                norms.append(math.hypot(float(w.batch()), float(sumD_now)))
                peaks.append(peak)
                continue
            S1 = sum(F(li) for _, _, li, new, _, _ in w.meta if new) + F(l_in)
            S2 = sum(F(li) ** 2 for _, _, li, new, _, _ in w.meta if new) + F(l_in) ** 2
            ttft = F(model.c1) + F(model.k1) * S1 + F(model.k1q) * S2
            ttft_ok = ttft <= F(model.ttft_slo)
            if abs(F(model.ttft_slo) - ttft) <= F(1, 10 ** 9) * max(abs(ttft), abs(F(model.ttft_slo))):
                close = True
            pre_ok = True
            ongoing = [F(model.decode_slo) * g - td for _, _, _, new, g, td in w.meta if not new]
            if use_d and ongoing:
                dl = F(model.theta) * min(ongoing)
                pre_ok = ttft <= dl
                if abs(ttft - dl) <= F(1, 10 ** 9) * max(abs(ttft), abs(dl)):
                    close = True
            feas.append(kv_ok and dec_ok and ttft_ok and pre_ok)
            sumD_now = sum(F(c) + gamma * F(r) for c, r, _, _, _, _ in w.meta)
            norms.append(math.hypot(float(w.batch()), float(sumD_now)))
            peaks.append(peak)
        order = sorted(range(len(workers)), key=lambda i: (-norms[i], i))
        chosen = next((i for i in order if feas[i]), -1)
        if chosen >= 0:
            w = workers[chosen]
            w.vecs.append(qv)
            w.meta.append([l_in, l_pred, l_in, True, 0, F(0)])
            placed[qi] = chosen
        out.append({"worker": chosen, "n_feasible": sum(feas), "peaks": peaks, "norms": norms,
                    "close": close})
        if heartbeat_every:
            since += 1
            if since == heartbeat_every:
                for w in workers:
                    w.heartbeat(model)
                since = 0
    apply_moves(len(queries))
    return out
