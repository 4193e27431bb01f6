"""Pins of the CPU oracle against the paper and against mathematics (no GPU).

Each test checks the oracle against something other than itself: a value the
paper prints, a closed form, the explicit footprint-vector definition of
constraint (e), Eq. 3/Eq. 4 evaluated in exact rationals, or Algorithm 1 run
literally with a floating-point capacity_norm.
"""
from __future__ import annotations

import dataclasses
import math
import json
import os

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl
from tests.brute import BruteWorker, Req, brute_place, demand_peak

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

# A model whose latency constraints never bind (only constraint (e) matters).
FREE = wl.Model(c1=0.0, k1=0.0, k1q=0.0, c3=0.0, c2=0.0, k2=1e-12, ttft_slo=1e9, decode_slo=1e9)


def run(W, M, residents, model, queries, H=0, check=True, t_dec=None):
    """residents: list per worker of (l_in, l_pred, g); t_dec: list per worker of
    the residents' decode times (constraint (d) on), or None."""
    off = np.zeros(W + 1, np.int64)
    rl, rp, rg, td = [], [], [], []
    for i in range(W):
        for k, (a, b, g) in enumerate(residents[i]):
            rl.append(a); rp.append(b); rg.append(g)
            if t_dec is not None:
                td.append(t_dec[i][k])
        off[i + 1] = len(rl)
    q = np.array(queries, np.int32).reshape(-1, 2)
    return ref.place(W, np.full(W, M, np.int64) if np.isscalar(M) else np.asarray(M, np.int64), off,
                     np.array(rl, np.int32), np.array(rp, np.int32), np.array(rg, np.int32), model,
                     q[:, 0], q[:, 1], heartbeat_every=H, check=check,
                     res_t_dec=None if t_dec is None else np.array(td, np.float64))


# --------------------------------------------------------------------------- paper's worked example
def test_fig3_worked_example():
    fx = json.load(open(os.path.join(GOLDEN, "fig3_example.json")))
    pr, dv = fx["printed"], fx["derived"]
    LP, LO = tuple(dv["long_prompt"]), tuple(dv["long_output"])
    kinds = {"long_prompt": LP, "long_output": LO}
    queries = [kinds[k] for k in pr["arrival_order"]]
    M = pr["kv_capacity"]
    # JSQ as described: prompts together, outputs together
    assert ref.kv_peak([LP[0], LP[0]], [LP[1], LP[1]]) == pr["jsq_peak_each_worker"]
    assert ref.kv_peak([LO[0], LO[0]], [LO[1], LO[1]]) == pr["jsq_peak_each_worker"]
    assert pr["jsq_peak_each_worker"] > M
    # Algorithm 1 with only the KV constraint binding reaches the printed best placement
    res = run(pr["n_workers"], M, [[], []], FREE, queries)
    assert list(res.worker) == [0, 0, 1, 1]
    assert list(res.peak) == [pr["best_peak_each_worker"]] * 2
    assert all(p <= M for p in res.peak)


# --------------------------------------------------------------------------- KV peak
def test_peak_equals_footprint_vector_sum():
    rng = np.random.default_rng(11)
    for _ in range(3000):
        n = int(rng.integers(0, 7))
        reqs = [Req(rng.integers(1, 9), rng.integers(1, 9)) for _ in range(n)]
        for r in reqs:
            r.g = int(rng.integers(0, r.l_pred))
        want = demand_peak([r.footprint() for r in reqs])
        got = ref.kv_peak([r.l_in + r.g for r in reqs], [r.l_pred - r.g for r in reqs])
        assert got == want


def test_lone_request_peak_closed_form():
    # a lone new request peaks at its last iteration: l_in + l_pred
    for lin, lp in [(1, 1), (4, 1), (1, 4), (300, 17), (32768, 4096)]:
        res = run(1, 10 ** 9, [[]], FREE, [(lin, lp)])
        assert res.kv_peak_chosen[0] == lin + lp
        assert res.peak[0] == lin + lp


def test_peak_ties_and_exact_capacity():
    # equal remaining lengths: all alive until the common end point
    assert ref.kv_peak([5, 7, 9], [3, 3, 3]) == (5 + 3) + (7 + 3) + (9 + 3)
    # capacity exactly reached is allowed (<= M), one more token is not
    res = run(1, 10, [[]], FREE, [(4, 1), (1, 4)])      # peak 7 after both
    assert list(res.worker) == [0, 0]
    res = run(1, 6, [[]], FREE, [(4, 1), (1, 4)])
    assert list(res.worker) == [0, -1]
    assert res.kv_excess_min[1] == 7 - 6


# --------------------------------------------------------------------------- whole placement vs brute force
def _random_model(rng):
    # coefficients chosen so that each constraint binds for some of the tiny cases
    return wl.Model(c1=float(rng.uniform(0.0, 0.2)), k1=float(rng.uniform(0.005, 0.05)),
                    k1q=float(rng.choice([0.0, rng.uniform(0.0, 0.005)])),
                    c3=float(rng.uniform(0.0, 0.1)), c2=float(rng.uniform(0.0, 0.05)),
                    k2=float(rng.uniform(0.002, 0.02)), ttft_slo=float(rng.uniform(0.3, 1.5)),
                    decode_slo=float(rng.uniform(0.2, 0.6)), theta=float(rng.choice([1.0, 0.75, 0.5])),
                    gamma_num=int(rng.integers(0, 3)), gamma_log2den=1)


@pytest.mark.parametrize("H", [0, 1, 3])
def test_placement_matches_bruteforce(H):
    rng = np.random.default_rng(100 + H)
    compared = 0
    for case in range(400):
        W = int(rng.integers(1, 5))
        model = _random_model(rng)
        residents = []
        for _ in range(W):
            rs = []
            for _ in range(int(rng.integers(0, 6))):
                lp = int(rng.integers(1, 9))
                rs.append((int(rng.integers(1, 9)), lp, int(rng.integers(0, lp))))
            residents.append(rs)
        M = [int(rng.integers(8, 60)) for _ in range(W)]
        queries = [(int(rng.integers(1, 9)), int(rng.integers(1, 9))) for _ in range(int(rng.integers(1, 12)))]
        res = run(W, M, residents, model, queries, H=H)
        bw = [BruteWorker(M[i], [Req(a, b, g) for (a, b, g) in residents[i]]) for i in range(W)]
        want = brute_place(bw, model, queries, heartbeat_every=H)
        for k, wq in enumerate(want):
            if wq["close"]:
                break  # fp64 rounding may legitimately decide from here on
            norms = sorted(wq["norms"])
            if any(0 < b - a <= 1e-12 * b for a, b in zip(norms, norms[1:])):
                break
            assert res.worker[k] == wq["worker"], (case, k)
            assert res.n_feasible[k] == wq["n_feasible"], (case, k)
            assert res.kv_excess_min[k] == min(p - m for p, m in zip(wq["peaks"], M)), (case, k)
            if wq["worker"] >= 0:
                assert res.kv_peak_chosen[k] == wq["peaks"][wq["worker"]]
            compared += 1
    assert compared > 1500


def _hb_from_period(Q, H):
    hb = np.zeros(Q, np.int32)
    if H > 0:
        hb[H::H] = 1
    return hb


@pytest.mark.parametrize("H", [1, 7, 100])
def test_heartbeats_per_query_equal_a_period(H):
    """hb_before = 1 at every H-th query is the same stream as heartbeat_every = H
    (whose heartbeat after the last query, when H divides Q, has no query to
    precede: the final states are compared only when it does not happen)."""
    t = wl.with_decode_history(wl.make_trace("hbq", 41, W=10, R=12, Q=703, kv_capacity=20000, model=wl.BASE_MODEL), 3)
    a = ref.place_trace(t, heartbeat_every=H, check=True)
    b = ref.place_hb(t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated, t.model,
                     t.q_l_in, t.q_l_pred, _hb_from_period(t.n_queries, H), check=True, res_t_dec=t.res_t_dec)
    fields = ["worker", "n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min"]
    if t.n_queries % H:
        fields += ["B", "sum_c", "sum_r", "peak"]
    for f in fields:
        assert np.array_equal(getattr(a, f), getattr(b, f)), f
    assert np.array_equal(a.ttft_chosen, b.ttft_chosen) and np.array_equal(a.tdec_chosen, b.tdec_chosen)


@pytest.mark.parametrize("use_d", [False, True])
def test_heartbeats_per_query_match_bruteforce(use_d):
    """Arrival-time heartbeats: any number of decode iterations (bursts, idle
    gaps) before a query, against the brute force, with and without (d)."""
    rng = np.random.default_rng(700 + int(use_d))
    compared = 0
    for case in range(300):
        W = int(rng.integers(1, 5))
        model = _random_model(rng)
        model = dataclasses.replace(model, c1=float(rng.uniform(0.0, 0.02)), k1=float(rng.uniform(0.0, 0.004)),
                                    ttft_slo=1.0)
        residents, t_dec = [], []
        for _ in range(W):
            rs, ts = [], []
            for _ in range(int(rng.integers(0, 6))):
                lp = int(rng.integers(1, 9))
                g = int(rng.integers(0, lp))
                rs.append((int(rng.integers(1, 9)), lp, g))
                ts.append(float(rng.uniform(0.0, 2.0)) * g * model.decode_slo)
            residents.append(rs)
            t_dec.append(ts)
        M = [int(rng.integers(8, 60)) for _ in range(W)]
        Q = int(rng.integers(1, 12))
        queries = [(int(rng.integers(1, 9)), int(rng.integers(1, 9))) for _ in range(Q)]
        hbb = rng.choice([0, 0, 0, 1, 2, 5], Q).astype(np.int32)
        off = np.zeros(W + 1, np.int64)
        rl, rp, rg, td = [], [], [], []
        for i in range(W):
            for k, (a, b, g) in enumerate(residents[i]):
                rl.append(a); rp.append(b); rg.append(g); td.append(t_dec[i][k])
            off[i + 1] = len(rl)
        q = np.array(queries, np.int32).reshape(-1, 2)
        res = ref.place_hb(W, np.asarray(M, np.int64), off, np.array(rl, np.int32), np.array(rp, np.int32),
                           np.array(rg, np.int32), model, q[:, 0], q[:, 1], hbb, check=True,
                           res_t_dec=np.array(td, np.float64) if use_d else None)
        bw = [BruteWorker(M[i], [Req(a, b, g, t_dec=t_dec[i][k]) for k, (a, b, g) in enumerate(residents[i])])
              for i in range(W)]
        want = brute_place(bw, model, queries, use_d=use_d, hb_before=hbb)
        for k, wq in enumerate(want):
            if wq["close"]:
                break
            norms = sorted(wq["norms"])
            if any(0 < b - a <= 1e-12 * b for a, b in zip(norms, norms[1:])):
                break
            assert res.worker[k] == wq["worker"], (case, k)
            assert res.n_feasible[k] == wq["n_feasible"], (case, k)
            compared += 1
    assert compared > 1000


def _moves_case(rng, use_d):
    W = int(rng.integers(2, 5))
    model = _random_model(rng)
    model = dataclasses.replace(model, c1=float(rng.uniform(0.0, 0.02)), k1=float(rng.uniform(0.0, 0.004)),
                                ttft_slo=float(rng.uniform(0.02, 0.06)))
    residents, t_dec = [], []
    for _ in range(W):
        rs, ts = [], []
        for _ in range(int(rng.integers(0, 5))):
            lp = int(rng.integers(1, 9))
            g = int(rng.integers(0, lp))
            rs.append((int(rng.integers(1, 9)), lp, g))
            ts.append(float(rng.uniform(0.0, 2.0)) * g * model.decode_slo)
        residents.append(rs)
        t_dec.append(ts)
    M = [int(rng.integers(20, 80)) for _ in range(W)]
    Q = int(rng.integers(2, 14))
    queries = [(int(rng.integers(1, 9)), int(rng.integers(1, 9))) for _ in range(Q)]
    hbb = rng.choice([0, 0, 1, 2], Q).astype(np.int32)
    off = np.zeros(W + 1, np.int64)
    rl, rp, rg, td = [], [], [], []
    for i in range(W):
        for k, (a, b, g) in enumerate(residents[i]):
            rl.append(a); rp.append(b); rg.append(g); td.append(t_dec[i][k])
        off[i + 1] = len(rl)
    q = np.array(queries, np.int32).reshape(-1, 2)
    args = (W, np.asarray(M, np.int64), off, np.array(rl, np.int32), np.array(rp, np.int32), np.array(rg, np.int32),
            model, q[:, 0], q[:, 1])
    td = np.array(td, np.float64) if use_d else None
    # moves before query k (inside a window or at its end), each of a request
    # placed earlier in the same window, chosen on the run with the moves so far
    # (earlier placements do not depend on later moves)
    moves = []
    for k in range(1, Q + 1):
        if rng.random() < 0.35:
            start = max([i for i in range(k) if i == 0 or hbb[i] > 0])
            r = ref.place_moves(*args, moves, hb_before=hbb, res_t_dec=td)
            cand = [j for j in range(start, k) if r.worker[j] >= 0]
            if cand:
                j = int(rng.choice(cand))
                y = int(rng.choice([w for w in range(W) if w != r.worker[j]]))
                moves.append((k, j, y))
    return args, hbb, td, moves, residents, t_dec, M, queries, model


@pytest.mark.parametrize("use_d", [False, True])
def test_moves_match_bruteforce(use_d):
    """Moving a request placed in the current window is placing it on the new
    worker: against the brute force with the same moves applied literally."""
    rng = np.random.default_rng(800 + int(use_d))
    compared = moved = 0
    for case in range(250):
        args, hbb, td, moves, residents, t_dec, M, queries, model = _moves_case(rng, use_d)
        res = ref.place_moves(*args, moves, hb_before=hbb, res_t_dec=td)
        W = args[0]
        bw = [BruteWorker(M[i], [Req(a, b, g, t_dec=t_dec[i][k]) for k, (a, b, g) in enumerate(residents[i])])
              for i in range(W)]
        want = brute_place(bw, model, queries, use_d=use_d, hb_before=hbb, moves=moves)
        moved += len(moves)
        for k, wq in enumerate(want):
            if wq["close"]:
                break
            norms = sorted(wq["norms"])
            if any(0 < b - a <= 1e-12 * b for a, b in zip(norms, norms[1:])):
                break
            assert res.worker[k] == wq["worker"], (case, k, moves)
            assert res.n_feasible[k] == wq["n_feasible"], (case, k)
            compared += 1
    assert compared > 800 and moved > 150


def test_move_there_and_back_is_no_move():
    rng = np.random.default_rng(810)
    n = 0
    for case in range(60):
        args, hbb, td, moves, *_ = _moves_case(rng, False)
        if not moves:
            continue
        e, j, y = moves[0]
        base = ref.place_moves(*args, [], hb_before=hbb)
        if base.worker[j] < 0:
            continue
        x = int(base.worker[j])
        back = ref.place_moves(*args, [(e, j, y), (e, j, x)], hb_before=hbb)
        for f in ("worker", "n_feasible", "B", "sum_c", "sum_r", "peak", "S1", "S2"):
            assert np.array_equal(getattr(base, f), getattr(back, f)), f
        n += 1
    assert n > 20


def test_move_outside_the_window_is_rejected():
    # moves before query k come before the heartbeats that precede it: the
    # request of query 0 can move before query 1, not before query 2 once a
    # heartbeat preceded query 1
    args = (2, np.array([100, 100], np.int64), np.zeros(3, np.int64), np.zeros(0, np.int32), np.zeros(0, np.int32),
            np.zeros(0, np.int32), FREE, np.array([3, 3, 3], np.int32), np.array([4, 4, 4], np.int32))
    hb = np.array([0, 1, 0], np.int32)
    ok = ref.place_moves(*args, [(1, 0, 1)], hb_before=hb)
    assert ok.worker[0] == 1
    with pytest.raises(RuntimeError):
        ref.place_moves(*args, [(2, 0, 1)], hb_before=hb)


@pytest.mark.parametrize("H", [0, 2])
def test_decode_workers_match_bruteforce(H):
    """Split-phase decode workers (infinite TTFT SLO): only (b) and (e), even
    with a decode history; against the brute force, and the TTFT limit of the
    same model with a finite SLO does bind in this population."""
    rng = np.random.default_rng(500 + H)
    compared = differ = 0
    for case in range(300):
        W = int(rng.integers(1, 5))
        model = _random_model(rng)
        model = dataclasses.replace(model, c1=float(rng.uniform(0.0, 0.02)), k1=float(rng.uniform(0.0, 0.004)),
                                    ttft_slo=0.03)
        dmodel = dataclasses.replace(model, ttft_slo=math.inf)
        residents, t_dec = [], []
        for _ in range(W):
            rs, ts = [], []
            for _ in range(int(rng.integers(0, 6))):
                lp = int(rng.integers(1, 9))
                g = int(rng.integers(0, lp))
                rs.append((int(rng.integers(1, 9)), lp, g))
                ts.append(float(rng.uniform(0.0, 2.0)) * g * model.decode_slo)
            residents.append(rs)
            t_dec.append(ts)
        M = [int(rng.integers(8, 60)) for _ in range(W)]
        queries = [(int(rng.integers(1, 9)), int(rng.integers(1, 9))) for _ in range(int(rng.integers(1, 12)))]
        res = run(W, M, residents, dmodel, queries, H=H, t_dec=t_dec)
        fin = run(W, M, residents, model, queries, H=H)
        differ += int(not np.array_equal(res.worker, fin.worker))
        bw = [BruteWorker(M[i], [Req(a, b, g) for (a, b, g) in residents[i]]) for i in range(W)]
        want = brute_place(bw, dmodel, queries, heartbeat_every=H)
        for k, wq in enumerate(want):
            if wq["close"]:
                break
            norms = sorted(wq["norms"])
            if any(0 < b - a <= 1e-12 * b for a, b in zip(norms, norms[1:])):
                break
            assert res.worker[k] == wq["worker"], (case, k)
            assert res.n_feasible[k] == wq["n_feasible"], (case, k)
            assert res.near_tie[k] == 0 or wq["close"]
            compared += 1
    assert compared > 1000 and differ > 30


@pytest.mark.parametrize("H", [0, 1, 3])
def test_preemption_limit_matches_bruteforce(H):
    # constraint (d) against the literal per-request decode history (exact
    # rationals, tokens and decode time accumulated request by request)
    rng = np.random.default_rng(300 + H)
    compared = blocked = 0
    for case in range(400):
        W = int(rng.integers(1, 5))
        model = _random_model(rng)
        model = dataclasses.replace(model, c1=float(rng.uniform(0.0, 0.02)), k1=float(rng.uniform(0.0, 0.004)),
                                    ttft_slo=1.0)
        residents, t_dec = [], []
        for _ in range(W):
            rs, ts = [], []
            for _ in range(int(rng.integers(0, 5))):
                lp = int(rng.integers(1, 9))
                g = int(rng.integers(0, lp))
                rs.append((int(rng.integers(1, 9)), lp, g))
                ts.append(float(g * model.decode_slo * rng.uniform(0.0, 1.2)))
            residents.append(rs)
            t_dec.append(ts)
        M = [int(rng.integers(8, 60)) for _ in range(W)]
        queries = [(int(rng.integers(1, 9)), int(rng.integers(1, 9))) for _ in range(int(rng.integers(1, 12)))]
        res = run(W, M, residents, model, queries, H=H, t_dec=t_dec)
        free = run(W, M, residents, model, queries, H=H)
        bw = [BruteWorker(M[i], [Req(a, b, g, t_dec=t_dec[i][k]) for k, (a, b, g) in enumerate(residents[i])])
              for i in range(W)]
        want = brute_place(bw, model, queries, heartbeat_every=H, use_d=True)
        for k, wq in enumerate(want):
            if wq["close"]:
                break
            norms = sorted(wq["norms"])
            if any(0 < b - a <= 1e-12 * b for a, b in zip(norms, norms[1:])):
                break
            assert res.worker[k] == wq["worker"], (case, k)
            assert res.n_feasible[k] == wq["n_feasible"], (case, k)
            blocked += int(res.n_feasible[k] < free.n_feasible[k]) if k == 0 else 0
            compared += 1
    assert compared > 1200
    assert blocked > 20  # the limit does bind in this population


def test_preemption_limit_worked_example():
    # one worker, one resident (l_in 10, l_pred 100, 10 tokens in 0.5 s), heartbeat
    # after every query, T_dec = 0.05 s: its slack is 10 * 0.05 - 0.5 = 0 at first.
    m = wl.Model(c1=0.001, k1=1e-3, k1q=0.0, c3=0.01, c2=0.001, k2=1e-4, ttft_slo=10.0, decode_slo=0.05)
    q = [(30, 5), (30, 5), (40, 5), (40, 5)]
    res = run(1, 10 ** 6, [[(10, 100, 10)]], m, q, H=1, t_dec=[[0.5]])
    # q0: prefill 0.031 s > 1.0 * 0 -> rejected.  Heartbeat 1 (batch 1, context 20):
    # t_iter = (0.01 + 0.001) + 1e-4 * 20 = 0.013, slack 0.037.
    # q1: 0.031 <= 0.037 -> placed.  Heartbeat 2 (batch 2, context 21 + 30):
    # t_iter = 0.012 + 0.0051 = 0.0171; the resident's slack 0.0699, q1's (its
    # first iteration) 0.05 - 0.0171 = 0.0329.
    # q2: 0.041 > 0.0329 -> rejected.  Heartbeat 3 (batch 2, context 22 + 31):
    # t_iter = 0.012 + 0.0053 = 0.0173, q1's slack 0.0329 + 0.0327 = 0.0656.
    # q3: 0.041 <= 0.0656 -> placed (decode: 1e-4 * 142.5 <= 0.037).
    assert list(res.worker) == [-1, 0, -1, 0]
    # without the decode history only (b), (c), (e) apply and every query fits
    assert list(run(1, 10 ** 6, [[(10, 100, 10)]], m, q, H=1).worker) == [0] * 4


def test_preemption_limit_needs_an_ongoing_request():
    # zero slack (nothing generated yet) blocks every prefill on its worker; a
    # worker with no ongoing request has no such limit, also once it holds
    # requests placed in the current heartbeat
    m = wl.Model(c1=0.01, k1=1e-5, k1q=0.0, c3=0.0, c2=0.0, k2=1e-9, ttft_slo=10.0, decode_slo=0.05)
    q = [(50, 10)] * 5
    res = run(2, 10 ** 6, [[(100, 50, 0)], []], m, q, t_dec=[[0.0], []])
    assert list(res.worker) == [1] * 5
    res = run(2, 10 ** 6, [[(100, 50, 0)], []], m, q)  # no history: the fuller worker
    assert list(res.worker) == [0] * 5


def test_heartbeat_is_one_iteration_shift():
    # after one decode iteration the demand seen from the new "now" is the old
    # demand vector without its first element
    rng = np.random.default_rng(5)
    for _ in range(500):
        rs = []
        for _ in range(int(rng.integers(1, 7))):
            lp = int(rng.integers(1, 9))
            rs.append((int(rng.integers(1, 9)), lp, int(rng.integers(0, lp))))
        vecs = [Req(a, b, g).footprint() for (a, b, g) in rs]
        K = max(len(v) for v in vecs)
        tot = [sum(v[k] if k < len(v) else 0 for v in vecs) for k in range(K)]
        # one query that fits nowhere (capacity 0) just to trigger the heartbeat
        res = run(1, 0, [rs], FREE, [(1, 1)], H=1)
        assert res.worker[0] == -1
        assert res.peak[0] == max(tot[1:], default=0)
        assert res.B[0] == sum(1 for v in vecs if len(v) > 1)


def test_alg1_sorted_scan_equals_exhaustive_on_workloads():
    # check=True makes the oracle run Algorithm 1 literally (sort, first
    # feasible) beside the exhaustive argmax and fail on any difference
    for name in ("tiny", "medium"):
        t = wl.make_config(name)
        ref.place_trace(t, check=True)


def test_committed_placements_respect_every_constraint():
    t = wl.make_config("medium")
    r = ref.place_trace(t)
    m = t.model
    placed = r.worker >= 0
    assert placed.sum() > 0
    assert np.all(r.kv_peak_chosen[placed] <= t.kv_capacity[r.worker[placed]])
    assert np.all(r.ttft_chosen[placed] <= m.ttft_slo)
    # Eq. 3 form of the decode check at theta = 1: T_d <= T_dec
    assert m.theta == 1.0
    assert np.all(r.tdec_chosen[placed] <= m.decode_slo * (1 + 1e-12))
    # no worker ends above capacity unless its residents already put it there
    start = ref.place_trace(t, q_slice=slice(0, 0))
    assert np.all(r.peak <= np.maximum(t.kv_capacity, start.peak))
    assert np.all(r.peak[start.peak <= t.kv_capacity] <= t.kv_capacity[start.peak <= t.kv_capacity])


def test_rejected_queries_leave_state_unchanged():
    t = wl.make_config("tiny")
    r = ref.place_trace(t)
    keep = r.worker >= 0
    # dropping the rejected queries from the stream changes nothing
    r2 = ref.place(t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated,
                   t.model, t.q_l_in[keep], t.q_l_pred[keep])
    assert np.array_equal(r2.worker, r.worker[keep])
    for f in ("B", "sum_c", "sum_r", "peak", "S1", "S2"):
        assert np.array_equal(getattr(r2, f), getattr(r, f))


def test_monotone_within_heartbeat():
    # a commit never lowers B, sum(D), S1, S2 or the peak, so a worker that was
    # infeasible for a query stays infeasible: evaluating a query at the
    # initial state admits at least as many workers as at any later state
    t = wl.make_config("medium")
    at_start = ref.place_trace(t, no_commit=True)
    seq = ref.place_trace(t)
    assert np.all(seq.n_feasible <= at_start.n_feasible)
    assert np.all(seq.kv_excess_min >= at_start.kv_excess_min)


def test_decode_margin_exactly_zero_is_feasible_and_near_tie():
    # k2 * sumD == theta*((T_dec - c3) - c2*b) exactly: lhs <= rhs holds
    m = dataclasses.replace(FREE, c3=0.0, c2=0.0, k2=0.5, decode_slo=5.0, theta=1.0, gamma_num=0)
    # sumD = l_in = 10 -> lhs = 5.0 = rhs
    res = run(1, 10 ** 6, [[]], m, [(10, 3), (1, 1)])
    assert res.worker[0] == 0 and res.near_tie[0] == 1
    assert res.worker[1] == -1 and res.near_tie[1] == 0


def test_tdec_chosen_worked_example():
    # Eq. 3 for the chosen worker's batch with the query in it, computed by hand.
    # Coefficients are powers of two, so every fp64 step below is exact.
    # Resident (l_in 10, l_pred 6, generated 2): context c = 12, remaining r = 4,
    # D = c + r/2 = 14.  Query 1 (5, 8): D = 5 + 8/2 = 9, batch b = 2:
    #   T_d = (c3 + c2*2) + k2*(14 + 9) = (0.25 + 0.25) + 0.0625*23 = 1.9375.
    # Query 2 (1, 2): D = 1 + 1 = 2, batch b = 3:
    #   T_d = (0.25 + 0.375) + 0.0625*25 = 2.1875.
    # With gamma = 1 (D = c + r): D = 16, 13, 3:
    #   T_d = 0.5 + 0.0625*29 = 2.3125, then 0.625 + 0.0625*32 = 2.625.
    m = dataclasses.replace(FREE, c3=0.25, c2=0.125, k2=0.0625, decode_slo=4.0, theta=1.0)
    res = run(1, 10 ** 6, [[(10, 6, 2)]], m, [(5, 8), (1, 2)])
    assert list(res.worker) == [0, 0]
    assert list(res.tdec_chosen) == [1.9375, 2.1875]
    m1 = dataclasses.replace(m, gamma_num=2, gamma_log2den=1)
    res = run(1, 10 ** 6, [[(10, 6, 2)]], m1, [(5, 8), (1, 2)])
    assert list(res.tdec_chosen) == [2.3125, 2.625]
    # a rejected query reports 0
    tight = dataclasses.replace(m, decode_slo=1.6)  # (1.6 - 0.25) - 0.25 = 1.1 < 0.0625 * 23
    res = run(1, 10 ** 6, [[(10, 6, 2)]], tight, [(5, 8)])
    assert res.worker[0] == -1 and res.tdec_chosen[0] == 0.0


def test_ttft_margin_exactly_zero_is_feasible():
    m = dataclasses.replace(FREE, c1=0.5, k1=0.25, k1q=0.0, ttft_slo=3.0)
    res = run(2, 10 ** 6, [[], []], m, [(10, 2), (1, 1)])
    assert res.worker[0] == 0 and res.ttft_chosen[0] == 3.0 and res.near_tie[0] == 1
    # the first worker's prefill budget is used up; the second one takes it
    assert res.worker[1] == 1


def test_decode_near_tie_band_is_relative():
    # lhs = k2 * l_in = 0.1 against rhs = T_dec: a margin of 2e-10 is 2e-9
    # relative (outside the 1e-9 band, although it is below 1e-9 in absolute
    # terms); a margin of 5e-11 is 5e-10 relative (inside)
    import math
    for margin, flagged in ((2e-10, 0), (5e-11, 1)):
        m = dataclasses.replace(FREE, c3=0.0, c2=0.0, k2=0.01, decode_slo=0.1 + margin, theta=1.0, gamma_num=0)
        lhs, rhs = 0.01 * 10, 0.1 + margin
        assert (abs(lhs - rhs) <= 1e-9 * max(abs(lhs), abs(rhs))) == bool(flagged)
        assert math.isclose(abs(lhs - rhs), margin, rel_tol=1e-6)
        res = run(1, 10 ** 6, [[]], m, [(10, 3)])
        assert res.worker[0] == 0 and res.near_tie[0] == flagged, margin


def test_capacity_norm_is_taken_before_placement():
    # Algorithm 1 sorts the bins by ||(B, sum D)||_2 before placing the query.
    # Worker 0: one request c=4, r=3 (sum D = 4 + 3/2); worker 1: three requests
    # c=1, r=1 (sum D = 3 * 3/2).  Before placement worker 0 ranks first; with the
    # query's batch slot already counted (B + 1) worker 1 would.
    import math
    assert math.hypot(1, 5.5) > math.hypot(3, 4.5)
    assert math.hypot(1 + 1, 5.5) < math.hypot(3 + 1, 4.5)
    res = run(2, 10 ** 6, [[(4, 3, 0)], [(1, 1, 0)] * 3], FREE, [(1, 1)])
    assert res.worker[0] == 0


def test_capacity_norm_ranking_picks_fullest_feasible():
    # worker 1 holds more context -> ranked first; worker 0 chosen only when 1 is full
    res = run(2, [100, 30], [[(2, 2, 0)], [(10, 5, 0)]], FREE, [(3, 3), (3, 3), (3, 3)])
    assert list(res.worker) == [1, 1, 0]


# --------------------------------------------------------------------------- App. A grouped placement
def test_router_share_within_one_query():
    """App. A: group i receives the share N_i / N_w of the stream.  After every
    prefix of h queries each group's count is strictly within one query of
    h * N_i / N_w (exact rationals), for random group sizes."""
    from fractions import Fraction
    rng = np.random.default_rng(77)
    for _ in range(300):
        G = int(rng.integers(1, 10))
        sizes = [int(x) for x in rng.integers(1, 40, G)]
        Nw = sum(sizes)
        Q = int(rng.integers(1, 400))
        g = ref.route_groups(sizes, Q)
        cnt = [0] * G
        for h, x in enumerate(g.tolist(), start=1):
            cnt[x] += 1
            for i in range(G):
                assert abs(cnt[i] - Fraction(h * sizes[i], Nw)) < 1, (sizes, h, i)


def test_router_equal_sizes_is_round_robin_and_worked_example():
    # equal groups: query x goes to group x mod G
    for G in (1, 2, 5):
        assert ref.route_groups([7] * G, 23).tolist() == [x % G for x in range(23)]
    # sizes [1, 2] (shares 1/3, 2/3), worked by hand: query 1: both below their
    # quota, larger N_i / (a_i + 1) is group 1 (2/1 > 1/1); query 2: counts (0, 1),
    # 1/1 = 2/2, tie to group 0; query 3: group 0 has 1 >= 3 * 1/3 (at quota),
    # so group 1; then the counts (1, 2) are the shares of h = 3 and it repeats
    assert ref.route_groups([1, 2], 9).tolist() == [1, 0, 1] * 3


@pytest.mark.parametrize("H", [0, 7])
def test_grouped_placement_is_each_groups_algorithm1(H):
    """Grouped placement equals, per group, Algorithm 1 over that group's
    workers and the queries the router sends it, with the cluster's heartbeats
    (after every H queries of the whole stream) counted before each of them."""
    rng = np.random.default_rng(31 + H)
    for _ in range(12):
        G = int(rng.integers(1, 5))
        sizes = [int(x) for x in rng.integers(1, 6, G)]
        W = sum(sizes)
        t = wl.make_trace("g", int(rng.integers(0, 10 ** 6)), W=W, R=int(rng.integers(0, 4)),
                          Q=int(rng.integers(1, 120)), kv_capacity=int(rng.choice([3000, 20000])),
                          model=wl.BASE_MODEL, in_dist=wl.SHORT_IN, out_dist=wl.SHORT_OUT)
        M = np.broadcast_to(np.asarray(t.kv_capacity, np.int64), (W,))
        got = ref.place_grouped(W, M, t.res_offsets, t.res_l_in, t.res_l_pred,
                                t.res_generated, t.model, sizes, t.q_l_in, t.q_l_pred, heartbeat_every=H)
        route = ref.route_groups(sizes, t.n_queries)
        wb = 0
        for g, n in enumerate(sizes):
            idx = np.flatnonzero(route == g)
            o0, o1 = int(t.res_offsets[wb]), int(t.res_offsets[wb + n])
            hb = np.diff(np.r_[0, idx // H]) if H else np.zeros(len(idx), np.int64)
            want = ref.place_hb(n, M[wb:wb + n], t.res_offsets[wb:wb + n + 1] - o0,
                                t.res_l_in[o0:o1], t.res_l_pred[o0:o1], t.res_generated[o0:o1], t.model,
                                t.q_l_in[idx], t.q_l_pred[idx], hb, check=True)
            assert got.worker[idx].tolist() == np.where(want.worker >= 0, want.worker + wb, -1).tolist()
            for f in ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min", "ttft_chosen", "tdec_chosen"):
                assert np.array_equal(getattr(got, f)[idx], getattr(want, f)), f
            wb += n


def test_sweep_equals_independent_places():
    s = wl.make_sweep("mini", 9, Q=300, worker_counts=(2, 3, 5), gpu_counts=(1, 2), base_capacity=6000,
                      model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)
    rej, first, workers = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, n_threads=2)
    for i, sc in enumerate(s.scenarios):
        r = ref.place(sc.n_workers, np.full(sc.n_workers, sc.kv_capacity, np.int64), None, None, None, None,
                      sc.model, s.q_l_in, s.q_l_pred)
        assert np.array_equal(r.worker, workers[i])
        assert rej[i] == int((r.worker < 0).sum())
        neg = np.flatnonzero(r.worker < 0)
        assert first[i] == (int(neg[0]) if len(neg) else -1)
    assert rej.min() < rej.max()


def test_sweep_with_heartbeats_equals_independent_places():
    """Per-scenario heartbeat periods: each scenario is the single-stream
    placement with that period (and the periods do change the result)."""
    s = wl.make_sweep("mini", 10, Q=400, worker_counts=(2, 3, 6), gpu_counts=(1, 2), base_capacity=6000,
                      model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)
    H = np.array([0, 1, 3, 17, 60, 400], np.int32)
    rej, first, workers = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, n_threads=2,
                                    heartbeat_every=H)
    for i, sc in enumerate(s.scenarios):
        r = ref.place(sc.n_workers, np.full(sc.n_workers, sc.kv_capacity, np.int64), None, None, None, None,
                      sc.model, s.q_l_in, s.q_l_pred, heartbeat_every=int(H[i]))
        assert np.array_equal(r.worker, workers[i])
        assert rej[i] == int((r.worker < 0).sum())
    r0, _, _ = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred)
    assert not np.array_equal(r0, rej)


def test_threads_do_not_change_results():
    t = wl.make_config("medium")
    a = ref.place_trace(t, n_threads=1)
    b = ref.place_trace(t, n_threads=4)
    for f in ("worker", "n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min", "ttft_chosen",
              "tdec_chosen", "B", "peak"):
        assert np.array_equal(getattr(a, f), getattr(b, f))


def test_invalid_inputs_rejected():
    with pytest.raises(RuntimeError):
        run(1, 10, [[(3, 2, 2)]], FREE, [(1, 1)])   # g must be < l_pred
    with pytest.raises(RuntimeError):
        run(1, 10, [[]], FREE, [(0, 1)])            # l_in >= 1


# ---------------------------------------------------------------------------
# Algorithm 2 (Sec. 4.3): re-balancing against output-length prediction errors

def _rb_model(c2=1e-4, k2=2e-7):
    return wl.Model(c1=0.0, k1=0.0, k1q=0.0, c3=0.0, c2=c2, k2=k2, ttft_slo=1.0, decode_slo=1.0, theta=1.0,
                    gamma_num=1, gamma_log2den=1)


def _rho(m):
    """rho = c2 / k2 as an exact fraction (both are doubles)."""
    from fractions import Fraction
    return Fraction(m.c2) / Fraction(m.k2)


def _val(pair, rho):
    """The real value a + rho * b of a pair the oracle reports."""
    return pair[0] + rho * pair[1]


def test_rebalance_sign_is_exact():
    """Every decision of the search is the sign of a + rho * b for integers a, b;
    the oracle's sign matches exact rational arithmetic, also for pairs chosen
    next to a zero of the expression."""
    from fractions import Fraction
    rng = np.random.default_rng(5)
    models = [_rb_model(c2=c2, k2=k2) for c2, k2 in ((1e-4, 2e-7), (1001 * 2.0 ** -23, 2.0 ** -22), (0.0, 1e-6),
                                                     (3e-5, 7e-7), (1e-3, 1e-12))]
    for m in models:
        rho = _rho(m)
        for _ in range(400):
            a = int(rng.integers(-2 ** 59, 2 ** 59)) >> int(rng.integers(0, 55))
            b = int(rng.integers(-2 ** 40, 2 ** 40)) >> int(rng.integers(0, 38))
            if m.c2 > 0 and rng.random() < 0.5:
                b = -round(Fraction(a) / rho) + int(rng.integers(-1, 2))  # a + rho * b near 0
                if abs(b) >= 2 ** 59:
                    continue
            v = a + rho * b
            assert ref.rb_sign(a, b, m) == (v > 0) - (v < 0), (a, b, m.c2, m.k2)
    # an exact zero: rho = 500.5, a = -1001, b = 2
    assert ref.rb_sign(-1001, 2, models[1]) == 0
    assert ref.rb_sign(-1000, 2, models[1]) == 1 and ref.rb_sign(-1002, 2, models[1]) == -1


def test_rebalance_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "rebalance_example.json")))
    from fractions import Fraction
    for ex in g["examples"]:
        m = _rb_model(**ex["model"])
        assert _rho(m) == Fraction(*ex["rho"]), ex["name"]
        o, n = ex["ongoing"], ex["new"]
        r = ref.rebalance(ex["W"], m, o["worker"], o["l_pred"], o["l_out"], o["l_real"], o["l_repred"],
                          n["l_pred"], n["worker"])
        e = ex["expected"]
        assert r.worker.tolist() == e["worker"], ex["name"]
        assert r.le.tolist() == e["le"] and r.be.tolist() == e["be"], ex["name"]
        assert r.moves.tolist() == e["moves"], ex["name"]
        assert list(r.obj_before) == e["obj_before"] and list(r.obj_after) == e["obj_after"], ex["name"]


def test_rebalance_errors_closed_forms():
    """All under-estimated: l^e = sum of the re-predictions, b^e = count; all
    over-estimated: l^e = sum(l_real - l_pred), b^e = -count; predictions that
    were right (l_out <= l_pred <= l_real) leave no error."""
    m = _rb_model()
    rng = np.random.default_rng(3)
    n = 50
    lp = rng.integers(10, 100, n)
    rp = rng.integers(100, 300, n)
    r = ref.rebalance(2, m, np.zeros(n), lp, lp + 1, lp + 5, rp, [], [])
    assert r.le.tolist() == [int(rp.sum()), 0] and r.be.tolist() == [n, 0]
    lr = lp - rng.integers(1, 9, n)
    r = ref.rebalance(2, m, np.ones(n), lp, lr, lr, rp, [], [])
    assert r.le.tolist() == [0, int((lr - lp).sum())] and r.be.tolist() == [0, -n]
    r = ref.rebalance(2, m, np.ones(n), lp, lp, lp + rng.integers(0, 9, n), rp, [], [])
    assert r.le.tolist() == [0, 0] and r.be.tolist() == [0, 0] and r.obj_before == (0, 0)


@pytest.mark.parametrize("seed", range(6))
def test_rebalance_two_workers_closed_form(seed):
    """Two workers, every new request on worker 0 with one length: k moves give
    the objective f(k) = |c0 - k d| + |c1 + k d| (d = l_pred + rho), a convex
    function of k, so the greedy search stops at the smallest minimiser of f
    over 0 .. n (moving a request back would lead to f(k - 1) > f(k))."""
    rng = np.random.default_rng(seed)
    m = _rb_model(c2=float(rng.choice([1e-4, 3e-5, 0.0, 1.7e-5])), k2=float(rng.choice([2e-7, 3.3e-7])))
    rho = _rho(m)
    nu, no, n = (int(x) for x in rng.integers(1, 30, 3))
    lpu = rng.integers(10, 50, nu)
    rpu = rng.integers(50, 400, nu)
    lpo = rng.integers(100, 400, no)
    lro = lpo - rng.integers(1, 90, no)
    L = int(rng.integers(5, 200))
    ow = np.r_[np.zeros(nu), np.ones(no)]
    r = ref.rebalance(2, m, ow, np.r_[lpu, lpo], np.r_[lpu + 1, lro], np.r_[lpu + 3, lro], np.r_[rpu, np.zeros(no)],
                      np.full(n, L), np.zeros(n))
    c0 = int(rpu.sum()) + rho * nu
    c1 = int((lro - lpo).sum()) - rho * no
    d = L + rho
    f = [abs(c0 - k * d) + abs(c1 + k * d) for k in range(n + 1)]
    kstar = min(range(n + 1), key=lambda k: (f[k], k))
    assert len(r.moves) == kstar
    assert _val(r.obj_before, rho) == f[0] and _val(r.obj_after, rho) == f[kstar]
    assert r.moves.tolist() == [[j, 1] for j in range(kstar)]
    assert (r.worker == 1).sum() == kstar


def _objective(le, be, rho):
    return sum(abs(int(a) + rho * int(b)) for a, b in zip(le, be))


@pytest.mark.parametrize("seed", range(25))
def test_rebalance_moves_replayed_by_bruteforce(seed):
    """Replay the move log: before each move, try every (placed request, other
    worker) on a copy of the state and recompute the whole objective in exact
    rationals (rho = c2 / k2 as a fraction); the applied move must reach the
    smallest objective, be the first such pair in request-then-worker order, and
    lower the objective.  At the end no move lowers it, unplaced requests
    stayed, and the reported errors and objectives match the replayed state."""
    rng = np.random.default_rng(100 + seed)
    W = int(rng.integers(1, 7))
    m = _rb_model(c2=float(rng.choice([1e-4, 2e-6, 0.0, 1.3e-4])), k2=float(rng.choice([2e-7, 1e-6, 2.9e-7])))
    n_old, n_new = int(rng.integers(0, 25)), int(rng.integers(0, 12))
    ow = rng.integers(0, W, n_old)
    lp = rng.integers(1, 60, n_old)
    lr = np.maximum(1, (lp * np.exp(rng.normal(0, 0.6, n_old))).astype(np.int64))
    lo = np.array([int(rng.integers(0, x + 1)) for x in lr], np.int64)
    rp = lp + rng.integers(0, 80, n_old)
    # lengths of the order of rho, where requests move more than once
    nlp = rng.integers(1, 300 if seed % 2 else 900, n_new)
    nw = rng.integers(-1, W, n_new)
    _replay_check(W, m, ow, lp, lo, lr, rp, nlp, nw)


def test_rebalance_request_may_move_again():
    """Nothing in the algorithm stops a request that moved from moving again
    once other moves changed the errors: on this input request 2 moves twice,
    and both moves are the largest decrease at their step (replayed in exact
    rationals)."""
    rng = np.random.default_rng(12935)
    W = int(rng.integers(2, 6))
    n_old, n_new = int(rng.integers(0, 20)), int(rng.integers(1, 10))
    ow = rng.integers(0, W, n_old)
    lp = rng.integers(1, 60, n_old)
    lr = np.maximum(1, (lp * np.exp(rng.normal(0, 0.8, n_old))).astype(np.int64))
    lo = np.array([int(rng.integers(0, x + 1)) for x in lr], np.int64)
    rp = lp + rng.integers(0, 80, n_old)
    nlp = rng.integers(1, 100, n_new)
    nw = rng.integers(0, W, n_new)
    r = _replay_check(W, _rb_model(c2=0.0), ow, lp, lo, lr, rp, nlp, nw)
    assert r.moves[:, 0].tolist().count(2) == 2


def _replay_check(W, m, ow, lp, lo, lr, rp, nlp, nw):
    rho = _rho(m)
    n_old, n_new = len(ow), len(nlp)
    r = ref.rebalance(W, m, ow, lp, lo, lr, rp, nlp, nw)
    # the errors, from the two tests of the algorithm, one request at a time
    le = [0] * W
    be = [0] * W
    for j in range(n_old):
        if lo[j] > lp[j]:
            le[ow[j]] += int(rp[j]); be[ow[j]] += 1
        if lr[j] < lp[j]:
            le[ow[j]] += int(lr[j] - lp[j]); be[ow[j]] -= 1
    assert _val(r.obj_before, rho) == _objective(le, be, rho)
    cur = [int(x) for x in nw]

    def after(j, y):
        le2, be2 = list(le), list(be)
        le2[cur[j]] -= int(nlp[j]); be2[cur[j]] -= 1
        le2[y] += int(nlp[j]); be2[y] += 1
        return _objective(le2, be2, rho)

    def candidates():
        return [(after(j, y), j, y) for j in range(n_new) if cur[j] >= 0 for y in range(W) if y != cur[j]]

    for j, y in r.moves.tolist():
        obj = _objective(le, be, rho)
        best = min(candidates())
        assert (best[1], best[2]) == (j, y) and best[0] < obj
        le[cur[j]] -= int(nlp[j]); be[cur[j]] -= 1
        le[y] += int(nlp[j]); be[y] += 1
        cur[j] = y
    obj = _objective(le, be, rho)
    assert all(o >= obj for o, _, _ in candidates())
    assert _val(r.obj_after, rho) == obj
    assert r.worker.tolist() == cur and r.le.tolist() == le and r.be.tolist() == be
    assert all(r.worker[j] == -1 for j in range(n_new) if nw[j] == -1)
    return r


def test_rebalance_rejects_invalid_input():
    m = _rb_model()
    with pytest.raises(RuntimeError):  # generated more than the real length
        ref.rebalance(2, m, [0], [10], [6], [5], [0], [], [])
    with pytest.raises(RuntimeError):  # worker out of range
        ref.rebalance(2, m, [2], [10], [1], [5], [0], [], [])
    with pytest.raises(RuntimeError):  # new request on a worker out of range
        ref.rebalance(2, m, [], [], [], [], [], [5], [2])
    with pytest.raises(RuntimeError):  # no decode slope: the error line is undefined
        ref.rebalance(2, _rb_model(k2=0.0), [], [], [], [], [], [], [])
    with pytest.raises(RuntimeError):  # rho = c2 / k2 above 1e9
        ref.rebalance(2, _rb_model(c2=1.0, k2=1e-10), [], [], [], [], [], [], [])

