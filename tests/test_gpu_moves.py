"""Moves of requests placed in the current heartbeat window (Algorithm 2
applied to the placement) on the GPU vs the oracle (needs an MI355X)."""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def aladdin():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin as mod
    return mod


def say(*a):
    print(*a, flush=True)


def oracle_args(t):
    return (t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated, t.model,
            t.q_l_in, t.q_l_pred)


def choose_moves(t, hb, rng, points):
    """Moves before the given query indices, each of 1-3 requests placed
    earlier in the same heartbeat window, chosen on the oracle run with the
    moves so far (earlier placements do not depend on later moves)."""
    moves = []
    for k in points:
        start = max([i for i in range(k) if i == 0 or hb[i] > 0])
        r = ref.place_moves(*oracle_args(t), moves, hb_before=hb, res_t_dec=t.res_t_dec)
        cand = [j for j in range(start, k) if r.worker[j] >= 0]
        for j in rng.choice(cand, size=min(len(cand), int(rng.integers(1, 4))), replace=False) if cand else []:
            y = int(rng.choice([w for w in range(t.n_workers) if w != r.worker[j]]))
            moves.append((k, int(j), y))
            r.worker[j] = y
    return moves


def run_gpu(aladdin, t, hb, moves, tile=256, slots=0):
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(t, slots_per_worker=slots)
    cuts = sorted({k for k, _, _ in moves} | {0, t.n_queries})
    worker = np.full(t.n_queries, -2, np.int32)
    diags = []
    for a, b in zip(cuts, cuts[1:]):
        batch = [m for m in moves if m[0] == a]
        if batch:
            ev.move_requests([t.q_l_in[j] for _, j, _ in batch], [t.q_l_pred[j] for _, j, _ in batch],
                             [worker[j] for _, j, _ in batch], [y for _, _, y in batch])
            for _, j, y in batch:
                worker[j] = y
        r = ev.place(t.q_l_in[a:b], t.q_l_pred[a:b], hb_before=hb[a:b])
        worker[a:b] = r.worker
        diags.append(r.diag)
    batch = [m for m in moves if m[0] == t.n_queries]
    if batch:
        ev.move_requests([t.q_l_in[j] for _, j, _ in batch], [t.q_l_pred[j] for _, j, _ in batch],
                         [worker[j] for _, j, _ in batch], [y for _, _, y in batch])
        for _, j, y in batch:
            worker[j] = y
    summ = ev.summary()
    ev.close()
    return worker, np.concatenate(diags), summ


@pytest.mark.parametrize("history", [False, True])
def test_moves_match_oracle(aladdin, history):
    t = wl.make_trace("moves", 51, W=10, R=12, Q=900, kv_capacity=20000, model=wl.BASE_MODEL, rate=60.0)
    if history:
        t = wl.with_decode_history(t, 13)
    hb = wl.heartbeats_from_arrivals(t.arrivals, t.model.decode_slo)
    rng = np.random.default_rng(52 + int(history))
    points = sorted(rng.choice(np.arange(1, t.n_queries + 1), size=25, replace=False).tolist())
    moves = choose_moves(t, hb, rng, points)
    say("moves", len(moves), "history", history)
    want = ref.place_moves(*oracle_args(t), moves, hb_before=hb, res_t_dec=t.res_t_dec)
    worker, diag, summ = run_gpu(aladdin, t, hb, moves)
    assert np.array_equal(worker, want.worker), np.flatnonzero(worker != want.worker)[:10]
    for f in ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min"):
        assert np.array_equal(diag[f].astype(np.int64), getattr(want, f).astype(np.int64)), f
    for f in ("B", "sum_c", "sum_r", "peak"):
        assert np.array_equal(summ[f].astype(np.int64), getattr(want, f)), f


def test_rebalance_then_move_matches_oracle(aladdin):
    """Algorithm 2 in the serving loop: place a heartbeat's requests with
    Algorithm 1, re-balance them against the residents' prediction errors
    (ald_rebalance), apply the moves (ald_move_requests), then go on placing."""
    import torch
    t = wl.make_trace("rb-loop", 53, W=16, R=20, Q=1200, kv_capacity=40000, model=wl.BASE_MODEL)
    n1 = 400
    hb = np.zeros(t.n_queries, np.int32)
    hb[n1] = 1  # the heartbeat after the re-balanced window
    rng = np.random.default_rng(54)
    # what the scheduler observed of the residents (the ongoing requests):
    # about a third decode past their prediction, a third finished before it
    lp = t.res_l_pred.astype(np.int64)
    kind = rng.integers(0, 3, lp.size)
    past = lp + rng.integers(1, 60, lp.size)
    early = np.maximum(1, lp - rng.integers(1, 60, lp.size))
    l_out = np.where(kind == 0, past, np.where(kind == 1, np.minimum(early, lp - 1), np.minimum(lp, 1)))
    l_out = np.maximum(0, l_out)
    l_real = np.where(kind == 0, past + 5, np.where(kind == 1, early, lp))
    l_out = np.minimum(l_out, l_real)
    old_worker = np.repeat(np.arange(t.n_workers), np.diff(t.res_offsets))
    ev = aladdin.Evaluator(0, tile=128)
    ev.load_trace(t)
    first = ev.place(t.q_l_in[:n1], t.q_l_pred[:n1], hb_before=hb[:n1])
    placed = first.worker.copy()
    batch = wl.RebalanceBatch("loop", [t.model], np.array([t.n_workers], np.int32),
                              np.array([0, lp.size], np.int64), old_worker.astype(np.int32), lp.astype(np.int32),
                              l_out.astype(np.int32), l_real.astype(np.int32),
                              np.rint(lp * 1.3).astype(np.int32), np.array([0, n1], np.int64),
                              t.q_l_pred[:n1].astype(np.int32), placed.astype(np.int32))
    rb = ev.rebalance(batch, want_log=True)
    k = int(rb["moves"][0])
    assert k > 0
    log = rb["log"][0]
    ev.move_requests(t.q_l_in[log[:, 0]], t.q_l_pred[log[:, 0]], placed[log[:, 0]], log[:, 1])
    placed[log[:, 0]] = log[:, 1]
    rest = ev.place(t.q_l_in[n1:], t.q_l_pred[n1:], hb_before=hb[n1:])
    summ = ev.summary()
    ev.close()
    want_rb = ref.rebalance(t.n_workers, t.model, old_worker, lp, l_out, l_real, np.rint(lp * 1.3),
                            t.q_l_pred[:n1], first.worker)
    assert want_rb.moves.tolist() == log.tolist()
    moves = [(n1, int(j), int(y)) for j, y in log]
    want = ref.place_moves(*oracle_args(t), moves, hb_before=hb)
    assert np.array_equal(np.concatenate([placed, rest.worker]), want.worker)
    for f in ("B", "sum_c", "sum_r", "peak"):
        assert np.array_equal(summ[f].astype(np.int64), getattr(want, f)), f


def test_move_outside_the_window_changes_nothing(aladdin):
    t = wl.make_trace("moves-bad", 55, W=4, R=3, Q=60, kv_capacity=20000, model=wl.BASE_MODEL)
    hb = np.zeros(t.n_queries, np.int32)
    hb[30] = 1
    ev = aladdin.Evaluator(0)
    ev.load_trace(t)
    a = ev.place(t.q_l_in[:31], t.q_l_pred[:31], hb_before=hb[:31])
    j = int(np.flatnonzero(a.worker[:30] >= 0)[0])  # placed before the heartbeat
    with pytest.raises(aladdin.AladdinError) as e:
        ev.move_requests([t.q_l_in[j]], [t.q_l_pred[j]], [a.worker[j]], [(a.worker[j] + 1) % 4])
    assert e.value.code == aladdin.ALD_EINVAL
    b = ev.place(t.q_l_in[31:], t.q_l_pred[31:], hb_before=hb[31:])
    ev.close()
    want = ref.place_hb(*oracle_args(t), hb)
    assert np.array_equal(np.concatenate([a.worker, b.worker]), want.worker)


def draw_moves_case(seed):
    rng = np.random.default_rng(9500 + seed)
    W = int(rng.choice([2, 3, 7, 20, 65, 130]))
    R = int(rng.choice([0, 5, 30]))
    Q = int(rng.integers(20, 600))
    model = wl.BASE_MODEL.scaled(float(rng.choice([0.5, 1.0, 2.0])))
    if rng.random() < 0.25:
        model = dataclasses.replace(model, ttft_slo=math.inf)  # decode workers
    elif rng.random() < 0.2:
        model = dataclasses.replace(model, k1=-1e-7, k1q=1e-9)  # the fp64 checks
    t = wl.make_trace("rmoves%d" % seed, 9600 + seed, W=W, R=R, Q=Q, kv_capacity=int(rng.choice([8000, 30000])),
                      model=model, in_dist=wl.SHORT_IN, out_dist=wl.SHORT_OUT, rate=float(rng.choice([20.0, 200.0])))
    if R > 0 and rng.random() < 0.4:
        t = wl.with_decode_history(t, 9700 + seed)
    if rng.random() < 0.7:
        hb = wl.heartbeats_from_arrivals(t.arrivals, model.decode_slo)
    else:
        hb = np.zeros(Q, np.int32)
    points = sorted(rng.choice(np.arange(1, Q + 1), size=min(Q, 8), replace=False).tolist())
    return t, hb, points, int(rng.choice([64, 256, 1024])), rng


@pytest.mark.parametrize("seed", range(24))
def test_random_moves_match_oracle(aladdin, seed):
    """Random configurations with moves between placement calls: GPU vs oracle."""
    t, hb, points, tile, rng = draw_moves_case(seed)
    moves = choose_moves(t, hb, rng, points)
    say("random moves", seed, "W", t.n_workers, "Q", t.n_queries, "moves", len(moves), "tile", tile,
        "history", t.res_t_dec is not None, "ttft", t.model.ttft_slo)
    want = ref.place_moves(*oracle_args(t), moves, hb_before=hb, res_t_dec=t.res_t_dec)
    # moves are not checked against the batch limit, so leave room for them
    slots = int(np.diff(t.res_offsets).max(initial=0)) + t.n_queries
    worker, diag, summ = run_gpu(aladdin, t, hb, moves, tile=tile, slots=slots)
    assert np.array_equal(worker, want.worker), np.flatnonzero(worker != want.worker)[:10]
    for f in ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min"):
        assert np.array_equal(diag[f].astype(np.int64), getattr(want, f).astype(np.int64)), f
    for f in ("B", "sum_c", "sum_r", "peak"):
        assert np.array_equal(summ[f].astype(np.int64), getattr(want, f)), f
