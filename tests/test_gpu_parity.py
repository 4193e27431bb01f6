"""GPU library vs CPU oracle, element by element (needs an MI355X).

Integer outputs (worker choice, feasible counts, KV peaks and excesses, final
worker sums) must match exactly.  fp64 latencies are computed with the same
operations in the same order on both sides and are expected bit-identical;
the contract tolerance is a relative 1e-9 and is what the assertion enforces,
with any bit difference reported separately.  Queries whose decode or TTFT
margin lies within that tolerance are flagged by both sides (near_tie) and
counted separately.
"""
from __future__ import annotations

import dataclasses
import hashlib
import json
import math
import os

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
FIELDS_INT = ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min")
FIELDS_FP = ("ttft_chosen", "tdec_chosen")
RTOL = 1e-9


@pytest.fixture(scope="module")
def aladdin():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin as mod
    return mod


def say(*a):
    print(*a, flush=True)


def gpu_place(aladdin, trace, tile=4096, diag=True, H=None, chunks=None, slots=0):
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(trace, slots_per_worker=slots)
    H = trace.heartbeat_every if H is None else H
    if chunks is None:
        res = ev.place(trace.q_l_in, trace.q_l_pred, H, diag=diag)
        worker, dg = res.worker, res.diag
    else:
        ws, ds = [], []
        for a, b in chunks:
            r = ev.place(trace.q_l_in[a:b], trace.q_l_pred[a:b], H, diag=diag)
            ws.append(r.worker)
            ds.append(r.diag)
        worker = np.concatenate(ws)
        dg = np.concatenate(ds) if diag else None
    summ = ev.summary()
    ev.close()
    return worker, dg, summ


def compare(worker, dg, summ, want, label=""):
    assert np.array_equal(worker, want.worker), (label, np.flatnonzero(worker != want.worker)[:10])
    if dg is not None:
        for f in FIELDS_INT:
            g = dg[f].astype(np.int64)
            w = getattr(want, f).astype(np.int64)
            assert np.array_equal(g, w), (label, f, np.flatnonzero(g != w)[:10])
        for f in FIELDS_FP:
            g, w = dg[f], getattr(want, f)
            assert np.allclose(g, w, rtol=RTOL, atol=0.0), (label, f)
            nbits = int((g.view(np.int64) != w.view(np.int64)).sum())
            if nbits:
                say("%s: %s within 1e-9 but %d values differ in the last bits" % (label, f, nbits))
    if summ is not None:
        for f in ("B", "sum_c", "sum_r", "peak"):
            assert np.array_equal(summ[f].astype(np.int64), getattr(want, f)), (label, f)


# ----------------------------------------------------------------------------- small workloads
@pytest.mark.parametrize("tile", [64, 256, 4096])
def test_tiny_matches_oracle(aladdin, tile):
    t = wl.make_config("tiny")
    say("tiny tile", tile)
    compare(*gpu_place(aladdin, t, tile=tile), ref.place_trace(t), "tiny/%d" % tile)


@pytest.mark.parametrize("tile", [64, 1024, 4096])
def test_medium_matches_oracle(aladdin, tile):
    t = wl.make_config("medium")
    say("medium tile", tile)
    compare(*gpu_place(aladdin, t, tile=tile), ref.place_trace(t), "medium/%d" % tile)


def test_medium_without_diagnostics_same_choices(aladdin):
    t = wl.make_config("medium")
    w, d, s = gpu_place(aladdin, t, tile=512, diag=False)
    assert d is None
    compare(w, None, s, ref.place_trace(t), "medium/nodiag")


def test_stream_continues_across_calls(aladdin):
    # one stream placed in four calls equals the whole stream at once
    t = wl.make_trace("chunks", 21, W=24, R=20, Q=1500, kv_capacity=30000, model=wl.BASE_MODEL,
                      heartbeat_every=37)
    cuts = [(0, 100), (100, 101), (101, 900), (900, 1500)]
    compare(*gpu_place(aladdin, t, tile=256, chunks=cuts), ref.place_trace(t), "chunks")


@pytest.mark.parametrize("k1,k1q", [(2e-5, -3e-10), (-1e-7, 1e-9)])
def test_ttft_not_monotone_in_lin(aladdin, k1, k1q):
    # with a negative prefill coefficient the TTFT check has no integer
    # threshold in l_in and every pair takes the exact fp64 path
    model = dataclasses.replace(wl.BASE_MODEL, k1=k1, k1q=k1q, ttft_slo=0.03)
    t = wl.make_trace("ttft_nm", 23, W=20, R=10, Q=900, kv_capacity=30000, model=model, heartbeat_every=50)
    compare(*gpu_place(aladdin, t, tile=128), ref.place_trace(t), "ttft_nm")


@pytest.mark.parametrize("case", ["integer", "fp64", "history"])
def test_decode_workers_match_oracle(aladdin, case):
    """Split-phase decode workers (TTFT SLO +inf): only (b) and (e) are checked;
    with the integer thresholds, with the fp64 checks (a negative prefill
    coefficient), and with a decode history that (d) must then ignore."""
    m = dataclasses.replace(wl.BASE_MODEL, ttft_slo=math.inf)
    if case == "fp64":
        m = dataclasses.replace(m, k1=-1e-7, k1q=1e-9)
    t = wl.make_trace("decode-" + case, 25, W=16, R=24, Q=3000, kv_capacity=30000, model=m, heartbeat_every=60)
    if case == "history":
        t = wl.with_decode_history(t, 11)
    say("decode workers", case)
    for tile in (64, 1024):
        compare(*gpu_place(aladdin, t, tile=tile), ref.place_trace(t), "decode/%s/%d" % (case, tile))
    # the same stream with a finite TTFT SLO places differently
    fin = dataclasses.replace(t, model=dataclasses.replace(m, ttft_slo=0.02))
    assert not np.array_equal(ref.place_trace(fin).worker, ref.place_trace(t).worker)


def oracle_hb(t, hb):
    return ref.place_hb(t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated, t.model,
                        t.q_l_in, t.q_l_pred, hb, res_t_dec=t.res_t_dec)


def test_decode_workers_with_history_many_residents(aladdin):
    """A decode worker's model ignores the decode history, so no per-request
    log of constraint (d) is kept: loading 9,000 residents with decode times
    must not write one (regression: the load once wrote the log whenever
    decode times were given, past the arrays sized for no log)."""
    m = dataclasses.replace(wl.BASE_MODEL, ttft_slo=math.inf)
    t = wl.with_decode_history(wl.make_trace("decode-wide", 27, W=300, R=30, Q=600, kv_capacity=30000, model=m), 14)
    say("decode workers with history, 300 x 30 residents")
    for tile in (128, 1024):
        compare(*gpu_place(aladdin, t, tile=tile), ref.place_trace(t), "decode-wide/%d" % tile)


@pytest.mark.parametrize("tile", [64, 1024])
def test_heartbeats_per_query_equal_a_period(aladdin, tile):
    t = wl.make_trace("hbq", 26, W=30, R=20, Q=2501, kv_capacity=30000, model=wl.BASE_MODEL)
    hb = np.zeros(t.n_queries, np.int32)
    hb[37::37] = 1
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(t)
    a = ev.place(t.q_l_in, t.q_l_pred, hb_before=hb)
    ev.close()
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(t)
    b = ev.place(t.q_l_in, t.q_l_pred, heartbeat_every=37)
    ev.close()
    assert np.array_equal(a.worker, b.worker)
    for f in FIELDS_INT + FIELDS_FP:
        assert np.array_equal(a.diag[f], b.diag[f]), f
    compare(a.worker, a.diag, None, oracle_hb(t, hb), "hb per query / %d" % tile)


@pytest.mark.parametrize("history", [False, True])
def test_arrival_time_heartbeats_match_oracle(aladdin, history):
    """Poisson arrivals, one decode iteration per T_dec: bursts (several queries
    per iteration) and gaps (several iterations per query), in three calls."""
    t = wl.make_trace("arrivals", 27, W=12, R=16, Q=3000, kv_capacity=20000, model=wl.BASE_MODEL, rate=60.0)
    if history:
        t = wl.with_decode_history(t, 12)
    hb = wl.heartbeats_from_arrivals(t.arrivals, t.model.decode_slo)
    assert hb.max() >= 2 and (hb == 0).mean() > 0.2
    say("arrival-time heartbeats, history", history, "iterations", int(hb.sum()))
    ev = aladdin.Evaluator(0, tile=256)
    ev.load_trace(t)
    ws, ds = [], []
    for a, b in [(0, 1), (1, 1700), (1700, 3000)]:
        r = ev.place(t.q_l_in[a:b], t.q_l_pred[a:b], hb_before=hb[a:b])
        ws.append(r.worker)
        ds.append(r.diag)
    summ = ev.summary()
    ev.close()
    compare(np.concatenate(ws), np.concatenate(ds), summ, oracle_hb(t, hb), "arrivals/%s" % history)


def test_decode_clock_past_2_24(aladdin):
    """Once l_pred + tau reaches 2^24 a block leaves the staged evaluation (its
    24-bit count-times-end product) for the exact path.  One heartbeat entry
    runs 2^24 - 3,000 decode iterations, then 1,000 run before each query, so
    the first queries are evaluated staged and the later ones are not."""
    W, Q = 8, 1500
    rng = np.random.default_rng(31)
    t = wl.Trace(name="tau24", seed=0, model=wl.BASE_MODEL, kv_capacity=np.full(W, 4000, np.int64),
                 res_offsets=np.arange(W + 1, dtype=np.int64), res_l_in=rng.integers(1, 50, W).astype(np.int32),
                 res_l_pred=rng.integers(1, 50, W).astype(np.int32), res_generated=np.zeros(W, np.int32),
                 q_l_in=rng.integers(1, 500, Q).astype(np.int32), q_l_pred=rng.integers(1, 900, Q).astype(np.int32),
                 arrivals=None, heartbeat_every=0)
    hb = np.full(Q, 1000, np.int32)
    hb[0] = (1 << 24) - 3000
    say("decode clock past 2^24: final tau", int(hb.astype(np.int64).sum()))
    ev = aladdin.Evaluator(0, tile=256)
    ev.load_trace(t, slots_per_worker=6)  # (slots + 1 times the final tau must stay below 2^27)
    r = ev.place(t.q_l_in, t.q_l_pred, hb_before=hb)
    summ = ev.summary()
    ev.close()
    want = oracle_hb(t, hb)
    assert (want.worker >= 0).sum() > Q // 2
    compare(r.worker, r.diag, summ, want, "tau past 2^24")


def test_block_qd_span_past_2_31(aladdin):
    """gamma = 256 / 2^8: qD = 256 (l_in + l_pred).  A query of l_in = 2^23 among
    short ones gives its block of 1,024 queries a qD span of at least 2^31, so
    that block leaves the staged evaluation (32-bit compares relative to the
    block's smallest qD) for the exact path; the tile's other blocks stay."""
    model = dataclasses.replace(wl.BASE_MODEL, gamma_num=256, gamma_log2den=8)
    t = wl.make_trace("qdspan", 41, W=40, R=4, Q=4096, kv_capacity=30000, model=model)
    ql, qp = t.q_l_in.copy(), t.q_l_pred.copy()
    ql[100], qp[100] = 1 << 23, 500
    ql[3000], qp[3000] = (1 << 23) + 5, 700
    assert 256 * (int(ql[100]) + int(qp[100])) - 256 * int((ql[:1024] + qp[:1024]).min()) >= 1 << 31
    t = dataclasses.replace(t, q_l_in=ql, q_l_pred=qp)
    say("qD span past 2^31 in blocks 0 and 2 of 4")
    want = ref.place_trace(t)
    assert (want.worker >= 0).sum() > 0 and want.worker[100] == -1 and want.worker[3000] == -1
    compare(*gpu_place(aladdin, t, tile=4096), want, "qD span")


@pytest.mark.parametrize("W,R,cap,dslo,slots", [(12, 900, 850_000, 1.0, 2000), (3, 4100, 3_800_000, 2.0, 5000)])
def test_workers_too_large_to_stage_match_oracle(aladdin, W, R, cap, dslo, slots):
    """Workers loaded with at least 768 requests take the evaluation variant
    that reads unstaged workers through their breakpoint tables in global
    memory: below 4,096 live requests by table (queries with l_pred past the
    table's 2,048 by search), from 4,096 on by search; heartbeats retire
    requests between tiles."""
    m = dataclasses.replace(wl.BASE_MODEL, ttft_slo=10.0, decode_slo=dslo)
    t = wl.make_trace("big%d" % R, 90 + R, W=W, R=R, Q=1500, kv_capacity=cap, model=m,
                      in_dist=(6.0, 1.0, 16, 4096), out_dist=(6.0, 1.0, 16, 4096))
    assert (t.q_l_pred > 2048).any() and (t.q_l_pred <= 2048).mean() > 0.8
    say("workers of", R, "requests, largest l_pred", int(t.q_l_pred.max()))
    want = ref.place_trace(t, heartbeat_every=50)
    assert 0 < (want.worker >= 0).sum() < t.n_queries
    compare(*gpu_place(aladdin, t, tile=4096, H=50, slots=slots), want, "big workers %d" % R)


def test_heartbeats_per_query_checked(aladdin):
    t = wl.make_trace("hbbad", 28, W=4, R=2, Q=10, kv_capacity=30000, model=wl.BASE_MODEL)
    ev = aladdin.Evaluator(0)
    ev.load_trace(t)
    hb = np.zeros(10, np.int32)
    hb[4] = -1
    with pytest.raises(aladdin.AladdinError) as e:
        ev.place(t.q_l_in, t.q_l_pred, hb_before=hb)
    assert e.value.code == aladdin.ALD_EINVAL
    ev.close()


@pytest.mark.parametrize("seed", range(3))
def test_unequal_capacities(aladdin, seed):
    # capacities differ between workers (some equal), some workers start empty:
    # empty workers are then ranked one by one instead of as one class
    rng = np.random.default_rng(3000 + seed)
    W = int(rng.integers(8, 48))
    R = rng.integers(0, 3, W) * rng.integers(0, 30, W)  # about a third empty
    t = wl.make_trace("capmix%d" % seed, 3100 + seed, W=W, R=0, Q=1500, kv_capacity=1, model=wl.BASE_MODEL,
                      heartbeat_every=int(rng.choice([0, 40])), R_per_worker=R)
    caps = rng.choice([9000, 16000, 16000, 30000, 60000], W).astype(np.int64)
    t = dataclasses.replace(t, kv_capacity=caps)
    compare(*gpu_place(aladdin, t, tile=int(rng.choice([64, 256]))), ref.place_trace(t), "capmix%d" % seed)


def test_more_workers_than_the_dirty_bitmap(aladdin):
    # 66,000 workers (the commit's LDS dirty bitmap covers 65,536) and a batch
    # limit of about three requests, so a tile dirties many workers
    model = dataclasses.replace(wl.BASE_MODEL, c2=0.012)
    t = wl.make_trace("wide", 24, W=66000, R=0, Q=420, kv_capacity=200000, model=model)
    got = gpu_place(aladdin, t, tile=256)
    want = ref.place_trace(t, n_threads=16)
    assert (want.worker >= 0).sum() > 200
    compare(*got, want, "wide")


def test_chunks_ending_on_heartbeats(aladdin):
    # calls that end exactly where a heartbeat falls: the next call must start
    # from summaries rebuilt at the advanced decode iteration
    t = wl.make_trace("hbchunks", 22, W=16, R=24, Q=700, kv_capacity=20000, model=wl.BASE_MODEL,
                      heartbeat_every=37)
    cuts = [(0, 37), (37, 74), (74, 111), (111, 333), (333, 370), (370, 700)]
    for tile in (64, 256):
        compare(*gpu_place(aladdin, t, tile=tile, chunks=cuts), ref.place_trace(t), "hbchunks tile %d" % tile)


@pytest.mark.parametrize("seed", range(12))
def test_random_ragged_traces(aladdin, seed):
    rng = np.random.default_rng(1000 + seed)
    W = int(rng.integers(1, 70))
    R = rng.integers(0, 60, W)
    H = int(rng.choice([0, 1, 5, 64, 333]))
    model = wl.BASE_MODEL.scaled(float(rng.uniform(0.3, 1.2)))
    model = dataclasses.replace(model, theta=float(rng.choice([1.0, 0.9, 0.5])),
                                gamma_num=int(rng.integers(0, 3)), gamma_log2den=1)
    t = wl.make_trace("rand%d" % seed, 2000 + seed, W=W, R=0, Q=int(rng.integers(1, 3000)),
                      kv_capacity=int(rng.integers(2000, 40000)), model=model, heartbeat_every=H,
                      R_per_worker=R)
    tile = int(rng.choice([64, 100, 256, 1000]))
    say("random seed", seed, "W", W, "Q", t.n_queries, "H", H, "tile", tile)
    compare(*gpu_place(aladdin, t, tile=tile), ref.place_trace(t), "rand%d" % seed)


# ----------------------------------------------------------------------------- adversarial cases
FREE = wl.Model(c1=0.0, k1=1e-12, k1q=0.0, c3=0.0, c2=1e-3, k2=1e-12, ttft_slo=1e9, decode_slo=1.0)


def _trace(W, M, residents, queries, model=FREE, H=0):
    counts = np.array([len(r) for r in residents], np.int64)
    off = np.zeros(W + 1, np.int64)
    off[1:] = np.cumsum(counts)
    flat = [x for r in residents for x in r] or [(1, 1, 0)]
    arr = np.array(flat, np.int32).reshape(-1, 3)[: int(counts.sum())]
    q = np.array(queries, np.int32).reshape(-1, 2)
    return wl.Trace(name="adv", seed=0, model=model, kv_capacity=np.asarray(M, np.int64) * np.ones(W, np.int64),
                    res_offsets=off, res_l_in=arr[:, 0].copy(), res_l_pred=arr[:, 1].copy(),
                    res_generated=arr[:, 2].copy(), q_l_in=q[:, 0].copy(), q_l_pred=q[:, 1].copy(),
                    arrivals=None, heartbeat_every=H)


def test_fig3_example_on_gpu(aladdin):
    fx = json.load(open(os.path.join(GOLDEN, "fig3_example.json")))
    LP, LO = fx["derived"]["long_prompt"], fx["derived"]["long_output"]
    t = _trace(2, fx["printed"]["kv_capacity"], [[], []], [LP, LO, LP, LO])
    w, d, s = gpu_place(aladdin, t, tile=64)
    assert list(w) == [0, 0, 1, 1]
    assert list(s["peak"]) == [fx["printed"]["best_peak_each_worker"]] * 2


def test_all_workers_identical_rank_ties(aladdin):
    # identical workers: ties everywhere, lowest index wins each time
    res = [[(50, 10, 3), (20, 30, 0)]] * 40
    q = [(30, 20)] * 300 + [(1, 1)] * 50
    t = _trace(40, 2000, res, q)
    compare(*gpu_place(aladdin, t, tile=128), ref.place_trace(t), "ties")


def test_peak_exactly_at_capacity(aladdin):
    # (4,1) then (1,4) gives a peak of exactly 7
    t = _trace(3, 7, [[], [], []], [(4, 1), (1, 4), (4, 1), (1, 4), (4, 1), (1, 4), (3, 3)])
    compare(*gpu_place(aladdin, t, tile=64), ref.place_trace(t), "exact-cap")


def test_many_commits_to_one_worker_in_one_tile(aladdin):
    # one roomy worker absorbs hundreds of placements inside a single tile
    t = _trace(5, [10 ** 6, 50, 50, 50, 50], [[], [], [], [], []], [(3, 2)] * 700)
    compare(*gpu_place(aladdin, t, tile=1024, slots=800), ref.place_trace(t), "one-worker")


def test_no_worker_ever_fits(aladdin):
    t = _trace(7, 10, [[(5, 5, 0)]] * 7, [(20, 20)] * 333)
    w, d, s = gpu_place(aladdin, t, tile=64)
    assert (w == -1).all()
    compare(w, d, s, ref.place_trace(t), "nothing-fits")


def test_single_worker_and_empty_residents(aladdin):
    t = _trace(1, 5000, [[]], [(int(a), int(b)) for a, b in zip(range(1, 200), range(200, 1, -1))])
    compare(*gpu_place(aladdin, t, tile=64), ref.place_trace(t), "single")


def test_heartbeat_every_query_drains_residents(aladdin):
    res = [[(10, 3, 1), (5, 2, 0), (7, 9, 8)] for _ in range(9)]
    q = [(2, 2)] * 400
    t = _trace(9, 40, res, q, H=1)
    compare(*gpu_place(aladdin, t, tile=64), ref.place_trace(t), "hb1")


def test_near_tie_margins_are_flagged(aladdin):
    # decode margin exactly zero for the first query
    m = wl.Model(c1=0.0, k1=0.0, k1q=0.0, c3=0.0, c2=0.0, k2=0.5, ttft_slo=1e9, decode_slo=5.0,
                 gamma_num=0, gamma_log2den=1)
    t = _trace(2, 10 ** 6, [[], []], [(10, 3), (1, 1), (9, 1)], model=m)
    w, d, s = gpu_place(aladdin, t, tile=64, slots=16)
    want = ref.place_trace(t)
    compare(w, d, s, want, "near-tie")
    assert d["near_tie"][0] == 1


@pytest.mark.parametrize("seed", [0, 1])
def test_near_tie_sets_with_integer_forms(aladdin, seed):
    # k1 > 0 and narrow bands: the evaluation takes near-tie margins from each
    # worker's exact integer near-tie sets.  The TTFT margin is zero where
    # S1 + l_in = 10 and the decode margin where sum(c) + l_in = 10, so the tie
    # sits at a different l_in on each worker as the workers fill.
    m = wl.Model(c1=0.0, k1=0.25, k1q=0.0, c3=0.0, c2=0.0, k2=0.5, ttft_slo=2.5, decode_slo=5.0,
                 gamma_num=0, gamma_log2den=1)
    rng = np.random.default_rng(seed)
    res = [[(int(rng.integers(1, 4)), int(rng.integers(1, 4)), 0)] for _ in range(6)] + [[], []]
    q = [(int(a), int(b)) for a, b in zip(rng.integers(1, 12, 300), rng.integers(1, 6, 300))]
    t = _trace(8, 10 ** 6, res, q, model=m)
    want = ref.place_trace(t)
    assert want.near_tie.sum() > 0
    for tile in (64, 4096):
        w, d, s = gpu_place(aladdin, t, tile=tile, slots=64)
        compare(w, d, s, want, "integer near-tie sets, tile %d" % tile)


# ----------------------------------------------------------------------------- constraint (d)
@pytest.mark.parametrize("tile", [64, 4096])
def test_decode_history_matches_oracle(aladdin, tile):
    t = wl.with_decode_history(wl.make_config("medium"), 7)
    want = ref.place_trace(t)
    assert 0 < int((want.worker >= 0).sum()) < 719  # the limit binds on part of the pool
    compare(*gpu_place(aladdin, t, tile=tile), want, "history medium tile %d" % tile)


def test_decode_history_without_diagnostics_same_choices(aladdin):
    t = wl.with_decode_history(wl.make_config("medium"), 8, 0.0, 0.6)
    w, _, s = gpu_place(aladdin, t, tile=256, diag=False)
    compare(w, None, s, ref.place_trace(t), "history no diag")


@pytest.mark.parametrize("tile", [64, 256, 4096])
def test_decode_history_across_heartbeats(aladdin, tile):
    # slack grows at every heartbeat and new requests join the ongoing set;
    # calls end on and between heartbeats
    t = wl.with_decode_history(wl.make_trace("hbhist", 23, W=16, R=24, Q=700, kv_capacity=20000,
                                             model=wl.BASE_MODEL, heartbeat_every=37), 9)
    want = ref.place_trace(t)
    assert int((want.worker >= 0).sum()) > 50
    cuts = [(0, 37), (37, 74), (74, 100), (100, 333), (333, 370), (370, 700)]
    compare(*gpu_place(aladdin, t, tile=tile, chunks=cuts), want, "history hb tile %d" % tile)
    compare(*gpu_place(aladdin, t, tile=tile), want, "history hb one call tile %d" % tile)


def test_decode_history_fp64_checks(aladdin):
    # a negative prefill coefficient: every pair takes the fp64 checks
    m = dataclasses.replace(wl.BASE_MODEL, k1=-1e-6, k1q=2e-9)
    t = wl.with_decode_history(wl.make_trace("hbneg", 24, W=12, R=16, Q=500, kv_capacity=20000, model=m,
                                             heartbeat_every=25), 10)
    compare(*gpu_place(aladdin, t, tile=64), ref.place_trace(t), "history fp64")


def test_decode_history_near_tie(aladdin):
    # the resident saved 2 * 0.5 - 0.5 = 0.5 s; a prefill of 0.25 * 2 = 0.5 s meets
    # constraint (d) exactly (feasible, flagged)
    m = wl.Model(c1=0.0, k1=0.25, k1q=0.0, c3=0.0, c2=0.0, k2=1e-9, ttft_slo=100.0, decode_slo=0.5)
    t = _trace(2, 10 ** 6, [[(4, 8, 2)], []], [(2, 3), (3, 3), (1, 1)], model=m)
    t = dataclasses.replace(t, res_t_dec=np.array([0.5]))
    want = ref.place_trace(t)
    assert want.near_tie[0] == 1 and want.worker[0] == 0
    compare(*gpu_place(aladdin, t, tile=64, slots=16), want, "history near tie")


def test_invalid_decode_history_is_rejected(aladdin):
    t = wl.make_config("tiny")
    for bad in (-1.0, float("nan"), float("inf")):
        td = np.full(t.n_resident, 0.1)
        td[3] = bad
        ev = aladdin.Evaluator(0)
        with pytest.raises(aladdin.AladdinError):
            ev.load_trace(dataclasses.replace(t, res_t_dec=td))
        ev.close()


def test_slots_exhausted_is_reported(aladdin):
    t = _trace(1, 10 ** 6, [[]], [(3, 2)] * 50)
    ev = aladdin.Evaluator(0, tile=64)
    ev.load_trace(t, slots_per_worker=8)
    with pytest.raises(aladdin.AladdinError) as ei:
        ev.place(t.q_l_in, t.q_l_pred, 0)
    assert ei.value.code == aladdin.ALD_ESLOTS
    ev.close()


def test_invalid_inputs_are_rejected(aladdin):
    t = _trace(2, 100, [[(3, 2, 0)], []], [(1, 1)])
    ev = aladdin.Evaluator(0, tile=64)
    bad = dataclasses.replace(t, res_generated=np.array([2], np.int32))  # g must be < l_pred
    with pytest.raises(aladdin.AladdinError) as ei:
        ev.load_trace(bad)
    assert ei.value.code == aladdin.ALD_EINVAL
    with pytest.raises(aladdin.AladdinError) as ei:
        ev.place([1], [1], 0)
    assert ei.value.code == aladdin.ALD_ESTATE
    ev.load_trace(t)
    with pytest.raises(aladdin.AladdinError) as ei:
        ev.place([0], [1], 0)
    assert ei.value.code == aladdin.ALD_EINVAL
    bad_model = dataclasses.replace(t, model=dataclasses.replace(FREE, decode_slo=0.0, c3=0.1))
    with pytest.raises(aladdin.AladdinError):
        ev.load_trace(bad_model)
    ev.close()


def test_invalid_query_late_in_stream_writes_nothing(aladdin):
    # a bad length in a later tile is caught before the first commit of the
    # call: outputs and worker state stay as they were, and the handle stays usable
    import torch
    t = wl.make_config("tiny")
    ev = aladdin.Evaluator(0, tile=64)
    ev.load_trace(t)
    before = ev.summary()
    dev = torch.device("cuda", 0)
    ql = np.array(t.q_l_in, np.int32)
    qp = np.array(t.q_l_pred, np.int32)
    for idx, field, val in ((200, "lin", 0), (255, "lp", (1 << 24) + 1), (130, "lin", -5)):
        a, b = ql.copy(), qp.copy()
        (a if field == "lin" else b)[idx] = val
        out = torch.full((len(a),), 12345, dtype=torch.int32, device=dev)
        dg = torch.full((len(a) * 40,), 7, dtype=torch.uint8, device=dev)
        with pytest.raises(aladdin.AladdinError) as ei:
            ev.place_device(torch.as_tensor(a).to(dev), torch.as_tensor(b).to(dev), 0, True, out, dg)
        assert ei.value.code == aladdin.ALD_EINVAL
        assert bool((out == 12345).all()) and bool((dg == 7).all())
        after = ev.summary()
        assert all(np.array_equal(before[k], after[k]) for k in before)
    res = ev.place(ql, qp, 0)
    ev.close()
    want = ref.place_trace(t)
    assert np.array_equal(res.worker, want.worker)


def test_sweep_small_matches_oracle(aladdin):
    s = wl.make_sweep("mini", 9, Q=700, worker_counts=(2, 3, 5, 16), gpu_counts=(1, 2), base_capacity=6000,
                      model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)
    ev = aladdin.Evaluator(0, tile=128)
    rej, first, workers, best = ev.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, want_answer=True)
    ev.close()
    orej, ofirst, oworkers = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True)
    assert np.array_equal(workers, oworkers)
    assert np.array_equal(rej, orej)
    assert np.array_equal(first, ofirst)
    assert best == ref.min_gpus(s.scenarios, orej)


@pytest.mark.parametrize("tile", [64, 1024])
def test_sweep_with_heartbeats_matches_oracle(aladdin, tile):
    s = wl.make_sweep("mini-hb", 10, Q=2500, worker_counts=(1, 2, 3, 5, 16, 40), gpu_counts=(1, 2), base_capacity=65536,
                      model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)
    H = np.array([0, 1, 2, 7, 25, 64, 100, 333, 1000, 2499, 2500, 5000], np.int32)
    say("sweep with heartbeats, tile", tile)
    ev = aladdin.Evaluator(0, tile=tile)
    rej, first, workers = ev.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, heartbeat_every=H)
    ev.close()
    orej, ofirst, oworkers = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, heartbeat_every=H,
                                       n_threads=4)
    assert np.array_equal(workers, oworkers)
    assert np.array_equal(rej, orej)
    assert np.array_equal(first, ofirst)


def test_sweep_heartbeat_arguments_checked(aladdin):
    s = wl.make_sweep("mini-hb", 11, Q=50, worker_counts=(2,), gpu_counts=(1,), base_capacity=6000,
                      model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)
    ev = aladdin.Evaluator(0)
    with pytest.raises(aladdin.AladdinError) as e:
        ev.sweep(s.scenarios, s.q_l_in, s.q_l_pred, heartbeat_every=[-1])
    assert e.value.code == aladdin.ALD_EINVAL
    ev.close()


def test_repeat_runs_bitwise_identical(aladdin):
    t = wl.make_config("medium")
    a = gpu_place(aladdin, t, tile=1024)
    b = gpu_place(aladdin, t, tile=1024)
    assert np.array_equal(a[0], b[0])
    assert a[1].tobytes() == b[1].tobytes()


# ----------------------------------------------------------------------------- full-size workloads
def _digest(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def _check_golden(name, worker, dg, summ):
    g = json.load(open(os.path.join(GOLDEN, "%s_oracle.json" % name)))
    assert int((worker >= 0).sum()) == g["placed"]
    assert _digest(worker.astype(np.int32)) == g["sha256"]["worker"]
    casts = {"n_feasible": np.int32, "near_tie": np.int32, "kv_peak_chosen": np.int64,
             "kv_excess_min": np.int64, "ttft_chosen": np.float64, "tdec_chosen": np.float64}
    for f, dt in casts.items():
        assert _digest(dg[f].astype(dt)) == g["sha256"][f], f
    for f in ("B", "sum_c", "sum_r", "peak"):
        assert _digest(summ[f].astype(np.int64)) == g["sha256"][f], f
    smp = g["sample"]
    idx = np.array(smp["index"])
    assert np.array_equal(worker[idx], np.array(smp["worker"]))
    for f in FIELDS_INT:
        assert np.array_equal(dg[f][idx].astype(np.int64), np.array(smp[f], np.int64)), f


def test_large_full_size(aladdin):
    t = wl.make_config("large")
    say("large: W=512 R=512 Q=65536")
    w, d, s = gpu_place(aladdin, t, tile=65536)
    _check_golden("large", w, d, s)
    # sampled queries recomputed by the oracle one by one at the initial state
    # (valid because no query of this stream is ever placed)
    idx = np.arange(0, t.n_queries, 4099)
    want = ref.place(t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated,
                     t.model, t.q_l_in[idx], t.q_l_pred[idx], no_commit=True)
    assert (w == -1).all()
    for f in FIELDS_INT:
        assert np.array_equal(d[f][idx].astype(np.int64), getattr(want, f).astype(np.int64)), f


def test_long_full_size(aladdin):
    t = wl.make_config("long")
    say("long: W=2048 R=1024 Q=131072 heartbeat 100")
    w, d, s = gpu_place(aladdin, t, tile=4096)
    _check_golden("long", w, d, s)


def test_sweep_full_size(aladdin):
    s = wl.make_config("sweep")
    say("sweep: 256 scenarios x 16384 queries")
    g = json.load(open(os.path.join(GOLDEN, "sweep_oracle.json")))
    ev = aladdin.Evaluator(0, tile=1024)
    rej, first, workers, best = ev.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, want_answer=True)
    ev.close()
    assert list(rej) == g["rejected"]
    assert list(first) == g["first_reject"]
    assert _digest(workers.astype(np.int32)) == g["sha256"]["worker"]
    # the answer, computed on the device, equals the oracle's
    assert best == (g["min_gpus"], g["min_gpus_scenario"])
    assert aladdin.smallest_feasible_cluster(s.scenarios, rej) == best


def test_sorted_layout_arrival_time_heartbeats_match_oracle(aladdin):
    # one-scenario tiles of 16,384+ queries evaluate in l_pred order; per-query
    # heartbeats end tiles at arbitrary queries, so chunks come out partial
    t = wl.make_trace("arrivals-sorted", 29, W=12, R=16, Q=20000, kv_capacity=20000, model=wl.BASE_MODEL, rate=60.0)
    hb = wl.heartbeats_from_arrivals(t.arrivals, t.model.decode_slo)
    say("sorted layout, arrival-time heartbeats, iterations", int(hb.sum()))
    ev = aladdin.Evaluator(0, tile=65536)
    ev.load_trace(t)
    r = ev.place(t.q_l_in, t.q_l_pred, hb_before=hb)
    summ = ev.summary()
    ev.close()
    compare(r.worker, r.diag, summ, oracle_hb(t, hb), "arrivals sorted")


def test_sorted_layout_decode_history_matches_oracle(aladdin):
    # constraint (d) takes the commit variants with the decode history
    t = wl.with_decode_history(wl.make_trace("hist-sorted", 30, W=24, R=24, Q=18000, kv_capacity=20000,
                                             model=wl.BASE_MODEL), 11)
    want = ref.place_trace(t)
    placed = int((want.worker >= 0).sum())
    say("sorted layout with a decode history, placed", placed)
    assert 0 < placed < 18000
    compare(*gpu_place(aladdin, t, tile=65536), want, "history sorted")
