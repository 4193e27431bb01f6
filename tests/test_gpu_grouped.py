"""Grouped placement (App. A) on the GPU vs the CPU oracle (needs an MI355X).

The reference is the oracle's grouped placement: its router sends group g the
share N_g / N_w of the stream, and each group places its queries on its own
workers with Algorithm 1, under the cluster's heartbeats (every H queries of
the whole stream)."""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu

FIELDS = ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min", "ttft_chosen", "tdec_chosen")


@pytest.fixture(scope="module")
def aladdin():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin as mod
    return mod


def say(*a):
    print(*a, flush=True)


def oracle_grouped(t, sizes, H):
    """Per query: global worker (or -1) and diagnostics over its group."""
    r = ref.place_grouped(t.n_workers, np.broadcast_to(np.asarray(t.kv_capacity, np.int64), (t.n_workers,)),
                          t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated, t.model, sizes, t.q_l_in,
                          t.q_l_pred, heartbeat_every=H, res_t_dec=t.res_t_dec)
    return r.worker, {f: getattr(r, f) for f in FIELDS}


def check(got, want_w, want_d, label):
    assert np.array_equal(got.worker, want_w), (label, np.flatnonzero(got.worker != want_w)[:10])
    for f in FIELDS:
        g, w = got.diag[f], want_d[f]
        if f.startswith(("ttft", "tdec")):
            assert np.allclose(g, w, rtol=1e-9, atol=0.0), (label, f)
        else:
            assert np.array_equal(g.astype(np.int64), w.astype(np.int64)), (label, f, np.flatnonzero(g != w)[:10])


CASES = [
    # (G, sizes, H, tile)
    (1, [40], 0, 256),
    (3, [10, 17, 13], 0, 64),
    (4, [10, 10, 10, 10], 48, 256),
    (5, [1, 2, 30, 3, 4], 60, 1024),
    (5, [1, 2, 30, 3, 4], 37, 128),
    (2, [39, 1], 7, 64),
]


@pytest.mark.parametrize("case", CASES, ids=["G%d-H%d-t%d" % (c[0], c[2], c[3]) for c in CASES])
def test_grouped_matches_oracle(aladdin, case):
    G, sizes, H, tile = case
    t = wl.make_trace("grouped", 31, W=40, R=16, Q=2400, kv_capacity=30000, model=wl.BASE_MODEL)
    say("grouped", case)
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(t)
    got = ev.place_grouped(sizes, t.q_l_in, t.q_l_pred, heartbeat_every=H)
    summ = ev.summary()
    ev.close()
    w, d = oracle_grouped(t, sizes, H)
    check(got, w, d, "grouped %s" % (case,))
    assert int((w >= 0).sum()) > 0 and (H > 0 or int((w >= 0).sum()) < t.n_queries)
    # every group takes its share of the stream (within one query)
    route = ref.route_groups(sizes, t.n_queries)
    wb = np.concatenate([[0], np.cumsum(sizes)])
    for g, n in enumerate(sizes):
        assert abs(int((route == g).sum()) - t.n_queries * n / sum(sizes)) < 1
        placed = w[route == g]
        assert np.all((placed == -1) | ((placed >= wb[g]) & (placed < wb[g + 1])))
    # one group is the ungrouped placement
    if G == 1:
        want = ref.place_trace(dataclasses.replace(t, heartbeat_every=H))
        assert np.array_equal(got.worker, want.worker)
        assert np.array_equal(summ["B"].astype(np.int64), want.B)


def test_grouped_in_calls_with_history(aladdin):
    """Calls continue one stream (the router's counts and the heartbeat clock
    carry over, also in the middle of a heartbeat window); constraint (d) with
    a decode history holds per group."""
    G, sizes, H = 3, [7, 11, 6], 30
    t = wl.with_decode_history(wl.make_trace("grouped-d", 32, W=24, R=12, Q=1800, kv_capacity=20000,
                                             model=wl.BASE_MODEL), 5)
    ev = aladdin.Evaluator(0, tile=128)
    ev.load_trace(t)
    parts, ds = [], []
    for a, b in [(0, 37), (37, 301), (301, 1800)]:
        r = ev.place_grouped(sizes, t.q_l_in[a:b], t.q_l_pred[a:b], heartbeat_every=H)
        parts.append(r.worker)
        ds.append(r.diag)
    ev.close()
    got = type(r)(worker=np.concatenate(parts), diag=np.concatenate(ds))
    w, d = oracle_grouped(t, sizes, H)
    check(got, w, d, "grouped calls")


def test_grouped_edge_cases(aladdin):
    """Fewer queries than groups (some groups get none), one worker per group,
    and a decode-worker model."""
    import math
    t = wl.make_trace("grouped-edge", 34, W=12, R=6, Q=900, kv_capacity=25000, model=wl.BASE_MODEL)
    for sizes, Q, H, model in (([3, 4, 5], 2, 0, None), ([1] * 12, 900, 0, None), ([1] * 12, 840, 24, None),
                               ([6, 6], 900, 0, dataclasses.replace(wl.BASE_MODEL, ttft_slo=math.inf))):
        tt = t if model is None else dataclasses.replace(t, model=model)
        tt = dataclasses.replace(tt, q_l_in=tt.q_l_in[:Q], q_l_pred=tt.q_l_pred[:Q], arrivals=None)
        say("grouped edge", sizes, Q, H)
        ev = aladdin.Evaluator(0, tile=128)
        ev.load_trace(tt)
        got = ev.place_grouped(sizes, tt.q_l_in, tt.q_l_pred, heartbeat_every=H)
        ev.close()
        w, d = oracle_grouped(tt, sizes, H)
        check(got, w, d, "edge %s Q=%d H=%d" % (sizes, Q, H))


def test_grouped_arguments_checked(aladdin):
    t = wl.make_trace("grouped-bad", 33, W=8, R=2, Q=100, kv_capacity=30000, model=wl.BASE_MODEL)
    ev = aladdin.Evaluator(0)
    ev.load_trace(t)
    bad = [([4, 3], 0, 100),       # sizes do not add up to W
           ([8, 0], 0, 10),        # empty group
           ([4, 4], -1, 10)]       # negative period
    for sizes, H, Q in bad:
        with pytest.raises(aladdin.AladdinError) as e:
            ev.place_grouped(sizes, t.q_l_in[:Q], t.q_l_pred[:Q], heartbeat_every=H)
        assert e.value.code == aladdin.ALD_EINVAL
    ev.close()


def draw_grouped(seed):
    rng = np.random.default_rng(9900 + seed)
    G = int(rng.integers(1, 7))
    sizes = [int(x) for x in rng.integers(1, 25, G)]
    W = sum(sizes)
    R = int(rng.choice([0, 5, 16]))
    model = wl.BASE_MODEL.scaled(float(rng.choice([0.5, 1.0, 2.0])))
    if rng.random() < 0.2:
        model = dataclasses.replace(model, ttft_slo=math.inf)
    elif rng.random() < 0.2:
        model = dataclasses.replace(model, k1=-1e-7, k1q=1e-9)
    H = int(rng.choice([0, 1, 5, 20, 33]))
    Q = int(rng.integers(1, 1500))
    t = wl.make_trace("rgrouped%d" % seed, 9950 + seed, W=W, R=R, Q=Q, kv_capacity=int(rng.choice([8000, 30000])),
                      model=model, in_dist=wl.SHORT_IN, out_dist=wl.SHORT_OUT)
    if R > 0 and rng.random() < 0.3:
        t = wl.with_decode_history(t, 9990 + seed)
    return t, sizes, H, int(rng.choice([64, 256, 1024]))


@pytest.mark.parametrize("seed", range(16))
def test_random_grouped_matches_oracle(aladdin, seed):
    """Random group counts and sizes, models, decode histories, heartbeats and tiles."""
    t, sizes, H, tile = draw_grouped(seed)
    say("random grouped", seed, "sizes", sizes, "H", H, "Q", t.n_queries, "tile", tile,
        "history", t.res_t_dec is not None, "ttft", t.model.ttft_slo)
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(t)
    got = ev.place_grouped(sizes, t.q_l_in, t.q_l_pred, heartbeat_every=H)
    ev.close()
    w, d = oracle_grouped(t, sizes, H)
    check(got, w, d, "random grouped %d" % seed)
