"""Randomised parity: many small configurations drawn from a seeded generator,
each placed on the GPU and by the oracle, compared exactly (needs an MI355X)."""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu

INT_FIELDS = ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min")


@pytest.fixture(scope="module")
def aladdin():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin as mod
    return mod


def draw(seed):
    rng = np.random.default_rng(9000 + seed)
    W = int(rng.choice([1, 2, 3, 7, 20, 65, 130, 300, 1030]))
    R = int(rng.choice([0, 1, 5, 30]))
    Q = int(rng.integers(1, 1500))
    model = wl.BASE_MODEL.scaled(float(rng.choice([0.5, 1.0, 2.0])))
    if rng.random() < 0.2:
        model = dataclasses.replace(model, ttft_slo=math.inf)
    elif rng.random() < 0.2:
        model = dataclasses.replace(model, k1=-1e-7, k1q=1e-9)  # the fp64 checks
    cap = int(rng.choice([8000, 30000, 120000]))
    t = wl.make_trace("rand%d" % seed, 9100 + seed, W=W, R=R, Q=Q, kv_capacity=cap, model=model,
                      in_dist=wl.SHORT_IN, out_dist=wl.SHORT_OUT, rate=float(rng.choice([20.0, 200.0])))
    if R > 0 and rng.random() < 0.3:
        t = wl.with_decode_history(t, 9200 + seed)
    mode = rng.choice(["none", "period", "clock"])
    H = int(rng.choice([1, 3, 50])) if mode == "period" else 0
    hb = wl.heartbeats_from_arrivals(t.arrivals, model.decode_slo) if mode == "clock" else None
    tile = int(rng.choice([64, 128, 1024, 4096]))
    diag = bool(rng.random() < 0.7)
    return t, H, hb, tile, diag


@pytest.mark.parametrize("seed", range(64))
def test_random_configuration_matches_oracle(aladdin, seed):
    t, H, hb, tile, diag = draw(seed)
    print("random", seed, "W", t.n_workers, "Q", t.n_queries, "H", H, "clock", hb is not None, "tile", tile,
          "diag", diag, "history", t.res_t_dec is not None, "ttft", t.model.ttft_slo, flush=True)
    ev = aladdin.Evaluator(0, tile=tile)
    ev.load_trace(t)
    got = ev.place(t.q_l_in, t.q_l_pred, heartbeat_every=H, diag=diag, hb_before=hb)
    summ = ev.summary()
    ev.close()
    if hb is None:
        want = ref.place_trace(t, heartbeat_every=H)
    else:
        want = ref.place_hb(t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated,
                            t.model, t.q_l_in, t.q_l_pred, hb, res_t_dec=t.res_t_dec)
    assert np.array_equal(got.worker, want.worker), np.flatnonzero(got.worker != want.worker)[:10]
    if diag:
        for f in INT_FIELDS:
            assert np.array_equal(got.diag[f].astype(np.int64), getattr(want, f).astype(np.int64)), f
        for f in ("ttft_chosen", "tdec_chosen"):
            assert np.allclose(got.diag[f], getattr(want, f), rtol=1e-9, atol=0.0), f
    # a trailing heartbeat of the periodic form happens after the last query
    if hb is not None or H == 0 or t.n_queries % H:
        for f in ("B", "sum_c", "sum_r", "peak"):
            assert np.array_equal(summ[f].astype(np.int64), getattr(want, f)), f


def draw_sweep(seed):
    rng = np.random.default_rng(9800 + seed)
    S = int(rng.integers(1, 24))
    scen, H = [], []
    for _ in range(S):
        model = wl.BASE_MODEL.scaled(float(rng.choice([0.5, 1.0, 2.0])))
        if rng.random() < 0.2:
            model = dataclasses.replace(model, ttft_slo=math.inf)
        elif rng.random() < 0.2:
            model = dataclasses.replace(model, k1=-1e-7, k1q=1e-9)
        scen.append(wl.Scenario(n_workers=int(rng.choice([1, 2, 3, 7, 20, 65, 130, 300])), gpus_per_worker=1,
                                kv_capacity=int(rng.choice([4000, 8000, 30000, 120000])), model=model))
        H.append(int(rng.choice([0, 1, 3, 17, 100])))
    Q = int(rng.integers(1, 1500))
    q_in = wl._lengths(rng, *wl.SHORT_IN, Q).astype(np.int32)
    q_pred = wl._lengths(rng, *wl.SHORT_OUT, Q).astype(np.int32)
    tile = int(rng.choice([64, 256, 1024, 4096]))
    return scen, np.array(H, np.int32), q_in, q_pred, tile


@pytest.mark.parametrize("seed", range(16))
def test_random_sweep_matches_oracle(aladdin, seed):
    """Random scenario sets (sizes, capacities, models, heartbeat periods) swept at once."""
    scen, H, q_in, q_pred, tile = draw_sweep(seed)
    print("random sweep", seed, "S", len(scen), "W", [s.n_workers for s in scen], "Q", q_in.size, "tile", tile,
          flush=True)
    ev = aladdin.Evaluator(0, tile=tile)
    rej, first, workers, best = ev.sweep(scen, q_in, q_pred, want_workers=True, heartbeat_every=H, want_answer=True)
    ev.close()
    orej, ofirst, oworkers = ref.sweep(scen, q_in, q_pred, want_workers=True, heartbeat_every=H)
    assert np.array_equal(workers, oworkers), np.argwhere(workers != oworkers)[:5]
    assert np.array_equal(rej, orej)
    assert np.array_equal(first, ofirst)
    assert best == ref.min_gpus(scen, orej)
