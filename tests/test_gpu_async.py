"""Stream-asynchronous placement (needs an MI355X).

ald_place_stream_async enqueues the tile rounds a call needs when no tile is
cut (plus spare rounds) and returns; a status word on the device tells how the
call ended.  A chain of such calls must place exactly what the oracle's one
arrival-order pass places (Algorithm 1, Sec. 4.2), also when rounds run out
(the call stops short, later calls are blocked, ald_place_resume finishes it
and the blocked calls are issued again), when heartbeats fall inside and
between calls, and when synchronous calls are mixed in."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu

INT_FIELDS = ("n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min")
SENTINEL = 12345


@pytest.fixture(scope="module")
def aladdin():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin as mod
    return mod


def trace(W, R, Q, cap, seed):
    return wl.make_trace("async", seed, W=W, R=R, Q=Q, kv_capacity=cap, model=wl.BASE_MODEL,
                         in_dist=wl.SHORT_IN, out_dist=wl.SHORT_OUT, rate=200.0)


def chunks(Q, n):
    edges = np.linspace(0, Q, n + 1).astype(int)
    return [(int(a), int(b)) for a, b in zip(edges[:-1], edges[1:])]


def run_async_chain(aladdin, ev, t, H, parts, spare, diag=True):
    """Issue every part asynchronously; on a short call resume it and issue the
    blocked parts again.  Returns the concatenated placement and diagnostics,
    and how many calls stopped short."""
    import torch
    dev = ev.device
    ql = torch.as_tensor(t.q_l_in, dtype=torch.int32, device=dev)
    qp = torch.as_tensor(t.q_l_pred, dtype=torch.int32, device=dev)
    Q = int(ql.numel())
    out = torch.full((Q,), -7, dtype=torch.int32, device=dev)
    dg = torch.zeros(Q * aladdin.DIAG_DTYPE.itemsize, dtype=torch.uint8, device=dev) if diag else None
    status = torch.full((len(parts),), SENTINEL, dtype=torch.int32, device=dev)
    short = 0
    todo = list(range(len(parts)))
    while todo:
        for k in todo:
            a, b = parts[k]
            ev.place_async(ql[a:b], qp[a:b], heartbeat_every=H, diag=diag, out=out[a:b],
                           diag_out=None if dg is None else dg[a * 40:b * 40], status=status[k:k + 1],
                           spare_rounds=spare)
        torch.cuda.synchronize()
        st = status.cpu().numpy()
        codes = st[todo]
        assert SENTINEL not in codes, codes
        bad = [i for i, c in enumerate(codes) if c != aladdin.ALD_OK]
        if not bad:
            break
        first = bad[0]
        # the first call that did not finish stopped short; every later one was blocked
        assert codes[first] == aladdin.ALD_EINCOMPLETE, codes
        assert all(c == aladdin.ALD_EBLOCKED for c in codes[first + 1:]), codes
        short += 1
        ev.resume()
        todo = todo[first + 1:]
        status[todo] = SENTINEL
    torch.cuda.synchronize()
    got_w = out.cpu().numpy()
    got_d = None if dg is None else dg.cpu().numpy().view(aladdin.DIAG_DTYPE)
    return got_w, got_d, short


def compare(got_w, got_d, summ, want, H, Q):
    assert np.array_equal(got_w, want.worker), np.flatnonzero(got_w != want.worker)[:10]
    if got_d is not None:
        for f in INT_FIELDS:
            assert np.array_equal(got_d[f].astype(np.int64), getattr(want, f).astype(np.int64)), f
        for f in ("ttft_chosen", "tdec_chosen"):
            assert np.allclose(got_d[f], getattr(want, f), rtol=1e-9, atol=0.0), f
    if H == 0 or Q % H:
        for f in ("B", "sum_c", "sum_r", "peak"):
            assert np.array_equal(summ[f].astype(np.int64), getattr(want, f)), f


CASES = [
    # W, residents per worker, Q, KV capacity, heartbeat period, parts, spare rounds
    (12, 5, 3000, 30000, 0, 6, 0),
    (12, 5, 3000, 30000, 50, 7, 0),
    (40, 3, 4000, 8000, 0, 5, 2),
    (64, 1, 4096, 8000, 100, 9, 0),
    (64, 1, 4096, 8000, 37, 4, 64),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_async_chain_matches_oracle(aladdin, case):
    W, R, Q, cap, H, n, spare = CASES[case]
    print("async chain case", case, "W", W, "R", R, "Q", Q, "cap", cap, "H", H, "parts", n, "spare", spare,
          flush=True)
    t = trace(W, R, Q, cap, 9100 + case)
    want = ref.place_trace(t, heartbeat_every=H)
    ev = aladdin.Evaluator(0, tile=4096)
    ev.load_trace(t)
    got_w, got_d, short = run_async_chain(aladdin, ev, t, H, chunks(Q, n), spare)
    summ = ev.summary()
    ev.close()
    print("calls that stopped short", short, flush=True)
    if case == 0:
        assert short > 0  # long tiles on a filling cluster: the resumption path was taken
    compare(got_w, got_d, summ, want, H, Q)


def test_async_without_cuts_needs_no_resume(aladdin):
    # a full cluster (capacity 1 token): every query is rejected, no worker
    # changes, so no tile is cut and the rounds enqueued are exactly enough,
    # heartbeats inside and between calls included
    t = trace(64, 2, 3000, 1, 9200)
    want = ref.place_trace(t, heartbeat_every=25)
    assert (want.worker < 0).all()
    ev = aladdin.Evaluator(0, tile=4096)
    ev.load_trace(t)
    got_w, got_d, short = run_async_chain(aladdin, ev, t, 25, chunks(3000, 8), 0)
    summ = ev.summary()
    ev.close()
    assert short == 0
    compare(got_w, got_d, summ, want, 25, 3000)


def test_sync_calls_after_async_ones(aladdin):
    import torch
    t = trace(12, 0, 3000, 8000, 9300)
    H = 0
    want = ref.place_trace(t, heartbeat_every=H)
    ev = aladdin.Evaluator(0, tile=4096)
    ev.load_trace(t)
    dev = ev.device
    ql = torch.as_tensor(t.q_l_in, dtype=torch.int32, device=dev)
    qp = torch.as_tensor(t.q_l_pred, dtype=torch.int32, device=dev)
    out = torch.full((3000,), -7, dtype=torch.int32, device=dev)
    dg = torch.zeros(3000 * 40, dtype=torch.uint8, device=dev)
    s = torch.full((2,), SENTINEL, dtype=torch.int32, device=dev)
    ev.place_async(ql[:1000], qp[:1000], H, True, out[:1000], dg[:40000], s[0:1], spare_rounds=0)
    ev.place_async(ql[1000:1500], qp[1000:1500], H, True, out[1000:1500], dg[40000:60000], s[1:2], spare_rounds=0)
    torch.cuda.synchronize()
    codes = s.cpu().numpy()
    assert codes[0] == aladdin.ALD_EINCOMPLETE and codes[1] == aladdin.ALD_EBLOCKED, codes
    # a synchronous call refuses to run over an unfinished asynchronous one and changes nothing
    with pytest.raises(aladdin.AladdinError) as e:
        ev.place_device(ql[1000:1500], qp[1000:1500], H, True, out[1000:1500], dg[40000:60000])
    assert e.value.code == aladdin.ALD_EINCOMPLETE
    ev.resume()
    ev.resume()  # nothing left: a no-op
    ev.place_device(ql[1000:2200], qp[1000:2200], H, True, out[1000:2200], dg[40000:88000])
    s[0] = SENTINEL
    ev.place_async(ql[2200:], qp[2200:], H, True, out[2200:], dg[88000:], s[0:1], spare_rounds=4096)
    torch.cuda.synchronize()
    assert int(s[0].item()) == aladdin.ALD_OK
    summ = ev.summary()
    ev.close()
    compare(out.cpu().numpy(), dg.cpu().numpy().view(aladdin.DIAG_DTYPE), summ, want, H, 3000)


def test_async_errors_and_empty_calls(aladdin):
    import torch
    t = trace(12, 5, 600, 30000, 9400)
    ev = aladdin.Evaluator(0, tile=4096)
    ev.load_trace(t)
    dev = ev.device
    before = ev.summary()
    s = torch.full((3,), SENTINEL, dtype=torch.int32, device=dev)
    empty = torch.empty(0, dtype=torch.int32, device=dev)
    ev.place_async(empty, empty, 0, False, status=s[0:1])
    bad = torch.as_tensor(t.q_l_in, dtype=torch.int32, device=dev).clone()
    bad[17] = 0  # a length outside [1, 2^24]
    qp = torch.as_tensor(t.q_l_pred, dtype=torch.int32, device=dev)
    out = torch.full((600,), -7, dtype=torch.int32, device=dev)
    ev.place_async(bad, qp, 0, True, out=out, status=s[1:2])
    ev.place_async(qp, qp, 0, True, status=s[2:3])
    torch.cuda.synchronize()
    codes = s.cpu().numpy()
    assert codes[0] == aladdin.ALD_OK and codes[1] == aladdin.ALD_EINVAL and codes[2] == aladdin.ALD_EBLOCKED, codes
    assert (out.cpu().numpy() == -7).all()  # nothing written
    # the failed call's error is reported once, then the handle works from where it stood
    with pytest.raises(aladdin.AladdinError) as e:
        ev.resume()
    assert e.value.code == aladdin.ALD_EINVAL
    after = ev.summary()
    for f in before:
        assert np.array_equal(before[f], after[f]), f
    with pytest.raises(aladdin.AladdinError) as e:
        ev.place_async(qp, qp, 0, True, status=s[0:1], spare_rounds=-1)
    assert e.value.code == aladdin.ALD_EINVAL
    got = ev.place(t.q_l_in, t.q_l_pred, heartbeat_every=0, diag=False)
    ev.close()
    want = ref.place_trace(t, heartbeat_every=0)
    assert np.array_equal(got.worker, want.worker)


def mini_sweep(seed, Q):
    return wl.make_sweep("mini-hb", seed, Q=Q, worker_counts=(1, 2, 3, 5, 16, 40), gpu_counts=(1, 2),
                         base_capacity=65536, model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)


def check_sweep(aladdin, s, got, H):
    rej, first, ow, best, status = got
    assert int(status.item()) == aladdin.ALD_OK
    S, Q = len(s.scenarios), len(s.q_l_in)
    orej, ofirst, oworkers = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, heartbeat_every=H,
                                       n_threads=4)
    assert np.array_equal(ow.cpu().numpy()[:S * Q].reshape(S, Q), oworkers)
    assert np.array_equal(rej.cpu().numpy(), orej)
    assert np.array_equal(first.cpu().numpy(), ofirst)
    b = best.cpu().numpy()
    assert ((None, -1) if b[0] < 0 else (int(b[0]), int(b[1]))) == ref.min_gpus(s.scenarios, orej)


def test_async_sweeps_back_to_back_match_oracle(aladdin):
    import torch
    s1, s2 = mini_sweep(21, 2500), mini_sweep(22, 1800)
    H2 = np.array([0, 1, 2, 7, 25, 64, 100, 333, 1000, 1799, 1800, 5000], np.int32)
    ev = aladdin.Evaluator(0, tile=1024)
    dev = ev.device
    q1 = [torch.as_tensor(x, dtype=torch.int32, device=dev) for x in (s1.q_l_in, s1.q_l_pred)]
    q2 = [torch.as_tensor(x, dtype=torch.int32, device=dev) for x in (s2.q_l_in, s2.q_l_pred)]
    # two sweeps in flight: the second lays its tables over the first's, after it on the stream
    g1 = ev.sweep_async(s1.scenarios, *q1, want_workers=True, spare_rounds=256)
    g2 = ev.sweep_async(s2.scenarios, *q2, want_workers=True, heartbeat_every=H2, spare_rounds=256)
    torch.cuda.synchronize()
    check_sweep(aladdin, s1, g1, None)
    check_sweep(aladdin, s2, g2, H2)
    # Long tiles on small clusters that fill up: the synchronous sweep cuts
    # tiles (its tile statistics say so), and without heartbeats every
    # scenario has the same tiles, so a sweep with no spare round cannot finish
    s3 = wl.make_sweep("async-cuts", 23, Q=3000, worker_counts=(6, 12, 40), gpu_counts=(1,), base_capacity=8000,
                       model=wl.BASE_MODEL, in_dist=wl.SHORT_IN, out_dist=wl.SHORT_OUT, rate=None)
    ev3 = aladdin.Evaluator(0, tile=4096)
    ev3.sweep(s3.scenarios, s3.q_l_in, s3.q_l_pred)
    st = ev3.tile_stats()
    print("sweep tile statistics", st, flush=True)
    assert st["cuts"] > 0
    q3 = [torch.as_tensor(x, dtype=torch.int32, device=dev) for x in (s3.q_l_in, s3.q_l_pred)]
    g = ev3.sweep_async(s3.scenarios, *q3, want_workers=True, spare_rounds=0)
    torch.cuda.synchronize()
    assert int(g[4].item()) == aladdin.ALD_EINCOMPLETE
    g = ev3.sweep_async(s3.scenarios, *q3, want_workers=True, spare_rounds=int(st["cuts"]))
    torch.cuda.synchronize()
    check_sweep(aladdin, s3, g, None)
    ev3.close()
    # a query length outside [1, 2^24]
    bad = q1[0].clone()
    bad[5] = 0
    g = ev.sweep_async(s1.scenarios, bad, q1[1], spare_rounds=4)
    torch.cuda.synchronize()
    assert int(g[4].item()) == aladdin.ALD_EINVAL
    with pytest.raises(aladdin.AladdinError) as e:
        ev.sweep_async(s1.scenarios, *q1, spare_rounds=-1)
    assert e.value.code == aladdin.ALD_EINVAL
    ev.close()


def test_async_chain_in_sorted_layout_matches_oracle(aladdin):
    # calls of at least 16,384 queries evaluate in l_pred order; rounds run
    # out (no spare rounds) and the stopped call is resumed
    t = trace(40, 3, 54000, 8000, 9500)
    want = ref.place_trace(t, heartbeat_every=0)
    ev = aladdin.Evaluator(0, tile=65536)
    ev.load_trace(t)
    got_w, got_d, short = run_async_chain(aladdin, ev, t, 0, chunks(54000, 3), 0)
    summ = ev.summary()
    ev.close()
    assert short > 0
    compare(got_w, got_d, summ, want, 0, 54000)


def test_async_calls_with_changing_heartbeat_periods_match_sync(aladdin):
    # the host projects the stream position of every asynchronous call
    # (heartbeats inside the call, and one already due when a call with a
    # shorter period starts); the first synchronous call afterwards checks the
    # projection against the device and fails on a difference
    import torch
    t = trace(16, 4, 2400, 30000, 9600)
    parts = [(0, 500, 50), (500, 900, 20), (900, 1300, 0), (1300, 1800, 37), (1800, 2400, 64)]
    res = []
    for mode in ("sync", "async"):
        ev = aladdin.Evaluator(0, tile=4096)
        ev.load_trace(t)
        dev = ev.device
        ql = torch.as_tensor(t.q_l_in, dtype=torch.int32, device=dev)
        qp = torch.as_tensor(t.q_l_pred, dtype=torch.int32, device=dev)
        out = torch.full((2400,), -7, dtype=torch.int32, device=dev)
        dg = torch.zeros(2400 * 40, dtype=torch.uint8, device=dev)
        s = torch.full((len(parts),), SENTINEL, dtype=torch.int32, device=dev)
        for k, (a, b, H) in enumerate(parts):
            if mode == "sync":
                ev.place_device(ql[a:b], qp[a:b], H, True, out[a:b], dg[a * 40:b * 40])
            else:
                ev.place_async(ql[a:b], qp[a:b], H, True, out[a:b], dg[a * 40:b * 40], s[k:k + 1],
                               spare_rounds=4096)
        summ = ev.summary()  # settles the asynchronous calls
        if mode == "async":
            assert (s.cpu().numpy() == aladdin.ALD_OK).all(), s
        res.append((out.cpu().numpy(), dg.cpu().numpy(), summ))
        ev.close()
    assert np.array_equal(res[0][0], res[1][0])
    assert np.array_equal(res[0][1], res[1][1])
    for f in res[0][2]:
        assert np.array_equal(res[0][2][f], res[1][2][f]), f
