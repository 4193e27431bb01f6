"""The caller-owned workspace (needs an MI355X): the library allocates no
device memory, calls run entirely from the workspace the caller attaches, a
call that does not fit is refused with ALD_ESPACE before doing anything, and
the loaded state moves with the workspace."""
from __future__ import annotations

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


def test_planned_size_is_enough(aladdin):
    """ald_workspace_size's figure runs the load and a whole-stream placement
    with diagnostics and per-query heartbeats without a refusal."""
    import torch
    t = wl.make_config("medium")
    ev = aladdin.Evaluator(0, tile=1024)
    n = aladdin.ald_workspace_size(ev.h, t.n_workers, int(t.res_offsets[-1]), aladdin.to_model(t.model), 0, False,
                                   t.n_queries)
    say("medium planned workspace", n)
    ws = torch.empty(n, dtype=torch.uint8, device=ev.device)
    aladdin.ald_set_workspace(ev.h, ws, n)
    ev.ws, ev.ws_bytes = ws, n
    ev.load_trace(t)
    got = ev.place(t.q_l_in, t.q_l_pred, 0, diag=True)
    assert ev.ws is ws  # no growth
    hb = np.zeros(t.n_queries, np.int32)
    hb[::97] = 1
    ev.load_trace(t)
    got_hb = ev.place(t.q_l_in, t.q_l_pred, hb_before=hb)
    assert ev.ws is ws
    ev.close()
    want = ref.place_trace(t)
    assert np.array_equal(got.worker, want.worker)
    assert np.array_equal(got.diag["kv_excess_min"], want.kv_excess_min)
    want_hb = ref.place_hb(t.n_workers, t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated,
                           t.model, t.q_l_in, t.q_l_pred, hb)
    assert np.array_equal(got_hb.worker, want_hb.worker)


def test_too_small_is_refused_and_reports_the_need(aladdin):
    import torch
    t = wl.make_config("tiny")
    ev = aladdin.Evaluator(0, tile=64)
    small = torch.empty(4096, dtype=torch.uint8, device=ev.device)
    aladdin.ald_set_workspace(ev.h, small)
    with pytest.raises(aladdin.AladdinError) as e:
        aladdin.ald_load_workers(ev.h, t.n_workers, aladdin.to_model(t.model),
                                 *[ev._dev(a, d) for a, d in ((t.kv_capacity, torch.int64), (t.res_offsets, torch.int64),
                                                              (t.res_l_in, torch.int32), (t.res_l_pred, torch.int32),
                                                              (t.res_generated, torch.int32))])
    assert e.value.code == aladdin.ALD_ESPACE
    need = aladdin.ald_workspace_needed(ev.h)
    assert need > 4096
    with pytest.raises(aladdin.AladdinError) as e:  # still nothing loaded
        ev.place(t.q_l_in, t.q_l_pred, 0)
    assert e.value.code == aladdin.ALD_ESTATE
    big = torch.empty(need, dtype=torch.uint8, device=ev.device)
    aladdin.ald_set_workspace(ev.h, big)
    ev.ws, ev.ws_bytes = big, need
    ev.load_trace(t)  # fits exactly
    assert ev.ws is big
    got = ev.place(t.q_l_in, t.q_l_pred, 0)  # grown by the Evaluator if the call needs more
    assert ev.ws_bytes >= need
    ev.close()
    assert np.array_equal(got.worker, ref.place_trace(t).worker)


def test_state_moves_with_the_workspace(aladdin):
    """Half a stream, a new workspace (the old one overwritten and released),
    the other half: the same placements as one run."""
    import torch
    t = wl.make_config("medium")
    ev = aladdin.Evaluator(0, tile=512)
    ev.load_trace(t)
    h = t.n_queries // 2
    a = ev.place(t.q_l_in[:h], t.q_l_pred[:h], 0)
    old = ev.ws
    ev.attach_workspace(ev.ws_bytes * 2)
    old.fill_(0xA5)  # the state was copied out before the stream reached this
    del old
    b = ev.place(t.q_l_in[h:], t.q_l_pred[h:], 0)
    summ = ev.summary()
    ev.close()
    want = ref.place_trace(t)
    assert np.array_equal(np.concatenate([a.worker, b.worker]), want.worker)
    assert np.array_equal(summ["B"].astype(np.int64), want.B)
    assert np.array_equal(summ["peak"].astype(np.int64), want.peak)


def test_sweep_planned_size(aladdin):
    import torch
    s = wl.make_sweep("ws-sweep", 21, Q=600, worker_counts=(2, 5, 16), gpu_counts=(1, 2), base_capacity=20000,
                      model=wl.BASE_MODEL, in_dist=wl.MID_IN, out_dist=wl.MID_OUT, rate=None)
    ev = aladdin.Evaluator(0, tile=256)
    arr = (aladdin.Scenario * len(s.scenarios))()
    for i, sc in enumerate(s.scenarios):
        arr[i] = aladdin.Scenario(sc.n_workers, sc.gpus_per_worker, sc.kv_capacity, aladdin.to_model(sc.model))
    n = aladdin.ald_sweep_workspace_size(ev.h, len(s.scenarios), arr, s.n_queries)
    ws = torch.empty(n, dtype=torch.uint8, device=ev.device)
    aladdin.ald_set_workspace(ev.h, ws, n)
    ev.ws, ev.ws_bytes = ws, n
    rej, first, _, best = ev.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_answer=True)
    assert ev.ws is ws
    ev.close()
    orej, ofirst, _ = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred)
    assert np.array_equal(rej, orej) and np.array_equal(first, ofirst)
    assert best == ref.min_gpus(s.scenarios, orej)
