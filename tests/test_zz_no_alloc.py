"""The allocation-free Algorithm 2 entry point (ald_rebalance_noalloc) against
ald_rebalance, through the C ABI (needs an MI355X).

Both run the same kernels on the same inputs; the allocation-free one keeps
its tables in the library's fixed device array instead of handle memory.  Two
calls in a row, the second with a smaller input, so that the second one runs
on the array as the first left it.  Everything is integer: outputs must be
identical."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu


def run(fn, h, b, dev):
    import torch

    from paper_2405_06856_amd import aladdin
    d32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32).to(dev)
    P = b.P
    Wt = int(np.sum(b.n_workers))
    models = (aladdin.Model * P)(*[aladdin.to_model(m) for m in b.models])
    nw = d32(b.new_worker)
    le = torch.full((Wt,), 7, dtype=torch.int64, device=dev)  # not zero: the call clears them
    be = torch.full((Wt,), -7, dtype=torch.int64, device=dev)
    mv = torch.empty(P, dtype=torch.int32, device=dev)
    obj = torch.empty(4 * P, dtype=torch.int64, device=dev)
    cap = int(4 * np.diff(b.new_offsets).max() + int(np.max(b.n_workers)))
    log = torch.empty(max(1, 2 * P * cap), dtype=torch.int32, device=dev)
    fn(h, P, b.n_workers, models, b.old_offsets, d32(b.old_worker), d32(b.old_l_pred), d32(b.old_l_out),
       d32(b.old_l_real), d32(b.old_l_repred), b.new_offsets, d32(b.new_l_pred), nw, le, be, mv, cap, log, obj)
    torch.cuda.synchronize()
    k = mv.cpu().numpy()
    lg = log.cpu().numpy()
    logs = [lg[2 * p * cap:2 * p * cap + 2 * int(k[p])].tolist() for p in range(P)]
    return {"worker": nw.cpu().numpy(), "le": le.cpu().numpy(), "be": be.cpu().numpy(), "moves": k,
            "obj": obj.cpu().numpy(), "logs": logs}


def test_noalloc_matches_allocating_entry_point():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin
    dev = torch.device("cuda", 0)
    h = aladdin.ald_create(0, torch.cuda.current_stream(dev).cuda_stream)
    ws = torch.empty(64 << 20, dtype=torch.uint8, device=dev)  # ald_rebalance's tables
    aladdin.ald_set_workspace(h, ws)
    try:
        big = wl.make_rebalance("noalloc big", 91, 24, 48, 20, 600, sigma_err=0.7)
        small = wl.make_rebalance("noalloc small", 92, 3, 9, 6, 40, sigma_err=0.6)
        for b in (big, small):
            print("noalloc case P=%d new=%d" % (b.P, int(b.new_offsets[-1])), flush=True)
            want = run(aladdin.ald_rebalance, h, b, dev)
            got = run(aladdin.ald_rebalance_noalloc, h, b, dev)
            for key in ("worker", "le", "be", "moves", "obj"):
                assert np.array_equal(got[key], want[key]), key
            assert got["logs"] == want["logs"]
            assert int(want["moves"].sum()) > 0
    finally:
        aladdin.ald_destroy(h)


def test_noalloc_rejects_what_does_not_fit():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin
    dev = torch.device("cuda", 0)
    h = aladdin.ald_create(0, torch.cuda.current_stream(dev).cuda_stream)
    try:
        b = wl.make_rebalance("noalloc tiny", 93, 2, 4, 3, 10)
        d32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32).to(dev)
        models = (aladdin.Model * b.P)(*[aladdin.to_model(m) for m in b.models])
        args = (h, b.P, b.n_workers, models, b.old_offsets, d32(b.old_worker), d32(b.old_l_pred), d32(b.old_l_out),
                d32(b.old_l_real), d32(b.old_l_repred), b.new_offsets, d32(b.new_l_pred), d32(b.new_worker))
        with pytest.raises(aladdin.AladdinError) as e:
            aladdin.ald_rebalance_noalloc(*args, None, None)  # no error arrays of the caller's
        assert e.value.code == aladdin.ALD_EINVAL
        # more problems than the fixed array holds
        P = 4097
        models_p = (aladdin.Model * P)(*([aladdin.to_model(b.models[0])] * P))
        z = torch.zeros(1, dtype=torch.int32, device=dev)
        le = torch.zeros(P, dtype=torch.int64, device=dev)
        with pytest.raises(aladdin.AladdinError) as e:
            aladdin.ald_rebalance_noalloc(h, P, np.ones(P, np.int32), models_p, np.zeros(P + 1, np.int64), z, z, z, z,
                                          z, np.zeros(P + 1, np.int64), z, z, le, le)
        assert e.value.code == aladdin.ALD_EINVAL
    finally:
        aladdin.ald_destroy(h)
