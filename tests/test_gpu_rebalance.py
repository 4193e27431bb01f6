"""Algorithm 2 (re-balancing) on the GPU vs the CPU oracle (needs an MI355X).

Everything is integer, so the new workers, per-worker errors, move logs and
objectives must match the oracle exactly."""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest

from oracle import ref
from paper_2405_06856_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2405_06856_amd import aladdin
    e = aladdin.Evaluator(0)
    yield e
    e.close()


def say(*a):
    print(*a, flush=True)


def check_against_oracle(batch, got, problems=None):
    wb = np.concatenate([[0], np.cumsum(batch.n_workers)])
    for p in (range(batch.P) if problems is None else problems):
        W = int(batch.n_workers[p])
        want = ref.rebalance(*batch.problem(p))
        n0, n1 = int(batch.new_offsets[p]), int(batch.new_offsets[p + 1])
        k = len(want.moves)
        assert got["worker"][n0:n1].tolist() == want.worker.tolist(), "problem %d: workers differ" % p
        assert got["le"][wb[p]:wb[p] + W].tolist() == want.le.tolist(), "problem %d: l^e differs" % p
        assert got["be"][wb[p]:wb[p] + W].tolist() == want.be.tolist(), "problem %d: b^e differs" % p
        assert int(got["moves"][p]) == k
        assert got["obj"][p].tolist() == [*want.obj_before, *want.obj_after]
        if "log" in got:
            assert got["log"][p].tolist() == want.moves.tolist()


SMALL = [
    # (name, P, W, R, n_new, sigma_err)
    ("one worker", 2, 1, 5, 9, 0.5),
    ("tiny", 3, 5, 4, 11, 0.8),
    ("mixed sizes", 4, [3, 64, 17, 1], [0, 9, 40, 3], [50, 0, 300, 7], 0.6),
    ("several waves of requests", 2, 33, 20, 2000, 0.7),
    ("many workers", 1, 4096, 2, 64, 0.9),
    ("3000 new requests", 2, 24, 6, [3000, 40], 0.7),
    ("most new requests", 1, 40, 8, 8192, 0.7),
    ("no prediction error", 2, 16, 30, 100, 0.0),
    # the largest problem the library takes (4096 workers, 8192 new requests):
    # the moves kernel's LDS at its maximum
    ("largest problem", 2, [4096, 8], [1, 3], [8192, 10], 0.02),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_rebalance_matches_oracle(ev, case):
    name, P, W, R, n_new, sig = case
    say("rebalance case", name)
    b = wl.make_rebalance(name, 40 + SMALL.index(case), P, W, R, n_new, sigma_err=sig)
    got = ev.rebalance(b, want_log=True)
    check_against_oracle(b, got)


def test_rebalance_models_per_problem(ev):
    """Each problem takes its own rho = c2 / k2, the real ratio of two doubles
    (not whole tokens): 0, about 150, 500.025, 2000 and exactly 500.5."""
    from fractions import Fraction
    b = wl.make_rebalance("rho", 7, 5, 24, 12, 400, sigma_err=0.7)
    base = b.models[0]
    b.models = [dataclasses.replace(base, c2=c2) for c2 in (0.0, 3e-5, 1.00005e-4, 4e-4)]
    b.models.append(dataclasses.replace(base, k2=2.0 ** -22, c2=1001 * 2.0 ** -23))
    rhos = [Fraction(m.c2) / Fraction(m.k2) for m in b.models]
    assert rhos[4] == Fraction(1001, 2) and abs(rhos[2] - Fraction(500025, 1000)) < Fraction(1, 10 ** 9)
    assert sum(r.denominator != 1 for r in rhos) >= 3
    got = ev.rebalance(b, want_log=True)
    check_against_oracle(b, got)


def test_rebalance_extreme_rho(ev):
    """rho exactly 500 (pairs such as (1000, 0) and (500, 1) then tie exactly,
    and the lowest index decides), about 10^9 (the largest ratio taken) and
    10^-12 (the batch term only breaks ties of lengths)."""
    from fractions import Fraction
    b = wl.make_rebalance("extreme rho", 61, 3, [40, 40, 40], [12, 12, 12], [300, 300, 300], sigma_err=0.7)
    base = b.models[0]
    b.models = [dataclasses.replace(base, k2=2.0 ** -22, c2=500 * 2.0 ** -22),
                dataclasses.replace(base, k2=1e-12, c2=999999999.5e-12),
                dataclasses.replace(base, k2=1.0, c2=1e-12)]
    rhos = [Fraction(m.c2) / Fraction(m.k2) for m in b.models]
    assert rhos[0] == 500 and abs(rhos[1] - 10 ** 9) < 1 and rhos[2] < Fraction(1, 10 ** 11)
    got = ev.rebalance(b, want_log=True)
    assert int(got["moves"].sum()) > 0
    check_against_oracle(b, got)


def test_rebalance_full_size(ev):
    """The 256-problem workload in the launch the benchmark times: every 16th
    problem against the oracle (the exhaustive oracle takes about half a second
    per problem), and on all of them the invariants (a move keeps sum l^e and
    sum b^e, the objective never grows)."""
    from fractions import Fraction
    b = wl.make_config("rebalance")
    say("rebalance full size", b.P)
    got = ev.rebalance(b, want_log=True)
    check_against_oracle(b, got, problems=range(0, b.P, 16))
    wb = np.concatenate([[0], np.cumsum(b.n_workers)])
    rho = Fraction(b.models[0].c2) / Fraction(b.models[0].k2)
    assert rho.denominator != 1  # the workload's rho is not a whole number of tokens
    for p in range(b.P):
        o = [int(x) for x in got["obj"][p]]
        assert o[2] + rho * o[3] <= o[0] + rho * o[1]
    assert int(got["moves"].sum()) > 0
    # a move takes its request's length and one batch slot from one worker to
    # another: the sums of l^e and of b^e over a problem's workers do not change
    for p in range(b.P):
        n0, n1 = int(b.new_offsets[p]), int(b.new_offsets[p + 1])
        changed = got["worker"][n0:n1] != b.new_worker[n0:n1]
        assert int(changed.sum()) <= int(got["moves"][p])
        want = ref.rebalance(*b.problem(p)[:7], [], [])  # the errors alone, no new requests
        assert int(got["le"][wb[p]:wb[p + 1]].sum()) == int(want.le.sum())
        assert int(got["be"][wb[p]:wb[p + 1]].sum()) == int(want.be.sum())


def test_rebalance_twice_in_a_row(ev):
    """Tables and error arrays are reused between calls of different sizes."""
    b1 = wl.make_rebalance("a", 11, 6, 50, 10, 700)
    b2 = wl.make_rebalance("b", 12, 2, 9, 3, 40)
    check_against_oracle(b1, ev.rebalance(b1, want_log=True))
    check_against_oracle(b2, ev.rebalance(b2, want_log=True))
    check_against_oracle(b1, ev.rebalance(b1))


def test_rebalance_invalid_input_changes_nothing(ev):
    from paper_2405_06856_amd import aladdin
    b = wl.make_rebalance("bad", 13, 3, 8, 5, 30)
    k = int(b.old_offsets[2]) + 1  # a request of the last problem
    b.old_l_out = b.old_l_out.copy()
    b.old_l_out[k] = b.old_l_real[k] + 1  # more tokens generated than the real length
    with pytest.raises(aladdin.AladdinError) as e:
        ev.rebalance(b)
    assert e.value.code == aladdin.ALD_EINVAL
    b2 = wl.make_rebalance("bad2", 14, 2, 8, 5, 30)
    b2.new_worker = b2.new_worker.copy()
    b2.new_worker[3] = 8  # worker out of range
    import torch
    t = torch
    nw = t.as_tensor(b2.new_worker).to(ev.device)
    before = nw.clone()
    models = (aladdin.Model * b2.P)(*[aladdin.to_model(m) for m in b2.models])
    d = lambda a: t.as_tensor(a, dtype=t.int32).to(ev.device)
    with pytest.raises(aladdin.AladdinError):
        aladdin.ald_rebalance(ev.h, b2.P, b2.n_workers, models, b2.old_offsets, d(b2.old_worker), d(b2.old_l_pred),
                              d(b2.old_l_out), d(b2.old_l_real), d(b2.old_l_repred), b2.new_offsets,
                              d(b2.new_l_pred), nw)
    assert t.equal(nw, before)
    # host-side checks: too many workers, a model without decode slope
    b3 = wl.make_rebalance("big", 15, 1, 4097, 0, 1)
    with pytest.raises(aladdin.AladdinError):
        ev.rebalance(b3)
    b4 = wl.make_rebalance("k2", 16, 1, 4, 2, 3)
    b4.models = [dataclasses.replace(b4.models[0], k2=0.0)]
    with pytest.raises(aladdin.AladdinError):
        ev.rebalance(b4)


@pytest.mark.parametrize("seed", range(16))
def test_random_rebalance_matches_oracle(ev, seed):
    """Random batches: problem counts, per-problem sizes, error spreads,
    unplaced shares and per-problem rho."""
    rng = np.random.default_rng(9400 + seed)
    P = int(rng.integers(1, 20))
    W = [int(x) for x in rng.choice([1, 2, 3, 9, 40, 300], P)]
    R = [int(x) for x in rng.choice([0, 1, 7, 60], P)]
    n_new = [int(x) for x in rng.choice([0, 1, 5, 80, 600], P)]
    b = wl.make_rebalance("random%d" % seed, 9450 + seed, P, W, R, n_new,
                          sigma_err=float(rng.choice([0.0, 0.3, 0.8, 1.5])), unplaced=float(rng.choice([0.0, 0.1, 0.5])))
    if rng.random() < 0.5:
        base = b.models[0]
        b.models = [dataclasses.replace(base, c2=float(rng.choice([0.0, 3e-5, 1e-4, 4e-4, 1.7e-5])),
                                        k2=float(rng.choice([2e-7, 3.1e-7]))) for _ in range(P)]
    say("random rebalance", seed, "P", P, "W", W[:6], "new", n_new[:6])
    got = ev.rebalance(b, want_log=True)
    check_against_oracle(b, got)
