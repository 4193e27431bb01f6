"""The oracle's pins have teeth: plant one plausible mistake at a time in a copy
of the oracle's C source (never in the oracle itself), build it, and require
that at least one pin of ``test_oracle.py`` fails against it (CPU only)."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

from oracle import ref
from tests import test_oracle as pins

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = open(ref.SRC).read()

# (name, original text, planted mistake)
MUTANTS = [
    ("kv end point one iteration early", "int64_t d_ = sumc + cnt * (t);", "int64_t d_ = sumc + cnt * ((t) - 1);"),
    ("query's own end point not checked", "sumc += cq; cnt += 1;\n        DEMAND_AT(rq);", "sumc += cq; cnt += 1;"),
    ("generated tokens not in the context", "add_request(&ws[i], lin + g, lp - g,", "add_request(&ws[i], lin, lp - g,"),
    ("remaining length ignores generated tokens", "add_request(&ws[i], lin + g, lp - g,",
     "add_request(&ws[i], lin + g, lp,"),
    ("batch size without the query", "const int64_t b = B + 1;", "const int64_t b = B;"),
    ("gamma applied to the context", "const int64_t DS = SC * ((int64_t)1 << gs) + gn * SR;",
     "const int64_t DS = SC * gn + SR * ((int64_t)1 << gs);"),
    ("TTFT without the query's prefill", "const int64_t S1 = w->S1 + lin;", "const int64_t S1 = w->S1;"),
    ("quadratic prefill term linear", "const int64_t S2 = w->S2 + lin * lin;", "const int64_t S2 = w->S2 + lin;"),
    ("ties to the highest index", "    return a < b;\n}", "    return a > b;\n}"),
    ("rank key after placement", "(unsigned __int128)(B * ((int64_t)1 << gs));",
     "(unsigned __int128)((B + 1) * ((int64_t)1 << gs));"),
    ("heartbeat keeps the prefill sums", "    w->S1 = 0;\n    w->S2 = 0;\n}", "}"),
    ("heartbeat evicts one iteration early", "if (w->r[i] >= 0) { keep = i + 1;", "if (w->r[i] > 0) { keep = i + 1;"),
    ("heartbeat does not grow contexts", "        w->c[i] += 1;\n", ""),
    ("near tie absolute", "return fabs(x - y) <= 1e-9 * m;", "return fabs(x - y) <= 1e-9;"),
    ("KV check strict", "o->kv_ok = o->peak <= w->M;", "o->kv_ok = o->peak < w->M;"),
    ("decode check strict", "o->dec_ok = o->lhs <= o->rhs;", "o->dec_ok = o->lhs < o->rhs;"),
    ("TTFT check strict", "o->ttft_ok = decode_only || o->ttft <= m->ttft_slo;",
     "o->ttft_ok = decode_only || o->ttft < m->ttft_slo;"),
    ("heartbeat counts only placements", "if (H > 0 && !no_commit) {\n            since_hb += 1;",
     "if (H > 0 && !no_commit && best >= 0) {\n            since_hb += 1;"),
    ("chosen decode time without the query's batch slot", "o->tdec = (m->c3 + m->c2 * (double)b) + m->k2 * sumD;",
     "o->tdec = (m->c3 + m->c2 * (double)B) + m->k2 * sumD;"),
    ("chosen decode time without the query's context", "o->tdec = (m->c3 + m->c2 * (double)b) + m->k2 * sumD;",
     "o->tdec = (m->c3 + m->c2 * (double)b) + m->k2 * ldexp((double)DS, -gs);"),
    ("smallest excess over feasible workers only", "if (ex < excess_min) excess_min = ex;",
     "if (pr[i].feasible && ex < excess_min) excess_min = ex;"),
    # constraint (d)
    ("(d) not part of feasibility", "o->feasible = o->kv_ok && o->dec_ok && o->ttft_ok && o->pre_ok;",
     "o->feasible = o->kv_ok && o->dec_ok && o->ttft_ok;"),
    ("(d) counts this heartbeat's requests as ongoing", "if (w->win[i] >= hb) continue;", "if (w->win[i] > hb) continue;"),
    ("(d) limit without theta", "const double lim = m->theta * smin;", "const double lim = smin;"),
    ("(d) new request starts at the worker's gain", "add_request(w, lin, lp, -w->phi, hb)", "add_request(w, lin, lp, 0.0, hb)"),
    ("(d) slack gain with the sign flipped", "w->phi = w->phi + (m->decode_slo - t_iter);",
     "w->phi = w->phi + (t_iter - m->decode_slo);"),
    ("(d) iteration time without the batch term", "(m->c3 + m->c2 * (double)w->n)", "(m->c3 + m->c2 * (double)(w->n - 1))"),
    ("(d) resident slack from the predicted length", "s0 = model->decode_slo * (double)g - res_tdec[k];",
     "s0 = model->decode_slo * (double)lp - res_tdec[k];"),
    ("one heartbeat fewer before a query", "k < hb_before[q]; ++k)", "k + 1 < hb_before[q]; ++k)"),
    ("a moved request keeps its prefill on the source", "    w->S1 -= lin;\n    w->S2 -= lin * lin;\n", ""),
    ("a moved request takes the source's slack origin", "add_request(v, lin, lp, -v->phi, hb)",
     "add_request(v, lin, lp, -w->phi, hb)"),
    # split-phase decode workers
    ("decode workers still check (d)", "if (use_d && !decode_only) {", "if (use_d) {"),
    ("decode workers flag TTFT near ties", "(!decode_only && near(o->ttft, m->ttft_slo))", "near(o->ttft, m->ttft_slo)"),
    # App. A grouped placement
    ("router splits the stream evenly", "if (!(counts[i] * Nw < h * (int64_t)N[i])) continue;",
     "if (!(counts[i] * G < h)) continue;"),
    ("router without the upper quota", "if (!(counts[i] * Nw < h * (int64_t)N[i])) continue;", ""),
    ("router ties to the highest group", "(int64_t)N[i] * (counts[best] + 1) > (int64_t)N[best] * (counts[i] + 1)",
     "(int64_t)N[i] * (counts[best] + 1) >= (int64_t)N[best] * (counts[i] + 1)"),
    ("grouped search over every worker", "            lo = gfirst[g];\n            hi = gfirst[g + 1];\n",
     "            lo = 0 * gfirst[g];\n            hi = W + 0 * gfirst[g + 1];\n"),
    # Algorithm 2
    ("A2 over-estimate error with the sign flipped", "c[i].a += (int64_t)old_lreal[j] - old_lpred[j]; c[i].b -= 1;",
     "c[i].a += (int64_t)old_lpred[j] - old_lreal[j]; c[i].b -= 1;"),
    ("A2 under-estimate counts the old prediction", "c[i].a += old_lrepred[j]; c[i].b += 1;",
     "c[i].a += old_lpred[j]; c[i].b += 1;"),
    ("A2 under-estimate test non-strict", "if (old_lout[j] > old_lpred[j])", "if (old_lout[j] >= old_lpred[j])"),
    ("A2 batch error left out of the line", "const __float128 y = (__float128)b * (__float128)m->c2;",
     "const __float128 y = 0 * (__float128)b * (__float128)m->c2;"),
    ("A2 rho rounded to whole tokens", "const __float128 y = (__float128)b * (__float128)m->c2;",
     "const __float128 y = (__float128)b * (__float128)(rint(m->c2 / m->k2) * m->k2);"),
    ("A2 a move shifts only the length", "const rb_pair d = {new_lpred[j], 1};", "const rb_pair d = {new_lpred[j], 0};"),
    ("A2 ties to the last pair", "if (rb_sign(diff.a, diff.b, m) > 0) { best = gain;",
     "if (rb_sign(diff.a, diff.b, m) >= 0 && rb_sign(gain.a, gain.b, m) > 0) { best = gain;"),
    ("A2 a request moves at most once", "        new_worker[bj] = by;\n",
     "        new_worker[bj] = by;\n        ((int32_t*)new_lpred)[bj] = 1 << 30;\n"),
    ("A2 the objective's absolute value taken on the length error only",
     "    if (rb_sign(u.a, u.b, m) < 0) { u.a = -u.a; u.b = -u.b; }",
     "    if (u.a < 0) { u.a = -u.a; u.b = -u.b; }"),
]

PINS = [
    pins.test_fig3_worked_example,
    pins.test_peak_equals_footprint_vector_sum,
    pins.test_lone_request_peak_closed_form,
    pins.test_peak_ties_and_exact_capacity,
    lambda: pins.test_placement_matches_bruteforce(0),
    lambda: pins.test_placement_matches_bruteforce(1),
    lambda: pins.test_placement_matches_bruteforce(3),
    pins.test_heartbeat_is_one_iteration_shift,
    pins.test_committed_placements_respect_every_constraint,
    pins.test_decode_margin_exactly_zero_is_feasible_and_near_tie,
    pins.test_tdec_chosen_worked_example,
    pins.test_ttft_margin_exactly_zero_is_feasible,
    pins.test_capacity_norm_ranking_picks_fullest_feasible,
    pins.test_decode_near_tie_band_is_relative,
    pins.test_capacity_norm_is_taken_before_placement,
    lambda: pins.test_preemption_limit_matches_bruteforce(0),
    lambda: pins.test_preemption_limit_matches_bruteforce(1),
    lambda: pins.test_preemption_limit_matches_bruteforce(3),
    pins.test_preemption_limit_worked_example,
    pins.test_preemption_limit_needs_an_ongoing_request,
    lambda: pins.test_heartbeats_per_query_match_bruteforce(False),
    lambda: pins.test_heartbeats_per_query_match_bruteforce(True),
    lambda: pins.test_moves_match_bruteforce(False),
    lambda: pins.test_moves_match_bruteforce(True),
    lambda: pins.test_decode_workers_match_bruteforce(0),
    lambda: pins.test_decode_workers_match_bruteforce(2),
    pins.test_router_share_within_one_query,
    pins.test_router_equal_sizes_is_round_robin_and_worked_example,
    lambda: pins.test_grouped_placement_is_each_groups_algorithm1(0),
    lambda: pins.test_grouped_placement_is_each_groups_algorithm1(7),
    pins.test_rebalance_sign_is_exact,
    pins.test_rebalance_worked_example,
    pins.test_rebalance_errors_closed_forms,
    pins.test_rebalance_request_may_move_again,
] + [lambda s=s: pins.test_rebalance_two_workers_closed_form(s) for s in range(6)] + [
    lambda s=s: pins.test_rebalance_moves_replayed_by_bruteforce(s) for s in range(25)]


def test_mutant_table_applies():
    for name, old, new in MUTANTS:
        assert SRC.count(old) >= 1, name


def first_catch(idx: int, workdir: str) -> str:
    """Build the oracle with mutant idx planted and run the pins until one
    fails; the failing pin's name, or "" when none does."""
    name, old, new = MUTANTS[idx]
    src = os.path.join(workdir, "mutant.c")
    with open(src, "w") as f:
        f.write(SRC.replace(old, new, 1))
    lib = os.path.join(workdir, "libmutant.so")
    subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
                           "-shared", "-o", lib, src, "-lm"])
    ref.SRC, ref.LIB, ref._lib = src, lib, None
    for pin in PINS:  # the first pin that fails is enough
        try:
            pin()
        except Exception as e:  # AssertionError, or an oracle error code
            return getattr(pin, "__name__", "bruteforce") + ": " + type(e).__name__
    return ""


@pytest.fixture(scope="module")
def catches(tmp_path_factory):
    """Every mutant, each in a process of its own (a few at a time)."""
    from concurrent.futures import ThreadPoolExecutor
    root = os.path.dirname(HERE)
    env = dict(os.environ, PYTHONPATH=root + os.pathsep + os.environ.get("PYTHONPATH", ""), OMP_NUM_THREADS="1")
    env.pop("ORACLE_LIB", None)

    # the directories first, in this thread: pytest's temp factory is not
    # safe to initialise from several threads at once
    dirs = [tmp_path_factory.mktemp("mutant%d" % i) for i in range(len(MUTANTS))]

    def run(idx):
        d = dirs[idx]
        out = subprocess.run([sys.executable, __file__, str(idx), str(d)], cwd=root, env=env, capture_output=True,
                             text=True, timeout=600)
        if out.returncode != 0:
            return "runner failed: " + out.stderr[-400:]
        return out.stdout.strip().splitlines()[-1] if out.stdout.strip() else ""

    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    with ThreadPoolExecutor(workers) as ex:
        return list(ex.map(run, range(len(MUTANTS))))


@pytest.mark.parametrize("idx", range(len(MUTANTS)), ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(idx, catches):
    name = MUTANTS[idx][0]
    assert catches[idx] and not catches[idx].startswith("runner failed"), \
        "no pin caught the planted mistake: %s (%s)" % (name, catches[idx])


if __name__ == "__main__":  # one mutant: python tests/test_oracle_mutants.py IDX WORKDIR
    print(first_catch(int(sys.argv[1]), sys.argv[2]))
