"""Write the stored expected results of the three large workloads.

Every value written here comes from the CPU oracle (``oracle/``) run on the
seeded workload generator; nothing comes from the GPU library.  The files are
digests (sha256 of the little-endian bytes of each output array) plus a sample
of full records, so that a GPU run can be compared bit for bit without running
the minutes-long oracle again.

    python tests/golden/make_golden.py [large|long|sweep ...] [--threads N]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import ref  # noqa: E402
from paper_2405_06856_amd import workloads as wl  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def digest(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def trace_digest(t) -> str:
    h = hashlib.sha256()
    for a in (t.kv_capacity, t.res_offsets, t.res_l_in, t.res_l_pred, t.res_generated, t.q_l_in, t.q_l_pred):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def sweep_digest(s) -> str:
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(s.q_l_in).tobytes())
    h.update(np.ascontiguousarray(s.q_l_pred).tobytes())
    for sc in s.scenarios:
        m = sc.model
        h.update(np.array([sc.n_workers, sc.gpus_per_worker, sc.kv_capacity], np.int64).tobytes())
        h.update(np.array([m.c1, m.k1, m.k1q, m.c3, m.c2, m.k2, m.ttft_slo, m.decode_slo, m.theta],
                          np.float64).tobytes())
    return h.hexdigest()


QUERY_FIELDS = ("worker", "n_feasible", "near_tie", "kv_peak_chosen", "kv_excess_min", "ttft_chosen",
                "tdec_chosen")
WORKER_FIELDS = ("B", "sum_c", "sum_r", "peak", "S1", "S2")


def sample_indices(Q: int, n: int = 64) -> np.ndarray:
    idx = np.unique(np.concatenate([np.arange(min(8, Q)), np.linspace(0, Q - 1, n).astype(np.int64)]))
    return idx


def record(res, idx):
    out = {"index": [int(i) for i in idx]}
    for f in QUERY_FIELDS:
        a = getattr(res, f)[idx]
        out[f] = [float(x).hex() for x in a] if a.dtype == np.float64 else [int(x) for x in a]
    return out


def make_place(name: str, threads: int):
    t = wl.make_config(name)
    t0 = time.time()
    res = ref.place_trace(t, n_threads=threads)
    dt = time.time() - t0
    placed = res.worker >= 0
    doc = {
        "what": "oracle results for workloads.make_config(%r)" % name,
        "written_by": "tests/golden/make_golden.py (oracle only)",
        "numpy": np.__version__,
        "inputs_sha256": trace_digest(t),
        "n_workers": t.n_workers, "n_queries": t.n_queries, "heartbeat_every": t.heartbeat_every,
        "placed": int(placed.sum()),
        "first_placed": int(np.argmax(placed)) if placed.any() else -1,
        "pairs": int(t.n_workers) * int(t.n_queries),
        "sha256": {f: digest(getattr(res, f)) for f in QUERY_FIELDS + WORKER_FIELDS},
        "sample": record(res, sample_indices(t.n_queries)),
        "oracle_seconds": round(dt, 1), "oracle_threads": threads,
    }
    with open(os.path.join(HERE, "%s_oracle.json" % name), "w") as f:
        json.dump(doc, f, indent=1)
    print(name, "placed", doc["placed"], "first", doc["first_placed"], "%.1fs" % dt, flush=True)


def make_sweep(threads: int):
    s = wl.make_config("sweep")
    t0 = time.time()
    rej, first, workers = ref.sweep(s.scenarios, s.q_l_in, s.q_l_pred, want_workers=True, n_threads=threads)
    dt = time.time() - t0
    gpus, idx = ref.min_gpus(s.scenarios, rej)
    doc = {
        "what": "oracle results for workloads.make_config('sweep')",
        "written_by": "tests/golden/make_golden.py (oracle only)",
        "numpy": np.__version__,
        "inputs_sha256": sweep_digest(s),
        "n_scenarios": len(s.scenarios), "n_queries": s.n_queries,
        "rejected": [int(x) for x in rej],
        "first_reject": [int(x) for x in first],
        "min_gpus": gpus, "min_gpus_scenario": idx,
        "min_gpus_ties": [i for i, (sc, r) in enumerate(zip(s.scenarios, rej))
                          if r == 0 and gpus is not None and sc.n_workers * sc.gpus_per_worker == gpus],
        "sha256": {"worker": digest(workers)},
        "oracle_seconds": round(dt, 1), "oracle_threads": threads,
    }
    with open(os.path.join(HERE, "sweep_oracle.json"), "w") as f:
        json.dump(doc, f, indent=1)
    print("sweep min_gpus", gpus, "scenario", idx, "%.1fs" % dt, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("configs", nargs="*", default=["large", "sweep", "long"])
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    a = ap.parse_args()
    ref.build()
    for c in a.configs:
        if c == "sweep":
            make_sweep(a.threads)
        else:
            make_place(c, a.threads)


if __name__ == "__main__":
    main()
