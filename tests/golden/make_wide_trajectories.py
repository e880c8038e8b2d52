"""Write tests/golden/wide_trajectories.json: the fp64 oracle's free-running ALS trajectory
(training RMSE after every half-sweep, paper Sec. 2.2 for the alternation and Sec. 4.1 for
the RMSE) on the two wide full-size workloads, so that the GPU test can compare its own
trajectory without running hours of host fp64 work on the GPU host.

    python tests/golden/make_wide_trajectories.py [--threads N] [--configs 4 5]

Only ``workload`` (the seeded inputs) and ``oracle`` are called. Each entry stores the
SHA-256 of the inputs the trajectory was computed from (row_ptr, col, val, U0, V0), so a
change of the generator makes the test fail instead of comparing against stale values.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workload  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "wide_trajectories.json")


def input_digests(r, U0, V0) -> dict:
    """SHA-256 of the exact bytes both implementations read."""
    out = {}
    for name, a in (("row_ptr", r.row_ptr), ("col", r.col), ("val", r.val), ("U0", U0),
                    ("V0", V0)):
        out[name] = hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
    return out


def trajectory(k: int, threads: int) -> dict:
    t0 = time.time()
    r = workload.make_config(k)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    print(f"{r.name}: generated in {time.time() - t0:.1f} s", flush=True)
    entry = {
        "name": r.name, "M": r.M, "N": r.N, "nnz": r.nnz, "D": r.D, "lambda": r.lam,
        "sweeps": r.sweeps, "order": "items then users",
        "sha256": input_digests(r, U0, V0),
        "rmse_after_items": [], "rmse_after_users": [], "flagged": [],
    }
    t = oracle.Trajectory(r.M, r.N, r.row_ptr, r.col, r.val, U0, V0, r.lam, threads=threads)
    for sweep in range(1, r.sweeps + 1):
        for side in ("items", "users"):
            ts = time.time()
            t.step(side)
            rm = t.rmse()
            entry[f"rmse_after_{side}"].append(rm)
            entry["flagged"].append(t.nflag)
            print(f"  sweep {sweep} {side}: rmse {rm:.12f} flagged {t.nflag} "
                  f"({time.time() - ts:.0f} s)", flush=True)
    return entry


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=0)
    ap.add_argument("--configs", type=int, nargs="+", default=[4, 5])
    a = ap.parse_args()
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            data = json.load(f)
    data["_about"] = ("fp64 oracle ALS trajectories (training RMSE after every half-sweep, "
                      "items then users) written by tests/golden/make_wide_trajectories.py "
                      "from oracle/ and workload/ only")
    for k in a.configs:
        data[str(k)] = trajectory(k, a.threads)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)
            f.write("\n")
        print(f"wrote {OUT} (config {k})", flush=True)


if __name__ == "__main__":
    main()
