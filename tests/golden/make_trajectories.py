"""Write the serial oracle's test-RMSE trajectory of a workload to
tests/golden/trajectory_<label>.json.

Section 3.2.4 compares schedules by the test RMSE reached after each epoch;
the batch-Hogwild! parity tests hold the GPU library's default launch to the
serial oracle's value after the same epoch.  Only the oracle and the seeded
input generator are used here: the samples are the workload's train/test
arrays, the initial factors are the oracle's own initialisation (uniform on
[0, 1/sqrt(k)) from the workload's seed), and every epoch is one serial pass
in array order with the workload's learning-rate schedule.

The file is rewritten after every epoch, so a long run can be stopped and
its finished epochs used.

    python tests/golden/make_trajectories.py netflix 20
    python tests/golden/make_trajectories.py netflix 20 --k 32 --label netflix_k32
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_1610_05838_amd import datagen  # noqa: E402


def oracle_digest() -> str:
    with open(oracle.SRC, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("workload")
    ap.add_argument("epochs", type=int)
    ap.add_argument("--k", type=int, default=0, help="override the trained rank")
    ap.add_argument("--label", default="")
    args = ap.parse_args()

    over = {"k": args.k} if args.k else {}
    w = datagen.workload(args.workload, **over)
    label = args.label or args.workload
    path = os.path.join(HERE, f"trajectory_{label}.json")
    dt = np.float16 if w["dtype"] == "fp16" else np.float32
    t0 = time.time()
    S, T = datagen.make(w)
    P, Q = oracle.init_factors(w["m"], w["n"], w["k"], w["seed"], dt)
    rec = {
        "cite": "Section 3.2.4: test RMSE after each epoch as the convergence measure; serial SGD "
                "(section 2.2 update, samples in array order) is the reference every Hogwild! run is held to",
        "made_by": "tests/golden/make_trajectories.py (oracle/ and the seeded generator only)",
        "oracle_c_sha256_16": oracle_digest(),
        "workload": args.workload,
        "m": w["m"], "n": w["n"], "k": w["k"], "dtype": w["dtype"],
        "ntrain": w["ntrain"], "ntest": w["ntest"], "seed": w["seed"],
        "lr": w["lr"], "decay": w["decay"], "lambda": w["lam"],
        "schedule": "lr * decay^t for epoch t = 0, 1, ...",
        "rmse_init": oracle.rmse(P, Q, T),
        "rmse": [],
        "epoch_seconds": [],
    }
    print(f"[{label}] data ready in {time.time() - t0:.1f}s, initial test rmse {rec['rmse_init']:.6f}", flush=True)
    for t in range(args.epochs):
        t1 = time.time()
        oracle.epoch_serial(P, Q, S, datagen.lr_at(w, t), w["lam"], w["lam"])
        rec["rmse"].append(oracle.rmse(P, Q, T))
        rec["epoch_seconds"].append(round(time.time() - t1, 1))
        tmp = path + ".tmp"
        with open(tmp, "w") as fh:
            json.dump(rec, fh, indent=1)
            fh.write("\n")
        os.replace(tmp, path)
        print(f"[{label}] epoch {t + 1}: test rmse {rec['rmse'][-1]:.6f} ({rec['epoch_seconds'][-1]} s)", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
