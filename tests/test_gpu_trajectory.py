"""The library's default batch-Hogwild! against the serial oracle's test-RMSE
trajectory at full size (section 3.2.4: test RMSE after each epoch is the
convergence measure; section 5.5.1: Hogwild! behaves like serial SGD only
when concurrent updates rarely share a row).

The expected values are tests/golden/trajectory_<label>.json, written by
tests/golden/make_trajectories.py from the oracle alone (serial SGD in array
order, the workload's learning-rate schedule, the oracle's initial factors).
The GPU run uses the same seeded samples and the library's initial factors
(bit-equal to the oracle's), with every option at its default except the
storage type, and must end within 1e-3 (binary32) / 5e-3 (binary16) of the
oracle's test RMSE after the same number of epochs.  Individual Hogwild!
runs are not deterministic; the per-epoch gaps are printed."""
import json
import os

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden")
TOL = {"fp32": 1e-3, "fp16": 5e-3}


def golden(label):
    with open(os.path.join(GOLD, f"trajectory_{label}.json")) as f:
        return json.load(f)


@pytest.fixture(scope="module")
def M():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1610_05838_amd import mfsgd
    mfsgd.lib()
    yield mfsgd
    mfsgd.finalize()


def run_default(M, gen, g, epochs):
    import torch
    w = gen.workload(g["workload"], k=g["k"])
    assert (w["m"], w["n"], w["ntrain"], w["ntest"], w["seed"]) == (g["m"], g["n"], g["ntrain"], g["ntest"], g["seed"])
    if w["draw"] == "independent":
        dS = gen.draw_to_device(w, 0, w["ntrain"])
        dT = gen.draw_to_device(w, w["ntrain"], w["ntest"])
    else:
        S, T = gen.make(w)
        dS, dT = M.samples_to_device(S), M.samples_to_device(T)
    M.reset_options()
    M.set_option("dtype", 1 if w["dtype"] == "fp16" else 0)
    M.init(w["m"], w["n"], w["k"], w["seed"])
    rm = []
    for t in range(epochs):
        M.epoch(dS, gen.lr_at(w, t), w["lam"], w["lam"], "hogwild")
        rm.append(M.rmse(dT))
    del dS, dT
    torch.cuda.empty_cache()
    return rm


@pytest.mark.parametrize("label", ["tiny", "netflix", "netflix_fp16", "yahoo", "netflix_k32"])
def test_default_hogwild_tracks_the_serial_oracle(M, gen, label):
    g = golden(label)
    want = g["rmse"]
    assert len(want) >= 5, "the trajectory needs at least 5 epochs"
    got = run_default(M, gen, g, len(want))
    gaps = [a - b for a, b in zip(got, want)]
    print(f"{label}: default batch-Hogwild! test rmse after {len(want)} epochs {got[-1]:.6f}, "
          f"oracle {want[-1]:.6f}; gap per epoch " + " ".join(f"{x:+.4f}" for x in gaps))
    assert abs(gaps[-1]) <= TOL[g["dtype"]]
