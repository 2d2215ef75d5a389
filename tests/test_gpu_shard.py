"""bench.py --shard G: one GPU's share of a G-GPU epoch (block partition of
the paper's section 4.1), run on this GPU at its real shape."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_shard_share_is_rank_zeros_blocks(gen):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    G = 4
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--shard", str(G),
                        "--steps", "1", "--warmup", "1"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads(r.stdout.strip().splitlines()[-1])
    w = gen.workload("tiny")
    S, _ = gen.make(w)
    mine = S[(S["u"].astype(np.int64) * G) // w["m"] == 0]
    per_wave = np.bincount((mine["v"].astype(np.int64) * G) // w["n"], minlength=G)
    assert d["gpus_emulated"] == G and d["share_samples"] == len(mine)
    assert d["wave_samples"] == per_wave.tolist()
    assert len(d["wave_ms"]) == G and all(x > 0 for x in d["wave_ms"])
    assert d["q_segment_bytes"] == -(-w["n"] // G) * w["k"] * 4
    assert d["projected_epoch_ms"] >= d["compute_ms_per_epoch"] > 0
