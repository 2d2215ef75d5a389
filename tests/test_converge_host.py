"""Host logic of converge.py (no GPU): the learning-rate schedules and the
scheme list."""
import math
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import converge  # noqa: E402


def test_paper_schedule_values():
    """Evaluation section: s_t = alpha / (1 + beta t^1.5) with the Netflix row
    (lambda 0.05, alpha 0.08, beta 0.3): s_0 = 0.08, s_1 = 0.08 / 1.3,
    s_4 = 0.08 / (1 + 0.3 * 8) = 0.08 / 3.4."""
    from paper_1610_05838_amd import datagen

    for name in ("netflix", "netflix_fp16"):
        lr, lam = converge.lr_schedule(datagen.workload(name), "paper")
        assert lam == 0.05
        assert lr(0) == pytest.approx(0.08, rel=1e-15)
        assert lr(1) == pytest.approx(0.08 / 1.3, rel=1e-15)
        assert lr(4) == pytest.approx(0.08 / 3.4, rel=1e-15)
        assert all(lr(t + 1) < lr(t) for t in range(30))
    lr, lam = converge.lr_schedule(datagen.workload("yahoo"), "paper")
    assert lam == 1.0 and lr(1) == pytest.approx(0.08 / 1.2, rel=1e-15)
    lr, lam = converge.lr_schedule(datagen.workload("hugewiki"), "paper")
    assert lam == 0.03 and lr(9) == pytest.approx(0.08 / (1 + 0.3 * 27), rel=1e-15)


def test_config_schedule_is_the_workloads():
    from paper_1610_05838_amd import datagen

    w = datagen.workload("netflix")
    lr, lam = converge.lr_schedule(w, "config")
    assert lam == w["lam"]
    assert lr(0) == pytest.approx(0.003) and lr(10) == pytest.approx(0.003 * math.pow(0.99, 10))


def test_schemes_and_labels():
    assert converge.parse_schemes("hogwild,wavefront:8,wavefront_det") == [
        ("hogwild", 0), ("wavefront", 8), ("wavefront_det", 0)]
    assert converge.label("wavefront", 32) == "wavefront s=32"
    with pytest.raises(SystemExit):
        converge.parse_schemes("hogwild,blocked")
    with pytest.raises(SystemExit):
        converge.stand_in("tiny")
