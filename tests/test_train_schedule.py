"""Warm-up density schedule of the training integration (host logic, CPU)."""
import pytest

from paper_2108_06004_amd.train import DensitySchedule, GlobalSketchSGD


def test_schedule_follows_the_warmup_then_the_target():
    # the paper's warm-up densities (Sec. IV) then a 0.1% target
    s = DensitySchedule(0.001, 0.1, [(0.25, 0.1), (0.0725, 0.03), (0.015, 0.01), (0.004, 0.01)])
    d = 65_536
    assert [s.k_at(e, d) for e in range(6)] == [16_384, 4_752, 984, 263, 66, 66]
    assert s.at(1) == (0.0725, 0.03) and s.at(10) == (0.001, 0.1)
    assert s.k_max(d) == 16_384


def test_schedule_k_is_clamped_to_one_and_d():
    assert DensitySchedule(1e-9, 0.1).k_at(0, 1000) == 1
    assert DensitySchedule(2.0, 0.1).k_at(0, 1000) == 1000


def test_trainer_rejects_unknown_variants_before_touching_the_device():
    s = DensitySchedule(0.01, 0.1)
    hp = {"a": [1], "b": [0], "a2": [1], "b2": [0]}
    with pytest.raises(ValueError):
        GlobalSketchSGD(100, 2, 1, 10, hp, s, selection="random")
    with pytest.raises(ValueError):
        GlobalSketchSGD(100, 2, 1, 10, hp, s, selection="heavymix", state="sketch")
