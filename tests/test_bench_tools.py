"""Host logic of bench.py that needs no GPU: the choice of the plan skew from
timed candidates (calibrate_skew), with the timing replaced by fixed values."""
import numpy as np
import pytest

import bench


class _FakeStepper:
    def __init__(self):
        self.runner = ("runner", 0)
        self.made = []

    def make_runner(self, skew):
        self.made.append(skew)
        return ("runner", skew)

    def step(self):
        pass

    class torch:
        class cuda:
            @staticmethod
            def synchronize():
                pass


def _calibrate(monkeypatch, kernel_us, **kw):
    st = _FakeStepper()
    rounds = []

    def fake_time_steps(stepper, steps, warmup):
        p = stepper.runner[1]
        rounds.append(p)
        return 0.0, 0.0, kernel_us[p] / 1e3
    monkeypatch.setattr(bench, "time_steps", fake_time_steps)
    return st, bench.calibrate_skew(st, **kw), rounds


def test_skew_calibration_takes_the_fastest(monkeypatch):
    us = {-40: 230.0, -20: 226.0, 0: 224.0, 20: 221.0, 40: 222.0}
    st, cal, rounds = _calibrate(monkeypatch, us)
    assert cal["chosen"] == 20 and st.runner == ("runner", 20)
    assert sorted(st.made) == [-40, -20, 20, 40]            # the stepper's own runner is the p = 0 one
    assert len(rounds) == 3 * len(us) and {float(v) for v in cal["kernel_us_median"].values()} == set(us.values())


def test_skew_calibration_keeps_equal_slices_below_the_gain_threshold(monkeypatch):
    us = {-40: 230.0, -20: 226.0, 0: 224.0, 20: 223.8, 40: 225.0}  # 0.09 % better: not enough
    st, cal, _ = _calibrate(monkeypatch, us)
    assert cal["chosen"] == 0 and st.runner == ("runner", 0)


def test_skew_calibration_rotates_the_order(monkeypatch):
    us = {p: 200.0 + abs(p) for p in (-40, -20, 0, 20, 40)}
    _, _, rounds = _calibrate(monkeypatch, us, rounds=3)
    firsts = [rounds[i * 5] for i in range(3)]
    assert firsts == [-40, -20, 0]                           # each round starts one candidate later
