"""Spatial controller (§4.4 Eq. (1), Algorithm 1 step 3): oracle pins, then the library against the oracle.

The paper prints no controller trace values, so the pins are the policy's own
closed forms and special cases: the EWMA of a constant, the clamps of rho,
the aggressive cap with no downstream activity, nearest-level snapping checked
by brute force, hysteresis, and one sequence worked by hand.
"""
import math

import numpy as np
import pytest

from oracle.controller import ControllerError, SpatialController, run, snap

LADDER = [64, 96, 128, 160, 192]


def make(gamma=0.4, sat=0.8, steps=1, ladder=LADDER, aggr=256, total=256):
    return SpatialController(total, aggr, ladder, gamma, sat, steps)


# ----------------------------------------------------------------------------- oracle pins

def test_ewma_of_a_constant_closed_form():
    c = make(gamma=0.3)
    c.step(True, 0.9)                      # B_hat_0 = first sample
    for t in range(1, 12):
        d = c.step(True, 0.2)
        assert d.pressure == pytest.approx(0.2 + (0.9 - 0.2) * (1 - 0.3) ** t, rel=1e-12)


def test_rho_clamps_to_ladder_ends():
    c = make(sat=0.5)
    assert c.step(True, 3.0).shared == 192          # rho clamps to 1: S_cap
    c = make(sat=0.5)
    d = c.step(True, -1.0)
    assert (d.rho, d.shared) == (0.0, 64)           # rho clamps to 0: S_min


def test_no_downstream_gives_aggressive_cap():
    c = make(aggr=224, total=256)
    for b in (0.0, 0.5, 5.0):
        d = c.step(False, b)
        assert (d.shared, d.down, d.level) == (224, 32, -1)


def test_snap_is_nearest_level_by_brute_force():
    rng = np.random.default_rng(7)
    for _ in range(500):
        ladder = sorted(set(int(v) for v in rng.integers(1, 256, size=rng.integers(1, 9))))
        x = float(rng.uniform(0, 260))
        i = snap(ladder, x)
        best = min(abs(s - x) for s in ladder)
        assert abs(ladder[i] - x) == best
        # ties go to the larger level
        assert all(not (abs(s - x) == best and s > ladder[i]) for s in ladder)
    assert snap([64, 128], 96.0) == 1
    assert snap([64, 128], 95.9) == 0


def test_hysteresis_keeps_one_level_moves_with_two_steps():
    c = make(gamma=1.0, sat=1.0, steps=2)   # gamma 1: B_hat = latest sample
    assert c.step(True, 0.0).shared == 64   # first step applies S_min
    d = c.step(True, 0.25)                   # target 96: one level, kept
    assert (d.shared, d.changed) == (64, False)
    d = c.step(True, 0.5)                    # target 128: two levels, applied
    assert (d.shared, d.changed, d.level) == (128, True, 2)
    d = c.step(True, 0.75)                   # target 160: one level, kept
    assert d.shared == 128
    d = c.step(True, 1.0)                    # 192: two levels
    assert d.shared == 192


def test_entering_corunning_from_aggressive_always_applies():
    c = make(gamma=1.0, sat=1.0, steps=4)
    assert c.step(False, 0.1).shared == 256
    d = c.step(True, 0.25)                   # previous cap is not a ladder level
    assert (d.shared, d.changed) == (96, True)


def test_worked_sequence_by_hand():
    # gamma 0.4, B_sat 0.8, ladder 64..192 in steps of 32, S_aggr = S_tot = 256.
    #   B_hat: 0.3 | 0.4*0.1+0.6*0.3 = 0.22 | 0.4*0.9+0.6*0.22 = 0.492 | 0.4*0.95+0.6*0.492 = 0.6752
    #   targets: aggressive | 64+0.275*128 = 99.2 -> 96 | 64+0.615*128 = 142.72 -> 128 | 64+0.844*128 = 172.03 -> 160
    d = run(make(), [0, 1, 1, 1], [0.3, 0.1, 0.9, 0.95])
    assert [x.shared for x in d] == [256, 96, 128, 160]
    assert [x.down for x in d] == [0, 160, 128, 96]
    assert [round(x.pressure, 6) for x in d] == [0.3, 0.22, 0.492, 0.6752]


def test_invalid_configurations_raise():
    with pytest.raises(ControllerError):
        make(ladder=[64, 64])
    with pytest.raises(ControllerError):
        make(ladder=[64, 256], aggr=256)          # S_cap must be below S_aggr
    with pytest.raises(ControllerError):
        make(gamma=0.0)
    with pytest.raises(ControllerError):
        make(sat=0.0)


# ----------------------------------------------------------------------------- library vs oracle

def _lib():
    from paper_2608_01785_amd import binding
    binding.lib()
    return binding


@pytest.mark.parametrize("cfg", [
    dict(total=256, aggr=256, ladder=[64, 96, 128, 160, 192], gamma=0.4, sat=0.8, steps=1),
    dict(total=256, aggr=224, ladder=[32, 64, 128], gamma=0.1, sat=0.5, steps=2),
    dict(total=128, aggr=120, ladder=[8, 16, 24, 32, 40, 48, 56, 64, 72, 80], gamma=0.9, sat=1.0, steps=3),
])
def test_library_matches_oracle_on_random_traces(cfg):
    B = _lib()
    rng = np.random.default_rng(11)
    n = 400
    active = (rng.uniform(size=n) < 0.7).astype(int)
    samples = rng.uniform(-0.1, 1.3, size=n)
    ref = run(SpatialController(cfg["total"], cfg["aggr"], cfg["ladder"], cfg["gamma"], cfg["sat"], cfg["steps"]),
              active, samples)
    ctrl = B.Controller(cfg["total"], cfg["aggr"], cfg["ladder"], cfg["gamma"], cfg["sat"], cfg["steps"])
    try:
        for a, b, r in zip(active, samples, ref):
            s = B.hs_controller_step(ctrl, bool(a), float(b))
            assert (s.shared_cus, s.down_cus, s.level, bool(s.changed)) == (r.shared, r.down, r.level, r.changed)
            assert s.pressure == r.pressure and s.rho == r.rho
    finally:
        ctrl.close()


def test_library_rejects_bad_input():
    B = _lib()
    for kw in (dict(ladder=[64, 32]), dict(ladder=[64, 256]), dict(ewma_weight=1.5), dict(saturation=-1.0),
               dict(hysteresis_steps=0)):
        args = dict(total_cus=256, aggressive_cus=256, ladder=[64, 128], ewma_weight=0.4, saturation=0.8,
                    hysteresis_steps=1)
        args.update(kw)
        with pytest.raises(B.HorizonError) as e:
            B.Controller(**args)
        assert e.value.status == B.HS_ERR_INVALID_ARG
    ctrl = B.Controller(256, 256, [64, 128], 0.4, 0.8, 1)
    try:
        with pytest.raises(B.HorizonError):
            B.hs_controller_step(ctrl, True, math.nan)
        s = B.hs_controller_step(ctrl, True, 0.0)  # the rejected sample left no trace
        assert (s.shared_cus, s.pressure) == (64, 0.0)
    finally:
        ctrl.close()
