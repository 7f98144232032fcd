"""Pins for the oracle's planner (Sec. 3.1, Eq. 2-4, 8-9) from closed forms,
printed numbers and invariants -- not from re-typing the oracle's formulas."""
import math

import numpy as np
import pytest

from oracle import planner
from paper_2608_16354_amd import inputs as I


def _stats(w, m):
    xy, yaw = I.poses(m, w.n_pose, w.dt)
    return planner.motion_statistics(xy, yaw)


def _D(w, m):
    p = I.scene_problem(w, m)
    return planner.scene_tables(p)


def test_stationary_plan_has_zero_motion():
    w = I.WORKLOADS["dit-12x1152-bf16"]
    L, Th = _stats(w, I.Motion(0.0, 0.0))
    assert L == 0.0 and Th == 0.0
    t = _D(w, I.Motion(0.0, 0.0))
    assert t.D == 0.0 and t.supported


@pytest.mark.parametrize("v,om", [(8.0, 0.0), (6.0, 0.25), (13.0, -0.2), (0.5, 0.3)])
def test_constant_motion_closed_form(v, om):
    # each 0.1 s step moves exactly v*dt along the current heading: L = v*T_h;
    # the heading changes by |om|*dt per step: Theta = |om|*T_h
    w = I.WORKLOADS["dit-30x1920-bf16"]
    L, Th = _stats(w, I.Motion(v, om))
    assert L == pytest.approx(v * w.horizon_s, rel=1e-12)
    assert Th == pytest.approx(abs(om) * w.horizon_s, rel=1e-12, abs=1e-12)


def test_motion_intensity_corners():
    # the moving-turn anchor maps to the upper corner: z = (1, 1) -> D = 1
    assert planner.motion_intensity(1.0, 1.0) == pytest.approx(1.0, abs=1e-15)
    # pure translation at the anchor speed: z = (1, 0) -> D = 1/sqrt(2)
    assert planner.motion_intensity(1.0, 0.0) == pytest.approx(1 / math.sqrt(2), abs=1e-15)
    assert planner.motion_intensity(0.0, 0.0) == 0.0


@pytest.mark.parametrize("name,D", [("dit-tiny-f32", 0.4 / math.sqrt(2)),
                                    ("dit-30x1920-bf16", math.sqrt(0.3 ** 2 + (1.2 / 1.44) ** 2) / math.sqrt(2)),
                                    ("dit-42x3072-bf16", math.sqrt(0.75 ** 2 + (0.42 / 1.44) ** 2) / math.sqrt(2))])
def test_workload_intensities(name, D):
    # tiny: 8 m/s over 1.2 s against a 20 m/s anchor -> zL = 0.4
    # target: 6 m/s, 0.25 rad/s over 4.8 s -> zL = 28.8/96, zTh = 1.2/1.44
    # wide: 15 m/s over 4.8 s, 0.15 rad/s for 2.8 s -> zL = 72/96, zTh = 0.42/1.44
    w = I.WORKLOADS[name]
    t = _D(w, w.motions[0])
    assert t.supported
    assert t.D == pytest.approx(D, rel=1e-12)
    assert round(t.D, 4) == {"dit-tiny-f32": 0.2828, "dit-30x1920-bf16": 0.6263,
                             "dit-42x3072-bf16": 0.5690}[name]


def test_support_gate():
    w = I.WORKLOADS["dit-30x1920-bf16"]
    assert not _D(w, I.Motion(25.0, 0.0)).supported           # faster than the moving anchor
    assert not _D(w, I.Motion(5.0, 0.4)).supported            # turns more than the anchor
    assert _D(w, I.Motion(19.9, 0.29)).supported
    # the gate is coordinatewise: a radially small point outside on one axis is rejected
    assert not planner.in_support(1.0001, 0.0)
    assert not planner.in_support(-1e-9, 0.5)
    assert planner.in_support(1.0, 1.0) and planner.in_support(0.0, 0.0)


def test_wrap_is_shortest_signed_angle():
    assert planner.wrap(0.1 + 2 * math.pi) == pytest.approx(0.1, abs=1e-12)
    assert planner.wrap(-0.1 - 4 * math.pi) == pytest.approx(-0.1, abs=1e-12)
    assert planner.wrap(math.pi) == pytest.approx(-math.pi)
    assert planner.wrap(-math.pi) == pytest.approx(-math.pi)
    # a heading crossing +-pi: 3.1 -> -3.1 is a left turn of 2*pi - 6.2 rad, not 6.2 rad
    L, Th = planner.motion_statistics([[0, 0], [1, 0], [2, 0]], [3.0, 3.1, -3.1])
    assert Th == pytest.approx(0.1 + (2 * math.pi - 6.2), abs=1e-12)
    assert L == 2.0


def test_one_sided_interpolation():
    q0 = [[1.0, 2.0], [3.0, 0.5]]
    q1 = [[2.0, 1.0], [3.0, 4.5]]
    # D = 0 keeps the low-motion anchor
    assert planner.interpolate(q0, q1, 0.0) == q0
    # D = 1 reaches max(q0, q1); an easier moving anchor never lowers the response
    assert planner.interpolate(q0, q1, 1.0) == [[2.0, 2.0], [3.0, 4.5]]
    assert planner.interpolate(q0, q1, 0.5) == [[1.5, 2.0], [3.0, 2.5]]


def test_envelope_and_increments_hand_example():
    s = 2.0 ** -40
    # responses 1.5, 0.5, 3.0 (x 2^-40 units): envelope 1.5, 1.5, 3.0 -> costs 1.5, 0, 1.5
    qt = [[3 * s, 1 * s, 6 * s], [0.0, 2 * s, 1 * s]]
    Q, c = planner.envelope_costs(qt)
    assert Q == [[3, 3, 6], [0, 2, 2]]
    assert c == [[3, 0, 3], [0, 2, 0]]


def test_fixed_point_rounds_half_to_even():
    s = 2.0 ** -40
    Q, c = planner.envelope_costs([[2.5 * s, 3.5 * s, 3.5 * s]])
    assert Q == [[2, 4, 4]] and c == [[2, 2, 0]]


@pytest.mark.parametrize("name", ["dit-tiny-f32", "dit-30x1920-bf16", "dit-12x1152-bf16"])
def test_scene_costs_telescope_and_are_nonnegative(name):
    w = I.WORKLOADS[name]
    p = I.scene_problem(w, w.motions[0])
    t = planner.scene_tables(p)
    qt = planner.interpolate(p.q0.tolist(), p.q1.tolist(), t.D)
    for j in range(w.K - 1):
        run = 0
        for h in range(w.h_max):
            assert t.chat_q[j][h] >= 0
            run += t.chat_q[j][h]
            # the sum of the increments is the largest response seen so far (Eq. 9)
            assert run == round(max(qt[j][: h + 1]) * 2.0 ** 40)


def test_synthetic_tables_exercise_envelope_and_interpolation():
    q0, q1 = I.response_tables(50, 3)
    # non-monotone in the age, so the envelope is active
    assert (q0[:, 1] < q0[:, 0]).all()
    # the moving anchor is easier early and harder late, so the one-sided max is active
    assert q1[0, 0] < q0[0, 0] and q1[-1, 0] > q0[-1, 0]
