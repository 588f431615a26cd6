"""Pins for oracle/neurons.py against closed forms of the LIF model."""
import math

import numpy as np
import pytest

from oracle.neurons import gain_bias, lif_rate, lif_step

TAU_RC, TAU_REF, DT = 0.02, 0.002, 0.001


def test_rate_closed_form_values():
    # r(J) = 1 / (tau_ref - tau_rc ln(1 - 1/J)); hand-evaluated:
    # r(2) = 1/(0.002 + 0.02 ln 2)      = 63.0400 Hz
    # r(5) = 1/(0.002 + 0.02 ln(5/4))   = 154.730 Hz
    r = lif_rate(np.array([2.0, 5.0]), TAU_RC, TAU_REF)
    assert r[0] == pytest.approx(63.0400, abs=5e-4)
    assert r[1] == pytest.approx(154.730, abs=5e-3)


def test_rate_matches_log_form_and_is_zero_below_threshold():
    J = np.linspace(-3.0, 60.0, 2001)
    r = lif_rate(J, TAU_RC, TAU_REF)
    above = J > 1
    ref = 1.0 / (TAU_REF - TAU_RC * np.log(1.0 - 1.0 / J[above]))
    np.testing.assert_allclose(r[above], ref, rtol=1e-13)
    assert np.all(r[~above] == 0.0)
    assert np.all(np.diff(r[above]) > 0)          # monotone in J
    assert r.max() < 1.0 / TAU_REF                 # refractory period caps the rate


@pytest.mark.parametrize("J", [1.2, 2.0, 5.0, 40.0])
def test_spike_steps_match_closed_form(J):
    """Constant J from V = 0: crossing j happens at t_j = t1 + (j-1)(tau_ref + t1),
    t1 = tau_rc ln(J/(J-1)); it is reported in step ceil(t_j / dt)."""
    n_steps = 5000
    V = np.zeros(1); ref = np.zeros(1)
    steps = []
    for k in range(1, n_steps + 1):
        s, V, ref = lif_step(np.array([J]), V, ref, DT, TAU_RC, TAU_REF, 1.0)
        if s[0] > 0:
            assert s[0] == pytest.approx(1.0 / DT)
            steps.append(k)
    t1 = TAU_RC * math.log(J / (J - 1.0))
    period = TAU_REF + t1
    expect = []
    j = 0
    while True:
        t = t1 + j * period
        k = math.ceil(t / DT - 1e-9)
        if k > n_steps:
            break
        expect.append(k)
        j += 1
    assert steps == expect
    # long-run rate equals the rate curve
    rate = len(steps) / (n_steps * DT)
    assert rate == pytest.approx(lif_rate(np.array([J]), TAU_RC, TAU_REF)[0], rel=2e-3)


@pytest.mark.parametrize("J", [-5.0, 0.0, 0.5, 1.0])
def test_subthreshold_never_spikes_and_converges(J):
    V = np.zeros(1); ref = np.zeros(1)
    for _ in range(3000):
        s, V, ref = lif_step(np.array([J]), V, ref, DT, TAU_RC, TAU_REF, 1.0)
        assert s[0] == 0.0
    assert V[0] == pytest.approx(max(J, 0.0), abs=1e-12)


def test_partial_refractory_integrates_remaining_time():
    # ref = 0.4 ms left: only 0.6 ms of integration this step
    J = np.array([3.0]); V = np.array([0.0]); ref = np.array([0.0004])
    s, V2, ref2 = lif_step(J, V, ref, DT, TAU_RC, TAU_REF, 1.0)
    assert s[0] == 0.0 and ref2[0] == 0.0
    assert V2[0] == pytest.approx(3.0 * (1 - math.exp(-0.0006 / TAU_RC)), rel=1e-14)
    # fully refractory: no integration
    s, V3, ref3 = lif_step(J, np.array([0.0]), np.array([0.0015]), DT, TAU_RC, TAU_REF, 1.0)
    assert V3[0] == 0.0 and ref3[0] == pytest.approx(0.0005)


def test_spike_sets_refractory_from_crossing_time():
    # start just below threshold: crossing time inside the step is recoverable
    J = np.array([2.0]); V0 = 0.99
    s, V, ref = lif_step(J, np.array([V0]), np.array([0.0]), DT, TAU_RC, TAU_REF, 2.5)
    t_cross = TAU_RC * math.log((J[0] - V0) / (J[0] - 1.0))
    assert s[0] == pytest.approx(2.5 / DT)
    assert V[0] == 0.0
    assert ref[0] == pytest.approx(TAU_REF - (DT - t_cross), rel=1e-12)


def test_gain_bias_invariants():
    rng = np.random.default_rng(0)
    m = rng.uniform(200, 400, 1000); c = rng.uniform(-0.99, 0.99, 1000)
    g, b = gain_bias(m, c, TAU_RC, TAU_REF)
    np.testing.assert_allclose(g * c + b, 1.0, rtol=0, atol=1e-12 * np.abs(g).max())
    np.testing.assert_allclose(lif_rate(g + b, TAU_RC, TAU_REF), m, rtol=1e-12)
    assert np.all(g > 0)


def test_soft_lif_rate_closed_forms():
    """Soft LIF rate: at J = 1, rho = sigma ln 2 exactly, so r = 1/(tau_ref +
    tau_rc ln(1 + 1/(sigma ln 2))); where J - 1 >> sigma, rho = J - 1 (to
    exp(-(J-1)/sigma)) and the curve is the LIF rate; as sigma -> 0 it tends
    to the LIF rate everywhere off threshold; far below threshold rho = sigma
    exp((J-1)/sigma) (relative error exp((J-1)/sigma)), so r = 1/(tau_ref +
    tau_rc ((1-J)/sigma - ln sigma)) up to that error; always positive and
    increasing."""
    from oracle.neurons import lif_rate, rate_output, soft_lif_rate
    trc, tref = 0.02, 0.002
    for s in (0.005, 0.02, 0.3):
        exp = 1.0 / (tref + trc * np.log1p(1.0 / (s * np.log(2.0))))
        assert soft_lif_rate(np.array([1.0]), trc, tref, s)[0] == pytest.approx(exp, rel=1e-13)
    J = 1.0 + np.array([0.8, 1.5, 4.0, 40.0])
    np.testing.assert_allclose(soft_lif_rate(J, trc, tref, 0.01), lif_rate(J, trc, tref), rtol=1e-13)
    Jo = np.array([0.2, 0.9, 1.05, 1.3, 3.0])
    prev = None
    for s in (1e-2, 1e-3, 1e-4):
        d = np.abs(soft_lif_rate(Jo, trc, tref, s) - lif_rate(Jo, trc, tref)).max()
        assert prev is None or d < prev
        prev = d
    assert prev < 0.06   # Hz, against rates of tens of Hz (the tail below threshold shrinks like sigma)
    far = np.array([-3.0, -0.5, 0.5])
    s = 0.01
    np.testing.assert_allclose(soft_lif_rate(far, trc, tref, s),
                               1.0 / (tref + trc * ((1.0 - far) / s - np.log(s))), rtol=1e-12)
    grid = np.linspace(-5, 5, 2001)
    r = soft_lif_rate(grid, trc, tref, 0.02)
    assert np.all(r > 0) and np.all(np.diff(r) > 0)
    np.testing.assert_array_equal(rate_output("softlif_rate", J, trc, tref, 0.5, 0.01),
                                  0.5 * soft_lif_rate(J, trc, tref, 0.01))


def test_relu_rate_and_gain_bias():
    """Rectified-linear neuron: r(J) = max(J, 0); gain and bias put J = 0 at the
    intercept and J = max_rate at x = 1.  Hand values: max_rate 200 Hz at
    intercept 0.5 gives gain 400 and bias -200."""
    from oracle.neurons import rate_output, relu_gain_bias, relu_rate
    assert list(relu_rate(np.array([-1.0, 0.0, 2.5]))) == [0.0, 0.0, 2.5]
    g, b = relu_gain_bias(np.array([200.0]), np.array([0.5]))
    assert g[0] == 400.0 and b[0] == -200.0
    rng = np.random.default_rng(7)
    m, c = rng.uniform(200, 400, 1000), rng.uniform(-1, 1, 1000)
    g, b = relu_gain_bias(m, c)
    np.testing.assert_allclose(relu_rate(g + b), m, rtol=1e-12)          # x = 1 fires at max_rate
    np.testing.assert_allclose(g * c + b, 0.0, atol=1e-9 * np.abs(g).max())  # x = intercept: J = 0
    assert np.all(relu_rate(g * (c - 1e-3) + b) == 0.0)                   # silent below the intercept
    np.testing.assert_array_equal(rate_output("relu", np.array([3.0, -2.0]), 0.02, 0.002, 0.5),
                                  [1.5, 0.0])
