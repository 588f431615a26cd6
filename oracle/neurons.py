"""Leaky integrate-and-fire neuron model (paper Sec. 2.1.3 names SimLIF and
Sec. 3.2 / 5.2.1 its rate approximation; the paper defers the equations to Nengo,
so they are stated here from the membrane equation dV/dt = (J - V) / tau_rc with
threshold 1, reset 0 and an absolute refractory period tau_ref).

Pins (tests/test_oracle_neurons.py):
  lif_rate        closed form 1/(tau_ref - tau_rc ln(1 - 1/J)); printed values
  lif_step        exact spike steps ceil(t_j / dt) for constant J; long-run rate
  gain_bias       r(g + b) == max_rate and g * intercept + b == 1
  relu_rate       max(J, 0) by definition; relu_gain_bias: g + b == max_rate and
                  g * intercept + b == 0 (tests/test_oracle_neurons.py)
  soft_lif_rate   at J = 1 the closed form 1/(tau_ref + tau_rc ln(1 + 1/(sigma ln 2)));
                  equal to lif_rate where J - 1 >> sigma; tends to lif_rate as
                  sigma -> 0; far below threshold 1/(tau_ref + tau_rc ((1 - J)/sigma
                  - ln sigma)) (tests/test_oracle_neurons.py)

A rectified-linear rate neuron (the neuron type of the memory storage and
retrieval example, Sec. 5.2) is also defined here: its output is amplitude *
max(J, 0), with no state.
"""
import numpy as np


def lif_rate(J, tau_rc, tau_ref):
    """Steady-state firing rate (Hz) of a LIF neuron driven by constant current J.

    Time to climb from 0 to threshold 1 is tau_rc * ln(J / (J - 1)); one period
    adds the refractory time.  Zero for J <= 1 (threshold never reached).
    """
    J = np.asarray(J, dtype=np.float64)
    out = np.zeros_like(J)
    m = J > 1.0
    out[m] = 1.0 / (tau_ref + tau_rc * np.log1p(1.0 / (J[m] - 1.0)))
    return out


def gain_bias(max_rates, intercepts, tau_rc, tau_ref):
    """Gain and bias so that a neuron starts firing at x = intercept and fires at
    max_rate at x = 1 (radius 1): J(x) = gain * x + bias.

    r(J_max) = max_rate gives J_max = 1 / (1 - exp((tau_ref - 1/max_rate) / tau_rc));
    J(intercept) = 1 and J(1) = J_max fix the line.
    """
    max_rates = np.asarray(max_rates, dtype=np.float64)
    intercepts = np.asarray(intercepts, dtype=np.float64)
    j_max = 1.0 / -np.expm1((tau_ref - 1.0 / max_rates) / tau_rc)
    gain = (j_max - 1.0) / (1.0 - intercepts)
    bias = 1.0 - gain * intercepts
    return gain, bias


def lif_step(J, V, ref, dt, tau_rc, tau_ref, amplitude, dtype=np.float64):
    """One timestep of the spiking LIF model, elementwise; returns (s, V, ref).

    V integrates exactly for the part of the step that is not refractory
    (dt - ref, clipped to [0, dt]).  Crossing 1 (strictly) emits one spike of
    height amplitude/dt; the crossing time is recovered from the overshoot by
    inverting the exponential approach, so the refractory period is measured from
    the crossing itself and not from the step boundary.  V is floored at 0.
    dtype: the arithmetic precision (float64; float32 only to measure what
    float32 arithmetic does to spike trains).
    """
    J = np.asarray(J, dtype=dtype)
    V = np.array(V, dtype=dtype, copy=True)
    ref = np.array(ref, dtype=dtype, copy=True)
    dt, tau_rc, tau_ref = dtype(dt), dtype(tau_rc), dtype(tau_ref)
    integ = np.clip(dt - ref, 0.0, dt)
    V = V - (J - V) * np.expm1(-integ / tau_rc)
    ref = np.maximum(ref - dt, 0.0)
    spiked = V > 1.0
    since = np.zeros_like(V)
    drive = J - 1.0
    ok = spiked & (drive > 0.0)
    q = np.zeros_like(V)
    q[ok] = (V[ok] - 1.0) / drive[ok]
    full = ok & (q >= 1.0)
    part = ok & (q < 1.0)
    since[full] = integ[full]
    since[part] = np.minimum(-tau_rc * np.log1p(-q[part]), integ[part])
    V = np.where(spiked, dtype(0.0), np.maximum(V, dtype(0.0)))
    ref = np.where(spiked, tau_ref - since, ref)
    s = np.where(spiked, dtype(amplitude) / dt, dtype(0.0))
    return s, V, ref


def relu_rate(J):
    """Rectified-linear rate: J above 0, else 0."""
    J = np.asarray(J, dtype=np.float64)
    return np.maximum(J, 0.0)


def relu_gain_bias(max_rates, intercepts):
    """Gain and bias of a rectified-linear neuron: J(x) = gain * x + bias is 0 at
    x = intercept (where it starts to respond) and max_rate at x = 1."""
    max_rates = np.asarray(max_rates, dtype=np.float64)
    intercepts = np.asarray(intercepts, dtype=np.float64)
    gain = max_rates / (1.0 - intercepts)
    bias = -gain * intercepts
    return gain, bias


def soft_lif_rate(J, tau_rc, tau_ref, sigma):
    """Smoothed LIF rate curve, the differentiable stand-in for the spiking LIF
    when a model is trained by gradient descent (paper Sec. 3.2 trains spiking
    models through a rate approximation; the smoothing is Hunsberger and
    Eliasmith's): the threshold nonlinearity max(J - 1, 0) inside the LIF rate
    curve becomes rho = sigma log(1 + exp((J - 1) / sigma)), so that
    r = 1 / (tau_ref + tau_rc log(1 + 1 / rho)) for every J.  Its slope stays
    bounded at threshold, where the exact curve's grows without bound; below
    threshold it decays slowly (log(1 + 1/rho) grows like (1 - J) / sigma).

    Evaluated with x = (J - 1) / sigma as log1p(1 / rho), rho = sigma
    softplus(x), for x >= -30; below, where softplus(x) = exp(x) to a relative
    exp(x) / 2, as log1p(rho) - log(rho) with log(rho) = log(sigma) + x, so
    that nothing overflows or underflows."""
    J = np.asarray(J, dtype=np.float64)
    x = (J - 1.0) / sigma
    far = x < -30.0
    rho = sigma * np.logaddexp(0.0, np.where(far, 0.0, x))
    q_near = np.log1p(1.0 / rho)
    q_far = np.log1p(sigma * np.exp(np.minimum(x, 0.0))) - (np.log(sigma) + x)
    q = np.where(far, q_far, q_near)
    return 1.0 / (tau_ref + tau_rc * q)


def rate_output(neuron_type, J, tau_rc, tau_ref, amplitude, sigma=0.0):
    """Output of a rate neuron: amplitude * r(J) with the LIF, the smoothed LIF
    (smoothing sigma) or the ReLU curve."""
    if neuron_type == "relu":
        return amplitude * relu_rate(J)
    if neuron_type == "softlif_rate":
        return amplitude * soft_lif_rate(J, tau_rc, tau_ref, sigma)
    return amplitude * lif_rate(J, tau_rc, tau_ref)


def lif_rate_output(J, tau_rc, tau_ref, amplitude):
    """Rate-mode neuron output: amplitude * r(J)."""
    return amplitude * lif_rate(J, tau_rc, tau_ref)
