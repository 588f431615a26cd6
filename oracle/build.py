"""Build step: turn a model description into the numbers a simulation uses
(paper Sec. 2.1.3: the builder turns front-end objects into signals and
operators; Sec. 3.2: decoders come from a least-squares optimisation over the
ensemble's evaluation points).

Readings where the paper is silent:
  * gain/bias from (max rate, intercept) by the LIF rate curve (neurons.gain_bias),
    or by the rectified-linear line for ReLU neurons (neurons.relu_gain_bias)
  * scaled encoders E_hat = diag(gain) E (radius 1)
  * activities A[m, i] = amplitude * r(gain_i e_i . x_m + bias_i) on the
    ensemble's eval points
  * ridge decoders (A^T A + M sigma^2 I) D = A^T f(X), sigma = reg * max(A),
    solved by Cholesky in float64

Pins (tests/test_oracle_build.py): normal-equation residual; agreement with
scipy.linalg.solve(assume_a='pos') and with numpy.linalg.lstsq on the stacked
system [A; sqrt(lambda) I].
"""
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, Optional, Tuple

import numpy as np
import scipy.linalg

from .neurons import gain_bias, rate_output, relu_gain_bias


def function_targets(function: str, X: np.ndarray) -> np.ndarray:
    """Target values f(X) for a decoded connection; X is [M, d]."""
    if function == "identity":
        return X.copy()
    if function == "product":
        return (X[:, 0] * X[:, 1])[:, None]
    raise ValueError(f"unknown function {function!r}")


def function_size(function: str, dims: int) -> int:
    return dims if function == "identity" else 1


def apply_function(function: str, x: np.ndarray) -> np.ndarray:
    """f applied to represented values x [B, d] (used by direct-mode ensembles)."""
    if function == "identity":
        return x.copy()
    if function == "product":
        return (x[:, 0] * x[:, 1])[:, None]
    raise ValueError(function)


def ensemble_gain_bias(ens):
    if ens.gains is not None:
        return np.asarray(ens.gains, np.float64), np.asarray(ens.biases, np.float64)
    if ens.neuron_type == "relu":
        return relu_gain_bias(ens.max_rates, ens.intercepts)
    return gain_bias(ens.max_rates, ens.intercepts, ens.tau_rc, ens.tau_ref)


def ensemble_activities(ens, gain, bias, X):
    """Rate-mode outputs [M, n] of the ensemble's neurons at represented values X."""
    J = (X @ np.asarray(ens.encoders, np.float64).T) * gain[None, :] + bias[None, :]
    return rate_output(ens.neuron_type, J, ens.tau_rc, ens.tau_ref, ens.amplitude, ens.sigma)


def ridge_decoders(A: np.ndarray, Y: np.ndarray, reg: float) -> np.ndarray:
    """Solve (A^T A + M (reg max A)^2 I) D = A^T Y by Cholesky (float64)."""
    M, n = A.shape
    sigma = reg * A.max()
    lam = M * sigma * sigma
    G = A.T @ A + lam * np.eye(n)
    factor = scipy.linalg.cho_factor(G, lower=True, check_finite=False)
    return scipy.linalg.cho_solve(factor, A.T @ Y, check_finite=False)


SOLVER_REG = 0.1   # sigma = 0.1 * max activity


@dataclass
class BuiltParams:
    gain: Dict[int, np.ndarray] = field(default_factory=dict)
    bias: Dict[int, np.ndarray] = field(default_factory=dict)
    scaled_encoders: Dict[int, np.ndarray] = field(default_factory=dict)   # [n, d]
    decoders: Dict[Tuple[int, str], np.ndarray] = field(default_factory=dict)  # [n, d_fn]


def build_params(spec, direct: frozenset = frozenset()) -> BuiltParams:
    """Gains, biases, scaled encoders and the decoders every connection or
    probe needs.  Decoders are keyed by (ensemble, function) and shared by every
    connection/probe that decodes the same function from the same ensemble."""
    P = BuiltParams()
    for i, ens in enumerate(spec.ensembles):
        if i in direct:
            continue
        g, b = ensemble_gain_bias(ens)
        P.gain[i], P.bias[i] = g, b
        P.scaled_encoders[i] = np.asarray(ens.encoders, np.float64) * g[:, None]
    needed = []
    for c in spec.connections:
        if c.pre[0] == "ens" and c.decoders is None:
            needed.append((c.pre[1], c.function))
    for p in spec.probes:
        if p.target[0] == "ens":
            needed.append((p.target[1], "identity"))
    todo = []
    for key in needed:
        if key not in todo and key[0] not in direct:
            todo.append(key)

    def solve(key):
        ei, fn = key
        ens = spec.ensembles[ei]
        X = np.asarray(ens.eval_points, np.float64)
        A = ensemble_activities(ens, P.gain[ei], P.bias[ei], X)
        return ridge_decoders(A, function_targets(fn, X), SOLVER_REG)

    # ensembles are independent; solve them concurrently (numpy releases the GIL)
    workers = min(len(todo), os.cpu_count() or 1) if len(todo) > 8 else 1
    if workers > 1:
        try:   # one BLAS thread per worker: parallelism comes from the ensembles
            from threadpoolctl import threadpool_limits
            limit = threadpool_limits(1)
        except Exception:
            limit = None
        try:
            with ThreadPoolExecutor(workers) as pool:
                results = list(pool.map(solve, todo))
        finally:
            if limit is not None:
                limit.restore_original_limits()
    else:
        results = [solve(k) for k in todo]
    for key, D in zip(todo, results):
        P.decoders[key] = D
    return P
