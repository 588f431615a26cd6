"""Pins for oracle/build.py: decoders against independent library solvers."""
import numpy as np
import pytest
import scipy.linalg

from oracle.build import build_params, ensemble_activities, ensemble_gain_bias, ridge_decoders
from synth import make_workload
from synth.configs import lif_ensemble


@pytest.mark.parametrize("d,fn", [(1, "identity"), (2, "product"), (16, "identity")])
def test_ridge_decoders_against_library_routines(d, fn):
    rng = np.random.default_rng(d)
    ens = lif_ensemble(rng, 120, d, 300, "lif")
    g, b = ensemble_gain_bias(ens)
    X = ens.eval_points
    A = ensemble_activities(ens, g, b, X)
    Y = X.copy() if fn == "identity" else (X[:, 0] * X[:, 1])[:, None]
    D = ridge_decoders(A, Y, 0.1)
    M, n = A.shape
    lam = M * (0.1 * A.max()) ** 2
    # normal-equation residual
    G = A.T @ A + lam * np.eye(n)
    res = np.abs(G @ D - A.T @ Y).max() / np.abs(A.T @ Y).max()
    assert res < 1e-10
    # symmetric-positive-definite solver
    D2 = scipy.linalg.solve(G, A.T @ Y, assume_a="pos")
    np.testing.assert_allclose(D, D2, rtol=1e-8, atol=1e-12 * np.abs(D).max())
    # least squares on the stacked system [A; sqrt(lam) I] D = [Y; 0]
    S = np.vstack([A, np.sqrt(lam) * np.eye(n)])
    T = np.vstack([Y, np.zeros((n, Y.shape[1]))])
    D3 = np.linalg.lstsq(S, T, rcond=None)[0]
    np.testing.assert_allclose(D, D3, rtol=1e-6, atol=1e-9 * np.abs(D).max())


def test_decoders_decode_identity_well():
    w = make_workload("c4", n_ens=2, n_steps=2, minibatch=1)
    P = build_params(w.spec)
    ens = w.spec.ensembles[0]
    A = ensemble_activities(ens, P.gain[0], P.bias[0], ens.eval_points)
    err = A @ P.decoders[(0, "identity")] - ens.eval_points
    assert np.sqrt(np.mean(err ** 2)) < 0.1


def test_decoders_shared_per_ensemble_and_function():
    w = make_workload("c1")
    P = build_params(w.spec)
    # recurrent connection and probe both decode the identity from ensemble 0
    assert list(P.decoders) == [(0, "identity")]
