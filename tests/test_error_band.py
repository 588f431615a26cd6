"""CPU pins of the rate-mode error band (tests/error_band.py): it steps
exactly the float64 oracle (identical probe records), and the oracle run in
float32 arithmetic -- a plain float32 simulator -- stays inside the band plus
1e-5 of each probe's peak, at test sizes on every workload and at the full
classifier and wide-array sizes (8 batch rows)."""
import numpy as np
import pytest

from oracle.sim import OracleSim
from synth import make_workload
from tests.error_band import BandSim
from tests.test_plan_cpu import SMALL


def _check(w, feeds, B, n):
    band = BandSim(w.spec, minibatch=B)
    band.run_steps(n, feeds)
    ref = OracleSim(w.spec, minibatch=B, param_dtype=np.float32)
    ref.run_steps(n, feeds)
    f32 = OracleSim(w.spec, minibatch=B, arith_dtype=np.float32)
    f32.run_steps(n, feeds)
    worst = 0.0
    for pi, p in enumerate(w.spec.probes):
        exp = ref.data(pi)
        assert np.array_equal(band.data(pi), exp)
        if p.target[0] == "neurons":
            continue
        dev = np.abs(f32.data(pi).astype(np.float64) - exp)
        lim = band.band(pi) + 1e-5 * np.abs(exp).max()
        assert np.all(dev <= lim), (pi, float((dev - lim).max()))
        worst = max(worst, float((dev / lim).max()))
    return worst


@pytest.mark.parametrize("neuron_type", ["lif_rate", "relu"])
@pytest.mark.parametrize("name", list(SMALL))
def test_band_contains_float32_run_small(name, neuron_type):
    w = make_workload(name, neuron_type=neuron_type, **SMALL[name])
    print(f"{name}: float32 deviation / band at most {_check(w, w.feeds, w.minibatch, w.n_steps):.2f}")


@pytest.mark.parametrize("name", ["c3", "c4"])
def test_band_contains_float32_run_full_size(name):
    w = make_workload(name, neuron_type="lif_rate")
    rows = np.arange(0, w.minibatch, 73)[:8]
    feeds = {k: f[rows] for k, f in w.feeds.items()}
    print(f"{name}: float32 deviation / band at most {_check(w, feeds, len(rows), w.n_steps):.2f}")


def test_band_refuses_spiking_neurons():
    w = make_workload("c1", n_steps=5)
    with pytest.raises(ValueError):
        BandSim(w.spec)
