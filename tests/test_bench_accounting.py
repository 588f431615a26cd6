"""The algorithmic work that bench.py divides by measured time, checked
against hand derivations from the workload shapes (sizes in bytes and flops
per timestep; float32)."""
import pytest

import bench
from synth import make_workload


def test_c5_bytes_per_step_by_hand():
    """5000 ensembles x 500 LIF x 16-D, B = 1: V and refractory time read and
    written (16 B per neuron), bias and encoders (17 floats per neuron),
    decoders (16 per neuron), 20,000 16x16 transforms and 100 16x32 input
    transforms, 320,000 + 1,600 filtered values read and written, 32 fed
    values."""
    w = make_workload("c5")
    N = 5000 * 500
    expect = (16 * N + 4 * N * 17 + 4 * N * 16 + 4 * (20000 * 256 + 100 * 16 * 32)
              + 8 * (20000 * 16 + 100 * 16) + 4 * 32)
    assert bench.compulsory_bytes_per_step(w) == expect


def test_c3_flops_per_step_by_hand():
    """784 -> 1024 -> 1024 -> 10 at B = 256: the three weight products plus the
    one-dimensional 'encoders' of the neuron-space layers (2 flops per neuron)."""
    w = make_workload("c3")
    B = 256
    expect = 2 * B * (1024 * 784 + 1024 * 1024 + 10 * 1024) + 2 * B * 2048
    got = bench.gemm_flops_per_step(w)
    assert got == pytest.approx(expect, rel=1e-3)


@pytest.mark.parametrize("name, mb, mflop", [("c2", 13.8, 10.2), ("c4", 846, 3321)])
def test_c2_c4_magnitudes(name, mb, mflop):
    """C2 and C4 bytes and flops per step, to 1%: 13.8 MB and 10.2 MFLOP (C2),
    846 MB and 3321 MFLOP (C4)."""
    w = make_workload(name)
    assert bench.compulsory_bytes_per_step(w) / 1e6 == pytest.approx(mb, rel=0.01)
    assert bench.gemm_flops_per_step(w) / 1e6 == pytest.approx(mflop, rel=0.01)


def test_c4_ensemble_gemm_flops_by_hand():
    """The matrix-core work of C4's fused ensembles: 200 ensembles x 500
    neurons x 512 batch rows, 16-D encoders (every ensemble has an input: the
    chain and the input node) and 16 decoded outputs, 2 flops per
    multiply-add."""
    w = make_workload("c4")
    assert bench.ensemble_gemm_flops_per_step(w) == 200 * 500 * 512 * 2 * (16 + 16)


def test_mean_ci95_matches_student_t():
    """95% interval of five values by hand: mean 2, sample sd 1.5811, t(0.975, 4)
    = 2.7764 -> half-width 1.9632."""
    m, h = bench.mean_ci95([0.0, 1.0, 2.0, 3.0, 4.0])
    assert m == pytest.approx(2.0)
    assert h == pytest.approx(2.7764451 * 1.5811388 / 5 ** 0.5, rel=1e-6)
