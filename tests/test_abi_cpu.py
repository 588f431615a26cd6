"""The C-ABI library on a machine without a GPU: it loads, exports every entry
point include/mergesim.h declares, and its host-side calls (model building,
planning, validation and error reporting) behave as documented."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_1805_11144_amd as M
from paper_1805_11144_amd import mergesim as MS
from synth import Connection, Ensemble, ModelSpec, Node, Probe, make_workload

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "mergesim.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ms_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = MS.load_library()
    names = declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n


def _status_of(fn):
    try:
        fn()
    except MS.MergesimError as e:
        return e.code, str(e)
    return 0, ""


def test_validation_errors_are_reported():
    m = M.Model()
    code, msg = _status_of(lambda: m.add_node(0))
    assert code == -1 and "size" in msg
    m.add_node(2)
    ens = Ensemble(n_neurons=3, dims=2, encoders=np.eye(3, 2), eval_points=np.zeros((1, 2)),
                   gains=np.ones(3), biases=np.ones(3))
    m.add_ensemble(ens)
    # transform of the wrong shape
    code, msg = _status_of(lambda: M.Plan(_with(m, Connection(pre=("node", 0), post=("ens", 0),
                                                               transform=np.ones((3, 2))))))
    assert code == -1 and "transform" in msg
    # out-of-range id
    code, msg = _status_of(lambda: M.Plan(_with(m, Connection(pre=("node", 5), post=("ens", 0)))))
    assert code == -1


def _with(model, conn):
    model.add_connection(conn)
    return model


def test_unfiltered_cycle_is_reported():
    spec = ModelSpec()
    spec.add_node(Node(size=1, passthrough=True))
    spec.add_node(Node(size=1, passthrough=True))
    spec.connect(Connection(pre=("node", 0), post=("node", 1)))
    spec.connect(Connection(pre=("node", 1), post=("node", 0)))
    code, msg = _status_of(lambda: M.Plan(M.model_from_spec(spec)))
    assert code == -2 and "cycle" in msg


def test_filtered_cycle_is_fine():
    w = make_workload("c1", n_steps=5)
    plan = M.Plan(M.model_from_spec(w.spec)).json()
    assert plan["groups"]


def test_decoder_solve_failure_is_numeric_error():
    spec = ModelSpec()
    spec.add_ensemble(Ensemble(n_neurons=4, dims=1, encoders=np.ones((4, 1)),
                               eval_points=np.full((10, 1), -1.0),
                               max_rates=np.full(4, 300.0), intercepts=np.full(4, 0.5)))
    spec.probe(Probe(target=("ens", 0)))
    code, msg = _status_of(lambda: M.Plan(M.model_from_spec(spec)))
    assert code == -6


def test_plan_json_sizes_with_zero_capacity():
    w = make_workload("c1", n_steps=5)
    plan = M.Plan(M.model_from_spec(w.spec))
    n = C.c_int64()
    MS._check(MS._LIB.ms_plan_export_json(plan.handle, None, 0, C.byref(n)))
    assert n.value > 100
    small = C.create_string_buffer(11)
    MS._check(MS._LIB.ms_plan_export_json(plan.handle, small, 11, C.byref(n)))
    assert len(small.value) == 10


def test_sim_creation_without_gpu_fails_cleanly():
    # the GPU driver's device node, checked without starting a GPU runtime in
    # this process (torch brings its own HIP runtime besides the library's)
    if os.path.exists("/dev/kfd"):
        pytest.skip("a GPU is present")
    w = make_workload("c1", n_steps=5)
    code, msg = _status_of(lambda: M.Simulator(M.model_from_spec(w.spec)))
    assert code in (-1, -4)


def test_sim_opts_defaults_and_decode_field():
    """ms_sim_opts_default fills the decode option (dense) at the offset the
    binding's structure declares; the event value marshals through."""
    o = MS.make_opts()
    assert o.decode == M.DECODE_DENSE and o.gemm_dtype == M.GEMM_F32
    assert MS.make_opts(decode="event").decode == M.DECODE_EVENT
