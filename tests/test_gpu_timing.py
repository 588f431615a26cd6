"""GPU: per-kernel timing of the stream-ordered launch driver
(ms_sim_set_timing / ms_sim_kernel_time), the basis of the benchmark's
roofline.  Each timed interval is one group's execution (from its first
kernel's start to its last kernel's end), so per operator type the busy time
is at most the run's device time, every type together at most the run, and
every launch of a type is counted."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from synth import make_workload

pytestmark = pytest.mark.gpu
MS = M.mergesim


@pytest.mark.parametrize("name,kw", [
    ("c5", dict(n_steps=50, n_ens=40, n_neurons=100, n_eval=200, n_input_targets=8, n_probed=4)),
    ("pes", dict(n_steps=50, minibatch=4, D=16, neurons_per_dim=40)),
])
def test_kernel_times_fit_in_the_run(name, kw):
    w = make_workload(name, **kw)
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, driver=M.DRIVER_STEPS,
                     probe_capacity_steps=2 * w.n_steps) as sim:
        sim.run_steps(w.n_steps, w.feeds)          # warm-up
        sim.set_timing(True)
        sim.run_steps(w.n_steps, w.feeds)
        run_ms = sim.last_run_ms()
        times = {t: sim.kernel_time(t) for t in range(14)}
        groups = sim.info()["groups_per_step"]
    total = sum(ms for ms, _ in times.values())
    launches = sum(n for _, n in times.values())
    print(f"{name}: run {run_ms:.3f} ms, timed groups {total:.3f} ms over {launches} launches; "
          + ", ".join(f"type {t}: {ms:.3f} ms / {n}" for t, (ms, n) in times.items() if n))
    assert launches >= w.n_steps * groups - w.n_steps   # groups with no rows are not launched
    assert all(ms >= 0 for ms, _ in times.values())
    assert total <= run_ms * 1.001 + 1e-3
    if name == "pes":
        ms, n = times[MS.OP_PES_DECODE_UPDATE]
        assert n == w.n_steps and ms > 0
