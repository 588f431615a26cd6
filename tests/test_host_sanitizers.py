"""The host part of the library (builder, decoder solves, IR, planner, sort,
window and step programs, JSON export, the model and plan calls) built with
AddressSanitizer and UndefinedBehaviorSanitizer and driven through the same C
ABI on every workload shape, every planner option set and the error paths: an
out-of-bounds access, a use after free or undefined behaviour aborts the run.

g++ builds the host sources only (no GPU code is involved); the run loads the
sanitizer runtime first in a child process, with leak checking off (the Python
interpreter's own allocations are not the library's)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

pytestmark = pytest.mark.slow

DRIVER = r'''
import sys
sys.path.insert(0, sys.argv[1])
import numpy as np
import paper_1805_11144_amd.mergesim as MS
MS.load_library(sys.argv[2], host_only=True)
from synth import make_workload, make_train
from synth.configs import lif_ensemble
from synth.spec import Connection

SMALL = dict(c1=dict(n_steps=5), c2=dict(n_steps=5, minibatch=2, D=8, n_neurons=20, n_eval=50),
             c3=dict(n_steps=5, minibatch=2, n_in=20, n_hidden=40, n_out=4),
             c4=dict(n_steps=5, minibatch=2, n_ens=5, n_neurons=30, dims=4, n_eval=60),
             c5=dict(n_steps=5, n_ens=40, n_neurons=30, n_eval=60),
             bg=dict(n_steps=5, D=6, n_neurons=10, n_eval=40),
             pes=dict(n_steps=5, minibatch=2, D=4, neurons_per_dim=10))
OPTS = [dict(), dict(planner=MS.PLANNER_GREEDY), dict(planner_depth=1), dict(sort=False), dict(simplify=False),
        dict(merge=False), dict(fuse=False), dict(fuse=MS.FUSE_ENSEMBLES), dict(fuse=MS.FUSE_SYNAPSES)]
n = 0
for name, kw in SMALL.items():
    for nt in (["lif", "lif_rate", "relu", "softlif_rate"] if name != "pes" else ["lif", "lif_rate"]):
        w = make_workload(name, neuron_type=nt, **kw)
        for o in OPTS:
            p = MS.Plan(MS.model_from_spec(w.spec), minibatch=w.minibatch, **o)
            j = p.json()
            for b in range(len(j["bases"])):
                p.base(b)
            n += 1
for kind in ("mlp", "chain", "cconv"):
    w, _ = make_train(kind, n_steps=4, minibatch=2, **({"n_in": 10, "n_hidden": 20, "n_out": 3} if kind == "mlp" else
                      {"n_ens": 3, "n_neurons": 20, "dims": 3, "n_eval": 40} if kind == "chain" else
                      {"D": 4, "n_neurons": 10, "n_eval": 40}))
    MS.Plan(MS.model_from_spec(w.spec), minibatch=2, fuse=False, simplify=False).json()
    n += 1
# error paths: a cycle without synapse, bad ids and shapes, a failing decoder solve
m = MS.Model()
a = m.add_node(1, passthrough=True)
b = m.add_node(1, passthrough=True)
m.add_connection(Connection(pre=("node", a), post=("node", b)))
m.add_connection(Connection(pre=("node", b), post=("node", a)))
try:
    MS.Plan(m)
    raise SystemExit("cycle not reported")
except MS.MergesimError:
    pass
for bad in (dict(pre=("node", 7), post=("ens", 0)), dict(pre=("ens", 0), post=("ens", 9)),
            dict(pre=("ens", 0), post=("ens", 0), transform=np.ones((3, 5)))):
    m = MS.Model()
    m.add_ensemble(lif_ensemble(np.random.default_rng(0), 10, 2, 30, "lif"))
    try:   # refused when added or when planned
        m.add_connection(Connection(**bad))
        MS.Plan(m)
        raise SystemExit(f"bad connection accepted: {bad}")
    except MS.MergesimError:
        pass
print("planned", n)
'''


def _build(tmp):
    from paper_1805_11144_amd import build_lib
    out = os.path.join(tmp, "libmergesim_host_san.so")
    srcs = [os.path.join(build_lib.CSRC, s) for s in build_lib.HOST_SOURCES]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-I" + build_lib.INCLUDE,
           *srcs, "-o", out, "-lpthread"]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout[-4000:]
    return out


def test_planner_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    lib = _build(str(tmp_path))
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], stdout=subprocess.PIPE, text=True).stdout.strip()
    ubsan = subprocess.run(["g++", "-print-file-name=libubsan.so"], stdout=subprocess.PIPE, text=True).stdout.strip()
    env = dict(os.environ, LD_PRELOAD=f"{asan}:{ubsan}", ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-c", DRIVER, ROOT, lib], stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, env=env, timeout=1200)
    tail = r.stdout[-6000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stdout and "runtime error" not in r.stdout, tail
    assert "planned" in r.stdout, tail
