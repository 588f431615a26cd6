"""ctypes binding of libmergesim (include/mergesim.h).  Marshalling only: every
step of the simulation runs in the library's HIP kernels."""
from __future__ import annotations

import ctypes as C
import json
import os
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmergesim.so")

MS_OK = 0
REF_NODE, REF_ENS, REF_NEURONS, REF_LEARNING = 0, 1, 2, 3
NEURON_LIF, NEURON_LIF_RATE, NEURON_RELU, NEURON_SOFTLIF_RATE = 0, 1, 2, 3
FN_IDENTITY, FN_PRODUCT = 0, 1
PLANNER_GREEDY, PLANNER_TREE = 0, 1
DRIVER_AUTO, DRIVER_STEPS, DRIVER_GRAPH, DRIVER_PERSISTENT, DRIVER_WINDOW = 0, 1, 2, 3, 4
GEMM_F32, GEMM_BF16 = 0, 1
FUSE_ENSEMBLES, FUSE_SYNAPSES = 1, 2
PROBE_READ_STATIC_MAX = 1 << 22
DECODE_DENSE, DECODE_EVENT = 0, 1
PARAM_GAIN, PARAM_BIAS, PARAM_DECODERS = 0, 1, 2
(STATE_VOLTAGE, STATE_REFRACTORY, STATE_SYNAPSE, STATE_PROBE_SYNAPSE, STATE_LEARNED_DECODERS,
 STATE_PES_ACTIVITY) = range(6)
(OP_FEED, OP_RESET, OP_COPY, OP_COPY_INC, OP_ELEMENTWISE_INC, OP_DOT_INC, OP_LIF, OP_LIF_RATE, OP_LOWPASS,
 OP_ENSEMBLE, OP_SYNAPSE_SCATTER, OP_LEARNED_DECODE, OP_PES, OP_PES_DECODE_UPDATE) = range(14)
OP_GRAD_WEIGHTS, OP_GRAD_INPUTS, OP_GRAD_OTHER, OP_GRAD_WEIGHTS_SMALL = 14, 15, 16, 17
TRAIN_ENCODERS, TRAIN_BIASES, TRAIN_DECODERS, TRAIN_CONN_DECODERS, TRAIN_TRANSFORM = range(5)

_dp = C.POINTER(C.c_double)
_fp = C.POINTER(C.c_float)
_i32 = C.c_int32
_i64 = C.c_int64


class EnsembleDesc(C.Structure):
    _fields_ = [("n_neurons", _i32), ("dims", _i32), ("neuron_type", _i32),
                ("tau_rc", C.c_double), ("tau_ref", C.c_double), ("amplitude", C.c_double),
                ("encoders", _dp), ("max_rates", _dp), ("intercepts", _dp), ("gains", _dp),
                ("biases", _dp), ("n_eval_points", _i32), ("eval_points", _dp), ("sigma", C.c_double)]


class ConnectionDesc(C.Structure):
    _fields_ = [("pre_kind", _i32), ("pre_id", _i32), ("pre_start", _i32), ("pre_stop", _i32),
                ("post_kind", _i32), ("post_id", _i32), ("post_start", _i32), ("post_stop", _i32),
                ("function", _i32), ("decoders", _dp), ("decoders_cols", _i32),
                ("transform_rows", _i32), ("transform_cols", _i32), ("transform", _dp),
                ("transform_scalar", C.c_double), ("synapse_tau", C.c_double)]


class ProbeDesc(C.Structure):
    _fields_ = [("target_kind", _i32), ("target_id", _i32), ("start", _i32), ("stop", _i32),
                ("synapse_tau", C.c_double)]


class SimOpts(C.Structure):
    _fields_ = [("dt", C.c_double), ("minibatch", _i32), ("unroll", _i32), ("planner", _i32),
                ("planner_depth", _i32), ("merge", _i32), ("sort", _i32), ("simplify", _i32),
                ("fuse", _i32),
                ("driver", _i32), ("device", _i32), ("stream", C.c_void_p),
                ("probe_capacity_steps", _i64), ("gemm_dtype", _i32), ("decode", _i32),
                ("spike_probe_bits", _i32)]


class Feed(C.Structure):
    _fields_ = [("node_id", _i32), ("on_device", _i32), ("data", _fp)]


class Target(C.Structure):
    _fields_ = [("probe_id", _i32), ("on_device", _i32), ("data", _fp)]


class MergesimError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"mergesim error {code}: {msg}")
        self.code = code


_LIB = None

# (name, argtypes, restype)
_SIGNATURES = [
    ("ms_model_create", [C.POINTER(C.c_void_p)], _i32),
    ("ms_model_destroy", [C.c_void_p], None),
    ("ms_model_add_node", [C.c_void_p, _i32, _dp, _i32, C.POINTER(_i32)], _i32),
    ("ms_model_add_ensemble", [C.c_void_p, C.POINTER(EnsembleDesc), C.POINTER(_i32)], _i32),
    ("ms_model_add_connection", [C.c_void_p, C.POINTER(ConnectionDesc), C.POINTER(_i32)], _i32),
    ("ms_model_add_probe", [C.c_void_p, C.POINTER(ProbeDesc), C.POINTER(_i32)], _i32),
    ("ms_model_set_pes", [C.c_void_p, _i32, C.c_double, C.c_double], _i32),
    ("ms_sim_opts_default", [C.POINTER(SimOpts)], None),
    ("ms_plan_create", [C.c_void_p, C.POINTER(SimOpts), C.POINTER(C.c_void_p)], _i32),
    ("ms_plan_destroy", [C.c_void_p], None),
    ("ms_plan_export_json", [C.c_void_p, C.c_char_p, _i64, C.POINTER(_i64)], _i32),
    ("ms_plan_get_param", [C.c_void_p, _i32, _i32, _i32, _dp, _i64, C.POINTER(_i64)], _i32),
    ("ms_plan_export_base", [C.c_void_p, _i32, _fp, _i64, C.POINTER(_i64)], _i32),
    ("ms_sim_create", [C.c_void_p, C.POINTER(SimOpts), C.POINTER(C.c_void_p)], _i32),
    ("ms_sim_destroy", [C.c_void_p], None),
    ("ms_sim_run_steps", [C.c_void_p, _i64, C.POINTER(Feed), _i32], _i32),
    ("ms_sim_sync", [C.c_void_p], _i32),
    ("ms_sim_steps", [C.c_void_p, C.POINTER(_i64)], _i32),
    ("ms_sim_probe_width", [C.c_void_p, _i32, C.POINTER(_i32)], _i32),
    ("ms_sim_probe_read", [C.c_void_p, _i32, _fp, _i64, _i32], _i32),
    ("ms_sim_probe_read_static", [C.c_void_p, _i32, _fp, _i64], _i32),
    ("ms_sim_probe_read_bits", [C.c_void_p, _i32, C.POINTER(C.c_uint32), _i64, _i32], _i32),
    ("ms_sim_reset", [C.c_void_p], _i32),
    ("ms_sim_get_state", [C.c_void_p, _i32, _i32, _fp, _i64], _i32),
    ("ms_sim_set_state", [C.c_void_p, _i32, _i32, _fp, _i64], _i32),
    ("ms_sim_last_run_ms", [C.c_void_p, C.POINTER(C.c_double)], _i32),
    ("ms_sim_set_timing", [C.c_void_p, _i32], _i32),
    ("ms_sim_kernel_time", [C.c_void_p, _i32, C.POINTER(C.c_double), C.POINTER(_i64)], _i32),
    ("ms_sim_info", [C.c_void_p, C.POINTER(_i32), C.POINTER(_i32)], _i32),
    ("ms_sim_set_check_feeds", [C.c_void_p, _i32], _i32),
    ("ms_sim_train_step", [C.c_void_p, _i64, C.POINTER(Feed), _i32, C.POINTER(Target), _i32, C.c_double,
                           _dp], _i32),
    ("ms_sim_train_param", [C.c_void_p, _i32, _i32, _i32, _i32, _fp, _i64, C.POINTER(_i64)], _i32),
    ("ms_sim_set_train_param", [C.c_void_p, _i32, _i32, _i32, _fp, _i64], _i32),
    ("ms_last_error", [], C.c_char_p),
]


def load_library(path: str = LIB_PATH, host_only: bool = False):
    """Load libmergesim.so; raise loudly if it has not been built.
    host_only: the library holds the host part only (model, plan and JSON
    calls; a sanitizer build of the planner), the simulator calls are absent."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: the HIP library has not been built "
                          "(run `python -c 'import __graft_entry__ as g; g.build()'`)")
    lib = C.CDLL(path)
    for name, args, res in _SIGNATURES:
        fn = getattr(lib, name, None)
        if fn is None and host_only and name.startswith("ms_sim_") and name != "ms_sim_opts_default":
            continue
        if fn is None:
            raise ImportError(f"{path} does not export {name}")
        fn.argtypes = args
        fn.restype = res
    _LIB = lib
    return lib


def _check(code):
    if code != MS_OK:
        msg = _LIB.ms_last_error()
        raise MergesimError(code, msg.decode() if msg else "")


def _dptr(a: Optional[np.ndarray]):
    if a is None:
        return None
    return a.ctypes.data_as(_dp)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


_KINDS = {"node": REF_NODE, "ens": REF_ENS, "neurons": REF_NEURONS, "learning": REF_LEARNING}


class Model:
    """A network description (Nodes, Ensembles, Connections, Probes)."""

    def __init__(self):
        self._lib = load_library()
        h = C.c_void_p()
        _check(self._lib.ms_model_create(C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _LIB is not None:
            _LIB.ms_model_destroy(self.handle)
            self.handle = None

    def add_node(self, size: int, value=None, passthrough=False) -> int:
        out = _i32()
        v = None if value is None else _f64(value)
        _check(self._lib.ms_model_add_node(self.handle, int(size), _dptr(v), int(bool(passthrough)),
                                           C.byref(out)))
        return out.value

    def add_ensemble(self, ens) -> int:
        keep = []

        def arr(x):
            if x is None:
                return None
            a = _f64(x)
            keep.append(a)
            return _dptr(a)
        d = EnsembleDesc()
        d.n_neurons, d.dims = int(ens.n_neurons), int(ens.dims)
        d.neuron_type = {"lif": NEURON_LIF, "lif_rate": NEURON_LIF_RATE, "relu": NEURON_RELU,
                         "softlif_rate": NEURON_SOFTLIF_RATE}[ens.neuron_type]
        d.sigma = float(getattr(ens, "sigma", 0.0))
        d.tau_rc, d.tau_ref, d.amplitude = float(ens.tau_rc), float(ens.tau_ref), float(ens.amplitude)
        d.encoders = arr(ens.encoders)
        if ens.gains is not None:
            d.gains, d.biases = arr(ens.gains), arr(ens.biases)
        else:
            d.max_rates, d.intercepts = arr(ens.max_rates), arr(ens.intercepts)
        ev = np.asarray(ens.eval_points) if ens.eval_points is not None else None
        d.n_eval_points = 0 if ev is None else int(ev.shape[0])
        d.eval_points = arr(ev)
        out = _i32()
        _check(self._lib.ms_model_add_ensemble(self.handle, C.byref(d), C.byref(out)))
        return out.value

    def add_connection(self, conn) -> int:
        keep = []
        d = ConnectionDesc()
        d.pre_kind, d.pre_id = _KINDS[conn.pre[0]], int(conn.pre[1])
        d.post_kind, d.post_id = _KINDS[conn.post[0]], int(conn.post[1])
        if conn.pre_slice is not None:
            d.pre_start, d.pre_stop = map(int, conn.pre_slice)
        if conn.post_slice is not None:
            d.post_start, d.post_stop = map(int, conn.post_slice)
        d.function = FN_PRODUCT if conn.function == "product" else FN_IDENTITY
        if conn.decoders is not None:
            dec = _f64(conn.decoders)
            keep.append(dec)
            d.decoders, d.decoders_cols = _dptr(dec), int(dec.shape[1])
        T = conn.transform
        if np.ndim(T) == 0:
            d.transform_scalar = float(T)
        else:
            t = _f64(T)
            keep.append(t)
            d.transform_rows, d.transform_cols = int(t.shape[0]), int(t.shape[1])
            d.transform = _dptr(t)
        d.synapse_tau = float(conn.synapse) if conn.synapse is not None else 0.0
        out = _i32()
        _check(self._lib.ms_model_add_connection(self.handle, C.byref(d), C.byref(out)))
        rule = getattr(conn, "learning_rule", None)
        if rule is not None:
            self.set_pes(out.value, rule.learning_rate, rule.pre_synapse)
        return out.value

    def set_pes(self, conn_id: int, learning_rate: float, pre_synapse=None) -> None:
        """PES learning on connection conn_id's decoders (ms_model_set_pes)."""
        _check(self._lib.ms_model_set_pes(self.handle, int(conn_id), float(learning_rate),
                                          0.0 if pre_synapse is None else float(pre_synapse)))

    def add_probe(self, probe) -> int:
        d = ProbeDesc()
        d.target_kind, d.target_id = _KINDS[probe.target[0]], int(probe.target[1])
        if getattr(probe, "neuron_slice", None) is not None:
            d.start, d.stop = map(int, probe.neuron_slice)
        d.synapse_tau = float(probe.synapse) if probe.synapse is not None else 0.0
        out = _i32()
        _check(self._lib.ms_model_add_probe(self.handle, C.byref(d), C.byref(out)))
        return out.value


def model_from_spec(spec) -> Model:
    """Marshal a plain-data model description (objects with the fields of
    synth.spec) into a library model, preserving object ids."""
    m = Model()
    for node in spec.nodes:
        m.add_node(node.size, None if node.passthrough else node.value, node.passthrough)
    for e in spec.ensembles:
        m.add_ensemble(e)
    for c in spec.connections:
        m.add_connection(c)
    for p in spec.probes:
        m.add_probe(p)
    return m


def make_opts(dt=0.001, minibatch=1, unroll=10, planner=PLANNER_TREE, planner_depth=3, merge=True,
              sort=True, simplify=True, fuse=True, driver=DRIVER_AUTO, device=0, stream=None,
              probe_capacity_steps=1000, gemm_dtype=None, decode=None, spike_probe_bits=False) -> SimOpts:
    o = SimOpts()
    load_library().ms_sim_opts_default(C.byref(o))
    o.dt, o.minibatch, o.unroll = float(dt), int(minibatch), int(unroll)
    o.planner, o.planner_depth = int(planner), int(planner_depth)
    o.merge, o.sort, o.simplify = int(bool(merge)), int(bool(sort)), int(bool(simplify))
    # True: every fusion (MS_FUSE_ENSEMBLES | MS_FUSE_SYNAPSES); False: none; an
    # int: the MS_FUSE_* bits
    o.fuse = (FUSE_ENSEMBLES | FUSE_SYNAPSES) if fuse is True else 0 if fuse is False else int(fuse)
    o.driver, o.device = int(driver), int(device)
    o.stream = stream
    o.probe_capacity_steps = int(probe_capacity_steps)
    if gemm_dtype is not None:
        o.gemm_dtype = {"f32": GEMM_F32, "bf16": GEMM_BF16}.get(gemm_dtype, gemm_dtype)
    if decode is not None:
        o.decode = {"dense": DECODE_DENSE, "event": DECODE_EVENT}.get(decode, decode)
    o.spike_probe_bits = int(bool(spike_probe_bits))
    return o


class Plan:
    """Host-only build + plan (no GPU): parameters and the merged plan."""

    def __init__(self, model: Model, **opts):
        self._lib = load_library()
        self.model = model
        h = C.c_void_p()
        o = make_opts(**opts)
        _check(self._lib.ms_plan_create(model.handle, C.byref(o), C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _LIB is not None:
            _LIB.ms_plan_destroy(self.handle)
            self.handle = None

    def json(self) -> dict:
        n = _i64()
        _check(self._lib.ms_plan_export_json(self.handle, None, 0, C.byref(n)))
        buf = C.create_string_buffer(n.value + 1)
        _check(self._lib.ms_plan_export_json(self.handle, buf, n.value + 1, C.byref(n)))
        return json.loads(buf.value.decode())

    def param(self, which: int, ensemble: int, function: int = FN_IDENTITY) -> np.ndarray:
        n = _i64()
        _check(self._lib.ms_plan_get_param(self.handle, which, ensemble, function, None, 0, C.byref(n)))
        out = np.empty(n.value, np.float64)
        _check(self._lib.ms_plan_get_param(self.handle, which, ensemble, function, _dptr(out), n.value,
                                           C.byref(n)))
        return out


def _plan_base(self, base: int) -> np.ndarray:
    n = _i64()
    _check(self._lib.ms_plan_export_base(self.handle, base, None, 0, C.byref(n)))
    out = np.empty(n.value, np.float32)
    _check(self._lib.ms_plan_export_base(self.handle, base, out.ctypes.data_as(_fp), n.value, C.byref(n)))
    return out


Plan.base = _plan_base


class Simulator:
    """GPU simulator (paper Sec. 3.1: Simulator(net, minibatch_size=...),
    run with data={node: [B, T, d]}, data[probe], reset())."""

    def __init__(self, model: Model, **opts):
        self._lib = load_library()
        self.model = model
        self.minibatch = int(opts.get("minibatch", 1))
        o = make_opts(**opts)
        h = C.c_void_p()
        _check(self._lib.ms_sim_create(model.handle, C.byref(o), C.byref(h)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None) and _LIB is not None:
            _LIB.ms_sim_destroy(self.handle)
            self.handle = None

    __del__ = close

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def _arrays(self, n_steps, items, Struct, key, what):
        """ctypes array of Struct (Feed or Target) for {id: [B, n_steps, w]}
        data (numpy, or torch tensors on the simulator's device), and the
        objects that keep the data alive."""
        arr = (Struct * max(1, len(items)))()
        keep = []
        for i, (ident, data) in enumerate(items.items()):
            setattr(arr[i], key, int(ident))
            if hasattr(data, "is_cuda") and data.is_cuda:
                t = data.contiguous()
                keep.append(t)
                arr[i].on_device = 1
                arr[i].data = C.cast(C.c_void_p(t.data_ptr()), _fp)
            else:
                a = np.ascontiguousarray(np.asarray(data, dtype=np.float32))
                if a.ndim != 3 or a.shape[0] != self.minibatch or a.shape[1] < n_steps:
                    raise ValueError(f"{what} for {ident} has shape {a.shape}")
                a = np.ascontiguousarray(a[:, :n_steps])
                keep.append(a)
                arr[i].on_device = 0
                arr[i].data = a.ctypes.data_as(_fp)
        return arr, keep

    def run_steps(self, n_steps: int, feeds: Optional[Dict[int, object]] = None):
        """Advance n_steps.  feeds: node id -> float32 [B, n_steps, size]
        (numpy array, or a torch tensor on the simulator's device)."""
        feeds = feeds or {}
        arr, keep = self._arrays(n_steps, feeds, Feed, "node_id", "feed")
        _check(self._lib.ms_sim_run_steps(self.handle, int(n_steps), arr, len(feeds)))
        del keep

    def train_step(self, n_steps: int, feeds: Optional[Dict[int, object]], targets: Dict[int, object],
                   learning_rate: float = 0.0) -> float:
        """One training step (ms_sim_train_step, paper Sec. 3.2): a run of
        n_steps from the initial state, the mean-squared-error objective of
        the probes in `targets` (probe id -> [B, n_steps, width]), its
        gradient through the run, and p <- p - learning_rate * dL/dp.
        Returns the objective.  Needs driver=DRIVER_WINDOW, fuse=False,
        simplify=False and rate neurons."""
        feeds = feeds or {}
        farr, fkeep = self._arrays(n_steps, feeds, Feed, "node_id", "feed")
        tarr, tkeep = self._arrays(n_steps, targets, Target, "probe_id", "target")
        loss = C.c_double()
        _check(self._lib.ms_sim_train_step(self.handle, int(n_steps), farr, len(feeds), tarr, len(targets),
                                           float(learning_rate), C.byref(loss)))
        del fkeep, tkeep
        return loss.value

    def train_param(self, which: int, ident: int, function: int = FN_IDENTITY, gradient: bool = False):
        """A trained parameter (TRAIN_*) or its gradient from the last
        train_step, float32, flat in the layout of ms_sim_train_param."""
        n = _i64()
        _check(self._lib.ms_sim_train_param(self.handle, which, ident, function, int(bool(gradient)), None, 0,
                                            C.byref(n)))
        out = np.empty(n.value, np.float32)
        _check(self._lib.ms_sim_train_param(self.handle, which, ident, function, int(bool(gradient)),
                                            out.ctypes.data_as(_fp), n.value, C.byref(n)))
        return out

    def set_train_param(self, which: int, ident: int, values, function: int = FN_IDENTITY) -> None:
        a = np.ascontiguousarray(np.asarray(values, np.float32).ravel())
        _check(self._lib.ms_sim_set_train_param(self.handle, which, ident, function, a.ctypes.data_as(_fp),
                                                a.size))

    def sync(self):
        _check(self._lib.ms_sim_sync(self.handle))

    @property
    def n_steps(self) -> int:
        n = _i64()
        _check(self._lib.ms_sim_steps(self.handle, C.byref(n)))
        return n.value

    def probe_width(self, probe: int) -> int:
        w = _i32()
        _check(self._lib.ms_sim_probe_width(self.handle, probe, C.byref(w)))
        return w.value

    def data(self, probe: int) -> np.ndarray:
        """Probe record [B, steps, width] (float32)."""
        w = self.probe_width(probe)
        T = self.n_steps
        out = np.empty((self.minibatch, T, w), np.float32)
        _check(self._lib.ms_sim_probe_read(self.handle, probe, out.ctypes.data_as(_fp), out.size, 0))
        return out

    def data_bits(self, probe: int) -> np.ndarray:
        """Spike probe record as bitmasks [B, steps, ceil(width / 32)] uint32
        (simulators created with spike_probe_bits=True)."""
        nw = (self.probe_width(probe) + 31) // 32
        out = np.empty((self.minibatch, self.n_steps, nw), np.uint32)
        _check(self._lib.ms_sim_probe_read_bits(self.handle, probe, out.ctypes.data_as(C.POINTER(C.c_uint32)),
                                                out.size, 0))
        return out

    def data_static(self, probe: int) -> np.ndarray:
        """Probe record [B, steps, width] read without any device allocation
        (ms_sim_probe_read_static; at most PROBE_READ_STATIC_MAX values)."""
        w = self.probe_width(probe)
        T = self.n_steps
        out = np.empty((self.minibatch, T, w), np.float32)
        _check(self._lib.ms_sim_probe_read_static(self.handle, probe, out.ctypes.data_as(_fp), out.size))
        return out

    def reset(self):
        _check(self._lib.ms_sim_reset(self.handle))

    def get_state(self, which: int, ident: int, width: int) -> np.ndarray:
        out = np.empty((self.minibatch, width), np.float32)
        _check(self._lib.ms_sim_get_state(self.handle, which, ident, out.ctypes.data_as(_fp), out.size))
        return out

    def set_state(self, which: int, ident: int, values) -> None:
        a = np.ascontiguousarray(np.asarray(values, np.float32))
        _check(self._lib.ms_sim_set_state(self.handle, which, ident, a.ctypes.data_as(_fp), a.size))

    def last_run_ms(self) -> float:
        v = C.c_double()
        _check(self._lib.ms_sim_last_run_ms(self.handle, C.byref(v)))
        return v.value

    def set_timing(self, on: bool) -> None:
        _check(self._lib.ms_sim_set_timing(self.handle, 1 if on else 0))

    def kernel_time(self, op_type: int):
        """(summed ms, launches) of operator type op_type (OP_*) in the last run."""
        ms, n = C.c_double(), _i64()
        _check(self._lib.ms_sim_kernel_time(self.handle, int(op_type), C.byref(ms), C.byref(n)))
        return ms.value, n.value

    def set_check_feeds(self, on: bool) -> None:
        """Refuse feeds that hold NaN or Inf (MS_E_NUMERIC) before each run."""
        _check(self._lib.ms_sim_set_check_feeds(self.handle, 1 if on else 0))

    def info(self):
        d, g = _i32(), _i32()
        _check(self._lib.ms_sim_info(self.handle, C.byref(d), C.byref(g)))
        return {"driver": d.value, "groups_per_step": g.value}
