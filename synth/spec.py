"""Plain-data description of a Nengo-style model (Network of Nodes, Ensembles,
Connections and Probes; paper Sec. 2.1.2) plus a workload (minibatch size,
number of timesteps, per-node input feeds shaped [batch, timesteps, dims],
paper Sec. 3.1).

Object references are (kind, index) pairs:
  ("node", i)      output of node i (or a passthrough node's summed input)
  ("ens", i)       decoded (represented) value of ensemble i      -- pre / probe
                   the ensemble's represented input                 -- post
  ("neurons", i)   spike output of ensemble i's neurons            -- pre / probe
                   the neurons' input current (scaled by gain)     -- post
  ("learning", c)  error input of connection c's learning rule     -- post only
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple, Union

import numpy as np

Ref = Tuple[str, int]


@dataclass
class Ensemble:
    n_neurons: int
    dims: int
    encoders: np.ndarray                 # [n, d] float64, rows of unit length
    eval_points: np.ndarray              # [M, d] float64, used by decoder solves
    max_rates: Optional[np.ndarray] = None   # [n] Hz
    intercepts: Optional[np.ndarray] = None  # [n]
    gains: Optional[np.ndarray] = None       # [n]; overrides max_rates/intercepts
    biases: Optional[np.ndarray] = None      # [n]
    neuron_type: str = "lif"             # "lif" (spiking) | "lif_rate" | "softlif_rate" | "relu"
    tau_rc: float = 0.02
    tau_ref: float = 0.002
    amplitude: float = 1.0
    sigma: float = 0.02                  # smoothing of the "softlif_rate" curve (ignored otherwise)


@dataclass
class Node:
    size: int
    value: Optional[np.ndarray] = None   # constant output when not fed (zeros if None)
    passthrough: bool = False            # output = sum of its inputs in the same step


@dataclass
class PES:
    """Prescribed Error Sensitivity rule on a decoded connection's output
    weights (paper Sec. 5.1, the pes benchmark; MacNeil and Eliasmith 2011).
    Every step each batch row's decoders move against the error:
    D <- D - (learning_rate * dt / n) * outer(pre activities, error), the pre
    activities lowpass-filtered with time constant pre_synapse (None: this
    step's activities)."""
    learning_rate: float = 1e-4
    pre_synapse: Optional[float] = 0.005


@dataclass
class Connection:
    pre: Ref
    post: Ref
    # scalar, or matrix of shape [post_slice_size, pre_slice_size (or function output size)]
    transform: Union[float, np.ndarray] = 1.0
    function: str = "identity"           # "identity" | "product" (x0*x1) for ("ens", i) pre
    decoders: Optional[np.ndarray] = None    # explicit [n, d_fn] decoders (skip the solve)
    synapse: Optional[float] = None      # lowpass time constant in s; None = no filter
    pre_slice: Optional[Tuple[int, int]] = None   # [start, stop) of the pre output
    post_slice: Optional[Tuple[int, int]] = None  # [start, stop) of the post input
    learning_rule: Optional[PES] = None  # decoded connections only: per-batch learned decoders


@dataclass
class Probe:
    target: Ref                          # ("node", i) | ("ens", i) decoded | ("neurons", i) spikes
    synapse: Optional[float] = None
    neuron_slice: Optional[Tuple[int, int]] = None  # for ("neurons", i) targets


@dataclass
class ModelSpec:
    nodes: List[Node] = field(default_factory=list)
    ensembles: List[Ensemble] = field(default_factory=list)
    connections: List[Connection] = field(default_factory=list)
    probes: List[Probe] = field(default_factory=list)
    dt: float = 0.001

    def add_node(self, node: Node) -> Ref:
        self.nodes.append(node)
        return ("node", len(self.nodes) - 1)

    def add_ensemble(self, ens: Ensemble) -> int:
        self.ensembles.append(ens)
        return len(self.ensembles) - 1

    def connect(self, conn: Connection) -> int:
        self.connections.append(conn)
        return len(self.connections) - 1

    def probe(self, probe: Probe) -> int:
        self.probes.append(probe)
        return len(self.probes) - 1


@dataclass
class Workload:
    name: str
    spec: ModelSpec
    minibatch: int
    n_steps: int
    feeds: Dict[int, np.ndarray]         # node index -> float32 [B, T, size]
    notes: str = ""

    @property
    def n_neurons(self) -> int:
        return int(sum(e.n_neurons for e in self.spec.ensembles))

    @property
    def neuron_steps(self) -> int:
        return self.n_neurons * self.n_steps * self.minibatch
