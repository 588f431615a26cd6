"""Seeded synthetic model descriptions and input feeds.

This package is shared test input: it draws the random parameters of the
benchmark-shaped models (encoders, firing-rate distributions, intercepts,
evaluation points, transforms, feeds) and holds none of the simulation's
arithmetic.  Both the CPU oracle and the GPU library consume what it returns.
"""
from .spec import Ensemble, Node, Connection, Probe, ModelSpec, Workload
from .configs import make_workload, make_train, CONFIG_NAMES

__all__ = ["Ensemble", "Node", "Connection", "Probe", "ModelSpec", "Workload",
           "make_workload", "make_train", "CONFIG_NAMES"]
