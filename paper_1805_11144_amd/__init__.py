"""mergesim: merged-operator spiking-network simulator for one MI355X.

The simulation runs in ``libmergesim.so`` (hand-written HIP kernels for gfx950
behind a C ABI, declared in include/mergesim.h).  This package is the thin
Python binding: argument marshalling only.
"""
from .mergesim import (Model, Plan, Simulator, MergesimError, load_library, model_from_spec,
                       DRIVER_AUTO, DRIVER_STEPS, DRIVER_GRAPH, DRIVER_PERSISTENT, DRIVER_WINDOW,
                       GEMM_F32, GEMM_BF16, PLANNER_GREEDY, PLANNER_TREE, DECODE_DENSE, DECODE_EVENT)

__all__ = ["Model", "Plan", "Simulator", "MergesimError", "load_library", "model_from_spec",
           "DRIVER_AUTO", "DRIVER_STEPS", "DRIVER_GRAPH", "DRIVER_PERSISTENT", "DRIVER_WINDOW",
           "GEMM_F32", "GEMM_BF16", "PLANNER_GREEDY", "PLANNER_TREE", "DECODE_DENSE", "DECODE_EVENT"]
