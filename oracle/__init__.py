"""CPU float64 oracle of the merged-operator simulation -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  The GPU library never
calls it and shares no code with it.

Contents
  neurons.py      LIF rate curve, exact-integration LIF step, gain/bias from
                  (max rate, intercept)
  build.py        per-ensemble parameters and least-squares decoders
  sim.py          unmerged, per-object float64 stepper (the definition of what
                  a timestep computes)
  scalar.py       pure-Python per-neuron interpreter used to brute-force-check
                  sim.py on tiny models
  planner_ref.py  independent implementation of operator merging, planning,
                  sorting and simplification (paper Sec. 4.2)
  train.py        objective, gradients and gradient-descent steps of a
                  rate-neuron model through the unrolled simulation (Sec. 3.2)

Parity status of each function is stated in its docstring; anything not pinned
by a closed form, a library routine or brute force says "parity unpinned".
"""
