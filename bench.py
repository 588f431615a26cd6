"""Throughput of the merged-operator simulation on one MI355X.

One bench step = one simulator run over a whole synthetic batch: reset, then
n_steps timesteps for all B batch rows (every merged operator of the hot path:
feeds, encoders, LIF, decoders, transforms, lowpass synapses, copies/scatters,
probes).  Inputs are resident in HBM (torch CUDA tensors) before timing.

Metric: neuron-timesteps/s = N_neurons * T * B / wall time per run.
Default workload: the circular-convolution-shaped net (128 product ensembles of
100 LIF neurons, 2-D, D = 64, B = 64, T = 1000).

Prints one JSON line.  --gpus > 1 is not supported (single-GPU build).
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_VALU_PEAK_TFLOPS = 78.6   # 256 CU x 4 SIMD x 16 lanes x 2 flop x 2.4 GHz, no packed FP32

WORKLOADS = {
    "c1": "integrator: 1 ensemble x 100 LIF, 1-D, recurrent lowpass 0.1, B=1, T=1000",
    "c2": "cconv-shaped: 128 product ensembles x 100 LIF (2-D), D=64 DFT transforms, "
          "lowpass 0.005, B=64, T=1000",
    "c3": "spiking MLP 784-1024-1024-10, Glorot-normal, lowpass 0.005, B=256, T=50",
    "c4": "wide array: 200 ensembles x 500 LIF x 16-D chain, B=512, T=500",
    "c5": "sparse graph: 5000 ensembles x 500 LIF x 16-D, fan-out 4, B=1, T=1000",
}


def compulsory_bytes_per_step(w):
    """Algorithmic HBM bytes of one timestep, time-major: V and refractory state
    read+written (16 B per neuron-instance), every weight/parameter read once,
    filter states read+written, feeds read, probes written (float32)."""
    spec, B = w.spec, w.minibatch
    n = sum(e.n_neurons for e in spec.ensembles if e.neuron_type == "lif")
    state = 16 * n * B
    params = 0
    for e in spec.ensembles:
        params += 4 * e.n_neurons * (1 + e.dims)               # bias + scaled encoders
    decoded = set()
    for c in spec.connections:
        params += 4 * int(np.size(c.transform))
        if c.pre[0] == "ens" and (c.pre[1], c.function) not in decoded:
            decoded.add((c.pre[1], c.function))
            params += 4 * spec.ensembles[c.pre[1]].n_neurons * (1 if c.function == "product" else
                                                                 spec.ensembles[c.pre[1]].dims)
    filt = 0
    for c in spec.connections:
        if c.synapse is not None:
            w_ = (c.post_slice[1] - c.post_slice[0]) if c.post_slice else (
                spec.nodes[c.post[1]].size if c.post[0] == "node" else
                spec.ensembles[c.post[1]].dims if c.post[0] == "ens" else spec.ensembles[c.post[1]].n_neurons)
            filt += 8 * w_ * B
    feeds = 4 * B * sum(f.shape[2] for f in w.feeds.values())
    return state + params + filt + feeds


def gemm_flops_per_step(w):
    spec, B = w.spec, w.minibatch
    f = 0
    for e in spec.ensembles:
        f += 2 * e.n_neurons * e.dims * B
    dec_done = set()
    for c in spec.connections:
        if c.pre[0] == "ens":
            key = (c.pre[1], c.function)
            if key not in dec_done:
                dec_done.add(key)
                e = spec.ensembles[c.pre[1]]
                f += 2 * e.n_neurons * (1 if c.function == "product" else e.dims) * B
        f += 2 * int(np.size(c.transform)) * B
    return f


def cpu_baseline(w, budget_s=15.0):
    """Time the float64 oracle on a bounded sample of the same workload."""
    from oracle.sim import OracleSim
    try:
        import threadpoolctl
        cores = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:
        cores = os.cpu_count() or 1
    sim = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    t0 = time.perf_counter()
    k = 0
    while k < w.n_steps and time.perf_counter() - t0 < budget_s:
        sim.run_steps(1, {i: f[:, k:k + 1] for i, f in w.feeds.items()})
        k += 1
    dt = time.perf_counter() - t0
    value = w.n_neurons * k * w.minibatch / dt
    return {"value": value, "unit": "neuron-timesteps/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {k} of {w.n_steps} timesteps, all {w.minibatch} batch rows, "
                      f"float64 numpy, {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c2", choices=sorted(WORKLOADS))
    ap.add_argument("--driver", default="auto", choices=["auto", "steps", "graph", "persistent", "window"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)

    import torch

    import paper_1805_11144_amd as M
    from synth import make_workload

    w = make_workload(args.config)
    model = M.model_from_spec(w.spec)
    driver = {"auto": M.DRIVER_AUTO, "steps": M.DRIVER_STEPS, "graph": M.DRIVER_GRAPH,
              "persistent": M.DRIVER_PERSISTENT, "window": M.DRIVER_WINDOW}[args.driver]
    dev = torch.device("cuda:0")
    t_build = time.perf_counter()
    sim = M.Simulator(model, minibatch=w.minibatch, driver=driver, unroll=20,
                      probe_capacity_steps=w.n_steps)
    t_build = time.perf_counter() - t_build
    feeds = {i: torch.from_numpy(f).to(dev) for i, f in w.feeds.items()}
    torch.cuda.synchronize()

    def one_run():
        sim.reset()
        sim.run_steps(w.n_steps, feeds)

    for _ in range(args.warmup):
        one_run()
    sim.sync()
    torch.cuda.synchronize()
    kernel_ms = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_run()
        kernel_ms.append(sim.last_run_ms())
    sim.sync()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    ms_per_step = 1000.0 * elapsed / args.steps
    neuron_steps = w.n_neurons * w.n_steps * w.minibatch
    value = neuron_steps / (elapsed / args.steps)
    info = sim.info()
    launch_ms = float(np.mean(kernel_ms))
    bytes_run = compulsory_bytes_per_step(w) * w.n_steps
    achieved_gbs = bytes_run / (launch_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved_gbs / HBM_PEAK_GBS, 4), "traffic": None,
                "kernel": {1: "per-group kernels", 2: "per-group kernels (hipGraph)",
                           3: "k_persistent", 4: "stage-major window kernels"}.get(info["driver"], "?"),
                "launch_ms": round(launch_ms, 4), "bytes_per_launch": int(bytes_run)}
    out = {
        "metric": "neuron-timesteps/sec (x minibatch) on 1 MI355X",
        "value": value, "unit": "neuron-timesteps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "name": args.config, "neurons": w.n_neurons,
                   "timesteps": w.n_steps, "minibatch": w.minibatch,
                   "driver": {1: "steps", 2: "graph", 3: "persistent", 4: "window"}.get(info["driver"]),
                   "groups_per_step": info["groups_per_step"], "build_s": round(t_build, 2)},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
