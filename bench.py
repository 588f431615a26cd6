"""Throughput of the merged-operator simulation on one MI355X.

One bench step = one simulator run over a whole synthetic batch: reset, then
n_steps timesteps for all B batch rows (every merged operator of the hot path:
feeds, encoders, LIF, decoders, transforms, lowpass synapses, copies/scatters,
probes).  Inputs are resident in HBM (torch CUDA tensors) before timing.

Metric: neuron-timesteps/s = N_neurons * T * B / wall time per run (the mean
over the timed runs, with a 95% confidence interval as in the paper's speed
measurements, Sec. 5.1).
Default workload: the wide ensemble array (200 ensembles x 500 LIF x 16-D in a
chain, B = 512, T = 500), the largest of the five workloads.

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
# VALU issue peak in wavefront instructions per second: a full-rate wave64
# instruction occupies a 16-lane SIMD for 4 cycles; 256 CU x 4 SIMD x 2.4 GHz / 4
VALU_ISSUE_PEAK = 256 * 4 * 2.4e9 / 4

WORKLOADS = {
    "c1": "integrator: 1 ensemble x 100 LIF, 1-D, recurrent lowpass 0.1, B=1, T=1000",
    "c2": "cconv-shaped: 128 product ensembles x 100 LIF (2-D), D=64 DFT transforms, "
          "lowpass 0.005, B=64, T=1000",
    "c3": "spiking MLP 784-1024-1024-10, Glorot-normal, lowpass 0.005, B=256, T=50",
    "c4": "wide array: 200 ensembles x 500 LIF x 16-D chain, B=512, T=500",
    "c5": "sparse graph: 5000 ensembles x 500 LIF x 16-D, fan-out 4, B=1, T=1000",
    "bg": "basal-ganglia-shaped: 5 arrays x 64 ensembles x 50 LIF (1-D), one-to-one and all-to-all "
          "array transforms, B=1, T=1000",
    "pes": "online learning: 192-D input -> 9600 LIF -> PES-learned decoders (one 9600x192 matrix "
           "per batch row), error lowpass 0.005, B=10, T=1000",
    "train": "training step: rate classifier 784-1024-1024-10 (smoothed LIF rate, sigma 0.02), lowpass 0.005, mean squared error "
             "on one-hot targets at every step, gradient through all T=50 steps, B=256, gradient-descent update",
}
TRAIN_LR = 1e-4


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
    learned = 0
    for c in spec.connections:
        params += 4 * int(np.size(c.transform))
        if c.learning_rule is not None:
            # per-batch-row decoders read and written every step, and the
            # activity filter state
            learned += pes_bytes_per_launch(spec, c, B)
            continue
        if c.pre[0] == "ens" and (c.pre[1], c.function) not in decoded:
            decoded.add((c.pre[1], c.function))
            params += 4 * spec.ensembles[c.pre[1]].n_neurons * (1 if c.function == "product" else
                                                                 spec.ensembles[c.pre[1]].dims)
    filt = 0
    for c in spec.connections:
        if c.synapse is not None:
            w_ = (c.post_slice[1] - c.post_slice[0]) if c.post_slice else _post_width(spec, c)
            filt += 8 * w_ * B
    feeds = 4 * B * sum(f.shape[2] for f in w.feeds.values())
    return state + params + filt + feeds + learned


def _post_width(spec, c):
    kind, i = c.post
    if kind == "node":
        return spec.nodes[i].size
    if kind == "ens":
        return spec.ensembles[i].dims
    if kind == "learning":
        lc = spec.connections[i]
        return np.asarray(lc.decoders).shape[1] if lc.decoders is not None else spec.ensembles[lc.pre[1]].dims
    return spec.ensembles[i].n_neurons


def pes_bytes_per_launch(spec, c, B):
    """Algorithmic bytes of one PES decode + update pass over one learned
    connection (n neurons, k outputs): the decoders read and written (8 n k B),
    the activities and their filter read (8 n B), the error read and the
    decoded output written (8 k B)."""
    n = spec.ensembles[c.pre[1]].n_neurons
    k = np.asarray(c.decoders).shape[1] if c.decoders is not None else spec.ensembles[c.pre[1]].dims
    return 8 * n * k * B + 8 * n * B + 8 * k * B


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


LIF_FLOPS = 21    # exact-integration LIF step: clamp 3, factor 2, voltage 3, refractory 2, threshold 1,
                  # overshoot 3, crossing time 4, resets 3 operations per neuron-step
RATE_FLOPS = 7    # rate LIF
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0   # dense


def ensemble_work_per_step(w):
    """(flops, bytes) of the fused ensemble operators in one timestep: per
    neuron and batch row the encoders (2d), bias (1), neuron update and fused
    decoders (2 per decoded dimension); bytes as a time-major pass moves them
    (parameters once, V/refractory state read and written, inputs and decoded
    outputs)."""
    spec, B = w.spec, w.minibatch
    ndec = {}
    for c in spec.connections:
        if c.pre[0] == "ens" and c.decoders is None:
            e = spec.ensembles[c.pre[1]]
            ndec.setdefault(c.pre[1], {})[c.function] = 1 if c.function == "product" else e.dims
    for p in spec.probes:
        if p.target[0] == "ens":
            ndec.setdefault(p.target[1], {})["identity"] = spec.ensembles[p.target[1]].dims
    flops = byts = 0
    for i, e in enumerate(spec.ensembles):
        nd = sum(ndec.get(i, {}).values())
        nf = LIF_FLOPS if e.neuron_type == "lif" else RATE_FLOPS
        flops += e.n_neurons * B * (2 * e.dims + 1 + nf + 2 * nd)
        byts += 4 * e.n_neurons * (e.dims + 1 + nd) + 4 * B * (e.dims + nd)
        if e.neuron_type == "lif":
            byts += 16 * e.n_neurons * B
    return flops, byts


def ensemble_gemm_flops_per_step(w):
    """Matrix-product flops of the fused ensemble operators in one timestep:
    per neuron and batch row 2 d for the encoders (ensembles with a
    represented input) and 2 per decoded output for the decoders -- the
    products that run on the matrix cores."""
    spec, B = w.spec, w.minibatch
    ndec = {}
    fed = set()
    for c in spec.connections:
        if c.pre[0] == "ens" and c.decoders is None:
            e = spec.ensembles[c.pre[1]]
            ndec.setdefault(c.pre[1], {})[c.function] = 1 if c.function == "product" else e.dims
        if c.post[0] == "ens":
            fed.add(c.post[1])
    for p in spec.probes:
        if p.target[0] == "ens":
            ndec.setdefault(p.target[1], {})["identity"] = spec.ensembles[p.target[1]].dims
    f = 0
    for i, e in enumerate(spec.ensembles):
        nd = sum(ndec.get(i, {}).values())
        f += 2 * e.n_neurons * B * ((e.dims if i in fed else 0) + nd)
    return f


def dot_flops_per_step(plan_json, B):
    """GEMM flops of the merged DotInc groups (2 M K per op and batch row)."""
    return sum(2 * g["M"] * g["K"] * len(g["w_row"]) * B for g in plan_json["groups"] if g["type"] == "DotInc")


def _oracle_leg(w, budget_s):
    """Oracle timesteps run within budget_s (after building it), and the time."""
    from oracle.sim import OracleSim
    sim = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    t0 = time.perf_counter()
    k = 0
    while k < w.n_steps and time.perf_counter() - t0 < budget_s:
        sim.run_steps(1, {i: f[:, k:k + 1] for i, f in w.feeds.items()})
        k += 1
    return k, time.perf_counter() - t0


def cpu_baseline(w, budget_s=12.0):
    """Time the float64 oracle on a bounded sample of the same workload: the
    first timesteps that fit in budget_s, all batch rows, extrapolated per
    timestep; once with the BLAS threads the host offers, once with one."""
    import threadpoolctl
    cores = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] or [1])
    k, dt = _oracle_leg(w, budget_s)
    with threadpoolctl.threadpool_limits(limits=1):
        k1, dt1 = _oracle_leg(w, budget_s)
    per = w.n_neurons * w.minibatch
    return {"value": per * k / dt, "unit": "neuron-timesteps/s", "cores": int(cores), "kind": "oracle",
            "sample": f"first {k} of {w.n_steps} timesteps, all {w.minibatch} batch rows, "
                      f"float64 numpy, {dt:.1f} s, {cores} BLAS threads",
            "single_thread": {"value": per * k1 / dt1, "cores": 1,
                              "sample": f"first {k1} of {w.n_steps} timesteps, {dt1:.1f} s, 1 thread"}}


def train_cpu_baseline(w, targets, budget_s=12.0):
    """Time the training oracle (float64 forward and reverse-mode gradient of
    the whole run, then the update) on a bounded sample: all steps of the
    first b batch rows, b doubled from 2 while a leg stays under a quarter of
    the budget; once with torch's CPU threads and once with one."""
    import torch
    from oracle.train import TrainOracle

    def leg():
        b, rate, dt = 2, 0.0, 0.0
        while True:
            sub = {i: f[:b] for i, f in w.feeds.items()}
            tg = {p: t[:b] for p, t in targets.items()}
            tr = TrainOracle(w.spec, b)
            t0 = time.perf_counter()
            _, g, _ = tr.loss_and_grads(w.n_steps, sub, tg)
            tr.sgd(g, TRAIN_LR)
            dt = time.perf_counter() - t0
            rate = w.n_neurons * w.n_steps * b / dt
            if dt > budget_s / 4 or 2 * b > w.minibatch:
                return b, rate, dt
            b *= 2
    threads = torch.get_num_threads()
    b, rate, dt = leg()
    torch.set_num_threads(1)
    try:
        b1, rate1, dt1 = leg()
    finally:
        torch.set_num_threads(threads)
    return {"value": rate, "unit": "neuron-timesteps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"one training step (all {w.n_steps} steps, gradient, update) of the first {b} of "
                      f"{w.minibatch} batch rows, float64 torch, {dt:.1f} s, {threads} threads",
            "single_thread": {"value": rate1, "cores": 1,
                              "sample": f"first {b1} batch rows, {dt1:.1f} s, 1 thread"}}


def train_roofline(M, sim, w, feeds, targets, plan_json):
    """Roofline of the largest operator kind of a training step, from HIP
    events with per-launch timing on (one extra step), and beside it the
    weight-gradient products on the matrix cores (k_t_dw).  Products: 2 M K
    flops per op, step and batch row, against the fp32 MFMA peak."""
    MS = M.mergesim
    sim.set_timing(True)
    sim.train_step(w.n_steps, feeds, targets, TRAIN_LR)
    times = {t: sim.kernel_time(t) for t in range(18)}
    sim.set_timing(False)
    TB = w.n_steps * w.minibatch
    dots = [g for g in plan_json["groups"] if g["type"] == "DotInc"]
    flops = lambda gs: sum(2 * g["M"] * g["K"] * len(g["w_row"]) for g in gs) * TB
    big = [g for g in dots if g["M"] >= 64 and g["K"] >= 64 and w.minibatch % 4 == 0]
    kinds = {MS.OP_DOT_INC: (flops(dots), "k_w_gemm2", "DotInc (forward)"),
             MS.OP_GRAD_WEIGHTS: (flops(big), "k_t_dw", "weight gradients")}

    def line(t):
        ms, n = times[t]
        work, kernel, op = kinds[t]
        ach = work / (ms * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": round(ach, 3), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": stored_traffic(kernel, "train"),
                "basis": "algorithmic", "kernel": kernel, "op": op, "launch_ms": round(ms / max(n, 1), 4),
                "launches": n, "busy_ms": round(ms, 4), "work_per_launch": int(work / max(n, 1))}
    top = max(times, key=lambda t: times[t][0])
    out = line(top) if top in kinds else {
        "bound": None, "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None,
        "kernel": f"timing kind {top}", "launch_ms": round(times[top][0] / max(times[top][1], 1), 4)}
    if top != MS.OP_GRAD_WEIGHTS and times[MS.OP_GRAD_WEIGHTS][1]:
        out["weight_gradients"] = line(MS.OP_GRAD_WEIGHTS)
    out["kinds_ms"] = {str(t): round(v[0], 4) for t, v in times.items() if v[1]}
    return out


def main_train(args):
    """One bench step = one training step of the classifier (ms_sim_train_step):
    a run from the initial state over the whole batch, the objective, its
    gradient through every step, and the update."""
    import torch

    import paper_1805_11144_amd as M
    from synth import make_train

    w, targets = make_train("mlp", **({"n_steps": args.timesteps} if args.timesteps else {}))
    model = M.model_from_spec(w.spec)
    dev = torch.device("cuda:0")
    opts = dict(driver=M.DRIVER_WINDOW, fuse=False, simplify=False)
    t_build = time.perf_counter()
    sim = M.Simulator(model, minibatch=w.minibatch, probe_capacity_steps=w.n_steps, **opts)
    t_build = time.perf_counter() - t_build
    feeds = {i: torch.from_numpy(f).to(dev) for i, f in w.feeds.items()}
    tg = {p: torch.from_numpy(t).to(dev) for p, t in targets.items()}
    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        del src, dst
    torch.cuda.synchronize()
    if args.counters_run:
        sim.train_step(w.n_steps, feeds, tg, TRAIN_LR)
        torch.cuda.synchronize()
        return
    for _ in range(args.warmup):
        sim.train_step(w.n_steps, feeds, tg, TRAIN_LR)
    torch.cuda.synchronize()
    run_ms, losses = [], []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        losses.append(sim.train_step(w.n_steps, feeds, tg, TRAIN_LR))   # returns when the step is done
        run_ms.append(sim.last_run_ms())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    neuron_steps = w.n_neurons * w.n_steps * w.minibatch
    run_mean, run_ci = mean_ci95(run_ms)
    plan_json = M.Plan(model, minibatch=w.minibatch, fuse=False, simplify=False).json()
    roofline = train_roofline(M, sim, w, feeds, tg, plan_json)
    out = {
        "metric": "training neuron-timesteps/sec (x minibatch) on 1 MI355X",
        "value": neuron_steps / (elapsed / args.steps), "unit": "neuron-timesteps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": 1000.0 * elapsed / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": WORKLOADS["train"], "name": "train", "neurons": w.n_neurons,
                   "timesteps": w.n_steps, "minibatch": w.minibatch, "driver": "window",
                   "learning_rate": TRAIN_LR, "build_s": round(t_build, 2),
                   "plan": {"fuse": False, "simplify": False}},
        "runs": {"device_ms": [round(x, 4) for x in run_ms], "mean_ms": round(run_mean, 4),
                 "ci95_ms": None if run_ci is None else round(run_ci, 4), "objective": losses},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = train_cpu_baseline(w, targets, args.cpu_budget)
    print(json.dumps(out))
    sim.close()


def mean_ci95(xs):
    """Mean and half-width of the 95% confidence interval (Student t)."""
    xs = np.asarray(xs, np.float64)
    if xs.size < 2:
        return float(xs.mean()), None
    from scipy import stats
    h = stats.t.ppf(0.975, xs.size - 1) * xs.std(ddof=1) / np.sqrt(xs.size)
    return float(xs.mean()), float(h)


def measure_roofline(M, model, w, sim, info, feeds, bf16=False, plan_opts=None, default_plan=True, event=False):
    """Roofline of the dominant kernel, timed with HIP events on the stream it
    runs on (one extra run with per-launch timing; the plain-launch driver
    stands in for the hipGraph driver, whose kernels are the same)."""
    T = w.n_steps
    drv = info["driver"]
    if drv == M.DRIVER_PERSISTENT:
        ms = sim.last_run_ms()
        b = compulsory_bytes_per_step(w) * T
        ach = b / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "k_persistent",
                "launch_ms": round(ms, 4), "launches": 1, "work_per_launch": int(b)}
    tsim = sim if drv in (M.DRIVER_WINDOW, M.DRIVER_STEPS) else \
        M.Simulator(model, minibatch=w.minibatch, driver=M.DRIVER_STEPS, probe_capacity_steps=T,
                    **(plan_opts or {}))
    tsim.set_timing(True)
    tsim.reset()
    tsim.run_steps(T, feeds)
    times = {t: tsim.kernel_time(t) for t in range(14)}
    tsim.set_timing(False)
    if tsim is not sim:
        tsim.close()
    top = max(times, key=lambda t: times[t][0])
    if bf16:      # the bf16 variant reports its products against the bf16 peak
        top = M.mergesim.OP_DOT_INC
    ms, n = times[top]
    window = drv == M.DRIVER_WINDOW
    if top == M.mergesim.OP_ENSEMBLE:
        flops, byts = ensemble_work_per_step(w)
        if window:    # state stays on chip across the window: the products bound it
            work, bound, peak, unit = ensemble_gemm_flops_per_step(w) * T, "mfma", FP32_MFMA_PEAK_TFLOPS, \
                "TFLOP/s"
            kernel = "k_w_ens"
        else:
            work, bound, peak, unit = byts * T, "hbm", HBM_PEAK_GBS, "GB/s"
            kernel = "k_ens_wg" if w.minibatch < 32 else "k_ens_tile"
    elif top == M.mergesim.OP_DOT_INC:
        work = dot_flops_per_step(M.Plan(model, minibatch=w.minibatch, **(plan_opts or {})).json(), w.minibatch) * T
        bound, peak, unit = "mfma", FP32_MFMA_PEAK_TFLOPS, "TFLOP/s"
        kernel = "k_w_gemm2" if window else "k_dot_inc"
        if bf16:
            peak, kernel = BF16_MFMA_PEAK_TFLOPS, "k_w_gemm_bf16"
    elif top in (M.mergesim.OP_PES_DECODE_UPDATE, M.mergesim.OP_LEARNED_DECODE, M.mergesim.OP_PES):
        work = sum(pes_bytes_per_launch(w.spec, c, w.minibatch) for c in w.spec.connections
                   if c.learning_rule is not None) * T
        bound, peak, unit, kernel = "hbm", HBM_PEAK_GBS, "GB/s", "k_pes"
    else:
        work, bound, peak, unit = compulsory_bytes_per_step(w) * T, "hbm", HBM_PEAK_GBS, "GB/s"
        kernel = f"op type {top}"
    basis = "algorithmic"
    if event and top == M.mergesim.OP_ENSEMBLE and not window:
        # event-driven decoding moves fewer bytes than the method's dense
        # work: its rate is reported from measured counter bytes, if taken
        rec = stored_traffic(kernel, w.name + "event")
        basis = "counter bytes"
        if rec is None:
            return {"bound": bound, "achieved": None, "peak": peak, "unit": unit, "frac": None,
                    "traffic": None, "basis": basis, "kernel": kernel, "op": "Ensemble",
                    "launch_ms": round(ms / max(n, 1), 4), "launches": n}
        work = rec * n
    scale = 1e12 if unit == "TFLOP/s" else 1e9
    ach = work / (ms * 1e-3) / scale
    op_names = {M.mergesim.OP_ENSEMBLE: "Ensemble", M.mergesim.OP_DOT_INC: "DotInc",
                M.mergesim.OP_PES_DECODE_UPDATE: "PESDecodeUpdate"}
    out = {"bound": bound, "achieved": round(ach, 3), "peak": peak, "unit": unit,
           "frac": round(ach / peak, 4),
           "traffic": stored_traffic(kernel, w.name + ("event" if event else "")) if default_plan else None,
           "basis": basis,
           "kernel": kernel, "op": op_names.get(top, str(top)), "launch_ms": round(ms / max(n, 1), 4),
           "launches": n, "busy_ms": round(ms, 4), "work_per_launch": int(work / max(n, 1))}
    sq = stored_sq(kernel, w.name) if default_plan else None
    if sq is not None and "SQ_INSTS_VALU" in sq:
        # VALU issue rate of the same kernel: wavefront instructions per launch
        # from the committed counter pass, over the launch time measured here
        rate = sq["SQ_INSTS_VALU"] / (ms * 1e-3 / max(n, 1))
        out["valu"] = {"insts_per_launch": int(sq["SQ_INSTS_VALU"]), "issue_per_s": rate,
                       "peak_per_s": VALU_ISSUE_PEAK, "frac": round(rate / VALU_ISSUE_PEAK, 4)}
    return out


def stored_sq(kernel, workload):
    """Per-launch shader counters of a kernel and workload from the committed
    counter summary, if it was taken from the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_sq.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    return rec["per_launch"] if rec.get("source_sha") == source_sha() else None


def stored_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter summary of this kernel
    and workload, if it was taken from the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    return rec["bytes_per_launch"] if rec.get("source_sha") == source_sha() else None


def source_sha():
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1805_11144_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hpp", ".hip", ".cpp")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


COPY_PROBE_BYTES = 256 << 20


def _counter_rows(d):
    import csv
    import glob
    rows = []
    for path in glob.glob(os.path.join(d, "**", "*counter_collection*.csv"), recursive=True):
        with open(path) as f:
            rows += list(csv.DictReader(f))
    if not rows:
        raise SystemExit(f"no counter_collection csv under {d}")
    return rows


def _per_dispatch(rows, counter):
    """kernel name -> list of per-dispatch counter values (bytes)."""
    out = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)   # KiB -> B
    return out


def summarize_traffic(args):
    """Per-launch HBM bytes of a kernel from FETCH_SIZE and WRITE_SIZE runs, each
    scaled by what the same counter reads for the 256 MiB calibration copy."""
    res = {}
    for kind, d, counter in (("fetch", args.summarize_traffic[0], "FETCH_SIZE"),
                             ("write", args.summarize_traffic[1], "WRITE_SIZE")):
        per = _per_dispatch(_counter_rows(d), counter)
        copies = [v for k, vals in per.items() if "copyBuffer" in k for v in vals]
        if not copies:
            raise SystemExit("calibration copy not found (run the profiled bench with --copy-probe)")
        scale = COPY_PROBE_BYTES / max(copies)
        names = [n for n in (args.match or args.kernel).split(",") if n]

        def hit(k):
            base = k.split("(")[0].split("<")[0].strip().split(" ")[-1]
            return any(base == n for n in names)
        vals = [v for k, vs in per.items() if hit(k) for v in vs]
        if not vals:
            raise SystemExit(f"kernels {names} not found in {d}")
        raw, launches = sum(vals) / len(vals), len(vals)
        if args.sum_kernels:
            # the kernels run together as one launch of the operator (one dispatch of
            # each per launch): a launch moves the sum of their per-dispatch averages
            by = {}
            for k, vs in per.items():
                if hit(k):
                    by.setdefault(k.split("(")[0].split("<")[0].strip().split(" ")[-1], []).extend(vs)
            counts = {len(vs) for vs in by.values()}
            if len(counts) != 1:
                raise SystemExit(f"--sum-kernels: dispatch counts differ {[(k, len(v)) for k, v in by.items()]}")
            raw, launches = sum(sum(vs) / len(vs) for vs in by.values()), counts.pop()
        res[kind] = {"raw_bytes_per_launch": raw, "scale": scale, "launches": launches,
                     "bytes_per_launch": scale * raw}
    workload = args.config + ("event" if args.event_decode else "")
    rec = {"kernel": args.kernel, "kernels_counted": names, "workload": workload,
           "bytes_per_launch": int(res["fetch"]["bytes_per_launch"] + res["write"]["bytes_per_launch"]),
           "fetch": res["fetch"], "write": res["write"], "source_sha": source_sha(), "command": args.command}
    path = os.path.join(ROOT, "profiles", f"{args.kernel}_{workload}_traffic.json")
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def summarize_sq(args):
    """Per-launch shader (SQ_*) counters of a kernel from one or more rocprofv3
    --pmc runs, averaged over its dispatches."""
    names = [n for n in (args.match or args.kernel).split(",") if n]

    def hit(k):
        base = k.split("(")[0].split("<")[0].strip().split(" ")[-1]
        return any(base == n for n in names)
    per = {}
    for d in args.summarize_sq:
        for r in _counter_rows(d):
            if hit(r["Kernel_Name"]):
                per.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    if not per:
        raise SystemExit(f"kernels {names} not found")
    rec = {"kernel": args.kernel, "kernels_counted": names, "workload": args.config,
           "per_launch": {k: sum(v) / len(v) for k, v in sorted(per.items())},
           "launches": {k: len(v) for k, v in sorted(per.items())},
           "source_sha": source_sha(), "command": args.command}
    path = os.path.join(ROOT, "profiles", f"{args.kernel}_{args.config}_sq.json")
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c4", choices=sorted(WORKLOADS))
    ap.add_argument("--driver", default="auto", choices=["auto", "steps", "graph", "persistent", "window"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gemm-dtype", default="f32", choices=["f32", "bf16"],
                    help="input precision of the large window products (bf16: fp32 accumulation)")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle stepping per leg of the CPU baseline (two legs)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="copy 256 MiB device to device before timing (calibrates HBM counters)")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) into profiles/<kernel>_<config>_traffic.json")
    ap.add_argument("--summarize-sq", nargs="+", metavar="PMC_DIR",
                    help="turn rocprofv3 --pmc runs of SQ_* counters into profiles/<kernel>_<config>_sq.json")
    ap.add_argument("--kernel", default="k_w_ens", help="kernel name prefix for --summarize-traffic")
    ap.add_argument("--command", default="", help="profiling command recorded by --summarize-traffic")
    ap.add_argument("--match", default="",
                    help="comma-separated kernel names counted by --summarize-traffic (default: --kernel); "
                         "list every kernel of the operator type the roofline times")
    ap.add_argument("--sum-kernels", action="store_true",
                    help="--summarize-traffic: the --match kernels are one operator launch (one dispatch "
                         "each); count their sum per launch")
    ap.add_argument("--timesteps", type=int, default=0,
                    help="override the workload's timesteps (counter passes: per-launch traffic of a "
                         "time-major kernel does not depend on the run length)")
    ap.add_argument("--unroll", type=int, default=20,
                    help="steps per hipGraph launch (the paper's unroll_simulation)")
    ap.add_argument("--planner", default="tree", choices=["tree", "greedy"],
                    help="operator-merging planner (ablation; default: tree search, depth 3)")
    ap.add_argument("--planner-depth", type=int, default=3)
    ap.add_argument("--no-merge", action="store_true", help="ablation: one group per operator")
    ap.add_argument("--no-sort", action="store_true", help="ablation: signals and operators in build order")
    ap.add_argument("--no-simplify", action="store_true", help="ablation: skip simplification")
    ap.add_argument("--no-fuse", action="store_true", help="ablation: no fused ensemble operators")
    ap.add_argument("--spike-bits", action="store_true",
                    help="record spike probes as one bit per neuron and step (window driver)")
    ap.add_argument("--event-decode", action="store_true",
                    help="event-driven decoding (reads the decoders of spiking neurons only); not the "
                         "method's dense work, so the roofline uses measured counter bytes")
    ap.add_argument("--counters-run", action="store_true",
                    help="one untimed run for a rocprofv3 --pmc pass (with --copy-probe); prints no JSON")
    args = ap.parse_args()
    if args.summarize_traffic:
        summarize_traffic(args)
        return
    if args.summarize_sq:
        summarize_sq(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)
    if args.config == "train":
        main_train(args)
        return

    import torch

    import paper_1805_11144_amd as M
    from synth import make_workload

    w = make_workload(args.config, **({"n_steps": args.timesteps} if args.timesteps else {}))
    model = M.model_from_spec(w.spec)
    driver = {"auto": M.DRIVER_AUTO, "steps": M.DRIVER_STEPS, "graph": M.DRIVER_GRAPH,
              "persistent": M.DRIVER_PERSISTENT, "window": M.DRIVER_WINDOW}[args.driver]
    dev = torch.device("cuda:0")
    t_build = time.perf_counter()
    plan_opts = dict(planner=M.PLANNER_TREE if args.planner == "tree" else M.PLANNER_GREEDY,
                     planner_depth=args.planner_depth, merge=not args.no_merge, sort=not args.no_sort,
                     simplify=not args.no_simplify, fuse=not args.no_fuse,
                     decode="event" if args.event_decode else "dense",
                     spike_probe_bits=args.spike_bits)
    sim = M.Simulator(model, minibatch=w.minibatch, driver=driver, unroll=args.unroll,
                      probe_capacity_steps=w.n_steps, gemm_dtype=args.gemm_dtype, **plan_opts)
    t_build = time.perf_counter() - t_build
    feeds = {i: torch.from_numpy(f).to(dev) for i, f in w.feeds.items()}
    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        del src, dst
    torch.cuda.synchronize()

    def one_run():
        sim.reset()
        sim.run_steps(w.n_steps, feeds)

    if args.counters_run:
        one_run()
        sim.sync()
        torch.cuda.synchronize()
        return
    for _ in range(args.warmup):
        one_run()
    sim.sync()
    torch.cuda.synchronize()
    run_ms = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_run()
        run_ms.append(sim.last_run_ms())   # HIP events around the run on its stream
    sim.sync()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    ms_per_step = 1000.0 * elapsed / args.steps
    neuron_steps = w.n_neurons * w.n_steps * w.minibatch
    value = neuron_steps / (elapsed / args.steps)
    run_mean, run_ci = mean_ci95(run_ms)
    info = sim.info()
    bf16 = args.gemm_dtype == "bf16"
    default_plan = (args.planner, args.planner_depth, args.no_merge, args.no_sort, args.no_simplify,
                    args.no_fuse) == ("tree", 3, False, False, False, False)
    roofline = measure_roofline(M, model, w, sim, info, feeds, bf16, plan_opts, default_plan,
                                event=args.event_decode)
    out = {
        "metric": "neuron-timesteps/sec (x minibatch) on 1 MI355X",
        "value": value, "unit": "neuron-timesteps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16/f32" if bf16 else "f32", "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "name": args.config, "neurons": w.n_neurons,
                   "timesteps": w.n_steps, "minibatch": w.minibatch,
                   "driver": {1: "steps", 2: "graph", 3: "persistent", 4: "window"}.get(info["driver"]),
                   "launches_per_window" if info["driver"] == M.DRIVER_WINDOW else "groups_per_step":
                       info["groups_per_step"], "build_s": round(t_build, 2),
                   "gemm_dtype": args.gemm_dtype, "unroll": args.unroll,
                   "plan": {"planner": args.planner, "depth": args.planner_depth, "merge": not args.no_merge,
                            "sort": not args.no_sort, "simplify": not args.no_simplify,
                            "fuse": not args.no_fuse},
                   "decode": "event" if args.event_decode else "dense", "spike_probe_bits": args.spike_bits},
        "runs": {"device_ms": [round(x, 4) for x in run_ms], "mean_ms": round(run_mean, 4),
                 "ci95_ms": None if run_ci is None else round(run_ci, 4),
                 "value_ci95": None if run_ci is None else
                 [neuron_steps / ((run_mean + run_ci) * 1e-3), neuron_steps / ((run_mean - run_ci) * 1e-3)]},
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
