"""Float64 CPU executor of an exported merged plan (test helper).

It runs the library's plan -- base-array layout, merged groups in plan order,
lowered index arrays and the float32 parameter values the GPU uses -- with
numpy in float64.  Compared with the unmerged oracle (parameters rounded to
float32), it checks that merging, planning, sorting, simplification and
lowering do not change the model's output (paper Sec. 4.2), without a GPU.
"""
import numpy as np

from oracle.neurons import soft_lif_rate


def _rows(op, n):
    if op is None:
        return None
    if "idx" in op:
        return np.asarray(op["idx"], np.int64)
    return op["start"] + np.arange(n, dtype=np.int64)


def _lif(J, V, ref, dt, trc, tref, amp):
    integ = np.clip(dt - ref, 0, dt)
    V = V - (J - V) * np.expm1(-integ / trc)
    ref = np.maximum(ref - dt, 0)
    spk = V > 1
    q = np.where(spk & (J > 1), (V - 1) / np.where(J > 1, J - 1, 1), 0.0)
    since = np.where(q >= 1, integ, np.minimum(-trc * np.log1p(-np.minimum(q, 0.999999999999)), integ))
    since = np.where(spk & (J > 1), since, 0.0)
    V = np.where(spk, 0.0, np.maximum(V, 0.0))
    ref = np.where(spk, tref - since, ref)
    return np.where(spk, amp / dt, 0.0), V, ref


def _rate(J, trc, tref, amp):
    r = np.zeros_like(J)
    m = J > 1
    r[m] = 1.0 / (np.broadcast_to(tref, J.shape)[m] +
                  np.broadcast_to(trc, J.shape)[m] * np.log1p(1.0 / (J[m] - 1.0)))
    return amp * r


def _vec(v, n):
    v = np.asarray(v, np.float64)
    return np.broadcast_to(v, (n,)) if v.size == 1 else v


def oracle_param(oracle, name):
    """Value of a parameter signal, by its canonical name, from the oracle."""
    owner, kind = name.split(".", 1)
    i = int(owner[1:])
    spec = oracle.spec
    if owner[0] == "e":
        if kind == "bias":
            return oracle.bias[i]
        if kind == "gain":
            return oracle.gain[i]
        if kind == "enc":
            return oracle.enc[i]
        if kind in ("Did", "Dprod"):
            return oracle.dec[(i, "identity" if kind == "Did" else "product")].T
    if owner[0] == "c":
        if kind == "T":
            return oracle.conn_T[i]
        if kind == "t":
            return np.array([oracle.conn_T[i]])
        if kind == "D":
            return oracle.conn_dec[i].T
    if owner[0] == "n" and kind == "value":
        return np.asarray(spec.nodes[i].value, np.float64)
    raise KeyError(name)


class PlanExecutor:
    """params_from: an OracleSim whose (float32-rounded) parameters replace the
    library's, so that only the plan itself is under test; None uses the
    library's exported float32 parameters."""

    def __init__(self, plan, spec, minibatch, params_from=None):
        self.j = plan.json()
        self.B = minibatch
        self.spec = spec
        self.params_from = params_from
        self.bases = []
        for bi, b in enumerate(self.j["bases"]):
            if b["name"] == "state":
                self.bases.append(None)
                self.state_base = bi
                # initial value of every row (learned decoders; zeros elsewhere)
                self.init = plan.base(bi).astype(np.float64).reshape(b["rows"])
            elif params_from is None:
                self.bases.append(plan.base(bi).astype(np.float64).reshape(b["rows"], b["cols"]))
            else:
                arr = np.zeros((b["rows"], b["cols"]))
                for sg in self.j["signals"]:
                    if sg["base"] == bi:
                        v = np.asarray(oracle_param(params_from, sg["name"]), np.float64)
                        arr[sg["offset"]:sg["offset"] + sg["rows"]] = v.reshape(sg["rows"], b["cols"])
                self.bases.append(arr)
        if params_from is not None:
            self._replace_constants(params_from, self.j["groups"])
            if self.j.get("window", {}).get("ok"):
                self._replace_constants(params_from, [ph["group"] for ph in self.j["window"]["phases"]])
        self.rows = self.j["bases"][self.state_base]["rows"]
        self.fed = [i for i, n in enumerate(spec.nodes) if not n.passthrough and n.value is None]
        self.dt = spec.dt
        self.reset()

    def _replace_constants(self, o, groups):
        """Reset values, neuron parameters and filter coefficients from the oracle."""
        for g in groups:
            if g["type"] == "Reset" and "values" in g:
                rows = {sg["name"]: sg["rows"] for sg in self.j["signals"]}
                dst = {"reset": "out", "resetx": "x", "resetid": "did", "resetprod": "dprod",
                       "resetv": "v", "resetd": "xd", "resete": "E"}
                vals = []
                for name in g["ops"]:
                    owner, kind = name.split(".", 1)
                    i = int(owner[1:])
                    if kind == "bias":
                        vals.append(o.bias[i])
                    elif kind == "const":
                        vals.append(np.asarray(self.spec.nodes[i].value, float))
                    else:
                        vals.append(np.zeros(rows[owner + "." + dst[kind]]))
                g["values"] = np.concatenate(vals).tolist()
            elif g["type"] in ("SimLIF", "SimLIFRate"):
                cols = {"tau_rc": [], "tau_ref": [], "amp": []}
                for name in g["ops"]:
                    e = self.spec.ensembles[int(name.split(".")[0][1:])]
                    for k in cols:
                        cols[k].append(np.full(e.n_neurons, getattr(e, "amplitude" if k == "amp" else k)))
                for k in cols:
                    g[k] = np.concatenate(cols[k]).tolist()
                if "sigma" in g:
                    g["sigma"] = np.concatenate([np.full(e.n_neurons, e.sigma) for e in
                                                 (self.spec.ensembles[int(name.split(".")[0][1:])]
                                                  for name in g["ops"])]).tolist()
            elif g["type"] == "Ensemble":
                ens = [self.spec.ensembles[int(name.split(".")[0][1:])] for name in g["ops"]]
                g["tau_rc"] = [e.tau_rc for e in ens]
                g["tau_ref"] = [e.tau_ref for e in ens]
                g["amp"] = [e.amplitude for e in ens]
            elif g["type"] in ("PES", "PESDecodeUpdate"):
                g["coef"] = [-o.pes_coef[int(name.split(".")[0][1:])] for name in g["ops"]
                             if name.endswith(".pes")]
            elif g["type"] == "Lowpass":
                ca, cb = [], []
                for name in g["ops"]:
                    owner, kind = name.split(".", 1)
                    i = int(owner[1:])
                    if kind == "presyn":      # a PES rule's activity filter
                        a, b = o.pes_a[i]
                        w = o.abar[i].shape[1]
                    else:
                        a, b = (o.conn_a[i] if owner[0] == "c" else o.probe_a[i])
                        w = (o.y[i] if owner[0] == "c" else o.yp[i]).shape[1]
                    ca.append(np.full(w, a)); cb.append(np.full(w, b))
                g["ca"] = np.concatenate(ca).tolist()
                g["cb"] = np.concatenate(cb).tolist()

    def reset(self):
        self.st = np.repeat(self.init[:, None], self.B, axis=1)
        if self.params_from is not None:      # learned decoders from the oracle's values
            for sg in self.j["signals"]:
                owner, kind = sg["name"].split(".", 1)
                if kind == "W":
                    W = self.params_from.conn_dec[int(owner[1:])]
                    self.st[sg["offset"]:sg["offset"] + sg["rows"]] = W.reshape(-1)[:, None]
        self.records = []

    def _src(self, arr, base, rows):
        if base == self.state_base:
            return arr[rows]
        return np.broadcast_to(self.bases[base][rows, 0][:, None], (len(rows), self.B))

    def step(self, feed_rows_values):
        st = self.st
        for g in self.j["groups"]:
            self.exec_group(g, st, st, st, st, feed_rows_values)
        self.records.append(st[np.asarray(self.j["probe_rows"], np.int64)].copy())

    def exec_group(self, g, cur, src, prev, pa, feed_rows_values):
        """One merged group for one step.  cur: this step's values (written);
        src: where the group's batched inputs are read; prev: the previous
        step's values (a filter's own output); pa: neuron state.  In the
        time-major layout all four are the same array."""
        t, n = g["type"], g["rows"]
        if t == "Feed":
            cur[_rows(g["dst"], n)] = feed_rows_values[np.asarray(g["feed_rows"])]
        elif t == "Reset":
            d = _rows(g["dst"], n)
            cur[d] = _vec(g["values"], n)[:, None] if "values" in g else 0.0
        elif t == "Copy":
            cur[_rows(g["dst"], n)] = self._src(src, g["src"]["base"], _rows(g["src"], n))
        elif t in ("CopyInc", "ElementwiseInc"):
            d = _rows(g["dst"], n)
            if "ptr" in g:
                ptr = np.asarray(g["ptr"])
                m = ptr[-1]
                seg = np.repeat(np.arange(n), np.diff(ptr))
            else:
                m = n
                seg = np.arange(n)
            vals = self._src(src, g["src"]["base"], _rows(g["src"], m))
            if t == "ElementwiseInc":
                vals = vals * self.bases[g["a"]["base"]][_rows(g["a"], m), 0][:, None]
            acc = np.zeros((n, self.B))
            np.add.at(acc, seg, vals)
            cur[d] += acc
        elif t == "DotInc":
            M, K = g["M"], g["K"]
            W = self.bases[self._weight_base(g)]
            for w0, x0, d0 in zip(g["w_row"], g["x_row"], g["d_row"]):
                Wm = W[w0:w0 + M, :K] if W.shape[1] == K else W[w0:w0 + M * K, 0].reshape(M, K)
                cur[d0:d0 + M] += Wm @ src[x0:x0 + K]
        elif t in ("LearnedDotInc", "PES", "PESDecodeUpdate"):
            M, K = g["M"], g["K"]
            for o in range(n):
                w0, x0 = g["w_row"][o], g["x_row"][o]
                W = cur[w0:w0 + K * M].reshape(K, M, self.B)      # row i*M + j: neuron i, output j
                if t != "PES":
                    d0 = g["d_row"][o]
                    cur[d0:d0 + M] += np.einsum("kmb,kb->mb", W, src[x0:x0 + K])
                if t != "LearnedDotInc":
                    a0 = g["act_row"][o] if t == "PESDecodeUpdate" else x0
                    e0 = g["e_row"][o]
                    W += g["coef"][o] * src[a0:a0 + K][:, None, :] * src[e0:e0 + M][None, :, :]
        elif t in ("SimLIF", "SimLIFRate"):
            J = src[_rows(g["src"], n)]
            trc = _vec(g["tau_rc"], n)[:, None]
            tref = _vec(g["tau_ref"], n)[:, None]
            amp = _vec(g["amp"], n)[:, None]
            if t == "SimLIFRate":
                if g.get("neuron") == 2:
                    out = amp * np.maximum(J, 0.0)
                elif g.get("neuron") == 3:
                    out = amp * soft_lif_rate(J, trc, tref, _vec(g["sigma"], n)[:, None])
                else:
                    out = _rate(J, trc, tref, amp)
            else:
                vr, rr = _rows(g["V"], n), _rows(g["ref"], n)
                out, pa[vr], pa[rr] = _lif(J, pa[vr].copy(), pa[rr].copy(), self.dt, trc, tref, amp)
            cur[_rows(g["dst"], n)] = out
        elif t == "Ensemble":
            trc_all = _vec(g["tau_rc"], n); tref_all = _vec(g["tau_ref"], n)
            amp_all = _vec(g["amp"], n)
            chain = np.asarray(g["chain"], np.int64).reshape(n, -1) if "chain" in g else None
            for k in range(n):
                nn = g["n"][k]
                b0 = g["bias_row"][k]
                J = np.repeat(self.bases[g["bias_base"]][b0:b0 + nn, 0][:, None], self.B, axis=1)
                if g["x_row"][k] >= 0:
                    d = g["d"]
                    E = self.bases[g["enc_base"]][g["enc_row"][k]:g["enc_row"][k] + nn]
                    if chain is not None and chain[k, 1] > 0:
                        # fused connection chain (window driver): x_t = y_{t-1}, y_t = a y_{t-1} + b W d_t
                        d0, K, w0, y0, Mc = (int(v) for v in chain[k, :5])
                        a, b = np.asarray(chain[k, 6:8], np.int32).view(np.float32).astype(np.float64)
                        Wc = self.bases[g["chain_wbase"]][w0:w0 + Mc, :K]
                        x = prev[y0:y0 + Mc].copy()
                        cur[y0:y0 + Mc] = a * prev[y0:y0 + Mc] + b * (Wc @ cur[d0:d0 + K])
                    else:
                        x = src[g["x_row"][k]:g["x_row"][k] + d]
                    J = J + E[:, :d] @ x
                if g["neuron"] == 0:
                    v0, r0 = g["V_row"][k], g["ref_row"][k]
                    s_, pa[v0:v0 + nn], pa[r0:r0 + nn] = _lif(J, pa[v0:v0 + nn].copy(),
                                                              pa[r0:r0 + nn].copy(), self.dt,
                                                              trc_all[k], tref_all[k], amp_all[k])
                elif g["neuron"] == 2:
                    s_ = amp_all[k] * np.maximum(J, 0.0)
                else:
                    s_ = _rate(J, trc_all[k], tref_all[k], amp_all[k])
                if g["s_row"][k] >= 0:
                    cur[g["s_row"][k]:g["s_row"][k] + nn] = s_
                for f, df in enumerate(g["df"]):
                    D = self.bases[g["D_base"][f]][g["D_row"][f][k]:g["D_row"][f][k] + df, :nn]
                    cur[g["d_row"][f][k]:g["d_row"][f][k] + df] = D @ s_
        elif t == "Lowpass":
            y, v = _rows(g["dst"], n), _rows(g["src"], n)
            cur[y] = _vec(g["ca"], n)[:, None] * prev[y] + _vec(g["cb"], n)[:, None] * src[v]
        else:
            raise ValueError(t)

    def _weight_base(self, g):
        sigs = self.j["signals"]
        # weight signals are named like the op's owner with .enc/.D*/.T
        name = g["ops"][0]
        owner, kind = name.split(".", 1)
        if kind == "enc":
            wname = owner + ".enc"
        elif kind.startswith("dec"):
            wname = owner + ".D" + kind[3:]
        else:   # transform
            wname = owner + ".T"
        for s in sigs:
            if s["name"] == wname:
                return s["base"]
        raise KeyError(wname)

    def run(self, n_steps, feeds):
        for k in range(n_steps):
            vals = np.concatenate([np.asarray(feeds[i][:, k, :], np.float64).T if i in feeds
                                   else np.zeros((self.spec.nodes[i].size, self.B))
                                   for i in self.fed], axis=0) if self.fed else np.zeros((0, self.B))
            self.step(vals)

    def data(self, probe):
        off = self.j["probe_offsets"]
        rec = np.stack(self.records, axis=0)        # [T, probe_rows, B]
        return np.transpose(rec[:, off[probe]:off[probe + 1], :], (2, 0, 1))


class WindowExecutor(PlanExecutor):
    """Runs the library's stage-major schedule (the plan's "window" section):
    every phase over a whole window of steps before the next phase, with
    versioned signals [rows][W+1][B] (block 0: carried in; block t+1: window
    step t) and neuron state in a private [rows][B] array."""

    def __init__(self, plan, spec, minibatch, window, params_from=None):
        super().__init__(plan, spec, minibatch, params_from)
        self.w = self.j["window"]
        assert self.w["ok"], self.w["why"]
        self.W = window
        self.reset()

    def reset(self):
        super().reset()
        if getattr(self, "w", None) is None:
            return
        self.va = np.zeros((self.w["rows_v"], self.W + 1, self.B))
        self.pa = np.zeros((self.w["rows_p"], self.B))

    def run(self, n_steps, feeds):
        vals_all = []
        for k in range(n_steps):
            vals_all.append(np.concatenate([np.asarray(feeds[i][:, k, :], np.float64).T if i in feeds
                                            else np.zeros((self.spec.nodes[i].size, self.B))
                                            for i in self.fed], axis=0) if self.fed
                            else np.zeros((0, self.B)))
        pr = np.asarray(self.w["probe_rows"], np.int64)
        t0 = 0
        while t0 < n_steps:
            tw = min(self.W, n_steps - t0)
            for ph in self.w["phases"]:
                g = ph["group"]
                for t in range(tw):
                    self.exec_group(g, self.va[:, t + 1], self.va[:, t + ph["src_blk"]], self.va[:, t],
                                    self.pa, vals_all[t0 + t])
            for t in range(tw):
                self.records.append(self.va[pr, t + 1].copy())
            self.va[:, 0] = self.va[:, tw]
            t0 += tw


class LaunchExecutor(PlanExecutor):
    """Runs the time-major step program of the launch drivers (the plan's
    "launch" section): merged ensemble groups and fused synapse groups, with
    the fused groups' pull-only prologue at the start of every run."""

    def __init__(self, plan, spec, minibatch, params_from=None):
        super().__init__(plan, spec, minibatch, params_from)
        self.lp = self.j["launch"]
        if params_from is not None:
            self._replace_constants(params_from, [g for g in self.lp["groups"] if g["type"] != "Reset"])
            # resets may have lost rows: their values row by row from the plan's
            reset_val = {}
            for g in self.j["groups"]:
                if g["type"] == "Reset":
                    n = g["rows"]
                    vals = _vec(g["values"], n) if "values" in g else np.zeros(n)
                    reset_val.update({int(r): float(v) for r, v in zip(_rows(g["dst"], n), vals)})
            for g in self.lp["groups"]:
                if g["type"] == "Reset" and "values" in g:
                    g["values"] = [reset_val[int(r)] for r in _rows(g["dst"], g["rows"])]
            # fused groups take each connection's coefficients from its first
            # filter row, as set in the plan's (oracle-valued) Lowpass groups
            coef = {}
            for g in self.j["groups"]:
                if g["type"] == "Lowpass":
                    n = g["rows"]
                    for y, a, b in zip(_rows(g["dst"], n), _vec(g["ca"], n), _vec(g["cb"], n)):
                        coef[int(y)] = (float(a), float(b))
            for g in self.lp["groups"] + ([self.lp["prologue"]] if self.lp["prologue"] else []):
                if g["type"] == "SynapseScatter":
                    conn = np.asarray(g["conn"], np.int64).reshape(-1, 8)
                    g["ab"] = [x for y0, v0 in conn[:, :2] for x in (coef[int(y0)] if v0 != -2 else (0.0, 0.0))]

    def step(self, feed_rows_values):
        st = self.st
        rec = None
        for g in self.lp["groups"]:
            if g["type"] == "SynapseScatter":
                r = self.exec_synapse(g, st, feed_rows_values)
                if g["probe"]:
                    rec = r
            else:
                self.exec_group(g, st, st, st, st, feed_rows_values)
        if rec is None:
            rec = st[np.asarray(self.j["probe_rows"], np.int64)].copy()
        else:   # a folded probe must have recorded every probe row
            assert not np.isnan(rec).any(), "probe rows the fused group did not record"
        self.records.append(rec)

    def run(self, n_steps, feeds):
        if self.lp["prologue"] is not None:
            self.exec_synapse(self.lp["prologue"], self.st)
        super().run(n_steps, feeds)

    def exec_synapse(self, g, st, feed_rows_values=None):
        """Per segment row i: for each connection in order, v (state row or
        weight row . inputs, the inputs from the state or from this step's
        feed values), y <- a y + b v (when updating), sum of the y; the sum is
        stored in the post row.  Returns the probe rows it recorded."""
        seg = np.asarray(g["seg"], np.int64).reshape(-1, 4)
        conn = np.asarray(g["conn"], np.int64).reshape(-1, 8)
        ab = np.asarray(g["ab"], np.float64).reshape(-1, 2)
        rec = np.full((len(self.j["probe_rows"]), self.B), np.nan)
        for dst, ln, c0, nc in seg:
            i = np.arange(ln)
            acc = np.zeros((ln, self.B))
            for c in range(c0, c0 + nc):
                y0, v0, x0, K, ws, w0, pr, staged = conn[c]
                y = st[y0 + i]
                if g["update"]:
                    if v0 != -2:
                        if v0 >= 0:
                            v = st[v0 + i]
                        elif ws == -2:      # elementwise: scale (float bits in w0) times input row x0 + i
                            scale = float(np.array([w0], np.int32).view(np.float32)[0])
                            v = scale * (feed_rows_values[x0 + i] if staged else st[x0 + i])
                        else:
                            W = self.bases[g["wbase"][ws]]
                            xin = feed_rows_values[x0:x0 + K] if staged else st[x0:x0 + K]
                            v = W[w0 + i, :K] @ xin
                        y = ab[c, 0] * y + ab[c, 1] * v
                        st[y0 + i] = y
                    if pr >= 0:
                        assert np.isnan(rec[pr + i]).all(), "probe row recorded twice"
                        rec[pr + i] = y
                acc = acc + y
            if dst >= 0:
                st[dst + i] = acc
        return rec
