// Model -> signals and operators (paper Sec. 2.1.3 and Fig. 2), plus the
// simplification pass (Sec. 4.2.4).
//
// The lowering is canonical: signals and operators are created in a fixed,
// documented order, and every one gets a stable name, so that plans can be
// compared operator by operator with an independent implementation.
//
// Per node i (id order):
//   signal  n<i>.out [size] batched
//   fed node:          FEED     n<i>.feed    sets n<i>.out from the feed buffer
//   constant node:     COPY     n<i>.const   n<i>.out = n<i>.value (param)
//   passthrough node:  RESET    n<i>.reset   n<i>.out = 0
// Per ensemble e (id order):
//   signals e<e>.J, e<e>.s [n] batched; LIF: e<e>.V, e<e>.ref [n] batched state;
//   param e<e>.bias [n]; with decoded-space input: e<e>.x [d] batched and param
//   e<e>.enc [n x d] (gain-scaled encoders); with neuron-space input: param
//   e<e>.gain [n]; per decoded function f used (first use by a connection, then
//   by a probe): e<e>.d<f> [d_f] batched and param e<e>.D<f> [d_f x n]
//   ops: RESET e<e>.resetx (x = 0); COPY e<e>.bias (J = bias);
//        DOT_INC e<e>.enc (J += enc x); LIF|LIF_RATE e<e>.neurons (J -> s);
//        per f: RESET e<e>.reset<f>, DOT_INC e<e>.dec<f> (d_f += D_f s)
// Per connection c (id order):
//   explicit decoders: c<c>.xd [cols] batched, param c<c>.D [cols x n];
//     RESET c<c>.resetd, DOT_INC c<c>.dec
//   c<c>.v [w] batched (w = post slice width); param c<c>.t [1] (scalar) or
//   c<c>.T [w x k]; with a synapse c<c>.y [w] batched state
//   ops: RESET c<c>.resetv; ELEM_INC (scalar) | DOT_INC (matrix) c<c>.transform
//        (v += T pre[slice]); LOWPASS c<c>.synapse (y <- a y + (1-a) v);
//        c<c>.deliver: COPY_INC into x / passthrough output, or ELEM_INC
//        (J += gain (.) value) for neuron-space posts
//   connection with a PES rule (decodes from ensemble e, n neurons, k
//   outputs): c<c>.xd [k] batched, c<c>.W [n*k] batched state (row i*k + j,
//   initially the decoders), with a pre synapse c<c>.a [n] batched state;
//     RESET c<c>.resetd, BDOT_INC c<c>.dec (xd += per-column W^T s),
//     RESET c<c>.resete, PES c<c>.pes (W += -kappa dt / n  act (x) E, act =
//     c<c>.a or e<e>.s), with a pre synapse LOWPASS c<c>.presyn (a <- p a +
//     (1-p) s); its error input c<c>.E [k] batched is created, in connection
//     order, before the first connection's signals; connections into
//     (MS_REF_LEARNING, c) deliver into it by COPY_INC
// Per probe p: with a synapse p<p>.y [w] batched state, LOWPASS p<p>.synapse.
#include <algorithm>
#include <cmath>

#include "host.hpp"

namespace ms {

namespace {

std::string fn_tag(int32_t fn) { return fn == MS_FN_PRODUCT ? "prod" : "id"; }

struct Builder {
  IR ir;
  const Model& m;
  std::map<std::string, int32_t> base_ids;

  explicit Builder(const Model& mm) : m(mm) {}

  int32_t base_for(SigClass cls, int32_t cols) {
    std::string name = cls == SC_BATCHED ? "state" : (cols == 1 ? "vec" : "mat" + std::to_string(cols));
    auto it = base_ids.find(name);
    if (it != base_ids.end()) return it->second;
    int32_t id = (int32_t)ir.bases.size();
    ir.bases.push_back({name, cls, cls == SC_BATCHED ? 1 : cols});
    base_ids[name] = id;
    return id;
  }

  int32_t batched(const std::string& name, int32_t rows, bool state) {
    Signal s;
    s.name = name; s.rows = rows; s.cols = 1; s.cls = SC_BATCHED; s.state = state;
    s.base = base_for(SC_BATCHED, 1);
    ir.sigs.push_back(std::move(s));
    return (int32_t)ir.sigs.size() - 1;
  }

  int32_t param(const std::string& name, int32_t rows, int32_t cols, std::vector<double> v) {
    Signal s;
    s.name = name; s.rows = rows; s.cols = cols; s.cls = SC_PARAM; s.value = std::move(v);
    s.base = base_for(SC_PARAM, cols);
    ir.sigs.push_back(std::move(s));
    return (int32_t)ir.sigs.size() - 1;
  }

  SRef whole(int32_t sig) { return SRef{sig, 0, ir.sigs[sig].rows}; }

  Op& add(OpType t, const std::string& name) {
    Op o;
    o.type = t;
    o.name = name;
    ir.ops.push_back(std::move(o));
    return ir.ops.back();
  }
};

void check(bool ok, const std::string& msg) {
  if (!ok) fail(MS_E_INVALID, msg);
}

}  // namespace

IR build_ir(const Model& m, const Built& bp, double dt) {
  Builder B(m);
  const int32_t nn = (int32_t)m.nodes.size(), ne = (int32_t)m.ens.size();
  const int32_t nc = (int32_t)m.conns.size();

  // ---- validation and usage scan
  std::vector<char> has_x(ne, 0), has_nin(ne, 0);
  std::vector<std::vector<int32_t>> fns(ne);   // decoded functions, first-use order
  auto use_fn = [&](int32_t e, int32_t fn) {
    if (std::find(fns[e].begin(), fns[e].end(), fn) == fns[e].end()) fns[e].push_back(fn);
  };
  auto ref_size = [&](int32_t kind, int32_t id, int32_t fn) -> int32_t {
    if (kind == MS_REF_NODE) {
      check(id >= 0 && id < nn, "node id out of range");
      return m.nodes[id].size;
    }
    check(id >= 0 && id < ne, "ensemble id out of range");
    if (kind == MS_REF_ENS) return function_size(fn, m.ens[id].d);
    check(kind == MS_REF_NEURONS, "bad reference kind");
    return m.ens[id].n;
  };
  std::vector<int32_t> pre_w(nc), post_w(nc), pre_full(nc), post_full(nc), learn_k(nc, 0);
  for (int32_t ci = 0; ci < nc; ++ci) {
    const ConnDesc& c = m.conns[ci];
    if (!c.learned) continue;
    check(c.pre_kind == MS_REF_ENS && c.pre_id >= 0 && c.pre_id < ne, "a learning connection decodes from an ensemble");
    check(c.pre_start == 0 && c.pre_stop == 0, "a learning connection takes no pre slice");
    learn_k[ci] = c.decoders.empty() ? function_size(c.function, m.ens[c.pre_id].d) : c.decoders_cols;
  }
  for (int32_t ci = 0; ci < nc; ++ci) {
    const ConnDesc& c = m.conns[ci];
    int32_t pf;
    if (c.pre_kind == MS_REF_ENS && !c.decoders.empty()) {
      check(c.pre_id >= 0 && c.pre_id < ne, "ensemble id out of range");
      check((int64_t)c.decoders.size() == (int64_t)m.ens[c.pre_id].n * c.decoders_cols &&
                c.decoders_cols > 0, "explicit decoders must be [n][cols]");
      pf = c.decoders_cols;
    } else {
      if (c.pre_kind == MS_REF_ENS) {
        check(c.function == MS_FN_IDENTITY || c.function == MS_FN_PRODUCT, "bad function");
        check(c.function != MS_FN_PRODUCT || m.ens[c.pre_id].d >= 2, "product needs dims >= 2");
      }
      pf = ref_size(c.pre_kind, c.pre_id, c.function);
    }
    int32_t qf;
    if (c.post_kind == MS_REF_LEARNING) {
      check(c.post_id >= 0 && c.post_id < nc && m.conns[c.post_id].learned,
            "connection into the learning rule of a connection that has none");
      qf = learn_k[c.post_id];
    } else {
      qf = ref_size(c.post_kind, c.post_id, MS_FN_IDENTITY);
    }
    if (c.post_kind == MS_REF_NODE) check(m.nodes[c.post_id].passthrough, "connection into a non-passthrough node");
    pre_full[ci] = pf; post_full[ci] = qf;
    int32_t p0 = c.pre_start, p1 = (c.pre_start == 0 && c.pre_stop == 0) ? pf : c.pre_stop;
    int32_t q0 = c.post_start, q1 = (c.post_start == 0 && c.post_stop == 0) ? qf : c.post_stop;
    check(0 <= p0 && p0 < p1 && p1 <= pf, "pre slice out of range");
    check(0 <= q0 && q0 < q1 && q1 <= qf, "post slice out of range");
    pre_w[ci] = p1 - p0; post_w[ci] = q1 - q0;
    if (c.t_rows == 0) {
      check(c.transform.empty(), "scalar transform with matrix data");
      check(pre_w[ci] == post_w[ci], "scalar transform needs equal pre/post widths");
    } else {
      check(c.t_rows == post_w[ci] && c.t_cols == pre_w[ci], "transform shape must be [post width][pre width]");
      check((int64_t)c.transform.size() == (int64_t)c.t_rows * c.t_cols, "transform size mismatch");
    }
    if (c.post_kind == MS_REF_ENS) has_x[c.post_id] = 1;
    if (c.post_kind == MS_REF_NEURONS) has_nin[c.post_id] = 1;
    if (c.pre_kind == MS_REF_ENS && c.decoders.empty() && !c.learned) use_fn(c.pre_id, c.function);
  }
  for (const ProbeDesc& p : m.probes) {
    int32_t w = ref_size(p.kind, p.id, MS_FN_IDENTITY);
    if (p.kind == MS_REF_NEURONS && !(p.start == 0 && p.stop == 0))
      check(0 <= p.start && p.start < p.stop && p.stop <= w, "probe neuron slice out of range");
    if (p.kind == MS_REF_ENS) use_fn(p.id, MS_FN_IDENTITY);
  }

  // ---- nodes
  std::vector<int32_t> node_out(nn);
  B.ir.feed_row_of_node.assign(nn, -1);
  for (int32_t i = 0; i < nn; ++i) B.ir.node_size.push_back(m.nodes[i].size);
  for (int32_t i = 0; i < nn; ++i) {
    const NodeDesc& nd = m.nodes[i];
    const std::string p = "n" + std::to_string(i);
    node_out[i] = B.batched(p + ".out", nd.size, false);
    if (nd.passthrough) {
      Op& o = B.add(OP_RESET, p + ".reset");
      o.dst = B.whole(node_out[i]);
    } else if (nd.constant) {
      int32_t v = B.param(p + ".value", nd.size, 1, nd.value);
      Op& o = B.add(OP_COPY, p + ".const");
      o.dst = B.whole(node_out[i]);
      o.src = B.whole(v);
    } else {
      B.ir.fed_nodes.push_back(i);
      B.ir.feed_row_of_node[i] = B.ir.feed_rows;
      B.ir.feed_rows += nd.size;
      Op& o = B.add(OP_FEED, p + ".feed");
      o.dst = B.whole(node_out[i]);
      o.node = i;
    }
  }

  // ---- ensembles
  std::vector<int32_t> eJ(ne), eS(ne), eX(ne, -1), eGain(ne, -1);
  std::map<std::pair<int32_t, int32_t>, int32_t> dec_sig;
  B.ir.ens_V.assign(ne, -1);
  B.ir.ens_ref.assign(ne, -1);
  for (int32_t e = 0; e < ne; ++e) {
    const EnsembleDesc& E = m.ens[e];
    const std::string p = "e" + std::to_string(e);
    eJ[e] = B.batched(p + ".J", E.n, false);
    eS[e] = B.batched(p + ".s", E.n, false);
    const bool lif = E.neuron_type == MS_NEURON_LIF;
    int32_t V = -1, R = -1;
    if (lif) {
      V = B.batched(p + ".V", E.n, true);
      R = B.batched(p + ".ref", E.n, true);
      B.ir.ens_V[e] = V;
      B.ir.ens_ref[e] = R;
    }
    int32_t bias = B.param(p + ".bias", E.n, 1, bp.bias[e]);
    int32_t enc = -1;
    if (has_x[e]) {
      eX[e] = B.batched(p + ".x", E.d, false);
      std::vector<double> ge((size_t)E.n * E.d);
      for (int32_t k = 0; k < E.n; ++k)
        for (int32_t j = 0; j < E.d; ++j)
          ge[(size_t)k * E.d + j] = bp.gain[e][k] * E.encoders[(size_t)k * E.d + j];
      enc = B.param(p + ".enc", E.n, E.d, std::move(ge));
    }
    if (has_nin[e]) eGain[e] = B.param(p + ".gain", E.n, 1, bp.gain[e]);
    std::vector<std::pair<int32_t, int32_t>> dec_params;   // (signal, param) per fn
    for (int32_t fn : fns[e]) {
      const int32_t df = function_size(fn, E.d);
      int32_t ds = B.batched(p + ".d" + fn_tag(fn), df, false);
      const std::vector<double>& D = bp.decoders.at({e, fn});   // [n][df]
      std::vector<double> Dt((size_t)df * E.n);
      for (int32_t k = 0; k < E.n; ++k)
        for (int32_t j = 0; j < df; ++j) Dt[(size_t)j * E.n + k] = D[(size_t)k * df + j];
      int32_t dp = B.param(p + ".D" + fn_tag(fn), df, E.n, std::move(Dt));
      dec_sig[{e, fn}] = ds;
      dec_params.push_back({ds, dp});
    }
    if (has_x[e]) {
      Op& o = B.add(OP_RESET, p + ".resetx");
      o.dst = B.whole(eX[e]);
    }
    {
      Op& o = B.add(OP_COPY, p + ".bias");
      o.dst = B.whole(eJ[e]);
      o.src = B.whole(bias);
    }
    if (has_x[e]) {
      Op& o = B.add(OP_DOT_INC, p + ".enc");
      o.dst = B.whole(eJ[e]);
      o.a = B.whole(enc);
      o.src = B.whole(eX[e]);
    }
    {
      Op& o = B.add(lif ? OP_LIF : OP_LIF_RATE, p + ".neurons");
      o.ntype = E.neuron_type;
      o.src = B.whole(eJ[e]);
      o.dst = B.whole(eS[e]);
      if (lif) { o.V = B.whole(V); o.ref = B.whole(R); }
      o.tau_rc = E.tau_rc; o.tau_ref = E.tau_ref; o.amp = E.amplitude; o.sigma = E.sigma;
    }
    for (size_t k = 0; k < fns[e].size(); ++k) {
      const std::string tag = fn_tag(fns[e][k]);
      Op& r = B.add(OP_RESET, p + ".reset" + tag);
      r.dst = B.whole(dec_params[k].first);
      Op& o = B.add(OP_DOT_INC, p + ".dec" + tag);
      o.dst = B.whole(dec_params[k].first);
      o.a = B.whole(dec_params[k].second);
      o.src = B.whole(eS[e]);
    }
  }

  // ---- connections
  B.ir.conn_y.assign(nc, -1);
  B.ir.conn_W.assign(nc, -1);
  B.ir.conn_act.assign(nc, -1);
  std::vector<int32_t> err_sig(nc, -1);
  for (int32_t ci = 0; ci < nc; ++ci)
    if (m.conns[ci].learned) err_sig[ci] = B.batched("c" + std::to_string(ci) + ".E", learn_k[ci], false);
  for (int32_t ci = 0; ci < nc; ++ci) {
    const ConnDesc& c = m.conns[ci];
    const std::string p = "c" + std::to_string(ci);
    // pre value signal
    int32_t pre_sig;
    if (c.learned) {
      const EnsembleDesc& E = m.ens[c.pre_id];
      const int32_t k = learn_k[ci];
      const std::vector<double>& D = c.decoders.empty() ? bp.decoders.at({c.pre_id, c.function}) : c.decoders;
      pre_sig = B.batched(p + ".xd", k, false);
      const int32_t W = B.batched(p + ".W", E.n * k, true);
      B.ir.sigs[W].value = D;   // [n][k] row-major: row i*k + j
      B.ir.conn_W[ci] = W;
      int32_t act = eS[c.pre_id];
      if (c.pes_tau > 0) {
        act = B.batched(p + ".a", E.n, true);
        B.ir.conn_act[ci] = act;
      }
      Op& r = B.add(OP_RESET, p + ".resetd");
      r.dst = B.whole(pre_sig);
      Op& o = B.add(OP_BDOT_INC, p + ".dec");
      o.dst = B.whole(pre_sig);
      o.a = B.whole(W);
      o.src = B.whole(eS[c.pre_id]);
      Op& re = B.add(OP_RESET, p + ".resete");
      re.dst = B.whole(err_sig[ci]);
      Op& u = B.add(OP_PES, p + ".pes");
      u.dst = B.whole(W);
      u.src = B.whole(act);
      u.a = B.whole(err_sig[ci]);
      u.coef_a = -c.pes_rate * dt / E.n;
      if (c.pes_tau > 0) {
        Op& f = B.add(OP_LOWPASS, p + ".presyn");
        f.dst = B.whole(act);
        f.src = B.whole(eS[c.pre_id]);
        const double a = std::exp(-dt / c.pes_tau);
        f.coef_a = a;
        f.coef_b = 1.0 - a;
      }
    } else if (c.pre_kind == MS_REF_NODE) {
      pre_sig = node_out[c.pre_id];
    } else if (c.pre_kind == MS_REF_NEURONS) {
      pre_sig = eS[c.pre_id];
    } else if (!c.decoders.empty()) {
      const EnsembleDesc& E = m.ens[c.pre_id];
      const int32_t cols = c.decoders_cols;
      pre_sig = B.batched(p + ".xd", cols, false);
      std::vector<double> Dt((size_t)cols * E.n);
      for (int32_t k = 0; k < E.n; ++k)
        for (int32_t j = 0; j < cols; ++j) Dt[(size_t)j * E.n + k] = c.decoders[(size_t)k * cols + j];
      int32_t dp = B.param(p + ".D", cols, E.n, std::move(Dt));
      Op& r = B.add(OP_RESET, p + ".resetd");
      r.dst = B.whole(pre_sig);
      Op& o = B.add(OP_DOT_INC, p + ".dec");
      o.dst = B.whole(pre_sig);
      o.a = B.whole(dp);
      o.src = B.whole(eS[c.pre_id]);
    } else {
      pre_sig = dec_sig.at({c.pre_id, c.function});
    }
    const int32_t p0 = c.pre_start;
    const int32_t q0 = c.post_start;
    const int32_t w = post_w[ci], k = pre_w[ci];
    int32_t v = B.batched(p + ".v", w, false);
    int32_t tsig;
    if (c.t_rows == 0)
      tsig = B.param(p + ".t", 1, 1, std::vector<double>{c.t_scalar});
    else
      tsig = B.param(p + ".T", w, k, c.transform);
    int32_t y = -1;
    if (c.synapse > 0) {
      y = B.batched(p + ".y", w, true);
      B.ir.conn_y[ci] = y;
    }
    {
      Op& r = B.add(OP_RESET, p + ".resetv");
      r.dst = B.whole(v);
    }
    {
      Op& o = B.add(c.t_rows == 0 ? OP_ELEM_INC : OP_DOT_INC, p + ".transform");
      o.dst = B.whole(v);
      o.a = B.whole(tsig);
      o.src = SRef{pre_sig, p0, k};
    }
    if (y >= 0) {
      Op& o = B.add(OP_LOWPASS, p + ".synapse");
      o.dst = B.whole(y);
      o.src = B.whole(v);
      const double a = std::exp(-dt / c.synapse);
      o.coef_a = a;
      o.coef_b = 1.0 - a;
    }
    const int32_t delivered = y >= 0 ? y : v;
    if (c.post_kind == MS_REF_LEARNING) {
      Op& o = B.add(OP_COPY_INC, p + ".deliver");
      o.dst = SRef{err_sig[c.post_id], q0, w};
      o.src = B.whole(delivered);
    } else if (c.post_kind == MS_REF_NEURONS) {
      Op& o = B.add(OP_ELEM_INC, p + ".deliver");
      o.dst = SRef{eJ[c.post_id], q0, w};
      o.a = SRef{eGain[c.post_id], q0, w};
      o.src = B.whole(delivered);
    } else {
      Op& o = B.add(OP_COPY_INC, p + ".deliver");
      o.dst = SRef{c.post_kind == MS_REF_ENS ? eX[c.post_id] : node_out[c.post_id], q0, w};
      o.src = B.whole(delivered);
    }
  }

  // ---- probes
  const int32_t np = (int32_t)m.probes.size();
  B.ir.probe_y.assign(np, -1);
  for (int32_t pi = 0; pi < np; ++pi) {
    const ProbeDesc& pd = m.probes[pi];
    SRef target;
    if (pd.kind == MS_REF_NODE) {
      target = B.whole(node_out[pd.id]);
    } else if (pd.kind == MS_REF_ENS) {
      target = B.whole(dec_sig.at({pd.id, MS_FN_IDENTITY}));
    } else {
      target = B.whole(eS[pd.id]);
      if (!(pd.start == 0 && pd.stop == 0)) target = SRef{eS[pd.id], pd.start, pd.stop - pd.start};
    }
    if (pd.synapse > 0) {
      const std::string p = "p" + std::to_string(pi);
      int32_t y = B.batched(p + ".y", target.len, true);
      B.ir.probe_y[pi] = y;
      Op& o = B.add(OP_LOWPASS, p + ".synapse");
      o.dst = B.whole(y);
      o.src = target;
      const double a = std::exp(-dt / pd.synapse);
      o.coef_a = a;
      o.coef_b = 1.0 - a;
      B.ir.probes.push_back({B.whole(y)});
    } else {
      B.ir.probes.push_back({target});
    }
  }
  return std::move(B.ir);
}

// Simplification (Sec. 4.2.4): y += x * 1 becomes y += x, and a copy from a
// signal that never changes (a parameter) becomes a reset to that constant.
void simplify_ir(IR& ir) {
  for (Op& o : ir.ops) {
    if (o.type == OP_ELEM_INC && o.a.len == 1 && o.dst.len >= 1) {
      const Signal& s = ir.sigs[o.a.sig];
      if (s.rows == 1 && s.value.size() == 1 && s.value[0] == 1.0 && o.src.len == o.dst.len) {
        o.type = OP_COPY_INC;
        o.a = SRef{};
      }
    } else if (o.type == OP_COPY && ir.sigs[o.src.sig].cls == SC_PARAM) {
      const Signal& s = ir.sigs[o.src.sig];
      o.type = OP_RESET;
      o.reset_value.assign(s.value.begin() + o.src.start, s.value.begin() + o.src.start + o.src.len);
      o.src = SRef{};
    }
  }
}

// Fuse each ensemble's bias reset, encoder DotInc, neuron update and (when
// small enough) its decoder resets and DotIncs into one ENS operator, so the
// input current and, when nothing else reads them, the spikes never reach
// memory.  Ensembles with neuron-space inputs keep their separate operators.
// The fused operator takes the place of the ensemble's bias operator; signals
// no operator or probe uses any more are dropped (order otherwise kept).
void fuse_ensembles(IR& ir) {
  std::map<std::string, int32_t> op_index;
  for (int32_t k = 0; k < (int32_t)ir.ops.size(); ++k) op_index[ir.ops[k].name] = k;
  auto find = [&](const std::string& n) -> int32_t {
    auto it = op_index.find(n);
    return it == op_index.end() ? -1 : it->second;
  };
  // readers of each signal other than decoder DotIncs of its own ensemble
  std::vector<int32_t> other_readers(ir.sigs.size(), 0);
  for (const Op& o : ir.ops) {
    const bool own_dec = o.type == OP_DOT_INC && o.name.size() > 4 &&
                         o.name.find(".dec") != std::string::npos && o.name[0] == 'e';
    if (!own_dec) {
      if (o.src.sig >= 0) other_readers[o.src.sig]++;
      if (o.a.sig >= 0) other_readers[o.a.sig]++;
    }
  }
  for (const auto& p : ir.probes) other_readers[p.src.sig]++;
  std::vector<int32_t> writers(ir.sigs.size(), 0);
  for (const Op& o : ir.ops)
    if (o.dst.sig >= 0 && o.type != OP_LIF && o.type != OP_LIF_RATE) writers[o.dst.sig]++;
  std::map<std::string, int32_t> sig_index;
  for (int32_t k = 0; k < (int32_t)ir.sigs.size(); ++k) sig_index[ir.sigs[k].name] = k;
  std::vector<char> drop(ir.ops.size(), 0);
  std::vector<std::pair<int32_t, Op>> fused;   // (position, op)
  for (int32_t e = 0;; ++e) {
    const std::string p = "e" + std::to_string(e);
    const int32_t kb = find(p + ".bias"), kn = find(p + ".neurons");
    if (kb < 0 || kn < 0) break;
    const Op& nop = ir.ops[kn];
    const int32_t J = nop.src.sig;
    // the fused kernels compute the LIF, LIF rate and ReLU curves only
    if (nop.type == OP_LIF_RATE && nop.ntype == MS_NEURON_SOFTLIF_RATE) continue;
    // J must be written only by the bias op and the encoder op
    const int32_t ke = find(p + ".enc");
    if (writers[J] != 1 + (ke >= 0 ? 1 : 0)) continue;
    Op f;
    f.type = OP_ENS;
    f.name = p + ".ens";
    f.ntype = nop.type == OP_LIF ? MS_NEURON_LIF : nop.ntype;
    f.n = nop.src.len;
    f.tau_rc = nop.tau_rc; f.tau_ref = nop.tau_ref; f.amp = nop.amp;
    f.V = nop.V; f.ref = nop.ref;
    f.bias = SRef{sig_index.at(p + ".bias"), 0, f.n};
    if (ke >= 0) { f.src = ir.ops[ke].src; f.a = ir.ops[ke].a; }
    // decoders
    std::vector<int32_t> dec_ops;
    int32_t total = 0;
    for (const char* tag : {"id", "prod"}) {
      const int32_t kr = find(p + ".reset" + tag), kd = find(p + ".dec" + tag);
      if (kr >= 0 && kd >= 0) { dec_ops.push_back(kr); dec_ops.push_back(kd); total += ir.ops[kd].dst.len; }
    }
    // keep the function order of first use (operator order)
    std::vector<int32_t> dec_pairs;
    for (size_t k = 0; k + 1 < dec_ops.size(); k += 2) dec_pairs.push_back(dec_ops[k + 1]);
    std::sort(dec_pairs.begin(), dec_pairs.end());
    const bool fuse_dec = total <= kMaxFusedDecoded;
    if (fuse_dec)
      for (int32_t kd : dec_pairs) f.decs.push_back({ir.ops[kd].a, ir.ops[kd].dst});
    // spikes stored only if something besides fused decoders reads them
    const int32_t S = nop.dst.sig;
    const bool s_needed = other_readers[S] > 0 || !fuse_dec;
    if (s_needed) f.dst = nop.dst;
    drop[kb] = 1; drop[kn] = 1;
    if (ke >= 0) drop[ke] = 1;
    if (fuse_dec)
      for (int32_t k : dec_ops) drop[k] = 1;
    fused.push_back({kb, f});
  }
  if (fused.empty()) return;
  std::vector<Op> ops;
  size_t fi = 0;
  for (int32_t k = 0; k < (int32_t)ir.ops.size(); ++k) {
    if (fi < fused.size() && fused[fi].first == k) { ops.push_back(fused[fi].second); ++fi; continue; }
    if (!drop[k]) ops.push_back(ir.ops[k]);
  }
  ir.ops.swap(ops);
  // drop signals nothing references any more
  std::vector<char> used(ir.sigs.size(), 0);
  auto mark = [&](const SRef& r) { if (r.sig >= 0) used[r.sig] = 1; };
  for (const Op& o : ir.ops) {
    mark(o.dst); mark(o.src); mark(o.a); mark(o.V); mark(o.ref); mark(o.bias);
    for (const auto& d : o.decs) { mark(d.first); mark(d.second); }
  }
  for (const auto& p : ir.probes) mark(p.src);
  std::vector<int32_t> remap(ir.sigs.size(), -1);
  std::vector<Signal> sigs;
  for (size_t s = 0; s < ir.sigs.size(); ++s)
    if (used[s]) { remap[s] = (int32_t)sigs.size(); sigs.push_back(std::move(ir.sigs[s])); }
  ir.sigs.swap(sigs);
  auto rm = [&](SRef& r) { if (r.sig >= 0) r.sig = remap[r.sig]; };
  for (Op& o : ir.ops) {
    rm(o.dst); rm(o.src); rm(o.a); rm(o.V); rm(o.ref); rm(o.bias);
    for (auto& d : o.decs) { rm(d.first); rm(d.second); }
  }
  for (auto& p : ir.probes) rm(p.src);
  for (auto* v : {&ir.ens_V, &ir.ens_ref, &ir.conn_y, &ir.probe_y, &ir.conn_W, &ir.conn_act})
    for (int32_t& x : *v) if (x >= 0) x = remap[x];
}

}  // namespace ms
