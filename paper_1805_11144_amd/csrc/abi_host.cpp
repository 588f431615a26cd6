// Host half of the C ABI: model description, host-only planning and error
// reporting.  Every entry point converts exceptions into an ms_status.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>

#include "host.hpp"

namespace ms {

namespace {
thread_local std::string g_last_error;
}

void set_last_error(const std::string& msg) { g_last_error = msg; }

[[noreturn]] void fail(ms_status code, const std::string& msg) { throw Error(code, msg); }

}  // namespace ms

struct ms_model {
  ms::Model m;
};

struct ms_plan {
  std::unique_ptr<ms::Plan> p;
  std::string json;
};

namespace {

using ms::guarded;

std::vector<double> copy_or_empty(const double* p, size_t n) {
  return p ? std::vector<double>(p, p + n) : std::vector<double>();
}

void need(bool ok, const char* msg) {
  if (!ok) ms::fail(MS_E_INVALID, msg);
}

}  // namespace

namespace ms {
PlanOpts plan_opts_from(const ms_sim_opts* o) {
  PlanOpts p;
  if (o) {
    p.planner = o->planner;
    p.depth = o->planner_depth;
    p.merge = o->merge != 0;
    p.sort = o->sort != 0;
    p.simplify = o->simplify != 0;
    p.fuse = (o->fuse & MS_FUSE_ENSEMBLES) != 0;
    p.fuse_synapse = (o->fuse & MS_FUSE_SYNAPSES) != 0;
    need(o->minibatch >= 1, "minibatch must be >= 1");
    p.minibatch = o->minibatch;
    need(p.planner == MS_PLANNER_GREEDY || p.planner == MS_PLANNER_TREE, "unknown planner");
    need(p.depth >= 1 && p.depth <= 8, "planner depth must be in [1, 8]");
  }
  return p;
}
const Model& model_of(const ms_model* m) { return m->m; }
}  // namespace ms

extern "C" {

const char* ms_last_error(void) { return ms::g_last_error.c_str(); }

void ms_sim_opts_default(ms_sim_opts* o) {
  if (!o) return;
  std::memset(o, 0, sizeof(*o));
  o->dt = 0.001;
  o->minibatch = 1;
  o->unroll = 10;
  o->planner = MS_PLANNER_TREE;
  o->planner_depth = 3;
  o->merge = 1;
  o->sort = 1;
  o->simplify = 1;
  o->fuse = MS_FUSE_ENSEMBLES | MS_FUSE_SYNAPSES;
  o->driver = MS_DRIVER_AUTO;
  o->device = 0;
  o->stream = nullptr;
  o->probe_capacity_steps = 1000;
  o->gemm_dtype = MS_GEMM_F32;
  o->decode = MS_DECODE_DENSE;
}

ms_status ms_model_create(ms_model** out) {
  return guarded([&] {
    need(out != nullptr, "out is NULL");
    *out = new ms_model();
  });
}

void ms_model_destroy(ms_model* m) { delete m; }

ms_status ms_model_add_node(ms_model* m, int32_t size, const double* value, int32_t passthrough,
                            int32_t* id_out) {
  return guarded([&] {
    need(m && id_out, "NULL argument");
    need(size > 0, "node size must be positive");
    ms::NodeDesc n;
    n.size = size;
    n.passthrough = passthrough != 0;
    n.constant = !n.passthrough && value != nullptr;
    if (n.constant) n.value.assign(value, value + size);
    m->m.nodes.push_back(std::move(n));
    *id_out = (int32_t)m->m.nodes.size() - 1;
  });
}

ms_status ms_model_add_ensemble(ms_model* m, const ms_ensemble_desc* d, int32_t* id_out) {
  return guarded([&] {
    need(m && d && id_out, "NULL argument");
    need(d->n_neurons > 0 && d->dims > 0, "ensemble needs n_neurons > 0 and dims > 0");
    need(d->neuron_type == MS_NEURON_LIF || d->neuron_type == MS_NEURON_LIF_RATE || d->neuron_type == MS_NEURON_RELU ||
             d->neuron_type == MS_NEURON_SOFTLIF_RATE,
         "unknown neuron type");
    need(d->neuron_type != MS_NEURON_SOFTLIF_RATE || d->sigma > 0, "the soft LIF rate needs sigma > 0");
    need(d->tau_rc > 0 && d->tau_ref >= 0, "tau_rc must be > 0 and tau_ref >= 0");
    need(d->encoders != nullptr, "encoders are required");
    const size_t n = (size_t)d->n_neurons;
    ms::EnsembleDesc e;
    e.n = d->n_neurons;
    e.d = d->dims;
    e.neuron_type = d->neuron_type;
    e.tau_rc = d->tau_rc;
    e.tau_ref = d->tau_ref;
    e.amplitude = d->amplitude;
    e.sigma = d->neuron_type == MS_NEURON_SOFTLIF_RATE ? d->sigma : 0.0;
    e.encoders.assign(d->encoders, d->encoders + n * d->dims);
    if (d->gains) {
      need(d->biases != nullptr, "gains given without biases");
      e.gains = copy_or_empty(d->gains, n);
      e.biases = copy_or_empty(d->biases, n);
    } else {
      need(d->max_rates && d->intercepts, "need gains+biases or max_rates+intercepts");
      e.max_rates = copy_or_empty(d->max_rates, n);
      e.intercepts = copy_or_empty(d->intercepts, n);
      for (size_t k = 0; k < n; ++k) {
        need(e.max_rates[k] > 0 && 1.0 / e.max_rates[k] > e.tau_ref, "max rate must be in (0, 1/tau_ref)");
        need(e.intercepts[k] < 1.0, "intercepts must be < 1");
      }
    }
    need(d->n_eval_points >= 0, "n_eval_points must be >= 0");
    e.n_eval = d->n_eval_points;
    if (e.n_eval > 0) {
      need(d->eval_points != nullptr, "eval_points is NULL");
      e.eval_points.assign(d->eval_points, d->eval_points + (size_t)e.n_eval * d->dims);
    }
    m->m.ens.push_back(std::move(e));
    *id_out = (int32_t)m->m.ens.size() - 1;
  });
}

ms_status ms_model_add_connection(ms_model* m, const ms_connection_desc* d, int32_t* id_out) {
  return guarded([&] {
    need(m && d && id_out, "NULL argument");
    ms::ConnDesc c;
    c.pre_kind = d->pre_kind; c.pre_id = d->pre_id; c.pre_start = d->pre_start; c.pre_stop = d->pre_stop;
    c.post_kind = d->post_kind; c.post_id = d->post_id;
    c.post_start = d->post_start; c.post_stop = d->post_stop;
    c.function = d->function;
    need(c.pre_kind >= 0 && c.pre_kind <= 2 && c.post_kind >= 0 && c.post_kind <= 3, "bad reference kind");
    if (d->decoders) {
      need(c.pre_kind == MS_REF_ENS, "explicit decoders need an ensemble pre");
      need(c.pre_id >= 0 && c.pre_id < (int32_t)m->m.ens.size(), "ensemble id out of range");
      need(d->decoders_cols > 0, "decoders_cols must be > 0");
      c.decoders.assign(d->decoders, d->decoders + (size_t)m->m.ens[c.pre_id].n * d->decoders_cols);
      c.decoders_cols = d->decoders_cols;
    }
    c.t_rows = d->transform_rows;
    c.t_cols = d->transform_cols;
    need(c.t_rows >= 0 && c.t_cols >= 0 && ((c.t_rows == 0) == (c.t_cols == 0)), "bad transform shape");
    if (c.t_rows > 0) {
      need(d->transform != nullptr, "transform data is NULL");
      c.transform.assign(d->transform, d->transform + (size_t)c.t_rows * c.t_cols);
    } else {
      c.t_scalar = d->transform_scalar;
    }
    c.synapse = d->synapse_tau;
    m->m.conns.push_back(std::move(c));
    *id_out = (int32_t)m->m.conns.size() - 1;
  });
}

ms_status ms_model_set_pes(ms_model* m, int32_t conn_id, double learning_rate, double pre_synapse_tau) {
  return guarded([&] {
    need(m != nullptr, "NULL argument");
    need(conn_id >= 0 && conn_id < (int32_t)m->m.conns.size(), "connection id out of range");
    ms::ConnDesc& c = m->m.conns[conn_id];
    need(c.pre_kind == MS_REF_ENS, "a learning rule needs a connection that decodes from an ensemble");
    need(c.pre_start == 0 && c.pre_stop == 0, "a learning connection takes no pre slice");
    need(!c.learned, "the connection already has a learning rule");
    need(learning_rate >= 0.0 && std::isfinite(learning_rate), "learning_rate must be finite and >= 0");
    c.learned = true;
    c.pes_rate = learning_rate;
    c.pes_tau = pre_synapse_tau;
  });
}

ms_status ms_model_add_probe(ms_model* m, const ms_probe_desc* d, int32_t* id_out) {
  return guarded([&] {
    need(m && d && id_out, "NULL argument");
    need(d->target_kind >= 0 && d->target_kind <= 2, "bad probe target kind");
    ms::ProbeDesc p;
    p.kind = d->target_kind; p.id = d->target_id; p.start = d->start; p.stop = d->stop;
    p.synapse = d->synapse_tau;
    m->m.probes.push_back(p);
    *id_out = (int32_t)m->m.probes.size() - 1;
  });
}

ms_status ms_plan_create(const ms_model* m, const ms_sim_opts* opts, ms_plan** out) {
  return guarded([&] {
    need(m && out, "NULL argument");
    ms_sim_opts def;
    ms_sim_opts_default(&def);
    const ms_sim_opts* o = opts ? opts : &def;
    need(o->dt > 0, "dt must be > 0");
    auto pl = new ms_plan();
    try {
      pl->p = ms::make_plan(m->m, o->dt, ms::plan_opts_from(o));
    } catch (...) {
      delete pl;
      throw;
    }
    *out = pl;
  });
}

void ms_plan_destroy(ms_plan* p) { delete p; }

ms_status ms_plan_export_json(const ms_plan* p, char* buf, int64_t cap, int64_t* len_out) {
  return guarded([&] {
    need(p && len_out, "NULL argument");
    auto* mp = const_cast<ms_plan*>(p);
    if (mp->json.empty()) mp->json = ms::plan_to_json(*p->p);
    *len_out = (int64_t)mp->json.size();
    if (buf && cap > 0) {
      const int64_t n = std::min<int64_t>(cap - 1, (int64_t)mp->json.size());
      std::memcpy(buf, mp->json.data(), (size_t)n);
      buf[n] = 0;
    }
  });
}

ms_status ms_plan_get_param(const ms_plan* p, int32_t which, int32_t ens, int32_t fn, double* out,
                            int64_t cap, int64_t* n_out) {
  return guarded([&] {
    need(p && n_out, "NULL argument");
    const ms::Built& b = p->p->built;
    need(ens >= 0 && ens < (int32_t)b.gain.size(), "ensemble id out of range");
    const std::vector<double>* v = nullptr;
    if (which == MS_PARAM_GAIN) v = &b.gain[ens];
    else if (which == MS_PARAM_BIAS) v = &b.bias[ens];
    else if (which == MS_PARAM_DECODERS) {
      auto it = b.decoders.find({ens, fn});
      need(it != b.decoders.end(), "no decoders built for this (ensemble, function)");
      v = &it->second;
    } else {
      need(false, "unknown parameter");
    }
    *n_out = (int64_t)v->size();
    if (out) {
      need(cap >= (int64_t)v->size(), "output capacity too small");
      std::memcpy(out, v->data(), v->size() * sizeof(double));
    }
  });
}

ms_status ms_plan_export_base(const ms_plan* p, int32_t base, float* out, int64_t cap, int64_t* n_out) {
  return guarded([&] {
    need(p && n_out, "NULL argument");
    const ms::Plan& P = *p->p;
    const ms::IR& ir = P.ir;
    need(base >= 0 && base < (int32_t)ir.bases.size(), "base id out of range");
    const int64_t cols = ir.bases[base].cols;   // 1 for the batched state base
    const int64_t n = P.base_rows[base] * cols;
    *n_out = n;
    if (!out) return;
    need(cap >= n, "output capacity too small");
    std::fill(out, out + n, 0.0f);
    for (size_t k = 0; k < ir.sigs.size(); ++k) {
      const ms::Signal& s = ir.sigs[k];
      if (s.base != base) continue;
      const int64_t off = P.sig_offset[k] * cols;
      for (size_t j = 0; j < s.value.size(); ++j) out[off + j] = (float)s.value[j];
    }
  });
}

}  // extern "C"
