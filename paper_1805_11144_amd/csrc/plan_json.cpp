// JSON export of a plan: base arrays, signal placement and the merged groups in
// execution order with their lowered operands.  Used by tests to compare the
// planner bit for bit with an independent implementation.
#include <sstream>

#include "host.hpp"

namespace ms {

namespace {

void jstr(std::ostringstream& o, const std::string& s) {
  o << '"';
  for (char c : s) {
    if (c == '"' || c == '\\') o << '\\';
    o << c;
  }
  o << '"';
}

template <class T>
void jarr(std::ostringstream& o, const std::vector<T>& v) {
  o << '[';
  for (size_t i = 0; i < v.size(); ++i) {
    if (i) o << ',';
    o << v[i];
  }
  o << ']';
}

void joperand(std::ostringstream& o, const LOperand& x) {
  o << "{\"base\":" << x.base;
  if (x.contiguous()) o << ",\"start\":" << x.start;
  else { o << ",\"idx\":"; jarr(o, x.idx); }
  o << '}';
}

void jgroup(std::ostringstream& o, const Plan& p, const LGroup& L) {
  const IR& ir = p.ir;
  o << "{\"type\":";
  jstr(o, op_type_name(L.type));
  o << ",\"key\":" << p.key_of_op[L.ops[0]] << ",\"ops\":[";
  for (size_t k = 0; k < L.ops.size(); ++k) {
    if (k) o << ',';
    jstr(o, ir.ops[L.ops[k]].name);
  }
  o << "],\"rows\":" << L.rows;
  if (L.type == OP_ENS) {
    o << ",\"d\":" << L.ens_d << ",\"neuron\":" << L.ens_type << ",\"enc_base\":" << L.a.base
      << ",\"bias_base\":" << L.ens_bias_base << ",\"D_base\":";
    jarr(o, L.ens_Dbase);
    o << ",\"n\":";
    jarr(o, L.ens_n);
    o << ",\"x_row\":"; jarr(o, L.ens_x);
    o << ",\"enc_row\":"; jarr(o, L.ens_enc);
    o << ",\"bias_row\":"; jarr(o, L.ens_bias);
    o << ",\"V_row\":"; jarr(o, L.ens_V);
    o << ",\"ref_row\":"; jarr(o, L.ens_ref);
    o << ",\"s_row\":"; jarr(o, L.ens_s);
    o << ",\"df\":"; jarr(o, L.ens_df);
    o << ",\"D_row\":[";
    for (size_t k = 0; k < L.ens_D.size(); ++k) { if (k) o << ','; jarr(o, L.ens_D[k]); }
    o << "],\"d_row\":[";
    for (size_t k = 0; k < L.ens_dd.size(); ++k) { if (k) o << ','; jarr(o, L.ens_dd[k]); }
    o << ']';
    o << ",\"tau_rc\":"; jarr(o, L.tau_rc);
    o << ",\"tau_ref\":"; jarr(o, L.tau_ref);
    o << ",\"amp\":"; jarr(o, L.amp);
    if (!L.ens_chain.empty()) {
      o << ",\"chain\":"; jarr(o, L.ens_chain);
      o << ",\"chain_wbase\":" << L.ens_chain_wbase;
    }
  } else if (L.type == OP_SYN_SCATTER) {
    o << ",\"update\":" << L.syn_update << ",\"probe\":" << L.syn_probe << ",\"seg\":";
    jarr(o, L.syn_seg);
    o << ",\"conn\":";
    jarr(o, L.syn_conn);
    o << ",\"ab\":";
    jarr(o, L.syn_ab);
    o << ",\"wbase\":";
    jarr(o, L.syn_wbase);
  } else if (L.type == OP_DOT_INC || L.type == OP_BDOT_INC || L.type == OP_PES || L.type == OP_PES_FUSED) {
    o << ",\"M\":" << L.M << ",\"K\":" << L.K << ",\"w_row\":";
    jarr(o, L.w_row);
    o << ",\"x_row\":";
    jarr(o, L.x_row);
    if (L.type != OP_PES) { o << ",\"d_row\":"; jarr(o, L.d_row); }
    if (L.type == OP_PES || L.type == OP_PES_FUSED) {
      o << ",\"e_row\":"; jarr(o, L.e_row);
      o << ",\"coef\":"; jarr(o, L.coef);
    }
    if (L.type == OP_PES_FUSED) { o << ",\"act_row\":"; jarr(o, L.act_row); }
  } else {
    o << ",\"dst\":";
    joperand(o, L.dst);
    if (L.src.base >= 0) { o << ",\"src\":"; joperand(o, L.src); }
    if (L.a.base >= 0) { o << ",\"a\":"; joperand(o, L.a); }
    if (L.V.base >= 0) { o << ",\"V\":"; joperand(o, L.V); }
    if (L.ref.base >= 0) { o << ",\"ref\":"; joperand(o, L.ref); }
    if (!L.ptr.empty()) { o << ",\"ptr\":"; jarr(o, L.ptr); }
    if (!L.feed_rows.empty()) { o << ",\"feed_rows\":"; jarr(o, L.feed_rows); }
    if (!L.values.empty()) { o << ",\"values\":"; jarr(o, L.values); }
    if (L.type == OP_LIF_RATE && L.ens_type != MS_NEURON_LIF_RATE) o << ",\"neuron\":" << L.ens_type;
    if (!L.sigma.empty()) { o << ",\"sigma\":"; jarr(o, L.sigma); }
    if (!L.tau_rc.empty()) {
      o << ",\"tau_rc\":"; jarr(o, L.tau_rc);
      o << ",\"tau_ref\":"; jarr(o, L.tau_ref);
      o << ",\"amp\":"; jarr(o, L.amp);
    }
    if (!L.ca.empty()) { o << ",\"ca\":"; jarr(o, L.ca); o << ",\"cb\":"; jarr(o, L.cb); }
  }
  o << '}';
}

}  // namespace

std::string plan_to_json(const Plan& p) {
  const IR& ir = p.ir;
  std::ostringstream o;
  o.precision(9);
  o << "{\"bases\":[";
  for (size_t b = 0; b < ir.bases.size(); ++b) {
    if (b) o << ',';
    o << "{\"name\":";
    jstr(o, ir.bases[b].name);
    o << ",\"rows\":" << p.base_rows[b] << ",\"cols\":" << ir.bases[b].cols << '}';
  }
  o << "],\"signals\":[";
  for (size_t s = 0; s < ir.sigs.size(); ++s) {
    if (s) o << ',';
    o << "{\"name\":";
    jstr(o, ir.sigs[s].name);
    o << ",\"base\":" << ir.sigs[s].base << ",\"offset\":" << p.sig_offset[s]
      << ",\"rows\":" << ir.sigs[s].rows << '}';
  }
  o << "],\"groups\":[";
  for (size_t g = 0; g < p.lowered.size(); ++g) {
    if (g) o << ',';
    jgroup(o, p, p.lowered[g]);
  }
  o << "],\"probe_rows\":";
  jarr(o, p.probe_src_rows);
  o << ",\"probe_offsets\":";
  jarr(o, p.probe_row_offset);
  o << ",\"feed_rows\":" << ir.feed_rows;
  const WindowPlan w = make_window_plan(p);
  o << ",\"window\":{\"ok\":" << (w.ok ? "true" : "false") << ",\"why\":";
  jstr(o, w.why);
  if (w.ok) {
    o << ",\"levels\":" << w.levels << ",\"rows_v\":" << w.rows_v << ",\"rows_p\":" << w.rows_p
      << ",\"sig_row\":";
    jarr(o, w.sig_row);
    std::vector<int> pv(w.priv.begin(), w.priv.end());
    o << ",\"priv\":";
    jarr(o, pv);
    o << ",\"probe_rows\":";
    jarr(o, w.probe_rows);
    o << ",\"phases\":[";
    for (size_t k = 0; k < w.phases.size(); ++k) {
      if (k) o << ',';
      o << "{\"level\":" << w.phases[k].level << ",\"src_blk\":" << w.phases[k].src_blk
        << ",\"a_blk\":" << w.phases[k].a_blk << ",\"exclusive\":" << (w.phases[k].exclusive ? "true" : "false")
        << ",\"group\":";
      jgroup(o, p, w.phases[k].g);
      o << '}';
    }
    o << ']';
  }
  o << '}';
  // the time-major step program of the launch drivers
  const LaunchPlan lp = make_launch_plan(p);
  o << ",\"launch\":{\"why\":";
  jstr(o, lp.why);
  o << ",\"groups\":[";
  for (size_t g = 0; g < lp.step.size(); ++g) {
    if (g) o << ',';
    jgroup(o, p, lp.step[g]);
  }
  o << "],\"prologue\":";
  if (lp.has_prologue) jgroup(o, p, lp.prologue);
  else o << "null";
  o << "}}";
  return o.str();
}

}  // namespace ms
