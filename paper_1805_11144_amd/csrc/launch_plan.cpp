// The step program of the time-major launch drivers: the plan's merged groups
// of one timestep, with consecutive independent fused-ensemble groups sharing
// a launch and (option MS_FUSE_SYNAPSES) the connection tail of the paper's
// Fig. 2 -- transform DotInc, synaptic filter, Copy of the filtered value into
// the post input -- fused into one group; a PES update runs in the same pass
// over the decoders as the decode that reads them, where the error is known
// by then.  Host code only.
#include <algorithm>
#include <map>
#include <set>

#include "host.hpp"

namespace ms {

namespace {

// ----------------------------------------------- consecutive ensemble groups

// Row ranges [first, last) of the state array that a fused-ensemble group
// reads (inputs) and writes (spikes, decoded outputs; voltage and refractory
// time count as both).
void ens_rows(const LGroup& g, std::vector<std::pair<int64_t, int64_t>>& rd,
              std::vector<std::pair<int64_t, int64_t>>& wr) {
  for (size_t k = 0; k < g.ens_n.size(); ++k) {
    const int64_t n = g.ens_n[k];
    if (g.ens_x[k] >= 0) rd.push_back({g.ens_x[k], g.ens_x[k] + g.ens_d});
    if (g.ens_V[k] >= 0) { wr.push_back({g.ens_V[k], g.ens_V[k] + n}); wr.push_back({g.ens_ref[k], g.ens_ref[k] + n}); }
    if (g.ens_s[k] >= 0) wr.push_back({g.ens_s[k], g.ens_s[k] + n});
    for (size_t f = 0; f < g.ens_dd.size(); ++f) wr.push_back({g.ens_dd[f][k], g.ens_dd[f][k] + g.ens_df[f]});
  }
}

bool ranges_meet(std::vector<std::pair<int64_t, int64_t>> a, std::vector<std::pair<int64_t, int64_t>> b) {
  std::sort(a.begin(), a.end());
  std::sort(b.begin(), b.end());
  size_t i = 0, j = 0;
  while (i < a.size() && j < b.size()) {
    if (a[i].second <= b[j].first) ++i;
    else if (b[j].second <= a[i].first) ++j;
    else return true;
  }
  return false;
}

// Two consecutive fused-ensemble groups can run as one launch when they share
// neuron type, decoded functions and parameter bases, their inputs (if both
// have any) have one width and encoder base, and neither touches a row the
// other writes.  The planner keeps them apart because their operator
// signatures differ (ensembles without input, ensembles whose spikes are
// stored), which would otherwise cost a launch each per step.
bool can_merge_ens(const LGroup& A, const LGroup& B) {
  if (A.type != OP_ENS || B.type != OP_ENS) return false;
  if (A.ens_type != B.ens_type || A.ens_df != B.ens_df || A.ens_Dbase != B.ens_Dbase ||
      A.ens_bias_base != B.ens_bias_base)
    return false;
  const bool ia = A.a.base >= 0 && A.ens_d > 0, ib = B.a.base >= 0 && B.ens_d > 0;
  if (ia && ib && (A.ens_d != B.ens_d || A.a.base != B.a.base)) return false;
  for (int32_t x : A.ens_x) if (x >= 0 && !ia) return false;
  for (int32_t x : B.ens_x) if (x >= 0 && !ib) return false;
  std::vector<std::pair<int64_t, int64_t>> ra, wa, rb, wb;
  ens_rows(A, ra, wa);
  ens_rows(B, rb, wb);
  return !ranges_meet(wa, rb) && !ranges_meet(wb, ra) && !ranges_meet(wa, wb);
}

void append_ens(LGroup& A, const LGroup& B) {
  const size_t na = A.ens_n.size(), nb = B.ens_n.size();
  auto params = [&](std::vector<float>& a, const std::vector<float>& b) {
    if (a.size() == 1 && b.size() == 1 && a[0] == b[0]) return;
    if (a.size() == 1) a.assign(na, a[0]);
    if (b.size() == 1) a.insert(a.end(), nb, b[0]);
    else a.insert(a.end(), b.begin(), b.end());
  };
  params(A.tau_rc, B.tau_rc);
  params(A.tau_ref, B.tau_ref);
  params(A.amp, B.amp);
  if (!(A.a.base >= 0 && A.ens_d > 0)) { A.ens_d = B.ens_d; A.a = B.a; A.src = B.src; }
  auto cat = [](std::vector<int32_t>& a, const std::vector<int32_t>& b) { a.insert(a.end(), b.begin(), b.end()); };
  cat(A.ops, B.ops);
  cat(A.ens_n, B.ens_n); cat(A.ens_x, B.ens_x); cat(A.ens_enc, B.ens_enc); cat(A.ens_bias, B.ens_bias);
  cat(A.ens_V, B.ens_V); cat(A.ens_ref, B.ens_ref); cat(A.ens_s, B.ens_s);
  for (size_t f = 0; f < A.ens_D.size(); ++f) { cat(A.ens_D[f], B.ens_D[f]); cat(A.ens_dd[f], B.ens_dd[f]); }
  A.rows += B.rows;
}

// ----------------------------------------------------- row access of a group

int64_t lrow(const LOperand& o, int64_t r) { return o.idx.empty() ? o.start + r : (int64_t)o.idx[r]; }

LOperand rows_operand(int32_t base, const std::vector<int32_t>& rows) {
  LOperand o;
  o.base = base;
  bool contig = true;
  for (size_t i = 1; i < rows.size() && contig; ++i) contig = rows[i] == rows[0] + (int32_t)i;
  if (contig) o.start = rows.empty() ? 0 : rows[0];
  else o.idx = rows;
  return o;
}


// Entries of an increment group (COPY_INC / ELEM_INC): ptr gives the entries of
// unique destination u, or one entry per destination without ptr.
int64_t n_entries(const LGroup& g) { return g.ptr.empty() ? g.rows : (int64_t)g.ptr.back(); }

// State rows a group reads and writes (state base `sb`); `wr` holds every row
// it stores to, increments included.
void accesses(const IR& ir, int32_t sb, const LGroup& g, std::vector<int64_t>& rd, std::vector<int64_t>& wr) {
  rd.clear();
  wr.clear();
  auto on_state = [&](const LOperand& o) { return o.base == sb; };
  auto rows_of = [&](const LOperand& o, int64_t n, std::vector<int64_t>& out) {
    if (!on_state(o)) return;
    for (int64_t r = 0; r < n; ++r) out.push_back(lrow(o, r));
  };
  (void)ir;
  switch (g.type) {
    case OP_FEED:
    case OP_RESET: rows_of(g.dst, g.rows, wr); break;
    case OP_COPY: rows_of(g.dst, g.rows, wr); rows_of(g.src, g.rows, rd); break;
    case OP_COPY_INC:
    case OP_ELEM_INC:
      rows_of(g.dst, g.rows, wr);
      rows_of(g.dst, g.rows, rd);
      rows_of(g.src, n_entries(g), rd);
      if (g.type == OP_ELEM_INC) rows_of(g.a, n_entries(g), rd);
      break;
    case OP_DOT_INC:
      for (int64_t o = 0; o < g.rows; ++o) {
        if (g.src.base == sb)
          for (int32_t k = 0; k < g.K; ++k) rd.push_back(g.x_row[o] + k);
        for (int32_t m = 0; m < g.M; ++m) { wr.push_back(g.d_row[o] + m); rd.push_back(g.d_row[o] + m); }
      }
      break;
    case OP_LIF:
      rows_of(g.src, g.rows, rd); rows_of(g.dst, g.rows, wr);
      rows_of(g.V, g.rows, rd); rows_of(g.V, g.rows, wr);
      rows_of(g.ref, g.rows, rd); rows_of(g.ref, g.rows, wr);
      break;
    case OP_LIF_RATE: rows_of(g.src, g.rows, rd); rows_of(g.dst, g.rows, wr); break;
    case OP_LOWPASS:
      rows_of(g.src, g.rows, rd); rows_of(g.dst, g.rows, rd); rows_of(g.dst, g.rows, wr);
      break;
    case OP_BDOT_INC:
    case OP_PES:
    case OP_PES_FUSED:
      for (int64_t o = 0; o < g.rows; ++o) {
        const int64_t nw = (int64_t)g.M * g.K;
        for (int64_t r = 0; r < nw; ++r) rd.push_back(g.w_row[o] + r);
        if (g.type != OP_BDOT_INC) for (int64_t r = 0; r < nw; ++r) wr.push_back(g.w_row[o] + r);
        for (int32_t k = 0; k < g.K; ++k) rd.push_back(g.x_row[o] + k);
        if (g.type == OP_PES_FUSED) for (int32_t k = 0; k < g.K; ++k) rd.push_back(g.act_row[o] + k);
        if (g.type != OP_BDOT_INC) for (int32_t m = 0; m < g.M; ++m) rd.push_back(g.e_row[o] + m);
        if (g.type != OP_PES)
          for (int32_t m = 0; m < g.M; ++m) { rd.push_back(g.d_row[o] + m); wr.push_back(g.d_row[o] + m); }
      }
      break;
    case OP_ENS:
      for (size_t k = 0; k < g.ens_n.size(); ++k) {
        const int64_t n = g.ens_n[k];
        if (g.ens_x[k] >= 0) for (int32_t q = 0; q < g.ens_d; ++q) rd.push_back(g.ens_x[k] + q);
        if (g.ens_V[k] >= 0)
          for (int64_t r = 0; r < n; ++r) {
            rd.push_back(g.ens_V[k] + r); wr.push_back(g.ens_V[k] + r);
            rd.push_back(g.ens_ref[k] + r); wr.push_back(g.ens_ref[k] + r);
          }
        if (g.ens_s[k] >= 0) for (int64_t r = 0; r < n; ++r) wr.push_back(g.ens_s[k] + r);
        for (size_t f = 0; f < g.ens_dd.size(); ++f)
          for (int32_t q = 0; q < g.ens_df[f]; ++q) wr.push_back(g.ens_dd[f][k] + q);
      }
      break;
    default: fail(MS_E_INVALID, "step program: unknown group type");
  }
}

// One connection of a fused segment: its value v for row i of the segment is
// either state row v + i, or the product of weight row w + i (slot ws, K wide)
// with input rows x .. x + K - 1, or (ws == -2, an elementwise transform) the
// scale whose float bits are w times input row x + i; its filter row is y + i.
// v == -2 marks a probe copy: row y is read and recorded, nothing updated.
// pr: the probe row that records row y (-1: none).
// stage: the inputs x .. x + K - 1 are rows of the step's feed staging
// buffer, not of the state (the node rows a Feed group fills from there).
struct Conn {
  int32_t y = -1, v = -1, x = -1, K = 0, ws = -1, w = -1, pr = -1, stage = 0;
  float a = 0.f, b = 0.f;
  bool next_of(const Conn& p) const {   // row i + 1 of the same arithmetic run as p
    if (y != p.y + 1 || a != p.a || b != p.b || (v < 0) != (p.v < 0) || stage != p.stage) return false;
    if ((pr < 0) != (p.pr < 0) || (pr >= 0 && pr != p.pr + 1)) return false;
    if (v == -2 || p.v == -2) return v == p.v;
    if (v >= 0) return v == p.v + 1;
    if (ws == -2 || p.ws == -2) return ws == p.ws && x == p.x + 1 && w == p.w;
    return ws == p.ws && x == p.x && K == p.K && w == p.w + 1;
  }
};

// Builds the fused group from the step's groups G, or explains why not.
struct Fuser {
  const Plan& p;
  const std::vector<LGroup>& G;
  int32_t sb = -1;
  int64_t nrows = 0;
  std::string why;

  Fuser(const Plan& pl, const std::vector<LGroup>& g) : p(pl), G(g) {
    for (size_t b = 0; b < p.ir.bases.size(); ++b)
      if (p.ir.bases[b].cls == SC_BATCHED) { sb = (int32_t)b; nrows = p.base_rows[b]; }
  }

  std::vector<int32_t> lidx;     // filter row -> index in the filter group, or -1
  std::vector<int32_t> vcount;   // how often the filter group reads each row as its input

  bool no(const std::string& w) { why = w; return false; }

  // value of row `row` of a one-column parameter base (the plan's float32 values)
  std::map<int32_t, std::vector<float>> pbase;
  float param_value(int32_t base, int64_t row) {
    auto it = pbase.find(base);
    if (it == pbase.end()) {
      std::vector<float> v((size_t)p.base_rows[base] * p.ir.bases[base].cols, 0.0f);
      for (size_t k = 0; k < p.ir.sigs.size(); ++k) {
        const Signal& sg = p.ir.sigs[k];
        if (sg.base != base) continue;
        const size_t off = (size_t)p.sig_offset[k] * p.ir.bases[base].cols;
        for (size_t j = 0; j < sg.value.size(); ++j) v[off + j] = (float)sg.value[j];
      }
      it = pbase.emplace(base, std::move(v)).first;
    }
    return it->second[(size_t)row * p.ir.bases[base].cols];
  }

  bool run(std::vector<LGroup>& out, LGroup& prologue);
  bool fuse_with(int32_t ci, std::vector<LGroup>& out, LGroup& prologue);
};

// The step must end with the filter group; the first CopyInc group that pulls
// only filtered values and passes every check of fuse_with is fused with it.
bool Fuser::run(std::vector<LGroup>& out, LGroup& prologue) {
  const int32_t n = (int32_t)G.size();
  if (sb < 0 || n == 0) return no("no batched signals");
  const LGroup& L = G[n - 1];
  if (L.type != OP_LOWPASS) return no("the step does not end with the synaptic filters");
  if (L.dst.base != sb || L.src.base != sb) return no("filter operands outside the state array");
  lidx.assign((size_t)nrows, -1);
  vcount.assign((size_t)nrows, 0);
  for (int64_t r = 0; r < L.rows; ++r) {
    const int64_t y = lrow(L.dst, r), v = lrow(L.src, r);
    if (lidx[y] >= 0) return no("a filter row updated twice");
    lidx[y] = (int32_t)r;
    ++vcount[v];
  }
  bool any = false;
  for (int32_t g = 0; g + 1 < n; ++g) {
    const LGroup& c = G[g];
    if (c.type != OP_COPY_INC || c.src.base != sb || c.dst.base != sb) continue;
    bool all = true;
    for (int64_t e = 0; e < n_entries(c) && all; ++e) all = lidx[lrow(c.src, e)] >= 0;
    if (!all) continue;
    any = true;
    if (fuse_with(g, out, prologue)) return true;
  }
  if (!any) return no("no copy of filtered values into post inputs");
  return false;
}

bool Fuser::fuse_with(int32_t ci, std::vector<LGroup>& out, LGroup& prologue) {
  const int32_t n = (int32_t)G.size();
  const LGroup& L = G[n - 1];
  const int64_t nl = L.rows;
  const LGroup& C = G[ci];
  std::vector<char> pulled((size_t)nl, 0), isdst((size_t)nrows, 0), probed((size_t)nrows, 0);
  for (int64_t e = 0; e < n_entries(C); ++e) {
    const int32_t r = lidx[lrow(C.src, e)];
    if (pulled[r]) return no("a filtered value copied twice");
    pulled[r] = 1;
  }
  for (int64_t u = 0; u < C.rows; ++u) isdst[lrow(C.dst, u)] = 1;
  for (int32_t r : p.probe_src_rows) probed[r] = 1;
  for (int64_t u = 0; u < C.rows; ++u) {
    const int64_t x = lrow(C.dst, u);
    if (probed[x]) return no("a probe reads a post input");
    if (lidx[x] >= 0 || vcount[x] > 0) return no("a post input is a filter row");
  }
  // every post input is reset to zero before the copy and touched by nothing
  // else before it; the resets of those rows go
  std::vector<char> reset0((size_t)nrows, 0);
  std::vector<int64_t> rd, wr;
  for (int32_t g = 0; g < ci; ++g) {
    const LGroup& q = G[g];
    if (q.type == OP_RESET && q.dst.base == sb) {
      for (int64_t r = 0; r < q.rows; ++r) {
        const int64_t x = lrow(q.dst, r);
        if (!isdst[x]) continue;
        if (!q.values.empty() && q.values[r] != 0.0f) return no("a post input reset to a nonzero value");
        reset0[x] = 1;
      }
      continue;
    }
    accesses(p.ir, sb, q, rd, wr);
    for (int64_t x : rd) if (isdst[x]) return no("a post input read before the copy");
    for (int64_t x : wr) if (isdst[x]) return no("a post input written before the copy");
  }
  for (int64_t u = 0; u < C.rows; ++u)
    if (!reset0[lrow(C.dst, u)]) return no("a post input not reset before the copy");

  // filter inputs computed here: written only by zero resets (before the
  // product) and by one row of one DotInc op with constant weights, read only
  // by the filter, not probed, and with inputs that nothing rewrites before
  // the filter's place
  // el: the row is the single entry of a CopyInc / ElementwiseInc (input row
  // ex times scale) rather than a row of a DotInc op
  struct Src {
    int32_t g = -1; int32_t op = -1; int32_t m = -1; int32_t writers = 0; int32_t first_reset = -1;
    bool el = false; int64_t ex = -1; float scale = 1.0f;
  };
  std::vector<Src> vs((size_t)nrows);
  std::vector<int32_t> readers((size_t)nrows, 0), last_writer((size_t)nrows, -1);
  for (int32_t g = 0; g + 1 < n; ++g) {
    const LGroup& q = G[g];
    accesses(p.ir, sb, q, rd, wr);
    if (q.type == OP_RESET && q.values.empty()) {
      for (int64_t x : wr) if (vcount[x] > 0 && vs[x].first_reset < 0) vs[x].first_reset = g;
    } else if (q.type == OP_DOT_INC) {
      for (int64_t o = 0; o < q.rows; ++o)
        for (int32_t m = 0; m < q.M; ++m) {
          Src& s = vs[q.d_row[o] + m];
          ++s.writers;
          s.g = g; s.op = (int32_t)o; s.m = m;
        }
      // reads of a DotInc's own destination (its accumulation) are not reads
      std::vector<int64_t> rd2;
      for (int64_t o = 0; o < q.rows; ++o)
        if (q.src.base == sb) for (int32_t k = 0; k < q.K; ++k) rd2.push_back(q.x_row[o] + k);
      rd.swap(rd2);
    } else if ((q.type == OP_COPY_INC || q.type == OP_ELEM_INC) && q.dst.base == sb && q.src.base == sb && g != ci) {
      // single-entry destinations that are filter inputs may fold (v = scale
      // x); the accumulation's read of its own destination is not a read
      const bool a_param = q.type == OP_COPY_INC || (q.a.base >= 0 && p.ir.bases[q.a.base].cls != SC_BATCHED);
      std::vector<int64_t> rd2;
      for (int64_t u = 0; u < q.rows; ++u) {
        const int64_t e0 = q.ptr.empty() ? u : q.ptr[u], e1 = q.ptr.empty() ? u + 1 : q.ptr[u + 1];
        const int64_t x = lrow(q.dst, u);
        for (int64_t e = e0; e < e1; ++e) {
          rd2.push_back(lrow(q.src, e));
          if (q.type == OP_ELEM_INC && !a_param) rd2.push_back(lrow(q.a, e));
        }
        if (vcount[x] == 0) continue;
        Src& sx = vs[x];
        if (e1 - e0 == 1 && a_param) {
          ++sx.writers;
          sx.g = g;
          sx.el = true;
          sx.ex = lrow(q.src, e0);
          sx.scale = q.type == OP_COPY_INC ? 1.0f : param_value(q.a.base, lrow(q.a, e0));
        } else {
          sx.writers += 2;
        }
      }
      rd.swap(rd2);
    } else {
      for (int64_t x : wr) if (vcount[x] > 0) vs[x].writers += 2;   // any other writer disqualifies
    }
    for (int64_t x : rd) ++readers[x];
    for (int64_t x : wr) last_writer[x] = g;
  }
  // which DotInc ops fold into the fused group
  std::map<std::pair<int32_t, int32_t>, bool> op_ok;   // (group, op) -> all rows eligible
  std::vector<int32_t> wslot_base;
  auto eligible = [&](int64_t v) {
    const Src& s = vs[v];
    if (s.writers != 1 || s.g < 0 || vcount[v] != 1 || readers[v] != 0 || probed[v]) return false;
    if (s.first_reset < 0 || s.first_reset > s.g) return false;
    if (s.el)   // input not rewritten after the copy, not written by the fused group
      return last_writer[s.ex] <= s.g && lidx[s.ex] < 0 && !isdst[s.ex];
    const LGroup& D = G[s.g];
    if (D.a.base < 0 || p.ir.bases[D.a.base].cls == SC_BATCHED) return false;
    if (D.src.base != sb) return false;
    if (D.K >= 64 && p.opts.minibatch <= 4) return false;   // that product sums in another order
    for (int32_t k = 0; k < D.K; ++k) {
      const int64_t x = D.x_row[s.op] + k;
      if (last_writer[x] > s.g) return false;        // input rewritten after the product
      if (lidx[x] >= 0 || isdst[x]) return false;    // input written by the fused group itself
    }
    return true;
  };
  std::vector<char> el_fold((size_t)nrows, 0);   // elementwise rows that fold, one by one
  for (int64_t r = 0; r < nl; ++r) {
    const int64_t v = lrow(L.src, r);
    const Src& s = vs[v];
    if (s.g < 0) continue;
    if (s.el) {
      el_fold[v] = eligible(v) ? 1 : 0;
      continue;
    }
    const auto key = std::make_pair(s.g, s.op);
    const bool ok = eligible(v);
    auto it = op_ok.find(key);
    op_ok[key] = (it == op_ok.end() ? true : it->second) && ok;
  }
  // an op folds only if every one of its rows feeds the filter
  for (auto& kv : op_ok) {
    const LGroup& D = G[kv.first.first];
    for (int32_t m = 0; m < D.M && kv.second; ++m) {
      const int64_t v = D.d_row[kv.first.second] + m;
      if (vcount[v] != 1 || !eligible(v)) kv.second = false;
    }
  }
  auto folded = [&](int64_t v) {
    const Src& s = vs[v];
    if (s.g < 0) return false;
    if (s.el) return el_fold[v] != 0;
    auto it = op_ok.find({s.g, s.op});
    return it != op_ok.end() && it->second;
  };
  auto slot_of = [&](int32_t base) -> int32_t {
    for (size_t k = 0; k < wslot_base.size(); ++k) if (wslot_base[k] == base) return (int32_t)k;
    if ((int32_t)wslot_base.size() == kSynSlots) return -1;
    wslot_base.push_back(base);
    return (int32_t)wslot_base.size() - 1;
  };
  // demote ops whose weight base finds no slot
  for (auto& kv : op_ok)
    if (kv.second && slot_of(G[kv.first.first].a.base) < 0) kv.second = false;
  // filter inputs read from the state must not be rows the fused group writes
  for (int64_t r = 0; r < nl; ++r) {
    const int64_t v = lrow(L.src, r);
    if (!folded(v) && (lidx[v] >= 0 || isdst[v])) return no("a filter reads a row the fused group writes");
  }
  // the probe copy folds into the fused group when every probe row records a
  // distinct row: a filter row is recorded by the lane that updates it, any
  // other probed row (final once the filters run, since post inputs are never
  // probed here) by a copy entry
  std::vector<int32_t> probe_of((size_t)nrows, -1);
  bool fold_probe = true;
  for (size_t pr = 0; pr < p.probe_src_rows.size(); ++pr) {
    int32_t& q = probe_of[p.probe_src_rows[pr]];
    if (q >= 0) fold_probe = false;
    q = (int32_t)pr;
  }
  // node rows filled by a Feed group and not rewritten after it: a folded
  // product reads them straight from the feed staging buffer
  std::vector<int32_t> feed_of((size_t)nrows, -1), feed_grp((size_t)nrows, -1);
  for (int32_t g = 0; g + 1 < n; ++g)
    if (G[g].type == OP_FEED && G[g].dst.base == sb)
      for (int64_t r = 0; r < G[g].rows; ++r) {
        const int64_t x = lrow(G[g].dst, r);
        feed_of[x] = G[g].feed_rows[r];
        feed_grp[x] = g;
      }
  auto staged = [&](int64_t x0, int32_t K) {
    for (int32_t k = 0; k < K; ++k) {
      const int64_t x = x0 + k;
      if (feed_of[x] < 0 || feed_of[x] != feed_of[x0] + k || last_writer[x] != feed_grp[x]) return false;
    }
    return K > 0;
  };
  auto conn_of = [&](int64_t r) {
    Conn c;
    c.y = (int32_t)lrow(L.dst, r);
    c.pr = fold_probe ? probe_of[c.y] : -1;
    c.a = L.ca.size() > 1 ? L.ca[r] : L.ca[0];
    c.b = L.cb.size() > 1 ? L.cb[r] : L.cb[0];
    const int64_t v = lrow(L.src, r);
    if (folded(v) && vs[v].el) {
      const Src& s = vs[v];
      c.ws = -2;
      c.K = 0;
      c.x = (int32_t)s.ex;
      c.w = __builtin_bit_cast(int32_t, s.scale);
      if (staged(c.x, 1)) {
        c.stage = 1;
        c.x = feed_of[c.x];
      }
    } else if (folded(v)) {
      const Src& s = vs[v];
      const LGroup& D = G[s.g];
      c.x = D.x_row[s.op];
      c.K = D.K;
      c.ws = slot_of(D.a.base);
      c.w = D.w_row[s.op] + s.m;
      if (staged(c.x, c.K)) {
        c.stage = 1;
        c.x = feed_of[c.x];
      }
    } else {
      c.v = (int32_t)v;
    }
    return c;
  };

  // segments: runs of up to kSynSeg consecutive post inputs whose connections
  // advance row by row, then the filter rows nothing pulls
  LGroup F;
  F.type = OP_SYN_SCATTER;
  F.ops = L.ops;
  std::vector<Conn> conns;
  auto flush = [&](int32_t dst, int32_t len, const std::vector<Conn>& first) {
    F.syn_seg.insert(F.syn_seg.end(), {dst, len, (int32_t)conns.size(), (int32_t)first.size()});
    conns.insert(conns.end(), first.begin(), first.end());
  };
  {
    std::vector<Conn> first, prev, cur;
    int32_t dst0 = -1, len = 0;
    for (int64_t u = 0; u < C.rows; ++u) {
      const int64_t e0 = C.ptr.empty() ? u : C.ptr[u], e1 = C.ptr.empty() ? u + 1 : C.ptr[u + 1];
      cur.clear();
      for (int64_t e = e0; e < e1; ++e) cur.push_back(conn_of(lidx[lrow(C.src, e)]));
      const int32_t x = (int32_t)lrow(C.dst, u);
      bool ext = len > 0 && len < kSynSeg && x == dst0 + len && cur.size() == prev.size();
      for (size_t j = 0; ext && j < cur.size(); ++j) ext = cur[j].next_of(prev[j]);
      if (!ext) {
        if (len > 0) flush(dst0, len, first);
        first = cur;
        dst0 = x;
        len = 0;
      }
      ++len;
      prev = cur;
    }
    if (len > 0) flush(dst0, len, first);
  }
  const int32_t npulled_seg = (int32_t)(F.syn_seg.size() / 4);
  {
    Conn first, prev;
    int32_t len = 0;
    for (int64_t r = 0; r < nl; ++r) {
      if (pulled[r]) continue;
      const Conn c = conn_of(r);
      if (len > 0 && len < kSynSeg && c.next_of(prev)) {
        ++len;
      } else {
        if (len > 0) flush(-1, len, {first});
        first = c;
        len = 1;
      }
      prev = c;
    }
    if (len > 0) flush(-1, len, {first});
  }
  if (fold_probe) {
    Conn first, prev;
    int32_t len = 0;
    for (size_t pr = 0; pr < p.probe_src_rows.size(); ++pr) {
      const int32_t src = p.probe_src_rows[pr];
      if (lidx[src] >= 0) continue;   // recorded where its filter is updated
      Conn c;
      c.y = src;
      c.v = -2;
      c.pr = (int32_t)pr;
      if (len > 0 && len < kSynSeg && c.next_of(prev)) {
        ++len;
      } else {
        if (len > 0) flush(-1, len, {first});
        first = c;
        len = 1;
      }
      prev = c;
    }
    if (len > 0) flush(-1, len, {first});
  }
  for (const Conn& c : conns) {
    F.syn_conn.insert(F.syn_conn.end(), {c.y, c.v, c.x, c.K, c.ws, c.w, c.pr, c.stage});
    F.syn_ab.push_back(c.a);
    F.syn_ab.push_back(c.b);
  }
  F.syn_probe = fold_probe ? 1 : 0;
  F.syn_wbase = wslot_base;
  F.rows = (int64_t)F.syn_seg.size() / 4;
  F.syn_update = 1;
  F.dst.base = sb;
  // the pull alone, for the start of a run
  prologue = F;
  prologue.syn_seg.resize((size_t)npulled_seg * 4);
  prologue.rows = npulled_seg;
  prologue.syn_update = 0;
  prologue.syn_probe = 0;

  // the rest of the step: resets without the post inputs and the folded
  // filter inputs, no CopyInc, DotIncs without the folded ops
  std::vector<char> drop_row((size_t)nrows, 0);
  for (int64_t u = 0; u < C.rows; ++u) drop_row[lrow(C.dst, u)] = 1;
  for (int64_t r = 0; r < nl; ++r) {
    const int64_t v = lrow(L.src, r);
    if (folded(v)) drop_row[v] = 1;
  }
  out.clear();
  for (int32_t g = 0; g + 1 < n; ++g) {
    const LGroup& q = G[g];
    if (g == ci) continue;
    if (q.type == OP_RESET && q.dst.base == sb) {
      std::vector<int32_t> keep;
      std::vector<float> vals;
      for (int64_t r = 0; r < q.rows; ++r) {
        const int64_t x = lrow(q.dst, r);
        if (drop_row[x]) continue;
        keep.push_back((int32_t)x);
        if (!q.values.empty()) vals.push_back(q.values[r]);
      }
      if (keep.empty()) continue;
      LGroup k = q;
      k.rows = (int64_t)keep.size();
      bool contig = true;
      for (size_t i = 1; i < keep.size() && contig; ++i) contig = keep[i] == keep[0] + (int32_t)i;
      k.dst.idx.clear();
      if (contig) k.dst.start = keep[0];
      else k.dst.idx = keep;
      k.values = vals;
      out.push_back(k);
      continue;
    }
    if ((q.type == OP_COPY_INC || q.type == OP_ELEM_INC) && q.dst.base == sb && q.src.base == sb) {
      // without the entries of folded rows (each the single entry of its row)
      std::vector<int32_t> dst, src, av, ptr{0};
      bool any = false;
      for (int64_t u = 0; u < q.rows; ++u) {
        const int64_t x = lrow(q.dst, u);
        if (drop_row[x]) { any = true; continue; }
        const int64_t e0 = q.ptr.empty() ? u : q.ptr[u], e1 = q.ptr.empty() ? u + 1 : q.ptr[u + 1];
        dst.push_back((int32_t)x);
        for (int64_t e = e0; e < e1; ++e) {
          src.push_back((int32_t)lrow(q.src, e));
          if (q.type == OP_ELEM_INC) av.push_back((int32_t)lrow(q.a, e));
        }
        ptr.push_back((int32_t)src.size());
      }
      if (!any) { out.push_back(q); continue; }
      if (dst.empty()) continue;
      LGroup k = q;
      k.ops.clear();
      for (int32_t oi : q.ops) {
        const Op& o = p.ir.ops[oi];
        if (!drop_row[p.sig_offset[o.dst.sig] + o.dst.start]) k.ops.push_back(oi);
      }
      if (k.ops.empty()) k.ops.push_back(q.ops[0]);
      k.rows = (int64_t)dst.size();
      k.dst = rows_operand(sb, dst);
      k.src = rows_operand(sb, src);
      if (q.type == OP_ELEM_INC) k.a = rows_operand(q.a.base, av);
      k.ptr = src.size() == dst.size() ? std::vector<int32_t>{} : ptr;
      out.push_back(k);
      continue;
    }
    if (q.type == OP_DOT_INC) {
      LGroup k = q;
      k.ops.clear(); k.w_row.clear(); k.x_row.clear(); k.d_row.clear();
      for (int64_t o = 0; o < q.rows; ++o) {
        auto it = op_ok.find({g, (int32_t)o});
        if (it != op_ok.end() && it->second) continue;
        k.ops.push_back(q.ops[o]);
        k.w_row.push_back(q.w_row[o]); k.x_row.push_back(q.x_row[o]); k.d_row.push_back(q.d_row[o]);
      }
      k.rows = (int64_t)k.w_row.size();
      if (k.rows > 0) out.push_back(k);
      continue;
    }
    out.push_back(q);
  }
  // a Feed group whose rows nothing reads any more (the products that read
  // them now take the staging buffer) goes
  {
    std::vector<char> read((size_t)nrows, 0);
    for (const LGroup& q : out) {
      accesses(p.ir, sb, q, rd, wr);
      for (int64_t x : rd) read[x] = 1;
    }
    for (int32_t r : p.probe_src_rows) read[r] = 1;
    for (size_t sgi = 0; sgi < F.syn_seg.size(); sgi += 4) {
      const int32_t len = F.syn_seg[sgi + 1], c0 = F.syn_seg[sgi + 2], nc = F.syn_seg[sgi + 3];
      for (int32_t c = c0; c < c0 + nc; ++c) {
        const Conn& q = conns[c];
        for (int32_t i = 0; i < len; ++i) {
          if (q.v >= 0) read[q.v + i] = 1;
          if (q.v == -2) read[q.y + i] = 1;
        }
        if (q.v == -1 && !q.stage && q.ws == -2) for (int32_t i = 0; i < len; ++i) read[q.x + i] = 1;
        if (q.v == -1 && !q.stage && q.ws != -2) for (int32_t k = 0; k < q.K; ++k) read[q.x + k] = 1;
      }
    }
    std::vector<LGroup> kept;
    for (LGroup& q : out) {
      bool needed = q.type != OP_FEED || q.dst.base != sb;
      for (int64_t r = 0; r < q.rows && !needed; ++r) needed = read[lrow(q.dst, r)] != 0;
      if (needed) kept.push_back(std::move(q));
    }
    out.swap(kept);
  }
  out.push_back(F);
  return true;
}

}  // namespace

std::vector<LGroup> merge_ens_groups(const std::vector<LGroup>& in) {
  std::vector<LGroup> out;
  for (const LGroup& g : in) {
    if (!out.empty() && can_merge_ens(out.back(), g)) append_ens(out.back(), g);
    else out.push_back(g);
  }
  return out;
}

namespace {

int32_t state_base(const Plan& p) {
  int32_t sb = -1;
  for (size_t b = 0; b < p.ir.bases.size(); ++b)
    if (p.ir.bases[b].cls == SC_BATCHED) sb = (int32_t)b;
  return sb;
}

bool overlap(const std::vector<int64_t>& a, const std::vector<int64_t>& b) {
  if (a.empty() || b.empty()) return false;
  std::set<int64_t> s(a.begin(), a.end());
  for (int64_t x : b) if (s.count(x)) return true;
  return false;
}


// A CopyInc group whose destinations are of two kinds -- all of a
// destination's entries pull filter rows of the last group and the filters
// neither read nor probes record the destination, or not -- splits into the
// pulls and the rest at the same place (they write different rows), so that
// the pulls can fuse with the filters.  A destination whose entries mix
// filtered and other values keeps the group whole.
void split_pulls(const Plan& p, std::vector<LGroup>& G) {
  const int32_t sb = state_base(p);
  if (sb < 0 || G.empty() || G.back().type != OP_LOWPASS) return;
  const LGroup& L = G.back();
  std::set<int64_t> filt, busy;   // filter rows; rows the filters read or probes record
  for (int64_t r = 0; r < L.rows; ++r) {
    filt.insert(lrow(L.dst, r));
    busy.insert(lrow(L.src, r));
    busy.insert(lrow(L.dst, r));
  }
  for (int32_t r : p.probe_src_rows) busy.insert(r);
  std::vector<LGroup> out;
  for (size_t gi = 0; gi < G.size(); ++gi) {
    const LGroup& q = G[gi];
    if (q.type != OP_COPY_INC || q.src.base != sb || q.dst.base != sb) { out.push_back(q); continue; }
    struct Part { std::vector<int32_t> dst, src, ptr{0}; std::set<int64_t> dset; };
    Part part[2];   // 0: pulls, 1: the rest
    bool mixed = false;
    for (int64_t u = 0; u < q.rows && !mixed; ++u) {
      const int64_t e0 = q.ptr.empty() ? u : q.ptr[u], e1 = q.ptr.empty() ? u + 1 : q.ptr[u + 1];
      int32_t nf = 0;
      for (int64_t e = e0; e < e1; ++e) nf += filt.count(lrow(q.src, e)) ? 1 : 0;
      if (nf != 0 && nf != e1 - e0) { mixed = true; break; }
      Part& P = part[nf && !busy.count(lrow(q.dst, u)) ? 0 : 1];
      P.dst.push_back((int32_t)lrow(q.dst, u));
      P.dset.insert(lrow(q.dst, u));
      for (int64_t e = e0; e < e1; ++e) P.src.push_back((int32_t)lrow(q.src, e));
      P.ptr.push_back((int32_t)P.src.size());
    }
    if (mixed || part[0].dst.empty() || part[1].dst.empty()) { out.push_back(q); continue; }
    for (Part& P : part) {
      LGroup g = q;
      g.rows = (int64_t)P.dst.size();
      g.dst = rows_operand(sb, P.dst);
      g.src = rows_operand(sb, P.src);
      g.ptr = P.src.size() == P.dst.size() ? std::vector<int32_t>{} : P.ptr;
      g.ops.clear();
      for (int32_t oi : q.ops) {
        const Op& o = p.ir.ops[oi];
        if (P.dset.count(p.sig_offset[o.dst.sig] + o.dst.start)) g.ops.push_back(oi);
      }
      out.push_back(std::move(g));
    }
  }
  G.swap(out);
}

// Groups after the last filter group that share no row with it (a PES update
// of decoders nothing else touches, say) move in front of it, so that the
// step ends with the filters.
void filters_last(const Plan& p, std::vector<LGroup>& G) {
  const int32_t sb = state_base(p);
  int32_t L = -1;
  for (int32_t g = 0; g < (int32_t)G.size(); ++g) if (G[g].type == OP_LOWPASS) L = g;
  if (L < 0 || L + 1 == (int32_t)G.size() || sb < 0) return;
  std::vector<int64_t> lr, lw, rd, wr;
  accesses(p.ir, sb, G[L], lr, lw);
  for (int32_t g = L + 1; g < (int32_t)G.size(); ++g) {
    accesses(p.ir, sb, G[g], rd, wr);
    if (overlap(lw, rd) || overlap(lw, wr) || overlap(lr, wr)) return;
  }
  LGroup f = std::move(G[L]);
  G.erase(G.begin() + L);
  G.push_back(std::move(f));
}

// A PES group whose ops are exactly those of a learned-decode group moves to
// the decode's place and runs with it as one pass over the decoders, when
// nothing between the two writes the error or activity rows the update reads
// or touches the decoders.
void fuse_pes(const Plan& p, std::vector<LGroup>& G) {
  const int32_t sb = state_base(p);
  if (sb < 0) return;
  std::vector<int64_t> rd, wr;
  for (int32_t pi = 0; pi < (int32_t)G.size(); ++pi) {
    if (G[pi].type != OP_PES) continue;
    const LGroup& P = G[pi];
    int32_t di = -1;
    for (int32_t g = 0; g < pi; ++g)
      if (G[g].type == OP_BDOT_INC && G[g].w_row == P.w_row && G[g].M == P.M && G[g].K == P.K &&
          G[g].a.base == sb && P.dst.base == sb && G[g].src.base == sb && P.src.base == sb && P.a.base == sb)
        di = g;
    if (di < 0) continue;
    std::vector<int64_t> need;   // rows the update reads besides the decoders
    for (int64_t o = 0; o < P.rows; ++o) {
      for (int32_t k = 0; k < P.K; ++k) need.push_back(P.x_row[o] + k);
      for (int32_t m = 0; m < P.M; ++m) need.push_back(P.e_row[o] + m);
    }
    std::vector<int64_t> wrows;
    for (int64_t o = 0; o < P.rows; ++o)
      for (int64_t r = 0; r < (int64_t)P.M * P.K; ++r) wrows.push_back(P.w_row[o] + r);
    bool ok = true;
    for (int32_t g = di + 1; g < pi && ok; ++g) {
      accesses(p.ir, sb, G[g], rd, wr);
      ok = !overlap(need, wr) && !overlap(wrows, wr) && !overlap(wrows, rd);
    }
    // the decode's own outputs are not among the rows the update reads
    std::vector<int64_t> drows;
    for (int64_t o = 0; o < P.rows; ++o)
      for (int32_t m = 0; m < P.M; ++m) drows.push_back(G[di].d_row[o] + m);
    ok = ok && !overlap(need, drows);
    if (!ok) continue;
    LGroup f = G[di];
    f.type = OP_PES_FUSED;
    f.act_row = P.x_row;
    f.e_row = P.e_row;
    f.coef = P.coef;
    f.ops.insert(f.ops.end(), P.ops.begin(), P.ops.end());
    G[di] = std::move(f);
    G.erase(G.begin() + pi);
    --pi;
  }
}

}  // namespace

LaunchPlan make_launch_plan(const Plan& p) {
  LaunchPlan lp;
  lp.step = merge_ens_groups(p.lowered);
  if (p.opts.fuse_synapse) {
    filters_last(p, lp.step);
    split_pulls(p, lp.step);
    Fuser f(p, lp.step);
    std::vector<LGroup> out;
    if (f.run(out, lp.prologue)) {
      lp.step = std::move(out);
      lp.has_prologue = lp.prologue.rows > 0;
    } else {
      lp.why = f.why;
    }
  }
  fuse_pes(p, lp.step);
  return lp;
}

}  // namespace ms
