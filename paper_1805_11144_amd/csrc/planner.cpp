// Graph optimisations of the paper's Sec. 4.2: operator merging, planning
// (greedy or bounded breadth-first tree search), signal/operator sorting
// (Alg. 1 meta-block sorting, Alg. 2 signal/operator sorting) and the final
// layout of signals in base arrays, followed by the lowering of every merged
// group to index arrays the GPU kernels consume.
//
// Readings where the paper leaves details open:
//  * dependencies: for every signal, the operators that set it run before those
//    that increment it, which run before those that read it, which run before
//    those that update it (Sec. 4.1.1: readers see a signal after all writes)
//  * merge key: operator type, base array of every operand, and for DotInc the
//    weight shape (M, K); neuron and filter parameters become per-row arrays
//  * candidates of one planning step: for each key, all ready operators with
//    that key; a plan's value is the number of operators it schedules in n
//    steps, and among equal counts the plan that finishes in fewer steps (so
//    an unbounded search returns a shortest plan); remaining ties prefer the
//    larger first group, then the lower key id (key ids in order of first
//    appearance in the operator list)
//  * read blocks: signals read by one group in one operand slot; block size =
//    total elements; ties go to the lower id.  Alg. 1 ranks the candidate
//    meta-blocks by the four criteria of Sec. 4.2.3 (a criterion no candidate
//    meets does not separate them), then by the lowest id.  Alg. 2 sorts
//    operators by (position of the read signal, slice start), permutes
//    signals only inside their meta-block, and makes at most 10 passes.
#include <algorithm>
#include <array>
#include <climits>
#include <cstring>
#include <numeric>
#include <set>
#include <tuple>

#include "host.hpp"

namespace ms {

const char* op_type_name(int32_t t) {
  static const char* n[] = {"Feed", "Reset", "Copy", "CopyInc", "ElementwiseInc",
                            "DotInc", "SimLIF", "SimLIFRate", "Lowpass", "Ensemble",
                            "SynapseScatter", "LearnedDotInc", "PES", "PESDecodeUpdate"};
  return (t >= 0 && t < OP_NTYPES) ? n[t] : "?";
}

namespace {

// Signals an operator reads, in slot order (the slots used for read blocks).
std::vector<SRef> read_slots(const Op& o) {
  switch (o.type) {
    case OP_COPY:
    case OP_COPY_INC: return {o.src};
    case OP_ELEM_INC:
    case OP_DOT_INC: return {o.a, o.src};
    case OP_LIF: return {o.src, o.V, o.ref};
    case OP_LIF_RATE: return {o.src};
    case OP_LOWPASS: return {o.src, o.dst};
    case OP_BDOT_INC: return {o.a, o.src};
    case OP_PES: return {o.src, o.a, o.dst};
    case OP_ENS: {
      std::vector<SRef> r;
      if (o.src.sig >= 0) { r.push_back(o.src); r.push_back(o.a); }
      r.push_back(o.bias);
      if (o.V.sig >= 0) { r.push_back(o.V); r.push_back(o.ref); }
      for (const auto& d : o.decs) r.push_back(d.first);
      return r;
    }
    default: return {};
  }
}

// sets / incs / reads / updates of batched signals
void access(const Op& o, std::vector<int32_t>& sets, std::vector<int32_t>& incs,
            std::vector<int32_t>& reads, std::vector<int32_t>& upds) {
  sets.clear(); incs.clear(); reads.clear(); upds.clear();
  switch (o.type) {
    case OP_FEED:
    case OP_RESET: sets.push_back(o.dst.sig); break;
    case OP_COPY: sets.push_back(o.dst.sig); reads.push_back(o.src.sig); break;
    case OP_COPY_INC: incs.push_back(o.dst.sig); reads.push_back(o.src.sig); break;
    case OP_ELEM_INC:
    case OP_DOT_INC: incs.push_back(o.dst.sig); reads.push_back(o.a.sig); reads.push_back(o.src.sig); break;
    case OP_LIF: reads.push_back(o.src.sig); sets.push_back(o.dst.sig);
      upds.push_back(o.V.sig); upds.push_back(o.ref.sig); break;
    case OP_LIF_RATE: reads.push_back(o.src.sig); sets.push_back(o.dst.sig); break;
    case OP_LOWPASS: reads.push_back(o.src.sig); upds.push_back(o.dst.sig); break;
    case OP_BDOT_INC: incs.push_back(o.dst.sig); reads.push_back(o.a.sig); reads.push_back(o.src.sig); break;
    case OP_PES: reads.push_back(o.src.sig); reads.push_back(o.a.sig); upds.push_back(o.dst.sig); break;
    case OP_ENS:
      if (o.src.sig >= 0) reads.push_back(o.src.sig);
      if (o.dst.sig >= 0) sets.push_back(o.dst.sig);
      for (const auto& d : o.decs) sets.push_back(d.second.sig);
      if (o.V.sig >= 0) { upds.push_back(o.V.sig); upds.push_back(o.ref.sig); }
      break;
    default: break;
  }
}

std::vector<int32_t> merge_key(const IR& ir, const Op& o) {
  auto b = [&](const SRef& r) { return r.sig >= 0 ? ir.sigs[r.sig].base : -1; };
  switch (o.type) {
    case OP_FEED: return {OP_FEED};
    case OP_RESET: return {OP_RESET, b(o.dst)};
    case OP_COPY:
    case OP_COPY_INC: return {o.type, b(o.dst), b(o.src)};
    case OP_ELEM_INC: return {OP_ELEM_INC, b(o.dst), b(o.a), b(o.src)};
    case OP_DOT_INC: return {OP_DOT_INC, b(o.dst), b(o.a), b(o.src), o.a.len, o.src.len};
    case OP_LIF: return {OP_LIF, b(o.src), b(o.dst), b(o.V), b(o.ref)};
    case OP_LIF_RATE: return {OP_LIF_RATE, b(o.src), b(o.dst), o.ntype};   // rate curve: LIF or ReLU
    case OP_LOWPASS: return {OP_LOWPASS, b(o.dst), b(o.src)};
    case OP_BDOT_INC: return {OP_BDOT_INC, b(o.dst), b(o.a), b(o.src), o.dst.len, o.src.len};
    case OP_PES: return {OP_PES, b(o.dst), b(o.src), b(o.a), o.a.len, o.src.len};
    case OP_ENS: {
      std::vector<int32_t> k = {OP_ENS, o.ntype, b(o.src), b(o.a), o.src.len, b(o.bias),
                                b(o.dst), b(o.V), b(o.ref)};
      for (const auto& d : o.decs) { k.push_back(b(d.first)); k.push_back(d.second.len); k.push_back(b(d.second)); }
      return k;
    }
    default: return {o.type};
  }
}

struct Graph {
  std::vector<std::vector<int32_t>> succ;
  std::vector<int32_t> indeg;
};

Graph dependency_graph(const IR& ir) {
  const int32_t no = (int32_t)ir.ops.size();
  const int32_t ns = (int32_t)ir.sigs.size();
  std::vector<std::array<std::vector<int32_t>, 4>> layers(ns);
  std::vector<int32_t> s, i, r, u;
  for (int32_t k = 0; k < no; ++k) {
    access(ir.ops[k], s, i, r, u);
    const std::vector<int32_t>* L[4] = {&s, &i, &r, &u};
    for (int l = 0; l < 4; ++l)
      for (int32_t sig : *L[l])
        if (ir.sigs[sig].cls == SC_BATCHED) {
          auto& v = layers[sig][l];
          if (v.empty() || v.back() != k) v.push_back(k);
        }
  }
  Graph g;
  g.succ.assign(no, {});
  g.indeg.assign(no, 0);
  for (int32_t sig = 0; sig < ns; ++sig) {
    if (layers[sig][0].size() > 1)
      fail(MS_E_INVALID, "signal " + ir.sigs[sig].name + " is set by more than one operator");
    const std::vector<int32_t>* prev = nullptr;
    for (int l = 0; l < 4; ++l) {
      const auto& cur = layers[sig][l];
      if (cur.empty()) continue;
      if (prev)
        for (int32_t a : *prev)
          for (int32_t bb : cur)
            if (a != bb) { g.succ[a].push_back(bb); g.indeg[bb]++; }
      prev = &cur;
    }
  }
  // cycle check (Kahn)
  std::vector<int32_t> deg = g.indeg, q;
  for (int32_t k = 0; k < no; ++k) if (deg[k] == 0) q.push_back(k);
  size_t seen = 0;
  while (seen < q.size()) {
    int32_t k = q[seen++];
    for (int32_t t : g.succ[k]) if (--deg[t] == 0) q.push_back(t);
  }
  if ((int32_t)q.size() != no)
    fail(MS_E_CYCLE, "the operator graph has a cycle (a loop of connections without a synapse)");
  return g;
}

// ------------------------------------------------------------------ planner
struct PlanSearch {
  const Graph& g;
  const std::vector<int32_t>& key;
  std::vector<int32_t> indeg;
  std::vector<std::vector<int32_t>> ready;   // per key

  PlanSearch(const Graph& gg, const std::vector<int32_t>& k, int32_t nkeys)
      : g(gg), key(k), indeg(gg.indeg), ready(nkeys) {
    for (int32_t o = 0; o < (int32_t)indeg.size(); ++o)
      if (indeg[o] == 0) ready[key[o]].push_back(o);
  }

  // schedule every ready op of key k; returns the scheduled list
  std::vector<int32_t> apply(int32_t k) {
    std::vector<int32_t> L;
    L.swap(ready[k]);
    for (int32_t o : L)
      for (int32_t t : g.succ[o])
        if (--indeg[t] == 0) ready[key[t]].push_back(t);
    return L;
  }
  void undo(int32_t k, std::vector<int32_t>& L) {
    for (auto it = L.rbegin(); it != L.rend(); ++it) {
      const auto& sc = g.succ[*it];
      for (auto jt = sc.rbegin(); jt != sc.rend(); ++jt) {
        int32_t t = *jt;
        if (indeg[t] == 0) ready[key[t]].pop_back();
        ++indeg[t];
      }
    }
    ready[k].swap(L);
  }

  // Best (operators scheduled, steps used) over all plans of at most `depth`
  // steps from the current state: more operators first, then fewer steps
  // (a plan that finishes everything early beats one that needs the horizon).
  struct Val {
    int64_t ops = 0, steps = 0;
    bool better(const Val& o) const { return ops != o.ops ? ops > o.ops : steps < o.steps; }
  };
  Val best(int depth) {
    Val v;
    if (depth <= 0) return v;
    for (int32_t k = 0; k < (int32_t)ready.size(); ++k) {
      const int64_t sz = (int64_t)ready[k].size();
      if (!sz) continue;
      Val cand;
      if (depth == 1) {
        cand = Val{sz, 1};
      } else {
        auto L = apply(k);
        Val rest = best(depth - 1);
        undo(k, L);
        cand = Val{sz + rest.ops, 1 + rest.steps};
      }
      if (cand.better(v) || v.steps == 0) v = cand;
    }
    return v;
  }
};

}  // namespace

std::vector<std::vector<int32_t>> plan_groups(const IR& ir, const std::vector<int32_t>& key,
                                              int32_t n_keys, const PlanOpts& o) {
  Graph g = dependency_graph(ir);
  PlanSearch ps(g, key, n_keys);
  const int depth = (o.planner == MS_PLANNER_GREEDY || !o.merge) ? 1 : std::max(1, o.depth);
  std::vector<std::vector<int32_t>> groups;
  size_t done = 0;
  while (done < ir.ops.size()) {
    int32_t best_k = -1;
    PlanSearch::Val best_v;
    int64_t best_sz = -1;
    for (int32_t k = 0; k < n_keys; ++k) {
      const int64_t sz = (int64_t)ps.ready[k].size();
      if (!sz) continue;
      PlanSearch::Val v{sz, 1};
      if (depth > 1) {
        auto L = ps.apply(k);
        PlanSearch::Val rest = ps.best(depth - 1);
        ps.undo(k, L);
        v = PlanSearch::Val{sz + rest.ops, 1 + rest.steps};
      }
      if (best_k < 0 || v.better(best_v) || (!best_v.better(v) && sz > best_sz)) {
        best_v = v; best_sz = sz; best_k = k;
      }
    }
    if (best_k < 0) fail(MS_E_CYCLE, "planner stalled (cycle)");
    auto L = ps.apply(best_k);
    std::sort(L.begin(), L.end());
    done += L.size();
    groups.push_back(std::move(L));
  }
  return groups;
}

namespace {

// ------------------------------------------------------------------ sorting
struct Block {
  int32_t group, slot, base;
  int64_t size = 0;
  std::vector<int32_t> sigs;          // distinct, first-occurrence order
};

struct SortState {
  std::vector<std::vector<int32_t>> order;   // per base: signal ids
  std::vector<int32_t> pos;                  // per signal: position in its base
  void reindex(int32_t base) {
    const auto& v = order[base];
    for (int32_t i = 0; i < (int32_t)v.size(); ++i) pos[v[i]] = i;
  }
};

void sort_plan(const IR& ir, std::vector<std::vector<int32_t>>& groups, SortState& st) {
  const int32_t ns = (int32_t)ir.sigs.size(), nb = (int32_t)ir.bases.size();
  // read blocks
  std::vector<Block> blocks;
  std::vector<std::vector<int32_t>> group_blocks(groups.size());
  for (int32_t gi = 0; gi < (int32_t)groups.size(); ++gi) {
    const Op& first = ir.ops[groups[gi][0]];
    const size_t nslots = read_slots(first).size();
    for (size_t sl = 0; sl < nslots; ++sl) {
      Block b;
      b.group = gi; b.slot = (int32_t)sl;
      std::set<int32_t> seen;
      for (int32_t oi : groups[gi]) {
        int32_t sig = read_slots(ir.ops[oi])[sl].sig;
        if (seen.insert(sig).second) {
          b.sigs.push_back(sig);
          b.size += (int64_t)ir.sigs[sig].rows * ir.sigs[sig].cols;
        }
      }
      b.base = ir.sigs[b.sigs[0]].base;
      group_blocks[gi].push_back((int32_t)blocks.size());
      blocks.push_back(std::move(b));
    }
  }
  const int32_t nblk = (int32_t)blocks.size();
  // membership of each signal
  std::vector<std::vector<int32_t>> member(ns);
  for (int32_t bi = 0; bi < nblk; ++bi)
    for (int32_t sig : blocks[bi].sigs) member[sig].push_back(bi);
  // meta-blocks per base, first appearance in canonical signal order
  std::map<std::pair<int32_t, std::vector<int32_t>>, int32_t> meta_id;
  std::vector<std::vector<int32_t>> meta_sigs, meta_set;
  std::vector<int32_t> meta_base;
  std::vector<int32_t> meta_of(ns, -1);
  for (int32_t sig = 0; sig < ns; ++sig) {
    auto k = std::make_pair(ir.sigs[sig].base, member[sig]);
    auto it = meta_id.find(k);
    int32_t id;
    if (it == meta_id.end()) {
      id = (int32_t)meta_sigs.size();
      meta_id[k] = id;
      meta_sigs.push_back({});
      meta_set.push_back(member[sig]);
      meta_base.push_back(ir.sigs[sig].base);
    } else {
      id = it->second;
    }
    meta_sigs[id].push_back(sig);
    meta_of[sig] = id;
  }
  auto larger_first = [&](int32_t x, int32_t y) {   // read blocks: size desc, id asc
    if (blocks[x].size != blocks[y].size) return blocks[x].size > blocks[y].size;
    return x < y;
  };
  auto holds = [&](int32_t m, int32_t blk) {
    return std::binary_search(meta_set[m].begin(), meta_set[m].end(), blk);
  };

  // ---- meta-block layout (Alg. 1), per base array.  Meta-blocks are placed
  // one after another; the next is the remaining one that best matches the
  // last placed, ranked by the four criteria of Sec. 4.2.3 in order of
  // precedence: holds the active read block; holds every read block of the
  // last; smallest Hamming distance to the last; holds the last's read blocks,
  // the larger the better (block by block, largest first); then lowest id.
  // The active block is the largest at first; once no remaining meta-block
  // holds it, the largest block of the last placed takes over for later
  // choices.
  st.order.assign(nb, {});
  st.pos.assign(ns, -1);
  for (int32_t base = 0; base < nb; ++base) {
    std::vector<int32_t> left;
    for (int32_t m = 0; m < (int32_t)meta_sigs.size(); ++m) if (meta_base[m] == base) left.push_back(m);
    std::vector<int32_t> base_blocks;
    for (int32_t bi = 0; bi < nblk; ++bi) if (blocks[bi].base == base) base_blocks.push_back(bi);
    std::vector<int32_t> placed;
    if (base_blocks.empty()) {
      placed = left;
    } else {
      int32_t active = *std::min_element(base_blocks.begin(), base_blocks.end(), larger_first);
      int32_t last = -1;   // before anything is placed: a meta-block holding the active block
      for (int32_t m : left) if (holds(m, active)) { last = m; break; }
      while (!left.empty()) {
        bool active_left = false;
        for (int32_t m : left) active_left = active_left || holds(m, active);
        std::vector<int32_t> last_blocks = meta_set[last];
        std::sort(last_blocks.begin(), last_blocks.end(), larger_first);
        // rank key: criteria 1-4 as small integers, then the id
        auto key = [&](int32_t m) {
          std::vector<int64_t> k;
          k.push_back(active_left && !holds(m, active) ? 1 : 0);
          k.push_back(std::includes(meta_set[m].begin(), meta_set[m].end(), meta_set[last].begin(),
                                    meta_set[last].end()) ? 0 : 1);
          std::vector<int32_t> diff;
          std::set_symmetric_difference(meta_set[m].begin(), meta_set[m].end(), meta_set[last].begin(),
                                        meta_set[last].end(), std::back_inserter(diff));
          k.push_back((int64_t)diff.size());
          for (int32_t blk : last_blocks) k.push_back(holds(m, blk) ? 0 : 1);
          k.push_back(m);
          return k;
        };
        int32_t best = left[0];
        std::vector<int64_t> best_key = key(best);
        for (size_t i = 1; i < left.size(); ++i) {
          std::vector<int64_t> k = key(left[i]);
          if (k < best_key) { best_key.swap(k); best = left[i]; }
        }
        if (!active_left && !last_blocks.empty()) active = last_blocks[0];
        left.erase(std::find(left.begin(), left.end(), best));
        placed.push_back(best);
        last = best;
      }
    }
    for (int32_t m : placed)
      for (int32_t sig : meta_sigs[m]) st.order[base].push_back(sig);
    st.reindex(base);
  }

  // ---- operators and signals inside meta-blocks (Alg. 2).  For one read
  // block: its group's operators take the order in which the block's signals
  // lie in memory; then every read block of that group has its signals
  // rearranged into the new operator order, each meta-block within its own
  // positions (the meta-block layout stays).  Blocks are visited smallest
  // first so that larger blocks settle last; passes repeat until one changes
  // nothing, at most 10.
  std::vector<int32_t> visit(nblk);
  std::iota(visit.begin(), visit.end(), 0);
  std::stable_sort(visit.begin(), visit.end(), [&](int32_t x, int32_t y) { return blocks[x].size < blocks[y].size; });
  std::vector<std::vector<int32_t>> metas_of(nblk);
  for (int32_t m = 0; m < (int32_t)meta_sigs.size(); ++m)
    for (int32_t bi : meta_set[m]) metas_of[bi].push_back(m);
  auto read_of = [&](int32_t op, int32_t slot) { return read_slots(ir.ops[op])[slot]; };
  auto ops_follow_layout = [&](const Block& b) {
    std::vector<int32_t>& ops = groups[b.group];
    std::stable_sort(ops.begin(), ops.end(), [&](int32_t x, int32_t y) {
      const SRef rx = read_of(x, b.slot), ry = read_of(y, b.slot);
      return std::make_pair(st.pos[rx.sig], rx.start) < std::make_pair(st.pos[ry.sig], ry.start);
    });
  };
  auto signals_follow_ops = [&](int32_t bi) {
    const Block& c = blocks[bi];
    std::map<int32_t, int32_t> rank;   // signal -> first operator (in group order) reading it
    for (int32_t op : groups[c.group]) rank.emplace(read_of(op, c.slot).sig, (int32_t)rank.size());
    for (int32_t m : metas_of[bi]) {
      std::vector<int32_t> spots, sigs = meta_sigs[m];
      for (int32_t sig : sigs) spots.push_back(st.pos[sig]);
      std::sort(spots.begin(), spots.end());
      std::sort(sigs.begin(), sigs.end(), [&](int32_t x, int32_t y) { return rank.at(x) < rank.at(y); });
      for (size_t i = 0; i < spots.size(); ++i) {
        st.order[c.base][spots[i]] = sigs[i];
        st.pos[sigs[i]] = spots[i];
      }
    }
  };
  for (int pass = 0; pass < 10; ++pass) {
    const auto groups_before = groups;
    const auto order_before = st.order;
    for (int32_t bi : visit) {
      ops_follow_layout(blocks[bi]);
      for (int32_t other : group_blocks[blocks[bi].group]) signals_follow_ops(other);
    }
    if (groups == groups_before && st.order == order_before) break;
  }
}

// ----------------------------------------------------------------- lowering
LOperand make_operand(int32_t base, const std::vector<int32_t>& rows) {
  LOperand o;
  o.base = base;
  bool contig = true;
  for (size_t i = 1; i < rows.size(); ++i)
    if (rows[i] != rows[0] + (int32_t)i) { contig = false; break; }
  if (contig) {
    o.start = rows.empty() ? 0 : rows[0];
  } else {
    o.idx = rows;
  }
  return o;
}

template <class T>
std::vector<float> uniform_or_rows(const std::vector<T>& v) {
  bool uni = true;
  for (size_t i = 1; i < v.size(); ++i) if ((float)v[i] != (float)v[0]) { uni = false; break; }
  std::vector<float> out;
  if (uni && !v.empty()) out.push_back((float)v[0]);
  else for (const T& x : v) out.push_back((float)x);
  return out;
}

// Lowers the operators `ops` of one merged group to row lists, with signal rows
// taken from `sig_offset` (row of each signal's first element in its base).
LGroup lower_group_at(const IR& ir, const std::vector<int64_t>& sig_offset, const std::vector<int32_t>& ops) {
  LGroup g;
  g.type = ir.ops[ops[0]].type;
  g.ops = ops;
  auto row = [&](const SRef& r, int32_t i) { return (int32_t)(sig_offset[r.sig] + r.start + i); };
  auto base = [&](const SRef& r) { return ir.sigs[r.sig].base; };
  const Op& f = ir.ops[ops[0]];
  switch (g.type) {
    case OP_FEED: {
      std::vector<int32_t> d, fr;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        for (int32_t i = 0; i < o.dst.len; ++i) {
          d.push_back(row(o.dst, i));
          fr.push_back(ir.feed_row_of_node[o.node] + i);
        }
      }
      g.rows = (int64_t)d.size();
      g.dst = make_operand(base(f.dst), d);
      g.feed_rows = fr;
      break;
    }
    case OP_RESET: {
      std::vector<int32_t> d;
      std::vector<double> val;
      bool any = false;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        for (int32_t i = 0; i < o.dst.len; ++i) {
          d.push_back(row(o.dst, i));
          double v = o.reset_value.empty() ? 0.0 : o.reset_value[i];
          any |= v != 0.0;
          val.push_back(v);
        }
      }
      g.rows = (int64_t)d.size();
      g.dst = make_operand(base(f.dst), d);
      if (any) for (double v : val) g.values.push_back((float)v);
      break;
    }
    case OP_COPY: {
      std::vector<int32_t> d, s;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        for (int32_t i = 0; i < o.dst.len; ++i) { d.push_back(row(o.dst, i)); s.push_back(row(o.src, i)); }
      }
      g.rows = (int64_t)d.size();
      g.dst = make_operand(base(f.dst), d);
      g.src = make_operand(base(f.src), s);
      break;
    }
    case OP_COPY_INC:
    case OP_ELEM_INC: {
      // entries in operator order; grouped by destination (first appearance)
      std::vector<int32_t> ed, es, ea;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        for (int32_t i = 0; i < o.dst.len; ++i) {
          ed.push_back(row(o.dst, i));
          es.push_back(row(o.src, i));
          if (g.type == OP_ELEM_INC) ea.push_back(row(o.a, o.a.len == 1 ? 0 : i));
        }
      }
      std::vector<int32_t> uniq;
      std::map<int32_t, int32_t> uid;
      std::vector<std::vector<int32_t>> ent;
      for (int32_t e = 0; e < (int32_t)ed.size(); ++e) {
        auto it = uid.find(ed[e]);
        int32_t u;
        if (it == uid.end()) { u = (int32_t)uniq.size(); uid[ed[e]] = u; uniq.push_back(ed[e]); ent.push_back({}); }
        else u = it->second;
        ent[u].push_back(e);
      }
      std::vector<int32_t> s2, a2;
      g.ptr.push_back(0);
      for (size_t u = 0; u < uniq.size(); ++u) {
        for (int32_t e : ent[u]) { s2.push_back(es[e]); if (!ea.empty()) a2.push_back(ea[e]); }
        g.ptr.push_back((int32_t)s2.size());
      }
      if (uniq.size() == ed.size()) g.ptr.clear();   // no repeated destination
      g.rows = (int64_t)uniq.size();
      g.dst = make_operand(base(f.dst), uniq);
      g.src = make_operand(base(f.src), s2);
      if (g.type == OP_ELEM_INC) g.a = make_operand(base(f.a), a2);
      break;
    }
    case OP_DOT_INC: {
      g.M = f.a.len;
      g.K = f.src.len;
      std::set<int32_t> dsts;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        g.w_row.push_back((int32_t)sig_offset[o.a.sig] + o.a.start);
        g.x_row.push_back(row(o.src, 0));
        g.d_row.push_back(row(o.dst, 0));
        if (!dsts.insert(o.dst.sig).second) fail(MS_E_INVALID, "DotInc group with repeated destination");
      }
      g.rows = (int64_t)ops.size();
      g.a.base = base(f.a);
      g.src.base = base(f.src);
      g.dst.base = base(f.dst);
      break;
    }
    case OP_LIF:
    case OP_LIF_RATE: {
      std::vector<int32_t> J, s, V, R;
      std::vector<double> trc, tref, amp, sig;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        for (int32_t i = 0; i < o.src.len; ++i) {
          J.push_back(row(o.src, i));
          s.push_back(row(o.dst, i));
          if (g.type == OP_LIF) { V.push_back(row(o.V, i)); R.push_back(row(o.ref, i)); }
          if (g.type == OP_LIF_RATE) g.ens_type = o.ntype;   // same in every op of the group (key)
          trc.push_back(o.tau_rc); tref.push_back(o.tau_ref); amp.push_back(o.amp); sig.push_back(o.sigma);
        }
      }
      if (g.type == OP_LIF_RATE && g.ens_type == MS_NEURON_SOFTLIF_RATE) g.sigma = uniform_or_rows(sig);
      g.rows = (int64_t)J.size();
      g.src = make_operand(base(f.src), J);
      g.dst = make_operand(base(f.dst), s);
      if (g.type == OP_LIF) { g.V = make_operand(base(f.V), V); g.ref = make_operand(base(f.ref), R); }
      g.tau_rc = uniform_or_rows(trc);
      g.tau_ref = uniform_or_rows(tref);
      g.amp = uniform_or_rows(amp);
      break;
    }
    case OP_LOWPASS: {
      std::vector<int32_t> y, v;
      std::vector<double> ca, cb;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        for (int32_t i = 0; i < o.dst.len; ++i) {
          y.push_back(row(o.dst, i)); v.push_back(row(o.src, i));
          ca.push_back(o.coef_a); cb.push_back(o.coef_b);
        }
      }
      g.rows = (int64_t)y.size();
      g.dst = make_operand(base(f.dst), y);
      g.src = make_operand(base(f.src), v);
      g.ca = uniform_or_rows(ca);
      g.cb = uniform_or_rows(cb);
      break;
    }
    case OP_BDOT_INC:
    case OP_PES: {
      // per op: decoders, activities, outputs (BDOT_INC) or error (PES)
      g.M = g.type == OP_BDOT_INC ? f.dst.len : f.a.len;
      g.K = f.src.len;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        if (g.type == OP_BDOT_INC) {
          g.w_row.push_back(row(o.a, 0));
          g.d_row.push_back(row(o.dst, 0));
        } else {
          g.w_row.push_back(row(o.dst, 0));
          g.e_row.push_back(row(o.a, 0));
          g.coef.push_back((float)o.coef_a);
        }
        g.x_row.push_back(row(o.src, 0));
      }
      g.rows = (int64_t)ops.size();
      g.dst.base = base(f.dst);
      g.src.base = base(f.src);
      g.a.base = base(f.a);
      break;
    }
    case OP_ENS: {
      g.rows = (int64_t)ops.size();
      g.ens_type = f.ntype;
      g.ens_d = f.src.sig >= 0 ? f.src.len : 0;
      for (const auto& d : f.decs) g.ens_df.push_back(d.second.len);
      g.ens_D.assign(f.decs.size(), {});
      g.ens_dd.assign(f.decs.size(), {});
      std::vector<double> trc, tref, amp;
      for (int32_t oi : ops) {
        const Op& o = ir.ops[oi];
        g.ens_n.push_back(o.n);
        g.ens_x.push_back(o.src.sig >= 0 ? row(o.src, 0) : -1);
        g.ens_enc.push_back(o.a.sig >= 0 ? (int32_t)sig_offset[o.a.sig] : -1);
        g.ens_bias.push_back(row(o.bias, 0));
        g.ens_V.push_back(o.V.sig >= 0 ? row(o.V, 0) : -1);
        g.ens_ref.push_back(o.ref.sig >= 0 ? row(o.ref, 0) : -1);
        g.ens_s.push_back(o.dst.sig >= 0 ? row(o.dst, 0) : -1);
        for (size_t k = 0; k < o.decs.size(); ++k) {
          g.ens_D[k].push_back((int32_t)sig_offset[o.decs[k].first.sig]);
          g.ens_dd[k].push_back(row(o.decs[k].second, 0));
        }
        trc.push_back(o.tau_rc); tref.push_back(o.tau_ref); amp.push_back(o.amp);
      }
      // operand bases for the runtime
      g.src.base = f.src.sig >= 0 ? base(f.src) : -1;
      g.a.base = f.a.sig >= 0 ? base(f.a) : -1;
      g.ens_bias_base = base(f.bias);
      g.tau_rc = uniform_or_rows(trc);
      g.tau_ref = uniform_or_rows(tref);
      g.amp = uniform_or_rows(amp);
      for (const auto& d : f.decs) g.ens_Dbase.push_back(base(d.first));
      break;
    }
    default: fail(MS_E_INVALID, "cannot lower operator type");
  }
  return g;
}

LGroup lower_group(const Plan& p, const std::vector<int32_t>& ops) { return lower_group_at(p.ir, p.sig_offset, ops); }

}  // namespace

// The connection chain of Fig. 2 in front of an ensemble -- a transform
// DotInc of a value d into v (reset to zero), the lowpass y <- a y + b v, and
// the Copy of y (the previous step's, as filters are read) into the
// ensemble's input x (reset to zero) -- fuses into the ensemble's window phase
// when each of v, y and x has no other reader or writer and no probe, the
// three operators are alone in their phases, the transform has constant
// weights with K, M <= 16, the lowpass a nonzero input gain b, and the
// ensemble takes one batch column per
// workgroup and one neuron per thread (more than 128 neurons, or minibatch 1;
// no ensemble of its phase above 512 neurons).  The ensemble kernel
// then computes x_t = y_{t-1}, y_t = a y_{t-1} + b W d_t itself, and writes
// only y's last step (the value the next window starts from); the three
// phases and the resets of v and x go.
static void fuse_window_chains(const Plan& p, WindowPlan& w, const std::vector<std::vector<int32_t>>& S,
                        const std::vector<std::vector<int32_t>>& I, const std::vector<std::vector<int32_t>>& R,
                        const std::vector<std::vector<int32_t>>& U) {
  const IR& ir = p.ir;
  const int32_t ns = (int32_t)ir.sigs.size();
  std::vector<char> probed(ns, 0);
  for (const auto& pr : ir.probes) probed[pr.src.sig] = 1;
  std::map<int32_t, int32_t> phase_of;
  for (size_t k = 0; k < w.phases.size(); ++k)
    for (int32_t op : w.phases[k].g.ops) phase_of[op] = (int32_t)k;
  auto whole = [&](const SRef& r) { return r.sig >= 0 && r.start == 0 && r.len == ir.sigs[r.sig].rows; };
  auto zero_reset_only = [&](int32_t sg) {
    if (S[sg].size() != 1) return false;
    const Op& o = ir.ops[S[sg][0]];
    if (o.type != OP_RESET || !whole(o.dst)) return false;
    for (double v : o.reset_value) if (v != 0.0) return false;
    return true;
  };
  auto alone = [&](int32_t op, int32_t blk) {
    auto it = phase_of.find(op);
    return it != phase_of.end() && w.phases[it->second].g.ops.size() == 1 && w.phases[it->second].src_blk == blk;
  };
  std::vector<char> drop_phase(w.phases.size(), 0);
  std::set<int64_t> drop_rows;   // window rows of v and x whose resets go
  for (int32_t e = 0; e < (int32_t)ir.ops.size(); ++e) {
    const Op& E = ir.ops[e];
    if (E.type != OP_ENS || E.src.sig < 0 || !whole(E.src)) continue;
    if (!(E.n > 128 || p.opts.minibatch == 1)) continue;
    const int32_t X = E.src.sig;
    if (!zero_reset_only(X) || I[X].size() != 1 || R[X] != std::vector<int32_t>{e} || !U[X].empty() || probed[X])
      continue;
    const int32_t c = I[X][0];
    const Op& C = ir.ops[c];
    if (C.type != OP_COPY_INC || !whole(C.dst) || !whole(C.src)) continue;
    const int32_t Y = C.src.sig;
    if (U[Y].size() != 1 || R[Y] != std::vector<int32_t>{c} || !S[Y].empty() || !I[Y].empty() || probed[Y]) continue;
    const int32_t f = U[Y][0];
    const Op& F = ir.ops[f];
    if (F.type != OP_LOWPASS || !whole(F.dst) || !whole(F.src)) continue;
    const int32_t V = F.src.sig;
    if (!zero_reset_only(V) || I[V].size() != 1 || R[V] != std::vector<int32_t>{f} || !U[V].empty() || probed[V])
      continue;
    const int32_t dd = I[V][0];
    const Op& D = ir.ops[dd];
    if (D.type != OP_DOT_INC || !whole(D.dst) || ir.sigs[D.a.sig].cls == SC_BATCHED ||
        ir.sigs[D.src.sig].cls != SC_BATCHED || w.priv[D.src.sig])
      continue;
    const int32_t M = D.dst.len, K = D.src.len;
    if (M > 16 || K > 16 || M != E.src.len) continue;
    if (!alone(dd, 1) || !alone(f, 1) || !alone(c, 0)) continue;
    if ((float)F.coef_b == 0.0f) continue;   // the kernel's unrolled filter divides by b
    auto ph = phase_of.find(e);
    if (ph == phase_of.end()) continue;
    LGroup& G = w.phases[ph->second].g;
    // the fused launch runs one column per workgroup and one neuron per thread
    if (*std::max_element(G.ens_n.begin(), G.ens_n.end()) > 512) continue;
    const int32_t wb = ir.sigs[D.a.sig].base;
    if (G.ens_chain_wbase >= 0 && G.ens_chain_wbase != wb) continue;
    const size_t k = (size_t)(std::find(G.ops.begin(), G.ops.end(), e) - G.ops.begin());
    if (G.ens_chain.empty()) G.ens_chain.assign(G.ops.size() * kChainInts, 0);
    int32_t* r = &G.ens_chain[k * kChainInts];
    r[0] = (int32_t)(w.sig_row[D.src.sig] + D.src.start);
    r[1] = K;
    r[2] = (int32_t)(p.sig_offset[D.a.sig] + D.a.start);
    r[3] = (int32_t)w.sig_row[Y];
    r[4] = M;
    r[5] = 0;
    const float a = (float)F.coef_a, b = (float)F.coef_b;
    std::memcpy(&r[6], &a, 4);
    std::memcpy(&r[7], &b, 4);
    G.ens_chain_wbase = wb;
    drop_phase[phase_of[dd]] = drop_phase[phase_of[f]] = drop_phase[phase_of[c]] = 1;
    for (int32_t i = 0; i < ir.sigs[V].rows; ++i) drop_rows.insert(w.sig_row[V] + i);
    for (int32_t i = 0; i < ir.sigs[X].rows; ++i) drop_rows.insert(w.sig_row[X] + i);
  }
  if (drop_rows.empty()) return;
  std::vector<WPhase> kept;
  for (size_t k = 0; k < w.phases.size(); ++k) {
    if (drop_phase[k]) continue;
    WPhase ph = w.phases[k];
    if (ph.g.type == OP_RESET) {
      std::vector<int32_t> rows;
      std::vector<float> vals;
      for (int64_t r = 0; r < ph.g.rows; ++r) {
        const int64_t x = ph.g.dst.idx.empty() ? ph.g.dst.start + r : ph.g.dst.idx[r];
        if (drop_rows.count(x)) continue;
        rows.push_back((int32_t)x);
        if (!ph.g.values.empty()) vals.push_back(ph.g.values[r]);
      }
      if (rows.empty()) continue;
      if ((int64_t)rows.size() != ph.g.rows) {
        ph.g.rows = (int64_t)rows.size();
        ph.g.dst = make_operand(ph.g.dst.base, rows);
        ph.g.values = vals;
        std::vector<int32_t> ops;   // the resets that still have rows
        for (int32_t op : ph.g.ops)
          if (!drop_rows.count(w.sig_row[ir.ops[op].dst.sig] + ir.ops[op].dst.start)) ops.push_back(op);
        ph.g.ops = ops;
      }
    }
    kept.push_back(std::move(ph));
  }
  w.phases.swap(kept);
}

// Stage-major schedule.  Per batched signal: the operators that set it run
// before those that increment it, which run before those that read it (all
// within a step); a signal that is updated (filter output) is read as the
// previous step's value, so its updater runs, for the whole window, before its
// readers.  Levels are longest paths in that graph; each level's operators run
// as the plan's merged groups restricted to the level.
WindowPlan make_window_plan(const Plan& p) {
  const IR& ir = p.ir;
  WindowPlan w;
  const int32_t no = (int32_t)ir.ops.size(), ns = (int32_t)ir.sigs.size();
  auto batched = [&](int32_t sg) { return sg >= 0 && ir.sigs[sg].cls == SC_BATCHED; };
  std::vector<std::vector<int32_t>> S(ns), I(ns), R(ns), U(ns);
  std::vector<int32_t> s_, i_, r_, u_;
  for (int32_t k = 0; k < no; ++k) {
    access(ir.ops[k], s_, i_, r_, u_);
    const std::vector<int32_t>* src[4] = {&s_, &i_, &r_, &u_};
    std::vector<std::vector<int32_t>>* dst[4] = {&S, &I, &R, &U};
    for (int l = 0; l < 4; ++l)
      for (int32_t sg : *src[l])
        if (batched(sg)) {
          auto& v = (*dst[l])[sg];
          if (v.empty() || v.back() != k) v.push_back(k);
        }
  }
  w.priv.assign(ns, 0);
  for (const Op& o : ir.ops)
    if ((o.type == OP_LIF || o.type == OP_ENS) && o.V.sig >= 0) { w.priv[o.V.sig] = 1; w.priv[o.ref.sig] = 1; }
  auto refuse = [&](const std::string& why) { w.ok = false; w.why = why; return w; };
  for (const Op& o : ir.ops)
    if (o.type == OP_PES) return refuse("online learning changes the decoders every step (" + o.name + ")");
  for (int32_t sg = 0; sg < ns; ++sg) {
    if (!batched(sg)) continue;
    if (w.priv[sg]) {
      if (U[sg].size() != 1 || !S[sg].empty() || !I[sg].empty() || !R[sg].empty())
        return refuse("neuron state " + ir.sigs[sg].name + " is accessed by other operators");
      continue;
    }
    if (!U[sg].empty() && (!S[sg].empty() || !I[sg].empty() || U[sg].size() > 1))
      return refuse("signal " + ir.sigs[sg].name + " is both updated and written");
    if (U[sg].empty() && S[sg].empty() && !I[sg].empty())
      return refuse("signal " + ir.sigs[sg].name + " accumulates across steps");
  }
  for (const auto& pr : ir.probes)
    if (w.priv[pr.src.sig]) return refuse("a probe reads neuron state");
  // graph: ops, then three ordering points per signal (after set, after
  // increments, after update)
  const int32_t nn = no + 3 * ns;
  std::vector<std::vector<int32_t>> succ(nn);
  for (int32_t sg = 0; sg < ns; ++sg) {
    if (!batched(sg) || w.priv[sg]) continue;
    const int32_t AS = no + 3 * sg, AI = AS + 1, AU = AS + 2;
    for (int32_t k : S[sg]) succ[k].push_back(AS);
    succ[AS].push_back(AI);
    for (int32_t k : I[sg]) { succ[AS].push_back(k); succ[k].push_back(AI); }
    if (!U[sg].empty()) {
      for (int32_t k : U[sg]) succ[k].push_back(AU);
      for (int32_t k : R[sg]) if (k != U[sg][0]) succ[AU].push_back(k);
    } else {
      for (int32_t k : R[sg]) succ[AI].push_back(k);
    }
  }
  std::vector<int32_t> indeg(nn, 0), dist(nn, 0);
  for (int32_t u = 0; u < nn; ++u) for (int32_t v : succ[u]) indeg[v]++;
  std::vector<int32_t> q;
  for (int32_t u = 0; u < nn; ++u) if (indeg[u] == 0) q.push_back(u);
  size_t head = 0;
  while (head < q.size()) {
    const int32_t u = q[head++];
    const int32_t fin = dist[u] + (u < no ? 1 : 0);
    for (int32_t v : succ[u]) {
      dist[v] = std::max(dist[v], fin);
      if (--indeg[v] == 0) q.push_back(v);
    }
  }
  if ((int32_t)q.size() != nn) return refuse("a cycle through synapse updates (recurrent connections)");
  // window rows: batched signals in layout order, private ones in their own array
  w.sig_row = p.sig_offset;
  std::vector<int32_t> order;
  for (int32_t sg = 0; sg < ns; ++sg) if (batched(sg)) order.push_back(sg);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return p.sig_offset[a] < p.sig_offset[b]; });
  for (int32_t sg : order) {
    if (w.priv[sg]) { w.sig_row[sg] = w.rows_p; w.rows_p += ir.sigs[sg].rows; }
    else { w.sig_row[sg] = w.rows_v; w.rows_v += ir.sigs[sg].rows; }
  }
  // phases
  int32_t maxl = 0;
  for (int32_t k = 0; k < no; ++k) maxl = std::max(maxl, dist[k]);
  w.levels = no ? maxl + 1 : 0;
  auto blk = [&](int32_t k, const SRef& r) {
    if (!batched(r.sig) || w.priv[r.sig] || U[r.sig].empty()) return 1;
    return U[r.sig][0] == k ? 1 : 0;
  };
  for (int32_t L = 0; L <= maxl && no; ++L) {
    for (const auto& grp : p.groups) {
      std::map<std::pair<int32_t, int32_t>, std::vector<int32_t>> parts;
      std::vector<std::pair<int32_t, int32_t>> part_order;
      for (int32_t k : grp) {
        if (dist[k] != L) continue;
        const Op& o = ir.ops[k];
        const int32_t sb = o.src.sig >= 0 ? blk(k, o.src) : 1;
        const int32_t ab = (o.type == OP_ELEM_INC && batched(o.a.sig)) ? blk(k, o.a) : 1;
        auto key = std::make_pair(sb, ab);
        if (!parts.count(key)) part_order.push_back(key);
        parts[key].push_back(k);
      }
      for (const auto& key : part_order) {
        WPhase ph;
        ph.g = lower_group_at(ir, w.sig_row, parts[key]);
        ph.level = L;
        ph.src_blk = key.first;
        ph.a_blk = key.second;
        w.phases.push_back(std::move(ph));
      }
    }
  }
  // phases of a level may run concurrently only if their written signals are disjoint
  for (size_t a = 0; a < w.phases.size();) {
    size_t e = a;
    while (e < w.phases.size() && w.phases[e].level == w.phases[a].level) ++e;
    std::map<int32_t, int32_t> writers;
    std::vector<std::set<int32_t>> wsets(e - a);
    for (size_t k = a; k < e; ++k) {
      for (int32_t op : w.phases[k].g.ops) {
        access(ir.ops[op], s_, i_, r_, u_);
        for (const auto* L : {&s_, &i_, &u_})
          for (int32_t sg : *L) if (batched(sg)) wsets[k - a].insert(sg);
      }
      for (int32_t sg : wsets[k - a]) writers[sg]++;
    }
    for (size_t k = a; k < e; ++k) {
      bool ex = true;
      for (int32_t sg : wsets[k - a]) ex = ex && writers[sg] == 1;
      w.phases[k].exclusive = ex;
    }
    a = e;
  }
  fuse_window_chains(p, w, S, I, R, U);
  for (const auto& pr : ir.probes)
    for (int32_t i = 0; i < pr.src.len; ++i) w.probe_rows.push_back((int32_t)(w.sig_row[pr.src.sig] + pr.src.start + i));
  w.ok = true;
  return w;
}

std::unique_ptr<Plan> make_plan(const Model& m, double dt, const PlanOpts& o) {
  auto p = std::make_unique<Plan>();
  p->opts = o;
  p->dt = dt;
  p->built = build_params(m);
  p->ir = build_ir(m, p->built, dt);
  if (o.simplify) simplify_ir(p->ir);
  if (o.fuse) fuse_ensembles(p->ir);
  IR& ir = p->ir;
  // merge keys in first-appearance order
  std::map<std::vector<int32_t>, int32_t> kid;
  p->key_of_op.resize(ir.ops.size());
  int32_t nkeys = 0;
  for (size_t k = 0; k < ir.ops.size(); ++k) {
    if (!o.merge) { p->key_of_op[k] = nkeys++; continue; }
    auto key = merge_key(ir, ir.ops[k]);
    auto it = kid.find(key);
    if (it == kid.end()) { kid[key] = nkeys; p->key_of_op[k] = nkeys++; }
    else p->key_of_op[k] = it->second;
  }
  p->groups = plan_groups(ir, p->key_of_op, nkeys, o);
  // layout
  SortState st;
  if (o.sort) {
    sort_plan(ir, p->groups, st);
  } else {
    st.order.assign(ir.bases.size(), {});
    st.pos.assign(ir.sigs.size(), -1);
    for (int32_t s = 0; s < (int32_t)ir.sigs.size(); ++s) st.order[ir.sigs[s].base].push_back(s);
  }
  p->sig_offset.assign(ir.sigs.size(), 0);
  p->base_rows.assign(ir.bases.size(), 0);
  for (size_t b = 0; b < ir.bases.size(); ++b) {
    int64_t off = 0;
    for (int32_t s : st.order[b]) { p->sig_offset[s] = off; off += ir.sigs[s].rows; }
    p->base_rows[b] = off;
  }
  for (const auto& g : p->groups) p->lowered.push_back(lower_group(*p, g));
  // probes
  p->probe_row_offset.push_back(0);
  for (const auto& pr : ir.probes) {
    for (int32_t i = 0; i < pr.src.len; ++i)
      p->probe_src_rows.push_back((int32_t)(p->sig_offset[pr.src.sig] + pr.src.start + i));
    p->probe_width.push_back(pr.src.len);
    p->probe_row_offset.push_back((int32_t)p->probe_src_rows.size());
  }
  return p;
}

}  // namespace ms
