// Training through the window driver (paper Sec. 3.2): objective on probe
// outputs, gradient back through every step of the unrolled simulation, and
// gradient descent on the trained parameters.  Part of runtime.hip's
// translation unit (it uses the simulator's internals).
//
// The forward pass is an ordinary window run: the versioned signals then hold
// every signal at every step, which is exactly what the backward pass reads.
// The backward pass runs, for each window phase in reverse order, the
// reverse of its merged group over all steps (kernels_train.hpp) on an
// adjoint array laid out like the versioned signals, and sums the parameter
// gradients over steps and batch columns.  Only adjoints that lead to a
// trained parameter are formed: a batched signal needs one when some chain of
// operators carries a trained parameter's influence into it.

namespace {

// Kind of trained parameter a parameter signal is, from its canonical name
// (ir.cpp): e<e>.enc, e<e>.bias, e<e>.D<fn>, c<c>.D, c<c>.T, c<c>.t; -1 if
// the signal is not trained (gains, node constants).
int32_t trained_kind(const std::string& name) {
  const size_t dot = name.find('.');
  if (dot == std::string::npos || dot < 2) return -1;
  const std::string obj = name.substr(0, dot), field = name.substr(dot + 1);
  if (obj[0] == 'e') {
    if (field == "enc") return MS_TRAIN_ENCODERS;
    if (field == "bias") return MS_TRAIN_BIASES;
    if (field == "Did" || field == "Dprod") return MS_TRAIN_DECODERS;
  } else if (obj[0] == 'c') {
    if (field == "D") return MS_TRAIN_CONN_DECODERS;
    if (field == "T" || field == "t") return MS_TRAIN_TRANSFORM;
  }
  return -1;
}

int32_t* upload_ints(ms_sim* s, const std::vector<int32_t>& v) {
  int32_t* d = dev_alloc<int32_t>(std::max<size_t>(1, v.size()));
  s->extra_allocs.push_back(d);
  if (!v.empty()) HIPCHECK(hipMemcpy(d, v.data(), v.size() * 4, hipMemcpyHostToDevice));
  return d;
}

int64_t lrow(const LOperand& o, int64_t r) { return o.idx.empty() ? o.start + r : o.idx[(size_t)r]; }

bool rows_distinct(std::vector<int64_t> rows) {
  std::sort(rows.begin(), rows.end());
  return std::adjacent_find(rows.begin(), rows.end()) == rows.end();
}

void setup_train(ms_sim* s) {
  if (s->driver != MS_DRIVER_WINDOW)
    fail(MS_E_STATE, "training runs on the window driver (create the simulator with driver = MS_DRIVER_WINDOW)");
  if (s->gemm_dtype != MS_GEMM_F32) fail(MS_E_STATE, "training needs fp32 products (gemm_dtype = MS_GEMM_F32)");
  const Plan& p = *s->plan;
  const IR& ir = p.ir;
  const WindowPlan& w = *s->wplan;
  if (p.opts.simplify)
    fail(MS_E_STATE, "training needs simplify = 0 (simplification turns parameters into operator constants)");
  const size_t ns = ir.sigs.size();
  std::vector<char> tr(ns, 0), need(ns, 0);
  for (size_t k = 0; k < ns; ++k)
    if (ir.sigs[k].cls == SC_PARAM && trained_kind(ir.sigs[k].name) >= 0) {
      tr[k] = 1;
      s->trained.push_back((int32_t)k);
    }
  auto dep = [&](const SRef& r) {
    return r.sig >= 0 && (ir.sigs[r.sig].cls == SC_PARAM ? tr[r.sig] != 0 : need[r.sig] != 0);
  };
  for (const WPhase& ph : w.phases)
    for (int32_t op : ph.g.ops) {
      const Op& o = ir.ops[op];
      switch (o.type) {
        case OP_FEED: case OP_RESET: break;
        case OP_COPY: case OP_COPY_INC: case OP_ELEM_INC: case OP_DOT_INC: case OP_LIF_RATE: case OP_LOWPASS:
          if (dep(o.src) || dep(o.a)) need[o.dst.sig] = 1;
          break;
        case OP_LIF:
          fail(MS_E_STATE, "training needs rate neurons: " + o.name + " is a spiking LIF update");
        case OP_ENS:
          fail(MS_E_STATE, "training needs fuse = 0: " + o.name + " is a fused ensemble operator");
        default:
          fail(MS_E_STATE, "operator " + o.name + " has no gradient (online learning is not trained)");
      }
    }
  s->gbase.assign(ir.bases.size(), nullptr);
  for (int32_t k : s->trained) {
    const int32_t b = ir.sigs[k].base;
    if (!s->gbase[b]) s->gbase[b] = dev_alloc<float>(std::max<size_t>(1, (size_t)p.base_rows[b] * ir.bases[b].cols));
  }
  auto any_of_ops = [&](const LGroup& g, auto&& pred) {
    for (int32_t op : g.ops) if (pred(ir.ops[op])) return true;
    return false;
  };
  for (size_t k = w.phases.size(); k-- > 0;) {
    const LGroup& g = w.phases[k].g;
    const Launch& l = s->wl[k];
    if (l.rows == 0) continue;
    TrainStep st;
    st.phase = k;
    st.type = l.type;
    switch (l.type) {
      case OP_COPY: case OP_COPY_INC: case OP_ELEM_INC: {
        TScatter& S = st.sc;
        S.dst = l.dst;
        S.x = l.src;
        S.ptr = l.ptr;
        S.xblk = l.src_blk;
        S.xp = l.src_bcast ? l.src_base : nullptr;
        S.gxp = l.src_bcast ? s->gbase[g.src.base] : nullptr;
        S.want_x = any_of_ops(g, [&](const Op& o) { return dep(o.src); }) ? 1 : 0;
        if (l.type == OP_ELEM_INC) {
          S.a = l.a;
          S.a_kind = l.a_bcast ? 1 : 2;
          S.ap = l.a_bcast ? l.a_base : nullptr;
          S.gap = l.a_bcast ? s->gbase[g.a.base] : nullptr;
          S.ablk = l.a_blk;
          S.want_a = any_of_ops(g, [&](const Op& o) { return dep(o.a); }) ? 1 : 0;
        }
        if (!S.want_x && !S.want_a) continue;
        const int64_t ne = g.ptr.empty() ? g.rows : (int64_t)g.ptr.back();
        std::vector<int64_t> xr, ar;
        for (int64_t e = 0; e < ne; ++e) {
          xr.push_back(lrow(g.src, e));
          if (l.type == OP_ELEM_INC) ar.push_back(lrow(g.a, e));
        }
        S.atomic = ((S.want_x && !l.src_bcast && !rows_distinct(xr)) ||
                    (S.want_a && S.a_kind == 2 && !rows_distinct(ar))) ? 1 : 0;
        break;
      }
      case OP_LIF_RATE:
        if (!any_of_ops(g, [&](const Op& o) { return dep(o.src); })) continue;
        break;
      case OP_LOWPASS: {
        if (!any_of_ops(g, [&](const Op& o) { return dep(o.src); })) continue;
        std::vector<int64_t> xr;
        for (int64_t r = 0; r < g.rows; ++r) xr.push_back(lrow(g.src, r));
        st.atomic = rows_distinct(xr) ? 0 : 1;
        break;
      }
      case OP_DOT_INC: {
        st.dx = any_of_ops(g, [&](const Op& o) { return dep(o.src); });
        st.dw = any_of_ops(g, [&](const Op& o) { return dep(o.a); });
        if (!st.dx && !st.dw) continue;
        if (l.src_blk != 1) fail(MS_E_STATE, "a product reading a filter's previous value has no gradient here");
        if (!l.a_bcast) fail(MS_E_STATE, "a product with batched weights has no gradient here");
        st.gw = st.dw ? s->gbase[g.a.base] : nullptr;
        if (st.dx) {
          const int64_t nops = l.rows;
          st.wt = dev_alloc<float>(std::max<size_t>(1, (size_t)nops * l.M * l.K));
          s->extra_allocs.push_back(st.wt);
          // ops whose input rows overlap go to different launches, so that each
          // launch adds every adjoint element from one work item
          std::vector<std::vector<int32_t>> colour;
          std::vector<std::vector<std::pair<int64_t, int64_t>>> spans;
          for (int64_t op = 0; op < nops; ++op) {
            const int64_t a0 = g.x_row[op], a1 = a0 + l.K;
            size_t c = 0;
            for (; c < colour.size(); ++c) {
              bool clash = false;
              for (const auto& sp : spans[c]) clash = clash || (a0 < sp.second && sp.first < a1);
              if (!clash) break;
            }
            if (c == colour.size()) { colour.emplace_back(); spans.emplace_back(); }
            colour[c].push_back((int32_t)op);
            spans[c].push_back({a0, a1});
          }
          for (const auto& ops : colour) {
            std::vector<int32_t> wr, xr, dr;
            for (int32_t op : ops) {
              wr.push_back(op * l.K);          // op's W^T block: rows op*K .. of M values
              xr.push_back(g.d_row[op]);       // reads the output adjoint
              dr.push_back(g.x_row[op]);       // adds into the input adjoint
            }
            Launch lx = l;
            lx.M = l.K;
            lx.K = l.M;
            lx.rows = (int64_t)ops.size();
            lx.a_base = st.wt;
            lx.a_bcast = true;
            lx.w16 = nullptr;
            lx.src_blk = 1;
            lx.w_row = upload_ints(s, wr);
            lx.x_row = upload_ints(s, xr);
            lx.d_row = upload_ints(s, dr);
            st.dx_l.push_back(lx);
          }
        }
        break;
      }
      default:
        continue;   // FEED, RESET: nothing flows back
    }
    s->tsteps.push_back(std::move(st));
  }
  s->train_ready = true;
}

// Adjoint array for the current window (reallocated when the window grows).
void ensure_adjoints(ms_sim* s) {
  const size_t n = (size_t)std::max<int64_t>(1, s->wplan->rows_v) * s->vs;
  if (s->ga && s->ga_n == n) return;
  if (s->ga) {
    HIPCHECK(hipStreamSynchronize(s->stream));
    HIPCHECK(hipFree(s->ga));
  }
  s->ga = dev_alloc<float>(n);
  s->ga_n = n;
}

constexpr int kLossBlocks = 256;

void run_backward(ms_sim* s, int32_t T) {
  const WView w{s->va, s->vs, s->B, T};
  const double tb = (double)T * s->B;
  hipStream_t q = s->stream;
  for (const TrainStep& st : s->tsteps) {
    const Launch& l = s->wl[st.phase];
    switch (st.type) {
      case OP_COPY: case OP_COPY_INC: case OP_ELEM_INC: {
        const int64_t chunk = 4096;
        const int64_t nch = ((int64_t)tb + chunk - 1) / chunk;
        if (l.rows > 2147483647 || nch > 65535) fail(MS_E_INVALID, "window too large for the gradient launch");
        time_begin(s, kTimeGradOther, q);
        hipLaunchKernelGGL(k_t_scatter, dim3((unsigned)l.rows, (unsigned)nch), dim3(256), 0, q, w, s->ga, st.sc, chunk);
        time_end(s, q);
        break;
      }
      case OP_LIF_RATE:
        time_begin(s, kTimeGradOther, q);
        hipLaunchKernelGGL(k_t_rate, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, s->ga, l.rows, l.src,
                           l.dst, l.np, l.src_blk);
        time_end(s, q);
        break;
      case OP_LOWPASS:
        time_begin(s, kTimeGradOther, q);
        hipLaunchKernelGGL(k_t_lowpass, dim3(grid_items((double)l.rows * s->B)), dim3(kBlock), 0, q, w, s->ga,
                           l.rows, l.dst, l.src, l.fp, l.src_blk, st.atomic);
        time_end(s, q);
        break;
      case OP_DOT_INC: {
        const int64_t nops = l.rows;
        if (st.dw) {
          const bool mfma = l.M >= 64 && l.K >= 64 && s->B % 4 == 0;
          time_begin(s, mfma ? kTimeGradW : kTimeGradWSmall, q);
          if (mfma) {
            const int32_t mt = (l.M + kDwM - 1) / kDwM, kt = (l.K + kDwK - 1) / kDwK;
            const int64_t tiles = (int64_t)mt * kt * nops;
            // column chunks: enough workgroups for two per CU twice over, chunks of at least 256 columns
            const int64_t want = std::max<int64_t>(1, (4 * (int64_t)s->n_cu + tiles - 1) / tiles);
            const int64_t nsplit = std::max<int64_t>(1, std::min<int64_t>(want, (int64_t)tb / 256));
            const int64_t cchunk = (((int64_t)tb + nsplit - 1) / nsplit + kDwC - 1) / kDwC * kDwC;
            const int64_t total = tiles * nsplit;
            if (total >= 2147483647LL - 8) fail(MS_E_INVALID, "weight gradient grid too large");
            hipLaunchKernelGGL(k_t_dw, dim3((unsigned)(8 * ((total + 7) / 8))), dim3(256), 0, q, w,
                               (const float*)s->ga, l.M, l.K, mt, kt, (int32_t)nops, (int32_t)nsplit, cchunk,
                               st.gw, l.w_row, l.x_row, l.d_row, l.src_blk);
          } else if (std::min(l.M, l.K) <= kSkM) {
            const bool long_m = l.K <= kSkM && l.M > l.K;
            const int64_t L = long_m ? l.M : l.K;
            // column chunks: about 32 waves per CU over all (op, long row, chunk)
            const int64_t want = std::max<int64_t>(1, (32 * (int64_t)s->n_cu + nops * L - 1) / (nops * L));
            const int64_t nch = std::max<int64_t>(1, std::min<int64_t>(want, ((int64_t)tb + 255) / 256));
            const int64_t cchunk = ((int64_t)tb + nch - 1) / nch;
            const int64_t nwaves = nops * L * nch;
            if ((nwaves + 3) / 4 >= 2147483647LL) fail(MS_E_INVALID, "weight gradient grid too large");
            hipLaunchKernelGGL(k_t_dw_skinny, dim3((unsigned)((nwaves + 3) / 4)), dim3(256), 0, q, w,
                               (const float*)s->ga, l.M, l.K, nwaves, (int32_t)nch, cchunk, st.gw, l.w_row, l.x_row,
                               l.d_row, l.src_blk, long_m ? 1 : 0);
          } else {
            const int64_t nout = nops * l.M * l.K;
            const int64_t cchunk = 256;
            const int64_t nch = ((int64_t)tb + cchunk - 1) / cchunk;
            if (nch > 65535) fail(MS_E_INVALID, "window too large for the gradient launch");
            hipLaunchKernelGGL(k_t_dw_small, dim3(grid_for(nout), (unsigned)nch), dim3(kBlock), 0, q, w,
                               (const float*)s->ga, l.M, l.K, nout, cchunk, st.gw, l.w_row, l.x_row, l.d_row,
                               l.src_blk);
          }
          time_end(s, q);
        }
        if (st.dx) {
          time_begin(s, kTimeGradX, q);
          const int64_t n = nops * l.M * l.K;
          hipLaunchKernelGGL(k_t_transpose, dim3(grid_for(n)), dim3(kBlock), 0, q, l.a_base, l.w_row, l.M, l.K, n,
                             st.wt);
          for (const Launch& lx : st.dx_l) launch_phase(s, lx, T, 0, q, s->ga);
          time_end(s, q);
        }
        break;
      }
      default: break;
    }
  }
}

// Device pointer and shape of trained parameter (which, id, function).
struct TrainParam { int32_t sig; float* p; float* g; int64_t rows, cols; bool transposed; };

TrainParam train_param(ms_sim* s, int32_t which, int32_t id, int32_t fn) {
  const Plan& p = *s->plan;
  const IR& ir = p.ir;
  std::string name;
  switch (which) {
    case MS_TRAIN_ENCODERS: name = "e" + std::to_string(id) + ".enc"; break;
    case MS_TRAIN_BIASES: name = "e" + std::to_string(id) + ".bias"; break;
    case MS_TRAIN_DECODERS:
      if (fn != MS_FN_IDENTITY && fn != MS_FN_PRODUCT) fail(MS_E_INVALID, "unknown function");
      name = "e" + std::to_string(id) + (fn == MS_FN_PRODUCT ? ".Dprod" : ".Did");
      break;
    case MS_TRAIN_CONN_DECODERS: name = "c" + std::to_string(id) + ".D"; break;
    case MS_TRAIN_TRANSFORM: name = "c" + std::to_string(id) + ".T"; break;
    default: fail(MS_E_INVALID, "unknown trained parameter kind");
  }
  int32_t sig = -1;
  for (size_t k = 0; k < ir.sigs.size() && sig < 0; ++k)
    if (ir.sigs[k].cls == SC_PARAM &&
        (ir.sigs[k].name == name || (which == MS_TRAIN_TRANSFORM && ir.sigs[k].name == "c" + std::to_string(id) + ".t")))
      sig = (int32_t)k;
  if (sig < 0) fail(MS_E_INVALID, "the model has no trained parameter " + name);
  const Signal& sg = ir.sigs[sig];
  const int64_t cols = ir.bases[sg.base].cols;
  const int64_t off = p.sig_offset[sig] * cols;
  TrainParam t{sig, s->base_ptr[sg.base] + off, nullptr, sg.rows, cols,
               which == MS_TRAIN_DECODERS || which == MS_TRAIN_CONN_DECODERS};
  if (s->train_ready && (size_t)sg.base < s->gbase.size() && s->gbase[sg.base]) t.g = s->gbase[sg.base] + off;
  return t;
}

}  // namespace

extern "C" {

ms_status ms_sim_train_step(ms_sim* s, int64_t n_steps, const ms_feed* feeds, int32_t n_feeds,
                            const ms_target* targets, int32_t n_targets, double learning_rate, double* loss_out) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    if (n_steps < 1) fail(MS_E_INVALID, "n_steps must be >= 1");
    if (n_feeds < 0 || (n_feeds > 0 && !feeds)) fail(MS_E_INVALID, "bad feeds");
    if (n_targets < 0 || (n_targets > 0 && !targets)) fail(MS_E_INVALID, "bad targets");
    if (!std::isfinite(learning_rate)) fail(MS_E_INVALID, "learning_rate must be finite");
    DeviceGuard dg(s->device);
    if (!s->train_ready) setup_train(s);
    const Plan& p = *s->plan;
    for (int32_t i = 0; i < n_targets; ++i) {
      const int32_t pid = targets[i].probe_id;
      if (pid < 0 || pid >= (int32_t)p.probe_width.size()) fail(MS_E_INVALID, "target for an unknown probe");
      if (!targets[i].data) fail(MS_E_INVALID, "target data is NULL");
    }
    ensure_window(s, n_steps);
    if (s->W < n_steps)
      fail(MS_E_INVALID, "training needs the whole run in one window: at most " + std::to_string(s->W) +
                             " steps for this model and minibatch");
    // forward from the initial state
    reset_state(s);
    ensure_capacity(s, n_steps);
    stage_feeds(s, n_steps, feeds, n_feeds);
    ensure_adjoints(s);
    const size_t nparts = (size_t)std::max<int32_t>(1, n_targets) * kLossBlocks;
    if (s->loss_part_n < nparts) {
      HIPCHECK(hipStreamSynchronize(s->stream));
      if (s->loss_part) HIPCHECK(hipFree(s->loss_part));
      s->loss_part = dev_alloc<float>(nparts);
      s->loss_part_n = nparts;
    }
    HIPCHECK(hipMemsetAsync(s->ctr + 1, 0, sizeof(int64_t), s->stream));
    s->tn = 0;
    HIPCHECK(hipEventRecord(s->ev0, s->stream));
    run_window(s, n_steps);
    s->steps_total += n_steps;
    // adjoints and gradients from zero
    HIPCHECK(hipMemsetAsync(s->ga, 0, s->ga_n * sizeof(float), s->stream));
    for (size_t b = 0; b < s->gbase.size(); ++b)
      if (s->gbase[b])
        HIPCHECK(hipMemsetAsync(s->gbase[b], 0, (size_t)p.base_rows[b] * p.ir.bases[b].cols * sizeof(float), s->stream));
    HIPCHECK(hipMemsetAsync(s->loss_part, 0, nparts * sizeof(float), s->stream));
    const int32_t T = (int32_t)n_steps;
    const WView w{s->va, s->vs, s->B, T};
    for (int32_t i = 0; i < n_targets; ++i) {
      const int32_t pid = targets[i].probe_id;
      const int32_t width = p.probe_width[pid];
      const size_t n = (size_t)s->B * T * width;
      if (n == 0) continue;
      const float* tg = targets[i].data;
      if (!targets[i].on_device) {
        if (s->tgt_n < n) {
          HIPCHECK(hipStreamSynchronize(s->stream));
          if (s->tgt_buf) HIPCHECK(hipFree(s->tgt_buf));
          s->tgt_buf = dev_alloc<float>(n);
          s->tgt_n = n;
        }
        HIPCHECK(hipMemcpyAsync(s->tgt_buf, tg, n * 4, hipMemcpyHostToDevice, s->stream));
        tg = s->tgt_buf;
      }
      const unsigned blocks = (unsigned)std::min<size_t>(kLossBlocks, (n + kBlock - 1) / kBlock);
      time_begin(s, kTimeGradOther, s->stream);
      hipLaunchKernelGGL(k_t_loss, dim3(blocks), dim3(kBlock), 0, s->stream, w, s->ga,
                         s->wprobe_src + p.probe_row_offset[pid], width, tg, (float)(1.0 / (double)n),
                         s->loss_part + (size_t)i * kLossBlocks);
      time_end(s, s->stream);
      if (!targets[i].on_device) HIPCHECK(hipStreamSynchronize(s->stream));   // tgt_buf reused
    }
    run_backward(s, T);
    if (learning_rate != 0.0) {
      time_begin(s, kTimeGradOther, s->stream);
      for (int32_t k : s->trained) {
        const Signal& sg = p.ir.sigs[k];
        const int64_t cols = p.ir.bases[sg.base].cols, off = p.sig_offset[k] * cols, n = (int64_t)sg.rows * cols;
        hipLaunchKernelGGL(k_t_sgd, dim3(grid_for(n)), dim3(kBlock), 0, s->stream, s->base_ptr[sg.base] + off,
                           (const float*)(s->gbase[sg.base] + off), n, (float)learning_rate);
      }
      time_end(s, s->stream);
    }
    HIPCHECK(hipGetLastError());
    HIPCHECK(hipEventRecord(s->ev1, s->stream));
    std::vector<float> parts(nparts);
    HIPCHECK(hipMemcpyAsync(parts.data(), s->loss_part, nparts * 4, hipMemcpyDeviceToHost, s->stream));
    HIPCHECK(hipStreamSynchronize(s->stream));
    double loss = 0.0;
    for (int32_t i = 0; i < n_targets; ++i) {
      const size_t n = (size_t)s->B * T * p.probe_width[targets[i].probe_id];
      double sum = 0.0;
      for (int k = 0; k < kLossBlocks; ++k) sum += parts[(size_t)i * kLossBlocks + k];
      if (n) loss += sum / (double)n;
    }
    if (loss_out) *loss_out = loss;
  });
}

ms_status ms_sim_train_param(ms_sim* s, int32_t which, int32_t id, int32_t fn, int32_t gradient, float* out,
                             int64_t cap, int64_t* n_out) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    DeviceGuard dg(s->device);
    const TrainParam t = train_param(s, which, id, fn);
    const int64_t n = t.rows * t.cols;
    if (n_out) *n_out = n;
    if (!out) return;
    if (cap < n) fail(MS_E_INVALID, "output capacity too small");
    std::vector<float> h((size_t)n, 0.0f);
    HIPCHECK(hipStreamSynchronize(s->stream));
    if (!gradient) HIPCHECK(hipMemcpy(h.data(), t.p, (size_t)n * 4, hipMemcpyDeviceToHost));
    else if (t.g) HIPCHECK(hipMemcpy(h.data(), t.g, (size_t)n * 4, hipMemcpyDeviceToHost));
    if (t.transposed) {   // stored [outputs][n], returned [n][outputs]
      for (int64_t r = 0; r < t.rows; ++r)
        for (int64_t c = 0; c < t.cols; ++c) out[c * t.rows + r] = h[(size_t)(r * t.cols + c)];
    } else {
      std::copy(h.begin(), h.end(), out);
    }
  });
}

ms_status ms_sim_set_train_param(ms_sim* s, int32_t which, int32_t id, int32_t fn, const float* in, int64_t n) {
  return guarded([&] {
    if (!s || !in) fail(MS_E_INVALID, "NULL argument");
    DeviceGuard dg(s->device);
    const TrainParam t = train_param(s, which, id, fn);
    if (n != t.rows * t.cols) fail(MS_E_INVALID, "parameter size mismatch");
    std::vector<float> h((size_t)n);
    if (t.transposed) {
      for (int64_t r = 0; r < t.rows; ++r)
        for (int64_t c = 0; c < t.cols; ++c) h[(size_t)(r * t.cols + c)] = in[c * t.rows + r];
    } else {
      std::copy(in, in + n, h.begin());
    }
    HIPCHECK(hipStreamSynchronize(s->stream));
    HIPCHECK(hipMemcpy(t.p, h.data(), (size_t)n * 4, hipMemcpyHostToDevice));
  });
}

}  // extern "C"
