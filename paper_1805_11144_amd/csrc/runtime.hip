// GPU runtime of mergesim: device base arrays, the merged-group kernels, the
// step drivers (stream-ordered launches, a hipGraph of `unroll` steps, and a
// persistent per-batch-column kernel), feeds, probes and state access.
//
// Data layout in HBM (paper Sec. 4.2.1: signals are concatenated along the
// first axis into base arrays):
//   state  float [rows][B]  every batched signal, minibatch contiguous
//   vec    float [rows]     per-row parameters (biases, gains, scalars)
//   mat<K> float [rows][K]  weight matrices with K columns
// Each merged group is one launch; a group's per-row operands are either a
// contiguous row range (a "slice") or an int32 index list.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include <mutex>

#include "host.hpp"
#include "kernels.hpp"
#include "kernels_window.hpp"
#include "kernels_train.hpp"

using namespace ms;

// Staging array of ms_sim_probe_read_static, which allocates nothing: one copy
// per GPU, held until the process ends.  In host code its name is only a
// handle; its device address (per device) comes from hipGetSymbolAddress.
static __device__ __align__(256) float scratch[MS_PROBE_READ_STATIC_MAX];

#define HIPCHECK(expr)                                                                    \
  do {                                                                                    \
    hipError_t _e = (expr);                                                               \
    if (_e != hipSuccess)                                                                 \
      ms::fail(MS_E_HIP, std::string(#expr) + ": " + hipGetErrorString(_e));              \
  } while (0)

namespace {

template <class T>
T* dev_alloc(size_t n) {
  if (n == 0) return nullptr;
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, n * sizeof(T));
  if (e != hipSuccess) fail(MS_E_OOM, std::string("hipMalloc failed: ") + hipGetErrorString(e));
  return (T*)p;
}

// Host mirror of one lowered group, with device pointers.
struct Launch {
  int32_t type = 0;
  int64_t rows = 0;
  Opnd dst, src, a, V, ref;
  const float* src_base = nullptr;   // base array of src (COPY*, ELEM_INC x)
  bool src_bcast = false;            // src base is a parameter base (no batch axis)
  const float* a_base = nullptr;     // ELEM_INC a / DOT_INC W base
  const int32_t* ptr = nullptr;      // CSR offsets (repeated destinations) or null
  const float* values = nullptr;     // RESET values or null (zeros)
  int32_t M = 0, K = 0;
  const int32_t* w_row = nullptr;
  const int32_t* x_row = nullptr;
  const int32_t* d_row = nullptr;
  NeuronParams np{};
  FilterParams fp{};
  const int32_t* feed_rows = nullptr;
  EnsDesc ens{};
  bool a_bcast = true;               // ELEM_INC a is a parameter base
  // window driver
  int32_t src_blk = 1, a_blk = 1;    // block offsets of src / a (1: this step, 0: previous step)
  int32_t nmax = 0, npt = 1, nthr = 64, ts = 16, cpw = 1, kch = 1;   // fused-ensemble launch shape
  int32_t enc_lds = 0, dec_lds = 0, rw = 0;   // rw: encoder/decoder fragments held in registers
  int32_t xs = 1, js = 1;            // LDS row strides of the inputs and currents (padded)
  size_t lds = 0;
  const uint16_t* w16 = nullptr;     // DOT_INC on bf16 MFMA: W rounded to bf16, op k at k*M*K
  // SYN_SCATTER
  const int32_t* syn_seg = nullptr;
  const SynConn* syn_conn = nullptr;
  SynW syn_w{};
  int32_t syn_update = 1;
  int32_t syn_probe = 0;
  // BDOT_INC / PES / PES_FUSED: per-op rows, chunking of the neurons
  int32_t ens_nmax = 0;              // ENS: most neurons of an op
  const int32_t* e_row = nullptr;
  const int32_t* act_row = nullptr;
  const float* coef = nullptr;
  int32_t pes_L = 0, pes_nch = 0;
};

// Backward work of one forward window phase (training, paper Sec. 3.2).
struct TrainStep {
  size_t phase = 0;                  // index into the window phases
  int32_t type = 0;
  TScatter sc{};                     // COPY / COPY_INC / ELEM_INC
  int32_t atomic = 0;                // LOWPASS: inputs shared by several rows
  bool dx = false, dw = false;       // DOT_INC: adjoint of the input, gradient of W
  std::vector<Launch> dx_l;          // products on W^T, input rows disjoint within each launch
  float* wt = nullptr;               // W^T, [nops * K][M]
  float* gw = nullptr;               // gradient base of W
};

}  // namespace

struct ms_sim {
  std::unique_ptr<Plan> plan;
  int32_t B = 1;
  int32_t device = 0;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  int32_t driver = MS_DRIVER_STEPS;
  int32_t unroll = 10;
  int32_t gemm_dtype = MS_GEMM_F32;
  int32_t decode = MS_DECODE_DENSE;
  float dt = 0.001f;
  // device memory
  std::vector<float*> base_ptr;      // per base id
  float* state = nullptr;
  size_t state_rows = 0;
  Strides S{1, 1};                   // element (r, b) at r * S.rs + b * S.cs
  int32_t* ipool = nullptr;
  float* fpool = nullptr;
  std::vector<Launch> launches;
  bool has_prologue = false;         // launch drivers: pull of the post inputs before each run
  Launch prologue;
  bool probe_folded = false;         // the step's fused synapse launch records the probes
  int64_t* ctr = nullptr;            // [0] steps recorded since reset, [1] step within run
  float* feed_stage = nullptr;       // [cap][feed_rows][B]
  int64_t feed_cap = 0;
  float* feed_tmp = nullptr;         // [B][T][size] upload buffer for host feeds
  size_t feed_tmp_elems = 0;
  float* probe_buf = nullptr;        // [cap][probe_rows][B]
  // spike probes recorded as bitmasks (window driver, opts spike_probe_bits):
  // per probe the spike value amplitude / dt, or 0 for a probe recorded as floats
  std::vector<float> spike_mag;
  std::vector<int32_t> bit_off;      // per probe: first word row in bits_buf, or -1
  int32_t bit_words = 0;             // word rows per step (0: no bit-recorded probe)
  uint32_t* bits_buf = nullptr;      // [cap][bit_words][B]
  int32_t* wbit_src = nullptr;       // [bit_words * 32]: window row of each bit, -1 pads
  int32_t* wprobe_fsrc = nullptr;    // float-recorded probe rows: window source rows
  int32_t* wprobe_fdst = nullptr;    // ... and their rows in probe_buf
  int32_t pr_float = 0;
  int64_t probe_cap = 0;
  int32_t probe_rows = 0;
  const int32_t* probe_src = nullptr;
  int64_t steps_total = 0;
  // graph driver
  hipGraphExec_t graph_exec = nullptr;
  hipGraph_t graph = nullptr;
  bool graph_valid = false;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  double last_ms = 0.0;
  // persistent driver
  PersistentProgram prog{};
  bool persistent_ok = false;
  size_t lds_limit = 0;              // dynamic LDS bytes one workgroup may use
  int32_t n_cu = 256;                // compute units of the device
  int32_t persistent_threads = 256;  // workgroup size of the persistent kernel
  int64_t scratch_n = 0;             // per-column scratch floats of the persistent kernel
  float* col_scratch = nullptr;      // global scratch when state is not LDS-resident
  std::vector<void*> extra_allocs;   // transposed weights and their offsets, extra pools
  // window driver
  std::unique_ptr<WindowPlan> wplan;
  std::vector<Launch> wl;            // phases in execution order
  float* va = nullptr;               // versioned signals [rows_v][(W+1)*B]
  float* pa = nullptr;               // neuron state [rows_p][B]
  int32_t W = 0;                     // steps per window
  int64_t vs = 0;                    // row stride of va
  const int32_t* wprobe_src = nullptr;
  // per-launch timing (ms_sim_set_timing)
  bool timing = false;
  std::vector<hipEvent_t> tev;       // event pool, pairs
  std::vector<int32_t> ttype;        // op type of each recorded pair
  size_t tn = 0;                     // pairs recorded in the last run
  bool tx = false, tx_first = false; // a launch-driver group is being timed (first kernel next)
  hipEvent_t tx_start = nullptr, tx_stop = nullptr;
  static constexpr int kSide = 3;    // extra streams for independent phases of one level
  hipStream_t side[kSide] = {};
  hipEvent_t side_ev[kSide + 1] = {};
  std::vector<std::vector<float>> host_bases;   // host copies of parameter bases
  float* init_vals = nullptr;        // initial values of batched state signals that have one
  std::vector<std::pair<int32_t, int64_t>> init_sigs;   // (signal, offset in init_vals)
  float* pes_part = nullptr;         // partial decodes of the learned-decoder launches
  size_t pes_part_n = 0, pes_part_cap = 0;
  // training (window driver)
  bool train_ready = false;
  std::vector<TrainStep> tsteps;     // backward order
  std::vector<int32_t> trained;      // trained parameter signals
  float* ga = nullptr;               // adjoints, laid out like va
  size_t ga_n = 0;
  std::vector<float*> gbase;         // per base: parameter gradients (null: nothing trained there)
  float* loss_part = nullptr;        // per-workgroup sums of squared differences
  size_t loss_part_n = 0;
  float* tgt_buf = nullptr;          // a target uploaded from the host
  size_t tgt_n = 0;
  // failure detection
  bool check_feeds = false;          // scan every feed for NaN / Inf before a run
  unsigned int* nonfinite = nullptr; // device count of non-finite feed values
};

namespace {

struct DeviceGuard {
  int prev = 0;
  explicit DeviceGuard(int dev) {
    HIPCHECK(hipGetDevice(&prev));
    if (prev != dev) HIPCHECK(hipSetDevice(dev));
  }
  ~DeviceGuard() {
    int cur = 0;
    if (hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

// Device address of `scratch` on each device, resolved once per device with
// that device current (at simulator creation).
std::mutex g_scratch_mu;
std::vector<float*> g_scratch_ptr;

float* scratch_on(int dev) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (dev < 0) fail(MS_E_INVALID, "device ordinal out of range");
  if ((size_t)dev >= g_scratch_ptr.size()) g_scratch_ptr.resize((size_t)dev + 1, nullptr);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    HIPCHECK(hipGetDevice(&cur));
    if (cur != dev) fail(MS_E_STATE, "static staging array resolved on another device");
    void* p = nullptr;
    HIPCHECK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) fail(MS_E_HIP, "hipGetSymbolAddress returned no address for the staging array");
    g_scratch_ptr[dev] = (float*)p;
  }
  return g_scratch_ptr[dev];
}

void destroy_graph(ms_sim* s) {
  if (s->graph_exec) (void)hipGraphExecDestroy(s->graph_exec);
  if (s->graph) (void)hipGraphDestroy(s->graph);
  s->graph_exec = nullptr;
  s->graph = nullptr;
  s->graph_valid = false;
}

void free_sim(ms_sim* s) {
  destroy_graph(s);
  auto f = [](void* p) { if (p) (void)hipFree(p); };
  f(s->state);
  for (size_t b = 0; b < s->base_ptr.size(); ++b)
    if (s->base_ptr[b] != s->state) f(s->base_ptr[b]);
  f(s->ipool); f(s->fpool); f(s->ctr); f(s->feed_stage); f(s->feed_tmp); f(s->probe_buf);
  f(s->prog.groups);
  f(s->col_scratch);
  f(s->va); f(s->pa);
  f(s->pes_part);
  f(s->init_vals);
  f(s->ga); f(s->loss_part); f(s->tgt_buf); f(s->nonfinite);
  f(s->bits_buf); f(s->wbit_src); f(s->wprobe_fsrc); f(s->wprobe_fdst);
  for (float* g : s->gbase) f(g);
  for (void* p : s->extra_allocs) f(p);
  if (s->ev0) (void)hipEventDestroy(s->ev0);
  if (s->ev1) (void)hipEventDestroy(s->ev1);
  for (hipEvent_t e : s->tev) (void)hipEventDestroy(e);
  for (int k = 0; k < ms_sim::kSide; ++k)
    if (s->side[k]) (void)hipStreamDestroy(s->side[k]);
  for (int k = 0; k <= ms_sim::kSide; ++k)
    if (s->side_ev[k]) (void)hipEventDestroy(s->side_ev[k]);
  if (s->own_stream && s->stream) (void)hipStreamDestroy(s->stream);
}

// Pools of int32 and float arrays uploaded once; offsets resolved to pointers later.
struct PoolBuilder {
  std::vector<int32_t> ints;
  std::vector<float> floats;
  int64_t add_i(const std::vector<int32_t>& v) {
    if (v.empty()) return -1;
    int64_t off = (int64_t)ints.size();
    ints.insert(ints.end(), v.begin(), v.end());
    while (ints.size() % 64) ints.push_back(0);   // keep arrays 256-byte aligned
    return off;
  }
  int64_t add_f(const std::vector<float>& v) {
    if (v.empty()) return -1;
    int64_t off = (int64_t)floats.size();
    floats.insert(floats.end(), v.begin(), v.end());
    while (floats.size() % 64) floats.push_back(0.f);
    return off;
  }
};

const std::vector<float>& host_param_base(ms_sim* s, int32_t base);

// Lowered groups -> launch records (index and parameter arrays uploaded into
// pools owned by the simulator); `extra_ints` is uploaded alongside and its
// device address returned in *extra_ptr.
void build_launches(ms_sim* s, const std::vector<LGroup>& groups, std::vector<Launch>& out,
                    const std::vector<int32_t>& extra_ints, const int32_t** extra_ptr) {
  Plan& p = *s->plan;
  const IR& ir = p.ir;
  // ---- lowered groups -> pools
  PoolBuilder pb;
  struct Offs { int64_t dst, src, a, V, ref, ptr, values, w, x, d, trc, tref, amp, ca, cb, feed, full, e, act, coef, sig; };
  std::vector<Offs> offs;
  for (const LGroup& g : groups) {
    Offs o{};
    o.dst = pb.add_i(g.dst.idx); o.src = pb.add_i(g.src.idx); o.a = pb.add_i(g.a.idx);
    o.V = pb.add_i(g.V.idx); o.ref = pb.add_i(g.ref.idx); o.ptr = pb.add_i(g.ptr);
    o.w = pb.add_i(g.w_row); o.x = pb.add_i(g.x_row); o.d = pb.add_i(g.d_row);
    o.e = pb.add_i(g.e_row); o.act = pb.add_i(g.act_row); o.coef = pb.add_f(g.coef);
    o.feed = pb.add_i(g.feed_rows);
    o.values = pb.add_f(g.values);
    const bool per_row_params = g.type != OP_ENS;
    o.trc = per_row_params && g.tau_rc.size() > 1 ? pb.add_f(g.tau_rc) : -1;
    o.full = -1;
    if (per_row_params && g.tau_rc.size() > 1) {
      std::vector<float> full(g.tau_rc.size());
      for (size_t k = 0; k < full.size(); ++k) full[k] = (float)std::expm1(-p.dt / (double)g.tau_rc[k]);
      o.full = pb.add_f(full);
    }
    o.tref = per_row_params && g.tau_ref.size() > 1 ? pb.add_f(g.tau_ref) : -1;
    o.sig = g.sigma.size() > 1 ? pb.add_f(g.sigma) : -1;
    o.amp = per_row_params && g.amp.size() > 1 ? pb.add_f(g.amp) : -1;
    o.ca = g.ca.size() > 1 ? pb.add_f(g.ca) : -1;
    o.cb = g.cb.size() > 1 ? pb.add_f(g.cb) : -1;
    offs.push_back(o);
  }
  // packed per-op records of fused ensemble groups (EnsOp, 17 x 4 bytes each)
  static_assert(sizeof(EnsOp) == 17 * 4, "EnsOp layout");
  std::vector<int64_t> ens_off(groups.size(), -1);
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    const LGroup& g = groups[gi];
    if (g.type != OP_ENS) continue;
    std::vector<int32_t> rec;
    for (size_t k = 0; k < g.ens_n.size(); ++k) {
      EnsOp e{};
      e.n = g.ens_n[k]; e.x = g.ens_x[k]; e.enc = g.ens_enc[k]; e.bias = g.ens_bias[k];
      e.V = g.ens_V[k]; e.ref = g.ens_ref[k]; e.s = g.ens_s[k];
      for (int f = 0; f < kMaxFns; ++f) {
        e.D[f] = f < (int)g.ens_D.size() ? g.ens_D[f][k] : 0;
        e.d[f] = f < (int)g.ens_dd.size() ? g.ens_dd[f][k] : 0;
      }
      const float trc = g.tau_rc.size() > 1 ? g.tau_rc[k] : g.tau_rc[0];
      e.tau_rc = trc;
      e.tau_ref = g.tau_ref.size() > 1 ? g.tau_ref[k] : g.tau_ref[0];
      e.amp = g.amp.size() > 1 ? g.amp[k] : g.amp[0];
      e.full = (float)std::expm1(-p.dt / (double)trc);
      e.inv_tau = (float)(1.0 / (double)trc);
      e.tau6 = (float)((double)trc / 6.0);
      const int32_t* w = reinterpret_cast<const int32_t*>(&e);
      rec.insert(rec.end(), w, w + 17);
    }
    ens_off[gi] = pb.add_i(rec);
  }
  // fused connection chains of window ensemble phases (8 words per op)
  std::vector<int64_t> chain_off(groups.size(), -1);
  for (size_t gi = 0; gi < groups.size(); ++gi)
    if (groups[gi].type == OP_ENS && !groups[gi].ens_chain.empty()) chain_off[gi] = pb.add_i(groups[gi].ens_chain);
  // fused synapse groups: segments, then connection records of 8 words
  static_assert(sizeof(SynConn) == 8 * 4, "SynConn layout");
  std::vector<int64_t> seg_off(groups.size(), -1), conn_off(groups.size(), -1);
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    const LGroup& g = groups[gi];
    if (g.type != OP_SYN_SCATTER) continue;
    seg_off[gi] = pb.add_i(g.syn_seg);
    std::vector<int32_t> rec;
    const size_t nc = g.syn_conn.size() / 8;
    for (size_t c = 0; c < nc; ++c) {
      const int32_t* q = &g.syn_conn[8 * c];
      if (q[0] < 0 || q[3] < 0 || q[3] > 0xffff || q[4] > 3 || q[4] < -2) fail(MS_E_INVALID, "fused synapse connection out of range");
      SynConn r{};
      r.y = q[0]; r.v = q[1]; r.x = q[2];
      r.kw = q[3] | (std::max(q[4], 0) << 16) | (q[7] ? 1 << 20 : 0) | (q[4] == -2 ? 1 << 21 : 0);
      r.w = q[5]; r.p = q[6];
      r.a = g.syn_ab[2 * c]; r.b = g.syn_ab[2 * c + 1];
      const int32_t* w = reinterpret_cast<const int32_t*>(&r);
      rec.insert(rec.end(), w, w + 8);
    }
    conn_off[gi] = pb.add_i(rec);
  }
  const int64_t extra_off = pb.add_i(extra_ints);
  int32_t* ipool = dev_alloc<int32_t>(std::max<size_t>(1, pb.ints.size()));
  float* fpool = dev_alloc<float>(std::max<size_t>(1, pb.floats.size()));
  s->extra_allocs.push_back(ipool);
  s->extra_allocs.push_back(fpool);
  if (!pb.ints.empty())
    HIPCHECK(hipMemcpy(ipool, pb.ints.data(), pb.ints.size() * 4, hipMemcpyHostToDevice));
  if (!pb.floats.empty())
    HIPCHECK(hipMemcpy(fpool, pb.floats.data(), pb.floats.size() * 4, hipMemcpyHostToDevice));
  auto ip = [&](int64_t off) -> const int32_t* { return off < 0 ? nullptr : ipool + off; };
  auto fp = [&](int64_t off) -> const float* { return off < 0 ? nullptr : fpool + off; };
  *extra_ptr = ip(extra_off);
  auto opnd = [&](const LOperand& L, int64_t off) { return Opnd{ip(off), L.start}; };
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    const LGroup& g = groups[gi];
    const Offs& o = offs[gi];
    Launch l;
    l.type = g.type;
    l.rows = g.rows;
    l.dst = opnd(g.dst, o.dst);
    l.src = opnd(g.src, o.src);
    l.a = opnd(g.a, o.a);
    l.V = opnd(g.V, o.V);
    l.ref = opnd(g.ref, o.ref);
    if (g.src.base >= 0) {
      l.src_base = s->base_ptr[g.src.base];
      l.src_bcast = ir.bases[g.src.base].cls != SC_BATCHED;
    }
    if (g.a.base >= 0) {
      l.a_base = s->base_ptr[g.a.base];
      l.a_bcast = ir.bases[g.a.base].cls != SC_BATCHED;
    }
    l.ptr = ip(o.ptr);
    l.values = fp(o.values);
    l.M = g.M; l.K = g.K;
    l.w_row = ip(o.w); l.x_row = ip(o.x); l.d_row = ip(o.d);
    l.feed_rows = ip(o.feed);
    if (g.type == OP_LIF || g.type == OP_LIF_RATE) {
      l.np.tau_rc = g.tau_rc[0]; l.np.tau_ref = g.tau_ref[0]; l.np.amp = g.amp[0];
      l.np.full = (float)std::expm1(-p.dt / (double)g.tau_rc[0]);
      l.np.tau_rc_r = fp(o.trc); l.np.tau_ref_r = fp(o.tref); l.np.amp_r = fp(o.amp);
      l.np.full_r = fp(o.full);
      l.np.relu = g.type == OP_LIF_RATE && g.ens_type == MS_NEURON_RELU ? 1 : 0;
      l.np.sigma = g.sigma.empty() ? 0.0f : g.sigma[0];
      l.np.sigma_r = fp(o.sig);
    }
    if (g.type == OP_LOWPASS) {
      l.fp.a = g.ca[0]; l.fp.b = g.cb[0];
      l.fp.a_r = fp(o.ca); l.fp.b_r = fp(o.cb);
    }
    if (g.type == OP_ENS) {
      EnsDesc& E = l.ens;
      if ((int)g.ens_df.size() > kMaxFns) fail(MS_E_INVALID, "fused ensemble with too many decoded functions");
      E.d = g.ens_d; E.ntype = g.ens_type; E.nf = (int32_t)g.ens_df.size(); E.ndec = 0;
      for (int f = 0; f < E.nf; ++f) { E.df[f] = g.ens_df[f]; E.ndec += g.ens_df[f]; }
      if (E.ndec > kMaxDec) fail(MS_E_INVALID, "fused ensemble decodes too many outputs");
      for (int f = 0; f < E.nf; ++f) {
        E.D[f] = s->base_ptr[g.ens_Dbase[f]];
        E.Dcols[f] = ir.bases[g.ens_Dbase[f]].cols;
      }
      E.enc = g.a.base >= 0 ? s->base_ptr[g.a.base] : nullptr;
      if (g.a.base >= 0 && g.ens_d > 0 && s->B < 32) {
        // per-op transposed encoder blocks for the lanes-over-neurons kernel
        const std::vector<float>& he = host_param_base(s, g.a.base);
        std::vector<float> t(he.size(), 0.0f);
        const int64_t d = g.ens_d;
        for (size_t k = 0; k < g.ens_n.size(); ++k) {
          if (g.ens_x[k] < 0 || g.ens_enc[k] < 0) continue;   // no input, no encoders
          const int64_t e0 = g.ens_enc[k], n = g.ens_n[k];
          for (int64_t r = 0; r < n; ++r)
            for (int64_t q = 0; q < d; ++q) t[(size_t)(e0 * d + q * n + r)] = he[(size_t)((e0 + r) * d + q)];
        }
        float* dt_ = dev_alloc<float>(std::max<size_t>(1, t.size()));
        HIPCHECK(hipMemcpy(dt_, t.data(), t.size() * 4, hipMemcpyHostToDevice));
        s->extra_allocs.push_back(dt_);
        E.encT = dt_;
      }
      if (s->decode == MS_DECODE_EVENT && g.ens_type == 0 && E.ndec > 0 && s->B < 32 &&
          (s->driver == MS_DRIVER_STEPS || s->driver == MS_DRIVER_GRAPH)) {
        // neuron-major decoders for event-driven decoding: op k's neuron r
        // holds its decoded outputs (function 0's rows, then function 1's) in
        // one row of dec_bucket(ndec) values, zero-padded
        const int64_t row = dec_bucket(E.ndec);
        int64_t nmax = 1;
        for (int32_t n : g.ens_n) nmax = std::max<int64_t>(nmax, n);
        std::vector<float> t((size_t)(g.ens_n.size() * nmax * row), 0.0f);
        for (int f = 0, q0 = 0; f < E.nf; q0 += E.df[f], ++f) {
          const std::vector<float>& hd = host_param_base(s, g.ens_Dbase[f]);
          const int64_t cols = E.Dcols[f];
          for (size_t k = 0; k < g.ens_n.size(); ++k)
            for (int32_t q = 0; q < E.df[f]; ++q)
              for (int64_t r = 0; r < g.ens_n[k]; ++r)
                t[(size_t)(((int64_t)k * nmax + r) * row + q0 + q)] =
                    hd[(size_t)(((int64_t)g.ens_D[f][k] + q) * cols + r)];
        }
        float* dd = dev_alloc<float>(t.size());
        HIPCHECK(hipMemcpy(dd, t.data(), t.size() * 4, hipMemcpyHostToDevice));
        s->extra_allocs.push_back(dd);
        E.decT = dd;
        E.dT_op = nmax * row;
        E.dT_row = (int32_t)row;
      }
      E.bias = s->base_ptr[g.ens_bias_base];
      E.ops = reinterpret_cast<const EnsOp*>(ipool + ens_off[gi]);
      if (chain_off[gi] >= 0) {
        E.chain = ip(chain_off[gi]);
        E.chain_w = s->base_ptr[g.ens_chain_wbase];
        E.chain_wcols = ir.bases[g.ens_chain_wbase].cols;
      }
      for (int32_t n : g.ens_n) l.ens_nmax = std::max(l.ens_nmax, n);
    }
    if (g.type == OP_BDOT_INC || g.type == OP_PES || g.type == OP_PES_FUSED) {
      // neurons per workgroup: about 2048 workgroups per launch, at least 4
      // neurons each, the chunk's activities (2 * L * B floats) within 64 KB of LDS
      if (s->S.rs != s->B || s->S.cs != 1) fail(MS_E_INVALID, "learned decoders need the launch drivers' state layout");
      const int64_t MB = (int64_t)g.M * s->B;
      const int64_t cblk = (MB + 255) / 256;
      if (g.rows > 65535 || cblk > 2147483647LL) fail(MS_E_INVALID, "learned-decoder group too large");
      const int64_t lmax = 8192 / s->B;
      if (lmax < 1) fail(MS_E_INVALID, "minibatch too large for learned decoders (at most 8192)");
      const int64_t want = std::max<int64_t>(1, 2048 / std::max<int64_t>(1, cblk * g.rows));
      int64_t L = std::max<int64_t>(4, (g.K + want - 1) / want);
      L = std::max<int64_t>(1, std::min<int64_t>(L, lmax));
      const int64_t nch = (g.K + L - 1) / L;
      if (nch > 65535) fail(MS_E_INVALID, "learned-decoder group has too many neurons for its minibatch");
      l.pes_L = (int32_t)L;
      l.pes_nch = (int32_t)nch;
      l.e_row = ip(o.e);
      l.act_row = ip(o.act);
      l.coef = fp(o.coef);
      if (g.type != OP_PES) s->pes_part_n = std::max(s->pes_part_n, (size_t)(g.rows * nch * MB));
    }
    if (g.type == OP_SYN_SCATTER) {
      if ((int)g.syn_wbase.size() > 4) fail(MS_E_INVALID, "fused synapse group with too many weight bases");
      l.syn_seg = ip(seg_off[gi]);
      l.syn_conn = reinterpret_cast<const SynConn*>(ip(conn_off[gi]));
      for (size_t k = 0; k < g.syn_wbase.size(); ++k) l.syn_w.w[k] = s->base_ptr[g.syn_wbase[k]];
      l.syn_update = g.syn_update;
      l.syn_probe = g.syn_probe;
    }
    out.push_back(l);
  }
  if (s->pes_part_n > s->pes_part_cap) {
    if (s->pes_part) HIPCHECK(hipFree(s->pes_part));
    s->pes_part = nullptr;
    s->pes_part = dev_alloc<float>(s->pes_part_n);
    s->pes_part_cap = s->pes_part_n;
  }
}

void setup_device(ms_sim* s) {
  Plan& p = *s->plan;
  const IR& ir = p.ir;
  const int32_t B = s->B;
  // ---- base arrays
  s->base_ptr.assign(ir.bases.size(), nullptr);
  for (size_t b = 0; b < ir.bases.size(); ++b) {
    const BaseArray& ba = ir.bases[b];
    if (ba.cls == SC_BATCHED) {
      s->state_rows = (size_t)p.base_rows[b];
      s->state = dev_alloc<float>(std::max<size_t>(1, s->state_rows * B));
      s->base_ptr[b] = s->state;
    } else {
      const size_t n = (size_t)p.base_rows[b] * ba.cols;
      std::vector<float> host(std::max<size_t>(1, n), 0.f);
      for (size_t k = 0; k < ir.sigs.size(); ++k) {
        const Signal& sg = ir.sigs[k];
        if (sg.base != (int32_t)b) continue;
        const size_t off = (size_t)p.sig_offset[k] * ba.cols;
        for (size_t j = 0; j < sg.value.size(); ++j) host[off + j] = (float)sg.value[j];
      }
      s->base_ptr[b] = dev_alloc<float>(host.size());
      HIPCHECK(hipMemcpy(s->base_ptr[b], host.data(), host.size() * sizeof(float), hipMemcpyHostToDevice));
      if (s->host_bases.size() <= b) s->host_bases.resize(b + 1);
      s->host_bases[b] = std::move(host);
    }
  }
  if (!s->state) {
    s->state = dev_alloc<float>(B);
  }
  // the persistent driver interprets the plan's groups one to one; the launch
  // drivers run the step program (merged ensemble launches, fused synapses)
  if (s->driver == MS_DRIVER_STEPS || s->driver == MS_DRIVER_GRAPH) {
    LaunchPlan lp = make_launch_plan(p);
    std::vector<LGroup> gs = std::move(lp.step);
    if (lp.has_prologue) gs.push_back(lp.prologue);
    build_launches(s, gs, s->launches, p.probe_src_rows, &s->probe_src);
    if (lp.has_prologue) {
      s->prologue = s->launches.back();
      s->launches.pop_back();
      s->has_prologue = true;
    }
    for (const Launch& l : s->launches) s->probe_folded |= l.type == OP_SYN_SCATTER && l.syn_probe;
  } else {
    build_launches(s, p.lowered, s->launches, p.probe_src_rows, &s->probe_src);
  }
  s->probe_rows = (int32_t)p.probe_src_rows.size();
  s->ctr = dev_alloc<int64_t>(2);
  HIPCHECK(hipMemset(s->ctr, 0, 2 * sizeof(int64_t)));
  HIPCHECK(hipMemset(s->state, 0, std::max<size_t>(1, s->state_rows) * B * sizeof(float)));
}

// -------------------------------------------------------------- launching
constexpr int kBlock = 256;
// Timing kinds beyond the operator types: the launches of a training step's
// backward pass (weight gradients, adjoints of product inputs, the rest).
constexpr int32_t kTimeGradW = OP_NTYPES, kTimeGradX = OP_NTYPES + 1, kTimeGradOther = OP_NTYPES + 2;
constexpr int32_t kTimeGradWSmall = OP_NTYPES + 3;
constexpr int32_t kTimedTypes = OP_NTYPES + 4;
static_assert(kTimeGradW == MS_OP_GRAD_WEIGHTS && kTimeGradX == MS_OP_GRAD_INPUTS &&
                  kTimeGradOther == MS_OP_GRAD_OTHER && kTimeGradWSmall == MS_OP_GRAD_WEIGHTS_SMALL,
              "timing kinds match the C ABI");

inline unsigned grid_for(int64_t n) { return (unsigned)std::max<int64_t>(1, (n + kBlock - 1) / kBlock); }

// Timing brackets around one launch of type `type` on stream q (no-ops unless
// timing is on).
// The next pair of timing events, for a launch of operator type `type`.
void time_slot(ms_sim* s, int32_t type) {
  if (2 * (s->tn + 1) > s->tev.size()) {
    for (int k = 0; k < 2; ++k) {
      hipEvent_t e = nullptr;
      HIPCHECK(hipEventCreate(&e));
      s->tev.push_back(e);
    }
  }
  if (s->ttype.size() <= s->tn) s->ttype.resize(s->tn + 1);
  s->ttype[s->tn] = type;
}

void time_begin(ms_sim* s, int32_t type, hipStream_t q) {
  if (!s->timing) return;
  time_slot(s, type);
  HIPCHECK(hipEventRecord(s->tev[2 * s->tn], q));
}

void time_end(ms_sim* s, hipStream_t q) {
  if (!s->timing) return;
  HIPCHECK(hipEventRecord(s->tev[2 * s->tn + 1], q));
  ++s->tn;
}

// Timing of one group of the launch drivers: its kernels are launched with
// hipExtLaunchKernelGGL, the first recording the begin event when it starts
// and each recording the end event when it ends (the last one counts), so
// that the interval is the group's execution, without the host's launch
// latency (which the stream-ordered driver would otherwise add whenever the
// GPU waits for the next launch).
void time_group_begin(ms_sim* s, int32_t type) {
  if (!s->timing) return;
  time_slot(s, type);
  s->tx = true;
  s->tx_first = true;
  s->tx_start = s->tev[2 * s->tn];
  s->tx_stop = s->tev[2 * s->tn + 1];
}

void time_group_end(ms_sim* s) {
  if (!s->timing) return;
  s->tx = false;
  ++s->tn;
}

// Kernel launch of a merged group: plain, or with the timing events of
// time_group_begin.
#define KL(kern, grid, block, lds, stream, ...)                                                          \
  do {                                                                                                  \
    if (s->tx) {                                                                                        \
      hipExtLaunchKernelGGL(kern, grid, block, lds, stream, s->tx_first ? s->tx_start : nullptr,        \
                            s->tx_stop, 0, __VA_ARGS__);                                               \
      s->tx_first = false;                                                                              \
    } else {                                                                                            \
      hipLaunchKernelGGL(kern, grid, block, lds, stream, __VA_ARGS__);                                  \
    }                                                                                                   \
  } while (0)

void launch_group(ms_sim* s, const Launch& l, int32_t du) {
  const int32_t B = s->B;
  if ((double)l.rows * (l.type == OP_DOT_INC ? l.M : 1) * B >= 4294967296.0)
    fail(MS_E_INVALID, "merged group too large for 32-bit work-item indexing");
  float* st = s->state;
  const Strides S = s->S;
  hipStream_t q = s->stream;
  if (l.rows == 0) return;
  const int64_t n = l.rows * B;
  switch (l.type) {
    case OP_FEED:
      KL(k_feed, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.dst,
                         l.feed_rows, (const float*)s->feed_stage, s->plan->ir.feed_rows, s->ctr, du);
      break;
    case OP_RESET:
      KL(k_reset, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.dst, l.values);
      break;
    case OP_COPY:
      KL(k_copy, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.dst,
                         l.src_base, l.src, (int)l.src_bcast);
      break;
    case OP_COPY_INC:
      KL(k_copy_inc, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.dst,
                         l.src_base, l.src, (int)l.src_bcast, l.ptr);
      break;
    case OP_ELEM_INC:
      KL(k_elem_inc, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.dst,
                         l.a_base, l.a, l.src_base, l.src, l.ptr);
      break;
    case OP_DOT_INC: {
      if (l.K >= 64 && B <= 4) {
        const int64_t waves = l.rows * (int64_t)l.M;
        KL(k_dot_inc_wave, dim3(grid_for(waves * 64)), dim3(kBlock), 0, q, st, S, B, l.rows,
                           l.M, l.K, l.a_base, l.w_row, l.x_row, l.d_row);
      } else {
        const int64_t work = l.rows * (int64_t)l.M * B;
        KL(k_dot_inc, dim3(grid_for(work)), dim3(kBlock), 0, q, st, S, B, l.rows, l.M, l.K,
                           l.a_base, l.w_row, l.x_row, l.d_row);
      }
      break;
    }
    case OP_LIF:
      KL(k_lif, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.src, l.dst,
                         l.V, l.ref, l.np, s->dt);
      break;
    case OP_LIF_RATE:
      KL(k_lif_rate, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.src,
                         l.dst, l.np);
      break;
    case OP_LOWPASS:
      KL(k_lowpass, dim3(grid_for(n)), dim3(kBlock), 0, q, st, S, B, l.rows, l.dst,
                         l.src, l.fp);
      break;
    case OP_SYN_SCATTER: {
      // one wavefront per (segment, batch column)
      const double items = (double)l.rows * 64 * B;
      if (items >= 4294967296.0) fail(MS_E_INVALID, "fused synapse group too large for 32-bit indexing");
      if (B == 1 && S.rs == 1)
        KL(k_syn_scatter<true>, dim3(grid_for((int64_t)items)), dim3(kBlock), 0, q, st, S, B,
                           (int32_t)l.rows, l.syn_seg, l.syn_conn, l.syn_w, l.syn_update,
                           l.syn_probe ? s->probe_buf : nullptr, s->probe_rows, (const float*)s->feed_stage,
                           s->plan->ir.feed_rows, (const int64_t*)s->ctr, du);
      else
        KL(k_syn_scatter<false>, dim3(grid_for((int64_t)items)), dim3(kBlock), 0, q, st, S, B,
                           (int32_t)l.rows, l.syn_seg, l.syn_conn, l.syn_w, l.syn_update,
                           l.syn_probe ? s->probe_buf : nullptr, s->probe_rows, (const float*)s->feed_stage,
                           s->plan->ir.feed_rows, (const int64_t*)s->ctr, du);
      break;
    }
    case OP_BDOT_INC:
    case OP_PES:
    case OP_PES_FUSED: {
      const int64_t MB = (int64_t)l.M * B;
      const dim3 grid((unsigned)((MB + 255) / 256), (unsigned)l.pes_nch, (unsigned)l.rows);
      const size_t lds = (size_t)2 * l.pes_L * B * sizeof(float);
      const PesOps P{l.w_row, l.x_row, l.d_row, l.e_row, l.act_row, l.coef};
      if (l.type == OP_BDOT_INC)
        KL(k_pes<0>, grid, dim3(256), lds, q, st, B, l.M, l.K, l.pes_L, P, s->pes_part, l.pes_nch);
      else if (l.type == OP_PES)
        KL(k_pes<1>, grid, dim3(256), lds, q, st, B, l.M, l.K, l.pes_L, P, s->pes_part, l.pes_nch);
      else
        KL(k_pes<2>, grid, dim3(256), lds, q, st, B, l.M, l.K, l.pes_L, P, s->pes_part, l.pes_nch);
      if (l.type != OP_PES) {
        HIPCHECK(hipGetLastError());
        KL(k_pes_reduce, dim3((unsigned)((MB + 31) / 32), (unsigned)l.rows), dim3(256), 0, q, st,
                           B, l.M, l.d_row, (const float*)s->pes_part, l.pes_nch);
      }
      break;
    }
    case OP_ENS: {
      // many neurons per op, no fused decoders, few batch columns: neuron
      // chunks of every op run in parallel, the batch in registers
      int32_t nw = 16;   // wavefronts per workgroup, within 64 KB of LDS
      while (nw >= 4 && (size_t)(l.ens.d + 64 * nw) * B * sizeof(float) > 65536) nw /= 2;
      if (B <= kBigCols && l.ens.ndec == 0 && l.ens.encT && l.ens_nmax >= 512 && nw >= 4 &&
          S.rs == B && S.cs == 1 && l.rows <= 65535) {
        const size_t big_lds = (size_t)(l.ens.d + 64 * nw) * B * sizeof(float);
        KL(k_ens_big, dim3((unsigned)((l.ens_nmax + kBigNeurons - 1) / kBigNeurons), (unsigned)l.rows),
                           dim3(64 * nw), big_lds, q, st, B, l.ens, s->dt);
      } else if (B >= 32) {
        KL(k_ens_tile, dim3((unsigned)l.rows, (unsigned)((B + 63) / 64)), dim3(256), 0, q, st, S,
                           B, l.ens, s->dt);
      } else if (l.ens.decT) {
        KL(k_ens_wg<true>, dim3((unsigned)l.rows, (unsigned)B), dim3(256), 0, q, st, S, l.ens, s->dt);
      } else {
        KL(k_ens_wg<false>, dim3((unsigned)l.rows, (unsigned)B), dim3(256), 0, q, st, S, l.ens, s->dt);
      }
      break;
    }
    default: fail(MS_E_INVALID, "unknown group type");
  }
}

// One timestep: the groups in plan order, then the probes.  The step is the
// du-th after the last advance of the device step counter; with advance set,
// the counter moves past this step afterwards (so a hipGraph of U steps
// advances it once, by U).
void launch_step(ms_sim* s, int32_t du = 0, bool advance = true) {
  for (const Launch& l : s->launches) {
    const bool t = s->driver == MS_DRIVER_STEPS && l.rows > 0;
    if (t) time_group_begin(s, l.type);
    launch_group(s, l, du);
    if (t) time_group_end(s);
  }
  const int64_t n = (int64_t)s->probe_rows * s->B;
  if (n > 0 && !s->probe_folded)
    hipLaunchKernelGGL(k_probe, dim3(grid_for(n)), dim3(kBlock), 0, s->stream, (const float*)s->state,
                       s->S, s->B, s->probe_rows, s->probe_src, s->probe_buf, s->ctr, du);
  if (advance) hipLaunchKernelGGL(k_advance, dim3(1), dim3(64), 0, s->stream, s->ctr, du + 1);
}

void ensure_graph(ms_sim* s) {
  if (s->graph_valid) return;
  destroy_graph(s);
  HIPCHECK(hipStreamBeginCapture(s->stream, hipStreamCaptureModeThreadLocal));
  try {
    for (int32_t u = 0; u < s->unroll; ++u) launch_step(s, u, u + 1 == s->unroll);
  } catch (...) {
    hipGraph_t g = nullptr;
    (void)hipStreamEndCapture(s->stream, &g);
    if (g) (void)hipGraphDestroy(g);
    throw;
  }
  HIPCHECK(hipStreamEndCapture(s->stream, &s->graph));
  HIPCHECK(hipGraphInstantiate(&s->graph_exec, s->graph, nullptr, nullptr, 0));
  s->graph_valid = true;
}

void ensure_capacity(ms_sim* s, int64_t n_steps) {
  const int32_t B = s->B;
  const int32_t fr = s->plan->ir.feed_rows;
  if (n_steps > s->feed_cap) {
    int64_t cap = std::max<int64_t>(n_steps, s->feed_cap * 2);
    if (s->feed_stage) HIPCHECK(hipFree(s->feed_stage));
    s->feed_stage = dev_alloc<float>(std::max<size_t>(1, (size_t)cap * fr * B));
    s->feed_cap = cap;
    destroy_graph(s);
    s->persistent_ok = false;
  }
  const int64_t need = s->steps_total + n_steps;
  if (need > s->probe_cap) {
    int64_t cap = std::max<int64_t>(need, s->probe_cap * 2);
    float* nb = dev_alloc<float>(std::max<size_t>(1, (size_t)cap * s->probe_rows * B));
    if (s->probe_buf) {
      if (s->steps_total > 0)
        HIPCHECK(hipMemcpyAsync(nb, s->probe_buf, (size_t)s->steps_total * s->probe_rows * B * 4,
                                hipMemcpyDeviceToDevice, s->stream));
      HIPCHECK(hipStreamSynchronize(s->stream));
      HIPCHECK(hipFree(s->probe_buf));
    }
    s->probe_buf = nb;
    if (s->bit_words > 0) {
      const size_t words = (size_t)s->bit_words * B;
      uint32_t* nbits = dev_alloc<uint32_t>((size_t)cap * words);
      if (s->bits_buf) {
        if (s->steps_total > 0)
          HIPCHECK(hipMemcpyAsync(nbits, s->bits_buf, (size_t)s->steps_total * words * 4, hipMemcpyDeviceToDevice,
                                  s->stream));
        HIPCHECK(hipStreamSynchronize(s->stream));
        HIPCHECK(hipFree(s->bits_buf));
      }
      s->bits_buf = nbits;
    }
    s->probe_cap = cap;
    destroy_graph(s);
    s->persistent_ok = false;
  }
}

// Failure detection (ms_sim_set_check_feeds): a feed holding NaN or Inf is
// refused before anything runs; host feeds are scanned on the host, device
// feeds by a counting kernel.
void check_feed(ms_sim* s, const ms_feed& f, size_t elems) {
  int64_t bad = 0;
  if (!f.on_device) {
    for (size_t k = 0; k < elems; ++k) bad += std::isfinite(f.data[k]) ? 0 : 1;
  } else {
    if (!s->nonfinite) s->nonfinite = dev_alloc<unsigned int>(1);
    HIPCHECK(hipMemsetAsync(s->nonfinite, 0, sizeof(unsigned int), s->stream));
    const unsigned blocks = (unsigned)std::min<size_t>(1024, (elems + kBlock - 1) / kBlock);
    hipLaunchKernelGGL(k_count_nonfinite, dim3(std::max(1u, blocks)), dim3(kBlock), 0, s->stream, f.data,
                       (int64_t)elems, s->nonfinite);
    unsigned int h = 0;
    HIPCHECK(hipMemcpyAsync(&h, s->nonfinite, sizeof(h), hipMemcpyDeviceToHost, s->stream));
    HIPCHECK(hipStreamSynchronize(s->stream));
    bad = h;
  }
  if (bad)
    fail(MS_E_NUMERIC, "feed for node " + std::to_string(f.node_id) + " holds " + std::to_string(bad) +
                           " non-finite values (NaN or Inf)");
}

void stage_feeds(ms_sim* s, int64_t n_steps, const ms_feed* feeds, int32_t n_feeds) {
  const IR& ir = s->plan->ir;
  const int32_t B = s->B;
  const int32_t fr = ir.feed_rows;
  if (fr == 0) return;
  if (s->check_feeds)
    for (int32_t i = 0; i < n_feeds; ++i) {
      const ms_feed& f = feeds[i];
      if (f.node_id < 0 || f.node_id >= (int32_t)ir.node_size.size() || !f.data) continue;   // refused below
      check_feed(s, f, (size_t)B * n_steps * ir.node_size[f.node_id]);
    }
  HIPCHECK(hipMemsetAsync(s->feed_stage, 0, (size_t)n_steps * fr * B * 4, s->stream));
  for (int32_t i = 0; i < n_feeds; ++i) {
    const ms_feed& f = feeds[i];
    if (f.node_id < 0 || f.node_id >= (int32_t)ir.feed_row_of_node.size() || ir.feed_row_of_node[f.node_id] < 0)
      fail(MS_E_INVALID, "feed for node " + std::to_string(f.node_id) + ", which is not an input node");
    if (!f.data) fail(MS_E_INVALID, "feed data is NULL");
    const int32_t nsize = ir.node_size[f.node_id];
    const size_t elems = (size_t)B * n_steps * nsize;
    const float* src = f.data;
    if (!f.on_device) {
      if (elems > s->feed_tmp_elems) {
        HIPCHECK(hipStreamSynchronize(s->stream));
        if (s->feed_tmp) HIPCHECK(hipFree(s->feed_tmp));
        s->feed_tmp = dev_alloc<float>(elems);
        s->feed_tmp_elems = elems;
      }
      HIPCHECK(hipMemcpyAsync(s->feed_tmp, f.data, elems * 4, hipMemcpyHostToDevice, s->stream));
      src = s->feed_tmp;
    }
    for (int64_t t_off = 0; t_off < n_steps; t_off += 65535) {   // grid z is at most 65535
      const int64_t nt = std::min<int64_t>(65535, n_steps - t_off);
      hipLaunchKernelGGL(k_stage_feed, dim3((unsigned)((nsize + 31) / 32), (unsigned)((B + 31) / 32), (unsigned)nt),
                         dim3(32, 8), 0, s->stream, src, B, n_steps, nsize, s->feed_stage, fr,
                         ir.feed_row_of_node[f.node_id], t_off);
    }
    if (!f.on_device) HIPCHECK(hipStreamSynchronize(s->stream));   // feed_tmp reused
  }
}

const std::vector<float>& host_param_base(ms_sim* s, int32_t base) {
  if (base < 0 || base >= (int32_t)s->host_bases.size() || s->host_bases[base].empty())
    fail(MS_E_INVALID, "parameter base not available on the host");
  return s->host_bases[base];
}

// Weight bytes read per step (every parameter base array).
int64_t param_bytes(const Plan& p) {
  int64_t n = 0;
  for (size_t b = 0; b < p.ir.bases.size(); ++b)
    if (p.ir.bases[b].cls != SC_BATCHED) n += p.base_rows[b] * p.ir.bases[b].cols * 4;
  return n;
}

// Stage-major when the model has no recurrence beyond each neuron's and filter's
// own state; otherwise the persistent per-column driver when one workgroup can
// hold a column's whole step cheaply (small weights, modest state), else
// launches.
bool has_learning(const Plan& p) {
  for (const Op& o : p.ir.ops) if (o.type == OP_PES) return true;
  return false;
}

int32_t choose_driver(const Plan& p, int32_t B, int32_t requested) {
  if (requested != MS_DRIVER_AUTO) return requested;
  if (has_learning(p)) return MS_DRIVER_GRAPH;
  if (make_window_plan(p).ok) return MS_DRIVER_WINDOW;
  const int64_t rows = p.base_rows.empty() ? 0 : p.base_rows[0];
  const int64_t wbytes = param_bytes(p);
  if (wbytes <= (1 << 20) && rows <= (1 << 17) && (B >= 8 || rows <= 8192)) return MS_DRIVER_PERSISTENT;
  return MS_DRIVER_GRAPH;
}

void setup_persistent(ms_sim* s) {
  s->persistent_threads = s->state_rows <= 4096 ? 256 : 1024;
  std::vector<GroupDesc> gd;
  for (size_t gi = 0; gi < s->launches.size(); ++gi) {
    const Launch& l = s->launches[gi];
    GroupDesc g{};
    g.type = l.type; g.M = l.M; g.K = l.K; g.bcast = l.src_bcast ? 1 : 0; g.rows = l.rows;
    g.tpr = 1;
    if (l.type == OP_DOT_INC) {
      // transposed copy of every op's [M][K] block, [K][M], in one buffer
      const int64_t blk = (int64_t)l.M * l.K;
      std::vector<float> wt((size_t)(blk * l.rows));
      std::vector<int64_t> off((size_t)l.rows);
      std::vector<int32_t> wrow((size_t)l.rows);
      HIPCHECK(hipMemcpy(wrow.data(), l.w_row, wrow.size() * 4, hipMemcpyDeviceToHost));
      const LGroup& lg = s->plan->lowered[gi];
      const std::vector<float>& host_w = host_param_base(s, lg.a.base);
      const int64_t cols = s->plan->ir.bases[lg.a.base].cols;
      for (int64_t op = 0; op < l.rows; ++op) {
        off[op] = op * blk;
        for (int32_t m = 0; m < l.M; ++m)
          for (int32_t k = 0; k < l.K; ++k)
            wt[(size_t)(op * blk + (int64_t)k * l.M + m)] =
                host_w[(size_t)(((int64_t)wrow[op] + m) * cols + (cols == 1 ? 0 : k)) + (cols == 1 ? k : 0)];
      }
      float* dwt = dev_alloc<float>(std::max<size_t>(1, wt.size()));
      int64_t* doff = dev_alloc<int64_t>(std::max<size_t>(1, off.size()));
      HIPCHECK(hipMemcpy(dwt, wt.data(), wt.size() * 4, hipMemcpyHostToDevice));
      HIPCHECK(hipMemcpy(doff, off.data(), off.size() * 8, hipMemcpyHostToDevice));
      s->extra_allocs.push_back(dwt);
      s->extra_allocs.push_back(doff);
      g.wt_base = dwt;
      g.wt_off = doff;
      const int64_t out_rows = l.rows * (int64_t)l.M;
      while (g.tpr < 64 && out_rows * g.tpr * 2 <= s->persistent_threads && g.tpr * 2 <= l.K) g.tpr *= 2;
      s->scratch_n = std::max<int64_t>(s->scratch_n, out_rows * g.tpr);
    }
    g.dst = l.dst; g.src = l.src; g.a = l.a; g.V = l.V; g.ref = l.ref;
    g.src_base = l.src_base; g.a_base = l.a_base; g.ptr = l.ptr; g.values = l.values;
    g.w_row = l.w_row; g.x_row = l.x_row; g.d_row = l.d_row; g.feed_row = l.feed_rows;
    g.np = l.np; g.fp = l.fp; g.ens = l.ens;
    gd.push_back(g);
  }
  int lds_max = 0;
  HIPCHECK(hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, s->device));
  s->lds_limit = (size_t)lds_max;
  if (s->lds_limit > 65536)
    HIPCHECK(hipFuncSetAttribute((const void*)k_persistent<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)s->lds_limit));
  s->prog.n_groups = (int32_t)gd.size();
  s->prog.groups = dev_alloc<GroupDesc>(std::max<size_t>(1, gd.size()));
  if (!gd.empty())
    HIPCHECK(hipMemcpy(s->prog.groups, gd.data(), gd.size() * sizeof(GroupDesc), hipMemcpyHostToDevice));
}

void run_persistent(ms_sim* s, int64_t n_steps) {
  const int64_t rows = (int64_t)std::max<size_t>(1, s->state_rows);
  const int threads = s->persistent_threads;
  const size_t lds = (size_t)(rows + s->scratch_n) * sizeof(float);
  if (lds <= s->lds_limit) {
    hipLaunchKernelGGL(k_persistent<true>, dim3(s->B), dim3(threads), lds, s->stream, s->state, rows, s->B,
                       (const GroupDesc*)s->prog.groups, s->prog.n_groups, n_steps, s->dt,
                       (const float*)s->feed_stage, s->plan->ir.feed_rows, s->probe_src, s->probe_rows,
                       s->probe_buf, s->steps_total, s->col_scratch, s->scratch_n);
  } else {
    if (!s->col_scratch && s->scratch_n > 0) s->col_scratch = dev_alloc<float>((size_t)s->scratch_n * s->B);
    hipLaunchKernelGGL(k_persistent<false>, dim3(s->B), dim3(threads), 0, s->stream, s->state, rows, s->B,
                       (const GroupDesc*)s->prog.groups, s->prog.n_groups, n_steps, s->dt,
                       (const float*)s->feed_stage, s->plan->ir.feed_rows, s->probe_src, s->probe_rows,
                       s->probe_buf, s->steps_total, s->col_scratch, s->scratch_n);
  }
  hipLaunchKernelGGL(k_set_ctr, dim3(1), dim3(64), 0, s->stream, s->ctr, s->steps_total + n_steps, n_steps);
}

// ------------------------------------------------------------ window driver
constexpr double kWindowBytes = 16.0 * (1 << 30);  // budget for the versioned signals (of 288 GB HBM)
constexpr int32_t kMaxWindow = 1024;

// Launch shape of a fused-ensemble phase: threads cover the largest op's
// neurons (at most 4 per thread), LDS holds a sub-window of inputs and outputs.
void ens_shape(ms_sim* s, Launch& l, const LGroup& g) {
  int32_t nmax = 1;
  for (int32_t n : g.ens_n) nmax = std::max(nmax, n);
  l.nmax = nmax;
  // batch columns per workgroup: one when the weights-in-registers kernel
  // applies (at most 512 neurons, d and decoded dimensions at most 16: its
  // sub-window needs one barrier; 128 product ensembles of 100 neurons,
  // minibatch 64, 1000 steps: 2.0 ms per run against 2.5 with 2 columns per
  // workgroup and weights in LDS); otherwise fill up to 256 threads (4
  // wavefronts) with whole columns, and an ensemble of more neurons takes one
  // column and up to 512 threads.  Small workgroups let a CU interleave more of
  // them around each one's barriers (2 columns per workgroup ran 1.47 ms
  // against 1.76 ms with 5)
  const bool rw_shape = nmax <= 512 && std::max<int32_t>(1, l.ens.d) <= 16 && l.ens.ndec <= 16;
  l.cpw = rw_shape ? 1 : (int32_t)std::max<int64_t>(1, std::min<int64_t>(s->B, 256 / nmax));
  l.nthr = (int32_t)std::min<int64_t>(512, ((int64_t)nmax * l.cpw + 63) / 64 * 64);
  l.npt = (int32_t)(((int64_t)nmax * l.cpw + l.nthr - 1) / l.nthr);
  if (l.npt > 8) fail(MS_E_INVALID, "ensemble too large for the window driver (more than 4096 neurons)");
  if (l.ens.d >= 32768 || l.ens.ndec >= 32768) fail(MS_E_INVALID, "ensemble dimensions too large for the window driver");
  l.npt = l.npt <= 1 ? 1 : l.npt <= 2 ? 2 : l.npt <= 4 ? 4 : 8;
  const int64_t nw = l.nthr / 64, dp = std::max<int32_t>(1, l.ens.d);
  // LDS row strides: inputs and currents are read and written by lanes 16
  // columns apart; padding the rows spreads those lanes over the banks
  l.xs = stride2mod4((int32_t)(4 * ((dp + 3) / 4)));   // whole k steps of 4
  l.js = nmax % 2 == 0 ? nmax + 1 : nmax;
  // sub-window: the longest (a multiple of 16, at most 64 steps) that keeps
  // about 32 wavefronts per CU resident within the CU's LDS and whose inputs
  // fit the per-thread prefetch registers (if none does, 16 steps, the rest of
  // the inputs loaded without prefetch); decoder products split the neurons
  // into kch chunks so that there are about as many units as wavefronts
  auto kch_of = [&](int64_t ts) { return std::max<int64_t>(1, nw / std::max<int64_t>(1, l.cpw * ts / 16)); };
  // per-op constants staged in LDS: biases always; encoders and decoders when
  // small (otherwise they are read through the caches)
  l.enc_lds = (int64_t)nmax * dp * 4 <= 16384 ? 1 : 0;
  l.dec_lds = (int64_t)l.ens.ndec * nmax * 4 <= 16384 ? 1 : 0;
  const int64_t consts = nmax + (l.enc_lds ? (int64_t)nmax * l.xs : 0) +
                        (l.dec_lds ? (int64_t)l.ens.ndec * stride2mod4(nmax) : 0);
  if (!g.ens_chain.empty() && (l.cpw != 1 || l.npt != 1))
    fail(MS_E_INVALID, "fused connection chain needs one column per workgroup and one neuron per thread");
  // fused connection chains keep the transform and filter fragments in LDS
  const int64_t chain_f = g.ens_chain.empty() ? 0 : 512;
  auto bytes = [&](int64_t ts) {
    const int64_t ncol = l.cpw * ts;
    return (ncol * (l.xs + l.js) + (ncol / 16) * kch_of(ts) * 256 + consts + chain_f) * (int64_t)sizeof(float);
  };
  const int64_t wgs = std::max<int64_t>(1, 32 / nw);
  int64_t ts = 64;
  while (ts > 16 && (bytes(ts) * wgs > (int64_t)s->lds_limit || l.cpw * ts * l.ens.d > (int64_t)kEnsXPre * l.nthr))
    ts -= 16;
  if (bytes(ts) > (int64_t)s->lds_limit) fail(MS_E_INVALID, "ensemble too large for the window driver's LDS staging");
  l.ts = (int32_t)ts;
  l.kch = (int32_t)kch_of(ts);
  l.lds = (size_t)bytes(ts);
  // keep each wavefront's encoder and decoder fragments in registers for the
  // whole window when they fit the kernel's register arrays (at most 4 neuron
  // tiles of 16 per wavefront, d <= 16, at most 16 k steps of 4 per decoder
  // chunk, each wavefront on one chunk), also when they would fit in LDS
  // (one column per workgroup; wavefront w owns neurons 64 w .. 64 w + 63 and
  // their 4 encoder tiles; two input buffers and two sets of per-wavefront
  // partial decodes)
  // (every slot a neuron row of the products: rows of nthr + 1 currents and
  // nthr biases, zero past the op's neurons)
  const int64_t ntile = ((int64_t)nmax + 15) / 16, rw_js = l.nthr + 1;
  const int64_t rw_lds = (2 * ts * l.xs + ts * rw_js + 2 * nw * (ts / 16) * 256 + l.nthr + chain_f) * (int64_t)sizeof(float);
  if (l.npt == 1 && l.cpw == 1 && ntile <= 4 * nw && dp <= 16 && l.ens.ndec <= 16 &&
      rw_lds <= (int64_t)s->lds_limit) {
    l.rw = 1;
    l.enc_lds = l.dec_lds = 0;
    l.js = (int32_t)rw_js;
    l.lds = (size_t)rw_lds;
  }
}

// Steps per window for a run of n_steps: as many as the run needs, up to the
// memory budget; the versioned array is reallocated (keeping block 0, the
// carried state) when a longer window is wanted.  Blocks 1..W are always
// written before they are read; block 0 starts at zero.
void ensure_window(ms_sim* s, int64_t n_steps) {
  const WindowPlan& w = *s->wplan;
  const int32_t B = s->B;
  const double per_step = (double)std::max<int64_t>(1, w.rows_v) * B * sizeof(float);
  const int64_t cap = (int64_t)std::max<double>(1.0, std::min<double>(kMaxWindow, std::floor(kWindowBytes / per_step) - 1));
  const int32_t want = (int32_t)std::min<int64_t>(cap, std::max<int64_t>(1, n_steps));
  if (s->va && want <= s->W) return;
  const int64_t rows = std::max<int64_t>(1, w.rows_v);
  const int64_t vs = (int64_t)(want + 1) * B;
  float* nva = dev_alloc<float>((size_t)rows * vs);
  HIPCHECK(hipMemsetAsync(nva, 0, (size_t)rows * vs * sizeof(float), s->stream));
  if (s->va) {
    HIPCHECK(hipMemcpy2DAsync(nva, vs * 4, s->va, s->vs * 4, (size_t)B * 4, rows, hipMemcpyDeviceToDevice, s->stream));
    HIPCHECK(hipStreamSynchronize(s->stream));
    HIPCHECK(hipFree(s->va));
  }
  s->va = nva;
  s->W = want;
  s->vs = vs;
}

// fp32 -> bf16, round to nearest even (NaN stays NaN)
uint16_t bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x7fffffu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Products that run on bf16 MFMA when the simulator asks for bf16 GEMMs: merged
// DotInc groups with constant weights, M >= 64, K >= 16, K % 8 == 0 and
// B % 4 == 0 (the others keep fp32).
bool bf16_product(const ms_sim* s, const Launch& l) {
  return l.type == OP_DOT_INC && l.a_bcast && l.M >= 64 && l.K >= 16 && l.K % 8 == 0 && s->B % 4 == 0;
}

// Bit-recorded spike probes: their rows leave the float record (the rows of the
// other probes keep their places in probe_buf) and their bits go to bits_buf,
// each probe padded to whole 32-neuron words.
static void setup_spike_bits(ms_sim* s, const WindowPlan& w) {
  const Plan& p = *s->plan;
  const int32_t pr = (int32_t)w.probe_rows.size();
  if (pr != s->probe_rows) fail(MS_E_INVALID, "window probe rows differ from the plan's");
  std::vector<int32_t> src((size_t)std::max(1, pr));
  if (pr > 0) HIPCHECK(hipMemcpy(src.data(), s->wprobe_src, (size_t)pr * 4, hipMemcpyDeviceToHost));
  std::vector<int32_t> bsrc, fsrc, fdst;
  s->bit_off.assign(p.probe_width.size(), -1);
  for (size_t pi = 0; pi < p.probe_width.size(); ++pi) {
    const int32_t off = p.probe_row_offset[pi], width = p.probe_width[pi];
    if (s->spike_mag[pi] != 0.0f && width > 0) {
      s->bit_off[pi] = (int32_t)(bsrc.size() / 32);
      for (int32_t j = 0; j < width; ++j) bsrc.push_back(src[(size_t)(off + j)]);
      while (bsrc.size() % 32) bsrc.push_back(-1);
    } else {
      for (int32_t j = 0; j < width; ++j) { fsrc.push_back(src[(size_t)(off + j)]); fdst.push_back(off + j); }
    }
  }
  s->bit_words = (int32_t)(bsrc.size() / 32);
  if (s->bit_words == 0) return;
  s->pr_float = (int32_t)fsrc.size();
  s->wbit_src = dev_alloc<int32_t>(bsrc.size());
  HIPCHECK(hipMemcpy(s->wbit_src, bsrc.data(), bsrc.size() * 4, hipMemcpyHostToDevice));
  s->wprobe_fsrc = dev_alloc<int32_t>(std::max<size_t>(1, fsrc.size()));
  s->wprobe_fdst = dev_alloc<int32_t>(std::max<size_t>(1, fdst.size()));
  if (!fsrc.empty()) {
    HIPCHECK(hipMemcpy(s->wprobe_fsrc, fsrc.data(), fsrc.size() * 4, hipMemcpyHostToDevice));
    HIPCHECK(hipMemcpy(s->wprobe_fdst, fdst.data(), fdst.size() * 4, hipMemcpyHostToDevice));
  }
}

void setup_window(ms_sim* s) {
  WindowPlan& w = *s->wplan;
  const int32_t B = s->B;
  if (B > 65535) fail(MS_E_INVALID, "minibatch too large for the window driver");
  int lds_max = 0;
  HIPCHECK(hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, s->device));
  s->lds_limit = (size_t)lds_max;
  HIPCHECK(hipDeviceGetAttribute(&s->n_cu, hipDeviceAttributeMultiprocessorCount, s->device));
  s->pa = dev_alloc<float>((size_t)std::max<int64_t>(1, w.rows_p) * B);
  ensure_window(s, 1);
  for (int k = 0; k < ms_sim::kSide; ++k) HIPCHECK(hipStreamCreateWithFlags(&s->side[k], hipStreamNonBlocking));
  for (int k = 0; k <= ms_sim::kSide; ++k) HIPCHECK(hipEventCreateWithFlags(&s->side_ev[k], hipEventDisableTiming));
  std::vector<LGroup> groups;
  for (const WPhase& ph : w.phases) groups.push_back(ph.g);
  build_launches(s, groups, s->wl, w.probe_rows, &s->wprobe_src);
  if (!s->spike_mag.empty()) setup_spike_bits(s, w);
  for (size_t k = 0; k < s->wl.size(); ++k) {
    Launch& l = s->wl[k];
    l.src_blk = w.phases[k].src_blk;
    l.a_blk = w.phases[k].a_blk;
    if (l.type == OP_ENS) {
      ens_shape(s, l, w.phases[k].g);
    }
    if (s->gemm_dtype == MS_GEMM_BF16 && bf16_product(s, l)) {
      // each op's [M][K] block of W, rounded to nearest even, packed op after op
      const LGroup& g = w.phases[k].g;
      const std::vector<float>& hw = host_param_base(s, g.a.base);
      std::vector<uint16_t> w16((size_t)l.rows * l.M * l.K);
      for (int64_t op = 0; op < l.rows; ++op)
        for (int64_t e = 0; e < (int64_t)l.M * l.K; ++e)
          w16[(size_t)(op * l.M * l.K + e)] = bf16_rne(hw[(size_t)((int64_t)g.w_row[op] * l.K + e)]);
      uint16_t* d = dev_alloc<uint16_t>(w16.size());
      s->extra_allocs.push_back(d);
      HIPCHECK(hipMemcpy(d, w16.data(), w16.size() * sizeof(uint16_t), hipMemcpyHostToDevice));
      l.w16 = d;
    }
  }
  if (s->lds_limit > 65536) {
    const void* wens[] = {(const void*)k_w_ens<1, false, false>, (const void*)k_w_ens<2, false, false>,
                          (const void*)k_w_ens<4, false, false>, (const void*)k_w_ens<8, false, false>,
                          (const void*)k_w_ens<1, true, false>,  (const void*)k_w_ens<1, false, true>,
                          (const void*)k_w_ens<1, true, true>};
    for (const void* f : wens)
      HIPCHECK(hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)s->lds_limit));
  }
  HIPCHECK(hipMemset(s->pa, 0, (size_t)std::max<int64_t>(1, w.rows_p) * B * sizeof(float)));
}

inline unsigned grid_items(double n) {
  if (n >= 4294967296.0) fail(MS_E_INVALID, "window phase too large for 32-bit work-item indexing");
  return (unsigned)std::max<int64_t>(1, ((int64_t)n + kBlock - 1) / kBlock);
}

// va: the versioned array the phase works on (null: the simulation's; the
// training pass runs products on the adjoints)
void launch_phase(ms_sim* s, const Launch& l, int32_t T, int64_t t0, hipStream_t q, float* va = nullptr) {
  if (l.rows == 0) return;
  const WView w{va ? va : s->va, s->vs, s->B, T};
  const double tb = (double)T * s->B;
  switch (l.type) {
    case OP_FEED:
      if (s->B % 4 == 0)
        hipLaunchKernelGGL(k_w_feed4, dim3(grid_items(l.rows * tb / 4)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.feed_rows, (const float*)s->feed_stage, s->plan->ir.feed_rows, t0);
      else
        hipLaunchKernelGGL(k_w_feed, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.feed_rows, (const float*)s->feed_stage, s->plan->ir.feed_rows, t0);
      break;
    case OP_RESET:
      if (s->B % 4 == 0)   // 16-byte aligned rows of every block: four entries per thread
        hipLaunchKernelGGL(k_w_reset4, dim3(grid_items(l.rows * tb / 4)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.values);
      else
        hipLaunchKernelGGL(k_w_reset, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, l.rows, l.dst, l.values);
      break;
    case OP_COPY:
      hipLaunchKernelGGL(k_w_copy, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                         l.src_base, l.src, (int)l.src_bcast, l.src_blk);
      break;
    case OP_COPY_INC:
      if (s->B % 4 == 0)
        hipLaunchKernelGGL(k_w_copy_inc4, dim3(grid_items(l.rows * tb / 4)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.src_base, l.src, (int)l.src_bcast, l.src_blk, l.ptr);
      else
        hipLaunchKernelGGL(k_w_copy_inc, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.src_base, l.src, (int)l.src_bcast, l.src_blk, l.ptr);
      break;
    case OP_ELEM_INC:
      if (s->B % 4 == 0)
        hipLaunchKernelGGL(k_w_elem_inc4, dim3(grid_items(l.rows * tb / 4)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.a_base, l.a, (int)l.a_bcast, l.a_blk, l.src_base, l.src, (int)l.src_bcast, l.src_blk,
                           l.ptr);
      else
        hipLaunchKernelGGL(k_w_elem_inc, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, l.rows, l.dst,
                           l.a_base, l.a, (int)l.a_bcast, l.a_blk, l.src_base, l.src, (int)l.src_bcast, l.src_blk,
                           l.ptr);
      break;
    case OP_DOT_INC:
      if (l.w16 || (l.K > 128 && l.M >= 64 && l.K % 4 == 0 && s->B % 4 == 0)) {
        // 128 x 128 tiles in XCD order: one flat grid padded to a multiple of 8.
        // Products with K <= 128 are bound by their output traffic and run
        // faster on the 64 x 64 tiles below (more workgroups in flight).
        const int32_t mtiles = (l.M + kG2M - 1) / kG2M;
        const double ntiles = std::ceil(tb / kG2N);
        const double total = ntiles * mtiles * (double)l.rows;
        if (total >= 2147483648.0 - 8) fail(MS_E_INVALID, "window product too large for the GEMM grid");
        if (l.w16) {
          const unsigned grid = (unsigned)(8 * (((int64_t)total + 7) / 8));
          hipLaunchKernelGGL(k_w_gemm_bf16, dim3(grid), dim3(256), 0, q, w, l.M, l.K, mtiles, (int32_t)ntiles,
                             (int32_t)l.rows, l.w16, l.x_row, l.d_row, l.src_blk);
        } else {
          // tail split: when every tile is resident at once (at most 4 per CU)
          // and the count is not a whole multiple of the CUs, the column tiles
          // beyond the last whole multiple run as 64 x 64 tiles
          const int64_t ncu = std::max<int32_t>(1, s->n_cu), tiles = (int64_t)total;
          const int64_t per_col = (int64_t)mtiles * l.rows;
          int64_t nbig = (int64_t)ntiles, small = 0;
          if (tiles > ncu && tiles <= 4 * ncu && tiles % ncu != 0) {
            const int64_t nb = (tiles / ncu) * ncu / per_col;
            if (nb >= 1 && nb < nbig) {
              nbig = nb;
              small = (int64_t)((l.M + kGemmBM - 1) / kGemmBM) * l.rows *
                      (((int64_t)tb - nb * kG2N + kGemmBN - 1) / kGemmBN);
            }
          }
          const int64_t gbig = 8 * ((nbig * per_col + 7) / 8);
          const unsigned grid = (unsigned)(gbig + 8 * ((small + 7) / 8));
          hipLaunchKernelGGL(k_w_gemm2, dim3(grid), dim3(256), 0, q, w, l.M, l.K, mtiles, (int32_t)nbig,
                             (int32_t)l.rows, l.a_base, l.w_row, l.x_row, l.d_row, l.src_blk, (uint32_t)gbig);
        }
      } else if (l.M <= kSkM && l.K >= 256) {
        const double ctiles = std::ceil(tb / 64);
        if (ctiles * l.rows >= 2147483648.0) fail(MS_E_INVALID, "window product too large for the grid");
        hipLaunchKernelGGL(k_w_skinny, dim3((unsigned)(ctiles * l.rows)), dim3(64 * kSkW), 0, q, w, l.M, l.K,
                           (int32_t)ctiles, l.a_base, l.w_row, l.x_row, l.d_row, l.src_blk);
      } else if (l.K >= 16) {
        const int32_t mtiles = (l.M + kGemmBM - 1) / kGemmBM;
        const double ntiles = std::ceil(tb / kGemmBN);
        if (ntiles >= 2147483648.0 || (double)mtiles * l.rows > 65535.0)
          fail(MS_E_INVALID, "window product too large for the GEMM grid");
        hipLaunchKernelGGL(k_w_gemm, dim3((unsigned)ntiles, (unsigned)(mtiles * l.rows)), dim3(256), 0, q, w, l.M,
                           l.K, mtiles, l.a_base, l.w_row, l.x_row, l.d_row, l.src_blk);
      } else {
        hipLaunchKernelGGL(k_w_dot, dim3(grid_items((double)l.rows * l.M * tb)), dim3(kBlock), 0, q, w, l.rows,
                           l.M, l.K, l.a_base, l.w_row, l.x_row, l.d_row, l.src_blk);
      }
      break;
    case OP_LIF:
      hipLaunchKernelGGL(k_w_lif, dim3(grid_items((double)l.rows * s->B)), dim3(kBlock), 0, q, w, l.rows, l.src,
                         l.dst, l.V, l.ref, s->pa, l.np, s->dt, l.src_blk);
      break;
    case OP_LIF_RATE:
      hipLaunchKernelGGL(k_w_lif_rate, dim3(grid_items(l.rows * tb)), dim3(kBlock), 0, q, w, l.rows, l.src, l.dst,
                         l.np, l.src_blk);
      break;
    case OP_LOWPASS:
      hipLaunchKernelGGL(k_w_lowpass, dim3(grid_items((double)l.rows * s->B)), dim3(kBlock), 0, q, w, l.rows,
                         l.dst, l.src, l.fp, l.src_blk);
      break;
    case OP_ENS: {
      // one flat grid in XCD order, padded to a multiple of 8
      const int64_t total = l.rows * ((s->B + l.cpw - 1) / l.cpw);
      if (total >= 2147483648LL - 8) fail(MS_E_INVALID, "too many ensemble workgroups");
      const dim3 grid((unsigned)(8 * ((total + 7) / 8)));
      const int32_t nops = (int32_t)l.rows;
#define MS_WENS(NPT, RW, CH)                                                                                    \
  hipLaunchKernelGGL((k_w_ens<NPT, RW, CH>), grid, dim3(l.nthr), l.lds, q, w, s->pa, l.ens, s->dt, l.nmax, l.ts, \
                     l.cpw, l.kch, l.src_blk, l.enc_lds, l.dec_lds, nops, l.xs, l.js)
      const bool ch = l.ens.chain != nullptr;   // fused chains: one neuron per thread (checked by ens_shape)
      if (l.rw && ch) MS_WENS(1, true, true);
      else if (l.rw) MS_WENS(1, true, false);
      else if (ch) MS_WENS(1, false, true);
      else if (l.npt == 1) MS_WENS(1, false, false);
      else if (l.npt == 2) MS_WENS(2, false, false);
      else if (l.npt == 4) MS_WENS(4, false, false);
      else MS_WENS(8, false, false);
#undef MS_WENS
      break;
    }
    default: fail(MS_E_INVALID, "unknown group type");
  }
}

void timed_phase(ms_sim* s, const Launch& l, int32_t T, int64_t t0, hipStream_t q) {
  if (l.rows == 0) return;
  time_begin(s, l.type, q);
  launch_phase(s, l, T, t0, q);
  time_end(s, q);
}

void run_window(ms_sim* s, int64_t n_steps) {
  const WindowPlan& w = *s->wplan;
  ensure_window(s, n_steps);
  for (int64_t t0 = 0; t0 < n_steps; t0 += s->W) {
    const int32_t T = (int32_t)std::min<int64_t>(s->W, n_steps - t0);
    // phases of one level are independent: spread them over the side streams
    for (size_t a = 0; a < s->wl.size();) {
      size_t e = a + 1;
      while (e < s->wl.size() && w.phases[e].level == w.phases[a].level) ++e;
      if (e - a == 1) {
        timed_phase(s, s->wl[a], T, t0, s->stream);
      } else {
        const int used = (int)std::min<size_t>(ms_sim::kSide, e - a - 1);
        HIPCHECK(hipEventRecord(s->side_ev[ms_sim::kSide], s->stream));
        for (int k = 0; k < used; ++k) HIPCHECK(hipStreamWaitEvent(s->side[k], s->side_ev[ms_sim::kSide], 0));
        size_t rr = 0;   // exclusive phases round-robin over the streams; the rest in order on the main stream
        for (size_t i = a; i < e; ++i) {
          if (!w.phases[i].exclusive) { timed_phase(s, s->wl[i], T, t0, s->stream); continue; }
          const size_t slot = rr++ % (size_t)(used + 1);
          timed_phase(s, s->wl[i], T, t0, slot == 0 ? s->stream : s->side[slot - 1]);
        }
        for (int k = 0; k < used; ++k) {
          HIPCHECK(hipEventRecord(s->side_ev[k], s->side[k]));
          HIPCHECK(hipStreamWaitEvent(s->stream, s->side_ev[k], 0));
        }
      }
      a = e;
    }
    const WView v{s->va, s->vs, s->B, T};
    const int32_t pr = (int32_t)w.probe_rows.size();
    if (s->bit_words > 0) {
      if (s->pr_float > 0)
        hipLaunchKernelGGL(k_w_probe_map, dim3(grid_items((double)s->pr_float * T * s->B)), dim3(kBlock), 0,
                           s->stream, v, (const int32_t*)s->wprobe_fsrc, (const int32_t*)s->wprobe_fdst, s->pr_float,
                           pr, s->probe_buf, s->steps_total + t0);
      hipLaunchKernelGGL(k_w_probe_bits, dim3(grid_items((double)s->bit_words * T * s->B)), dim3(kBlock), 0,
                         s->stream, v, (const int32_t*)s->wbit_src, s->bit_words, s->bits_buf, s->steps_total + t0);
    } else if (pr > 0 && s->B % 4 == 0)
      hipLaunchKernelGGL(k_w_probe4, dim3(grid_items((double)pr * T * s->B / 4)), dim3(kBlock), 0, s->stream, v,
                         s->wprobe_src, pr, s->probe_buf, s->steps_total + t0);
    else if (pr > 0)
      hipLaunchKernelGGL(k_w_probe, dim3(grid_items((double)pr * T * s->B)), dim3(kBlock), 0, s->stream, v,
                         s->wprobe_src, pr, s->probe_buf, s->steps_total + t0);
    if (w.rows_v > 0)
      hipLaunchKernelGGL(k_w_carry, dim3(grid_items((double)w.rows_v * s->B)), dim3(kBlock), 0, s->stream, v,
                         w.rows_v);
  }
  hipLaunchKernelGGL(k_set_ctr, dim3(1), dim3(64), 0, s->stream, s->ctr, s->steps_total + n_steps, n_steps);
}

}  // namespace

static void state_copy(ms_sim* s, int32_t sig, float* host, bool to_device);

// Batched state signals with an initial value (learned decoders) get it in
// every batch column; the rest of the state starts at zero.  The values are
// uploaded once and broadcast on the device (the window driver's state is
// written through state_copy).
static void init_state(ms_sim* s) {
  const IR& ir = s->plan->ir;
  if (s->init_sigs.empty()) {
    std::vector<float> h;
    for (int32_t k = 0; k < (int32_t)ir.sigs.size(); ++k) {
      const Signal& sg = ir.sigs[k];
      if (sg.cls != SC_BATCHED || sg.value.empty()) continue;
      if ((int64_t)sg.value.size() != sg.rows) fail(MS_E_INVALID, "initial value size mismatch for " + sg.name);
      s->init_sigs.push_back({k, (int64_t)h.size()});
      h.insert(h.end(), sg.value.begin(), sg.value.end());
    }
    if (h.empty()) return;
    s->init_vals = dev_alloc<float>(h.size());
    HIPCHECK(hipMemcpy(s->init_vals, h.data(), h.size() * sizeof(float), hipMemcpyHostToDevice));
  }
  for (const auto& is : s->init_sigs) {
    const Signal& sg = ir.sigs[is.first];
    if (s->driver == MS_DRIVER_WINDOW) {
      std::vector<float> h((size_t)sg.rows * s->B);
      for (int64_t b = 0; b < s->B; ++b)
        for (int64_t r = 0; r < sg.rows; ++r) h[(size_t)(b * sg.rows + r)] = (float)sg.value[(size_t)r];
      state_copy(s, is.first, h.data(), true);
      continue;
    }
    const int64_t n = sg.rows * s->B;
    hipLaunchKernelGGL(k_init_rows, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s->stream, s->state, s->S,
                       s->B, s->plan->sig_offset[is.first], sg.rows, (const float*)(s->init_vals + is.second));
    HIPCHECK(hipGetLastError());
  }
}

extern "C" {

// MS_LOG (any value but "0"): the plan summary on stderr when a simulator is
// created: the driver, the merged groups it launches per step (per window for
// the window driver) with their sizes and kernels' shapes, and the bytes of
// state and parameters.
static void log_sim(const ms_sim* s) {
  const char* e = std::getenv("MS_LOG");
  if (!e || !*e || std::strcmp(e, "0") == 0) return;
  const Plan& p = *s->plan;
  const bool win = s->driver == MS_DRIVER_WINDOW;
  const std::vector<Launch>& ls = win ? s->wl : s->launches;
  static const char* dn[] = {"auto", "steps", "graph", "persistent", "window"};
  int64_t state_b = 0, param_b = 0;
  for (size_t b = 0; b < p.ir.bases.size(); ++b)
    (p.ir.bases[b].cls == SC_BATCHED ? state_b : param_b) += p.base_rows[b] * p.ir.bases[b].cols * 4;
  std::fprintf(stderr, "mergesim: driver %s, minibatch %d, %zu signals, %zu operators in %zu merged groups; "
               "%zu launches per %s; state %lld B per batch column, parameters %lld B\n",
               dn[s->driver], s->B, p.ir.sigs.size(), p.ir.ops.size(), p.groups.size(), ls.size(),
               win ? "window" : "step", (long long)state_b, (long long)param_b);
  for (size_t k = 0; k < ls.size(); ++k) {
    const Launch& l = ls[k];
    std::fprintf(stderr, "mergesim:   %2zu %-16s rows %lld", k, op_type_name(l.type), (long long)l.rows);
    if (l.type == OP_DOT_INC) std::fprintf(stderr, ", W %d x %d", l.M, l.K);
    if (l.type == OP_ENS)
      std::fprintf(stderr, ", <= %d neurons, %d threads, %d columns per workgroup%s%s", l.nmax, l.nthr, l.cpw,
                   l.rw ? ", weights in registers" : "", l.ens.chain ? ", fused chain" : "");
    if (win) std::fprintf(stderr, ", level %d", s->wplan->phases[k].level);
    std::fprintf(stderr, "\n");
  }
}

ms_status ms_sim_create(const ms_model* model, const ms_sim_opts* opts, ms_sim** out) {
  return guarded([&] {
    if (!model || !out) fail(MS_E_INVALID, "NULL argument");
    ms_sim_opts def;
    ms_sim_opts_default(&def);
    const ms_sim_opts* o = opts ? opts : &def;
    if (!(o->dt > 0)) fail(MS_E_INVALID, "dt must be > 0");
    if (o->minibatch < 1) fail(MS_E_INVALID, "minibatch must be >= 1");
    if (o->unroll < 1) fail(MS_E_INVALID, "unroll must be >= 1");
    if (o->driver < MS_DRIVER_AUTO || o->driver > MS_DRIVER_WINDOW) fail(MS_E_INVALID, "unknown driver");
    if (o->gemm_dtype != MS_GEMM_F32 && o->gemm_dtype != MS_GEMM_BF16) fail(MS_E_INVALID, "unknown gemm_dtype");
    if (o->decode != MS_DECODE_DENSE && o->decode != MS_DECODE_EVENT) fail(MS_E_INVALID, "unknown decode");
    int ndev = 0;
    HIPCHECK(hipGetDeviceCount(&ndev));
    if (o->device < 0 || o->device >= ndev) fail(MS_E_INVALID, "device ordinal out of range");
    auto s = new ms_sim();
    try {
      s->B = o->minibatch;
      s->device = o->device;
      s->unroll = o->unroll;
      s->dt = (float)o->dt;
      s->gemm_dtype = o->gemm_dtype;
      s->decode = o->decode;
      s->plan = make_plan(model_of(model), o->dt, plan_opts_from(o));
      if (o->spike_probe_bits) {
        const Model& m = model_of(model);
        s->spike_mag.assign(m.probes.size(), 0.0f);
        for (size_t i = 0; i < m.probes.size(); ++i) {
          const ProbeDesc& pd = m.probes[i];
          if (pd.kind == MS_REF_NEURONS && pd.synapse <= 0.0 && m.ens[(size_t)pd.id].neuron_type == MS_NEURON_LIF)
            s->spike_mag[i] = (float)m.ens[(size_t)pd.id].amplitude / (float)o->dt;
        }
      }
      DeviceGuard dg(s->device);
      if (o->stream) {
        s->stream = (hipStream_t)o->stream;
      } else {
        HIPCHECK(hipStreamCreateWithFlags(&s->stream, hipStreamNonBlocking));
        s->own_stream = true;
      }
      HIPCHECK(hipEventCreate(&s->ev0));
      HIPCHECK(hipEventCreate(&s->ev1));
      s->driver = choose_driver(*s->plan, s->B, o->driver);
      if (s->driver == MS_DRIVER_PERSISTENT && has_learning(*s->plan))
        fail(MS_E_INVALID, "the persistent driver cannot run a model with learning rules");
      if (s->gemm_dtype == MS_GEMM_BF16 && s->driver != MS_DRIVER_WINDOW)
        fail(MS_E_INVALID, "bf16 products run on the window driver only");
      if (o->spike_probe_bits && s->driver != MS_DRIVER_WINDOW)
        fail(MS_E_INVALID, "spike probes are recorded as bits by the window driver only");
      // persistent: one workgroup per batch column -> column-major state
      s->S = s->driver == MS_DRIVER_PERSISTENT ? Strides{1, (int64_t)std::max<int64_t>(1, s->plan->base_rows.empty() ? 1 : s->plan->base_rows[0])}
                                               : Strides{(int64_t)s->B, 1};
      if (s->driver == MS_DRIVER_WINDOW) {
        s->wplan = std::make_unique<WindowPlan>(make_window_plan(*s->plan));
        if (!s->wplan->ok) fail(MS_E_INVALID, "the window driver cannot run this model: " + s->wplan->why);
      }
      (void)scratch_on(s->device);   // the static staging array's address on this device
      setup_device(s);
      if (s->driver == MS_DRIVER_PERSISTENT) setup_persistent(s);
      if (s->driver == MS_DRIVER_WINDOW) setup_window(s);
      ensure_capacity(s, std::max<int64_t>(1, o->probe_capacity_steps));
      init_state(s);
      HIPCHECK(hipStreamSynchronize(s->stream));
      log_sim(s);
    } catch (...) {
      free_sim(s);
      delete s;
      throw;
    }
    *out = s;
  });
}

void ms_sim_destroy(ms_sim* s) {
  if (!s) return;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(s->device);
  if (s->stream) (void)hipStreamSynchronize(s->stream);
  free_sim(s);
  (void)hipSetDevice(prev);
  delete s;
}

ms_status ms_sim_run_steps(ms_sim* s, int64_t n_steps, const ms_feed* feeds, int32_t n_feeds) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    if (n_steps < 0) fail(MS_E_INVALID, "n_steps must be >= 0");
    if (n_feeds < 0 || (n_feeds > 0 && !feeds)) fail(MS_E_INVALID, "bad feeds");
    if (n_steps == 0) return;
    DeviceGuard dg(s->device);
    ensure_capacity(s, n_steps);
    stage_feeds(s, n_steps, feeds, n_feeds);
    HIPCHECK(hipMemsetAsync(s->ctr + 1, 0, sizeof(int64_t), s->stream));
    s->tn = 0;
    HIPCHECK(hipEventRecord(s->ev0, s->stream));
    if (s->driver == MS_DRIVER_PERSISTENT) {
      run_persistent(s, n_steps);
    } else if (s->driver == MS_DRIVER_WINDOW) {
      run_window(s, n_steps);
    } else if (s->driver == MS_DRIVER_GRAPH) {
      ensure_graph(s);
      if (s->has_prologue) launch_group(s, s->prologue, 0);
      int64_t k = 0;
      for (; k + s->unroll <= n_steps; k += s->unroll) HIPCHECK(hipGraphLaunch(s->graph_exec, s->stream));
      for (; k < n_steps; ++k) launch_step(s);
    } else {
      if (s->has_prologue) {
        time_group_begin(s, OP_SYN_SCATTER);
        launch_group(s, s->prologue, 0);
        time_group_end(s);
      }
      for (int64_t k = 0; k < n_steps; ++k) launch_step(s);
    }
    HIPCHECK(hipGetLastError());
    HIPCHECK(hipEventRecord(s->ev1, s->stream));
    s->steps_total += n_steps;
  });
}

ms_status ms_sim_sync(ms_sim* s) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    DeviceGuard dg(s->device);
    HIPCHECK(hipStreamSynchronize(s->stream));
  });
}

ms_status ms_sim_last_run_ms(ms_sim* s, double* ms_out) {
  return guarded([&] {
    if (!s || !ms_out) fail(MS_E_INVALID, "NULL argument");
    DeviceGuard dg(s->device);
    HIPCHECK(hipEventSynchronize(s->ev1));
    float ms = 0.f;
    HIPCHECK(hipEventElapsedTime(&ms, s->ev0, s->ev1));
    *ms_out = ms;
  });
}

ms_status ms_sim_set_timing(ms_sim* s, int32_t on) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    s->timing = on != 0;
  });
}

ms_status ms_sim_kernel_time(ms_sim* s, int32_t op_type, double* ms_out, int64_t* launches_out) {
  return guarded([&] {
    if (!s || !ms_out) fail(MS_E_INVALID, "NULL argument");
    if (op_type < 0 || op_type >= kTimedTypes) fail(MS_E_INVALID, "unknown operator type");
    if (s->driver != MS_DRIVER_WINDOW && s->driver != MS_DRIVER_STEPS)
      fail(MS_E_STATE, "per-kernel timing needs the WINDOW or STEPS driver");
    DeviceGuard dg(s->device);
    HIPCHECK(hipEventSynchronize(s->ev1));
    // launch intervals relative to the start of the run, then their union
    std::vector<std::pair<double, double>> iv;
    for (size_t k = 0; k < s->tn; ++k) {
      if (s->ttype[k] != op_type) continue;
      float a = 0.f, b = 0.f;
      HIPCHECK(hipEventElapsedTime(&a, s->ev0, s->tev[2 * k]));
      HIPCHECK(hipEventElapsedTime(&b, s->ev0, s->tev[2 * k + 1]));
      iv.push_back({a, std::max(a, b)});
    }
    std::sort(iv.begin(), iv.end());
    double busy = 0.0, lo = 0.0, hi = -1.0;
    for (const auto& x : iv) {
      if (x.first > hi) {
        if (hi > lo) busy += hi - lo;
        lo = x.first;
        hi = x.second;
      } else {
        hi = std::max(hi, x.second);
      }
    }
    if (hi > lo) busy += hi - lo;
    *ms_out = busy;
    if (launches_out) *launches_out = (int64_t)iv.size();
  });
}

ms_status ms_sim_steps(const ms_sim* s, int64_t* out) {
  return guarded([&] {
    if (!s || !out) fail(MS_E_INVALID, "NULL argument");
    *out = s->steps_total;
  });
}

ms_status ms_sim_set_check_feeds(ms_sim* s, int32_t on) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    s->check_feeds = on != 0;
  });
}

ms_status ms_sim_info(const ms_sim* s, int32_t* driver_out, int32_t* groups_out) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    if (driver_out) *driver_out = s->driver;
    if (groups_out) *groups_out = (int32_t)(s->driver == MS_DRIVER_WINDOW ? s->wl.size() : s->launches.size());
  });
}

ms_status ms_sim_probe_width(const ms_sim* s, int32_t probe, int32_t* w) {
  return guarded([&] {
    if (!s || !w) fail(MS_E_INVALID, "NULL argument");
    if (probe < 0 || probe >= (int32_t)s->plan->probe_width.size()) fail(MS_E_INVALID, "probe id out of range");
    *w = s->plan->probe_width[probe];
  });
}

ms_status ms_sim_probe_read(ms_sim* s, int32_t probe, float* out, int64_t cap, int32_t out_on_device) {
  return guarded([&] {
    if (!s || !out) fail(MS_E_INVALID, "NULL argument");
    const Plan& p = *s->plan;
    if (probe < 0 || probe >= (int32_t)p.probe_width.size()) fail(MS_E_INVALID, "probe id out of range");
    const int32_t w = p.probe_width[probe];
    const int64_t T = s->steps_total;
    const int64_t n = (int64_t)s->B * T * w;
    if (cap < n) fail(MS_E_INVALID, "probe output capacity too small");
    if (n == 0) return;
    DeviceGuard dg(s->device);
    float* tmp = out_on_device ? out : dev_alloc<float>((size_t)n);
    if (!s->bit_off.empty() && s->bit_off[probe] >= 0)
      hipLaunchKernelGGL(k_bits_extract, dim3(grid_for(n)), dim3(kBlock), 0, s->stream,
                         (const uint32_t*)s->bits_buf, s->B, T, s->bit_words, s->bit_off[probe], w,
                         s->spike_mag[probe], tmp);
    else
      hipLaunchKernelGGL(k_probe_extract, dim3(grid_for(n)), dim3(kBlock), 0, s->stream,
                         (const float*)s->probe_buf, s->B, T, s->probe_rows, p.probe_row_offset[probe], w, tmp);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && !out_on_device)
      e = hipMemcpyAsync(out, tmp, (size_t)n * 4, hipMemcpyDeviceToHost, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (!out_on_device) (void)hipFree(tmp);
    if (e != hipSuccess) fail(MS_E_HIP, std::string("probe read: ") + hipGetErrorString(e));
  });
}

ms_status ms_sim_probe_read_static(ms_sim* s, int32_t probe, float* out, int64_t cap) {
  return guarded([&] {
    if (!s || !out) fail(MS_E_INVALID, "NULL argument");
    const Plan& p = *s->plan;
    if (probe < 0 || probe >= (int32_t)p.probe_width.size()) fail(MS_E_INVALID, "probe id out of range");
    const int32_t w = p.probe_width[probe];
    const int64_t T = s->steps_total;
    const int64_t n = (int64_t)s->B * T * w;
    if (cap < n) fail(MS_E_INVALID, "probe output capacity too small");
    if (n > MS_PROBE_READ_STATIC_MAX)
      fail(MS_E_INVALID, "probe record of " + std::to_string(n) + " values exceeds the static staging array (" +
                             std::to_string(MS_PROBE_READ_STATIC_MAX) + " values); use ms_sim_probe_read");
    if (n == 0) return;
    DeviceGuard dg(s->device);
    float* stage = scratch_on(s->device);
    if (!s->bit_off.empty() && s->bit_off[probe] >= 0)
      hipLaunchKernelGGL(k_bits_extract, dim3(grid_for(n)), dim3(kBlock), 0, s->stream,
                         (const uint32_t*)s->bits_buf, s->B, T, s->bit_words, s->bit_off[probe], w,
                         s->spike_mag[probe], stage);
    else
      hipLaunchKernelGGL(k_probe_extract, dim3(grid_for(n)), dim3(kBlock), 0, s->stream,
                         (const float*)s->probe_buf, s->B, T, s->probe_rows, p.probe_row_offset[probe], w, stage);
    HIPCHECK(hipGetLastError());
    HIPCHECK(hipMemcpyAsync(out, stage, (size_t)n * 4, hipMemcpyDeviceToHost, s->stream));
    HIPCHECK(hipStreamSynchronize(s->stream));
  });
}

ms_status ms_sim_probe_read_bits(ms_sim* s, int32_t probe, uint32_t* out, int64_t cap, int32_t out_on_device) {
  return guarded([&] {
    if (!s || !out) fail(MS_E_INVALID, "NULL argument");
    const Plan& p = *s->plan;
    if (probe < 0 || probe >= (int32_t)p.probe_width.size()) fail(MS_E_INVALID, "probe id out of range");
    if (s->bit_off.empty() || s->bit_off[probe] < 0)
      fail(MS_E_INVALID, "probe " + std::to_string(probe) + " is not recorded as spike bits");
    const int32_t nw = (p.probe_width[probe] + 31) / 32;
    const int64_t T = s->steps_total;
    const int64_t n = (int64_t)s->B * T * nw;
    if (cap < n) fail(MS_E_INVALID, "probe output capacity too small");
    if (n == 0) return;
    DeviceGuard dg(s->device);
    uint32_t* tmp = out_on_device ? out : dev_alloc<uint32_t>((size_t)n);
    hipLaunchKernelGGL(k_bits_words, dim3(grid_for(n)), dim3(kBlock), 0, s->stream, (const uint32_t*)s->bits_buf,
                       s->B, T, s->bit_words, s->bit_off[probe], nw, tmp);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && !out_on_device)
      e = hipMemcpyAsync(out, tmp, (size_t)n * 4, hipMemcpyDeviceToHost, s->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(s->stream);
    if (!out_on_device) (void)hipFree(tmp);
    if (e != hipSuccess) fail(MS_E_HIP, std::string("probe read: ") + hipGetErrorString(e));
  });
}

// The initial state (ms_sim_reset), queued on the simulator's stream.
static void reset_state(ms_sim* s) {
  HIPCHECK(hipMemsetAsync(s->state, 0, std::max<size_t>(1, s->state_rows) * s->B * 4, s->stream));
  if (s->va)   // block 0 (the carried state); the other blocks are written before they are read
    HIPCHECK(hipMemset2DAsync(s->va, s->vs * 4, 0, (size_t)s->B * 4, std::max<int64_t>(1, s->wplan->rows_v), s->stream));
  if (s->pa) HIPCHECK(hipMemsetAsync(s->pa, 0, (size_t)std::max<int64_t>(1, s->wplan->rows_p) * s->B * 4, s->stream));
  HIPCHECK(hipMemsetAsync(s->ctr, 0, 2 * sizeof(int64_t), s->stream));
  init_state(s);
  s->steps_total = 0;
}

ms_status ms_sim_reset(ms_sim* s) {
  return guarded([&] {
    if (!s) fail(MS_E_INVALID, "NULL sim");
    DeviceGuard dg(s->device);
    reset_state(s);
    HIPCHECK(hipStreamSynchronize(s->stream));
  });
}

// Copies one state signal between the device state and a host buffer laid out
// [B][rows], touching only that signal's elements.  Row-major state (rs = B,
// cs = 1) holds the signal as one block of rows*B floats; column-major state
// (rs = 1) holds B columns of rows floats, cs floats apart.
static void state_copy(ms_sim* s, int32_t sig, float* host, bool to_device) {
  const int64_t rows = s->plan->ir.sigs[sig].rows, B = s->B;
  const int64_t r0 = s->plan->sig_offset[sig];
  DeviceGuard dg(s->device);
  HIPCHECK(hipStreamSynchronize(s->stream));
  if (s->driver == MS_DRIVER_WINDOW) {
    // block 0 of a versioned signal (the value the next window starts from), or
    // the private neuron state
    const WindowPlan& w = *s->wplan;
    const int64_t row = w.sig_row[sig];
    float* dev = w.priv[sig] ? s->pa + row * B : s->va + row * s->vs;
    const size_t pitch = (size_t)(w.priv[sig] ? B : s->vs) * 4;
    std::vector<float> h((size_t)(rows * B));
    if (to_device) {
      for (int64_t b = 0; b < B; ++b)
        for (int64_t r = 0; r < rows; ++r) h[(size_t)(r * B + b)] = host[(size_t)(b * rows + r)];
      HIPCHECK(hipMemcpy2D(dev, pitch, h.data(), B * 4, B * 4, rows, hipMemcpyHostToDevice));
    } else {
      HIPCHECK(hipMemcpy2D(h.data(), B * 4, dev, pitch, B * 4, rows, hipMemcpyDeviceToHost));
      for (int64_t b = 0; b < B; ++b)
        for (int64_t r = 0; r < rows; ++r) host[(size_t)(b * rows + r)] = h[(size_t)(r * B + b)];
    }
    return;
  }
  if (s->S.cs == 1) {
    if (s->S.rs != B) fail(MS_E_STATE, "unexpected state layout");
    float* dev = s->state + r0 * B;
    std::vector<float> h((size_t)(rows * B));
    if (to_device) {
      for (int64_t b = 0; b < B; ++b)
        for (int64_t r = 0; r < rows; ++r) h[(size_t)(r * B + b)] = host[(size_t)(b * rows + r)];
      HIPCHECK(hipMemcpy(dev, h.data(), h.size() * 4, hipMemcpyHostToDevice));
    } else {
      HIPCHECK(hipMemcpy(h.data(), dev, h.size() * 4, hipMemcpyDeviceToHost));
      for (int64_t b = 0; b < B; ++b)
        for (int64_t r = 0; r < rows; ++r) host[(size_t)(b * rows + r)] = h[(size_t)(r * B + b)];
    }
  } else {
    if (s->S.rs != 1 || s->S.cs < r0 + rows) fail(MS_E_STATE, "unexpected state layout");
    float* dev = s->state + r0;
    if (to_device)
      HIPCHECK(hipMemcpy2D(dev, s->S.cs * 4, host, rows * 4, rows * 4, B, hipMemcpyHostToDevice));
    else
      HIPCHECK(hipMemcpy2D(host, rows * 4, dev, s->S.cs * 4, rows * 4, B, hipMemcpyDeviceToHost));
  }
}

static int32_t state_signal(const ms_sim* s, int32_t which, int32_t id) {
  const IR& ir = s->plan->ir;
  auto pick = [&](const std::vector<int32_t>& v) -> int32_t {
    if (id < 0 || id >= (int32_t)v.size() || v[id] < 0) fail(MS_E_INVALID, "no such state for this id");
    return v[id];
  };
  switch (which) {
    case MS_STATE_VOLTAGE: return pick(ir.ens_V);
    case MS_STATE_REFRACTORY: return pick(ir.ens_ref);
    case MS_STATE_SYNAPSE: return pick(ir.conn_y);
    case MS_STATE_PROBE_SYNAPSE: return pick(ir.probe_y);
    case MS_STATE_LEARNED_DECODERS: return pick(ir.conn_W);
    case MS_STATE_PES_ACTIVITY: return pick(ir.conn_act);
    default: fail(MS_E_INVALID, "unknown state kind");
  }
}

ms_status ms_sim_get_state(ms_sim* s, int32_t which, int32_t id, float* out, int64_t cap) {
  return guarded([&] {
    if (!s || !out) fail(MS_E_INVALID, "NULL argument");
    const int32_t sig = state_signal(s, which, id);
    if (cap < (int64_t)s->plan->ir.sigs[sig].rows * s->B) fail(MS_E_INVALID, "state output capacity too small");
    state_copy(s, sig, out, false);
  });
}

ms_status ms_sim_set_state(ms_sim* s, int32_t which, int32_t id, const float* in, int64_t n_elems) {
  return guarded([&] {
    if (!s || !in) fail(MS_E_INVALID, "NULL argument");
    const int32_t sig = state_signal(s, which, id);
    if (n_elems != (int64_t)s->plan->ir.sigs[sig].rows * s->B) fail(MS_E_INVALID, "state size mismatch");
    state_copy(s, sig, const_cast<float*>(in), true);
  });
}

}  // extern "C"

#include "train_host.hpp"
