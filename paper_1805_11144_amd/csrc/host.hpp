// Host-side data structures of mergesim: the model description, the build
// step's parameters, the signal/operator IR, the merged plan and its lowering
// into per-group index arrays.  No HIP here: everything in this header runs on
// the CPU and is testable without a GPU.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <stdexcept>
#include <string>
#include <utility>
#include <vector>

#include "mergesim.h"

namespace ms {

// Error carrying an ms_status; caught at the C ABI boundary.
struct Error : std::runtime_error {
  ms_status code;
  Error(ms_status c, const std::string& m) : std::runtime_error(m), code(c) {}
};
[[noreturn]] void fail(ms_status code, const std::string& msg);
void set_last_error(const std::string& msg);

// ------------------------------------------------------------------ model
struct NodeDesc {
  int32_t size = 0;
  bool passthrough = false;
  bool constant = false;          // value given
  std::vector<double> value;      // [size]
};

struct EnsembleDesc {
  int32_t n = 0, d = 0, neuron_type = MS_NEURON_LIF;
  double tau_rc = 0.02, tau_ref = 0.002, amplitude = 1.0;
  double sigma = 0.0;             // smoothing of the soft LIF rate curve
  std::vector<double> encoders;   // [n*d]
  std::vector<double> max_rates, intercepts, gains, biases;
  int32_t n_eval = 0;
  std::vector<double> eval_points;  // [M*d]
};

struct ConnDesc {
  int32_t pre_kind = 0, pre_id = 0, pre_start = 0, pre_stop = 0;
  int32_t post_kind = 0, post_id = 0, post_start = 0, post_stop = 0;
  int32_t function = MS_FN_IDENTITY;
  std::vector<double> decoders;   // explicit [n*cols] or empty
  int32_t decoders_cols = 0;
  int32_t t_rows = 0, t_cols = 0;
  std::vector<double> transform;  // [rows*cols] or empty (scalar)
  double t_scalar = 1.0;
  double synapse = 0.0;           // <= 0: none
  bool learned = false;           // PES on its decoders
  double pes_rate = 0.0;          // kappa
  double pes_tau = 0.0;           // pre activity filter; <= 0: none
};

struct ProbeDesc {
  int32_t kind = 0, id = 0, start = 0, stop = 0;
  double synapse = 0.0;
};

struct Model {
  std::vector<NodeDesc> nodes;
  std::vector<EnsembleDesc> ens;
  std::vector<ConnDesc> conns;
  std::vector<ProbeDesc> probes;
};

// Size of the value a reference denotes (node output, decoded function,
// neurons) -- used for validation of slices and transforms.
int32_t function_size(int32_t fn, int32_t dims);

// ------------------------------------------------------------------ build
struct Built {
  std::vector<std::vector<double>> gain, bias;          // per ensemble [n]
  // decoders keyed by (ensemble, function): [n * d_fn]
  std::map<std::pair<int32_t, int32_t>, std::vector<double>> decoders;
};
Built build_params(const Model& m);

// --------------------------------------------------------------------- IR
enum SigClass : int32_t { SC_BATCHED = 0, SC_PARAM = 1 };

struct Signal {
  std::string name;
  int32_t rows = 0;
  int32_t cols = 1;               // params: matrix width (1 for vectors)
  SigClass cls = SC_BATCHED;
  bool state = false;             // persists across steps (V, ref, filters)
  std::vector<double> value;      // params: [rows*cols]; batched state: initial value
                                  // [rows] of every batch column (empty: zeros)
  int32_t base = -1;              // base array id (assigned by the IR builder)
};

enum OpType : int32_t {
  OP_FEED = 0,
  OP_RESET = 1,
  OP_COPY = 2,          // dst = src
  OP_COPY_INC = 3,      // dst += src
  OP_ELEM_INC = 4,      // dst += a (.) x
  OP_DOT_INC = 5,       // dst += W x
  OP_LIF = 6,
  OP_LIF_RATE = 7,
  OP_LOWPASS = 8,
  OP_ENS = 9,           // fused ensemble: J = bias + enc x; LIF; d_f = D_f s
  OP_SYN_SCATTER = 10,  // fused connection tail (launch drivers only, never in a plan's
                        // groups): transform, lowpass update, pull into the post inputs
  OP_BDOT_INC = 11,     // dst[j] += sum_i src[i] W[i*k + j], W a batched signal (per-row decoders)
  OP_PES = 12,          // W[i*k + j] += coef * src[i] * a[j] (update: after W's readers)
  OP_PES_FUSED = 13,    // BDOT_INC and PES of the same connections in one pass (launch drivers)
  OP_NTYPES = 14
};

// Fused decoders of one ensemble operator are limited to this many outputs in
// total (they are accumulated in registers); larger ones stay separate.
constexpr int32_t kMaxFusedDecoded = 16;
const char* op_type_name(int32_t t);

// A reference to rows [start, start+len) of a signal.
struct SRef {
  int32_t sig = -1;
  int32_t start = 0;
  int32_t len = 0;
};

struct Op {
  OpType type;
  std::string name;
  SRef dst;            // RESET/COPY/COPY_INC/ELEM_INC/DOT_INC dst; LIF s; LOWPASS y
  SRef src;            // COPY src; ELEM_INC x; DOT_INC x; LIF J; LOWPASS v
  SRef a;              // ELEM_INC a (len 1 = broadcast scalar); DOT_INC W (rows M, cols K)
  SRef V, ref;         // LIF state
  int32_t node = -1;   // FEED: node id
  std::vector<double> reset_value;  // RESET: [dst.len] (empty = zeros)
  SRef bias;                        // ENS: bias parameter [n]
  std::vector<std::pair<SRef, SRef>> decs;  // ENS: (decoder param [d_f x n], output d_f)
  int32_t ntype = 0;                // ENS, LIF_RATE: MS_NEURON_*
  int32_t n = 0;                    // ENS: neurons
  double tau_rc = 0, tau_ref = 0, amp = 0;  // LIF params
  double sigma = 0;                         // LIF_RATE, soft LIF rate: smoothing
  double coef_a = 0, coef_b = 0;            // LOWPASS y = coef_a y + coef_b v; PES coef_a
};

struct BaseArray {
  std::string name;   // "state", "vec", "mat<K>"
  SigClass cls;
  int32_t cols;
};

struct IR {
  std::vector<Signal> sigs;
  std::vector<Op> ops;
  std::vector<BaseArray> bases;
  // feed layout: fed nodes in id order, each [size] rows of the staging buffer
  std::vector<int32_t> fed_nodes;       // node ids
  std::vector<int32_t> feed_row_of_node;  // per node: first staging row or -1
  int32_t feed_rows = 0;
  std::vector<int32_t> node_size;       // per node
  // probes: probed signal rows
  struct ProbeSrc { SRef src; };
  std::vector<ProbeSrc> probes;
  // state signals for get/set state
  std::vector<int32_t> ens_V, ens_ref;     // per ensemble signal id or -1
  std::vector<int32_t> conn_y;             // per connection signal id or -1
  std::vector<int32_t> probe_y;            // per probe signal id or -1
  std::vector<int32_t> conn_W, conn_act;   // per connection: learned decoders, PES activity filter
};
IR build_ir(const Model& m, const Built& b, double dt);
void simplify_ir(IR& ir);
void fuse_ensembles(IR& ir);

// ------------------------------------------------------------------- plan
struct PlanOpts {
  int32_t planner = MS_PLANNER_TREE;
  int32_t depth = 3;
  bool merge = true, sort = true, simplify = true, fuse = true;
  bool fuse_synapse = true;    // time-major step program: fused synapse filter + scatter
  int32_t minibatch = 1;       // B, which picks the product kernel of a launch
};

// One operand of a lowered group: rows in its base array, either a contiguous
// range starting at `start` (idx empty) or an explicit index list.
struct LOperand {
  int32_t base = -1;
  int64_t start = 0;
  std::vector<int32_t> idx;
  bool contiguous() const { return idx.empty(); }
};

struct LGroup {
  OpType type;
  std::vector<int32_t> ops;     // op ids in execution order
  int64_t rows = 0;             // per-row work items (DOT_INC: number of ops)
  // per-row operands (meaning depends on type, see lower_group)
  LOperand dst, src, a, V, ref;
  // CSR for increments with repeated destinations (COPY_INC / ELEM_INC):
  // unique destinations `dst` (rows = number of unique), entries ptr[u]..ptr[u+1]
  std::vector<int32_t> ptr;
  // DOT_INC
  int32_t M = 0, K = 0;
  std::vector<int32_t> w_row, x_row, d_row;   // per op
  // BDOT_INC (M = k outputs, K = n neurons): per op w_row (first row of the
  // batched decoders, row i*k + j), x_row (activities), d_row (outputs).
  // PES: per op w_row, x_row (activities or their filter), e_row (error),
  // coef (-kappa dt / n).  PES_FUSED: both, d_row the outputs and x_row the
  // activities the decode reads, act_row the activities the update reads.
  std::vector<int32_t> e_row, act_row;
  std::vector<float> coef;
  // RESET values (empty: zeros)
  std::vector<float> values;
  // LIF / LIF_RATE parameters: uniform (size 1) or per row
  std::vector<float> tau_rc, tau_ref, amp;
  std::vector<float> sigma;     // LIF_RATE of soft LIF rate neurons: smoothing (uniform or per row)
  // LOWPASS coefficients: uniform (size 1) or per row
  std::vector<float> ca, cb;
  // FEED: staging rows per destination row
  std::vector<int32_t> feed_rows;
  // ENS: per-op rows (x_row -1 when the ensemble has no decoded input, s_row -1
  // when the spikes are not stored); decoder rows per fused function
  int32_t ens_d = 0, ens_type = 0;
  std::vector<int32_t> ens_n, ens_x, ens_enc, ens_bias, ens_V, ens_ref, ens_s;
  std::vector<int32_t> ens_df;                       // per function
  std::vector<std::vector<int32_t>> ens_D, ens_dd;   // [function][op]
  std::vector<int32_t> ens_Dbase;                    // per function
  int32_t ens_bias_base = -1;
  // ENS, window driver: per op kChainInts ints (empty: no op has one) -- the
  // op's input x is the connection chain of Fig. 2 fused in (x_t = y_{t-1},
  // y_t = a y_{t-1} + b W d_t): d first row (window row) and K, W first row
  // in the weight base ens_chain_wbase (M rows of K), y first row (window
  // row), M, then the float bits of a and b; K = 0 for an op without one
  std::vector<int32_t> ens_chain;
  int32_t ens_chain_wbase = -1;
  // SYN_SCATTER: segments of at most kSynSeg consecutive rows, 4 ints each
  // (first destination row or -1 for none, length, first connection, number of
  // connections); connections 8 ints each (first filter row y, first value row v
  // or -1 when the value is computed here or -2 for a probe copy of row y,
  // first input row x, K, weight slot, first weight row, first probe row or -1,
  // 1 when the inputs are rows of the feed staging buffer)
  // plus 2 floats (a, b: y <- a y + b v); weight bases per slot; syn_update 0:
  // pull only (no filter update, no probe); syn_probe 1: the group records
  // every probe row of the step (the separate probe copy is dropped)
  std::vector<int32_t> syn_seg, syn_conn, syn_wbase;
  std::vector<float> syn_ab;
  int32_t syn_update = 1;
  int32_t syn_probe = 0;
};

constexpr int32_t kChainInts = 8; // ints per op of a fused window connection chain
constexpr int32_t kSynSeg = 16;   // rows per segment of a fused synapse group
constexpr int32_t kSynSlots = 4;  // weight bases one fused synapse group may read

struct Plan {
  PlanOpts opts;
  double dt = 0.001;
  Built built;
  IR ir;
  std::vector<std::vector<int32_t>> groups;      // op ids per group, execution order
  std::vector<int64_t> sig_offset;               // row offset of each signal in its base
  std::vector<int64_t> base_rows;                // rows per base array
  std::vector<int32_t> key_of_op;
  std::vector<LGroup> lowered;
  // probe lowering: source row (state base) per probe row; probe row offsets
  std::vector<int32_t> probe_src_rows;
  std::vector<int32_t> probe_row_offset;         // per probe, + total at end
  std::vector<int32_t> probe_width;
};

// ------------------------------------------------- stage-major (window) schedule
// A model whose operators form no cycle once every synapse update is taken as
// an edge from one step to the next (feedforward chains and layers; every
// recurrence is an element's own state: neuron voltage/refractory time, a
// filter's output) can run stage by stage: each merged group over a whole
// window of timesteps before the groups that depend on it.  Signals read by
// other operators are then stored once per step of the window ("versioned":
// [rows][(W+1)*B], block 0 holding the value carried in from the previous
// window, block t+1 the value of window step t); neuron state stays in a
// private [rows][B] array.
struct WPhase {
  LGroup g;               // lowered with window row numbering
  int32_t level = 0;
  int32_t src_blk = 1;    // src rows: 1 = this step's value, 0 = the previous step's
  int32_t a_blk = 1;      // the same for a batched ElementwiseInc `a`
  bool exclusive = false; // no other phase of its level writes a signal it writes
};

struct WindowPlan {
  bool ok = false;
  std::string why;                   // why the model cannot run stage by stage
  std::vector<int64_t> sig_row;      // per signal: row in its window array (parameters: row in their base)
  std::vector<char> priv;            // per signal: in the private array
  int64_t rows_v = 0, rows_p = 0;
  int32_t levels = 0;
  std::vector<WPhase> phases;        // execution order
  std::vector<int32_t> probe_rows;   // versioned rows of the probe sources, probe-row order
};

WindowPlan make_window_plan(const Plan& p);

// ------------------------------------------------- time-major step program
// The groups one timestep of the launch drivers (plain launches, hipGraph)
// runs, in order.  Consecutive independent fused-ensemble groups share a
// launch.  With fuse_synapse, the connections' tail of Fig. 2 -- transform
// (DotInc), synaptic filter (Lowpass, last in the step) and the copy of the
// filtered value into the post input at the start of the next step (Reset +
// CopyInc) -- becomes one SYN_SCATTER group at the filter's place: per post
// input row it computes each incoming connection's value, updates the filter
// and sums the filtered values, in the CopyInc's order.  The pull thereby
// moves from the start of step k + 1 to the end of step k; nothing reads those
// rows in between, and `prologue` (pull only) sets them at the start of every
// run from the filter state.
struct LaunchPlan {
  std::vector<LGroup> step;
  bool has_prologue = false;
  LGroup prologue;
  std::string why;   // why no fusion took place (empty when it did or was off)
};
LaunchPlan make_launch_plan(const Plan& p);
std::vector<LGroup> merge_ens_groups(const std::vector<LGroup>& in);

std::unique_ptr<Plan> make_plan(const Model& m, double dt, const PlanOpts& o);
std::string plan_to_json(const Plan& p);

PlanOpts plan_opts_from(const ms_sim_opts* o);
const Model& model_of(const ms_model* m);

// Run f, converting exceptions into an ms_status and the thread-local message.
template <class F>
ms_status guarded(F&& f) {
  try {
    f();
    return MS_OK;
  } catch (const Error& e) {
    set_last_error(e.what());
    return e.code;
  } catch (const std::bad_alloc&) {
    set_last_error("host allocation failed");
    return MS_E_OOM;
  } catch (const std::exception& e) {
    set_last_error(e.what());
    return MS_E_INVALID;
  }
}

// Planner internals exposed for tests through the JSON export.
std::vector<std::vector<int32_t>> plan_groups(const IR& ir, const std::vector<int32_t>& key,
                                              int32_t n_keys, const PlanOpts& o);

}  // namespace ms
