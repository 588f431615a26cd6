/*
 * mergesim -- merged-operator spiking-network simulator for one MI355X (gfx950).
 *
 * C ABI.  Every entry point returns an ms_status (0 = MS_OK, negative = error)
 * except the destroy functions and ms_last_error.  No C++ exception crosses this
 * boundary.  On error, ms_last_error() returns a thread-local message describing
 * the last failure of a call made on the calling thread.
 *
 * The operation follows the problem statement of the NengoDL paper
 * (Rasmussen 2018):
 *   - a model is a Network of Nodes, Ensembles, Connections and Probes
 *     (Sec. 2.1.2); the builder lowers it to Signals and Operators (Sec. 2.1.3,
 *     Fig. 2: a connection is DotInc -> synaptic filter -> Copy into the post);
 *   - the simulator merges signals into base arrays and operators into groups,
 *     plans the group order, sorts signals for contiguous reads and simplifies
 *     special cases (Sec. 4.2, Alg. 1 and Alg. 2);
 *   - run(n_steps) advances the simulation with per-node input feeds shaped
 *     [minibatch][timesteps][dims] (Sec. 3.1); probes record one sample per
 *     step, read back as [minibatch][timesteps][dims]; reset() restores the
 *     initial state (Sec. 3.1).
 *
 * Ownership: the caller owns every array it passes in; the library copies model
 * descriptions during the ms_model_add_* call and copies feeds during
 * ms_sim_run_steps.  The library owns ms_model, ms_plan and ms_sim objects and
 * every device buffer it allocates.  Probe reads copy into caller memory.
 *
 * Randomness: the library draws no random numbers; every random parameter
 * (encoders, rates, intercepts, evaluation points, transforms) is an input.
 *
 * Precision: the build step (gains, biases, decoder solves) runs in double on
 * the host; the simulation stores parameters and state in float32 on the GPU
 * and accumulates products in float32.
 */
#ifndef MERGESIM_H
#define MERGESIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ms_status;

#define MS_OK 0
#define MS_E_INVALID (-1)   /* bad shape, id, range or option */
#define MS_E_CYCLE (-2)     /* a cycle of connections without a synapse */
#define MS_E_OOM (-3)       /* host or device allocation failed */
#define MS_E_HIP (-4)       /* a HIP runtime call failed; message kept */
#define MS_E_STATE (-5)     /* call not valid in the object's current state */
#define MS_E_NUMERIC (-6)   /* decoder solve failed (matrix not positive definite) */

typedef struct ms_model ms_model;
typedef struct ms_plan ms_plan;
typedef struct ms_sim ms_sim;

/* Reference kinds used by connections and probes. */
#define MS_REF_NODE 0     /* node output (pre) / passthrough node input (post) */
#define MS_REF_ENS 1      /* decoded value (pre) / represented input (post)    */
#define MS_REF_NEURONS 2  /* spike output (pre) / input current times gain (post) */
#define MS_REF_LEARNING 3 /* post only: error input of the learning rule of
                             connection post_id (see ms_model_set_pes) */

#define MS_NEURON_LIF 0       /* spiking LIF, exact integration */
#define MS_NEURON_LIF_RATE 1  /* LIF rate curve amplitude * r(J) */
#define MS_NEURON_RELU 2      /* rectified linear: amplitude * max(J, 0); gain and bias
                                 from max_rates/intercepts put J = 0 at the intercept
                                 and J = max_rate at x = 1 (no state) */
#define MS_NEURON_SOFTLIF_RATE 3  /* smoothed LIF rate, the differentiable stand-in for
                                 the spiking LIF in training (Sec. 3.2 trains spiking
                                 models through a rate approximation): amplitude /
                                 (tau_ref + tau_rc log(1 + 1/rho)), rho = sigma
                                 log(1 + exp((J - 1) / sigma)); gain and bias as for
                                 LIF; never fused (MS_FUSE_ENSEMBLES skips it) */

#define MS_FN_IDENTITY 0  /* decode x (d outputs) */
#define MS_FN_PRODUCT 1   /* decode x0 * x1 (1 output, needs dims >= 2) */

/* ------------------------------------------------------------------ model */

/* Ensemble description (paper Sec. 2.1.2 "a group of neurons").
 * encoders [n][d] row-major; either gains+biases [n] are given, or
 * max_rates+intercepts [n] (then gain and bias are computed so that the
 * neuron starts firing at intercept and fires at max_rate at x = 1).
 * eval_points [M][d]: where decoders are fitted (needed only if something
 * decodes from this ensemble without explicit decoders).
 * tau_rc, tau_ref in seconds; amplitude scales the neuron output
 * (spike height amplitude/dt, rate amplitude * r(J)). */
typedef struct {
  int32_t n_neurons;
  int32_t dims;
  int32_t neuron_type;          /* MS_NEURON_* */
  double tau_rc, tau_ref, amplitude;
  const double* encoders;       /* [n][d] */
  const double* max_rates;      /* [n] or NULL if gains given */
  const double* intercepts;     /* [n] or NULL if gains given */
  const double* gains;          /* [n] or NULL */
  const double* biases;         /* [n] or NULL */
  int32_t n_eval_points;
  const double* eval_points;    /* [M][d] or NULL */
  double sigma;                 /* smoothing of MS_NEURON_SOFTLIF_RATE (> 0); ignored otherwise */
} ms_ensemble_desc;

/* Connection description (paper Sec. 2.1.2 "Connection", Fig. 2).
 * The value sent is v = T * pre[pre_start:pre_stop] (a start == stop == 0
 * slice means the whole object).  Pre kinds: node output, an ensemble's decoded
 * function (MS_FN_*, decoders solved on the ensemble's eval points unless
 * explicit decoders [n][decoders_cols] are given), or an ensemble's spikes.
 * T is a matrix [transform_rows][transform_cols] (rows = post slice size,
 * cols = pre slice size) or, when transform_rows == 0, the scalar
 * transform_scalar.  synapse_tau > 0 adds a lowpass filter (one-step delay);
 * synapse_tau <= 0 delivers v within the same step.  Post kinds: a passthrough
 * node, an ensemble's represented input, or an ensemble's neurons (added to the
 * input current after multiplying by the neuron gains). */
typedef struct {
  int32_t pre_kind, pre_id, pre_start, pre_stop;
  int32_t post_kind, post_id, post_start, post_stop;
  int32_t function;             /* MS_FN_*, used when pre_kind == MS_REF_ENS */
  const double* decoders;       /* explicit [n][decoders_cols] or NULL */
  int32_t decoders_cols;
  int32_t transform_rows, transform_cols;
  const double* transform;      /* [rows][cols] or NULL for a scalar */
  double transform_scalar;
  double synapse_tau;           /* seconds; <= 0 means no synapse */
} ms_connection_desc;

/* Probe description (paper Sec. 3.1 sim.data[probe]).  Targets: node output,
 * an ensemble's decoded identity, or spikes of neurons [start, stop) of an
 * ensemble (start == stop == 0: all).  synapse_tau > 0 filters the probed
 * value with a lowpass before recording. */
typedef struct {
  int32_t target_kind, target_id;
  int32_t start, stop;
  double synapse_tau;
} ms_probe_desc;

ms_status ms_model_create(ms_model** out);
void ms_model_destroy(ms_model* model);

/* A node of `size` outputs.  value == NULL: an input node whose output is
 * supplied by a feed at every run call (zeros when no feed is given).
 * value != NULL: a constant node (copied).  passthrough != 0: the node's output
 * is the sum of its incoming connections in the same step (value ignored). */
ms_status ms_model_add_node(ms_model* model, int32_t size, const double* value,
                            int32_t passthrough, int32_t* id_out);
ms_status ms_model_add_ensemble(ms_model* model, const ms_ensemble_desc* desc,
                                int32_t* id_out);
ms_status ms_model_add_connection(ms_model* model, const ms_connection_desc* desc,
                                  int32_t* id_out);
ms_status ms_model_add_probe(ms_model* model, const ms_probe_desc* desc, int32_t* id_out);

/* Online learning with the Prescribed Error Sensitivity rule (paper Sec. 5.1,
 * the pes benchmark: an ensemble's output weights updated as the simulation
 * runs; Fig. 7: each batch element then needs its own weight matrix).
 * Connection `conn_id` must decode from an ensemble (pre_kind MS_REF_ENS, no
 * pre slice); its decoders D [n][k] (explicit, or solved for its function)
 * become the initial value of per-batch-element decoders D^b, which every step
 * changes by
 *     D^b <- D^b - (learning_rate * dt / n) * outer(a^b, e^b)
 * after the connection has decoded with them.  e^b [k] is the sum of the
 * connections whose post is (MS_REF_LEARNING, conn_id) (a filtered one
 * delivers its state as left by the previous step); a^b [n] is the pre
 * neurons' output lowpass-filtered with pre_synapse_tau, as left by the
 * previous step, or this step's output when pre_synapse_tau <= 0.  Models
 * with learning run on the STEPS and GRAPH drivers (MS_DRIVER_AUTO picks
 * GRAPH; PERSISTENT and WINDOW give MS_E_INVALID).  MS_E_INVALID for a
 * connection that does not decode from neurons, has a pre slice or already
 * learns, and for learning_rate < 0. */
ms_status ms_model_set_pes(ms_model* model, int32_t conn_id, double learning_rate,
                           double pre_synapse_tau);

/* ---------------------------------------------------------------- options */

#define MS_PLANNER_GREEDY 0   /* schedule the largest ready group next (tree n = 1) */
#define MS_PLANNER_TREE 1     /* bounded breadth-first tree search (Sec. 4.2.2) */

#define MS_DRIVER_AUTO 0      /* library picks per model */
#define MS_DRIVER_STEPS 1     /* one launch per merged group, stream-ordered */
#define MS_DRIVER_GRAPH 2     /* hipGraph of `unroll` steps, replayed */
#define MS_DRIVER_PERSISTENT 3 /* one launch per run: each workgroup owns batch
                                  columns and executes every group of every step */
#define MS_DRIVER_WINDOW 4    /* stage-major: each merged group runs over a window of
                                 steps before the groups that depend on it.  Only for
                                 models with no recurrence other than each neuron's and
                                 filter's own state (feedforward layers and chains; the
                                 one-step synapse delay separates the stages); other
                                 models get MS_E_INVALID with the reason.  Same results
                                 as the time-major drivers: every operator still sees
                                 exactly the values of its own step (Sec. 4.1). */

/* Input precision of the dense window products (Sec. 3.1 lets the user pick the
 * simulation dtype; the paper's choices are float32/float64, bf16 is this
 * library's addition for matrix cores).  MS_GEMM_BF16 makes the window driver
 * run every merged DotInc group with constant weights, M >= 64, K >= 16,
 * K % 8 == 0 and minibatch % 4 == 0 on bf16 MFMA: the weights are rounded to
 * bf16 (nearest even) once at creation, the signal operand as it is read,
 * products accumulate in fp32 and are added to the fp32 destination.  All
 * other operators stay fp32.  Any other driver with MS_GEMM_BF16 is
 * MS_E_INVALID. */
#define MS_GEMM_F32 0
#define MS_GEMM_BF16 1

/* Decoding of spiking ensembles (the `decode` option).  MS_DECODE_DENSE, the
 * method as the paper merges it, computes every decoded output as the full
 * product of the decoders with the ensemble's output vector (Sec. 2, the
 * decoder DotInc of each connection).  MS_DECODE_EVENT reads only the decoder
 * columns of neurons that spiked in the step, from a neuron-major copy of the
 * decoders made at creation (as much device memory again as the decoders):
 * a neuron that does not spike contributes an exact zero, so the outputs are
 * equal to the dense ones (up to the sign of a zero sum).  It applies to the
 * small-minibatch fused-ensemble kernel of the time-major drivers (steps and
 * graph, minibatch < 32) and to spiking ensembles; elsewhere decoding stays
 * dense.  Other values are MS_E_INVALID. */
#define MS_DECODE_DENSE 0
#define MS_DECODE_EVENT 1

/* Operator fusion (the `fuse` option).  The paper merges operators of one type
 * (Sec. 4.2.1); these fuse operators of different types that always run
 * together, with the same results:
 *   MS_FUSE_ENSEMBLES: each ensemble's bias reset, encoder DotInc, neuron
 *     update and decoder DotIncs become one operator (J is never stored);
 *   MS_FUSE_SYNAPSES: in the time-major launch drivers (STEPS, GRAPH), the
 *     tail of the connections of Fig. 2 -- transform DotInc, synaptic filter
 *     and the Copy of the filtered value into the post input (with that
 *     input's reset) -- becomes one launch at the filter's place at the end of
 *     the step, which also sums the filtered values into the post inputs of
 *     the next step (every run starts with a launch that sums them from the
 *     filter state).  Applied to the connections whose signals allow it (each
 *     filtered value copied once, post inputs touched by nothing else before
 *     the copy, no probe on them); the others keep their separate operators. */
#define MS_FUSE_ENSEMBLES 1
#define MS_FUSE_SYNAPSES 2

typedef struct {
  double dt;                  /* seconds, default 0.001 */
  int32_t minibatch;          /* B >= 1, default 1 */
  int32_t unroll;             /* steps per graph launch, default 10 */
  int32_t planner;            /* MS_PLANNER_*, default TREE */
  int32_t planner_depth;      /* tree search depth n, default 3 */
  int32_t merge;              /* 0: one operator per group (no merging) */
  int32_t sort;               /* 0: keep signals/operators in build order */
  int32_t simplify;           /* 0: skip simplification */
  int32_t fuse;               /* operator fusion, a set of MS_FUSE_* bits (default
                                 both; 0 keeps every operator of the lowered model
                                 separate) */
  int32_t driver;             /* MS_DRIVER_* */
  int32_t device;             /* HIP device ordinal */
  void* stream;               /* hipStream_t to run on, NULL = library-owned */
  int64_t probe_capacity_steps; /* initial probe/feed staging capacity */
  int32_t gemm_dtype;         /* MS_GEMM_F32 (default) or MS_GEMM_BF16 */
  int32_t decode;             /* MS_DECODE_DENSE (default) or MS_DECODE_EVENT */
  int32_t spike_probe_bits;   /* 1: spike probes (MS_REF_NEURONS targets of
                                 spiking LIF ensembles, no synapse) are recorded
                                 as one bit per neuron and step (window driver
                                 only; see ms_sim_probe_read_bits); default 0 */
} ms_sim_opts;

/* Fill `opts` with the defaults listed above. */
void ms_sim_opts_default(ms_sim_opts* opts);

/* ------------------------------------------------------------------- plan */

/* Host-only build + plan (no GPU needed): computes gains, biases and decoders
 * in double, lowers the model to signals and operators, and runs merging,
 * planning, sorting and simplification.  The plan is a snapshot; later edits of
 * the model do not affect it. */
ms_status ms_plan_create(const ms_model* model, const ms_sim_opts* opts, ms_plan** out);
void ms_plan_destroy(ms_plan* plan);

/* The plan as a JSON document (base arrays, signal placement, operator groups in
 * execution order with their operators and index arrays).  Writes at most `cap`
 * bytes including the terminating NUL; *len_out receives the full length
 * (without NUL), so a call with cap == 0 sizes the buffer. */
ms_status ms_plan_export_json(const ms_plan* plan, char* buf, int64_t cap, int64_t* len_out);

#define MS_PARAM_GAIN 0       /* [n] */
#define MS_PARAM_BIAS 1       /* [n] */
#define MS_PARAM_DECODERS 2   /* [n][d_fn] for (ensemble, function) */

/* Copy a built parameter (double, as computed by the build step) into `out`
 * (capacity `cap` doubles); *n_out receives the element count. */
ms_status ms_plan_get_param(const ms_plan* plan, int32_t which, int32_t ensemble,
                            int32_t function, double* out, int64_t cap, int64_t* n_out);

/* Copy parameter base array `base` (ids as in the JSON export) as the float32
 * values the simulation uses: [rows][cols] row-major.  For the batched state
 * array: the value each row starts from in every batch column (zero except
 * the learned decoders of PES connections).  *n_out receives the element
 * count; out == NULL sizes it. */
ms_status ms_plan_export_base(const ms_plan* plan, int32_t base, float* out, int64_t cap,
                              int64_t* n_out);

/* -------------------------------------------------------------- simulator */

ms_status ms_sim_create(const ms_model* model, const ms_sim_opts* opts, ms_sim** out);
void ms_sim_destroy(ms_sim* sim);

/* One input feed: data laid out [minibatch][n_steps][node size] float32;
 * on_device != 0 means `data` is a device pointer on the simulator's device. */
typedef struct {
  int32_t node_id;
  int32_t on_device;
  const float* data;
} ms_feed;

/* Advance the simulation n_steps timesteps (paper Sec. 3.1 sim.run).  Steps
 * continue from the current state; probes append.  Feeds for input nodes not
 * listed read zeros.  Asynchronous with respect to the host unless a probe or
 * state read follows; ms_sim_sync waits. */
ms_status ms_sim_run_steps(ms_sim* sim, int64_t n_steps, const ms_feed* feeds, int32_t n_feeds);
/* Wait until every launch of earlier ms_sim_run_steps calls has finished (the
 * paper's run_steps returns with the steps done, Sec. 3.1; here the wait is
 * explicit so that runs can be queued). */
ms_status ms_sim_sync(ms_sim* sim);

/* Number of steps recorded since creation or the last reset (the time axis of
 * the probe data, Sec. 3.1). */
ms_status ms_sim_steps(const ms_sim* sim, int64_t* n_steps_out);

/* Probe width: values per batch row per step, the last axis of the probe data
 * [batch, steps, width] (Sec. 3.1). */
ms_status ms_sim_probe_width(const ms_sim* sim, int32_t probe_id, int32_t* width_out);

/* Copy probe `probe_id`'s record, [minibatch][steps][width] float32, into `out`
 * (host memory unless out_on_device != 0).  cap_elems must be at least
 * minibatch * steps * width. */
ms_status ms_sim_probe_read(ms_sim* sim, int32_t probe_id, float* out, int64_t cap_elems,
                            int32_t out_on_device);

/* Spike probe record as bitmasks (paper Sec. 3.1 sim.data of a spike probe;
 * a spiking neuron's output is 0 or amplitude / dt, so one bit per neuron and
 * step holds it).  Only for a simulator created with spike_probe_bits = 1 and a
 * probe recorded that way (else MS_E_INVALID); ms_sim_probe_read of such a
 * probe expands the bits to the values.  out: [minibatch][steps][nw] uint32,
 * nw = ceil(width / 32); bit j of word k is neuron 32 k + j of the probe (bits
 * past the width are 0).  cap_words >= minibatch * steps * nw, else
 * MS_E_INVALID.  out_on_device: out is device memory on the simulator's GPU;
 * otherwise host memory (the call then allocates a device staging buffer). */
ms_status ms_sim_probe_read_bits(ms_sim* sim, int32_t probe_id, uint32_t* out, int64_t cap_words,
                                 int32_t out_on_device);

/* Probe read that allocates nothing, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Same result as ms_sim_probe_read into host memory (out:
 * host buffer, [minibatch][steps][width] float32, cap_elems at least
 * minibatch * steps * width), but the device-side transposition is staged in a
 * fixed array of MS_PROBE_READ_STATIC_MAX floats (16 MiB) that each GPU the
 * library runs on holds until the process ends, instead of a temporary
 * allocation.  A record larger than that is MS_E_INVALID (use
 * ms_sim_probe_read).  Every simulator on one GPU shares that GPU's array:
 * calls that overlap on one GPU (several host threads) race.  Returns after
 * the copy into `out` has finished. */
#define MS_PROBE_READ_STATIC_MAX (1 << 22)
ms_status ms_sim_probe_read_static(ms_sim* sim, int32_t probe_id, float* out, int64_t cap_elems);

/* Restore the initial state (V = 0, refractory 0, filters 0, learned
 * decoders back to their initial value) and clear probes (paper Sec. 3.1
 * sim.reset()). */
ms_status ms_sim_reset(ms_sim* sim);

/* State access for checkpoint/resume and injected-state tests.  Host buffers.
 *   MS_STATE_VOLTAGE, MS_STATE_REFRACTORY: id = ensemble, [minibatch][n_neurons]
 *   MS_STATE_SYNAPSE: id = connection with a synapse, [minibatch][post width]
 *   MS_STATE_PROBE_SYNAPSE: id = probe with a synapse, [minibatch][width] */
#define MS_STATE_VOLTAGE 0
#define MS_STATE_REFRACTORY 1
#define MS_STATE_SYNAPSE 2
#define MS_STATE_PROBE_SYNAPSE 3
#define MS_STATE_LEARNED_DECODERS 4  /* id = learning connection, [minibatch][n][k] (D^b) */
#define MS_STATE_PES_ACTIVITY 5      /* id = learning connection with a pre synapse,
                                        [minibatch][n] (a^b) */
ms_status ms_sim_get_state(ms_sim* sim, int32_t which, int32_t id, float* out, int64_t cap_elems);
ms_status ms_sim_set_state(ms_sim* sim, int32_t which, int32_t id, const float* in, int64_t n_elems);

/* Per-run timing of the last ms_sim_run_steps (HIP events on the simulator's
 * stream around the simulation launches, excluding feed staging); ms.  The
 * quantity behind the speed comparisons of Sec. 5.1 (simulation time of a
 * run, repeated and averaged). */
ms_status ms_sim_last_run_ms(ms_sim* sim, double* ms_out);

/* Failure detection for the caller's data (not a part of the paper's method):
 * with on != 0, every later ms_sim_run_steps and ms_sim_train_step first
 * scans each feed for NaN and Inf (host feeds on the host, device feeds with
 * a counting kernel and a wait) and returns MS_E_NUMERIC, naming the node and
 * the count, before anything runs.  Off by default (the scan reads every feed
 * once more).  Setting the environment variable MS_LOG (to anything but "0")
 * prints a summary of the plan on stderr when a simulator is created: the
 * driver, the merged groups launched per step (per window on the window
 * driver) with their sizes, and the bytes of state and parameters. */
ms_status ms_sim_set_check_feeds(ms_sim* sim, int32_t on);

/* The driver actually used (MS_DRIVER_STEPS/GRAPH/PERSISTENT/WINDOW) and the
 * number of merged groups executed per step (WINDOW: launches per window) --
 * the count that operator merging reduces (Sec. 4.2, Fig. 8). */
ms_status ms_sim_info(const ms_sim* sim, int32_t* driver_out, int32_t* groups_per_step_out);

/* Merged operator types (the groups a plan is made of, paper Sec. 4.2). */
#define MS_OP_FEED 0
#define MS_OP_RESET 1
#define MS_OP_COPY 2
#define MS_OP_COPY_INC 3
#define MS_OP_ELEMENTWISE_INC 4
#define MS_OP_DOT_INC 5
#define MS_OP_LIF 6
#define MS_OP_LIF_RATE 7
#define MS_OP_LOWPASS 8
#define MS_OP_ENSEMBLE 9  /* fused bias + encoders + neurons + decoders of an ensemble */
#define MS_OP_SYNAPSE_SCATTER 10  /* fused transform + lowpass + copy into post inputs */
#define MS_OP_LEARNED_DECODE 11   /* decoding with per-batch-element decoders */
#define MS_OP_PES 12              /* the PES update of those decoders */
#define MS_OP_PES_DECODE_UPDATE 13 /* both in one pass over the decoders (launch drivers,
                                      when the error is known before the decode) */

/* Per-kernel timing for measurement (the cost of each kind of merged operator
 * group, Sec. 4.2 and 5.1).  With timing on (on != 0), every merged group's
 * launch is timed: on the STEPS driver its kernels are launched with
 * hipExtLaunchKernelGGL, the first recording the group's begin event when it
 * starts executing and each recording the end event when it finishes, so that
 * host launch latency is not counted; on the WINDOW driver HIP events are
 * recorded on the stream the launch runs on.  ms_sim_kernel_time then returns,
 * for operator type `op_type` (MS_OP_*) during the last ms_sim_run_steps call
 * (it waits for that call to finish), the busy time in ms -- the length of the
 * union of those launches' intervals, so that launches running at once on
 * different streams count once (it equals the summed durations when they do
 * not overlap) -- and the number of launches.  Only the WINDOW and STEPS
 * drivers time individual launches (MS_E_STATE otherwise).  Timing adds event
 * records to every launch: leave it off for throughput runs. */
ms_status ms_sim_set_timing(ms_sim* sim, int32_t on);
ms_status ms_sim_kernel_time(ms_sim* sim, int32_t op_type, double* ms_out, int64_t* launches_out);

/* ------------------------------------------------------------- training */

/* Training by gradient descent (paper Sec. 3.2: an objective on probe outputs
 * minimised with a gradient-descent optimiser, the gradient taken through
 * every step of the unrolled simulation).
 *
 * One call of ms_sim_train_step:
 *   1. restores the initial state (as ms_sim_reset, probes cleared) and runs
 *      n_steps with the feeds (as ms_sim_run_steps; the probes record them);
 *   2. computes the objective: for each target, the mean over minibatch rows,
 *      steps and probe dimensions of (probe value - target)^2, summed over
 *      the targets (mean squared error);
 *   3. computes dL/dp for every trained parameter, through all n_steps;
 *   4. if learning_rate != 0, updates each trained parameter p <- p -
 *      learning_rate * dL/dp.
 * *loss_out (if not NULL) receives the objective of step 2 (double); the call
 * returns after the step has finished.
 *
 * Trained parameters: each ensemble's gain-scaled encoders [n][d] and biases
 * [n]; each (ensemble, function)'s solved decoders (shared by every
 * connection and probe that decodes that function); each connection's
 * explicit decoders and its transform (matrix or scalar).  Gains of
 * neuron-space inputs, node constants and filter coefficients stay fixed.
 *
 * Requirements (MS_E_STATE otherwise, with the reason): the simulator runs on
 * MS_DRIVER_WINDOW with fp32 products, was created with fuse = 0 and
 * simplify = 0 (fusion and simplification turn parameters into parts of
 * other operators or into constants), its ensembles use rate neurons
 * (MS_NEURON_LIF_RATE or MS_NEURON_RELU: the spiking LIF has no useful
 * derivative) and it has no learning rule; n_steps must fit in one window of
 * the window driver (its versioned signals hold every step for the backward
 * pass).  Memory: the backward pass holds one more array the size of the
 * window's versioned signals, plus gradients the size of the trained
 * parameter bases.
 *
 * Targets: data [minibatch][n_steps][probe width] float32, host memory
 * unless on_device != 0. */
typedef struct {
  int32_t probe_id;
  int32_t on_device;
  const float* data;
} ms_target;

ms_status ms_sim_train_step(ms_sim* sim, int64_t n_steps, const ms_feed* feeds, int32_t n_feeds,
                            const ms_target* targets, int32_t n_targets, double learning_rate,
                            double* loss_out);

#define MS_TRAIN_ENCODERS 0       /* id = ensemble: [n][d] gain-scaled encoders */
#define MS_TRAIN_BIASES 1         /* id = ensemble: [n] */
#define MS_TRAIN_DECODERS 2       /* id = ensemble, function = MS_FN_*: [n][d_fn] */
#define MS_TRAIN_CONN_DECODERS 3  /* id = connection with explicit decoders: [n][cols] */
#define MS_TRAIN_TRANSFORM 4      /* id = connection: [rows][cols], or [1] for a scalar */

/* Read a trained parameter's current value (gradient == 0) or its gradient
 * from the last ms_sim_train_step (gradient != 0; zeros before the first),
 * as float32 in the layout listed above, into host memory `out` (capacity
 * `cap` floats; out == NULL sizes it).  *n_out receives the element count.
 * MS_E_INVALID if the model has no such parameter. */
ms_status ms_sim_train_param(ms_sim* sim, int32_t which, int32_t id, int32_t function, int32_t gradient,
                             float* out, int64_t cap, int64_t* n_out);
/* Overwrite a trained parameter (checkpoint restore; n must equal its element
 * count).  Later runs and training steps use the new values. */
ms_status ms_sim_set_train_param(ms_sim* sim, int32_t which, int32_t id, int32_t function, const float* in,
                                 int64_t n);

/* Timing kinds of a training step's backward pass for ms_sim_kernel_time
 * (with timing on, the forward groups are timed under their MS_OP_* types as
 * in ms_sim_run_steps): */
#define MS_OP_GRAD_WEIGHTS 14  /* weight gradients of merged DotInc groups with both sides
                                  of W at least 64 (matrix-core products) */
#define MS_OP_GRAD_INPUTS 15   /* adjoints of the DotInc inputs (products with W^T) */
#define MS_OP_GRAD_OTHER 16    /* objective, elementwise, neuron and filter reverses, update */
#define MS_OP_GRAD_WEIGHTS_SMALL 17  /* weight gradients of the other DotInc groups */

const char* ms_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MERGESIM_H */
