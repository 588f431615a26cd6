// Device code of mergesim: one kernel per merged operator type (paper
// Sec. 4.2.1: a merged group reads its operands as one gather from the base
// arrays, computes once, and writes once), plus the persistent per-batch-column
// interpreter that runs every group of every step in a single launch.
//
// Batched signals live in the `state` base array; element (row r, batch b) is at
// st[r * rs + b * cs].  Launch drivers use rs = B, cs = 1 (minibatch
// contiguous, coalesced across the batch); the persistent driver uses rs = 1,
// cs = rows (each batch column contiguous, coalesced across rows, since one
// workgroup owns one column).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

// Pointers read out of device-resident descriptors are generic pointers to the
// compiler; casting them back to the global address space turns flat memory
// instructions (which also wait on LDS traffic) into global loads.
template <class T>
using gptr = const __attribute__((address_space(1))) T*;
template <class T>
__device__ __forceinline__ gptr<T> G(const T* p) {
  return (gptr<T>)p;
}

// A record of a table that no kernel writes while it runs (group descriptors,
// per-op records), read word by word through the constant address space.  At a
// workgroup-uniform address the compiler then issues scalar loads; through a
// generic pointer it must use vector loads in any kernel that also stores,
// since it cannot prove the table unchanged.
template <class T>
using kptr = const __attribute__((address_space(4))) T*;
template <class T>
__device__ __forceinline__ T kload(const T* p) {
  static_assert(sizeof(T) % 4 == 0, "records of whole 32-bit words");
  struct Words {
    int32_t v[sizeof(T) / 4];
  } x;
  kptr<int32_t> w = (kptr<int32_t>)p;
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) x.v[i] = w[i];
  return __builtin_bit_cast(T, x);
}

// Row of the r-th work item of an operand: slice start + r, or idx[r].
struct Opnd {
  const int32_t* idx;
  int64_t start;
};

__device__ __forceinline__ int64_t rowof(const Opnd& o, int64_t r) {
  return o.idx ? (int64_t)G(o.idx)[r] : o.start + r;
}

struct NeuronParams {
  float tau_rc, tau_ref, amp;                     // uniform values
  float full;                                     // expm1(-dt / tau_rc), uniform
  const float *tau_rc_r, *tau_ref_r, *amp_r;      // per-row values or null
  const float* full_r;                            // per-row expm1(-dt / tau_rc) or null
  int32_t relu;                                   // rate neurons: 1 = rectified linear
  float sigma;                                    // rate neurons: > 0 = soft LIF rate, its smoothing
  const float* sigma_r;                           // per-row smoothing or null
};

// log(1 + y) for y >= 0 from the hardware log2 (v_log_f32, about 1 ulp):
// with u = 1 + y rounded, log(u) * y / (u - 1) cancels the rounding of u
// (Kahan's method; a few ulp), and y itself where u rounds to 1.
__device__ __forceinline__ float log1p_hw(float y) {
  const float u = 1.0f + y;
  if (u == 1.0f) return y;
  return __builtin_amdgcn_logf(u) * 0.69314718055994531f * (y / (u - 1.0f));
}

// Soft LIF rate curve r(J) (without amplitude): the LIF rate with max(J - 1, 0)
// replaced by rho = s log(1 + exp(x)), x = (J - 1) / s.  For x >= -15,
// log(1 + 1/rho) is evaluated directly from rho = s softplus(x); below, where
// softplus(x) = exp(x) to a relative exp(x) / 2 < 2e-7, as log1p(rho) -
// log(rho) with log(rho) = log(s) + x, so nothing overflows or underflows.
// exp(x) comes from the hardware exp2 (v_exp_f32) of x log2(e), whose rounding
// adds a relative |x| 2^-24 (at most 1e-6 here); reciprocals from v_rcp_f32.
// Also returns rho'/rho and rho for the derivative.
__device__ __forceinline__ float soft_lif_rate(float j, float tau_rc, float tau_ref, float s, float* dlog,
                                               float* rho_out) {
  constexpr float kLog2e = 1.44269504088896341f;
  const float inv_s = __builtin_amdgcn_rcpf(s);
  const float x = (j - 1.0f) * inv_s;
  float q, rho;
  if (x < -15.0f) {
    rho = s * __builtin_amdgcn_exp2f(x * kLog2e);
    q = log1p_hw(rho) - (__builtin_amdgcn_logf(s) * 0.69314718055994531f + x);
    *dlog = inv_s;   // sigmoid(x) / (s softplus(x)) = 1 / s to 2e-7
  } else {
    const float e = __builtin_amdgcn_exp2f(x * kLog2e);
    const float sp = x > 15.0f ? x + __builtin_amdgcn_exp2f(-x * kLog2e) : log1p_hw(e);
    rho = s * sp;
    q = log1p_hw(__builtin_amdgcn_rcpf(rho));
    *dlog = x > 15.0f ? __builtin_amdgcn_rcpf(rho) : e * __builtin_amdgcn_rcpf((1.0f + e) * rho);
  }
  *rho_out = rho;
  return __builtin_amdgcn_rcpf(tau_ref + tau_rc * q);
}

struct FilterParams {
  float a, b;                 // y = a y + b v (uniform)
  const float *a_r, *b_r;     // per-row or null
};

struct Strides {
  int64_t rs, cs;
};

__device__ __forceinline__ int64_t at(const Strides& s, int64_t r, int64_t b) {
  return r * s.rs + b * s.cs;
}

// --------------------------------------------------------- per-item bodies
// Each body computes one (row, batch) work item of a merged group.

__device__ __forceinline__ float neuron_update(int ntype, float j, float& v, float& rf, float tau_rc,
                                               float tau_ref, float amp, float full, float dt,
                                               float inv_tau);

__device__ __forceinline__ void lif_item(float* st, const Strides& S, int64_t r, int64_t b,
                                         const Opnd& J, const Opnd& s, const Opnd& V, const Opnd& R,
                                         const NeuronParams& np, float dt) {
  const float tau_rc = np.tau_rc_r ? G(np.tau_rc_r)[r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? G(np.tau_ref_r)[r] : np.tau_ref;
  const float amp = np.amp_r ? G(np.amp_r)[r] : np.amp;
  const float full = np.full_r ? G(np.full_r)[r] : np.full;
  const int64_t jv = at(S, rowof(J, r), b), vv = at(S, rowof(V, r), b), rv = at(S, rowof(R, r), b);
  float v = st[vv], rf = st[rv];
  const float out = neuron_update(0, st[jv], v, rf, tau_rc, tau_ref, amp, full, dt, 1.0f / tau_rc);
  st[vv] = v;
  st[rv] = rf;
  st[at(S, rowof(s, r), b)] = out;
}

__device__ __forceinline__ void lif_rate_item(float* st, const Strides& S, int64_t r, int64_t b,
                                              const Opnd& J, const Opnd& s, const NeuronParams& np) {
  const float tau_rc = np.tau_rc_r ? G(np.tau_rc_r)[r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? G(np.tau_ref_r)[r] : np.tau_ref;
  const float amp = np.amp_r ? G(np.amp_r)[r] : np.amp;
  const float j = st[at(S, rowof(J, r), b)];
  float out = 0.0f;
  if (np.relu) {
    out = amp * fmaxf(j, 0.0f);
  } else if (np.sigma > 0.0f) {
    float dl, rho;
    out = amp * soft_lif_rate(j, tau_rc, tau_ref, np.sigma_r ? G(np.sigma_r)[r] : np.sigma, &dl, &rho);
  } else if (j > 1.0f) {
    out = amp / (tau_ref + tau_rc * log1pf(1.0f / (j - 1.0f)));
  }
  st[at(S, rowof(s, r), b)] = out;
}

// One lowpass step y <- a y + c v with its rounding fixed (c v rounded, then
// a y added in one fma), so that every kernel that runs a filter, fused or
// not, gives the same bits.
__device__ __forceinline__ float lowpass_step(float a, float y, float c, float v) { return fmaf(a, y, c * v); }

__device__ __forceinline__ void lowpass_item(float* st, const Strides& S, int64_t r, int64_t b,
                                             const Opnd& y, const Opnd& v, const FilterParams& fp) {
  const float a = fp.a_r ? G(fp.a_r)[r] : fp.a;
  const float c = fp.b_r ? G(fp.b_r)[r] : fp.b;
  const int64_t yi = at(S, rowof(y, r), b);
  st[yi] = lowpass_step(a, st[yi], c, st[at(S, rowof(v, r), b)]);
}

__device__ __forceinline__ float src_val(const float* base, const Strides& S, int bcast, int64_t row,
                                         int64_t b) {
  return bcast ? G(base)[row] : base[at(S, row, b)];
}

// dst (+)= sum of src entries of unique destination u (ptr == null: one entry)
__device__ __forceinline__ void copy_inc_item(float* st, const Strides& S, int64_t u, int64_t b,
                                              const Opnd& dst, const float* src_base, const Opnd& src,
                                              int bcast, const int32_t* ptr) {
  const int64_t di = at(S, rowof(dst, u), b);
  float acc = st[di];
  if (ptr) {
    for (int32_t e = G(ptr)[u]; e < G(ptr)[u + 1]; ++e) acc += src_val(src_base, S, bcast, rowof(src, e), b);
  } else {
    acc += src_val(src_base, S, bcast, rowof(src, u), b);
  }
  st[di] = acc;
}

__device__ __forceinline__ void elem_inc_item(float* st, const Strides& S, int64_t u, int64_t b,
                                              const Opnd& dst, const float* a_base, const Opnd& a,
                                              const float* x_base, const Opnd& x, const int32_t* ptr) {
  const int64_t di = at(S, rowof(dst, u), b);
  float acc = st[di];
  if (ptr) {
    for (int32_t e = G(ptr)[u]; e < G(ptr)[u + 1]; ++e) acc += G(a_base)[rowof(a, e)] * x_base[at(S, rowof(x, e), b)];
  } else {
    acc += G(a_base)[rowof(a, u)] * x_base[at(S, rowof(x, u), b)];
  }
  st[di] = acc;
}

// one output row m of op `op` for batch b: dst[m] += W[m, :] . x
__device__ __forceinline__ void dot_row_item(float* st, const Strides& S, int64_t op, int32_t m, int64_t b,
                                             int32_t K, const float* W, const int32_t* w_row,
                                             const int32_t* x_row, const int32_t* d_row) {
  gptr<float> w = G(W) + ((int64_t)G(w_row)[op] + m) * K;
  const int64_t x0 = G(x_row)[op];
  float acc = 0.0f;
  if ((K & 3) == 0) {
    // weight rows are 16-byte aligned when K is a multiple of 4: four at a time
    typedef float f4v __attribute__((ext_vector_type(4)));
    const __attribute__((address_space(1))) f4v* w4 = (const __attribute__((address_space(1))) f4v*)w;
    for (int32_t k4 = 0; k4 < K / 4; ++k4) {
      const f4v wv = w4[k4];
      const int64_t k = 4 * (int64_t)k4;
      acc += wv[0] * st[at(S, x0 + k, b)];
      acc += wv[1] * st[at(S, x0 + k + 1, b)];
      acc += wv[2] * st[at(S, x0 + k + 2, b)];
      acc += wv[3] * st[at(S, x0 + k + 3, b)];
    }
  } else {
    for (int32_t k = 0; k < K; ++k) acc += w[k] * st[at(S, x0 + k, b)];
  }
  st[at(S, (int64_t)G(d_row)[op] + m, b)] += acc;
}

// ------------------------------------------------------ fused ensemble ops
// One merged group of fused ensemble operators.  Per op: n neurons, rows of its
// represented input x (d rows, -1: none), gain-scaled encoders (row of the
// [n x d] block in the encoder base), bias, state V / refractory, spikes (-1:
// not stored) and, per fused function f, the decoder block [df[f] x n] and the
// output rows.  Neuron parameters are uniform or per op.
constexpr int kMaxFns = 2;
constexpr int kMaxDec = 16;   // total decoded outputs of one fused op

// Rows of one fused op, packed so a wavefront fetches them with one scalar load.
struct EnsOp {
  int32_t n, x, enc, bias, V, ref, s;
  float inv_tau;                      // 1 / tau_rc
  int32_t D[kMaxFns], d[kMaxFns];
  float tau_rc, tau_ref, amp, full;   // neuron parameters of this op
  float tau6;                         // tau_rc / 6 (the spike-time series' scale)
};

struct EnsDesc {
  int32_t d, ntype, nf, ndec;
  int32_t df[kMaxFns];
  const EnsOp* ops;
  const float* enc;      // encoder base [rows][d]
  const float* encT;     // the same encoders with each op's block stored [d][n] (or null)
  const float* bias;     // bias base (vector)
  const float* D[kMaxFns];  // decoder bases [rows][n]
  int32_t Dcols[kMaxFns];   // row stride of each decoder base
  // event-driven decoding (spiking, or null): op k's decoders neuron-major,
  // neuron r's decoded outputs at decT[k * dT_op + r * dT_row + q], rows padded
  // with zeros to dT_row = dec_bucket(ndec) values
  const float* decT;
  int64_t dT_op;
  int32_t dT_row;
  // window driver: fused connection chains into the ops' inputs (per op 8
  // ints, see k_w_ens; null: none) and their transforms' weight base
  const int32_t* chain;
  const float* chain_w;
  int32_t chain_wcols;
};


// exp(x) - 1 for -1/16 <= x <= 0 (the partial-step integration factor):
// degree-6 Taylor polynomial, truncation error below 1e-11 relative.
__device__ __forceinline__ float expm1_small(float x) {
  float p = 1.0f / 720.0f;
  p = fmaf(p, x, 1.0f / 120.0f);
  p = fmaf(p, x, 1.0f / 24.0f);
  p = fmaf(p, x, 1.0f / 6.0f);
  p = fmaf(p, x, 0.5f);
  p = fmaf(p, x, 1.0f);
  return p * x;
}

// -ln(1 - q) for 0 <= q <= 1/16 (the crossing time's logarithm): the series
// q (1 + q/2 + q^2/3 + ... + q^6/7), truncation below 1e-9 relative.  Unlike
// a logarithm of the rounded 1 - q, it keeps full relative precision for
// small q, where an error of one ulp of 1 would move the end of the
// refractory period by about tau_rc * 6e-8 s.
__device__ __forceinline__ float neg_log1m_small(float q) {
  float p = 1.0f / 7.0f;
  p = fmaf(p, q, 1.0f / 6.0f);
  p = fmaf(p, q, 1.0f / 5.0f);
  p = fmaf(p, q, 1.0f / 4.0f);
  p = fmaf(p, q, 1.0f / 3.0f);
  p = fmaf(p, q, 0.5f);
  p = fmaf(p, q, 1.0f);
  return p * q;
}

// LIF (or rate) update of one neuron for input current j; V, rf updated in place.
// Spiking: exact integration over the non-refractory part of the step (the
// whole-step factor `full` = expm1(-dt/tau_rc) is precomputed; a partial step
// uses the polynomial above or expm1f), strict threshold 1, crossing time from
// the overshoot q = (V - 1)/(J - 1) (the hardware reciprocal, v_rcp_f32, about
// one ulp; -ln(1 - q) from the series above for q <= 1/16, log1pf otherwise),
// reset to 0, refractory period measured from the crossing.  Rate:
// amplitude / (tau_ref + tau_rc log1p(1/(J-1))).
__device__ __forceinline__ float neuron_update(int ntype, float j, float& v, float& rf, float tau_rc,
                                               float tau_ref, float amp, float full, float dt,
                                               float inv_tau) {
  if (ntype == 2) return amp * fmaxf(j, 0.0f);   // rectified linear
  if (ntype != 0) {
    return j > 1.0f ? amp / (tau_ref + tau_rc * log1pf(1.0f / (j - 1.0f))) : 0.0f;
  }
  const float integ = fminf(fmaxf(dt - rf, 0.0f), dt);
  float e = full;
  if (rf > 0.0f) {
    const float x = -integ * inv_tau;
    e = x >= -0.0625f ? expm1_small(x) : expm1f(x);
  }
  v = v - (j - v) * e;
  rf = fmaxf(rf - dt, 0.0f);
  if (v > 1.0f) {
    float since = 0.0f;
    const float drive = j - 1.0f;
    if (drive > 0.0f) {
      const float q = (v - 1.0f) * __builtin_amdgcn_rcpf(drive);
      since = q >= 1.0f ? integ
                        : fminf(tau_rc * (q <= 0.0625f ? neg_log1m_small(q) : -log1pf(-q)), integ);
    }
    v = 0.0f;
    rf = tau_ref - since;
    return amp / dt;
  }
  v = fmaxf(v, 0.0f);
  return 0.0f;
}

// Shorter polynomials for the branch-free update below, where |x| <= 1/16 and
// 0 <= q <= 1/16: expm1 to degree 5 (truncation below 2e-9 relative) and
// -ln(1 - q) = q (1 + q/2 + ... + q^5/6) (truncation below 1e-8 relative),
// both well under float32 rounding.
__device__ __forceinline__ float expm1_bf(float x) {
  float p = 1.0f / 120.0f;
  p = fmaf(p, x, 1.0f / 24.0f);
  p = fmaf(p, x, 1.0f / 6.0f);
  p = fmaf(p, x, 0.5f);
  p = fmaf(p, x, 1.0f);
  return p * x;
}

// 6 (-ln(1 - q)) / q to the same order, 6 + 3q + 2q^2 + 1.5q^3 + 1.2q^4 + q^5:
// with the leading coefficient 1 the first Horner step is an add of a
// literal, so no constant has to sit in a register.
__device__ __forceinline__ float neg_log1m6_bf(float q) {
  float p = q + 1.2f;
  p = fmaf(p, q, 1.5f);
  p = fmaf(p, q, 2.0f);
  p = fmaf(p, q, 3.0f);
  return fmaf(p, q, 6.0f);
}

// Branch-free form of the spiking update above for dt / tau_rc <= 1/16, with
// every path computed and the results selected, so that lanes whose neurons
// spike or sit in their refractory period do not serialise the wavefront:
//   * the partial-step factor comes from the polynomial on every lane (at a
//     whole step it is expm1(-dt / tau_rc) to within rounding, so the
//     refractory state needs no select);
//   * a crossing's overshoot ratio q stays below 1 - exp(-1/16) < 1/16 on any
//     trajectory from V <= 1, so -ln(1 - q) comes from the series;
//   * the crossing time is min(tau_rc (-ln(1 - q)), integ) when J > 1: the
//     series grows with q, and for q >= 1 (a voltage above threshold set from
//     outside) it exceeds tau_rc >= 16 dt >= integ, so the clamp of the
//     crossing to the start of the step needs no test of its own.
// The series is evaluated as (tau_rc / 6) q (6 + 3q + ... + q^5).  Clamps are
// v_med3 (no operand canonicalisation), the refractory countdown
// reuses dt - rf negated (exact), and (V - 1) / (J - 1) is one fma on the
// reciprocal (V - 1 is exact for V in [1/2, 2]; elsewhere the fma rounds once
// where the product of the rounded difference rounded twice).
// Returns the neuron output (amp_dt = amplitude / dt or 0).
// tau6 = tau_rc / 6.
__device__ __forceinline__ float lif_update_bf(float j, float& v, float& rf, float tau6, float tau_ref,
                                               float amp_dt, float dt, float inv_tau) {
  const float t = dt - rf;
  const float integ = __builtin_amdgcn_fmed3f(t, 0.0f, dt);           // clamp to [0, dt]
  const float e = expm1_bf(-integ * inv_tau);
  v = v - (j - v) * e;
  const float rf_next = __builtin_amdgcn_fmed3f(-t, 0.0f, __builtin_inff());   // max(rf - dt, 0)
  const float drive = j - 1.0f;
  const float r = __builtin_amdgcn_rcpf(drive);
  const float q = fmaf(v, r, -r);
  // the crossing time, clamped to [0, integ] (a crossing has q > 0), computed
  // on every lane: the empty asm statement takes it as an operand, so that the
  // compiler selects instead of branching on J > 1 (a branch runs both sides
  // anyway when the lanes disagree)
  float since = __builtin_amdgcn_fmed3f(tau6 * (q * neg_log1m6_bf(q)), 0.0f, integ);
  __asm__ volatile("" : "+v"(since));
  since = drive > 0.0f ? since : 0.0f;
  const bool spk = v > 1.0f;
  const float vpos = __builtin_amdgcn_fmed3f(v, 0.0f, __builtin_inff());
  v = spk ? 0.0f : vpos;
  rf = spk ? tau_ref - since : rf_next;
  return spk ? amp_dt : 0.0f;
}

// Sum over the 64 lanes of a wavefront, returned in every lane.  DPP moves
// fold quads, half-rows and rows of 16 lanes; the four row sums are read with
// readlane.  All lanes must be active.
__device__ __forceinline__ float wave_sum(float x) {
  int xi = __builtin_bit_cast(int, x);
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(xi, 0xB1, 0xF, 0xF, true));   // quad [1,0,3,2]
  xi = __builtin_bit_cast(int, x);
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(xi, 0x4E, 0xF, 0xF, true));   // quad [2,3,0,1]
  xi = __builtin_bit_cast(int, x);
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(xi, 0x141, 0xF, 0xF, true));  // row_half_mirror
  xi = __builtin_bit_cast(int, x);
  x += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(xi, 0x140, 0xF, 0xF, true));  // row_mirror
  xi = __builtin_bit_cast(int, x);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 0)) +
         __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 16)) +
         __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 32)) +
         __builtin_bit_cast(float, __builtin_amdgcn_readlane(xi, 48));
}

template <class P>
__device__ __forceinline__ EnsOp op_from_words(P w) {
  EnsOp o;
  o.n = w[0]; o.x = w[1]; o.enc = w[2]; o.bias = w[3]; o.V = w[4]; o.ref = w[5]; o.s = w[6];
  o.inv_tau = __builtin_bit_cast(float, w[7]);
  o.D[0] = w[8]; o.D[1] = w[9]; o.d[0] = w[10]; o.d[1] = w[11];
  o.tau_rc = __builtin_bit_cast(float, w[12]);
  o.tau_ref = __builtin_bit_cast(float, w[13]);
  o.amp = __builtin_bit_cast(float, w[14]);
  o.full = __builtin_bit_cast(float, w[15]);
  o.tau6 = __builtin_bit_cast(float, w[16]);
  return o;
}

__device__ __forceinline__ EnsOp load_op(const EnsOp* ops, int op) {
  return op_from_words(G(reinterpret_cast<const int32_t*>(ops + op)));
}

// The same record at a wavefront-uniform index, through scalar loads (kload).
__device__ __forceinline__ EnsOp load_op_uniform(const EnsOp* ops, int op) {
  return op_from_words((kptr<int32_t>)reinterpret_cast<const int32_t*>(ops + op));
}

// Decoded-output bucket: the smallest of 0, 1, 2, 4, 8, 16 that holds n outputs.
__host__ __device__ __forceinline__ int dec_bucket(int n) {
  return n <= 0 ? 0 : n <= 1 ? 1 : n <= 2 ? 2 : n <= 4 ? 4 : n <= 8 ? 8 : 16;
}

// Ensemble inputs up to this many dimensions are held in registers for the
// whole neuron loop (they would otherwise be re-read for every neuron, since
// the loop stores state through the same pointer).
constexpr int kMaxXReg = 16;

__device__ __forceinline__ void load_input(float (&xr)[kMaxXReg], const float* st, const Strides& S, int32_t x,
                                           int64_t b, int d) {
#pragma unroll
  for (int k = 0; k < kMaxXReg; ++k) xr[k] = k < d ? st[at(S, x + k, b)] : 0.0f;
}

// J = bias + sum_k enc[k] x[k], accumulated in order k = 0..d-1.
__device__ __forceinline__ float input_current(float j, gptr<float> enc, const float (&xr)[kMaxXReg],
                                               const float* st, const Strides& S, int32_t x, int64_t b, int d) {
  if (d <= kMaxXReg) {
#pragma unroll
    for (int k = 0; k < kMaxXReg; ++k)
      if (k < d) j += enc[k] * xr[k];
  } else {
    for (int k = 0; k < d; ++k) j += enc[k] * st[at(S, x + k, b)];
  }
  return j;
}

// One fused op, one batch column, processed by one wavefront (lanes over
// neurons); NDEC >= total decoded outputs (extra slots repeat the last row and
// are never stored).  The decoded outputs are reduced across the wavefront
// and written by lane 0.  V/refractory/x/s/d live in `st` (strides S, column b).
template <int NDEC>
__device__ __forceinline__ void ens_op_wave_t(float* st, const Strides& S, int64_t b, const EnsDesc& E,
                                              const EnsOp& o, int lane, float dt) {
  const int d = o.x >= 0 ? E.d : 0, ndec = E.ndec, df0 = E.df[0];   // ops without input: J = bias
  gptr<float> enc = G(E.enc) + (int64_t)o.enc * d;
  gptr<float> bias = G(E.bias) + o.bias;
  gptr<float> D0 = G(E.D[0]) + (int64_t)o.D[0] * E.Dcols[0];
  gptr<float> D1 = G(E.D[E.nf > 1 ? 1 : 0]) + (int64_t)o.D[E.nf > 1 ? 1 : 0] * E.Dcols[E.nf > 1 ? 1 : 0];
  const int64_t s0 = E.Dcols[0], s1 = E.Dcols[E.nf > 1 ? 1 : 0];
  float acc[NDEC > 0 ? NDEC : 1];
#pragma unroll
  for (int q = 0; q < NDEC; ++q) acc[q] = 0.0f;
  for (int r = lane; r < o.n; r += 64) {
    float j = bias[r];
    for (int k = 0; k < d; ++k) j += enc[(int64_t)r * d + k] * st[at(S, o.x + k, b)];
    float v = 0.0f, rf = 0.0f;
    if (E.ntype == 0) { v = st[at(S, o.V + r, b)]; rf = st[at(S, o.ref + r, b)]; }
    const float sp = neuron_update(E.ntype, j, v, rf, o.tau_rc, o.tau_ref, o.amp, o.full, dt, o.inv_tau);
    if (E.ntype == 0) { st[at(S, o.V + r, b)] = v; st[at(S, o.ref + r, b)] = rf; }
    if (o.s >= 0) st[at(S, o.s + r, b)] = sp;
#pragma unroll
    for (int q = 0; q < NDEC; ++q) {
      const int qq = q < ndec ? q : ndec - 1;
      gptr<float> row = qq < df0 ? D0 + (int64_t)qq * s0 : D1 + (int64_t)(qq - df0) * s1;
      acc[q] += row[r] * sp;
    }
  }
#pragma unroll
  for (int q = 0; q < NDEC; ++q) {
    const float t = wave_sum(acc[q]);
    if (lane == 0 && q < ndec) {
      const int dr = q < df0 ? o.d[0] + q : o.d[1] + (q - df0);
      st[at(S, dr, b)] = t;
    }
  }
}

__device__ __forceinline__ void ens_op_wave(float* st, const Strides& S, int64_t b, const EnsDesc& E, int op,
                                            int lane, float dt) {
  const EnsOp o = load_op_uniform(E.ops, op);
  switch (dec_bucket(E.ndec)) {
    case 0: ens_op_wave_t<0>(st, S, b, E, o, lane, dt); break;
    case 1: ens_op_wave_t<1>(st, S, b, E, o, lane, dt); break;
    case 2: ens_op_wave_t<2>(st, S, b, E, o, lane, dt); break;
    case 4: ens_op_wave_t<4>(st, S, b, E, o, lane, dt); break;
    case 8: ens_op_wave_t<8>(st, S, b, E, o, lane, dt); break;
    default: ens_op_wave_t<16>(st, S, b, E, o, lane, dt); break;
  }
}

// ----------------------------------------------------------- launch kernels
// Work items are (row, batch) pairs flattened as row * B + b; the host checks
// that rows * B fits in 32 bits so the split uses 32-bit division.
#define GRID_ITEM(n)                                                        \
  const uint32_t _i = blockIdx.x * blockDim.x + threadIdx.x;                \
  if (_i >= (uint32_t)(n)) return;                                          \
  const uint32_t _r = _i / (uint32_t)B, _b = _i - _r * (uint32_t)B;

__global__ void k_reset(float* st, Strides S, int32_t B, int64_t rows, Opnd dst, const float* values) {
  GRID_ITEM(rows * B);
  st[at(S, rowof(dst, _r), _b)] = values ? values[_r] : 0.0f;
}

__global__ void k_copy(float* st, Strides S, int32_t B, int64_t rows, Opnd dst, const float* src_base,
                       Opnd src, int bcast) {
  GRID_ITEM(rows * B);
  st[at(S, rowof(dst, _r), _b)] = src_val(src_base, S, bcast, rowof(src, _r), _b);
}

__global__ void k_copy_inc(float* st, Strides S, int32_t B, int64_t rows, Opnd dst, const float* src_base,
                           Opnd src, int bcast, const int32_t* ptr) {
  GRID_ITEM(rows * B);
  copy_inc_item(st, S, _r, _b, dst, src_base, src, bcast, ptr);
}

__global__ void k_elem_inc(float* st, Strides S, int32_t B, int64_t rows, Opnd dst, const float* a_base,
                           Opnd a, const float* x_base, Opnd x, const int32_t* ptr) {
  GRID_ITEM(rows * B);
  elem_inc_item(st, S, _r, _b, dst, a_base, a, x_base, x, ptr);
}

// thread per (op, m, b)
__global__ void k_dot_inc(float* st, Strides S, int32_t B, int64_t nops, int32_t M, int32_t K,
                          const float* W, const int32_t* w_row, const int32_t* x_row, const int32_t* d_row) {
  GRID_ITEM(nops * M * B);
  const uint32_t op = _r / (uint32_t)M;
  dot_row_item(st, S, op, (int32_t)(_r - op * (uint32_t)M), _b, K, W, w_row, x_row, d_row);
}

// wave per (op, m): lanes split K, reduced across the wavefront; loops over b.
__global__ void k_dot_inc_wave(float* st, Strides S, int32_t B, int64_t nops, int32_t M, int32_t K,
                               const float* W, const int32_t* w_row, const int32_t* x_row,
                               const int32_t* d_row) {
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / warpSize;
  const int lane = threadIdx.x % warpSize;
  if (wave >= nops * M) return;
  const int64_t op = wave / M;
  const int32_t m = (int32_t)(wave % M);
  const float* w = W + ((int64_t)w_row[op] + m) * K;
  const int64_t x0 = x_row[op];
  const int64_t d = (int64_t)d_row[op] + m;
  for (int64_t b = 0; b < B; ++b) {
    float acc = 0.0f;
    for (int32_t k = lane; k < K; k += warpSize) acc += w[k] * st[at(S, x0 + k, b)];
    for (int off = warpSize / 2; off > 0; off >>= 1) acc += __shfl_down(acc, off);
    if (lane == 0) st[at(S, d, b)] += acc;
  }
}

__global__ void k_lif(float* st, Strides S, int32_t B, int64_t rows, Opnd J, Opnd s, Opnd V, Opnd R,
                      NeuronParams np, float dt) {
  GRID_ITEM(rows * B);
  lif_item(st, S, _r, _b, J, s, V, R, np, dt);
}

__global__ void k_lif_rate(float* st, Strides S, int32_t B, int64_t rows, Opnd J, Opnd s, NeuronParams np) {
  GRID_ITEM(rows * B);
  lif_rate_item(st, S, _r, _b, J, s, np);
}

__global__ void k_lowpass(float* st, Strides S, int32_t B, int64_t rows, Opnd y, Opnd v, FilterParams fp) {
  GRID_ITEM(rows * B);
  lowpass_item(st, S, _r, _b, y, v, fp);
}

// Fused ensembles, small minibatch: one workgroup of 256 threads per (op,
// batch column); threads over neurons.  Decoded partial sums are reduced
// within each wavefront, then across the four wavefronts in LDS.
template <int NDEC, bool EVD>
__device__ __forceinline__ void ens_wg_t(float* st, const Strides& S, const EnsDesc& E, float dt,
                                         float (*red)[kMaxDec]) {
  const int op = blockIdx.x;
  const int64_t b = blockIdx.y;
  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  const EnsOp o = load_op(E.ops, op);
  const int d = o.x >= 0 ? E.d : 0, ndec = E.ndec, df0 = E.df[0];   // ops without input: J = bias
  gptr<float> enc = G(E.enc) + (int64_t)o.enc * d;
  gptr<float> bias = G(E.bias) + o.bias;
  gptr<float> D0 = G(E.D[0]) + (int64_t)o.D[0] * E.Dcols[0];
  gptr<float> D1 = G(E.D[E.nf > 1 ? 1 : 0]) + (int64_t)o.D[E.nf > 1 ? 1 : 0] * E.Dcols[E.nf > 1 ? 1 : 0];
  const int64_t s0 = E.Dcols[0], s1 = E.Dcols[E.nf > 1 ? 1 : 0];
  float acc[NDEC > 0 ? NDEC : 1];
#pragma unroll
  for (int q = 0; q < NDEC; ++q) acc[q] = 0.0f;
  float xr[kMaxXReg];
  load_input(xr, st, S, o.x, b, d);
  // with the transposed copy, encoder k of adjacent neurons is adjacent in memory
  gptr<float> encT = G(E.encT) + (int64_t)o.enc * d;
  const bool tr = E.encT != nullptr && d > 0 && d <= kMaxXReg;
  // event-driven decoding (EVD, E.decT set) reads a neuron's decoders only
  // when it spikes
  constexpr bool evd = EVD;
  gptr<float> dT = G(E.decT) + (int64_t)op * E.dT_op;
  for (int r = threadIdx.x; r < o.n; r += 256) {
    // every load of this neuron is issued before any arithmetic or store: the
    // encoders with the index clamped to d - 1 (the extra terms meet xr[k] = 0),
    // the bias, the state and (dense decoding) the decoder entries
    float ev[kMaxXReg], dv[NDEC > 0 ? NDEC : 1];
    if (tr) {
#pragma unroll
      for (int k = 0; k < kMaxXReg; ++k) ev[k] = encT[(int64_t)(k < d ? k : d - 1) * o.n + r];
    }
    const float bj = bias[r];
    float v = 0.0f, rf = 0.0f;
    if (E.ntype == 0) { v = st[at(S, o.V + r, b)]; rf = st[at(S, o.ref + r, b)]; }
    if constexpr (!evd) {
#pragma unroll
      for (int q = 0; q < NDEC; ++q) {
        const int qq = q < ndec ? q : ndec - 1;
        gptr<float> row = qq < df0 ? D0 + (int64_t)qq * s0 : D1 + (int64_t)(qq - df0) * s1;
        dv[q] = row[r];
      }
    }
    float j;
    if (tr) {
      j = bj;
#pragma unroll
      for (int k = 0; k < kMaxXReg; ++k) j += ev[k] * xr[k];
    } else {
      j = input_current(bj, enc + (int64_t)r * d, xr, st, S, o.x, b, d);
    }
    const float sp = neuron_update(E.ntype, j, v, rf, o.tau_rc, o.tau_ref, o.amp, o.full, dt, o.inv_tau);
    if (E.ntype == 0) { st[at(S, o.V + r, b)] = v; st[at(S, o.ref + r, b)] = rf; }
    if (o.s >= 0) st[at(S, o.s + r, b)] = sp;
    if constexpr (evd) {   // a silent neuron adds exact zeros, as in the dense sum
      if (sp != 0.0f) {
        if constexpr (NDEC >= 4) {
          typedef float f4v __attribute__((ext_vector_type(4)));
#pragma unroll
          for (int q4 = 0; q4 < NDEC / 4; ++q4) {
            const f4v t = *(const __attribute__((address_space(1))) f4v*)(dT + (int64_t)r * NDEC + 4 * q4);
#pragma unroll
            for (int e = 0; e < 4; ++e) dv[4 * q4 + e] = t[e];
          }
        } else {
#pragma unroll
          for (int q = 0; q < NDEC; ++q) dv[q] = dT[(int64_t)r * NDEC + q];
        }
      } else {
#pragma unroll
        for (int q = 0; q < NDEC; ++q) dv[q] = 0.0f;
      }
    }
#pragma unroll
    for (int q = 0; q < NDEC; ++q) acc[q] += dv[q] * sp;
  }
#pragma unroll
  for (int q = 0; q < NDEC; ++q) {
    const float t = wave_sum(acc[q]);
    if (lane == 0) red[wave][q] = t;
  }
  __syncthreads();
  const int q = threadIdx.x;
  if (q < ndec) {
    const float t = red[0][q] + red[1][q] + red[2][q] + red[3][q];
    const int dr = q < df0 ? o.d[0] + q : o.d[1] + (q - df0);
    st[at(S, dr, b)] = t;
  }
}

template <bool EVD>
__global__ void __launch_bounds__(256) k_ens_wg(float* st, Strides S, EnsDesc E, float dt) {
  __shared__ float red[4][kMaxDec];
  switch (dec_bucket(E.ndec)) {
    case 0: ens_wg_t<0, EVD>(st, S, E, dt, red); break;
    case 1: ens_wg_t<1, EVD>(st, S, E, dt, red); break;
    case 2: ens_wg_t<2, EVD>(st, S, E, dt, red); break;
    case 4: ens_wg_t<4, EVD>(st, S, E, dt, red); break;
    case 8: ens_wg_t<8, EVD>(st, S, E, dt, red); break;
    default: ens_wg_t<16, EVD>(st, S, E, dt, red); break;
  }
}

// Fused ensembles without fused decoders, with many neurons and a small
// minibatch (B <= 16), in the launch drivers' layout (element (r, b) at
// r * B + b).  Such neurons are independent, so a workgroup takes 64
// neurons of one op for every batch column: its 4 wavefronts split the input
// dimensions in four, lanes are neurons, the batch columns are held in
// registers.  The input x[q][b] is staged in LDS once per workgroup, and each
// transposed encoder value (coalesced across lanes) feeds B products.  The
// four partial currents meet in LDS; then the workgroup runs the neuron
// update for its 64 x B (neuron, column) pairs, consecutive threads taking
// consecutive columns.  The workgroup has nw wavefronts (blockDim.x = 64 nw),
// which split the input dimensions nw ways.  Dynamic LDS: (d + 64 nw) * B
// floats.
constexpr int kBigCols = 16, kBigNeurons = 64;

__global__ void __launch_bounds__(1024) k_ens_big(float* __restrict__ st, int32_t B, EnsDesc E, float dt) {
  extern __shared__ float big_lds[];
  const EnsOp o = load_op(E.ops, blockIdx.y);
  const int32_t i0 = (int32_t)blockIdx.x * kBigNeurons;
  if (i0 >= o.n) return;   // the whole workgroup
  const int32_t d = o.x >= 0 ? E.d : 0;
  float* xs = big_lds;
  float* part = big_lds + (size_t)d * B;   // [wave][neuron][column]
  const int32_t nt = blockDim.x, nw = nt / 64;
  for (int32_t t = threadIdx.x; t < d * B; t += nt) xs[t] = st[(int64_t)o.x * B + t];
  __syncthreads();
  const int32_t lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  float acc[kBigCols];
#pragma unroll
  for (int b = 0; b < kBigCols; ++b) acc[b] = 0.0f;
  if (i0 + lane < o.n && d > 0) {
    const int32_t dq = (d + nw - 1) / nw, q0 = wave * dq, q1 = min(d, q0 + dq);
    gptr<float> encT = G(E.encT) + (int64_t)o.enc * d + i0 + lane;   // (q, r) at q * n + r
    int32_t q = q0;
    for (; q + 4 <= q1; q += 4) {   // four loads in flight, then their products
      float e[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) e[k] = encT[(int64_t)(q + k) * o.n];
#pragma unroll
      for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int b = 0; b < kBigCols; ++b)
          if (b < B) acc[b] = fmaf(e[k], xs[(q + k) * B + b], acc[b]);
    }
    for (; q < q1; ++q) {
      const float e = encT[(int64_t)q * o.n];
#pragma unroll
      for (int b = 0; b < kBigCols; ++b)
        if (b < B) acc[b] = fmaf(e, xs[q * B + b], acc[b]);
    }
  }
#pragma unroll
  for (int b = 0; b < kBigCols; ++b)
    if (b < B) part[(wave * kBigNeurons + lane) * B + b] = acc[b];
  __syncthreads();
  const int32_t nb = min(kBigNeurons, o.n - i0) * B;
  for (int32_t p = threadIdx.x; p < nb; p += nt) {
    const int32_t r = p / B, b = p - r * B, i = i0 + r;
    float sum = 0.0f;
    for (int32_t w = 0; w < nw; ++w) sum += part[(w * kBigNeurons + r) * B + b];
    const float j = G(E.bias)[o.bias + i] + sum;
    float v = 0.0f, rf = 0.0f;
    if (E.ntype == 0) {
      v = st[(int64_t)(o.V + i) * B + b];
      rf = st[(int64_t)(o.ref + i) * B + b];
    }
    const float sp = neuron_update(E.ntype, j, v, rf, o.tau_rc, o.tau_ref, o.amp, o.full, dt, o.inv_tau);
    if (E.ntype == 0) {
      st[(int64_t)(o.V + i) * B + b] = v;
      st[(int64_t)(o.ref + i) * B + b] = rf;
    }
    if (o.s >= 0) st[(int64_t)(o.s + i) * B + b] = sp;
  }
}

// Fused ensembles, large minibatch: one workgroup (4 wavefronts) per (op, tile
// of 64 batch columns); lanes are batch columns, wavefronts split the neurons;
// encoder and decoder weights are wavefront-uniform loads; decoded partial
// sums are combined across wavefronts in LDS.
template <int NDEC>
__device__ __forceinline__ void ens_tile_t(float* st, const Strides& S, int32_t B, const EnsDesc& E, float dt,
                                           float (*red)[kMaxDec][64]) {
  const int op = blockIdx.x;
  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  const int64_t b = (int64_t)blockIdx.y * 64 + lane;
  const bool live = b < B;
  const EnsOp o = load_op(E.ops, op);
  const int d = o.x >= 0 ? E.d : 0, ndec = E.ndec, df0 = E.df[0];   // ops without input: J = bias
  gptr<float> enc = G(E.enc) + (int64_t)o.enc * d;
  gptr<float> bias = G(E.bias) + o.bias;
  gptr<float> D0 = G(E.D[0]) + (int64_t)o.D[0] * E.Dcols[0];
  gptr<float> D1 = G(E.D[E.nf > 1 ? 1 : 0]) + (int64_t)o.D[E.nf > 1 ? 1 : 0] * E.Dcols[E.nf > 1 ? 1 : 0];
  const int64_t s0 = E.Dcols[0], s1 = E.Dcols[E.nf > 1 ? 1 : 0];
  const int64_t bb = live ? b : 0;
  float acc[NDEC > 0 ? NDEC : 1];
#pragma unroll
  for (int q = 0; q < NDEC; ++q) acc[q] = 0.0f;
  for (int r = wave; r < o.n; r += 4) {
    float j = bias[r];
    for (int k = 0; k < d; ++k) j += enc[(int64_t)r * d + k] * st[at(S, o.x + k, bb)];
    float v = 0.0f, rf = 0.0f;
    if (E.ntype == 0) { v = st[at(S, o.V + r, bb)]; rf = st[at(S, o.ref + r, bb)]; }
    const float sp = neuron_update(E.ntype, j, v, rf, o.tau_rc, o.tau_ref, o.amp, o.full, dt, o.inv_tau);
    if (live) {
      if (E.ntype == 0) { st[at(S, o.V + r, b)] = v; st[at(S, o.ref + r, b)] = rf; }
      if (o.s >= 0) st[at(S, o.s + r, b)] = sp;
    }
#pragma unroll
    for (int q = 0; q < NDEC; ++q) {
      const int qq = q < ndec ? q : ndec - 1;
      gptr<float> row = qq < df0 ? D0 + (int64_t)qq * s0 : D1 + (int64_t)(qq - df0) * s1;
      acc[q] += row[r] * sp;
    }
  }
#pragma unroll
  for (int q = 0; q < NDEC; ++q) red[wave][q][lane] = acc[q];
  __syncthreads();
  if (wave == 0 && live) {
    for (int q = 0; q < ndec; ++q) {
      const float t = red[0][q][lane] + red[1][q][lane] + red[2][q][lane] + red[3][q][lane];
      const int dr = q < df0 ? o.d[0] + q : o.d[1] + (q - df0);
      st[at(S, dr, b)] = t;
    }
  }
}

__global__ void __launch_bounds__(256) k_ens_tile(float* st, Strides S, int32_t B, EnsDesc E, float dt) {
  __shared__ float red[4][kMaxDec][64];
  switch (dec_bucket(E.ndec)) {
    case 0: ens_tile_t<0>(st, S, B, E, dt, red); break;
    case 1: ens_tile_t<1>(st, S, B, E, dt, red); break;
    case 2: ens_tile_t<2>(st, S, B, E, dt, red); break;
    case 4: ens_tile_t<4>(st, S, B, E, dt, red); break;
    case 8: ens_tile_t<8>(st, S, B, E, dt, red); break;
    default: ens_tile_t<16>(st, S, B, E, dt, red); break;
  }
}

// ------------------------------------------- fused synapse filter + scatter
// The connection tail of Fig. 2 for a merged set of connections, at the end
// of a timestep: for every post input row, each incoming connection's value
// (a state row, or weight row . input rows computed here), its lowpass update
// y <- a y + b v, and the sum of the updated y in the order of the CopyInc it
// replaces, stored as the post input of the next step.  Segment: {post row or
// -1, rows, first connection, connections}; a connection record is 8 words
// {y, v, x, K | slot << 16 | staged << 20, w, probe row, a, b}: segment row i
// reads or updates row y + i and takes its value from row v + i (v >= 0), or
// computes it from weight row w + i of slot `slot` and the K inputs from row
// x on (v == -1; rows of the state, or with `staged` rows of this step's feed
// staging buffer), or only records row y + i (v == -2, a probe copy); with a
// probe row p >= 0 the updated (or copied) value of row i also goes to probe
// row p + i of this step.  update == 0 only sums (the pull at the start of a
// run).
//
// One wavefront per (segment, batch column): lane 16 j + i takes row i and,
// in chunk q, connections 8 q + j and 8 q + j + 4, whose loads are all issued
// before their arithmetic; the next chunk's records are fetched meanwhile.
// Row i's sum adds the chunk's values in connection order, read from lanes
// i, i + 16, i + 32, i + 48 (first and second connection of each lane).
// kw: K | weight slot << 16 | staged inputs << 20 | elementwise << 21 (then w
// holds the float bits of the scale)
struct SynConn {
  int32_t y, v, x, kw, w, p;
  float a, b;
};
struct SynW {
  const float* w[4];
};
constexpr int kSynRows = 16, kSynLanes = 4, kSynPerLane = 2, kSynChunk = kSynLanes * kSynPerLane;

// sum_k w[k] x[k] in k order (the DotInc kernel's order); x[k] at xp[k * xs]
// (UNIT: xs = 1, the inputs at fixed offsets from one address)
template <int KK, bool UNIT>
__device__ __forceinline__ float syn_dot_fixed(gptr<float> wr, const float* xp, int64_t xs, float d = 0.0f) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  const __attribute__((address_space(1))) f4v* w4 = (const __attribute__((address_space(1))) f4v*)wr;
  f4v wv[KK / 4];
  float xv[KK];
#pragma unroll
  for (int k4 = 0; k4 < KK / 4; ++k4) wv[k4] = w4[k4];
#pragma unroll
  for (int k = 0; k < KK; ++k) xv[k] = xp[UNIT ? k : k * xs];
#pragma unroll
  for (int k4 = 0; k4 < KK / 4; ++k4) {
    d += wv[k4][0] * xv[4 * k4];
    d += wv[k4][1] * xv[4 * k4 + 1];
    d += wv[k4][2] * xv[4 * k4 + 2];
    d += wv[k4][3] * xv[4 * k4 + 3];
  }
  return d;
}

template <bool UNIT>
__device__ __forceinline__ float syn_dot(gptr<float> wr, const float* xp, int64_t xs, int32_t K) {
  if (K == 16) return syn_dot_fixed<16, UNIT>(wr, xp, xs);
  if (K == 32) {   // two blocks of 16 (fewer registers), the sum still in k order
    const float d0 = syn_dot_fixed<16, UNIT>(wr, xp, xs);
    return syn_dot_fixed<16, UNIT>(wr + 16, xp + (UNIT ? 16 : 16 * xs), xs, d0);
  }
  float d = 0.0f;
  if ((K & 3) == 0) {
    typedef float f4v __attribute__((ext_vector_type(4)));
    const __attribute__((address_space(1))) f4v* w4 = (const __attribute__((address_space(1))) f4v*)wr;
    for (int32_t k4 = 0; k4 < K / 4; ++k4) {
      const f4v wq = w4[k4];
      const int64_t k = 4 * (int64_t)k4;
      d += wq[0] * xp[k * xs];
      d += wq[1] * xp[(k + 1) * xs];
      d += wq[2] * xp[(k + 2) * xs];
      d += wq[3] * xp[(k + 3) * xs];
    }
  } else {
    for (int32_t k = 0; k < K; ++k) d += wr[k] * xp[(int64_t)k * xs];
  }
  return d;
}

struct SynRec {
  int32_t y, v, x, kw, w, p, a, b;
};

__device__ __forceinline__ SynRec syn_rec(const SynConn* conn, int32_t c, bool live) {
  SynRec r{-3, -3, 0, 0, 0, -1, 0, 0};
  if (live) {
    typedef int i4v __attribute__((ext_vector_type(4)));
    const __attribute__((address_space(1))) i4v* q = (const __attribute__((address_space(1))) i4v*)(conn + c);
    const i4v u = q[0], w = q[1];
    r = SynRec{u[0], u[1], u[2], u[3], w[0], w[1], w[2], w[3]};
  }
  return r;
}

// UNIT: one batch column (B = 1, row stride 1), so a connection's inputs are
// consecutive floats.
template <bool UNIT>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(UNIT ? 5 : 1))) k_syn_scatter(float* st, Strides S, int32_t B, int32_t nseg,
                                                     const int32_t* seg, const SynConn* conn, SynW W,
                                                     int32_t update, float* probe, int32_t probe_rows,
                                                     const float* stage, int32_t feed_rows, const int64_t* ctr,
                                                     int32_t du) {
  const uint32_t wv = (blockIdx.x * blockDim.x + threadIdx.x) / 64;
  // slots per lane: one when the inputs are consecutive (fewer registers, more
  // wavefronts resident), kSynPerLane otherwise
  constexpr int PL = UNIT ? 1 : kSynPerLane, CH = kSynLanes * PL;
  const int lane = threadIdx.x % 64, i = lane % kSynRows, j = lane / kSynRows;
  const uint32_t sg = wv / (uint32_t)B, b = wv - sg * (uint32_t)B;
  if (sg >= (uint32_t)nseg) return;   // the whole wavefront leaves together
  typedef int i4v __attribute__((ext_vector_type(4)));
  const i4v sd = *(const __attribute__((address_space(1))) i4v*)(G(seg) + 4 * (int64_t)sg);
  const bool row = i < sd[1];
  const int32_t c0 = sd[2], nc = sd[3];
  // run-relative step (feed staging) and absolute step (probe record)
  const int64_t tr = update ? ctr[1] + du : 0, ta = update ? ctr[0] + du : 0;
  SynRec nxt[PL];
#pragma unroll
  for (int h = 0; h < PL; ++h) nxt[h] = syn_rec(conn, c0 + j + kSynLanes * h, row && j + kSynLanes * h < nc);
  float acc = 0.0f;
  for (int32_t q0 = 0; q0 < nc; q0 += CH) {
    SynRec cur[PL];
#pragma unroll
    for (int h = 0; h < PL; ++h) cur[h] = nxt[h];
#pragma unroll
    for (int h = 0; h < PL; ++h) {
      const int32_t q = q0 + CH + j + kSynLanes * h;
      nxt[h] = syn_rec(conn, c0 + q, row && q < nc);
    }
    // values (loads of both connections first, then the products)
    float y[PL], v[PL];
#pragma unroll
    for (int h = 0; h < PL; ++h) {
      const SynRec& r = cur[h];
      y[h] = 0.0f;
      v[h] = 0.0f;
      if (r.y == -3) continue;   // no connection in this slot
      y[h] = st[at(S, (int64_t)r.y + i, b)];
      if (!update || r.v == -2) continue;
      if (r.v >= 0) {
        v[h] = st[at(S, (int64_t)r.v + i, b)];
      } else if (r.kw & (1 << 21)) {   // elementwise transform: scale (bits in w) times input row x + i
        const float xi = (r.kw >> 20) & 1 ? stage[(tr * feed_rows + r.x + i) * B + b] : st[at(S, (int64_t)r.x + i, b)];
        v[h] = 0.0f + __builtin_bit_cast(float, r.w) * xi;   // the increment adds into a reset row
      } else {
        const int32_t K = r.kw & 0xffff, ws = (r.kw >> 16) & 15, staged = (r.kw >> 20) & 1;
        gptr<float> wr = G(W.w[ws]) + ((int64_t)r.w + i) * K;
        const float* xp = staged ? stage + (tr * feed_rows + r.x) * B + b : st + at(S, r.x, b);
        const int64_t xs = staged ? (int64_t)B : S.rs;
        v[h] = 0.0f + syn_dot<UNIT>(wr, xp, xs, K);   // the DotInc adds into a reset row
      }
    }
#pragma unroll
    for (int h = 0; h < PL; ++h) {
      const SynRec& r = cur[h];
      if (r.y == -3 || !update) continue;
      if (r.v != -2) {
        y[h] = lowpass_step(__builtin_bit_cast(float, r.a), y[h], __builtin_bit_cast(float, r.b), v[h]);
        st[at(S, (int64_t)r.y + i, b)] = y[h];
      }
      if (probe && r.p >= 0) probe[(ta * probe_rows + r.p + i) * B + b] = y[h];
    }
    // every lane takes part in the exchange; only lanes j == 0 keep a sum
#pragma unroll
    for (int jj = 0; jj < CH; ++jj) {
      const float u = __shfl(y[jj / kSynLanes], i + kSynRows * (jj % kSynLanes), 64);
      if (q0 + jj < nc) acc += u;
    }
  }
  if (j == 0 && row && sd[0] >= 0) st[at(S, (int64_t)sd[0] + i, b)] = acc;
}

// ------------------------------------------------------------- PES learning
// Online learning of a decoded connection's output weights (paper Sec. 5.1,
// the pes benchmark), one decoder matrix per batch column (Fig. 7).  Op o's
// decoders for neuron i, output j, batch column b sit at state row
// w[o] + i*M + j, column b; in the launch drivers' layout (element (r, b) at
// r * B + b) neuron i's decoders are the M*B consecutive floats at
// (w[o] + i*M) * B, indexed by c = j*B + b.  One pass over them computes the
// decode d[j, b] += sum_i x[i, b] W[i, j, b] (MODE 0), the PES update
// W[i, j, b] += coef * act[i, b] * e[j, b] (MODE 1, act = the x rows), or
// both (MODE 2: decode with the old value, store the new), so that the
// decoders are read once and written once per step.
struct PesOps {
  const int32_t* w;     // first decoder row
  const int32_t* x;     // activities the decode reads (MODE 1: the update's)
  const int32_t* d;     // decoded outputs (MODE 0, 2)
  const int32_t* e;     // error rows (MODE 1, 2)
  const int32_t* act;   // activities the update reads (MODE 2)
  const float* coef;    // -kappa dt / n (MODE 1, 2)
};

// grid (ceil(M*B / 256), chunks, ops); each workgroup takes neurons
// [chunk * L, min(K, chunk * L + L)) of 256 columns c; the chunk's activity
// rows (L*B floats each) are staged in LDS (dynamic, 2*L*B floats).  Partial
// decodes go to part[(o * nch + chunk) * M*B + c], summed by k_pes_reduce.
template <int MODE>
__global__ void __launch_bounds__(256) k_pes(float* __restrict__ st, int32_t B, int32_t M, int32_t K,
                                             int32_t L, PesOps P, float* __restrict__ part, int32_t nch) {
  extern __shared__ float pes_lds[];
  float* s_x = pes_lds;
  float* s_a = pes_lds + (size_t)L * B;
  const int32_t o = blockIdx.z, ch = blockIdx.y;
  const int32_t MB = M * B;
  const int32_t c = (int32_t)blockIdx.x * 256 + (int32_t)threadIdx.x;
  const int32_t i0 = ch * L, n = min(K, i0 + L) - i0;
  const int64_t xb = ((int64_t)P.x[o] + i0) * B;
  const int64_t ab = MODE == 2 ? ((int64_t)P.act[o] + i0) * B : xb;
  for (int32_t t = threadIdx.x; t < n * B; t += 256) {
    if (MODE != 1) s_x[t] = st[xb + t];
    if (MODE != 0) s_a[t] = st[ab + t];
  }
  __syncthreads();
  if (c >= MB) return;
  const int32_t b = c % B;
  float e = 0.f, coef = 0.f;
  if (MODE != 0) {
    e = st[(int64_t)P.e[o] * B + c];
    coef = P.coef[o];
  }
  float* w = st + ((int64_t)P.w[o] + (int64_t)i0 * M) * B + c;
  const int64_t stp = MB;
  float acc0 = 0.f, acc1 = 0.f;
  int32_t i = 0;
  for (; i + 4 <= n; i += 4) {
    const float w0 = w[0], w1 = w[stp], w2 = w[2 * stp], w3 = w[3 * stp];
    if (MODE != 1) {
      acc0 = fmaf(s_x[i * B + b], w0, acc0);
      acc1 = fmaf(s_x[(i + 1) * B + b], w1, acc1);
      acc0 = fmaf(s_x[(i + 2) * B + b], w2, acc0);
      acc1 = fmaf(s_x[(i + 3) * B + b], w3, acc1);
    }
    if (MODE != 0) {
      w[0] = fmaf(coef * s_a[i * B + b], e, w0);
      w[stp] = fmaf(coef * s_a[(i + 1) * B + b], e, w1);
      w[2 * stp] = fmaf(coef * s_a[(i + 2) * B + b], e, w2);
      w[3 * stp] = fmaf(coef * s_a[(i + 3) * B + b], e, w3);
    }
    w += 4 * stp;
  }
  for (; i < n; ++i) {
    const float w0 = w[0];
    if (MODE != 1) acc0 = fmaf(s_x[i * B + b], w0, acc0);
    if (MODE != 0) w[0] = fmaf(coef * s_a[i * B + b], e, w0);
    w += stp;
  }
  if (MODE != 1) part[((int64_t)o * nch + ch) * MB + c] = acc0 + acc1;
}

// d[o] rows += the sum over chunks of the partial decodes, in a fixed order:
// a workgroup takes 32 columns of one op; its 8 slices of 32 threads each sum
// every 8th chunk (4 accumulators), and the 8 slice sums are added in slice
// order.  grid (ceil(M*B / 32), ops).
__global__ void __launch_bounds__(256) k_pes_reduce(float* __restrict__ st, int32_t B, int32_t M, const int32_t* d,
                                                    const float* __restrict__ part, int32_t nch) {
  __shared__ float red[8][32];
  const int64_t MB = (int64_t)M * B;
  const int32_t o = blockIdx.y, col = threadIdx.x % 32, slice = threadIdx.x / 32;
  const int64_t c = (int64_t)blockIdx.x * 32 + col;
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  if (c < MB) {
    const float* p = part + (int64_t)o * nch * MB + c;
    int32_t ch = slice;
    for (; ch + 24 < nch; ch += 32) {
      a0 += p[(int64_t)ch * MB];
      a1 += p[(int64_t)(ch + 8) * MB];
      a2 += p[(int64_t)(ch + 16) * MB];
      a3 += p[(int64_t)(ch + 24) * MB];
    }
    for (; ch < nch; ch += 8) a0 += p[(int64_t)ch * MB];
  }
  red[slice][col] = (a0 + a1) + (a2 + a3);
  __syncthreads();
  if (slice == 0 && c < MB) {
    float t = red[0][col];
#pragma unroll
    for (int k = 1; k < 8; ++k) t += red[k][col];
    st[(int64_t)d[o] * B + c] += t;
  }
}

// node output <- feed staging [step][feed_rows][B] at the run-relative step
// ctr[1] + du (du: the step's place among the steps launched since the counter
// last advanced)
__global__ void k_feed(float* st, Strides S, int32_t B, int64_t rows, Opnd dst, const int32_t* feed_row,
                       const float* stage, int32_t feed_rows, const int64_t* ctr, int32_t du) {
  GRID_ITEM(rows * B);
  const int64_t t = ctr[1] + du;
  st[at(S, rowof(dst, _r), _b)] = stage[(t * feed_rows + feed_row[_r]) * B + _b];
}

// probe buffer [step][probe_rows][B] at the absolute step ctr[0] + du
__global__ void k_probe(const float* st, Strides S, int32_t B, int32_t rows, const int32_t* src, float* buf,
                        const int64_t* ctr, int32_t du) {
  GRID_ITEM((int64_t)rows * B);
  buf[((ctr[0] + du) * rows + _r) * B + _b] = st[at(S, src[_r], _b)];
}

__global__ void k_advance(int64_t* ctr, int32_t n) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctr[0] += n;
    ctr[1] += n;
  }
}

// Rows [row0, row0 + rows) of the state get vals[r] in every batch column
// (initial values of learned decoders, on creation and reset).
__global__ void k_init_rows(float* st, Strides S, int32_t B, int64_t row0, int64_t rows, const float* vals) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows * B) return;
  const int64_t r = t / B, b = t - r * B;
  st[at(S, row0 + r, b)] = vals[r];
}

__global__ void k_set_ctr(int64_t* ctr, int64_t c0, int64_t c1) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctr[0] = c0;
    ctr[1] = c1;
  }
}

// count of non-finite values among x[0..n) (grid-stride; one atomic per workgroup)
__global__ void __launch_bounds__(256) k_count_nonfinite(const float* x, int64_t n, unsigned int* count) {
  __shared__ unsigned int c;
  if (threadIdx.x == 0) c = 0;
  __syncthreads();
  unsigned int mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    mine += isfinite(x[i]) ? 0u : 1u;
  if (mine) atomicAdd(&c, mine);
  __syncthreads();
  if (threadIdx.x == 0 && c) atomicAdd(count, c);
}

// feed [B][T][size] -> staging [T][feed_rows][B] rows [row0, row0+size)
#define GRID_FLAT(n)                                                        \
  const int64_t _i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;        \
  if (_i >= (n)) return;

// feed [B][T][size] -> staging [T][feed_rows][B] at rows row0..row0+size: per
// step a [B x size] -> [size x B] transpose through a 32 x 33 LDS tile, so that
// both the reads (along size) and the writes (along B) are coalesced.
// Grid (ceil(size/32), ceil(B/32), steps of this chunk), block 32 x 8; steps
// t_off + blockIdx.z.
__global__ void __launch_bounds__(256) k_stage_feed(const float* src, int32_t B, int64_t T, int32_t size,
                                                    float* stage, int32_t feed_rows, int32_t row0, int64_t t_off) {
  __shared__ float tile[32][33];
  const int64_t t = t_off + blockIdx.z;
  const int j0 = blockIdx.x * 32, b0 = blockIdx.y * 32;
  const int tx = threadIdx.x, ty = threadIdx.y;
  for (int r = ty; r < 32; r += 8) {
    const int b = b0 + r, j = j0 + tx;
    if (b < B && j < size) tile[r][tx] = src[((int64_t)b * T + t) * size + j];
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int j = j0 + r, b = b0 + tx;
    if (j < size && b < B) stage[(t * feed_rows + row0 + j) * B + b] = tile[tx][r];
  }
}

// probe buffer [T][probe_rows][B] -> out [B][T][w] for rows [off, off+w)
__global__ void k_probe_extract(const float* buf, int32_t B, int64_t T, int32_t probe_rows, int32_t off,
                                int32_t w, float* out) {
  GRID_FLAT((int64_t)B * T * w);
  const int64_t j = _i % w;
  const int64_t t = (_i / w) % T;
  const int64_t b = _i / ((int64_t)w * T);
  out[_i] = buf[(t * probe_rows + off + j) * B + b];
}

// A bit-recorded spike probe read out as values: out[b][t][i] (the layout of
// every probe read) is `mag` (amplitude / dt) where bit i of step t, column b
// is set, else 0.  The probe's words start at word row `off` of `words` per step.
__global__ void k_bits_extract(const uint32_t* bits, int32_t B, int64_t T, int32_t words, int32_t off, int32_t width,
                               float mag, float* out) {
  const int64_t n = (int64_t)B * T * width;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t j = (int32_t)(i % width);
  const int64_t t = (i / width) % T, b = i / ((int64_t)width * T);
  const uint32_t m = G(bits)[(t * words + off + j / 32) * B + b];
  out[i] = ((m >> (j % 32)) & 1u) ? mag : 0.0f;
}

// The same probe's words, [b][t][k] for k < nw (bit j of word k: neuron 32 k + j).
__global__ void k_bits_words(const uint32_t* bits, int32_t B, int64_t T, int32_t words, int32_t off, int32_t nw,
                             uint32_t* out) {
  const int64_t n = (int64_t)B * T * nw;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t k = (int32_t)(i % nw);
  const int64_t t = (i / nw) % T, b = i / ((int64_t)nw * T);
  out[i] = G(bits)[(t * words + off + k) * B + b];
}

// ----------------------------------------------------- persistent interpreter
// A merged group as the persistent kernel sees it (device-resident array).
struct GroupDesc {
  int32_t type;
  int32_t M, K, tpr;
  const float* wt_base;    // DOT_INC: transposed weights
  const int64_t* wt_off;   // DOT_INC: per-op offset of the [K][M] block
  int32_t bcast;
  int64_t rows;
  Opnd dst, src, a, V, ref;
  const float* src_base;
  const float* a_base;
  const int32_t* ptr;
  const float* values;
  const int32_t* w_row;
  const int32_t* x_row;
  const int32_t* d_row;
  const int32_t* feed_row;
  NeuronParams np;
  FilterParams fp;
  EnsDesc ens;
};

struct PersistentProgram {
  GroupDesc* groups;     // device array
  int32_t n_groups;
};

// Every group of every step for one batch column per workgroup; groups are
// separated by workgroup barriers (operators inside a group are independent by
// construction, and groups run in plan order).  Probes record after each step.
// LDS = true: the column's whole state is copied into LDS at the start, every
// group works on LDS for all steps, and it is written back at the end.
template <bool LDS>
__global__ void __launch_bounds__(1024)
k_persistent(float* state, int64_t rows, int32_t B, const GroupDesc* groups, int32_t ng, int64_t n_steps,
             float dt, const float* stage, int32_t feed_rows, const int32_t* probe_src, int32_t probe_rows,
             float* probe_buf, int64_t t0, float* scratch_g, int64_t scratch_n) {
  extern __shared__ float lds[];
  const int64_t col = blockIdx.x;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int lane = tid % warpSize, wave = tid / warpSize, nwaves = nt / warpSize;
  // column-major state: column `col` occupies rows [col * rows, (col + 1) * rows)
  float* gcol = state + col * rows;
  float* st = LDS ? lds : gcol;
  float* scratch = LDS ? lds + rows : scratch_g + col * scratch_n;
  const Strides S{1, 0};
  const int64_t b = 0;
  if (LDS) {
    for (int64_t r = tid; r < rows; r += nt) lds[r] = gcol[r];
    __syncthreads();
  }
  for (int64_t k = 0; k < n_steps; ++k) {
    for (int32_t g = 0; g < ng; ++g) {
      // descriptor fields through kload: scalar loads of a table the kernel never writes
      const GroupDesc* gp = groups + g;
      const int64_t nrow = kload(&gp->rows);
      switch (kload(&gp->type)) {
        case ms::OP_FEED: {
          const Opnd dst = kload(&gp->dst);
          gptr<int32_t> fr = ::G(kload(&gp->feed_row));
          for (int64_t r = tid; r < nrow; r += nt) st[rowof(dst, r)] = stage[(k * feed_rows + fr[r]) * B + col];
          break;
        }
        case ms::OP_RESET: {
          const Opnd dst = kload(&gp->dst);
          const float* values = kload(&gp->values);
          for (int64_t r = tid; r < nrow; r += nt) st[rowof(dst, r)] = values ? ::G(values)[r] : 0.0f;
          break;
        }
        case ms::OP_COPY: {
          const Opnd dst = kload(&gp->dst), src = kload(&gp->src);
          const int32_t bcast = kload(&gp->bcast);
          gptr<float> sb = ::G(kload(&gp->src_base));
          for (int64_t r = tid; r < nrow; r += nt)
            st[rowof(dst, r)] = bcast ? sb[rowof(src, r)] : st[rowof(src, r)];
          break;
        }
        case ms::OP_COPY_INC: {
          const Opnd dst = kload(&gp->dst), src = kload(&gp->src);
          const int32_t bcast = kload(&gp->bcast);
          gptr<float> sb = ::G(kload(&gp->src_base));
          const int32_t* ptr = kload(&gp->ptr);
          for (int64_t r = tid; r < nrow; r += nt) {
            const int64_t di = rowof(dst, r);
            float acc = st[di];
            if (ptr) {
              for (int32_t e = ::G(ptr)[r]; e < ::G(ptr)[r + 1]; ++e)
                acc += bcast ? sb[rowof(src, e)] : st[rowof(src, e)];
            } else {
              acc += bcast ? sb[rowof(src, r)] : st[rowof(src, r)];
            }
            st[di] = acc;
          }
          break;
        }
        case ms::OP_ELEM_INC: {
          const Opnd dst = kload(&gp->dst), src = kload(&gp->src), a = kload(&gp->a);
          gptr<float> ab = ::G(kload(&gp->a_base));
          const int32_t* ptr = kload(&gp->ptr);
          for (int64_t r = tid; r < nrow; r += nt) {
            const int64_t di = rowof(dst, r);
            float acc = st[di];
            if (ptr) {
              for (int32_t e = ::G(ptr)[r]; e < ::G(ptr)[r + 1]; ++e) acc += ab[rowof(a, e)] * st[rowof(src, e)];
            } else {
              acc += ab[rowof(a, r)] * st[rowof(src, r)];
            }
            st[di] = acc;
          }
          break;
        }
        case ms::OP_DOT_INC: {
          // Weights are stored transposed per op ([K][M], wt_base) so that
          // lanes over output rows read consecutive weights.  The K range is
          // split into tpr parts; part-major work items keep lanes of a
          // wavefront on consecutive rows; parts > 1 add their partial sums
          // through the LDS scratch after the state.
          const uint32_t M = (uint32_t)kload(&gp->M), K = (uint32_t)kload(&gp->K), tpr = (uint32_t)kload(&gp->tpr);
          gptr<float> wt_base = ::G(kload(&gp->wt_base));
          gptr<int64_t> wt_off = ::G(kload(&gp->wt_off));
          gptr<int32_t> x_row = ::G(kload(&gp->x_row)), d_row = ::G(kload(&gp->d_row));
          const uint32_t total = (uint32_t)nrow * M;
          const uint32_t chunk = (K + tpr - 1) / tpr;
          for (uint32_t t = tid; t < total * tpr; t += (uint32_t)nt) {
            const uint32_t part = t / total, rowi = t - part * total;
            const uint32_t op = rowi / M, m = rowi - op * M;
            gptr<float> w = wt_base + wt_off[op];
            const int64_t x0 = x_row[op];
            const uint32_t k0 = part * chunk, k1 = min(K, k0 + chunk);
            float acc = 0.0f;
            for (uint32_t kk = k0; kk < k1; ++kk) acc += w[(int64_t)kk * M + m] * st[x0 + kk];
            if (tpr == 1) st[(int64_t)d_row[op] + m] += acc;
            else scratch[t] = acc;
          }
          if (tpr > 1) {
            __syncthreads();
            for (uint32_t rowi = tid; rowi < total; rowi += (uint32_t)nt) {
              const uint32_t op = rowi / M, m = rowi - op * M;
              float acc = 0.0f;
              for (uint32_t p2 = 0; p2 < tpr; ++p2) acc += scratch[p2 * total + rowi];
              st[(int64_t)d_row[op] + m] += acc;
            }
          }
          break;
        }
        case ms::OP_LIF: {
          const Opnd src = kload(&gp->src), dst = kload(&gp->dst), V = kload(&gp->V), ref = kload(&gp->ref);
          const NeuronParams np = kload(&gp->np);
          for (int64_t r = tid; r < nrow; r += nt) lif_item(st, S, r, b, src, dst, V, ref, np, dt);
          break;
        }
        case ms::OP_LIF_RATE: {
          const Opnd src = kload(&gp->src), dst = kload(&gp->dst);
          const NeuronParams np = kload(&gp->np);
          for (int64_t r = tid; r < nrow; r += nt) lif_rate_item(st, S, r, b, src, dst, np);
          break;
        }
        case ms::OP_LOWPASS: {
          const Opnd dst = kload(&gp->dst), src = kload(&gp->src);
          const FilterParams fp = kload(&gp->fp);
          for (int64_t r = tid; r < nrow; r += nt) lowpass_item(st, S, r, b, dst, src, fp);
          break;
        }
        case ms::OP_ENS: {
          const EnsDesc E = kload(&gp->ens);
          for (int op = wave; op < nrow; op += nwaves) ens_op_wave(st, S, b, E, op, lane, dt);
          break;
        }
        default: break;
      }
      __syncthreads();
    }
    for (int32_t r = tid; r < probe_rows; r += nt)
      probe_buf[((t0 + k) * probe_rows + r) * B + col] = st[::G(probe_src)[r]];
    __syncthreads();
  }
  if (LDS) {
    for (int64_t r = tid; r < rows; r += nt) gcol[r] = lds[r];
  }
}
