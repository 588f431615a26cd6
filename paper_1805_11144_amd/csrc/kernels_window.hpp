// Stage-major (window) kernels: one launch runs a merged group for every step
// of a window of T timesteps.
//
// Versioned signals live in `va`: element (row, block k, batch column b) at
// va[row * vs + k * B + b] with vs = (W + 1) * B; block 0 holds the value
// carried in from the previous window, block t + 1 the value of window step t.
// An operand read at block offset `blk` = 1 sees this step's value, 0 the
// previous step's (a filter output read before its update).  Neuron state
// (voltage, refractory time) lives in `pa` as [rows][B].
//
// Groups without a recurrence (feeds, resets, copies, increments, products,
// rate neurons) are time-parallel: one work item per (row, step, column), the
// (step, column) pair flattened as c = t * B + b so that block t + blk of a row
// is va[row * vs + blk * B + c].  Filters and spiking neurons carry their
// state through the window in registers, one work item per (row, column).
#pragma once

#include "kernels.hpp"

#include <type_traits>

struct WView {
  float* va;
  int64_t vs;      // row stride of va, (W + 1) * B
  int32_t B;
  int32_t T;       // steps of this window
};

__device__ __forceinline__ int64_t vat(const WView& w, int64_t row, int64_t c) { return row * w.vs + c; }

// Work item i of rows x (T * B): row and flattened (step, column) index.  The
// host checks that rows * T * B fits in 32 bits.
#define W_ITEM(rows)                                                           \
  const uint32_t _i = blockIdx.x * blockDim.x + threadIdx.x;                   \
  const uint32_t _tb = (uint32_t)w.T * (uint32_t)w.B;                          \
  if (_i >= (uint32_t)(rows) * _tb) return;                                    \
  const uint32_t _r = _i / _tb, _c = _i - _r * _tb;

__device__ __forceinline__ float w_src(const WView& w, const float* param, int bcast, int64_t row, int blk,
                                       uint32_t c) {
  return bcast ? G(param)[row] : w.va[vat(w, row, (int64_t)blk * w.B + c)];
}

// node rows <- staged feed [step][feed_rows][B] at run step t0 + t
__global__ void k_w_feed(WView w, int64_t rows, Opnd dst, const int32_t* feed_row, const float* stage,
                         int32_t feed_rows, int64_t t0) {
  W_ITEM(rows);
  const uint32_t t = _c / (uint32_t)w.B, b = _c - t * (uint32_t)w.B;
  w.va[vat(w, rowof(dst, _r), w.B + _c)] = stage[((t0 + t) * feed_rows + G(feed_row)[_r]) * w.B + b];
}

__global__ void k_w_reset(WView w, int64_t rows, Opnd dst, const float* values) {
  W_ITEM(rows);
  w.va[vat(w, rowof(dst, _r), w.B + _c)] = values ? G(values)[_r] : 0.0f;
}

__global__ void k_w_copy(WView w, int64_t rows, Opnd dst, const float* param, Opnd src, int bcast, int sblk) {
  W_ITEM(rows);
  w.va[vat(w, rowof(dst, _r), w.B + _c)] = w_src(w, param, bcast, rowof(src, _r), sblk, _c);
}

// dst += sum of the src entries of unique destination u (ptr == null: one entry)
__global__ void k_w_copy_inc(WView w, int64_t rows, Opnd dst, const float* param, Opnd src, int bcast, int sblk,
                             const int32_t* ptr) {
  W_ITEM(rows);
  const int64_t di = vat(w, rowof(dst, _r), w.B + _c);
  float acc = w.va[di];
  if (ptr) {
    for (int32_t e = G(ptr)[_r]; e < G(ptr)[_r + 1]; ++e) acc += w_src(w, param, bcast, rowof(src, e), sblk, _c);
  } else {
    acc += w_src(w, param, bcast, rowof(src, _r), sblk, _c);
  }
  w.va[di] = acc;
}

// dst += a (.) x, entries grouped by destination as in k_w_copy_inc
__global__ void k_w_elem_inc(WView w, int64_t rows, Opnd dst, const float* a_param, Opnd a, int a_bcast, int ablk,
                             const float* x_param, Opnd x, int x_bcast, int xblk, const int32_t* ptr) {
  W_ITEM(rows);
  const int64_t di = vat(w, rowof(dst, _r), w.B + _c);
  float acc = w.va[di];
  if (ptr) {
    for (int32_t e = G(ptr)[_r]; e < G(ptr)[_r + 1]; ++e)
      acc += w_src(w, a_param, a_bcast, rowof(a, e), ablk, _c) * w_src(w, x_param, x_bcast, rowof(x, e), xblk, _c);
  } else {
    acc += w_src(w, a_param, a_bcast, rowof(a, _r), ablk, _c) * w_src(w, x_param, x_bcast, rowof(x, _r), xblk, _c);
  }
  w.va[di] = acc;
}

// dst[m] += W[m, :] . x for every op, output row and (step, column)
__global__ void k_w_dot(WView w, int64_t nops, int32_t M, int32_t K, const float* Wt, const int32_t* w_row,
                        const int32_t* x_row, const int32_t* d_row, int xblk) {
  W_ITEM(nops * M);
  const uint32_t op = _r / (uint32_t)M, m = _r - op * (uint32_t)M;
  gptr<float> wr = G(Wt) + ((int64_t)G(w_row)[op] + m) * K;
  const int64_t x0 = G(x_row)[op];
  const int64_t xc = (int64_t)xblk * w.B + _c;
  float acc = 0.0f;
  for (int32_t k = 0; k < K; ++k) acc += wr[k] * w.va[vat(w, x0 + k, xc)];
  w.va[vat(w, (int64_t)G(d_row)[op] + m, w.B + _c)] += acc;
}

__global__ void k_w_lif_rate(WView w, int64_t rows, Opnd J, Opnd s, NeuronParams np, int jblk) {
  W_ITEM(rows);
  const float tau_rc = np.tau_rc_r ? G(np.tau_rc_r)[_r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? G(np.tau_ref_r)[_r] : np.tau_ref;
  const float amp = np.amp_r ? G(np.amp_r)[_r] : np.amp;
  const float j = w.va[vat(w, rowof(J, _r), (int64_t)jblk * w.B + _c)];
  float out = 0.0f;
  if (np.relu) {
    out = amp * fmaxf(j, 0.0f);
  } else if (np.sigma > 0.0f) {
    float dl, rho;
    out = amp * soft_lif_rate(j, tau_rc, tau_ref, np.sigma_r ? G(np.sigma_r)[_r] : np.sigma, &dl, &rho);
  } else if (j > 1.0f) {
    out = amp / (tau_ref + tau_rc * log1pf(1.0f / (j - 1.0f)));
  }
  w.va[vat(w, rowof(s, _r), w.B + _c)] = out;
}

// Work item per (row, column): state carried through the window.
#define W_ROWCOL(rows)                                                         \
  const uint32_t _i = blockIdx.x * blockDim.x + threadIdx.x;                   \
  if (_i >= (uint32_t)(rows) * (uint32_t)w.B) return;                          \
  const uint32_t _r = _i / (uint32_t)w.B, _b = _i - _r * (uint32_t)w.B;

__global__ void k_w_lif(WView w, int64_t rows, Opnd J, Opnd s, Opnd V, Opnd R, float* pa, NeuronParams np,
                        float dt, int jblk) {
  W_ROWCOL(rows);
  const float tau_rc = np.tau_rc_r ? G(np.tau_rc_r)[_r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? G(np.tau_ref_r)[_r] : np.tau_ref;
  const float amp = np.amp_r ? G(np.amp_r)[_r] : np.amp;
  const float full = np.full_r ? G(np.full_r)[_r] : np.full;
  const int64_t vi = rowof(V, _r) * w.B + _b, ri = rowof(R, _r) * w.B + _b;
  float v = pa[vi], rf = pa[ri];
  const int64_t jr = rowof(J, _r) * w.vs + (int64_t)jblk * w.B + _b;
  const int64_t sr = rowof(s, _r) * w.vs + w.B + _b;
  const float inv_tau = 1.0f / tau_rc;
  if (dt * inv_tau <= 0.0625f) {
    const float amp_dt = amp / dt, tau6 = tau_rc * (1.0f / 6.0f);
    for (int32_t t = 0; t < w.T; ++t) {
      const float j = w.va[jr + (int64_t)t * w.B];
      w.va[sr + (int64_t)t * w.B] = lif_update_bf(j, v, rf, tau6, tau_ref, amp_dt, dt, inv_tau);
    }
  } else {
    for (int32_t t = 0; t < w.T; ++t) {
      const float j = w.va[jr + (int64_t)t * w.B];
      w.va[sr + (int64_t)t * w.B] = neuron_update(0, j, v, rf, tau_rc, tau_ref, amp, full, dt, inv_tau);
    }
  }
  pa[vi] = v;
  pa[ri] = rf;
}

// y(t) = a y(t - 1) + b v(t) through the window; y(-1) is block 0
__global__ void k_w_lowpass(WView w, int64_t rows, Opnd y, Opnd v, FilterParams fp, int vblk) {
  W_ROWCOL(rows);
  const float a = fp.a_r ? G(fp.a_r)[_r] : fp.a;
  const float c = fp.b_r ? G(fp.b_r)[_r] : fp.b;
  const int64_t yr = rowof(y, _r) * w.vs + _b;
  const int64_t vr = rowof(v, _r) * w.vs + (int64_t)vblk * w.B + _b;
  float yv = w.va[yr];
  // inputs of 32 (then 8) steps are loaded before they are consumed, so the
  // loads of a chunk are in flight together; the recurrence itself is one FMA
  // per step, in step order, whatever the window length
  int32_t t = 0;
  for (; t + 32 <= w.T; t += 32) {
    float vin[32];
#pragma unroll
    for (int u = 0; u < 32; ++u) vin[u] = w.va[vr + (int64_t)(t + u) * w.B];
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      yv = lowpass_step(a, yv, c, vin[u]);
      w.va[yr + (int64_t)(t + u + 1) * w.B] = yv;
    }
  }
  for (; t + 8 <= w.T; t += 8) {
    float vin[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) vin[u] = w.va[vr + (int64_t)(t + u) * w.B];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      yv = lowpass_step(a, yv, c, vin[u]);
      w.va[yr + (int64_t)(t + u + 1) * w.B] = yv;
    }
  }
  for (; t < w.T; ++t) {
    yv = lowpass_step(a, yv, c, w.va[vr + (int64_t)t * w.B]);
    w.va[yr + (int64_t)(t + 1) * w.B] = yv;
  }
}

// probe buffer [step][probe_rows][B] <- block t + 1 of the probed rows
__global__ void k_w_probe(WView w, const int32_t* src, int32_t probe_rows, float* buf, int64_t step0) {
  W_ITEM(probe_rows);
  const uint32_t t = _c / (uint32_t)w.B, b = _c - t * (uint32_t)w.B;
  buf[((step0 + t) * probe_rows + _r) * w.B + b] = w.va[vat(w, G(src)[_r], w.B + _c)];
}

// k_w_probe for a subset of the probe rows: entry i copies window row src[i]
// into row dst[i] of the probe buffer, which holds `stride` rows per step.
__global__ void k_w_probe_map(WView w, const int32_t* src, const int32_t* dst, int32_t n, int32_t stride, float* buf,
                              int64_t step0) {
  W_ITEM(n);
  const uint32_t t = _c / (uint32_t)w.B, b = _c - t * (uint32_t)w.B;
  buf[((step0 + t) * stride + G(dst)[_r]) * w.B + b] = w.va[vat(w, G(src)[_r], w.B + _c)];
}

// Spike probes as bitmasks (a spiking neuron's output is 0 or amplitude / dt):
// word k of a step and batch column has bit j set when the neuron recorded at
// src[32 k + j] spiked (a nonzero output); entries of -1 pad a probe to whole
// words and stay 0.  Lanes run over batch columns, so each of the 32 reads of
// a thread is one coalesced row segment across its wavefront.
__global__ void k_w_probe_bits(WView w, const int32_t* src, int32_t words, uint32_t* bits, int64_t step0) {
  W_ITEM(words);
  const uint32_t t = _c / (uint32_t)w.B, b = _c - t * (uint32_t)w.B;
  gptr<int32_t> rs = G(src) + (int64_t)_r * 32;
  uint32_t m = 0;
#pragma unroll 8
  for (int j = 0; j < 32; ++j) {
    const int32_t r = rs[j];
    if (r >= 0 && w.va[vat(w, r, w.B + _c)] != 0.0f) m |= 1u << j;
  }
  bits[((step0 + t) * words + _r) * w.B + b] = m;
}

// block 0 <- block T for every row (the values the next window starts from)
__global__ void k_w_carry(WView w, int64_t rows) {
  W_ROWCOL(rows);
  const int64_t r0 = (int64_t)_r * w.vs + _b;
  w.va[r0] = w.va[r0 + (int64_t)w.T * w.B];
}

// ------------------------------------------------- fused ensembles over a window
// One workgroup per (op, group of cpw batch columns), for the whole window, in
// sub-windows of ts steps (a multiple of 16).  A thread slot g = tid + j*blockDim
// (j < NPT) owns neuron g % nmax of column g / nmax; its voltage and refractory
// time stay in registers for the whole window.  The "columns" of the two
// products below are the (batch column, step) pairs c*ts + s of a sub-window.
// Per sub-window:
//   1. input currents J = E x + bias on MFMA (v_mfma_f32_16x16x4f32; A lane l:
//      row l%16, k l/16; B lane l: k l/16, column l%16; result register v:
//      row 4(l/16) + v, column l%16), one (16-neuron tile, 16-column tile)
//      unit per wavefront at a time, written to LDS as [column][neuron];
//   2. every slot advances its neuron through the sub-window, overwriting each
//      J in LDS with the neuron's output -- no synchronisation between steps,
//      since a neuron depends only on its own past;
//   3. decoded outputs, [ndec x n] by [n x columns], on MFMA: units are
//      (16-column tile, chunk of neurons), partial tiles summed in LDS.
// The next sub-window's inputs are fetched into registers before step 1 and
// stored to LDS after it, so their latency overlaps the work.
typedef float mfma_f4x __attribute__((ext_vector_type(4)));
constexpr int kEnsXPre = 4;        // prefetched input values per thread

// Workgroups are numbered for the XCDs (workgroup g runs on XCD g % 8): XCD x
// takes a contiguous run of (op, column group), column group fastest, so the
// column groups of one op share their input and output lines in one L2.  The
// grid is padded to a multiple of eight; padding workgroups return at once.
//
// RW (weights in registers): each wavefront keeps, for the whole window, the
// encoder fragments of its neuron tiles (tiles wave, wave + nw, ..., at most 4
// tiles of k <= 16) and the decoder fragments of its neuron chunk (chunk
// wave % kch, at most 16 k steps), loaded once from global memory.  The units
// of both products are then assigned so that a wavefront only meets its own
// fragments; every unit accumulates in the same order as without RW, so the
// results are the same bit for bit.  Used when encoders and decoders are too
// large to stage in LDS.
constexpr int kRwTiles = 4, kRwKd = 4, kRwKs = 16;

// One neuron's updates through tsv steps of its LDS column (stride js), each
// current replaced by the neuron's output: blocks of 8 steps read their
// currents first, so that one LDS wait covers a block and the addresses are
// fixed offsets from one register.
template <class F>
__device__ __forceinline__ void sweep_cell(float* cell, int32_t js, int tsv, F&& upd) {
  int st = 0;
  for (; st + 8 <= tsv; st += 8) {
    float* c = cell + st * js;
    float jv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) jv[u] = c[u * js];
#pragma unroll
    for (int u = 0; u < 8; ++u) c[u * js] = upd(jv[u]);
  }
  for (; st < tsv; ++st) cell[st * js] = upd(cell[st * js]);
}

// The connection chain of Fig. 2 fused into an ensemble's input (window
// driver; one wavefront, one batch column b0): for window steps t0 .. t0 + tsn
// - 1, x_t = y_{t-1} and y_t = a y_{t-1} + b v_t with v_t = W d_t, d_t the
// upstream value (K rows from drow, block t + 1) and W the M x K transform.
// Over a tile of 16 steps s = 0 .. 15 starting from y_{-1} = y0 the filter
// unrolls to y_s = sum_{j <= s} b a^(s-j) v'_j with v'_0 = v_0 + (a / b) y0
// and v'_j = v_j otherwise, so a tile is two 16 x 16 products on MFMA and no
// sequential loop: V'^T = D^T W^T (plus the y0 term), then Y^T = L^T V'^T
// with L[j][s] = b a^(s-j) for j <= s, else 0.  The second product sums over
// j in the order j = 4 (l / 16) + kk, which is the layout the first one
// leaves its result in, so V'^T passes between them in registers.
// Fragments (lane l, m = l % 16, g = l / 16): wa[kk] = W[m][4 kk + g] and
// la[kk] = L[4 g + kk][m] (kept in LDS, Cf[kk][l] and Cf[4 + kk][l]), the
// upstream values of a tile D[4 kk + g][m] (kk = 0 .. 3), and ycur = y0[m]; the result lane l holds y_{4 g + q} for output
// m, which it stores as x one step later into Xdst[step * xs + m].
// chain_load fetches the first tile's upstream values early, so that their
// latency overlaps other work; later tiles (sub-windows of more than 16
// steps) are loaded when they are used.
constexpr int kChainPre = 4;

// Per-lane view of a chain's upstream values: lane l reads rows drow + 4 kk +
// l / 16 at window step l % 16 of a tile, from base (its value at block 1 of
// row drow + l / 16) plus kk * kstride + t * B; K inputs, M outputs.
struct ChainCtx {
  const float* base;
  int64_t kstride;
  int32_t K, M;
};

__device__ __forceinline__ void chain_load(const WView& w, const ChainCtx& cc, int32_t t0, int32_t tsn, int lane,
                                           float (&pre)[kChainPre]) {
#pragma unroll
  for (int kk = 0; kk < kChainPre; ++kk)
    pre[kk] = (4 * kk + lane / 16 < cc.K && lane % 16 < tsn) ? cc.base[kk * cc.kstride + (int64_t)t0 * w.B] : 0.0f;
}

__device__ __forceinline__ void chain_inputs(const WView& w, const ChainCtx& cc, int32_t t0, int32_t tsn, float* Xdst,
                                             int32_t xs, float& ycur, int lane, const float* Cf, float c0,
                                             const float (&pre)[kChainPre]) {
  const int m = lane % 16, g = lane / 16;
  float wa[4], la[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    wa[kk] = Cf[kk * 64 + lane];
    la[kk] = Cf[(4 + kk) * 64 + lane];
  }
  for (int32_t ct = 0; 16 * ct < tsn; ++ct) {
    const int32_t n = min(16, tsn - 16 * ct);   // steps of this tile
    float dv[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      dv[kk] = ct == 0 ? pre[kk]
                       : (4 * kk + g < cc.K && 16 * ct + m < tsn)
                             ? cc.base[kk * cc.kstride + (int64_t)(t0 + 16 * ct) * w.B]
                             : 0.0f;
    mfma_f4x v = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) v = __builtin_amdgcn_mfma_f32_16x16x4f32(dv[kk], wa[kk], v, 0, 0, 0);
    if (g == 0) v[0] += c0 * ycur;   // the carried state enters with step 0
    mfma_f4x y = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) y = __builtin_amdgcn_mfma_f32_16x16x4f32(la[kk], v[kk], y, 0, 0, 0);
    if (m < cc.M) {
      if (g == 0) Xdst[(16 * ct) * xs + m] = ycur;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (4 * g + q + 1 < n) Xdst[(16 * ct + 4 * g + q + 1) * xs + m] = y[q];
    }
    const int ql = (n - 1) % 4;   // y of the tile's last step, from lane 16 ((n - 1) / 4) + m
    const float last = ql == 0 ? y[0] : ql == 1 ? y[1] : ql == 2 ? y[2] : y[3];
    ycur = __shfl(last, 16 * ((n - 1) / 4) + m);
  }
}

// Smallest stride >= x that is 2 mod 4: rows of that stride put lanes i and
// i + 1 of a 16-lane group (rows i, i + 1; two adjacent columns per group)
// in 32 different banks.
__host__ __device__ inline int32_t stride2mod4(int32_t x) { return x + ((6 - x % 4) % 4); }

template <int NPT, bool RW, bool CHAIN>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(CHAIN ? 4 : 1))) k_w_ens(WView w, float* pa, EnsDesc E, float dt, int32_t nmax,
                                               int32_t ts, int32_t cpw, int32_t kch, int xblk, int enc_lds,
                                               int dec_lds, int32_t nops, int32_t xs, int32_t js) {
  extern __shared__ float lds[];
  const uint32_t ncg = ((uint32_t)w.B + cpw - 1) / cpw, total = (uint32_t)nops * ncg, chunk = (total + 7) / 8;
  const uint32_t L = (blockIdx.x % 8) * chunk + blockIdx.x / 8;
  if (L >= total) return;
  const int op = (int)(L / ncg);
  const int b0 = (int)(L - (uint32_t)op * ncg) * cpw;
  const int tid = threadIdx.x, nthr = blockDim.x, lane = tid % 64, wave = tid / 64, nw = nthr / 64;
  const EnsOp o = load_op(E.ops, op);
  const int n = o.n;
  const int d = o.x >= 0 ? E.d : 0, ndec = E.ndec, df0 = E.df[0];
  const int dp = E.d > 0 ? E.d : 1;
  const int ncol = cpw * ts, ctiles = ncol / 16;
  // LDS rows are padded (xs >= dp, js >= nmax) so that the products' lanes,
  // 16 columns apart, fall into different banks
  // RW keeps a second input buffer (the next sub-window's) and two sets of
  // per-wavefront partial decodes, so that a sub-window needs one barrier
  float* X = lds;                                   // [ncol][xs]
  float* Xn = X + (RW ? ncol * xs : 0);             // RW: the other input buffer
  float* Jb = Xn + ncol * xs;                       // [ncol][js]: currents, then outputs
  float* red = Jb + (int64_t)ncol * js;             // [ctiles][kch][16][16]; RW: [2][nw][ctiles][16][16]
  // [nmax] biases (RW: [nthr], zero past n), then [nmax][xs] encoders
  float* Bl = red + (RW ? 2 * nw * ctiles * 256 : ctiles * kch * 256);
  float* El = Bl + (RW ? nthr : nmax);              // rows of stride xs
  const int ds = stride2mod4(nmax);
  float* Dl = El + (enc_lds ? nmax * xs : 0);       // [ndec][ds] decoders (dec_lds)
  // fused connection chain into this op's input (K = crec[1] > 0), computed by
  // wavefront 0 alone
  // (its record is read once here: rows, sizes, coefficients)
  int32_t crec[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (CHAIN && E.chain) {
    gptr<int32_t> cg = G(E.chain) + (int64_t)op * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) crec[i] = cg[i];
  }
  const bool chain = CHAIN && crec[1] > 0;   // compiled out of the kernels without chains
  gptr<float> enc = G(E.enc) + (int64_t)o.enc * E.d;
  gptr<float> bias = G(E.bias) + o.bias;
  gptr<float> D0 = G(E.D[0]) + (int64_t)o.D[0] * E.Dcols[0];
  gptr<float> D1 = G(E.D[E.nf > 1 ? 1 : 0]) + (int64_t)o.D[E.nf > 1 ? 1 : 0] * E.Dcols[E.nf > 1 ? 1 : 0];
  const int64_t s0 = E.Dcols[0], s1 = E.Dcols[E.nf > 1 ? 1 : 0];
  const bool spiking = E.ntype == 0;
  const bool bf = spiking && dt * o.inv_tau <= 0.0625f;   // branch-free spiking update applies
  const float amp_dt = o.amp / dt, tau6 = o.tau6;
  const float* xsrc = w.va + (int64_t)(o.x >= 0 ? o.x : 0) * w.vs + (int64_t)xblk * w.B;
  // neuron state of this thread's slots
  float v[NPT], rf[NPT];
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    const int g = tid + j * nthr, c = g / nmax, r = g - c * nmax;
    const bool live = spiking && c < cpw && b0 + c < w.B && r < n;
    v[j] = live ? pa[(int64_t)(o.V + r) * w.B + b0 + c] : 0.0f;
    rf[j] = live ? pa[(int64_t)(o.ref + r) * w.B + b0 + c] : 0.0f;
  }
  auto stage_x = [&](int i, int32_t tb, int tsv) -> float {   // input value i of the sub-window at tb
    const int col = i / d, k = i - col * d, c = col / ts, st = col - c * ts;
    return (st < tsv && b0 + c < w.B) ? xsrc[(int64_t)k * w.vs + (int64_t)(tb + st) * w.B + b0 + c] : 0.0f;
  };
  // chain: W and L fragments and the carried filter state (wavefront 0)
  float* Cf = Dl + (dec_lds ? ndec * ds : 0);       // [8][64] chain fragments
  float ycur = 0.0f, c0 = 0.0f;
  ChainCtx cc{w.va, 4 * w.vs, crec[1], crec[4]};
  if (chain && wave == 0) {
    const int32_t K = crec[1], M = crec[4];
    const float a = __builtin_bit_cast(float, crec[6]), b = __builtin_bit_cast(float, crec[7]);
    gptr<float> Wc = G(E.chain_w) + (int64_t)crec[2] * E.chain_wcols;
    const int m = lane % 16, g = lane / 16;
    cc.base = w.va + (int64_t)(crec[0] + g) * w.vs + (int64_t)(m + 1) * w.B + b0;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int k = 4 * kk + g, j = 4 * g + kk;
      Cf[kk * 64 + lane] = (m < M && k < K) ? Wc[(int64_t)m * E.chain_wcols + k] : 0.0f;
      double p = b;   // b a^(m - j), powers formed in double
      for (int e = j; e < m; ++e) p *= (double)a;
      Cf[(4 + kk) * 64 + lane] = j <= m ? (float)p : 0.0f;
    }
    c0 = a / b;   // b != 0 (the planner fuses no chain without it)
    if (m < M && b0 < w.B) ycur = w.va[(int64_t)(crec[3] + m) * w.vs + b0];
  }
  {
    const int tsv = min(ts, w.T);
    if (chain) {
      if (wave == 0 && b0 < w.B) {
        float cpre0[kChainPre];
        chain_load(w, cc, 0, tsv, lane, cpre0);
        chain_inputs(w, cc, 0, tsv, X, xs, ycur, lane, Cf, c0, cpre0);
      }
    } else {
      for (int i = tid; i < ncol * d; i += nthr) {
        const int col = i / d, k = i - col * d;
        X[col * xs + k] = stage_x(i, 0, tsv);
      }
    }
  }
  // per-op constants: biases always, encoders and decoders when they fit
  if (RW) {
    // every slot of the workgroup is a neuron row of the products: rows past
    // n get zero bias (and zero encoder and decoder entries), so that they
    // compute zeros and the sub-window loop needs no per-lane tests; the
    // input columns past d up to the k steps' 4 kd are zero as well
    Bl[tid] = tid < n ? bias[tid] : 0.0f;
    const int dpad = 4 * ((d + 3) / 4) - d;
    for (int i = tid; i < 2 * ncol * dpad; i += nthr) {
      const int col = i / dpad, k = d + (i - col * dpad);
      X[col * xs + k] = 0.0f;   // X and Xn, which follows it
    }
  } else {
    for (int r = tid; r < n; r += nthr) Bl[r] = bias[r];
  }
  if (enc_lds)
    for (int i = tid; i < n * d; i += nthr) El[(i / d) * xs + i % d] = enc[(int64_t)i];
  if (dec_lds)
    for (int i = tid; i < ndec * n; i += nthr) {
      const int q = i / n, r = i - q * n;
      Dl[q * ds + r] = (q < df0 ? D0 + (int64_t)q * s0 : D1 + (int64_t)(q - df0) * s1)[r];
    }
  __syncthreads();
  const int ntile = (n + 15) / 16, kd = (d + 3) / 4;
  const int qa = lane % 16;
  gptr<float> drow = qa < df0 ? D0 + (int64_t)qa * s0 : D1 + (int64_t)(qa - df0) * s1;
  const int ksteps = (n + 4 * kch - 1) / (4 * kch);
  // Slots that stay fixed for the whole window, so that the sub-window loop
  // does no integer division: input value tid + c*nthr of a sub-window is
  // step st, column cc, dimension k, packed st | cc << 7 | k << 16, -1 past the
  // inputs or for a column beyond B (which keeps the zeros staged above), with
  // its LDS index in xlds; output tid is step st, column c, decoded dimension
  // q, packed the same way (st | c << 7 | q << 16), -1 past the outputs.  The
  // host keeps ts <= 64, cpw <= 512 and d, ndec < 32768.
  int32_t xslot[kEnsXPre], xlds[kEnsXPre];
#pragma unroll
  for (int c = 0; c < kEnsXPre; ++c) {
    const int i = tid + c * nthr;
    if (!chain && i < ncol * d) {
      const int col = i / d, k = i - col * d, cc = col / ts, st = col - cc * ts;
      xslot[c] = b0 + cc < w.B ? st | (cc << 7) | (k << 16) : -1;
      xlds[c] = col * xs + k;
    } else {
      xslot[c] = -1;
      xlds[c] = 0;
    }
  }
  int32_t oslot = -1;
  if (tid < ndec * ncol) {
    const int q = tid / ncol, col = tid - q * ncol, c = col / ts;
    oslot = (col - c * ts) | (c << 7) | (q << 16);
  }
  float ae[RW ? kRwTiles : 1][RW ? kRwKd : 1], ad[RW ? kRwKs : 1];
  if constexpr (RW) {
    // one column per workgroup, slot tid = neuron tid: wavefront `wave` owns
    // neurons 64 wave .. 64 wave + 63, i.e. encoder tiles 4 wave .. 4 wave + 3
    // and the decoder entries of those neurons
#pragma unroll
    for (int i = 0; i < kRwTiles; ++i)
#pragma unroll
      for (int kk = 0; kk < kRwKd; ++kk) {
        const int ra = 16 * (kRwTiles * wave + i) + lane % 16, k = 4 * kk + lane / 16;
        ae[i][kk] = (ra < n && k < d) ? enc[(int64_t)ra * E.d + k] : 0.0f;
      }
#pragma unroll
    for (int ks = 0; ks < kRwKs; ++ks) {
      const int r = 64 * wave + 4 * ks + lane / 16;
      ad[ks] = (qa < ndec && r < n) ? drow[r] : 0.0f;
    }
  }
  (void)ksteps;
  if constexpr (RW) {
    // Per sub-window, each wavefront alone: the currents of its own neurons
    // (MFMA) into LDS, their updates through the sub-window, their share of
    // the decoded outputs (MFMA) into its partial buffer, and its share of the
    // next inputs into the other input buffer; then one barrier, after which
    // the partials of every wavefront are added in wavefront order.  A
    // wavefront reads only LDS rows it wrote itself until that barrier.
    int xb = 0;
    const int oq = tid / ncol, ocol = tid - oq * ncol;   // this thread's first decoded output
    float* const odst = oq < ndec ? w.va + (int64_t)(oq < df0 ? o.d[0] + oq : o.d[1] + (oq - df0)) * w.vs +
                                        (int64_t)(ocol + 1) * w.B + b0
                                  : w.va;
    for (int32_t t0 = 0; t0 < w.T; t0 += ts) {
      const int tsv = min(ts, w.T - t0);
      const int32_t t1 = t0 + ts;
      const int tsn = t1 < w.T ? min(ts, w.T - t1) : 0;
      float xpre[kEnsXPre];
      if (!chain) {
#pragma unroll
        for (int c = 0; c < kEnsXPre; ++c) {
          const int32_t ps = xslot[c], st = ps & 127;
          xpre[c] = (ps >= 0 && st < tsn)
                        ? xsrc[(int64_t)(ps >> 16) * w.vs + (int64_t)(t1 + st) * w.B + b0 + ((ps >> 7) & 511)]
                        : 0.0f;
        }
      }
      float cpre[kChainPre];   // the next sub-window's upstream values (chain, wavefront 0)
      if (chain && wave == 0 && tsn > 0 && b0 < w.B) chain_load(w, cc, t1, tsn, lane, cpre);
      const float* Xc = xb ? Xn : X;
      float* Xo = xb ? X : Xn;
      float* rb = red + xb * nw * ctiles * 256;
      // 1. currents of this wavefront's neurons (all four tiles: rows past n
      // compute zeros), loads and stores at fixed offsets from one address
      // (all kRwKd k steps when d > 12: no test per step)
      auto currents = [&](auto full) {
#pragma unroll
        for (int i = 0; i < kRwTiles; ++i) {
          const int r0 = 16 * (kRwTiles * wave + i) + 4 * (lane / 16);
          for (int ct = 0; ct < ctiles; ++ct) {
            const int col = 16 * ct + lane % 16;
            const float* xr = Xc + col * xs + lane / 16;
            mfma_f4x acc = {Bl[r0], Bl[r0 + 1], Bl[r0 + 2], Bl[r0 + 3]};   // J = bias + E x
#pragma unroll
            for (int kk = 0; kk < kRwKd; ++kk)
              if (decltype(full)::value || kk < kd)
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(ae[i][kk], xr[4 * kk], acc, 0, 0, 0);
            float* jr = Jb + col * js + r0;
#pragma unroll
            for (int q = 0; q < 4; ++q) jr[q] = acc[q];
          }
        }
      };
      if (kd == kRwKd)
        currents(std::true_type{});
      else
        currents(std::false_type{});
      // 2. its neurons through the sub-window (slot tid: neuron tid, column 0;
      // slots past n carry zero state and current, and output zeros)
      if (b0 < w.B) {
        float* cell = Jb + tid;
        if (bf)
          sweep_cell(cell, js, tsv, [&](float j) {
            return lif_update_bf(j, v[0], rf[0], tau6, o.tau_ref, amp_dt, dt, o.inv_tau);
          });
        else
          for (int st = 0; st < tsv; ++st)
            cell[st * js] = neuron_update(E.ntype, cell[st * js], v[0], rf[0], o.tau_rc, o.tau_ref, o.amp, o.full,
                                          dt, o.inv_tau);
      }
      // 3. its neurons' share of the decoded outputs
      for (int ct = 0; ndec > 0 && ct < ctiles; ++ct) {
        const int col = 16 * ct + lane % 16;
        mfma_f4x acc = {0.0f, 0.0f, 0.0f, 0.0f};
        const float* sr = Jb + col * js + 64 * wave + lane / 16;
#pragma unroll
        for (int ks = 0; ks < kRwKs; ++ks) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(ad[ks], sr[4 * ks], acc, 0, 0, 0);
#pragma unroll
        for (int q = 0; q < 4; ++q) rb[((wave * ctiles + ct) * 16 + 4 * (lane / 16) + q) * 16 + lane % 16] = acc[q];
      }
      // 4. the next sub-window's inputs into the other buffer
      if (chain && wave == 0 && tsn > 0 && b0 < w.B)
        chain_inputs(w, cc, t1, tsn, Xo, xs, ycur, lane, Cf, c0, cpre);
      if (!chain) {
#pragma unroll
        for (int c = 0; c < kEnsXPre; ++c)
          if (tsn > 0 && xslot[c] >= 0) Xo[xlds[c]] = xpre[c];
      }
      if (tsn > 0 && !chain) {
        for (int i = tid + kEnsXPre * nthr; i < ncol * d; i += nthr) {
          const int col = i / d, k = i - col * d;
          Xo[col * xs + k] = stage_x(i, t1, tsn);
        }
      }
      __syncthreads();
      // 5. decoded outputs: the wavefronts' partials in wavefront order (the
      // first output of each thread from its precomputed slot)
      if (b0 < w.B)
        for (int i = tid; i < ndec * ncol; i += nthr) {
          int q = oq, col = ocol;
          float* dst = odst;
          if (i != tid) {
            q = i / ncol, col = i - q * ncol;
            dst = w.va + (int64_t)(q < df0 ? o.d[0] + q : o.d[1] + (q - df0)) * w.vs + (int64_t)(col + 1) * w.B + b0;
          }
          if (col < tsv) {
            const float* pr = rb + ((col / 16) * 16 + q) * 16 + col % 16;
            float sum = 0.0f;
            for (int ww = 0; ww < nw; ++ww) sum += pr[ww * ctiles * 256];
            dst[(int64_t)t0 * w.B] = sum;
          }
        }
      if (o.s >= 0) {   // neuron outputs of every wavefront, then a barrier before they are overwritten
        for (int i = tid; i < ncol * n; i += nthr) {
          const int r = i / ncol, st = i - r * ncol;
          if (st < tsv && b0 < w.B)
            w.va[(int64_t)(o.s + r) * w.vs + (int64_t)(t0 + st + 1) * w.B + b0] = Jb[st * js + r];
        }
        __syncthreads();
      }
      xb ^= 1;
    }
  } else
  for (int32_t t0 = 0; t0 < w.T; t0 += ts) {
    const int tsv = min(ts, w.T - t0);
    // 0. fetch the next sub-window's inputs
    const int32_t t1 = t0 + ts;
    const int tsn = t1 < w.T ? min(ts, w.T - t1) : 0;
    float xpre[kEnsXPre];
#pragma unroll
    for (int c = 0; c < kEnsXPre; ++c) {
      const int32_t ps = xslot[c], st = ps & 127;
      xpre[c] = (ps >= 0 && st < tsn)
                    ? xsrc[(int64_t)(ps >> 16) * w.vs + (int64_t)(t1 + st) * w.B + b0 + ((ps >> 7) & 511)]
                    : 0.0f;
    }
    float cpre[kChainPre];   // the next sub-window's upstream values (chain, wavefront 0)
    if (chain && wave == 0 && tsn > 0 && b0 < w.B) chain_load(w, cc, t1, tsn, lane, cpre);
    // 1. J = E x + bias
    for (int u = wave; u < ntile * ctiles; u += nw) {
      const int nt = u / ctiles, ct = u - nt * ctiles;
      const int col = 16 * ct + lane % 16;
      const int rb0 = 16 * nt + 4 * (lane / 16);
      mfma_f4x acc;   // J = bias + E x (rows past n unused)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[q] = rb0 + q < n ? Bl[rb0 + q] : 0.0f;
      for (int kk = 0; kk < kd; ++kk) {
        const int ra = 16 * nt + lane % 16, k = 4 * kk + lane / 16;
        const float a = (ra < n && k < d) ? (enc_lds ? El[ra * xs + k] : enc[(int64_t)ra * E.d + k]) : 0.0f;
        const float xb = k < d ? X[col * xs + k] : 0.0f;
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, xb, acc, 0, 0, 0);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = rb0 + q;
        if (r < n) Jb[col * js + r] = acc[q];
      }
    }
    __syncthreads();
    // next inputs into LDS (every read of this sub-window's X is done)
    if (chain && wave == 0 && tsn > 0 && b0 < w.B)
      chain_inputs(w, cc, t1, tsn, X, xs, ycur, lane, Cf, c0, cpre);
#pragma unroll
    for (int c = 0; c < kEnsXPre; ++c)
      if (tsn > 0 && xslot[c] >= 0) X[xlds[c]] = xpre[c];
    if (tsn > 0 && !chain) {   // inputs beyond the prefetch registers
      for (int i = tid + kEnsXPre * nthr; i < ncol * d; i += nthr) {
        const int col = i / d, k = i - col * d;
        X[col * xs + k] = stage_x(i, t1, tsn);
      }
    }
    // 2. neurons through the sub-window
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const int g = tid + j * nthr, c = g / nmax, r = g - c * nmax;
      if (c < cpw && b0 + c < w.B && r < n) {
        float* cell = Jb + (int64_t)c * ts * js + r;
        if (bf) {
          sweep_cell(cell, js, tsv, [&](float jc) {
            return lif_update_bf(jc, v[j], rf[j], tau6, o.tau_ref, amp_dt, dt, o.inv_tau);
          });
        } else {
          for (int st = 0; st < tsv; ++st)
            cell[st * js] = neuron_update(E.ntype, cell[st * js], v[j], rf[j], o.tau_rc, o.tau_ref, o.amp,
                                            o.full, dt, o.inv_tau);
        }
      }
    }
    __syncthreads();
    // 3. decoded outputs
    if (ndec > 0) {
      for (int u = wave; u < ctiles * kch; u += nw) {
        const int ct = u / kch, kc = u - ct * kch;
        const int col = 16 * ct + lane % 16;
        mfma_f4x acc = {0.0f, 0.0f, 0.0f, 0.0f};
        for (int ks = 0; ks < ksteps; ++ks) {
          const int r = 4 * (kc + kch * ks) + lane / 16;
          const float a = (qa < ndec && r < n) ? (dec_lds ? Dl[qa * ds + r] : drow[r]) : 0.0f;
          const float sb = r < n ? Jb[col * js + r] : 0.0f;
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, sb, acc, 0, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) red[(u * 16 + 4 * (lane / 16) + q) * 16 + lane % 16] = acc[q];
      }
    }
    __syncthreads();
    for (int i = tid; i < ndec * ncol; i += nthr) {
      int q, c, st;
      if (i == tid) {
        st = oslot & 127, c = (oslot >> 7) & 511, q = oslot >> 16;
      } else {
        const int cl = i - (q = i / ncol) * ncol;
        c = cl / ts, st = cl - c * ts;
      }
      const int col = c * ts + st;
      if (st < tsv && b0 + c < w.B) {
        float sum = 0.0f;
        for (int kc = 0; kc < kch; ++kc) sum += red[(((col / 16) * kch + kc) * 16 + q) * 16 + col % 16];
        const int dr = q < df0 ? o.d[0] + q : o.d[1] + (q - df0);
        w.va[(int64_t)dr * w.vs + (int64_t)(t0 + st + 1) * w.B + b0 + c] = sum;
      }
    }
    if (o.s >= 0) {
      // neuron outputs: adjacent lanes take adjacent batch columns, then steps,
      // so that a wavefront's stores fall into few cache lines
      for (int i = tid; i < ncol * n; i += nthr) {
        const int r = i / ncol, rem = i - r * ncol, st = rem / cpw, c = rem - st * cpw;
        if (st < tsv && b0 + c < w.B)
          w.va[(int64_t)(o.s + r) * w.vs + (int64_t)(t0 + st + 1) * w.B + b0 + c] = Jb[(c * ts + st) * js + r];
      }
    }
    __syncthreads();
  }
  if (chain && wave == 0 && lane < crec[4] && b0 < w.B)   // the filter state the next window starts from
    w.va[(int64_t)(crec[3] + lane) * w.vs + (int64_t)w.T * w.B + b0] = ycur;
  if (spiking) {
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const int g = tid + j * nthr, c = g / nmax, r = g - c * nmax;
      if (c < cpw && b0 + c < w.B && r < n) {
        pa[(int64_t)(o.V + r) * w.B + b0 + c] = v[j];
        pa[(int64_t)(o.ref + r) * w.B + b0 + c] = rf[j];
      }
    }
  }
}

// ------------------------------------------------- products on fp32 MFMA
// dst[m][c] += sum_k W[m][k] x[k][c] for every op of a merged DotInc group and
// every (step, column) c of the window: per op a dense M x K by K x (T*B)
// product.  Workgroup tile 64 x 64 (M x columns), K in slices of 16 staged in
// LDS; each of the four wavefronts owns a 32 x 32 quarter and accumulates it
// with v_mfma_f32_32x32x2f32 (A lane l: row l%32, k l/32; B lane l: k l/32,
// column l%32; result register v: row 8(v/4) + 4(l/32) + v%4, column l%32).
typedef float mfma_f16x __attribute__((ext_vector_type(16)));

constexpr int kGemmBM = 64, kGemmBN = 64, kGemmBK = 16;

// One 64 x 64 tile (rows m0.., columns c0.. of the window) of op's product,
// by a workgroup of 256 threads, staging through As and Bs.
__device__ __forceinline__ void gemm64_tile(const WView& w, int32_t M, int32_t K, const float* Wt,
                                            const int32_t* w_row, const int32_t* x_row, const int32_t* d_row,
                                            int xblk, int op, int64_t m0, int64_t c0,
                                            float (*As)[kGemmBM + 4], float (*Bs)[kGemmBN + 4]) {
  const int64_t N = (int64_t)w.T * w.B;
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int wm = wave / 2, wn = wave % 2;
  gptr<float> A = G(Wt) + (int64_t)G(w_row)[op] * K;
  const float* X = w.va + (int64_t)G(x_row)[op] * w.vs + (int64_t)xblk * w.B;
  float* C = w.va + (int64_t)G(d_row)[op] * w.vs + w.B;
  mfma_f16x acc;
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
  for (int32_t k0 = 0; k0 < K; k0 += kGemmBK) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + q * 256;
      const int mm = idx / kGemmBK, kk = idx % kGemmBK;
      const int64_t m = m0 + mm;
      const int32_t k = k0 + kk;
      As[kk][mm] = (m < M && k < K) ? A[m * K + k] : 0.0f;
      const int kb = idx / kGemmBN, jj = idx % kGemmBN;
      const int32_t kx = k0 + kb;
      const int64_t c = c0 + jj;
      Bs[kb][jj] = (kx < K && c < N) ? X[(int64_t)kx * w.vs + c] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < kGemmBK; kk += 2) {
      const float a = As[kk + lane / 32][wm * 32 + lane % 32];
      const float b = Bs[kk + lane / 32][wn * 32 + lane % 32];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
    __syncthreads();
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int64_t m = m0 + wm * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
    const int64_t c = c0 + wn * 32 + lane % 32;
    if (m < M && c < N) C[m * w.vs + c] += acc[v];
  }
}

__global__ void __launch_bounds__(256) k_w_gemm(WView w, int32_t M, int32_t K, int32_t mtiles, const float* Wt,
                                                const int32_t* w_row, const int32_t* x_row, const int32_t* d_row,
                                                int xblk) {
  __shared__ float As[kGemmBK][kGemmBM + 4];
  __shared__ float Bs[kGemmBK][kGemmBN + 4];
  const int op = blockIdx.y / mtiles, mt = blockIdx.y - op * mtiles;
  gemm64_tile(w, M, K, Wt, w_row, x_row, d_row, xblk, op, (int64_t)mt * kGemmBM, (int64_t)blockIdx.x * kGemmBN,
              As, Bs);
}

// Products with few rows and a deep K (M <= 16, K >= 256): one lane per
// (step, column) of the window, all M rows per lane.  The eight wavefronts of
// a workgroup take eight contiguous ranges of K and meet in LDS, where their
// partial sums are added in wavefront order (the result does not depend on
// timing).  W is read at wave-uniform addresses.
constexpr int kSkM = 16, kSkW = 8;

__global__ void __launch_bounds__(512) k_w_skinny(WView w, int32_t M, int32_t K, int32_t ctiles, const float* Wt,
                                                  const int32_t* w_row, const int32_t* x_row, const int32_t* d_row,
                                                  int xblk) {
  __shared__ float red[kSkW][kSkM][64];
  const int64_t N = (int64_t)w.T * w.B;
  const int op = blockIdx.x / ctiles;
  const int64_t c0 = (int64_t)(blockIdx.x - op * ctiles) * 64;
  const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  const int64_t c = c0 + lane;
  const bool live = c < N;
  const int32_t kper = (K + kSkW - 1) / kSkW;
  const int32_t kb = min(K, wave * kper), ke = min(K, kb + kper);
  gptr<float> A = G(Wt) + (int64_t)G(w_row)[op] * K;
  const float* X = w.va + (int64_t)G(x_row)[op] * w.vs + (int64_t)xblk * w.B;
  float acc[kSkM];
#pragma unroll
  for (int m = 0; m < kSkM; ++m) acc[m] = 0.0f;
  int32_t k = kb;
  // 32 (then 8) input rows are loaded before they are used, so that their
  // loads are in flight together; each sum still runs over k in order
  for (; k + 32 <= ke; k += 32) {
    float xv[32];
#pragma unroll
    for (int u = 0; u < 32; ++u) xv[u] = live ? X[(int64_t)(k + u) * w.vs + c] : 0.0f;
#pragma unroll
    for (int m = 0; m < kSkM; ++m)
      if (m < M) {
#pragma unroll
        for (int u = 0; u < 32; ++u) acc[m] += A[(int64_t)m * K + k + u] * xv[u];
      }
  }
  for (; k + 8 <= ke; k += 8) {
    float xv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) xv[u] = live ? X[(int64_t)(k + u) * w.vs + c] : 0.0f;
#pragma unroll
    for (int m = 0; m < kSkM; ++m)
      if (m < M) {
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[m] += A[(int64_t)m * K + k + u] * xv[u];
      }
  }
  for (; k < ke; ++k) {
    const float x = live ? X[(int64_t)k * w.vs + c] : 0.0f;
#pragma unroll
    for (int m = 0; m < kSkM; ++m)
      if (m < M) acc[m] += A[(int64_t)m * K + k] * x;
  }
#pragma unroll
  for (int m = 0; m < kSkM; ++m) red[wave][m][lane] = acc[m];
  __syncthreads();
  float* C = w.va + (int64_t)G(d_row)[op] * w.vs + w.B;
  for (int i = threadIdx.x; i < M * 64; i += blockDim.x) {
    const int m = i / 64, l = i % 64;
    float sum = 0.0f;
#pragma unroll
    for (int v = 0; v < kSkW; ++v) sum += red[v][m][l];
    if (c0 + l < N) C[(int64_t)m * w.vs + c0 + l] += sum;
  }
}

// Tile order of the large products.  Workgroups are handed to the eight XCDs
// round robin (workgroup g to XCD g % 8); renumbering g so that XCD x receives
// the contiguous run x*chunk .. of (op, column tile, row tile), row tile
// fastest, lets the row tiles that share a column tile of x run back to back
// on one XCD and read that tile from its L2.  The grid is padded to a multiple
// of eight; the padding workgroups return at once.
struct TileIdx { int op, mt, nt; bool live; };
__device__ __forceinline__ TileIdx xcd_tile(uint32_t mtiles, uint32_t ntiles, uint32_t nops, uint32_t g) {
  const uint32_t total = mtiles * ntiles * nops, chunk = (total + 7) / 8;
  const uint32_t L = (g % 8) * chunk + g / 8;
  TileIdx t{0, 0, 0, L < total};
  if (!t.live) return t;
  t.mt = (int)(L % mtiles);
  const uint32_t rest = L / mtiles;
  t.nt = (int)(rest % ntiles);
  t.op = (int)(rest / ntiles);
  return t;
}

// Larger products: workgroup tile 128 x 128, K in slices of 16, double-buffered
// LDS; each of the four wavefronts owns a 64 x 64 quarter as 2 x 2 blocks of
// v_mfma_f32_32x32x2f32.  The next slice is fetched into registers (four
// float4 per thread) while the current one is multiplied.  Used when K and B
// are multiples of 4 (so rows of W and of x are 16-byte aligned).
constexpr int kG2M = 128, kG2N = 128, kG2K = 16;

//
// Tail split: when the 128 x 128 tiles number a little more than a whole
// multiple of the CUs, the last column tiles would leave most CUs idle while
// a few finish one extra tile.  The launch then covers only the first ntiles
// column tiles with 128 x 128 tiles (workgroups 0 .. gbig-1) and the columns
// after them with 64 x 64 tiles (workgroups gbig ..), a quarter of the work
// each, which the CUs take up beside their large tiles.  Both tile sizes add
// k in the same order (slices of 16, pairs on v_mfma_f32_32x32x2f32), so the
// split does not change any result.
__global__ void __launch_bounds__(256, 4) k_w_gemm2(WView w, int32_t M, int32_t K, int32_t mtiles, int32_t ntiles,
                                                 int32_t nops, const float* Wt, const int32_t* w_row,
                                                 const int32_t* x_row, const int32_t* d_row, int xblk,
                                                 uint32_t gbig) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  __shared__ float As[2][kG2K][kG2M + 4];
  __shared__ float Bs[2][kG2K][kG2N + 4];
  const int64_t N = (int64_t)w.T * w.B;
  if (blockIdx.x >= gbig) {   // 64 x 64 tiles of the columns after the large tiles
    const int64_t cs = (int64_t)ntiles * kG2N;
    const uint32_t mt2 = (uint32_t)((M + kGemmBM - 1) / kGemmBM);
    const uint32_t nt2 = (uint32_t)((N - cs + kGemmBN - 1) / kGemmBN);
    const TileIdx st = xcd_tile(mt2, nt2, nops, blockIdx.x - gbig);
    if (!st.live) return;
    gemm64_tile(w, M, K, Wt, w_row, x_row, d_row, xblk, st.op, (int64_t)st.mt * kGemmBM,
                cs + (int64_t)st.nt * kGemmBN, (float(*)[kGemmBM + 4]) & As[0][0][0],
                (float(*)[kGemmBN + 4]) & Bs[0][0][0]);
    return;
  }
  const TileIdx ti = xcd_tile(mtiles, ntiles, nops, blockIdx.x);
  if (!ti.live) return;
  const int op = ti.op, mt = ti.mt;
  const int64_t m0 = (int64_t)mt * kG2M, c0 = (int64_t)ti.nt * kG2N;
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int wm = wave / 2, wn = wave % 2;
  gptr<float> A = G(Wt) + (int64_t)G(w_row)[op] * K;
  const float* X = w.va + (int64_t)G(x_row)[op] * w.vs + (int64_t)xblk * w.B;
  float* C = w.va + (int64_t)G(d_row)[op] * w.vs + w.B;
  // fetch assignment: A slice 128 x 16 = 512 float4 (row mm, k4), B slice 16 x 128 = 512 float4 (k, col4)
  f4v ra[2], rb[2];
  auto fetch = [&](int32_t k0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + q * 256;
      const int mm = idx / 4, k4 = idx % 4;
      const int64_t m = m0 + mm;
      const int32_t k = k0 + 4 * k4;
      f4v va = {0.0f, 0.0f, 0.0f, 0.0f};
      if (m < M) {
        if (k + 3 < K) {
          va = *(const __attribute__((address_space(1))) f4v*)(A + m * K + k);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) va[e] = k + e < K ? A[m * K + k + e] : 0.0f;
        }
      }
      ra[q] = va;
      const int kb = idx / 32, j4 = idx % 32;
      const int32_t kx = k0 + kb;
      const int64_t c = c0 + 4 * j4;
      f4v vb = {0.0f, 0.0f, 0.0f, 0.0f};
      if (kx < K) {
        if (c + 3 < N) {
          vb = *(const f4v*)(X + (int64_t)kx * w.vs + c);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) vb[e] = c + e < N ? X[(int64_t)kx * w.vs + c + e] : 0.0f;
        }
      }
      rb[q] = vb;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + q * 256;
      const int mm = idx / 4, k4 = idx % 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) As[buf][4 * k4 + e][mm] = ra[q][e];
      const int kb = idx / 32, j4 = idx % 32;
#pragma unroll
      for (int e = 0; e < 4; ++e) Bs[buf][kb][4 * j4 + e] = rb[q][e];
    }
  };
  mfma_f16x acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
  fetch(0);
  stash(0);
  __syncthreads();
  int buf = 0;
  for (int32_t k0 = 0; k0 < K; k0 += kG2K) {
    const bool more = k0 + kG2K < K;
    if (more) fetch(k0 + kG2K);
#pragma unroll
    for (int kk = 0; kk < kG2K; kk += 2) {
      float a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[buf][kk + lane / 32][wm * 64 + i * 32 + lane % 32];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = Bs[buf][kk + lane / 32][wn * 64 + j * 32 + lane % 32];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) stash(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t m = m0 + wm * 64 + i * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
        const int64_t c = c0 + wn * 64 + j * 32 + lane % 32;
        if (m < M && c < N) C[m * w.vs + c] += acc[i][j][v];
      }
}

// The same products with bf16 inputs and fp32 accumulation (v_mfma_f32_32x32x16_bf16):
// W arrives already rounded to bf16, one [M][K] block per op (op k at k*M*K);
// x is rounded to nearest even as it is staged.  Workgroup tile 128 x 128, K in
// slices of 64, double-buffered; LDS keeps both operands k-contiguous ([m][k]
// and [column][k], rows padded to 72 values) so that each lane reads its eight
// k values of a fragment as one 16-byte word.  A lane l supplies row (or
// column) l%32 and k values 8(l/32) .. 8(l/32)+7 of each 16-wide k step; the
// result layout is that of the fp32 32 x 32 products.  Needs K % 8 == 0 and
// B % 4 == 0.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
constexpr int kGbM = 128, kGbN = 128, kGbK = 32, kGbP = 40, kGbU = kGbK / 16;
static_assert(kGemmBK == kG2K && kGemmBK * (kGemmBM + 4) <= 2 * kG2K * (kG2M + 4) &&
                  kGemmBK * (kGemmBN + 4) <= 2 * kG2K * (kG2N + 4),
              "the tail tiles of k_w_gemm2 add k in the same slices and fit its LDS arrays");
static_assert(kGbM == kG2M && kGbN == kG2N, "the two large-product kernels share their tile grid");

__global__ void __launch_bounds__(256, 3) k_w_gemm_bf16(WView w, int32_t M, int32_t K, int32_t mtiles,
                                                     int32_t ntiles, int32_t nops, const uint16_t* W16,
                                                     const int32_t* x_row, const int32_t* d_row, int xblk) {
  __shared__ __attribute__((aligned(16))) __bf16 As[2][kGbM][kGbP];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[2][kGbN][kGbP];
  const TileIdx ti = xcd_tile(mtiles, ntiles, nops, blockIdx.x);
  if (!ti.live) return;
  const int64_t N = (int64_t)w.T * w.B;
  const int op = ti.op, mt = ti.mt;
  const int64_t m0 = (int64_t)mt * kGbM, c0 = (int64_t)ti.nt * kGbN;
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int wm = wave / 2, wn = wave % 2;
  const uint16_t* A = W16 + (int64_t)op * M * K;
  const float* X = w.va + (int64_t)G(x_row)[op] * w.vs + (int64_t)xblk * w.B;
  float* C = w.va + (int64_t)G(d_row)[op] * w.vs + w.B;
  // fetch assignment: A slice 128 x 64 and B slice 64 x 128 are 1024 units of
  // eight k values each; thread tid takes units tid + 256 q (q < 4) of both
  bf16x8 ra[kGbU], rb[kGbU];
  auto fetch = [&](int32_t k0) {
#pragma unroll
    for (int q = 0; q < kGbU; ++q) {
      const int idx = tid + q * 256;
      const int mm = idx / (kGbK / 8), k8 = idx % (kGbK / 8);
      const int64_t m = m0 + mm;
      const int32_t k = k0 + 8 * k8;
      bf16x8 va = {};
      if (m < M && k < K) va = *(const bf16x8*)(A + m * K + k);
      ra[q] = va;
      const int cc = idx % kGbN, kb = idx / kGbN;
      const int64_t c = c0 + cc;
      const int32_t kx = k0 + 8 * kb;
      bf16x8 vb = {};
      if (c < N && kx < K) {
#pragma unroll
        for (int e = 0; e < 8; ++e) vb[e] = (__bf16)X[(int64_t)(kx + e) * w.vs + c];
      }
      rb[q] = vb;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int q = 0; q < kGbU; ++q) {
      const int idx = tid + q * 256;
      *(bf16x8*)&As[buf][idx / (kGbK / 8)][8 * (idx % (kGbK / 8))] = ra[q];
      *(bf16x8*)&Bs[buf][idx % kGbN][8 * (idx / kGbN)] = rb[q];
    }
  };
  mfma_f16x acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
  fetch(0);
  stash(0);
  __syncthreads();
  int buf = 0;
  for (int32_t k0 = 0; k0 < K; k0 += kGbK) {
    const bool more = k0 + kGbK < K;
    if (more) fetch(k0 + kGbK);
#pragma unroll
    for (int ks = 0; ks < kGbK; ks += 16) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = *(const bf16x8*)&As[buf][wm * 64 + i * 32 + lane % 32][ks + 8 * (lane / 32)];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = *(const bf16x8*)&Bs[buf][wn * 64 + j * 32 + lane % 32][ks + 8 * (lane / 32)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) stash(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t m = m0 + wm * 64 + i * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
        const int64_t c = c0 + wn * 64 + j * 32 + lane % 32;
        if (m < M && c < N) C[m * w.vs + c] += acc[i][j][v];
      }
}

// Four consecutive (step, column) entries per thread (needs T*B % 4 == 0 and
// B % 4 == 0, so every row of every block is 16-byte aligned).
typedef float w_f4 __attribute__((ext_vector_type(4)));
#define W_ITEM4(rows)                                                          \
  const uint32_t _i = blockIdx.x * blockDim.x + threadIdx.x;                   \
  const uint32_t _q = ((uint32_t)w.T * (uint32_t)w.B) / 4;                     \
  if (_i >= (uint32_t)(rows) * _q) return;                                     \
  const uint32_t _r = _i / _q, _c = 4 * (_i - _r * _q);

__device__ __forceinline__ w_f4& w4(const WView& w, int64_t row, int64_t c) {
  return *(w_f4*)(w.va + row * w.vs + c);
}

__global__ void k_w_reset4(WView w, int64_t rows, Opnd dst, const float* values) {
  W_ITEM4(rows);
  const float v = values ? G(values)[_r] : 0.0f;
  w4(w, rowof(dst, _r), w.B + _c) = w_f4{v, v, v, v};
}

// k_w_probe, four entries per thread; the probe buffer is not read again
// before the host copies it out, so its stores bypass the caches
__global__ void k_w_probe4(WView w, const int32_t* src, int32_t probe_rows, float* buf, int64_t step0) {
  W_ITEM4(probe_rows);
  const uint32_t t = _c / (uint32_t)w.B, b = _c - t * (uint32_t)w.B;
  const w_f4 v = w4(w, G(src)[_r], w.B + _c);
  __builtin_nontemporal_store(v, (w_f4*)(buf + ((step0 + t) * probe_rows + _r) * w.B + b));
}

__device__ __forceinline__ w_f4 w_src4(const WView& w, const float* param, int bcast, int64_t row, int blk,
                                       uint32_t c) {
  if (bcast) {
    const float v = G(param)[row];
    return w_f4{v, v, v, v};
  }
  return w4(w, row, (int64_t)blk * w.B + c);
}

// k_w_feed, four entries per thread (B a multiple of 4: the staged rows are
// 16-byte aligned as well)
__global__ void k_w_feed4(WView w, int64_t rows, Opnd dst, const int32_t* feed_row, const float* stage,
                          int32_t feed_rows, int64_t t0) {
  W_ITEM4(rows);
  const uint32_t t = _c / (uint32_t)w.B, b = _c - t * (uint32_t)w.B;
  w4(w, rowof(dst, _r), w.B + _c) = *(const w_f4*)(stage + ((t0 + t) * feed_rows + G(feed_row)[_r]) * w.B + b);
}

// k_w_elem_inc, four entries per thread (each entry the same sum, in the same order)
__global__ void k_w_elem_inc4(WView w, int64_t rows, Opnd dst, const float* a_param, Opnd a, int a_bcast, int ablk,
                              const float* x_param, Opnd x, int x_bcast, int xblk, const int32_t* ptr);

__global__ void k_w_copy_inc4(WView w, int64_t rows, Opnd dst, const float* param, Opnd src, int bcast, int sblk,
                              const int32_t* ptr) {
  W_ITEM4(rows);
  w_f4& d = w4(w, rowof(dst, _r), w.B + _c);
  w_f4 acc = d;
  if (ptr) {
    for (int32_t e = G(ptr)[_r]; e < G(ptr)[_r + 1]; ++e) acc += w_src4(w, param, bcast, rowof(src, e), sblk, _c);
  } else {
    acc += w_src4(w, param, bcast, rowof(src, _r), sblk, _c);
  }
  d = acc;
}

__global__ void k_w_elem_inc4(WView w, int64_t rows, Opnd dst, const float* a_param, Opnd a, int a_bcast, int ablk,
                              const float* x_param, Opnd x, int x_bcast, int xblk, const int32_t* ptr) {
  W_ITEM4(rows);
  w_f4& d = w4(w, rowof(dst, _r), w.B + _c);
  w_f4 acc = d;
  if (ptr) {
    for (int32_t e = G(ptr)[_r]; e < G(ptr)[_r + 1]; ++e)
      acc += w_src4(w, a_param, a_bcast, rowof(a, e), ablk, _c) * w_src4(w, x_param, x_bcast, rowof(x, e), xblk, _c);
  } else {
    acc += w_src4(w, a_param, a_bcast, rowof(a, _r), ablk, _c) * w_src4(w, x_param, x_bcast, rowof(x, _r), xblk, _c);
  }
  d = acc;
}
