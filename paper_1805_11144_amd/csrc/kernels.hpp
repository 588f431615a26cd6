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

// Row of the r-th work item of an operand: slice start + r, or idx[r].
struct Opnd {
  const int32_t* idx;
  int64_t start;
};

__device__ __forceinline__ int64_t rowof(const Opnd& o, int64_t r) {
  return o.idx ? (int64_t)o.idx[r] : o.start + r;
}

struct NeuronParams {
  float tau_rc, tau_ref, amp;                     // uniform values
  float full;                                     // expm1(-dt / tau_rc), uniform
  const float *tau_rc_r, *tau_ref_r, *amp_r;      // per-row values or null
  const float* full_r;                            // per-row expm1(-dt / tau_rc) or null
};

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

__device__ __forceinline__ void lif_item(float* st, const Strides& S, int64_t r, int64_t b,
                                         const Opnd& J, const Opnd& s, const Opnd& V, const Opnd& R,
                                         const NeuronParams& np, float dt) {
  const float tau_rc = np.tau_rc_r ? np.tau_rc_r[r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? np.tau_ref_r[r] : np.tau_ref;
  const float amp = np.amp_r ? np.amp_r[r] : np.amp;
  const int64_t jv = at(S, rowof(J, r), b), vv = at(S, rowof(V, r), b), rv = at(S, rowof(R, r), b);
  const float j = st[jv];
  float v = st[vv];
  float rf = st[rv];
  // integrate exactly over the non-refractory part of the step; a neuron that
  // is not refractory integrates the whole step with the precomputed factor
  const float integ = fminf(fmaxf(dt - rf, 0.0f), dt);
  const float e = rf <= 0.0f ? (np.full_r ? np.full_r[r] : np.full) : expm1f(-integ / tau_rc);
  v = v - (j - v) * e;
  rf = fmaxf(rf - dt, 0.0f);
  float out = 0.0f;
  if (v > 1.0f) {
    // time since the threshold crossing, from the overshoot
    float since = 0.0f;
    const float drive = j - 1.0f;
    if (drive > 0.0f) {
      const float q = (v - 1.0f) / drive;
      since = q >= 1.0f ? integ : fminf(-tau_rc * log1pf(-q), integ);
    }
    v = 0.0f;
    rf = tau_ref - since;
    out = amp / dt;
  } else {
    v = fmaxf(v, 0.0f);
  }
  st[vv] = v;
  st[rv] = rf;
  st[at(S, rowof(s, r), b)] = out;
}

__device__ __forceinline__ void lif_rate_item(float* st, const Strides& S, int64_t r, int64_t b,
                                              const Opnd& J, const Opnd& s, const NeuronParams& np) {
  const float tau_rc = np.tau_rc_r ? np.tau_rc_r[r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? np.tau_ref_r[r] : np.tau_ref;
  const float amp = np.amp_r ? np.amp_r[r] : np.amp;
  const float j = st[at(S, rowof(J, r), b)];
  float out = 0.0f;
  if (j > 1.0f) out = amp / (tau_ref + tau_rc * log1pf(1.0f / (j - 1.0f)));
  st[at(S, rowof(s, r), b)] = out;
}

__device__ __forceinline__ void lowpass_item(float* st, const Strides& S, int64_t r, int64_t b,
                                             const Opnd& y, const Opnd& v, const FilterParams& fp) {
  const float a = fp.a_r ? fp.a_r[r] : fp.a;
  const float c = fp.b_r ? fp.b_r[r] : fp.b;
  const int64_t yi = at(S, rowof(y, r), b);
  st[yi] = a * st[yi] + c * st[at(S, rowof(v, r), b)];
}

__device__ __forceinline__ float src_val(const float* base, const Strides& S, int bcast, int64_t row,
                                         int64_t b) {
  return bcast ? base[row] : base[at(S, row, b)];
}

// dst (+)= sum of src entries of unique destination u (ptr == null: one entry)
__device__ __forceinline__ void copy_inc_item(float* st, const Strides& S, int64_t u, int64_t b,
                                              const Opnd& dst, const float* src_base, const Opnd& src,
                                              int bcast, const int32_t* ptr) {
  const int64_t di = at(S, rowof(dst, u), b);
  float acc = st[di];
  if (ptr) {
    for (int32_t e = ptr[u]; e < ptr[u + 1]; ++e) acc += src_val(src_base, S, bcast, rowof(src, e), b);
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
    for (int32_t e = ptr[u]; e < ptr[u + 1]; ++e) acc += a_base[rowof(a, e)] * x_base[at(S, rowof(x, e), b)];
  } else {
    acc += a_base[rowof(a, u)] * x_base[at(S, rowof(x, u), b)];
  }
  st[di] = acc;
}

// one output row m of op `op` for batch b: dst[m] += W[m, :] . x
__device__ __forceinline__ void dot_row_item(float* st, const Strides& S, int64_t op, int32_t m, int64_t b,
                                             int32_t K, const float* W, const int32_t* w_row,
                                             const int32_t* x_row, const int32_t* d_row) {
  const float* w = W + ((int64_t)w_row[op] + m) * K;
  const int64_t x0 = x_row[op];
  float acc = 0.0f;
  for (int32_t k = 0; k < K; ++k) acc += w[k] * st[at(S, x0 + k, b)];
  st[at(S, (int64_t)d_row[op] + m, b)] += acc;
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

// node output <- feed staging [step][feed_rows][B] at the run-relative step ctr[1]
__global__ void k_feed(float* st, Strides S, int32_t B, int64_t rows, Opnd dst, const int32_t* feed_row,
                       const float* stage, int32_t feed_rows, const int64_t* ctr) {
  GRID_ITEM(rows * B);
  const int64_t t = ctr[1];
  st[at(S, rowof(dst, _r), _b)] = stage[(t * feed_rows + feed_row[_r]) * B + _b];
}

// probe buffer [step][probe_rows][B] at the absolute step ctr[0]
__global__ void k_probe(const float* st, Strides S, int32_t B, int32_t rows, const int32_t* src, float* buf,
                        const int64_t* ctr) {
  GRID_ITEM((int64_t)rows * B);
  buf[(ctr[0] * rows + _r) * B + _b] = st[at(S, src[_r], _b)];
}

__global__ void k_advance(int64_t* ctr) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctr[0] += 1;
    ctr[1] += 1;
  }
}

__global__ void k_set_ctr(int64_t* ctr, int64_t c0, int64_t c1) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctr[0] = c0;
    ctr[1] = c1;
  }
}

// feed [B][T][size] -> staging [T][feed_rows][B] rows [row0, row0+size)
#define GRID_FLAT(n)                                                        \
  const int64_t _i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;        \
  if (_i >= (n)) return;

__global__ void k_stage_feed(const float* src, int32_t B, int64_t T, int32_t size, float* stage,
                             int32_t feed_rows, int32_t row0) {
  GRID_FLAT((int64_t)B * T * size);
  const int64_t j = _i % size;
  const int64_t t = (_i / size) % T;
  const int64_t b = _i / (size * T);
  stage[(t * feed_rows + row0 + j) * B + b] = src[_i];
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

// ----------------------------------------------------- persistent interpreter
// A merged group as the persistent kernel sees it (device-resident array).
struct GroupDesc {
  int32_t type;
  int32_t M, K;
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
};

struct PersistentProgram {
  GroupDesc* groups;     // device array
  int32_t n_groups;
};

// Every group of every step for one batch column per workgroup; groups are
// separated by workgroup barriers (operators inside a group are independent by
// construction, and groups run in plan order).  Probes record after each step.
__global__ void __launch_bounds__(1024)
k_persistent(float* st, Strides S, int32_t B, const GroupDesc* groups, int32_t ng, int64_t n_steps, float dt,
             const float* stage, int32_t feed_rows, const int32_t* probe_src, int32_t probe_rows,
             float* probe_buf, int64_t t0) {
  const int64_t b = blockIdx.x;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int lane = tid % warpSize, wave = tid / warpSize, nwaves = nt / warpSize;
  for (int64_t k = 0; k < n_steps; ++k) {
    for (int32_t g = 0; g < ng; ++g) {
      const GroupDesc& G = groups[g];
      const int64_t rows = G.rows;
      switch (G.type) {
        case ms::OP_FEED:
          for (int64_t r = tid; r < rows; r += nt)
            st[at(S, rowof(G.dst, r), b)] = stage[(k * feed_rows + G.feed_row[r]) * B + b];
          break;
        case ms::OP_RESET:
          for (int64_t r = tid; r < rows; r += nt) st[at(S, rowof(G.dst, r), b)] = G.values ? G.values[r] : 0.0f;
          break;
        case ms::OP_COPY:
          for (int64_t r = tid; r < rows; r += nt)
            st[at(S, rowof(G.dst, r), b)] = src_val(G.src_base, S, G.bcast, rowof(G.src, r), b);
          break;
        case ms::OP_COPY_INC:
          for (int64_t r = tid; r < rows; r += nt) copy_inc_item(st, S, r, b, G.dst, G.src_base, G.src, G.bcast, G.ptr);
          break;
        case ms::OP_ELEM_INC:
          for (int64_t r = tid; r < rows; r += nt)
            elem_inc_item(st, S, r, b, G.dst, G.a_base, G.a, G.src_base, G.src, G.ptr);
          break;
        case ms::OP_DOT_INC: {
          const uint32_t total = (uint32_t)(rows * G.M);
          const uint32_t M = (uint32_t)G.M;
          if (G.K >= 32) {
            for (uint32_t t = wave; t < total; t += nwaves) {
              const uint32_t op = t / M;
              const int32_t m = (int32_t)(t - op * M);
              const float* w = G.a_base + ((int64_t)G.w_row[op] + m) * G.K;
              const int64_t x0 = G.x_row[op];
              float acc = 0.0f;
              for (int32_t kk = lane; kk < G.K; kk += warpSize) acc += w[kk] * st[at(S, x0 + kk, b)];
              for (int off = warpSize / 2; off > 0; off >>= 1) acc += __shfl_down(acc, off);
              if (lane == 0) st[at(S, (int64_t)G.d_row[op] + m, b)] += acc;
            }
          } else {
            for (uint32_t t = tid; t < total; t += nt) {
              const uint32_t op = t / M;
              dot_row_item(st, S, op, (int32_t)(t - op * M), b, G.K, G.a_base, G.w_row, G.x_row, G.d_row);
            }
          }
          break;
        }
        case ms::OP_LIF:
          for (int64_t r = tid; r < rows; r += nt) lif_item(st, S, r, b, G.src, G.dst, G.V, G.ref, G.np, dt);
          break;
        case ms::OP_LIF_RATE:
          for (int64_t r = tid; r < rows; r += nt) lif_rate_item(st, S, r, b, G.src, G.dst, G.np);
          break;
        case ms::OP_LOWPASS:
          for (int64_t r = tid; r < rows; r += nt) lowpass_item(st, S, r, b, G.dst, G.src, G.fp);
          break;
        default: break;
      }
      __syncthreads();
    }
    for (int32_t r = tid; r < probe_rows; r += nt)
      probe_buf[((t0 + k) * probe_rows + r) * B + b] = st[at(S, probe_src[r], b)];
    __syncthreads();
  }
}
