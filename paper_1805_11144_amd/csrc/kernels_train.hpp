// Gradient kernels of the window driver: training by gradient descent on an
// objective over probe outputs, the gradient taken back through every step of
// the unrolled simulation (paper Sec. 3.2).  Each kernel runs the reverse of
// one merged group over a whole window of steps.
//
// Adjoints live in `ga`, laid out like the versioned signals (element (row,
// block k, column b) at row * vs + k * B + b): block t + 1 of a row holds
// dL/d(the row's value at window step t); block 0, the adjoint of the value
// carried in, is not used.  A group that reads operand x at block t + blk and
// writes its output at block t + 1 adds (d output / d x) * ga[output, t + 1]
// into ga[x, t + blk].  The groups run in the reverse of the forward schedule,
// so every reader of an output has added its share before the output's
// writer runs backwards.  Parameter gradients live in arrays shaped like the
// parameter bases; they sum over every step and batch column and are added
// with atomics (their order, and so their last bits, is not fixed).
#pragma once

#include "kernels_window.hpp"

__device__ __forceinline__ void t_add(float* p, float v, int atomic) {
  if (atomic) atomicAdd(p, v);
  else *p += v;
}

// Sum of v over a workgroup of 256 threads (4 wavefronts); every thread calls
// it; the sum is returned to thread 0.
__device__ __forceinline__ float t_block_sum(float v, float* red4) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_down(v, o, 64);
  __syncthreads();   // red4 may still be read from the previous call
  if (threadIdx.x % 64 == 0) red4[threadIdx.x / 64] = v;
  __syncthreads();
  return threadIdx.x == 0 ? (red4[0] + red4[1]) + (red4[2] + red4[3]) : 0.0f;
}

// Objective of one probe with a target: rows[j] (j < width) are the probed
// window rows, tgt is [B][T][width] for the window's steps, scale = 1 / (B T
// width).  Each element adds 2 scale (value - target) to the adjoint of the
// probed value (atomically: two probes may read one row); each workgroup
// writes its sum of squared differences to part[blockIdx.x].
__global__ void __launch_bounds__(256) k_t_loss(WView w, float* ga, const int32_t* rows, int32_t width,
                                                const float* tgt, float scale, float* part) {
  __shared__ float red[4];
  const int64_t n = (int64_t)w.B * w.T * width;
  float acc = 0.0f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = i % width, t = (i / width) % w.T, b = i / ((int64_t)width * w.T);
    const int64_t e = (int64_t)G(rows)[j] * w.vs + (t + 1) * w.B + b;
    const float d = w.va[e] - G(tgt)[i];
    acc = fmaf(d, d, acc);
    atomicAdd(&ga[e], 2.0f * scale * d);
  }
  const float s = t_block_sum(acc, red);
  if (threadIdx.x == 0) part[blockIdx.x] = s;
}

// Reverse of COPY (dst = x), COPY_INC (dst += x) and ELEMENTWISE_INC
// (dst += a (.) x), entries grouped by unique destination as in the forward
// kernels: for destination u = blockIdx.x, each entry e and the columns of
// chunk blockIdx.y, with g = ga[dst u],
//   ga[x e] += a g      (x batched, wanted)   or  dW[x e] += sum a g   (x a parameter, trained)
//   ga[a e] += x g      (a batched, wanted)   or  dW[a e] += sum x g   (a a parameter, trained)
// (a = 1 for the copies).  Batched adjoints are added atomically when two
// entries share a row.
struct TScatter {
  Opnd dst, x, a;
  const int32_t* ptr;          // CSR over unique destinations, or null (entry e = destination u)
  const float* xp;             // x's parameter base (x a parameter), else null
  float* gxp;                  // its gradient
  const float* ap;             // a's parameter base (a a parameter), else null
  float* gap;
  int32_t a_kind;              // 0 none (a = 1), 1 parameter, 2 batched
  int32_t xblk, ablk;
  int32_t want_x, want_a;      // adjoint or gradient of x / a wanted
  int32_t atomic;
};

__global__ void __launch_bounds__(256) k_t_scatter(WView w, float* ga, TScatter S, int64_t chunk) {
  __shared__ float red[4];
  const int64_t u = blockIdx.x;
  const int64_t N = (int64_t)w.T * w.B;
  const int64_t c0 = (int64_t)blockIdx.y * chunk, c1 = min(N, c0 + chunk);
  const int64_t gd = rowof(S.dst, u) * w.vs + w.B;
  const int32_t e0 = S.ptr ? G(S.ptr)[u] : (int32_t)u, e1 = S.ptr ? G(S.ptr)[u + 1] : (int32_t)u + 1;
  const bool xpar = S.xp != nullptr;
  for (int32_t e = e0; e < e1; ++e) {
    const int64_t xr = rowof(S.x, e);
    const int64_t ar = S.a_kind ? rowof(S.a, e) : 0;
    const float xv0 = xpar ? G(S.xp)[xr] : 0.0f;
    const float av0 = S.a_kind == 1 ? G(S.ap)[ar] : 1.0f;
    const int64_t xo = xr * w.vs + (int64_t)S.xblk * w.B, ao = ar * w.vs + (int64_t)S.ablk * w.B;
    float sx = 0.0f, sa = 0.0f;
    for (int64_t c = c0 + threadIdx.x; c < c1; c += blockDim.x) {
      const float g = ga[gd + c];
      const float av = S.a_kind == 2 ? w.va[ao + c] : av0;
      if (S.want_x) {
        if (xpar) sx = fmaf(av, g, sx);
        else t_add(&ga[xo + c], av * g, S.atomic);
      }
      if (S.want_a) {
        const float xv = xpar ? xv0 : w.va[xo + c];
        if (S.a_kind == 1) sa = fmaf(xv, g, sa);
        else t_add(&ga[ao + c], xv * g, S.atomic);
      }
    }
    if (S.want_x && xpar) {
      const float t = t_block_sum(sx, red);
      if (threadIdx.x == 0) atomicAdd(&S.gxp[xr], t);
    }
    if (S.want_a && S.a_kind == 1) {
      const float t = t_block_sum(sa, red);
      if (threadIdx.x == 0) atomicAdd(&S.gap[ar], t);
    }
  }
}

// Reverse of a rate neuron s = amplitude r(J) at every (row, step, column):
// ga[J] += r'(J) ga[s].  LIF rate: r = 1 / (tau_ref + tau_rc log(1 + 1/(J-1)))
// above J = 1, so r' = tau_rc r^2 / (J (J - 1)); 0 for J <= 1.  Soft LIF rate
// (J - 1 smoothed into rho): r' = tau_rc r^2 (rho'/rho) / (1 + rho).  ReLU: 1
// above J = 0, else 0.  J rows are distinct within a group.
__global__ void k_t_rate(WView w, float* ga, int64_t rows, Opnd J, Opnd s, NeuronParams np, int jblk) {
  W_ITEM(rows);
  const float tau_rc = np.tau_rc_r ? G(np.tau_rc_r)[_r] : np.tau_rc;
  const float tau_ref = np.tau_ref_r ? G(np.tau_ref_r)[_r] : np.tau_ref;
  const float amp = np.amp_r ? G(np.amp_r)[_r] : np.amp;
  const int64_t jo = vat(w, rowof(J, _r), (int64_t)jblk * w.B + _c);
  const float g = ga[vat(w, rowof(s, _r), w.B + _c)];
  const float j = w.va[jo];
  float d = 0.0f;
  if (np.relu) {
    d = j > 0.0f ? amp : 0.0f;
  } else if (np.sigma > 0.0f) {
    float dl, rho;
    const float r = soft_lif_rate(j, tau_rc, tau_ref, np.sigma_r ? G(np.sigma_r)[_r] : np.sigma, &dl, &rho);
    d = amp * tau_rc * r * r * dl / (1.0f + rho);
  } else if (j > 1.0f) {
    const float r = 1.0f / (tau_ref + tau_rc * log1pf(1.0f / (j - 1.0f)));
    d = amp * tau_rc * r * r / (j * (j - 1.0f));
  }
  ga[jo] += d * g;
}

// Reverse of the lowpass y(t) = a y(t - 1) + b x(t) through the window, one
// work item per (row, column), steps in reverse: mu(t) = ga[y, t + 1] +
// a mu(t + 1) is dL/dy(t) with every later step's dependence included, and
// x(t) receives b mu(t).
__global__ void k_t_lowpass(WView w, float* ga, int64_t rows, Opnd y, Opnd x, FilterParams fp, int xblk,
                            int atomic) {
  W_ROWCOL(rows);
  const float a = fp.a_r ? G(fp.a_r)[_r] : fp.a;
  const float c = fp.b_r ? G(fp.b_r)[_r] : fp.b;
  const int64_t yr = rowof(y, _r) * w.vs + _b;
  const int64_t xr = rowof(x, _r) * w.vs + (int64_t)xblk * w.B + _b;
  float mu = 0.0f;
  for (int32_t t = w.T - 1; t >= 0; --t) {
    mu = fmaf(a, mu, ga[yr + (int64_t)(t + 1) * w.B]);
    t_add(&ga[xr + (int64_t)t * w.B], c * mu, atomic);
  }
}

// Each op's [M][K] weight block transposed: Wt[(op K + k) M + m] = W[(w_row[op] + m) K + k]
// (the products that carry adjoints back to the inputs multiply by W^T).
__global__ void k_t_transpose(const float* W, const int32_t* w_row, int32_t M, int32_t K, int64_t n, float* Wt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t mk = (int64_t)M * K;
  const int64_t op = i / mk, r = i - op * mk, k = r / M, m = r - k * M;
  Wt[i] = G(W)[((int64_t)G(w_row)[op] + m) * K + k];
}

// Weight gradients of a merged DotInc group, dW[op][m][k] = sum over the
// window's (step, column) pairs c of ga[d_row + m, c] x[x_row + k, c]: a
// product whose reduction runs along the contiguous axis of both operands.
// Workgroup tile 128 (m) x 128 (k); the columns are split into nsplit chunks
// of cchunk (a multiple of 16) so that the launch fills the chip; each chunk's
// tile is added to dW with atomics.  Columns in slices of 16, double-buffered
// in LDS, the next slice fetched into registers (float4 along the columns)
// while the current one is multiplied; each wavefront owns a 64 x 64 quarter
// as 2 x 2 blocks of v_mfma_f32_32x32x2f32.  Needs B % 4 == 0.  Workgroups
// are numbered for the XCDs as in the forward products: a contiguous run of
// (m tile fastest, k tile, op, chunk) per XCD, so tiles that share a column
// chunk read it from one L2.
constexpr int kDwM = 128, kDwK = 128, kDwC = 16;

__global__ void __launch_bounds__(256, 2) k_t_dw(WView w, const float* ga, int32_t M, int32_t K, int32_t mtiles,
                                              int32_t ktiles, int32_t nops, int32_t nsplit, int64_t cchunk,
                                              float* gW, const int32_t* w_row, const int32_t* x_row,
                                              const int32_t* d_row, int xblk) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  __shared__ float As[2][kDwC][kDwM + 4];
  __shared__ float Bs[2][kDwC][kDwK + 4];
  const uint32_t total = (uint32_t)mtiles * ktiles * nops * nsplit, chunk8 = (total + 7) / 8;
  const uint32_t L = (blockIdx.x % 8) * chunk8 + blockIdx.x / 8;
  if (L >= total) return;
  const int mt = (int)(L % mtiles);
  uint32_t rest = L / mtiles;
  const int kt = (int)(rest % ktiles);
  rest /= ktiles;
  const int op = (int)(rest % nops), sp = (int)(rest / nops);
  const int64_t N = (int64_t)w.T * w.B;
  const int64_t cb = (int64_t)sp * cchunk, ce = min(N, cb + cchunk);
  if (cb >= ce) return;
  const int64_t m0 = (int64_t)mt * kDwM, k0 = (int64_t)kt * kDwK;
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  const int wm = wave / 2, wn = wave % 2;
  const float* Y = ga + (int64_t)G(d_row)[op] * w.vs + w.B;
  const float* X = w.va + (int64_t)G(x_row)[op] * w.vs + (int64_t)xblk * w.B;
  f4v ra[2], rb[2];
  // 128 rows x 16 columns of each operand: 512 float4, two per thread
  auto fetch = [&](int64_t c0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + q * 256;
      const int rr = idx / 4, c4 = idx % 4;
      const int64_t c = c0 + 4 * c4;
      f4v a = {0.0f, 0.0f, 0.0f, 0.0f}, b = {0.0f, 0.0f, 0.0f, 0.0f};
      if (c < ce) {   // c and ce are multiples of 4
        if (m0 + rr < M) a = *(const f4v*)(Y + (m0 + rr) * w.vs + c);
        if (k0 + rr < K) b = *(const f4v*)(X + (k0 + rr) * w.vs + c);
      }
      ra[q] = a;
      rb[q] = b;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + q * 256;
      const int rr = idx / 4, c4 = idx % 4;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        As[buf][4 * c4 + e][rr] = ra[q][e];
        Bs[buf][4 * c4 + e][rr] = rb[q][e];
      }
    }
  };
  mfma_f16x acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
  fetch(cb);
  stash(0);
  __syncthreads();
  int buf = 0;
  for (int64_t c0 = cb; c0 < ce; c0 += kDwC) {
    const bool more = c0 + kDwC < ce;
    if (more) fetch(c0 + kDwC);
#pragma unroll
    for (int kk = 0; kk < kDwC; kk += 2) {
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
  float* dW = gW + (int64_t)G(w_row)[op] * K;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t m = m0 + wm * 64 + i * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
        const int64_t k = k0 + wn * 64 + j * 32 + lane % 32;
        if (m < M && k < K) atomicAdd(&dW[m * K + k], acc[i][j][v]);
      }
}

// Weight gradients of skinny blocks, one side (M or K) at most kSkM: each
// wavefront takes one row of the long side and cchunk columns; its lanes walk
// the columns (coalesced), each keeping partial sums against every row of the
// short side (those rows are shared by all wavefronts and stay in cache); the
// wavefront then sums each partial over its lanes and adds it atomically.
// long_m != 0: the long side is M (rows of the output adjoint).
__global__ void __launch_bounds__(256) k_t_dw_skinny(WView w, const float* ga, int32_t M, int32_t K, int64_t nwaves,
                                                     int32_t nch, int64_t cchunk, float* gW, const int32_t* w_row,
                                                     const int32_t* x_row, const int32_t* d_row, int xblk,
                                                     int long_m) {
  const int64_t wv = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (wv >= nwaves) return;   // whole wavefronts leave together
  const int32_t L = long_m ? M : K, S = long_m ? K : M;
  const int64_t ch = wv % nch, rest = wv / nch;
  const int64_t l = rest % L, op = rest / L;
  const int64_t N = (int64_t)w.T * w.B;
  const int64_t c0 = ch * cchunk, c1 = min(N, c0 + cchunk);
  const float* Y = ga + (int64_t)G(d_row)[op] * w.vs + w.B;
  const float* X = w.va + (int64_t)G(x_row)[op] * w.vs + (int64_t)xblk * w.B;
  const float* lrow = long_m ? Y + l * w.vs : X + l * w.vs;
  const float* srow = long_m ? X : Y;
  float acc[kSkM];
#pragma unroll
  for (int s = 0; s < kSkM; ++s) acc[s] = 0.0f;
  for (int64_t c = c0 + lane; c < c1; c += 64) {
    const float lv = lrow[c];
#pragma unroll
    for (int s = 0; s < kSkM; ++s)
      if (s < S) acc[s] = fmaf(lv, srow[(int64_t)s * w.vs + c], acc[s]);
  }
  float* dW = gW + (int64_t)G(w_row)[op] * K;
#pragma unroll
  for (int s = 0; s < kSkM; ++s) {
    if (s >= S) break;
    float v = acc[s];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) atomicAdd(&dW[long_m ? l * K + s : (int64_t)s * K + l], v);
  }
}

// The same gradients for small blocks (M or K below a tile, or B % 4 != 0):
// one work item per (op, m, k) and column chunk blockIdx.y of cchunk columns.
__global__ void k_t_dw_small(WView w, const float* ga, int32_t M, int32_t K, int64_t nout, int64_t cchunk, float* gW,
                             const int32_t* w_row, const int32_t* x_row, const int32_t* d_row, int xblk) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nout) return;
  const int64_t mk = (int64_t)M * K;
  const int64_t op = i / mk, r = i - op * mk, m = r / K, k = r - m * K;
  const int64_t N = (int64_t)w.T * w.B;
  const int64_t c0 = (int64_t)blockIdx.y * cchunk, c1 = min(N, c0 + cchunk);
  const float* y = ga + ((int64_t)G(d_row)[op] + m) * w.vs + w.B;
  const float* x = w.va + ((int64_t)G(x_row)[op] + k) * w.vs + (int64_t)xblk * w.B;
  float acc = 0.0f;
  for (int64_t c = c0; c < c1; ++c) acc = fmaf(y[c], x[c], acc);
  atomicAdd(&gW[((int64_t)G(w_row)[op] + m) * K + k], acc);
}

// Gradient descent on one parameter range: p <- p - lr g.
__global__ void k_t_sgd(float* p, const float* g, int64_t n, float lr) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = fmaf(-lr, g[i], p[i]);
}
