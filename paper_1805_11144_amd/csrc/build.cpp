// Build step in double precision: gains, biases and least-squares decoders.
//
// The paper defers the neuron and decoder definitions to Nengo (Sec. 2.1.3,
// Sec. 3.2 "least squares optimization"); they are stated here from the
// LIF membrane equation dV/dt = (J - V) / tau_rc (threshold 1, reset 0,
// refractory tau_ref):
//   rate r(J) = 1 / (tau_ref + tau_rc * log1p(1 / (J - 1)))  for J > 1, else 0
//   gain/bias put the firing onset at the intercept and the maximum rate at x = 1
//   decoders solve (A^T A + M sigma^2 I) D = A^T f(X), sigma = 0.1 max(A),
//   A = amplitude * r(gain e.x + bias) on the ensemble's eval points, by Cholesky.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <thread>

#include "host.hpp"

namespace ms {

namespace {

double lif_rate(double J, double tau_rc, double tau_ref) {
  if (!(J > 1.0)) return 0.0;
  return 1.0 / (tau_ref + tau_rc * std::log1p(1.0 / (J - 1.0)));
}

// Smoothed LIF rate: max(J - 1, 0) replaced by rho = sigma log(1 + exp(x)),
// x = (J - 1) / sigma; log(1 + 1/rho) directly for x >= -30, and below (where
// softplus(x) = exp(x) to a relative exp(x) / 2) as log1p(rho) - log(rho) with
// log(rho) = log(sigma) + x.
double soft_lif_rate(double J, double tau_rc, double tau_ref, double sigma) {
  const double x = (J - 1.0) / sigma;
  double q;
  if (x < -30.0) {
    q = std::log1p(sigma * std::exp(x)) - (std::log(sigma) + x);
  } else {
    const double sp = x > 30.0 ? x + std::log1p(std::exp(-x)) : std::log1p(std::exp(x));
    q = std::log1p(1.0 / (sigma * sp));
  }
  return 1.0 / (tau_ref + tau_rc * q);
}

// rate curve of the ensemble's neuron type (spiking LIF decodes from its rates)
double rate_of(const EnsembleDesc& e, double J) {
  if (e.neuron_type == MS_NEURON_RELU) return J > 0.0 ? J : 0.0;
  if (e.neuron_type == MS_NEURON_SOFTLIF_RATE) return soft_lif_rate(J, e.tau_rc, e.tau_ref, e.sigma);
  return lif_rate(J, e.tau_rc, e.tau_ref);
}

// G = A^T A (lower triangle filled, then mirrored), A is [M][n] row-major.
void gram(const std::vector<double>& A, int M, int n, std::vector<double>& G) {
  // transpose so every entry is a contiguous dot product of length M
  std::vector<double> At((size_t)n * M);
  for (int m = 0; m < M; ++m)
    for (int i = 0; i < n; ++i) At[(size_t)i * M + m] = A[(size_t)m * n + i];
  G.assign((size_t)n * n, 0.0);
  int i = 0;
  for (; i + 1 < n; i += 2) {
    const double* a0 = &At[(size_t)i * M];
    const double* a1 = a0 + M;
    // i is even, so j (even) reaches i and the 2x2 block covers the diagonal
    for (int j = 0; j <= i; j += 2) {
      const double* b0 = &At[(size_t)j * M];
      const double* b1 = b0 + M;
      double s00 = 0, s01 = 0, s10 = 0, s11 = 0;
      for (int m = 0; m < M; ++m) {
        s00 += a0[m] * b0[m]; s01 += a0[m] * b1[m];
        s10 += a1[m] * b0[m]; s11 += a1[m] * b1[m];
      }
      G[(size_t)i * n + j] = s00; G[(size_t)i * n + j + 1] = s01;
      G[(size_t)(i + 1) * n + j] = s10; G[(size_t)(i + 1) * n + j + 1] = s11;
    }
  }
  for (; i < n; ++i) {
    const double* a0 = &At[(size_t)i * M];
    for (int j = 0; j <= i; ++j) {
      const double* b0 = &At[(size_t)j * M];
      double s = 0;
      for (int m = 0; m < M; ++m) s += a0[m] * b0[m];
      G[(size_t)i * n + j] = s;
    }
  }
  for (int r = 0; r < n; ++r)
    for (int c = r + 1; c < n; ++c) G[(size_t)r * n + c] = G[(size_t)c * n + r];
}

// In-place Cholesky G = L L^T (lower).  Returns false if not positive definite.
bool cholesky(std::vector<double>& G, int n) {
  for (int j = 0; j < n; ++j) {
    double* gj = &G[(size_t)j * n];
    double s = gj[j];
    for (int k = 0; k < j; ++k) s -= gj[k] * gj[k];
    if (!(s > 0.0)) return false;
    double d = std::sqrt(s);
    gj[j] = d;
    for (int i = j + 1; i < n; ++i) {
      double* gi = &G[(size_t)i * n];
      double t = gi[j];
      for (int k = 0; k < j; ++k) t -= gi[k] * gj[k];
      gi[j] = t / d;
    }
  }
  return true;
}

std::vector<double> solve_decoders(const EnsembleDesc& e, const std::vector<double>& gain,
                                   const std::vector<double>& bias, int32_t fn, bool* ok) {
  const int n = e.n, d = e.d, M = e.n_eval;
  std::vector<double> A((size_t)M * n);
  double amax = 0.0;
  for (int m = 0; m < M; ++m) {
    const double* x = &e.eval_points[(size_t)m * d];
    for (int i = 0; i < n; ++i) {
      const double* en = &e.encoders[(size_t)i * d];
      double dot = 0.0;
      for (int k = 0; k < d; ++k) dot += en[k] * x[k];
      double v = e.amplitude * rate_of(e, gain[i] * dot + bias[i]);
      A[(size_t)m * n + i] = v;
      amax = std::max(amax, v);
    }
  }
  const int dout = function_size(fn, d);
  std::vector<double> Y((size_t)M * dout);
  for (int m = 0; m < M; ++m) {
    const double* x = &e.eval_points[(size_t)m * d];
    if (fn == MS_FN_IDENTITY)
      for (int k = 0; k < d; ++k) Y[(size_t)m * dout + k] = x[k];
    else
      Y[m] = x[0] * x[1];
  }
  std::vector<double> G;
  gram(A, M, n, G);
  const double sigma = 0.1 * amax;
  const double lam = (double)M * sigma * sigma;
  for (int i = 0; i < n; ++i) G[(size_t)i * n + i] += lam;
  // rhs = A^T Y  [n][dout]
  std::vector<double> R((size_t)n * dout, 0.0);
  for (int m = 0; m < M; ++m)
    for (int i = 0; i < n; ++i) {
      const double a = A[(size_t)m * n + i];
      if (a == 0.0) continue;
      for (int k = 0; k < dout; ++k) R[(size_t)i * dout + k] += a * Y[(size_t)m * dout + k];
    }
  if (!cholesky(G, n)) { *ok = false; return {}; }
  // forward: L z = R ; backward: L^T D = z
  for (int k = 0; k < dout; ++k) {
    for (int i = 0; i < n; ++i) {
      double t = R[(size_t)i * dout + k];
      const double* gi = &G[(size_t)i * n];
      for (int j = 0; j < i; ++j) t -= gi[j] * R[(size_t)j * dout + k];
      R[(size_t)i * dout + k] = t / gi[i];
    }
    for (int i = n - 1; i >= 0; --i) {
      double t = R[(size_t)i * dout + k];
      for (int j = i + 1; j < n; ++j) t -= G[(size_t)j * n + i] * R[(size_t)j * dout + k];
      R[(size_t)i * dout + k] = t / G[(size_t)i * n + i];
    }
  }
  *ok = true;
  return R;
}

}  // namespace

int32_t function_size(int32_t fn, int32_t dims) { return fn == MS_FN_PRODUCT ? 1 : dims; }

Built build_params(const Model& m) {
  Built b;
  const size_t ne = m.ens.size();
  b.gain.resize(ne);
  b.bias.resize(ne);
  for (size_t i = 0; i < ne; ++i) {
    const EnsembleDesc& e = m.ens[i];
    if (!e.gains.empty()) {
      b.gain[i] = e.gains;
      b.bias[i] = e.biases;
      continue;
    }
    b.gain[i].resize(e.n);
    b.bias[i].resize(e.n);
    for (int k = 0; k < e.n && e.neuron_type == MS_NEURON_RELU; ++k) {
      // rectified linear: J = 0 at the intercept, J = max_rate at x = 1
      const double g = e.max_rates[k] / (1.0 - e.intercepts[k]);
      b.gain[i][k] = g;
      b.bias[i][k] = -g * e.intercepts[k];
    }
    for (int k = 0; k < e.n && e.neuron_type != MS_NEURON_RELU; ++k) {
      const double jmax = 1.0 / -std::expm1((e.tau_ref - 1.0 / e.max_rates[k]) / e.tau_rc);
      const double g = (jmax - 1.0) / (1.0 - e.intercepts[k]);
      b.gain[i][k] = g;
      b.bias[i][k] = 1.0 - g * e.intercepts[k];
    }
  }
  // decoders needed: connections from decoded ensembles (without explicit
  // decoders) and decoded probes; shared per (ensemble, function)
  std::vector<std::pair<int32_t, int32_t>> need;
  auto want = [&](int32_t e, int32_t fn) {
    auto key = std::make_pair(e, fn);
    if (std::find(need.begin(), need.end(), key) == need.end()) need.push_back(key);
  };
  for (const ConnDesc& c : m.conns)
    if (c.pre_kind == MS_REF_ENS && c.decoders.empty()) want(c.pre_id, c.function);
  for (const ProbeDesc& p : m.probes)
    if (p.kind == MS_REF_ENS) want(p.id, MS_FN_IDENTITY);
  std::vector<std::vector<double>> out(need.size());
  std::vector<char> ok(need.size(), 1);
  std::atomic<size_t> next{0};
  auto worker = [&]() {
    for (;;) {
      size_t k = next.fetch_add(1);
      if (k >= need.size()) break;
      const auto& key = need[k];
      bool good = true;
      out[k] = solve_decoders(m.ens[key.first], b.gain[key.first], b.bias[key.first],
                              key.second, &good);
      ok[k] = good;
    }
  };
  unsigned nt = std::max(1u, std::thread::hardware_concurrency());
  nt = std::min<unsigned>(nt, (unsigned)std::max<size_t>(1, need.size()));
  std::vector<std::thread> pool;
  for (unsigned t = 1; t < nt; ++t) pool.emplace_back(worker);
  worker();
  for (auto& t : pool) t.join();
  for (size_t k = 0; k < need.size(); ++k) {
    if (!ok[k])
      fail(MS_E_NUMERIC, "decoder solve failed for ensemble " + std::to_string(need[k].first) +
                             " (no active neuron on the eval points?)");
    b.decoders[need[k]] = std::move(out[k]);
  }
  return b;
}

}  // namespace ms
