// Host side of the library: status and error reporting, the pattern
// distribution search (Sec. III-C, Alg. 1), the per-iteration pattern sampler
// (Sec. III-D) and tile bitmaps (Sec. III-B).
//
// This file must be compiled without fast-math: the sampler's inverse CDF is a
// chain of fp64 additions and comparisons whose exact IEEE results every
// implementation of the sampler has to reproduce bit for bit.

#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "ard_internal.hpp"

namespace ard {

static thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

void clear_error() { g_last_error.clear(); }

int check_row_plan(const ard_row_plan* plan, int32_t n, const char* what, bool needs_list) {
  if (plan == nullptr) return ARD_OK;
  if (plan->n != n)
    return fail(ARD_ERR_INVALID_ARG, "%s: plan covers %d neurons, layer has %d", what, plan->n, n);
  if (plan->period < 1 || plan->offset < 0 || plan->offset >= plan->period)
    return fail(ARD_ERR_INVALID_ARG, "%s: invalid pattern (period %d, offset %d)", what,
                plan->period, plan->offset);
  if (plan->kept != kept_count(n, plan->period, plan->offset))
    return fail(ARD_ERR_INVALID_ARG, "%s: kept %d does not match the pattern", what, plan->kept);
  if (needs_list && plan->period > 1 && plan->kept > 0 && plan->d_idx == nullptr)
    return fail(ARD_ERR_INVALID_ARG, "%s: d_idx is NULL (this call reads the kept-index list)", what);
  return ARD_OK;
}

// ---------------------------------------------------------------------------
// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): a Weyl sequence with the
// golden-ratio increment, each state passed through a 64-bit finaliser.
// ---------------------------------------------------------------------------
struct SplitMix64 {
  uint64_t state;
  uint64_t next() {
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  // 53 random bits as a double in [0, 1).
  double uniform() { return static_cast<double>(next() >> 11) * 0x1.0p-53; }
  // Unbiased integer in [0, n): reject draws below 2^64 mod n, then reduce.
  uint64_t below(uint64_t n) {
    const uint64_t threshold = (0 - n) % n;  // == 2^64 mod n
    uint64_t w = next();
    while (w < threshold) w = next();
    return w % n;
  }
};

constexpr int kStreamBits = 24;
constexpr int kIterBits = 40;

static int make_stream(uint64_t seed, uint32_t stream, uint64_t iter, SplitMix64* g) {
  if (stream >= (1u << kStreamBits))
    return fail(ARD_ERR_INVALID_ARG, "stream %u must be < 2^24", stream);
  if (iter >= (1ull << kIterBits))
    return fail(ARD_ERR_INVALID_ARG, "iter must be < 2^40");
  g->state = seed ^ ((static_cast<uint64_t>(stream) << kIterBits) | iter);
  return ARD_OK;
}

// ---------------------------------------------------------------------------
// Alg. 1 pieces. log d_i is taken as v_i - logsumexp(v), which stays finite
// even where exp underflows d_i to zero.
// ---------------------------------------------------------------------------
struct SearchState {
  int n;
  double p, lam1, lam2;
  std::vector<double> pu, d, logd, g;

  void softmax(const std::vector<double>& v) {
    double vmax = v[0];
    for (int i = 1; i < n; ++i) vmax = v[i] > vmax ? v[i] : vmax;
    double z = 0.0;
    for (int i = 0; i < n; ++i) z += std::exp(v[i] - vmax);
    const double lse = vmax + std::log(z);
    for (int i = 0; i < n; ++i) {
      logd[i] = v[i] - lse;
      d[i] = std::exp(logd[i]);
    }
  }
  double mean_rate() const {
    double mu = 0.0;
    for (int i = 0; i < n; ++i) mu += d[i] * pu[i];
    return mu;
  }
  double loss() const {
    const double e_p = (mean_rate() - p) * (mean_rate() - p);
    double e_n = 0.0;
    for (int i = 0; i < n; ++i)
      if (d[i] > 0.0) e_n += d[i] * logd[i];
    return lam1 * e_p + lam2 * e_n / n;
  }
  // g = dL/dd
  void grad_d() {
    const double mu = mean_rate();
    for (int i = 0; i < n; ++i) g[i] = 2.0 * lam1 * (mu - p) * pu[i] + (lam2 / n) * (logd[i] + 1.0);
  }
};

}  // namespace ard

using namespace ard;

extern "C" {

const char* ard_status_string(int status) {
  switch (status) {
    case ARD_OK: return "ARD_OK";
    case ARD_ERR_INVALID_ARG: return "ARD_ERR_INVALID_ARG";
    case ARD_ERR_UNSUPPORTED: return "ARD_ERR_UNSUPPORTED";
    case ARD_ERR_HIP: return "ARD_ERR_HIP";
    case ARD_ERR_NOT_CONVERGED: return "ARD_ERR_NOT_CONVERGED";
    case ARD_ERR_WORKSPACE: return "ARD_ERR_WORKSPACE";
    default: return "ARD_ERR_UNKNOWN";
  }
}

const char* ard_last_error(void) { return g_last_error.c_str(); }

int ard_version(void) { return ARD_VERSION; }

void ard_search_opts_default(ard_search_opts* opts) {
  if (!opts) return;
  opts->n_max = 16;
  opts->mode = ARD_SEARCH_PLAIN;
  opts->lambda1 = 0.99;
  opts->lr = 10.0;
  opts->threshold = 1e-15;
  opts->max_iters = 1000000;
}

int ard_search_distribution(double p, const ard_search_opts* opts_in, double* K_out,
                            ard_search_info* info) {
  clear_error();
  ard_search_opts opts;
  if (opts_in)
    opts = *opts_in;
  else
    ard_search_opts_default(&opts);
  if (!K_out) return fail(ARD_ERR_INVALID_ARG, "K_out is NULL");
  const int n = opts.n_max;
  if (n < 1 || n > (1 << 20)) return fail(ARD_ERR_INVALID_ARG, "n_max %d out of range", n);
  if (opts.mode != ARD_SEARCH_PLAIN && opts.mode != ARD_SEARCH_MIRROR)
    return fail(ARD_ERR_INVALID_ARG, "unknown search mode %d", opts.mode);
  if (!(opts.lambda1 > 0.0 && opts.lambda1 < 1.0))
    return fail(ARD_ERR_INVALID_ARG, "lambda1 must lie in (0, 1)");
  if (!(opts.lr > 0.0)) return fail(ARD_ERR_INVALID_ARG, "lr must be positive");
  if (!(opts.threshold >= 0.0)) return fail(ARD_ERR_INVALID_ARG, "threshold must be >= 0");
  if (opts.max_iters < 1) return fail(ARD_ERR_INVALID_ARG, "max_iters must be >= 1");
  const double p_max = static_cast<double>(n - 1) / n;
  if (!(p >= 0.0) || (p > 0.0 && !(p < p_max)))
    return fail(ARD_ERR_INVALID_ARG, "rate %g unreachable with periods 1..%d (need 0 <= p < %g)",
                p, n, p_max);

  SearchState s;
  s.n = n;
  s.p = p;
  s.lam1 = opts.lambda1;
  s.lam2 = 1.0 - opts.lambda1;
  s.pu.resize(n);
  s.d.assign(n, 0.0);
  s.logd.assign(n, 0.0);
  s.g.assign(n, 0.0);
  for (int i = 0; i < n; ++i) s.pu[i] = static_cast<double>(i) / (i + 1);  // (i'-1)/i', i' = i+1

  if (p == 0.0) {  // no dropout: every iteration uses period 1
    for (int i = 0; i < n; ++i) K_out[i] = i == 0 ? 1.0 : 0.0;
    if (info) {
      info->iters = 0;
      info->loss = 0.0;
      info->p_global = 0.0;
      info->kkt_residual = 0.0;
      info->converged = 1;
      info->reserved = 0;
    }
    return ARD_OK;
  }

  std::vector<double> v(n, 0.0);
  double prev = 0.0, cur = 0.0;
  int64_t it = 0;
  bool converged = false;
  for (it = 1; it <= opts.max_iters; ++it) {
    s.softmax(v);
    cur = s.loss();
    if (it > 1 && std::fabs(cur - prev) < opts.threshold) {
      converged = true;
      break;
    }
    prev = cur;
    s.grad_d();
    if (opts.mode == ARD_SEARCH_PLAIN) {
      // chain rule through softmax: dL/dv_j = d_j (g_j - sum_i d_i g_i)
      double dg = 0.0;
      for (int i = 0; i < n; ++i) dg += s.d[i] * s.g[i];
      for (int i = 0; i < n; ++i) v[i] -= opts.lr * s.d[i] * (s.g[i] - dg);
    } else {
      for (int i = 0; i < n; ++i) v[i] -= opts.lr * s.g[i];
    }
  }
  if (!converged) {
    it = opts.max_iters;
    s.softmax(v);
    cur = s.loss();
  }
  s.grad_d();
  double gmin = s.g[0], gmax = s.g[0];
  for (int i = 1; i < n; ++i) {
    gmin = s.g[i] < gmin ? s.g[i] : gmin;
    gmax = s.g[i] > gmax ? s.g[i] : gmax;
  }
  for (int i = 0; i < n; ++i) K_out[i] = s.d[i];
  if (info) {
    info->iters = it;
    info->loss = cur;
    info->p_global = s.mean_rate();
    info->kkt_residual = gmax - gmin;
    info->converged = converged ? 1 : 0;
    info->reserved = 0;
  }
  if (!converged)
    return fail(ARD_ERR_NOT_CONVERGED, "search did not converge in %lld iterations",
                static_cast<long long>(opts.max_iters));
  return ARD_OK;
}

int ard_sample_row_pattern(const double* K, int32_t n_max, uint64_t seed, uint32_t stream,
                           uint64_t iter, ard_row_pattern* out) {
  clear_error();
  if (!K || !out) return fail(ARD_ERR_INVALID_ARG, "NULL argument");
  if (n_max < 1) return fail(ARD_ERR_INVALID_ARG, "n_max must be >= 1");
  int last_positive = 0;
  for (int i = 0; i < n_max; ++i) {
    if (!(K[i] >= 0.0)) return fail(ARD_ERR_INVALID_ARG, "K[%d] is negative or NaN", i);
    if (K[i] > 0.0) last_positive = i + 1;
  }
  if (last_positive == 0) return fail(ARD_ERR_INVALID_ARG, "K has no positive entry");
  SplitMix64 g;
  int st = make_stream(seed, stream, iter, &g);
  if (st != ARD_OK) return st;
  // inverse CDF over sequential partial sums C_i = C_{i-1} + K_i
  const double u = g.uniform();
  int period = 0;
  double c = 0.0;
  for (int i = 0; i < n_max; ++i) {
    c = c + K[i];
    if (u < c) {
      period = i + 1;
      break;
    }
  }
  if (period == 0) period = last_positive;
  out->period = period;
  out->offset = static_cast<int32_t>(g.below(static_cast<uint64_t>(period)));
  return ARD_OK;
}

int32_t ard_row_kept(int32_t n, int32_t period, int32_t offset) {
  if (n < 0 || period < 1 || offset < 0 || offset >= period) return -1;
  return kept_count(n, period, offset);
}

int ard_tile_bitmap_tdp(int32_t tiles_n, int32_t tiles_k, int32_t period, int32_t offset,
                        uint32_t* bits) {
  clear_error();
  if (!bits) return fail(ARD_ERR_INVALID_ARG, "bits is NULL");
  if (tiles_n < 1 || tiles_k < 1 || static_cast<int64_t>(tiles_n) * tiles_k > (1 << 30))
    return fail(ARD_ERR_INVALID_ARG, "invalid tile grid %d x %d", tiles_n, tiles_k);
  if (period < 1 || offset < 0 || offset >= period)
    return fail(ARD_ERR_INVALID_ARG, "invalid pattern (period %d, offset %d)", period, offset);
  const int64_t total = static_cast<int64_t>(tiles_n) * tiles_k;
  std::memset(bits, 0, sizeof(uint32_t) * ((total + 31) / 32));
  for (int64_t t = offset; t < total; t += period) bits[t / 32] |= 1u << (t % 32);
  return ARD_OK;
}

int ard_tile_bitmap_bernoulli(int32_t tiles_n, int32_t tiles_k, double p, uint64_t seed,
                              uint32_t stream, uint64_t iter, uint32_t* bits) {
  clear_error();
  if (!bits) return fail(ARD_ERR_INVALID_ARG, "bits is NULL");
  if (tiles_n < 1 || tiles_k < 1 || static_cast<int64_t>(tiles_n) * tiles_k > (1 << 30))
    return fail(ARD_ERR_INVALID_ARG, "invalid tile grid %d x %d", tiles_n, tiles_k);
  if (!(p >= 0.0 && p <= 1.0)) return fail(ARD_ERR_INVALID_ARG, "p must lie in [0, 1]");
  SplitMix64 g;
  int st = make_stream(seed, stream, iter, &g);
  if (st != ARD_OK) return st;
  const int64_t total = static_cast<int64_t>(tiles_n) * tiles_k;
  std::memset(bits, 0, sizeof(uint32_t) * ((total + 31) / 32));
  for (int64_t t = 0; t < total; ++t)
    if (g.uniform() >= p) bits[t / 32] |= 1u << (t % 32);
  return ARD_OK;
}

int32_t ard_bitmap_popcount(const uint32_t* bits, int32_t total) {
  if (!bits || total < 0) return -1;
  int32_t c = 0;
  for (int32_t w = 0; w < total / 32; ++w) c += __builtin_popcount(bits[w]);
  if (total % 32) c += __builtin_popcount(bits[total / 32] & ((1u << (total % 32)) - 1u));
  return c;
}

}  // extern "C"
