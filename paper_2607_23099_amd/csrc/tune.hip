// Offline auto-tuning (Sec. IV-A) and the Dirichlet reverse modelling of Alg. 1 (Sec. III-A).
//
// Random numbers come from a counter-based Philox4x32-10 generator (Salmon, Moraes, Dror,
// Shaw, SC'11) keyed by the caller's seed, so every draw is addressed by a counter
// (n, e, sample, tag) and Alg. 1 sees the same random numbers at every bisection step.
// Gamma variates use Marsaglia and Tsang's method (ACM TOMS 2000) for shape alpha + 1 with a
// Box-Muller normal, boosted to shape alpha by U^(1/alpha) in log space, so Dirichlet samples
// never underflow even at alpha = 0.03.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <numeric>
#include <vector>

#include "common.h"

namespace {

struct Philox {
  uint32_t k0, k1;
  explicit Philox(uint64_t seed) : k0((uint32_t)seed), k1((uint32_t)(seed >> 32)) {}
  void block(uint32_t n, uint32_t e, uint32_t s, uint32_t tag, uint32_t out[4]) const {
    uint32_t x0 = n, x1 = e, x2 = s, x3 = tag, a = k0, b = k1;
    for (int r = 0; r < 10; ++r) {
      const uint64_t m0 = (uint64_t)0xD2511F53u * x0;
      const uint64_t m1 = (uint64_t)0xCD9E8D57u * x2;
      const uint32_t n0 = (uint32_t)(m1 >> 32) ^ x1 ^ a;
      const uint32_t n2 = (uint32_t)(m0 >> 32) ^ x3 ^ b;
      x0 = n0;
      x1 = (uint32_t)m1;
      x2 = n2;
      x3 = (uint32_t)m0;
      a += 0x9E3779B9u;
      b += 0xBB67AE85u;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
  }
  // Two uniforms in (0, 1), 53-bit, from one block.
  void uniforms(uint32_t n, uint32_t e, uint32_t s, uint32_t tag, double& u0, double& u1) const {
    uint32_t r[4];
    block(n, e, s, tag, r);
    const double inv = 1.0 / 9007199254740992.0;
    u0 = ((double)(((uint64_t)(r[0] >> 5) << 26) | (r[1] >> 6)) + 0.5) * inv;
    u1 = ((double)(((uint64_t)(r[2] >> 5) << 26) | (r[3] >> 6)) + 0.5) * inv;
  }
};

// log of a Gamma(alpha) variate, draw (e, s).
double log_gamma(const Philox& g, double alpha, uint32_t e, uint32_t s) {
  const double d = alpha + 1.0 - 1.0 / 3.0;
  const double c = 1.0 / std::sqrt(9.0 * d);
  double val = 0.0;
  for (uint32_t i = 0;; ++i) {
    double u1, u2, ua, ub;
    g.uniforms(2 * i, e, s, 0, u1, u2);
    g.uniforms(2 * i + 1, e, s, 0, ua, ub);
    const double z = std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586 * u2);
    double v = 1.0 + c * z;
    if (v <= 0.0) continue;
    v = v * v * v;
    if (std::log(ua) < 0.5 * z * z + d - d * v + d * std::log(v)) {
      val = d * v;
      break;
    }
  }
  double b0, b1;
  g.uniforms(0, e, s, 1, b0, b1);
  return std::log(val) + std::log(b0) / alpha;
}

// log p of one Dirichlet(alpha 1_E) sample.
void dirichlet_logp(const Philox& g, double alpha, int32_t E, uint32_t s, std::vector<double>& lp) {
  lp.resize(E);
  double mx = -INFINITY;
  for (int32_t e = 0; e < E; ++e) {
    lp[e] = log_gamma(g, alpha, (uint32_t)e, s);
    mx = std::max(mx, lp[e]);
  }
  double z = 0.0;
  for (int32_t e = 0; e < E; ++e) z += std::exp(lp[e] - mx);
  const double lz = mx + std::log(z);
  for (int32_t e = 0; e < E; ++e) lp[e] -= lz;
}

// Mean Effective Experts (Eq. (2) applied to p) of S samples of Dir(alpha).
double mean_effexp(const Philox& g, int32_t E, double alpha, int32_t S, std::vector<double>& lp) {
  double acc = 0.0;
  for (int32_t s = 0; s < S; ++s) {
    dirichlet_logp(g, alpha, E, (uint32_t)s, lp);
    double mx = *std::max_element(lp.begin(), lp.end());
    double z = 0.0;
    for (double v : lp) z += std::exp(v - mx);
    double s1 = 0.0, s2 = 0.0;
    for (double v : lp) {
      const double p = std::exp(v - mx) / z;
      s1 += p;
      s2 += p * p;
    }
    acc += s1 * s1 / s2;
  }
  return acc / S;
}

// Gumbel-top-k experts of token t under log p (keys from uniforms tagged 2), softmax gates of
// N(0,1) logits (tag 3), written to id[0..k) and w[0..k).
void gumbel_token(const Philox& g, const std::vector<double>& lp, uint32_t t, int32_t k, uint32_t s,
                  std::vector<double>& key, std::vector<int32_t>& idx, int32_t* id, float* w) {
  const int32_t E = (int32_t)lp.size();
  for (int32_t e = 0; e < E; e += 2) {
    double u0, u1;
    g.uniforms(t, (uint32_t)e, s, 2, u0, u1);
    key[e] = lp[e] - std::log(-std::log(u0));
    if (e + 1 < E) key[e + 1] = lp[e + 1] - std::log(-std::log(u1));
  }
  std::iota(idx.begin(), idx.end(), 0);
  std::partial_sort(idx.begin(), idx.begin() + k, idx.end(), [&](int32_t a, int32_t b) {
    return key[a] > key[b] || (key[a] == key[b] && a < b);
  });
  double zs = 0.0, lg[DAMOE_MAX_K];
  for (int32_t j = 0; j < k; ++j) {
    double u0, u1;
    g.uniforms(t, (uint32_t)j, s, 3, u0, u1);
    lg[j] = std::sqrt(-2.0 * std::log(u0)) * std::cos(6.283185307179586 * u1);
  }
  const double m = *std::max_element(lg, lg + k);
  for (int32_t j = 0; j < k; ++j) zs += std::exp(lg[j] - m);
  for (int32_t j = 0; j < k; ++j) {
    id[j] = idx[j];
    w[j] = (float)(std::exp(lg[j] - m) / zs);
  }
}

// Routing of T tokens for a layer of E_local experts.  Without expert parallelism (ep <= 1)
// the tokens are drawn directly (E_local = lp.size()).  With ep > 1, lp is over the global
// pool of E_local * ep experts and the layer is the rank holding experts [0, E_local): global
// tokens are drawn in turn, those with at least one local slot are kept with the other slots
// masked (-1), until T are kept (bounded; rows left over are fully masked).
void sample_routing(const Philox& g, const std::vector<double>& lp, int32_t T, int32_t k, int32_t E_local,
                    int32_t ep, uint32_t s, std::vector<int32_t>& ids, std::vector<float>& w) {
  const int32_t Eg = (int32_t)lp.size();
  ids.assign((size_t)T * k, -1);
  w.assign((size_t)T * k, 0.f);
  std::vector<double> key(Eg);
  std::vector<int32_t> idx(Eg);
  if (ep <= 1) {
    for (int32_t t = 0; t < T; ++t)
      gumbel_token(g, lp, (uint32_t)t, k, s, key, idx, ids.data() + (size_t)t * k, w.data() + (size_t)t * k);
    return;
  }
  int32_t kept = 0;
  std::vector<int32_t> id(k);
  std::vector<float> wt(k);
  for (uint32_t t = 0; kept < T && t < (uint32_t)T * 1024u; ++t) {
    gumbel_token(g, lp, t, k, s, key, idx, id.data(), wt.data());
    bool local = false;
    for (int32_t j = 0; j < k; ++j) local = local || id[j] < E_local;
    if (!local) continue;
    for (int32_t j = 0; j < k; ++j) {
      ids[(size_t)kept * k + j] = id[j] < E_local ? id[j] : -1;
      w[(size_t)kept * k + j] = wt[j];
    }
    ++kept;
  }
}

// Routing of T tokens whose groups of `group` consecutive tokens share one row: group r draws
// one Gumbel-top-k row under lp (as token r of sample_routing) and every token of the group
// takes its ids and gates.
void repeated_routing(const Philox& g, const std::vector<double>& lp, int32_t T, int32_t k, int32_t group,
                      uint32_t s, std::vector<int32_t>& ids, std::vector<float>& w) {
  const int32_t E = (int32_t)lp.size();
  ids.assign((size_t)T * k, -1);
  w.assign((size_t)T * k, 0.f);
  std::vector<double> key(E);
  std::vector<int32_t> idx(E);
  for (int32_t t = 0; t < T; ++t) {
    if (t % group == 0) {
      gumbel_token(g, lp, (uint32_t)(t / group), k, s, key, idx, ids.data() + (size_t)t * k,
                   w.data() + (size_t)t * k);
    } else {
      std::copy_n(ids.data() + (size_t)(t - 1) * k, k, ids.data() + (size_t)t * k);
      std::copy_n(w.data() + (size_t)(t - 1) * k, k, w.data() + (size_t)t * k);
    }
  }
}

void exemplar(const std::vector<std::vector<int32_t>>& counts, int32_t E, int32_t* Q) {
  std::vector<double> c(E, 0.0);
  for (const auto& v : counts) {
    std::vector<int32_t> s(v);
    std::sort(s.begin(), s.end(), std::greater<int32_t>());
    double nn = 0.0;
    for (int32_t x : s) nn += (double)x * x;
    if (nn <= 0.0) continue;
    nn = std::sqrt(nn);
    for (int32_t r = 0; r < E; ++r) c[r] += s[r] / nn / (double)counts.size();
  }
  double n = 0.0;
  for (double x : c) n += x * x;
  n = std::sqrt(n);
  for (int32_t r = 0; r < E; ++r) Q[r] = (int32_t)std::nearbyint(n > 0.0 ? c[r] / n * 32768.0 : 0.0);
}

#define TRY_HIP(x)                                         \
  do {                                                     \
    if ((x) != hipSuccess) {                               \
      st = DAMOE_ERR_HIP;                                  \
      goto done;                                           \
    }                                                      \
  } while (0)
#define TRY(x)                                             \
  do {                                                     \
    if ((st = (x)) != DAMOE_OK) goto done;                 \
  } while (0)

// The kernel class a variant runs on, of the kClasses that a fused call launches separately:
// the stream and tiled variants share one kernel, the big-tile, fp8-MFMA and deep-ring
// variants have kernels of their own, and the fp8-MFMA deep-ring variant, which runs the
// deep-ring GEMM1 and the fp8-MFMA GEMM2, counts as a class of its own.  A fused call whose candidates span several classes
// launches all of them, and those the device did not choose return at once.
constexpr int32_t kClasses = 5;
int32_t kernel_class(int32_t v) {
  switch (damoe::variant(v).kind) {
    case damoe::kBig: return 1;
    case damoe::kBig8: return 2;
    case damoe::kDeep: return 3;
    case damoe::kDeep8: return 4;
    default: return 0;
  }
}

}  // namespace

extern "C" {

// Alg. 1's root: the mean Effective Experts of Dir(alpha) grows with alpha (Sec. III-A), so the
// concentration reaching `target` is bracketed in [1e-6, 1e6] and the bracket is halved on a log
// scale (alpha spans twelve decades and the skews of interest sit between 0.03 and 10), at most
// `iters` times, until its ends agree to a relative 1e-12; the geometric centre of the bracket
// is returned.  The draws are the same at every alpha (common random numbers), so the mean is a
// deterministic function of alpha.
double damoe_alpha_search(int32_t E, double target, int32_t samples, int32_t iters, uint64_t seed) {
  if (E < 1 || samples < 1 || iters < 1) return NAN;
  const Philox g(seed);
  std::vector<double> lp;
  double log_lo = std::log(1e-6), log_hi = std::log(1e6);
  for (int32_t t = 0; t < iters && log_hi - log_lo > 1e-12; ++t) {
    const double log_c = 0.5 * (log_lo + log_hi);
    const bool below = mean_effexp(g, E, std::exp(log_c), samples, lp) < target;
    (below ? log_lo : log_hi) = log_c;
  }
  return std::exp(0.5 * (log_lo + log_hi));
}

damoe_status damoe_tune(const damoe_layer* L, const damoe_tune_config* cfg, damoe_table** out,
                        hipStream_t stream) {
  if (!L || !cfg || !out || !cfg->bucket_T || cfg->n_buckets < 1 || !cfg->skew_X || cfg->n_skews < 1 ||
      cfg->samples < 1 || cfg->reps < 1 || !cfg->x)
    return DAMOE_ERR_INVALID_ARG;
  *out = nullptr;
  const int32_t E = L->E, k = L->k, H = L->H;
  const int32_t nv = damoe_num_variants();
  int32_t T_max = 0;
  for (int32_t b = 0; b < cfg->n_buckets; ++b) T_max = std::max(T_max, cfg->bucket_T[b]);
  const size_t ws_bytes = damoe_workspace_size(L, T_max);
  if (ws_bytes == 0) return DAMOE_ERR_INVALID_ARG;
  // Expert parallelism: the layer is one rank's share of a global pool of E * ep experts.
  if (cfg->ep < 0 || cfg->ep > 64) return DAMOE_ERR_INVALID_ARG;
  // Repeated-row exemplars (not combined with expert parallelism).
  if (cfg->n_repeat < 0 || cfg->n_repeat > 64 || (cfg->n_repeat > 0 && (!cfg->repeat_f || cfg->ep > 1)))
    return DAMOE_ERR_INVALID_ARG;
  for (int32_t r = 0; r < cfg->n_repeat; ++r)
    if (cfg->repeat_f[r] < 1 || cfg->repeat_f[r] > 100) return DAMOE_ERR_INVALID_ARG;
  if (cfg->flush_mib < 0 || cfg->flush_mib > 16384) return DAMOE_ERR_INVALID_ARG;
  const size_t flush_bytes = (size_t)cfg->flush_mib << 20;
  const int32_t ep = cfg->ep > 1 ? cfg->ep : 1;
  const int32_t Eg = E * ep;
  const int32_t a_samples = cfg->alpha_samples > 0 ? cfg->alpha_samples : 64;
  const int32_t a_iters = cfg->alpha_iters > 0 ? cfg->alpha_iters : 60;
  const Philox g(cfg->seed);

  damoe_status st = DAMOE_OK;
  void* ws = nullptr;
  int32_t *d_ids = nullptr, *d_counts = nullptr, *d_off = nullptr, *d_perm = nullptr, *d_inv = nullptr,
          *d_bucket = nullptr;
  float* d_w = nullptr;
  uint64_t* d_nd = nullptr;
  uint16_t* d_y = nullptr;
  int32_t* d_vid = nullptr;
  void* d_flush = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  std::vector<int32_t> t_bucket, t_nex, t_noda, t_kid, t_Q;
  std::vector<double> alphas(cfg->n_skews);
  std::vector<double> noop(kClasses, 0.0);  // ms
  std::vector<double> lp;
  std::vector<int32_t> ids;
  std::vector<float> w;
  const size_t A_max = (size_t)T_max * k;

  TRY_HIP(hipMalloc(&ws, ws_bytes));
  TRY_HIP(hipMalloc(&d_ids, sizeof(int32_t) * A_max));
  TRY_HIP(hipMalloc(&d_w, sizeof(float) * A_max));
  TRY_HIP(hipMalloc(&d_counts, sizeof(int32_t) * E));
  TRY_HIP(hipMalloc(&d_off, sizeof(int32_t) * (E + 1)));
  TRY_HIP(hipMalloc(&d_perm, sizeof(int32_t) * A_max));
  TRY_HIP(hipMalloc(&d_inv, sizeof(int32_t) * A_max));
  TRY_HIP(hipMalloc(&d_nd, sizeof(uint64_t) * 2));
  TRY_HIP(hipMalloc(&d_bucket, sizeof(int32_t)));
  TRY_HIP(hipMalloc(&d_y, sizeof(uint16_t) * (size_t)T_max * H));
  TRY_HIP(hipMalloc(&d_vid, sizeof(int32_t)));
  if (flush_bytes) TRY_HIP(hipMalloc(&d_flush, flush_bytes));
  TRY_HIP(hipMemset(ws, 0, ws_bytes));
  TRY_HIP(hipEventCreate(&e0));
  TRY_HIP(hipEventCreate(&e1));

  // Alg. 1 once per skew: the ddist:X target is E / X.
  for (int32_t j = 0; j < cfg->n_skews; ++j) {
    alphas[j] = damoe_alpha_search(Eg, (double)Eg / cfg->skew_X[j], a_samples, a_iters, cfg->seed);
    if (cfg->verbose) std::fprintf(stderr, "damoe_tune: ddist:%.2f -> alpha %.5g\n", cfg->skew_X[j], alphas[j]);
  }

  // Cost of a launched class that runs nothing, per class c: a fused call whose candidates are
  // a reference variant of another class and c's first variant, with the device-side id on the
  // reference, against the reference alone; paired runs (each behind the cache flush) on one
  // uniform routing of a single token, the median difference.  The cost does not depend on
  // the call's size, and at one token it is not buried in the run-to-run spread of the GEMMs
  // (at T = 2048 that spread is about 100 us).  Charged below to the per-exemplar choices of
  // a bucket whose kernels span several classes.
  {
    const int32_t T = 1;
    int32_t first_of[kClasses];
    for (int32_t c = 0; c < kClasses; ++c) first_of[c] = -1;
    for (int32_t v = nv - 1; v >= 0; --v)
      if (damoe_variant_supports(v, L->wdtype)) first_of[kernel_class(v)] = v;
    lp.assign(Eg, -std::log((double)Eg));
    sample_routing(g, lp, T, k, E, ep, 0x9000000u, ids, w);
    TRY_HIP(hipMemcpyAsync(d_ids, ids.data(), sizeof(int32_t) * ids.size(), hipMemcpyHostToDevice, stream));
    TRY_HIP(hipMemcpyAsync(d_w, w.data(), sizeof(float) * w.size(), hipMemcpyHostToDevice, stream));
    TRY(damoe_route_histogram(d_ids, T, k, E, d_counts, d_off, d_perm, d_inv, d_nd, d_bucket, ws, ws_bytes,
                              stream));
    for (int32_t c = 0; c < kClasses; ++c) {
      if (first_of[c] < 0) continue;
      int32_t ref = -1;
      for (int32_t o = 0; o < kClasses && ref < 0; ++o)
        if (o != c && first_of[o] >= 0) ref = first_of[o];
      if (ref < 0) continue;
      const uint32_t mask = (1u << ref) | (1u << first_of[c]);
      TRY_HIP(hipMemcpyAsync(d_vid, &ref, sizeof(int32_t), hipMemcpyHostToDevice, stream));
      const int32_t nrep = 2 * cfg->reps + 1;
      std::vector<float> diff(nrep);
      for (int32_t r = 0; r < nrep; ++r) {
        float t2[2];
        for (int32_t m = 0; m < 2; ++m) {
          if (d_flush) TRY_HIP(hipMemsetAsync(d_flush, r & 0xFF, flush_bytes, stream));
          TRY_HIP(hipEventRecord(e0, stream));
          TRY(damoe_fused_moe(L, cfg->x, d_w, T, d_perm, d_inv, d_vid, m == 0 ? ref : -1, m == 0 ? 0u : mask, d_y,
                              ws, ws_bytes, stream));
          TRY_HIP(hipEventRecord(e1, stream));
          TRY_HIP(hipEventSynchronize(e1));
          TRY_HIP(hipEventElapsedTime(&t2[m], e0, e1));
        }
        diff[r] = t2[1] - t2[0];
      }
      std::nth_element(diff.begin(), diff.begin() + nrep / 2, diff.end());
      noop[c] = std::max(0.0, (double)diff[nrep / 2]);
      if (cfg->verbose)
        std::fprintf(stderr, "damoe_tune: launched class of %s, not chosen: %.1f us\n",
                     damoe_variant_name(first_of[c]), noop[c] * 1e3);
    }
  }

  for (int32_t b = 0; b < cfg->n_buckets; ++b) {
    const int32_t T = cfg->bucket_T[b];
    // Latency of every variant on one routing: median of reps forced runs.
    auto time_routing = [&](std::vector<double>& lat_v, std::vector<int32_t>* counts_out) -> damoe_status {
      if (hipMemcpyAsync(d_ids, ids.data(), sizeof(int32_t) * ids.size(), hipMemcpyHostToDevice, stream) ||
          hipMemcpyAsync(d_w, w.data(), sizeof(float) * w.size(), hipMemcpyHostToDevice, stream))
        return DAMOE_ERR_HIP;
      damoe_status s2 = damoe_route_histogram(d_ids, T, k, E, d_counts, d_off, d_perm, d_inv, d_nd,
                                              d_bucket, ws, ws_bytes, stream);
      if (s2 != DAMOE_OK) return s2;
      if (counts_out) {
        counts_out->resize(E);
        if (hipMemcpyAsync(counts_out->data(), d_counts, sizeof(int32_t) * E, hipMemcpyDeviceToHost, stream))
          return DAMOE_ERR_HIP;
      }
      lat_v.assign(nv, INFINITY);
      std::vector<float> reps(cfg->reps);
      for (int32_t v = 0; v < nv; ++v) {
        if (!damoe_variant_supports(v, L->wdtype)) continue;
        // warm-up
        s2 = damoe_fused_moe(L, cfg->x, d_w, T, d_perm, d_inv, nullptr, v, 0u, d_y, ws, ws_bytes, stream);
        if (s2 != DAMOE_OK) return s2;
        for (int32_t r = 0; r < cfg->reps; ++r) {
          // The tuner is synchronous and never captured, so a memset is a fine way to evict.
          if (d_flush && hipMemsetAsync(d_flush, r & 0xFF, flush_bytes, stream)) return DAMOE_ERR_HIP;
          if (hipEventRecord(e0, stream)) return DAMOE_ERR_HIP;
          s2 = damoe_fused_moe(L, cfg->x, d_w, T, d_perm, d_inv, nullptr, v, 0u, d_y, ws, ws_bytes, stream);
          if (s2 != DAMOE_OK) return s2;
          if (hipEventRecord(e1, stream) || hipEventSynchronize(e1)) return DAMOE_ERR_HIP;
          float ms = 0.f;
          if (hipEventElapsedTime(&ms, e0, e1)) return DAMOE_ERR_HIP;
          reps[r] = ms;
        }
        std::nth_element(reps.begin(), reps.begin() + cfg->reps / 2, reps.end());
        lat_v[v] = reps[cfg->reps / 2];
      }
      return hipStreamSynchronize(stream) == hipSuccess ? DAMOE_OK : DAMOE_ERR_HIP;
    };

    t_bucket.push_back(T);
    int32_t n_added = 0;
    const size_t first_ex = t_kid.size();
    std::vector<std::vector<double>> skew_mean;  // [skew][variant] mean latency over the samples
    for (int32_t j = 0; j < cfg->n_skews; ++j) {
      std::vector<std::vector<int32_t>> cs;
      std::vector<double> mean(nv, 0.0), lat;
      for (int32_t s = 0; s < cfg->samples; ++s) {
        const uint32_t sid = 0x10000u + ((uint32_t)b << 20) + ((uint32_t)j << 10) + (uint32_t)s;
        dirichlet_logp(g, alphas[j], Eg, sid, lp);
        sample_routing(g, lp, T, k, E, ep, sid, ids, w);
        std::vector<int32_t> c;
        TRY(time_routing(lat, &c));
        cs.push_back(c);
        for (int32_t v = 0; v < nv; ++v) mean[v] += lat[v] / cfg->samples;
      }
      int32_t best = 0;
      for (int32_t v = 1; v < nv; ++v)
        if (mean[v] < mean[best]) best = v;
      t_kid.push_back(best);
      t_Q.resize(t_Q.size() + E);
      exemplar(cs, E, t_Q.data() + t_Q.size() - E);
      skew_mean.push_back(mean);
      ++n_added;
      if (cfg->verbose)
        std::fprintf(stderr, "damoe_tune: T=%d ddist:%.2f -> %s (%.1f us)\n", T, cfg->skew_X[j],
                     damoe_variant_name(best), mean[best] * 1e3);
    }
    // Repeated-row exemplars: groups of max(1, round(f T / 100)) consecutive tokens share one
    // row under a Dirichlet(1) p (round half to even).  Their sorted histograms are step-shaped,
    // unlike every Dirichlet exemplar, so without them the match takes an exemplar of another
    // shape for such batches.
    for (int32_t r = 0; r < cfg->n_repeat; ++r) {
      const int32_t group = std::max(1, (int32_t)std::nearbyint(cfg->repeat_f[r] * (double)T / 100.0));
      std::vector<std::vector<int32_t>> cs;
      std::vector<double> mean(nv, 0.0), lat;
      for (int32_t s = 0; s < cfg->samples; ++s) {
        const uint32_t sid = 0x4000000u + ((uint32_t)b << 16) + ((uint32_t)r << 8) + (uint32_t)s;
        dirichlet_logp(g, 1.0, Eg, sid, lp);
        repeated_routing(g, lp, T, k, group, sid, ids, w);
        std::vector<int32_t> c;
        TRY(time_routing(lat, &c));
        cs.push_back(c);
        for (int32_t v = 0; v < nv; ++v) mean[v] += lat[v] / cfg->samples;
      }
      int32_t best = 0;
      for (int32_t v = 1; v < nv; ++v)
        if (mean[v] < mean[best]) best = v;
      t_kid.push_back(best);
      t_Q.resize(t_Q.size() + E);
      exemplar(cs, E, t_Q.data() + t_Q.size() - E);
      skew_mean.push_back(mean);
      ++n_added;
      if (cfg->verbose)
        std::fprintf(stderr, "damoe_tune: T=%d repeat:%d%% -> %s (%.1f us)\n", T, cfg->repeat_f[r],
                     damoe_variant_name(best), mean[best] * 1e3);
    }
    t_nex.push_back(n_added);
    // Skews whose exemplars quantise to the same vector are the same distribution to the
    // dispatcher (it can only ever pick the first of them): they share one kernel, the one
    // with the fastest mean over all of their samples.
    for (int32_t j = 0; j < n_added; ++j) {
      std::vector<double> pooled(nv, 0.0);
      int32_t members = 0;
      for (int32_t u = 0; u < n_added; ++u) {
        if (!std::equal(t_Q.begin() + (first_ex + j) * E, t_Q.begin() + (first_ex + j + 1) * E,
                        t_Q.begin() + (first_ex + u) * E))
          continue;
        for (int32_t v = 0; v < nv; ++v) pooled[v] += skew_mean[u][v];
        ++members;
      }
      if (members > 1) {
        int32_t best = 0;
        for (int32_t v = 1; v < nv; ++v)
          if (pooled[v] < pooled[best]) best = v;
        t_kid[first_ex + j] = best;
      }
    }
    // Cost of the exemplar match itself: route + match on a one-bucket table of this bucket's
    // exemplars whose kernels differ (so every call scores them), minus route alone, both on
    // the last routing timed above.  The per-exemplar choice is kept only when its mean over
    // the bucket's samples, charged this cost, beats the best single variant; otherwise every
    // exemplar maps to that variant and the online step skips the match.
    {
      std::vector<int32_t> kid_probe(n_added), noda_probe(1, 0), bt(1, T), nex(1, n_added);
      for (int32_t j = 0; j < n_added; ++j) kid_probe[j] = j & 1;
      damoe_table_desc pd{};
      pd.E = E;
      pd.k = k;
      pd.H = L->H;
      pd.I = L->I;
      pd.wdtype = L->wdtype;
      pd.n_buckets = 1;
      pd.bucket_T = bt.data();
      pd.n_ex = nex.data();
      pd.Q = t_Q.data() + first_ex * E;
      pd.kid = kid_probe.data();
      pd.noda = noda_probe.data();
      damoe_table* probe = nullptr;
      TRY(damoe_table_create(&pd, &probe));
      const int32_t nrep = 2 * cfg->reps + 1;
      std::vector<float> t_route(nrep), t_match(nrep);
      damoe_status s3 = DAMOE_OK;
      for (int32_t r = 0; r < nrep && s3 == DAMOE_OK; ++r) {
        for (int32_t m = 0; m < 2 && s3 == DAMOE_OK; ++m) {
          if (hipEventRecord(e0, stream)) s3 = DAMOE_ERR_HIP;
          if (s3 == DAMOE_OK)
            s3 = m == 0 ? damoe_route_histogram(d_ids, T, k, E, d_counts, d_off, d_perm, d_inv, d_nd, d_bucket,
                                                ws, ws_bytes, stream)
                        : damoe_route_dispatch(probe, d_ids, T, k, E, d_counts, d_off, d_perm, d_inv, d_nd,
                                               d_bucket, d_vid, ws, ws_bytes, stream);
          float ms = 0.f;
          if (s3 == DAMOE_OK && (hipEventRecord(e1, stream) || hipEventSynchronize(e1) ||
                                 hipEventElapsedTime(&ms, e0, e1)))
            s3 = DAMOE_ERR_HIP;
          (m == 0 ? t_route : t_match)[r] = ms;
        }
      }
      damoe_table_destroy(probe);
      TRY(s3);
      std::nth_element(t_route.begin(), t_route.begin() + nrep / 2, t_route.end());
      std::nth_element(t_match.begin(), t_match.begin() + nrep / 2, t_match.end());
      const double match_cost = std::max(0.0, (double)t_match[nrep / 2] - (double)t_route[nrep / 2]);
      // Mean over the bucket's exemplars of a choice of kernels: their latencies, the match when
      // they differ, and for each exemplar the launches of the bucket's other kernel classes.
      auto cost_of = [&](const std::vector<int32_t>& kid) {
        uint32_t classes = 0;
        bool differ = false;
        for (int32_t j = 0; j < n_added; ++j) {
          classes |= 1u << kernel_class(kid[j]);
          differ = differ || kid[j] != kid[0];
        }
        double c = differ ? match_cost : 0.0;
        for (int32_t j = 0; j < n_added; ++j) {
          c += skew_mean[j][kid[j]] / n_added;
          for (int32_t o = 0; o < kClasses; ++o)
            if (((classes >> o) & 1u) && o != kernel_class(kid[j])) c += noop[o] / n_added;
        }
        return c;
      };
      std::vector<int32_t> kid_ad(t_kid.begin() + first_ex, t_kid.end());
      const double adaptive = cost_of(kid_ad);
      std::vector<double> single(nv, 0.0);
      for (int32_t j = 0; j < n_added; ++j)
        for (int32_t v = 0; v < nv; ++v) single[v] += skew_mean[j][v] / n_added;
      int32_t best = 0;
      for (int32_t v = 1; v < nv; ++v)
        if (single[v] < single[best]) best = v;
      // The per-exemplar choice restricted to one kernel class (exemplars that quantise alike
      // pooled as above): one launch per GEMM, the match only if the kernels still differ.
      std::vector<int32_t> chosen(n_added, best);
      double chosen_cost = single[best];
      const char* how = " -> single variant";
      if (adaptive < chosen_cost) {
        chosen = kid_ad;
        chosen_cost = adaptive;
        how = "";
      }
      for (int32_t c = 0; c < kClasses; ++c) {
        std::vector<int32_t> kid_c(n_added, -1);
        for (int32_t j = 0; j < n_added; ++j) {
          double bv = INFINITY;
          for (int32_t v = 0; v < nv; ++v) {
            if (kernel_class(v) != c || !damoe_variant_supports(v, L->wdtype)) continue;
            double pooled = 0.0;
            for (int32_t u = 0; u < n_added; ++u)
              if (std::equal(t_Q.begin() + (first_ex + j) * E, t_Q.begin() + (first_ex + j + 1) * E,
                             t_Q.begin() + (first_ex + u) * E))
                pooled += skew_mean[u][v];
            if (pooled < bv) {
              bv = pooled;
              kid_c[j] = v;
            }
          }
        }
        if (kid_c[0] < 0) continue;  // no variant of this class runs these weights
        const double cc = cost_of(kid_c);
        if (cc < chosen_cost) {
          chosen = kid_c;
          chosen_cost = cc;
          how = " -> one kernel class";
        }
      }
      std::copy(chosen.begin(), chosen.end(), t_kid.begin() + first_ex);
      if (cfg->verbose)
        std::fprintf(stderr, "damoe_tune: T=%d match %.1f us; adaptive %.1f us vs %s %.1f us; chosen %.1f us%s\n",
                     T, match_cost * 1e3, adaptive * 1e3, damoe_variant_name(best), single[best] * 1e3,
                     chosen_cost * 1e3, how);
    }
    // Distribution-unaware baseline: the fastest variant under uniform routing.
    {
      std::vector<double> mean(nv, 0.0), lat;
      lp.assign(Eg, -std::log((double)Eg));
      for (int32_t s = 0; s < cfg->samples; ++s) {
        const uint32_t sid = 0x8000000u + ((uint32_t)b << 10) + (uint32_t)s;
        sample_routing(g, lp, T, k, E, ep, sid, ids, w);
        TRY(time_routing(lat, nullptr));
        for (int32_t v = 0; v < nv; ++v) mean[v] += lat[v] / cfg->samples;
      }
      int32_t best = 0;
      for (int32_t v = 1; v < nv; ++v)
        if (mean[v] < mean[best]) best = v;
      t_noda.push_back(best);
      if (cfg->verbose)
        std::fprintf(stderr, "damoe_tune: T=%d uniform (noda) -> %s\n", T, damoe_variant_name(best));
    }
  }
  {
    damoe_table_desc d{};
    d.E = E;
    d.k = k;
    d.H = L->H;
    d.I = L->I;
    d.wdtype = L->wdtype;
    d.n_buckets = (int32_t)t_bucket.size();
    d.bucket_T = t_bucket.data();
    d.n_ex = t_nex.data();
    d.Q = t_Q.data();
    d.kid = t_kid.data();
    d.noda = t_noda.data();
    st = damoe_table_create(&d, out);
  }
done:
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(ws);
  (void)hipFree(d_ids);
  (void)hipFree(d_w);
  (void)hipFree(d_counts);
  (void)hipFree(d_off);
  (void)hipFree(d_perm);
  (void)hipFree(d_inv);
  (void)hipFree(d_nd);
  (void)hipFree(d_bucket);
  (void)hipFree(d_y);
  (void)hipFree(d_vid);
  (void)hipFree(d_flush);
  return st;
}

}  // extern "C"
