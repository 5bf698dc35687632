// Offline statistics and communication-aware replica placement (Table I):
// host code of the C ABI.  The calibration record is what a full-depth,
// exact pass of the stack writes into its trace (routed experts,
// importances, per-layer exit confidences); the statistics follow
// Sec. IV-C Eq. (26)-(27) and Sec. V-E Eq. (38), the replication Eq. (28)
// and Table I, lines 9-13.  Every function validates its arguments first
// and writes nothing on error.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <queue>
#include <vector>

#include "trimmoe.h"

namespace {

bool finite_nonneg(double v) { return v >= 0.0 && !isinf(v); }

// Eq. (28): lambda * rho * (z / mean bandwidth + mean latency), the means
// over the servers that currently host expert (l, k)
double benefit(int M, int N, int E, const double* lambda, const double* rho, const double* z,
               const double* bandwidth, const double* latency, const uint8_t* x, int m, int l,
               int k) {
  double bsum = 0.0, tsum = 0.0;
  int hosts = 0;
  for (int n = 0; n < M; ++n)
    if (x[((size_t)n * N + l) * E + k]) {
      bsum += bandwidth[(size_t)m * M + n];
      tsum += latency[(size_t)m * M + n];
      ++hosts;
    }
  const double b_bar = bsum / hosts, t_bar = tsum / hosts;
  return lambda[(size_t)l * E + k] * rho[(size_t)m * N + l] * (z[l] / b_bar + t_bar);
}

struct Cand {
  double b;
  int l, k, m;
  uint32_t version;  // placements of (l, k) when the benefit was computed
};

// heap order: larger benefit first, then lower l, k, m
struct CandLess {
  bool operator()(const Cand& a, const Cand& c) const {
    if (a.b != c.b) return a.b < c.b;
    if (a.l != c.l) return a.l > c.l;
    if (a.k != c.k) return a.k > c.k;
    return a.m > c.m;
  }
};

}  // namespace

extern "C" {

int trimmoe_calib_exit_layers(int32_t n_layers, int32_t n_tokens, const float* xi, float p_exit,
                              int32_t* exit_layer) {
  if (!xi || !exit_layer) return TRIMMOE_ERR_NULL;
  if (n_layers < 1 || n_tokens < 0) return TRIMMOE_ERR_SHAPE;
  if (isnan(p_exit)) return TRIMMOE_ERR_POLICY;
  for (int q = 0; q < n_tokens; ++q) {
    int ex = n_layers;
    for (int l = 0; l + 1 < n_layers; ++l) {
      const float v = xi[(size_t)l * n_tokens + q];
      if (!isnan(v) && v >= p_exit) {
        ex = l;
        break;
      }
    }
    exit_layer[q] = ex;
  }
  return TRIMMOE_OK;
}

int trimmoe_calib_stats(int32_t n_layers, int32_t n_tokens, int32_t n_experts, int32_t top_k,
                        const int16_t* target, const float* importance,
                        const int32_t* exit_layer, const float* theta, double* pi, double* act,
                        double* sigma, double* lambda) {
  if (!target || !importance || !exit_layer || !theta || !pi || !act || !sigma || !lambda)
    return TRIMMOE_ERR_NULL;
  const int N = n_layers, Q = n_tokens, E = n_experts, k = top_k;
  if (N < 1 || Q < 1 || E < 1 || E > TRIMMOE_MAX_EXPERTS || k < 1 || k > TRIMMOE_MAX_TOPK)
    return TRIMMOE_ERR_SHAPE;
  for (size_t i = 0; i < (size_t)N * Q * k; ++i)
    if (target[i] < 0 || target[i] >= E) return TRIMMOE_ERR_SHAPE;
  std::vector<double> routed(E), above(E);
  std::vector<uint8_t> seen(E);
  for (int l = 0; l < N; ++l) {
    std::fill(routed.begin(), routed.end(), 0.0);
    std::fill(above.begin(), above.end(), 0.0);
    int active = 0;
    for (int q = 0; q < Q; ++q) {
      if (exit_layer[q] < l) continue;
      ++active;
      const int16_t* s = target + ((size_t)l * Q + q) * k;
      const bool over = importance[(size_t)l * Q + q] > theta[l];
      std::fill(seen.begin(), seen.end(), 0);
      for (int r = 0; r < k; ++r) {
        if (seen[s[r]]) continue;  // the routed set: each expert once
        seen[s[r]] = 1;
        routed[s[r]] += 1.0;
        if (over) above[s[r]] += 1.0;
      }
    }
    pi[l] = (double)active / Q;  // Eq. (26)
    for (int e = 0; e < E; ++e) {
      const size_t i = (size_t)l * E + e;
      act[i] = active ? routed[e] / active : 0.0;
      sigma[i] = routed[e] > 0.0 ? above[e] / routed[e] : 0.0;  // Eq. (27)
      lambda[i] = pi[l] * sigma[i] * act[i];
    }
  }
  return TRIMMOE_OK;
}

int trimmoe_calib_transitions(int32_t n_layers, int32_t n_tokens, int32_t n_experts,
                              int32_t top_k, const int16_t* target, const int32_t* exit_layer,
                              int32_t trans_b, int16_t* trans_to, float* trans_p) {
  if (!target || !exit_layer || !trans_to || !trans_p) return TRIMMOE_ERR_NULL;
  const int N = n_layers, Q = n_tokens, E = n_experts, k = top_k, B = trans_b;
  if (N < 2 || Q < 0 || E < 1 || E > TRIMMOE_MAX_EXPERTS || k < 1 || k > TRIMMOE_MAX_TOPK ||
      B < 1 || B > E)
    return TRIMMOE_ERR_SHAPE;
  for (size_t i = 0; i < (size_t)N * Q * k; ++i)
    if (target[i] < 0 || target[i] >= E) return TRIMMOE_ERR_SHAPE;
  std::vector<int64_t> counts((size_t)E * E);
  std::vector<int> order(E);
  for (int l = 0; l + 1 < N; ++l) {
    std::fill(counts.begin(), counts.end(), 0);
    // Eq. (38): every (routed at l, routed at l + 1) pair of a token active
    // at both layers counts once
    for (int q = 0; q < Q; ++q) {
      if (exit_layer[q] < l + 1) continue;
      const int16_t* a = target + ((size_t)l * Q + q) * k;
      const int16_t* b = target + ((size_t)(l + 1) * Q + q) * k;
      for (int r = 0; r < k; ++r)
        for (int s = 0; s < k; ++s) ++counts[(size_t)a[r] * E + b[s]];
    }
    for (int e = 0; e < E; ++e) {
      const int64_t* c = counts.data() + (size_t)e * E;
      for (int f = 0; f < E; ++f) order[f] = f;
      // the B most frequent next experts, ties to the lower id
      std::stable_sort(order.begin(), order.end(), [&](int u, int v) { return c[u] > c[v]; });
      int64_t total = 0;
      int kept = 0;
      for (; kept < B && c[order[kept]] > 0; ++kept) total += c[order[kept]];
      int16_t* to = trans_to + ((size_t)l * E + e) * B;
      float* pr = trans_p + ((size_t)l * E + e) * B;
      for (int j = 0; j < B; ++j) {
        to[j] = j < kept ? (int16_t)order[j] : (int16_t)-1;
        pr[j] = j < kept ? (float)((double)c[order[j]] / (double)total) : 0.f;
      }
    }
  }
  return TRIMMOE_OK;
}

int trimmoe_place_replicas(int32_t n_servers, int32_t n_layers, int32_t n_experts,
                           const double* lambda, const double* rho, const double* z,
                           const double* nbytes, const double* capacity,
                           const double* bandwidth, const double* latency, uint8_t* x,
                           int32_t* n_placed) {
  if (!lambda || !rho || !z || !nbytes || !capacity || !bandwidth || !latency || !x || !n_placed)
    return TRIMMOE_ERR_NULL;
  const int M = n_servers, N = n_layers, E = n_experts;
  if (M < 1 || N < 1 || E < 1) return TRIMMOE_ERR_SHAPE;
  for (size_t i = 0; i < (size_t)N * E; ++i)
    if (!finite_nonneg(lambda[i]) || !(nbytes[i] > 0.0) || isinf(nbytes[i]))
      return TRIMMOE_ERR_POLICY;
  for (size_t i = 0; i < (size_t)M * N; ++i)
    if (!finite_nonneg(rho[i])) return TRIMMOE_ERR_POLICY;
  for (int l = 0; l < N; ++l)
    if (!finite_nonneg(z[l])) return TRIMMOE_ERR_POLICY;
  for (size_t i = 0; i < (size_t)M * M; ++i)
    if (!(bandwidth[i] > 0.0) || isinf(bandwidth[i]) || !finite_nonneg(latency[i]))
      return TRIMMOE_ERR_POLICY;
  // the baseline must satisfy (c.1)-(c.3) (the premise of Property 1)
  std::vector<double> used(M, 0.0);
  for (int m = 0; m < M; ++m) {
    if (!finite_nonneg(capacity[m])) return TRIMMOE_ERR_POLICY;
    for (int l = 0; l < N; ++l)
      for (int k = 0; k < E; ++k) {
        const uint8_t v = x[((size_t)m * N + l) * E + k];
        if (v > 1) return TRIMMOE_ERR_SHAPE;
        if (v) used[m] += nbytes[(size_t)l * E + k];
      }
    if (used[m] > capacity[m]) return TRIMMOE_ERR_SHAPE;
  }
  for (int l = 0; l < N; ++l)
    for (int k = 0; k < E; ++k) {
      bool placed = false;
      for (int m = 0; m < M; ++m) placed |= x[((size_t)m * N + l) * E + k] != 0;
      if (!placed) return TRIMMOE_ERR_SHAPE;
    }

  // Table I, lines 10-13, with the candidates in a max-heap.  A placement
  // of (l, k) changes the host set behind the benefit of every other
  // server's copy of (l, k), so those are recomputed and pushed again; older
  // entries of (l, k) are dropped when they surface.  Residual memory only
  // shrinks, so a candidate that no longer fits is dropped for good; a
  // non-positive benefit stays non-positive (its sign is that of
  // lambda * rho), so such candidates are never pushed.
  std::vector<uint32_t> version((size_t)N * E, 0);
  std::priority_queue<Cand, std::vector<Cand>, CandLess> heap;
  auto push_expert = [&](int l, int k) {
    for (int m = 0; m < M; ++m) {
      if (x[((size_t)m * N + l) * E + k]) continue;
      const double b = benefit(M, N, E, lambda, rho, z, bandwidth, latency, x, m, l, k);
      if (b > 0.0) heap.push(Cand{b, l, k, m, version[(size_t)l * E + k]});
    }
  };
  for (int l = 0; l < N; ++l)
    for (int k = 0; k < E; ++k) push_expert(l, k);
  int placed = 0;
  while (!heap.empty()) {
    const Cand c = heap.top();
    heap.pop();
    const size_t lk = (size_t)c.l * E + c.k;
    if (c.version != version[lk]) continue;
    if (x[((size_t)c.m * N + c.l) * E + c.k]) continue;
    if (used[c.m] + nbytes[lk] > capacity[c.m]) continue;
    x[((size_t)c.m * N + c.l) * E + c.k] = 1;
    used[c.m] += nbytes[lk];
    ++placed;
    ++version[lk];
    push_expert(c.l, c.k);
  }
  *n_placed = placed;
  return TRIMMOE_OK;
}

}  // extern "C"
