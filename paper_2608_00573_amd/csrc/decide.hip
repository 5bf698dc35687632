// Decision-side kernels of the adaptive-depth MoE step (gfx950):
//   substitution table, routing + online decision, bucketing of the executed
//   (token, expert) rows, row permutation, weighted combine, exit gate and
//   the stable compaction of the active-token list.
//
// The decision rule is TrimMoE's online algorithm (arXiv 2608.00573,
// Sec. V, Algorithm 2 in Table II) at look-ahead horizon H = 1:
//   * routing / importance:        Sec. III-B, Eq. (4)
//   * substitution loss:           Sec. III-A, Eq. (3)
//   * skip degradation:            Sec. III-B, Eq. (5), rho(I) = min(1, s_l I)
//   * execute / skip cost:         Sec. V-A, Eq. (31), (32)
//   * feasible action set:         Sec. V-B, Eq. (34)
//   * transmission necessity:      Sec. V-C, Eq. (35) + importance threshold
//   * argmin and state update:     Sec. V-E, Eq. (40)-(42)
//   * exit gate:                   Sec. III-C, Eq. (8), (9)
// With top-k > 1 every routed slot is resolved on its own under the one
// per-token budget; the only useful substitute of a remote slot is its
// minimum-Q local expert (same delay, least budget); ties: lower expert id
// in top-k, then fewer substitutions, then the lower slot bitmask, and
// execute before skip.  Comparisons are non-strict as printed (Eq. (8),
// (34), Sec. V-C).
#include <math.h>

#include "common.h"

namespace trimmoe {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int RB = kRouteTokens;
constexpr int KMAX = TRIMMOE_MAX_TOPK;

// ----------------------------------------------------------- state reset --
__global__ void k_state_reset(int T, int N, float* d_acc, int32_t* active_idx,
                              int32_t* n_active, int32_t* exit_layer, float* xi) {
  int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t == 0) *n_active = T;
  if (t < T) {
    d_acc[t] = 0.f;
    active_idx[t] = t;
    exit_layer[t] = N;
    xi[t] = __int_as_float(0x7fc00000);
  }
}

// ------------------------------------------------ trace: inactive default --
// Rows of the layers p's trace pointers start at, one per blockIdx.y.
__global__ void k_trace_fill(LayerParams p) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const size_t y = blockIdx.y, rowT = y * p.T, rowTk = rowT * p.k;
  const float qnan = __int_as_float(0x7fc00000);
  if (blockIdx.x == 0 && threadIdx.x < kCounters && p.tr_counters)
    p.tr_counters[y * kCounters + threadIdx.x] = 0;
  if (t >= p.T) return;
  if (p.tr_action) p.tr_action[rowT + t] = TRIMMOE_ACT_INACTIVE;
  for (int s = 0; s < p.k; ++s) {
    const size_t o = rowTk + (size_t)t * p.k + s;
    if (p.tr_target) p.tr_target[o] = -1;
    if (p.tr_exec) p.tr_exec[o] = -1;
    if (p.tr_kind) p.tr_kind[o] = TRIMMOE_KIND_NONE;
    if (p.tr_gate) p.tr_gate[o] = qnan;
  }
  if (p.tr_importance) p.tr_importance[rowT + t] = qnan;
  if (p.tr_xi) p.tr_xi[rowT + t] = qnan;
  if (p.tr_d_acc) p.tr_d_acc[rowT + t] = qnan;
}

// ------------------------------------------- route + decide (one layer) --
constexpr int kRouteWaves = 8;  // wavefronts of a route block

// K splits of the router logits: enough (column tile, K range) items for the
// wavefronts of a route block, each range a multiple of 32
static __host__ __device__ inline int route_ks(int E, int d) {
  const int nct = (E + 15) / 16;
  int ks = 1;
  while (nct * ks < kRouteWaves) ks *= 2;
  while (ks > 1 && d % (32 * ks) != 0) ks /= 2;
  return ks;
}

// Eq. (3): best local substitute c(e) = argmin over local j != e with
// Sim[e][j] >= sim_min of Q(e, j) = min(1, phi_scale (1 - Sim[e][j]) / 2),
// ties to the lower j (-1: none), and its Q.  One wavefront per row e: each
// lane scans j = lane, lane + 64, ... in order, then a butterfly takes the
// least (Q, j) pair, which is what a serial scan that keeps the first least
// Q returns (Q is never NaN: fminf(1, NaN) = 1).  Every lane gets the result.
__device__ inline void best_substitute(const float* sim, const uint8_t* local, int E, int e,
                                       float phi_scale, float sim_min, int lane, int& c,
                                       float& q) {
  int best = E;
  float bq = 0.f;
  for (int j = lane; j < E; j += 64) {
    const float sv = sim[(size_t)e * E + j];
    if (j == e || !local[j] || !(sv >= sim_min)) continue;
    const float qj = fminf(1.f, phi_scale * (1.f - sv) * 0.5f);
    if (best == E || qj < bq) {
      best = j;
      bq = qj;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float oq = __shfl_xor(bq, off);
    const int oj = __shfl_xor(best, off);
    if (oj < E && (best == E || oq < bq || (oq == bq && oj < best))) {
      best = oj;
      bq = oq;
    }
  }
  c = best < E ? best : -1;
  q = best < E ? bq : 0.f;
}

// Under look-ahead a remote slot may run its target or any of its local
// substitute candidates (the C = la_subs of least Q with Sim >= sim_min, in
// ascending (Q, j) order): Eq. (34) admits every feasible one, and the
// cost-to-go depends on which expert runs.  One wavefront per row e: C
// rounds, each taking the least (Q, j) after the previous pick (lanes scan
// j = lane, lane + 64, ..., then a butterfly).  c[r] = -1 past the last.
__device__ inline void best_candidates(const float* sim, const uint8_t* local, int E, int e,
                                       float phi_scale, float sim_min, int lane, int C,
                                       int16_t* c, float* q) {
  int pj = -1;
  float pq = -1.f;
  for (int r = 0; r < C; ++r) {
    int best = E;
    float bq = 0.f;
    for (int j = lane; j < E; j += 64) {
      const float sv = sim[(size_t)e * E + j];
      if (j == e || !local[j] || !(sv >= sim_min)) continue;
      const float qj = fminf(1.f, phi_scale * (1.f - sv) * 0.5f);
      const bool after = qj > pq || (qj == pq && j > pj);
      if (after && (best == E || qj < bq)) {
        best = j;
        bq = qj;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float oq = __shfl_xor(bq, off);
      const int oj = __shfl_xor(best, off);
      if (oj < E && (best == E || oq < bq || (oq == bq && oj < best))) {
        best = oj;
        bq = oq;
      }
    }
    if (lane == 0) {
      c[r] = (int16_t)(best < E ? best : -1);
      q[r] = best < E ? bq : 0.f;
    }
    if (best == E) {
      for (int t = r + 1; t < C; ++t)
        if (lane == 0) c[t] = -1;
      break;
    }
    pj = best;
    pq = bq;
  }
}

// ------------------------------------------------ look-ahead (Eq. (39)) --
// Cost-to-go of a token over the later layers of the horizon.  The token
// never moves (one GPU), so it depends on an action only through the
// experts the slots run (sources of the next-layer transitions) and the
// budget the action leaves.  Level j is layer + j; its placement and
// candidate lists are at [j - 1], the transitions out of level j at [j].
// Every slot moves independently (a tuple's probability is the product of
// its slots'); the token's current importance stands in for later ones;
// exits are not predicted.  All arrays live in the route block's LDS.
struct LaView {
  int E, k, B, ntup, C;       // ntup = B^k next-layer tuples; C candidates per row
  const uint8_t* mask;        // [horizon - 1][E]
  const int16_t* cand;        // [horizon - 1][E][C], -1 = none
  const float* candq;         // [horizon - 1][E][C]
  const int16_t* tto;         // [horizon - 1][E * B], -1 = padding
  const float* tp;            // [horizon - 1][E * B]
  const float* theta;         // [horizon - 1]
  const float* slope;         // [horizon - 1]
  float wt, wd, tl, tr;
};

// next-layer tuple `it` of sources x out of level j: targets and probability
// (slot 0 is the most significant digit; padding entries give 0)
__device__ inline float la_tuple(const LaView& v, int j, const int* x, int it, int* tau) {
  const int16_t* to = v.tto + (size_t)j * v.E * v.B;
  const float* pr = v.tp + (size_t)j * v.E * v.B;
  int div = v.ntup;
  float prob = 1.f;
  for (int s = 0; s < v.k; ++s) {
    div /= v.B;
    const int dgt = (it / div) % v.B;
    const int t = to[x[s] * v.B + dgt];
    tau[s] = t < 0 ? 0 : t;
    prob = t < 0 ? 0.f : prob * pr[x[s] * v.B + dgt];
  }
  return prob;
}

// candidates of a row of C entries (-1 padded, ascending Q) that fit the
// budget on their own: D + Q <= b.  An option using any other one is
// infeasible (Q >= 0 only adds), so leaving them out of the enumeration
// changes no decision, and the options that remain keep their order.
__device__ inline int la_nfit(const int16_t* row, const float* rq, int C, float D, float b) {
  int n = 0;
  while (n < C && row[n] >= 0 && D + rq[n] <= b) ++n;
  return n;
}

// Execute option o of a token: slots in rank order, the remote ones with
// candidates (ranks rs[0..nsub), radices rad[u] = 1 + candidates) as mixed-
// radix digits, rs[0] the lowest; digit d > 0 runs candidate d - 1 of the
// slot's row.  Writes the experts run into x and returns the summed Q;
// *mask gets the substituted ranks.
__device__ inline float la_option(int o, int k, const int* tau, const int* rs, const int* rad,
                                  int nsub, const int16_t* cand, const float* candq, int C,
                                  int* x, int* mask) {
  for (int s = 0; s < k; ++s) x[s] = tau[s];
  float sq = 0.f;
  int m = 0;
  for (int u = 0; u < nsub; ++u) {
    const int d = o % rad[u];
    o /= rad[u];
    if (d > 0) {
      const int s = rs[u];
      const size_t at = (size_t)tau[s] * C + d - 1;
      x[s] = cand[at];
      sq += candq[at];
      m |= 1 << s;
    }
  }
  *mask = m;
  return sq;
}

template <int R>
__device__ float la_phi(const LaView& v, int j, const int* x, float D, float I, float b);

// least per-step cost plus cost-to-go (R more levels) of the options at
// level j for routed targets tau with D-hat = D: the rule of Eq. (31),
// (32), (34), (35) and the importance admission at layer + j
template <int R>
__device__ float la_inner(const LaView& v, int j, const int* tau, float D, float I, float b) {
  const int lev = j - 1;
  const uint8_t* mask = v.mask + (size_t)lev * v.E;
  const int16_t* cand = v.cand + (size_t)lev * v.E * v.C;
  const float* candq = v.candq + (size_t)lev * v.E * v.C;
  int n_loc = 0, n_rem = 0, nsub = 0, nopt = 1;
  int rs[TRIMMOE_MAX_LOOKAHEAD_TOPK], rad[TRIMMOE_MAX_LOOKAHEAD_TOPK];
  for (int s = 0; s < v.k; ++s) {
    const int e = tau[s];
    if (mask[e]) {
      ++n_loc;
    } else {
      ++n_rem;
      const int n = la_nfit(cand + (size_t)e * v.C, candq + (size_t)e * v.C, v.C, D, b);
      if (n > 0) {
        rs[nsub] = s;
        rad[nsub++] = 1 + n;
        nopt *= 1 + n;
      }
    }
  }
  float best = __builtin_inff();
  bool all_local = false;
  for (int o = 0; o < nopt; ++o) {
    int x[TRIMMOE_MAX_LOOKAHEAD_TOPK], m;
    const float sq = la_option(o, v.k, tau, rs, rad, nsub, cand, candq, v.C, x, &m);
    if (D + sq <= b) {
      const int ns = __popc(m);
      if (ns == n_rem) all_local = true;
      float f = v.wt * ((float)(n_loc + ns) * v.tl + (float)(n_rem - ns) * v.tr) +
                (b > 0.f ? v.wd * sq / b : 0.f);
      if constexpr (R > 0) f += la_phi<R>(v, j, x, D + sq, I, b);
      best = fminf(best, f);
    }
  }
  if (!all_local) {
    const float lam = fminf(1.f, v.slope[lev] * I);
    if (I <= v.theta[lev] && D + lam <= b) {
      float f = b > 0.f ? v.wd * lam / b : 0.f;
      if constexpr (R > 0) f += la_phi<R>(v, j, tau, D + lam, I, b);
      best = fminf(best, f);
    }
  }
  return best;
}

// Phi^(R): expectation over the next layer's tuples of la_inner<R - 1>
template <int R>
__device__ float la_phi(const LaView& v, int j, const int* x, float D, float I, float b) {
  float acc = 0.f;
  for (int it = 0; it < v.ntup; ++it) {
    int tau[TRIMMOE_MAX_LOOKAHEAD_TOPK];
    const float prob = la_tuple(v, j, x, it, tau);
    if (prob != 0.f) acc += prob * la_inner<R - 1>(v, j + 1, tau, D, I, b);
  }
  return acc;
}

// la_inner at level 1 with `rem` further levels (horizon - 2)
__device__ inline float la_inner_top(const LaView& v, int rem, const int* tau, float D, float I,
                                     float b) {
  if (rem == 0) return la_inner<0>(v, 1, tau, D, I, b);
  if (rem == 1) return la_inner<1>(v, 1, tau, D, I, b);
  return la_inner<2>(v, 1, tau, D, I, b);
}

// options of a token at the layer itself: (1 + C)^k execute options at most,
// plus the skip
__host__ __device__ inline int la_opt_max(int C, int k) {
  int n = 1;
  for (int s = 0; s < k; ++s) n *= 1 + C;
  return n + 1;
}

// A route block's look-ahead LDS, after the logits: 4-byte arrays first,
// then 2-byte, then bytes.  base == NULL only measures.  Returns bytes.
struct LaLds {
  float *tp, *candq, *theta, *slope;  // later layers (see LaView)
  float* candq0;                      // [E][C] this layer's candidate losses
  float* branch;                      // [waves][opt_max B^k] first-level values
  float* phi;                         // [RB][opt_max] cost-to-go per option
  float *tokI, *tokD, *tokB;          // [RB] importance, D-hat, budget
  int* nopt;                          // [RB] execute options
  int16_t *tto, *cand, *cand0;        // cand0: [E][C] this layer's candidates
  uint8_t *mask, *skipok;             // skipok: [RB] skip admitted at this layer
};

__host__ __device__ inline int la_ntup(int B, int k) {
  int n = 1;
  for (int s = 0; s < k; ++s) n *= B;
  return n;
}

__host__ __device__ inline size_t la_carve(char* base, int E, int B, int k, int nlev, int C,
                                           LaLds* o) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* q = base ? base + off : nullptr;
    off += (bytes + 3) & ~(size_t)3;
    return q;
  };
  const size_t opts = (size_t)la_opt_max(C, k);
  LaLds tmp;
  LaLds& L = o ? *o : tmp;
  L.tp = (float*)take((size_t)nlev * E * B * 4);
  L.candq = (float*)take((size_t)nlev * E * C * 4);
  L.theta = (float*)take((size_t)nlev * 4);
  L.slope = (float*)take((size_t)nlev * 4);
  L.candq0 = (float*)take((size_t)E * C * 4);
  L.branch = (float*)take((size_t)kRouteWaves * opts * la_ntup(B, k) * 4);
  L.phi = (float*)take((size_t)RB * opts * 4);
  L.tokI = (float*)take((size_t)RB * 4);
  L.tokD = (float*)take((size_t)RB * 4);
  L.tokB = (float*)take((size_t)RB * 4);
  L.nopt = (int*)take((size_t)RB * 4);
  L.tto = (int16_t*)take((size_t)nlev * E * B * 2);
  L.cand = (int16_t*)take((size_t)nlev * E * C * 2);
  L.cand0 = (int16_t*)take((size_t)E * C * 2);
  L.mask = (uint8_t*)take((size_t)nlev * E);
  L.skipok = (uint8_t*)take((size_t)RB);
  return off;
}

// One block = RB active tokens.  Phase 0: the layer's substitute table
// (and, with look-ahead, the later layers' tables and transitions), one
// wavefront per expert row.  Phase 1: router logits into LDS (MFMA 16x16x32
// bf16 tiles, or fp32 FMA).  Phase 2: top-k and softmax weights with a lane
// group per token, then one thread per token runs the decision; with
// look-ahead (LA) the block first evaluates the cost-to-go of every
// candidate action of its tokens, one wavefront per token, its lanes over
// (action, next-layer tuple) branches.  Phase 3: per-block expert histogram
// for the bucketing.
template <bool BF16, bool LA>
__global__ __launch_bounds__(64 * kRouteWaves) void k_route(LayerParams p) {
  extern __shared__ float zs[];  // [route_ks][RB][E] logits, K partial sums; then LaLds
  __shared__ int s_cnt[TRIMMOE_MAX_EXPERTS];
  __shared__ int16_t s_subc[TRIMMOE_MAX_EXPERTS];  // best substitute (H = 1)
  __shared__ float s_subq[TRIMMOE_MAX_EXPERTS];
  __shared__ int s_xcnt;
  __shared__ int sS[RB][KMAX];
  __shared__ float sW[RB][KMAX];    // slot weights in rank order
  __shared__ int sRsub[RB][KMAX];   // ranks of substitutable remote slots
  __shared__ int sRad[RB][KMAX];    // their radices: 1 + candidates
  __shared__ int sNsub[RB];
  __shared__ int sRx[RB][KMAX];     // merged rows: expert
  __shared__ float sRw[RB][KMAX];   // merged rows: summed weight
  __shared__ float sI[RB];          // importance: summed weight of the picks

  const int n_a = *p.n_active;
  const int base = blockIdx.x * p.rb;
  if (base >= n_a) return;
  const int nt = min(p.rb, n_a - base);
  const int E = p.E, d = p.d, k = p.k;
  for (int e = threadIdx.x; e < E; e += blockDim.x) s_cnt[e] = 0;
  if (threadIdx.x == 0) s_xcnt = 0;
  // the decision's per-expert and per-token inputs, loaded here so that
  // their latency overlaps the substitute table and the router logits
  // instead of adding round trips after them
  __shared__ uint8_t s_local[TRIMMOE_MAX_EXPERTS];
  __shared__ float s_bias[TRIMMOE_MAX_EXPERTS];
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    s_local[e] = p.local_mask[e] ? 1 : 0;
    s_bias[e] = p.b_router ? p.b_router[e] : 0.f;
  }
  int t_pre = 0;
  float d_pre = 0.f, budget_pre = 0.f;
  if ((int)threadIdx.x < nt) {
    t_pre = p.active_idx[base + threadIdx.x];
    d_pre = p.d_acc[t_pre];
    budget_pre = p.budget_tok ? p.budget_tok[t_pre] : p.budget;
  }

  // Eq. (3): the layer's substitute table, one wavefront per expert
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int e = wave; e < E; e += kRouteWaves) {
    int c;
    float q;
    best_substitute(p.sim, p.local_mask, E, e, p.phi_scale, p.sim_min, lane, c, q);
    if (lane == 0) {
      s_subc[e] = (int16_t)c;
      s_subq[e] = q;
    }
  }

  LaLds la;
  LaView lv;
  const int nlev = LA ? p.horizon - 1 : 0;
  if constexpr (LA) {
    const int B = p.trans_b, C = p.la_subs;
    const int ks = BF16 ? route_ks(E, d) : 1;
    la_carve(reinterpret_cast<char*>(zs + (size_t)ks * RB * E), E, B, k, nlev, C, &la);
    // this layer's candidate lists, then the later layers': placement,
    // candidate lists, theta and slope; the transitions out of this layer
    // and every later one but the last
    for (int e = wave; e < E; e += kRouteWaves)
      best_candidates(p.sim, p.local_mask, E, e, p.phi_scale, p.sim_min, lane, C,
                      la.cand0 + (size_t)e * C, la.candq0 + (size_t)e * C);
    for (int idx = wave; idx < nlev * E; idx += kRouteWaves) {
      const int j = idx / E, e = idx % E;
      best_candidates(p.la_sim[j], p.la_mask[j], E, e, p.phi_scale, p.sim_min, lane, C,
                      la.cand + (size_t)idx * C, la.candq + (size_t)idx * C);
      if (lane == 0) la.mask[idx] = p.la_mask[j][e] ? 1 : 0;
    }
    for (int idx = threadIdx.x; idx < nlev * E * B; idx += blockDim.x) {
      const int j = idx / (E * B), r = idx % (E * B);
      const int t = p.la_tto[j][r];
      const bool ok = t >= 0 && t < E;  // anything else is padding
      la.tto[idx] = (int16_t)(ok ? t : -1);
      la.tp[idx] = ok ? p.la_tp[j][r] : 0.f;
    }
    if (threadIdx.x < nlev) {
      la.theta[threadIdx.x] = p.la_theta[threadIdx.x];
      la.slope[threadIdx.x] = p.la_slope[threadIdx.x];
    }
    lv = LaView{E, k, B, la_ntup(B, k), C, la.mask, la.cand, la.candq, la.tto, la.tp,
                la.theta, la.slope, p.omega_t, 1.f - p.omega_t, p.t_local, p.t_remote};
  }

  if constexpr (BF16) {
    // logits of RB = 32 tokens x E experts with 16x16x32 MFMAs: a wavefront
    // takes one 16-expert column tile and one K range for both 16-token row
    // tiles, so each expert row is read once per 32 tokens.  With few column
    // tiles the K range is split (route_ks) so that all wavefronts work;
    // the partial sums are added in K order.  The k-steps run in groups of
    // four whose loads are issued one group ahead (clamped to the last group:
    // in bounds, unused).  Rows past the live tokens / experts load a clamped
    // valid row (never stored).
    const bf16_t* h = static_cast<const bf16_t*>(p.h);
    const bf16_t* W = static_cast<const bf16_t*>(p.w_router);
    const int nct = (E + 15) >> 4, ks = route_ks(E, d), dk = d / ks;
    const int tl = lane & 15, kl = 8 * (lane >> 4);
    const int t0 = p.active_idx[base + min(tl, nt - 1)];
    const int t1 = p.active_idx[base + min(16 + tl, nt - 1)];
    for (int w = wave; w < nct * ks; w += kRouteWaves) {
      const int ct = w % nct, kq = w / nct;
      const int e = ct * 16 + tl;
      const bf16_t* h0 = h + (size_t)t0 * d + kq * dk + kl;
      const bf16_t* h1 = h + (size_t)t1 * d + kq * dk + kl;
      const bf16_t* wr = W + (size_t)min(e, E - 1) * d + kq * dk + kl;
      f32x4_t acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
      const int ng = dk / 128;  // full groups of four k-steps
      if (ng > 0) {
        bf16x8_t a0[4], a1[4], b[4], n0[4], n1[4], nb[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          a0[u] = *reinterpret_cast<const bf16x8_t*>(h0 + 32 * u);
          a1[u] = *reinterpret_cast<const bf16x8_t*>(h1 + 32 * u);
          b[u] = *reinterpret_cast<const bf16x8_t*>(wr + 32 * u);
        }
        for (int g = 0; g < ng; ++g) {
          const int o = min(g + 1, ng - 1) * 128;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            n0[u] = *reinterpret_cast<const bf16x8_t*>(h0 + o + 32 * u);
            n1[u] = *reinterpret_cast<const bf16x8_t*>(h1 + o + 32 * u);
            nb[u] = *reinterpret_cast<const bf16x8_t*>(wr + o + 32 * u);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], b[u], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[u], b[u], acc1, 0, 0, 0);
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            a0[u] = n0[u];
            a1[u] = n1[u];
            b[u] = nb[u];
          }
        }
      }
      // the remaining 0..3 k-steps: every load issued before the first MFMA
      // (offsets clamped to the last k-step: in bounds; their MFMAs are skipped)
      const int rem = (dk - ng * 128) / 32;
      if (rem > 0) {
        bf16x8_t a0[3], a1[3], b[3];
#pragma unroll
        for (int u = 0; u < 3; ++u) {
          const int o = ng * 128 + 32 * min(u, rem - 1);
          a0[u] = *reinterpret_cast<const bf16x8_t*>(h0 + o);
          a1[u] = *reinterpret_cast<const bf16x8_t*>(h1 + o);
          b[u] = *reinterpret_cast<const bf16x8_t*>(wr + o);
        }
#pragma unroll
        for (int u = 0; u < 3; ++u) {
          if (u < rem) {
            acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], b[u], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[u], b[u], acc1, 0, 0, 0);
          }
        }
      }
      // accumulator: column = lane % 16 (expert), row = 4 * (lane / 16) + r (token)
      float* dst = zs + (size_t)kq * RB * E;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 4 * (lane >> 4) + r;
        if (e < E && row < nt) dst[row * E + e] = acc0[r];
        if (e < E && 16 + row < nt) dst[(16 + row) * E + e] = acc1[r];
      }
    }
    if (ks > 1) {
      __syncthreads();
      for (int idx = threadIdx.x; idx < nt * E; idx += blockDim.x) {
        float v = zs[idx];
        for (int q = 1; q < ks; ++q) v += zs[(size_t)q * RB * E + idx];
        zs[idx] = v;
      }
    }
  } else {
    const float* h = static_cast<const float*>(p.h);
    const float* W = static_cast<const float*>(p.w_router);
    for (int idx = threadIdx.x; idx < nt * E; idx += blockDim.x) {
      const int i = idx / E, e = idx % E;
      const int t = p.active_idx[base + i];
      const float* hr = h + (size_t)t * d;
      const float* wr = W + (size_t)e * d;
      float acc = 0.f;
      for (int j = 0; j < d; ++j) acc = fmaf(hr[j], wr[j], acc);
      zs[i * E + e] = acc;
    }
  }
  __syncthreads();

  // Eq. (4) per token, G lanes per token (G the least power of two >= E, at
  // most 64; a wavefront takes 64 / G tokens at once), each lane over
  // experts e = g, g + G, ...: biased logits (NaN ranks last), the top-k in
  // rank order (larger logit first, ties to the lower id; each pick is the
  // best logit ranked strictly after the previous one) and the softmax
  // weights of the picks.  Butterflies stay inside the lane group.
  {
    int G = 1;
    while (G < E && G < 64) G <<= 1;
    const int tpw = 64 / G, g = lane & (G - 1);
    for (int t0 = wave * tpw; t0 < nt; t0 += kRouteWaves * tpw) {
      const int ti = t0 + lane / G;
      if (ti >= nt) continue;
      float* z = zs + ti * E;
      const float ninf = -__builtin_inff();
      for (int e = g; e < E; e += G) {
        const float v = z[e] + s_bias[e];
        z[e] = (v == v) ? v : ninf;
      }
      float vprev = 0.f, vtop[KMAX];
      int iprev = -1;
#pragma unroll
      for (int r = 0; r < KMAX; ++r) {
        if (r >= k) break;
        int be = E;
        float bv = 0.f;
        for (int e = g; e < E; e += G) {
          const float v = z[e];
          const bool after = (r == 0) || (v < vprev) || (v == vprev && e > iprev);
          if (after && (be == E || v > bv)) {
            be = e;
            bv = v;
          }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          if (off >= G) continue;
          const float ov = __shfl_xor(bv, off);
          const int oe = __shfl_xor(be, off);
          if (oe < E && (be == E || ov > bv || (ov == bv && oe < be))) {
            be = oe;
            bv = ov;
          }
        }
        if (g == 0) sS[ti][r] = be < E ? be : -1;
        vtop[r] = bv;
        vprev = bv;
        iprev = be;
      }
      // p_e = exp(z_e - max) / sum over all E; the lane partials of the sum
      // are added in a fixed butterfly, so every lane of the group holds it
      const float zmax = vtop[0];
      float sum = 0.f;
      for (int e = g; e < E; e += G) sum += expf(z[e] - zmax);
#pragma unroll
      for (int off = 32; off > 0; off >>= 1)
        if (off < G) sum += __shfl_xor(sum, off);
      if (g == 0) {
        float imp = 0.f;
#pragma unroll
        for (int r = 0; r < KMAX; ++r) {
          if (r >= k) break;
          const float pr = expf(vtop[r] - zmax) / sum;
          sW[ti][r] = pr;
          imp += pr;
        }
        if (p.normalize)
          for (int r = 0; r < k; ++r) sW[ti][r] = sW[ti][r] / imp;
        sI[ti] = imp;
      }
    }
  }
  __syncthreads();

  const int i = threadIdx.x;
  int pos = 0, t = 0, n_loc = 0, n_rem = 0, nsub = 0, nopt = 1;
  float I = 0.f, budget = 0.f, D = 0.f;
  // each remote slot's candidates: its best substitute at H = 1 (A13), its
  // C = la_subs least-loss local candidates under look-ahead
  const int C = LA ? p.la_subs : 1;
  const int16_t* cand = LA ? la.cand0 : s_subc;
  const float* candq = LA ? la.candq0 : s_subq;
  if (i < nt) {
    pos = base + i;
    t = t_pre;
    I = sI[i];

    budget = budget_pre;
    D = d_pre;
    // resolve slots: local exact, or remote with or without candidates that
    // fit the budget
    for (int r = 0; r < k; ++r) {
      const int e = sS[i][r];
      if (s_local[e]) {
        ++n_loc;
      } else {
        ++n_rem;
        const int n = la_nfit(cand + (size_t)e * C, candq + (size_t)e * C, C, D, budget);
        if (n > 0) {
          sRsub[i][nsub] = r;
          sRad[i][nsub++] = 1 + n;
          nopt *= 1 + n;
        }
      }
    }
    sNsub[i] = nsub;
  }

  if constexpr (LA) {
    // Eq. (39)-(40): cost-to-go of every candidate action of the block's
    // tokens.  Options 0 .. nopt - 1 execute (la_option's mixed-radix
    // numbering over the substitutable remote slots); option nopt skips.
    // Every branch (option, next-layer tuple) is one lane's work; a
    // wavefront takes one token at a time and sums the branches of each
    // option in tuple order.
    const int opt_max = la_opt_max(C, k);
    if (i < nt) {
      la.tokI[i] = I;
      la.tokD[i] = D;
      la.tokB[i] = budget;
      la.nopt[i] = nopt;
      // the skip is a candidate iff Gamma > 0 (no feasible all-local
      // assignment, Eq. (35): the cheapest one takes every slot's least-loss
      // candidate), I <= theta and the budget admits Lambda
      float sq_all = 0.f;
      for (int u = 0; u < nsub; ++u) sq_all += candq[(size_t)sS[i][sRsub[i][u]] * C];
      const bool all_local = nsub == n_rem && D + sq_all <= budget;  // as the enumeration finds
      const float lam = fminf(1.f, p.skip_slope * I);
      la.skipok[i] = !all_local && I <= p.theta && D + lam <= budget;
    }
    __syncthreads();
    // tokens in flight per round and wavefronts per token (a block of few
    // tokens gives each token several wavefronts)
    const int tpr = min(p.rb, kRouteWaves), wpt = kRouteWaves / tpr;
    const int slot = wave / wpt, wsub = wave % wpt;
    const int ntup = lv.ntup, rem = nlev - 1;
    float* br = la.branch + (size_t)slot * opt_max * ntup;
    for (int r = 0; r * tpr < p.rb; ++r) {
      const int ti = slot + tpr * r;
      const int nall = ti < nt ? la.nopt[ti] + 1 : 0;  // with the skip
      for (int it = wsub * 64 + lane; it < nall * ntup; it += wpt * 64) {
        const int o = it / ntup, tup = it % ntup;
        const float Dt = la.tokD[ti], bt = la.tokB[ti], It = la.tokI[ti];
        int x[TRIMMOE_MAX_LOOKAHEAD_TOPK];
        float charge;
        bool feasible;
        if (o < nall - 1) {
          int m;
          charge = la_option(o, k, sS[ti], sRsub[ti], sRad[ti], sNsub[ti], cand, candq, C, x,
                             &m);
          feasible = Dt + charge <= bt;
        } else {
          for (int s = 0; s < k; ++s) x[s] = sS[ti][s];
          charge = fminf(1.f, p.skip_slope * It);
          feasible = la.skipok[ti] != 0;
        }
        float val = 0.f;
        if (feasible) {
          int tau[TRIMMOE_MAX_LOOKAHEAD_TOPK];
          const float prob = la_tuple(lv, 0, x, tup, tau);
          if (prob != 0.f) val = prob * la_inner_top(lv, rem, tau, Dt + charge, It, bt);
        }
        br[it] = val;
      }
      __syncthreads();
      if (wsub == 0)
        for (int o = lane; o < nall; o += 64) {
          float acc = 0.f;
          for (int u = 0; u < ntup; ++u) acc += br[o * ntup + u];
          la.phi[ti * opt_max + o] = acc;
        }
      __syncthreads();
    }
  }

  if (i < nt) {
    const float wt = p.omega_t, wd = 1.f - p.omega_t;
    const float* phi = LA ? la.phi + i * la_opt_max(C, k) : nullptr;
    // Eq. (34) + Eq. (31): every way of serving the remote slots (target or
    // a candidate) within the budget
    bool have = false, all_local = false;
    float bf = 0.f, bsq = 0.f;
    int bns = 0, bmask = 0, bo = 0, bx[KMAX];
    for (int o = 0; o < nopt; ++o) {
      int x[KMAX], mask;
      const float sq = la_option(o, k, sS[i], sRsub[i], sRad[i], nsub, cand, candq, C, x, &mask);
      if (!(D + sq <= budget)) continue;
      const int ns = __popc(mask);
      if (ns == n_rem) all_local = true;
      float f = wt * ((float)(n_loc + ns) * p.t_local + (float)(n_rem - ns) * p.t_remote) +
                (budget > 0.f ? wd * sq / budget : 0.f);
      if constexpr (LA) f += phi[o];  // Eq. (40): per-step cost + cost-to-go
      const bool better =
          !have || f < bf ||
          (f == bf && (ns < bns || (ns == bns && (mask < bmask || (mask == bmask && o < bo)))));
      if (better) {
        have = true;
        bf = f;
        bns = ns;
        bmask = mask;
        bo = o;
        bsq = sq;
        for (int s = 0; s < k; ++s) bx[s] = x[s];
      }
    }
    // Eq. (35) + importance threshold + Eq. (32): skip admission and choice
    const float lam = fminf(1.f, p.skip_slope * I);
    bool skip = false;
    if (!all_local && I <= p.theta && D + lam <= budget) {
      float fs = budget > 0.f ? wd * lam / budget : 0.f;
      if constexpr (LA) fs += phi[nopt];
      skip = fs < bf;
    }
    if (!have) skip = false;  // unreachable: the empty assignment is feasible

    // per-slot execution and merged rows (a substitute keeps its target's weight)
    int nrows = 0, nsubst = 0, nremote = 0, nroute_remote = 0;
    for (int r = 0; r < k; ++r) {
      const int e = sS[i][r];
      nroute_remote += !s_local[e];
      int x = -1, kind = TRIMMOE_KIND_NONE;
      if (!skip) {
        if ((bmask >> r) & 1) {
          x = bx[r];
          kind = TRIMMOE_KIND_SUBST;
          ++nsubst;
        } else {
          x = e;
          kind = s_local[e] ? TRIMMOE_KIND_LOCAL : TRIMMOE_KIND_REMOTE;
          if (kind == TRIMMOE_KIND_REMOTE) ++nremote;
        }
        int j = 0;
        for (; j < nrows; ++j)
          if (sRx[i][j] == x) break;
        if (j < nrows) {
          sRw[i][j] += sW[i][r];  // merge duplicates in rank order
        } else {
          sRx[i][nrows] = x;
          sRw[i][nrows] = sW[i][r];
          ++nrows;
        }
      }
      if (p.tr_target) p.tr_target[(size_t)t * k + r] = (int16_t)e;
      if (p.tr_exec) p.tr_exec[(size_t)t * k + r] = (int16_t)x;
      if (p.tr_kind) p.tr_kind[(size_t)t * k + r] = (int8_t)kind;
      if (p.tr_gate) p.tr_gate[(size_t)t * k + r] = sW[i][r];
    }
    for (int j = 0; j < k; ++j) {
      p.tok_exec[(size_t)pos * k + j] = j < nrows ? sRx[i][j] : -1;
      p.tok_w[(size_t)pos * k + j] = j < nrows ? sRw[i][j] : 0.f;
    }
    const float dnew = D + (skip ? lam : bsq);  // Eq. (41) / (42)
    p.d_acc[t] = dnew;
    p.tok_action[pos] = skip ? TRIMMOE_ACT_SKIP : TRIMMOE_ACT_EXEC;
    p.tok_keep[pos] = 1;
    for (int j = 0; j < nrows; ++j) atomicAdd(&s_cnt[sRx[i][j]], 1);
    if (!skip) atomicAdd(&s_xcnt, 1);
    if (p.tr_action) p.tr_action[t] = skip ? TRIMMOE_ACT_SKIP : TRIMMOE_ACT_EXEC;
    if (p.tr_importance) p.tr_importance[t] = I;
    if (p.tr_d_acc) p.tr_d_acc[t] = dnew;
    if (p.tr_counters) {
      atomicAdd(&p.tr_counters[0], 1);
      atomicAdd(&p.tr_counters[skip ? 2 : 1], 1);
      if (nsubst) atomicAdd(&p.tr_counters[4], nsubst);
      if (nremote) atomicAdd(&p.tr_counters[5], nremote);
      if (nroute_remote) atomicAdd(&p.tr_counters[8], nroute_remote);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) p.blk_cnt[(size_t)blockIdx.x * E + e] = s_cnt[e];
  if (threadIdx.x == 0) p.blk_xcnt[blockIdx.x] = s_xcnt;
}

// ------------------------------------------- expert offsets and tile list --
// Exclusive scan of a value per thread over a 1024-thread block (wavefront
// prefix with shuffles, then the 16 wavefront totals); returns the block
// total in *total.
__device__ __forceinline__ int block_exclusive_scan(int v, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
      const int c = s_wave[w];
      s_wave[w] = run;
      run += c;
    }
    s_wave[16] = run;
  }
  __syncthreads();
  const int r = s_wave[wave] + x - v;
  *total = s_wave[16];
  __syncthreads();
  return r;
}

// Per-expert offsets of every route block's rows, expert row offsets, the
// grouped-GEMM tile list and the executed-token offsets, in one block of
// 1024 threads: thread (segment g, expert e) sums its run of route blocks,
// the segments of an expert are scanned in order, and the expert totals
// and block exec counts go through block-wide scans.
__global__ __launch_bounds__(1024) void k_scan(LayerParams p) {
  __shared__ int s_seg[1024];
  __shared__ int s_wave[17];
  __shared__ int s_tot[TRIMMOE_MAX_EXPERTS];
  __shared__ int s_off[TRIMMOE_MAX_EXPERTS];
  __shared__ int s_toff[TRIMMOE_MAX_EXPERTS];
  const int n_a = *p.n_active;
  const int nb = (n_a + p.rb - 1) / p.rb;
  const int E = p.E;
  int ep = 1;
  while (ep < E) ep <<= 1;
  const int S = 1024 / ep;               // segments per expert
  const int L = (nb + S - 1) / S;        // route blocks per segment
  const int e = threadIdx.x % ep, g = threadIdx.x / ep;
  const int b0 = g * L, b1 = min(nb, b0 + L);
  // the counts of a segment are read in chunks of 8, every load of a chunk
  // before its stores, so the loads of a chunk are in flight together
  constexpr int CH = 8;
  int sum = 0;
  if (e < E)
    for (int b = b0; b < b1; b += CH) {
      int c[CH];
#pragma unroll
      for (int u = 0; u < CH; ++u) c[u] = b + u < b1 ? p.blk_cnt[(size_t)(b + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < CH; ++u) sum += c[u];
    }
  s_seg[g * ep + e] = sum;
  __syncthreads();
  if (e < E) {
    int run = 0;
    for (int q = 0; q < g; ++q) run += s_seg[q * ep + e];
    for (int b = b0; b < b1; b += CH) {
      int c[CH];
#pragma unroll
      for (int u = 0; u < CH; ++u) c[u] = b + u < b1 ? p.blk_cnt[(size_t)(b + u) * E + e] : 0;
#pragma unroll
      for (int u = 0; u < CH; ++u)
        if (b + u < b1) {
          p.blk_off[(size_t)(b + u) * E + e] = run;
          run += c[u];
        }
    }
    if (g == S - 1) s_tot[e] = run;
  }
  __syncthreads();
  // expert row offsets and tile offsets (threads 0..E-1 carry one expert)
  int total = 0, ttotal = 0;
  const int tot = threadIdx.x < E ? s_tot[threadIdx.x] : 0;
  const int off = block_exclusive_scan(tot, s_wave, &total);
  const int nt_e = (tot + p.bm - 1) / p.bm;
  const int toff = block_exclusive_scan(nt_e, s_wave, &ttotal);
  if (threadIdx.x < E) {
    s_off[threadIdx.x] = off;
    s_toff[threadIdx.x] = toff;
    p.exp_off[threadIdx.x] = off;
    p.exp_toff[threadIdx.x] = toff;
    for (int u = 0; u < nt_e; ++u)
      p.tiles[toff + u] = make_int4(threadIdx.x, off + u * p.bm, off + tot, 0);
  }
  // executed-token offsets of the route blocks
  int xrun = 0;
  for (int c0 = 0; c0 < nb; c0 += 1024) {
    const int b = c0 + threadIdx.x;
    const int v = b < nb ? p.blk_xcnt[b] : 0;
    int chunk = 0;
    const int o = block_exclusive_scan(v, s_wave, &chunk);
    if (b < nb) p.blk_xoff[b] = xrun + o;
    xrun += chunk;
  }
  if (threadIdx.x == 0) {
    p.exp_off[E] = total;
    p.counts[kCntRows] = total;
    int nt_all = 0, distinct = 0;
    for (int x = 0; x < E; ++x) {
      nt_all += (s_tot[x] + p.bm - 1) / p.bm;
      distinct += s_tot[x] > 0;
    }
    p.counts[kCntTiles] = nt_all;
    p.counts[kCntExec] = xrun;
    if (p.tr_counters) {
      p.tr_counters[6] = total;
      p.tr_counters[7] = distinct;
    }
  }
}

// ------------------------------------------------- stable row permutation --
// bounds of the fused scan: block histogram entries (route blocks x experts)
// and route blocks a bucket block holds in LDS
constexpr int kFusedScanEntries = 4096;
constexpr int kFusedScanBlocks = 1024;
// Row of (active position pos, merged row j with expert e) =
//   exp_off[e] + (rows of e in earlier blocks) + (rows of e earlier in block),
// i.e. rows of one expert stay in token order.  No hidden state is copied:
// row_src[row] names the token whose h row the grouped GEMM gathers, and
// exec_list / exec_pos list the executed tokens in active order.
//
// FUSED (small route grids, bucket_fused_scan): no k_scan launch.  Every
// bucket block reads all block histograms into LDS and derives the offsets
// it needs (its own per-expert run starts, the expert row offsets, its
// executed-token offset) with the same integer sums k_scan makes; block 0
// also writes the layer's expert offsets, tile list and counters.
__device__ __forceinline__ void fused_scan(const LayerParams& p, int nb, int* s_cnt, int* s_x,
                                           int* s_seg, int* s_wave, int* s_off, int* s_xoff) {
  const int E = p.E, tid = threadIdx.x, b_me = blockIdx.x;
  const int n_c = nb * E;
  for (int i = tid; i < n_c; i += blockDim.x) s_cnt[i] = p.blk_cnt[i];
  for (int b = tid; b < nb; b += blockDim.x) s_x[b] = p.blk_xcnt[b];
  __syncthreads();
  // thread (segment g, expert e) sums its run of blocks; the segment holding
  // this block also sums the blocks before it
  int ep = 1;
  while (ep < E) ep <<= 1;
  const int S = blockDim.x / ep, L = (nb + S - 1) / S;
  const int e = tid % ep, g = tid / ep;
  const int b0 = g * L, b1 = min(nb, b0 + L);
  int sum = 0, before = 0;
  if (e < E)
    for (int b = b0; b < b1; ++b) {
      if (b == b_me) before = sum;
      sum += s_cnt[b * E + e];
    }
  s_seg[g * ep + e] = sum;
  if (e < E && b_me >= b0 && b_me < b1) s_off[e] = before;  // in-segment part
  __syncthreads();
  int tot = 0, pre = 0;
  if (tid < E) {
    const int gme = L > 0 ? b_me / L : 0;
    for (int q = 0; q < S; ++q) {
      const int v = s_seg[q * ep + tid];
      if (q < gme) pre += v;
      tot += v;
    }
    pre += b_me < nb ? s_off[tid] : 0;
  }
  __syncthreads();
  int total = 0, ttotal = 0;
  const int off = block_exclusive_scan(tot, s_wave, &total);
  const int nt_e = (tot + p.bm - 1) / p.bm;
  const int toff = block_exclusive_scan(nt_e, s_wave, &ttotal);
  if (tid < E) s_off[tid] = off + pre;
  // executed-token offset of this block, and the layer's executed total
  int xrun = 0;
  for (int c0 = 0; c0 < nb; c0 += blockDim.x) {
    const int b = c0 + tid;
    const int v = b < nb ? s_x[b] : 0;
    int chunk = 0;
    const int o = block_exclusive_scan(v, s_wave, &chunk);
    if (b == b_me) *s_xoff = xrun + o;
    xrun += chunk;
  }
  if (b_me == 0) {
    if (tid < E) {
      p.exp_off[tid] = off;
      p.exp_toff[tid] = toff;
      for (int u = 0; u < nt_e; ++u) p.tiles[toff + u] = make_int4(tid, off + u * p.bm, off + tot, 0);
    }
    const int distinct = __syncthreads_count(tid < E && tot > 0);
    if (tid == 0) {
      p.exp_off[E] = total;
      p.counts[kCntRows] = total;
      p.counts[kCntTiles] = ttotal;
      p.counts[kCntExec] = xrun;
      if (p.tr_counters) {
        p.tr_counters[6] = total;
        p.tr_counters[7] = distinct;
      }
    }
  }
}

template <bool FUSED>
__global__ __launch_bounds__(256) void k_bucket(LayerParams p) {
  static_assert(RB <= 32 && RB * KMAX <= 256, "token masks and one thread per slot");
  __shared__ unsigned s_emask[TRIMMOE_MAX_EXPERTS];  // block tokens holding a row of e
  __shared__ int s_off[TRIMMOE_MAX_EXPERTS];         // the block's first row of e
  __shared__ unsigned s_xmask;                       // block tokens that execute
  __shared__ int s_xoff;                             // the block's first executed token
  const int n_a = *p.n_active;
  const int base = blockIdx.x * p.rb;
  const int k = p.k, E = p.E;
  const int tid = threadIdx.x;
  if constexpr (FUSED) {
    __shared__ int s_cnt[kFusedScanEntries];
    __shared__ int s_x[kFusedScanBlocks];
    __shared__ int s_seg[256];
    __shared__ int s_wave[17];
    const int nb = (n_a + p.rb - 1) / p.rb;
    if (blockIdx.x > 0 && base >= n_a) return;  // block 0 writes the layer's offsets
    fused_scan(p, nb, s_cnt, s_x, s_seg, s_wave, s_off, &s_xoff);
    if (base >= n_a) return;
    for (int e = tid; e < E; e += blockDim.x) s_emask[e] = 0u;
  } else {
    if (base >= n_a) return;
    for (int e = tid; e < E; e += blockDim.x) {
      s_emask[e] = 0u;
      s_off[e] = p.exp_off[e] + p.blk_off[(size_t)blockIdx.x * E + e];
    }
    if (tid == 0) s_xoff = p.blk_xoff[blockIdx.x];
  }
  const int nt = min(p.rb, n_a - base);
  if (tid == 0) s_xmask = 0u;
  __syncthreads();
  // thread (token i, slot j); a token's merged rows are distinct experts
  // packed at the front of its slots, so the rows of e before token i's
  // are one per earlier block token that holds e
  const int i = tid / k, j = tid - (tid / k) * k;
  const int pos = base + i;
  int e = -1;
  if (tid < nt * k) {
    e = p.tok_exec[(size_t)pos * k + j];
    if (e >= 0) atomicOr(&s_emask[e], 1u << i);
  }
  if (tid < nt && p.tok_action[base + tid] == TRIMMOE_ACT_EXEC) atomicOr(&s_xmask, 1u << tid);
  __syncthreads();
  if (e >= 0) {
    const int row = s_off[e] + __popc(s_emask[e] & ((1u << i) - 1u));
    p.tok_row[(size_t)pos * k + j] = row;
    p.row_src[row] = p.active_idx[pos];
  }
  if (tid < nt && ((s_xmask >> tid) & 1u)) {
    const int xidx = s_xoff + __popc(s_xmask & ((1u << tid) - 1u));
    p.exec_list[xidx] = p.active_idx[base + tid];
    p.exec_pos[xidx] = base + tid;
  }
}

// ------------------------------------------------ weighted combine (R4) --
// h[t] <- round(h[t] + sum_rows w * Y[row] (+ shared Y)), summed in rank
// order in fp32 (each row's K-split slices first, in slice order) and
// rounded once; the new row also goes to hx, the exit head's compact input.
// One thread handles 8 consecutive features of one token.  Skipped and
// inactive tokens are untouched.
template <typename ST>
__global__ __launch_bounds__(256) void k_combine(LayerParams p) {
  const int n_x = p.counts[kCntExec];
  const int per_tok = p.d / 8;
  const size_t total = (size_t)n_x * per_tok;
  ST* h = static_cast<ST*>(p.h);
  for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (size_t)gridDim.x * blockDim.x) {
    const int j = (int)(idx / per_tok), c = (int)(idx % per_tok) * 8;
    const int pos = p.exec_pos[j];
    const int t = p.exec_list[j];
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.f;
    for (int s = 0; s < p.k; ++s) {
      const int e = p.tok_exec[(size_t)pos * p.k + s];
      if (e < 0) break;
      const int row = p.tok_row[(size_t)pos * p.k + s];
      const float w = p.tok_w[(size_t)pos * p.k + s];
      const float4* y = reinterpret_cast<const float4*>(p.y_buf + (size_t)row * p.d + c);
      float4 v0 = y[0], v1 = y[1];
      for (int q = 1; q < p.down_splits; ++q) {
        const float4* yq = reinterpret_cast<const float4*>(p.y_buf + q * p.y_split_stride +
                                                           (size_t)row * p.d + c);
        const float4 a0 = yq[0], a1 = yq[1];
        v0.x += a0.x; v0.y += a0.y; v0.z += a0.z; v0.w += a0.w;
        v1.x += a1.x; v1.y += a1.y; v1.z += a1.z; v1.w += a1.w;
      }
      // large-group down GEMM: the later K pieces of a cut tile, in order
      if (p.sk_flag) {
        const int rt = row - p.exp_off[e];
        const int mt = p.exp_toff[e] + rt / p.bm;
        const int word = p.sk_flag[mt * ((p.d + 255) >> 8) + (c >> 8)];
        for (int q = 1; q < (word & 15); ++q) {
          const float4* yq = reinterpret_cast<const float4*>(
              p.sk_part + (size_t)((word >> 4) + q - 1) * 65536 + (rt % p.bm) * 256 + (c & 255));
          const float4 a0 = yq[0], a1 = yq[1];
          v0.x += a0.x; v0.y += a0.y; v0.z += a0.z; v0.w += a0.w;
          v1.x += a1.x; v1.y += a1.y; v1.z += a1.z; v1.w += a1.w;
        }
      }
      acc[0] += w * v0.x; acc[1] += w * v0.y; acc[2] += w * v0.z; acc[3] += w * v0.w;
      acc[4] += w * v1.x; acc[5] += w * v1.y; acc[6] += w * v1.z; acc[7] += w * v1.w;
    }
    if (p.Fs > 0) {
      const float4* ys = reinterpret_cast<const float4*>(p.y_s + (size_t)j * p.d + c);
      const float4 a0 = ys[0], a1 = ys[1];
      acc[0] += a0.x; acc[1] += a0.y; acc[2] += a0.z; acc[3] += a0.w;
      acc[4] += a1.x; acc[5] += a1.y; acc[6] += a1.z; acc[7] += a1.w;
    }
    // 8 elements = 16 bytes (bf16) or 32 bytes (fp32) per row access: rows
    // start at multiples of d (a multiple of 8) in 16-byte aligned buffers
    ST* hr = h + (size_t)t * p.d + c;
    ST* xr = static_cast<ST*>(p.hx) + (size_t)j * p.d + c;
    if constexpr (sizeof(ST) == 2) {
      union {
        uint4 v;
        ST e[8];
      } in, out;
      in.v = *reinterpret_cast<const uint4*>(hr);
#pragma unroll
      for (int u = 0; u < 8; ++u) out.e[u] = from_f32<ST>(to_f32<ST>(in.e[u]) + acc[u]);
      *reinterpret_cast<uint4*>(hr) = out.v;
      *reinterpret_cast<uint4*>(xr) = out.v;
    } else {
      float4* h4 = reinterpret_cast<float4*>(hr);
      float4* x4 = reinterpret_cast<float4*>(xr);
      float4 a0 = h4[0], a1 = h4[1];
      a0.x += acc[0]; a0.y += acc[1]; a0.z += acc[2]; a0.w += acc[3];
      a1.x += acc[4]; a1.y += acc[5]; a1.z += acc[6]; a1.w += acc[7];
      h4[0] = a0; h4[1] = a1;
      x4[0] = a0; x4[1] = a1;
    }
  }
}

// -------------------------------------------- exit confidence and gate --
// xi = 1 / sum_tiles s_i 2^(m_i - M) (softmax max-probability from the
// per-tile partial maxima, kept in base 2, and sums), or sigmoid of the
// single logit;
// exit iff xi >= p_J (Eq. (8)).  One wavefront per executed token.
__global__ __launch_bounds__(256) void k_exit_reduce(LayerParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + wave;
  const int n_x = p.counts[kCntExec];
  if (j >= n_x) return;
  const int nv = p.n_vtiles;
  const float2* pr = p.partials + (size_t)j * nv;
  // the token's ids are read first, so their latency overlaps the partials'
  const int t = p.exec_list[j];
  const int pos = p.exec_pos[j];
  float m = -__builtin_inff();
  for (int u = lane; u < nv; u += 64) m = fmaxf(m, pr[u].x);
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  // partial maxima are in base 2 (max z * log2 e)
  float s = 0.f;
  for (int u = lane; u < nv; u += 64) {
    const float2 v = pr[u];
    if (v.y > 0.f) s += v.y * exp2f(v.x - m);
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) {
    const float xi = p.conf_mode == TRIMMOE_CONF_SIGMOID
                         ? 1.f / (1.f + exp2f(-m))  // m = logit * log2 e
                         : 1.f / s;
    p.xi[t] = xi;
    if (p.tr_xi) p.tr_xi[t] = xi;
    const float pj = p.p_exit_tok ? p.p_exit_tok[t] : p.p_exit;
    if (xi >= pj) {
      p.exit_layer[t] = p.layer;
      p.tok_keep[pos] = 0;
    }
  }
}

// ------------------------------------- stable compaction of active list --
// In place, one block, chunk by chunk: every write of a chunk lands before
// the chunk's own start, and all its reads finish before the first write.
// Positions come from a wavefront ballot/popcount plus the scanned
// wavefront totals.
__global__ __launch_bounds__(1024) void k_compact(LayerParams p) {
  __shared__ int s_wave[17];
  const int n_a = *p.n_active;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int out = 0;
  for (int c0 = 0; c0 < n_a; c0 += 1024) {
    const int i = c0 + threadIdx.x;
    const bool keep = i < n_a && p.tok_keep[i];
    const int idx = i < n_a ? p.active_idx[i] : 0;
    const unsigned long long m = __ballot(keep);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[wave] = __popcll(m);
    __syncthreads();
    if (threadIdx.x == 0) {
      int run = 0;
      for (int w = 0; w < 16; ++w) {
        const int c = s_wave[w];
        s_wave[w] = run;
        run += c;
      }
      s_wave[16] = run;
    }
    __syncthreads();
    if (keep) p.active_idx[out + s_wave[wave] + before] = idx;
    out += s_wave[16];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *p.n_active = out;
    if (p.tr_counters) p.tr_counters[3] = n_a - out;
  }
}

// -------------------------------------------------------------- launchers --
static inline int cdiv(int a, int b) { return (a + b - 1) / b; }

hipError_t launch_state_reset(const trimmoe_model* m, const trimmoe_state* s, hipStream_t st) {
  const int T = s->n_tokens;
  hipLaunchKernelGGL(k_state_reset, dim3(cdiv(T > 0 ? T : 1, 256)), dim3(256), 0, st, T,
                     m->n_layers, s->d_acc, s->active_idx, s->n_active, s->exit_layer, s->xi);
  return hipGetLastError();
}

hipError_t launch_trace_fill(const LayerParams& p, int n_layers, hipStream_t st) {
  hipLaunchKernelGGL(k_trace_fill, dim3(cdiv(p.T > 0 ? p.T : 1, 256), n_layers), dim3(256), 0, st,
                     p);
  return hipGetLastError();
}

size_t route_lds_bytes(bool bf16, int E, int d, int horizon, int trans_b, int k, int la_subs) {
  size_t lds = (size_t)(bf16 ? route_ks(E, d) : 1) * RB * E * sizeof(float);
  if (horizon > 1) lds += la_carve(nullptr, E, trans_b, k, horizon - 1, la_subs, nullptr);
  return lds;
}

hipError_t launch_route(const LayerParams& p, bool bf16, hipStream_t st) {
  const int nb = cdiv(p.T, p.rb);
  const size_t lds = route_lds_bytes(bf16, p.E, p.d, p.horizon, p.trans_b, p.k, p.la_subs);
  const dim3 grid(nb), block(64 * kRouteWaves);
  if (p.horizon > 1) {
    auto kern = bf16 ? k_route<true, true> : k_route<false, true>;
    if (lds > 65536) {
      const hipError_t e =
          hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, grid, block, lds, st, p);
  } else if (bf16) {
    hipLaunchKernelGGL((k_route<true, false>), grid, block, lds, st, p);
  } else {
    hipLaunchKernelGGL((k_route<false, false>), grid, block, lds, st, p);
  }
  return hipGetLastError();
}

// the bucket blocks derive the scan themselves when every block histogram
// fits in their LDS (one launch fewer per layer)
static bool bucket_fused_scan(const LayerParams& p) {
  const int nb = cdiv(p.T, p.rb);
  return nb <= kFusedScanBlocks && (size_t)nb * p.E <= (size_t)kFusedScanEntries;
}

hipError_t launch_scan(const LayerParams& p, hipStream_t st) {
  if (bucket_fused_scan(p)) return hipSuccess;
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_bucket(const LayerParams& p, hipStream_t st) {
  if (bucket_fused_scan(p))
    hipLaunchKernelGGL(k_bucket<true>, dim3(cdiv(p.T, p.rb)), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_bucket<false>, dim3(cdiv(p.T, p.rb)), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_combine(const LayerParams& p, bool bf16, hipStream_t st) {
  const int nb = cdiv(p.T * (p.d / 8), 256) < 4096 ? cdiv(p.T * (p.d / 8), 256) : 4096;
  if (bf16)
    hipLaunchKernelGGL(k_combine<bf16_t>, dim3(nb), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_combine<float>, dim3(nb), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_exit_reduce(const LayerParams& p, hipStream_t st) {
  hipLaunchKernelGGL(k_exit_reduce, dim3(cdiv(p.T, 4)), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_compact(const LayerParams& p, hipStream_t st) {
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, st, p);
  return hipGetLastError();
}


// --------------------------------- runtime feedback observations (window) --
// Sums over one stack pass, added to stats[0..5] = tokens, exits, confidence
// at exit, budget utilisation D-hat / budget, executed-slot delay, and the
// reference delay of full-depth exact execution (Sec. V-D Eq. (37), Sec. V-F
// Eq. (43), normalised as in Eq. (21)).  The reference prices each layer at
// T k slots of the mean routed-target delay of the tokens active there; a
// layer no token reached takes the mean over the whole pass.  One block,
// fixed summation order: repeated runs give identical sums.
__global__ __launch_bounds__(1024) void k_window_stats(WindowArgs w) {
  __shared__ double s_red[3][1024];
  double v[3] = {0.0, 0.0, 0.0};  // exits, confidence at exit, utilisation
  for (int t = threadIdx.x; t < w.T; t += 1024) {
    if (w.exit_layer[t] < w.N) {
      v[0] += 1.0;
      v[1] += (double)w.xi[t];
    }
    const double b = w.budget_tok ? (double)w.budget_tok[t] : (double)w.budget;
    if (b > 0.0) v[2] += (double)w.d_acc[t] / b;
  }
#pragma unroll
  for (int i = 0; i < 3; ++i) s_red[i][threadIdx.x] = v[i];
  __syncthreads();
  for (int stride = 512; stride > 0; stride >>= 1) {
    if (threadIdx.x < stride)
#pragma unroll
      for (int i = 0; i < 3; ++i) s_red[i][threadIdx.x] += s_red[i][threadIdx.x + stride];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double tl = w.t_local, tr = w.t_remote;
    double delay = 0.0, routed = 0.0, routed_remote = 0.0;
    for (int l = 0; l < w.N; ++l) {
      // executed tokens, remote exact slots; routed slots, their remote targets
      const int* c = w.counters + kCounters * l;
      const double slots = (double)c[1] * w.k;
      delay += (slots - c[5]) * tl + (double)c[5] * tr;
      routed += (double)c[0] * w.k;
      routed_remote += (double)c[8];
    }
    double ref = 0.0;
    if (routed > 0.0) {
      const double pooled = ((routed - routed_remote) * tl + routed_remote * tr) / routed;
      for (int l = 0; l < w.N; ++l) {
        const int* c = w.counters + kCounters * l;
        const double r = (double)c[0] * w.k;
        const double mean = r > 0.0 ? ((r - c[8]) * tl + (double)c[8] * tr) / r : pooled;
        ref += (double)w.T * w.k * mean;
      }
    }
    w.stats[0] += (double)w.T;
    w.stats[1] += s_red[0][0];
    w.stats[2] += s_red[1][0];
    w.stats[3] += s_red[2][0];
    w.stats[4] += delay;
    w.stats[5] += ref;
  }
}

hipError_t launch_window_stats(const WindowArgs& w, hipStream_t st) {
  hipLaunchKernelGGL(k_window_stats, dim3(1), dim3(1024), 0, st, w);
  return hipGetLastError();
}

}  // namespace trimmoe
