// C ABI of libtrimmoe: argument validation, workspace carving and the
// per-layer launch sequence of the adaptive-depth MoE step.  The declared
// interface and its conventions are in include/trimmoe.h.
//
// Launch sequence of one layer, all on the caller's stream and sized for
// the worst case (every kernel reads the live counts from device memory
// and retires early, so the host never waits on the device):
//   [trace fill] -> substitution table -> route+decide -> offsets/tiles ->
//   row bucketing -> up/gate GEMM (gathers h rows) -> down GEMM (-> shared
//   expert) -> combine (updates h) -> (not the last layer) exit GEMM
//   (gathers the executed tokens' h rows) -> exit gate -> compaction.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <mutex>

#include "common.h"

using namespace trimmoe;

// Workspace of trimmoe_stack_forward_static: a file-scope device array, one
// copy per device (each device that loads the library holds it until the
// process ends).  In host code its name is only a stand-in for the symbol:
// the device address comes from hipGetSymbolAddress (static_scratch below)
// and is what kernels and copies receive.
static __device__ __align__(256) char scratch[TRIMMOE_STATIC_SCRATCH_BYTES];

namespace {

inline int cdiv(int a, int b) { return (a + b - 1) / b; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int validate_model(const trimmoe_model* m) {
  if (!m || !m->layers) return TRIMMOE_ERR_NULL;
  if (m->dtype != TRIMMOE_F32 && m->dtype != TRIMMOE_BF16) return TRIMMOE_ERR_DTYPE;
  if (m->act != TRIMMOE_ACT_RELU && m->act != TRIMMOE_ACT_SWIGLU) return TRIMMOE_ERR_DTYPE;
  if (m->conf_mode != TRIMMOE_CONF_SOFTMAX && m->conf_mode != TRIMMOE_CONF_SIGMOID)
    return TRIMMOE_ERR_DTYPE;
  if (m->normalize_topk != 0 && m->normalize_topk != 1) return TRIMMOE_ERR_SHAPE;
  if (m->n_layers < 1 || m->d_model < 1 || m->n_experts < 1 ||
      m->n_experts > TRIMMOE_MAX_EXPERTS || m->top_k < 1 || m->top_k > TRIMMOE_MAX_TOPK ||
      m->top_k > m->n_experts || m->d_ff < 1 || m->d_ff_shared < 0 || m->vocab_exit < 1)
    return TRIMMOE_ERR_SHAPE;
  if (m->conf_mode == TRIMMOE_CONF_SIGMOID && m->vocab_exit != 1) return TRIMMOE_ERR_SHAPE;
  if (m->dtype == TRIMMOE_BF16) {
    if (m->d_model % 64 || m->d_ff % 64 || m->d_ff_shared % 64) return TRIMMOE_ERR_SHAPE;
  } else {
    if (m->d_model % 8) return TRIMMOE_ERR_SHAPE;
  }
  const bool swiglu = m->act == TRIMMOE_ACT_SWIGLU;
  for (int l = 0; l < m->n_layers; ++l) {
    const trimmoe_layer& L = m->layers[l];
    if (!L.w_router || !L.w_up || !L.w_down || !L.w_exit || !L.local_mask || !L.sim)
      return TRIMMOE_ERR_NULL;
    if (swiglu && !L.w_gate) return TRIMMOE_ERR_NULL;
    if (m->d_ff_shared > 0 && (!L.ws_up || !L.ws_gate || !L.ws_down)) return TRIMMOE_ERR_NULL;
    const void* mats[] = {L.w_router, L.w_up, L.w_down, L.w_exit,
                          swiglu ? L.w_gate : L.w_up,
                          m->d_ff_shared ? L.ws_up : L.w_up,
                          m->d_ff_shared ? L.ws_gate : L.w_up,
                          m->d_ff_shared ? L.ws_down : L.w_up};
    for (const void* q : mats)
      if (!aligned16(q)) return TRIMMOE_ERR_SHAPE;
    if (isnan(L.theta) || !(L.skip_slope >= 0.f) || isinf(L.skip_slope)) return TRIMMOE_ERR_POLICY;
  }
  return TRIMMOE_OK;
}

int validate_policy(const trimmoe_policy* p) {
  if (!p) return TRIMMOE_ERR_NULL;
  if (isnan(p->p_exit) || isnan(p->sim_min)) return TRIMMOE_ERR_POLICY;
  if (!(p->budget >= 0.f) || isinf(p->budget)) return TRIMMOE_ERR_POLICY;
  if (!(p->omega_t >= 0.f && p->omega_t <= 1.f)) return TRIMMOE_ERR_POLICY;
  if (!(p->t_local >= 0.f) || !(p->t_remote >= 0.f) || isinf(p->t_local) || isinf(p->t_remote))
    return TRIMMOE_ERR_POLICY;
  if (!(p->phi_scale >= 0.f) || isinf(p->phi_scale)) return TRIMMOE_ERR_POLICY;
  if (p->horizon < 1 || p->horizon > TRIMMOE_MAX_HORIZON) return TRIMMOE_ERR_POLICY;
  if (p->horizon > 1 && (p->la_subs < 1 || p->la_subs > TRIMMOE_MAX_LA_SUBS))
    return TRIMMOE_ERR_POLICY;
  return TRIMMOE_OK;
}

// The look-ahead's limits (policy.horizon > 1): its work per token grows as
// O^H * B^(k (H - 1)) cost evaluations, O = (1 + la_subs)^k + 1 options per
// level.  Layers first..last run;
// layer l reads the transitions of layers l .. l + H - 2 (not past N - 2).
int validate_lookahead(const trimmoe_model* m, const trimmoe_policy* p, int first, int last) {
  // the horizon the first layer run sees (later layers see no more)
  const int H = std::min(p->horizon, m->n_layers - first);
  if (H <= 1) return TRIMMOE_OK;
  const int k = m->top_k, B = m->trans_b;
  if (k > TRIMMOE_MAX_LOOKAHEAD_TOPK || B < 1 || B > TRIMMOE_MAX_TRANS_B) return TRIMMOE_ERR_SHAPE;
  double tuples = 1.0;
  for (int s = 0; s < k; ++s) tuples *= B;
  const double opts = pow(1.0 + p->la_subs, k) + 1.0;
  if (opts * tuples > kMaxBranches) return TRIMMOE_ERR_SHAPE;
  if (pow(opts, H) * pow(tuples, H - 1) > (double)(1 << 23)) return TRIMMOE_ERR_SHAPE;
  if (route_lds_bytes(m->dtype == TRIMMOE_BF16, m->n_experts, m->d_model, H, B, k, p->la_subs) >
      kRouteLdsMax)
    return TRIMMOE_ERR_SHAPE;
  const int end = std::min(last + H - 1, m->n_layers - 1);
  for (int l = first; l < end; ++l)
    if (!m->layers[l].trans_to || !m->layers[l].trans_p) return TRIMMOE_ERR_NULL;
  return TRIMMOE_OK;
}

int validate_state(const trimmoe_model* m, const trimmoe_state* s) {
  if (!s) return TRIMMOE_ERR_NULL;
  if (s->n_tokens < 0) return TRIMMOE_ERR_SHAPE;
  if (!s->h || !s->d_acc || !s->active_idx || !s->n_active || !s->exit_layer || !s->xi)
    return TRIMMOE_ERR_NULL;
  if (!aligned16(s->h)) return TRIMMOE_ERR_SHAPE;
  (void)m;
  return TRIMMOE_OK;
}

// Rows of split-K partial slices (splits x rows) the routed down GEMM may
// use for any batch of at most T tokens.  The split count depends on the
// row-tile count and is not monotone in it (a smaller batch can need more
// slice rows than a larger one), so take the largest product over every
// tile count up to T's, each at its largest batch.
size_t down_slice_rows_max(const trimmoe_model* m, int T) {
  const int E = m->n_experts, k = m->top_k;
  const long long R = (long long)T * k;
  if (m->dtype != TRIMMOE_BF16) return (size_t)R;
  const int tiles_T = cdiv((int)R, kGemmBM) + E;
  long long best = R * down_splits(tiles_T, m->d_model, m->d_ff);
  for (int tiles = E + 1; tiles < tiles_T; ++tiles) {
    // largest batch whose row count gives this many tiles
    const long long Tt = std::min<long long>(T, (long long)(tiles - E) * kGemmBM / k);
    best = std::max(best, Tt * k * down_splits(tiles, m->d_model, m->d_ff));
  }
  return (size_t)best;
}

// Per-(token, vocabulary tile) exit partials for any batch of at most T
// tokens: decode-sized batches use finer vocabulary tiles, so the largest of
// them can need more than a slightly larger batch.
size_t exit_partials_max(const trimmoe_model* m, int T) {
  const bool bf16 = m->dtype == TRIMMOE_BF16;
  size_t n = (size_t)T * cdiv(m->vocab_exit, exit_tile_rows(bf16, T));
  const int Ts = std::min(T, kExitSmallTokens);
  return std::max(n, (size_t)Ts * cdiv(m->vocab_exit, exit_tile_rows(bf16, Ts)));
}

// Carve the workspace (base == NULL: only measure).  Returns total bytes,
// which never decrease as T grows: a workspace carved for T tokens serves
// every smaller batch.
size_t carve(const trimmoe_model* m, int T, char* base, LayerParams* p) {
  const bool bf16 = m->dtype == TRIMMOE_BF16;
  const int E = m->n_experts, k = m->top_k, d = m->d_model, F = m->d_ff, Fs = m->d_ff_shared;
  const size_t es = bf16 ? 2 : 4;
  const int Tm = T > 0 ? T : 1;
  const size_t R = (size_t)Tm * k;
  const int nblk = route_blocks_max(Tm);
  const int max_tiles = (int)cdiv((int)R, kGemmBM) + E;
  const int n_vtiles = cdiv(m->vocab_exit, exit_tile_rows(bf16, Tm));
  size_t off = 0;
  auto take = [&](size_t bytes) -> void* {
    void* q = base ? base + off : nullptr;
    off = align256(off + bytes);
    return q;
  };
  LayerParams tmp;
  LayerParams& P = p ? *p : tmp;
  P.tok_exec = (int32_t*)take(R * 4);
  P.tok_w = (float*)take(R * 4);
  P.tok_row = (int32_t*)take(R * 4);
  P.tok_action = (int32_t*)take((size_t)Tm * 4);
  P.tok_keep = (int32_t*)take((size_t)Tm * 4);
  P.exec_list = (int32_t*)take((size_t)Tm * 4);
  P.exec_pos = (int32_t*)take((size_t)Tm * 4);
  P.blk_cnt = (int32_t*)take((size_t)nblk * E * 4);
  P.blk_off = (int32_t*)take((size_t)nblk * E * 4);
  P.blk_xcnt = (int32_t*)take((size_t)nblk * 4);
  P.blk_xoff = (int32_t*)take((size_t)nblk * 4);
  P.exp_off = (int32_t*)take((size_t)(E + 1) * 4);
  P.counts = (int32_t*)take(kCntSlots * 4);
  P.tiles = (int4*)take((size_t)max_tiles * 16);
  P.exp_toff = (int32_t*)take((size_t)E * 4);
  // the large-group core (and its cut down-GEMM tiles) is open to some batch
  // of at most Tm tokens once Tm k >= kBigRowsPerExpert E
  const bool big_any = bf16 && R >= (size_t)kBigRowsPerExpert * E;
  P.sk_flag = (int32_t*)take((size_t)max_tiles * cdiv(d, 256) * 4);
  P.sk_part = big_any ? (float*)take((size_t)kSkSlots * 256 * 256 * 4) : nullptr;
  P.row_src = (int32_t*)take(R * 4);
  P.act_buf = take(R * F * es);
  const int splits = bf16 ? down_splits(max_tiles, d, F) : 1;
  P.y_buf = (float*)take(down_slice_rows_max(m, Tm) * d * 4);
  P.y_split_stride = R * d;
  P.down_splits = splits;
  P.act_s = Fs ? take((size_t)Tm * Fs * es) : nullptr;
  P.y_s = Fs ? (float*)take((size_t)Tm * d * 4) : nullptr;
  P.hx = take((size_t)Tm * d * es);
  P.partials = (float2*)take(exit_partials_max(m, Tm) * 8);
  P.n_vtiles = n_vtiles;
  P.max_tiles = max_tiles;
  return off;
}

void fill_params(LayerParams& P, const trimmoe_model* m, int l, const trimmoe_policy* pol,
                 const trimmoe_state* s, const trimmoe_trace* tr) {
  const trimmoe_layer& L = m->layers[l];
  const int T = s->n_tokens, k = m->top_k;
  P.N = m->n_layers;
  P.d = m->d_model;
  P.E = m->n_experts;
  P.k = k;
  P.F = m->d_ff;
  P.Fs = m->d_ff_shared;
  P.V = m->vocab_exit;
  P.act = m->act;
  P.conf_mode = m->conf_mode;
  P.normalize = m->normalize_topk;
  P.layer = l;
  P.w_router = L.w_router;
  P.b_router = L.b_router;
  P.w_up = L.w_up;
  P.w_gate = m->act == TRIMMOE_ACT_SWIGLU ? L.w_gate : nullptr;
  P.w_down = L.w_down;
  P.ws_up = L.ws_up;
  P.ws_gate = L.ws_gate;
  P.ws_down = L.ws_down;
  P.w_exit = L.w_exit;
  P.b_exit = L.b_exit;
  P.local_mask = L.local_mask;
  P.sim = L.sim;
  P.theta = L.theta;
  P.skip_slope = L.skip_slope;
  P.p_exit = pol->p_exit;
  P.budget = pol->budget;
  P.omega_t = pol->omega_t;
  P.t_local = pol->t_local;
  P.t_remote = pol->t_remote;
  P.phi_scale = pol->phi_scale;
  P.sim_min = pol->sim_min;
  P.p_exit_tok = pol->p_exit_tok;
  P.budget_tok = pol->budget_tok;
  P.horizon = std::min(pol->horizon, m->n_layers - l);
  P.la_subs = P.horizon > 1 ? pol->la_subs : 1;
  P.trans_b = m->trans_b;
  P.rb = route_block_tokens(T, P.horizon > 1);
  P.bm = expert_tile_rows(m->dtype == TRIMMOE_BF16, T, k, m->n_experts, m->d_model, m->d_ff);
  // the large-group down GEMM cuts the tiles of its last round along K
  // instead of splitting every tile
  if (P.bm == kBigBM) {
    P.down_splits = 1;
  } else {
    P.sk_flag = nullptr;
    P.sk_part = nullptr;
  }
  for (int j = 0; j < kMaxLookahead; ++j) {
    const bool later = j + 1 < P.horizon;  // layer l + j + 1 is looked at
    const trimmoe_layer* Lj = later ? &m->layers[l + j + 1] : nullptr;
    P.la_mask[j] = Lj ? Lj->local_mask : nullptr;
    P.la_sim[j] = Lj ? Lj->sim : nullptr;
    P.la_theta[j] = Lj ? Lj->theta : 0.f;
    P.la_slope[j] = Lj ? Lj->skip_slope : 0.f;
    P.la_tto[j] = j + 1 < P.horizon ? m->layers[l + j].trans_to : nullptr;
    P.la_tp[j] = j + 1 < P.horizon ? m->layers[l + j].trans_p : nullptr;
  }
  P.T = T;
  P.h = s->h;
  P.d_acc = s->d_acc;
  P.active_idx = s->active_idx;
  P.n_active = s->n_active;
  P.exit_layer = s->exit_layer;
  P.xi = s->xi;
  const size_t rowT = (size_t)l * T, rowTk = (size_t)l * T * k;
  P.tr_action = tr && tr->action ? tr->action + rowT : nullptr;
  P.tr_target = tr && tr->target ? tr->target + rowTk : nullptr;
  P.tr_exec = tr && tr->exec ? tr->exec + rowTk : nullptr;
  P.tr_kind = tr && tr->kind ? tr->kind + rowTk : nullptr;
  P.tr_gate = tr && tr->gate ? tr->gate + rowTk : nullptr;
  P.tr_importance = tr && tr->importance ? tr->importance + rowT : nullptr;
  P.tr_xi = tr && tr->xi ? tr->xi + rowT : nullptr;
  P.tr_d_acc = tr && tr->d_acc ? tr->d_acc + rowT : nullptr;
  P.tr_counters = tr && tr->counters ? tr->counters + (size_t)l * kCounters : nullptr;
}

bool any_trace(const trimmoe_trace* tr) {
  return tr && (tr->action || tr->target || tr->exec || tr->kind || tr->gate || tr->importance ||
                tr->xi || tr->d_acc || tr->counters);
}

int check_workspace(const trimmoe_model* m, const trimmoe_state* s, void* ws, size_t bytes) {
  if (!ws) return TRIMMOE_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) & 255) return TRIMMOE_ERR_WORKSPACE;
  if (bytes < carve(m, s->n_tokens, nullptr, nullptr)) return TRIMMOE_ERR_WORKSPACE;
  return TRIMMOE_OK;
}

namespace {
// engine-clock record of later GEMM launches (trimmoe_set_clock_record) and
// the device it lives on: launches on any other device record nothing
std::mutex g_clock_mu;
unsigned long long* g_clock_rec = nullptr;
int g_clock_dev = -1;

unsigned long long* clock_record_for(int dev) {
  std::lock_guard<std::mutex> lock(g_clock_mu);
  return dev == g_clock_dev ? g_clock_rec : nullptr;
}
}  // namespace

// ev: NULL, or TRIMMOE_TIMED_CLASSES + 1 events recorded around the classes;
// fill_layers: trace rows of this many layers from l on get their inactive
// defaults first (a stack pass fills all of them at layer 0)
int run_layer(const trimmoe_model* m, int l, const trimmoe_policy* pol, const trimmoe_state* s,
              const trimmoe_trace* tr, void* ws, hipStream_t st, hipEvent_t* ev,
              int fill_layers) {
  if (s->n_tokens == 0) return TRIMMOE_OK;
  LayerParams P;
  memset(&P, 0, sizeof(P));
  carve(m, s->n_tokens, static_cast<char*>(ws), &P);
  fill_params(P, m, l, pol, s, tr);
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      ncu <= 0)
    return TRIMMOE_ERR_HIP;
  P.n_cu = ncu;
  P.clk = clock_record_for(dev);
  const bool bf16 = m->dtype == TRIMMOE_BF16;
  const bool last = l == m->n_layers - 1;
#define TRIMMOE_TRY(x) \
  if ((x) != hipSuccess) return TRIMMOE_ERR_HIP
#define TRIMMOE_MARK(i) \
  if (ev) TRIMMOE_TRY(hipEventRecord(ev[i], st))
  TRIMMOE_MARK(0);
  if (fill_layers > 0 && any_trace(tr)) TRIMMOE_TRY(launch_trace_fill(P, fill_layers, st));
  TRIMMOE_TRY(launch_route(P, bf16, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_ROUTE + 1);
  TRIMMOE_TRY(launch_scan(P, st));
  TRIMMOE_TRY(launch_bucket(P, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_BUCKET + 1);
  TRIMMOE_TRY(launch_expert_up(P, bf16, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_UP + 1);
  TRIMMOE_TRY(launch_expert_down(P, bf16, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_DOWN + 1);
  if (P.Fs > 0) TRIMMOE_TRY(launch_shared_expert(P, bf16, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_SHARED + 1);
  TRIMMOE_TRY(launch_combine(P, bf16, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_COMBINE + 1);
  if (!last) TRIMMOE_TRY(launch_exit_head(P, bf16, st));
  TRIMMOE_MARK(TRIMMOE_CLASS_EXIT + 1);
  if (!last) {
    TRIMMOE_TRY(launch_exit_reduce(P, st));
    TRIMMOE_TRY(launch_compact(P, st));
  }
  TRIMMOE_MARK(TRIMMOE_CLASS_GATE + 1);
#undef TRIMMOE_MARK
#undef TRIMMOE_TRY
  return TRIMMOE_OK;
}

int stack(const trimmoe_model* m, const trimmoe_policy* p, trimmoe_state* s,
          trimmoe_trace* trace, void* workspace, size_t workspace_bytes, void* stream,
          void* const* events, int32_t n_events) {
  int rc = validate_model(m);
  if (rc) return rc;
  if ((rc = validate_policy(p))) return rc;
  if ((rc = validate_lookahead(m, p, 0, m->n_layers - 1))) return rc;
  if ((rc = validate_state(m, s))) return rc;
  if ((rc = check_workspace(m, s, workspace, workspace_bytes))) return rc;
  const int per = TRIMMOE_TIMED_CLASSES + 1;
  if (events) {
    if (n_events != m->n_layers * per) return TRIMMOE_ERR_SHAPE;
    for (int i = 0; i < n_events; ++i)
      if (!events[i]) return TRIMMOE_ERR_NULL;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s->n_tokens == 0) return TRIMMOE_OK;
  if (launch_state_reset(m, s, st) != hipSuccess) return TRIMMOE_ERR_HIP;
  for (int l = 0; l < m->n_layers; ++l) {
    hipEvent_t* ev = events ? reinterpret_cast<hipEvent_t*>(const_cast<void**>(events)) + l * per
                            : nullptr;
    if ((rc = run_layer(m, l, p, s, trace, workspace, st, ev, l == 0 ? m->n_layers : 0)))
      return rc;
  }
  return TRIMMOE_OK;
}

}  // namespace

extern "C" {

int trimmoe_abi_version(void) { return TRIMMOE_ABI_VERSION; }

const char* trimmoe_status_str(int status) {
  switch (status) {
    case TRIMMOE_OK: return "ok";
    case TRIMMOE_ERR_NULL: return "required pointer is NULL";
    case TRIMMOE_ERR_SHAPE: return "unsupported or inconsistent shape or alignment";
    case TRIMMOE_ERR_DTYPE: return "unknown dtype, activation or confidence mode";
    case TRIMMOE_ERR_POLICY: return "policy scalar out of range or NaN";
    case TRIMMOE_ERR_LAYER: return "layer index out of range";
    case TRIMMOE_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case TRIMMOE_ERR_HIP: return "HIP kernel launch failed";
    default: return "unknown status";
  }
}

int trimmoe_workspace_size(const trimmoe_model* m, int32_t max_tokens, size_t* bytes_out) {
  if (!bytes_out) return TRIMMOE_ERR_NULL;
  int rc = validate_model(m);
  if (rc) return rc;
  if (max_tokens < 0) return TRIMMOE_ERR_SHAPE;
  // the carve never shrinks as the token count grows, so this covers every
  // batch of at most max_tokens tokens
  *bytes_out = carve(m, max_tokens, nullptr, nullptr);
  return TRIMMOE_OK;
}

int trimmoe_state_reset(const trimmoe_model* m, trimmoe_state* s, void* stream) {
  int rc = validate_model(m);
  if (rc) return rc;
  if ((rc = validate_state(m, s))) return rc;
  if (s->n_tokens == 0) return TRIMMOE_OK;
  if (launch_state_reset(m, s, static_cast<hipStream_t>(stream)) != hipSuccess) return TRIMMOE_ERR_HIP;
  return TRIMMOE_OK;
}

int trimmoe_layer_step(const trimmoe_model* m, int32_t layer, const trimmoe_policy* p,
                       trimmoe_state* s, trimmoe_trace* trace, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int rc = validate_model(m);
  if (rc) return rc;
  if ((rc = validate_policy(p))) return rc;
  if (layer < 0 || layer >= m->n_layers) return TRIMMOE_ERR_LAYER;
  if ((rc = validate_lookahead(m, p, layer, layer))) return rc;
  if ((rc = validate_state(m, s))) return rc;
  if ((rc = check_workspace(m, s, workspace, workspace_bytes))) return rc;
  return run_layer(m, layer, p, s, trace, workspace, static_cast<hipStream_t>(stream), nullptr,
                   1);
}

int trimmoe_stack_forward(const trimmoe_model* m, const trimmoe_policy* p, trimmoe_state* s,
                          trimmoe_trace* trace, void* workspace, size_t workspace_bytes,
                          void* stream) {
  return stack(m, p, s, trace, workspace, workspace_bytes, stream, nullptr, 0);
}

int trimmoe_set_clock_record(uint64_t* rec) {
  static_assert(sizeof(uint64_t) == sizeof(unsigned long long), "64-bit record words");
  int dev = -1;
  if (rec && hipGetDevice(&dev) != hipSuccess) return TRIMMOE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_clock_mu);
  g_clock_rec = reinterpret_cast<unsigned long long*>(rec);
  g_clock_dev = rec ? dev : -1;
  return TRIMMOE_OK;
}

int trimmoe_stack_forward_timed(const trimmoe_model* m, const trimmoe_policy* p,
                                trimmoe_state* s, trimmoe_trace* trace, void* workspace,
                                size_t workspace_bytes, void* stream, void* const* events,
                                int32_t n_events) {
  if (!events) return TRIMMOE_ERR_NULL;
  return stack(m, p, s, trace, workspace, workspace_bytes, stream, events, n_events);
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per device, once looked up

// The current device's copy of `scratch`: its address is looked up once per
// device, with that device current, and kept.
int static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TRIMMOE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
      return TRIMMOE_ERR_HIP;
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return TRIMMOE_OK;
}
}  // namespace

int trimmoe_stack_forward_static(const trimmoe_model* m, const trimmoe_policy* p,
                                 trimmoe_state* s, trimmoe_trace* trace, void* stream) {
  // every argument check first (no HIP call before them), then the size limit
  int rc = validate_model(m);
  if (rc) return rc;
  if ((rc = validate_policy(p))) return rc;
  if ((rc = validate_lookahead(m, p, 0, m->n_layers - 1))) return rc;
  if ((rc = validate_state(m, s))) return rc;
  const size_t need = carve(m, s->n_tokens, nullptr, nullptr);
  if (need > TRIMMOE_STATIC_SCRATCH_BYTES) return TRIMMOE_ERR_WORKSPACE;
  if (s->n_tokens == 0) return TRIMMOE_OK;
  void* ws = nullptr;
  if ((rc = static_scratch(&ws))) return rc;
  // the carve needs no cleared memory: every kernel writes what it reads
  // later in the same layer before reading it
  return stack(m, p, s, trace, ws, TRIMMOE_STATIC_SCRATCH_BYTES, stream, nullptr, 0);
}

int trimmoe_window_stats(const trimmoe_model* m, const trimmoe_policy* p, const trimmoe_state* s,
                         const trimmoe_trace* trace, double* stats, void* stream) {
  int rc = validate_model(m);
  if (rc) return rc;
  if ((rc = validate_policy(p))) return rc;
  if ((rc = validate_state(m, s))) return rc;
  if (!trace || !trace->counters || !stats) return TRIMMOE_ERR_NULL;
  WindowArgs w{s->n_tokens, m->n_layers, m->top_k, s->exit_layer, s->xi, s->d_acc,
               p->budget_tok, p->budget, p->t_local, p->t_remote, trace->counters, stats};
  return launch_window_stats(w, static_cast<hipStream_t>(stream)) == hipSuccess ? TRIMMOE_OK
                                                                                  : TRIMMOE_ERR_HIP;
}

int trimmoe_feedback_update(trimmoe_policy* p, const double* stats, double eta, double kappa,
                            double p_floor) {
  if (!p || !stats) return TRIMMOE_ERR_NULL;
  if (validate_policy(p)) return TRIMMOE_ERR_POLICY;
  if (!(eta >= 0.0) || !(kappa >= 0.0) || isinf(eta) || isinf(kappa) ||
      !(p_floor >= 0.0 && p_floor <= 1.0))
    return TRIMMOE_ERR_POLICY;
  for (int i = 0; i < 6; ++i)
    if (!(stats[i] >= 0.0) || isinf(stats[i])) return TRIMMOE_ERR_POLICY;
  const double tokens = stats[0], exits = stats[1], xi_exit = stats[2], util = stats[3],
               delay = stats[4], delay_ref = stats[5];
  double pj = p->p_exit;
  if (exits > 0.0) {  // Eq. (37): towards the mean confidence at exit, within [p_floor, 1]
    pj += eta * (xi_exit / exits - pj);
    pj = pj < p_floor ? p_floor : (pj > 1.0 ? 1.0 : pj);
  }
  double omega_d = 1.0 - p->omega_t;
  if (tokens > 0.0 && delay_ref > 0.0) {  // Eq. (43): budget utilisation vs normalised delay
    omega_d += kappa * (util / tokens - delay / delay_ref);
    omega_d = omega_d < 0.0 ? 0.0 : (omega_d > 1.0 ? 1.0 : omega_d);
  }
  p->p_exit = (float)pj;
  p->omega_t = (float)(1.0 - omega_d);
  return TRIMMOE_OK;
}

// ----------------------------------------- exit-head training (Sec. IV-A) --
namespace {
size_t argmax_ws(bool bf16, int V, int n_rows, int* n_vtiles) {
  const int rows = n_rows > 0 ? n_rows : 1;
  const int nvt = cdiv(V, bf16 ? exit_tile_rows(true, rows) : kExitTileF32);
  if (n_vtiles) *n_vtiles = nvt;
  return 256 + align256((size_t)rows * nvt * sizeof(float2));
}
size_t train_ws(int n_rows) {
  const int rows = n_rows > 0 ? n_rows : 1;
  return align256((size_t)rows * 4) + align256((size_t)rows * 8);
}
bool head_dims_ok(int dtype, int d) {
  if (dtype == TRIMMOE_BF16) return d >= 64 && d % 64 == 0;
  return dtype == TRIMMOE_F32 && d >= 1;
}
}  // namespace

int trimmoe_head_argmax_workspace_size(int32_t dtype, int32_t vocab, int32_t n_rows,
                                       size_t* bytes) {
  if (!bytes) return TRIMMOE_ERR_NULL;
  if (dtype != TRIMMOE_F32 && dtype != TRIMMOE_BF16) return TRIMMOE_ERR_DTYPE;
  if (vocab < 1 || n_rows < 0) return TRIMMOE_ERR_SHAPE;
  *bytes = argmax_ws(dtype == TRIMMOE_BF16, vocab, n_rows, nullptr);
  return TRIMMOE_OK;
}

int trimmoe_head_argmax(int32_t dtype, int32_t vocab, int32_t d_model, int32_t n_rows,
                        const void* w_head, const float* b_head, const void* h, int32_t* argmax,
                        void* workspace, size_t workspace_bytes, void* stream) {
  if (!w_head || !h || !argmax || !workspace) return TRIMMOE_ERR_NULL;
  if (dtype != TRIMMOE_F32 && dtype != TRIMMOE_BF16) return TRIMMOE_ERR_DTYPE;
  if (vocab < 1 || n_rows < 0 || !head_dims_ok(dtype, d_model)) return TRIMMOE_ERR_SHAPE;
  const bool bf16 = dtype == TRIMMOE_BF16;
  if (bf16 && (!aligned16(w_head) || !aligned16(h))) return TRIMMOE_ERR_SHAPE;
  int nvt = 0;
  if (reinterpret_cast<uintptr_t>(workspace) & 255) return TRIMMOE_ERR_WORKSPACE;
  if (workspace_bytes < argmax_ws(bf16, vocab, n_rows, &nvt)) return TRIMMOE_ERR_WORKSPACE;
  if (n_rows == 0) return TRIMMOE_OK;
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return TRIMMOE_ERR_HIP;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t* n_dev = static_cast<int32_t*>(workspace);
  float2* partials = reinterpret_cast<float2*>(static_cast<char*>(workspace) + 256);
  if (launch_set_int(n_dev, n_rows, st) != hipSuccess ||
      launch_head_argmax_partials(bf16, w_head, b_head, h, n_dev, n_rows, vocab, d_model, nvt,
                                  partials, ncu, st) != hipSuccess ||
      launch_argmax_reduce(partials, nvt, n_rows, argmax, st) != hipSuccess)
    return TRIMMOE_ERR_HIP;
  return TRIMMOE_OK;
}

int trimmoe_consistency_labels(int32_t n_rows, const int32_t* pred, const int32_t* ref,
                               uint8_t* labels, void* stream) {
  if (!pred || !ref || !labels) return TRIMMOE_ERR_NULL;
  if (n_rows < 0) return TRIMMOE_ERR_SHAPE;
  if (launch_consistency(pred, ref, n_rows, labels, static_cast<hipStream_t>(stream)) !=
      hipSuccess)
    return TRIMMOE_ERR_HIP;
  return TRIMMOE_OK;
}

int trimmoe_train_exit_head_workspace_size(int32_t n_rows, size_t* bytes) {
  if (!bytes) return TRIMMOE_ERR_NULL;
  if (n_rows < 0) return TRIMMOE_ERR_SHAPE;
  *bytes = train_ws(n_rows);
  return TRIMMOE_OK;
}

int trimmoe_train_exit_head(int32_t dtype, int32_t d_model, int32_t n_rows, const void* h,
                            const uint8_t* labels, int32_t epochs, float lr, float* w, float* c,
                            float* loss, void* workspace, size_t workspace_bytes, void* stream) {
  if (!h || !labels || !w || !c || !workspace) return TRIMMOE_ERR_NULL;
  if (dtype != TRIMMOE_F32 && dtype != TRIMMOE_BF16) return TRIMMOE_ERR_DTYPE;
  if (n_rows < 1 || epochs < 0 || !head_dims_ok(dtype, d_model)) return TRIMMOE_ERR_SHAPE;
  if (!(lr >= 0.f) || isinf(lr)) return TRIMMOE_ERR_POLICY;
  if (reinterpret_cast<uintptr_t>(workspace) & 255) return TRIMMOE_ERR_WORKSPACE;
  if (workspace_bytes < train_ws(n_rows)) return TRIMMOE_ERR_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  float* r = static_cast<float*>(workspace);
  double* row_loss = reinterpret_cast<double*>(static_cast<char*>(workspace) +
                                               align256((size_t)n_rows * 4));
  for (int e = 0; e < epochs; ++e)
    if (launch_bce_step(dtype == TRIMMOE_BF16, h, labels, n_rows, d_model, lr, w, c, r, row_loss,
                        loss ? loss + e : nullptr, st) != hipSuccess)
      return TRIMMOE_ERR_HIP;
  return TRIMMOE_OK;
}

}  // extern "C"
