/*
 * trimmoe.h -- C ABI of the adaptive-depth MoE step (TrimMoE, arXiv
 * 2608.00573) on one AMD Instinct MI355X (gfx950).
 *
 * One call of trimmoe_layer_step runs, for every still-active token, the
 * online decision of the paper's Algorithm 2 (Table II) at look-ahead
 * horizon H = 1 and the MoE layer it selects:
 *
 *   route   router logits, top-k, layer importance I (Sec. III-B, Eq. (4))
 *   decide  substitution of remote experts by local ones (Eq. (3)), skip
 *           admission and costs (Eq. (5), (31), (32), (34), (35), the
 *           importance threshold of Sec. V-C), budget update (Eq. (41),
 *           (42))
 *   FFN     grouped expert FFN over the executed (token, expert) rows, the
 *           weighted combine and the residual update (a skipped layer is the
 *           identity path, Sec. III-B)
 *   exit    exit-head confidence xi (Eq. (7)) after an executed layer and
 *           the exit gate xi >= p_J (Eq. (8), (9)); exited tokens are
 *           removed from the active list.
 *
 * Conventions
 *  - Every pointer inside trimmoe_layer, trimmoe_state and trimmoe_trace is a
 *    DEVICE pointer on the current HIP device; trimmoe_model,
 *    trimmoe_policy and the layer array are HOST structs read during the
 *    call only.  Matrices are row-major and contiguous, 16-byte aligned.
 *  - dtype TRIMMOE_BF16: weights and h are bf16 (2-byte words); routed and
 *    shared activations are rounded to bf16 before the down projection and
 *    h is rounded to bf16 once per executed layer.  TRIMMOE_F32: all fp32.
 *  - All arguments are validated before anything is enqueued; on any error
 *    nothing is launched and no output is modified.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *    is the null stream).  TRIMMOE_OK means "enqueued"; kernel faults
 *    surface at the caller's next synchronisation.
 *  - The library never allocates, frees or synchronises.  The caller owns
 *    the workspace (size from trimmoe_workspace_size); the one exception is
 *    trimmoe_stack_forward_static, whose workspace is a fixed device array
 *    per device held by the library.  Calls that share a workspace or a
 *    state must be ordered on one stream.
 */
#ifndef TRIMMOE_H
#define TRIMMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TRIMMOE_ABI_VERSION 6

/* status codes */
#define TRIMMOE_OK 0
#define TRIMMOE_ERR_NULL (-1)      /* a required pointer is NULL             */
#define TRIMMOE_ERR_SHAPE (-2)     /* unsupported or inconsistent dimensions */
#define TRIMMOE_ERR_DTYPE (-3)     /* unknown dtype / activation / mode      */
#define TRIMMOE_ERR_POLICY (-4)    /* NaN or out-of-range policy scalar      */
#define TRIMMOE_ERR_LAYER (-5)     /* layer index out of range               */
#define TRIMMOE_ERR_WORKSPACE (-6) /* workspace NULL, misaligned or too small */
#define TRIMMOE_ERR_HIP (-7)       /* a kernel launch was rejected by HIP    */

#define TRIMMOE_F32 0
#define TRIMMOE_BF16 1

#define TRIMMOE_ACT_RELU 0   /* E(x) = W_down relu(W_up x)                    */
#define TRIMMOE_ACT_SWIGLU 1 /* E(x) = W_down (silu(W_gate x) * (W_up x))     */

#define TRIMMOE_CONF_SOFTMAX 0 /* xi = max softmax(W_exit h + b), V >= 2     */
#define TRIMMOE_CONF_SIGMOID 1 /* xi = sigmoid(w . h + b), W_exit is [1, d]  */

/* limits checked by validation */
#define TRIMMOE_MAX_EXPERTS 256
#define TRIMMOE_MAX_TOPK 8
/* look-ahead (policy.horizon > 1): H <= 4, top_k <= 4, 1 <= trans_b <= 8,
 * 1 <= la_subs <= 4, and with O = (1 + la_subs)^k + 1 options per token:
 * O * trans_b^k <= 1024 first-level branches per token,
 * O^H * trans_b^(k (H - 1)) <= 2^23 cost evaluations per token, and the route
 * block's look-ahead tables within 148 KB of LDS */
#define TRIMMOE_MAX_HORIZON 4
#define TRIMMOE_MAX_LOOKAHEAD_TOPK 4
#define TRIMMOE_MAX_TRANS_B 8
#define TRIMMOE_MAX_LA_SUBS 4

/* actions recorded in the trace */
#define TRIMMOE_ACT_INACTIVE 0
#define TRIMMOE_ACT_EXEC 1
#define TRIMMOE_ACT_SKIP 2

/* per-slot kinds recorded in the trace */
#define TRIMMOE_KIND_NONE (-1)   /* token inactive or layer skipped          */
#define TRIMMOE_KIND_LOCAL 0     /* target expert, resident on this GPU      */
#define TRIMMOE_KIND_SUBST 1     /* local substitute of a remote target      */
#define TRIMMOE_KIND_REMOTE 2    /* remote target executed exactly           */

/*
 * One MoE layer.  E = n_experts, d = d_model, F = d_ff, Fs = d_ff_shared,
 * V = vocab_exit (1 in sigmoid mode).  Weight element type = model dtype.
 */
typedef struct trimmoe_layer {
  const void* w_router;   /* [E, d]   router (Sec. III-B)                       */
  const float* b_router;  /* [E] fp32 or NULL                                   */
  const void* w_up;       /* [E, F, d]                                          */
  const void* w_gate;     /* [E, F, d] (SwiGLU) or NULL (ReLU)                  */
  const void* w_down;     /* [E, d, F]                                          */
  const void* ws_up;      /* [Fs, d] shared expert (SwiGLU) or NULL if Fs == 0  */
  const void* ws_gate;    /* [Fs, d]                                            */
  const void* ws_down;    /* [d, Fs]                                            */
  const void* w_exit;     /* [V, d]   exit head h_l (Eq. (7))                   */
  const float* b_exit;    /* [V] fp32 or NULL                                   */
  const uint8_t* local_mask; /* [E]  1 = expert resident on this GPU (Eq. (1)) */
  const float* sim;       /* [E, E] fp32 expert similarity Sim_l (Eq. (3))      */
  float theta;            /* importance threshold theta_l (Eq. (24), Sec. V-C)  */
  float skip_slope;       /* s_l of the skip degradation rho(I)=min(1,s_l I)    */
  /* Expert transitions P_l from this layer to the next (Eq. (38)), read by
   * the look-ahead only (policy.horizon > 1: the decision at layer l reads
   * P_l .. P_{l+H-2}, never the last layer's, and those must be non-NULL):
   * row e holds trans_b (target, probability) entries; target -1
   * (probability 0) pads a row.  Device memory, caller-owned.             */
  const int16_t* trans_to; /* [E, trans_b] next-layer expert or -1           */
  const float* trans_p;    /* [E, trans_b] probabilities, each row sums to 1 */
} trimmoe_layer;

typedef struct trimmoe_model {
  int32_t n_layers;       /* N                                                  */
  int32_t d_model;        /* d; bf16: multiple of 64, f32: multiple of 8        */
  int32_t n_experts;      /* E, 1..256                                          */
  int32_t top_k;          /* k, 1..min(8, E)                                    */
  int32_t d_ff;           /* F; bf16: multiple of 64                            */
  int32_t d_ff_shared;    /* Fs, 0 = no shared expert; bf16: multiple of 64     */
  int32_t vocab_exit;     /* V                                                  */
  int32_t dtype;          /* TRIMMOE_F32 | TRIMMOE_BF16                         */
  int32_t act;            /* TRIMMOE_ACT_RELU | TRIMMOE_ACT_SWIGLU              */
  int32_t conf_mode;      /* TRIMMOE_CONF_SOFTMAX | TRIMMOE_CONF_SIGMOID        */
  int32_t normalize_topk; /* 1: slot weight p_e / I, 0: p_e                     */
  const trimmoe_layer* layers; /* host array of N layers                        */
  int32_t trans_b;        /* entries per transition row (0: no transitions)     */
} trimmoe_model;

/*
 * Online policy (Sec. V).  Costs: execute = omega_t * sum of per-slot
 * delays (t_local or t_remote) + (1 - omega_t) * sum Q / budget (Eq. (31));
 * skip = (1 - omega_t) * Lambda / budget (Eq. (32)).  Q(e, j) =
 * min(1, phi_scale * (1 - Sim[e][j]) / 2) (Eq. (3)); a local expert j is a
 * feasible substitute of e when Sim[e][j] >= sim_min.
 *
 * With horizon H > 1 every candidate action also carries the cost-to-go
 * Phi^(H-1) of Eq. (39) and the action minimising the sum is taken
 * (Eq. (40)): the expected least cost of the next H - 1 layers, each slot's
 * next target drawn from the transition row of the expert the slot runs
 * (its routed target after a skip), starting from the budget the action
 * leaves.  The token's importance at this layer stands in for later ones,
 * exits are not predicted inside the recursion, and the token never moves
 * (one GPU: the location in Eq. (39) is always this device).  Under the
 * look-ahead each remote slot may run its target or any of its la_subs
 * least-loss local substitutes (Sim >= sim_min, ties to the lower id), at
 * this layer and at every level of the recursion: Eq. (34) admits every
 * feasible one, and the cost-to-go depends on the expert run.  At H = 1 only
 * the least-loss one can be optimal and la_subs is not read.
 */
typedef struct trimmoe_policy {
  float p_exit;      /* confidence requirement p_J (Eq. (8))               */
  float budget;      /* per-token degradation budget D_i (Eq. (33)), >= 0   */
  float omega_t;     /* delay weight in [0, 1]; omega_D = 1 - omega_t       */
  float t_local;     /* normalised delay of a local slot, >= 0              */
  float t_remote;    /* normalised delay of a remote slot, >= 0             */
  float phi_scale;   /* phi(x) = min(1, phi_scale * x), >= 0                */
  float sim_min;     /* similarity floor of feasible substitutes            */
  const float* p_exit_tok; /* [T] device, per-token p_J, or NULL            */
  const float* budget_tok; /* [T] device, per-token budget, or NULL         */
  int32_t horizon;   /* look-ahead horizon H, 1..TRIMMOE_MAX_HORIZON (Sec. V-E,
                        Eq. (39), (40)); 1 = the myopic rule                */
  int32_t la_subs;   /* H > 1: local substitute candidates per remote slot,
                        1..TRIMMOE_MAX_LA_SUBS (the least-loss ones); not
                        read at H = 1                                      */
} trimmoe_policy;

/*
 * Per-token state, all device memory owned by the caller.  T = n_tokens.
 *   h          [T, d]  hidden states; updated in place; an exited token
 *                      keeps its state at exit time (Eq. (8)).
 *   d_acc      [T] f32 accumulated degradation D-hat (Eq. (41), (42)).
 *   active_idx [T] i32 tokens still active, ascending; first *n_active used.
 *   n_active   [1] i32 number of active tokens (device).
 *   exit_layer [T] i32 0-based layer after which the token exited, or N.
 *   xi         [T] f32 last evaluated confidence, NaN if none yet.
 */
typedef struct trimmoe_state {
  int32_t n_tokens;
  void* h;
  float* d_acc;
  int32_t* active_idx;
  int32_t* n_active;
  int32_t* exit_layer;
  float* xi;
} trimmoe_state;

/*
 * Optional per-layer decision record (device memory, NULL = not written).
 * Row l of each array covers layer l; entries of tokens inactive at layer l
 * are written as: action 0, target/exec -1, kind -1, gate/importance/xi/
 * d_acc NaN.  exec[t][s] is the expert slot s runs (target, substitute, or
 * -1 if skipped); kind per the TRIMMOE_KIND_* codes; gate is the slot
 * weight; xi is NaN where no confidence was evaluated; d_acc is D-hat
 * after the layer.  counters[l][0..8] = active, executed, skipped, exited,
 * substituted slots, remote slots, merged rows, distinct experts, and remote
 * targets among the routed slots of the active tokens (what exact execution
 * of every active token would send remote); counters[l][9..15] are zero.
 */
typedef struct trimmoe_trace {
  int8_t* action;      /* [N, T]    */
  int16_t* target;     /* [N, T, k] */
  int16_t* exec;       /* [N, T, k] */
  int8_t* kind;        /* [N, T, k] */
  float* gate;         /* [N, T, k] */
  float* importance;   /* [N, T]    */
  float* xi;           /* [N, T]    */
  float* d_acc;        /* [N, T]    */
  int32_t* counters;   /* [N, 16]   */
} trimmoe_trace;

/* TRIMMOE_ABI_VERSION of the built library. */
int trimmoe_abi_version(void);

/* Static text for a status code (never NULL). */
const char* trimmoe_status_str(int status);

/*
 * Bytes of workspace that trimmoe_layer_step / trimmoe_stack_forward need
 * for up to max_tokens tokens (written to *bytes_out).  The workspace must
 * be 256-byte aligned.  Host-only; validates the model like the steps do.
 */
int trimmoe_workspace_size(const trimmoe_model* m, int32_t max_tokens,
                           size_t* bytes_out);

/*
 * Algorithm 2 initialisation (Table II, first loop): d_acc = 0, every token
 * active in index order, n_active = T, exit_layer = N, xi = NaN.  h is not
 * touched.
 */
int trimmoe_state_reset(const trimmoe_model* m, trimmoe_state* s, void* stream);

/*
 * One MoE layer `layer` (0-based) for the active tokens of `s` (Algorithm 2
 * at H = 1, Eq. (3)-(9), (31)-(35), (40)-(42)).  Reads the active list and
 * n_active on the device (no host round trip); updates h, d_acc,
 * active_idx, n_active, exit_layer and xi.  The confidence of layer N-1 is
 * not evaluated.  trace may be NULL.
 */
int trimmoe_layer_step(const trimmoe_model* m, int32_t layer,
                       const trimmoe_policy* p, trimmoe_state* s,
                       trimmoe_trace* trace, void* workspace,
                       size_t workspace_bytes, void* stream);

/* trimmoe_state_reset followed by trimmoe_layer_step for l = 0 .. N-1. */
int trimmoe_stack_forward(const trimmoe_model* m, const trimmoe_policy* p,
                          trimmoe_state* s, trimmoe_trace* trace,
                          void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * trimmoe_stack_forward without a caller workspace and without any
 * allocation, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * The caller still passes the model, policy, state and optional trace.
 *
 * The workspace is a library-owned device array of
 * TRIMMOE_STATIC_SCRATCH_BYTES bytes, one per device, created when the
 * library's code object is loaded on that device and held until the process
 * ends; its address is looked up (hipGetSymbolAddress) at the first call on
 * each device.  A batch whose workspace (trimmoe_workspace_size of n_tokens)
 * exceeds that size is rejected with TRIMMOE_ERR_WORKSPACE before anything
 * is enqueued; other errors as trimmoe_stack_forward, plus TRIMMOE_ERR_HIP
 * if the array cannot be located.  No memory is allocated or freed (no
 * hipMalloc, no allocating library routine); nothing needs clearing between
 * calls (the array keeps the last call's contents, which no call reads).
 * All calls on one device share its array: calls that may overlap on one
 * device (different streams, or different host threads without ordering)
 * race and must be serialised by the caller.
 */
#define TRIMMOE_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int trimmoe_stack_forward_static(const trimmoe_model* m, const trimmoe_policy* p,
                                 trimmoe_state* s, trimmoe_trace* trace, void* stream);

/*
 * Kernel classes of one layer, in launch order, as timed by
 * trimmoe_stack_forward_timed.
 */
#define TRIMMOE_TIMED_CLASSES 8
#define TRIMMOE_CLASS_ROUTE 0    /* substitution table + route/decide       */
#define TRIMMOE_CLASS_BUCKET 1   /* expert offsets/tiles + row permutation  */
#define TRIMMOE_CLASS_UP 2       /* grouped up/gate GEMM + activation       */
#define TRIMMOE_CLASS_DOWN 3     /* grouped down GEMM                       */
#define TRIMMOE_CLASS_SHARED 4   /* shared expert up + down GEMMs           */
#define TRIMMOE_CLASS_COMBINE 5  /* weighted combine + residual             */
#define TRIMMOE_CLASS_EXIT 6     /* exit-head GEMM with softmax partials    */
#define TRIMMOE_CLASS_GATE 7     /* exit gate + active-list compaction      */

/*
 * trimmoe_stack_forward, additionally recording caller-created HIP events
 * (hipEvent_t passed as void*, created with timing enabled) on `stream`:
 * events[l * (TRIMMOE_TIMED_CLASSES + 1) + c] before kernel class c of layer
 * l and events[l * (TRIMMOE_TIMED_CLASSES + 1) + c + 1] after it (a class
 * with no launch gives two back-to-back records).  n_events must be
 * N * (TRIMMOE_TIMED_CLASSES + 1).  For measurement: the work is identical
 * to trimmoe_stack_forward; nothing is synchronised.
 */
int trimmoe_stack_forward_timed(const trimmoe_model* m, const trimmoe_policy* p,
                                trimmoe_state* s, trimmoe_trace* trace,
                                void* workspace, size_t workspace_bytes,
                                void* stream, void* const* events,
                                int32_t n_events);

/*
 * Engine-clock record of the GEMM kernels (measurement; no passage of the
 * method).  While set, each block of a bf16 GEMM launch of class c
 * (TRIMMOE_CLASS_UP, _DOWN, _SHARED or _EXIT) adds to rec[2 c] the core clock
 * cycles and to rec[2 c + 1] the ticks of the 100 MHz constant clock that
 * pass between its start and the end of its last tile (blocks with no tile
 * add nothing), so 100 MHz * rec[2 c] / rec[2 c + 1] is the mean engine clock
 * the class ran at.  rec: device memory of 2 * TRIMMOE_TIMED_CLASSES uint64
 * words on the current device, zeroed and owned by the caller, which keeps
 * it allocated while set; NULL stops recording.  The setting is process-wide
 * and applies to layer steps issued after the call on that device (the
 * record is read when a layer's launches are issued; launches on other
 * devices record nothing); the work and results are otherwise identical.
 * Returns TRIMMOE_OK, or TRIMMOE_ERR_HIP when the current device cannot be
 * queried.
 */
int trimmoe_set_clock_record(uint64_t* rec);


/*
 * Runtime feedback (Sec. V-D Eq. (37), Sec. V-F Eq. (43)) over an
 * observation window of stack passes.
 *
 * trimmoe_window_stats adds one pass's observations to stats[0..5] (device
 * memory, 6 doubles, caller-owned and caller-zeroed at the start of a
 * window): tokens, tokens that exited, sum of their confidence at exit, sum
 * over tokens of D-hat / budget (0 where the budget is 0), delay of the
 * executed slots (t_local per local exact or substitute slot, t_remote per
 * remote exact slot), and the reference delay of full-depth exact
 * execution on the same placement (Eq. (21)): per layer, T * k times the
 * mean per-slot delay of the routed targets of the tokens active there
 * (the mean over the whole pass for a layer no token reached; 0 for an
 * empty pass).  Reads the state left by the pass and trace->counters (the
 * only trace field needed); one small kernel on `stream`, fixed summation
 * order.
 */
int trimmoe_window_stats(const trimmoe_model* m, const trimmoe_policy* p,
                         const trimmoe_state* s, const trimmoe_trace* trace,
                         double* stats, void* stream);

/*
 * Host-only update of p->p_exit and p->omega_t from a window's stats
 * (host copy of the 6 doubles above):
 *   Eq. (37): p_J <- clip(p_J + eta (xi_exit_mean - p_J), [p_floor, 1]),
 *             unchanged when no token exited;
 *   Eq. (43): omega_D <- clip(omega_D + kappa (D_mean - T_norm), [0, 1]),
 *             omega_T <- 1 - omega_D, with D_mean = stats[3] / stats[0] and
 *             T_norm = stats[4] / stats[5]; unchanged when stats[0] or
 *             stats[5] is 0.
 * eta, kappa >= 0, p_floor in [0, 1]; stats finite and >= 0; else
 * TRIMMOE_ERR_POLICY and *p unchanged.
 */
int trimmoe_feedback_update(trimmoe_policy* p, const double* stats, double eta,
                            double kappa, double p_floor);

/*
 * Offline statistics and replica placement (Table I), host-only functions:
 * all pointers are host memory owned by the caller; arguments are checked
 * before anything is written.
 *
 * A calibration record is what a full-depth exact pass of the stack writes
 * into its trace (budget 0 and a confidence requirement above 1, so that
 * nothing is skipped, substituted or exited): trace->target [N, Q, k],
 * trace->importance [N, Q], trace->xi [N, Q] (NaN where not evaluated).
 *
 * trimmoe_calib_exit_layers: per calibration token, the first layer l < N - 1
 * whose confidence xi[l][q] >= p_exit (0-based), else N: the layer after
 * which the exit gate of Eq. (8) would let it leave.
 */
int trimmoe_calib_exit_layers(int32_t n_layers, int32_t n_tokens, const float* xi, float p_exit,
                              int32_t* exit_layer);

/*
 * Execution-frequency statistics of Sec. IV-C: pi[l] (Eq. (26)) the
 * fraction of tokens active entering layer l (exit_layer[q] >= l);
 * act[l][e] the fraction of those whose routed set contains e; sigma[l][e]
 * (Eq. (27)) the fraction of the latter whose importance exceeds theta[l]
 * (0 when none); lambda = pi * sigma * act.  target [N, Q, k] int16 in
 * [0, E); outputs fp64, [N] and [N, E].
 */
int trimmoe_calib_stats(int32_t n_layers, int32_t n_tokens, int32_t n_experts, int32_t top_k,
                        const int16_t* target, const float* importance,
                        const int32_t* exit_layer, const float* theta, double* pi, double* act,
                        double* sigma, double* lambda);

/*
 * Expert transition statistics P_l (Eq. (38)) for l < N - 1 from a
 * calibration record, in the layout the look-ahead reads: row e of layer l
 * holds the trans_b most frequent next-layer experts (ties to the lower
 * id), probabilities renormalised over them, padded with (-1, 0).  With
 * top-k every (routed at l, routed at l + 1) pair of a token active at both
 * layers counts once.  trans_to / trans_p: [N - 1, E, trans_b];
 * 1 <= trans_b <= E.
 */
int trimmoe_calib_transitions(int32_t n_layers, int32_t n_tokens, int32_t n_experts,
                              int32_t top_k, const int16_t* target, const int32_t* exit_layer,
                              int32_t trans_b, int16_t* trans_to, float* trans_p);

/*
 * Communication-aware greedy replication (Table I, lines 9-13): starting
 * from the baseline deployment x [M, N, E] (1 = expert (l, e) on server m),
 * which must satisfy (c.1)-(c.3), repeatedly place the replica of largest
 * redundancy benefit B = lambda[l][e] * rho[m][l] * (z[l] / mean bandwidth
 * + mean latency) (Eq. (28); means over the servers hosting the expert,
 * from bandwidth / latency [M, M]) among the pairs not yet placed that fit
 * the server's residual memory (capacity [M], nbytes [N, E]); ties to the
 * lower layer, expert, server; stop when no positive benefit fits.  x is
 * updated in place; *n_placed = replicas added.  By Property 1 the result
 * satisfies (c.1)-(c.3).  A baseline that violates them: TRIMMOE_ERR_SHAPE;
 * negative, NaN or infinite inputs (bandwidth must be > 0):
 * TRIMMOE_ERR_POLICY.  Row x[m] of the result is the local_mask of every
 * layer for a device playing server m.
 */
int trimmoe_place_replicas(int32_t n_servers, int32_t n_layers, int32_t n_experts,
                           const double* lambda, const double* rho, const double* z,
                           const double* nbytes, const double* capacity,
                           const double* bandwidth, const double* latency, uint8_t* x,
                           int32_t* n_placed);

/*
 * Exit-head training (Sec. IV-A) on cached hidden states.  Device memory,
 * caller-owned; work is enqueued on `stream`; arguments are checked before
 * anything is enqueued.
 *
 * trimmoe_head_argmax: argmax[q] = argmax_v (w_head[v] . h[q] + b_head[v])
 * over the V rows of an output head w_head [V, d] (ties to the lower v): the
 * prediction of a representation, from which the consistency labels of
 * Eq. (22) follow.  h [n_rows, d] and w_head in `dtype` (bf16: d a multiple
 * of 64, both 16-byte aligned); b_head fp32 [V] or NULL; argmax int32
 * [n_rows].  Needs a 256-byte aligned workspace of
 * trimmoe_head_argmax_workspace_size(dtype, V, n_rows) bytes.
 */
int trimmoe_head_argmax_workspace_size(int32_t dtype, int32_t vocab, int32_t n_rows,
                                       size_t* bytes);
int trimmoe_head_argmax(int32_t dtype, int32_t vocab, int32_t d_model, int32_t n_rows,
                        const void* w_head, const float* b_head, const void* h, int32_t* argmax,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * trimmoe_consistency_labels: Eq. (22), labels[q] = (pred[q] == ref[q]) for
 * the predictions of one layer and of full depth (int32 [n_rows] each, from
 * trimmoe_head_argmax); labels uint8 [n_rows].
 */
int trimmoe_consistency_labels(int32_t n_rows, const int32_t* pred, const int32_t* ref,
                               uint8_t* labels, void* stream);

/*
 * trimmoe_train_exit_head: `epochs` steps of full-batch gradient descent of
 * the exit head xi = sigmoid(w . h + c) on the binary cross-entropy of
 * Eq. (23) against labels[q] in {0, 1} (uint8 [n_rows]):
 * w -= lr * mean_q (xi_q - y_q) h_q and c -= lr * mean_q (xi_q - y_q).
 * w (fp32 [d]) and c (fp32 [1]) hold the start on entry and the trained head
 * on return; loss (fp32 [epochs], or NULL) receives Eq. (23) at the weights
 * each epoch starts from.  h [n_rows, d] in `dtype` (bf16: d a multiple of
 * 64).  Sums run in a fixed order in fp64: repeated runs give identical
 * weights.  Needs a 256-byte aligned workspace of
 * trimmoe_train_exit_head_workspace_size(n_rows) bytes.
 */
int trimmoe_train_exit_head_workspace_size(int32_t n_rows, size_t* bytes);
int trimmoe_train_exit_head(int32_t dtype, int32_t d_model, int32_t n_rows, const void* h,
                            const uint8_t* labels, int32_t epochs, float lr, float* w, float* c,
                            float* loss, void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TRIMMOE_H */
