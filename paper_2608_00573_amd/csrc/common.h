// Internal definitions shared by the HIP kernels and the host launcher of
// libtrimmoe (adaptive-depth MoE step, gfx950).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "trimmoe.h"

namespace trimmoe {

typedef uint16_t bf16_t;

// ---------------------------------------------------------------- tiling --
// tokens handled by one block of the route and permute kernels (at most;
// with look-ahead a small batch uses fewer per block: route_block_tokens)
constexpr int kRouteTokens = 32;
// route blocks the look-ahead aims for: one per CU
constexpr int kLookaheadBlocks = 256;

// tokens per route block for a batch of T tokens: kRouteTokens, or with
// look-ahead the power of two that gives about kLookaheadBlocks blocks
inline int route_block_tokens(int T, bool lookahead) {
  if (!lookahead) return kRouteTokens;
  int rb = 1;
  while (rb < kRouteTokens && 2 * rb * kLookaheadBlocks <= T) rb *= 2;
  return rb;
}
// route blocks the workspace provides for batches of up to T tokens
inline int route_blocks_max(int T) {
  const int full = (T + kRouteTokens - 1) / kRouteTokens;
  const int la = T < 2 * kLookaheadBlocks ? T : 2 * kLookaheadBlocks;
  return full > la ? full : la;
}
// rows of an expert group covered by one grouped-GEMM tile: kGemmBM, or
// kBigBM for the large-group core (bf16 batches with at least
// kBigRowsPerExpert rows per expert on average)
constexpr int kGemmBM = 128;
constexpr int kBigBM = 256;
constexpr int kBigRowsPerExpert = 1024;
// the large-group down GEMM cuts the tiles of its last round into at most
// kSkPieces runs of K slices, with at most kSkSlots 256 x 256 extra partials
constexpr int kSkPieces = 8;
constexpr int kSkSlots = 256;
// the dense shared-expert GEMMs use the large-group core from this many tokens
constexpr int kBigDenseTokens = 2048;
// the large-group core addresses its operands with 32-bit byte offsets
inline bool big_offsets_fit(long long rows, long long cols) {
  return rows * cols * 2 < (1ll << 31);
}
inline int expert_tile_rows(bool bf16, int T, int k, int E, int d, int F) {
  const long long R = (long long)T * k;
  return bf16 && R >= (long long)kBigRowsPerExpert * E && big_offsets_fit(T, d) &&
                 big_offsets_fit(R, F)
             ? kBigBM
             : kGemmBM;
}
inline bool big_dense(bool bf16, int T, int d, int Fs) {
  return bf16 && T >= kBigDenseTokens && big_offsets_fit(T, d) && big_offsets_fit(T, Fs);
}
// the exit head uses the large-group core for wide models and large batches
// (its 256-row vocabulary tiles match kExitTileBF16)
constexpr int kBigExitTokens = 1024;
constexpr int kBigExitDModel = 2048;
inline bool big_exit(bool bf16, int T, int V, int d) {
  return bf16 && T >= kBigExitTokens && d >= kBigExitDModel && big_offsets_fit(V, d) &&
         big_offsets_fit(T, d);
}
// batches of this many tokens or more use the 256-token exit-head tile
constexpr int kWideTokens = 4096;
constexpr int kGemmBN = 128;
constexpr int kGemmBK = 64;
// vocabulary rows of one exit-head tile (bf16 MFMA path / fp32 path); bf16
// batches of kExitSmallTokens or fewer use kExitTileBF16Small-row tiles, so
// that a decode-sized batch still spreads W_exit over every CU
constexpr int kExitTileBF16 = 256;
constexpr int kExitTileBF16Small = 128;
constexpr int kExitSmallTokens = 64;
constexpr int kExitTileF32 = 16;

inline int exit_tile_rows(bool bf16, int T) {
  return bf16 ? (T <= kExitSmallTokens ? kExitTileBF16Small : kExitTileBF16) : kExitTileF32;
}
// fp32 GEMM tile
constexpr int kF32Tile = 16;
// per-layer trace counters (row stride of trimmoe_trace.counters)
constexpr int kCounters = 16;
// look-ahead: later layers a decision looks at, and first-level branches
// (candidate action, next-layer target tuple) per token
constexpr int kMaxLookahead = TRIMMOE_MAX_HORIZON - 1;
constexpr int kMaxBranches = 1024;

// slots of the small device counter block in the workspace
enum CountSlot {
  kCntRows = 0,   // merged (token, expert) rows of this layer
  kCntTiles = 1,  // grouped-GEMM row tiles
  kCntExec = 2,   // executed tokens
  kCntSlots = 8
};

// --------------------------------------------------------------- numbers --
__device__ __forceinline__ float bf2f(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// fp32 -> bf16, round to nearest, ties to even (NaN stays NaN)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f2bf(v); }

// --------------------------------------------------- per-layer arguments --
// Everything one layer's kernels need, passed by value.
struct LayerParams {
  // model
  int N, d, E, k, F, Fs, V, act, conf_mode, normalize, layer;
  // layer tensors
  const void* w_router;
  const float* b_router;
  const void* w_up;
  const void* w_gate;
  const void* w_down;
  const void* ws_up;
  const void* ws_gate;
  const void* ws_down;
  const void* w_exit;
  const float* b_exit;
  const uint8_t* local_mask;
  const float* sim;
  float theta, skip_slope;
  // policy
  float p_exit, budget, omega_t, t_local, t_remote, phi_scale, sim_min;
  const float* p_exit_tok;
  const float* budget_tok;
  // look-ahead (Eq. (39)): la_*[j - 1] describe layer + j for j = 1 ..
  // horizon - 1; la_tto/la_tp[j] the transitions from layer + j to the next
  int horizon;  // effective horizon: min(policy horizon, N - layer)
  int la_subs;  // look-ahead: local substitute candidates per remote slot (1 at H = 1)
  int trans_b;
  int rb;       // tokens per route block (route, scan and bucket agree on it)
  int bm;       // rows per expert tile of the grouped GEMMs (kGemmBM or kBigBM)
  const uint8_t* la_mask[kMaxLookahead];
  const float* la_sim[kMaxLookahead];
  float la_theta[kMaxLookahead], la_slope[kMaxLookahead];
  const int16_t* la_tto[kMaxLookahead];
  const float* la_tp[kMaxLookahead];
  // state
  int T;
  void* h;
  float* d_acc;
  int32_t* active_idx;
  int32_t* n_active;
  int32_t* exit_layer;
  float* xi;
  // trace (already offset to this layer's rows; all NULL when no trace)
  int8_t* tr_action;
  int16_t* tr_target;
  int16_t* tr_exec;
  int8_t* tr_kind;
  float* tr_gate;
  float* tr_importance;
  float* tr_xi;
  float* tr_d_acc;
  int32_t* tr_counters;
  // workspace
  int32_t* tok_exec;   // [T*k] merged rows per active position, -1 padded
  float* tok_w;        // [T*k]
  int32_t* tok_row;    // [T*k] permuted row of each merged row
  int32_t* tok_action; // [T]   ACT_EXEC / ACT_SKIP per active position
  int32_t* tok_keep;   // [T]   1 = still active after this layer
  int32_t* exec_list;  // [T]   token id of each executed token (active order)
  int32_t* exec_pos;   // [T]   active position of each executed token
  int32_t* blk_cnt;    // [nblk*E]
  int32_t* blk_off;    // [nblk*E]
  int32_t* blk_xcnt;   // [nblk]
  int32_t* blk_xoff;   // [nblk]
  int32_t* exp_off;    // [E+1]
  int32_t* counts;     // [kCntSlots]
  int4* tiles;         // [max_tiles] (expert, row begin, row end, 0)
  int32_t* exp_toff;   // [E]   first tile of each expert in `tiles`
  int32_t* sk_flag;    // [max_tiles * cdiv(d, 256)] large-group down GEMM: per tile,
                       // 0 (whole) or (first compact partial << 4 | pieces) when
                       // its K slices were cut; NULL when the layer's down GEMM
                       // is not on that core
  float* sk_part;      // [kSkSlots][256][256] compact partials of later pieces
  int32_t* row_src;    // [T*k] token whose h row feeds each permuted row
  void* act_buf;       // [T*k, F]
  float* y_buf;        // [down_splits][T*k, d] partial down-projection slices
  size_t y_split_stride;  // elements between slices of y_buf
  int down_splits;     // K splits of the routed down GEMM (bf16 path)
  void* act_s;         // [T, Fs]
  float* y_s;          // [T, d]
  void* hx;            // [T, d]    updated rows of executed tokens (exit input)
  float2* partials;    // [T, n_vtiles] (max, sum exp) per vocabulary tile
  int n_vtiles;
  int max_tiles;
  int n_cu;            // compute units of the device (persistent grids)
  // engine-clock record (measurement): [class][2] sums of core cycles and
  // 100 MHz ticks per GEMM block, or NULL
  unsigned long long* clk;
};

// observations of one stack pass for the runtime feedback rules
struct WindowArgs {
  int T, N, k;
  const int32_t* exit_layer;  // [T]
  const float* xi;            // [T]
  const float* d_acc;         // [T]
  const float* budget_tok;    // [T] or NULL
  float budget, t_local, t_remote;
  const int32_t* counters;    // trace counters [N, kCounters]
  double* stats;              // [6], accumulated
};

// launchers (decide.hip)
hipError_t launch_state_reset(const trimmoe_model* m, const trimmoe_state* s,
                              hipStream_t st);
// inactive defaults of the trace rows of n_layers consecutive layers, from
// the layer p's trace pointers point at
hipError_t launch_trace_fill(const LayerParams& p, int n_layers, hipStream_t st);
hipError_t launch_route(const LayerParams& p, bool bf16, hipStream_t st);
hipError_t launch_scan(const LayerParams& p, hipStream_t st);
hipError_t launch_bucket(const LayerParams& p, hipStream_t st);
hipError_t launch_combine(const LayerParams& p, bool bf16, hipStream_t st);
hipError_t launch_exit_reduce(const LayerParams& p, hipStream_t st);
hipError_t launch_compact(const LayerParams& p, hipStream_t st);
// exit-head training (Sec. IV-A): per-tile (max logit, row) partials of an
// output head over rows of hidden states (head.hip reduces them to argmax)
hipError_t launch_head_argmax_partials(bool bf16, const void* W, const float* bias, const void* H,
                                       const int* n_rows_dev, int n_rows, int V, int K,
                                       int n_vtiles, float2* partials, int n_cu, hipStream_t st);
hipError_t launch_argmax_reduce(const float2* partials, int n_vtiles, int n_rows, int32_t* out,
                                hipStream_t st);
hipError_t launch_consistency(const int32_t* pred, const int32_t* ref, int n_rows,
                              uint8_t* labels, hipStream_t st);
// *p = v on the stream (a kernel, so that the call can be captured)
hipError_t launch_set_int(int32_t* p, int v, hipStream_t st);
// one full-batch descent step of the sigmoid exit head on BCE (Eq. (23)):
// residuals r = sigmoid(w . h + c) - y and per-row losses, then the update
hipError_t launch_bce_step(bool bf16, const void* H, const uint8_t* y, int n_rows, int d,
                           float lr, float* w, float* c, float* r, double* row_loss,
                           float* loss_out, hipStream_t st);
hipError_t launch_window_stats(const WindowArgs& w, hipStream_t st);

// launchers (gemm.hip)
hipError_t launch_expert_up(const LayerParams& p, bool bf16, hipStream_t st);
hipError_t launch_expert_down(const LayerParams& p, bool bf16, hipStream_t st);
hipError_t launch_shared_expert(const LayerParams& p, bool bf16, hipStream_t st);
hipError_t launch_exit_head(const LayerParams& p, bool bf16, hipStream_t st);
int down_splits(int max_tiles, int N, int K);
// dynamic LDS of a route block (logits, and the look-ahead tables at H > 1)
size_t route_lds_bytes(bool bf16, int E, int d, int horizon, int trans_b, int k, int la_subs);
// dynamic LDS a route block may take next to its static arrays (about 10 KB;
// gfx950: 160 KB per workgroup)
constexpr size_t kRouteLdsMax = 148 * 1024;

}  // namespace trimmoe
