// Matrix kernels of the adaptive-depth MoE step (gfx950):
//   * grouped expert FFN over the executed (token, expert) rows:
//       up/gate GEMM with the activation fused in the epilogue, output bf16
//       (SwiGLU: silu(G) * U; ReLU: relu(U)), then the down GEMM, output fp32;
//   * exit head (Sec. III-C, Eq. (7)): logits = W_exit h for the executed
//     tokens, reduced in the epilogue to a per-(token, vocabulary tile)
//     (max, sum exp) pair so the logits never reach memory.
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation, 128x128 block
// tiles of 4 wavefronts (64x64 each), K staged through LDS in 64-wide slices
// with double buffering.  Both operands are K-contiguous ("NT"): A is
// [M, K], B is [N, K] and C = A B^T.  Block ids are remapped so that each
// XCD works on a contiguous run of tiles ordered in 8-tile-tall column
// patches, which keeps the operand slices of concurrent blocks in that
// XCD's L2.  fp32 path: plain FMA kernels for fp32 models.
#include <math.h>

#include "common.h"

namespace trimmoe {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int BM = kGemmBM, BN = kGemmBN, BK = kGemmBK;
constexpr int LDSK = BK + 8;  // padded LDS row (144 B): conflict-free b128 reads
constexpr int kPatch = 8;     // tiles per patch column in the block order
constexpr int kXcd = 8;       // XCDs of an MI355X; blocks are dealt round-robin

static_assert(BM == 128 && BN == 128 && BK == 64, "tile mapping below assumes 128x128x64");

// -------------------------------------------------- block order remapping --
// Hardware deals block b to XCD b % 8.  Give XCD x the contiguous logical
// range [x*q + min(x, r), ...) of the `total` live tiles (a bijection on
// [0, total)), then read the logical index in patch order: kPatch M-tiles of
// one N-tile, then the next N-tile.
__device__ __forceinline__ bool map_tile(int b, int total, int n_mt, int n_nt, int& mt, int& nt) {
  if (b >= total) return false;
  const int q = total / kXcd, r = total % kXcd;
  const int x = b % kXcd, i = b / kXcd;
  const int L = x * q + min(x, r) + i;
  const int span = kPatch * n_nt;
  const int g = L / span, w = L % span;
  const int gm = min(kPatch, n_mt - g * kPatch);
  nt = w / gm;
  mt = g * kPatch + w % gm;
  return true;
}

// --------------------------------------------------------------- mainloop --
template <bool DUAL>
struct Smem {
  bf16_t a[2][BM * LDSK];
  bf16_t b0[2][BN * LDSK];
  bf16_t b1[DUAL ? 2 : 1][DUAL ? BN * LDSK : 8];
};

// acc0 += A B0^T, acc1 += A B1^T over the full K.  A and B* point at the
// first row of the tile; rows at or beyond a_valid / b_valid read as zero.
template <bool DUAL>
__device__ __forceinline__ void gload(const bf16_t* __restrict__ A, int a_valid,
                                      const bf16_t* __restrict__ B0,
                                      const bf16_t* __restrict__ B1, int b_valid, int K, int k0,
                                      int lr, int lc, uint4 (&ra)[4], uint4 (&rb0)[4],
                                      uint4 (&rb1)[4]) {
  // Rows past the valid range load a clamped (valid) row and are zeroed by
  // a value select, so every load is unconditional and nothing needs memory.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = lr + 32 * i;
    const int rowa = min(row, a_valid - 1), rowb = min(row, b_valid - 1);
    uint4 va = *reinterpret_cast<const uint4*>(A + (size_t)rowa * K + k0 + lc);
    uint4 vb0 = *reinterpret_cast<const uint4*>(B0 + (size_t)rowb * K + k0 + lc);
    const bool oka = row < a_valid, okb = row < b_valid;
    ra[i] = make_uint4(oka ? va.x : 0u, oka ? va.y : 0u, oka ? va.z : 0u, oka ? va.w : 0u);
    rb0[i] = make_uint4(okb ? vb0.x : 0u, okb ? vb0.y : 0u, okb ? vb0.z : 0u, okb ? vb0.w : 0u);
    if constexpr (DUAL) {
      uint4 vb1 = *reinterpret_cast<const uint4*>(B1 + (size_t)rowb * K + k0 + lc);
      rb1[i] = make_uint4(okb ? vb1.x : 0u, okb ? vb1.y : 0u, okb ? vb1.z : 0u, okb ? vb1.w : 0u);
    }
  }
}

template <bool DUAL>
__device__ __forceinline__ void sstore(Smem<DUAL>& sm, int s, int lr, int lc, const uint4 (&ra)[4],
                                       const uint4 (&rb0)[4], const uint4 (&rb1)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = lr + 32 * i;
    *reinterpret_cast<uint4*>(&sm.a[s][row * LDSK + lc]) = ra[i];
    *reinterpret_cast<uint4*>(&sm.b0[s][row * LDSK + lc]) = rb0[i];
    if constexpr (DUAL) *reinterpret_cast<uint4*>(&sm.b1[s][row * LDSK + lc]) = rb1[i];
  }
}

template <bool DUAL>
__device__ __forceinline__ void mma_slice(const Smem<DUAL>& sm, int s, int wm, int wn, int fr,
                                          int fk, f32x16_t (&acc0)[2][2],
                                          f32x16_t (&acc1)[2][2]) {
#pragma unroll
  for (int ks = 0; ks < BK / 16; ++ks) {
    bf16x8_t af[2], bf0[2], bf1[2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
      af[mi] = *reinterpret_cast<const bf16x8_t*>(&sm.a[s][(wm * 64 + mi * 32 + fr) * LDSK + ks * 16 + fk]);
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      bf0[ni] = *reinterpret_cast<const bf16x8_t*>(&sm.b0[s][(wn * 64 + ni * 32 + fr) * LDSK + ks * 16 + fk]);
      if constexpr (DUAL)
        bf1[ni] = *reinterpret_cast<const bf16x8_t*>(&sm.b1[s][(wn * 64 + ni * 32 + fr) * LDSK + ks * 16 + fk]);
    }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        acc0[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bf0[ni], acc0[mi][ni], 0, 0, 0);
        if constexpr (DUAL)
          acc1[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bf1[ni], acc1[mi][ni], 0, 0, 0);
      }
  }
}

template <bool DUAL>
__device__ __forceinline__ void mma_mainloop(const bf16_t* __restrict__ A, int a_valid,
                                             const bf16_t* __restrict__ B0,
                                             const bf16_t* __restrict__ B1, int b_valid, int K,
                                             f32x16_t (&acc0)[2][2], f32x16_t (&acc1)[2][2],
                                             Smem<DUAL>& sm) {
  const int tid = threadIdx.x;
  const int lr = tid >> 3, lc = (tid & 7) * 8;  // load row / column (elements)
  const int wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 31, fk = (lane >> 5) * 8;  // fragment row, k offset
  uint4 ra[4], rb0[4], rb1[4];
  const f32x16_t zacc = {};
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      acc0[mi][ni] = zacc;
      if constexpr (DUAL) acc1[mi][ni] = zacc;
    }

  const int nk = K / BK;
  gload<DUAL>(A, a_valid, B0, B1, b_valid, K, 0, lr, lc, ra, rb0, rb1);
  sstore<DUAL>(sm, 0, lr, lc, ra, rb0, rb1);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload<DUAL>(A, a_valid, B0, B1, b_valid, K, (kt + 1) * BK, lr, lc, ra, rb0, rb1);
    mma_slice<DUAL>(sm, kt & 1, wm, wn, fr, fk, acc0, acc1);
    if (kt + 1 < nk) sstore<DUAL>(sm, (kt + 1) & 1, lr, lc, ra, rb0, rb1);
    __syncthreads();
  }
}

// accumulator element -> tile-local (row, col)
__device__ __forceinline__ int acc_row(int wm, int mi, int r, int lane) {
  return wm * 64 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
__device__ __forceinline__ int acc_col(int wn, int ni, int lane) { return wn * 64 + ni * 32 + (lane & 31); }

// ------------------------------------------------------ grouped FFN GEMMs --
// Rows come in expert groups; tile list entry = (expert, row begin, row end).
// Dense mode (shared expert): one group, rows [0, *dense_rows).
struct FfnArgs {
  const bf16_t* X;          // [rows, K]
  const bf16_t* W0;         // expert 0 of [E, N, K] (up, or down)
  const bf16_t* W1;         // gate, same layout, or NULL
  size_t w_stride;          // elements between experts
  int K, N;
  const int4* tiles;        // grouped mode
  const int* n_tiles;       // grouped mode: live tiles (device)
  const int* dense_rows;    // dense mode: live rows (device), else NULL
  void* out;                // up: bf16 [rows, N]; down: f32 [rows, N]
  int act;                  // up: TRIMMOE_ACT_*
};

template <bool DUAL, bool UP>
__global__ __launch_bounds__(256) void k_ffn_mma(FfnArgs a) {
  __shared__ Smem<DUAL> sm;
  const int n_nt = (a.N + BN - 1) / BN;
  int n_mt;
  if (a.dense_rows)
    n_mt = (*a.dense_rows + BM - 1) / BM;
  else
    n_mt = *a.n_tiles;
  int mt, ntile;
  if (!map_tile(blockIdx.x, n_mt * n_nt, n_mt, n_nt, mt, ntile)) return;
  int e, m0, m1;
  if (a.dense_rows) {
    e = 0;
    m0 = mt * BM;
    m1 = *a.dense_rows;
  } else {
    const int4 tl = a.tiles[mt];
    e = tl.x;
    m0 = tl.y;
    m1 = tl.z;
  }
  const int n0 = ntile * BN;
  const int a_valid = min(BM, m1 - m0);
  const int b_valid = min(BN, a.N - n0);
  const bf16_t* W0 = a.W0 + (size_t)e * a.w_stride + (size_t)n0 * a.K;
  const bf16_t* W1 = DUAL ? a.W1 + (size_t)e * a.w_stride + (size_t)n0 * a.K : nullptr;
  f32x16_t acc0[2][2], acc1[2][2];
  mma_mainloop<DUAL>(a.X + (size_t)m0 * a.K, a_valid, W0, W1, b_valid, a.K, acc0, acc1, sm);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int col = acc_col(wn, ni, lane);
      if (col >= b_valid) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = acc_row(wm, mi, r, lane);
        if (row >= a_valid) continue;
        const size_t o = (size_t)(m0 + row) * a.N + n0 + col;
        if constexpr (UP) {
          const float u = acc0[mi][ni][r];
          float v;
          if constexpr (DUAL) {
            const float g = acc1[mi][ni][r];
            v = g / (1.f + expf(-g)) * u;  // silu(g) * u
          } else {
            v = fmaxf(u, 0.f);
          }
          static_cast<bf16_t*>(a.out)[o] = f2bf(v);
        } else {
          static_cast<float*>(a.out)[o] = acc0[mi][ni][r];
        }
      }
    }
}

// ----------------------------------------------------------- exit head --
// M = vocabulary (A = W_exit [V, d]), N = executed tokens (B = hx [n_x, d]).
// Epilogue: for every token column, max and sum exp over the tile's
// vocabulary rows (bias added), written as one partial per vocabulary tile.
struct ExitArgs {
  const bf16_t* W;   // [V, K]
  const bf16_t* H;   // [n_x, K]
  const float* bias; // [V] or NULL
  const int* n_exec; // device
  int V, K, n_vtiles;
  float2* partials;  // [n_x, n_vtiles]
};

__global__ __launch_bounds__(256) void k_exit_mma(ExitArgs a) {
  __shared__ Smem<false> sm;
  __shared__ float2 s_part[2][BN];  // per wm half: (max, sum) per token column
  const int n_x = *a.n_exec;
  const int n_mt = a.n_vtiles, n_nt = (n_x + BN - 1) / BN;
  int mt, nt;
  if (!map_tile(blockIdx.x, n_mt * n_nt, n_mt, n_nt, mt, nt)) return;
  const int v0 = mt * BM, j0 = nt * BN;
  const int a_valid = min(BM, a.V - v0);
  const int b_valid = min(BN, n_x - j0);
  f32x16_t acc0[2][2], acc1[2][2];
  mma_mainloop<false>(a.W + (size_t)v0 * a.K, a_valid, a.H + (size_t)j0 * a.K, nullptr, b_valid,
                      a.K, acc0, acc1, sm);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const float ninf = -__builtin_inff();
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    float m = ninf;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = acc_row(wm, mi, r, lane);
        float x = acc0[mi][ni][r];
        if (row < a_valid) {
          if (a.bias) x += a.bias[v0 + row];
        } else {
          x = ninf;
        }
        acc0[mi][ni][r] = x;
        m = fmaxf(m, x);
      }
    m = fmaxf(m, __shfl_xor(m, 32));
    float s = 0.f;
    if (m != ninf) {
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += expf(acc0[mi][ni][r] - m);
    }
    s += __shfl_xor(s, 32);
    if (lane < 32) s_part[wm][acc_col(wn, ni, lane)] = make_float2(m, s);
  }
  __syncthreads();
  const int c = threadIdx.x;
  if (c < b_valid) {
    const float2 p0 = s_part[0][c], p1 = s_part[1][c];
    const float M = fmaxf(p0.x, p1.x);
    float S = 0.f;
    if (p0.y > 0.f) S += p0.y * expf(p0.x - M);
    if (p1.y > 0.f) S += p1.y * expf(p1.x - M);
    a.partials[(size_t)(j0 + c) * a.n_vtiles + mt] = make_float2(M, S);
  }
}

// ------------------------------------------------------------- fp32 path --
constexpr int FT = kF32Tile;

// out[m][n] = X[m] . W[e][n] over a 128-row group tile, 16 columns per block.
template <bool UP>
__global__ __launch_bounds__(256) void k_ffn_f32(const float* X, const float* W0, const float* W1,
                                                 size_t w_stride, int K, int N, const int4* tiles,
                                                 const int* n_tiles, const int* dense_rows,
                                                 void* out, int act) {
  const int n_nt = (N + FT - 1) / FT;
  const int n_mt = dense_rows ? (*dense_rows + BM - 1) / BM : *n_tiles;
  const int mt = blockIdx.x / n_nt, ntile = blockIdx.x % n_nt;
  if (mt >= n_mt) return;
  int e, m0, m1;
  if (dense_rows) {
    e = 0;
    m0 = mt * BM;
    m1 = *dense_rows;
  } else {
    const int4 tl = tiles[mt];
    e = tl.x;
    m0 = tl.y;
    m1 = tl.z;
  }
  const int tx = threadIdx.x % FT, ty = threadIdx.x / FT;
  const int n = ntile * FT + tx;
  if (n >= N) return;
  const float* w0 = W0 + (size_t)e * w_stride + (size_t)n * K;
  const float* w1 = W1 ? W1 + (size_t)e * w_stride + (size_t)n * K : nullptr;
  for (int m = m0 + ty; m < min(m0 + BM, m1); m += 256 / FT) {
    const float* x = X + (size_t)m * K;
    float u = 0.f, g = 0.f;
    for (int j = 0; j < K; ++j) {
      u = fmaf(x[j], w0[j], u);
      if (w1) g = fmaf(x[j], w1[j], g);
    }
    if constexpr (UP) {
      const float v = act == TRIMMOE_ACT_SWIGLU ? g / (1.f + expf(-g)) * u : fmaxf(u, 0.f);
      static_cast<float*>(out)[(size_t)m * N + n] = v;
    } else {
      static_cast<float*>(out)[(size_t)m * N + n] = u;
    }
  }
}

// exit head, fp32: block = 16 vocabulary rows x 16 tokens
__global__ __launch_bounds__(256) void k_exit_f32(const float* W, const float* H, const float* bias,
                                                  const int* n_exec, int V, int K, int n_vtiles,
                                                  float2* partials) {
  __shared__ float s_z[FT][FT + 1];
  const int n_x = *n_exec;
  const int vt = blockIdx.x % n_vtiles, jt = blockIdx.x / n_vtiles;
  if (jt * FT >= n_x) return;
  const int tv = threadIdx.x / FT, tj = threadIdx.x % FT;
  const int v = vt * FT + tv, j = jt * FT + tj;
  float z = -__builtin_inff();
  if (v < V && j < n_x) {
    const float* w = W + (size_t)v * K;
    const float* h = H + (size_t)j * K;
    float acc = 0.f;
    for (int c = 0; c < K; ++c) acc = fmaf(w[c], h[c], acc);
    z = acc + (bias ? bias[v] : 0.f);
  }
  s_z[tv][tj] = z;
  __syncthreads();
  if (threadIdx.x < FT) {
    const int jj = jt * FT + threadIdx.x;
    if (jj < n_x) {
      float m = -__builtin_inff();
      for (int u = 0; u < FT; ++u) m = fmaxf(m, s_z[u][threadIdx.x]);
      float s = 0.f;
      if (m != -__builtin_inff())
        for (int u = 0; u < FT; ++u) s += expf(s_z[u][threadIdx.x] - m);
      partials[(size_t)jj * n_vtiles + vt] = make_float2(m, s);
    }
  }
}

// ------------------------------------------------------------- launchers --
static inline int cdiv(int a, int b) { return (a + b - 1) / b; }

static hipError_t ffn_pass(const LayerParams& p, bool bf16, bool up, bool shared, hipStream_t st) {
  const int K = up ? p.d : (shared ? p.Fs : p.F);
  const int N = up ? (shared ? p.Fs : p.F) : p.d;
  const bool dual = up && (shared || p.act == TRIMMOE_ACT_SWIGLU);
  const void* w0 = shared ? (up ? p.ws_up : p.ws_down) : (up ? p.w_up : p.w_down);
  const void* w1 = dual ? (shared ? p.ws_gate : p.w_gate) : nullptr;
  const size_t w_stride = shared ? 0 : (size_t)N * K;
  const void* X = up ? (shared ? p.xs : p.x_perm) : (shared ? p.act_s : p.act_buf);
  void* out = up ? (shared ? p.act_s : p.act_buf) : (shared ? (void*)p.y_s : (void*)p.y_buf);
  const int* dense = shared ? &p.counts[kCntExec] : nullptr;
  const int max_mt = shared ? cdiv(p.T, BM) : p.max_tiles;
  const int act = shared ? TRIMMOE_ACT_SWIGLU : p.act;
  if (max_mt <= 0) return hipSuccess;
  if (bf16) {
    FfnArgs a{static_cast<const bf16_t*>(X), static_cast<const bf16_t*>(w0),
              static_cast<const bf16_t*>(w1), w_stride, K, N, p.tiles, &p.counts[kCntTiles],
              dense, out, act};
    const dim3 grid(max_mt * cdiv(N, BN));
    if (up && dual)
      hipLaunchKernelGGL((k_ffn_mma<true, true>), grid, dim3(256), 0, st, a);
    else if (up)
      hipLaunchKernelGGL((k_ffn_mma<false, true>), grid, dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((k_ffn_mma<false, false>), grid, dim3(256), 0, st, a);
  } else {
    const dim3 grid(max_mt * cdiv(N, FT));
    if (up)
      hipLaunchKernelGGL(k_ffn_f32<true>, grid, dim3(256), 0, st, static_cast<const float*>(X),
                         static_cast<const float*>(w0), static_cast<const float*>(w1), w_stride, K,
                         N, p.tiles, &p.counts[kCntTiles], dense, out, act);
    else
      hipLaunchKernelGGL(k_ffn_f32<false>, grid, dim3(256), 0, st, static_cast<const float*>(X),
                         static_cast<const float*>(w0), nullptr, w_stride, K, N, p.tiles,
                         &p.counts[kCntTiles], dense, out, act);
  }
  return hipGetLastError();
}

hipError_t launch_expert_up(const LayerParams& p, bool bf16, hipStream_t st) {
  return ffn_pass(p, bf16, true, false, st);
}

hipError_t launch_expert_down(const LayerParams& p, bool bf16, hipStream_t st) {
  return ffn_pass(p, bf16, false, false, st);
}

hipError_t launch_shared_expert(const LayerParams& p, bool bf16, hipStream_t st) {
  hipError_t e = ffn_pass(p, bf16, true, true, st);
  if (e != hipSuccess) return e;
  return ffn_pass(p, bf16, false, true, st);
}

hipError_t launch_exit_head(const LayerParams& p, bool bf16, hipStream_t st) {
  if (p.T <= 0) return hipSuccess;
  if (bf16) {
    ExitArgs a{static_cast<const bf16_t*>(p.w_exit), static_cast<const bf16_t*>(p.hx), p.b_exit,
               &p.counts[kCntExec], p.V, p.d, p.n_vtiles, p.partials};
    const dim3 grid(p.n_vtiles * cdiv(p.T, BN));
    hipLaunchKernelGGL(k_exit_mma, grid, dim3(256), 0, st, a);
  } else {
    const dim3 grid(p.n_vtiles * cdiv(p.T, FT));
    hipLaunchKernelGGL(k_exit_f32, grid, dim3(256), 0, st, static_cast<const float*>(p.w_exit),
                       static_cast<const float*>(p.hx), p.b_exit, &p.counts[kCntExec], p.V, p.d,
                       p.n_vtiles, p.partials);
  }
  return hipGetLastError();
}

}  // namespace trimmoe
