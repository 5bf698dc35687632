// Matrix kernels of the adaptive-depth MoE step (gfx950):
//   * grouped expert FFN over the executed (token, expert) rows:
//       up/gate GEMM with the activation fused in the epilogue, output bf16
//       (SwiGLU: silu(G) * U; ReLU: relu(U)), then the down GEMM, output fp32
//       (optionally split along K into partial slices that the combine
//       kernel sums in a fixed order);
//   * exit head (Sec. III-C, Eq. (7)): logits = W_exit h for the executed
//     tokens, reduced in the epilogue to a per-(token, vocabulary tile)
//     (max, sum exp) pair so the logits never reach memory.
//
// bf16 path.  Both operands are K-contiguous ("NT"): A is [M, K], B is
// [N, K], C = A B^T, fp32 accumulation in v_mfma_f32_32x32x16_bf16.  A block
// is 4 wavefronts in a 2x2 grid; K advances in 64-wide slices (one 128-byte
// row segment per operand row).  Each thread stages its 16-byte pieces of a
// slice in registers; two register sets and two LDS buffers keep the global
// loads of slices kt+1 and kt+2 in flight while the MFMAs consume slice kt,
// and the compiler only waits for the one older set it is about to store.
// In LDS a row segment keeps its eight 16-byte chunks XOR-swizzled by
// (row & 7), so 8 consecutive rows' 16-byte fragment reads (and the
// 128-byte row writes) hit distinct banks.  Rows past the valid range load a
// clamped valid row (never stored).  Block ids are remapped so that each XCD
// works on a contiguous run of tiles taken in 8-tile-tall column patches.
//
// fp32 path: plain FMA kernels for fp32 models.
#include <math.h>

#include "common.h"

namespace trimmoe {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

constexpr int BK = kGemmBK;  // 64 bf16 = one 128-byte row segment
constexpr int kPatch = 8;    // tiles per patch column in the block order
constexpr int kXcd = 8;      // XCDs of an MI355X; blocks are dealt round-robin

static_assert(BK == 64, "the LDS layout assumes 128-byte row segments");

// -------------------------------------------------- block order remapping --
// Hardware deals block b to XCD b % 8.  Give XCD x the contiguous logical
// range [x*q + min(x, r), ...) of the `total` live tiles (a bijection on
// [0, total)), then read the logical index in patch order: kPatch M-tiles of
// one N-tile, then the next N-tile; the K split (if any) is the slowest index.
__device__ __forceinline__ bool map_tile(int b, int n_mt, int n_nt, int n_split, int& mt, int& nt,
                                         int& sp) {
  const int per = n_mt * n_nt, total = per * n_split;
  if (b >= total) return false;
  const int q = total / kXcd, r = total % kXcd;
  const int x = b % kXcd, i = b / kXcd;
  int L = x * q + min(x, r) + i;
  sp = L / per;
  L -= sp * per;
  const int span = kPatch * n_nt;
  const int g = L / span, w = L % span;
  const int gm = min(kPatch, n_mt - g * kPatch);
  nt = w / gm;
  mt = g * kPatch + w % gm;
  return true;
}

// ---------------------------------------------------------- pipelined core --
// BM x BN block tile, NB B operands sharing A, GM x GN wavefronts
template <int BM_, int BN_, int NB_, int GM_, int GN_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, NB = NB_, GM = GM_, GN = GN_;
  static constexpr int THREADS = 64 * GM * GN;
  static constexpr int WM = BM / GM, WN = BN / GN;  // wavefront tile
  static constexpr int TM = WM / 32, TN = WN / 32;  // MFMA tiles per wavefront
  static constexpr int A_BYTES = BM * 128, B_BYTES = BN * 128;
  static constexpr int STAGE = A_BYTES + NB * B_BYTES;
  static constexpr int LDS = 2 * STAGE;
  static constexpr int ROWS_PER_PASS = THREADS / 8;  // 8 threads per 128-byte row
  static constexpr int A_PT = BM / ROWS_PER_PASS, B_PT = BN / ROWS_PER_PASS;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wavefront tile");
  static_assert(BM % ROWS_PER_PASS == 0 && BN % ROWS_PER_PASS == 0, "load passes");
  static_assert(LDS <= 160 * 1024, "LDS");
};

template <class T>
struct Regs {
  u32x4_t a[T::A_PT];
  u32x4_t b0[T::B_PT];
  u32x4_t b1[T::NB == 2 ? T::B_PT : 1];
};

// A / B* point at row 0 of their matrices.  Tile row r of A is matrix row
// a_idx[r] (a gather through a token list) or a_row0 + r; likewise for B.
struct CoreArgs {
  const bf16_t* A;
  const bf16_t* B0;
  const bf16_t* B1;
  const int* a_idx;
  const int* b_idx;
  int a_row0, b_row0;
  int a_valid, b_valid, K, k_begin, nk;
};

// Per-thread source pointers: thread t loads chunk t%8 of tile rows
// t/8 + i * ROWS_PER_PASS; rows past the valid range use the last valid row.
template <class T>
struct Ptrs {
  const bf16_t* a[T::A_PT];
  const bf16_t* b0[T::B_PT];
  const bf16_t* b1[T::NB == 2 ? T::B_PT : 1];
};

template <class T>
__device__ __forceinline__ void make_ptrs(Ptrs<T>& q, const CoreArgs& c) {
  const int t = threadIdx.x;
  const size_t col = (size_t)c.k_begin + 8 * (t & 7);
#pragma unroll
  for (int i = 0; i < T::A_PT; ++i) {
    const int r = min((t >> 3) + T::ROWS_PER_PASS * i, c.a_valid - 1);
    const int src = c.a_idx ? c.a_idx[r] : c.a_row0 + r;
    q.a[i] = c.A + (size_t)src * c.K + col;
  }
#pragma unroll
  for (int i = 0; i < T::B_PT; ++i) {
    const int r = min((t >> 3) + T::ROWS_PER_PASS * i, c.b_valid - 1);
    const int src = c.b_idx ? c.b_idx[r] : c.b_row0 + r;
    q.b0[i] = c.B0 + (size_t)src * c.K + col;
    if constexpr (T::NB == 2) q.b1[i] = c.B1 + (size_t)src * c.K + col;
  }
}

template <class T>
__device__ __forceinline__ void gload(Regs<T>& r, const Ptrs<T>& q, int kt) {
  const int o = kt * BK;
#pragma unroll
  for (int i = 0; i < T::A_PT; ++i) r.a[i] = *reinterpret_cast<const u32x4_t*>(q.a[i] + o);
#pragma unroll
  for (int i = 0; i < T::B_PT; ++i) {
    r.b0[i] = *reinterpret_cast<const u32x4_t*>(q.b0[i] + o);
    if constexpr (T::NB == 2) r.b1[i] = *reinterpret_cast<const u32x4_t*>(q.b1[i] + o);
  }
}

// 16-byte chunk c of row r sits at chunk c ^ swz(r): 8 consecutive rows, or
// 16 consecutive rows split by parity, then touch distinct bank groups.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

template <class T>
__device__ __forceinline__ void sstore(char* sb, const Regs<T>& r) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < T::A_PT; ++i) {
    const int row = (t >> 3) + i * T::ROWS_PER_PASS;
    *reinterpret_cast<u32x4_t*>(sb + row * 128 + (((t & 7) ^ swz(row)) << 4)) = r.a[i];
  }
#pragma unroll
  for (int i = 0; i < T::B_PT; ++i) {
    const int row = (t >> 3) + i * T::ROWS_PER_PASS;
    const int off = row * 128 + (((t & 7) ^ swz(row)) << 4);
    *reinterpret_cast<u32x4_t*>(sb + T::A_BYTES + off) = r.b0[i];
    if constexpr (T::NB == 2) *reinterpret_cast<u32x4_t*>(sb + T::A_BYTES + T::B_BYTES + off) = r.b1[i];
  }
}

// store piece p of register set r (A rows first, then B0, then B1) into LDS
// stage sb, at the swizzled position sstore uses
template <class T>
__device__ __forceinline__ void sstore_piece(char* sb, const Regs<T>& r, int p) {
  const int t = threadIdx.x;
  if (p < T::A_PT) {
    const int row = (t >> 3) + p * T::ROWS_PER_PASS;
    *reinterpret_cast<u32x4_t*>(sb + row * 128 + (((t & 7) ^ swz(row)) << 4)) = r.a[p];
    return;
  }
  p -= T::A_PT;
  const int i = p % T::B_PT, which = p / T::B_PT;
  const int row = (t >> 3) + i * T::ROWS_PER_PASS;
  const int off = T::A_BYTES + which * T::B_BYTES + row * 128 + (((t & 7) ^ swz(row)) << 4);
  if (which == 0) *reinterpret_cast<u32x4_t*>(sb + off) = r.b0[i];
  else if constexpr (T::NB == 2) *reinterpret_cast<u32x4_t*>(sb + off) = r.b1[i];
}

// One BK slice from LDS stage sb.  Fragments for k-step ks+1 are read while
// the MFMAs of k-step ks run, and the next slice's register set rn goes into
// stage nxt, spread over the k-steps so that the LDS writes overlap
// the MFMAs instead of stalling every wavefront at once; nxt was last read
// before the previous barrier, so it is free.
template <class T>
__device__ __forceinline__ void mma_slice(const char* sb, char* nxt, const Regs<T>& rn,
                                          int wm, int wn, int lane,
                                          f32x16_t (&acc0)[T::TM][T::TN],
                                          f32x16_t (&acc1)[T::TM][T::TN]) {
  constexpr int KS = BK / 16;
  constexpr int NP = T::A_PT + T::B_PT * T::NB;
  const int fr = lane & 31, hi = lane >> 5;
  const int sw = swz(fr);  // fragment rows are 32-aligned offsets plus fr
  bf16x8_t a[2][T::TM], b0[2][T::TN], b1[2][T::NB == 2 ? T::TN : 1];
  auto frag = [&](int ks, int buf) {
    const int ch = ((2 * ks + hi) ^ sw) << 4;
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
      a[buf][i] = *reinterpret_cast<const bf16x8_t*>(sb + (wm * T::WM + i * 32 + fr) * 128 + ch);
#pragma unroll
    for (int j = 0; j < T::TN; ++j) {
      const int o = T::A_BYTES + (wn * T::WN + j * 32 + fr) * 128 + ch;
      b0[buf][j] = *reinterpret_cast<const bf16x8_t*>(sb + o);
      if constexpr (T::NB == 2) b1[buf][j] = *reinterpret_cast<const bf16x8_t*>(sb + T::B_BYTES + o);
    }
  };
  frag(0, 0);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < KS) frag(ks + 1, buf ^ 1);
#pragma unroll
    for (int p = ks * NP / KS; p < (ks + 1) * NP / KS; ++p) sstore_piece<T>(nxt, rn, p);
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
      for (int j = 0; j < T::TN; ++j) {
        acc0[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][i], b0[buf][j], acc0[i][j], 0, 0, 0);
        if constexpr (T::NB == 2)
          acc1[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[buf][i], b1[buf][j], acc1[i][j], 0, 0, 0);
      }
  }
}

// acc0 = A B0^T, acc1 = A B1^T over c.nk slices starting at column c.k_begin.
// Slice kt is computed from LDS buffer kt % 2 while register set (kt+1) % 2
// holds slice kt+1 and set kt % 2 receives slice kt+2.  Every refill load is
// issued unconditionally (past the end it re-reads the last slice, unused),
// so the compiler's load counting stays exact and each LDS store waits only
// for its own, older register set.
template <class T>
__device__ __forceinline__ void gemm_core(char* lds0, char* lds1, const CoreArgs& c,
                                          f32x16_t (&acc0)[T::TM][T::TN],
                                          f32x16_t (&acc1)[T::TM][T::TN]) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave / T::GN, wn = wave % T::GN;
  const f32x16_t z = {};
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j) {
      acc0[i][j] = z;
      if constexpr (T::NB == 2) acc1[i][j] = z;
    }
  Ptrs<T> q;
  make_ptrs<T>(q, c);
  Regs<T> r0, r1;
  const int nk = c.nk, last = c.nk - 1;
  gload<T>(r0, q, 0);
  gload<T>(r1, q, min(1, last));
  sstore<T>(lds0, r0);
  __syncthreads();
  gload<T>(r0, q, min(2, last));
  for (int kt = 0; kt < nk; kt += 2) {
    mma_slice<T>(lds0, lds1, r1, wm, wn, lane, acc0, acc1);  // slice kt; store kt + 1
    __syncthreads();
    gload<T>(r1, q, min(kt + 3, last));
    if (kt + 1 < nk) mma_slice<T>(lds1, lds0, r0, wm, wn, lane, acc0, acc1);
    else sstore<T>(lds0, r0);                                        // slice kt + 2
    __syncthreads();
    gload<T>(r0, q, min(kt + 4, last));
  }
}

#define TRIMMOE_STAGES(T)                               \
  __shared__ __align__(16) char lds_buf0[T::STAGE];     \
  __shared__ __align__(16) char lds_buf1[T::STAGE]

// accumulator element -> tile-local (row, col)
template <class T>
__device__ __forceinline__ int acc_row(int wm, int i, int r, int lane) {
  return wm * T::WM + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
template <class T>
__device__ __forceinline__ int acc_col(int wn, int j, int lane) {
  return wn * T::WN + j * 32 + (lane & 31);
}

// ------------------------------------------------ direct-to-LDS pipeline --
// gfx950's global_load_lds_dwordx4 moves a wavefront's 64 x 16 bytes from
// global memory straight into LDS at a wave-uniform base (lane l at base +
// 16 l): no staging VGPRs and no ds_write, which is what the register-staged
// core above spends most of its non-MFMA issue time on.  Three LDS stages
// form a ring: slice g+2 is in flight while slice g is computed and slice
// g+1 has landed.  Lane l of the DMA that covers tile rows r..r+7 loads row
// r + l/8, chunk (l % 8) ^ swz(row), so the LDS image is the same swizzled
// layout the fragment reads expect.
//
// Waits are explicit.  The compiler cannot tell that a DMA into one stage
// does not alias a read of another, and would wait for every outstanding DMA
// before each fragment read; the fragment reads are therefore inline-asm
// ds_read_b128, and
//   * lgkm_wait<N> (s_waitcnt lgkmcnt(N)) takes the fragments as in/out
//     operands, so the MFMAs that use them cannot be scheduled above it;
//   * slice_barrier<N> (s_waitcnt vmcnt(N) lgkmcnt(0); s_barrier) ends a
//     slice: this wave's DMAs older than the last N have landed and its
//     fragment reads are done, and after the barrier the same holds for all
//     waves, so the next stage may be read and the oldest one rewritten.
// Only LDS DMAs and rare stores are outstanding vector-memory operations in
// these loops; extra newer operations only make a vmcnt wait stricter.
typedef __attribute__((address_space(3))) char lds_char;

__device__ __forceinline__ void dma16(const bf16_t* g, char* l) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)(g),
                                   (lds_char*)(l), 16, 0, 0);
}

__device__ __forceinline__ uint32_t lds_addr(const char* p) {
  return (uint32_t)(uintptr_t)(const lds_char*)(p);
}

__device__ __forceinline__ bf16x8_t lds_read(uint32_t a) {
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
  return v;
}

// the four 32 x 16 fragments one wavefront multiplies per k-step: two A
// fragments (rows +0, +32) and two B fragments (columns +0, +32 of one
// operand, or the same columns of two operands)
struct Frag4 {
  bf16x8_t a0, a1, b0, b1;
};

template <int N>
__device__ __forceinline__ void lgkm_wait(Frag4& f) {
  asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(f.a0), "+v"(f.a1), "+v"(f.b0), "+v"(f.b1) : "n"(N));
}

template <int N>
__device__ __forceinline__ void slice_barrier(Frag4& f) {
  asm volatile("s_waitcnt vmcnt(%4) lgkmcnt(0)\n\ts_barrier"
               : "+v"(f.a0), "+v"(f.a1), "+v"(f.b0), "+v"(f.b1) : "n"(N) : "memory");
}

// barrier for plain LDS traffic that leaves the DMA stream in flight
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <class T>
struct DmaTile {
  static_assert(T::TM == 2 && T::TN * T::NB == 2, "Frag4 holds 2 x 2 fragments per k-step");
  static constexpr int NDMA = T::A_PT + T::B_PT * T::NB;  // DMAs per thread per slice
  static constexpr int LDS = 3 * T::STAGE;
  static_assert(LDS + 8 * 1024 <= 160 * 1024, "three stages plus epilogue scratch");
};

// per-lane global sources of one tile: A rows, then B0 rows (then B1 rows)
template <class T>
struct DPtrs {
  const bf16_t* a[T::A_PT];
  const bf16_t* b[T::B_PT * T::NB];
};

template <class T>
__device__ __forceinline__ void make_dptrs(DPtrs<T>& q, const CoreArgs& c) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < T::A_PT; ++i) {
    const int row = (t >> 3) + T::ROWS_PER_PASS * i;
    const int r = min(row, c.a_valid - 1);
    const int src = c.a_idx ? c.a_idx[r] : c.a_row0 + r;
    q.a[i] = c.A + (size_t)src * c.K + c.k_begin + 8 * ((t & 7) ^ swz(row));
  }
#pragma unroll
  for (int i = 0; i < T::B_PT; ++i) {
    const int row = (t >> 3) + T::ROWS_PER_PASS * i;
    const int r = min(row, c.b_valid - 1);
    const size_t off = (size_t)(c.b_idx ? c.b_idx[r] : c.b_row0 + r) * c.K + c.k_begin +
                       8 * ((t & 7) ^ swz(row));
    q.b[i] = c.B0 + off;
    if constexpr (T::NB == 2) q.b[T::B_PT + i] = c.B1 + off;
  }
}

// DMA slice kt of the tile into stage st
template <class T>
__device__ __forceinline__ void dma_slice(char* st, const DPtrs<T>& q, int kt) {
  const int w = threadIdx.x >> 6;
  const int o = kt * BK;
#pragma unroll
  for (int i = 0; i < T::A_PT; ++i) dma16(q.a[i] + o, st + (T::ROWS_PER_PASS * i + 8 * w) * 128);
#pragma unroll
  for (int i = 0; i < T::B_PT * T::NB; ++i)
    dma16(q.b[i] + o, st + T::A_BYTES + (i / T::B_PT) * T::B_BYTES +
                          (T::ROWS_PER_PASS * (i % T::B_PT) + 8 * w) * 128);
}

// per-lane LDS offsets of a wavefront's fragments within a stage
template <class T>
struct FragAddr {
  uint32_t a, b, ch[4];
  __device__ __forceinline__ FragAddr(int wm, int wn, int lane) {
    const int fr = lane & 31, hi = lane >> 5;
    a = (wm * T::WM + fr) * 128;
    b = T::A_BYTES + (wn * T::WN + fr) * 128;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) ch[ks] = ((2 * ks + hi) ^ swz(fr)) << 4;
  }
  __device__ __forceinline__ void read(Frag4& f, uint32_t stage, int ks) const {
    constexpr uint32_t kB1 = T::NB == 2 ? T::B_BYTES : 32 * 128;
    const uint32_t pa = stage + a + ch[ks], pb = stage + b + ch[ks];
    f.a0 = lds_read(pa);
    f.a1 = lds_read(pa + 32 * 128);
    f.b0 = lds_read(pb);
    f.b1 = lds_read(pb + kB1);
  }
};

// acc[i][j] += A_i B_j^T for the k-step held in f
__device__ __forceinline__ void mma4(const Frag4& f, f32x16_t (&acc)[2][2]) {
  acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a0, f.b0, acc[0][0], 0, 0, 0);
  acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a0, f.b1, acc[0][1], 0, 0, 0);
  acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a1, f.b0, acc[1][0], 0, 0, 0);
  acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a1, f.b1, acc[1][1], 0, 0, 0);
}

// One slice from stage cur (its k-step-0 fragments already in f0), with the
// next slice's k-step-0 fragments read from stage nxt under the last
// k-step's MFMAs.  `issue` starts the DMA of the slice two ahead.
template <class T, class Issue>
__device__ __forceinline__ void dma_slice_mma(const FragAddr<T>& fa, uint32_t cur, uint32_t nxt,
                                              Frag4& f0, Frag4& f1, f32x16_t (&acc)[2][2],
                                              Issue issue) {
  issue();
  fa.read(f1, cur, 1);
  lgkm_wait<4>(f0);
  mma4(f0, acc);
  fa.read(f0, cur, 2);
  lgkm_wait<4>(f1);
  mma4(f1, acc);
  fa.read(f1, cur, 3);
  lgkm_wait<4>(f0);
  mma4(f0, acc);
  slice_barrier<DmaTile<T>::NDMA>(f1);
  fa.read(f0, nxt, 0);
  mma4(f1, acc);
}

// ------------------------------------------------------ grouped FFN GEMMs --
// Rows come in expert groups; tile list entry = (expert, row begin, row end).
// Dense mode (shared expert): one group, rows [0, *dense_rows).
struct FfnArgs {
  const bf16_t* X;        // [rows, K], or h [T, K] when x_idx is set
  const int* x_idx;       // row -> source row of X (gather), or NULL
  const bf16_t* W0;       // expert 0 of [E, N, K] (up, or down)
  const bf16_t* W1;       // gate, same layout, or NULL
  size_t w_stride;        // elements between experts
  int K, N;
  const int4* tiles;      // grouped mode
  const int* n_tiles;     // grouped mode: live tiles (device)
  const int* dense_rows;  // dense mode: live rows (device), else NULL
  void* out;              // up: bf16 [rows, N]; down: f32 [split][rows_cap, N]
  size_t split_stride;    // elements between split slices of `out`
  int n_split;            // K splits (down GEMM); 1 otherwise
  int act;                // up: TRIMMOE_ACT_*
};

template <class T, bool UP>
__global__ __launch_bounds__(T::THREADS) void k_ffn_mma(FfnArgs a) {
  TRIMMOE_STAGES(T);
  const int n_nt = (a.N + T::BN - 1) / T::BN;
  const int n_mt = a.dense_rows ? (*a.dense_rows + T::BM - 1) / T::BM : *a.n_tiles;
  int mt, ntile, sp;
  if (!map_tile(blockIdx.x, n_mt, n_nt, a.n_split, mt, ntile, sp)) return;
  int e, m0, m1;
  if (a.dense_rows) {
    e = 0;
    m0 = mt * T::BM;
    m1 = *a.dense_rows;
  } else {
    const int4 tl = a.tiles[mt];
    e = tl.x;
    m0 = tl.y;
    m1 = tl.z;
  }
  const int n0 = ntile * T::BN;
  const int a_valid = min(T::BM, m1 - m0);
  const int b_valid = min(T::BN, a.N - n0);
  const bf16_t* W0 = a.W0 + (size_t)e * a.w_stride + (size_t)n0 * a.K;
  const bf16_t* W1 = T::NB == 2 ? a.W1 + (size_t)e * a.w_stride + (size_t)n0 * a.K : nullptr;
  const int nk = (a.K / BK) / a.n_split;
  f32x16_t acc0[T::TM][T::TN], acc1[T::TM][T::TN];
  gemm_core<T>(lds_buf0, lds_buf1,
               CoreArgs{a.X, W0, W1, a.x_idx ? a.x_idx + m0 : nullptr, nullptr, m0, 0, a_valid,
                        b_valid, a.K, sp * nk * BK, nk},
               acc0, acc1);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / T::GN, wn = wave % T::GN;
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j) {
      const int col = acc_col<T>(wn, j, lane);
      if (col >= b_valid) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = acc_row<T>(wm, i, r, lane);
        if (row >= a_valid) continue;
        const size_t o = (size_t)(m0 + row) * a.N + n0 + col;
        if constexpr (UP) {
          const float u = acc0[i][j][r];
          float v;
          if constexpr (T::NB == 2) {
            const float g = acc1[i][j][r];
            v = g / (1.f + expf(-g)) * u;  // silu(g) * u
          } else {
            v = fmaxf(u, 0.f);
          }
          static_cast<bf16_t*>(a.out)[o] = f2bf(v);
        } else {
          static_cast<float*>(a.out)[sp * a.split_stride + o] = acc0[i][j][r];
        }
      }
    }
}

// ----------------------------------------------------------- exit head --
// M = vocabulary (A = W_exit [V, d]), N = executed tokens (B = hx [n_x, d],
// the executed tokens' updated rows written by the combine kernel).
// Epilogue: for every token column, max and sum exp over the tile's
// vocabulary rows (bias added), written as one partial per vocabulary tile
// as (max z * log2 e, sum exp(z - max z)).
//
// Persistent: the grid has one block per CU; block b walks the tiles
// tb + i0, tb + i0 + bx, ... of its XCD's contiguous tile range (bx = blocks
// on that XCD), so the bx blocks of an XCD work on bx consecutive tiles of
// the patch order at any time.  Its K slices form one continuous load
// stream across tiles: the first slices of the next tile are already in
// flight while the current tile's epilogue runs.
struct ExitArgs {
  const bf16_t* W;    // [V, K]
  const bf16_t* H;    // [n_x, K]
  const float* bias;  // [V] or NULL
  const int* n_exec;  // device
  int V, K, n_vtiles;
  float2* partials;   // [n_x, n_vtiles]
};

using ExitTile = Tile<kExitTileBF16, 128, 1, 4, 2>;

struct ExitSched {
  int tb, i0, bx, n_mt, n_nt, n_x, nk;
  // tile j of this block -> vocabulary tile mt, token tile nt (patch order)
  __device__ __forceinline__ void decode(int j, int& mt, int& nt) const {
    const int L = tb + i0 + j * bx;
    const int span = kPatch * n_nt;
    const int g = L / span, w = L % span;
    const int gm = min(kPatch, n_mt - g * kPatch);
    nt = w / gm;
    mt = g * kPatch + w % gm;
  }
};

__device__ __forceinline__ void exit_epilogue(int j, const ExitSched& S, const ExitArgs& a,
                                              f32x16_t (&acc)[2][2],
                                              float2 (&s_part)[ExitTile::GM][ExitTile::BN]) {
  using T = ExitTile;
  int mt, nt;
  S.decode(j, mt, nt);
  const int v0 = mt * T::BM, j0 = nt * T::BN;
  const int a_valid = min(T::BM, a.V - v0);
  const int b_valid = min(T::BN, S.n_x - j0);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / T::GN, wn = wave % T::GN;
  // partials in base 2: y = z * log2(e), so exp(z - max z) = exp2(y - max y)
  // is one FMA and one v_exp_f32 per logit; the pair stored is (max y, sum)
  const float ninf = -__builtin_inff();
  const float kLog2e = 1.4426950408889634f;
  const bool full = a_valid == T::BM && !a.bias;
#pragma unroll
  for (int jj = 0; jj < T::TN; ++jj) {
    float m = ninf;
    if (full) {
#pragma unroll
      for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float y = acc[i][jj][r] * kLog2e;
          acc[i][jj][r] = y;
          m = fmaxf(m, y);
        }
    } else {
#pragma unroll
      for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = acc_row<T>(wm, i, r, lane);
          float y = acc[i][jj][r];
          if (a.bias) y += a.bias[v0 + min(row, a_valid - 1)];
          y = row < a_valid ? y * kLog2e : ninf;
          acc[i][jj][r] = y;
          m = fmaxf(m, y);
        }
    }
    m = fmaxf(m, __shfl_xor(m, 32));
    float sum = 0.f;
    if (m != ninf) {
#pragma unroll
      for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += __builtin_amdgcn_exp2f(acc[i][jj][r] - m);
    }
    sum += __shfl_xor(sum, 32);
    if (lane < 32) s_part[wm][acc_col<T>(wn, jj, lane)] = make_float2(m, sum);
  }
  lds_barrier();
  const int c = threadIdx.x;
  if (c < b_valid) {
    float M = s_part[0][c].x;
#pragma unroll
    for (int g = 1; g < T::GM; ++g) M = fmaxf(M, s_part[g][c].x);
    float S2 = 0.f;
#pragma unroll
    for (int g = 0; g < T::GM; ++g) {
      const float2 v = s_part[g][c];
      if (v.y > 0.f) S2 += v.y * __builtin_amdgcn_exp2f(v.x - M);
    }
    a.partials[(size_t)(j0 + c) * a.n_vtiles + mt] = make_float2(M, S2);
  }
  const f32x16_t z = {};
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int jj = 0; jj < T::TN; ++jj) acc[i][jj] = z;
}

__global__ __launch_bounds__(ExitTile::THREADS) void k_exit_mma(ExitArgs a) {
  using T = ExitTile;
  __shared__ __align__(16) char lds[DmaTile<T>::LDS];
  __shared__ float2 s_part[T::GM][T::BN];  // per wavefront row: (max, sum) per token column
  const int n_x = *a.n_exec;
  ExitSched S;
  S.n_mt = a.n_vtiles;
  S.n_nt = (n_x + T::BN - 1) / T::BN;
  S.n_x = n_x;
  S.nk = a.K / BK;
  const int total = S.n_mt * S.n_nt;
  // XCD groups (fewer when the grid is smaller than the XCD count)
  const int nx = min(kXcd, (int)gridDim.x);
  const int x = blockIdx.x % nx;
  S.i0 = blockIdx.x / nx;
  S.bx = ((int)gridDim.x - x + nx - 1) / nx;
  const int q = total / nx, r = total % nx;
  S.tb = x * q + min(x, r);
  const int te = S.tb + q + (x < r ? 1 : 0);
  if (S.tb + S.i0 >= te) return;
  const int ntiles = (te - (S.tb + S.i0) + S.bx - 1) / S.bx;
  const int nk = S.nk, G = ntiles * nk;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const FragAddr<T> fa(wave / T::GN, wave % T::GN, lane);
  const uint32_t st0 = lds_addr(lds);
  f32x16_t acc[2][2];
  const f32x16_t z = {};
  acc[0][0] = acc[0][1] = acc[1][0] = acc[1][1] = z;

  // DMA stream: next slice to issue is slice dk of tile dj; past the end the
  // last slice is issued again (in bounds, never read)
  DPtrs<T> qp;
  int dj = 0, dk = 0, lt = -1;
  auto issue = [&](int stage) {
    if (dj != lt) {
      int mt, nt;
      S.decode(dj, mt, nt);
      const CoreArgs c{a.W, a.H, nullptr, nullptr, nullptr, mt * T::BM, nt * T::BN,
                       min(T::BM, a.V - mt * T::BM), min(T::BN, S.n_x - nt * T::BN), a.K, 0, nk};
      make_dptrs<T>(qp, c);
      lt = dj;
    }
    dma_slice<T>(lds + stage * T::STAGE, qp, dk);
    if (++dk == nk) {
      if (dj + 1 < ntiles) {
        ++dj;
        dk = 0;
      } else {
        dk = nk - 1;
      }
    }
  };

  Frag4 f0, f1;
  issue(0);
  issue(1);
  slice_barrier<DmaTile<T>::NDMA>(f1);
  fa.read(f0, st0, 0);
  int sx = 0, kk = 0, j = 0;  // stage, slice within the tile, tile of the compute stream
  for (int g = 0; g < G; ++g) {
    const int sn = sx == 2 ? 0 : sx + 1, sp = sn == 2 ? 0 : sn + 1;
    dma_slice_mma<T>(fa, st0 + sx * T::STAGE, st0 + sn * T::STAGE, f0, f1, acc,
                     [&] { issue(sp); });
    if (++kk == nk) {
      exit_epilogue(j, S, a, acc, s_part);
      kk = 0;
      ++j;
    }
    sx = sn;
  }
}

// ------------------------------------------------------------- fp32 path --
constexpr int FT = kF32Tile;

// out[m][n] = X[m] . W[e][n] over a 128-row group tile, 16 columns per block.
template <bool UP>
__global__ __launch_bounds__(256) void k_ffn_f32(const float* X, const int* x_idx, const float* W0,
                                                 const float* W1, size_t w_stride, int K, int N,
                                                 const int4* tiles, const int* n_tiles,
                                                 const int* dense_rows, void* out, int act) {
  const int n_nt = (N + FT - 1) / FT;
  const int n_mt = dense_rows ? (*dense_rows + kGemmBM - 1) / kGemmBM : *n_tiles;
  const int mt = blockIdx.x / n_nt, ntile = blockIdx.x % n_nt;
  if (mt >= n_mt) return;
  int e, m0, m1;
  if (dense_rows) {
    e = 0;
    m0 = mt * kGemmBM;
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
  for (int m = m0 + ty; m < min(m0 + kGemmBM, m1); m += 256 / FT) {
    const float* x = X + (size_t)(x_idx ? x_idx[m] : m) * K;
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
__global__ __launch_bounds__(256) void k_exit_f32(const float* W, const float* H, const int* tok,
                                                  const float* bias, const int* n_exec, int V,
                                                  int K, int n_vtiles, float2* partials) {
  __shared__ float s_z[FT][FT + 1];
  const int n_x = *n_exec;
  const int vt = blockIdx.x % n_vtiles, jt = blockIdx.x / n_vtiles;
  if (jt * FT >= n_x) return;
  const int tv = threadIdx.x / FT, tj = threadIdx.x % FT;
  const int v = vt * FT + tv, j = jt * FT + tj;
  float z = -__builtin_inff();
  if (v < V && j < n_x) {
    const float* w = W + (size_t)v * K;
    const float* h = H + (size_t)tok[j] * K;
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
      // partials are kept in base 2: (max z * log2 e, sum exp(z - max z))
      partials[(size_t)jj * n_vtiles + vt] = make_float2(m * 1.4426950408889634f, s);
    }
  }
}

// ------------------------------------------------------------- launchers --
static inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Tile shapes of the expert GEMMs (BM rows of an expert group x BN outputs)
using UpDualTile = Tile<kGemmBM, 128, 2, 2, 4>;  // SwiGLU: up and gate share A
using UpTile = Tile<kGemmBM, 256, 1, 2, 4>;      // ReLU
using DownTile = Tile<kGemmBM, 128, 1, 2, 2>;

// K splits of the routed down GEMM: enough blocks to cover the CUs twice,
// each split keeping at least 8 K slices.
int down_splits(int max_tiles, int N, int K) {
  const int tiles = max_tiles * cdiv(N, DownTile::BN);
  const int nk = K / BK;
  int s = 1;
  while (s < 4 && tiles * s < 512 && nk % (2 * s) == 0 && nk / (2 * s) >= 8) s *= 2;
  return s;
}

template <class T, bool UP>
static void launch_ffn_mma(const FfnArgs& a, int max_mt, hipStream_t st) {
  const dim3 grid(max_mt * cdiv(a.N, T::BN) * a.n_split);
  hipLaunchKernelGGL((k_ffn_mma<T, UP>), grid, dim3(T::THREADS), 0, st, a);
}

static hipError_t ffn_pass(const LayerParams& p, bool bf16, bool up, bool shared, hipStream_t st) {
  const int K = up ? p.d : (shared ? p.Fs : p.F);
  const int N = up ? (shared ? p.Fs : p.F) : p.d;
  const bool dual = up && (shared || p.act == TRIMMOE_ACT_SWIGLU);
  const void* w0 = shared ? (up ? p.ws_up : p.ws_down) : (up ? p.w_up : p.w_down);
  const void* w1 = dual ? (shared ? p.ws_gate : p.w_gate) : nullptr;
  const size_t w_stride = shared ? 0 : (size_t)N * K;
  // up projections gather h rows: routed rows through row_src, shared-expert
  // rows through the executed-token list
  const void* X = up ? p.h : (shared ? p.act_s : p.act_buf);
  const int* x_idx = up ? (shared ? p.exec_list : p.row_src) : nullptr;
  void* out = up ? (shared ? p.act_s : p.act_buf) : (shared ? (void*)p.y_s : (void*)p.y_buf);
  const int* dense = shared ? &p.counts[kCntExec] : nullptr;
  const int max_mt = shared ? cdiv(p.T, kGemmBM) : p.max_tiles;
  const int act = shared ? TRIMMOE_ACT_SWIGLU : p.act;
  if (max_mt <= 0) return hipSuccess;
  if (bf16) {
    const int n_split = (!up && !shared) ? p.down_splits : 1;
    FfnArgs a{static_cast<const bf16_t*>(X), x_idx, static_cast<const bf16_t*>(w0),
              static_cast<const bf16_t*>(w1), w_stride, K, N, p.tiles, &p.counts[kCntTiles],
              dense, out, p.y_split_stride, n_split, act};
    if (up && dual)
      launch_ffn_mma<UpDualTile, true>(a, max_mt, st);
    else if (up)
      launch_ffn_mma<UpTile, true>(a, max_mt, st);
    else
      launch_ffn_mma<DownTile, false>(a, max_mt, st);
  } else {
    const dim3 grid(max_mt * cdiv(N, FT));
    if (up)
      hipLaunchKernelGGL(k_ffn_f32<true>, grid, dim3(256), 0, st, static_cast<const float*>(X),
                         x_idx, static_cast<const float*>(w0), static_cast<const float*>(w1),
                         w_stride, K, N, p.tiles, &p.counts[kCntTiles], dense, out, act);
    else
      hipLaunchKernelGGL(k_ffn_f32<false>, grid, dim3(256), 0, st, static_cast<const float*>(X),
                         x_idx, static_cast<const float*>(w0), nullptr, w_stride, K, N, p.tiles,
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
    // persistent: one block per CU (at most one tile per block in the worst case)
    const int max_tiles = p.n_vtiles * cdiv(p.T, ExitTile::BN);
    const dim3 grid(min(max_tiles, p.n_cu));
    hipLaunchKernelGGL(k_exit_mma, grid, dim3(ExitTile::THREADS), 0, st, a);
  } else {
    const dim3 grid(p.n_vtiles * cdiv(p.T, FT));
    hipLaunchKernelGGL(k_exit_f32, grid, dim3(256), 0, st, static_cast<const float*>(p.w_exit),
                       static_cast<const float*>(p.h), p.exec_list, p.b_exit, &p.counts[kCntExec],
                       p.V, p.d, p.n_vtiles, p.partials);
  }
  return hipGetLastError();
}

}  // namespace trimmoe
