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
// is 8 wavefronts; each owns a 64 x 64 output patch (or 64 x 32 of two B
// operands) and multiplies two A by two B fragments per 16-wide k-step.  K
// advances in 64-wide slices (one 128-byte row segment per operand row)
// that gfx950's direct-to-LDS loads bring into a three-stage LDS ring two
// slices ahead.  In LDS a row segment keeps its eight 16-byte chunks
// XOR-swizzled by (row & 7) ^ ((row >> 3) & 1), so the fragment reads of 8
// consecutive rows hit distinct banks.  Rows past the valid range load a
// clamped valid row (their results are never stored).  Grids are persistent
// (one block per CU); each block streams the K slices of its tiles
// back to back, tiles taken from its XCD's contiguous range in patch order.
//
// Large expert groups, the dense shared expert of large batches and the exit
// head of wide models run on a second bf16 core (4 wavefronts, 256 x 256
// tiles in v_mfma_f32_16x16x32_bf16; described with its kernels).
//
// fp32 path: plain FMA kernels for fp32 models.
#include <math.h>

#include "common.h"

namespace trimmoe {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int BK = kGemmBK;  // 64 bf16 = one 128-byte row segment
constexpr int kPatch = 8;    // M-tiles per patch column in the tile order
constexpr int kXcd = 8;      // XCDs of an MI355X; blocks are dealt round-robin

static_assert(BK == 64, "the LDS layout assumes 128-byte row segments");

// ------------------------------------------------------------ tile shapes --
// BM x BN block tile, NB B operands sharing A, GM x GN wavefronts
template <int BM_, int BN_, int NB_, int GM_, int GN_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, NB = NB_, GM = GM_, GN = GN_;
  static constexpr int THREADS = 64 * GM * GN;
  static constexpr int WM = BM / GM, WN = BN / GN;  // wavefront tile
  static constexpr int TM = WM / 32, TN = WN / 32;  // MFMA tiles per wavefront
  static constexpr int A_BYTES = BM * 128, B_BYTES = BN * 128;
  static constexpr int STAGE = A_BYTES + NB * B_BYTES;
  static constexpr int ROWS_PER_PASS = THREADS / 8;  // 8 threads per 128-byte row
  static constexpr int A_PT = BM / ROWS_PER_PASS, B_PT = BN / ROWS_PER_PASS;
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wavefront tile");
  static_assert(BM % ROWS_PER_PASS == 0 && BN % ROWS_PER_PASS == 0, "load passes");
};

// 16-byte chunk c of row r sits at chunk c ^ swz(r): 8 consecutive rows, or
// 16 consecutive rows split by parity, then touch distinct bank groups.
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

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
// 16 l): no staging VGPRs and no ds_write (the two things a register-staged
// operand path spends most of its non-MFMA issue time on).  Three LDS stages
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

// one k-step's fragments of a wavefront: TM A fragments (rows +32 i) and
// TN * NB B fragments (operand o, columns +32 j at index o * TN + j)
template <class T>
struct Frags {
  bf16x8_t a[T::TM];
  bf16x8_t b[T::TN * T::NB];
};

// ties every fragment register to the asm statement just before it (volatile
// asm keeps its order), so no MFMA reading one is scheduled above that wait
template <class T>
__device__ __forceinline__ void frags_after(Frags<T>& f) {
#pragma unroll
  for (int i = 0; i < T::TM; ++i) asm volatile("" : "+v"(f.a[i]));
#pragma unroll
  for (int j = 0; j < T::TN * T::NB; ++j) asm volatile("" : "+v"(f.b[j]));
}

template <int N, class T>
__device__ __forceinline__ void lgkm_wait(Frags<T>& f) {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N));
  frags_after(f);
}

template <int N, class T>
__device__ __forceinline__ void slice_barrier(Frags<T>& f) {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
  frags_after(f);
}

// barrier for plain LDS traffic that leaves the DMA stream in flight
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Ring depth: three stages (two slices in flight ahead of the one being
// computed) when they fit next to 8 KB of epilogue scratch, else two.
template <class T>
struct DmaTile {
  static constexpr int NF = T::TM + T::TN * T::NB;        // fragment reads per k-step
  static constexpr int NDMA = T::A_PT + T::B_PT * T::NB;  // DMAs per thread per slice
  static constexpr int STAGES = 3 * T::STAGE + 8 * 1024 <= 160 * 1024 ? 3 : 2;
  static constexpr int DEPTH = STAGES - 1;                // slices issued ahead
  static constexpr int LDS = STAGES * T::STAGE;
  static_assert(LDS + 8 * 1024 <= 160 * 1024, "stages plus epilogue scratch");
  static_assert(NF <= 15 && NDMA * (DEPTH - 1) <= 63, "waitcnt fields");
};

// per-lane global sources of one tile: A rows, then B0 rows (then B1 rows)
template <class T>
struct DPtrs {
  const bf16_t* a[T::A_PT];
  const bf16_t* b[T::B_PT * T::NB];
};

// tile row a thread's i-th A / B DMA covers, and the 16-byte chunk it loads
__device__ __forceinline__ int dma_row(int i, int rows_per_pass) {
  return ((int)threadIdx.x >> 3) + rows_per_pass * i;
}
__device__ __forceinline__ int dma_col(int row) { return 8 * (((int)threadIdx.x & 7) ^ swz(row)); }

// A rows a_src[i] (matrix rows, already clamped) of A; B rows b_row0 + r,
// r clamped to b_valid - 1, of B0 (and B1); K columns from k_begin
template <class T>
__device__ __forceinline__ void make_dptrs(DPtrs<T>& q, const bf16_t* A, const int (&a_src)[T::A_PT],
                                           const bf16_t* B0, const bf16_t* B1, int b_row0,
                                           int b_valid, int K, int k_begin) {
#pragma unroll
  for (int i = 0; i < T::A_PT; ++i) {
    const int row = dma_row(i, T::ROWS_PER_PASS);
    q.a[i] = A + (size_t)a_src[i] * K + k_begin + dma_col(row);
  }
#pragma unroll
  for (int i = 0; i < T::B_PT; ++i) {
    const int row = dma_row(i, T::ROWS_PER_PASS);
    const size_t off = (size_t)(b_row0 + min(row, b_valid - 1)) * K + k_begin + dma_col(row);
    q.b[i] = B0 + off;
    if constexpr (T::NB == 2) q.b[T::B_PT + i] = B1 + off;
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
  __device__ __forceinline__ void read(Frags<T>& f, uint32_t stage, int ks) const {
    const uint32_t pa = stage + a + ch[ks], pb = stage + b + ch[ks];
#pragma unroll
    for (int i = 0; i < T::TM; ++i) f.a[i] = lds_read(pa + i * 32 * 128);
#pragma unroll
    for (int o = 0; o < T::NB; ++o)
#pragma unroll
      for (int j = 0; j < T::TN; ++j) f.b[o * T::TN + j] = lds_read(pb + o * T::B_BYTES + j * 32 * 128);
  }
};

template <class T>
using Acc = f32x16_t[T::TM][T::TN * T::NB];

// acc[i][j] += A_i B_j^T for the k-step held in f
template <class T>
__device__ __forceinline__ void mma_step(const Frags<T>& f, Acc<T>& acc) {
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN * T::NB; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
}

// One slice from stage cur (its k-step-0 fragments already in f0), with the
// next slice's k-step-0 fragments read from stage nxt under the last
// k-step's MFMAs.  `issue` starts the DMA of the slice DEPTH ahead; the
// barrier waits for the DMAs of the next slice only.
template <class T, class Issue>
__device__ __forceinline__ void dma_slice_mma(const FragAddr<T>& fa, uint32_t cur, uint32_t nxt,
                                              Frags<T>& f0, Frags<T>& f1, Acc<T>& acc,
                                              Issue issue) {
  using D = DmaTile<T>;
  issue();
  fa.read(f1, cur, 1);
  lgkm_wait<D::NF>(f0);
  mma_step<T>(f0, acc);
  fa.read(f0, cur, 2);
  lgkm_wait<D::NF>(f1);
  mma_step<T>(f1, acc);
  fa.read(f1, cur, 3);
  lgkm_wait<D::NF>(f0);
  mma_step<T>(f0, acc);
  slice_barrier<D::NDMA * (D::DEPTH - 1)>(f1);
  fa.read(f0, nxt, 0);
  mma_step<T>(f1, acc);
}

// ------------------------------------------------------- tile scheduling --
// Persistent grids: one block per CU (or fewer).  The live tiles (a count
// known only on the device) are split into contiguous ranges, one per XCD
// (hardware deals block b to XCD b % 8); block b walks tiles tb + i0,
// tb + i0 + bx, ... of its XCD's range (bx = blocks on that XCD), so the
// blocks of an XCD work on consecutive tiles and share its L2.  A tile index
// is read in patch order: kPatch M-tiles of one N-tile, then the next
// N-tile; the K split (if any) is the slowest index.
struct TileSched {
  int tb, i0, bx, n_mt, n_nt;
  // false when this block has no tile, else its tile count in ntiles
  __device__ __forceinline__ bool init(int n_mt_, int n_nt_, int n_split, int& ntiles) {
    return init_total(n_mt_ * n_nt_ * n_split, n_mt_, n_nt_, ntiles);
  }
  // the first `total` tile indices only
  __device__ __forceinline__ bool init_total(int total, int n_mt_, int n_nt_, int& ntiles) {
    n_mt = n_mt_;
    n_nt = n_nt_;
    const int nx = min(kXcd, (int)gridDim.x);  // fewer groups for a small grid
    const int x = blockIdx.x % nx;
    i0 = blockIdx.x / nx;
    bx = ((int)gridDim.x - x + nx - 1) / nx;
    const int q = total / nx, r = total % nx;
    tb = x * q + min(x, r);
    const int te = tb + q + (x < r ? 1 : 0);
    if (tb + i0 >= te) return false;
    ntiles = (te - (tb + i0) + bx - 1) / bx;
    return true;
  }
  __device__ __forceinline__ void decode(int j, int& mt, int& nt, int& sp) const {
    decode_abs(tb + i0 + j * bx, mt, nt, sp);
  }
  // tile index L of the whole patch order
  __device__ __forceinline__ void decode_abs(int L, int& mt, int& nt, int& sp) const {
    const int per = n_mt * n_nt;
    sp = L / per;
    L -= sp * per;
    const int span = kPatch * n_nt;
    const int g = L / span, w = L % span;
    const int gm = min(kPatch, n_mt - g * kPatch);
    nt = w / gm;
    mt = g * kPatch + w % gm;
  }
};

// A persistent block's GEMM over its ntiles tiles of nk slices each: one
// continuous stream of K slices through the DMA ring, so the next tile's
// first slices are in flight while the current tile's epilogue runs.
// Src supplies, for tile j of the block:
//   Desc desc(int j)                      descriptor (may load from memory);
//                                         Desc::pick(c, x, y) = c ? x : y
//   void rows(const Desc&, int (&)[A_PT]) per-thread A source rows (may load)
//   void ptrs(DPtrs<T>&, const Desc&, const int (&)[A_PT])
//   void epilogue(const Desc&, Acc<T>&)
// Descriptors are loaded two tiles and rows one tile ahead of their use, so
// the compiler's load-count waits for them never drain the DMA ring.
template <class T, class Src>
__device__ __forceinline__ void dma_gemm_stream(char* lds, int ntiles, int nk, const Src& src) {
  using Desc = typename Src::Desc;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const FragAddr<T> fa(wave / T::GN, wave % T::GN, lane);
  const uint32_t st0 = lds_addr(lds);
  using D = DmaTile<T>;
  Acc<T> acc;
  const f32x16_t z = {};
  auto zero = [&] {
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
      for (int j = 0; j < T::TN * T::NB; ++j) acc[i][j] = z;
  };
  zero();

  // DMA side: slice dk of tile dj through pointers qp; n1 / n2 describe
  // tiles dj+1 / dj+2 and rn1 holds the A rows of dj+1
  // start-up: the three descriptor loads go out together, and the first
  // slice's DMA right after tile 0's rows, before tile 1's rows are needed
  const int last = ntiles - 1;
  DPtrs<T> qp;
  int rows[T::A_PT], rn1[T::A_PT];
  Desc c0 = src.desc(0);
  Desc n1 = src.desc(min(1, last));
  Desc n2 = src.desc(min(2, last));
  src.rows(c0, rows);
  src.ptrs(qp, c0, rows);
  int dj = 0, dk = 0;
  // compute side: c0 describes tile jc; c1 / c2 tiles jc+1 / jc+2 once the
  // DMA side has entered them (it runs at most DEPTH <= 2 slices ahead)
  Desc c1 = n1, c2 = n2;
  int jc = 0;
  // the DMA side enters a tile when it issues the tile's first slice, at
  // most DEPTH <= 2 slices ahead of the compute side, so dj - jc is 1 or 2
  auto issue = [&](int stage) {
    if (dk == nk) {
      if (dj == last) {  // past the end: the last slice again (in bounds, never read)
        dk = nk - 1;
      } else {
        ++dj;
        dk = 0;
        src.ptrs(qp, n1, rn1);
        const bool next = dj == jc + 1;  // field-wise selects: no indexed copy
        c1 = Desc::pick(next, n1, c1);
        c2 = Desc::pick(next, c2, n1);
        src.rows(n2, rn1);
        n1 = n2;
        n2 = src.desc(min(dj + 2, last));
      }
    }
    dma_slice<T>(lds + stage * T::STAGE, qp, dk);
    ++dk;
  };

  Frags<T> f0, f1;
  issue(0);
  src.rows(n1, rn1);  // first needed when the stream enters tile 1
#pragma unroll
  for (int s = 1; s < D::DEPTH; ++s) issue(s);
  slice_barrier<D::NDMA * (D::DEPTH - 1)>(f1);
  fa.read(f0, st0, 0);
  const int G = ntiles * nk;
  int sx = 0, kk = 0;  // stage of the slice being computed, its index in the tile
  for (int g = 0; g < G; ++g) {
    const int sn = sx + 1 == D::STAGES ? 0 : sx + 1;
    const int sp = (sx + D::DEPTH) % D::STAGES;  // stage of slice g + DEPTH
    dma_slice_mma<T>(fa, st0 + sx * T::STAGE, st0 + sn * T::STAGE, f0, f1, acc,
                     [&] { issue(sp); });
    if (++kk == nk) {
      src.epilogue(c0, acc);
      zero();
      c0 = c1;
      c1 = c2;
      ++jc;
      kk = 0;
    }
    sx = sn;
  }
}

// ----------------------------------------------- activation helpers --
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float swap_pair(float v) {
  // lane l reads lane l ^ 1 (quad_perm [1, 0, 3, 2])
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xb1, 0xf,
                                                             0xf, false));
}

// The values of lanes l and l ^ 16 (lanes_xor16) or l and l ^ 32
// (lanes_xor32) in every lane, by gfx950's permlane swaps instead of an LDS
// exchange: (a, b) is (own, other) in lanes 0..15 (xor16: every even row of
// 16 lanes) or 0..31 (xor32) and (other, own) in the rest, so a commutative
// reduction of a and b gives every lane the pair's result.  The two results
// are copied out of the returned pair before the bit casts: a bit cast of
// the subscripted second element read the first one.
struct LanePair {
  float a, b;
};
__device__ __forceinline__ LanePair lanes_xor16(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const unsigned r0 = r[0], r1 = r[1];
  return {__builtin_bit_cast(float, r0), __builtin_bit_cast(float, r1)};
}
__device__ __forceinline__ LanePair lanes_xor32(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned r0 = r[0], r1 = r[1];
  return {__builtin_bit_cast(float, r0), __builtin_bit_cast(float, r1)};
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// silu(g) u = g u / (1 + e^-g) with the hardware exp2 and reciprocal (about
// 1 ulp each in fp32; callers round the result to bf16)
__device__ __forceinline__ float silu_mul(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-g * 1.4426950408889634f)) * u;
}

// ------------------------------------------------------ grouped FFN GEMMs --
// Row tiles come from the device tile list (expert, first row, end row) of
// the expert-sorted rows, or (dense mode, shared expert) cover the first
// *dense_rows rows.  A rows are gathered through x_idx (the token whose h
// row feeds each sorted row) when it is set.
// Engine-clock record (measurement only): with a record set, a block adds the
// core clock cycles (s_memtime) and the 100 MHz constant-clock ticks
// (s_memrealtime) between its start and the end of its work to rec[0] and
// rec[1]; their ratio is the mean engine clock under the kernel.  The start
// values are subtracted at once (modulo 2^64) and the end values added at
// the end, so nothing is held in registers in between.
__device__ __forceinline__ void clock_mark(unsigned long long* rec, bool start) {
  if (rec && threadIdx.x == 0) {
    const unsigned long long t = __builtin_amdgcn_s_memtime();
    const unsigned long long r = __builtin_amdgcn_s_memrealtime();
    atomicAdd(rec, start ? 0ull - t : t);
    atomicAdd(rec + 1, start ? 0ull - r : r);
  }
}

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
  int* sk_flag;           // large-group down GEMM: per-tile piece words (see SkPlan), or NULL
  float* sk_part;         // ... and the compact partials of pieces 1.. of cut tiles
  unsigned long long* clk;  // engine-clock record of this class (see clock_mark), or NULL
};

template <class T, bool UP>
struct FfnSrc {
  struct Desc {
    int e, m0, m1, nt, sp;
    static __device__ __forceinline__ Desc pick(bool c, const Desc& x, const Desc& y) {
      return Desc{c ? x.e : y.e, c ? x.m0 : y.m0, c ? x.m1 : y.m1, c ? x.nt : y.nt,
                  c ? x.sp : y.sp};
    }
  };
  const FfnArgs& a;
  const TileSched& S;
  int dense_m1;  // dense mode: live rows
  int nk;

  __device__ __forceinline__ Desc desc(int j) const {
    int mt, nt, sp;
    S.decode(j, mt, nt, sp);
    if (a.dense_rows) return Desc{0, mt * T::BM, dense_m1, nt, sp};
    const int4 tl = a.tiles[mt];
    return Desc{tl.x, tl.y, tl.z, nt, sp};
  }
  __device__ __forceinline__ void rows(const Desc& d, int (&src)[T::A_PT]) const {
#pragma unroll
    for (int i = 0; i < T::A_PT; ++i) {
      const int r = d.m0 + min(dma_row(i, T::ROWS_PER_PASS), d.m1 - d.m0 - 1);
      src[i] = a.x_idx ? a.x_idx[r] : r;
    }
  }
  __device__ __forceinline__ void ptrs(DPtrs<T>& q, const Desc& d,
                                       const int (&src)[T::A_PT]) const {
    const size_t wo = (size_t)d.e * a.w_stride;
    const int n0 = d.nt * T::BN;
    make_dptrs<T>(q, a.X, src, a.W0 + wo, T::NB == 2 ? a.W1 + wo : nullptr, n0,
                  min(T::BN, a.N - n0), a.K, d.sp * nk * BK);
  }
  __device__ __forceinline__ void epilogue(const Desc& d, Acc<T>& acc) const {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / T::GN, wn = wave % T::GN;
    const int n0 = d.nt * T::BN;
    const int a_valid = min(T::BM, d.m1 - d.m0);
    const int b_valid = min(T::BN, a.N - n0);
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
          const size_t o = (size_t)(d.m0 + row) * a.N + n0 + col;
          if constexpr (UP) {
            const float u = acc[i][j][r];
            float v;
            if constexpr (T::NB == 2) {
              v = silu_mul(acc[i][T::TN + j][r], u);  // gate of the same column
            } else {
              v = fmaxf(u, 0.f);
            }
            static_cast<__bf16*>(a.out)[o] = (__bf16)v;
          } else {
            static_cast<float*>(a.out)[d.sp * a.split_stride + o] = acc[i][j][r];
          }
        }
      }
  }
};

template <class T, bool UP>
__global__ __launch_bounds__(T::THREADS) void k_ffn_mma(FfnArgs a) {
  __shared__ __align__(16) char lds[DmaTile<T>::LDS];
  const int n_nt = (a.N + T::BN - 1) / T::BN;
  const int dense_m1 = a.dense_rows ? *a.dense_rows : 0;
  const int n_mt = a.dense_rows ? (dense_m1 + T::BM - 1) / T::BM : *a.n_tiles;
  TileSched S;
  int ntiles;
  if (!S.init(n_mt, n_nt, a.n_split, ntiles)) return;
  clock_mark(a.clk, true);
  const int nk = (a.K / BK) / a.n_split;
  const FfnSrc<T, UP> src{a, S, dense_m1, nk};
  dma_gemm_stream<T>(lds, ntiles, nk, src);
  clock_mark(a.clk, false);
}

// ------------------------------------------ large-group expert GEMMs --
// Expert groups of prefill batches (about a thousand rows or more per expert),
// the dense shared expert of large batches and the exit head of wide models
// (k_exit_big, below) use a second core with 256 x 256 block tiles and 4
// wavefronts, one per SIMD, each owning a 128 x 128 output patch: 8 x 8
// accumulators of 16 x 16 in AGPRs, multiplied in v_mfma_f32_16x16x32_bf16.
// A k-step of 32 reads 16 fragments for 64 MFMAs (half the LDS bytes per
// MFMA of the 64 x 64 patches) and a 64-wide K slice moves 64 KB for
// 256 x 256 outputs (2/3 of the bytes per MFMA of the 128 x 256 block).  The
// chip does not hold its peak clock under a dense MFMA load, and the
// 16 x 16 x 32 form keeps a higher one than 32 x 32 x 16 at nearly the same
// share of the cycles (a loop of MFMAs alone: about 2.1 GHz against 1.8),
// which is why this core uses it.  With one wavefront per SIMD no other
// wavefront fills the MFMA pipe while this one waits, so the instruction
// stream is laid out explicitly (sched_barrier keeps the compiler from
// regrouping it; the MFMAs are inline asm on AGPR operands, so the register
// allocator cannot move accumulators inside the loop):
//   * a k-step issues its 64 MFMAs row by row (tile (i, j) = (T / 8, T % 8)).
//     The next k-step's B fragments go to a second register set, read one
//     after each of the first 8 MFMAs; its a_i replaces this k-step's a_i
//     right after that fragment's last MFMA (8 i + 7), so A needs one set.
//     Each MFMA waits for its own fragments with a partial lgkmcnt;
//   * both operands go straight to LDS through buffer-to-LDS DMAs (a
//     wavefront's 64 x 16 bytes land at a wave-uniform base; 32-bit row
//     offsets, the K position in the scalar offset), so no VGPRs and no
//     ds_write are spent on them.  A (the gathered activations) has two
//     32 KB stages and B (the weights) a ring of three.  During slice g the
//     first k-step brings the second half of A of slice g + 1, the last
//     k-step (after the barrier, into the A stage slice g leaves) the first
//     half of A of slice g + 2, and both bring B of slice g + 2: 16 DMAs per
//     thread spread over the slice, since a DMA of a whole 64 KB slice at
//     once asks the texture path for about 128 B/clk per CU against the
//     ~50 B/clk it sustains, and its stalls land on the MFMA issue;
//   * one barrier per slice, before MFMA 32 of the last k-step: it waits for
//     this slice's reads and every DMA of slice g + 1, and the next slice's
//     first fragments are read after it, one after each following MFMA.
// Blocks are persistent and walk their XCD's contiguous tile range as the
// other core does; each tile runs its own prologue and epilogue.
namespace big {
constexpr int BM = 256, BN = 256, THREADS = 256;
constexpr int RB = 128;                  // bytes of a row segment (64 bf16)
constexpr int AB = BM * RB;              // A rows of a slice (32 KB)
constexpr int BB = BN * RB;              // B rows of a slice (32 KB)
constexpr int BS = 3;                    // B stages (DMA ring)
constexpr int B0 = 2 * AB;               // first B stage, after the two A stages
constexpr int LDS = 2 * AB + BS * BB;    // 160 KB
constexpr int RPP = THREADS / 8;         // rows per fetch pass (8 threads per 128-byte row)
}  // namespace big

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// a wavefront's fragments of one 32-wide k-step: A rows +16 i, B columns +16 j
struct FragA {
  bf16x8_t a[8];
};
struct FragB {
  bf16x8_t b[8];
};
// its 128 x 128 patch: 8 x 8 accumulators of 16 x 16 (lane: column l % 16,
// rows 4 (l / 16) .. + 4)
using AccBig = f32x4_t[8][8];

__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

template <int N>
__device__ __forceinline__ void lgkm_le() {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N));
}

// fragment read with a constant byte offset from a per-lane LDS address
template <int OFF>
__device__ __forceinline__ bf16x8_t lds_read_at(uint32_t a) {
  bf16x8_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "n"(OFF));
  return v;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p) {
  // raw buffer, no range limit: every offset is clamped to a valid row first
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)0xffffffff,
                                           0x00020000);
}

// a buffer of no records: every load from it returns zeros
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc_empty(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, 0, 0x00020000);
}

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// A 32-wide k-step issues its 64 MFMAs row by row (tile (i, j) = (T / 8,
// T % 8)): a_i is last used by MFMA 8 i + 7, so the next k-step's a_i is read
// into the same registers right after it, while the b fragments alternate
// between two sets.  Per MFMA slot T: the lgkmcnt wait before it (-1: none;
// the value counts the LDS reads issued after the ones it needs, capped at
// the counter's 15, which only waits longer), and the fragment read after it
// (q = 2 n for a_n, 2 n + 1 for b_n; -1: none; the first k-step also reads
// the next a_0 after MFMA 7), for the first k-step of a slice (0) and the
// last (1: its reads, of the next slice, follow the slice barrier before
// MFMA 32).  The first k-step waits on the last k-step's read order and the
// last k-step on the first's.
constexpr int kWait0[64] = {
    14, 13, 12, 11, 10, 10, 10, 10,  // MFMAs 0..7
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 8..15
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 16..23
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 24..31
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 32..39
    15, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 40..47
    15, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 48..55
    15, -1, -1, -1, -1, -1, -1, -1   // MFMAs 56..63
};
constexpr int kWait1[64] = {
     7, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 0..7
     6, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 8..15
     5, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 16..23
     4, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 24..31
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 32..39
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 40..47
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 48..55
    -1, -1, -1, -1, -1, -1, -1, -1   // MFMAs 56..63
};
constexpr int kRead0[64] = {
     1,  3,  5,  7,  9, 11, 13, 15,  // MFMAs 0..7
    -1, -1, -1, -1, -1, -1, -1,  2,  // MFMAs 8..15
    -1, -1, -1, -1, -1, -1, -1,  4,  // MFMAs 16..23
    -1, -1, -1, -1, -1, -1, -1,  6,  // MFMAs 24..31
    -1, -1, -1, -1, -1, -1, -1,  8,  // MFMAs 32..39
    -1, -1, -1, -1, -1, -1, -1, 10,  // MFMAs 40..47
    -1, -1, -1, -1, -1, -1, -1, 12,  // MFMAs 48..55
    -1, -1, -1, -1, -1, -1, -1, 14   // MFMAs 56..63
};
constexpr int kRead1[64] = {
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 0..7
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 8..15
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 16..23
    -1, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 24..31
     0,  1,  2,  3,  4,  5,  6,  7,  // MFMAs 32..39
     8,  9, -1, 11, -1, 13, -1, 15,  // MFMAs 40..47
    10, -1, -1, -1, -1, -1, -1, -1,  // MFMAs 48..55
    12, -1, -1, -1, -1, -1, -1, 14   // MFMAs 56..63
};

// B fragment j of a wavefront: LDS row offset from its first B row.  DUAL:
// columns j = 0..3 of the up operand (rows 0..127 of the B stage), j = 4..7
// the same columns of the gate operand (rows 128..255).
template <bool DUAL>
constexpr int big_brow(int j) {
  return DUAL ? (j < 4 ? 16 * j : 128 + 16 * (j - 4)) : 16 * j;
}

// fragment read Q of a k-step: a_{Q/2} for even Q, b_{Q/2} for odd Q
template <bool DUAL, int Q>
__device__ __forceinline__ void big_read(FragA& fa, FragB& fb, uint32_t pa, uint32_t pb) {
  if constexpr (Q >= 0) {
    if constexpr (Q & 1)
      fb.b[Q >> 1] = lds_read_at<big_brow<DUAL>(Q >> 1) * big::RB>(pb);
    else
      fa.a[Q >> 1] = lds_read_at<(Q >> 1) * 16 * big::RB>(pa);
    sched_fence();
  }
}

// Per-thread operand rows of one tile: row u < 8 is A row r0 + 32 u (gathered,
// clamped), u >= 8 B row r0 + 32 (u - 8) (clamped to the valid columns); byte
// offsets of the thread's 16-byte chunk within their buffers at K = k0
struct BigRows {
  __amdgpu_buffer_rsrc_t ra, rb0, rb1, none;
  uint32_t off[16];
};

// the buffers one slice is fetched from: a slice past the last one reads the
// empty buffer, so it lands as zeros and adds nothing
struct BigSrc {
  __amdgpu_buffer_rsrc_t ra, rb0, rb1;
  uint32_t ko;
  __device__ __forceinline__ BigSrc(const BigRows& q, int kt, int nk) {
    const bool live = kt < nk;
    ra = live ? q.ra : q.none;
    rb0 = live ? q.rb0 : q.none;
    rb1 = live ? q.rb1 : q.none;
    ko = live ? kt * big::RB : 0;
  }
};

// B row group u (0..7) of the wave straight into B stage `bst` (LDS address):
// lane l lands at bst + (8 w + 32 u) * 128 + 16 l, which is row 8 w + 32 u +
// l / 8, chunk slot l % 8 (the thread's fetch chunk is the swizzled one)
template <bool DUAL>
__device__ __forceinline__ void big_dma(uint32_t bst, int wave, const BigRows& q, const BigSrc& b,
                                        int u) {
  const __amdgpu_buffer_rsrc_t& rs = DUAL && u >= 4 ? b.rb1 : b.rb0;
  const uint32_t dst = bst + (uint32_t)((8 * wave + big::RPP * u) * big::RB);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_char*)(uintptr_t)dst, 16, q.off[8 + u], b.ko, 0,
                                           0);
}

// A row group u (0..7) of the wave straight into A stage `ast`
__device__ __forceinline__ void big_dma_a(uint32_t ast, int wave, const BigRows& q, const BigSrc& b,
                                          int u) {
  const uint32_t dst = ast + (uint32_t)((8 * wave + big::RPP * u) * big::RB);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(b.ra, (lds_char*)(uintptr_t)dst, 16, q.off[u], b.ko, 0, 0);
}

// MFMA slot T of a k-step (LAST: the second of the slice) from fragments fa,
// fb, with the next k-step's reads into fa (rotating) and fn: the wait, the
// MFMA, the reads; in the first k-step the A DMAs of the next slice (rows
// 4..7 of each thread) after MFMAs 16, 20, 24, 28; in the last the slice
// barrier before MFMA 32 and the A DMAs of the slice after next (rows 0..3,
// into the A stage this slice leaves) after MFMAs 32, 36, 40, 44; in both
// the B DMAs of the slice after next after MFMAs 18, 26, 50, 58 (rows 0..3
// in the first, 4..7 in the last).  The barrier waits for the next slice's
// A DMAs (the last issued at MFMA 28 of the first k-step, followed by 4 B
// DMAs) and its B DMAs (issued a slice earlier).
template <int T, bool LAST, bool DUAL, class DmaA, class DmaB>
__device__ __forceinline__ void big_slot(FragA& fa, FragB& fb, FragB& fn, AccBig& acc,
                                         uint32_t pa, uint32_t pb, DmaA& dma_a, DmaB& dma_b) {
  constexpr int i = T / 8, j = T % 8;
  constexpr int w = LAST ? kWait1[T] : kWait0[T];
  if constexpr (w >= 0) {
    lgkm_le<w>();
    asm volatile("" : "+v"(fa.a[i]), "+v"(fb.b[j]));
    sched_fence();
  }
  if constexpr (LAST && T == 32) {
    asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    asm volatile("" : "+v"(fa.a[i]), "+v"(fb.b[j]));
    sched_fence();
  }
  // the accumulators stay in AGPRs (with the builtin the allocator moved some
  // through VGPRs inside the loop)
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
               : "+a"(acc[i][j])
               : "v"(fa.a[i]), "v"(fb.b[j]));
  sched_fence();
  big_read<DUAL, LAST ? kRead1[T] : kRead0[T]>(fa, fn, pa, pb);
  // the first k-step's a_0 for the next k-step, after its last use
  if constexpr (!LAST && T == 7) big_read<DUAL, 0>(fa, fn, pa, pb);
  if constexpr (!LAST && (T == 16 || T == 20 || T == 24 || T == 28)) {
    dma_a(4 + (T - 16) / 4);
    sched_fence();
  }
  if constexpr (LAST && (T == 32 || T == 36 || T == 40 || T == 44)) {
    dma_a((T - 32) / 4);
    sched_fence();
  }
  if constexpr (T == 18 || T == 26 || T == 50 || T == 58) {
    dma_b((LAST ? 4 : 0) + (T == 18 ? 0 : T == 26 ? 1 : T == 50 ? 2 : 3));
    sched_fence();
  }
  if constexpr (T < 63) big_slot<T + 1, LAST, DUAL>(fa, fb, fn, acc, pa, pb, dma_a, dma_b);
}

// LDS of the large-group core: A stages at s0 and s0 + AB (slice parity), B
// stages at s0 + B0 + BB * (slice mod 3)
struct BigLds {
  uint32_t s0;
  __device__ __forceinline__ uint32_t a(int g) const { return s0 + (g & 1) * big::AB; }
  __device__ __forceinline__ uint32_t b(int g) const { return s0 + big::B0 + (g % 3) * big::BB; }
};

// One 64-wide slice g: two k-steps of 32 from A stage g & 1 and B stage
// g mod 3
template <bool DUAL>
__device__ __forceinline__ void big_half(const BigLds& L, int g, int wave, const BigRows& q,
                                         int nk, AccBig& acc, const uint32_t (&a_lane)[2],
                                         const uint32_t (&b_lane)[2], FragA& fa, FragB& fb0,
                                         FragB& fb1) {
  const uint32_t ca = L.a(g), cb = L.b(g), na = L.a(g + 1), nb = L.b(g + 1), db = L.b(g + 2);
  const BigSrc sa(q, g + 1, nk), sb(q, g + 2, nk);
  auto dma_a = [&](int u) { big_dma_a(na, wave, q, sa, u); };
  auto dma_a2 = [&](int u) { big_dma_a(ca, wave, q, sb, u); };
  auto dma_b = [&](int u) { big_dma<DUAL>(db, wave, q, sb, u); };
  big_slot<0, false, DUAL>(fa, fb0, fb1, acc, ca + a_lane[1], cb + b_lane[1], dma_a, dma_b);
  big_slot<0, true, DUAL>(fa, fb1, fb0, acc, na + a_lane[0], nb + b_lane[0], dma_a2, dma_b);
}

// C tile += A rows x B rows over nk slices from the rows' K origin; returns
// with every load landed and every wave past its last LDS access
template <bool DUAL>
__device__ __forceinline__ void big_tile(char* lds, const BigRows& q, int nk, AccBig& acc,
                                         const uint32_t (&a_lane)[2],
                                         const uint32_t (&b_lane)[2]) {
  const BigLds L{lds_addr(lds)};
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  {
    const BigSrc s0(q, 0, nk), s1(q, 1, nk);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      big_dma_a(L.a(0), wave, q, s0, u);
      sched_fence();
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      big_dma<DUAL>(L.b(0), wave, q, s0, u);
      sched_fence();
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      big_dma<DUAL>(L.b(1), wave, q, s1, u);
      sched_fence();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      big_dma_a(L.a(1), wave, q, s1, u);
      sched_fence();
    }
  }
  // A and B of slice 0 have landed (12 newer operations: B of slice 1 and
  // the first half of its A)
  asm volatile("s_waitcnt vmcnt(12)\n\ts_barrier" ::: "memory");
  // the first k-step's fragments, in the order the last k-step of a slice
  // reads them (the first k-step's waits count on it)
  FragA fa;
  FragB fb0, fb1;
  const uint32_t pa = L.a(0) + a_lane[0], pb = L.b(0) + b_lane[0];
  big_read<DUAL, 0>(fa, fb0, pa, pb);
  big_read<DUAL, 1>(fa, fb0, pa, pb);
  big_read<DUAL, 2>(fa, fb0, pa, pb);
  big_read<DUAL, 3>(fa, fb0, pa, pb);
  big_read<DUAL, 4>(fa, fb0, pa, pb);
  big_read<DUAL, 5>(fa, fb0, pa, pb);
  big_read<DUAL, 6>(fa, fb0, pa, pb);
  big_read<DUAL, 7>(fa, fb0, pa, pb);
  big_read<DUAL, 8>(fa, fb0, pa, pb);
  big_read<DUAL, 9>(fa, fb0, pa, pb);
  big_read<DUAL, 11>(fa, fb0, pa, pb);
  big_read<DUAL, 13>(fa, fb0, pa, pb);
  big_read<DUAL, 15>(fa, fb0, pa, pb);
  big_read<DUAL, 10>(fa, fb0, pa, pb);
  big_read<DUAL, 12>(fa, fb0, pa, pb);
  big_read<DUAL, 14>(fa, fb0, pa, pb);
  for (int g = 0; g < nk; ++g)
    big_half<DUAL>(L, g, wave, q, nk, acc, a_lane, b_lane, fa, fb0, fb1);
  // The last k-step read the first fragments of the slice past the end
  // (never used).  Those reads land whenever the LDS returns them, which the
  // compiler cannot see: the wait for them takes their registers as inputs,
  // so no other value is put there before they have landed.
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)"
               :
               : "v"(fa.a[0]), "v"(fa.a[1]), "v"(fa.a[2]), "v"(fa.a[3]), "v"(fa.a[4]),
                 "v"(fa.a[5]), "v"(fa.a[6]), "v"(fa.a[7])
               : "memory");
  asm volatile("" ::"v"(fb0.b[0]), "v"(fb0.b[1]), "v"(fb0.b[2]), "v"(fb0.b[3]), "v"(fb0.b[4]),
               "v"(fb0.b[5]), "v"(fb0.b[6]), "v"(fb0.b[7]));
  // the last MFMAs' results must be in their AGPRs before anything reads
  // them, and the compiler does not see the inline MFMAs' write latency: the
  // wait states follow in an asm statement that takes the last row of
  // accumulators (the other rows were written at least 8 MFMAs earlier).
  // The compiler may still place its own accumulator copies between the
  // loop and this statement, so the emitted code is checked for any access
  // to an MFMA's destination within 19 wait states of it.
  asm volatile("s_barrier\n\ts_nop 7\n\ts_nop 7"
               : "+a"(acc[7][0]), "+a"(acc[7][1]), "+a"(acc[7][2]), "+a"(acc[7][3]),
                 "+a"(acc[7][4]), "+a"(acc[7][5]), "+a"(acc[7][6]), "+a"(acc[7][7])
               :
               : "memory");
}

// ---------------------------------------------- large-group epilogues --
// Activation tile (MODE 0 SwiGLU: silu(g) u with g, u from accumulators j + 4
// and j; MODE 1 ReLU) as bf16 through LDS, so that it leaves as 16-byte row
// chunks instead of one 2-byte store per element.  A lane holds one column
// of 4 rows per accumulator; lanes c and c ^ 1 swap one value of each row
// pair (rows r, r + 1) so that each holds two adjacent columns of one row,
// which v_cvt_pk_bf16_f32 packs (round to nearest even) into one dword of
// the LDS image [256 rows][NT columns].  Every wave's LDS accesses of the
// tile's last slice are done when this runs (the main loop ends on a
// barrier), and it ends on a barrier before the next tile's operands go to
// LDS.
template <int MODE>
__device__ __forceinline__ void big_store_act(char* lds, const FfnArgs& a, AccBig& acc, int m0,
                                              int n0, int a_valid, int b_valid, int wm, int wn,
                                              int lane) {
  constexpr bool DUAL = MODE == 0;
  constexpr int NT = DUAL ? 128 : 256;      // output columns of the tile
  constexpr int RS = NT * 2 + (DUAL ? 16 : 0);  // LDS bytes per row (padded when it fits)
  static_assert(256 * RS <= big::LDS, "activation tile fits the stages");
  const int c = lane & 15, h = lane >> 4;
  const bool odd = c & 1;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < (DUAL ? 4 : 8); ++j) {
      const int col = (DUAL ? wn * 64 : wn * 128) + 16 * j + (c & ~1);
#pragma unroll
      for (int r = 0; r < 4; r += 2) {
        float v0, v1;
        if constexpr (DUAL) {
          v0 = silu_mul(acc[i][j + 4][r], acc[i][j][r]);
          v1 = silu_mul(acc[i][j + 4][r + 1], acc[i][j][r + 1]);
        } else {
          v0 = fmaxf(acc[i][j][r], 0.f);
          v1 = fmaxf(acc[i][j][r + 1], 0.f);
        }
        const float got = swap_pair(odd ? v0 : v1);
        const uint32_t w = odd ? pack_bf16x2(got, v1) : pack_bf16x2(v0, got);
        const int row = wm * 128 + 16 * i + 4 * h + r + (odd ? 1 : 0);
        *reinterpret_cast<uint32_t*>(lds + row * RS + col * 2) = w;
      }
    }
  __syncthreads();
  // 16-byte chunks of the valid rows and columns (N is a multiple of 64, so
  // a chunk is valid or not as a whole)
  constexpr int CPR = NT / 8;
  int N = a.N;
  asm volatile("" : "+s"(N));  // per-tile value: keeps the offsets below inside the tile loop
  const __amdgpu_buffer_rsrc_t ro = buf_rsrc(static_cast<bf16_t*>(a.out) + (size_t)m0 * N + n0);
#pragma unroll 4
  for (int idx = threadIdx.x; idx < 256 * CPR; idx += big::THREADS) {
    const int row = idx / CPR, ch = idx % CPR;
    if (row < a_valid && ch * 8 < b_valid) {
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(lds + row * RS + ch * 16);
      __builtin_amdgcn_raw_buffer_store_b128(v, ro, (uint32_t)((row * N + ch * 8) * 2), 0, 0);
    }
  }
  __syncthreads();
}

// fp32 down partials straight from the accumulators: per store, 16 lanes
// write 64 contiguous bytes of each of 4 rows.  Addresses are a per-lane
// 32-bit offset from the tile's first element plus a wave-uniform one per
// accumulator row (an SGPR), so nothing per element is kept across tiles;
// full tiles skip the per-element bounds tests.
template <bool CHECK>
__device__ __forceinline__ void big_store_partial_rows(AccBig& acc, __amdgpu_buffer_rsrc_t ro,
                                                       uint32_t voff, int N, int rl, int cl,
                                                       int a_valid, int b_valid) {
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (CHECK && cl + 16 * j >= b_valid) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int dr = 16 * i + r;
        if (CHECK && rl + dr >= a_valid) continue;
        // through a VGPR: stored straight from the accumulator registers, every
        // element of a block came out as its first one
        float v = acc[i][j][r];
        asm volatile("" : "+v"(v));
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), ro, voff,
                                              (uint32_t)((dr * N + 16 * j) * 4), 0);
      }
    }
}

// tile partials to `out` (the tile's first element; rows ld floats apart)
__device__ __forceinline__ void big_store_partial(float* out, int ld, AccBig& acc, int a_valid,
                                                  int b_valid, int wm, int wn, int lane) {
  asm volatile("" : "+s"(ld));  // per-tile value: keeps the offsets below inside the tile loop
  const int c = lane & 15, h = lane >> 4;
  const int rl = wm * 128 + 4 * h, cl = wn * 128 + c;  // the lane's first row and column
  const __amdgpu_buffer_rsrc_t ro = buf_rsrc(out);
  const uint32_t voff = (uint32_t)((rl * ld + cl) * 4);
  if (a_valid == big::BM && b_valid == big::BN)
    big_store_partial_rows<false>(acc, ro, voff, ld, rl, cl, a_valid, b_valid);
  else
    big_store_partial_rows<true>(acc, ro, voff, ld, rl, cl, a_valid, b_valid);
}

// Down GEMM of the large-group core (routed experts): with one tile per CU
// and round, the persistent grid's last round is often nearly empty (a
// layer's row tiles x column tiles rarely divide by the CU count).  The
// tiles of full rounds run whole; each of the nr < P tiles left over is cut
// into s equal runs of its K slices (s the largest power of two up to
// kSkPieces with s nr <= P, and at most kSkSlots extra partials), so the
// last round takes 1/s of a tile's time.  All pieces of that round start
// together and pieces with the same K run stay in step, as whole tiles do.
// Piece 0 of a cut tile writes the partial slot of its rows and the tile's
// word (base slot << 4 | s; 0 for a whole tile); piece q > 0 writes the
// compact 256 x 256 partial base + q - 1.  The combine adds them in piece
// order (deterministic).
struct SkPlan {
  int dp, nr, s;  // whole tiles, tiles cut, pieces per cut tile
  __device__ __forceinline__ SkPlan(int nt_all, int P) {
    nr = nt_all % P;
    s = 1;
    while (nr > 0 && s < kSkPieces && 2 * s * nr <= P && nr * (2 * s - 1) <= kSkSlots) s *= 2;
    if (s == 1) nr = 0;
    dp = nt_all - nr;
  }
};

// MODE 0: SwiGLU up and gate (NB operands W0 / W1, 128 output columns per
// tile), MODE 1: ReLU up, MODE 2: down (fp32 out; K splits, or stream-K
// pieces when a.sk_flag is set)
template <int MODE>
__global__ __launch_bounds__(big::THREADS) void k_ffn_big(FfnArgs a) {
  constexpr bool DUAL = MODE == 0;
  constexpr int NT = DUAL ? 128 : 256;  // output columns per tile
  __shared__ __align__(16) char lds[big::LDS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n_nt = (a.N + NT - 1) / NT;
  const int dense_m1 = a.dense_rows ? *a.dense_rows : 0;
  const int n_mt = a.dense_rows ? (dense_m1 + big::BM - 1) / big::BM : *a.n_tiles;
  const bool sk = MODE == 2 && a.sk_flag != nullptr;
  // per-lane LDS offsets of the fragments, per 32-wide k-step (row l % 16,
  // 16-byte chunk 4 ks + l / 16 of the slice, swizzled)
  const int fr = lane & 15, hk = lane >> 4;
  uint32_t a_lane[2], b_lane[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const uint32_t ch = ((4 * ks + hk) ^ swz(fr)) << 4;
    a_lane[ks] = (wm * 128 + fr) * big::RB + ch;
    b_lane[ks] = ((DUAL ? wn * 64 : wn * 128) + fr) * big::RB + ch;
  }
  // operand rows of this thread: r0 + 32 u; it fetches the 16-byte chunk cc
  // of each row segment and writes it to chunk slot tid & 7 of the LDS row,
  // so the stage holds the swizzled layout the fragment reads expect
  const int r0 = tid >> 3;
  const int cc = 8 * ((tid & 7) ^ swz(r0));
  const __amdgpu_buffer_rsrc_t ra = buf_rsrc(a.X);
  AccBig acc;
  // output tile (mt, nt) over K slices [ka, ka + nkp) into partial slot sp
  // of its rows, or (cslot >= 0, down GEMM) compact partial cslot
  auto piece = [&](int mt, int nt, int ka, int nkp, int sp, int cslot) {
    int e = 0, m0, m1;
    if (a.dense_rows) {
      m0 = mt * big::BM;
      m1 = dense_m1;
    } else {
      const int4 tl = a.tiles[mt];
      e = __builtin_amdgcn_readfirstlane(tl.x);
      m0 = __builtin_amdgcn_readfirstlane(tl.y);
      m1 = __builtin_amdgcn_readfirstlane(tl.z);
    }
    const int n0 = nt * NT;
    const int a_valid = min(big::BM, m1 - m0), b_valid = min(NT, a.N - n0);
    const int k0 = ka * BK;
    BigRows q;
    q.ra = ra;
    q.none = buf_rsrc_empty(a.X);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int r = m0 + min(r0 + big::RPP * u, a_valid - 1);
      const int src = a.x_idx ? a.x_idx[r] : r;
      q.off[u] = (uint32_t)(((size_t)src * a.K + k0 + cc) * 2);
    }
    const size_t wo = (size_t)e * a.w_stride + (size_t)n0 * a.K;
    q.rb0 = buf_rsrc(a.W0 + wo);
    q.rb1 = buf_rsrc(DUAL ? a.W1 + wo : a.W0 + wo);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int col = DUAL ? r0 + big::RPP * (u & 3) : r0 + big::RPP * u;
      q.off[8 + u] = (uint32_t)(((size_t)min(col, b_valid - 1) * a.K + k0 + cc) * 2);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = f32x4_t{};
    big_tile<DUAL>(lds, q, nkp, acc, a_lane, b_lane);
    if constexpr (MODE == 2) {
      if (cslot >= 0)
        big_store_partial(a.sk_part + (size_t)cslot * big::BM * big::BN, big::BN, acc, a_valid,
                          b_valid, wm, wn, lane);
      else
        big_store_partial(static_cast<float*>(a.out) + sp * a.split_stride + (size_t)m0 * a.N + n0,
                          a.N, acc, a_valid, b_valid, wm, wn, lane);
    } else {
      big_store_act<MODE>(lds, a, acc, m0, n0, a_valid, b_valid, wm, wn, lane);
    }
  };
  if (!sk) {
    TileSched S;
    int ntiles;
    if (!S.init(n_mt, n_nt, a.n_split, ntiles)) return;
    clock_mark(a.clk, true);
    const int nk = (a.K / BK) / a.n_split;
    for (int jt = 0; jt < ntiles; ++jt) {
      int mt, nt, sp;
      S.decode(jt, mt, nt, sp);
      piece(mt, nt, sp * nk, nk, sp, -1);
    }
    clock_mark(a.clk, false);
    return;
  }
  const int P = gridDim.x, nk = a.K / BK;
  clock_mark(a.clk, true);
  const SkPlan plan(n_mt * n_nt, P);
  // whole tiles, in the usual XCD-range order
  TileSched S;
  int ntiles;
  if (S.init_total(plan.dp, n_mt, n_nt, ntiles)) {
    for (int jt = 0; jt < ntiles; ++jt) {
      int mt, nt, sp;
      S.decode(jt, mt, nt, sp);
      piece(mt, nt, 0, nk, 0, -1);
      if (tid == 0) a.sk_flag[mt * n_nt + nt] = 0;
    }
  }
  // the cut tiles of the last round: CU v (numbered XCD by XCD) takes piece
  // v % s of tile v / s
  const int nx = min(kXcd, P), x = blockIdx.x % nx;
  const int v = x * (P / nx) + min(x, P % nx) + (int)blockIdx.x / nx;
  if (v < plan.nr * plan.s) {
    const int t = v / plan.s, q = v % plan.s;
    const int k0 = q * nk / plan.s, k1 = (q + 1) * nk / plan.s;
    int mt, nt, sp;
    S.n_mt = n_mt;
    S.n_nt = n_nt;
    S.decode_abs(plan.dp + t, mt, nt, sp);
    const int base = t * (plan.s - 1);
    piece(mt, nt, k0, k1 - k0, 0, q == 0 ? -1 : base + q - 1);
    if (q == 0 && tid == 0) a.sk_flag[mt * n_nt + nt] = (base << 4) | plan.s;
  }
  clock_mark(a.clk, false);
}

// ----------------------------------------------------------- exit head --
// M = vocabulary (A = W_exit [V, d]), N = executed tokens (B = hx [n_x, d],
// the executed tokens' updated rows written by the combine kernel).
// Epilogue: for every token column, max and sum exp over the tile's
// vocabulary rows (bias added), written as one partial per vocabulary tile
// as (max z * log2 e, sum exp(z - max z)).
struct ExitArgs {
  const bf16_t* W;    // [V, K]
  const bf16_t* H;    // [n_x, K]
  const float* bias;  // [V] or NULL
  const int* n_exec;  // device
  int V, K, n_vtiles;
  float2* partials;   // [n_x, n_vtiles]
  unsigned long long* clk;  // engine-clock record (see clock_mark), or NULL
};

using ExitTile = Tile<kExitTileBF16, 128, 1, 4, 2>;
// 256 tokens per tile for large batches: 64 x 128 wavefront tiles read 3/4 of
// the LDS bytes per MFMA of the 64 x 64 ones and the DMA writes 2/3, which
// brings a k-step's LDS traffic (~125 B/clk at the MFMA peak) under the LDS
// bandwidth (128 B/clk; the 128-token tile needs ~172).  It runs a two-stage
// ring (the 128-token tile keeps three stages, and its finer token tiles
// balance the persistent grid better at small n_x)
using ExitWide = Tile<kExitTileBF16, 256, 1, 4, 2>;
// decode-sized batches (kExitSmallTokens or fewer): 32 token columns, 128
// vocabulary rows, so the tiles cover the CUs and the MFMA work is not 4x
// padding; W_exit streaming (HBM) bounds it
using ExitSmall = Tile<kExitTileBF16Small, 32, 1, 4, 1>;

template <class T, bool ARGMAX = false>
struct ExitSrc {
  struct Desc {
    int mt, nt;
    static __device__ __forceinline__ Desc pick(bool c, const Desc& x, const Desc& y) {
      return Desc{c ? x.mt : y.mt, c ? x.nt : y.nt};
    }
  };
  const ExitArgs& a;
  const TileSched& S;
  int n_x;
  float2 (*s_part)[T::BN];  // [GM][BN] LDS exchange of the epilogue

  __device__ __forceinline__ Desc desc(int j) const {
    int mt, nt, sp;
    S.decode(j, mt, nt, sp);
    return Desc{mt, nt};
  }
  __device__ __forceinline__ void rows(const Desc& d, int (&src)[T::A_PT]) const {
    const int v0 = d.mt * T::BM, a_valid = min(T::BM, a.V - v0);
#pragma unroll
    for (int i = 0; i < T::A_PT; ++i) src[i] = v0 + min(dma_row(i, T::ROWS_PER_PASS), a_valid - 1);
  }
  __device__ __forceinline__ void ptrs(DPtrs<T>& q, const Desc& d,
                                       const int (&src)[T::A_PT]) const {
    const int j0 = d.nt * T::BN;
    make_dptrs<T>(q, a.W, src, a.H, nullptr, j0, min(T::BN, n_x - j0), a.K, 0);
  }
  __device__ __forceinline__ void epilogue(const Desc& d, Acc<T>& acc) const {
    if constexpr (ARGMAX)
      epilogue_argmax(d, acc);
    else
      epilogue_softmax(d, acc);
  }
  // per (token, vocabulary tile): the largest logit and its vocabulary row
  // (ties to the lower row), the row stored as the float's bit pattern
  __device__ __forceinline__ void epilogue_argmax(const Desc& d, Acc<T>& acc) const {
    const int v0 = d.mt * T::BM, j0 = d.nt * T::BN;
    const int a_valid = min(T::BM, a.V - v0);
    const int b_valid = min(T::BN, n_x - j0);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / T::GN, wn = wave % T::GN;
#pragma unroll
    for (int jj = 0; jj < T::TN; ++jj) {
      float m = -__builtin_inff();
      int mi = 0x7fffffff;
#pragma unroll
      for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = acc_row<T>(wm, i, r, lane);
          float y = acc[i][jj][r];
          if (a.bias) y += a.bias[v0 + min(row, a_valid - 1)];
          if (row < a_valid && (y > m || (y == m && row < mi))) {
            m = y;
            mi = row;
          }
        }
      // the better of the two row halves (ties to the lower row); lanes 0..31,
      // the ones that store it, hold their own candidate in a
      const LanePair pm = lanes_xor32(m), pi = lanes_xor32(__int_as_float(mi));
      const int ia = __float_as_int(pi.a), ib = __float_as_int(pi.b);
      const bool take_b = pm.b > pm.a || (pm.b == pm.a && ib < ia);
      m = take_b ? pm.b : pm.a;
      mi = take_b ? ib : ia;
      if (lane < 32) s_part[wm][acc_col<T>(wn, jj, lane)] = make_float2(m, __int_as_float(mi));
    }
    lds_barrier();
    const int c = threadIdx.x;
    if (c < b_valid) {
      float M = s_part[0][c].x;
      int R = __float_as_int(s_part[0][c].y);
#pragma unroll
      for (int g = 1; g < T::GM; ++g) {
        const float2 v = s_part[g][c];
        const int rv = __float_as_int(v.y);
        if (v.x > M || (v.x == M && rv < R)) {
          M = v.x;
          R = rv;
        }
      }
      a.partials[(size_t)(j0 + c) * a.n_vtiles + d.mt] = make_float2(M, __int_as_float(v0 + R));
    }
  }
  __device__ __forceinline__ void epilogue_softmax(const Desc& d, Acc<T>& acc) const {
    const int v0 = d.mt * T::BM, j0 = d.nt * T::BN;
    const int a_valid = min(T::BM, a.V - v0);
    const int b_valid = min(T::BN, n_x - j0);
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
      {
        const LanePair pm = lanes_xor32(m);
        m = fmaxf(pm.a, pm.b);
      }
      float sum = 0.f;
      if (m != ninf) {
#pragma unroll
        for (int i = 0; i < T::TM; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) sum += __builtin_amdgcn_exp2f(acc[i][jj][r] - m);
      }
      {
        const LanePair ps = lanes_xor32(sum);
        sum = ps.a + ps.b;
      }
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
      a.partials[(size_t)(j0 + c) * a.n_vtiles + d.mt] = make_float2(M, S2);
    }
  }
};

template <class T, bool ARGMAX = false>
__global__ __launch_bounds__(T::THREADS) void k_exit_mma(ExitArgs a) {
  __shared__ __align__(16) char lds[DmaTile<T>::LDS];
  __shared__ float2 s_part[T::GM][T::BN];  // per wavefront row: (max, sum) per token column
  const int n_x = *a.n_exec;
  TileSched S;
  int ntiles;
  if (!S.init(a.n_vtiles, (n_x + T::BN - 1) / T::BN, 1, ntiles)) return;
  clock_mark(a.clk, true);
  const ExitSrc<T, ARGMAX> src{a, S, n_x, s_part};
  dma_gemm_stream<T>(lds, ntiles, a.K / BK, src);
  clock_mark(a.clk, false);
}

// Exit head on the large-group core (large d): 256 vocabulary rows x 256
// executed tokens per tile, the same softmax partials as the epilogue above.
// A wavefront reduces its 128 rows of a token column (64 per lane, then the
// other half-wavefront); the two row halves meet in LDS.

// operand rows of tile j: vocabulary rows (A) and executed-token rows (B),
// clamped to the valid ones
__device__ __forceinline__ void exit_big_rows(BigRows& q, const ExitArgs& a, const TileSched& S,
                                              int n_x, int j, int r0, int cc) {
  int vt, tt, sp;
  S.decode(j, vt, tt, sp);
  const int v0 = vt * big::BM, c0 = tt * big::BN;
  const int a_valid = min(big::BM, a.V - v0), b_valid = min(big::BN, n_x - c0);
  q.rb0 = buf_rsrc(a.H + (size_t)c0 * a.K);
  q.rb1 = q.rb0;
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    q.off[u] = (uint32_t)(((size_t)(v0 + min(r0 + big::RPP * u, a_valid - 1)) * a.K + cc) * 2);
    q.off[8 + u] = (uint32_t)(((size_t)min(r0 + big::RPP * u, b_valid - 1) * a.K + cc) * 2);
  }
}

// partials in base 2 (y = z log2 e) of tile j: per token column the largest y
// and the sum of 2^(y - max y) over the tile's vocabulary rows.  Two passes
// over the accumulators (the logit z is recomputed, nothing written back):
// the largest z, then sum 2^(z log2 e - max y), one FMA and one v_exp_f32
// per logit.  A lane holds 4 rows of one token column per accumulator; the
// four row groups of a column (lanes l, l ^ 16, l ^ 32, l ^ 48) combine by
// lane exchange, the two row halves of the tile in LDS.  Partial tiles (last
// vocabulary tile, or a bias) take the bias and row mask in both passes.
// The tile's loads have all landed by now, so the LDS exchange waits for LDS
// work only.
__device__ __forceinline__ void exit_big_epilogue(const ExitArgs& a, const TileSched& S, int n_x,
                                                  int jt, const AccBig& acc,
                                                  float2 (*s_part)[big::BN], int wm, int wn,
                                                  int lane) {
  int vt, tt, sp;
  S.decode(jt, vt, tt, sp);
  const int v0 = vt * big::BM, c0 = tt * big::BN;
  const int a_valid = min(big::BM, a.V - v0), b_valid = min(big::BN, n_x - c0);
  const int h = lane >> 4;
  const float ninf = -__builtin_inff();
  const float kLog2e = 1.4426950408889634f;
  const bool full = a_valid == big::BM && !a.bias;
  // this lane's rows are wm * 128 + 4 h + o, o = 16 i + r; row o is valid for
  // o < lim, and bias row min(o, lim - 1) stays in range
  const int lim = a_valid - (wm * 128 + 4 * h);
  const float* bias = a.bias ? a.bias + v0 + wm * 128 + 4 * h : nullptr;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    float mz = ninf;
    if (full) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) mz = fmaxf(mz, acc[i][j][r]);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int o = 16 * i + r;
          const float b = bias ? bias[min(o, lim - 1)] : 0.f;
          mz = fmaxf(mz, o < lim ? acc[i][j][r] + b : ninf);
        }
    }
    {
      const LanePair p16 = lanes_xor16(mz);
      mz = fmaxf(p16.a, p16.b);
      const LanePair p32 = lanes_xor32(mz);
      mz = fmaxf(p32.a, p32.b);
    }
    const float m = mz * kLog2e;
    float sum = 0.f;
    if (mz != ninf) {
      if (full) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) sum += __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, -m));
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int o = 16 * i + r;
            const float b = bias ? bias[min(o, lim - 1)] : 0.f;
            const float e = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r] + b, kLog2e, -m));
            sum += o < lim ? e : 0.f;
          }
      }
    }
    {
      const LanePair p16 = lanes_xor16(sum);
      sum = p16.a + p16.b;
      const LanePair p32 = lanes_xor32(sum);
      sum = p32.a + p32.b;
    }
    if (lane < 16) s_part[wm][wn * 128 + 16 * j + lane] = make_float2(m, sum);
  }
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  const int c = threadIdx.x;
  if (c < b_valid) {
    const float2 p0 = s_part[0][c], p1 = s_part[1][c];
    const float M = fmaxf(p0.x, p1.x);
    float S2 = 0.f;
    if (p0.y > 0.f) S2 += p0.y * __builtin_amdgcn_exp2f(p0.x - M);
    if (p1.y > 0.f) S2 += p1.y * __builtin_amdgcn_exp2f(p1.x - M);
    a.partials[(size_t)(c0 + c) * a.n_vtiles + vt] = make_float2(M, S2);
  }
  // s_part is rewritten by the next epilogue only after the next tile's
  // slice barriers
}

__global__ __launch_bounds__(big::THREADS) void k_exit_big(ExitArgs a) {
  __shared__ __align__(16) char lds[big::LDS];
  // per row half: (max y, sum) per token column, in the last B stage (free
  // while the epilogue runs; the next tile writes it only after its first
  // slice barrier)
  float2(*s_part)[big::BN] = reinterpret_cast<float2(*)[big::BN]>(lds + big::B0 + 2 * big::BB);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n_x = *a.n_exec;
  TileSched S;
  int ntiles;
  if (!S.init(a.n_vtiles, (n_x + big::BN - 1) / big::BN, 1, ntiles)) return;
  clock_mark(a.clk, true);
  const int nk = a.K / BK;
  const int fr = lane & 15, hk = lane >> 4;
  uint32_t a_lane[2], b_lane[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const uint32_t ch = ((4 * ks + hk) ^ swz(fr)) << 4;
    a_lane[ks] = (wm * 128 + fr) * big::RB + ch;
    b_lane[ks] = (wn * 128 + fr) * big::RB + ch;
  }
  const int r0 = tid >> 3;
  const int cc = 8 * ((tid & 7) ^ swz(r0));
  BigRows q;
  q.ra = buf_rsrc(a.W);
  q.none = buf_rsrc_empty(a.W);
  AccBig acc;
  for (int jt = 0; jt < ntiles; ++jt) {
    exit_big_rows(q, a, S, n_x, jt, r0, cc);
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = f32x4_t{};
    big_tile<false>(lds, q, nk, acc, a_lane, b_lane);
    exit_big_epilogue(a, S, n_x, jt, acc, s_part, wm, wn, lane);
  }
  clock_mark(a.clk, false);
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
template <bool ARGMAX = false>
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
    const float* h = H + (size_t)(tok ? tok[j] : j) * K;
    float acc = 0.f;
    for (int c = 0; c < K; ++c) acc = fmaf(w[c], h[c], acc);
    z = acc + (bias ? bias[v] : 0.f);
  }
  s_z[tv][tj] = z;
  __syncthreads();
  if (threadIdx.x < FT) {
    const int jj = jt * FT + threadIdx.x;
    if (jj < n_x && ARGMAX) {
      // the largest logit of the tile and its row (ties to the lower row)
      float m = -__builtin_inff();
      int mi = vt * FT;
      for (int u = 0; u < FT && vt * FT + u < V; ++u)
        if (s_z[u][threadIdx.x] > m) {
          m = s_z[u][threadIdx.x];
          mi = vt * FT + u;
        }
      partials[(size_t)jj * n_vtiles + vt] = make_float2(m, __int_as_float(mi));
    } else if (jj < n_x) {
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

// Tile shapes of the expert GEMMs (BM rows of an expert group x BN outputs).
// Three-stage rings: the expert weights stream from HBM, and two slices in
// flight measured faster than 256-row two-stage tiles even for large groups.
using UpDualTile = Tile<kGemmBM, 128, 2, 2, 4>;  // SwiGLU: up and gate share A
using UpTile = Tile<kGemmBM, 256, 1, 2, 4>;      // ReLU
using DownTile = Tile<kGemmBM, 256, 1, 2, 4>;

// K splits of the routed down GEMM, only for a tile bound under two tiles
// per CU (1, 2 or 4, each split keeping at least 8 K slices): the fewest
// slices on the busiest CU of a 256-CU persistent grid, and on a tie the
// fewer splits (fewer fp32 partial slices to write and for the combine to
// read).
int down_splits(int max_tiles, int N, int K) {
  constexpr int kCu = 256;
  const int tiles = max_tiles * cdiv(N, DownTile::BN);
  const int nk = K / BK;
  if (tiles >= 2 * kCu) return 1;
  int best = 1;
  long best_cost = (long)cdiv(tiles, kCu) * nk;
  for (int s = 2; s <= 4; s *= 2) {
    if (nk % s != 0 || nk / s < 8) break;
    const long cost = (long)cdiv(tiles * s, kCu) * (nk / s);
    if (cost < best_cost) {
      best = s;
      best_cost = cost;
    }
  }
  return best;
}

// persistent: at most one block per CU, none beyond the tile bound
template <class T, bool UP>
static void launch_ffn_mma(const FfnArgs& a, int max_mt, int n_cu, hipStream_t st) {
  const dim3 grid(min(max_mt * cdiv(a.N, T::BN) * a.n_split, n_cu));
  hipLaunchKernelGGL((k_ffn_mma<T, UP>), grid, dim3(T::THREADS), 0, st, a);
}

// persistent: at most one block per CU, none beyond the tile bound
template <int MODE>
static void launch_ffn_big(const FfnArgs& a, int max_mt, int n_cu, hipStream_t st) {
  const int nt = cdiv(a.N, MODE == 0 ? 128 : big::BN);
  // cut tiles of the down GEMM: up to kSkPieces pieces each
  const dim3 grid(min(max_mt * nt * (a.sk_flag ? kSkPieces : a.n_split), n_cu));
  hipLaunchKernelGGL(k_ffn_big<MODE>, grid, dim3(big::THREADS), 0, st, a);
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
    // large groups: the routed tile list was built with kBigBM rows per tile
    const bool big = shared ? big_dense(true, p.T, p.d, p.Fs) : p.bm == kBigBM;
    FfnArgs a{static_cast<const bf16_t*>(X), x_idx, static_cast<const bf16_t*>(w0),
              static_cast<const bf16_t*>(w1), w_stride, K, N, p.tiles, &p.counts[kCntTiles],
              dense, out, p.y_split_stride, n_split, act,
              (!up && !shared && big) ? p.sk_flag : nullptr, p.sk_part,
              p.clk ? p.clk + 2 * (shared ? TRIMMOE_CLASS_SHARED
                                          : up ? TRIMMOE_CLASS_UP : TRIMMOE_CLASS_DOWN)
                    : nullptr};
    if (big) {
      const int big_mt = shared ? cdiv(p.T, kBigBM) : cdiv(p.T * p.k, kBigBM) + p.E;
      if (up && dual)
        launch_ffn_big<0>(a, big_mt, p.n_cu, st);
      else if (up)
        launch_ffn_big<1>(a, big_mt, p.n_cu, st);
      else
        launch_ffn_big<2>(a, big_mt, p.n_cu, st);
    } else if (up && dual)
      launch_ffn_mma<UpDualTile, true>(a, max_mt, p.n_cu, st);
    else if (up)
      launch_ffn_mma<UpTile, true>(a, max_mt, p.n_cu, st);
    else
      launch_ffn_mma<DownTile, false>(a, max_mt, p.n_cu, st);
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
               &p.counts[kCntExec], p.V, p.d, p.n_vtiles, p.partials,
               p.clk ? p.clk + 2 * TRIMMOE_CLASS_EXIT : nullptr};
    // persistent: at most one block per CU, none beyond the tile bound
    if (big_exit(true, p.T, p.V, p.d)) {
      const dim3 grid(min(p.n_vtiles * cdiv(p.T, big::BN), p.n_cu));
      hipLaunchKernelGGL(k_exit_big, grid, dim3(big::THREADS), 0, st, a);
    } else if (p.T <= kExitSmallTokens) {
      const dim3 grid(min(p.n_vtiles * cdiv(p.T, ExitSmall::BN), p.n_cu));
      hipLaunchKernelGGL(k_exit_mma<ExitSmall>, grid, dim3(ExitSmall::THREADS), 0, st, a);
    } else if (p.T >= kWideTokens) {
      const dim3 grid(min(p.n_vtiles * cdiv(p.T, ExitWide::BN), p.n_cu));
      hipLaunchKernelGGL(k_exit_mma<ExitWide>, grid, dim3(ExitWide::THREADS), 0, st, a);
    } else {
      const dim3 grid(min(p.n_vtiles * cdiv(p.T, ExitTile::BN), p.n_cu));
      hipLaunchKernelGGL(k_exit_mma<ExitTile>, grid, dim3(ExitTile::THREADS), 0, st, a);
    }
  } else {
    const dim3 grid(p.n_vtiles * cdiv(p.T, FT));
    hipLaunchKernelGGL(k_exit_f32<false>, grid, dim3(256), 0, st, static_cast<const float*>(p.w_exit),
                       static_cast<const float*>(p.h), p.exec_list, p.b_exit, &p.counts[kCntExec],
                       p.V, p.d, p.n_vtiles, p.partials);
  }
  return hipGetLastError();
}

hipError_t launch_head_argmax_partials(bool bf16, const void* W, const float* bias, const void* H,
                                       const int* n_rows_dev, int n_rows, int V, int K,
                                       int n_vtiles, float2* partials, int n_cu, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  if (bf16) {
    ExitArgs a{static_cast<const bf16_t*>(W), static_cast<const bf16_t*>(H), bias, n_rows_dev, V,
               K, n_vtiles, partials};
    if (n_rows <= kExitSmallTokens) {
      const dim3 grid(min(n_vtiles * cdiv(n_rows, ExitSmall::BN), n_cu));
      hipLaunchKernelGGL((k_exit_mma<ExitSmall, true>), grid, dim3(ExitSmall::THREADS), 0, st, a);
    } else if (n_rows >= kWideTokens) {
      const dim3 grid(min(n_vtiles * cdiv(n_rows, ExitWide::BN), n_cu));
      hipLaunchKernelGGL((k_exit_mma<ExitWide, true>), grid, dim3(ExitWide::THREADS), 0, st, a);
    } else {
      const dim3 grid(min(n_vtiles * cdiv(n_rows, ExitTile::BN), n_cu));
      hipLaunchKernelGGL((k_exit_mma<ExitTile, true>), grid, dim3(ExitTile::THREADS), 0, st, a);
    }
  } else {
    const dim3 grid(n_vtiles * cdiv(n_rows, FT));
    hipLaunchKernelGGL(k_exit_f32<true>, grid, dim3(256), 0, st, static_cast<const float*>(W),
                       static_cast<const float*>(H), nullptr, bias, n_rows_dev, V, K, n_vtiles,
                       partials);
  }
  return hipGetLastError();
}

}  // namespace trimmoe
