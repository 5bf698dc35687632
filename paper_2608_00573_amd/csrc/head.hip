// Exit-head training of Sec. IV-A on cached hidden states: the prediction of
// a representation (argmax of an output head, for the consistency labels of
// Eq. (22)) and full-batch gradient descent of the sigmoid exit head on the
// binary cross-entropy of Eq. (23).  Reductions run in a fixed order (fp64
// accumulators), so repeated runs give identical weights.
#include "common.h"

namespace trimmoe {

namespace {
inline int cdiv(int a, int b) { return (a + b - 1) / b; }
}  // namespace

__global__ void k_set_int(int32_t* p, int v) { *p = v; }

hipError_t launch_set_int(int32_t* p, int v, hipStream_t st) {
  hipLaunchKernelGGL(k_set_int, dim3(1), dim3(1), 0, st, p, v);
  return hipGetLastError();
}

// argmax over the vocabulary tiles of one row: the largest logit, ties to
// the lower vocabulary row.  One wavefront per row.
__global__ __launch_bounds__(256) void k_argmax_reduce(const float2* partials, int n_vtiles,
                                                       int n_rows, int32_t* out) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = blockIdx.x * 4 + wave;
  if (q >= n_rows) return;
  const float2* pr = partials + (size_t)q * n_vtiles;
  float m = -__builtin_inff();
  int mi = 0x7fffffff;
  for (int u = lane; u < n_vtiles; u += 64) {
    const float2 v = pr[u];
    const int r = __float_as_int(v.y);
    if (v.x > m || (v.x == m && r < mi)) {
      m = v.x;
      mi = r;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o);
    const int r2 = __shfl_xor(mi, o);
    if (m2 > m || (m2 == m && r2 < mi)) {
      m = m2;
      mi = r2;
    }
  }
  if (lane == 0) out[q] = mi;
}

hipError_t launch_argmax_reduce(const float2* partials, int n_vtiles, int n_rows, int32_t* out,
                                hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_argmax_reduce, dim3(cdiv(n_rows, 4)), dim3(256), 0, st, partials,
                     n_vtiles, n_rows, out);
  return hipGetLastError();
}

// Eq. (22): labels[q] = 1 where the layer's prediction equals the full-depth one
__global__ void k_consistency(const int32_t* pred, const int32_t* ref, int n_rows,
                              uint8_t* labels) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q < n_rows) labels[q] = pred[q] == ref[q] ? 1 : 0;
}

hipError_t launch_consistency(const int32_t* pred, const int32_t* ref, int n_rows,
                              uint8_t* labels, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_consistency, dim3(cdiv(n_rows, 256)), dim3(256), 0, st, pred, ref, n_rows,
                     labels);
  return hipGetLastError();
}

// Logit z = w . h + c of every row (one wavefront per row, fixed butterfly),
// the residual sigmoid(z) - y of the gradient and the row's loss
// max(z, 0) - y z + log(1 + exp(-|z|)) of Eq. (23).
template <typename T>
__global__ __launch_bounds__(256) void k_bce_logits(const T* H, const uint8_t* y, int n_rows, int d,
                                                    const float* w, const float* c, float* r,
                                                    double* row_loss) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = blockIdx.x * 4 + wave;
  if (q >= n_rows) return;
  const T* h = H + (size_t)q * d;
  float acc = 0.f;
  for (int k = lane; k < d; k += 64) acc = fmaf(w[k], to_f32<T>(h[k]), acc);
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) {
    const float z = acc + *c;
    const float label = y[q] ? 1.f : 0.f;
    r[q] = 1.f / (1.f + expf(-z)) - label;
    const double zd = z;
    row_loss[q] = fmax(zd, 0.0) - (double)label * zd + log1p(exp(-fabs(zd)));
  }
}

// w[k] -= lr * sum_q r[q] h[q][k] / Q, one column per thread, rows in order;
// block 0 also moves c by lr * mean r and writes the mean loss.
template <typename T>
__global__ __launch_bounds__(256) void k_bce_update(const T* H, int n_rows, int d, float lr,
                                                    const float* r, const double* row_loss,
                                                    float* w, float* c, float* loss_out) {
  __shared__ double s_r[256], s_l[256];
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k < d) {
    double g = 0.0;
    for (int q = 0; q < n_rows; ++q) g += (double)r[q] * (double)to_f32<T>(H[(size_t)q * d + k]);
    w[k] -= lr * (float)(g / n_rows);
  }
  if (blockIdx.x != 0) return;
  double sr = 0.0, sl = 0.0;
  for (int q = threadIdx.x; q < n_rows; q += 256) {
    sr += (double)r[q];
    sl += row_loss[q];
  }
  s_r[threadIdx.x] = sr;
  s_l[threadIdx.x] = sl;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      s_r[threadIdx.x] += s_r[threadIdx.x + s];
      s_l[threadIdx.x] += s_l[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *c -= lr * (float)(s_r[0] / n_rows);
    if (loss_out) *loss_out = (float)(s_l[0] / n_rows);
  }
}

hipError_t launch_bce_step(bool bf16, const void* H, const uint8_t* y, int n_rows, int d,
                           float lr, float* w, float* c, float* r, double* row_loss,
                           float* loss_out, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  const dim3 g1(cdiv(n_rows, 4)), g2(cdiv(d, 256)), b(256);
  if (bf16) {
    hipLaunchKernelGGL(k_bce_logits<bf16_t>, g1, b, 0, st, static_cast<const bf16_t*>(H), y,
                       n_rows, d, w, c, r, row_loss);
    hipLaunchKernelGGL(k_bce_update<bf16_t>, g2, b, 0, st, static_cast<const bf16_t*>(H), n_rows,
                       d, lr, r, row_loss, w, c, loss_out);
  } else {
    hipLaunchKernelGGL(k_bce_logits<float>, g1, b, 0, st, static_cast<const float*>(H), y, n_rows,
                       d, w, c, r, row_loss);
    hipLaunchKernelGGL(k_bce_update<float>, g2, b, 0, st, static_cast<const float*>(H), n_rows,
                       d, lr, r, row_loss, w, c, loss_out);
  }
  return hipGetLastError();
}

}  // namespace trimmoe
