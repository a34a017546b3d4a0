// alpha-CROWN state kernels (paper, Sec. 2.1: the lower slopes of unstable ReLU neurons
// become parameters in [0, 1], raised by gradient steps; Sec. 4.6: one slope per layer,
// specification row, input and neuron).  Every specification bound is a coefficient row
// (unit, q): q < m the lower bound of row q, q >= m the negated upper bound of row q - m, so
// every row maximises its own lower bound.  The per-layer state arrays are [M_pad][ld] with
// the GEMM's row and column padding.
#include "kernels.h"

namespace vcr {

// column of neuron n (this layer's order) in the compact per-row layout
__device__ __forceinline__ int64_t compact_col(const AlphaLayer &l, int64_t n) {
  if (l.hwc_C == 0) return n;
  const int64_t pos = n / l.hwc_C;
  return (n - pos * l.hwc_C) * l.hwc_HW + pos;
}

__global__ void k_alpha_init(AlphaLayer l, const float *alpha_init, int64_t n_total, int32_t rows, int32_t rows_pad,
                             int32_t rows_per_unit) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)rows_pad * l.ld) return;
  const int64_t row = idx / l.ld;
  const int32_t n = (int32_t)(idx - row * l.ld);
  float a = 0.f;
  if (row < rows && n < l.n) {
    // unstable neurons (t > 0) take the given slope, the others keep their fixed one
    const int64_t u = row / rows_per_unit;
    const float4 prm = l.P[u * l.ldp + n];
    a = (alpha_init && prm.z > 0.f) ? alpha_init[row * n_total + l.col0 + compact_col(l, n)] : prm.x;
  }
  l.alpha[idx] = a;
  l.best[idx] = a;
  l.mom[idx] = 0.f;
  l.vel[idx] = 0.f;
  l.grad[idx] = 0.f;
  l.pre[idx] = 0.f;   // coefficients a pass does not record (stable neurons) read as 0
}

hipError_t launch_alpha_init(const AlphaLayer &l, const float *alpha_init, int64_t n_total, int32_t rows,
                             int32_t rows_pad, int32_t rows_per_unit, hipStream_t s) {
  const int64_t n = (int64_t)rows_pad * l.ld;
  hipLaunchKernelGGL(k_alpha_init, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, l, alpha_init, n_total, rows,
                     rows_pad, rows_per_unit);
  return hipGetLastError();
}

// E0 = c - sign(a) r: the vertex where a . x is smallest (the centre where a = 0)
__global__ void k_alpha_vertex(const float *pre0, int64_t ld0, const float *c0, const float *r0, int32_t rows_pad,
                               int32_t rows_per_unit, int32_t units, float *E0) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)rows_pad * ld0) return;
  const int64_t row = idx / ld0;
  const int64_t i = idx - row * ld0;
  int64_t u = row / rows_per_unit;
  u = u < units ? u : units - 1;
  const float a = pre0[idx];
  const float c = c0[u * ld0 + i], r = r0[u * ld0 + i];
  E0[idx] = a > 0.f ? c - r : (a < 0.f ? c + r : c);
}

hipError_t launch_alpha_vertex(const float *pre0, int64_t ld0, const float *c0, const float *r0, int32_t rows_pad,
                               int32_t rows_per_unit, int32_t units, float *E0, hipStream_t s) {
  const int64_t n = (int64_t)rows_pad * ld0;
  hipLaunchKernelGGL(k_alpha_vertex, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, pre0, ld0, c0, r0, rows_pad,
                     rows_per_unit, units, E0);
  return hipGetLastError();
}

__global__ void k_alpha_best(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad, int32_t rows,
                             int32_t m, int32_t first, float *best_val, int32_t *flag, float *hist_lb,
                             float *hist_ub) {
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= rows) return;
  float sp = 0.f;
  for (int p = 0; p < n_parts; ++p) sp += cpart[(int64_t)p * M_pad + row];
  const float v = beta[row] + sp;
  const bool better = first || v > best_val[row];
  if (better) best_val[row] = v;
  flag[row] = better ? 1 : 0;
  const int64_t u = row / (2 * m);
  const int32_t q = (int32_t)(row - u * 2 * m);
  if (hist_lb) {
    if (q < m)
      hist_lb[u * m + q] = v;
    else
      hist_ub[u * m + q - m] = -v;
  }
}

hipError_t launch_alpha_best(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad, int32_t rows,
                             int32_t m, int32_t first, float *best_val, int32_t *flag, float *hist_lb,
                             float *hist_ub, hipStream_t s) {
  hipLaunchKernelGGL(k_alpha_best, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, beta, cpart, n_parts, M_pad,
                     rows, m, first, best_val, flag, hist_lb, hist_ub);
  return hipGetLastError();
}

// The slope-state kernels run one thread per 4 consecutive columns of a row (ld is a multiple
// of 128), workgroups of 256 threads covering 1024 columns of one row.
constexpr int ALPHA_COLS_PER_BLOCK = 1024;

// best <- alpha on the rows whose bound improved (flag)
__global__ void k_alpha_keep(AlphaLayer l, const int32_t *flag, int32_t blocks_per_row) {
  const int32_t row = blockIdx.x / blocks_per_row;
  const int64_t n0 = (int64_t)(blockIdx.x - row * blocks_per_row) * ALPHA_COLS_PER_BLOCK + threadIdx.x * 4;
  if (n0 >= l.ld || !flag[row]) return;
  const int64_t idx = (int64_t)row * l.ld + n0;
  *reinterpret_cast<float4 *>(l.best + idx) = *reinterpret_cast<const float4 *>(l.alpha + idx);
}

hipError_t launch_alpha_keep(const AlphaLayer &l, const int32_t *flag, int32_t rows, hipStream_t s) {
  if (l.ld % 4) return hipErrorInvalidValue;
  const int32_t bpr = (int32_t)((l.ld + ALPHA_COLS_PER_BLOCK - 1) / ALPHA_COLS_PER_BLOCK);
  hipLaunchKernelGGL(k_alpha_keep, dim3((unsigned)((int64_t)rows * bpr)), dim3(256), 0, s, l, flag, bpr);
  return hipGetLastError();
}

// Adam (bias-corrected moments) then projection onto [0, 1].  Only unstable neurons move:
// the gradient pass writes a zero gradient at every other column (stable neurons, split
// neurons made stable), whose moments therefore stay zero and whose step is exactly 0, and
// their slopes start at lambda in {0, 1}, which the projection keeps; so no relaxation
// parameter is read here and the result is the same as skipping those columns.  With flag, the rows whose bound improved first
// keep their current slopes in best (the keep step folded into the same pass over the state).
typedef float adam_f32x4 __attribute__((ext_vector_type(4)));
__global__ void k_alpha_adam(AlphaLayer l, const int32_t *flag, int32_t blocks_per_row, float lr, float beta1,
                             float beta2, float eps, float c1, float c2) {
  const int32_t row = blockIdx.x / blocks_per_row;
  const int64_t n0 = (int64_t)(blockIdx.x - row * blocks_per_row) * ALPHA_COLS_PER_BLOCK + threadIdx.x * 4;
  if (n0 >= l.ld) return;
  const int64_t idx = (int64_t)row * l.ld + n0;
  const float4 a4 = *reinterpret_cast<const float4 *>(l.alpha + idx);
  if (flag && flag[row]) *reinterpret_cast<float4 *>(l.best + idx) = a4;
  if (n0 >= l.n) return;
  // the gradient and the moments are touched once per step: streamed past the caches
  const adam_f32x4 g4 = __builtin_nontemporal_load(reinterpret_cast<const adam_f32x4 *>(l.grad + idx));
  const adam_f32x4 m4 = __builtin_nontemporal_load(reinterpret_cast<const adam_f32x4 *>(l.mom + idx));
  const adam_f32x4 v4 = __builtin_nontemporal_load(reinterpret_cast<const adam_f32x4 *>(l.vel + idx));
  float a[4] = {a4.x, a4.y, a4.z, a4.w}, g[4] = {g4[0], g4[1], g4[2], g4[3]};
  float mo[4] = {m4[0], m4[1], m4[2], m4[3]}, ve[4] = {v4[0], v4[1], v4[2], v4[3]};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (n0 + e >= l.n) continue;   // padding
    mo[e] = beta1 * mo[e] + (1.f - beta1) * g[e];
    ve[e] = beta2 * ve[e] + (1.f - beta2) * g[e] * g[e];
    const float t = a[e] + lr * (mo[e] * c1) / (sqrtf(ve[e] * c2) + eps);
    a[e] = fminf(fmaxf(t, 0.f), 1.f);
  }
  __builtin_nontemporal_store(adam_f32x4{mo[0], mo[1], mo[2], mo[3]}, reinterpret_cast<adam_f32x4 *>(l.mom + idx));
  __builtin_nontemporal_store(adam_f32x4{ve[0], ve[1], ve[2], ve[3]}, reinterpret_cast<adam_f32x4 *>(l.vel + idx));
  *reinterpret_cast<float4 *>(l.alpha + idx) = make_float4(a[0], a[1], a[2], a[3]);
}

hipError_t launch_alpha_adam(const AlphaLayer &l, const int32_t *flag, int32_t rows, int32_t rows_per_unit, float lr,
                             float beta1, float beta2, float eps, float c1, float c2, hipStream_t s) {
  if (l.ld % 4) return hipErrorInvalidValue;
  const int32_t bpr = (int32_t)((l.ld + ALPHA_COLS_PER_BLOCK - 1) / ALPHA_COLS_PER_BLOCK);
  (void)rows_per_unit;   // the relaxation parameters are not needed (see k_alpha_adam)
  hipLaunchKernelGGL(k_alpha_adam, dim3((unsigned)((int64_t)rows * bpr)), dim3(256), 0, s, l, flag, bpr, lr, beta1,
                     beta2, eps, c1, c2);
  return hipGetLastError();
}

__global__ void k_alpha_final(const float *best_val, int32_t units, int32_t m, const int32_t *unit_flags, float *lb,
                              float *ub) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)units * m) return;
  const int64_t u = idx / m;
  const int64_t q = idx - u * m;
  float l = best_val[u * 2 * m + q], h = -best_val[u * 2 * m + m + q];
  const int32_t f = unit_flags ? unit_flags[u] : 0;
  if (f == 1) {
    l = INFINITY;
    h = -INFINITY;
  } else if (f == 2) {
    l = h = NAN;
  }
  lb[idx] = l;
  ub[idx] = h;
}

hipError_t launch_alpha_final(const float *best_val, int32_t units, int32_t m, const int32_t *unit_flags, float *lb,
                              float *ub, hipStream_t s) {
  const int64_t n = (int64_t)units * m;
  hipLaunchKernelGGL(k_alpha_final, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, best_val, units, m,
                     unit_flags, lb, ub);
  return hipGetLastError();
}

__global__ void k_beta_init(BetaState b, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  b.beta[i] = 0.f;
  b.mom[i] = 0.f;
  b.vel[i] = 0.f;
  b.grad[i] = 0.f;
}

hipError_t launch_beta_init(const BetaState &b, int32_t rows_pad, hipStream_t s) {
  const int64_t n = (int64_t)rows_pad * b.S;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_beta_init, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, b, n);
  return hipGetLastError();
}

__global__ void k_beta_adam(BetaState b, int64_t n, float lr, float beta1, float beta2, float eps, float c1,
                            float c2) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float g = b.grad[i];   // 0 for unused slots (never written)
  const float mo = beta1 * b.mom[i] + (1.f - beta1) * g;
  const float ve = beta2 * b.vel[i] + (1.f - beta2) * g * g;
  b.mom[i] = mo;
  b.vel[i] = ve;
  b.beta[i] = fmaxf(b.beta[i] + lr * (mo * c1) / (sqrtf(ve * c2) + eps), 0.f);
}

hipError_t launch_beta_adam(const BetaState &b, int32_t rows, float lr, float beta1, float beta2, float eps,
                            float c1, float c2, hipStream_t s) {
  const int64_t n = (int64_t)rows * b.S;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_beta_adam, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, b, n, lr, beta1, beta2, eps, c1,
                     c2);
  return hipGetLastError();
}

__global__ void k_alpha_out(AlphaLayer l, int32_t rows, int32_t m, int64_t n_total, float *alpha_out,
                            float *grad_out) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)rows * l.n) return;
  const int64_t row = idx / l.n;
  const int64_t n = idx - row * l.n;
  const int64_t q = row % (2 * m);
  const int64_t src = row * l.ld + n, dst = row * n_total + l.col0 + compact_col(l, n);
  if (alpha_out) alpha_out[dst] = l.best[src];
  if (grad_out) grad_out[dst] = q < m ? l.grad[src] : -l.grad[src];
}

hipError_t launch_alpha_out(const AlphaLayer &l, int32_t rows, int32_t m, int64_t n_total, float *alpha_out,
                            float *grad_out, hipStream_t s) {
  const int64_t n = (int64_t)rows * l.n;
  hipLaunchKernelGGL(k_alpha_out, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, l, rows, m, n_total, alpha_out,
                     grad_out);
  return hipGetLastError();
}

}  // namespace vcr
