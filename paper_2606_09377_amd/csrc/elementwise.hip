// Bandwidth-bound kernels of the CROWN path: the input box, IBP (paper, Sec. 2.1, IBP),
// the ReLU relaxation (Sec. 2.1, CROWN), the first coefficient rows of every backward
// pass, the fixed-order row reductions that finish a bound, and the split table of
// branch-and-bound subdomains.
//
// Relaxation parameters of a ReLU on [l, u] are packed as float4 (lam, s, t, b) (relax.h),
// b being the bias of the dense layer that produces the ReLU's input, which the
// backward pass adds next.  All reductions run in a fixed order (sequential or a fixed
// butterfly), so every bound is reproducible bit for bit and independent of batching.
#include "kernels.h"
#include "relax.h"
#include "../../include/vcrown.h"

namespace vcr {

__device__ __forceinline__ float wave_sum(float x) {
  // fixed butterfly over the 64 lanes of a wavefront
  x += __shfl_xor(x, 32);
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 8);
  x += __shfl_xor(x, 4);
  x += __shfl_xor(x, 2);
  x += __shfl_xor(x, 1);
  return x;
}

// ------------------------------------------------------------------------------------
__global__ void k_fill(float *p, int64_t n, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

hipError_t launch_fill(float *p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

__global__ void k_copy(float *dst, const float *src, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

hipError_t launch_copy(float *dst, const float *src, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_copy, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dst, src, n);
  return hipGetLastError();
}

__global__ void k_store_ptrs(const PtrTable t, int32_t n, const float **dst) {
  const int i = threadIdx.x;
  if (i < n) dst[i] = t.p[i];
}

hipError_t launch_store_ptrs(const PtrTable &t, int32_t n, const float **dst, hipStream_t s) {
  if (n < 0 || n > PTR_TABLE_MAX) return hipErrorInvalidValue;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_store_ptrs, dim3(1), dim3(PTR_TABLE_MAX), 0, s, t, n, dst);
  return hipGetLastError();
}

// Wt[j][i] = W[i][j] for i < rows, j < cols, zero elsewhere; Wt is rows_t x ldt.
// With rows == 0 the same kernel zero-pads a plain copy (see launch_transpose_pad).
__global__ void k_transpose_pad(const float *W, int32_t rows, int32_t cols, float *Wt, int64_t ldt,
                                int64_t rows_t) {
  __shared__ float tile[32][33];
  const int64_t j0 = (int64_t)blockIdx.y * 32;   // Wt row block (W column)
  const int64_t i0 = (int64_t)blockIdx.x * 32;   // Wt column block (W row)
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int k = ty; k < 32; k += 8) {
    const int64_t wi = i0 + k, wj = j0 + tx;
    tile[k][tx] = (wi < rows && wj < cols) ? W[wi * cols + wj] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int64_t tj = j0 + k, ti = i0 + tx;
    if (tj < rows_t && ti < ldt) Wt[tj * ldt + ti] = tile[tx][k];
  }
}

hipError_t launch_transpose_pad(const float *W, int32_t rows, int32_t cols, float *Wt, int64_t ldt,
                                int64_t rows_t, hipStream_t s) {
  dim3 grid((unsigned)((ldt + 31) / 32), (unsigned)((rows_t + 31) / 32));
  hipLaunchKernelGGL(k_transpose_pad, grid, dim3(256), 0, s, W, rows, cols, Wt, ldt, rows_t);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Input box (paper, Sec. 1.1): lo = max(fl(x0 - eps), clip_lo), hi = min(fl(x0 + eps),
// clip_hi), stored as centre c = (lo + hi) / 2 and radius r = (hi - lo) / 2; padding
// columns are zero.
__global__ void k_box(const float *x0, int32_t B, int32_t n0, int64_t ld0, float eps, int32_t clip_on,
                      float clip_lo, float clip_hi, float *c0, float *r0) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * ld0) return;
  const int64_t b = idx / ld0, j = idx - b * ld0;
  float c = 0.f, r = 0.f;
  if (j < n0) {
    const float x = x0[b * n0 + j];
    float lo = __fsub_rn(x, eps), hi = __fadd_rn(x, eps);
    if (clip_on) {
      lo = fmaxf(lo, clip_lo);
      hi = fminf(hi, clip_hi);
    }
    c = __fmul_rn(__fadd_rn(lo, hi), 0.5f);
    r = __fmul_rn(__fsub_rn(hi, lo), 0.5f);
  }
  c0[idx] = c;
  r0[idx] = r;
}

hipError_t launch_box(const float *x0, int32_t B, int32_t n0, int64_t ld0, float eps, int32_t clip_on,
                      float clip_lo, float clip_hi, float *c0, float *r0, hipStream_t s) {
  const int64_t n = (int64_t)B * ld0;
  hipLaunchKernelGGL(k_box, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x0, B, n0, ld0, eps,
                     clip_on, clip_lo, clip_hi, c0, r0);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// IBP through a dense layer in centre/radius form: c' = W c + b, r' = |W| r, which is the
// interval step W+ l + W- u + b, W+ u + W- l + b with l = c - r, u = c + r.  With relu_in
// the input is first passed through ReLU: [max(l, 0), max(u, 0)].
// Both products run on the matrix cores (v_mfma_f32_16x16x4f32, operands straight from global
// memory).  A workgroup owns a block of 16 inputs x 16 outputs, so even one input spreads over
// n_out / 16 compute units; its IBP_KS waves split K into contiguous runs of whole 32-wide K
// tiles (many short runs in flight hide the memory latency), and their partial sums are added
// in wave order through LDS.  The K split depends on n_in only, so an input's bounds do not
// depend on the batch it is in.  Per K tile lane l supplies the 8 consecutive k at 8 (l / 16);
// the loads of the next two tiles are in flight while a tile is multiplied.
typedef float ibp_f32x4 __attribute__((ext_vector_type(4)));
constexpr int IBP_KS = 16;

__global__ __launch_bounds__(64 * IBP_KS) void k_ibp_dense(const float *Wp, int64_t ldw, const float *bias,
                                                           int32_t n_out, int32_t n_in, const float *cin,
                                                           const float *rin, int64_t ld_in, int32_t relu_in,
                                                           float *cout, float *rout, int64_t ld_out, int32_t B) {
  __shared__ float red[IBP_KS][2][4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int o0 = blockIdx.x * 16, b0 = blockIdx.y * 16;
  const int n_kt = (n_in + 31) / 32;
  const int per = (n_kt + IBP_KS - 1) / IBP_KS;
  const int t0 = wave * per, t1 = min(n_kt, t0 + per);
  const bool bval = b0 + r16 < B;
  const float *crow = cin + (int64_t)(bval ? b0 + r16 : 0) * ld_in;
  const float *rrow = rin + (int64_t)(bval ? b0 + r16 : 0) * ld_in;
  // columns past n_out compute on the last real row and are stored as zeros (Wp may hold only
  // n_out rows)
  const float *wrow = Wp + (int64_t)min(o0 + r16, n_out - 1) * ldw;
  ibp_f32x4 accc = {0.f, 0.f, 0.f, 0.f}, accr = {0.f, 0.f, 0.f, 0.f};
  // two K tiles in flight: slot 0 holds the even tiles of the run, slot 1 the odd ones
  float4 nc[2][2], nr[2][2], nw[2][2];
  auto load = [&](int t, float4 (&bc)[2], float4 (&br)[2], float4 (&bw)[2]) {
    const int kb = t * 32 + kg * 8;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      bw[j] = *reinterpret_cast<const float4 *>(wrow + kb + 4 * j);
      bc[j] = bval ? *reinterpret_cast<const float4 *>(crow + kb + 4 * j) : make_float4(0.f, 0.f, 0.f, 0.f);
      br[j] = bval ? *reinterpret_cast<const float4 *>(rrow + kb + 4 * j) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto step = [&](int t, float4 (&bc)[2], float4 (&br)[2], float4 (&bw)[2]) {
    const int kb = t * 32 + kg * 8;
    float c[8], r[8], w[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in = kb + j < n_in;   // past n_in: zero, whatever the padding holds
      const float4 c4 = bc[j / 4], r4 = br[j / 4], w4 = bw[j / 4];
      const float cs = (j & 3) == 0 ? c4.x : (j & 3) == 1 ? c4.y : (j & 3) == 2 ? c4.z : c4.w;
      const float rs = (j & 3) == 0 ? r4.x : (j & 3) == 1 ? r4.y : (j & 3) == 2 ? r4.z : r4.w;
      const float ws = (j & 3) == 0 ? w4.x : (j & 3) == 1 ? w4.y : (j & 3) == 2 ? w4.z : w4.w;
      float cj = in ? cs : 0.f, rj = in ? rs : 0.f;
      if (relu_in) {
        const float lo = fmaxf(cj - rj, 0.f), hi = fmaxf(cj + rj, 0.f);
        cj = (lo + hi) * 0.5f;
        rj = (hi - lo) * 0.5f;
      }
      c[j] = cj;
      r[j] = rj;
      w[j] = in ? ws : 0.f;
    }
    if (t + 2 < t1) load(t + 2, bc, br, bw);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      accc = __builtin_amdgcn_mfma_f32_16x16x4f32(c[j], w[j], accc, 0, 0, 0);
      accr = __builtin_amdgcn_mfma_f32_16x16x4f32(r[j], fabsf(w[j]), accr, 0, 0, 0);
    }
  };
  if (t0 < t1) load(t0, nc[0], nr[0], nw[0]);
  if (t0 + 1 < t1) load(t0 + 1, nc[1], nr[1], nw[1]);
  for (int t = t0; t < t1; t += 2) {
    step(t, nc[0], nr[0], nw[0]);
    if (t + 1 < t1) step(t + 1, nc[1], nr[1], nw[1]);
  }
  if (wave > 0) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      red[wave][0][v][lane] = accc[v];
      red[wave][1][v][lane] = accr[v];
    }
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll 1
  for (int w = 1; w < IBP_KS; ++w)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      accc[v] += red[w][0][v][lane];
      accr[v] += red[w][1][v][lane];
    }
  // entry v of a lane: input b0 + 4 (lane / 16) + v, output o0 + lane % 16
  const int o = o0 + r16;
  const bool real = o < n_out;
  const float bo = real ? bias[o] : 0.f;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int b = b0 + 4 * kg + v;
    if (b >= B) continue;
    cout[(int64_t)b * ld_out + o] = real ? accc[v] + bo : 0.f;
    rout[(int64_t)b * ld_out + o] = real ? accr[v] : 0.f;
  }
}

hipError_t launch_ibp_dense(const float *Wp, int64_t ldw, const float *b, int32_t n_out, int32_t n_in,
                            const float *cin, const float *rin, int64_t ld_in, int32_t relu_in,
                            float *cout, float *rout, int64_t ld_out, int32_t B, hipStream_t s) {
  // whole K tiles are read from every row: both pitches must cover them
  const int64_t k_pad = (int64_t)(n_in + 31) / 32 * 32;
  if (ld_out % 16 || ldw < k_pad || ld_in < k_pad || ldw % 4 || ld_in % 4) return hipErrorInvalidValue;
  dim3 grid((unsigned)(ld_out / 16), (unsigned)((B + 15) / 16));
  hipLaunchKernelGGL(k_ibp_dense, grid, dim3(64 * IBP_KS), 0, s, Wp, ldw, b, n_out, n_in, cin, rin, ld_in,
                     relu_in, cout, rout, ld_out, B);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// First ReLU layer: its pre-activation is one affine map of the input, whose exact range
// over the box is the IBP interval [c - r, c + r].
__global__ void k_layer_from_ibp(const float *c, const float *r, int64_t ld, int32_t n, int32_t B,
                                 const float *bias, float *L, float *U, float4 *P, int64_t ldp, int32_t rule) {
  // one thread per (input, column) of P, padding columns included (they get zeros)
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * ldp) return;
  const int64_t b = idx / ldp, i = idx - b * ldp;
  if (i >= n) {
    P[idx] = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  const float cc = c[b * ld + i], rr = r[b * ld + i];
  const float l = cc - rr, u = cc + rr;
  L[b * n + i] = l;
  U[b * n + i] = u;
  P[idx] = relax_params(l, u, bias[i], rule);
}

hipError_t launch_layer_from_ibp(const float *c, const float *r, int64_t ld, int32_t n, int32_t B,
                                 const float *bias, float *L, float *U, float4 *P, int64_t ldp,
                                 int32_t lam_rule, hipStream_t s) {
  if (ldp < n) return hipErrorInvalidValue;
  const int64_t tot = (int64_t)B * ldp;
  hipLaunchKernelGGL(k_layer_from_ibp, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, c, r, ld, n, B,
                     bias, L, U, P, ldp, lam_rule);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// First rows of a backward pass.  Row (unit u, direction d, i) starts as
// (d ? -1 : 1) * src[i, :] (a weight row W_k[i] or a spec row (C W_L)[i]) with constant
// (d ? -1 : 1) * src_bias[i]; the ReLU just below is relaxed with the lower rule and its
// constants (relaxation intercepts and the bias of the dense layer below) are added; a split
// neuron takes its fixed relaxation from the unit's split entries (the last entry of a column
// wins).  Padding rows are zero.
//
// A write-bound kernel: each wavefront owns IR consecutive rows and walks the columns in
// blocks of 256 NCH.  A lane keeps the relaxation parameters of its 4 NCH columns of the block
// in registers while it writes those columns of all its rows (reloading them only where the
// unit changes), so the parameters are read once per row group instead of once per row.  Each
// lane adds its columns in ascending order (carrying its running sum across column blocks in
// LDS), whatever IR and NCH are, so the row constants have the same bits for every launch shape.
// PLAIN: no split table, no per-row slopes and no copy of the unrelaxed rows (fewer registers).
typedef float nt_f32x4 __attribute__((ext_vector_type(4)));
template <int NCH, int IR, bool PLAIN>
__global__ __launch_bounds__(256) void k_init_rows(const InitArgs a) {
  __shared__ float carry[4][IR][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t row0 = ((int32_t)blockIdx.x * 4 + wave) * IR;
  const int32_t rpu = 2 * a.n_src;
  const bool has_splits = !PLAIN && a.splits.D > 0;
  const float *alpha = PLAIN ? nullptr : a.alpha;
  float *pre = PLAIN ? nullptr : a.pre;
  for (int64_t cb = 0; cb < a.ldo; cb += 256 * NCH) {
    const bool first = cb == 0, last = cb + 256 * NCH >= a.ldo;
    float4 prm[NCH][4];
    int32_t held = -1;
    // the unit's split entries at this ReLU (the unit is wave-uniform), folded into prm when
    // the unit changes; smask marks this lane's split columns of the block (bit 4 j + e)
    int e0 = 0, ne = 0;
    uint32_t smask = 0;
#pragma unroll 1
    for (int r = 0; r < IR; ++r) {
      const int32_t row = row0 + r;
      float *orow = a.out + (int64_t)row * a.ldo + cb + lane * 4;
      float *prow = pre ? pre + (int64_t)row * a.ldo + cb + lane * 4 : nullptr;
      if (row >= a.M) {
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          if (cb + j * 256 + lane * 4 >= a.ldo) continue;
          *reinterpret_cast<float4 *>(orow + j * 256) = make_float4(0.f, 0.f, 0.f, 0.f);
          if (prow) *reinterpret_cast<float4 *>(prow + j * 256) = make_float4(0.f, 0.f, 0.f, 0.f);
        }
        if (last && lane == 0) a.beta[row] = 0.f;
        continue;
      }
      const int32_t u = row / rpu;
      const int32_t r2 = row - u * rpu;
      const int dir = r2 >= a.n_src;
      const int32_t i = r2 - dir * a.n_src;
      const float sgn = dir ? -1.f : 1.f;
      const int64_t srow = a.per_unit_src ? (int64_t)u * a.n_src + i : i;
      const int32_t pu = a.param_per_unit ? u : 0;
      const int32_t key = has_splits ? u : pu;   // split units carry their own overrides
      if (key != held) {
        const float4 *P = a.P + (int64_t)pu * a.ldp + cb + lane * 4;
#pragma unroll
        for (int j = 0; j < NCH; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            prm[j][e] = cb + j * 256 + lane * 4 < a.ldo ? P[j * 256 + e] : make_float4(0.f, 0.f, 0.f, 0.f);
        if (has_splits) {
          smask = 0;
          e0 = a.splits.off[u * (a.splits.R + 1) + a.relu_index];
          ne = a.splits.off[u * (a.splits.R + 1) + a.relu_index + 1] - e0;
          for (int k = 0; k < ne; ++k) {   // in order: the last entry of a column wins
            const int64_t o = a.splits.ent_n[u * a.splits.S + e0 + k] - (cb + lane * 4);
            if (o < 0 || o >= 256 * NCH || (o & 255) >= 4) continue;   // not this lane's column
            const float4 ov = a.splits.ent_p[u * a.splits.S + e0 + k];
            const int jo = (int)(o >> 8), eo = (int)(o & 3);
#pragma unroll
            for (int j = 0; j < NCH; ++j)
#pragma unroll
              for (int e = 0; e < 4; ++e)
                if (j == jo && e == eo) {
                  prm[j][e].x = ov.x;
                  prm[j][e].y = ov.y;
                  prm[j][e].z = ov.z;
                }
            smask |= 1u << (4 * jo + eo);
          }
        }
        held = key;
      }
      const float *src = a.src + srow * a.ld_src + cb + lane * 4;
      float4 w[NCH];
#pragma unroll
      for (int j = 0; j < NCH; ++j)
        w[j] = cb + j * 256 + lane * 4 < a.ldo ? *reinterpret_cast<const float4 *>(src + j * 256)
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
      float acc = first ? 0.f : carry[wave][r][lane];
#pragma unroll
      for (int j = 0; j < NCH; ++j) {
        const int64_t c = cb + j * 256 + lane * 4;
        if (c >= a.ldo) continue;
        const float wv[4] = {w[j].x, w[j].y, w[j].z, w[j].w};
        float4 al4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (alpha) al4 = *reinterpret_cast<const float4 *>(alpha + (int64_t)row * a.ld_alpha + c);
        const float alv[4] = {al4.x, al4.y, al4.z, al4.w};
        float ov[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float4 q = prm[j][e];
          int ent = -1;
          float sterm = 0.f;
          if (has_splits && a.splits.beta && ((smask >> (4 * j + e)) & 1u)) {
            // a split column (rare): its entry for the beta term, the last match as above
            for (int k = 0; k < ne; ++k)
              if (a.splits.ent_n[u * a.splits.S + e0 + k] == (int)(c + e)) {
                ent = e0 + k;
                sterm = a.splits.ent_p[u * a.splits.S + e0 + k].w;
              }
          }
          const float x = sgn * wv[e];
          float lam = q.x;
          if (alpha && q.z > 0.f) lam = alv[e];
          float ap = x > 0.f ? x * lam : x * q.y;
          if (ent >= 0 && a.splits.beta) ap += a.splits.beta[(int64_t)row * a.splits.S + ent] * sterm;
          acc += fminf(x, 0.f) * q.z + ap * q.w;
          ov[e] = ap;
        }
        // streaming stores: the rows are read back only by the next GEMM, long after
        __builtin_nontemporal_store(nt_f32x4{ov[0], ov[1], ov[2], ov[3]},
                                    reinterpret_cast<nt_f32x4 *>(orow + j * 256));
        if (prow)
          __builtin_nontemporal_store(nt_f32x4{sgn * wv[0], sgn * wv[1], sgn * wv[2], sgn * wv[3]},
                                      reinterpret_cast<nt_f32x4 *>(prow + j * 256));
      }
      if (!last) {
        carry[wave][r][lane] = acc;  // each lane only ever touches its own slot
        continue;
      }
      acc = wave_sum(acc);
      if (lane == 0) a.beta[row] = sgn * a.src_bias[srow] + acc;
    }
  }
}

template <int NCH, int IR>
static void launch_init_rows_t(const InitArgs &a, int32_t M_pad, hipStream_t s) {
  const dim3 grid((unsigned)(M_pad / (4 * IR)));
  if (a.splits.D == 0 && !a.alpha && !a.pre)
    hipLaunchKernelGGL((k_init_rows<NCH, IR, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_init_rows<NCH, IR, false>), grid, dim3(256), 0, s, a);
}

template <int NCH>
static void launch_init_rows_n(const InitArgs &a, int32_t M_pad, hipStream_t s) {
  if (M_pad >= 32768)
    launch_init_rows_t<NCH, 16>(a, M_pad, s);
  else if (M_pad >= 4096)
    launch_init_rows_t<NCH, 4>(a, M_pad, s);
  else
    launch_init_rows_t<NCH, 1>(a, M_pad, s);
}

hipError_t launch_init_rows(const InitArgs &a, hipStream_t s) {
  if (a.ldo % 4) return hipErrorInvalidValue;
  const int32_t M_pad = (int32_t)rows_pad(a.M);  // a multiple of 128: every row group is whole
  if (a.ldo <= 256)
    launch_init_rows_n<1>(a, M_pad, s);
  else if (a.ldo <= 512)
    launch_init_rows_n<2>(a, M_pad, s);
  else
    launch_init_rows_n<4>(a, M_pad, s);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// beta[row] += sum_p part[p][row], p ascending.
__global__ void k_rowsum(float *beta, const float *part, int32_t n_parts, int32_t M_pad, int32_t M) {
  const int64_t row = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (row >= M) return;
  float s = 0.f;
  for (int p = 0; p < n_parts; ++p) s += part[(int64_t)p * M_pad + row];
  beta[row] += s;
}

hipError_t launch_rowsum(float *beta, const float *part, int32_t n_parts, int32_t M_pad, int32_t M,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_rowsum, dim3((unsigned)((M + 255) / 256)), dim3(256), 0, s, beta, part, n_parts, M_pad, M);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Bounds of one ReLU layer's pre-activations from the finished backward pass: lower rows
// (b, 0, i) give l, negated upper rows (b, 1, i) give -u; then intersection with IBP and
// the relaxation for the passes above.
__global__ void k_finalize_layer(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad,
                                 int32_t B, int32_t n, const float *ibp_c, const float *ibp_r, int64_t ld_ibp,
                                 int32_t intersect, const float *bias_next, float *L, float *U, float4 *P,
                                 int64_t ldp, int32_t rule) {
  // one thread per (input, column) of P, padding columns included (they get zeros)
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)B * ldp) return;
  const int64_t b = idx / ldp, i = idx - b * ldp;
  if (i >= n) {
    P[idx] = make_float4(0.f, 0.f, 0.f, 0.f);
    return;
  }
  const int64_t ml = b * 2 * n + i, mu = ml + n;
  float sl = 0.f, su = 0.f;
  for (int p = 0; p < n_parts; ++p) {
    sl += cpart[(int64_t)p * M_pad + ml];
    su += cpart[(int64_t)p * M_pad + mu];
  }
  float l = beta[ml] + sl;
  float u = -(beta[mu] + su);
  if (intersect) {
    const float c = ibp_c[b * ld_ibp + i], r = ibp_r[b * ld_ibp + i];
    l = fmaxf(l, c - r);
    u = fminf(u, c + r);
  }
  L[b * n + i] = l;
  U[b * n + i] = u;
  P[idx] = relax_params(l, u, bias_next[i], rule);
}

hipError_t launch_finalize_layer(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad,
                                 int32_t B, int32_t n, const float *ibp_c, const float *ibp_r,
                                 int64_t ld_ibp, int32_t intersect, const float *bias_next,
                                 float *L, float *U, float4 *P, int64_t ldp, int32_t lam_rule, hipStream_t s) {
  if (ldp < n) return hipErrorInvalidValue;
  const int64_t tot = (int64_t)B * ldp;
  hipLaunchKernelGGL(k_finalize_layer, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, beta, cpart,
                     n_parts, M_pad, B, n, ibp_c, ibp_r, ld_ibp, intersect, bias_next, L, U, P, ldp, lam_rule);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Spec rows folded into the last dense layer: CW[b, i, :] = C[b, i, :] W_L and
// Cb[b, i] = C[b, i, :] b_L (sequential over the output neurons).
__global__ void k_spec_cw(const float *C, int32_t B, int32_t m, int32_t n_out, const float *Wp, int64_t ldw,
                          const float *bias, int32_t n_in, float *CW, int64_t ld_cw, float *Cb) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t rows = (int64_t)B * m;
  if (idx >= rows * ld_cw) return;
  const int64_t row = idx / ld_cw, n = idx - row * ld_cw;
  const float *c = C + row * n_out;
  float s = 0.f;
  if (n < n_in)
    for (int o = 0; o < n_out; ++o) s += c[o] * Wp[(int64_t)o * ldw + n];
  CW[idx] = s;
  if (n == 0) {
    float sb = 0.f;
    for (int o = 0; o < n_out; ++o) sb += c[o] * bias[o];
    Cb[row] = sb;
  }
}

hipError_t launch_spec_cw(const float *C, int32_t B, int32_t m, int32_t n_out, const float *Wp,
                          int64_t ldw, const float *b, int32_t n_in, float *CW, int64_t ld_cw,
                          float *Cb, hipStream_t s) {
  const int64_t tot = (int64_t)B * m * ld_cw;
  hipLaunchKernelGGL(k_spec_cw, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, C, B, m, n_out, Wp, ldw,
                     b, n_in, CW, ld_cw, Cb);
  return hipGetLastError();
}

// lb = CW . c - |CW| . r + Cb, ub = CW . c + |CW| . r + Cb over an input interval given as
// centre/radius (optionally passed through ReLU first).  One wavefront per spec row.
__global__ __launch_bounds__(256) void k_spec_direct(const float *CW, int64_t ld_cw, const float *Cb, int32_t B,
                                                     int32_t m, int32_t n_in, const float *c, const float *r,
                                                     int64_t ld_in, int32_t relu_in, float *lb, float *ub) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= (int64_t)B * m) return;
  const int64_t b = row / m;
  float dc = 0.f, dr = 0.f;
  for (int64_t k = lane; k < n_in; k += 64) {
    const float w = CW[row * ld_cw + k];
    float cc = c[b * ld_in + k], rr = r[b * ld_in + k];
    if (relu_in) {
      const float lo = fmaxf(cc - rr, 0.f), hi = fmaxf(cc + rr, 0.f);
      cc = (lo + hi) * 0.5f;
      rr = (hi - lo) * 0.5f;
    }
    dc += w * cc;
    dr += fabsf(w) * rr;
  }
  dc = wave_sum(dc);
  dr = wave_sum(dr);
  if (lane == 0) {
    lb[row] = dc - dr + Cb[row];
    ub[row] = dc + dr + Cb[row];
  }
}

hipError_t launch_spec_direct(const float *CW, int64_t ld_cw, const float *Cb, int32_t B, int32_t m,
                              int32_t n_in, const float *c, const float *r, int64_t ld_in,
                              int32_t relu_in, float *lb, float *ub, hipStream_t s) {
  const int64_t rows = (int64_t)B * m;
  hipLaunchKernelGGL(k_spec_direct, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, CW, ld_cw, Cb, B, m,
                     n_in, c, r, ld_in, relu_in, lb, ub);
  return hipGetLastError();
}

// Final bounds per spec row: lb = beta + sum of concretization partials of the lower row,
// ub = -(same for the negated row).  Infeasible units give (+inf, -inf), invalid ones NaN.
__global__ void k_finalize_spec(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad,
                                int32_t units, int32_t m, const int32_t *flags, float *lb, float *ub) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)units * m) return;
  const int64_t u = idx / m, i = idx - u * m;
  const int64_t ml = u * 2 * m + i, mu = ml + m;
  float sl = 0.f, su = 0.f;
  for (int p = 0; p < n_parts; ++p) {
    sl += cpart[(int64_t)p * M_pad + ml];
    su += cpart[(int64_t)p * M_pad + mu];
  }
  float l = beta[ml] + sl;
  float h = -(beta[mu] + su);
  const int f = flags ? flags[u] : 0;
  if (f == 1) {
    l = __int_as_float(0x7f800000);
    h = -l;
  } else if (f == 2) {
    l = __int_as_float(0x7fc00000);
    h = l;
  }
  lb[idx] = l;
  ub[idx] = h;
}

hipError_t launch_finalize_spec(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad,
                                int32_t units, int32_t m, const int32_t *unit_flags, float *lb,
                                float *ub, hipStream_t s) {
  const int64_t tot = (int64_t)units * m;
  hipLaunchKernelGGL(k_finalize_spec, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, beta, cpart,
                     n_parts, M_pad, units, m, unit_flags, lb, ub);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Split table of branch-and-bound subdomains (paper, Sec. 2.1, complete verification).
// One thread per domain validates its entries, clamps each split neuron's root interval
// (active: l <- max(l, 0); inactive: u <- min(u, 0)), marks the domain infeasible if an
// interval becomes empty, and stores the entries sorted by ReLU with their relaxation.
constexpr int MAX_SPLITS = VCR_MAX_SPLITS;   // split slots per subdomain (the ABI limit)

__global__ void k_split_prepare(const SplitPrepArgs a) {
  const int d = blockIdx.x * blockDim.x + threadIdx.x;
  if (d >= a.D) return;
  int er[MAX_SPLITS], en[MAX_SPLITS], es[MAX_SPLITS];
  bool invalid = a.S > MAX_SPLITS;
  int cnt = 0;
  for (int k = 0; k < a.S && !invalid; ++k) {
    const int r = a.relu_id[(int64_t)d * a.S + k];
    const int j = a.neuron[(int64_t)d * a.S + k];
    const int sg = a.sign[(int64_t)d * a.S + k];
    if (r == -1) continue;   // an unused slot
    if (r < 0 || r >= a.R || (sg != 1 && sg != -1)) {
      invalid = true;
      break;
    }
    if (j < 0 || j >= a.relu_n[r]) {
      invalid = true;
      break;
    }
    for (int e = 0; e < cnt; ++e)
      if (er[e] == r && en[e] == j) invalid = true;
    // insertion keeps entries sorted by ReLU (stable)
    int pos = cnt;
    while (pos > 0 && er[pos - 1] > r) {
      er[pos] = er[pos - 1];
      en[pos] = en[pos - 1];
      es[pos] = es[pos - 1];
      --pos;
    }
    er[pos] = r;
    en[pos] = j;
    es[pos] = sg;
    ++cnt;
  }
  int32_t *off = a.off + (int64_t)d * (a.R + 1);
  if (invalid) {
    for (int r = 0; r <= a.R; ++r) off[r] = 0;
    a.flags[d] = 2;
    atomicAdd(a.n_invalid, 1);
    return;
  }
  bool infeasible = false;
  int e = 0;
  for (int r = 0; r <= a.R; ++r) {
    while (e < cnt && er[e] < r) ++e;
    off[r] = e;
  }
  for (int k = 0; k < cnt; ++k) {
    float l = a.L[er[k]][en[k]], u = a.U[er[k]][en[k]];
    if (es[k] > 0)
      l = fmaxf(l, 0.f);
    else
      u = fminf(u, 0.f);
    if (l > u) infeasible = true;
    int jn = en[k];
    if (a.hwc_C && a.hwc_C[er[k]] > 0) {   // (c, y, x) -> (y, x, c)
      const int C = a.hwc_C[er[k]], HW = a.relu_n[er[k]] / C;
      jn = (jn % HW) * C + jn / HW;
    }
    a.ent_n[(int64_t)d * a.S + k] = jn;
    float4 q = relax_params(l, u, 0.f, a.lam_rule);
    q.w = es[k] > 0 ? -1.f : 1.f;   // sign of the split's Lagrangian term
    a.ent_p[(int64_t)d * a.S + k] = q;
  }
  for (int k = cnt; k < a.S; ++k) {   // unused slots (never matched: off[] ends at cnt)
    a.ent_n[(int64_t)d * a.S + k] = -1;
    a.ent_p[(int64_t)d * a.S + k] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  a.flags[d] = infeasible ? 1 : 0;
}

hipError_t launch_split_prepare(const SplitPrepArgs &a, hipStream_t s) {
  if (a.D <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_split_prepare, dim3((unsigned)((a.D + 63) / 64)), dim3(64), 0, s, a);
  return hipGetLastError();
}

// Number of unstable neurons (l < 0 < u) in n entries.
__global__ void k_count_unstable(const float *L, const float *U, int64_t n, int32_t *count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int v = (i < n && L[i] < 0.f && U[i] > 0.f) ? 1 : 0;
  v += __shfl_xor(v, 32);
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 8);
  v += __shfl_xor(v, 4);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 1);
  if ((threadIdx.x & 63) == 0 && v) atomicAdd(count, v);
}

hipError_t launch_count_unstable(const float *L, const float *U, int64_t n, int32_t *count, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_count_unstable, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, L, U, n, count);
  return hipGetLastError();
}

// Non-finite values (NaN, +-inf) among n floats, added to *count (the VCR_OPT_CHECK_FINITE
// scan of a call's inputs).  One atomic per workgroup that found any.
__global__ void k_count_nonfinite(const float *p, int64_t n, int32_t *count) {
  __shared__ int32_t blk;
  if (threadIdx.x == 0) blk = 0;
  __syncthreads();
  int32_t mine = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    mine += isfinite(p[i]) ? 0 : 1;
  if (mine) atomicAdd(&blk, mine);
  __syncthreads();
  if (threadIdx.x == 0 && blk) atomicAdd(count, blk);
}

hipError_t launch_count_nonfinite(const float *p, int64_t n, int32_t *count, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(k_count_nonfinite, dim3((unsigned)blocks), dim3(256), 0, s, p, n, count);
  return hipGetLastError();
}

}  // namespace vcr
