// CROWN backward through convolutions (paper, Sec. 4.8 extends bound propagation to
// BoundConv; the step is the transpose of the convolution applied to every coefficient
// row), residual additions and flatten, on windowed coefficient rows.
//
// Coefficient rows of a convolutional node are stored channels-last, one square window per
// row: A[r][u][w][c], u, w in [0, S), c in [0, C).  A row that starts at one neuron (c0, i, j)
// of a 3x3 convolution output is nonzero only inside that neuron's receptive field, so the
// window has half-size h around the row's anchor (i, j) (scaled to the node's resolution)
// and grows by one per stride-1 3x3 convolution (2h + 1 through stride 2).  Rows of a
// dense node (spec rows, fully connected neurons) use the whole image: origin 0, S = H.
// Window positions outside the image are the convolution's zero padding: the transposed
// convolution computes and writes only the positions inside the image, and every reader of a
// window (the next transposed convolution, the stem, the constant terms) takes the positions
// outside it as zero without reading them.
//
// The transposed convolution of one row is an implicit GEMM:
//   out[(r, u, w), ci] = sum_{tap=(ky,kx), co} A_out[r][u'][w'][co] * W[co][ci][ky][kx]
//   u' = (u + delta - ky) / stride (only when divisible and inside the source window)
// with M = rows x S_in^2 (windowed rows: the positions inside the image), N = C_in,
// K = 9 C_out, run per class of output positions (the positions that the same taps reach:
// stride parity and the window's border ring) over that class's taps only.  The weights are repacked at load time as
// Bt[ci][tap * C_out + co] (K-contiguous).  The epilogue applies, per output element at
// global position (gy, gx):
//   outside the image          -> 0
//   + residual (same node, smaller window aligned on the same anchor)
//   relaxation (lam, s, t, b)  -> a' and the constant terms min(a,0) t + a' b, where the
//                                 parameters are the ReLU's at (unit, gy, gx, ci), or the
//                                 identity (1, 1, 0, b[ci]) when the node is not a ReLU
// and reduces the constants over the tile's columns into one partial per GEMM row.
#include "conv.h"
#include "relax.h"
#include "lds_dma.h"
#include "row_sums.h"
#include "splits.h"

#include <algorithm>
#include <vector>

namespace vcr {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv d) {
  // floor(n / d) for n < 2^31 with the precomputed magic of FastDiv
  const uint64_t t = (uint64_t)__umulhi(n, d.mul) + n;
  return (uint32_t)(t >> d.shift);
}

// floor(a / b) for b > 0 and any sign of a
__host__ __device__ inline int floor_div(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

// Class positions i in [0, n) of one axis whose image coordinate o + u0 + ustep i lies in
// [0, H): the interval [*lo, *hi) (empty: *lo == *hi)
__host__ __device__ inline void clip_range(int o, int u0, int ustep, int n, int H, int *lo, int *hi) {
  const int l = min(max(-floor_div(o + u0, ustep), 0), n);
  const int h = min(max(floor_div(H - 1 - o - u0, ustep) + 1, 0), n);
  *lo = l;
  *hi = max(h, l);
}

// Tables of a clipped class, per anchor a < Ha: tab[0][a] = first inside position of the
// y axis, tab[1][a] = inside y positions of the anchors before a (tab[1][Ha]: all of them),
// tab[2], tab[3] the same for x.  Built by one wave (lane a), an inclusive scan across lanes.
typedef int ClipTab[4][CONVT_CLIP_MAX + 1];
__device__ __forceinline__ void clip_tables(const ConvTArgs &p, const ConvClass &cl, ClipTab &tab, int lane) {
#pragma unroll
  for (int ax = 0; ax < 2; ++ax) {
    int lo = 0, hi = 0;
    if (lane < p.Ha)
      clip_range(lane * p.scale - p.h_in, ax ? cl.w0 : cl.u0, ax ? cl.wstep : cl.ustep, ax ? cl.nx : cl.ny, p.H_in,
                 &lo, &hi);
    int x = hi - lo;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o);
      if (lane >= o) x += y;
    }
    if (lane < p.Ha) {
      tab[2 * ax][lane] = lo;
      tab[2 * ax + 1][lane + 1] = x;
    }
    if (lane == 0) tab[2 * ax + 1][0] = 0;
  }
}

// GEMM row m < cl.M of a class -> coefficient row r, class position (iy, ix) and, for
// windowed rows (Ha > 0), the row's anchor index a_y Ha + a_x
__device__ __forceinline__ void convt_row(const ConvTArgs &p, const ConvClass &cl, const ClipTab &tab, uint32_t m,
                                          uint32_t *r, int *iy, int *ix, int *anc) {
  if (cl.clip) {
    const int Wx = tab[3][p.Ha];
    const uint32_t cyc = fdiv(m, cl.div_yx);   // cycles of Ha^2 rows
    int rem = (int)(m - cyc * (uint32_t)(tab[1][p.Ha] * Wx));
    int ay = 0, ax = 0;
#pragma unroll
    for (int b = CONVT_CLIP_MAX / 2; b > 0; b >>= 1)   // last anchor with prefix * Wx <= rem
      if (ay + b < p.Ha && tab[1][ay + b] * Wx <= rem) ay += b;
    rem -= tab[1][ay] * Wx;
    const int wy = tab[1][ay + 1] - tab[1][ay];
#pragma unroll
    for (int b = CONVT_CLIP_MAX / 2; b > 0; b >>= 1)
      if (ax + b < p.Ha && wy * tab[3][ax + b] <= rem) ax += b;
    rem -= wy * tab[3][ax];
    const int wx = tab[3][ax + 1] - tab[3][ax];   // > 0: ax is the last anchor below rem
    const int ky = rem / wx;
    *anc = ay * p.Ha + ax;
    *r = cyc * (uint32_t)(p.Ha * p.Ha) + (uint32_t)*anc;
    *iy = tab[0][ay] + ky;
    *ix = tab[2][ax] + rem - ky * wx;
  } else {
    const uint32_t rr = fdiv(m, cl.div_yx);
    const uint32_t pos = m - rr * (uint32_t)(cl.ny * cl.nx);
    const uint32_t y = fdiv(pos, cl.div_x);
    *r = rr;
    *iy = (int)y;
    *ix = (int)(pos - y * (uint32_t)cl.nx);
    *anc = p.Ha > 0 ? (int)(rr % (uint32_t)(p.Ha * p.Ha)) : 0;
  }
}

// Tile shapes: BM x BN outputs per workgroup of 4 wave64 arranged WM x WN, each wave
// owning (BM / WM) x (BN / WN) as 32 x 32 MFMA blocks; BK-deep K tiles through
// double-buffered LDS (rows unpadded, chunks swizzled by lds_swz).  A K tile never straddles
// two taps (C_out is a multiple of 32).

// Source of the zeros that taps outside the source window load
__device__ __attribute__((aligned(16))) float g_zero4[4] = {0.f, 0.f, 0.f, 0.f};   // never written

// LDS stages of the transposed convolution's operand tiles (three cost a workgroup per
// compute unit on the 256 x 64 tiles and measured 9% slower)
constexpr int CONVT_NS = 2;



// Epilogue shared by the transposed-convolution kernels: relaxation (or identity), residual,
// constant terms per GEMM row for the tile m0.. of class cl, columns n0..; acc holds the
// MB x NB 32 x 32 MFMA blocks of wave (wm, wn); scratch is >= 24 BM bytes of free LDS.
template <int BM, int BN, int WM, int WN, bool RELU, bool AL, bool SPL>
__device__ __forceinline__ void convt_epilogue(const ConvTArgs &p, const ConvClass &cl, const ClipTab &tab,
                                               const f32x16 (&acc)[BM / WM / 32][BN / WN / 32], int m0, int n0,
                                               int nt, float *scratch) {
  constexpr int MB = BM / WM / 32, NB = BN / WN / 32;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN, r32 = lane & 31;
  // Row information of the tile's BM GEMM rows is computed once, a row per thread, into
  // LDS (the operand buffers are free after the main loop's last barrier).  A lane holds 16
  // rows of each 32 x 32 block as 4 groups of 4 consecutive rows; the relaxation parameters
  // and residual terms of the next group are loaded while the current group is relaxed and
  // stored, so the epilogue waits on global memory about once instead of once per group.
  static_assert(BM % 256 == 0 || BM < 256, "rows are spread over the 256 threads");
  int64_t *s_ob = reinterpret_cast<int64_t *>(scratch);      // output offset
  int64_t *s_rb = s_ob + BM;                                 // residual offset, or -1
  int *s_pb = reinterpret_cast<int *>(s_rb + BM);            // parameter offset, -1 outside the image
  int *s_mo = s_pb + BM;                                     // partial-sum index, -1 past M
  int *s_rr = s_mo + BM;                                     // coefficient row (split lookups)
  const int S_in2 = p.S_in * p.S_in;
  const float4 *__restrict__ Pp = p.P_pos;
  const float *__restrict__ resp = p.res;
  float *__restrict__ outp = p.out;
  const float *__restrict__ alp = p.alpha;
  float *__restrict__ prep = p.pre;
  for (int tr = tid; tr < BM; tr += 256) {
    const int m = m0 + tr;
    const bool valid = m < cl.M;
    uint32_t r = 0;
    int iy = 0, ix = 0, anc = 0;
    if (valid) convt_row(p, cl, tab, (uint32_t)m, &r, &iy, &ix, &anc);
    const int u = cl.u0 + iy * cl.ustep;
    const int w = cl.w0 + ix * cl.wstep;
    const int4 an = p.rows[r];   // (unit, anchor y, anchor x, -)
    const int gy = p.dense ? u : an.y * p.scale - p.h_in + u;
    const int gx = p.dense ? w : an.z * p.scale - p.h_in + w;
    const bool inside = valid && gy >= 0 && gx >= 0 && gy < p.H_in && gx < p.H_in;
    const int du = u - p.res_off, dw = w - p.res_off;
    s_mo[tr] = valid ? (int)r * S_in2 + u * p.S_in + w : -1;
    s_rr[tr] = (int)r;
    s_ob[tr] = (int64_t)r * p.row_stride_in + ((int64_t)u * p.S_in + w) * p.C_in;
    s_pb[tr] = inside ? ((an.x * p.H_in + gy) * p.H_in + gx) * p.C_in : -1;
    s_rb[tr] = inside && resp && du >= 0 && dw >= 0 && du < p.res_S && dw < p.res_S
                    ? (int64_t)r * p.res_row_stride + ((int64_t)du * p.res_S + dw) * p.C_in
                    : -1;
  }
  __syncthreads();

  const int half = lane >> 5;
  const int lrow0 = wm * (BM / WM) + half * 4;   // + 32 i + 8 g + t
  int ncol[NB];
  float bn[NB];   // no ReLU at this node: identity, constant term a b[n]
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    ncol[j] = n0 + wn * (BN / WN) + j * 32 + r32;
    bn[j] = (!RELU && ncol[j] < p.C_in) ? p.bias[ncol[j]] : 0.f;
  }
  // A ReLU step's relaxation parameters of group q = 4 i + g go into buffer b, one group
  // ahead of their use.  Lanes with nothing to load (outside the image, past C_in) read
  // element 0, a finite parameter that meets a zero coefficient: no select on a loaded value,
  // 32-bit offsets from one base.  An identity step (the only kind with a residual) loads its
  // residual terms instead, RD groups ahead into a ring of RD + 1 buffers (8 floats each).
  constexpr int NG = MB * 4;
  float4 prm[2][NB][4];
  constexpr int RD = 3;
  float rvb[RD + 1][NB][4];
  auto fetch = [&](int q, int b) {
    const int lr = lrow0 + (q >> 2) * 32 + (q & 3) * 8;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if constexpr (RELU) {
        const int pb = s_pb[lr + t];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const uint32_t off = (ncol[j] < p.C_in && pb >= 0) ? (uint32_t)(pb + ncol[j]) : 0u;
          prm[b][j][t] = Pp[off];
        }
      } else {
        const int64_t rb = s_rb[lr + t];
#pragma unroll
        for (int j = 0; j < NB; ++j)
          rvb[b % (RD + 1)][j][t] = resp ? *((ncol[j] < p.C_in && rb >= 0) ? resp + rb + ncol[j] : g_zero4) : 0.f;
      }
    }
  };
  fetch(0, 0);
  if constexpr (!RELU) {
#pragma unroll
    for (int q = 1; q < RD && q < NG; ++q) fetch(q, q);
  }
  float rp[16];
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    const int i = q >> 2, g = q & 3, b = q & 1;
    const int lr = lrow0 + i * 32 + g * 8;
    float rv[NB][4];   // residual terms of this group
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        if constexpr (RELU) {   // (a ReLU step has no residual: resp is null)
          const int64_t rb = s_rb[lr + t];
          rv[j][t] = resp ? *((ncol[j] < p.C_in && rb >= 0) ? resp + rb + ncol[j] : g_zero4) : 0.f;
        } else {
          rv[j][t] = rvb[q % (RD + 1)][j][t];
        }
      }
    }
    if constexpr (RELU) {
      if (q + 1 < NG) fetch(q + 1, b ^ 1);
    } else {
      if (q + RD < NG) fetch(q + RD, q + RD);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int pb = s_pb[lr + t], mo = s_mo[lr + t];
      const int64_t ob = s_ob[lr + t];
      float x = 0.f;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const float a = acc[i][j][g * 4 + t] + rv[j][t];
        const bool store = mo >= 0 && ncol[j] < p.C_in;
        float ap = 0.f;
        if (pb >= 0) {   // inside the image: relax (or identity) and constant terms
          if constexpr (RELU) {
            float4 q = prm[b][j][t];
            int ent = -1;
            float sterm = 0.f;
            if constexpr (SPL) {   // subdomains: a split neuron's clamped relaxation
              if (store) q = split_override(p.splits, s_rr[lr + t], p.relu_index, pb + ncol[j], q, &ent, &sterm);
            }
            float lam = q.x;
            if constexpr (AL) {   // alpha-CROWN: the row's own slope at unstable neurons, whose
                                  // coefficients before relaxation are recorded (the gradient
                                  // pass reads them there only)
              if (store && q.z > 0.f) {
                lam = alp[ob + ncol[j]];
                prep[ob + ncol[j]] = a;
              }
            }
            ap = a > 0.f ? a * lam : a * q.y;
            if constexpr (SPL) {   // beta-CROWN: the split's multiplier term
              if (ent >= 0 && p.splits.beta) ap += p.splits.beta[(int64_t)s_rr[lr + t] * p.splits.S + ent] * sterm;
            }
            x += fminf(a, 0.f) * q.z + ap * q.w;
          } else {
            ap = a;
            x += a * bn[j];
          }
        }
        // non-temporal: the next step streams these coefficients back from HBM anyway (GBs
        // per step), and caching them evicts the source rows this kernel's gathers re-read
        if (store) __builtin_nontemporal_store(ap, outp + ob + ncol[j]);
      }
      rp[g * 4 + t] = x;
    }
    if (g == 3) {   // the lane's 16 rows of block i: reduce over the 32 columns, one partial each
      const float x = half_wave_row_sums(rp, r32);
      if ((r32 & 1) == 0) {   // lane 2 v stores row v
        const int v = r32 >> 1;
        const int mo = s_mo[lrow0 + i * 32 + (v >> 2) * 8 + (v & 3)];
        if (mo >= 0) p.part[(int64_t)(nt * WN + wn) * p.M_pad + mo] = x;
      }
    }
  }
}

// RELU: the destination node feeds a ReLU (relaxation parameters P_pos), else the identity
// with a per-channel constant (bias).  AL (with RELU, dense windows): alpha-CROWN's per-row
// slopes and the record of the coefficients before relaxation.
template <int BM, int BN, int BK, int WM, int WN, int MINB, bool RELU, bool AL = false, bool SPL = false>
__global__ __launch_bounds__(256, MINB) void k_convt(const ConvTArgs p) {
  static_assert(BK == 16 || BK == 32, "LDS swizzle assumes 4 or 8 chunks per row");
  static_assert(BN / WN == 64, "a wave's constant-term partial covers 64 columns (N_pad / 64 partials)");
  constexpr int CPR = BK / 4;                 // 16-byte chunks per tile row
  constexpr int MB = BM / WM / 32, NB = BN / WN / 32;
  constexpr int TPR = CPR;                    // threads per tile row (one chunk each)
  constexpr int RPP = 256 / TPR;              // tile rows per load pass
  constexpr int QA = BM / RPP, QB = BN / RPP;
  __shared__ __attribute__((aligned(16))) float As[CONVT_NS][BM * BK];
  __shared__ __attribute__((aligned(16))) float Bs[CONVT_NS][BN * BK];
  __shared__ ClipTab tab;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  // parity class of this workgroup (wave-uniform selects, no indexed argument access)
  const int bid = blockIdx.x;
  const int c = (bid >= p.cls[1].blk0) + (bid >= p.cls[2].blk0) + (bid >= p.cls[3].blk0);
  const ConvClass cl = c == 0 ? p.cls[0] : c == 1 ? p.cls[1] : c == 2 ? p.cls[2] : p.cls[3];
  const int n_nt = p.N_pad / BN;
  const int lb = bid - cl.blk0;
  const int mt = lb / n_nt, nt = lb - mt * n_nt;
  const int m0 = mt * BM, n0 = nt * BN;
  const int sh = p.stride == 2 ? 1 : 0;
  if (cl.clip) {   // workgroup-uniform
    if (wave == 0) clip_tables(p, cl, tab, lane);
    __syncthreads();
  }

  // Per tile row: its source row pointer and its class position (iy, ix).  Tap (ty, tx) of
  // the class reads source position (iy + dy, ix + dx) with a wave-uniform shift (dy, dx);
  // of a windowed source only the positions inside the image, [ylo, ylo + yl) x [xlo, xlo +
  // xl) of the window, are read (the pointer and coordinates are taken relative to ylo, xlo).
  // The operand tiles go from global memory straight into LDS (global_load_lds_dwordx4: the
  // 64 lanes of one load fill 1 KB of LDS in lane order, 64 / TPR whole tile rows).  Lane
  // (row lrow, chunk slot tid % TPR) therefore loads the logical chunk that the swizzle puts
  // into that slot: dcol = (slot ^ swz(lrow)) * 4 (the same for the rows lrow + RPP q).
  const int lrow = tid / TPR;
  const int dcol = (((tid % TPR)) ^ lds_swz<BK>(lrow)) * 4;
  constexpr int WROWS = 64 / TPR;   // tile rows of one wave's load
  // LDS byte addresses of this wave's first tile rows in stage 0 (M0 of its loads)
  const uint32_t a_lds = lds_addr(&As[0][0]) + (uint32_t)(wave * WROWS * BK * 4);
  const uint32_t b_lds = lds_addr(&Bs[0][0]) + (uint32_t)(wave * WROWS * BK * 4);
  static_assert(RPP % 16 == 0, "the swizzle (period 16 rows) repeats with the rows of a load pass");
  const float *a_row[QA];
  int ys[QA], xs[QA], yl[QA], xl[QA];
#pragma unroll
  for (int q = 0; q < QA; ++q) {
    const uint32_t m = (uint32_t)(m0 + lrow + RPP * q);
    const bool valid = m < (uint32_t)cl.M;
    uint32_t r = 0;
    int iy = 0, ix = 0, anc = 0;
    if (valid) convt_row(p, cl, tab, m, &r, &iy, &ix, &anc);
    int ylo = 0, xlo = 0, yn = p.S_out, xn = p.S_out;
    if (p.src_scale > 0 && valid) {   // windowed source (Ha > 0): anchor from the row index
      const int ay = anc / p.Ha, ax = anc - ay * p.Ha;
      const int oy = ay * p.src_scale - p.src_h, ox = ax * p.src_scale - p.src_h;
      ylo = max(0, -oy);
      xlo = max(0, -ox);
      yn = max(0, min(p.S_out, p.H_out - oy) - ylo);
      xn = max(0, min(p.S_out, p.H_out - ox) - xlo);
    }
    a_row[q] = p.A + (valid ? (int64_t)r * p.row_stride_out + ((int64_t)ylo * p.S_out + xlo) * p.C_out : 0);
    ys[q] = valid ? iy - ylo : -(1 << 20);   // an invalid row matches no tap
    xs[q] = ix - xlo;
    yl[q] = yn;
    xl[q] = xn;
  }
  const float *Bg = p.Bt + (int64_t)(n0 + lrow) * p.ldb + dcol;
  // K order: pairs of channel blocks outer, tap, then the block of the pair: the shifted
  // re-reads of one source block follow each other within a few K tiles (they hit the caches
  // instead of HBM), and the two halves of a 128-byte line (32 channels) are read by
  // consecutive K tiles (the second from L1)
  const int ntap = cl.nty * cl.ntx;
  const bool pairs = (p.C_out / BK) % 2 == 0;
  auto gload = [&](int kt, int buf) {
    int cb, t;
    if (pairs) {
      const int grp = kt / (2 * ntap), rem = kt - grp * 2 * ntap;
      t = rem >> 1;
      cb = grp * 2 + (rem & 1);
    } else {
      cb = kt / ntap;
      t = kt - cb * ntap;
    }
    const int co0 = cb * BK;
    const int ty = t / cl.ntx, tx = t - ty * cl.ntx;
    const int ky = cl.ky0 + cl.kys * ty, kx = cl.kx0 + cl.kxs * tx;
    const int dy = (cl.u0 + p.delta - ky) >> sh, dx = (cl.w0 + p.delta - kx) >> sh;   // exact
    const int co = co0 + dcol;
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int yy = ys[q] + dy, xx = xs[q] + dx;
      const bool ok = (unsigned)yy < (unsigned)yl[q] && (unsigned)xx < (unsigned)xl[q];
      // positions outside the source window or the image read a zero block
      const float *src = ok ? a_row[q] + (yy * p.S_out + xx) * p.C_out + co : g_zero4;
      dma16(src, a_lds + (uint32_t)(buf * (int)sizeof(As[0]) + RPP * q * BK * 4));
    }
    const int kb = (3 * ky + kx) * p.C_out + co0;
#pragma unroll
    for (int q = 0; q < QB; ++q)
      dma16(Bg + (int64_t)q * RPP * p.ldb + kb, b_lds + (uint32_t)(buf * (int)sizeof(Bs[0]) + RPP * q * BK * 4));
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int KT = cl.nty * cl.ntx * p.C_out / BK;
  // two LDS stages: K tile kt + 1 is in flight while tile kt is multiplied.  Its loads go out
  // right after the barrier that frees its stage, before this wave waits for tile kt's own
  // loads (a second barrier then publishes tile kt): the gathers wait on the L2, and issuing
  // them as early as possible is what counts here (issuing them after the operand reads, or
  // spread over the MFMA steps, measured 5-8% slower)
  constexpr int LPT = QA + QB;   // loads per thread per K tile
  gload(0, 0);
  // operand reads: lane (r32, half) takes chunks half * CPR / 2 + h, h < CPR / 2, of row r32
  const int r32 = lane & 31, sw = lds_swz<BK>(r32);
  int roff[CPR / 2];
#pragma unroll
  for (int h = 0; h < CPR / 2; ++h) roff[h] = ((((lane >> 5) * (CPR / 2)) + h) ^ sw) * 4;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt % CONVT_NS;
    static_assert(CONVT_NS == 2, "two barriers per tile: the next tile's loads go out before this one has landed");
    barrier_only();   // every wave is done with tile kt - 1: its stage is free
    if (kt + 1 < KT) {
      gload(kt + 1, cur ^ 1);
      wait_vmcnt<LPT>();   // this wave's part of tile kt has landed
    } else {
      wait_vmcnt<0>();
    }
    barrier_only();   // every wave's part of tile kt is in LDS
    const float *as = As[cur] + (wm * (BM / WM) + r32) * BK;
    const float *bs = Bs[cur] + (wn * (BN / WN) + r32) * BK;
#pragma unroll
    for (int h = 0; h < CPR / 2; ++h) {
      f32x4 a[MB], b[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = *reinterpret_cast<const f32x4 *>(as + i * 32 * BK + roff[h]);
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j] = *reinterpret_cast<const f32x4 *>(bs + j * 32 * BK + roff[h]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
  }
  __syncthreads();   // every wave is done with the operand buffers, which the epilogue reuses

  // ---- epilogue ----
  static_assert(28 * BM <= (int)sizeof(As), "epilogue row information must fit the A buffers");
  convt_epilogue<BM, BN, WM, WN, RELU, AL, SPL>(p, cl, tab, acc, m0, n0, nt, &As[0][0]);
}

// Classes of one axis: positions u of the destination window with the same taps ky, as an
// arithmetic progression of positions and of taps.
struct AxisClass {
  int u0, ustep, n, k0, ks, nk;
};

static bool axis_classes(int S_in, int S_out, int stride, int delta, std::vector<AxisClass> &out) {
  out.clear();
  std::vector<AxisClass> open;   // classes that can still grow
  for (int u = 0; u < S_in; ++u) {
    int taps[3], nt = 0;
    for (int ky = 0; ky < 3; ++ky) {
      const int q = u + delta - ky;
      if (q < 0 || q % stride) continue;
      if (q / stride < S_out) taps[nt++] = ky;
    }
    if (nt == 0) return false;   // a position no tap reaches (not produced by these shapes)
    const int ks = nt > 1 ? taps[1] - taps[0] : 1;
    for (int i = 2; i < nt; ++i)
      if (taps[i] - taps[i - 1] != ks) return false;
    bool joined = false;
    for (AxisClass &c : open) {   // same taps, next position of the progression
      if (c.k0 == taps[0] && c.nk == nt && c.ks == ks && u == c.u0 + stride * c.n) {
        ++c.n;
        joined = true;
        break;
      }
    }
    if (!joined) open.push_back({u, stride, 1, taps[0], ks, nt});
  }
  out = open;
  return true;
}

// The classes of a transposed convolution (axis classes of rows times those of columns) and
// their dispatches, up to four consecutive classes each.  (One dispatch of all classes, the
// longest first, measured 1.7% slower on the ResNet: a border-ring tile gathers a position or
// two from each of its 256 rows' windows, and mixing them with the interior tiles of other
// rows costs L2 locality.)
struct ConvtDispatch {
  std::vector<int> cls;   // indices into the class list
};

static bool convt_axes(const ConvTArgs &a, std::vector<AxisClass> &cu) {
  if (!axis_classes(a.S_in, a.S_out, a.stride, a.delta, cu) || cu.empty()) return false;
  for (const AxisClass &c : cu)   // the gather's row offset assumes ustep = stride for n > 1
    if (c.n > 1 && c.ustep != a.stride) return false;
  return true;
}

static ConvClass class_geometry(const std::vector<AxisClass> &cu, int idx) {
  const AxisClass &yu = cu[idx / cu.size()], &xw = cu[idx % cu.size()];   // square windows
  ConvClass k{};
  k.u0 = yu.u0;
  k.ustep = yu.ustep;
  k.ny = yu.n;
  k.ky0 = yu.k0;
  k.kys = yu.ks;
  k.nty = yu.nk;
  k.w0 = xw.u0;
  k.wstep = xw.ustep;
  k.nx = xw.n;
  k.kx0 = xw.k0;
  k.kxs = xw.ks;
  k.ntx = xw.nk;
  return k;
}

bool convt_clipped(const ConvTArgs &a) {
  return !a.dense && a.Ha > 0 && a.Ha <= CONVT_CLIP_MAX && a.R % (a.Ha * a.Ha) == 0;
}

// Inside positions of one axis of a class, summed over the anchors (clipped classes)
static int64_t clip_total(const ConvTArgs &a, int u0, int ustep, int n) {
  int64_t t = 0;
  for (int an = 0; an < a.Ha; ++an) {
    int lo, hi;
    clip_range(an * a.scale - a.h_in, u0, ustep, n, a.H_in, &lo, &hi);
    t += hi - lo;
  }
  return t;
}

static bool convt_plan(const ConvTArgs &a, std::vector<AxisClass> &cu, std::vector<ConvtDispatch> &plan) {
  plan.clear();
  if (a.C_out % 32 || a.R <= 0 || a.N_pad <= 0 || (a.stride != 1 && a.stride != 2)) return false;
  if ((int64_t)a.R * a.S_in * a.S_in > a.M_pad) return false;
  // windowed sources feed windows, in windowed passes (anchors from the row index)
  if (a.src_scale > 0 && (a.H_out <= 0 || a.dense || a.Ha <= 0 || a.R % (a.Ha * a.Ha))) return false;
  if (!convt_axes(a, cu)) return false;
  const int total = (int)(cu.size() * cu.size());
  for (int f = 0; f < total; f += 4) {
    ConvtDispatch d;
    for (int idx = f; idx < std::min(total, f + 4); ++idx) d.cls.push_back(idx);
    plan.push_back(d);
  }
  return true;
}

// Fills a.cls for dispatch d with BM-row tiles and n_nt column tiles; returns the number of
// workgroups (or -1).
static int64_t convt_fill(ConvTArgs &a, const std::vector<AxisClass> &cu, const ConvtDispatch &d, int BM, int BN) {
  if (a.N_pad % BN) return -1;
  const int n_nt = a.N_pad / BN;
  a.n_cls = (int)d.cls.size();
  int64_t blk = 0;
  for (int c = 0; c < 4; ++c) {
    ConvClass &k = a.cls[c];
    k = ConvClass{};
    if (c >= a.n_cls) {
      k.blk0 = 0x7fffffff;
      continue;
    }
    k = class_geometry(cu, d.cls[c]);
    int64_t M = (int64_t)a.R * k.ny * k.nx;
    uint32_t per = (uint32_t)(k.ny * k.nx);   // GEMM rows per coefficient row (clipped: per cycle)
    if (convt_clipped(a)) {
      const int64_t T = clip_total(a, k.u0, k.ustep, k.ny) * clip_total(a, k.w0, k.wstep, k.nx);
      M = (int64_t)(a.R / (a.Ha * a.Ha)) * T;
      per = (uint32_t)std::max<int64_t>(T, 1);
      k.clip = 1;
    }
    if (M >= ((int64_t)1 << 31)) return -1;
    k.M = (int32_t)M;
    k.div_yx = make_fastdiv(per);
    k.div_x = make_fastdiv((uint32_t)k.nx);
    k.blk0 = (int32_t)blk;
    blk += (M + BM - 1) / BM * n_nt;
  }
  return blk > 0x7fffffff ? -1 : blk;
}

uint64_t convt_part_flops(const ConvTArgs &a, int part) {
  std::vector<AxisClass> cu;
  std::vector<ConvtDispatch> plan;
  if (!convt_plan(a, cu, plan) || part < 0 || part >= (int)plan.size()) return 0;
  uint64_t f = 0;   // every position times the taps that reach it: the necessary multiply-adds
  const bool win = !a.dense && a.Ha > 0 && a.R % (a.Ha * a.Ha) == 0;
  const int sh = a.stride == 2 ? 1 : 0;
  // windowed rows: per axis and anchor, the (position, tap) pairs whose destination and source
  // both lie inside the image; a row's count is the product of its two axes'
  auto axis_pairs = [&](int u0, int ustep, int n, int k0, int ks, int nk) {
    int64_t t = 0;
    for (int an = 0; an < a.Ha; ++an) {
      int lo, hi;
      clip_range(an * a.scale - a.h_in, u0, ustep, n, a.H_in, &lo, &hi);
      const int os = an * a.src_scale - a.src_h;
      for (int i = lo; i < hi; ++i)
        for (int tk = 0; tk < nk; ++tk) {
          const int ys = i + ((u0 + a.delta - (k0 + ks * tk)) >> sh);   // source window position
          t += a.src_scale <= 0 || (os + ys >= 0 && os + ys < a.H_out);
        }
    }
    return t;
  };
  for (int idx : plan[part].cls) {
    const ConvClass k = class_geometry(cu, idx);
    if (win)
      f += 2ull * (uint64_t)(a.R / (a.Ha * a.Ha)) * (uint64_t)axis_pairs(k.u0, k.ustep, k.ny, k.ky0, k.kys, k.nty) *
           (uint64_t)axis_pairs(k.w0, k.wstep, k.nx, k.kx0, k.kxs, k.ntx) * (uint64_t)a.C_out * (uint64_t)a.C_in;
    else
      f += 2ull * (uint64_t)a.R * (uint64_t)(k.ny * k.nx) * (uint64_t)(k.nty * k.ntx) * (uint64_t)a.C_out *
           (uint64_t)a.C_in;
  }
  return f;
}

int convt_launches(const ConvTArgs &a) {
  std::vector<AxisClass> cu;
  std::vector<ConvtDispatch> plan;
  return convt_plan(a, cu, plan) ? (int)plan.size() : -1;
}

hipError_t launch_convt_part(const ConvTArgs &a0, int part, hipStream_t s) {
  std::vector<AxisClass> cu;
  std::vector<ConvtDispatch> plan;
  if (!convt_plan(a0, cu, plan) || part < 0 || part >= (int)plan.size()) return hipErrorInvalidValue;
  const ConvtDispatch &d = plan[part];
  ConvTArgs a = a0;
  const bool al = a.alpha || a.pre;
  const bool spl = a.splits.D > 0;
  if (al && (!a.alpha || !a.pre || !a.P_pos || !a.dense)) return hipErrorInvalidValue;
  if (spl && (!a.P_pos || !a.dense || a.splits.rows_per_domain <= 0)) return hipErrorInvalidValue;
  const dim3 blk256(256);
  if (a.N_pad % 128 == 0) {   // 128 x 128 tiles, 2 x 2 waves of 64 x 64
    const int64_t blk = convt_fill(a, cu, d, 128, 128);
    if (blk < 0) return hipErrorInvalidValue;
    const dim3 g((unsigned)blk);
    if (blk > 0 && al && spl)
      hipLaunchKernelGGL((k_convt<128, 128, 16, 2, 2, 2, true, true, true>), g, blk256, 0, s, a);
    else if (blk > 0 && spl)
      hipLaunchKernelGGL((k_convt<128, 128, 16, 2, 2, 2, true, false, true>), g, blk256, 0, s, a);
    else if (blk > 0 && al)
      hipLaunchKernelGGL((k_convt<128, 128, 16, 2, 2, 2, true, true>), g, blk256, 0, s, a);
    else if (blk > 0 && a.P_pos)
      hipLaunchKernelGGL((k_convt<128, 128, 16, 2, 2, 3, true>), dim3((unsigned)blk), dim3(256), 0, s, a);
    else if (blk > 0)
      hipLaunchKernelGGL((k_convt<128, 128, 16, 2, 2, 3, false>), dim3((unsigned)blk), dim3(256), 0, s, a);
  } else {                           // 256 x 64 tiles, 4 x 1 waves of 64 x 64
    const int64_t blk = convt_fill(a, cu, d, 256, 64);
    if (blk < 0) return hipErrorInvalidValue;
    const dim3 g((unsigned)blk);
    if (blk > 0 && al && spl)
      hipLaunchKernelGGL((k_convt<256, 64, 16, 4, 1, 2, true, true, true>), g, blk256, 0, s, a);
    else if (blk > 0 && spl)
      hipLaunchKernelGGL((k_convt<256, 64, 16, 4, 1, 2, true, false, true>), g, blk256, 0, s, a);
    else if (blk > 0 && al)
      hipLaunchKernelGGL((k_convt<256, 64, 16, 4, 1, 2, true, true>), g, blk256, 0, s, a);
    else if (blk > 0 && a.P_pos)
      hipLaunchKernelGGL((k_convt<256, 64, 16, 4, 1, 3, true>), dim3((unsigned)blk), dim3(256), 0, s, a);
    else if (blk > 0)
      hipLaunchKernelGGL((k_convt<256, 64, 16, 4, 1, 3, false>), dim3((unsigned)blk), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_convt(const ConvTArgs &a, hipStream_t s) {
  const int n = convt_launches(a);
  if (n < 0) return hipErrorInvalidValue;
  for (int k = 0; k < n; ++k) {
    const hipError_t e = launch_convt_part(a, k, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ------------------------------------------------------------------------------------
// Transposed stem convolution onto the network input (at most 4 input channels), fused with
// the concretization.  With few input channels the contraction is regrouped so that the
// matrix cores see a useful N: per source position s of a coefficient row
//   G[s][ci * 9 + tap] = sum_co A_out[r][s][co] W[co][ci][tap]        (GEMM, N = 9 C_in, K = C_out)
// and every input-window position (u, w) then gathers the taps that reach it,
//   a[ci] = sum over taps (ky, kx) reaching (u, w) of G[s(u, w, ky, kx)][ci * 9 + 3 ky + kx]
//   part[(r, u, w)] = sum_ci a c[unit][ci][gy][gx] - |a| r[unit][ci][gy][gx]   (inside the image)
// W's own layout [co][ci][3][3] is the B operand [K][N].  A workgroup takes several whole
// rows (small windows) or a strip of destination rows of one row (large windows); the
// source positions' G stays in LDS between the two phases.
constexpr int STEM_LDS_FLOATS = 10752;
constexpr int64_t STEM_GRID = 4096;   // workgroups; each takes every gridDim-th work item
// destination positions per thread (fewer with four input channels: register budget)
constexpr int stem_dpt(int cin) { return cin == 4 ? 1 : 4; }

template <int CIN>
__global__ __launch_bounds__(256, 3) void k_stem(const StemArgs p) {
  constexpr int NB = CIN * 9 > 32 ? 2 : 1;   // 32-column MFMA blocks of N
  constexpr int GP = 32 * NB + 1;            // G row pitch (odd: the gather reads hit distinct banks)
  constexpr int NW = CIN * 9;
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int WTP = p.C_out + 4;               // transposed weights, k contiguous
  float *wt = lds;                           // [32 NB][WTP]
  float *G = lds + 32 * NB * WTP;            // [source positions][GP]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 32 * NB * p.C_out; i += 256) {
    const int n = i / p.C_out, k = i - n * p.C_out;
    wt[n * WTP + k] = n < NW ? p.W[(int64_t)k * NW + n] : 0.f;
  }
  __syncthreads();
  // work items (row groups x strips), the weights staged once for all of them
  const int n_items = (p.R + p.rpw - 1) / p.rpw * p.n_strips;
  for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int rg = item / p.n_strips, st = item - rg * p.n_strips;
    const int r0 = rg * p.rpw;
    const int rows = min(p.rpw, p.R - r0);
    const int u_lo = st * p.strip, u_hi = min(p.S_in, u_lo + p.strip);
    // source rows reached from destination rows [u_lo, u_hi): y = (u + delta - ky) / stride
    const int lo_num = max(0, u_lo + p.delta - 2);
    const int y_lo = (lo_num + p.stride - 1) / p.stride;
    const int y_hi = min(p.S_out - 1, (u_hi - 1 + p.delta) / p.stride);
    const int n_row_src = (y_hi >= y_lo ? y_hi - y_lo + 1 : 0) * p.S_out;
    const int n_src = rows * n_row_src;

    // destination positions of this thread (at most stem_dpt): their box terms are loaded
    // before the GEMM phase, so the loads complete under it
    const int nu = u_hi - u_lo;
    const int per_rl = nu * p.S_in;
    constexpr int STEM_DPT = stem_dpt(CIN);
    const int n_dst = rows * per_rl;   // <= 256 STEM_DPT (launch_stem)
    bool live[STEM_DPT];
    float bc[STEM_DPT][CIN], br[STEM_DPT][CIN];
#pragma unroll
    for (int q = 0; q < STEM_DPT; ++q) {
      const int d = tid + 256 * q;
      live[q] = false;
      if (d < n_dst) {
        const int rl = d / per_rl, rem = d - rl * per_rl;
        const int uu = rem / p.S_in;
        const int u = u_lo + uu, w = rem - uu * p.S_in;
        const int4 an = p.rows[r0 + rl];
        const int gy = p.dense ? u : an.y * p.scale - p.h_in + u;
        const int gx = p.dense ? w : an.z * p.scale - p.h_in + w;
        live[q] = gy >= 0 && gx >= 0 && gy < p.H_in && gx < p.H_in;
        if (live[q]) {
#pragma unroll
          for (int ci = 0; ci < CIN; ++ci) {
            const int64_t bi = (int64_t)an.x * p.ld_box + ((int64_t)ci * p.H_in + gy) * p.H_in + gx;
            bc[q][ci] = p.c0[bi];
            br[q][ci] = p.r0[bi];
          }
        }
      }
    }


    // ---- G = A_src W: each wave takes 32-position blocks, two at a time (blocks b and b + 4),
    // as one stream of steps (block pair, 32-channel chunk); lane (r32, half) feeds the MFMAs
    // with 16 consecutive k of its position per chunk, identically for both operands.  Two
    // register sets: step s + 1 is requested before step s is multiplied (past the last step
    // the request repeats it: every request unconditional, so each multiply waits for its own
    // step only).
    const int r32 = lane & 31, half = lane >> 5;
    const int n_blk = (n_src + 31) / 32;
    const int KC = p.C_out / 32;
    const int n_pairs = wave < n_blk ? (n_blk - wave + 7) / 8 : 0;
    const int S = n_pairs * KC;   // wave-uniform
    auto load_step = [&](int st, f32x4 (&a)[2][4]) {
      st = min(st, S - 1);
      const int pr = st / KC, kc = st - pr * KC;
      const int b0 = wave + 8 * pr;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        // positions past the last one repeat it: their G rows are never gathered
        const int pi = min((b0 + 4 * q) * 32 + r32, n_src - 1);
        const int rl = pi / n_row_src, sp = pi - rl * n_row_src;
        const float *src = p.A + (int64_t)(r0 + rl) * p.row_stride_out + ((int64_t)y_lo * p.S_out + sp) * p.C_out +
                           kc * 32 + half * 16;
#pragma unroll
        for (int h = 0; h < 4; ++h) a[q][h] = *reinterpret_cast<const f32x4 *>(src + 4 * h);
      }
    };
    f32x16 acc[2][NB];
    auto mma_step = [&](int st, const f32x4 (&a)[2][4]) {
      const int pr = st / KC, kc = st - pr * KC;
      if (kc == 0) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[q][j][v] = 0.f;
      }
      f32x4 b[NB][4];
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int h = 0; h < 4; ++h)
          b[j][h] = *reinterpret_cast<const f32x4 *>(wt + (32 * j + r32) * WTP + kc * 32 + half * 16 + 4 * h);
#pragma unroll
      for (int h = 0; h < 4; ++h)
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int j = 0; j < NB; ++j)
              acc[q][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[q][h][e], b[j][h][e], acc[q][j], 0, 0, 0);
      if (kc == KC - 1) {   // the pair is done: lane holds rows 8 g + 4 half + t (v = 4 g + t)
        const int b0 = wave + 8 * pr;
        const bool two = b0 + 4 < n_blk;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          if (q == 1 && !two) break;
#pragma unroll
          for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
              G[((b0 + 4 * q) * 32 + (v >> 2) * 8 + half * 4 + (v & 3)) * GP + 32 * j + r32] = acc[q][j][v];
        }
      }
    };
    if (S > 0) {
      f32x4 a0[2][4], a1[2][4];
      load_step(0, a0);
      // an opaque copy: otherwise the loop head merges this load and the loop's into one
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int h = 0; h < 4; ++h) asm volatile("" : "+v"(a0[q][h]));
      for (int st = 0;; st += 2) {
        load_step(st + 1, a1);
        __builtin_amdgcn_sched_barrier(0);
        mma_step(st, a0);
        __builtin_amdgcn_sched_barrier(0);
        if (st + 1 >= S) break;
        load_step(st + 2, a0);
        __builtin_amdgcn_sched_barrier(0);
        mma_step(st + 1, a1);
        __builtin_amdgcn_sched_barrier(0);
        if (st + 2 >= S) break;
      }
    }
    __syncthreads();

    // ---- gather the taps of every destination position and concretize
    const int S_in2 = p.S_in * p.S_in;
#pragma unroll
    for (int q = 0; q < STEM_DPT; ++q) {
      const int d = tid + 256 * q;
      if (d >= n_dst) break;
      const int rl = d / per_rl, rem = d - rl * per_rl;
      const int uu = rem / p.S_in;
      const int u = u_lo + uu, w = rem - uu * p.S_in;
      float part = 0.f;
      if (live[q]) {   // inside the image
        // source window positions inside the source image: [ylo, yhi) x [xlo, xhi)
        int ylo = 0, yhi = p.S_out, xlo = 0, xhi = p.S_out;
        if (p.src_scale > 0) {
          const int4 an = p.rows[r0 + rl];
          const int oy = an.y * p.src_scale - p.src_h, ox = an.z * p.src_scale - p.src_h;
          ylo = max(0, -oy);
          xlo = max(0, -ox);
          yhi = min(p.S_out, p.H_src - oy);
          xhi = min(p.S_out, p.H_src - ox);
        }
        float a[CIN];
#pragma unroll
        for (int ci = 0; ci < CIN; ++ci) a[ci] = 0.f;
#pragma unroll
        for (int ky = 0; ky < 3; ++ky) {
          int yy = u + p.delta - ky;
          if (yy < 0 || (yy & (p.stride - 1))) continue;
          yy /= p.stride;
          if (yy < ylo || yy >= yhi) continue;
#pragma unroll
          for (int kx = 0; kx < 3; ++kx) {
            int xx = w + p.delta - kx;
            if (xx < 0 || (xx & (p.stride - 1))) continue;
            xx /= p.stride;
            if (xx < xlo || xx >= xhi) continue;
            const float *g = G + (rl * n_row_src + (yy - y_lo) * p.S_out + xx) * GP + 3 * ky + kx;
#pragma unroll
            for (int ci = 0; ci < CIN; ++ci) a[ci] += g[9 * ci];
          }
        }
#pragma unroll
        for (int ci = 0; ci < CIN; ++ci) part += a[ci] * bc[q][ci] - fabsf(a[ci]) * br[q][ci];
        if (p.vtx) {   // dense windows: (u, w) is the image position
          float *v = p.vtx + (int64_t)(r0 + rl) * p.ld_vtx + (u * p.H_in + w) * CIN;
#pragma unroll
          for (int ci = 0; ci < CIN; ++ci)
            v[ci] = a[ci] > 0.f ? bc[q][ci] - br[q][ci] : (a[ci] < 0.f ? bc[q][ci] + br[q][ci] : bc[q][ci]);
        }
      }
      p.part[(int64_t)(r0 + rl) * S_in2 + u * p.S_in + w] = part;
    }
    __syncthreads();   // G is rewritten by the next item
  }
}

template <int CIN>
hipError_t launch_stem_t(StemArgs a, hipStream_t s) {
  constexpr int NB = CIN * 9 > 32 ? 2 : 1;
  constexpr int GP = 32 * NB + 1;
  if (a.C_out <= 0 || a.C_out % 32 || a.R <= 0 || (a.stride != 1 && a.stride != 2) || a.S_out <= 0 || a.S_in <= 0)
    return hipErrorInvalidValue;
  if (a.vtx && (!a.dense || a.S_in != a.H_in || a.ld_vtx < (int64_t)a.H_in * a.H_in * CIN))
    return hipErrorInvalidValue;
  if (a.src_scale > 0 && (a.dense || a.H_src <= 0)) return hipErrorInvalidValue;
  const int64_t wt_floats = 32 * NB * (int64_t)(a.C_out + 4);
  // 42 KB of LDS per workgroup (three workgroups per CU), 64 KB for wide weights
  int64_t src_max = ((STEM_LDS_FLOATS - wt_floats) / GP) & ~(int64_t)31;
  if (src_max < 64) src_max = ((16384 - wt_floats) / GP) & ~(int64_t)31;
  if (src_max < 32) return hipErrorInvalidValue;
  auto src_positions = [&](int u_lo, int u_hi) {   // the kernel's source-row range, times S_out
    const int y_lo = (std::max(0, u_lo + a.delta - 2) + a.stride - 1) / a.stride;
    const int y_hi = std::min(a.S_out - 1, (u_hi - 1 + a.delta) / a.stride);
    return (int64_t)(y_hi >= y_lo ? y_hi - y_lo + 1 : 0) * a.S_out;
  };
  const int64_t full = src_positions(0, a.S_in);
  const int64_t dst_max = 256 * stem_dpt(CIN), S_in2 = (int64_t)a.S_in * a.S_in;
  if (full <= src_max && S_in2 <= dst_max) {   // whole rows
    a.rpw = (int32_t)std::max<int64_t>(1, std::min(src_max / std::max<int64_t>(full, 1), dst_max / S_in2));
    a.strip = a.S_in;
  } else {                                     // one row, strips of destination rows
    a.rpw = 1;
    a.strip = 0;
    for (int h = std::min<int64_t>(a.S_in, dst_max / a.S_in); h >= 1 && !a.strip; --h) {
      bool fits = true;
      for (int u0 = 0; u0 < a.S_in && fits; u0 += h) fits = src_positions(u0, std::min(a.S_in, u0 + h)) <= src_max;
      if (fits) a.strip = h;
    }
    if (!a.strip) return hipErrorInvalidValue;
  }
  a.n_strips = (a.S_in + a.strip - 1) / a.strip;
  const int64_t items = ((int64_t)a.R + a.rpw - 1) / a.rpw * a.n_strips;
  if (items > 0x7fffffff) return hipErrorInvalidValue;
  const int64_t grid = std::min<int64_t>(items, STEM_GRID);
  const size_t lds = sizeof(float) * (size_t)(wt_floats + src_max * GP);
  hipLaunchKernelGGL((k_stem<CIN>), dim3((unsigned)grid), dim3(256), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_stem(const StemArgs &a, hipStream_t s) {
  switch (a.C_in) {
    case 1: return launch_stem_t<1>(a, s);
    case 2: return launch_stem_t<2>(a, s);
    case 3: return launch_stem_t<3>(a, s);
    case 4: return launch_stem_t<4>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// ------------------------------------------------------------------------------------
// First rows of a pass that starts at a 3x3 convolution's output neurons: row (unit, dir,
// c0, i, j) is (dir ? -1 : 1) W[c0][ci][u][w] on the convolution's input window around
// (stride i, stride j), zero outside the image; relaxed (or identity) like the GEMM
// epilogue; beta = (dir ? -1 : 1) b[c0] + the window's constant terms.  Rows are ordered
// (unit, dir, c0, position); the 2 INIT_CONV_G rows of one unit and position with start
// channels c0 in one group of INIT_CONV_G (both directions) share their window and so their
// relaxation parameters, which are the bulk of the reads: a wave takes those rows, loads each
// parameter once for all of them, and writes each row with the lanes across the channels
// (weights tap-major, [c0][u][w][ci]: contiguous channel loads).  A row's constant is summed
// positions outer, a lane's channels inner, then a fixed butterfly.
constexpr int INIT_CONV_G = 4;   // start channels per wave (8 rows)

__global__ __launch_bounds__(256) void k_init_conv(const ConvInitArgs a) {
  const int lane = threadIdx.x & 63;
  const int HW = a.H_src * a.H_src;
  const int64_t n_src = (int64_t)a.C_src * HW;
  const int n_grp = a.C_src / INIT_CONV_G;
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t units = a.R / (2 * n_src);
  if (wv >= units * n_grp * HW) return;   // wave-uniform
  const int64_t ug = wv / HW;
  const int pos = (int)(wv - ug * HW);
  const int64_t ul = ug / n_grp;
  const int cg = (int)(ug - ul * n_grp);
  const int64_t r0 = ul * 2 * n_src + (int64_t)cg * INIT_CONV_G * HW + pos;   // dir 0, first c0 of the group
  const int4 an = a.rows[r0];   // the same unit and anchor for all the wave's rows
  const int S = a.S;
  const int64_t row_len = (int64_t)S * S * a.C_in;
  float acc[2][INIT_CONV_G];
#pragma unroll
  for (int d = 0; d < 2; ++d)
#pragma unroll
    for (int e = 0; e < INIT_CONV_G; ++e) acc[d][e] = 0.f;
  for (int u = 0; u < S; ++u)
    for (int w = 0; w < S; ++w) {
      const int gy = an.y * a.scale - a.h + u, gx = an.z * a.scale - a.h + w;
      const bool in = gy >= 0 && gx >= 0 && gy < a.H_in && gx < a.H_in;
      const float4 *P = a.P_pos ? a.P_pos + (((int64_t)an.x * a.H_in + gy) * a.H_in + gx) * a.C_in : nullptr;
      const int64_t po = (int64_t)(u * S + w) * a.C_in;
      for (int ci = lane; ci < a.C_in; ci += 64) {
        float4 prm = make_float4(0.f, 0.f, 0.f, 0.f);
        if (in) prm = P ? P[ci] : make_float4(1.f, 1.f, 0.f, a.bias_next[ci]);
#pragma unroll
        for (int e = 0; e < INIT_CONV_G; ++e) {
          const int c0 = cg * INIT_CONV_G + e;
          const float wt = in ? a.W[((int64_t)c0 * 9 + u * 3 + w) * a.C_in + ci] : 0.f;
#pragma unroll
          for (int d = 0; d < 2; ++d) {
            const float x = d ? -wt : wt;
            float ap = 0.f;
            if (in) {
              ap = x > 0.f ? x * prm.x : x * prm.y;
              acc[d][e] += fminf(x, 0.f) * prm.z + ap * prm.w;
            }
            const int64_t r = r0 + d * n_src + (int64_t)e * HW;
            __builtin_nontemporal_store(ap, a.out + r * row_len + po + ci);   // read back only by the next GEMM
          }
        }
      }
    }
  // the eight rows' sums over the wave (lane 8 k ends with row k = INIT_CONV_G d + e)
  static_assert(2 * INIT_CONV_G == 8, "one value per row of the wave's eight");
  float rows8[8];
#pragma unroll
  for (int d = 0; d < 2; ++d)
#pragma unroll
    for (int e = 0; e < INIT_CONV_G; ++e) rows8[d * INIT_CONV_G + e] = acc[d][e];
  const float x = wave_sums8(rows8, lane);
  if ((lane & 7) == 0) {
    const int k = lane >> 3, d = k / INIT_CONV_G, e = k - d * INIT_CONV_G;
    const int c0 = cg * INIT_CONV_G + e;
    a.beta[r0 + d * n_src + (int64_t)e * HW] = (d ? -1.f : 1.f) * a.b[c0] + x;
  }
}

hipError_t launch_init_conv(const ConvInitArgs &a, hipStream_t s) {
  const int64_t n_src = (int64_t)a.C_src * a.H_src * a.H_src;
  // whole units of 2 n_src rows, start channels in groups, a 3 x 3 window
  if (a.C_src % INIT_CONV_G || a.S != 3 || n_src <= 0 || a.R % (2 * n_src)) return hipErrorInvalidValue;
  const int64_t waves = a.R / 2 / INIT_CONV_G;
  if ((waves + 3) / 4 > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_init_conv, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Constant terms of a pass: beta[r] += sum over the row's positions and the column parts.
// G = 2^lg lanes share a row (lane j sums positions j, j + G, ... over all parts), then add
// their sums by a fixed butterfly: consecutive lanes read consecutive positions.
__global__ void k_rowsum_win(float *beta, const float *part, int32_t n_parts, int64_t M_pad, int64_t R,
                             int32_t per_row, int32_t lg, WinClip cw) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t r = t >> lg;
  const int G = 1 << lg, j = (int)(t & (G - 1));
  float s = 0.f;
  if (r < R) {
    int oy = 0, ox = 0;   // clipped rows: the window's origin in the image
    if (cw.Ha > 0) {
      const int an = (int)(r % (cw.Ha * cw.Ha));
      oy = an / cw.Ha * cw.scale - cw.h;
      ox = an % cw.Ha * cw.scale - cw.h;
    }
    for (int q = j; q < per_row; q += G) {
      if (cw.Ha > 0) {   // positions outside the image have no partial sums
        const int u = q / cw.S, w = q - u * cw.S;
        if ((unsigned)(oy + u) >= (unsigned)cw.H || (unsigned)(ox + w) >= (unsigned)cw.H) continue;
      }
      const int64_t m = r * per_row + q;
#pragma unroll 4
      for (int p = 0; p < n_parts; ++p) s += part[p * M_pad + m];   // loads issued ahead of the adds
    }
  }
  for (int o = G >> 1; o > 0; o >>= 1) s += __shfl_xor(s, o);   // every lane takes part
  if (r < R && j == 0) beta[r] += s;
}

hipError_t launch_rowsum_win(float *beta, const float *part, int32_t n_parts, int64_t M_pad, int64_t R,
                             int32_t per_row, hipStream_t s, WinClip clip) {
  if (R <= 0) return hipSuccess;
  if (clip.Ha > 0 && (clip.S <= 0 || (int64_t)clip.S * clip.S != per_row || R % ((int64_t)clip.Ha * clip.Ha)))
    return hipErrorInvalidValue;
  int lg = 0;
  while (lg < 6 && (2 << lg) <= per_row) ++lg;
  const int64_t n = R << lg;
  hipLaunchKernelGGL(k_rowsum_win, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, beta, part, n_parts, M_pad, R,
                     per_row, lg, clip);
  return hipGetLastError();
}

// Row table of a pass: row r -> (unit, anchor y, anchor x) for rows that start at the
// neurons of a (C, H, W) node in (unit, direction, c, y, x) order; dense rows get anchor 0.
__global__ void k_row_table(int4 *rows, int64_t R, int32_t rows_per_unit, int32_t C, int32_t H, int32_t Wd,
                            int32_t windowed, int32_t unit0) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  const int u = (int)(r / rows_per_unit);
  int ay = 0, ax = 0;
  if (windowed) {
    const int n = C * H * Wd;
    const int q = (int)(r - (int64_t)u * rows_per_unit) % n;
    const int hw = q % (H * Wd);
    ay = hw / Wd;
    ax = hw % Wd;
  }
  rows[r] = make_int4(u + unit0, ay, ax, 0);
}

hipError_t launch_row_table(int4 *rows, int64_t R, int32_t rows_per_unit, int32_t C, int32_t H, int32_t W,
                            int32_t windowed, int32_t unit0, hipStream_t s) {
  hipLaunchKernelGGL(k_row_table, dim3((unsigned)((R + 255) / 256)), dim3(256), 0, s, rows, R, rows_per_unit, C, H,
                     W, windowed, unit0);
  return hipGetLastError();
}

// Bounds of a convolutional ReLU layer from its finished pass: neuron q = (c, y, x) of unit
// b has rows (b, 0, q) (lower) and (b, 1, q) (negated upper); intersection with IBP; the
// relaxation is stored channels-last [b][y][x][c] for the windowed epilogues above.
__global__ void k_finalize_conv(const float *beta, int32_t B, int32_t C, int32_t H, const float *ibp_c,
                                const float *ibp_r, int64_t ld_ibp, int32_t intersect, const float *bias_next,
                                float *L, float *U, float4 *P, int32_t rule) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = (int64_t)C * H * H;
  if (idx >= B * n) return;
  const int64_t b = idx / n, q = idx - b * n;
  float l = beta[b * 2 * n + q];
  float u = -beta[b * 2 * n + n + q];
  if (intersect) {
    const int64_t j = b * ld_ibp + q;
    l = fmaxf(l, ibp_c[j] - ibp_r[j]);
    u = fminf(u, ibp_c[j] + ibp_r[j]);
  }
  L[idx] = l;
  U[idx] = u;
  const int c = (int)(q / (H * H)), hw = (int)(q % (H * H));
  const float4 prm = relax_params(l, u, bias_next ? bias_next[c] : 0.f, rule);
  P[(b * H * H + hw) * C + c] = prm;
}

hipError_t launch_finalize_conv(const float *beta, int32_t B, int32_t C, int32_t H, const float *ibp_c,
                                const float *ibp_r, int64_t ld_ibp, int32_t intersect, const float *bias_next,
                                float *L, float *U, float4 *P, int32_t lam_rule, hipStream_t s) {
  const int64_t tot = (int64_t)B * C * H * H;
  hipLaunchKernelGGL(k_finalize_conv, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, beta, B, C, H, ibp_c,
                     ibp_r, ld_ibp, intersect, bias_next, L, U, P, lam_rule);
  return hipGetLastError();
}

// A ReLU layer whose input is one convolution of the network input: its exact range over
// the box is the IBP interval [c - r, c + r]; relaxation stored channels-last.
__global__ void k_conv_layer_from_ibp(const float *ibp_c, const float *ibp_r, int64_t ld_ibp, int32_t B, int32_t C,
                                      int32_t H, const float *bias_next, float *L, float *U, float4 *P,
                                      int32_t rule) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = (int64_t)C * H * H;
  if (idx >= B * n) return;
  const int64_t b = idx / n, q = idx - b * n;
  const float cc = ibp_c[b * ld_ibp + q], rr = ibp_r[b * ld_ibp + q];
  const float l = cc - rr, u = cc + rr;
  L[idx] = l;
  U[idx] = u;
  const int c = (int)(q / (H * H)), hw = (int)(q % (H * H));
  const float4 prm = relax_params(l, u, bias_next[c], rule);
  P[(b * H * H + hw) * C + c] = prm;
}

hipError_t launch_conv_layer_from_ibp(const float *ibp_c, const float *ibp_r, int64_t ld_ibp, int32_t B, int32_t C,
                                      int32_t H, const float *bias_next, float *L, float *U, float4 *P,
                                      int32_t lam_rule, hipStream_t s) {
  const int64_t tot = (int64_t)B * C * H * H;
  hipLaunchKernelGGL(k_conv_layer_from_ibp, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, ibp_c, ibp_r,
                     ld_ibp, B, C, H, bias_next, L, U, P, lam_rule);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// IBP of a convolution in centre/radius form, c' = conv(W, c) + b, r' = conv(|W|, r), over
// CHW tensors, as an implicit GEMM on the matrix cores: out[co][pos] = sum_k W[co][k] x[k][pos]
// with k = (ci, ky, kx) (the weights' own K-contiguous order) and x[k][pos] the input value
// the tap reaches (0 in the padding).  A workgroup of 4 waves owns 32 output channels x 32
// output positions of one input: each wave takes a quarter of K (v_mfma_f32_32x32x2f32, the
// weights as the A operand, the gathered input as the B operand, so a lane's 32 consecutive
// positions are coalesced), and the four partial tiles are added in wave order through LDS,
// so every output has one fixed summation order (independent of the batch).
constexpr int IBPC_WAVES = 4;

__global__ __launch_bounds__(64 * IBPC_WAVES) void k_ibp_conv(const float *W, const float *bias, int32_t Co,
                                                             int32_t Ci, int32_t Hin, int32_t Hout, int32_t stride,
                                                             int32_t pad, const float *cin, const float *rin,
                                                             int64_t ld_in, float *cout, float *rout, int64_t ld_out) {
  __shared__ float red[IBPC_WAVES][32][64];   // per wave: 16 centre + 16 radius values per lane
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int P = Hout * Hout, K = Ci * 9;
  const int n_pt = (P + 31) / 32;
  const int b = blockIdx.x / n_pt, p0 = (blockIdx.x - b * n_pt) * 32;
  const int co0 = blockIdx.y * 32;
  const int l32 = lane & 31, kh = lane >> 5;
  // this lane's weight row (A operand) and output position (B operand)
  const int co = co0 + l32;
  const float *wrow = W + (int64_t)(co < Co ? co : 0) * K;
  const int pos = p0 + l32;
  const int oy = pos / Hout, ox = pos - oy * Hout;
  const int y0 = oy * stride - pad, x0 = ox * stride - pad;
  const bool pos_ok = pos < P, co_ok = co < Co;
  const float *cb = cin + (int64_t)b * ld_in, *rb = rin + (int64_t)b * ld_in;
  // this wave's quarter of K, in steps of 2 (one MFMA each for the centre and the radius)
  const int steps = (K + 1) / 2, per = (steps + IBPC_WAVES - 1) / IBPC_WAVES;
  const int s0 = wave * per, s1 = min(steps, s0 + per);
  f32x16 ac, ar;
#pragma unroll
  for (int v = 0; v < 16; ++v) ac[v] = ar[v] = 0.f;
  for (int st = s0; st < s1; ++st) {
    const int k = 2 * st + kh;
    float w = 0.f, xc = 0.f, xr = 0.f;
    if (k < K) {
      w = co_ok ? wrow[k] : 0.f;
      const int ci = k / 9, tap = k - ci * 9;
      const int ky = tap / 3, kx = tap - ky * 3;
      const int iy = y0 + ky, ix = x0 + kx;
      if (pos_ok && (unsigned)iy < (unsigned)Hin && (unsigned)ix < (unsigned)Hin) {
        const int64_t o = ((int64_t)ci * Hin + iy) * Hin + ix;
        xc = cb[o];
        xr = rb[o];
      }
    }
    ac = __builtin_amdgcn_mfma_f32_32x32x2f32(w, xc, ac, 0, 0, 0);
    ar = __builtin_amdgcn_mfma_f32_32x32x2f32(fabsf(w), xr, ar, 0, 0, 0);
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    red[wave][v][lane] = ac[v];
    red[wave][16 + v][lane] = ar[v];
  }
  __syncthreads();
  // thread t adds value v = 8 (t / 64) .. + 8 of lane t % 64 over the waves, in wave order;
  // lane l's value v is output channel 8 (v / 4) + 4 (l / 32) + v % 4 of the tile at position l % 32
  const int t = threadIdx.x, tl = t & 63, vq = t >> 6;
  const int op = p0 + (tl & 31);
  for (int j = 0; j < 8; ++j) {
    const int v = vq * 8 + j;   // 0..31: centre 0..15, radius 16..31
    float x = 0.f;
#pragma unroll
    for (int w = 0; w < IBPC_WAVES; ++w) x += red[w][v][tl];
    const int vv = v & 15;
    const int oc = co0 + 8 * (vv >> 2) + 4 * (tl >> 5) + (vv & 3);
    if (oc < Co && op < P) {
      if (v < 16)
        cout[(int64_t)b * ld_out + (int64_t)oc * P + op] = x + bias[oc];
      else
        rout[(int64_t)b * ld_out + (int64_t)oc * P + op] = x;
    }
  }
}

hipError_t launch_ibp_conv(const float *W, const float *bias, int32_t Co, int32_t Ci, int32_t Hin, int32_t Hout,
                           int32_t stride, int32_t pad, const float *cin, const float *rin, int64_t ld_in,
                           float *cout, float *rout, int64_t ld_out, int32_t B, hipStream_t s) {
  const int64_t n_pt = ((int64_t)Hout * Hout + 31) / 32;
  if (B <= 0 || B * n_pt > 0x7fffffff) return hipErrorInvalidValue;
  dim3 grid((unsigned)(B * n_pt), (unsigned)((Co + 31) / 32));
  hipLaunchKernelGGL(k_ibp_conv, grid, dim3(64 * IBPC_WAVES), 0, s, W, bias, Co, Ci, Hin, Hout, stride, pad, cin, rin,
                     ld_in, cout, rout, ld_out);
  return hipGetLastError();
}

// IBP of ReLU (interval [max(l,0), max(u,0)]) and of a sum, in centre/radius form.
__global__ void k_ibp_relu(const float *cin, const float *rin, float *cout, float *rout, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float lo = fmaxf(cin[i] - rin[i], 0.f), hi = fmaxf(cin[i] + rin[i], 0.f);
  cout[i] = (lo + hi) * 0.5f;
  rout[i] = (hi - lo) * 0.5f;
}

__global__ void k_ibp_add(const float *c1, const float *r1, const float *c2, const float *r2, float *cout,
                          float *rout, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  cout[i] = c1[i] + c2[i];
  rout[i] = r1[i] + r2[i];
}

hipError_t launch_ibp_relu(const float *cin, const float *rin, float *cout, float *rout, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_ibp_relu, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, cin, rin, cout, rout, n);
  return hipGetLastError();
}

hipError_t launch_ibp_add(const float *c1, const float *r1, const float *c2, const float *r2, float *cout,
                          float *rout, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_ibp_add, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, c1, r1, c2, r2, cout, rout, n);
  return hipGetLastError();
}

// Conv weights repacked for the transposed-convolution GEMM: Bt[ci][tap * Co + co] =
// W[co][ci][tap] for ci < Ci, zero rows up to Ci_pad.
__global__ void k_repack_convt(const float *W, int32_t Co, int32_t Ci, int32_t Ci_pad, float *Bt) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t K = 9 * (int64_t)Co;
  if (idx >= Ci_pad * K) return;
  const int ci = (int)(idx / K), k = (int)(idx % K);
  const int tap = k / Co, co = k % Co;
  Bt[idx] = ci < Ci ? W[((int64_t)co * Ci + ci) * 9 + tap] : 0.f;
}

hipError_t launch_repack_convt(const float *W, int32_t Co, int32_t Ci, int32_t Ci_pad, float *Bt, hipStream_t s) {
  const int64_t tot = (int64_t)Ci_pad * 9 * Co;
  hipLaunchKernelGGL(k_repack_convt, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, W, Co, Ci, Ci_pad, Bt);
  return hipGetLastError();
}

// Dense weight columns from flatten (C, H, W) order to channels-last (H, W, C) order.
__global__ void k_permute_hwc(const float *W, int32_t rows, int32_t C, int32_t HW, float *Wo, int64_t ldo) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n = (int64_t)C * HW;
  if (idx >= rows * ldo) return;
  const int64_t o = idx / ldo, j = idx % ldo;   // j = hw * C + c
  float v = 0.f;
  if (j < n) {
    const int64_t hw = j / C, c = j % C;
    v = W[o * n + c * HW + hw];
  }
  Wo[idx] = v;
}

hipError_t launch_permute_hwc(const float *W, int32_t rows, int32_t C, int32_t HW, float *Wo, int64_t ldo,
                              hipStream_t s) {
  const int64_t tot = (int64_t)rows * ldo;
  hipLaunchKernelGGL(k_permute_hwc, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, W, rows, C, HW, Wo, ldo);
  return hipGetLastError();
}

// Identity relaxation with a per-channel bias for channels-last columns: P[j] =
// (1, 1, 0, b[j % C]) for j < n, zero beyond.
__global__ void k_identity_params(const float *b, int32_t C, int64_t n, int64_t ld, float4 *P) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= ld) return;
  P[j] = j < n ? make_float4(1.f, 1.f, 0.f, b ? b[j % C] : 0.f) : make_float4(0.f, 0.f, 0.f, 0.f);
}

hipError_t launch_identity_params(const float *b, int32_t C, int64_t n, int64_t ld, float4 *P, hipStream_t s) {
  hipLaunchKernelGGL(k_identity_params, dim3((unsigned)((ld + 255) / 256)), dim3(256), 0, s, b, C, n, ld, P);
  return hipGetLastError();
}

// Relaxation parameters of a dense-output ReLU from channels-last bounds stay in the MLP
// layout [b][n]; a ReLU on a conv node keeps [b][y][x][c].  Both are produced by the
// finalize kernels.

FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  f.shift = l;
  f.mul = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
  if (d == 1) {
    f.mul = 0;
    f.shift = 0;
  }
  return f;
}


// ------------------------------------------------------------------------------------
// Forward 3x3 convolution (pad 1, stride 1 or 2) of channels-last images: alpha-CROWN's
// gradient pass evaluates the relaxed network forward from each coefficient row's box vertex
// (every row is one image).  Implicit GEMM with M = rows x Ho^2 output positions, N = Co,
// K = 9 Ci (tap outer, 16 input channels per K tile), the same LDS tiling and MFMA blocking
// as the transposed convolution above; inputs with at most 4 channels (the network input)
// take a plain per-output kernel instead.

// One output element: D = acc + bias (+ residual), then the identity or the ReLU line
// selected by the recorded coefficient's sign (lam D where it is positive, s D + t where it
// is negative, s D where it is 0), with the slope gradient at unstable neurons.  ob, pb, rb:
// the element's row offsets into out (and alpha, pre, grad), P and res, without the channel.
__device__ __forceinline__ void fwd_apply(const FwdConvArgs &p, int64_t r, int64_t ob, int64_t pb, int64_t rb,
                                          int32_t n, float D) {
  if (p.res) D += p.res[rb + n];
  const int64_t off = ob + n;
  if (p.P) {
    float4 prm = p.P[pb + n];
    if (p.splits.D > 0) {   // subdomains (unit 0 only: pb + n is the neuron's index)
      int ent = -1;
      float sterm = 0.f;
      prm = split_override(p.splits, (int)r, p.relu_index, (int)(pb + n), prm, &ent, &sterm);
      if (ent >= 0 && p.splits.grad_beta) p.splits.grad_beta[r * p.splits.S + ent] = sterm * D;
    }
    // every load issued without waiting on the parameters (a stable neuron's lines all give
    // s D whatever its recorded coefficient, which the spec pass leaves at 0 there)
    const float al = p.alpha[off], an = p.pre[off];
    const bool unst = prm.z > 0.f;
    const float lam = unst ? al : prm.x;
    p.out[off] = an > 0.f ? lam * D : prm.y * D + (an < 0.f ? prm.z : 0.f);
    p.grad[off] = (unst && an > 0.f) ? an * D : 0.f;
  } else {
    p.out[off] = D;
  }
}

// row offsets of coefficient row r at output position pos
__device__ __forceinline__ void fwd_offsets(const FwdConvArgs &p, int64_t r, int32_t pos, int64_t *ob, int64_t *pb,
                                            int64_t *rb) {
  const int64_t q = (int64_t)pos * p.Co;
  int64_t u = 0;
  if (p.P) {
    u = r / p.rows_per_unit;
    u = u < p.units ? u : p.units - 1;
  }
  *ob = r * p.out_rs + q;
  *pb = u * ((int64_t)p.Ho * p.Ho * p.Co) + q;
  *rb = r * p.res_rs + q;
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256, 2) void k_fwd_conv(const FwdConvArgs p, FastDiv div_pos) {
  constexpr int BK = 16, CPR = BK / 4, TPR = CPR, RPP = 256 / TPR;
  constexpr int MB = BM / WM / 32, NB = BN / WN / 32;
  constexpr int QA = BM / RPP, QB = BN / RPP;
  __shared__ __attribute__((aligned(16))) float As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * BK];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int n_nt = (p.Co + BN - 1) / BN;
  const int mt = blockIdx.x / n_nt, nt = blockIdx.x - mt * n_nt;
  const int m0 = mt * BM, n0 = nt * BN;
  const int HW = p.Ho * p.Ho;
  const uint32_t Mtot = (uint32_t)p.rows * (uint32_t)HW;

  // operand tiles straight into LDS (global_load_lds): lane (row lrow, chunk slot tid % TPR)
  // fetches the logical chunk dcol that the swizzle puts into its slot
  constexpr int WROWS = 64 / TPR;
  // LDS byte addresses of this wave's first tile rows in stage 0 (M0 of its loads)
  const uint32_t a_lds = lds_addr(&As[0][0]) + (uint32_t)(wave * WROWS * BK * 4);
  const uint32_t b_lds = lds_addr(&Bs[0][0]) + (uint32_t)(wave * WROWS * BK * 4);
  static_assert(RPP % 16 == 0, "rows of one load pass share the swizzle");
  const int lrow = tid / TPR;
  const int dcol = ((tid % TPR) ^ lds_swz<BK>(lrow)) * 4;
  const float *a_row[QA];
  int yi0[QA], xi0[QA];
#pragma unroll
  for (int q = 0; q < QA; ++q) {
    const uint32_t m = (uint32_t)(m0 + lrow + RPP * q);
    const bool valid = m < Mtot;
    const uint32_t r = valid ? fdiv(m, div_pos) : 0u;
    const int pos = (int)(m - r * (uint32_t)HW);
    const int yo = pos / p.Ho, xo = pos - yo * p.Ho;
    a_row[q] = p.in + (int64_t)r * p.in_rs;
    yi0[q] = valid ? yo * p.stride - 1 : -(1 << 20);   // an invalid row reads zeros only
    xi0[q] = xo * p.stride - 1;
  }
  const float *b_row[QB];
#pragma unroll
  for (int q = 0; q < QB; ++q) {
    const int co = n0 + lrow + RPP * q;
    b_row[q] = co < p.Co ? p.Wk + (int64_t)co * 9 * p.Ci + dcol : nullptr;
  }
  const int cpt = p.Ci / BK;   // K tiles per tap
  // K order: pairs of 16-channel blocks (one 128-byte line of a position) outer, then the
  // tap, then the block of the pair, so a tile's shifted re-reads of a line follow each
  // other within a few K tiles (as in the transposed convolution)
  const bool pairs = cpt % 2 == 0;
  auto gload = [&](int kt, int buf) {
    int t, cb;
    if (pairs) {
      const int grp = kt / 18, rem = kt - grp * 18;
      t = rem >> 1;
      cb = 2 * grp + (rem & 1);
    } else {
      cb = kt / 9;
      t = kt - cb * 9;
    }
    const int c0 = cb * BK;
    const int ky = t / 3, kx = t - ky * 3;
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int yy = yi0[q] + ky, xx = xi0[q] + kx;
      const bool ok = (unsigned)yy < (unsigned)p.Hi && (unsigned)xx < (unsigned)p.Hi;
      const float *src = ok ? a_row[q] + ((int64_t)yy * p.Hi + xx) * p.Ci + c0 + dcol : g_zero4;
      dma16(src, a_lds + (uint32_t)(buf * (int)sizeof(As[0]) + RPP * q * BK * 4));
    }
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const float *src = b_row[q] ? b_row[q] + t * p.Ci + c0 : g_zero4;
      dma16(src, b_lds + (uint32_t)(buf * (int)sizeof(Bs[0]) + RPP * q * BK * 4));
    }
  };
  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  const int KT = 9 * cpt;
  gload(0, 0);
  const int r32 = lane & 31, sw = lds_swz<BK>(r32);
  int roff[CPR / 2];
#pragma unroll
  for (int h = 0; h < CPR / 2; ++h) roff[h] = ((((lane >> 5) * (CPR / 2)) + h) ^ sw) * 4;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    barrier_only();   // every wave is done with tile kt - 1: its stage is free
    if (kt + 1 < KT) {
      gload(kt + 1, cur ^ 1);
      wait_vmcnt<QA + QB>();   // this wave's part of tile kt has landed
    } else {
      wait_vmcnt<0>();
    }
    barrier_only();   // every wave's part of tile kt is in LDS
    const float *as = As[cur] + (wm * (BM / WM) + r32) * BK;
    const float *bs = Bs[cur] + (wn * (BN / WN) + r32) * BK;
#pragma unroll
    for (int h = 0; h < CPR / 2; ++h) {
      f32x4 a[MB], b[NB];
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = *reinterpret_cast<const f32x4 *>(as + i * 32 * BK + roff[h]);
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j] = *reinterpret_cast<const f32x4 *>(bs + j * 32 * BK + roff[h]);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
    }
  }
  __syncthreads();   // every wave is done with the operand buffers, which the epilogue reuses
  // epilogue: the offsets of every tile row once (a row per thread), through the free A
  // buffer; -1 marks rows past the end
  static_assert(28 * BM <= (int)sizeof(As), "row offsets must fit the A buffers");
  int64_t *s_ob = reinterpret_cast<int64_t *>(&As[0][0]);
  int64_t *s_pb = s_ob + BM;
  int64_t *s_rb = s_pb + BM;
  int *s_r = reinterpret_cast<int *>(s_rb + BM);
  for (int tr = tid; tr < BM; tr += 256) {
    const uint32_t m = (uint32_t)(m0 + tr);
    if (m < Mtot) {
      const uint32_t r = fdiv(m, div_pos);
      fwd_offsets(p, r, (int)(m - r * (uint32_t)HW), &s_ob[tr], &s_pb[tr], &s_rb[tr]);
      s_r[tr] = (int)r;
    } else {
      s_ob[tr] = -1;
    }
  }
  __syncthreads();
  const int half = lane >> 5;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int n = n0 + wn * (BN / WN) + j * 32 + r32;
    if (n >= p.Co) continue;
    const float bn = p.bias[n];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int lr = wm * (BM / WM) + i * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
        const int64_t ob = s_ob[lr];
        if (ob >= 0) fwd_apply(p, s_r[lr], ob, s_pb[lr], s_rb[lr], n, acc[i][j][v] + bn);
      }
  }
}

// Inputs with CIN <= 4 channels (the network input): a thread per output position and four
// consecutive output channels (its 9 CIN inputs loaded once for the four), the weights staged
// in LDS channels fastest, [tap][ci][Co], read as float4.  Workgroups take 256 such items of
// one row (blockIdx.x) and stride over the rows (blockIdx.y).
template <int CIN>
__global__ __launch_bounds__(256) void k_fwd_conv_small(const FwdConvArgs p) {
  extern __shared__ __attribute__((aligned(16))) float wl[];
  const int tid = threadIdx.x;
  for (int i = tid; i < 9 * CIN * p.Co; i += 256) {
    const int co = i % p.Co, k = i / p.Co;   // k = tap * CIN + ci
    wl[i] = p.Wk[(int64_t)co * 9 * CIN + k];
  }
  __syncthreads();
  const int HW = p.Ho * p.Ho, G = p.Co / 4;
  const int local = blockIdx.x * 256 + tid;
  if (local >= HW * G) return;
  const int pos = local / G, n0 = 4 * (local - pos * G);
  const int yo = pos / p.Ho, xo = pos - yo * p.Ho;
  const float4 bn = *reinterpret_cast<const float4 *>(p.bias + n0);
  for (int64_t r = blockIdx.y; r < p.rows; r += gridDim.y) {
    const float *x = p.in + r * p.in_rs;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int ky = 0; ky < 3; ++ky) {
      const int yy = yo * p.stride - 1 + ky;
      if ((unsigned)yy >= (unsigned)p.Hi) continue;
#pragma unroll
      for (int kx = 0; kx < 3; ++kx) {
        const int xx = xo * p.stride - 1 + kx;
        if ((unsigned)xx >= (unsigned)p.Hi) continue;
        const float *xs = x + (yy * p.Hi + xx) * CIN;
#pragma unroll
        for (int ci = 0; ci < CIN; ++ci) {
          const float xv = xs[ci];
          const float4 w = *reinterpret_cast<const float4 *>(&wl[((ky * 3 + kx) * CIN + ci) * p.Co + n0]);
          acc.x += xv * w.x;
          acc.y += xv * w.y;
          acc.z += xv * w.z;
          acc.w += xv * w.w;
        }
      }
    }
    int64_t ob, pb, rb;
    fwd_offsets(p, r, pos, &ob, &pb, &rb);
    fwd_apply(p, r, ob, pb, rb, n0, acc.x + bn.x);
    fwd_apply(p, r, ob, pb, rb, n0 + 1, acc.y + bn.y);
    fwd_apply(p, r, ob, pb, rb, n0 + 2, acc.z + bn.z);
    fwd_apply(p, r, ob, pb, rb, n0 + 3, acc.w + bn.w);
  }
}

hipError_t launch_fwd_conv(const FwdConvArgs &a, hipStream_t s) {
  if (a.rows <= 0 || a.Co <= 0 || a.Ci <= 0 || a.Hi <= 0 || (a.stride != 1 && a.stride != 2) ||
      a.Ho != (a.Hi - 1) / a.stride + 1 || !a.in || !a.Wk || !a.bias || !a.out)
    return hipErrorInvalidValue;
  if (a.P && (!a.alpha || !a.pre || !a.grad || a.rows_per_unit <= 0 || a.units <= 0 || a.res))
    return hipErrorInvalidValue;
  if (a.splits.D > 0 && (!a.P || a.units != 1 || a.splits.rows_per_domain <= 0)) return hipErrorInvalidValue;
  const int64_t HW = (int64_t)a.Ho * a.Ho;
  if (a.out_rs < HW * a.Co || a.in_rs < (int64_t)a.Hi * a.Hi * a.Ci || (a.res && a.res_rs < HW * a.Co))
    return hipErrorInvalidValue;
  if (a.Ci <= 4) {
    const size_t lds = sizeof(float) * 9 * (size_t)a.Ci * a.Co;
    if (lds > 65536 || HW * a.Co >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    if (a.Co % 4) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((HW * (a.Co / 4) + 255) / 256), (unsigned)std::min<int64_t>(a.rows, 256));
    switch (a.Ci) {
      case 1: hipLaunchKernelGGL(k_fwd_conv_small<1>, grid, dim3(256), lds, s, a); break;
      case 2: hipLaunchKernelGGL(k_fwd_conv_small<2>, grid, dim3(256), lds, s, a); break;
      case 3: hipLaunchKernelGGL(k_fwd_conv_small<3>, grid, dim3(256), lds, s, a); break;
      default: hipLaunchKernelGGL(k_fwd_conv_small<4>, grid, dim3(256), lds, s, a); break;
    }
    return hipGetLastError();
  }
  if (a.Ci % 16 || a.in_rs % 4) return hipErrorInvalidValue;   // 16-byte operand loads
  const int64_t M = (int64_t)a.rows * HW;
  if (M >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  const FastDiv dp = make_fastdiv((uint32_t)HW);
  if (a.Co % 128 == 0) {
    const int64_t blk = (M + 127) / 128 * (a.Co / 128);
    hipLaunchKernelGGL((k_fwd_conv<128, 128, 2, 2>), dim3((unsigned)blk), dim3(256), 0, s, a, dp);
  } else {
    const int64_t blk = (M + 255) / 256 * ((a.Co + 63) / 64);
    hipLaunchKernelGGL((k_fwd_conv<256, 64, 4, 1>), dim3((unsigned)blk), dim3(256), 0, s, a, dp);
  }
  return hipGetLastError();
}

__global__ void k_fwd_add(const float *x, int64_t xs, const float *y, int64_t ys, float *out, int64_t os,
                          int32_t rows, int64_t n) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)rows * n) return;
  const int64_t r = idx / n, i = idx - r * n;
  out[r * os + i] = x[r * xs + i] + y[r * ys + i];
}

hipError_t launch_fwd_add(const float *x, int64_t xs, const float *y, int64_t ys, float *out, int64_t os,
                          int32_t rows, int64_t n, hipStream_t s) {
  if (rows <= 0 || n <= 0) return hipSuccess;
  const int64_t tot = (int64_t)rows * n;
  hipLaunchKernelGGL(k_fwd_add, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, s, x, xs, y, ys, out, os, rows, n);
  return hipGetLastError();
}

}  // namespace vcr
