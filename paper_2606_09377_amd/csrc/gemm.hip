// fp32 MFMA GEMM of the CROWN backward step (paper, Sec. 2.1, equation "crown"; the
// per-layer step A <- A Lambda_i W_i of Sec. 3.3.2), with the next ReLU's relaxation and
// the bias accumulation fused into the epilogue.
//
// One launch computes, for coefficient rows A' (already relaxed for layer j) and the layer
// weight W_j (given transposed, Bt = W_j^T, so both operands are K-contiguous):
//
//   a   = (A' W_j)[row, n]                           coefficient on h_{j-1}, neuron n
//   EPI_RELAX      : a'  = a > 0 ? lam a : s a       lower rule of ReLU j-1 at neuron n
//                    out[row, n] = a'
//                    part[row] += min(a, 0) t + a' b_{j-1}[n]
//                    (the relaxation intercept and the next linear layer's bias, i.e. the
//                    constant terms this neuron adds to the bound)
//   EPI_CONCRETIZE : part[row] += a c[n] - |a| r[n]  (j = 1: minimum of a . x over the box
//                    with centre c and radius r); A_0 itself is never written
//   EPI_AFFINE     : out[row, n] = a + bias[n], with |Bt| instead of Bt when abs_b (the IBP
//                    step c' = W c + b, r' = |W| r on the matrix cores)
//   EPI_FORWARD    : out[row, n] = the relaxation line of ReLU k at D = a + b_k[n] chosen
//                    by the sign of the backward coefficient, and its alpha gradient
//                    (alpha-CROWN's gradient pass: A' = E_{k-1}, Bt = W_k)
//
// alpha-CROWN (Sec. 2.1) replaces lam by a per-row slope at unstable neurons and records the
// coefficients before relaxation; see kernels.h.
//
// Upper bounds run through the same code on negated rows (max f = -min(-f)).
//
// Tiling for gfx950: 256 threads = 4 wave64 in a 2 x 2 grid, each wave owns a 64 x 64
// block of the 128 x 128 tile as 2 x 2 v_mfma_f32_32x32x2f32 accumulators (64 fp32 each
// lane).  K advances 32 at a time through double-buffered LDS (rows padded to 36 floats so
// the 128-bit LDS reads of 8/16 consecutive lanes hit distinct banks).  Each lane consumes
// 16 consecutive k of its operand rows per K tile, so every MFMA operand comes from one
// 128-bit LDS read (the k order inside a tile is permuted identically for A and B, which
// leaves the contraction unchanged).  Partial sums per row are reduced over the 32 columns
// a lane group holds with a fixed butterfly, so results are deterministic and do not depend
// on which other rows share the tile.
#include "kernels.h"
#include "lds_dma.h"
#include "row_sums.h"
#include "splits.h"

namespace vcr {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int TPR = BK / 4;             // staging threads per tile row (one 16-byte chunk each)
constexpr int RPP = 256 / TPR;          // tile rows per staging pass
constexpr int SQ = 128 / RPP;           // staging passes per 128-row tile
constexpr int GEMM_MINB = BK == 32 ? 2 : 3;   // workgroups per CU the registers are sized for
constexpr int NTHREADS = 256;
constexpr int GROUP_M = 8;

__device__ __forceinline__ void map_tile(int bid, int G, int n_mt, int n_nt, int &mt, int &nt) {
  // Workgroup ids are spread over the 8 XCDs round robin; hand each XCD a contiguous range
  // of logical tiles so the tiles sharing operands also share that XCD's L2.
  const int x = bid & 7, t = bid >> 3;
  const int q = G >> 3, rem = G & 7;
  const int logical = x * q + min(x, rem) + t;
  // Grouped order: GROUP_M row blocks sweep every column tile together.
  const int per_group = GROUP_M * n_nt;
  const int g = logical / per_group;
  const int first_m = g * GROUP_M;
  const int gm = min(GROUP_M, n_mt - first_m);
  const int idx = logical - g * per_group;
  mt = first_m + idx % gm;
  nt = idx / gm;
}


// Split lookups of one tile through LDS: flags[d - d0][n - n0] is the entry index of
// (domain d, neuron n) at this ReLU, or -1.  All threads of the workgroup build it once, so
// the per-element lookup is one LDS read instead of a walk over the domain's entries in
// global memory.  Tiles spanning more than SPLIT_ND domains keep the global walk.
constexpr int SPLIT_ND = 16;
struct TileSplits {
  const signed char *flags;   // null: look up in global memory
  int d0, n0, cols;
};

__device__ __forceinline__ TileSplits tile_splits_build(const SplitTable &st, int relu, int m0, int tile_rows,
                                                        int n0, int cols, signed char *lds) {
  TileSplits t{nullptr, 0, n0, cols};
  if (st.D <= 0 || !lds) return t;   // uniform over the workgroup
  const int d0 = min(m0 / st.rows_per_domain, st.D - 1);
  const int d1 = min((m0 + tile_rows - 1) / st.rows_per_domain, st.D - 1);
  const int nd = d1 - d0 + 1;
  if (nd > SPLIT_ND) return t;
  for (int i = threadIdx.x; i < nd * cols; i += blockDim.x) lds[i] = -1;
  __syncthreads();
  for (int i = threadIdx.x; i < nd * st.S; i += blockDim.x) {
    const int dl = i / st.S, e = i - dl * st.S, d = d0 + dl;
    const int e0 = st.off[d * (st.R + 1) + relu], e1 = st.off[d * (st.R + 1) + relu + 1];
    if (e >= e0 && e < e1) {
      const int n = st.ent_n[d * st.S + e];
      if (n >= n0 && n < n0 + cols) lds[dl * cols + (n - n0)] = (signed char)e;
    }
  }
  __syncthreads();
  t.flags = lds;
  t.d0 = d0;
  return t;
}

// split_override through the tile's table when there is one (the same entry, so the same
// parameters)
__device__ __forceinline__ float4 split_lookup(const SplitTable &st, const TileSplits &t, int row, int relu, int n,
                                               float4 prm, int *ent = nullptr, float *sterm = nullptr) {
  if (!t.flags) return split_override(st, row, relu, n, prm, ent, sterm);
  int d = row / st.rows_per_domain;
  d = d < st.D ? d : st.D - 1;
  const int e = t.flags[(d - t.d0) * t.cols + (n - t.n0)];
  if (e >= 0) {
    const float4 q = st.ent_p[d * st.S + e];
    prm.x = q.x;
    prm.y = q.y;
    prm.z = q.z;
    if (ent) {
      *ent = e;
      *sterm = q.w;
    }
  }
  return prm;
}

// Epilogue of one wave: MB blocks of 32 rows from tile-relative row wrow of the tile at m0
// (tile_rows high), 64 columns from col0 (one partial sum per row and 64 columns, so every
// tiling gives the same bits), accumulators acc[MB][2].
//
// NBJ = 1: the wave holds only column block bj1 (0 or 1) of the 64; the two waves of the
// workgroup combine their row sums through xpart (LDS, 16 x 64 floats) in the order a wave
// holding both blocks uses, so the bits do not change.
//
// The arrays the epilogue reads and writes arrive as restrict-qualified parameters of the body,
// so the compiler may issue the loads of later rows before the stores of earlier ones.
template <bool FWD, bool AL, bool AFF, int MB, int NBJ>
__device__ __forceinline__ void gemm_epilogue_body(const GemmArgs &p, f32x16 (&acc)[MB][NBJ], int m0, int wrow,
                                                   int col0, int lane, int tile_rows, int bj1, float *xpart,
                                                   const float4 *__restrict__ Pp, const float *__restrict__ c0p,
                                                   const float *__restrict__ r0p, const float *__restrict__ alpha_t,
                                                   float *__restrict__ pre_t, float *__restrict__ out_t,
                                                   float *__restrict__ grad_t, const float *__restrict__ sbeta,
                                                   float *__restrict__ gbeta, const float *__restrict__ biasp,
                                                   float *__restrict__ partp, const TileSplits &ts) {
  const int r32 = lane & 31;
  // 32x32 accumulator layout: lane holds column (lane % 32) and rows
  // 8 (v / 4) + 4 (lane / 32) + (v % 4), v = 0..15.
  const int half = lane >> 5;
  const bool uniform_unit = (p.rows_per_unit % tile_rows) == 0;
  int unit_tile = m0 / p.rows_per_unit;
  unit_tile = unit_tile < p.n_units ? unit_tile : p.n_units - 1;
  const bool has_splits = p.splits.D > 0;

  const int ld32 = (int)(p.mode == EPI_CONCRETIZE ? p.ld_pre : p.ldo);

  float rp[MB][16];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) rp[i][v] = 0.f;

  if constexpr (AFF) {
    // plain affine map (the IBP step on the matrix cores): out = A Bt^T (+ bias)
#pragma unroll
    for (int jj = 0; jj < NBJ; ++jj) {
      const int bj = NBJ == 2 ? jj : bj1;
      const int n = col0 + bj * 32 + r32;
      const float bn = biasp ? biasp[n] : 0.f;
#pragma unroll
      for (int bi = 0; bi < MB; ++bi)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int lr = wrow + bi * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
          out_t[lr * ld32 + n] = acc[bi][jj][v] + bn;
        }
    }
    return;
  }
#pragma unroll
  for (int jj = 0; jj < NBJ; ++jj) {
    const int bj = NBJ == 2 ? jj : bj1;
    const int n = col0 + bj * 32 + r32;
    if constexpr (FWD) {
      // the relaxed network evaluated forward: D = W_k E + b_k, then the line of ReLU k that
      // the backward pass chose for this row (by the sign of its coefficient)
      float4 prm_tile = make_float4(0.f, 0.f, 0.f, 0.f);
      if (uniform_unit) prm_tile = Pp[(int64_t)unit_tile * p.ldp + n];
#pragma unroll
      for (int bi = 0; bi < MB; ++bi) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int lr = wrow + bi * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
          const int row = m0 + lr;
          const int off = lr * ld32 + n;
          float4 prm = prm_tile;
          if (!uniform_unit) {
            int u = row / p.rows_per_unit;
            u = u < p.n_units ? u : p.n_units - 1;
            prm = Pp[(int64_t)u * p.ldp + n];
          }
          int ent = -1;
          float sterm = 0.f;
          if (has_splits) prm = split_lookup(p.splits, ts, row, p.relu_index, n, prm, &ent, &sterm);
          const bool unst = prm.z > 0.f;
          const float al = alpha_t[off];   // loaded for every row: no load waits on prm
          const float lam = unst ? al : prm.x;
          const float an = pre_t[off];
          const float D = acc[bi][jj][v] + prm.w;
          if (ent >= 0 && gbeta) gbeta[(int64_t)row * p.splits.S + ent] = sterm * D;
          const float E = an > 0.f ? lam * D : prm.y * D + (an < 0.f ? prm.z : 0.f);
          out_t[off] = E;
          grad_t[off] = (unst && an > 0.f) ? an * D : 0.f;
        }
      }
    } else if (p.mode == EPI_RELAX) {
      float4 prm_tile = make_float4(0.f, 0.f, 0.f, 0.f);
      if (uniform_unit) prm_tile = Pp[(int64_t)unit_tile * p.ldp + n];
#pragma unroll
      for (int bi = 0; bi < MB; ++bi) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int lr = wrow + bi * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
          const int row = m0 + lr;
          const int off = lr * ld32 + n;
          float4 prm = prm_tile;
          if (!uniform_unit) {
            int u = row / p.rows_per_unit;
            u = u < p.n_units ? u : p.n_units - 1;
            prm = Pp[(int64_t)u * p.ldp + n];
          }
          int ent = -1;
          float sterm = 0.f;
          if (has_splits) {
            if constexpr (AL)
              prm = split_lookup(p.splits, ts, row, p.relu_index, n, prm, &ent, &sterm);
            else
              prm = split_lookup(p.splits, ts, row, p.relu_index, n, prm);
          }
          const float a = acc[bi][jj][v];
          float lam = prm.x;
          if constexpr (AL) {
            if (alpha_t) {
              const float al = alpha_t[off];
              lam = prm.z > 0.f ? al : lam;
            }
          }
          float ap = a > 0.f ? a * lam : a * prm.y;
          if constexpr (AL) {
            if (ent >= 0 && sbeta) ap += sbeta[(int64_t)row * p.splits.S + ent] * sterm;
          }
          out_t[off] = ap;
          if constexpr (AL) {
            if (pre_t) pre_t[off] = a;
          }
          rp[bi][v] += fminf(a, 0.f) * prm.z + ap * prm.w;
        }
      }
    } else {
      float c_tile = 0.f, r_tile = 0.f;
      if (uniform_unit) {
        c_tile = c0p[(int64_t)unit_tile * p.ldc + n];
        r_tile = r0p[(int64_t)unit_tile * p.ldc + n];
      }
#pragma unroll
      for (int bi = 0; bi < MB; ++bi) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int lr = wrow + bi * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
          const int row = m0 + lr;
          float c = c_tile, r = r_tile;
          if (!uniform_unit) {
            int u = row / p.rows_per_unit;
            u = u < p.n_units ? u : p.n_units - 1;
            c = c0p[(int64_t)u * p.ldc + n];
            r = r0p[(int64_t)u * p.ldc + n];
          }
          const float a = acc[bi][jj][v];
          if constexpr (AL) {
            if (pre_t) pre_t[lr * ld32 + n] = a;
          }
          rp[bi][v] += a * c - fabsf(a) * r;
        }
      }
    }
  }

  if constexpr (FWD) return;
  if constexpr (NBJ == 1) {
    if (bj1 == 1) {
#pragma unroll
      for (int v = 0; v < 16; ++v) xpart[v * 64 + lane] = rp[0][v];
    }
    __syncthreads();
    if (bj1 == 1) return;
#pragma unroll
    for (int v = 0; v < 16; ++v) rp[0][v] += xpart[v * 64 + lane];
  }
  // fixed butterfly over the 32 lanes that share rows (as a reduce-scatter: lane 2 v ends
  // with row v's sum)
  float *dst = partp + (int64_t)(col0 / PART_COLS) * p.M_pad;
  const int v = r32 >> 1;
#pragma unroll
  for (int bi = 0; bi < MB; ++bi) {
    const float x = half_wave_row_sums(rp[bi], r32);
    if ((r32 & 1) == 0) dst[m0 + wrow + bi * 32 + (v >> 2) * 8 + half * 4 + (v & 3)] = x;
  }
}

// Stores and row-wise loads address the tile from a wave-uniform base with 32-bit lane offsets
// (every row-indexed array of one launch shares the pitch ld).
// tn0, tcols: the workgroup tile's first column and width; sflag: free LDS for the tile's
// split table (SPLIT_ND x tcols bytes), or null.  Every thread of the workgroup calls this.
template <bool FWD, bool AL, bool AFF, int MB, int NBJ = 2>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs &p, f32x16 (&acc)[MB][NBJ], int m0, int wrow, int col0,
                                              int lane, int tile_rows, int bj1, float *xpart, int tn0, int tcols,
                                              signed char *sflag) {
  const int64_t ld = p.mode == EPI_CONCRETIZE ? p.ld_pre : p.ldo;
  const int64_t tbase = (int64_t)m0 * ld;
  TileSplits ts{nullptr, 0, tn0, tcols};
  if (!AFF && p.mode != EPI_CONCRETIZE) ts = tile_splits_build(p.splits, p.relu_index, m0, tile_rows, tn0, tcols, sflag);
  gemm_epilogue_body<FWD, AL, AFF, MB, NBJ>(
      p, acc, m0, wrow, col0, lane, tile_rows, bj1, xpart, p.P, p.c0, p.r0, p.alpha ? p.alpha + tbase : nullptr,
      p.pre ? p.pre + tbase : nullptr, p.mode == EPI_CONCRETIZE ? nullptr : p.out + tbase,
      p.grad ? p.grad + tbase : nullptr, p.splits.beta, p.splits.grad_beta, p.bias, p.part, ts);
}

// Instantiations: FWD selects the forward epilogue (alpha-CROWN's gradient pass); otherwise the
// relax and concretize epilogues share one kernel and the mode is read at run time (this keeps
// the register allocation of the relax epilogue spill-free).  AL adds the alpha-CROWN extras
// (per-row slopes, stored coefficients) to the backward epilogues.
template <bool FWD, bool AL, bool AFF = false>
__global__ __launch_bounds__(NTHREADS, GEMM_MINB) void k_gemm(const GemmArgs p) {
  __shared__ __attribute__((aligned(16))) float As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * BK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n_mt = p.M_pad / BM, n_nt = p.N_pad / BN;
  int mt, nt;
  map_tile(blockIdx.x, n_mt * n_nt, n_mt, n_nt, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;

  // Operand tiles go from global memory straight into LDS (rows unpadded, chunks swizzled by
  // lds_swz): one load of a wave fills 64 / TPR whole rows, lane order, so lane (row lrow,
  // chunk slot tid % TPR) fetches the logical chunk that the swizzle puts into its slot (the
  // same for the rows lrow + RPP q, the swizzle repeating every 16 rows)
  static_assert(RPP % 16 == 0, "rows of one load pass share the swizzle");
  constexpr int WROWS = 64 / TPR;
  const int lrow = tid / TPR;
  const int dcol = ((tid % TPR) ^ lds_swz<BK>(lrow)) * 4;
  const float *Ag = p.A + (int64_t)(m0 + lrow) * p.lda + dcol;
  const float *Bg = p.Bt + (int64_t)(n0 + lrow) * p.ldb + dcol;
  const int64_t a_step = RPP * p.lda, b_step = RPP * p.ldb;
  auto issue = [&](int kt, int buf) {
    const int k0 = kt * BK;
#pragma unroll
    for (int q = 0; q < SQ; ++q) {
      dma16(Ag + q * a_step + k0, &As[buf][(wave * WROWS + RPP * q) * BK]);
      dma16(Bg + q * b_step + k0, &Bs[buf][(wave * WROWS + RPP * q) * BK]);
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // lane (r32, half) reads the 16 consecutive k half * 16 .. + 15 of its row: logical chunks
  // half * 4 + h, h < 4 (rows r32 and r32 + 32 of a 64-row block share the swizzle)
  const int r32 = lane & 31, sw = lds_swz<BK>(r32);
  int roff[BK / 8];
#pragma unroll
  for (int h = 0; h < BK / 8; ++h) roff[h] = ((((lane >> 5) * (BK / 8)) + h) ^ sw) * 4;
  const int a_off0 = (wm * 64 + r32) * BK;
  const int a_off1 = a_off0 + 32 * BK;
  const int b_off0 = (wn * 64 + r32) * BK;
  const int b_off1 = b_off0 + 32 * BK;

  const int KT = p.K / BK;
  issue(0, 0);
  static_assert(SQ == BK / 8, "one load pass per operand read step");
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    wait_vmcnt<0>();
    barrier_only();   // every wave's part of tile kt is in LDS; the other stage is free
    const bool more = kt + 1 < KT;
    const int k1 = (kt + 1) * BK;
    const float *as = As[cur];
    const float *bs = Bs[cur];
#pragma unroll
    for (int h = 0; h < BK / 8; ++h) {
      const f32x4 a0 = *reinterpret_cast<const f32x4 *>(as + a_off0 + roff[h]);
      const f32x4 a1 = *reinterpret_cast<const f32x4 *>(as + a_off1 + roff[h]);
      f32x4 b0 = *reinterpret_cast<const f32x4 *>(bs + b_off0 + roff[h]);
      f32x4 b1 = *reinterpret_cast<const f32x4 *>(bs + b_off1 + roff[h]);
      if (more) {   // the next tile's loads spread over the MFMA steps, one pass per step
        dma16(Ag + h * a_step + k1, &As[cur ^ 1][(wave * WROWS + RPP * h) * BK]);
        dma16(Bg + h * b_step + k1, &Bs[cur ^ 1][(wave * WROWS + RPP * h) * BK]);
      }
      if constexpr (AFF) {
        if (p.abs_b) {
          b0 = __builtin_elementwise_abs(b0);
          b1 = __builtin_elementwise_abs(b1);
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[e], b0[e], acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[e], b1[e], acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[e], b0[e], acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[e], b1[e], acc[1][1], 0, 0, 0);
      }
    }
  }
  __syncthreads();   // every wave is done with the operand buffers, which the epilogue reuses

  // ---- epilogue ---------------------------------------------------------------------
  gemm_epilogue<FWD, AL, AFF, 2>(p, acc, m0, wm * 64, n0 + wn * 64, lane, BM, 0, nullptr, n0, BN,
                                 reinterpret_cast<signed char *>(&As[0][0]));
}

// Small launches (few row tiles): a workgroup of two waves owns a 32 x 64 tile, each wave one
// 32-column block, and reads its MFMA operands straight from global memory (no LDS operand
// staging), K tiles in a ring of four register sets (three in flight).  Each lane takes the same 16 consecutive k of
// its row per K tile as in k_gemm, each accumulator sees the same MFMA sequence, and the row
// sums of the two blocks are added in k_gemm's order, so both kernels give the same bits.
constexpr int SM_BM = 32, SM_BN = 64;
constexpr int64_t SMALL_GRID = 512;   // 128 x 128 tiles below which the small kernel runs

template <bool FWD, bool AL, bool AFF = false>
__global__ __launch_bounds__(128) void k_gemm_small(const GemmArgs p) {
  __shared__ float xpart[16 * 64];
  __shared__ signed char sflag[SPLIT_ND * SM_BN];
  const int lane = threadIdx.x & 63, bj = threadIdx.x >> 6;
  const int n_mt = p.M_pad / SM_BM, n_nt = p.N_pad / SM_BN;
  int mt, nt;
  map_tile(blockIdx.x, n_mt * n_nt, n_mt, n_nt, mt, nt);
  const int m0 = mt * SM_BM, n0 = nt * SM_BN;
  const int r32 = lane & 31, kq = (lane >> 5) * (BK / 2);
  const float *Ag = p.A + (int64_t)(m0 + r32) * p.lda + kq;
  const float *Bg = p.Bt + (int64_t)(n0 + bj * 32 + r32) * p.ldb + kq;
  f32x16 acc[1][1];
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[0][0][v] = 0.f;
  const int KT_LAST = p.K / BK - 1;   // >= 0: launch_gemm requires K > 0, a multiple of BK
  // K tiles in a ring of four register sets (three in flight while one is multiplied): a
  // lone wave per tile has no other way to hide the latency.  The ring is unrolled (no copies
  // between sets, which would wait for every load in flight) and every request is
  // unconditional, past the last tile repeating it (cache hits, never multiplied), so each
  // multiply waits for its own tile only.
  typedef f32x4 KSet[2][BK / 8];   // [0]: A, [1]: B
  auto load = [&](int kt, KSet &r) {
    const int k0 = min(kt, KT_LAST) * BK;
#pragma unroll
    for (int h = 0; h < BK / 8; ++h) {
      r[0][h] = *reinterpret_cast<const f32x4 *>(Ag + k0 + 4 * h);
      r[1][h] = *reinterpret_cast<const f32x4 *>(Bg + k0 + 4 * h);
    }
  };
  auto mma = [&](KSet &r) {
#pragma unroll
    for (int h = 0; h < BK / 8; ++h) {
      f32x4 bb = r[1][h];
      if constexpr (AFF) {
        if (p.abs_b) bb = __builtin_elementwise_abs(bb);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(r[0][h][e], bb[e], acc[0][0], 0, 0, 0);
    }
  };
  KSet s0, s1, s2, s3;
  load(0, s0);
  load(1, s1);
  load(2, s2);
  // opaque copies: otherwise the loop head merges these loads with the loop's (a phi of loads
  // becomes a load of a phi), which undoes the ring
#pragma unroll
  for (int h = 0; h < BK / 8; ++h) asm volatile("" : "+v"(s0[0][h]), "+v"(s0[1][h]), "+v"(s1[0][h]), "+v"(s1[1][h]), "+v"(s2[0][h]), "+v"(s2[1][h]));
  // whole rounds of four tiles (no exit inside a round: the loop head then knows which loads
  // are in flight), then the last one to three tiles, already requested
  const int KT = KT_LAST + 1;
  int kt = 0;
  for (; kt + 4 <= KT; kt += 4) {
    load(kt + 3, s3);
    __builtin_amdgcn_sched_barrier(0);
    mma(s0);
    __builtin_amdgcn_sched_barrier(0);
    load(kt + 4, s0);
    __builtin_amdgcn_sched_barrier(0);
    mma(s1);
    __builtin_amdgcn_sched_barrier(0);
    load(kt + 5, s1);
    __builtin_amdgcn_sched_barrier(0);
    mma(s2);
    __builtin_amdgcn_sched_barrier(0);
    load(kt + 6, s2);
    __builtin_amdgcn_sched_barrier(0);
    mma(s3);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (kt < KT) mma(s0);
  if (kt + 1 < KT) mma(s1);
  if (kt + 2 < KT) mma(s2);
  gemm_epilogue<FWD, AL, AFF, 1, 1>(p, acc, m0, 0, n0, lane, SM_BM, bj, xpart, n0, SM_BN, sflag);
}

// Mid-size launches (fewer than MID_MAX_GRID 128 x 128 tiles, at least MID_GRID 64 x 64 ones):
// 64 x 64 tiles staged
// through double-buffered LDS like k_gemm, four waves of 32 x 32.  Each accumulator sees
// k_gemm's MFMA sequence and the two column waves of a row block add their row sums in
// k_gemm's order (through LDS), so the bits are k_gemm's; the operands cross the L2 half as
// often as in the small-tile kernel.
constexpr int MD_BM = 64, MD_BN = 64;
constexpr int64_t MID_GRID = 256;   // 64 x 64 tiles from which the mid-size kernel runs
// It also runs instead of k_gemm below MID_MAX_GRID 128 x 128 tiles when the last of k_gemm's
// rounds of 512 workgroups (what fits the chip) would be at most half full (576 tiles: a
// second round of 64): four times as many 64 x 64 tiles fill the chip evenly.  Whole or
// nearly whole rounds stay on k_gemm, which is faster per tile.
constexpr int64_t MID_MAX_GRID = 1536;
constexpr int64_t GEMM_ROUND = 512;

template <bool FWD, bool AL, bool AFF = false>
__global__ __launch_bounds__(256) void k_gemm_mid(const GemmArgs p) {
  __shared__ __attribute__((aligned(16))) float As[2][MD_BM * BK];
  __shared__ __attribute__((aligned(16))) float Bs[2][MD_BN * BK];
  __shared__ float xpart[2][16 * 64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int n_mt = p.M_pad / MD_BM, n_nt = p.N_pad / MD_BN;
  int mt, nt;
  map_tile(blockIdx.x, n_mt * n_nt, n_mt, n_nt, mt, nt);
  const int m0 = mt * MD_BM, n0 = nt * MD_BN;

  // operand tiles straight into LDS as in k_gemm (rows unpadded, chunks swizzled by lds_swz;
  // lane (row lrow, chunk slot tid % TPR) fetches the chunk that lands in its slot)
  constexpr int MQ = MD_BM / RPP;
  constexpr int WROWS = 64 / TPR;
  const int lrow = tid / TPR;
  const int dcol = ((tid % TPR) ^ lds_swz<BK>(lrow)) * 4;
  const float *Ag = p.A + (int64_t)(m0 + lrow) * p.lda + dcol;
  const float *Bg = p.Bt + (int64_t)(n0 + lrow) * p.ldb + dcol;
  const int64_t a_step = RPP * p.lda, b_step = RPP * p.ldb;
  auto issue = [&](int kt, int buf) {
    const int k0 = kt * BK;
#pragma unroll
    for (int q = 0; q < MQ; ++q) {
      dma16(Ag + q * a_step + k0, &As[buf][(wave * WROWS + RPP * q) * BK]);
      dma16(Bg + q * b_step + k0, &Bs[buf][(wave * WROWS + RPP * q) * BK]);
    }
  };

  f32x16 acc[1][1];
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[0][0][v] = 0.f;
  const int KT = p.K / BK;
  // lane (r32, half) reads k half * 16 .. + 15 of its row (logical chunks half * 4 + h)
  const int r32 = lane & 31, sw = lds_swz<BK>(r32);
  int roff[BK / 8];
#pragma unroll
  for (int h = 0; h < BK / 8; ++h) roff[h] = ((((lane >> 5) * (BK / 8)) + h) ^ sw) * 4;
  const int a_off = (wm * 32 + r32) * BK, b_off = (wn * 32 + r32) * BK;
  issue(0, 0);
  static_assert(MQ <= BK / 8, "the load passes fit the operand read steps");
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    wait_vmcnt<0>();
    barrier_only();   // every wave's part of tile kt is in LDS; the other stage is free
    const bool more = kt + 1 < KT;
    const int k1 = (kt + 1) * BK;
#pragma unroll
    for (int h = 0; h < BK / 8; ++h) {
      const f32x4 a = *reinterpret_cast<const f32x4 *>(As[cur] + a_off + roff[h]);
      f32x4 b = *reinterpret_cast<const f32x4 *>(Bs[cur] + b_off + roff[h]);
      if (more && h < MQ) {   // the next tile's loads spread over the MFMA steps
        dma16(Ag + h * a_step + k1, &As[cur ^ 1][(wave * WROWS + RPP * h) * BK]);
        dma16(Bg + h * b_step + k1, &Bs[cur ^ 1][(wave * WROWS + RPP * h) * BK]);
      }
      if constexpr (AFF) {
        if (p.abs_b) b = __builtin_elementwise_abs(b);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[e], b[e], acc[0][0], 0, 0, 0);
    }
  }
  __syncthreads();   // every wave is done with the operand buffers, which the epilogue reuses
  gemm_epilogue<FWD, AL, AFF, 1, 1>(p, acc, m0, wm * 32, n0, lane, MD_BM, wn, xpart[wm], n0, MD_BN,
                                    reinterpret_cast<signed char *>(&As[0][0]));
}

int gemm_kind(const GemmArgs &a) {
  if (a.M_pad <= 0 || a.N_pad <= 0) return 0;
  const int64_t grid = (int64_t)(a.M_pad / BM) * (a.N_pad / BN);
  const int64_t mid = (int64_t)(a.M_pad / MD_BM) * (a.N_pad / MD_BN);
  const int64_t last = grid % GEMM_ROUND;
  const bool ragged = grid < MID_MAX_GRID && last > 0 && last <= GEMM_ROUND / 2;
  if ((grid < SMALL_GRID || ragged) && mid >= MID_GRID) return 3;
  return grid < SMALL_GRID ? 2 : 0;
}

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s) {
  if (a.M_pad % BM || a.N_pad % BN || a.K % BK || a.K <= 0 || a.M_pad <= 0 || a.N_pad <= 0)
    return hipErrorInvalidValue;
  // the epilogue's row-indexed arrays share one pitch and use 32-bit offsets within a tile
  const int64_t ld = a.mode == EPI_CONCRETIZE ? a.ld_pre : a.ldo;
  if (a.mode != EPI_CONCRETIZE && ((a.alpha && a.ld_alpha != a.ldo) || (a.pre && a.ld_pre != a.ldo)))
    return hipErrorInvalidValue;
  if (a.mode == EPI_FORWARD && (!a.alpha || !a.pre || !a.grad || !a.out)) return hipErrorInvalidValue;
  if (a.mode == EPI_AFFINE && (!a.out || a.alpha || a.pre)) return hipErrorInvalidValue;
  if ((int64_t)BM * ld + a.N_pad >= ((int64_t)1 << 31) || (ld < a.N_pad && (a.mode != EPI_CONCRETIZE || a.pre)))
    return hipErrorInvalidValue;
  const int64_t grid = (int64_t)(a.M_pad / BM) * (a.N_pad / BN);
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  const bool al = a.alpha || a.pre;
  if (a.mode != EPI_RELAX && a.mode != EPI_CONCRETIZE && a.mode != EPI_FORWARD && a.mode != EPI_AFFINE)
    return hipErrorInvalidValue;
  const int64_t mid = (int64_t)(a.M_pad / MD_BM) * (a.N_pad / MD_BN);
  if (gemm_kind(a) == 3) {
    // too few 128 x 128 tiles to fill the chip, enough of 64 x 64 (same bits)
    const dim3 g((unsigned)mid), t(256);
    if (a.mode == EPI_AFFINE)
      hipLaunchKernelGGL((k_gemm_mid<false, false, true>), g, t, 0, s, a);
    else if (a.mode == EPI_FORWARD)
      hipLaunchKernelGGL((k_gemm_mid<true, true>), g, t, 0, s, a);
    else if (al)
      hipLaunchKernelGGL((k_gemm_mid<false, true>), g, t, 0, s, a);
    else
      hipLaunchKernelGGL((k_gemm_mid<false, false>), g, t, 0, s, a);
    return hipGetLastError();
  }
  if (grid < SMALL_GRID) {
    // too few tiles of either size: 32 x 64 tiles, two waves each (same bits)
    const int64_t sg = (int64_t)(a.M_pad / SM_BM) * (a.N_pad / SM_BN);
    const dim3 g((unsigned)sg), t(128);
    if (a.mode == EPI_AFFINE)
      hipLaunchKernelGGL((k_gemm_small<false, false, true>), g, t, 0, s, a);
    else if (a.mode == EPI_FORWARD)
      hipLaunchKernelGGL((k_gemm_small<true, true>), g, t, 0, s, a);
    else if (al)
      hipLaunchKernelGGL((k_gemm_small<false, true>), g, t, 0, s, a);
    else
      hipLaunchKernelGGL((k_gemm_small<false, false>), g, t, 0, s, a);
    return hipGetLastError();
  }
  const dim3 g((unsigned)grid), t(NTHREADS);
  if (a.mode == EPI_AFFINE)
    hipLaunchKernelGGL((k_gemm<false, false, true>), g, t, 0, s, a);
  else if (a.mode == EPI_FORWARD)
    hipLaunchKernelGGL((k_gemm<true, true>), g, t, 0, s, a);
  else if (al)
    hipLaunchKernelGGL((k_gemm<false, true>), g, t, 0, s, a);
  else
    hipLaunchKernelGGL((k_gemm<false, false>), g, t, 0, s, a);
  return hipGetLastError();
}

}  // namespace vcr
