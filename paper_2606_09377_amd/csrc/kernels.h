// Internal launch interface of the vcrown HIP kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vcr {

// GEMM tile: BM x BN output per workgroup, BK deep K steps; every padded width is a
// multiple of LD_ALIGN so a padded row is whole tiles in both the K and the N role.
constexpr int BM = 128;
constexpr int BN = 128;
constexpr int BK = 32;
constexpr int LD_ALIGN = 128;
constexpr int PART_COLS = 64;   // columns summed into one bias partial (one wave's slab)

inline int64_t ld_of(int64_t n) { return (n + LD_ALIGN - 1) / LD_ALIGN * LD_ALIGN; }
inline int64_t rows_pad(int64_t m) { return (m + BM - 1) / BM * BM; }

// Per-domain ReLU overrides for branch-and-bound subdomains, built on the device.
struct SplitTable {
  const int32_t *off = nullptr;   // [D][R+1] start of each ReLU's entries in ent_*
  const int32_t *ent_n = nullptr; // [D][S] neuron of each entry (sorted by ReLU)
  const float4 *ent_p = nullptr;  // [D][S] (lam, s, t, S) after the split is applied; S = -1 for
                                  // an active split (z >= 0), +1 for an inactive one (z <= 0)
  int32_t R = 0, S = 0, D = 0;
  int32_t rows_per_domain = 0;
  // beta-CROWN (optional): per-row multipliers of the entries, beta[row * S + e] >= 0; the
  // term beta S z of each split is added to the coefficient of z; in the forward epilogue
  // grad_beta[row * S + e] receives S z at the row's vertex
  const float *beta = nullptr;
  float *grad_beta = nullptr;
};

enum EpiMode : int32_t { EPI_RELAX = 0, EPI_CONCRETIZE = 1, EPI_FORWARD = 2, EPI_AFFINE = 3 };

struct GemmArgs {
  const float *A;      // M_pad x lda, coefficient rows (already relaxed), zero padded
  const float *Bt;     // N_pad x ldb, the layer weight transposed, zero padded
  int64_t lda, ldb;
  int32_t M;           // real rows (rows >= M are padding)
  int32_t M_pad;       // multiple of BM
  int32_t K;           // multiple of BK (padded)
  int32_t N_pad;       // multiple of BN
  int32_t mode;        // EpiMode
  // relax epilogue: out = relax(A Bt^T) with the per-unit parameters of the next ReLU
  float *out;
  int64_t ldo;
  const float4 *P;     // [units][ldp] (lam, s, t, bias of the layer below)
  int64_t ldp;
  int32_t relu_index;  // which ReLU the parameters belong to (split lookup)
  SplitTable splits;   // D == 0: no splits
  // concretize epilogue: partial sums of a.c - |a|.r per row
  const float *c0, *r0;
  int64_t ldc;
  int32_t rows_per_unit;   // rows of one input (intermediate: 2 n_k; final: 2 m)
  int32_t n_units;         // number of inputs that own rows (clamp for padding rows)
  float *part;             // [N_pad / PART_COLS][M_pad] per-row partial sums (null: EPI_FORWARD)
  // alpha-CROWN (all optional):
  //   alpha [M_pad][ld_alpha]: per-row lower slope of the ReLU relaxed in the epilogue, used
  //   at its unstable neurons (t > 0) instead of lam;
  //   pre [M_pad][ld_pre]: receives the coefficient a before relaxation (EPI_RELAX,
  //   EPI_CONCRETIZE); in EPI_FORWARD it is read: the sign of the coefficient on the ReLU's
  //   output that selected its line;
  //   EPI_FORWARD: D = (A Bt^T)[row, n] + b (P.w), out = the selected line at D
  //   (a > 0: lam D; else s D, plus t when a < 0), grad [M_pad][ld_alpha] = a D at
  //   unstable neurons with a > 0, else 0.
  const float *alpha;
  int64_t ld_alpha;
  float *pre;
  int64_t ld_pre;
  float *grad;
  // EPI_AFFINE: out = A Bt^T + bias (bias [N_pad] or null), Bt taken elementwise-absolute
  // when abs_b (IBP: c' = W c + b, r' = |W| r)
  const float *bias;
  int32_t abs_b;
};

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s);
// The kernel launch_gemm runs for these arguments: 0 k_gemm, 2 k_gemm_small, 3 k_gemm_mid.
int gemm_kind(const GemmArgs &a);

// ---- bandwidth-bound kernels -------------------------------------------------------
hipError_t launch_fill(float *p, int64_t n, float v, hipStream_t s);
hipError_t launch_transpose_pad(const float *W, int32_t rows, int32_t cols, float *Wt, int64_t ldt,
                                int64_t rows_t, hipStream_t s);
hipError_t launch_box(const float *x0, int32_t B, int32_t n0, int64_t ld0, float eps, int32_t clip_on,
                      float clip_lo, float clip_hi, float *c0, float *r0, hipStream_t s);
// Wp: the weights, n_out rows of pitch ldw (>= n_in rounded up to 32, zero padded); cin, rin:
// [B][ld_in]; cout, rout: [B][ld_out], ld_out a multiple of 16
hipError_t launch_ibp_dense(const float *Wp, int64_t ldw, const float *b, int32_t n_out, int32_t n_in,
                            const float *cin, const float *rin, int64_t ld_in, int32_t relu_in,
                            float *cout, float *rout, int64_t ld_out, int32_t B, hipStream_t s);
// lam_rule: the lower-slope rule of unstable neurons (VCR_OPT_LAMBDA_RULE values, relax.h)
hipError_t launch_layer_from_ibp(const float *c, const float *r, int64_t ld, int32_t n, int32_t B,
                                 const float *bias, float *L, float *U, float4 *P, int64_t ldp,
                                 int32_t lam_rule, hipStream_t s);
struct InitArgs {
  const float *src;      // source rows (W_k, or C W_L per input)
  int64_t ld_src;
  int32_t n_src;         // rows of one direction (n_k or m)
  int32_t per_unit_src;  // 1: unit u reads rows u*n_src + i (spec per input); 0: shared rows
  const float *src_bias; // (n_src) or (units * n_src) like src
  int32_t n_cols;        // real columns (width of the layer below)
  int64_t ldo;           // output row stride (padded)
  int32_t M;             // rows = units * 2 * n_src
  int32_t units;
  const float4 *P;       // params of the ReLU below, [param_units][ldp]
  int64_t ldp;
  int32_t param_per_unit;  // 1: unit u uses P row u; 0: row 0 (BaB: all domains share the root)
  int32_t relu_index;
  SplitTable splits;
  float *out;            // M_pad x ldo
  float *beta;           // M_pad
  const float *alpha;    // optional per-row lower slopes [M_pad][ld_alpha] (unstable neurons)
  int64_t ld_alpha;
  float *pre;            // optional: receives the rows before relaxation [M_pad][ldo]
};
hipError_t launch_init_rows(const InitArgs &a, hipStream_t s);
hipError_t launch_rowsum(float *beta, const float *part, int32_t n_parts, int32_t M_pad, int32_t M,
                         hipStream_t s);
hipError_t launch_finalize_layer(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad,
                                 int32_t B, int32_t n, const float *ibp_c, const float *ibp_r,
                                 int64_t ld_ibp, int32_t intersect, const float *bias_next,
                                 float *L, float *U, float4 *P, int64_t ldp, int32_t lam_rule, hipStream_t s);
hipError_t launch_spec_cw(const float *C, int32_t B, int32_t m, int32_t n_out, const float *Wp,
                          int64_t ldw, const float *b, int32_t n_in, float *CW, int64_t ld_cw,
                          float *Cb, hipStream_t s);
hipError_t launch_spec_direct(const float *CW, int64_t ld_cw, const float *Cb, int32_t B, int32_t m,
                              int32_t n_in, const float *c, const float *r, int64_t ld_in,
                              int32_t relu_in, float *lb, float *ub, hipStream_t s);
hipError_t launch_finalize_spec(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad,
                                int32_t units, int32_t m, const int32_t *unit_flags, float *lb,
                                float *ub, hipStream_t s);
struct SplitPrepArgs {
  const int32_t *relu_id, *neuron;
  const int8_t *sign;
  int32_t D, S, R;
  const int32_t *relu_n;     // [R] neurons per ReLU (device)
  const float *const *L;     // [R] device pointers to the root's lower bounds
  const float *const *U;     // [R] upper bounds
  int32_t *off;              // [D][R+1]
  int32_t *ent_n;            // [D][S]
  float4 *ent_p;             // [D][S]
  int32_t *flags;            // [D] 0 ok, 1 infeasible, 2 invalid
  int32_t *n_invalid;        // one counter
  int32_t lam_rule;          // lower-slope rule of unstable neurons (relax.h)
  // optional [R] (device): channels of a ReLU on a convolution output, 0 for flat ones.  The
  // split neurons come in (C, H, W) order (as L and U are laid out); ent_n then holds their
  // channels-last index, the one the convolution epilogues look up
  const int32_t *hwc_C;
};
hipError_t launch_split_prepare(const SplitPrepArgs &a, hipStream_t s);
hipError_t launch_count_unstable(const float *L, const float *U, int64_t n, int32_t *count, hipStream_t s);
hipError_t launch_count_nonfinite(const float *p, int64_t n, int32_t *count, hipStream_t s);
hipError_t launch_copy(float *dst, const float *src, int64_t n, hipStream_t s);
// dst[i] = ptrs[i] for i < n <= PTR_TABLE_MAX, the table travelling as a kernel argument (no
// host buffer has to outlive the launch)
constexpr int PTR_TABLE_MAX = 128;
struct PtrTable {
  const float *p[PTR_TABLE_MAX];
};
hipError_t launch_store_ptrs(const PtrTable &t, int32_t n, const float **dst, hipStream_t s);

// ---- alpha-CROWN (alpha.hip) --------------------------------------------------------
// Rows are (unit, q), q < 2m: q < m the lower bound of spec row q, q >= m the negated upper
// bound of spec row q - m; every row maximises its own lower bound.
struct AlphaLayer {
  float *alpha, *mom, *vel, *best, *grad, *pre;   // [M_pad][ld] each
  const float4 *P;                                // [units][ldp] relaxation of this ReLU
  int64_t ld, ldp;
  int32_t n, col0;                                // neurons, first column in the compact layout
  // channels-last neurons (ReLUs on convolution outputs): neuron (y, x, c) is column
  // (y W + x) C + c here and c H W + y W + x in the compact layout; 0 for flat neurons
  int32_t hwc_C, hwc_HW;
};
// alpha <- alpha_init (compact [units][2m][n_total]) or lam (P.x); mom = vel = grad = pre = 0
hipError_t launch_alpha_init(const AlphaLayer &l, const float *alpha_init, int64_t n_total, int32_t rows,
                             int32_t rows_pad, int32_t rows_per_unit, hipStream_t s);
// E0 = c - sign(pre0) r per row (the box vertex that attains the row's bound)
hipError_t launch_alpha_vertex(const float *pre0, int64_t ld0, const float *c0, const float *r0, int32_t rows_pad,
                               int32_t rows_per_unit, int32_t units, float *E0, hipStream_t s);
// row bound = beta + sum of the concretization partials (the order of the final reduction);
// best/flag update, optional history [units][m] lb and ub of this evaluation
hipError_t launch_alpha_best(const float *beta, const float *cpart, int32_t n_parts, int32_t M_pad, int32_t rows,
                             int32_t m, int32_t first, float *best_val, int32_t *flag, float *hist_lb,
                             float *hist_ub, hipStream_t s);
// best <- alpha where the row improved
hipError_t launch_alpha_keep(const AlphaLayer &l, const int32_t *flag, int32_t rows, hipStream_t s);
// one projected Adam step (ascent) at unstable neurons; c1 = 1 / (1 - beta1^t), c2 = 1 / (1 - beta2^t);
// with flag, first the keep step above on the same rows
hipError_t launch_alpha_adam(const AlphaLayer &l, const int32_t *flag, int32_t rows, int32_t rows_per_unit, float lr,
                             float beta1, float beta2, float eps, float c1, float c2, hipStream_t s);
// lb / ub from the best row values; with unit_flags (subdomains): 1 infeasible -> lb = +inf,
// ub = -inf; 2 invalid splits -> NaN
hipError_t launch_alpha_final(const float *best_val, int32_t units, int32_t m, const int32_t *unit_flags, float *lb,
                              float *ub, hipStream_t s);
// beta-CROWN multipliers [M_pad][S] with their Adam moments and gradient
struct BetaState {
  float *beta, *mom, *vel, *grad;
  int32_t S;
};
hipError_t launch_beta_init(const BetaState &b, int32_t rows_pad, hipStream_t s);
// one projected Adam step (ascent) on the multipliers of real split entries: beta >= 0
hipError_t launch_beta_adam(const BetaState &b, int32_t rows, float lr, float beta1, float beta2, float eps,
                            float c1, float c2, hipStream_t s);
// compact outputs: slopes of the best bound and the last gradient (d ub / d alpha for the
// upper rows, so the sign of the negated rows is undone)
hipError_t launch_alpha_out(const AlphaLayer &l, int32_t rows, int32_t m, int64_t n_total, float *alpha_out,
                            float *grad_out, hipStream_t s);

}  // namespace vcr
