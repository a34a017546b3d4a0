// Internal launch interface of the convolutional-path kernels (not part of the C ABI).
#pragma once

#include "kernels.h"

namespace vcr {

// floor(n / d) by multiply-high (n < 2^31), computed on the host
struct FastDiv {
  uint32_t mul = 0, shift = 0;
};
FastDiv make_fastdiv(uint32_t d);

// One class of output positions of a transposed convolution: the positions of the
// destination window that receive the same set of taps.  With stride 2 a position (u, w)
// only receives the taps whose (ky, kx) have the parity of (u + delta, w + delta); at the
// window's border ring, taps whose source falls outside the source window are missing too.
// Each class runs as a GEMM over its own taps only, so no all-zero K tile is computed (the
// executed flops are the algorithmic ones).  Positions: u = u0 + ustep iy, w = w0 + wstep ix
// (ustep = stride unless ny = 1); taps (ky0 + kys ty, kx0 + kxs tx).
//
// Windowed destinations are clipped to the image: a class then holds only the (row, position)
// pairs whose destination lies inside the image, rows outer and positions (iy, ix) inner as
// before.  Row r's anchor is (a_y, a_x) = ((r mod Ha^2) / Ha, r mod Ha); per anchor the inside
// positions of an axis are an interval [lo(a), lo(a) + n(a)), so one cycle of Ha^2 rows holds
// T = (sum_a n_y(a)) (sum_a n_x(a)) pairs and the kernel finds a pair's anchors by a search
// over the prefix sums of n(a).
constexpr int CONVT_CLIP_MAX = 64;   // anchors per axis (one wave builds the tables)
struct ConvClass {
  int32_t blk0;              // first workgroup of the class (classes are consecutive)
  int32_t M;                 // GEMM rows of the class: R ny nx, or (R / Ha^2) T clipped
  int32_t clip;              // 1: positions outside the image are left out (div_yx divides by T)
  int32_t ny, nx, u0, w0, ustep, wstep;
  int32_t nty, ntx, ky0, kx0, kys, kxs;
  FastDiv div_yx, div_x;
};

struct ConvTArgs {
  const float *A;          // source windows [R][S_out][S_out][C_out]
  int64_t row_stride_out;  // S_out^2 C_out
  int32_t S_out, C_out;
  const float *Bt;         // [N_pad][ldb], ldb = 9 C_out: Bt[ci][(3 ky + kx) C_out + co]
  int64_t ldb;
  int32_t N_pad;
  int32_t C_in, S_in, H_in;  // destination channels, window size, image size
  int64_t row_stride_in;     // S_in^2 C_in
  int32_t stride, delta;
  int32_t R;                 // coefficient rows
  int32_t M_pad;             // partial-sum pitch (>= R S_in^2)
  const int4 *rows;          // per coefficient row: (unit, anchor y, anchor x, -)
  int32_t dense, scale, h_in;  // window origin = anchor * scale - h_in (dense: 0)
  // windowed destinations: anchors per axis of the pass (rows in (cycle, a_y, a_x) order, the
  // row table's anchors); with 0 < Ha <= CONVT_CLIP_MAX and R a multiple of Ha^2 only the
  // window positions inside the image are computed and written (the others are never read:
  // windowed sources are masked to the image, and the constant terms skip them)
  int32_t Ha;
  // windowed sources (src_scale > 0, in windowed passes: Ha > 0): the source window's origin
  // is anchor * src_scale - src_h on an H_out image; source positions outside it read as zero
  int32_t src_scale, src_h, H_out;
  const float *res;          // optional residual windows on the same node
  int64_t res_row_stride;
  int32_t res_S, res_off;
  const float4 *P_pos;       // ReLU parameters [unit][H][H][C_in], or null (identity)
  const float *bias;         // identity: constant per channel
  float *out;                // [R][S_in][S_in][C_in]
  float *part;               // [N_pad / 64][M_pad]
  // alpha-CROWN (dense windows with a ReLU only): per-row lower slopes at unstable neurons,
  // and the coefficients before relaxation (recorded at unstable neurons only), both laid
  // out like out
  const float *alpha;
  float *pre;
  // branch-and-bound subdomains of one input (dense windows with a ReLU; every row belongs
  // to unit 0, so a parameter's offset is its neuron's channels-last index): the split
  // table of this ReLU (relu_index) and, with splits.beta, the multipliers' terms
  SplitTable splits;
  int32_t relu_index;
  // filled by launch_convt
  int32_t n_cls;
  ConvClass cls[4];
};
hipError_t launch_convt(const ConvTArgs &a, hipStream_t s);
// The transposed convolution runs as classes of output positions (the taps that reach them),
// four per dispatch: the number of dispatches (or -1 for unsupported shapes), dispatch `part`
// alone, and its flops (2 per multiply-add of a position and a tap that reaches it).
int convt_launches(const ConvTArgs &a);
hipError_t launch_convt_part(const ConvTArgs &a, int part, hipStream_t s);
// Algorithmic flops of dispatch `part`: 2 per multiply-add of a destination position and a tap
// whose source position both lie inside the image (windowed rows clipped to the image).
uint64_t convt_part_flops(const ConvTArgs &a, int part);
// Whether the launch computes only the window positions inside the image
bool convt_clipped(const ConvTArgs &a);

struct StemArgs {
  const float *A;
  int64_t row_stride_out;
  int32_t S_out, C_out;
  const float *W;          // [C_out][C_in][3][3]
  int32_t C_in, S_in, H_in, stride, delta;
  int32_t R;               // rows
  int32_t rpw, strip, n_strips;  // rows per workgroup, destination rows per strip, strips
                                 // per row (chosen by launch_stem)
  const int4 *rows;
  int32_t dense, scale, h_in;
  // windowed sources (src_scale > 0): source window origin anchor * src_scale - src_h on an
  // H_src image; positions outside the image are not gathered
  int32_t src_scale, src_h, H_src;
  const float *c0, *r0;    // box centre / radius, CHW per unit
  int64_t ld_box;          // floats per unit in c0 / r0
  float *part;             // [R][S_in^2]
  // optional (dense windows): the box vertex where each row's linear function is smallest,
  // c - sign(a) r per input neuron (the centre where a = 0), channels-last [R][ld_vtx]
  float *vtx;
  int64_t ld_vtx;
};
hipError_t launch_stem(const StemArgs &a, hipStream_t s);

struct ConvInitArgs {
  const float *W;          // start convolution, taps outer: [C_src][3][3][C_in]
  const float *b;          // its bias
  int32_t C_src, H_src;    // start node shape (C_src, H_src, H_src)
  int32_t C_in, H_in;      // the convolution's input node
  int32_t S, h, scale;     // window 3, half 1, stride
  int64_t R;
  const int4 *rows;
  const float4 *P_pos;     // ReLU below (channels-last) or null
  const float *bias_next;  // identity constants per input channel
  float *out;
  float *beta;
};
hipError_t launch_init_conv(const ConvInitArgs &a, hipStream_t s);

// Forward 3x3 convolution (pad 1) of `rows` channels-last images, the gradient pass of
// alpha-CROWN: out = conv(in) + bias (+ res), or with a ReLU line: the line of that ReLU the
// backward pass chose for the row (by the sign of the coefficient `pre` it recorded), and the
// slope gradient pre * D at unstable neurons whose coefficient is positive (else 0).
struct FwdConvArgs {
  const float *in;         // [rows][in_rs]: (Hi, Hi, Ci) channels-last
  int64_t in_rs;
  int32_t Ci, Hi;
  const float *Wk;         // [Co][3][3][Ci]
  const float *bias;       // [Co]
  int32_t Co, Ho, stride;
  int32_t rows;
  const float *res;        // optional [rows][res_rs], (Ho, Ho, Co): added to D
  int64_t res_rs;
  const float4 *P;         // optional ReLU parameters [units][Ho][Ho][Co]
  int32_t rows_per_unit, units;
  const float *alpha, *pre;  // [rows][out_rs] with P
  float *grad;               // [rows][out_rs] with P
  float *out;              // [rows][out_rs], (Ho, Ho, Co)
  int64_t out_rs;
  // with P, subdomains of one input (units = 1): the split table of this ReLU (relu_index);
  // with splits.grad_beta, each split's multiplier gradient S z at the row's vertex
  SplitTable splits;
  int32_t relu_index;
};
hipError_t launch_fwd_conv(const FwdConvArgs &a, hipStream_t s);
// out = x + y over rows of n values (the add node in the gradient pass)
hipError_t launch_fwd_add(const float *x, int64_t xs, const float *y, int64_t ys, float *out, int64_t os,
                          int32_t rows, int64_t n, hipStream_t s);
// Window positions of clipped rows (Ha > 0): row r's window of S x S positions at origin
// anchor * scale - h, anchor ((r mod Ha^2) / Ha, r mod Ha); positions outside the H x H image
// hold no partial sums.
struct WinClip {
  int32_t Ha = 0, scale = 1, h = 0, S = 0, H = 0;
};
hipError_t launch_rowsum_win(float *beta, const float *part, int32_t n_parts, int64_t M_pad, int64_t R,
                             int32_t per_row, hipStream_t s, WinClip clip = WinClip{});
hipError_t launch_row_table(int4 *rows, int64_t R, int32_t rows_per_unit, int32_t C, int32_t H, int32_t W,
                            int32_t windowed, int32_t unit0, hipStream_t s);
hipError_t launch_finalize_conv(const float *beta, int32_t B, int32_t C, int32_t H, const float *ibp_c,
                                const float *ibp_r, int64_t ld_ibp, int32_t intersect, const float *bias_next,
                                float *L, float *U, float4 *P, int32_t lam_rule, hipStream_t s);
hipError_t launch_conv_layer_from_ibp(const float *ibp_c, const float *ibp_r, int64_t ld_ibp, int32_t B, int32_t C,
                                      int32_t H, const float *bias_next, float *L, float *U, float4 *P,
                                      int32_t lam_rule, hipStream_t s);
hipError_t launch_ibp_conv(const float *W, const float *bias, int32_t Co, int32_t Ci, int32_t Hin, int32_t Hout,
                           int32_t stride, int32_t pad, const float *cin, const float *rin, int64_t ld_in,
                           float *cout, float *rout, int64_t ld_out, int32_t B, hipStream_t s);
hipError_t launch_ibp_relu(const float *cin, const float *rin, float *cout, float *rout, int64_t n, hipStream_t s);
hipError_t launch_ibp_add(const float *c1, const float *r1, const float *c2, const float *r2, float *cout,
                          float *rout, int64_t n, hipStream_t s);
hipError_t launch_repack_convt(const float *W, int32_t Co, int32_t Ci, int32_t Ci_pad, float *Bt, hipStream_t s);
hipError_t launch_permute_hwc(const float *W, int32_t rows, int32_t C, int32_t HW, float *Wo, int64_t ldo,
                              hipStream_t s);
hipError_t launch_identity_params(const float *b, int32_t C, int64_t n, int64_t ld, float4 *P, hipStream_t s);

}  // namespace vcr
