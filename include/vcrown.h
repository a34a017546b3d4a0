/*
 * vcrown — batched CROWN linear bound propagation on ReLU networks, for AMD Instinct
 * MI355X (gfx950).  C ABI.
 *
 * The problem (paper, Sec. 1.1): a network f : R^n -> R^m, an admissible input set, here
 * the L-infinity ball ||x - x0||_inf <= eps intersected with a clip box (local
 * robustness), and linear output properties given as a specification matrix C (the
 * linear constraints of the VNN-LIB format, Sec. 1.2).  The library returns, for every
 * row c of C, a lower and an upper bound on c . f(x) that hold for every x in the set.
 *
 * Methods (paper, Sec. 2.1):
 *   - IBP: intervals propagated layer by layer, l_y = W+ l + W- u + b, u_y = W+ u + W- l + b;
 *   - CROWN: a backward pass composing the layer weights with diagonal ReLU slope matrices
 *     (different slopes for the lower and the upper branch) into linear functions
 *     A_L x + b_L <= f(x) <= A_U x + b_U (equation "crown"), which are then minimised /
 *     maximised over the box.  "Full" CROWN: every ReLU's pre-activation bounds come from
 *     such a backward pass from that layer to the input, intersected with the IBP bounds;
 *   - branch-and-bound subdomains (Sec. 2.1, complete verification): each subdomain fixes
 *     some ReLUs to the active (z >= 0) or inactive (z <= 0) state; subdomains of one root
 *     input are bounded in one batched pass (Sec. 2.4, batch BaB).
 *
 * Conventions shared by every entry point:
 *   - All tensors are float32, dense, row-major (C order).  Device pointers must come from
 *     the context's device and be 16-byte aligned.
 *   - Work is queued on the context's stream (vcr_set_stream; default: the null stream).
 *     Entry points return once the work is queued; outputs are valid after the stream is
 *     synchronised.  Entry points that must read device results say "synchronises".
 *   - Every call returns a vcr_status.  On an error nothing is queued, the outputs are left
 *     untouched and vcr_last_error() describes the failure.  No C++ exception crosses the
 *     ABI.  An asynchronous device fault is reported as VCR_ERR_DEVICE by a later call.
 *   - A context is not thread-safe; use one context per host thread / stream.
 */
#ifndef VCROWN_H
#define VCROWN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VCR_ABI_VERSION 3   /* 2: vcr_stats gained timed_mid_*; 3: vcr_crown_bounds_noalloc */

typedef struct vcr_ctx vcr_ctx;

typedef enum {
  VCR_OK = 0,
  VCR_ERR_ARG = 1,          /* invalid argument value (null pointer, eps < 0, bad split) */
  VCR_ERR_SHAPE = 2,        /* sizes inconsistent with the loaded network */
  VCR_ERR_STATE = 3,        /* call out of order (e.g. bounds before vcr_load_net) */
  VCR_ERR_OOM = 4,          /* device allocation failed or exceeds the workspace cap */
  VCR_ERR_DEVICE = 5,       /* HIP runtime error (including an earlier asynchronous fault) */
  VCR_ERR_UNSUPPORTED = 6   /* valid request the library does not implement */
} vcr_status;

/* Node kinds of a feed-forward network given in topological order. */
typedef enum {
  VCR_DENSE = 0,     /* y = W x + b, W (out_features, d_in) row-major, b (out_features) */
  VCR_CONV2D = 1,    /* 2-D cross-correlation, W (out_ch, C_in, kh, kw), b (out_ch), zero padding */
  VCR_RELU = 2,      /* y = max(x, 0) elementwise */
  VCR_ADD = 3,       /* y = in0 + in1 (same shape) */
  VCR_FLATTEN = 4    /* (C, H, W) -> C*H*W in C, H, W order */
} vcr_op;

typedef struct {
  int32_t op;             /* vcr_op */
  int32_t in0, in1;       /* producer node ids, -1 = the network input; in1 only for VCR_ADD */
  int32_t out_features;   /* VCR_DENSE */
  int32_t out_ch, kh, kw, stride, pad;  /* VCR_CONV2D */
  const float *W, *b;     /* HOST pointers, copied by vcr_load_net; PyTorch layouts */
} vcr_node;

/* Branch-and-bound subdomains of one root input (paper, Sec. 2.1.1 and Sec. 2.4).
 * n_domains x per_domain entries each, DEVICE pointers, row-major by domain:
 *   relu_id[d*per_domain + k]  index of the ReLU node among the network's ReLU nodes, in
 *                              node order (0 = first ReLU);
 *   neuron[...]                flat index into that ReLU's tensor ((C, H, W) order for a
 *                              ReLU on a convolution output);
 *   sign[...]                  +1: the pre-activation is fixed to z >= 0 (active),
 *                              -1: fixed to z <= 0 (inactive).
 * A split slot with relu_id -1 is unused (skipped).
 * A domain's intermediate bounds are the root pass's, with each split neuron's interval
 * clamped (l <- max(l, 0) for +1, u <- min(u, 0) for -1).  A domain whose clamped interval
 * is empty (l > u) is infeasible and gets lb = +inf, ub = -inf (not an error).  A domain
 * with an out-of-range entry, a sign other than +-1 or a neuron repeated gets NaN bounds and
 * is counted in vcr_stats.invalid_domains. */
#define VCR_MAX_SPLITS 64   /* split slots per subdomain (per_domain <= VCR_MAX_SPLITS) */

typedef struct {
  int32_t n_domains, per_domain;
  const int32_t *relu_id;
  const int32_t *neuron;
  const int8_t *sign;
} vcr_splits;

/* Options (vcr_set_option). */
enum {
  VCR_OPT_CLIP_ENABLE = 1,          /* 1 (default): intersect the eps-ball with [CLIP_LO, CLIP_HI] */
  VCR_OPT_CLIP_LO = 2,              /* default 0.0 */
  VCR_OPT_CLIP_HI = 3,              /* default 1.0 */
  VCR_OPT_INTERSECT_IBP = 4,        /* 1 (default): intersect CROWN intermediate bounds with IBP */
  VCR_OPT_WORKSPACE_CAP_BYTES = 5,  /* device workspace cap; 0 (default) = no cap.  Inputs
                                       (or domains) are processed in chunks that fit. */
  VCR_OPT_SYNC_CHECK = 6,           /* 1: synchronise after each call and report device errors
                                       and invalid split domains as the call's status */
  VCR_OPT_TIME_GEMM = 7,            /* 1: bracket every backward-step GEMM launch (dense and
                                       transposed-convolution) with HIP events
                                       on the context's stream; vcr_get_stats reports their summed
                                       duration.  Setting the option (either value) resets the sums. */
  VCR_OPT_GRAPH = 8,                /* 1: vcr_crown_bounds without splits records its kernel launches
                                       into a HIP graph (captured on a private stream after one
                                       ordinary call with the same arguments) and, while the
                                       arguments, options, network and workspace stay the same,
                                       replays the graph on the context's stream instead of
                                       launching kernel by kernel.  Ignored while TIME_GEMM is on. */
  VCR_OPT_CHECK_FINITE = 9,         /* 1: every bounds call first scans x0 and C on the device for NaN
                                       and infinite values and fails with VCR_ERR_ARG (nothing else
                                       queued, outputs untouched) if it finds any; the scan
                                       synchronises the stream.  0 (default): no scan, and a
                                       non-finite input gives undefined bounds (Sec. 1.1 defines the
                                       input set for finite centres only). */
  VCR_OPT_LAMBDA_RULE = 10          /* lower slope lambda of unstable ReLU neurons (Sec. 2.1 only
                                       requires lambda in [0, 1], every value being sound):
                                       VCR_LAMBDA_ADAPTIVE (default), VCR_LAMBDA_ZERO, VCR_LAMBDA_ONE,
                                       VCR_LAMBDA_SAME_SLOPE.  Applies to every ReLU layer, to split
                                       neurons' relaxations and to alpha-CROWN's initial slopes. */
};

/* Values of VCR_OPT_LAMBDA_RULE.  For an unstable neuron (l < 0 < u) with upper line slope
 * s = u / (u - l): ADAPTIVE takes lambda = 1 if u > -l else 0 (a tie gives 0); ZERO 0; ONE 1;
 * SAME_SLOPE lambda = s. */
enum {
  VCR_LAMBDA_ADAPTIVE = 0,
  VCR_LAMBDA_ZERO = 1,
  VCR_LAMBDA_ONE = 2,
  VCR_LAMBDA_SAME_SLOPE = 3
};

typedef struct {
  double ms_last_call;              /* host wall time of the last bounds call (queue + wait if SYNC_CHECK) */
  uint64_t gemm_flops_last_call;    /* algorithmic fp32 GEMM flops of the last call (2 per MAC): the
                                       backward steps, and the IBP steps of large layers, which
                                       run as GEMMs */
  uint64_t peak_workspace_bytes;    /* largest device workspace held so far */
  uint64_t workspace_bytes;         /* current device workspace */
  int32_t n_chunks_last_call;       /* input (or domain) chunks used by the last call */
  int32_t invalid_domains;          /* domains rejected by the last split call (synchronises) */
  int32_t n_relu;                   /* ReLU nodes of the loaded network */
  int32_t unstable[64];             /* unstable neurons per ReLU node, summed over inputs, last
                                       CROWN call (synchronises); first min(n_relu, 64) valid */
  /* with VCR_OPT_TIME_GEMM: dense GEMM launches (A W steps) timed since the option was set,
   * their summed device duration and their algorithmic flops */
  uint64_t timed_gemm_launches;
  double timed_gemm_ms;
  uint64_t timed_gemm_flops;
  /* the same for the transposed-convolution GEMM launches (algorithmic flops: 2 per
   * multiply-add of the convolution's scatter form over the source window) */
  uint64_t timed_conv_launches;
  double timed_conv_ms;
  uint64_t timed_conv_flops;
  uint64_t net_bytes;               /* device memory holding the loaded network's weights */
  /* the dense GEMM launches too small to fill the chip, which run a small-tile kernel (not
   * included in timed_gemm_*) */
  uint64_t timed_small_launches;
  double timed_small_ms;
  uint64_t timed_small_flops;
  /* the dense GEMM launches of middle size (too few 128 x 128 tiles, enough 64 x 64 ones),
   * which run a 64 x 64 tile kernel (not included in the two above) */
  uint64_t timed_mid_launches;
  double timed_mid_ms;
  uint64_t timed_mid_flops;
} vcr_stats;

/* ABI version compiled into the library (VCR_ABI_VERSION). */
int32_t vcr_abi_version(void);

/* Create a context on HIP device `hip_device`.  hip_device = -1 creates a validation-only
 * context without a device: vcr_load_net checks the network and the bounds calls check
 * their arguments, then return VCR_ERR_STATE instead of queueing work. */
vcr_status vcr_create(int32_t hip_device, vcr_ctx **out);
void vcr_destroy(vcr_ctx *ctx);

/* Message of the last failed call; owned by the context, valid until its next call. */
const char *vcr_last_error(const vcr_ctx *ctx);

/* Use the caller's hipStream_t for all later work (NULL = the null stream). */
vcr_status vcr_set_stream(vcr_ctx *ctx, void *hip_stream);

vcr_status vcr_set_option(vcr_ctx *ctx, int32_t key, double value);

/* Size limits checked by vcr_load_net (VCR_ERR_SHAPE beyond them): elements of the input or
 * of any node's output, and weights of one dense or convolution layer (kernels up to 64 x 64). */
#define VCR_MAX_NODE_ELEMENTS ((int64_t)1 << 30)
#define VCR_MAX_LAYER_WEIGHTS ((int64_t)1 << 32)

/* Load (copy) a network.  nodes[0..n) in topological order; the last node is the output and
 * must be VCR_DENSE.  in_chw is the input shape (C, H, W); for a flat input use
 * (n0, 1, 1).  Weight pointers are host memory and are not retained.  Replaces any
 * previously loaded network.  Synchronises. */
vcr_status vcr_load_net(vcr_ctx *ctx, const vcr_node *nodes, int32_t n, const int32_t in_chw[3]);

/* IBP bounds on C f(x) (paper, Sec. 2.1, IBP), C folded into the last dense layer.
 *   x0  device (B, n0)      centres of the eps-balls (flat input, C,H,W order)
 *   eps scalar >= 0         L-infinity radius; the box is fl32(x0 -/+ eps) then clipped
 *   C   device (B, m, n_out) one specification matrix per input
 *   lb, ub device (B, m)    outputs */
vcr_status vcr_ibp_bounds(vcr_ctx *ctx, const float *x0, int32_t B, float eps,
                          const float *C, int32_t m, float *lb, float *ub);

/* Full CROWN bounds on C f(x) (paper, Sec. 2.1, equation "crown").
 * Without splits (splits == NULL): as vcr_ibp_bounds, outputs (B, m).
 * With splits: B must be 1; the root pass runs on x0 and every subdomain is bounded with
 * the final pass; C is (1, m, n_out) and lb, ub are (n_domains, m). */
vcr_status vcr_crown_bounds(vcr_ctx *ctx, const float *x0, int32_t B, float eps,
                            const float *C, int32_t m, const vcr_splits *splits,
                            float *lb, float *ub);

/* alpha-CROWN (paper, Sec. 2.1): the lower slope of every unstable ReLU neuron becomes a
 * parameter alpha in [0, 1], one per (ReLU layer, specification bound, input, neuron)
 * (the alpha tensors of Sec. 4.6), raised by gradient steps on the bound it enters.
 *
 * Slope arrays use the compact layout [B][2m][n_total]: row q < m holds the slopes of the
 * lower bound of specification row q, row m + q those of its upper bound; the columns are
 * the neurons of every ReLU node in node order (n_total = sum of their sizes), each node's
 * neurons in its own (C, H, W) order.  Entries of neurons that are not unstable are ignored
 * on input and report the fixed slope on output. */
typedef struct {
  int32_t iters;            /* optimisation steps after the first evaluation (>= 0) */
  float lr;                 /* Adam step size (> 0) */
  float beta1, beta2;       /* Adam moment decays, in [0, 1) */
  float adam_eps;           /* Adam denominator guard (> 0) */
  const float *alpha_init;  /* device [B][2m][n_total] in [0, 1], or NULL: CROWN's lambda */
  float *alpha_out;         /* device [B][2m][n_total] or NULL: slopes of each best bound */
  float *grad_out;          /* device [B][2m][n_total] or NULL: d bound / d alpha at the last
                               evaluated slopes (d lb for lower rows, d ub for upper rows) */
  float *lb_hist, *ub_hist; /* device [iters + 1][B][m] each, or NULL: every evaluation */
} vcr_alpha_opts;

/* alpha-CROWN bounds on C f(x): the intermediate bounds are full CROWN's (as
 * vcr_crown_bounds, IBP-intersected when that option is on); the final pass is evaluated
 * iters + 1 times, with projected Adam steps on the slopes in between (ascent on every
 * lower bound, descent on every upper bound), and each bound is the best one evaluated.
 * Every network vcr_crown_bounds takes: dense/relu chains, and convolutional networks with
 * residual additions and flatten (VCR_ERR_UNSUPPORTED, with the reason in vcr_last_error,
 * for a ReLU whose input is not a convolution or dense node, or an add of the network
 * input); x0, C, lb, ub as in vcr_crown_bounds without splits.  All arrays are caller-owned
 * device memory. */
vcr_status vcr_alpha_crown_bounds(vcr_ctx *ctx, const float *x0, int32_t B, float eps,
                                  const float *C, int32_t m, const vcr_alpha_opts *opts,
                                  float *lb, float *ub);

/* Number of ReLU neurons over all ReLU nodes of the loaded network (n_total above). */
int64_t vcr_relu_neurons(const vcr_ctx *ctx);

/* beta-CROWN on branch-and-bound subdomains (paper, Sec. 2.2, the alpha-beta-CROWN verifier): every split
 * g <= 0 (g = -z for an active split, g = z for an inactive one) enters the bound of its
 * subdomain with a multiplier beta >= 0 (f + beta g for a lower bound, f - beta g for an upper
 * one), one per (split, specification bound); the multipliers and the lower slopes alpha
 * (as in vcr_alpha_crown_bounds) are optimised jointly by projected Adam steps, and each bound
 * is the best one evaluated (the first evaluation is CROWN's, as vcr_crown_bounds with the
 * same splits).  Intermediate bounds: the root's full CROWN, with each split neuron's interval
 * clamped.  Every network vcr_crown_bounds takes (dense/relu chains and convolutional
 * networks, as vcr_alpha_crown_bounds). */
typedef struct {
  int32_t iters;            /* optimisation steps after the first evaluation (>= 0) */
  float lr_alpha, lr_beta;  /* Adam step sizes (> 0) */
  float beta1, beta2;       /* Adam moment decays, in [0, 1) */
  float adam_eps;           /* Adam denominator guard (> 0) */
  float *lb_hist, *ub_hist; /* device [iters + 1][n_domains][m] each, or NULL */
} vcr_beta_opts;

/* x0 (1, n0) and C (1, m, n_out) as in vcr_crown_bounds with splits; lb, ub (n_domains, m).
 * A split slot with relu_id -1 is unused (subdomains of different depths in one array). */
vcr_status vcr_beta_crown_bounds(vcr_ctx *ctx, const float *x0, float eps, const float *C, int32_t m,
                                 const vcr_splits *splits, const vcr_beta_opts *opts,
                                 float *lb, float *ub);

/* Fixed-batch branch-and-bound (paper, Sec. 2.1 complete verification; Sec. 2.2; Sec. 3.4.4: a
 * fixed number of subdomains per round, no early stop) on the property C f(x) > 0 for every row of
 * C over the eps-ball around x0.  The root is bounded by alpha-CROWN; unverified subdomains
 * wait first-in first-out; each round takes up to `batch` of them, splits each on the first
 * neuron of the priority order that it has not split yet into an active and an inactive
 * child, bounds the children with beta-CROWN and keeps those with a non-positive lower bound
 * (infeasible children are dropped).  Verified when no subdomain is left; otherwise unknown
 * after max_rounds, or when a subdomain has no neuron left to split.  The root's
 * intermediate bounds and relaxation are computed in the first round and reused in the later
 * ones. */
typedef struct {
  int32_t batch;            /* subdomains split per round (>= 1) */
  int32_t max_rounds;       /* in [0, VCR_MAX_SPLITS]: a subdomain gains one split per round
                               and holds at most VCR_MAX_SPLITS (VCR_ERR_ARG otherwise) */
  vcr_beta_opts bound;      /* bounding of the root and of every subdomain (hist ignored) */
  const int32_t *order_relu;    /* host [order_len]: split priority (ReLU node position,  */
  const int32_t *order_neuron;  /* neuron), or NULL: the root's unstable neurons by        */
  int32_t order_len;            /* decreasing chord intercept -u l / (u - l)               */
} vcr_bab_opts;

typedef struct {
  int32_t verified;         /* 1: the property holds on the whole ball */
  int32_t rounds;           /* rounds run */
  int64_t evaluated;        /* subdomains bounded (the root not counted) */
  int64_t remaining;        /* unverified subdomains left */
  float root_min_lb;        /* smallest lower bound of the root (alpha-CROWN) */
  float worst_lb;           /* smallest lower bound over the remaining subdomains (+inf if none) */
} vcr_bab_result;

/* x0, C device as above (one input).  round_log: host [max_rounds][4] or NULL, per round
 * (subdomains taken, children bounded, children verified, subdomains left).  Synchronises
 * once per round. */
vcr_status vcr_bab_verify(vcr_ctx *ctx, const float *x0, float eps, const float *C, int32_t m,
                          const vcr_bab_opts *opts, vcr_bab_result *result, int64_t *round_log);

/* Allocation-free variant of vcr_crown_bounds without splits, for callers that cannot
 * allocate device memory during a call (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, results and errors as
 * vcr_crown_bounds(ctx, x0, B, eps, C, m, NULL, lb, ub), bit for bit; the call allocates
 * nothing: its workspace is a fixed device array of VCR_NOALLOC_SCRATCH_BYTES per GPU (held
 * from the library's first use on that GPU until the process ends), shared by every context
 * on that GPU.  Inputs are processed in chunks that fit the scratch (and the workspace cap
 * option, if smaller); a call whose single input does not fit fails with VCR_ERR_OOM before
 * queueing work (for example the 3072-8192x4 MLP, or convolutional networks beyond a few
 * channels at small images).  The call clears the part of the scratch it uses before use.
 * Calls that overlap on one GPU (other streams, threads or contexts) race on the scratch;
 * vcr_get_layer_bounds after this call reads the scratch and is valid until the next call of
 * this entry point on the same GPU.  VCR_OPT_TIME_GEMM and VCR_OPT_GRAPH do not apply. */
#define VCR_NOALLOC_SCRATCH_BYTES ((uint64_t)256 << 20)
vcr_status vcr_crown_bounds_noalloc(vcr_ctx *ctx, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                                    float *lb, float *ub);

/* Pre-activation bounds of ReLU node `relu_id` (0-based among ReLU nodes) from the last
 * CROWN call, for every input: l, u device (B, numel).  Queued on the stream. */
vcr_status vcr_get_layer_bounds(vcr_ctx *ctx, int32_t relu_id, float *l, float *u);

/* Device bytes a bounds call of this size would hold (without a cap). */
vcr_status vcr_workspace_bytes(vcr_ctx *ctx, int32_t B, int32_t m, int32_t n_domains, uint64_t *bytes);

/* Statistics; synchronises the stream. */
vcr_status vcr_get_stats(vcr_ctx *ctx, vcr_stats *out);

#ifdef __cplusplus
}
#endif
#endif /* VCROWN_H */
