// Internal context of the vcrown library, shared by the MLP path (api.cpp) and the
// convolutional-network path (graph.cpp).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <memory>
#include <string>
#include <utility>
#include <vector>

#include "../../include/vcrown.h"
#include "kernels.h"

namespace vcr {
struct GraphNet;   // the convolutional-network path (graph.cpp)
void destroy_graph(GraphNet *g);
}

namespace vcr_internal {

struct DenseLayer {
  int32_t n_in = 0, n_out = 0;
  int64_t ld_in = 0, ld_out = 0;
  float *Wp = nullptr;   // n_out x ld_in, zero padded
  float *Bt = nullptr;   // ld_in x ld_out, Bt[n][k] = W[k][n], zero padded
  float *b = nullptr;    // ld_out, zero padded
};

struct Workspace {
  char *base = nullptr;
  size_t cap = 0, used = 0;
};

}  // namespace vcr_internal

using vcr_internal::DenseLayer;
using vcr_internal::Workspace;

struct vcr_ctx {
  int32_t device = -1;
  hipStream_t stream = nullptr;
  std::string err;
  // options
  int32_t clip_on = 1;
  float clip_lo = 0.f, clip_hi = 1.f;
  int32_t intersect = 1;
  uint64_t ws_cap = 0;
  int32_t sync_check = 0;
  int32_t check_finite = 0;
  int32_t lambda_rule = 0;          // VCR_OPT_LAMBDA_RULE (relax.h)
  // network
  bool loaded = false;
  int32_t n0 = 0;
  std::vector<DenseLayer> layers;   // the MLP chain
  std::vector<int32_t> relu_n;      // neurons per ReLU node
  int32_t n_out = 0;                // outputs of the loaded network (the last dense node)
  // workspace
  Workspace ws;
  uint64_t peak_ws = 0;
  uint64_t net_bytes = 0;   // device memory holding the loaded network (weights in their layouts)
  // last call
  int32_t last_B = 0;
  std::vector<float *> lastL, lastU;
  int32_t *d_counters = nullptr;    // [0, 64) unstable counts, [64] invalid domains, [65] non-finite inputs
  // branch-and-bound loop: device split arrays and bounds of one round (outside the
  // workspace, which every bounding call carves anew)
  void *bab_buf = nullptr;
  size_t bab_cap = 0;
  // the root's intermediate bounds and relaxation (one input), kept by the loop's first
  // subdomain call and copied back by the later rounds instead of being recomputed (the
  // rounds share the root input)
  bool bab_reuse = false, root_cached = false;
  float *root_cache = nullptr;
  size_t root_cache_cap = 0;
  bool last_had_splits = false;
  double ms_last = 0.0;
  uint64_t flops_last = 0;
  int32_t chunks_last = 0;
  // convolutional-network path (null for MLPs)
  vcr::GraphNet *graph = nullptr;
  // HIP graph replay of a repeated call (VCR_OPT_GRAPH)
  int32_t use_graph = 0;
  uint64_t net_epoch = 0;
  hipStream_t cap_stream = nullptr;
  hipGraphExec_t gexec = nullptr;
  std::vector<uint64_t> gkey;
  // timing of the GEMM launches (VCR_OPT_TIME_GEMM); kind 0 = dense k_gemm, 1 = conv k_convt,
  // 2 = dense k_gemm_small, 3 = dense k_gemm_mid
  int32_t time_gemm = 0;
  std::vector<hipEvent_t> ev_pool;      // pairs: start, stop
  size_t ev_used = 0;                   // events recorded but not yet read
  uint64_t timed_launches[4] = {0, 0, 0, 0}, timed_flops[4] = {0, 0, 0, 0};
  double timed_ms[4] = {0.0, 0.0, 0.0, 0.0};
  std::vector<std::pair<uint64_t, int>> pending;  // (flops, kind) of each recorded pair
  // the device's allocation-free scratch (vcr_crown_bounds_noalloc): its device address on
  // this context's device, resolved at vcr_create, and its size
  char *scratch = nullptr;
  size_t scratch_bytes = 0;
};

inline vcr_status fail(vcr_ctx *c, vcr_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  c->err = buf;
  return st;
}

#define HIP_TRY(c, expr)                                                                      \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess) return fail((c), VCR_ERR_DEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// A dense GEMM launch timed under the kernel it runs (k_gemm, k_gemm_small or k_gemm_mid).
#define TIMED_GEMM(c, s, flops, args)                                                            \
  timed_launch((c), (s), vcr::gemm_kind(args), (flops), [&] { return vcr::launch_gemm((args), (s)); })

// Reads every recorded timing pair into the sums (waits for the last one).
vcr_status timing_fold(vcr_ctx *c);

// Launches through `launch` (a callable returning hipError_t); with VCR_OPT_TIME_GEMM on, the
// launch is bracketed by HIP events on stream s and counted under `kind` with `flops`.
template <class F>
vcr_status timed_launch(vcr_ctx *c, hipStream_t s, int kind, uint64_t flops, F &&launch) {
  if (!c->time_gemm) {
    HIP_TRY(c, launch());
    return VCR_OK;
  }
  if (c->ev_used + 2 > c->ev_pool.size()) {
    hipEvent_t e0, e1;
    HIP_TRY(c, hipEventCreate(&e0));
    HIP_TRY(c, hipEventCreate(&e1));
    c->ev_pool.push_back(e0);
    c->ev_pool.push_back(e1);
  }
  HIP_TRY(c, hipEventRecord(c->ev_pool[c->ev_used], s));
  HIP_TRY(c, launch());
  HIP_TRY(c, hipEventRecord(c->ev_pool[c->ev_used + 1], s));
  c->ev_used += 2;
  c->pending.emplace_back(flops, kind);
  if (c->ev_used >= 4096) return timing_fold(c);   // keeps the pool bounded
  return VCR_OK;
}

inline size_t al(size_t x) { return (x + 255) / 256 * 256; }

// Sub-allocation from the workspace.  With a null base it only counts bytes, which is how
// the planners size a call: the same carve code runs for sizing and for the real layout.
template <class T>
T *take(Workspace &w, size_t count) {
  size_t b = al(sizeof(T) * (count > 0 ? count : 1));
  T *p = w.base ? reinterpret_cast<T *>(w.base + w.used) : nullptr;
  w.used += b;
  return p;
}

template <class T>
T *take(vcr_ctx *c, size_t count) {
  return take<T>(c->ws, count);
}

vcr_status ensure_ws(vcr_ctx *c, size_t bytes);

namespace vcr {
// Resolves the device address of the allocation-free scratch on c's device (current) into
// c->scratch / c->scratch_bytes (noalloc.hip).
vcr_status noalloc_setup(vcr_ctx *c);
// vcr_crown_bounds without splits, run in the caller-given device memory [base, base + bytes)
// instead of the context's workspace: no device allocation (api.cpp).
vcr_status crown_bounds_in(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m, float *lb,
                           float *ub, char *base, size_t bytes);
}  // namespace vcr
