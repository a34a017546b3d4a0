// C ABI of vcrown: network loading, argument validation, the batching planner and the
// sequence of kernel launches of one bounds call.
//
// One CROWN call on an MLP  z_k = W_k h_{k-1} + b_k,  h_k = ReLU(z_k),  f = z_L:
//   1. box (centre/radius) and one pure IBP forward pass over all layers;
//   2. ReLU 1: bounds of z_1 = the exact box range of one affine map (equals IBP);
//   3. ReLU k >= 2: rows [W_k; -W_k] for every input (the lower and the negated upper
//      bound of every neuron of z_k), relaxed through ReLU k-1, then one GEMM per layer
//      W_{k-1} .. W_2 whose epilogue relaxes the next ReLU, and a last GEMM with W_1 whose
//      epilogue concretizes over the box; finally l, u, intersection with IBP and the new
//      relaxation;
//   4. the spec pass: rows [C W_L; -C W_L] per input through the same chain.
// With branch-and-bound splits the root input runs 1-3 once; step 4 then runs over all
// subdomains, whose relaxations differ from the root's only at their split neurons.
//
// Rows never straddle inputs within a GEMM row block of an intermediate pass (2 n_k rows
// per input), every output element has its own fixed-order K sum, and every reduction
// runs in a fixed order: bounds are bitwise independent of batch size and chunking.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <string>
#include <vector>

#include "conv.h"
#include "ctx.h"

using namespace vcr;

namespace vcr {
vcr_status graph_load(vcr_ctx *c, const vcr_node *nodes, int32_t n, const int32_t in_chw[3],
                      const std::vector<std::vector<int64_t>> &sh);
vcr_status graph_crown(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                       const vcr_splits *splits, float *lb, float *ub);
vcr_status graph_ibp(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m, float *lb,
                     float *ub);
vcr_status graph_alpha(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                       const vcr_alpha_opts &o, int64_t n_total, float *lb, float *ub);
vcr_status graph_beta(vcr_ctx *c, const float *x0, float eps, const float *C, int32_t m, const vcr_splits *splits,
                      const vcr_alpha_opts &o, int64_t n_total, float lr_beta, float *lb, float *ub);
size_t graph_workspace_bytes(vcr_ctx *c, int32_t B, int32_t m, int32_t D, int32_t S, bool alpha);
vcr_status graph_plan(vcr_ctx *c, int32_t B, int32_t m, int *chunk_out, size_t *bytes_out, bool alpha);
}  // namespace vcr

namespace {

void free_layers(vcr_ctx *c) {
  for (auto &L : c->layers) {
    if (L.Wp) (void)hipFree(L.Wp);
    if (L.Bt) (void)hipFree(L.Bt);
    if (L.b) (void)hipFree(L.b);
  }
  c->layers.clear();
}

void free_ws(vcr_ctx *c) {
  if (c->ws.base) (void)hipFree(c->ws.base);
  c->ws = Workspace{};
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ---- workspace planning ------------------------------------------------------------
struct Plan {
  int32_t B = 0, m = 0, D = 0;
  int32_t alpha = 0;        // alpha-CROWN state for the spec pass
  int32_t chunk_in = 0;     // inputs per intermediate-pass chunk
  int32_t chunk_units = 0;  // inputs (or domains) per spec-pass chunk
  size_t bytes = 0;
};


int64_t max_inter_rows_per_input(const vcr_ctx *c) {
  int64_t r = 0;
  const int L = (int)c->layers.size();
  for (int k = 1; k < L - 1; ++k) r = std::max<int64_t>(r, 2 * (int64_t)c->layers[k].n_out);
  return r;
}

size_t carve_bytes(const vcr_ctx *c, const Plan &p, int32_t S);

vcr_status make_plan(vcr_ctx *c, int32_t B, int32_t m, int32_t D, int32_t S, Plan *p, int32_t alpha = 0) {
  p->B = B;
  p->m = m;
  p->D = D;
  p->alpha = alpha;
  const int64_t rpi = max_inter_rows_per_input(c);
  const int32_t spec_units = D > 0 ? D : B;
  const int32_t root_B = D > 0 ? 1 : B;
  auto need = [&](int32_t ci, int32_t cu) {
    Plan q = *p;
    q.chunk_in = ci;
    q.chunk_units = cu;
    return carve_bytes(c, q, S);
  };
  int32_t ci = std::max(root_B, 1), cu = std::max(spec_units, 1);
  if (c->ws_cap > 0) {
    while (need(ci, cu) > c->ws_cap && (ci > 1 || cu > 1)) {
      // shrink the larger row block first
      if (rpi * ci >= 2 * (int64_t)m * cu && ci > 1)
        ci = (ci + 1) / 2;
      else if (cu > 1)
        cu = (cu + 1) / 2;
      else
        ci = (ci + 1) / 2;
    }
    if (need(ci, cu) > c->ws_cap)
      return fail(c, VCR_ERR_OOM, "workspace cap %llu bytes is below the minimum plan (%llu bytes)",
                  (unsigned long long)c->ws_cap, (unsigned long long)need(ci, cu));
  }
  p->chunk_in = ci;
  p->chunk_units = cu;
  p->bytes = need(ci, cu);
  return VCR_OK;
}

}  // namespace

vcr_status ensure_ws(vcr_ctx *c, size_t bytes) {
  if (c->ws.cap >= bytes) {
    c->ws.used = 0;
    return VCR_OK;
  }
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  free_ws(c);
  void *p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(c, VCR_ERR_OOM, "hipMalloc(%llu) failed: %s", (unsigned long long)bytes, hipGetErrorString(e));
  }
  c->ws.base = static_cast<char *>(p);
  c->ws.cap = bytes;
  c->ws.used = 0;
  c->peak_ws = std::max<uint64_t>(c->peak_ws, bytes);
  // the A buffers' padding rows/columns are read by the GEMM: start from zeros
  HIP_TRY(c, launch_fill(reinterpret_cast<float *>(p), (int64_t)(bytes / 4), 0.f, c->stream));
  return VCR_OK;
}

namespace {


// ---- validation ---------------------------------------------------------------------
vcr_status validate_net(vcr_ctx *c, const vcr_node *nodes, int32_t n, const int32_t in_chw[3],
                        std::vector<std::vector<int64_t>> *shapes_out) {
  if (!nodes || n <= 0 || !in_chw) return fail(c, VCR_ERR_ARG, "empty network");
  if (in_chw[0] <= 0 || in_chw[1] <= 0 || in_chw[2] <= 0) return fail(c, VCR_ERR_SHAPE, "bad input shape");
  if ((int64_t)in_chw[0] * in_chw[1] * in_chw[2] > VCR_MAX_NODE_ELEMENTS)
    return fail(c, VCR_ERR_SHAPE, "the input exceeds the limit of %lld elements", (long long)VCR_MAX_NODE_ELEMENTS);
  std::vector<std::vector<int64_t>> sh;
  const std::vector<int64_t> in_shape = {in_chw[0], in_chw[1], in_chw[2]};
  auto shape_of = [&](int32_t i) -> const std::vector<int64_t> & { return i == -1 ? in_shape : sh[i]; };
  auto numel = [](const std::vector<int64_t> &s) {
    int64_t p = 1;
    for (auto v : s) p *= v;
    return p;
  };
  for (int32_t i = 0; i < n; ++i) {
    const vcr_node &nd = nodes[i];
    if (nd.in0 < -1 || nd.in0 >= i) return fail(c, VCR_ERR_ARG, "node %d: in0=%d is not an earlier node", i, nd.in0);
    const std::vector<int64_t> s = shape_of(nd.in0);   // a copy: sh grows below
    switch (nd.op) {
      case VCR_DENSE: {
        if (!nd.W || !nd.b) return fail(c, VCR_ERR_ARG, "node %d: dense without weights", i);
        if (nd.out_features <= 0) return fail(c, VCR_ERR_SHAPE, "node %d: out_features <= 0", i);
        sh.push_back({nd.out_features, 1, 1});
        break;
      }
      case VCR_CONV2D: {
        if (!nd.W || !nd.b) return fail(c, VCR_ERR_ARG, "node %d: conv without weights", i);
        if (nd.out_ch <= 0 || nd.kh <= 0 || nd.kw <= 0 || nd.stride <= 0 || nd.pad < 0)
          return fail(c, VCR_ERR_SHAPE, "node %d: bad conv geometry", i);
        const int64_t ho = (s[1] + 2 * nd.pad - nd.kh) / nd.stride + 1;
        const int64_t wo = (s[2] + 2 * nd.pad - nd.kw) / nd.stride + 1;
        if (ho <= 0 || wo <= 0) return fail(c, VCR_ERR_SHAPE, "node %d: conv output is empty", i);
        sh.push_back({nd.out_ch, ho, wo});
        break;
      }
      case VCR_RELU:
        sh.push_back(s);
        break;
      case VCR_ADD: {
        if (nd.in1 < -1 || nd.in1 >= i) return fail(c, VCR_ERR_ARG, "node %d: in1=%d is not an earlier node", i, nd.in1);
        if (shape_of(nd.in1) != s) return fail(c, VCR_ERR_SHAPE, "node %d: add inputs differ in shape", i);
        sh.push_back(s);
        break;
      }
      case VCR_FLATTEN:
        sh.push_back({numel(s), 1, 1});
        break;
      default:
        return fail(c, VCR_ERR_ARG, "node %d: unknown op %d", i, nd.op);
    }
    // size limits: kernel index arithmetic is 32-bit within a row and 64-bit across rows
    if (numel(sh.back()) > VCR_MAX_NODE_ELEMENTS)
      return fail(c, VCR_ERR_SHAPE, "node %d: %lld elements exceed the limit of %lld", i, (long long)numel(sh.back()),
                  (long long)VCR_MAX_NODE_ELEMENTS);
    const int64_t weights = nd.op == VCR_DENSE    ? (int64_t)nd.out_features * numel(s)
                            : nd.op == VCR_CONV2D ? (int64_t)nd.out_ch * s[0] * nd.kh * nd.kw
                                                  : 0;
    if ((nd.op == VCR_DENSE || nd.op == VCR_CONV2D) &&
        (nd.out_features > VCR_MAX_NODE_ELEMENTS || nd.kh > 64 || nd.kw > 64 || weights > VCR_MAX_LAYER_WEIGHTS))
      return fail(c, VCR_ERR_SHAPE, "node %d: %lld weights exceed the limit of %lld", i, (long long)weights,
                  (long long)VCR_MAX_LAYER_WEIGHTS);
  }
  if (nodes[n - 1].op != VCR_DENSE) return fail(c, VCR_ERR_ARG, "the output node must be dense");
  *shapes_out = sh;
  return VCR_OK;
}

// The dense path handles the MLP chain dense (relu dense)*; UNSUPPORTED otherwise (the caller
// then loads the network on the graph path).
vcr_status check_chain(vcr_ctx *c, const vcr_node *nodes, int32_t n, const int32_t in_chw[3],
                       const std::vector<std::vector<int64_t>> &sh) {
  if (in_chw[1] != 1 || in_chw[2] != 1)
    return fail(c, VCR_ERR_UNSUPPORTED, "the dense path takes flat inputs only (got a %dx%dx%d input)",
                in_chw[0], in_chw[1], in_chw[2]);
  (void)sh;
  for (int32_t i = 0; i < n; ++i) {
    const vcr_node &nd = nodes[i];
    const bool want_dense = (i % 2 == 0);
    if (want_dense) {
      if (nd.op != VCR_DENSE || nd.in0 != i - 1)
        return fail(c, VCR_ERR_UNSUPPORTED,
                    "node %d: the dense path takes chains dense (relu dense)* only", i);
    } else {
      if (nd.op != VCR_RELU || nd.in0 != i - 1)
        return fail(c, VCR_ERR_UNSUPPORTED,
                    "node %d: the dense path takes chains dense (relu dense)* only", i);
    }
  }
  return VCR_OK;
}

}  // namespace

// =====================================================================================
vcr_status timing_fold(vcr_ctx *c) {
  if (!c->ev_used) return VCR_OK;
  HIP_TRY(c, hipEventSynchronize(c->ev_pool[c->ev_used - 1]));
  for (size_t q = 0; q + 1 < c->ev_used; q += 2) {
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, c->ev_pool[q], c->ev_pool[q + 1]));
    const auto &pk = c->pending[q / 2];
    c->timed_ms[pk.second] += ms;
    c->timed_flops[pk.second] += pk.first;
    ++c->timed_launches[pk.second];
  }
  c->ev_used = 0;
  c->pending.clear();
  return VCR_OK;
}

extern "C" {

int32_t vcr_abi_version(void) { return VCR_ABI_VERSION; }

vcr_status vcr_create(int32_t hip_device, vcr_ctx **out) {
  if (!out) return VCR_ERR_ARG;
  *out = nullptr;
  vcr_ctx *c = new (std::nothrow) vcr_ctx();
  if (!c) return VCR_ERR_OOM;
  c->device = hip_device;
  if (hip_device >= 0) {
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || hip_device >= n) {
      delete c;
      return VCR_ERR_DEVICE;
    }
    if (hipSetDevice(hip_device) != hipSuccess) {
      delete c;
      return VCR_ERR_DEVICE;
    }
    if (hipMalloc(&c->d_counters, 80 * sizeof(int32_t)) != hipSuccess) {
      delete c;
      return VCR_ERR_OOM;
    }
    if (vcr::noalloc_setup(c) != VCR_OK) {
      (void)hipFree(c->d_counters);
      delete c;
      return VCR_ERR_DEVICE;
    }
  } else if (hip_device != -1) {
    delete c;
    return VCR_ERR_ARG;
  }
  *out = c;
  return VCR_OK;
}

void vcr_destroy(vcr_ctx *c) {
  if (!c) return;
  if (c->device >= 0) {
    (void)hipSetDevice(c->device);
    (void)hipStreamSynchronize(c->stream);
    free_layers(c);
    free_ws(c);
    if (c->d_counters) (void)hipFree(c->d_counters);
    if (c->bab_buf) (void)hipFree(c->bab_buf);
    if (c->root_cache) (void)hipFree(c->root_cache);
    for (auto e : c->ev_pool) (void)hipEventDestroy(e);
    if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
    if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  }
  destroy_graph(c->graph);
  delete c;
}

const char *vcr_last_error(const vcr_ctx *c) { return c ? c->err.c_str() : "null context"; }

vcr_status vcr_set_stream(vcr_ctx *c, void *s) {
  if (!c) return VCR_ERR_ARG;
  c->stream = static_cast<hipStream_t>(s);
  return VCR_OK;
}

vcr_status vcr_set_option(vcr_ctx *c, int32_t key, double v) {
  if (!c) return VCR_ERR_ARG;
  if (!std::isfinite(v)) return fail(c, VCR_ERR_ARG, "option %d: value is not finite", key);
  switch (key) {
    case VCR_OPT_CLIP_ENABLE: c->clip_on = v != 0.0; break;
    case VCR_OPT_CLIP_LO: c->clip_lo = (float)v; break;
    case VCR_OPT_CLIP_HI: c->clip_hi = (float)v; break;
    case VCR_OPT_INTERSECT_IBP: c->intersect = v != 0.0; break;
    case VCR_OPT_WORKSPACE_CAP_BYTES:
      if (v < 0) return fail(c, VCR_ERR_ARG, "workspace cap < 0");
      c->ws_cap = (uint64_t)v;
      break;
    case VCR_OPT_SYNC_CHECK: c->sync_check = v != 0.0; break;
    case VCR_OPT_CHECK_FINITE: c->check_finite = v != 0.0; break;
    case VCR_OPT_LAMBDA_RULE:
      if (v != VCR_LAMBDA_ADAPTIVE && v != VCR_LAMBDA_ZERO && v != VCR_LAMBDA_ONE && v != VCR_LAMBDA_SAME_SLOPE)
        return fail(c, VCR_ERR_ARG, "lambda rule %g is not one of VCR_LAMBDA_*", v);
      c->lambda_rule = (int32_t)v;
      break;
    case VCR_OPT_GRAPH:
      c->use_graph = v != 0.0;
      if (!c->use_graph && c->gexec) {
        (void)hipGraphExecDestroy(c->gexec);
        c->gexec = nullptr;
      }
      break;
    case VCR_OPT_TIME_GEMM:
      if (c->device >= 0 && c->ev_used) (void)hipStreamSynchronize(c->stream);
      c->time_gemm = v != 0.0;
      c->ev_used = 0;
      c->pending.clear();
      for (int k = 0; k < 4; ++k) {
        c->timed_launches[k] = c->timed_flops[k] = 0;
        c->timed_ms[k] = 0.0;
      }
      break;
    default: return fail(c, VCR_ERR_ARG, "unknown option %d", key);
  }
  return VCR_OK;
}

vcr_status vcr_load_net(vcr_ctx *c, const vcr_node *nodes, int32_t n, const int32_t in_chw[3]) {
  if (!c) return VCR_ERR_ARG;
  ++c->net_epoch;   // any recorded graph refers to the previous weights
  if (c->gexec) {
    (void)hipGraphExecDestroy(c->gexec);
    c->gexec = nullptr;
  }
  std::vector<std::vector<int64_t>> sh;
  vcr_status st = validate_net(c, nodes, n, in_chw, &sh);
  if (st != VCR_OK) return st;
  c->n_out = nodes[n - 1].out_features;
  // dense weight shapes must match their inputs
  for (int32_t i = 0; i < n; ++i) {
    if (nodes[i].op != VCR_DENSE) continue;
    const auto &s = nodes[i].in0 == -1 ? std::vector<int64_t>{in_chw[0], in_chw[1], in_chw[2]} : sh[nodes[i].in0];
    if (s[1] != 1 || s[2] != 1)
      return fail(c, VCR_ERR_SHAPE, "node %d: dense input must be flat (insert a flatten node)", i);
  }
  st = check_chain(c, nodes, n, in_chw, sh);
  if (st == VCR_ERR_UNSUPPORTED) {
    // not an MLP chain: the convolutional-network path
    const std::string mlp_err = c->err;
    if (c->device >= 0) {
      HIP_TRY(c, hipSetDevice(c->device));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
      free_layers(c);
      free_ws(c);
    }
    c->loaded = false;
    c->layers.clear();
    st = graph_load(c, nodes, n, in_chw, sh);
    if (st != VCR_OK) return st;
    c->loaded = true;
    return VCR_OK;
  }
  if (st != VCR_OK) return st;
  destroy_graph(c->graph);
  c->graph = nullptr;
  if (c->device < 0) {
    // validation-only context: remember the shapes for argument checks
    c->loaded = true;
    c->n0 = in_chw[0];
    c->layers.clear();
    c->relu_n.clear();
    int64_t prev = in_chw[0];
    for (int32_t i = 0; i < n; ++i) {
      if (nodes[i].op == VCR_DENSE) {
        DenseLayer L;
        L.n_in = (int32_t)prev;
        L.n_out = nodes[i].out_features;
        L.ld_in = ld_of(L.n_in);
        L.ld_out = ld_of(L.n_out);
        c->layers.push_back(L);
        prev = L.n_out;
      } else {
        c->relu_n.push_back((int32_t)prev);
      }
    }
    return VCR_OK;
  }
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  free_layers(c);
  free_ws(c);
  c->loaded = false;
  c->relu_n.clear();
  c->n0 = in_chw[0];
  int64_t prev = in_chw[0];
  float *staging = nullptr;
  for (int32_t i = 0; i < n; ++i) {
    if (nodes[i].op == VCR_RELU) {
      c->relu_n.push_back((int32_t)prev);
      continue;
    }
    DenseLayer L;
    L.n_in = (int32_t)prev;
    L.n_out = nodes[i].out_features;
    L.ld_in = ld_of(L.n_in);
    L.ld_out = ld_of(L.n_out);
    const size_t wbytes = sizeof(float) * (size_t)L.n_out * L.n_in;
    HIP_TRY(c, hipMalloc(&staging, wbytes));
    HIP_TRY(c, hipMemcpy(staging, nodes[i].W, wbytes, hipMemcpyHostToDevice));
    HIP_TRY(c, hipMalloc(&L.Wp, sizeof(float) * (size_t)L.ld_out * L.ld_in));
    HIP_TRY(c, hipMalloc(&L.Bt, sizeof(float) * (size_t)L.ld_in * L.ld_out));
    HIP_TRY(c, hipMalloc(&L.b, sizeof(float) * (size_t)L.ld_out));
    c->layers.push_back(L);
    // Wp: row-major copy, zero-padded to [ld_out][ld_in] (a transpose of the transpose); the
    // alpha-CROWN gradient pass uses it as a GEMM operand
    HIP_TRY(c, launch_transpose_pad(staging, L.n_out, L.n_in, L.Bt, L.ld_out, L.ld_in, c->stream));
    HIP_TRY(c, launch_transpose_pad(L.Bt, (int32_t)L.ld_in, (int32_t)L.ld_out, L.Wp, L.ld_in, L.ld_out, c->stream));
    HIP_TRY(c, launch_fill(L.b, L.ld_out, 0.f, c->stream));
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    HIP_TRY(c, hipMemcpy(L.b, nodes[i].b, sizeof(float) * L.n_out, hipMemcpyHostToDevice));
    HIP_TRY(c, hipFree(staging));
    staging = nullptr;
    prev = L.n_out;
  }
  HIP_TRY(c, hipDeviceSynchronize());
  c->net_bytes = 0;
  for (const DenseLayer &L : c->layers)
    c->net_bytes += sizeof(float) * (2 * (uint64_t)L.ld_in * L.ld_out + (uint64_t)L.ld_out);
  c->loaded = true;
  return VCR_OK;
}

}  // extern "C"

namespace {

struct CallBufs {
  float *c0, *r0;
  std::vector<float *> ibp_c, ibp_r, Lb, Ub;
  std::vector<float4 *> P;
  float *CW, *Cb;
  float *A[2], *beta, *part, *cpart;
  // splits
  int32_t *off, *ent_n, *flags;
  float4 *ent_p;
  const float **Lptr, **Uptr;
  int32_t *relu_n;
  // alpha-CROWN (one entry per ReLU), the input-layer coefficients, the best row bounds
  std::vector<AlphaLayer> al;
  float *pre0, *best_val;
  int32_t *flag;
  float *tmp_c, *tmp_r;   // ReLU'd IBP inputs of large layers
  // beta-CROWN multipliers of the split entries [rows][S] and their Adam state
  float *mul, *mul_mom, *mul_vel, *mul_grad;
};

vcr_status check_common(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                        const float *lb, const float *ub) {
  if (!c->loaded) return fail(c, VCR_ERR_STATE, "no network loaded");
  if (B <= 0) return fail(c, VCR_ERR_ARG, "B must be > 0");
  if (m <= 0) return fail(c, VCR_ERR_ARG, "m must be > 0");
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(c, VCR_ERR_ARG, "eps must be finite and >= 0");
  if (!x0 || !C || !lb || !ub) return fail(c, VCR_ERR_ARG, "null tensor pointer");
  if (!aligned16(x0) || !aligned16(C) || !aligned16(lb) || !aligned16(ub))
    return fail(c, VCR_ERR_ARG, "tensor pointers must be 16-byte aligned");
  if ((int64_t)B * m > (int64_t)1 << 30) return fail(c, VCR_ERR_SHAPE, "B * m too large");
  if (c->clip_on && !(c->clip_lo <= c->clip_hi)) return fail(c, VCR_ERR_ARG, "clip_lo > clip_hi");
  return VCR_OK;
}

// VCR_OPT_CHECK_FINITE: count the non-finite values of x0 (B x n0) and C (B x m x n_out) on
// the device before anything else is queued (synchronises).
vcr_status check_finite_inputs(vcr_ctx *c, const float *x0, int32_t B, const float *C, int32_t m) {
  if (!c->check_finite || c->device < 0) return VCR_OK;
  HIP_TRY(c, hipSetDevice(c->device));
  int32_t *cnt = c->d_counters + 65;
  HIP_TRY(c, launch_fill(reinterpret_cast<float *>(cnt), 1, 0.f, c->stream));
  HIP_TRY(c, launch_count_nonfinite(x0, (int64_t)B * c->n0, cnt, c->stream));
  HIP_TRY(c, launch_count_nonfinite(C, (int64_t)B * m * c->n_out, cnt, c->stream));
  int32_t host = 0;
  HIP_TRY(c, hipMemcpyAsync(&host, cnt, sizeof(int32_t), hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  if (host > 0) return fail(c, VCR_ERR_ARG, "x0 or C holds %d non-finite value(s)", host);
  return VCR_OK;
}

// IBP through dense layer W (c' = W c + b, r' = |W| r, after a ReLU on the input when
// relu_in).  Large layers run as two fp32 MFMA GEMMs; the choice depends on the layer's size
// only, so an input's bounds do not depend on the batch it is in.  cin/rin and cout/rout
// hold rows_pad(B) rows; tmp_c/tmp_r (same shape as cin) take the ReLU'd input.
constexpr int64_t IBP_MFMA_MIN_WEIGHTS = (int64_t)1 << 24;
bool ibp_on_mfma(const DenseLayer &W) { return (int64_t)W.n_out * W.n_in >= IBP_MFMA_MIN_WEIGHTS; }

vcr_status ibp_layer(vcr_ctx *c, const DenseLayer &W, const float *cin, const float *rin, bool relu_in, float *cout,
                     float *rout, int32_t B, float *tmp_c, float *tmp_r, hipStream_t s, uint64_t *flops = nullptr) {
  if (!ibp_on_mfma(W)) {
    HIP_TRY(c, launch_ibp_dense(W.Wp, W.ld_in, W.b, W.n_out, W.n_in, cin, rin, W.ld_in, relu_in, cout, rout, W.ld_out,
                                B, s));
    return VCR_OK;
  }
  const int64_t M_pad = rows_pad(B);
  if (relu_in) {
    HIP_TRY(c, launch_ibp_relu(cin, rin, tmp_c, tmp_r, M_pad * W.ld_in, s));
    cin = tmp_c;
    rin = tmp_r;
  }
  GemmArgs g{};
  g.lda = W.ld_in;
  g.Bt = W.Wp;
  g.ldb = W.ld_in;
  g.M = B;
  g.M_pad = (int32_t)M_pad;
  g.K = (int32_t)W.ld_in;
  g.N_pad = (int32_t)W.ld_out;
  g.mode = EPI_AFFINE;
  g.ldo = W.ld_out;
  g.rows_per_unit = (int32_t)M_pad;
  g.n_units = 1;
  g.A = cin;
  g.out = cout;
  g.bias = W.b;
  const uint64_t gf = 2ull * (uint64_t)B * (uint64_t)W.n_out * (uint64_t)W.n_in;
  if (flops) *flops += 2 * gf;
  vcr_status st = TIMED_GEMM(c, s, gf, g);
  if (st != VCR_OK) return st;
  g.A = rin;
  g.out = rout;
  g.bias = nullptr;
  g.abs_b = 1;
  return TIMED_GEMM(c, s, gf, g);
}

bool any_ibp_relu_on_mfma(const vcr_ctx *c) {
  for (size_t k = 1; k + 1 < c->layers.size(); ++k)
    if (ibp_on_mfma(c->layers[k])) return true;
  return false;
}

void carve(const vcr_ctx *c, Workspace &w, const Plan &p, int32_t S, CallBufs *bf) {
  const int L = (int)c->layers.size();
  const int32_t B = p.B;
  const int64_t Bp = rows_pad(B);   // IBP arrays are GEMM operands on large layers
  const int64_t ld0 = ld_of(c->n0);
  bf->c0 = take<float>(w, (size_t)Bp * ld0);
  bf->r0 = take<float>(w, (size_t)Bp * ld0);
  bf->ibp_c.clear(); bf->ibp_r.clear(); bf->Lb.clear(); bf->Ub.clear(); bf->P.clear();
  for (int k = 0; k < L - 1; ++k) {
    const int64_t ld = c->layers[k].ld_out, n = c->layers[k].n_out;
    bf->ibp_c.push_back(take<float>(w, (size_t)Bp * ld));
    bf->ibp_r.push_back(take<float>(w, (size_t)Bp * ld));
    bf->Lb.push_back(take<float>(w, (size_t)B * n));
    bf->Ub.push_back(take<float>(w, (size_t)B * n));
    bf->P.push_back(take<float4>(w, (size_t)B * ld));
  }
  const int64_t ldcw = L >= 2 ? c->layers[L - 1].ld_in : ld0;
  bf->CW = take<float>(w, (size_t)B * p.m * ldcw);
  bf->Cb = take<float>(w, (size_t)B * p.m);
  if (p.D > 0) {
    const int R = (int)c->relu_n.size();
    bf->off = take<int32_t>(w, (size_t)p.D * (R + 1));
    bf->ent_n = take<int32_t>(w, (size_t)p.D * S);
    bf->ent_p = take<float4>(w, (size_t)p.D * S);
    bf->flags = take<int32_t>(w, p.D);
    bf->Lptr = take<const float *>(w, 2 * R);
    bf->Uptr = bf->Lptr ? bf->Lptr + R : nullptr;   // null while only counting bytes
    bf->relu_n = take<int32_t>(w, R);
  }
  const int64_t rpi = max_inter_rows_per_input(c);
  const int64_t rows = std::max<int64_t>({rpi * p.chunk_in, 2 * (int64_t)p.m * p.chunk_units, 1});
  int64_t ldmax = 0;
  for (int k = 0; k < L - 1; ++k) ldmax = std::max(ldmax, c->layers[k].ld_out);
  if (p.alpha) ldmax = std::max(ldmax, ld0);   // the gradient pass starts at the input
  const int64_t mp = rows_pad(rows);
  bf->al.clear();
  if (p.alpha) {
    const int64_t ra = rows_pad(2 * (int64_t)p.m * p.chunk_units);
    int32_t col0 = 0;
    for (int k = 0; k < L - 1; ++k) {
      AlphaLayer a{};
      a.ld = c->layers[k].ld_out;
      a.ldp = a.ld;
      a.n = c->layers[k].n_out;
      a.col0 = col0;
      col0 += a.n;
      a.alpha = take<float>(w, (size_t)ra * a.ld);
      a.mom = take<float>(w, (size_t)ra * a.ld);
      a.vel = take<float>(w, (size_t)ra * a.ld);
      a.best = take<float>(w, (size_t)ra * a.ld);
      a.grad = take<float>(w, (size_t)ra * a.ld);
      a.pre = take<float>(w, (size_t)ra * a.ld);
      bf->al.push_back(a);
    }
    bf->pre0 = take<float>(w, (size_t)ra * ld0);
    bf->best_val = take<float>(w, (size_t)ra);
    bf->flag = take<int32_t>(w, (size_t)ra);
    bf->mul = bf->mul_mom = bf->mul_vel = bf->mul_grad = nullptr;
    if (p.D > 0 && S > 0) {
      bf->mul = take<float>(w, (size_t)ra * S);
      bf->mul_mom = take<float>(w, (size_t)ra * S);
      bf->mul_vel = take<float>(w, (size_t)ra * S);
      bf->mul_grad = take<float>(w, (size_t)ra * S);
    }
  }
  bf->A[0] = take<float>(w, (size_t)mp * std::max<int64_t>(ldmax, 1));
  bf->A[1] = take<float>(w, (size_t)mp * std::max<int64_t>(ldmax, 1));
  bf->beta = take<float>(w, (size_t)mp);
  bf->part = take<float>(w, (size_t)mp * std::max<int64_t>(ldmax / PART_COLS, 1));
  bf->cpart = take<float>(w, (size_t)mp * (ld0 / PART_COLS));
  bf->tmp_c = bf->tmp_r = nullptr;
  if (any_ibp_relu_on_mfma(c)) {
    bf->tmp_c = take<float>(w, (size_t)Bp * std::max<int64_t>(ldmax, 1));
    bf->tmp_r = take<float>(w, (size_t)Bp * std::max<int64_t>(ldmax, 1));
  }
}

size_t carve_bytes(const vcr_ctx *c, const Plan &p, int32_t S) {
  Workspace w;
  CallBufs bf;
  carve(c, w, p, S, &bf);
  return w.used;
}

// One backward pass through layers j = top .. 1 for `units` units of rows_per_unit rows
// that start in A[0] (already relaxed for ReLU top-1... i.e. coefficients on z_top).
// Leaves beta with the constants and cpart with the concretization partials.
vcr_status run_chain(vcr_ctx *c, CallBufs &bf, int top, int32_t M, int32_t rows_per_unit, int32_t units,
                     int32_t unit0, int32_t param_per_unit, const SplitTable &st, uint64_t *flops,
                     bool with_alpha = false) {
  const int32_t M_pad = (int32_t)rows_pad(M);
  int cur = 0;
  for (int j = top; j >= 1; --j) {
    const DenseLayer &W = c->layers[j - 1];   // layer j: z_j = W_j h_{j-1} + b_j
    GemmArgs g{};
    g.A = bf.A[cur];
    g.lda = W.ld_out;
    g.Bt = W.Bt;
    g.ldb = W.ld_out;
    g.M = M;
    g.M_pad = M_pad;
    g.K = (int32_t)W.ld_out;
    g.N_pad = (int32_t)W.ld_in;
    g.rows_per_unit = param_per_unit ? rows_per_unit : M_pad;
    g.n_units = param_per_unit ? units : 1;
    g.splits = st;
    const int64_t pu0 = param_per_unit ? unit0 : 0;
    if (j >= 2) {
      const int r = j - 2;   // ReLU on z_{j-1}
      g.mode = EPI_RELAX;
      g.out = bf.A[cur ^ 1];
      g.ldo = W.ld_in;
      g.P = bf.P[r] + pu0 * W.ld_in;
      g.ldp = W.ld_in;
      g.relu_index = r;
      g.part = bf.part;
      if (with_alpha) {
        g.alpha = bf.al[r].alpha;
        g.ld_alpha = bf.al[r].ld;
        g.pre = bf.al[r].pre;
        g.ld_pre = bf.al[r].ld;
      }
    } else {
      g.mode = EPI_CONCRETIZE;
      g.c0 = bf.c0 + pu0 * ld_of(c->n0);
      g.r0 = bf.r0 + pu0 * ld_of(c->n0);
      g.ldc = ld_of(c->n0);
      g.part = bf.cpart;
      if (with_alpha) {
        g.pre = bf.pre0;
        g.ld_pre = ld_of(c->n0);
      }
    }
    const uint64_t gf = 2ull * (uint64_t)M * (uint64_t)W.n_out * (uint64_t)W.n_in;
    {
      const vcr_status st = TIMED_GEMM(c, c->stream, gf, g);
      if (st != VCR_OK) return st;
    }
    *flops += gf;
    if (j >= 2) {
      HIP_TRY(c, launch_rowsum(bf.beta, bf.part, (int32_t)(W.ld_in / PART_COLS), M_pad, M, c->stream));
      cur ^= 1;
    }
  }
  return VCR_OK;
}

struct AlphaCall {
  vcr_alpha_opts o;
  int64_t n_total;
  float lr_beta = 0.f;   // subdomains (beta-CROWN): step size of the multipliers
};

// alpha-CROWN final pass (after the intermediate bounds are fixed) over every chunk of units:
// inputs, or subdomains of the root input (beta-CROWN: each split adds a multiplier).  Each
// step evaluates the bounds with the current slopes and multipliers (backward chain with
// per-row slopes and split terms, keeping the coefficients before each relaxation), keeps
// each row's best, then runs the gradient pass (the relaxed network forward from each row's
// box vertex) and one projected Adam step on both.
vcr_status alpha_spec(vcr_ctx *c, CallBufs &bf, const Plan &p, const AlphaCall &ac, int32_t units, int32_t m,
                      int32_t S, float *lb, float *ub, uint64_t *flops, int32_t *chunks) {
  const int L = (int)c->layers.size();
  const int R = L - 1;
  const bool dom = p.D > 0;   // subdomains of one root input (shared relaxation, split table)
  const DenseLayer &WL = c->layers[L - 1];
  const int64_t ld0 = ld_of(c->n0);
  hipStream_t s = c->stream;
  const vcr_alpha_opts &o = ac.o;
  const int Rn = (int)c->relu_n.size();
  for (int32_t u0 = 0; u0 < units; u0 += p.chunk_units) {
    const int32_t uc = std::min(p.chunk_units, units - u0);
    const int32_t rpu = 2 * m;
    const int32_t M = rpu * uc;
    const int32_t M_pad = (int32_t)rows_pad(M);
    // per-unit parameters (inputs) or the root's for every row (subdomains)
    const int32_t prpu = dom ? M_pad : rpu;
    const int64_t pu0 = dom ? 0 : u0;
    const int32_t pun = dom ? 1 : uc;
    SplitTable tab{};
    BetaState bs{bf.mul, bf.mul_mom, bf.mul_vel, bf.mul_grad, S};
    if (dom) {
      tab.off = bf.off + (int64_t)u0 * (Rn + 1);
      tab.ent_n = bf.ent_n + (int64_t)u0 * S;
      tab.ent_p = bf.ent_p + (int64_t)u0 * S;
      tab.R = Rn;
      tab.S = S;
      tab.D = uc;
      tab.rows_per_domain = rpu;
      tab.beta = S > 0 ? bf.mul : nullptr;
      HIP_TRY(c, launch_beta_init(bs, M_pad, s));
    }
    std::vector<AlphaLayer> al = bf.al;
    for (int r = 0; r < R; ++r) {
      al[r].P = bf.P[r] + pu0 * al[r].ld;
      HIP_TRY(c, launch_alpha_init(al[r], o.alpha_init ? o.alpha_init + (int64_t)u0 * rpu * ac.n_total : nullptr,
                                   ac.n_total, M, M_pad, prpu, s));
    }
    for (int32_t t = 0; t <= o.iters; ++t) {
      // evaluate
      InitArgs ia{};
      ia.src = bf.CW + (dom ? 0 : (int64_t)u0 * m * WL.ld_in);
      ia.ld_src = WL.ld_in;
      ia.n_src = m;
      ia.per_unit_src = dom ? 0 : 1;
      ia.src_bias = bf.Cb + (dom ? 0 : (int64_t)u0 * m);
      ia.n_cols = WL.n_in;
      ia.ldo = WL.ld_in;
      ia.M = M;
      ia.units = uc;
      ia.P = al[R - 1].P;
      ia.ldp = WL.ld_in;
      ia.param_per_unit = dom ? 0 : 1;
      ia.relu_index = R - 1;
      ia.splits = tab;
      ia.out = bf.A[0];
      ia.beta = bf.beta;
      ia.alpha = al[R - 1].alpha;
      ia.ld_alpha = al[R - 1].ld;
      ia.pre = al[R - 1].pre;
      HIP_TRY(c, launch_init_rows(ia, s));
      vcr_status st = run_chain(c, bf, L - 1, M, rpu, uc, dom ? 0 : u0, dom ? 0 : 1, tab, flops, true);
      if (st != VCR_OK) return st;
      HIP_TRY(c, launch_alpha_best(bf.beta, bf.cpart, (int32_t)(ld0 / PART_COLS), M_pad, M, m, t == 0, bf.best_val,
                                   bf.flag, o.lb_hist ? o.lb_hist + ((int64_t)t * units + u0) * m : nullptr,
                                   o.ub_hist ? o.ub_hist + ((int64_t)t * units + u0) * m : nullptr, s));
      const bool step = t < o.iters;
      // rows that improved keep their slopes: here after the last evaluation, otherwise inside
      // the Adam step below (the gradient pass leaves the slopes unchanged)
      if (!step)
        for (int r = 0; r < R; ++r) HIP_TRY(c, launch_alpha_keep(al[r], bf.flag, M, s));
      if (!step && !o.grad_out) break;
      // gradient: E_0 = the row's box vertex, then E_k = line_k(W_k E_{k-1} + b_k)
      HIP_TRY(c, launch_alpha_vertex(bf.pre0, ld0, bf.c0 + pu0 * ld0, bf.r0 + pu0 * ld0, M_pad, prpu, pun, bf.A[0], s));
      SplitTable ftab = tab;
      ftab.grad_beta = dom && S > 0 ? bf.mul_grad : nullptr;
      for (int k = 1; k <= R; ++k) {
        const DenseLayer &W = c->layers[k - 1];
        GemmArgs g{};
        g.A = bf.A[(k - 1) & 1];
        g.lda = W.ld_in;
        g.Bt = W.Wp;
        g.ldb = W.ld_in;
        g.M = M;
        g.M_pad = M_pad;
        g.K = (int32_t)W.ld_in;
        g.N_pad = (int32_t)W.ld_out;
        g.mode = EPI_FORWARD;
        g.out = bf.A[k & 1];
        g.ldo = W.ld_out;
        g.P = al[k - 1].P;
        g.ldp = W.ld_out;
        g.rows_per_unit = prpu;
        g.n_units = pun;
        g.relu_index = k - 1;
        g.splits = ftab;
        g.alpha = al[k - 1].alpha;
        g.ld_alpha = al[k - 1].ld;
        g.pre = al[k - 1].pre;
        g.ld_pre = al[k - 1].ld;
        g.grad = al[k - 1].grad;
        const uint64_t gf = 2ull * (uint64_t)M * (uint64_t)W.n_out * (uint64_t)W.n_in;
        st = TIMED_GEMM(c, s, gf, g);
        if (st != VCR_OK) return st;
        *flops += gf;
      }
      if (!step) break;
      const double c1 = 1.0 / (1.0 - std::pow((double)o.beta1, (double)(t + 1)));
      const double c2 = 1.0 / (1.0 - std::pow((double)o.beta2, (double)(t + 1)));
      for (int r = 0; r < R; ++r)
        HIP_TRY(c, launch_alpha_adam(al[r], bf.flag, M, prpu, o.lr, o.beta1, o.beta2, o.adam_eps, (float)c1,
                                     (float)c2, s));
      if (dom && S > 0)
        HIP_TRY(c, launch_beta_adam(bs, M, ac.lr_beta, o.beta1, o.beta2, o.adam_eps, (float)c1, (float)c2, s));
    }
    HIP_TRY(c, launch_alpha_final(bf.best_val, uc, m, dom ? bf.flags + u0 : nullptr, lb + (int64_t)u0 * m,
                                  ub + (int64_t)u0 * m, s));
    if (o.alpha_out || o.grad_out)
      for (int r = 0; r < R; ++r)
        HIP_TRY(c, launch_alpha_out(al[r], M, m, ac.n_total,
                                    o.alpha_out ? o.alpha_out + (int64_t)u0 * rpu * ac.n_total : nullptr,
                                    o.grad_out ? o.grad_out + (int64_t)u0 * rpu * ac.n_total : nullptr, s));
    ++*chunks;
  }
  return VCR_OK;
}

vcr_status crown_impl(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                      const vcr_splits *splits, float *lb, float *ub,
                      const AlphaCall *ac = nullptr) {
  const int L = (int)c->layers.size();
  const int R = (int)c->relu_n.size();
  const int32_t D = splits ? splits->n_domains : 0;
  const int32_t S = splits ? splits->per_domain : 0;
  Plan p;
  vcr_status st = make_plan(c, B, m, D, S, &p, ac ? 1 : 0);
  if (st != VCR_OK) return st;
  if (c->device < 0) {
    // report the plan the call would have run
    const int32_t units = D > 0 ? D : B;
    const int32_t rootB = D > 0 ? 1 : B;
    const int32_t n_inter = std::max(L - 2, 0);
    c->chunks_last = n_inter * ((rootB + p.chunk_in - 1) / p.chunk_in) + (L >= 2 ? (units + p.chunk_units - 1) / p.chunk_units : 0);
    return fail(c, VCR_ERR_STATE, "validation-only context: no device work");
  }
  HIP_TRY(c, hipSetDevice(c->device));
  c->lastL.clear();   // the previous call's layer bounds live in the workspace
  c->lastU.clear();
  st = ensure_ws(c, p.bytes);
  if (st != VCR_OK) return st;
  CallBufs bf;
  carve(c, c->ws, p, S, &bf);
  if (c->ws.used > c->ws.cap) return fail(c, VCR_ERR_OOM, "internal: workspace plan too small");
  uint64_t flops = 0;
  int32_t chunks = 0;
  hipStream_t s = c->stream;
  const int64_t ld0 = ld_of(c->n0);

  // the root steps 1-3 of a branch-and-bound round: copied from the loop's first round
  const bool use_cache = D > 0 && c->bab_reuse && c->root_cached;
  const bool fill_cache = D > 0 && c->bab_reuse && !c->root_cached;
  size_t cache_floats = 0;
  for (int r = 0; r < R && D > 0; ++r) cache_floats += 2 * (size_t)c->relu_n[r] + 4 * (size_t)c->layers[r].ld_out;
  auto cache_copy = [&](bool to_cache) -> vcr_status {
    size_t o = 0;
    for (int r = 0; r < R; ++r) {
      const int64_t n = c->relu_n[r], np = 4 * c->layers[r].ld_out;
      float *cl = c->root_cache + o, *cu = cl + n, *cp = cu + n;
      float *pp = reinterpret_cast<float *>(bf.P[r]);
      HIP_TRY(c, launch_copy(to_cache ? cl : bf.Lb[r], to_cache ? bf.Lb[r] : cl, n, s));
      HIP_TRY(c, launch_copy(to_cache ? cu : bf.Ub[r], to_cache ? bf.Ub[r] : cu, n, s));
      HIP_TRY(c, launch_copy(to_cache ? cp : pp, to_cache ? pp : cp, np, s));
      o += 2 * n + np;
    }
    return VCR_OK;
  };

  // 1. box and IBP
  HIP_TRY(c, launch_box(x0, B, c->n0, ld0, eps, c->clip_on, c->clip_lo, c->clip_hi, bf.c0, bf.r0, s));
  if (use_cache) {
    st = cache_copy(false);
    if (st != VCR_OK) return st;
  }
  for (int k = 0; k < L - 1 && !use_cache; ++k) {
    const DenseLayer &W = c->layers[k];
    const float *cin = k == 0 ? bf.c0 : bf.ibp_c[k - 1];
    const float *rin = k == 0 ? bf.r0 : bf.ibp_r[k - 1];
    st = ibp_layer(c, W, cin, rin, k > 0, bf.ibp_c[k], bf.ibp_r[k], B, bf.tmp_c, bf.tmp_r, s, &flops);
    if (st != VCR_OK) return st;
  }
  // 2. first ReLU
  if (L >= 2 && !use_cache)
    HIP_TRY(c, launch_layer_from_ibp(bf.ibp_c[0], bf.ibp_r[0], c->layers[0].ld_out, c->layers[0].n_out, B,
                                     c->layers[0].b, bf.Lb[0], bf.Ub[0], bf.P[0], c->layers[0].ld_out, c->lambda_rule, s));
  // 3. ReLU k >= 2 (layer index k: z_k = layers[k-1]); relu r = k-1
  for (int k = 2; k <= L - 1 && !use_cache; ++k) {
    const DenseLayer &Wk = c->layers[k - 1];
    const int32_t n = Wk.n_out;
    for (int32_t b0 = 0; b0 < B; b0 += p.chunk_in) {
      const int32_t bc = std::min(p.chunk_in, B - b0);
      const int32_t M = 2 * n * bc;
      InitArgs ia{};
      ia.src = Wk.Wp;
      ia.ld_src = Wk.ld_in;
      ia.n_src = n;
      ia.per_unit_src = 0;
      ia.src_bias = Wk.b;
      ia.n_cols = Wk.n_in;
      ia.ldo = Wk.ld_in;
      ia.M = M;
      ia.units = bc;
      ia.P = bf.P[k - 2] + (int64_t)b0 * Wk.ld_in;
      ia.ldp = Wk.ld_in;
      ia.param_per_unit = 1;
      ia.relu_index = k - 2;
      ia.out = bf.A[0];
      ia.beta = bf.beta;
      HIP_TRY(c, launch_init_rows(ia, s));
      st = run_chain(c, bf, k - 1, M, 2 * n, bc, b0, 1, SplitTable{}, &flops);
      if (st != VCR_OK) return st;
      HIP_TRY(c, launch_finalize_layer(bf.beta, bf.cpart, (int32_t)(ld0 / PART_COLS), (int32_t)rows_pad(M), bc, n,
                                       bf.ibp_c[k - 1] + (int64_t)b0 * Wk.ld_out,
                                       bf.ibp_r[k - 1] + (int64_t)b0 * Wk.ld_out, Wk.ld_out, c->intersect, Wk.b,
                                       bf.Lb[k - 1] + (int64_t)b0 * n, bf.Ub[k - 1] + (int64_t)b0 * n,
                                       bf.P[k - 1] + (int64_t)b0 * Wk.ld_out, Wk.ld_out, c->lambda_rule, s));
      ++chunks;
    }
  }
  if (fill_cache) {
    if (c->root_cache_cap < cache_floats) {
      HIP_TRY(c, hipStreamSynchronize(s));
      if (c->root_cache) HIP_TRY(c, hipFree(c->root_cache));
      c->root_cache = nullptr;
      c->root_cache_cap = 0;
      HIP_TRY(c, hipMalloc(&c->root_cache, sizeof(float) * cache_floats));
      c->root_cache_cap = cache_floats;
    }
    st = cache_copy(true);
    if (st != VCR_OK) return st;
    c->root_cached = true;
  }
  // 4. spec pass
  const DenseLayer &WL = c->layers[L - 1];
  const int32_t Bs = D > 0 ? 1 : B;
  HIP_TRY(c, launch_spec_cw(C, Bs, m, WL.n_out, WL.Wp, WL.ld_in, WL.b, WL.n_in, bf.CW, WL.ld_in, bf.Cb, s));
  SplitTable tab{};
  if (D > 0) {
    // the per-ReLU bound pointers for the split preparation: as a kernel argument when they
    // fit one (no wait), else copied from a host array that must outlive the copy
    std::vector<const float *> hp(2 * R);
    for (int r = 0; r < R; ++r) {
      hp[r] = bf.Lb[r];
      hp[R + r] = bf.Ub[r];
    }
    const bool by_arg = 2 * R <= PTR_TABLE_MAX;
    if (by_arg) {
      PtrTable pt{};
      for (int i = 0; i < 2 * R; ++i) pt.p[i] = hp[i];
      HIP_TRY(c, launch_store_ptrs(pt, 2 * R, bf.Lptr, s));
    } else {
      HIP_TRY(c, hipMemcpyAsync(bf.Lptr, hp.data(), sizeof(void *) * 2 * R, hipMemcpyHostToDevice, s));
    }
    HIP_TRY(c, hipMemcpyAsync(bf.relu_n, c->relu_n.data(), sizeof(int32_t) * R, hipMemcpyHostToDevice, s));
    HIP_TRY(c, launch_fill(reinterpret_cast<float *>(c->d_counters), 80, 0.f, s));
    SplitPrepArgs sp{};
    sp.relu_id = splits->relu_id;
    sp.neuron = splits->neuron;
    sp.sign = splits->sign;
    sp.D = D;
    sp.S = S;
    sp.R = R;
    sp.relu_n = bf.relu_n;
    sp.L = bf.Lptr;
    sp.U = bf.Uptr;
    sp.off = bf.off;
    sp.ent_n = bf.ent_n;
    sp.ent_p = bf.ent_p;
    sp.flags = bf.flags;
    sp.n_invalid = c->d_counters + 64;
    sp.lam_rule = c->lambda_rule;
    HIP_TRY(c, launch_split_prepare(sp, s));
    if (!by_arg) HIP_TRY(c, hipStreamSynchronize(s));   // hp must outlive its copy
  }
  const int32_t units = D > 0 ? D : B;
  if (ac) {
    st = alpha_spec(c, bf, p, *ac, units, m, S, lb, ub, &flops, &chunks);
    if (st != VCR_OK) return st;
  } else if (L == 1) {
    HIP_TRY(c, launch_spec_direct(bf.CW, WL.ld_in, bf.Cb, B, m, WL.n_in, bf.c0, bf.r0, ld0, 0, lb, ub, s));
  } else {
    for (int32_t u0 = 0; u0 < units; u0 += p.chunk_units) {
      const int32_t uc = std::min(p.chunk_units, units - u0);
      const int32_t M = 2 * m * uc;
      if (D > 0) {
        tab.off = bf.off + (int64_t)u0 * (R + 1);
        tab.ent_n = bf.ent_n + (int64_t)u0 * S;
        tab.ent_p = bf.ent_p + (int64_t)u0 * S;
        tab.R = R;
        tab.S = S;
        tab.D = uc;
        tab.rows_per_domain = 2 * m;
      }
      InitArgs ia{};
      ia.src = bf.CW + (D > 0 ? 0 : (int64_t)u0 * m * WL.ld_in);
      ia.ld_src = WL.ld_in;
      ia.n_src = m;
      ia.per_unit_src = D > 0 ? 0 : 1;
      ia.src_bias = bf.Cb + (D > 0 ? 0 : (int64_t)u0 * m);
      ia.n_cols = WL.n_in;
      ia.ldo = WL.ld_in;
      ia.M = M;
      ia.units = uc;
      ia.P = bf.P[L - 2] + (D > 0 ? 0 : (int64_t)u0 * WL.ld_in);
      ia.ldp = WL.ld_in;
      ia.param_per_unit = D > 0 ? 0 : 1;
      ia.relu_index = L - 2;
      ia.splits = tab;
      ia.out = bf.A[0];
      ia.beta = bf.beta;
      HIP_TRY(c, launch_init_rows(ia, s));
      st = run_chain(c, bf, L - 1, M, 2 * m, uc, D > 0 ? 0 : u0, D > 0 ? 0 : 1, tab, &flops);
      if (st != VCR_OK) return st;
      HIP_TRY(c, launch_finalize_spec(bf.beta, bf.cpart, (int32_t)(ld0 / PART_COLS), (int32_t)rows_pad(M), uc, m,
                                      D > 0 ? bf.flags + u0 : nullptr, lb + (int64_t)u0 * m,
                                      ub + (int64_t)u0 * m, s));
      ++chunks;
    }
  }
  c->last_B = D > 0 ? 1 : B;
  c->lastL.assign(bf.Lb.begin(), bf.Lb.end());
  c->lastU.assign(bf.Ub.begin(), bf.Ub.end());
  c->last_had_splits = D > 0;
  c->flops_last = flops;
  c->chunks_last = chunks;
  return VCR_OK;
}

vcr_status after_call(vcr_ctx *c, vcr_status st, std::chrono::steady_clock::time_point t0) {
  if (st == VCR_OK && c->sync_check) {
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) st = fail(c, VCR_ERR_DEVICE, "device error: %s", hipGetErrorString(e));
    if (st == VCR_OK && c->last_had_splits) {
      int32_t inv = 0;
      e = hipMemcpy(&inv, c->d_counters + 64, sizeof(int32_t), hipMemcpyDeviceToHost);
      if (e != hipSuccess) st = fail(c, VCR_ERR_DEVICE, "device error: %s", hipGetErrorString(e));
      else if (inv > 0) st = fail(c, VCR_ERR_ARG, "%d subdomain(s) have invalid splits (NaN bounds)", inv);
    }
  }
  c->ms_last = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  return st;
}

}  // namespace

extern "C" {

vcr_status vcr_crown_bounds(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                            const vcr_splits *splits, float *lb, float *ub) {
  if (!c) return VCR_ERR_ARG;
  const auto t0 = std::chrono::steady_clock::now();
  vcr_status st = check_common(c, x0, B, eps, C, m, lb, ub);
  if (st != VCR_OK) return st;
  if (splits) {
    if (B != 1) return fail(c, VCR_ERR_ARG, "splits need exactly one root input (B = 1)");
    if (splits->n_domains <= 0 || splits->per_domain < 0 || splits->per_domain > VCR_MAX_SPLITS)
      return fail(c, VCR_ERR_ARG, "bad split sizes (n_domains > 0, 0 <= per_domain <= 64)");
    if (splits->per_domain > 0 && (!splits->relu_id || !splits->neuron || !splits->sign))
      return fail(c, VCR_ERR_ARG, "null split array");
    if (c->relu_n.empty()) return fail(c, VCR_ERR_ARG, "splits need at least one ReLU");
    if ((int64_t)splits->n_domains * m > (int64_t)1 << 30) return fail(c, VCR_ERR_SHAPE, "n_domains * m too large");
  }
  st = check_finite_inputs(c, x0, B, C, m);
  if (st != VCR_OK) return st;
  auto run = [&]() {
    return c->graph ? graph_crown(c, x0, B, eps, C, m, splits, lb, ub) : crown_impl(c, x0, B, eps, C, m, splits, lb, ub);
  };
  if (!c->use_graph || splits || c->time_gemm || c->device < 0) return after_call(c, run(), t0);
  // graph replay: the key names everything a recorded launch sequence depends on
  std::vector<uint64_t> key = {(uint64_t)(uintptr_t)x0, (uint64_t)B, (uint64_t)*reinterpret_cast<const uint32_t *>(&eps),
                               (uint64_t)(uintptr_t)C, (uint64_t)m, (uint64_t)(uintptr_t)lb, (uint64_t)(uintptr_t)ub,
                               (uint64_t)c->clip_on, (uint64_t)*reinterpret_cast<const uint32_t *>(&c->clip_lo),
                               (uint64_t)*reinterpret_cast<const uint32_t *>(&c->clip_hi), (uint64_t)c->intersect,
                               c->ws_cap, c->net_epoch, (uint64_t)(uintptr_t)c->ws.base, (uint64_t)c->ws.cap,
                               (uint64_t)c->lambda_rule};
  if (c->gexec && key == c->gkey) {
    HIP_TRY(c, hipSetDevice(c->device));
    HIP_TRY(c, hipGraphLaunch(c->gexec, c->stream));
    return after_call(c, VCR_OK, t0);
  }
  // one ordinary call (allocates the workspace and produces this call's results) ...
  st = run();
  if (st != VCR_OK) return after_call(c, st, t0);
  // ... then the same launches recorded on a private stream
  if (c->gexec) {
    (void)hipGraphExecDestroy(c->gexec);
    c->gexec = nullptr;
  }
  if (!c->cap_stream) HIP_TRY(c, hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking));
  key[13] = (uint64_t)(uintptr_t)c->ws.base;
  key[14] = (uint64_t)c->ws.cap;
  hipStream_t user = c->stream;
  c->stream = c->cap_stream;
  hipGraph_t g = nullptr;
  hipError_t e = hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal);
  if (e == hipSuccess) {
    st = run();
    hipError_t e2 = hipStreamEndCapture(c->cap_stream, &g);
    if (e == hipSuccess) e = e2;
  }
  c->stream = user;
  if (st != VCR_OK || e != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    (void)hipGetLastError();
    if (st == VCR_OK) st = fail(c, VCR_ERR_DEVICE, "graph capture failed: %s", hipGetErrorString(e));
    return after_call(c, st, t0);
  }
  e = hipGraphInstantiate(&c->gexec, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (e != hipSuccess) {
    c->gexec = nullptr;
    return after_call(c, fail(c, VCR_ERR_DEVICE, "graph instantiation failed: %s", hipGetErrorString(e)), t0);
  }
  c->gkey = key;
  return after_call(c, VCR_OK, t0);
}

}  // extern "C"

// vcr_crown_bounds (no splits) with the workspace replaced by [base, base + bytes), which the
// caller owns: the plan is chunked to fit it (VCR_ERR_OOM when even one input does not), the
// bytes the plan uses are cleared by a fill kernel (the A buffers' padding is read by the
// GEMMs), and nothing is allocated: no workspace growth, no timing events (TIME_GEMM is
// ignored for the call), no graph capture.  The context's own workspace is left as it was.
vcr_status vcr::crown_bounds_in(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                                float *lb, float *ub, char *base, size_t bytes) {
  const auto t0 = std::chrono::steady_clock::now();
  vcr_status st = check_common(c, x0, B, eps, C, m, lb, ub);
  if (st != VCR_OK) return st;
  if (c->device < 0) return fail(c, VCR_ERR_STATE, "validation-only context: no device work");
  if (!base || bytes == 0) return fail(c, VCR_ERR_STATE, "no scratch memory on this device");
  st = check_finite_inputs(c, x0, B, C, m);
  if (st != VCR_OK) return st;
  HIP_TRY(c, hipSetDevice(c->device));
  // plan under the scratch size (or the user's cap, if smaller): the same plan the call makes
  const uint64_t user_cap = c->ws_cap;
  const uint64_t cap = user_cap > 0 ? std::min<uint64_t>(user_cap, bytes) : bytes;
  c->ws_cap = cap;
  size_t need = 0;
  if (c->graph) {
    int chunk = 0;
    st = graph_plan(c, B, m, &chunk, &need, false);
  } else {
    Plan p;
    st = make_plan(c, B, m, 0, 0, &p);
    need = p.bytes;
  }
  c->ws_cap = user_cap;
  if (st != VCR_OK)
    return fail(c, VCR_ERR_OOM, "the call does not fit the %llu-byte scratch even one input at a time (%s)",
                (unsigned long long)cap, c->err.c_str());
  const Workspace own = c->ws;
  const int32_t timing = c->time_gemm;
  c->ws = Workspace{base, cap, 0};
  c->ws_cap = cap;
  c->time_gemm = 0;
  struct Restore {
    vcr_ctx *c;
    Workspace own;
    uint64_t cap;
    int32_t timing;
    ~Restore() {
      c->ws = own;
      c->ws_cap = cap;
      c->time_gemm = timing;
    }
  } restore{c, own, user_cap, timing};
  // the scratch keeps the last call's contents: clear what this call's plan uses
  HIP_TRY(c, launch_fill(reinterpret_cast<float *>(base), (int64_t)(need / 4), 0.f, c->stream));
  st = c->graph ? graph_crown(c, x0, B, eps, C, m, nullptr, lb, ub) : crown_impl(c, x0, B, eps, C, m, nullptr, lb, ub);
  return after_call(c, st, t0);
}

extern "C" {

vcr_status vcr_ibp_bounds(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                          float *lb, float *ub) {
  if (!c) return VCR_ERR_ARG;
  const auto t0 = std::chrono::steady_clock::now();
  vcr_status st = check_common(c, x0, B, eps, C, m, lb, ub);
  if (st != VCR_OK) return st;
  if (c->device < 0) return fail(c, VCR_ERR_STATE, "validation-only context: no device work");
  st = check_finite_inputs(c, x0, B, C, m);
  if (st != VCR_OK) return st;
  if (c->graph) return after_call(c, graph_ibp(c, x0, B, eps, C, m, lb, ub), t0);
  HIP_TRY(c, hipSetDevice(c->device));
  const int L = (int)c->layers.size();
  const int64_t ld0 = ld_of(c->n0);
  const int64_t Bp = rows_pad(B);   // GEMM operands on large layers
  int64_t ldmax = 1;
  for (int k = 0; k < L - 1; ++k) ldmax = std::max(ldmax, c->layers[k].ld_out);
  const bool tmp = any_ibp_relu_on_mfma(c);
  size_t bytes = 2 * al(sizeof(float) * Bp * ld0);
  for (int k = 0; k < L - 1; ++k) bytes += 2 * al(sizeof(float) * Bp * c->layers[k].ld_out);
  bytes += al(sizeof(float) * B * m * c->layers[L - 1].ld_in) + al(sizeof(float) * B * m);
  if (tmp) bytes += 2 * al(sizeof(float) * Bp * ldmax);
  c->lastL.clear();   // this call reuses the workspace that held them
  c->lastU.clear();
  st = ensure_ws(c, bytes);
  if (st != VCR_OK) return st;
  hipStream_t s = c->stream;
  float *c0 = take<float>(c, (size_t)Bp * ld0), *r0 = take<float>(c, (size_t)Bp * ld0);
  std::vector<float *> cc, rr;
  for (int k = 0; k < L - 1; ++k) {
    cc.push_back(take<float>(c, (size_t)Bp * c->layers[k].ld_out));
    rr.push_back(take<float>(c, (size_t)Bp * c->layers[k].ld_out));
  }
  const DenseLayer &WL = c->layers[L - 1];
  float *CW = take<float>(c, (size_t)B * m * WL.ld_in), *Cb = take<float>(c, (size_t)B * m);
  float *tc = tmp ? take<float>(c, (size_t)Bp * ldmax) : nullptr, *tr = tmp ? take<float>(c, (size_t)Bp * ldmax) : nullptr;
  HIP_TRY(c, launch_box(x0, B, c->n0, ld0, eps, c->clip_on, c->clip_lo, c->clip_hi, c0, r0, s));
  for (int k = 0; k < L - 1; ++k) {
    const DenseLayer &W = c->layers[k];
    st = ibp_layer(c, W, k == 0 ? c0 : cc[k - 1], k == 0 ? r0 : rr[k - 1], k > 0, cc[k], rr[k], B, tc, tr, s);
    if (st != VCR_OK) return st;
  }
  HIP_TRY(c, launch_spec_cw(C, B, m, WL.n_out, WL.Wp, WL.ld_in, WL.b, WL.n_in, CW, WL.ld_in, Cb, s));
  HIP_TRY(c, launch_spec_direct(CW, WL.ld_in, Cb, B, m, WL.n_in, L >= 2 ? cc[L - 2] : c0, L >= 2 ? rr[L - 2] : r0,
                                WL.ld_in, L >= 2, lb, ub, s));
  return after_call(c, VCR_OK, t0);
}

vcr_status vcr_alpha_crown_bounds(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                                  const vcr_alpha_opts *opts, float *lb, float *ub) {
  if (!c) return VCR_ERR_ARG;
  const auto t0 = std::chrono::steady_clock::now();
  vcr_status st = check_common(c, x0, B, eps, C, m, lb, ub);
  if (st != VCR_OK) return st;
  if (!opts) return fail(c, VCR_ERR_ARG, "null alpha options");
  if (c->relu_n.empty()) return fail(c, VCR_ERR_ARG, "alpha-CROWN needs at least one ReLU");
  const vcr_alpha_opts &o = *opts;
  if (o.iters < 0 || o.iters > 1000000) return fail(c, VCR_ERR_ARG, "iters must be in [0, 1e6]");
  if (!(o.lr > 0.f) || !std::isfinite(o.lr)) return fail(c, VCR_ERR_ARG, "lr must be finite and > 0");
  if (!(o.beta1 >= 0.f && o.beta1 < 1.f) || !(o.beta2 >= 0.f && o.beta2 < 1.f))
    return fail(c, VCR_ERR_ARG, "beta1 and beta2 must be in [0, 1)");
  if (!(o.adam_eps > 0.f) || !std::isfinite(o.adam_eps)) return fail(c, VCR_ERR_ARG, "adam_eps must be finite and > 0");
  if ((o.lb_hist == nullptr) != (o.ub_hist == nullptr)) return fail(c, VCR_ERR_ARG, "lb_hist and ub_hist go together");
  AlphaCall ac{o, 0};
  for (int32_t n : c->relu_n) ac.n_total += n;
  if ((int64_t)B * 2 * m * ac.n_total > ((int64_t)1 << 40)) return fail(c, VCR_ERR_SHAPE, "alpha tensors too large");
  st = check_finite_inputs(c, x0, B, C, m);
  if (st != VCR_OK) return st;
  if (c->graph) return after_call(c, graph_alpha(c, x0, B, eps, C, m, o, ac.n_total, lb, ub), t0);
  return after_call(c, crown_impl(c, x0, B, eps, C, m, nullptr, lb, ub, &ac), t0);
}

}  // extern "C"

namespace {

vcr_status check_splits(vcr_ctx *c, const vcr_splits *splits, int32_t m) {
  if (splits->n_domains <= 0 || splits->per_domain < 0 || splits->per_domain > VCR_MAX_SPLITS)
    return fail(c, VCR_ERR_ARG, "bad split sizes (n_domains > 0, 0 <= per_domain <= 64)");
  if (splits->per_domain > 0 && (!splits->relu_id || !splits->neuron || !splits->sign))
    return fail(c, VCR_ERR_ARG, "null split array");
  if (c->relu_n.empty()) return fail(c, VCR_ERR_ARG, "splits need at least one ReLU");
  if ((int64_t)splits->n_domains * m > (int64_t)1 << 30) return fail(c, VCR_ERR_SHAPE, "n_domains * m too large");
  return VCR_OK;
}

vcr_status check_beta_opts(vcr_ctx *c, const vcr_beta_opts *o) {
  if (!o) return fail(c, VCR_ERR_ARG, "null beta options");
  if (o->iters < 0 || o->iters > 1000000) return fail(c, VCR_ERR_ARG, "iters must be in [0, 1e6]");
  if (!(o->lr_alpha > 0.f) || !std::isfinite(o->lr_alpha) || !(o->lr_beta > 0.f) || !std::isfinite(o->lr_beta))
    return fail(c, VCR_ERR_ARG, "lr_alpha and lr_beta must be finite and > 0");
  if (!(o->beta1 >= 0.f && o->beta1 < 1.f) || !(o->beta2 >= 0.f && o->beta2 < 1.f))
    return fail(c, VCR_ERR_ARG, "beta1 and beta2 must be in [0, 1)");
  if (!(o->adam_eps > 0.f) || !std::isfinite(o->adam_eps)) return fail(c, VCR_ERR_ARG, "adam_eps must be finite and > 0");
  if ((o->lb_hist == nullptr) != (o->ub_hist == nullptr)) return fail(c, VCR_ERR_ARG, "lb_hist and ub_hist go together");
  return VCR_OK;
}

AlphaCall alpha_call_of(const vcr_ctx *c, const vcr_beta_opts &b, bool hist) {
  AlphaCall ac{};
  ac.o.iters = b.iters;
  ac.o.lr = b.lr_alpha;
  ac.o.beta1 = b.beta1;
  ac.o.beta2 = b.beta2;
  ac.o.adam_eps = b.adam_eps;
  if (hist) {
    ac.o.lb_hist = b.lb_hist;
    ac.o.ub_hist = b.ub_hist;
  }
  for (int32_t n : c->relu_n) ac.n_total += n;
  ac.lr_beta = b.lr_beta;
  return ac;
}

// device memory of one branch-and-bound round (split arrays, bounds), grown on demand
vcr_status bab_reserve(vcr_ctx *c, size_t bytes) {
  if (c->bab_cap >= bytes) return VCR_OK;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  if (c->bab_buf) HIP_TRY(c, hipFree(c->bab_buf));
  c->bab_buf = nullptr;
  c->bab_cap = 0;
  HIP_TRY(c, hipMalloc(&c->bab_buf, bytes));
  c->bab_cap = bytes;
  return VCR_OK;
}

struct Split {
  int32_t r, j, sg;
};

}  // namespace

extern "C" {

vcr_status vcr_beta_crown_bounds(vcr_ctx *c, const float *x0, float eps, const float *C, int32_t m,
                                 const vcr_splits *splits, const vcr_beta_opts *opts, float *lb, float *ub) {
  if (!c) return VCR_ERR_ARG;
  const auto t0 = std::chrono::steady_clock::now();
  vcr_status st = check_common(c, x0, 1, eps, C, m, lb, ub);
  if (st != VCR_OK) return st;
  if (!splits) return fail(c, VCR_ERR_ARG, "null splits");
  st = check_splits(c, splits, m);
  if (st != VCR_OK) return st;
  st = check_beta_opts(c, opts);
  if (st != VCR_OK) return st;
  st = check_finite_inputs(c, x0, 1, C, m);
  if (st != VCR_OK) return st;
  AlphaCall ac = alpha_call_of(c, *opts, true);
  if (c->graph)
    return after_call(c, graph_beta(c, x0, eps, C, m, splits, ac.o, ac.n_total, ac.lr_beta, lb, ub), t0);
  return after_call(c, crown_impl(c, x0, 1, eps, C, m, splits, lb, ub, &ac), t0);
}

vcr_status vcr_bab_verify(vcr_ctx *c, const float *x0, float eps, const float *C, int32_t m, const vcr_bab_opts *opts,
                          vcr_bab_result *res, int64_t *round_log) {
  if (!c) return VCR_ERR_ARG;
  const auto t0 = std::chrono::steady_clock::now();
  if (!opts || !res) return fail(c, VCR_ERR_ARG, "null options or result");
  if (!c->loaded) return fail(c, VCR_ERR_STATE, "no network loaded");
  if (c->relu_n.empty()) return fail(c, VCR_ERR_ARG, "branch and bound needs at least one ReLU");
  if (opts->batch < 1 || opts->max_rounds < 0) return fail(c, VCR_ERR_ARG, "batch must be >= 1, max_rounds >= 0");
  // a subdomain gains one split per round, and the split table holds VCR_MAX_SPLITS
  if (opts->max_rounds > VCR_MAX_SPLITS)
    return fail(c, VCR_ERR_ARG, "max_rounds %d exceeds %d: a subdomain would hold more splits than the table",
                opts->max_rounds, VCR_MAX_SPLITS);
  if (m <= 0 || !x0 || !C) return fail(c, VCR_ERR_ARG, "bad property");
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(c, VCR_ERR_ARG, "eps must be finite and >= 0");
  if (!aligned16(x0) || !aligned16(C)) return fail(c, VCR_ERR_ARG, "tensor pointers must be 16-byte aligned");
  vcr_status st = check_beta_opts(c, &opts->bound);
  if (st != VCR_OK) return st;
  const int R = (int)c->relu_n.size();
  if (opts->order_len < 0 || (opts->order_len > 0 && (!opts->order_relu || !opts->order_neuron)))
    return fail(c, VCR_ERR_ARG, "bad split order");
  for (int32_t k = 0; k < opts->order_len; ++k)
    if (opts->order_relu[k] < 0 || opts->order_relu[k] >= R || opts->order_neuron[k] < 0 ||
        opts->order_neuron[k] >= c->relu_n[opts->order_relu[k]])
      return fail(c, VCR_ERR_ARG, "split order entry %d out of range", k);
  if (c->device < 0) return fail(c, VCR_ERR_STATE, "validation-only context: no device work");
  st = check_finite_inputs(c, x0, 1, C, m);
  if (st != VCR_OK) return st;
  HIP_TRY(c, hipSetDevice(c->device));
  hipStream_t s = c->stream;
  *res = vcr_bab_result{};
  const AlphaCall ac = alpha_call_of(c, opts->bound, false);
  // alpha-CROWN (no splits) or beta-CROWN (subdomains) on either network path
  auto bound = [&](const vcr_splits *sp, float *l, float *u) -> vcr_status {
    if (!c->graph) return crown_impl(c, x0, 1, eps, C, m, sp, l, u, &ac);
    return sp ? graph_beta(c, x0, eps, C, m, sp, ac.o, ac.n_total, ac.lr_beta, l, u)
              : graph_alpha(c, x0, 1, eps, C, m, ac.o, ac.n_total, l, u);
  };

  // root: alpha-CROWN
  st = bab_reserve(c, sizeof(float) * 2 * (size_t)m);
  if (st != VCR_OK) return st;
  float *d_lb = static_cast<float *>(c->bab_buf), *d_ub = d_lb + m;
  st = bound(nullptr, d_lb, d_ub);
  if (st != VCR_OK) return st;
  std::vector<float> h_lb(m);
  HIP_TRY(c, hipMemcpyAsync(h_lb.data(), d_lb, sizeof(float) * m, hipMemcpyDeviceToHost, s));
  // the split order: given, or the root's unstable neurons by decreasing chord intercept
  std::vector<std::pair<int32_t, int32_t>> order;
  if (opts->order_len > 0) {
    for (int32_t k = 0; k < opts->order_len; ++k) order.emplace_back(opts->order_relu[k], opts->order_neuron[k]);
  } else {
    struct Cand {
      double score;
      int32_t r, j;
    };
    std::vector<Cand> cand;
    for (int r = 0; r < R; ++r) {
      const int32_t n = c->relu_n[r];
      std::vector<float> l(n), u(n);
      HIP_TRY(c, hipMemcpyAsync(l.data(), c->lastL[r], sizeof(float) * n, hipMemcpyDeviceToHost, s));
      HIP_TRY(c, hipMemcpyAsync(u.data(), c->lastU[r], sizeof(float) * n, hipMemcpyDeviceToHost, s));
      HIP_TRY(c, hipStreamSynchronize(s));
      for (int32_t j = 0; j < n; ++j)
        if (l[j] < 0.f && u[j] > 0.f) cand.push_back({-(double)u[j] * (double)l[j] / ((double)u[j] - (double)l[j]), r, j});
    }
    std::stable_sort(cand.begin(), cand.end(), [](const Cand &a, const Cand &b) { return a.score > b.score; });
    for (const Cand &k : cand) order.emplace_back(k.r, k.j);
  }
  HIP_TRY(c, hipStreamSynchronize(s));
  float root_min = INFINITY;
  for (float v : h_lb) root_min = std::min(root_min, v);
  res->root_min_lb = root_min;
  bool all_pos = true;
  for (float v : h_lb) all_pos = all_pos && v > 0.f;
  if (all_pos) {
    res->verified = 1;
    res->worst_lb = INFINITY;
    c->ms_last = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return VCR_OK;
  }
  std::deque<std::vector<Split>> queue;
  std::deque<float> queue_lb;
  queue.emplace_back();
  queue_lb.push_back(root_min);
  // every round bounds subdomains of the same root: its steps 1-3 run in the first round only
  struct ReuseScope {
    vcr_ctx *c;
    explicit ReuseScope(vcr_ctx *cc) : c(cc) { c->bab_reuse = true; c->root_cached = false; }
    ~ReuseScope() { c->bab_reuse = false; c->root_cached = false; }
  } reuse_scope(c);
  for (int32_t rnd = 0; rnd < opts->max_rounds && !queue.empty(); ++rnd) {
    const size_t take = std::min<size_t>((size_t)opts->batch, queue.size());
    std::vector<std::vector<Split>> kids;
    bool stuck = false;
    for (size_t k = 0; k < take; ++k) {
      std::vector<Split> dom = std::move(queue.front());
      const float dlb = queue_lb.front();
      queue.pop_front();
      queue_lb.pop_front();
      const std::pair<int32_t, int32_t> *nxt = nullptr;
      for (const auto &o : order) {
        bool used = false;
        for (const Split &q : dom) used = used || (q.r == o.first && q.j == o.second);
        if (!used) {
          nxt = &o;
          break;
        }
      }
      if (!nxt) {   // nothing left to split: stays unverified
        stuck = true;
        queue.push_back(std::move(dom));
        queue_lb.push_back(dlb);
        continue;
      }
      for (int sg : {1, -1}) {
        std::vector<Split> ch = dom;
        ch.push_back({nxt->first, nxt->second, sg});
        kids.push_back(std::move(ch));
      }
    }
    int64_t pruned = 0;
    if (!kids.empty()) {
      const int32_t D = (int32_t)kids.size();
      int32_t S = 0;
      for (const auto &k : kids) S = std::max<int32_t>(S, (int32_t)k.size());
      std::vector<int32_t> hr((size_t)D * S, -1), hn((size_t)D * S, 0);
      std::vector<int8_t> hs((size_t)D * S, 1);
      for (int32_t d = 0; d < D; ++d)
        for (size_t e = 0; e < kids[d].size(); ++e) {
          hr[(size_t)d * S + e] = kids[d][e].r;
          hn[(size_t)d * S + e] = kids[d][e].j;
          hs[(size_t)d * S + e] = (int8_t)kids[d][e].sg;
        }
      const size_t nb = (size_t)D * S;
      const size_t off_n = al(sizeof(int32_t) * nb), off_s = off_n + al(sizeof(int32_t) * nb);
      const size_t off_lb = off_s + al(nb), off_ub = off_lb + al(sizeof(float) * D * m);
      st = bab_reserve(c, off_ub + al(sizeof(float) * D * m));
      if (st != VCR_OK) return st;
      char *base = static_cast<char *>(c->bab_buf);
      int32_t *d_r = reinterpret_cast<int32_t *>(base), *d_n = reinterpret_cast<int32_t *>(base + off_n);
      int8_t *d_s = reinterpret_cast<int8_t *>(base + off_s);
      float *k_lb = reinterpret_cast<float *>(base + off_lb), *k_ub = reinterpret_cast<float *>(base + off_ub);
      HIP_TRY(c, hipMemcpyAsync(d_r, hr.data(), sizeof(int32_t) * nb, hipMemcpyHostToDevice, s));
      HIP_TRY(c, hipMemcpyAsync(d_n, hn.data(), sizeof(int32_t) * nb, hipMemcpyHostToDevice, s));
      HIP_TRY(c, hipMemcpyAsync(d_s, hs.data(), nb, hipMemcpyHostToDevice, s));
      vcr_splits sp{D, S, d_r, d_n, d_s};
      st = bound(&sp, k_lb, k_ub);
      if (st != VCR_OK) return st;
      std::vector<float> kl((size_t)D * m);
      HIP_TRY(c, hipMemcpyAsync(kl.data(), k_lb, sizeof(float) * D * m, hipMemcpyDeviceToHost, s));
      HIP_TRY(c, hipStreamSynchronize(s));
      for (int32_t d = 0; d < D; ++d) {
        bool ok = true;
        float mn = INFINITY;
        for (int32_t q = 0; q < m; ++q) {
          const float v = kl[(size_t)d * m + q];
          if (std::isnan(v)) return fail(c, VCR_ERR_DEVICE, "internal: NaN bound of a subdomain");
          ok = ok && v > 0.f;
          mn = std::min(mn, v);
        }
        if (ok) {
          ++pruned;
        } else {
          queue.push_back(std::move(kids[d]));
          queue_lb.push_back(mn);
        }
      }
      res->evaluated += D;
    }
    res->rounds = rnd + 1;
    if (round_log) {
      round_log[4 * rnd + 0] = (int64_t)take;
      round_log[4 * rnd + 1] = (int64_t)kids.size();
      round_log[4 * rnd + 2] = pruned;
      round_log[4 * rnd + 3] = (int64_t)queue.size();
    }
    if (stuck && kids.empty()) break;
  }
  res->remaining = (int64_t)queue.size();
  res->verified = queue.empty() ? 1 : 0;
  res->worst_lb = INFINITY;
  for (float v : queue_lb) res->worst_lb = std::min(res->worst_lb, v);
  c->ms_last = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  return VCR_OK;
}

int64_t vcr_relu_neurons(const vcr_ctx *c) {
  if (!c) return 0;
  int64_t n = 0;
  for (int32_t k : c->relu_n) n += k;
  return n;
}

vcr_status vcr_get_layer_bounds(vcr_ctx *c, int32_t relu_id, float *l, float *u) {
  if (!c) return VCR_ERR_ARG;
  if (c->lastL.empty()) return fail(c, VCR_ERR_STATE, "no CROWN call yet");
  if (relu_id < 0 || relu_id >= (int32_t)c->lastL.size()) return fail(c, VCR_ERR_ARG, "relu_id out of range");
  if (!l || !u) return fail(c, VCR_ERR_ARG, "null output");
  const int64_t n = (int64_t)c->last_B * c->relu_n[relu_id];
  HIP_TRY(c, launch_copy(l, c->lastL[relu_id], n, c->stream));
  HIP_TRY(c, launch_copy(u, c->lastU[relu_id], n, c->stream));
  return VCR_OK;
}

vcr_status vcr_workspace_bytes(vcr_ctx *c, int32_t B, int32_t m, int32_t n_domains, uint64_t *bytes) {
  if (!c || !bytes) return VCR_ERR_ARG;
  if (!c->loaded) return fail(c, VCR_ERR_STATE, "no network loaded");
  if (B <= 0 || m <= 0 || n_domains < 0) return fail(c, VCR_ERR_ARG, "bad sizes");
  if (c->graph) {
    *bytes = graph_workspace_bytes(c, B, m, n_domains, n_domains > 0 ? VCR_MAX_SPLITS : 0, false);
    return VCR_OK;
  }
  const uint64_t cap = c->ws_cap;
  c->ws_cap = 0;
  Plan p;
  vcr_status st = make_plan(c, B, m, n_domains, 64, &p);
  c->ws_cap = cap;
  if (st != VCR_OK) return st;
  *bytes = p.bytes;
  return VCR_OK;
}

vcr_status vcr_get_stats(vcr_ctx *c, vcr_stats *out) {
  if (!c || !out) return VCR_ERR_ARG;
  std::memset(out, 0, sizeof(*out));
  out->ms_last_call = c->ms_last;
  out->gemm_flops_last_call = c->flops_last;
  out->peak_workspace_bytes = c->peak_ws;
  out->workspace_bytes = c->ws.cap;
  out->n_chunks_last_call = c->chunks_last;
  out->n_relu = (int32_t)c->relu_n.size();
  out->net_bytes = c->net_bytes;
  if (c->device < 0) return VCR_OK;
  HIP_TRY(c, hipSetDevice(c->device));
  {
    const vcr_status st = timing_fold(c);
    if (st != VCR_OK) return st;
  }
  out->timed_gemm_launches = c->timed_launches[0];
  out->timed_gemm_ms = c->timed_ms[0];
  out->timed_gemm_flops = c->timed_flops[0];
  out->timed_conv_launches = c->timed_launches[1];
  out->timed_conv_ms = c->timed_ms[1];
  out->timed_conv_flops = c->timed_flops[1];
  out->timed_small_launches = c->timed_launches[2];
  out->timed_small_ms = c->timed_ms[2];
  out->timed_small_flops = c->timed_flops[2];
  out->timed_mid_launches = c->timed_launches[3];
  out->timed_mid_ms = c->timed_ms[3];
  out->timed_mid_flops = c->timed_flops[3];
  if (c->lastL.empty()) return VCR_OK;
  int32_t *cnt = c->d_counters;
  const int R = std::min<int>((int)c->lastL.size(), 64);
  HIP_TRY(c, launch_fill(reinterpret_cast<float *>(cnt), 64, 0.f, c->stream));   // keeps [64] (invalid domains)
  for (int r = 0; r < R; ++r)
    HIP_TRY(c, launch_count_unstable(c->lastL[r], c->lastU[r], (int64_t)c->last_B * c->relu_n[r], cnt + r, c->stream));
  int32_t host[80];
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  HIP_TRY(c, hipMemcpy(host, cnt, sizeof(host), hipMemcpyDeviceToHost));
  for (int r = 0; r < R; ++r) out->unstable[r] = host[r];
  out->invalid_domains = c->last_had_splits ? host[64] : 0;
  return VCR_OK;
}

}  // extern "C"
