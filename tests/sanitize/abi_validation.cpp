// Host-side exercise of the vcrown C ABI on a validation-only context (no GPU), built with
// AddressSanitizer and UndefinedBehaviorSanitizer on the host code (tests/sanitize/build.sh):
// every argument check, the network validator and both planners (MLP and convolutional)
// run, on fixed cases and on seeded random node lists.  Any sanitizer report aborts the
// program; a wrong status makes it exit 1.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/vcrown.h"

namespace {

int g_fail = 0;

#define EXPECT(cond)                                                              \
  do {                                                                            \
    if (!(cond)) {                                                                \
      std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond);    \
      ++g_fail;                                                                   \
    }                                                                             \
  } while (0)

// a host buffer standing in for device memory (16-byte aligned, never dereferenced by a
// validation-only context)
struct Buf {
  std::vector<float> v;
  explicit Buf(size_t n) : v(n + 8, 0.f) {}
  float *p() {
    uintptr_t a = reinterpret_cast<uintptr_t>(v.data());
    return reinterpret_cast<float *>((a + 15) & ~uintptr_t(15));
  }
};

// owned host weights for a node list
struct Net {
  std::vector<vcr_node> nodes;
  std::vector<std::vector<float>> store;
  int32_t chw[3] = {1, 1, 1};
  const float *arr(size_t n) {
    store.emplace_back(n > 0 ? n : 1, 0.01f);
    return store.back().data();
  }
  void dense(int32_t in0, int32_t out, int64_t n_in) {
    vcr_node d{};
    d.op = VCR_DENSE;
    d.in0 = in0;
    d.in1 = -1;
    d.out_features = out;
    d.W = arr((size_t)out * (size_t)n_in);
    d.b = arr((size_t)out);
    nodes.push_back(d);
  }
  void conv(int32_t in0, int32_t out, int32_t cin, int32_t k, int32_t stride, int32_t pad) {
    vcr_node d{};
    d.op = VCR_CONV2D;
    d.in0 = in0;
    d.in1 = -1;
    d.out_ch = out;
    d.kh = d.kw = k;
    d.stride = stride;
    d.pad = pad;
    d.W = arr((size_t)out * cin * k * k);
    d.b = arr((size_t)out);
    nodes.push_back(d);
  }
  void op(int32_t kind, int32_t in0, int32_t in1 = -1) {
    vcr_node d{};
    d.op = kind;
    d.in0 = in0;
    d.in1 = in1;
    nodes.push_back(d);
  }
  vcr_status load(vcr_ctx *c) { return vcr_load_net(c, nodes.data(), (int32_t)nodes.size(), chw); }
};

Net mlp(std::vector<int32_t> dims) {
  Net n;
  n.chw[0] = dims[0];
  for (size_t i = 1; i < dims.size(); ++i) {
    n.dense((int32_t)n.nodes.size() - 1, dims[i], dims[i - 1]);
    if (i + 1 < dims.size()) n.op(VCR_RELU, (int32_t)n.nodes.size() - 1);
  }
  return n;
}

Net resnet(int32_t hw, int32_t c1, int32_t c2) {
  Net n;
  n.chw[0] = 3;
  n.chw[1] = n.chw[2] = hw;
  n.conv(-1, c1, 3, 3, 1, 1);                      // 0
  n.conv(0, c1, c1, 3, 1, 1);                      // 1
  n.op(VCR_RELU, 1);                               // 2
  n.conv(2, c1, c1, 3, 1, 1);                      // 3
  n.op(VCR_ADD, 0, 3);                             // 4
  n.conv(4, c2, c1, 3, 2, 1);                      // 5
  n.op(VCR_RELU, 5);                               // 6
  n.op(VCR_FLATTEN, 6);                            // 7
  const int32_t h2 = (hw - 1) / 2 + 1;
  n.dense(7, 16, (int64_t)c2 * h2 * h2);           // 8
  n.op(VCR_RELU, 8);                               // 9
  n.dense(9, 10, 16);                              // 10
  return n;
}

vcr_status crown(vcr_ctx *c, int32_t B, int32_t m, int32_t n0, int32_t nout, float eps, const vcr_splits *sp) {
  const int32_t rows = sp ? sp->n_domains : B;
  Buf x((size_t)std::max(B, 1) * n0), C((size_t)std::max(B, 1) * std::max(m, 1) * nout);
  Buf lb((size_t)std::max(rows, 1) * std::max(m, 1)), ub((size_t)std::max(rows, 1) * std::max(m, 1));
  return vcr_crown_bounds(c, x.p(), B, eps, C.p(), m, sp, lb.p(), ub.p());
}

void fixed_cases() {
  vcr_ctx *c = nullptr;
  EXPECT(vcr_create(-2, &c) == VCR_ERR_ARG);
  EXPECT(vcr_create(-1, nullptr) == VCR_ERR_ARG);
  EXPECT(std::strcmp(vcr_last_error(nullptr), "null context") == 0);
  EXPECT(vcr_create(-1, &c) == VCR_OK && c);
  EXPECT(vcr_abi_version() == VCR_ABI_VERSION);
  // options
  EXPECT(vcr_set_option(c, 99, 1.0) == VCR_ERR_ARG);
  EXPECT(vcr_set_option(c, VCR_OPT_CLIP_LO, NAN) == VCR_ERR_ARG);
  EXPECT(vcr_set_option(c, VCR_OPT_WORKSPACE_CAP_BYTES, -1.0) == VCR_ERR_ARG);
  EXPECT(vcr_set_option(c, VCR_OPT_LAMBDA_RULE, 4.0) == VCR_ERR_ARG);
  EXPECT(vcr_set_option(c, VCR_OPT_LAMBDA_RULE, VCR_LAMBDA_SAME_SLOPE) == VCR_OK);
  EXPECT(vcr_set_option(c, VCR_OPT_CHECK_FINITE, 1.0) == VCR_OK);
  EXPECT(vcr_set_option(c, VCR_OPT_TIME_GEMM, 1.0) == VCR_OK);
  EXPECT(vcr_set_option(c, VCR_OPT_TIME_GEMM, 0.0) == VCR_OK);
  // calls before a network
  EXPECT(crown(c, 1, 9, 784, 10, 0.01f, nullptr) == VCR_ERR_STATE);
  vcr_stats st;
  EXPECT(vcr_get_stats(c, &st) == VCR_OK);
  Buf l(16), u(16);
  EXPECT(vcr_get_layer_bounds(c, 0, l.p(), u.p()) == VCR_ERR_STATE);
  // networks
  EXPECT(vcr_load_net(c, nullptr, 3, nullptr) == VCR_ERR_ARG);
  Net a = mlp({784, 256, 256, 10});
  EXPECT(a.load(c) == VCR_OK);
  EXPECT(vcr_relu_neurons(c) == 512);
  EXPECT(crown(c, 2, 9, 784, 10, 0.01f, nullptr) == VCR_ERR_STATE);   // valid: stops before device work
  EXPECT(crown(c, 0, 9, 784, 10, 0.01f, nullptr) == VCR_ERR_ARG);
  EXPECT(crown(c, 1, 0, 784, 10, 0.01f, nullptr) == VCR_ERR_ARG);
  EXPECT(crown(c, 1, 9, 784, 10, -1.f, nullptr) == VCR_ERR_ARG);
  EXPECT(crown(c, 1, 9, 784, 10, NAN, nullptr) == VCR_ERR_ARG);
  EXPECT(crown(c, 1, 9, 784, 10, INFINITY, nullptr) == VCR_ERR_ARG);
  {
    Buf x(784), C(90), lb(9), ub(9);
    EXPECT(vcr_crown_bounds(c, nullptr, 1, 0.1f, C.p(), 9, nullptr, lb.p(), ub.p()) == VCR_ERR_ARG);
    EXPECT(vcr_crown_bounds(c, x.p() + 1, 1, 0.1f, C.p(), 9, nullptr, lb.p(), ub.p()) == VCR_ERR_ARG);   // misaligned
    EXPECT(vcr_ibp_bounds(c, x.p(), 1, 0.1f, C.p(), 9, lb.p(), ub.p()) == VCR_ERR_STATE);
    EXPECT(vcr_crown_bounds_noalloc(c, x.p(), 1, 0.1f, C.p(), 9, lb.p(), ub.p()) == VCR_ERR_STATE);
    // B * m beyond the limit: rejected before any buffer is touched
    EXPECT(vcr_crown_bounds(c, x.p(), 1 << 20, 0.1f, C.p(), 1 << 20, nullptr, lb.p(), ub.p()) == VCR_ERR_SHAPE);
  }
  // splits
  std::vector<int32_t> rid(4 * 8, 0), neu(4 * 8, 1);
  std::vector<int8_t> sg(4 * 8, 1);
  vcr_splits sp{4, 8, rid.data(), neu.data(), sg.data()};
  EXPECT(crown(c, 1, 9, 784, 10, 0.02f, &sp) == VCR_ERR_STATE);
  EXPECT(crown(c, 2, 9, 784, 10, 0.02f, &sp) == VCR_ERR_ARG);
  vcr_splits sp_big{4, VCR_MAX_SPLITS + 1, rid.data(), neu.data(), sg.data()};
  EXPECT(crown(c, 1, 9, 784, 10, 0.02f, &sp_big) == VCR_ERR_ARG);
  vcr_splits sp_null{4, 8, nullptr, neu.data(), sg.data()};
  EXPECT(crown(c, 1, 9, 784, 10, 0.02f, &sp_null) == VCR_ERR_ARG);
  vcr_splits sp_zero{0, 8, rid.data(), neu.data(), sg.data()};
  EXPECT(crown(c, 1, 9, 784, 10, 0.02f, &sp_zero) == VCR_ERR_ARG);
  // planning sizes
  uint64_t bytes = 0;
  EXPECT(vcr_workspace_bytes(c, 64, 9, 0, &bytes) == VCR_OK && bytes > 0);
  EXPECT(vcr_workspace_bytes(c, 1, 9, 4096, &bytes) == VCR_OK && bytes > 0);
  EXPECT(vcr_workspace_bytes(c, 0, 9, 0, &bytes) == VCR_ERR_ARG);
  EXPECT(vcr_set_option(c, VCR_OPT_WORKSPACE_CAP_BYTES, 6 << 20) == VCR_OK);
  EXPECT(crown(c, 64, 9, 784, 10, 0.01f, nullptr) == VCR_ERR_STATE);   // chunked plan
  EXPECT(vcr_get_stats(c, &st) == VCR_OK && st.n_chunks_last_call > 2);
  EXPECT(vcr_set_option(c, VCR_OPT_WORKSPACE_CAP_BYTES, 1024) == VCR_OK);
  EXPECT(crown(c, 64, 9, 784, 10, 0.01f, nullptr) == VCR_ERR_OOM);     // below the minimum plan
  EXPECT(vcr_set_option(c, VCR_OPT_WORKSPACE_CAP_BYTES, 0) == VCR_OK);
  // alpha, beta, branch and bound options
  {
    Buf x(784), C(90), lb(9), ub(9);
    vcr_alpha_opts ao{};
    ao.iters = 5;
    ao.lr = 0.1f;
    ao.beta1 = 0.9f;
    ao.beta2 = 0.999f;
    ao.adam_eps = 1e-8f;
    EXPECT(vcr_alpha_crown_bounds(c, x.p(), 1, 0.01f, C.p(), 9, &ao, lb.p(), ub.p()) == VCR_ERR_STATE);
    ao.lr = 0.f;
    EXPECT(vcr_alpha_crown_bounds(c, x.p(), 1, 0.01f, C.p(), 9, &ao, lb.p(), ub.p()) == VCR_ERR_ARG);
    EXPECT(vcr_alpha_crown_bounds(c, x.p(), 1, 0.01f, C.p(), 9, nullptr, lb.p(), ub.p()) == VCR_ERR_ARG);
    vcr_beta_opts bo{5, 0.1f, 0.05f, 0.9f, 0.999f, 1e-8f, nullptr, nullptr};
    EXPECT(vcr_beta_crown_bounds(c, x.p(), 0.02f, C.p(), 9, &sp, &bo, lb.p(), ub.p()) == VCR_ERR_STATE);
    EXPECT(vcr_beta_crown_bounds(c, x.p(), 0.02f, C.p(), 9, nullptr, &bo, lb.p(), ub.p()) == VCR_ERR_ARG);
    vcr_bab_opts bb{};
    bb.batch = 4;
    bb.max_rounds = 3;
    bb.bound = bo;
    vcr_bab_result res;
    int64_t log[4 * VCR_MAX_SPLITS];
    EXPECT(vcr_bab_verify(c, x.p(), 0.02f, C.p(), 9, &bb, &res, log) == VCR_ERR_STATE);
    bb.max_rounds = VCR_MAX_SPLITS + 1;
    EXPECT(vcr_bab_verify(c, x.p(), 0.02f, C.p(), 9, &bb, &res, log) == VCR_ERR_ARG);
    bb.max_rounds = 3;
    int32_t orr[2] = {0, 5}, orn[2] = {1, 1};
    bb.order_relu = orr;
    bb.order_neuron = orn;
    bb.order_len = 2;
    EXPECT(vcr_bab_verify(c, x.p(), 0.02f, C.p(), 9, &bb, &res, log) == VCR_ERR_ARG);   // ReLU 5 out of range
  }
  // a convolutional network (the graph planner, validation mode)
  Net r = resnet(8, 32, 64);
  EXPECT(r.load(c) == VCR_OK);
  EXPECT(vcr_workspace_bytes(c, 2, 9, 0, &bytes) == VCR_OK && bytes > 0);
  EXPECT(crown(c, 2, 9, 3 * 64, 10, 0.01f, nullptr) == VCR_ERR_STATE);
  // subdomains of one input (CROWN, beta-CROWN) and the loop: planned, then no device work
  EXPECT(crown(c, 1, 9, 3 * 64, 10, 0.01f, &sp) == VCR_ERR_STATE);
  EXPECT(vcr_workspace_bytes(c, 1, 9, sp.n_domains, &bytes) == VCR_OK && bytes > 0);
  {
    Buf x(3 * 64), C(9 * 10), lb(9 * sp.n_domains), ub(9 * sp.n_domains);
    vcr_beta_opts bo{};
    bo.iters = 3;
    bo.lr_alpha = 0.1f;
    bo.lr_beta = 0.05f;
    bo.beta1 = 0.9f;
    bo.beta2 = 0.999f;
    bo.adam_eps = 1e-8f;
    EXPECT(vcr_beta_crown_bounds(c, x.p(), 0.02f, C.p(), 9, &sp, &bo, lb.p(), ub.p()) == VCR_ERR_STATE);
    vcr_bab_opts bb{};
    bb.batch = 4;
    bb.max_rounds = 3;
    bb.bound = bo;
    vcr_bab_result res;
    EXPECT(vcr_bab_verify(c, x.p(), 0.02f, C.p(), 9, &bb, &res, nullptr) == VCR_ERR_STATE);
  }
  Net bad = resnet(8, 32, 64);
  bad.nodes[4].in1 = 5;   // not an earlier node
  EXPECT(bad.load(c) == VCR_ERR_ARG);
  Net odd = resnet(8, 32, 64);
  odd.nodes[1].kh = odd.nodes[1].kw = 5;   // same output shape, a kernel size the library lacks
  odd.nodes[1].pad = 2;
  EXPECT(odd.load(c) == VCR_ERR_UNSUPPORTED);
  Net shrink = resnet(8, 32, 64);
  shrink.nodes[1].kh = shrink.nodes[1].kw = 5;   // 6x6 output: the residual add no longer matches
  EXPECT(shrink.load(c) == VCR_ERR_SHAPE);
  vcr_destroy(c);
}

// MLPs of extreme widths: the validation-only context records shapes without reading the
// weights, so one small buffer stands in for every weight array; planning must not overflow
void extreme_sizes() {
  static float w[64];
  const int32_t widths[] = {1 << 20, 1 << 24, (1 << 30) - 1, INT32_MAX};
  for (int32_t n0 : {16, 1 << 20})
  for (int32_t wd : widths) {
    vcr_ctx *c = nullptr;
    EXPECT(vcr_create(-1, &c) == VCR_OK);
    vcr_node nd[3] = {};
    nd[0].op = VCR_DENSE;
    nd[0].in0 = -1;
    nd[0].out_features = wd;
    nd[0].W = nd[0].b = w;
    nd[1].op = VCR_RELU;
    nd[1].in0 = 0;
    nd[2].op = VCR_DENSE;
    nd[2].in0 = 1;
    nd[2].out_features = 10;
    nd[2].W = nd[2].b = w;
    const int32_t chw[3] = {n0, 1, 1};
    const vcr_status st = vcr_load_net(c, nd, 3, chw);
    // accepted exactly when every tensor and weight matrix is within the limits
    const bool fits = (int64_t)wd <= VCR_MAX_NODE_ELEMENTS && (int64_t)wd * n0 <= VCR_MAX_LAYER_WEIGHTS;
    EXPECT(st == (fits ? VCR_OK : VCR_ERR_SHAPE));
    if (st == VCR_OK) {
      uint64_t bytes = 0;
      const vcr_status ws = vcr_workspace_bytes(c, 1 << 10, 1 << 10, 0, &bytes);
      EXPECT(ws == VCR_OK || ws == VCR_ERR_SHAPE);
      Buf x(16), C(16), lb(16), ub(16);
      const vcr_status cs = vcr_crown_bounds(c, x.p(), 1, 0.1f, C.p(), 9, nullptr, lb.p(), ub.p());
      EXPECT(cs == VCR_ERR_STATE || cs == VCR_ERR_SHAPE);
    }
    vcr_destroy(c);
  }
}

// seeded random node lists: every load returns a status; valid ones are planned and bounded
uint64_t g_rng = 0x9e3779b97f4a7c15ull;
uint32_t rnd(uint32_t n) {
  g_rng = g_rng * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(g_rng >> 33) % n;
}

void fuzz(int rounds) {
  int ok = 0;
  for (int it = 0; it < rounds; ++it) {
    vcr_ctx *c = nullptr;
    if (vcr_create(-1, &c) != VCR_OK) {
      ++g_fail;
      return;
    }
    Net n;
    const bool conv = rnd(2);
    const bool plausible = rnd(2);   // mostly well-formed networks, so the planners run
    n.chw[0] = conv ? 1 + rnd(4) : 1 + rnd(64);
    n.chw[1] = n.chw[2] = conv ? 2 + rnd(10) : 1;
    if (conv && rnd(8) == 0) n.chw[2] = n.chw[1] + 1;   // non-square
    std::vector<std::vector<int64_t>> shp;              // C, H, W of each node (the harness's own view)
    const int len = 1 + rnd(9);
    bool flat = !conv;
    for (int i = 0; i < len; ++i) {
      int32_t in0 = (int32_t)rnd(i + 2) - 1 - (rnd(16) == 0 ? 3 : 0);   // sometimes invalid
      if (plausible) in0 = i - 1;
      std::vector<int64_t> s = in0 == -1 ? std::vector<int64_t>{n.chw[0], n.chw[1], n.chw[2]}
                                         : (in0 >= 0 && in0 < i ? shp[in0] : std::vector<int64_t>{1, 1, 1});
      const int64_t numel = s[0] * s[1] * s[2];
      int kind = rnd(5);
      if (plausible) {
        if (i == len - 1) kind = VCR_DENSE;
        else if (!flat) kind = i == 0 ? VCR_CONV2D : (rnd(3) == 0 ? VCR_FLATTEN : (rnd(2) ? VCR_RELU : VCR_CONV2D));
        else kind = i % 2 == 0 ? VCR_DENSE : VCR_RELU;
        if (kind == VCR_RELU && i > 0 && n.nodes[i - 1].op == VCR_RELU) kind = flat ? VCR_DENSE : VCR_CONV2D;
      }
      if (kind == VCR_DENSE || i == len - 1) {
        const int32_t out = 1 + rnd(40);
        n.dense(in0, out, numel);
        shp.push_back({out, 1, 1});
        flat = true;
      } else if (kind == VCR_CONV2D) {
        const int32_t out = 32 * (1 + rnd(2));
        const int32_t k = plausible || rnd(4) ? 3 : 1 + rnd(5), st = 1 + rnd(2), pad = plausible || rnd(4) ? 1 : rnd(3);
        n.conv(in0, out, (int32_t)s[0], k, st, pad);
        shp.push_back({out, std::max<int64_t>((s[1] + 2 * pad - k) / st + 1, 0), std::max<int64_t>((s[2] + 2 * pad - k) / st + 1, 0)});
      } else if (kind == VCR_ADD) {
        n.op(VCR_ADD, in0, (int32_t)rnd(i + 1) - 1);
        shp.push_back(s);
      } else if (kind == VCR_FLATTEN) {
        n.op(VCR_FLATTEN, in0);
        shp.push_back({numel, 1, 1});
        flat = true;
      } else {
        n.op(VCR_RELU, in0);
        shp.push_back(s);
      }
    }
    const vcr_status st = n.load(c);
    EXPECT(st >= VCR_OK && st <= VCR_ERR_UNSUPPORTED);
    if (st == VCR_OK) {
      ++ok;
      uint64_t bytes = 0;
      const int32_t B = 1 + rnd(8), m = 1 + rnd(12);
      const int32_t nout = n.nodes.back().out_features;
      EXPECT(vcr_workspace_bytes(c, B, m, 0, &bytes) == VCR_OK);
      const vcr_status cs = crown(c, B, m, n.chw[0] * n.chw[1] * n.chw[2], nout, 0.01f, nullptr);
      EXPECT(cs == VCR_ERR_STATE || cs == VCR_ERR_UNSUPPORTED);
    }
    vcr_destroy(c);
  }
  std::printf("fuzz: %d of %d random networks loaded\n", ok, rounds);
}

}  // namespace

int main(int argc, char **argv) {
  const int rounds = argc > 1 ? std::atoi(argv[1]) : 2000;
  fixed_cases();
  extreme_sizes();
  fuzz(rounds);
  if (g_fail) {
    std::fprintf(stderr, "%d check(s) failed\n", g_fail);
    return 1;
  }
  std::printf("abi validation: all checks passed\n");
  return 0;
}
