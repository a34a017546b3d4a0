// Full CROWN on feed-forward networks with convolutions, residual additions and flatten
// (the convolutional path of the library; MLP chains take the path in api.cpp).
//
// For every ReLU layer (in node order) and for the spec rows, a backward pass is planned
// once at load time by walking the node DAG from the pass's start node down to the input:
//   * the start rows are materialised by an init step (a convolution's kernel slice per
//     output neuron, a dense layer's weight rows, or C W_out for the spec rows);
//   * a convolution or dense node is expanded by one GEMM (transposed convolution on
//     windowed rows, or the dense GEMM), whose epilogue writes the coefficients of the node
//     below: relaxed through the ReLU when that node is a ReLU output, otherwise passed
//     through, plus any other contribution to that node (the identity branch of a residual
//     block) added at the aligned window position;
//   * an add node forwards its coefficients to both inputs; flatten forwards them to the
//     convolutional node it reshapes (rows are kept channels-last throughout);
//   * the last convolution onto the network input is the stem kernel, which concretizes
//     over the box instead of writing coefficients.
// Constant terms are accounted where a coefficient tensor is materialised: the relaxation
// intercepts, and the bias of every node whose coefficients equal that tensor (the node
// itself, and inputs of an add that receive nothing else).  Every step writes per-row
// partial sums that a fixed-order reduction adds to the row constant.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <functional>
#include <map>
#include <vector>

#include "conv.h"
#include "ctx.h"

namespace vcr {

namespace {

struct GNode {
  int op = 0, in0 = -1, in1 = -1;
  int C = 0, H = 1;            // output shape (C, H, H); flat nodes have H = 1
  bool flat = false;
  int64_t numel = 0;
  // conv
  int Ci = 0, Hi = 0, stride = 1;
  // parameters (device)
  float *W = nullptr;          // conv [Co][Ci][3][3]; dense [out][in] original columns
  float *Bt = nullptr;         // conv [Ci_pad][9 Co]; dense [ld(in)][ld(out)] (HWC order if hwc_in)
  float *Wp = nullptr;         // dense [out][ld(in)] original column order (IBP, spec fold)
  float *Wh = nullptr;         // dense [out][ld(in)] HWC column order when hwc_in (init rows)
  float *Wk = nullptr;         // conv [Co][3][3][Ci]: channels contiguous per tap (init rows)
  float *b = nullptr;          // bias, zero padded to ld(out) for dense
  std::vector<float> hb;       // host copy of the bias
  int Ci_pad = 0;
  int64_t ld_in = 0, ld_out = 0;
  bool hwc_in = false;         // dense whose input is a flatten of a convolutional node
  int relu_index = -1;
  std::vector<int> cons;
};

// A coefficient tensor on a node: flat rows (flat nodes) or square windows (conv nodes).
struct Coef {
  int node = -1;
  int slot = -1;
  bool flat = false, dense = false;
  int h = 0, scale = 1;        // window half-size and anchor scale (windowed rows)
  int C = 0, H = 1;
  int64_t row_stride = 0;      // floats per row
  int S() const { return flat ? 1 : (dense ? H : 2 * h + 1); }
};

enum StepKind { ST_INIT_CONV, ST_INIT_FLAT, ST_INIT_SPEC, ST_CONVT, ST_STEM, ST_DENSE };

struct Step {
  StepKind kind;
  int node = -1;               // the node expanded (or the start node for inits)
  Coef src, dst, res;
  bool has_res = false;
  int relu = -1;               // ReLU node whose relaxation is applied to dst, or -1
  int bias_off = -1;           // identity constants (per channel / per column) in the bias arena
  int pid_off = -1;            // identity float4 params (flat / dense-window columns) in the param arena
};

struct PassPlan {
  int start = -1;              // start node (conv / dense), or the output node for the spec pass
  bool spec = false;
  bool windowed = false;       // rows anchored on the start node's neurons
  bool direct = false;         // the start node reads the input: bounds are the exact IBP box range
  int relu = -1;               // ReLU whose input bounds this pass computes (-1: spec)
  std::vector<Step> steps;
  std::vector<int64_t> slot_floats;   // floats per row each slot needs
  int64_t rows_per_unit_mult = 0;      // rows per unit = 2 * this (numel or m)
};

// One step of alpha-CROWN's gradient pass: the relaxed network evaluated forward on every
// coefficient row, each row its own image (the box vertex where the row's bound is attained).
enum FwdKind { FW_CONV, FW_DENSE, FW_ADD };

struct FwdStep {
  FwdKind kind;
  int node = -1;               // node evaluated
  int in = -1;                 // node whose values it reads (-1: the input vertex)
  int res = -1;                // second summand (FW_CONV: a residual fused into the epilogue)
  int out = -1;                // node whose values it writes: node, the ReLU it feeds, or the add
  int relu = -1;               // ReLU index whose line (and slope gradient) is applied, or -1
};

}  // namespace

struct GraphNet {
  int in_C = 0, in_H = 0;
  int64_t n0 = 0;
  std::vector<GNode> nodes;
  std::vector<int> relus;      // ReLU node ids in order
  std::vector<PassPlan> passes;  // one per ReLU (in order) + the spec pass last
  float *bias_arena = nullptr;
  float4 *param_arena = nullptr;
  // alpha-CROWN on the spec pass (empty alpha_why: supported)
  std::string alpha_why;
  std::vector<int64_t> alpha_ld;          // per ReLU index: floats per row of its slope state
  std::vector<FwdStep> fwd;               // gradient pass
  std::vector<int> val_slot;              // per node: slot of its forward values, or -1
  std::vector<int64_t> val_rs;            // per node: floats per row of its forward values
  std::vector<int64_t> fwd_slot_floats;   // floats per row of every slot
  // device [2 R]: neurons of every ReLU node, then its channels (0 for flat nodes), for the
  // split preparation of subdomains
  int32_t *d_relu_info = nullptr;
};

void destroy_graph(GraphNet *g) {
  if (!g) return;
  for (auto &n : g->nodes) {
    for (float *p : {n.W, n.Bt, n.Wp, n.Wh, n.Wk, n.b})
      if (p) (void)hipFree(p);
  }
  if (g->bias_arena) (void)hipFree(g->bias_arena);
  if (g->param_arena) (void)hipFree(g->param_arena);
  if (g->d_relu_info) (void)hipFree(g->d_relu_info);
  delete g;
}

namespace {

// ---- planning -------------------------------------------------------------------------
struct Planner {
  vcr_ctx *c;
  GraphNet *g;
  std::vector<float> host_bias;      // bias arena contents
  std::vector<float4> host_params;   // param arena contents
  std::string why;

  bool unsupported(const char *fmt, ...) {
    char buf[400];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    why = buf;
    return false;
  }

  // consumers of u that are ancestors-or-self of the pass start
  int reach_cons(const std::vector<char> &reach, int u) {
    int k = 0;
    for (int cn : g->nodes[u].cons) k += reach[cn] ? 1 : 0;
    return k;
  }

  // constants per channel (conv node) or per column (flat node) carried by a coefficient
  // tensor materialised on node v
  void alias_bias(const std::vector<char> &reach, int v, std::vector<float> &acc) {
    const GNode &n = g->nodes[v];
    if (n.op == VCR_DENSE || n.op == VCR_CONV2D) {
      for (size_t i = 0; i < acc.size() && i < n.hb.size(); ++i) acc[i] += n.hb[i];
    } else if (n.op == VCR_ADD) {
      for (int u : {n.in0, n.in1})
        if (u >= 0 && reach_cons(reach, u) == 1) alias_bias(reach, u, acc);
    } else if (n.op == VCR_FLATTEN) {
      if (n.in0 >= 0 && reach_cons(reach, n.in0) == 1) alias_bias(reach, n.in0, acc);
    }
  }

  int push_bias(const std::vector<float> &b) {
    const int off = (int)host_bias.size();
    host_bias.insert(host_bias.end(), b.begin(), b.end());
    while (host_bias.size() % 64) host_bias.push_back(0.f);
    return off;
  }

  // identity params for ld columns whose constant is b[j % C] (channels-last) for j < n
  int push_params(const std::vector<float> &b, int C, int64_t n, int64_t ld) {
    const int off = (int)host_params.size();
    for (int64_t j = 0; j < ld; ++j)
      host_params.push_back(j < n ? make_float4(1.f, 1.f, 0.f, b[j % C]) : make_float4(0.f, 0.f, 0.f, 0.f));
    return off;
  }

  // where coefficients produced for node v land: through a ReLU they are relaxed onto its
  // input; through flatten they are the convolutional node's dense window
  // v: the node directly below the expanded one.  Returns the node that receives the
  // coefficients (*dst), the ReLU relaxed on the way (*relu, or -1) and whether a flatten was
  // crossed (the coefficients are then the convolutional node's channels-last dense window).
  bool destination(const std::vector<char> &reach, int v, int *dst, int *relu, bool *flat_cross = nullptr) {
    *relu = -1;
    if (flat_cross) *flat_cross = false;
    if (g->nodes[v].op == VCR_FLATTEN) {
      const int u = g->nodes[v].in0;
      if (u < 0 || g->nodes[u].flat) return unsupported("flatten of a flat node or of the input");
      if (reach_cons(reach, u) != 1) return unsupported("node %d feeds a flatten and other nodes", u);
      if (flat_cross) *flat_cross = true;
      v = u;
    }
    *dst = v;
    const GNode &n = g->nodes[v];
    if (n.op == VCR_RELU) {
      if (reach_cons(reach, v) != 1) return unsupported("ReLU node %d feeds more than one node", v);
      const int z = n.in0;
      if (z < 0) return unsupported("a ReLU directly on the network input");
      if (g->nodes[z].op != VCR_CONV2D && g->nodes[z].op != VCR_DENSE)
        return unsupported("ReLU node %d: its input must be a convolution or a dense node", v);
      if (reach_cons(reach, z) != 1) return unsupported("node %d feeds a ReLU and other nodes", z);
      *relu = v;
      *dst = z;
    }
    return true;
  }

  // slot allocation with reference counts
  std::vector<int> refcnt;
  std::vector<int64_t> *slot_floats;
  int alloc_slot(int64_t floats) {
    for (size_t i = 0; i < refcnt.size(); ++i)
      if (refcnt[i] == 0) {
        refcnt[i] = 1;
        (*slot_floats)[i] = std::max((*slot_floats)[i], floats);
        return (int)i;
      }
    refcnt.push_back(1);
    slot_floats->push_back(floats);
    return (int)refcnt.size() - 1;
  }
  void release(int s) {
    if (s >= 0) --refcnt[s];
  }

  Coef make_coef(int node, bool windowed_rows, int h, int scale) {
    const GNode &n = g->nodes[node];
    Coef k;
    k.node = node;
    k.flat = n.flat;
    k.C = n.flat ? (int)n.numel : n.C;
    k.H = n.flat ? 1 : n.H;
    if (n.flat) {
      k.row_stride = ld_of(n.numel);
    } else {
      k.dense = !windowed_rows;
      k.h = h;
      k.scale = scale;
      const int S = k.S();
      k.row_stride = (int64_t)S * S * n.C;
    }
    return k;
  }

  bool plan(PassPlan &pp) {
    const int nn = (int)g->nodes.size();
    refcnt.clear();
    slot_floats = &pp.slot_floats;
    std::vector<char> reach(nn, 0);
    reach[pp.start] = 1;
    for (int i = pp.start; i >= 0; --i) {
      if (!reach[i]) continue;
      const GNode &n = g->nodes[i];
      if (n.in0 >= 0) reach[n.in0] = 1;
      if (n.op == VCR_ADD && n.in1 >= 0) reach[n.in1] = 1;
    }
    std::map<int, std::vector<Coef>> pend;
    const GNode &s = g->nodes[pp.start];
    if (!pp.spec && s.in0 == -1) {
      // one affine map of the input: its range over the box is exact in IBP
      pp.direct = true;
      return true;
    }
    // ---- init
    {
      Step st;
      st.node = pp.start;
      int v = s.in0, dst, relu;
      if (v < 0) return unsupported("the start node reads the network input directly");
      const int via = v;
      bool crossed = false;
      if (!destination(reach, v, &dst, &relu, &crossed)) return false;
      bool windowed = false;
      int h = 0, scale = 1;
      if (s.op == VCR_CONV2D && !pp.spec) {
        st.kind = ST_INIT_CONV;
        windowed = true;
        h = 1;
        scale = s.stride;
        pp.windowed = true;
      } else {
        st.kind = pp.spec ? ST_INIT_SPEC : ST_INIT_FLAT;
        if (s.op != VCR_DENSE) return unsupported("the start node %d must be dense or conv", pp.start);
      }
      if (crossed && st.kind == ST_INIT_CONV) return unsupported("flatten below a convolution");
      st.relu = relu;
      st.dst = make_coef(dst, windowed, h, scale);
      if (st.kind != ST_INIT_CONV && !st.dst.flat) st.dst.row_stride = ld_of(g->nodes[dst].numel);
      st.dst.slot = alloc_slot(st.dst.row_stride);
      std::vector<float> b(st.dst.C, 0.f);
      if (relu < 0) {
        alias_bias(reach, via, b);
        if (st.kind == ST_INIT_CONV) st.bias_off = push_bias(b);
        else st.pid_off = push_params(b, st.dst.C, g->nodes[dst].numel, st.dst.row_stride);
      }
      pend[dst].push_back(st.dst);
      pp.steps.push_back(st);
    }
    // ---- walk
    for (int n = nn - 1; n >= 0; --n) {
      auto it = pend.find(n);
      if (it == pend.end() || it->second.empty()) continue;
      if (it->second.size() != 1)
        return unsupported("node %d receives several coefficient tensors with no GEMM to sum them", n);
      const Coef A = it->second[0];
      pend.erase(it);
      const GNode &nd = g->nodes[n];
      if (nd.op == VCR_ADD) {
        for (int u : {nd.in0, nd.in1}) {
          if (u < 0) return unsupported("add of the network input");
          Coef f = A;
          f.node = u;
          pend[u].push_back(f);
          ++refcnt[A.slot];
        }
        release(A.slot);
        continue;
      }
      if (nd.op == VCR_FLATTEN) {
        Coef f = A;
        f.node = nd.in0;
        pend[nd.in0].push_back(f);
        continue;
      }
      if (nd.op == VCR_RELU) return unsupported("ReLU node %d reached without a producing GEMM", n);
      Step st;
      st.node = n;
      st.src = A;
      const int v = nd.in0;
      if (nd.op == VCR_CONV2D) {
        if (A.flat) return unsupported("flat coefficients on convolution node %d", n);
        if (v < 0) {
          if (nd.Ci > 4) return unsupported("the first convolution must have at most 4 input channels");
          st.kind = ST_STEM;
          st.dst = A;   // descriptor of the input window filled below
          st.dst.node = -1;
          st.dst.C = nd.Ci;
          st.dst.H = nd.Hi;
          if (!A.dense) {
            st.dst.h = nd.stride * A.h + 1;
            st.dst.scale = nd.stride * A.scale;
          } else {
            st.dst.H = nd.Hi;
          }
          pp.steps.push_back(st);
          release(A.slot);
          continue;
        }
        st.kind = ST_CONVT;
      } else {   // dense
        if (!A.flat) return unsupported("windowed coefficients on dense node %d", n);
        if (v < 0) return unsupported("a dense node on the network input");
        st.kind = ST_DENSE;
      }
      int dst, relu;
      bool crossed = false;
      if (!destination(reach, v, &dst, &relu, &crossed)) return false;
      const int via = v;
      if (crossed && st.kind != ST_DENSE) return unsupported("flatten below a convolution");
      st.relu = relu;
      // destination window
      if (st.kind == ST_CONVT) {
        if (!A.dense) st.dst = make_coef(dst, true, nd.stride * A.h + 1, nd.stride * A.scale);
        else st.dst = make_coef(dst, false, 0, 1);
      } else {
        st.dst = make_coef(dst, false, 0, 1);
        if (!st.dst.flat) st.dst.row_stride = ld_of(g->nodes[dst].numel);
      }
      // the other contributions to dst must all be pending already (summed here); a ReLU
      // target's only consumer is its ReLU (checked by destination())
      if (relu < 0)
        for (int cn : g->nodes[dst].cons)
          if (reach[cn] && cn < n && cn != via)
            return unsupported("node %d: contributions from node %d arrive after the GEMM of node %d", dst, cn, n);
      auto pit = pend.find(dst);
      if (pit != pend.end() && !pit->second.empty()) {
        if (pit->second.size() > 1) return unsupported("node %d: more than one residual", dst);
        if (relu >= 0) return unsupported("residual into a ReLU input");
        st.res = pit->second[0];
        st.has_res = true;
        if (st.res.dense != st.dst.dense || st.res.flat || st.dst.flat) return unsupported("residual layout mismatch");
        if (!st.dst.dense && (st.res.scale != st.dst.scale || st.res.h > st.dst.h))
          return unsupported("residual window mismatch at node %d", dst);
        pend.erase(pit);
      }
      st.dst.slot = alloc_slot(st.dst.row_stride);
      if (relu < 0) {
        std::vector<float> b(st.dst.C, 0.f);
        alias_bias(reach, via, b);
        if (st.kind == ST_CONVT) st.bias_off = push_bias(b);
        else st.pid_off = push_params(b, st.dst.C, g->nodes[dst].numel, st.dst.row_stride);
      }
      pp.steps.push_back(st);
      release(A.slot);
      if (st.has_res) release(st.res.slot);
      pend[dst].push_back(st.dst);
    }
    if (!pend.empty()) return unsupported("coefficients left on node %d", pend.begin()->first);
    if (pp.steps.empty() || pp.steps.back().kind != ST_STEM)
      return unsupported("the backward pass does not end at a convolution on the network input");
    return true;
  }
};

// ---- alpha-CROWN plan -----------------------------------------------------------------------
// The slope state of every ReLU is laid out like the coefficient rows that the spec pass
// relaxes through it, so the relaxation, the recorded coefficients and the gradient pass all
// share one row layout.  The gradient pass evaluates nodes in order up to the last ReLU,
// fusing each ReLU line into the convolution or dense node below it and each add into the
// convolution that produces its later summand; value buffers are reused once their last
// reader has run.  Returns an empty string, or why the net has no alpha-CROWN plan.
std::string plan_alpha(GraphNet *g) {
  const int nn = (int)g->nodes.size();
  const int R = (int)g->relus.size();
  const PassPlan &sp = g->passes.back();
  g->alpha_ld.assign(R, 0);
  for (const Step &st : sp.steps) {
    if (st.relu < 0) continue;
    if (st.kind == ST_CONVT && !st.dst.dense) return "windowed rows in the spec pass";
    g->alpha_ld[g->nodes[st.relu].relu_index] = st.dst.row_stride;
  }
  for (int r = 0; r < R; ++r)
    if (g->alpha_ld[r] <= 0 || g->alpha_ld[r] % 4) return "a ReLU the spec pass does not relax";
  auto src = [&](int v) { return v >= 0 && g->nodes[v].op == VCR_FLATTEN ? g->nodes[v].in0 : v; };
  g->val_rs.assign(nn, 0);
  for (int i = 0; i < nn; ++i) {
    const GNode &n = g->nodes[i];
    g->val_rs[i] = n.op == VCR_RELU ? g->alpha_ld[n.relu_index] : ld_of(n.numel);
  }
  const int last = g->relus.back();
  std::vector<char> written(nn, 0), fused_add(nn, 0);
  g->fwd.clear();
  for (int i = 0; i < last; ++i) {
    const GNode &nd = g->nodes[i];
    if (nd.op == VCR_FLATTEN) continue;
    if (nd.op == VCR_RELU) {
      if (!written[i]) return "a ReLU whose input is not a convolution or dense node";
      continue;
    }
    if (nd.op == VCR_ADD) {
      if (fused_add[i]) continue;
      FwdStep f;
      f.kind = FW_ADD;
      f.node = i;
      f.in = src(nd.in0);
      f.res = src(nd.in1);
      f.out = i;
      if (f.in < 0 || f.res < 0) return "an add of the network input";
      g->fwd.push_back(f);
      written[i] = 1;
      continue;
    }
    FwdStep f;
    f.kind = nd.op == VCR_CONV2D ? FW_CONV : FW_DENSE;
    f.node = i;
    f.in = src(nd.in0);
    f.out = i;
    if (nd.cons.size() == 1) {
      const int cn = nd.cons[0];
      const GNode &c = g->nodes[cn];
      if (c.op == VCR_RELU) {
        f.out = cn;
        f.relu = c.relu_index;
      } else if (c.op == VCR_ADD && f.kind == FW_CONV) {
        const int other = c.in0 == i ? c.in1 : c.in0;
        if (other >= 0 && other < i && written[src(other)] && !g->nodes[other].flat) {
          f.res = src(other);
          f.out = cn;
          fused_add[cn] = 1;
        }
      }
    }
    if (f.kind == FW_DENSE) {
      if (f.in < 0) return "a dense node on the network input";
      if (g->val_rs[f.in] != nd.ld_in) return "dense input rows of another width";
      if (f.relu >= 0 && g->alpha_ld[f.relu] != nd.ld_out) return "dense ReLU rows of another width";
    }
    if (f.kind == FW_CONV && f.in >= 0 && g->nodes[f.in].flat) return "a convolution of a flat node";
    g->fwd.push_back(f);
    written[f.out] = 1;
  }
  for (int r : g->relus)
    if (!written[r]) return "a ReLU whose input is not a convolution or dense node";
  // value slots: a step's output never shares a slot with its inputs
  std::vector<int> last_use(nn, -1);
  for (int k = 0; k < (int)g->fwd.size(); ++k)
    for (int v : {g->fwd[k].in, g->fwd[k].res})
      if (v >= 0) last_use[v] = k;
  g->val_slot.assign(nn, -1);
  g->fwd_slot_floats.clear();
  std::vector<char> busy;
  for (int k = 0; k < (int)g->fwd.size(); ++k) {
    const int o = g->fwd[k].out;
    int sl = -1;
    for (size_t j = 0; j < busy.size() && sl < 0; ++j)
      if (!busy[j]) sl = (int)j;
    if (sl < 0) {
      sl = (int)busy.size();
      busy.push_back(0);
      g->fwd_slot_floats.push_back(0);
    }
    busy[sl] = 1;
    g->fwd_slot_floats[sl] = std::max(g->fwd_slot_floats[sl], g->val_rs[o]);
    g->val_slot[o] = sl;
    for (int v : {g->fwd[k].in, g->fwd[k].res})
      if (v >= 0 && last_use[v] == k) busy[g->val_slot[v]] = 0;
  }
  return std::string();
}

// ---- call-time buffers ------------------------------------------------------------------
struct GBufs {
  float *c0 = nullptr, *r0 = nullptr;
  std::vector<float *> ic, ir;     // IBP centre / radius per node [B][ld(numel)]
  std::vector<float *> L, U;       // per ReLU [B][numel]
  std::vector<float4 *> P;         // per ReLU: [B][H][H][C] or [B][ld(n)]
  float *CW = nullptr, *Cb = nullptr;
  std::vector<float *> slots;
  float *beta = nullptr, *part = nullptr;
  int4 *rows = nullptr;
  // alpha-CROWN: slope state per ReLU, best row bounds, improvement flags, the rows' box
  // vertices and the gradient pass's value slots
  std::vector<AlphaLayer> al;
  float *best_val = nullptr;
  int32_t *flag = nullptr;
  float *vtx = nullptr;
  std::vector<float *> fslots;
  // subdomains: the split table, per-domain flags, the root's bound pointers for the split
  // preparation, and (beta-CROWN) the multipliers with their Adam moments and gradient
  int32_t *off = nullptr, *ent_n = nullptr, *flags = nullptr;
  float4 *ent_p = nullptr;
  const float **Lptr = nullptr;
  float *mul = nullptr, *mul_mom = nullptr, *mul_vel = nullptr, *mul_grad = nullptr;
};

// Sizes of a call: B root inputs, m spec rows; ci inputs per chunk of the intermediate passes,
// cs units per chunk of the spec pass (inputs, or subdomains when D > 0, with S splits each)
struct GShape {
  int B = 1, m = 1, ci = 1, cs = 1, D = 0, S = 0;
  bool alpha = false;
};

struct GPlanSize {
  int chunk = 1;
  size_t bytes = 0;
};

int64_t max_rows_per_unit(const GraphNet *g, int m) {
  int64_t r = 2 * (int64_t)m;
  for (auto &pp : g->passes)
    if (!pp.spec) r = std::max<int64_t>(r, 2 * pp.rows_per_unit_mult);
  return r;
}

int64_t max_part_per_row(const GraphNet *g) {
  // GEMM rows per coefficient row times partial columns, over all steps
  int64_t best = 1;
  for (auto &pp : g->passes)
    for (auto &st : pp.steps) {
      if (st.kind == ST_CONVT) {
        const int S = st.dst.S();
        best = std::max<int64_t>(best, (int64_t)S * S * (g->nodes[st.node].Ci_pad / 64));
      } else if (st.kind == ST_STEM) {
        const int S = st.dst.dense ? st.dst.H : 2 * st.dst.h + 1;
        best = std::max<int64_t>(best, (int64_t)S * S);
      } else if (st.kind == ST_DENSE) {
        best = std::max<int64_t>(best, g->nodes[st.node].ld_in / PART_COLS);
      }
    }
  return best;
}

size_t carve_graph(const vcr_ctx *c, const GraphNet *g, Workspace &w, const GShape &sh, GBufs *bf) {
  const int B = sh.B, m = sh.m;
  const bool alpha = sh.alpha;
  const int nn = (int)g->nodes.size();
  const int64_t ld0 = ld_of(g->n0);
  bf->c0 = take<float>(w, (size_t)B * ld0);
  bf->r0 = take<float>(w, (size_t)B * ld0);
  bf->ic.assign(nn, nullptr);
  bf->ir.assign(nn, nullptr);
  for (int i = 0; i < nn; ++i) {
    const GNode &n = g->nodes[i];
    if (n.op == VCR_FLATTEN) continue;   // aliases its input
    bf->ic[i] = take<float>(w, (size_t)B * ld_of(n.numel));
    bf->ir[i] = take<float>(w, (size_t)B * ld_of(n.numel));
  }
  bf->L.clear();
  bf->U.clear();
  bf->P.clear();
  for (int r : g->relus) {
    const GNode &n = g->nodes[r];
    bf->L.push_back(take<float>(w, (size_t)B * n.numel));
    bf->U.push_back(take<float>(w, (size_t)B * n.numel));
    // channels-last parameters are read up to the padded row width of a dense window: keep a
    // zero tail after the last unit
    bf->P.push_back(take<float4>(w, (size_t)B * (n.flat ? ld_of(n.numel) : n.numel) + LD_ALIGN));
  }
  const GNode &out = g->nodes[nn - 1];
  bf->CW = take<float>(w, (size_t)B * m * out.ld_in);
  bf->Cb = take<float>(w, (size_t)B * m);
  const int64_t rows = std::max(max_rows_per_unit(g, m) * sh.ci, 2 * (int64_t)m * sh.cs);
  size_t nslots = 0;
  for (auto &pp : g->passes) nslots = std::max(nslots, pp.slot_floats.size());
  bf->slots.assign(nslots, nullptr);
  for (size_t s = 0; s < nslots; ++s) {
    int64_t f = 0;
    for (auto &pp : g->passes) {
      if (s >= pp.slot_floats.size()) continue;
      const int64_t pr = pp.spec ? 2 * (int64_t)m * sh.cs : 2 * pp.rows_per_unit_mult * sh.ci;
      // whole GEMM row blocks: the dense GEMM reads and writes padding rows
      f = std::max<int64_t>(f, pp.slot_floats[s] * rows_pad(pr));
    }
    bf->slots[s] = take<float>(w, (size_t)f);
  }
  bf->beta = take<float>(w, (size_t)rows_pad(rows));
  bf->part = take<float>(w, (size_t)((rows + 128) * max_part_per_row(g)));
  bf->rows = take<int4>(w, (size_t)rows);
  bf->al.clear();
  bf->fslots.clear();
  const int64_t ra = rows_pad(2 * (int64_t)m * sh.cs);
  const int R = (int)g->relus.size();
  bf->off = bf->ent_n = bf->flags = nullptr;
  bf->ent_p = nullptr;
  bf->Lptr = nullptr;
  bf->mul = bf->mul_mom = bf->mul_vel = bf->mul_grad = nullptr;
  if (sh.D > 0) {
    bf->off = take<int32_t>(w, (size_t)sh.D * (R + 1));
    bf->ent_n = take<int32_t>(w, (size_t)sh.D * std::max(sh.S, 1));
    bf->ent_p = take<float4>(w, (size_t)sh.D * std::max(sh.S, 1));
    bf->flags = take<int32_t>(w, (size_t)sh.D);
    bf->Lptr = take<const float *>(w, (size_t)2 * R);
    if (alpha && sh.S > 0)
      for (float **q : {&bf->mul, &bf->mul_mom, &bf->mul_vel, &bf->mul_grad}) *q = take<float>(w, (size_t)ra * sh.S);
  }
  if (alpha) {
    int32_t col0 = 0;
    for (size_t r = 0; r < g->relus.size(); ++r) {
      const GNode &n = g->nodes[g->relus[r]];
      AlphaLayer a{};
      a.ld = g->alpha_ld[r];
      a.ldp = n.flat ? ld_of(n.numel) : n.numel;   // the layout of P above
      a.n = (int32_t)n.numel;
      a.col0 = col0;
      a.hwc_C = n.flat ? 0 : n.C;
      a.hwc_HW = n.flat ? 0 : n.H * n.H;
      col0 += a.n;
      for (float **q : {&a.alpha, &a.mom, &a.vel, &a.best, &a.grad, &a.pre}) *q = take<float>(w, (size_t)ra * a.ld);
      bf->al.push_back(a);
    }
    bf->best_val = take<float>(w, (size_t)ra);
    bf->flag = take<int32_t>(w, (size_t)ra);
    bf->vtx = take<float>(w, (size_t)ra * ld_of(g->n0));
    for (int64_t f : g->fwd_slot_floats) bf->fslots.push_back(take<float>(w, (size_t)(ra * f)));
  }
  (void)c;
  return w.used;
}

}  // namespace

// =========================================================================================
// load

vcr_status graph_load(vcr_ctx *c, const vcr_node *nodes, int32_t n, const int32_t in_chw[3],
                      const std::vector<std::vector<int64_t>> &sh) {
  if (in_chw[1] != in_chw[2]) return fail(c, VCR_ERR_UNSUPPORTED, "only square inputs are supported");
  GraphNet *g = new GraphNet();
  std::unique_ptr<GraphNet, void (*)(GraphNet *)> guard(g, destroy_graph);
  c->net_bytes = 0;
  g->in_C = in_chw[0];
  g->in_H = in_chw[1];
  g->n0 = (int64_t)in_chw[0] * in_chw[1] * in_chw[2];
  g->nodes.resize(n);
  int n_input_readers = 0;
  for (int i = 0; i < n; ++i) {
    const vcr_node &d = nodes[i];
    GNode &gn = g->nodes[i];
    gn.op = d.op;
    gn.in0 = d.in0;
    gn.in1 = d.op == VCR_ADD ? d.in1 : -1;
    const auto &s = sh[i];
    const std::vector<int64_t> in_shape = {in_chw[0], in_chw[1], in_chw[2]};
    const auto &si = d.in0 == -1 ? in_shape : sh[d.in0];
    if (d.in0 == -1) ++n_input_readers;
    if (d.op == VCR_ADD && d.in1 == -1) ++n_input_readers;
    gn.numel = s[0] * s[1] * s[2];
    if (d.op == VCR_DENSE || d.op == VCR_FLATTEN || ((d.op == VCR_RELU) && si[1] == 1 && si[2] == 1 &&
                                                   (d.in0 >= 0 && g->nodes[d.in0].flat))) {
      gn.flat = true;
      gn.C = (int)gn.numel;
      gn.H = 1;
    } else {
      gn.C = (int)s[0];
      gn.H = (int)s[1];
      if (s[1] != s[2]) return fail(c, VCR_ERR_UNSUPPORTED, "node %d: only square feature maps are supported", i);
    }
    if (d.op == VCR_CONV2D) {
      if (d.kh != 3 || d.kw != 3 || d.pad != 1 || (d.stride != 1 && d.stride != 2))
        return fail(c, VCR_ERR_UNSUPPORTED, "node %d: convolutions must be 3x3, pad 1, stride 1 or 2", i);
      gn.Ci = (int)si[0];
      gn.Hi = (int)si[1];
      gn.stride = d.stride;
      if (d.out_ch % 32) return fail(c, VCR_ERR_UNSUPPORTED, "node %d: output channels must be a multiple of 32", i);
      if (d.in0 != -1 && gn.Ci % 32)
        return fail(c, VCR_ERR_UNSUPPORTED, "node %d: input channels must be a multiple of 32", i);
      if (d.in0 >= 0 && g->nodes[d.in0].flat) return fail(c, VCR_ERR_UNSUPPORTED, "node %d: conv of a flat node", i);
    }
    if (d.op == VCR_RELU && d.in0 == -1) return fail(c, VCR_ERR_UNSUPPORTED, "a ReLU on the network input");
    if (d.op == VCR_ADD && (gn.flat || (d.in0 >= 0 && g->nodes[d.in0].flat)))
      return fail(c, VCR_ERR_UNSUPPORTED, "node %d: add of flat nodes", i);
    if (d.op == VCR_DENSE && d.in0 >= 0) {
      const GNode &src = g->nodes[d.in0];
      if (src.op == VCR_FLATTEN) gn.hwc_in = true;
      else if (!src.flat) return fail(c, VCR_ERR_SHAPE, "node %d: dense input must be flat (insert a flatten node)", i);
    }
    if (d.op == VCR_DENSE && d.in0 == -1) return fail(c, VCR_ERR_UNSUPPORTED, "dense first layers use the MLP path");
    if (d.in0 >= 0) g->nodes[d.in0].cons.push_back(i);
    if (d.op == VCR_ADD && d.in1 >= 0) g->nodes[d.in1].cons.push_back(i);
    if (d.op == VCR_RELU) {
      gn.relu_index = (int)g->relus.size();
      g->relus.push_back(i);
    }
  }
  if (n_input_readers != 1) return fail(c, VCR_ERR_UNSUPPORTED, "exactly one node may read the network input");
  const bool dev = c->device >= 0;
  if (dev) HIP_TRY(c, hipSetDevice(c->device));
  hipStream_t s = c->stream;
  // upload parameters
  for (int i = 0; i < n; ++i) {
    const vcr_node &d = nodes[i];
    GNode &gn = g->nodes[i];
    if (d.op == VCR_CONV2D) gn.hb.assign(d.b, d.b + gn.C);
    if (d.op == VCR_DENSE) {
      const int64_t nin = d.in0 >= 0 ? g->nodes[d.in0].numel : g->n0;
      gn.ld_in = ld_of(nin);
      gn.ld_out = ld_of(d.out_features);
      gn.hb.assign(d.b, d.b + d.out_features);
    }
    if (d.op == VCR_CONV2D) gn.Ci_pad = (gn.Ci + 63) / 64 * 64;
    if (!dev) continue;
    if (d.op == VCR_CONV2D) {
      const int Co = gn.C, Ci = gn.Ci;
      const size_t wn = (size_t)Co * Ci * 9;
      HIP_TRY(c, hipMalloc(&gn.W, wn * 4));
      c->net_bytes += wn * 4;
      HIP_TRY(c, hipMemcpy(gn.W, d.W, wn * 4, hipMemcpyHostToDevice));
      {
        std::vector<float> wk(wn);
        for (int co = 0; co < Co; ++co)
          for (int ci = 0; ci < Ci; ++ci)
            for (int t = 0; t < 9; ++t) wk[((size_t)co * 9 + t) * Ci + ci] = d.W[((size_t)co * Ci + ci) * 9 + t];
        HIP_TRY(c, hipMalloc(&gn.Wk, wn * 4));
        c->net_bytes += wn * 4;
        HIP_TRY(c, hipMemcpy(gn.Wk, wk.data(), wn * 4, hipMemcpyHostToDevice));
      }
      HIP_TRY(c, hipMalloc(&gn.b, (size_t)Co * 4));
      c->net_bytes += (size_t)Co * 4;
      HIP_TRY(c, hipMemcpy(gn.b, d.b, (size_t)Co * 4, hipMemcpyHostToDevice));
      HIP_TRY(c, hipMalloc(&gn.Bt, (size_t)gn.Ci_pad * 9 * Co * 4));
      c->net_bytes += (size_t)gn.Ci_pad * 9 * Co * 4;
      HIP_TRY(c, launch_repack_convt(gn.W, Co, Ci, gn.Ci_pad, gn.Bt, s));
    } else if (d.op == VCR_DENSE) {
      const int64_t nin = d.in0 >= 0 ? g->nodes[d.in0].numel : g->n0;
      const int64_t nout = d.out_features;
      float *staging = nullptr;
      HIP_TRY(c, hipMalloc(&staging, (size_t)nout * nin * 4));
      HIP_TRY(c, hipMemcpy(staging, d.W, (size_t)nout * nin * 4, hipMemcpyHostToDevice));
      // Wp and Wh have zero rows up to ld(out): the gradient pass runs them as GEMM operands
      HIP_TRY(c, hipMalloc(&gn.Wp, (size_t)gn.ld_out * gn.ld_in * 4));
      c->net_bytes += (size_t)gn.ld_out * gn.ld_in * 4;
      HIP_TRY(c, hipMalloc(&gn.Bt, (size_t)gn.ld_in * gn.ld_out * 4));
      c->net_bytes += (size_t)gn.ld_in * gn.ld_out * 4;
      // Wp = W with zero-padded rows (via the transposed copy)
      HIP_TRY(c, launch_transpose_pad(staging, (int32_t)nout, (int32_t)nin, gn.Bt, gn.ld_out, gn.ld_in, s));
      HIP_TRY(c, launch_transpose_pad(gn.Bt, (int32_t)gn.ld_in, (int32_t)gn.ld_out, gn.Wp, gn.ld_in, gn.ld_out, s));
      if (gn.hwc_in) {
        const GNode &fl = g->nodes[d.in0];
        const GNode &cv = g->nodes[fl.in0];
        HIP_TRY(c, hipMalloc(&gn.Wh, (size_t)gn.ld_out * gn.ld_in * 4));
        c->net_bytes += (size_t)gn.ld_out * gn.ld_in * 4;
        HIP_TRY(c, launch_permute_hwc(staging, (int32_t)nout, cv.C, cv.H * cv.H, gn.Wh, gn.ld_in, s));
        if (gn.ld_out > nout)
          HIP_TRY(c, launch_fill(gn.Wh + (size_t)nout * gn.ld_in, (gn.ld_out - nout) * gn.ld_in, 0.f, s));
        HIP_TRY(c, launch_transpose_pad(gn.Wh, (int32_t)nout, (int32_t)gn.ld_in, gn.Bt, gn.ld_out, gn.ld_in, s));
      }
      HIP_TRY(c, hipMalloc(&gn.b, (size_t)gn.ld_out * 4));
      c->net_bytes += (size_t)gn.ld_out * 4;
      HIP_TRY(c, launch_fill(gn.b, gn.ld_out, 0.f, s));
      HIP_TRY(c, hipStreamSynchronize(s));
      HIP_TRY(c, hipMemcpy(gn.b, d.b, (size_t)nout * 4, hipMemcpyHostToDevice));
      HIP_TRY(c, hipFree(staging));
    }
  }
  // plan every pass
  Planner pl{c, g};
  for (int r : g->relus) {
    PassPlan pp;
    pp.start = g->nodes[r].in0;
    pp.relu = r;
    pp.rows_per_unit_mult = g->nodes[pp.start].numel;
    if (!pl.plan(pp)) return fail(c, VCR_ERR_UNSUPPORTED, "ReLU node %d: %s", r, pl.why.c_str());
    g->passes.push_back(pp);
  }
  {
    PassPlan pp;
    pp.start = n - 1;
    pp.spec = true;
    if (!pl.plan(pp)) return fail(c, VCR_ERR_UNSUPPORTED, "spec pass: %s", pl.why.c_str());
    g->passes.push_back(pp);
  }
  g->alpha_why = g->relus.empty() ? std::string("no ReLU") : plan_alpha(g);
  // the first ReLU's input must be reachable from the box by one pass like the others:
  // every pass ends at the stem (checked by the planner)
  if (dev && !pl.host_bias.empty()) {
    HIP_TRY(c, hipMalloc(&g->bias_arena, pl.host_bias.size() * 4));
    c->net_bytes += pl.host_bias.size() * 4;
    HIP_TRY(c, hipMemcpy(g->bias_arena, pl.host_bias.data(), pl.host_bias.size() * 4, hipMemcpyHostToDevice));
  }
  if (dev && !pl.host_params.empty()) {
    HIP_TRY(c, hipMalloc(&g->param_arena, pl.host_params.size() * sizeof(float4)));
    c->net_bytes += pl.host_params.size() * sizeof(float4);
    HIP_TRY(c, hipMemcpy(g->param_arena, pl.host_params.data(), pl.host_params.size() * sizeof(float4),
                         hipMemcpyHostToDevice));
  }
  if (dev && !g->relus.empty()) {
    std::vector<int32_t> info;
    for (int r : g->relus) info.push_back((int32_t)g->nodes[r].numel);
    for (int r : g->relus) info.push_back(g->nodes[r].flat ? 0 : g->nodes[r].C);
    HIP_TRY(c, hipMalloc(&g->d_relu_info, info.size() * sizeof(int32_t)));
    c->net_bytes += info.size() * sizeof(int32_t);
    HIP_TRY(c, hipMemcpy(g->d_relu_info, info.data(), info.size() * sizeof(int32_t), hipMemcpyHostToDevice));
  }
  if (dev) HIP_TRY(c, hipDeviceSynchronize());
  destroy_graph(c->graph);
  c->graph = guard.release();
  c->relu_n.clear();
  for (int r : g->relus) c->relu_n.push_back((int32_t)g->nodes[r].numel);
  c->n0 = (int32_t)g->n0;
  return VCR_OK;
}

// =========================================================================================
// calls

namespace {

vcr_status run_ibp(vcr_ctx *c, GraphNet *g, GBufs &bf, int B) {
  hipStream_t s = c->stream;
  const int nn = (int)g->nodes.size();
  const int64_t ld0 = ld_of(g->n0);
  for (int i = 0; i < nn; ++i) {
    GNode &n = g->nodes[i];
    float *ci_c = n.in0 == -1 ? bf.c0 : bf.ic[n.in0];
    float *ci_r = n.in0 == -1 ? bf.r0 : bf.ir[n.in0];
    const int64_t ld_i = n.in0 == -1 ? ld0 : ld_of(g->nodes[n.in0].numel);
    const int64_t ld_o = ld_of(n.numel);
    switch (n.op) {
      case VCR_CONV2D:
        HIP_TRY(c, launch_ibp_conv(n.W, n.b, n.C, n.Ci, n.Hi, n.H, n.stride, 1, ci_c, ci_r, ld_i, bf.ic[i], bf.ir[i],
                                   ld_o, B, s));
        break;
      case VCR_RELU:
        HIP_TRY(c, launch_ibp_relu(ci_c, ci_r, bf.ic[i], bf.ir[i], (int64_t)B * ld_o, s));
        break;
      case VCR_ADD:
        HIP_TRY(c, launch_ibp_add(ci_c, ci_r, bf.ic[n.in1], bf.ir[n.in1], bf.ic[i], bf.ir[i], (int64_t)B * ld_o, s));
        break;
      case VCR_FLATTEN:
        bf.ic[i] = ci_c;
        bf.ir[i] = ci_r;
        break;
      case VCR_DENSE:
        HIP_TRY(c, launch_ibp_dense(n.Wp, n.ld_in, n.b, (int32_t)n.numel, (int32_t)ld_i, ci_c, ci_r, n.ld_in, 0,
                                    bf.ic[i], bf.ir[i], n.ld_out, B, s));
        break;
    }
  }
  return VCR_OK;
}

float4 *relu_P(GraphNet *g, GBufs &bf, int relu_node) { return bf.P[g->nodes[relu_node].relu_index]; }

// One pass over `units` units starting at absolute unit u0.  Leaves the row constants
// (complete bounds) in bf.beta.  With alpha (the spec pass of alpha-CROWN) every relaxation
// takes the rows' slopes at unstable neurons and records the coefficients before it, and the
// stem writes each row's box vertex.
vcr_status run_pass(vcr_ctx *c, GraphNet *g, GBufs &bf, const PassPlan &pp, int u0, int units, int m,
                    uint64_t *flops, bool alpha = false, const SplitTable *tab = nullptr) {
  hipStream_t s = c->stream;
  const GNode &start = g->nodes[pp.start];
  const int64_t rpu = pp.spec ? 2 * (int64_t)m : 2 * pp.rows_per_unit_mult;
  const int64_t R = rpu * units;
  // subdomains (tab, spec pass only): units are domains u0.. of one input, whose parameters,
  // box and spec rows are unit 0's
  const bool dom = tab != nullptr;
  const int pu0 = dom ? 0 : u0;
  if (dom) {
    if (!pp.spec || R >= ((int64_t)1 << 31)) return fail(c, VCR_ERR_UNSUPPORTED, "internal: subdomain pass");
    HIP_TRY(c, launch_row_table(bf.rows, R, (int32_t)R, start.C, start.H, start.H, 0, 0, s));
  } else {
    HIP_TRY(c, launch_row_table(bf.rows, R, (int32_t)rpu, start.C, start.H, start.H, pp.windowed ? 1 : 0, u0, s));
  }
  auto ridx = [&](int relu_node) { return g->nodes[relu_node].relu_index; };
  auto slot = [&](const Coef &k) { return bf.slots[k.slot]; };
  for (const Step &st : pp.steps) {
    const GNode &nd = g->nodes[st.node];
    switch (st.kind) {
      case ST_INIT_CONV: {
        ConvInitArgs a{};
        a.W = nd.Wk;
        a.b = nd.b;
        a.C_src = nd.C;
        a.H_src = nd.H;
        a.C_in = nd.Ci;
        a.H_in = nd.Hi;
        a.S = 3;
        a.h = 1;
        a.scale = nd.stride;
        a.R = R;
        a.rows = bf.rows;
        a.P_pos = st.relu >= 0 ? relu_P(g, bf, st.relu) : nullptr;
        a.bias_next = st.bias_off >= 0 ? g->bias_arena + st.bias_off : nullptr;
        a.out = slot(st.dst);
        a.beta = bf.beta;
        HIP_TRY(c, launch_init_conv(a, s));
        break;
      }
      case ST_INIT_FLAT:
      case ST_INIT_SPEC: {
        InitArgs ia{};
        const bool spec = st.kind == ST_INIT_SPEC;
        const float *W = nd.hwc_in ? nd.Wh : nd.Wp;
        ia.src = spec ? bf.CW + (int64_t)pu0 * m * nd.ld_in : W;
        ia.ld_src = nd.ld_in;
        ia.n_src = spec ? m : (int32_t)nd.numel;
        ia.per_unit_src = spec && !dom ? 1 : 0;
        ia.src_bias = spec ? bf.Cb + (int64_t)pu0 * m : nd.b;
        ia.n_cols = (int32_t)g->nodes[st.dst.node].numel;
        ia.ldo = st.dst.row_stride;
        ia.M = (int32_t)R;
        ia.units = units;
        if (st.relu >= 0) {
          // flat ReLU parameters have the padded row width per unit; channels-last ones numel
          const int64_t ldp = st.dst.flat ? st.dst.row_stride : g->nodes[st.dst.node].numel;
          ia.P = relu_P(g, bf, st.relu) + (int64_t)pu0 * ldp;
          ia.ldp = ldp;
          ia.param_per_unit = dom ? 0 : 1;
          if (dom) {
            ia.splits = *tab;
            ia.relu_index = ridx(st.relu);
          }
        } else {
          ia.P = g->param_arena + st.pid_off;
          ia.ldp = st.dst.row_stride;
          ia.param_per_unit = 0;
        }
        ia.out = slot(st.dst);
        ia.beta = bf.beta;
        if (ia.ldo != nd.ld_in) return fail(c, VCR_ERR_UNSUPPORTED, "internal: init row width mismatch");
        if (alpha && st.relu >= 0) {
          const AlphaLayer &l = bf.al[g->nodes[st.relu].relu_index];
          if (l.ld != ia.ldo) return fail(c, VCR_ERR_UNSUPPORTED, "internal: slope row width mismatch");
          ia.alpha = l.alpha;
          ia.ld_alpha = l.ld;
          ia.pre = l.pre;
        }
        HIP_TRY(c, launch_init_rows(ia, s));
        break;
      }
      case ST_CONVT: {
        ConvTArgs a{};
        a.A = slot(st.src);
        a.row_stride_out = st.src.row_stride;
        a.S_out = st.src.S();
        a.C_out = nd.C;
        a.Bt = nd.Bt;
        a.ldb = 9 * (int64_t)nd.C;
        a.N_pad = nd.Ci_pad;
        a.C_in = nd.Ci;
        a.S_in = st.dst.S();
        a.H_in = nd.Hi;
        a.row_stride_in = st.dst.row_stride;
        a.stride = nd.stride;
        a.delta = st.src.dense ? 1 : 0;
        const int64_t M = R * a.S_in * a.S_in;
        if (M >= (int64_t)1 << 31) return fail(c, VCR_ERR_UNSUPPORTED, "pass too large for one launch (%lld GEMM rows)",
                                               (long long)M);
        a.R = (int32_t)R;
        a.M_pad = (int32_t)rows_pad(M);
        a.rows = bf.rows;
        a.dense = st.dst.dense ? 1 : 0;
        a.scale = st.dst.scale;
        a.h_in = st.dst.h;
        // windowed passes: rows (unit, direction, c, a_y, a_x) anchored on the start node's
        // H x H grid, so row r's anchor is r mod H^2
        a.Ha = pp.windowed && !dom && !st.dst.dense ? start.H : 0;
        if (!st.src.dense) {
          a.src_scale = st.src.scale;
          a.src_h = st.src.h;
          a.H_out = nd.H;
        }
        if (st.has_res) {
          a.res = slot(st.res);
          a.res_row_stride = st.res.row_stride;
          a.res_S = st.res.S();
          a.res_off = st.dst.dense ? 0 : st.dst.h - st.res.h;
        }
        a.P_pos = st.relu >= 0 ? relu_P(g, bf, st.relu) : nullptr;
        a.bias = st.bias_off >= 0 ? g->bias_arena + st.bias_off : nullptr;
        a.out = slot(st.dst);
        a.part = bf.part;
        if (alpha && st.relu >= 0) {
          const AlphaLayer &l = bf.al[g->nodes[st.relu].relu_index];
          if (!st.dst.dense || l.ld != st.dst.row_stride)
            return fail(c, VCR_ERR_UNSUPPORTED, "internal: slope row width mismatch");
          a.alpha = l.alpha;
          a.pre = l.pre;
        }
        if (dom && st.relu >= 0) {
          a.splits = *tab;
          a.relu_index = ridx(st.relu);
        }
        const int parts = convt_launches(a);
        if (parts < 0) return fail(c, VCR_ERR_UNSUPPORTED, "internal: transposed convolution shape");
        for (int k = 0; k < parts; ++k) {
          const uint64_t cf = convt_part_flops(a, k);
          const vcr_status st2 = timed_launch(c, s, 1, cf, [&] { return launch_convt_part(a, k, s); });
          if (st2 != VCR_OK) return st2;
          *flops += cf;
        }
        WinClip cw;
        if (convt_clipped(a)) cw = WinClip{a.Ha, a.scale, a.h_in, a.S_in, a.H_in};
        HIP_TRY(c, launch_rowsum_win(bf.beta, bf.part, a.N_pad / 64, a.M_pad, R, a.S_in * a.S_in, s, cw));
        break;
      }
      case ST_STEM: {
        StemArgs a{};
        a.A = slot(st.src);
        a.row_stride_out = st.src.row_stride;
        a.S_out = st.src.S();
        a.C_out = nd.C;
        a.W = nd.W;
        a.C_in = nd.Ci;
        a.S_in = st.src.dense ? nd.Hi : 2 * st.dst.h + 1;
        a.H_in = nd.Hi;
        a.stride = nd.stride;
        a.delta = st.src.dense ? 1 : 0;
        a.R = (int32_t)R;

        a.rows = bf.rows;
        a.dense = st.src.dense ? 1 : 0;
        a.scale = st.dst.scale;
        a.h_in = st.dst.h;
        if (!st.src.dense) {
          a.src_scale = st.src.scale;
          a.src_h = st.src.h;
          a.H_src = nd.H;
        }
        a.c0 = bf.c0;
        a.r0 = bf.r0;
        a.ld_box = ld_of(g->n0);
        a.part = bf.part;
        if (alpha) {
          a.vtx = bf.vtx;
          a.ld_vtx = ld_of(g->n0);
        }
        HIP_TRY(c, launch_stem(a, s));
        HIP_TRY(c, launch_rowsum_win(bf.beta, bf.part, 1, 0, R, a.S_in * a.S_in, s));
        *flops += 2ull * (uint64_t)R * a.S_out * a.S_out * 9ull * (uint64_t)nd.C * (uint64_t)nd.Ci;
        break;
      }
      case ST_DENSE: {
        GemmArgs ga{};
        ga.A = slot(st.src);
        ga.lda = nd.ld_out;
        ga.Bt = nd.Bt;
        ga.ldb = nd.ld_out;
        ga.M = (int32_t)R;
        ga.M_pad = (int32_t)rows_pad(R);
        ga.K = (int32_t)nd.ld_out;
        ga.N_pad = (int32_t)nd.ld_in;
        ga.mode = EPI_RELAX;
        ga.out = slot(st.dst);
        ga.ldo = nd.ld_in;
        if (st.relu >= 0) {
          const int64_t ldp = st.dst.flat ? nd.ld_in : g->nodes[st.dst.node].numel;
          ga.P = relu_P(g, bf, st.relu) + (int64_t)pu0 * ldp;
          ga.ldp = ldp;
          ga.rows_per_unit = dom ? ga.M_pad : (int32_t)rpu;
          ga.n_units = dom ? 1 : units;
          if (dom) {
            ga.splits = *tab;
            ga.relu_index = ridx(st.relu);
          }
        } else {
          ga.P = g->param_arena + st.pid_off;
          ga.ldp = 0;
          ga.rows_per_unit = ga.M_pad;
          ga.n_units = 1;
        }
        ga.part = bf.part;
        if (st.dst.row_stride != nd.ld_in) return fail(c, VCR_ERR_UNSUPPORTED, "internal: dense output width mismatch");
        if (alpha && st.relu >= 0) {
          const AlphaLayer &l = bf.al[g->nodes[st.relu].relu_index];
          if (l.ld != nd.ld_in) return fail(c, VCR_ERR_UNSUPPORTED, "internal: slope row width mismatch");
          ga.alpha = l.alpha;
          ga.ld_alpha = l.ld;
          ga.pre = l.pre;
          ga.ld_pre = l.ld;
        }
        const uint64_t df = 2ull * (uint64_t)R * (uint64_t)nd.numel * (uint64_t)g->nodes[nd.in0].numel;
        {
          const vcr_status st2 = TIMED_GEMM(c, s, df, ga);
          if (st2 != VCR_OK) return st2;
        }
        HIP_TRY(c, launch_rowsum_win(bf.beta, bf.part, (int32_t)(nd.ld_in / PART_COLS), ga.M_pad, R, 1, s));
        *flops += df;
        break;
      }
    }
  }
  return VCR_OK;
}

// alpha-CROWN's gradient pass over the M rows of `units` units from unit u0: the relaxed
// network evaluated forward from each row's box vertex (bf.vtx, written by the spec pass),
// each ReLU replaced by the line the row's coefficient selected, which leaves the slope
// gradients in bf.al[].grad.
vcr_status run_forward(vcr_ctx *c, GraphNet *g, GBufs &bf, int u0, int units, int32_t M, int32_t rpu,
                       uint64_t *flops, const SplitTable *ftab = nullptr) {
  hipStream_t s = c->stream;
  // subdomains: every row takes unit 0's relaxation, split neurons their own, and the
  // multipliers' gradients are written where a split neuron's value is formed
  const bool dom = ftab != nullptr;
  if (dom) u0 = 0;
  const int64_t ld0 = ld_of(g->n0);
  auto val = [&](int v) { return v < 0 ? bf.vtx : bf.fslots[g->val_slot[v]]; };
  auto rs = [&](int v) { return v < 0 ? ld0 : g->val_rs[v]; };
  for (const FwdStep &f : g->fwd) {
    const GNode &nd = g->nodes[f.node];
    switch (f.kind) {
      case FW_CONV: {
        FwdConvArgs a{};
        a.in = val(f.in);
        a.in_rs = rs(f.in);
        a.Ci = nd.Ci;
        a.Hi = nd.Hi;
        a.Wk = nd.Wk;
        a.bias = nd.b;
        a.Co = nd.C;
        a.Ho = nd.H;
        a.stride = nd.stride;
        a.rows = M;
        if (f.res >= 0) {
          a.res = val(f.res);
          a.res_rs = rs(f.res);
        }
        if (f.relu >= 0) {
          const AlphaLayer &l = bf.al[f.relu];
          a.P = bf.P[f.relu] + (int64_t)u0 * l.ldp;
          a.rows_per_unit = dom ? M : rpu;
          a.units = dom ? 1 : units;
          a.alpha = l.alpha;
          a.pre = l.pre;
          a.grad = l.grad;
          if (dom) {
            a.splits = *ftab;
            a.relu_index = f.relu;
          }
        }
        a.out = val(f.out);
        a.out_rs = rs(f.out);
        HIP_TRY(c, launch_fwd_conv(a, s));
        *flops += 2ull * (uint64_t)M * (uint64_t)nd.numel * 9ull * (uint64_t)nd.Ci;
        break;
      }
      case FW_DENSE: {
        GemmArgs ga{};
        ga.A = val(f.in);
        ga.lda = nd.ld_in;
        ga.Bt = nd.hwc_in ? nd.Wh : nd.Wp;
        ga.ldb = nd.ld_in;
        ga.M = M;
        ga.M_pad = (int32_t)rows_pad(M);
        ga.K = (int32_t)nd.ld_in;
        ga.N_pad = (int32_t)nd.ld_out;
        ga.out = val(f.out);
        ga.ldo = nd.ld_out;
        if (f.relu >= 0) {
          const AlphaLayer &l = bf.al[f.relu];
          ga.mode = EPI_FORWARD;
          ga.P = bf.P[f.relu] + (int64_t)u0 * l.ldp;
          ga.ldp = l.ldp;
          ga.rows_per_unit = dom ? ga.M_pad : rpu;
          ga.n_units = dom ? 1 : units;
          if (dom) {
            ga.splits = *ftab;
            ga.relu_index = f.relu;
          }
          ga.alpha = l.alpha;
          ga.ld_alpha = l.ld;
          ga.pre = l.pre;
          ga.ld_pre = l.ld;
          ga.grad = l.grad;
        } else {
          ga.mode = EPI_AFFINE;
          ga.bias = nd.b;
          ga.rows_per_unit = ga.M_pad;
          ga.n_units = 1;
        }
        const uint64_t df = 2ull * (uint64_t)M * (uint64_t)nd.numel * (uint64_t)g->nodes[f.in].numel;
        const vcr_status st = TIMED_GEMM(c, s, df, ga);
        if (st != VCR_OK) return st;
        *flops += df;
        break;
      }
      case FW_ADD:
        HIP_TRY(c, launch_fwd_add(val(f.in), rs(f.in), val(f.res), rs(f.res), val(f.out), rs(f.out), M, nd.numel, s));
        break;
    }
  }
  return VCR_OK;
}

struct GraphAlphaCall {
  vcr_alpha_opts o;
  int64_t n_total = 0;
  float lr_beta = 0.f;   // subdomains (beta-CROWN): step size of the multipliers
};

// The split table of domains d0 .. d0 + dc - 1 (a slice of the one the split preparation
// wrote for all domains); with S > 0 and beta, the multipliers of those rows.
SplitTable domain_table(const GraphNet *g, const GBufs &bf, int d0, int dc, int m, int S, bool beta) {
  const int R = (int)g->relus.size();
  SplitTable t{};
  t.off = bf.off + (int64_t)d0 * (R + 1);
  t.ent_n = bf.ent_n + (int64_t)d0 * S;
  t.ent_p = bf.ent_p + (int64_t)d0 * S;
  t.R = R;
  t.S = S;
  t.D = dc;
  t.rows_per_domain = 2 * m;
  t.beta = beta && S > 0 ? bf.mul : nullptr;
  return t;
}

// alpha-CROWN on the spec pass, per chunk of units: evaluate with the current slopes (the
// spec pass with per-row slopes), keep each row's best bound, run the gradient pass and one
// projected Adam step; T steps give T + 1 evaluations.  The slope kernels are the MLP path's.
// Units are inputs, or with D > 0 subdomains of the one input (beta-CROWN: the split
// multipliers are optimised with the slopes, and infeasible domains report lb = +inf).
vcr_status alpha_spec_graph(vcr_ctx *c, GraphNet *g, GBufs &bf, const PassPlan &pp, int units_total, int m,
                            int chunk, int D, int S, const GraphAlphaCall &ac, float *lb, float *ub, uint64_t *flops,
                            int *chunks) {
  hipStream_t s = c->stream;
  const vcr_alpha_opts &o = ac.o;
  const int R = (int)g->relus.size();
  const int32_t rpu = 2 * m;
  const bool dom = D > 0;
  for (int u0 = 0; u0 < units_total; u0 += chunk) {
    const int units = std::min(chunk, units_total - u0);
    const int32_t M = rpu * units;
    const int32_t M_pad = (int32_t)rows_pad(M);
    // per-unit parameters (inputs) or the root's for every row (subdomains)
    const int32_t prpu = dom ? M_pad : rpu;
    const int64_t pu0 = dom ? 0 : u0;
    for (int r = 0; r < R; ++r) {
      bf.al[r].P = bf.P[r] + pu0 * bf.al[r].ldp;
      HIP_TRY(c, launch_alpha_init(bf.al[r], o.alpha_init ? o.alpha_init + (int64_t)u0 * rpu * ac.n_total : nullptr,
                                   ac.n_total, M, M_pad, prpu, s));
    }
    SplitTable tab{}, ftab{};
    BetaState bs{bf.mul, bf.mul_mom, bf.mul_vel, bf.mul_grad, S};
    if (dom) {
      tab = domain_table(g, bf, u0, units, m, S, true);
      ftab = tab;
      ftab.grad_beta = S > 0 ? bf.mul_grad : nullptr;
      if (S > 0) HIP_TRY(c, launch_beta_init(bs, M_pad, s));
    }
    // value rows are read at their padded width: zero once, the padding is never written
    for (size_t k = 0; k < bf.fslots.size(); ++k)
      HIP_TRY(c, launch_fill(bf.fslots[k], (int64_t)M_pad * g->fwd_slot_floats[k], 0.f, s));
    HIP_TRY(c, launch_fill(bf.vtx, (int64_t)M_pad * ld_of(g->n0), 0.f, s));
    for (int32_t t = 0; t <= o.iters; ++t) {
      vcr_status st = run_pass(c, g, bf, pp, u0, units, m, flops, true, dom ? &tab : nullptr);
      if (st != VCR_OK) return st;
      HIP_TRY(c, launch_alpha_best(bf.beta, nullptr, 0, M_pad, M, m, t == 0, bf.best_val, bf.flag,
                                   o.lb_hist ? o.lb_hist + ((int64_t)t * units_total + u0) * m : nullptr,
                                   o.ub_hist ? o.ub_hist + ((int64_t)t * units_total + u0) * m : nullptr, s));
      const bool step = t < o.iters;
      if (!step)
        for (int r = 0; r < R; ++r) HIP_TRY(c, launch_alpha_keep(bf.al[r], bf.flag, M, s));
      if (!step && !o.grad_out) break;
      st = run_forward(c, g, bf, u0, units, M, rpu, flops, dom ? &ftab : nullptr);
      if (st != VCR_OK) return st;
      if (!step) break;
      const double c1 = 1.0 / (1.0 - std::pow((double)o.beta1, (double)(t + 1)));
      const double c2 = 1.0 / (1.0 - std::pow((double)o.beta2, (double)(t + 1)));
      for (int r = 0; r < R; ++r)
        HIP_TRY(c, launch_alpha_adam(bf.al[r], bf.flag, M, prpu, o.lr, o.beta1, o.beta2, o.adam_eps, (float)c1,
                                     (float)c2, s));
      if (dom && S > 0)
        HIP_TRY(c, launch_beta_adam(bs, M, ac.lr_beta, o.beta1, o.beta2, o.adam_eps, (float)c1, (float)c2, s));
    }
    HIP_TRY(c, launch_alpha_final(bf.best_val, units, m, dom ? bf.flags + u0 : nullptr, lb + (int64_t)u0 * m,
                                  ub + (int64_t)u0 * m, s));
    if (o.alpha_out || o.grad_out)
      for (int r = 0; r < R; ++r)
        HIP_TRY(c, launch_alpha_out(bf.al[r], M, m, ac.n_total,
                                    o.alpha_out ? o.alpha_out + (int64_t)u0 * rpu * ac.n_total : nullptr,
                                    o.grad_out ? o.grad_out + (int64_t)u0 * rpu * ac.n_total : nullptr, s));
    ++*chunks;
  }
  return VCR_OK;
}

}  // namespace

namespace {

// The call shape under the workspace cap: inputs (or subdomains) per chunk, halved from the
// whole batch until the plan fits (VCR_ERR_OOM when one unit does not).  Subdomains share one
// root input, whose intermediate passes run once.
vcr_status plan_shape(vcr_ctx *c, GShape sh, GShape *out, size_t *bytes_out) {
  GraphNet *g = c->graph;
  const int units = sh.D > 0 ? sh.D : sh.B;
  sh.ci = sh.D > 0 ? 1 : units;
  sh.cs = units;
  Workspace probe;
  GBufs tmp;
  size_t need = carve_graph(c, g, probe, sh, &tmp);
  if (c->ws_cap > 0) {
    while (need > c->ws_cap && sh.cs > 1) {
      sh.cs = (sh.cs + 1) / 2;
      if (sh.D == 0) sh.ci = sh.cs;
      Workspace pw;
      need = carve_graph(c, g, pw, sh, &tmp);
    }
    if (need > c->ws_cap)
      return fail(c, VCR_ERR_OOM, "workspace cap %llu bytes is below the minimum plan (%llu bytes)",
                  (unsigned long long)c->ws_cap, (unsigned long long)need);
  }
  *out = sh;
  *bytes_out = need;
  return VCR_OK;
}

}  // namespace

// Inputs per chunk and workspace bytes of a CROWN call of B inputs
vcr_status graph_plan(vcr_ctx *c, int32_t B, int32_t m, int *chunk_out, size_t *bytes_out, bool alpha) {
  GShape sh;
  sh.B = B;
  sh.m = m;
  sh.alpha = alpha;
  GShape out;
  const vcr_status st = plan_shape(c, sh, &out, bytes_out);
  if (st == VCR_OK) *chunk_out = out.cs;
  return st;
}

namespace {

// The split table of every subdomain from the root's bounds (in the workspace), written by
// the split preparation; flags per domain, invalid ones counted in the context's counters.
vcr_status prepare_splits(vcr_ctx *c, GraphNet *g, GBufs &bf, const vcr_splits *splits) {
  hipStream_t s = c->stream;
  const int R = (int)g->relus.size();
  if (2 * R > PTR_TABLE_MAX) return fail(c, VCR_ERR_UNSUPPORTED, "subdomains need at most %d ReLU nodes", PTR_TABLE_MAX / 2);
  PtrTable pt{};
  for (int r = 0; r < R; ++r) {
    pt.p[r] = bf.L[r];
    pt.p[R + r] = bf.U[r];
  }
  HIP_TRY(c, launch_store_ptrs(pt, 2 * R, bf.Lptr, s));
  HIP_TRY(c, launch_fill(reinterpret_cast<float *>(c->d_counters), 80, 0.f, s));
  SplitPrepArgs sp{};
  sp.relu_id = splits->relu_id;
  sp.neuron = splits->neuron;
  sp.sign = splits->sign;
  sp.D = splits->n_domains;
  sp.S = splits->per_domain;
  sp.R = R;
  sp.relu_n = g->d_relu_info;
  sp.hwc_C = g->d_relu_info + R;
  sp.L = bf.Lptr;
  sp.U = bf.Lptr + R;
  sp.off = bf.off;
  sp.ent_n = bf.ent_n;
  sp.ent_p = bf.ent_p;
  sp.flags = bf.flags;
  sp.n_invalid = c->d_counters + 64;
  sp.lam_rule = c->lambda_rule;
  HIP_TRY(c, launch_split_prepare(sp, s));
  return VCR_OK;
}

// Full CROWN (intermediate passes of every ReLU layer, then the spec pass) on B inputs, or
// with splits on subdomains of the one input (the root's intermediate bounds, each split
// neuron's interval clamped), or with ac alpha-CROWN on the spec pass (with splits:
// beta-CROWN).
vcr_status graph_run(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m, float *lb,
                     float *ub, const vcr_splits *splits, const GraphAlphaCall *ac) {
  GraphNet *g = c->graph;
  const int nn = (int)g->nodes.size();
  const GNode &out = g->nodes[nn - 1];
  GShape sh;
  sh.B = B;
  sh.m = m;
  sh.alpha = ac != nullptr;
  sh.D = splits ? splits->n_domains : 0;
  sh.S = splits ? splits->per_domain : 0;
  size_t need = 0;
  vcr_status st = plan_shape(c, sh, &sh, &need);
  if (st != VCR_OK) return st;
  const int units_total = sh.D > 0 ? sh.D : B;
  if (c->device < 0) {
    c->chunks_last = ((int)g->passes.size() - 1) * ((B + sh.ci - 1) / sh.ci) + (units_total + sh.cs - 1) / sh.cs;
    return fail(c, VCR_ERR_STATE, "validation-only context: no device work");
  }
  HIP_TRY(c, hipSetDevice(c->device));
  c->lastL.clear();
  c->lastU.clear();
  st = ensure_ws(c, need);
  if (st != VCR_OK) return st;
  GBufs bf;
  carve_graph(c, g, c->ws, sh, &bf);
  hipStream_t s = c->stream;
  const int64_t ld0 = ld_of(g->n0);
  // the rounds of a branch-and-bound loop bound subdomains of one root: its box, bounds and
  // relaxation (all the subdomain pass reads of it) are computed in the first round and
  // copied back in the later ones
  const bool use_cache = splits && c->bab_reuse && c->root_cached;
  const bool fill_cache = splits && c->bab_reuse && !c->root_cached;
  auto cache_copy = [&](bool to_cache) -> vcr_status {
    size_t o = 0;
    auto move = [&](float *ws_buf, size_t n) -> vcr_status {
      float *cb = c->root_cache + o;
      HIP_TRY(c, launch_copy(to_cache ? cb : ws_buf, to_cache ? ws_buf : cb, (int64_t)n, s));
      o += n;
      return VCR_OK;
    };
    vcr_status e = move(bf.c0, ld0);
    if (e == VCR_OK) e = move(bf.r0, ld0);
    for (size_t r = 0; r < g->relus.size() && e == VCR_OK; ++r) {
      const GNode &n = g->nodes[g->relus[r]];
      e = move(bf.L[r], n.numel);
      if (e == VCR_OK) e = move(bf.U[r], n.numel);
      if (e == VCR_OK) e = move(reinterpret_cast<float *>(bf.P[r]), 4 * (n.flat ? ld_of(n.numel) : n.numel));
    }
    return e;
  };
  size_t cache_floats = 2 * ld0;
  for (int r : g->relus) {
    const GNode &n = g->nodes[r];
    cache_floats += 2 * n.numel + 4 * (n.flat ? ld_of(n.numel) : n.numel);
  }
  if (use_cache) {
    st = cache_copy(false);
    if (st != VCR_OK) return st;
  } else {
    HIP_TRY(c, launch_box(x0, B, (int32_t)g->n0, ld0, eps, c->clip_on, c->clip_lo, c->clip_hi, bf.c0, bf.r0, s));
    st = run_ibp(c, g, bf, B);
    if (st != VCR_OK) return st;
  }
  HIP_TRY(c, launch_spec_cw(C, B, m, (int32_t)out.numel, out.hwc_in ? out.Wh : out.Wp, out.ld_in, out.b,
                            (int32_t)g->nodes[out.in0].numel, bf.CW, out.ld_in, bf.Cb, s));
  uint64_t flops = 0;
  int chunks = 0;
  for (const PassPlan &pp : g->passes) {
    if (use_cache && !pp.spec) continue;
    if (pp.spec && fill_cache) {
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
    if (pp.spec) {
      if (splits) {
        st = prepare_splits(c, g, bf, splits);
        if (st != VCR_OK) return st;
      }
      if (ac) {
        st = alpha_spec_graph(c, g, bf, pp, units_total, m, sh.cs, sh.D, sh.S, *ac, lb, ub, &flops, &chunks);
        if (st != VCR_OK) return st;
        continue;
      }
      for (int u0 = 0; u0 < units_total; u0 += sh.cs) {
        const int units = std::min(sh.cs, units_total - u0);
        SplitTable tab{};
        if (splits) tab = domain_table(g, bf, u0, units, m, sh.S, false);
        st = run_pass(c, g, bf, pp, u0, units, m, &flops, false, splits ? &tab : nullptr);
        if (st != VCR_OK) return st;
        ++chunks;
        HIP_TRY(c, launch_finalize_spec(bf.beta, nullptr, 0, 0, units, m, splits ? bf.flags + u0 : nullptr,
                                        lb + (int64_t)u0 * m, ub + (int64_t)u0 * m, s));
      }
      continue;
    }
    if (pp.direct) {
      const GNode &z = g->nodes[pp.start];
      const int ri = g->nodes[pp.relu].relu_index;
      const int64_t ldz = ld_of(z.numel);
      if (!z.flat)
        HIP_TRY(c, launch_conv_layer_from_ibp(bf.ic[pp.start], bf.ir[pp.start], ldz, B, z.C, z.H, z.b, bf.L[ri],
                                              bf.U[ri], bf.P[ri], c->lambda_rule, s));
      else
        HIP_TRY(c, launch_layer_from_ibp(bf.ic[pp.start], bf.ir[pp.start], ldz, (int32_t)z.numel, B, z.b, bf.L[ri],
                                         bf.U[ri], bf.P[ri], ldz, c->lambda_rule, s));
      continue;
    }
    for (int u0 = 0; u0 < B; u0 += sh.ci) {
      const int units = std::min(sh.ci, B - u0);
      st = run_pass(c, g, bf, pp, u0, units, m, &flops);
      if (st != VCR_OK) return st;
      ++chunks;
      const GNode &z = g->nodes[pp.start];
      const int ri = g->nodes[pp.relu].relu_index;
      const int64_t ldz = ld_of(z.numel);
      if (!z.flat) {
        HIP_TRY(c, launch_finalize_conv(bf.beta, units, z.C, z.H, bf.ic[pp.start] + (int64_t)u0 * ldz,
                                        bf.ir[pp.start] + (int64_t)u0 * ldz, ldz, c->intersect,
                                        z.b, bf.L[ri] + (int64_t)u0 * z.numel, bf.U[ri] + (int64_t)u0 * z.numel,
                                        bf.P[ri] + (int64_t)u0 * z.numel, c->lambda_rule, s));
      } else {
        HIP_TRY(c, launch_finalize_layer(bf.beta, nullptr, 0, 0, units, (int32_t)z.numel,
                                         bf.ic[pp.start] + (int64_t)u0 * ldz, bf.ir[pp.start] + (int64_t)u0 * ldz,
                                         ldz, c->intersect, z.b, bf.L[ri] + (int64_t)u0 * z.numel,
                                         bf.U[ri] + (int64_t)u0 * z.numel, bf.P[ri] + (int64_t)u0 * ldz, ldz,
                                         c->lambda_rule, s));
      }
    }
  }
  c->last_B = B;
  c->lastL.assign(bf.L.begin(), bf.L.end());
  c->lastU.assign(bf.U.begin(), bf.U.end());
  c->last_had_splits = splits != nullptr;
  c->flops_last = flops;
  c->chunks_last = chunks;
  return VCR_OK;
}

}  // namespace

vcr_status graph_crown(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                       const vcr_splits *splits, float *lb, float *ub) {
  return graph_run(c, x0, B, eps, C, m, lb, ub, splits, nullptr);
}

vcr_status graph_alpha(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m,
                       const vcr_alpha_opts &o, int64_t n_total, float *lb, float *ub) {
  if (!c->graph->alpha_why.empty())
    return fail(c, VCR_ERR_UNSUPPORTED, "alpha-CROWN on this network: %s", c->graph->alpha_why.c_str());
  GraphAlphaCall ac;
  ac.o = o;
  ac.n_total = n_total;
  return graph_run(c, x0, B, eps, C, m, lb, ub, nullptr, &ac);
}

vcr_status graph_beta(vcr_ctx *c, const float *x0, float eps, const float *C, int32_t m, const vcr_splits *splits,
                      const vcr_alpha_opts &o, int64_t n_total, float lr_beta, float *lb, float *ub) {
  if (!c->graph->alpha_why.empty())
    return fail(c, VCR_ERR_UNSUPPORTED, "beta-CROWN on this network: %s", c->graph->alpha_why.c_str());
  GraphAlphaCall ac;
  ac.o = o;
  ac.n_total = n_total;
  ac.lr_beta = lr_beta;
  return graph_run(c, x0, 1, eps, C, m, lb, ub, splits, &ac);
}

vcr_status graph_ibp(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C, int32_t m, float *lb,
                     float *ub) {
  GraphNet *g = c->graph;
  const int nn = (int)g->nodes.size();
  const GNode &out = g->nodes[nn - 1];
  Workspace probe;
  GBufs tmp;
  GShape sh;
  sh.B = B;
  sh.m = m;
  const size_t need = carve_graph(c, g, probe, sh, &tmp);
  HIP_TRY(c, hipSetDevice(c->device));
  c->lastL.clear();
  c->lastU.clear();
  vcr_status st = ensure_ws(c, need);
  if (st != VCR_OK) return st;
  GBufs bf;
  carve_graph(c, g, c->ws, sh, &bf);
  hipStream_t s = c->stream;
  HIP_TRY(c, launch_box(x0, B, (int32_t)g->n0, ld_of(g->n0), eps, c->clip_on, c->clip_lo, c->clip_hi, bf.c0, bf.r0, s));
  st = run_ibp(c, g, bf, B);
  if (st != VCR_OK) return st;
  const int src = out.in0;
  HIP_TRY(c, launch_spec_cw(C, B, m, (int32_t)out.numel, out.Wp, out.ld_in, out.b, (int32_t)g->nodes[src].numel,
                            bf.CW, out.ld_in, bf.Cb, s));
  HIP_TRY(c, launch_spec_direct(bf.CW, out.ld_in, bf.Cb, B, m, (int32_t)g->nodes[src].numel, bf.ic[src], bf.ir[src],
                                out.ld_in, 0, lb, ub, s));
  return VCR_OK;
}

size_t graph_workspace_bytes(vcr_ctx *c, int32_t B, int32_t m, int32_t D, int32_t S, bool alpha) {
  Workspace probe;
  GBufs tmp;
  GShape sh;
  sh.B = D > 0 ? 1 : B;
  sh.m = m;
  sh.D = D;
  sh.S = S;
  sh.ci = D > 0 ? 1 : B;
  sh.cs = D > 0 ? D : B;
  sh.alpha = alpha && c->graph->alpha_why.empty();
  return carve_graph(c, c->graph, probe, sh, &tmp);
}

}  // namespace vcr
