// Primitive-graph IR: shape inference (Korch, Section 3 primitive
// definitions), DAG finalization, reachability and convexity (Definition 1).
#include "ir.h"

#include <algorithm>
#include <set>
#include <sstream>

namespace korch {

int64_t numel(const Shape& s) {
  int64_t n = 1;
  for (auto d : s) n *= d;
  return n;
}

std::string shape_str(const Shape& s) {
  std::ostringstream o;
  o << "[";
  for (size_t i = 0; i < s.size(); ++i) o << (i ? "," : "") << s[i];
  o << "]";
  return o.str();
}

int dtype_bytes(int dtype) { return dtype == KORCH_F32 ? 4 : 2; }

const char* dtype_name(int dtype) {
  switch (dtype) {
    case KORCH_F32: return "f32";
    case KORCH_F16: return "f16";
    case KORCH_BF16: return "bf16";
  }
  return "?";
}

Kind op_kind(int op) {
  if (op == KORCH_INPUT) return Kind::Input;
  if (op >= KORCH_NEG && op <= KORCH_IDENTITY) return Kind::Unary;
  if (op >= KORCH_ADD && op <= KORCH_MIN) return Kind::Binary;
  if (op >= KORCH_REDUCE_SUM && op <= KORCH_REDUCE_MAX) return Kind::Reduce;
  if (op == KORCH_BROADCAST) return Kind::Broadcast;
  if (op >= KORCH_TRANSPOSE && op <= KORCH_FILL) return Kind::Layout;
  if (op == KORCH_MATMUL || op == KORCH_CONV2D) return Kind::Linear;
  fail(KORCH_E_ARG, "unknown op code " + std::to_string(op));
}

bool is_elementwise(int op) {
  Kind k = op_kind(op);
  return k == Kind::Unary || k == Kind::Binary;
}

const char* op_name(int op) {
  switch (op) {
    case KORCH_INPUT: return "input";
    case KORCH_NEG: return "neg";
    case KORCH_EXP: return "exp";
    case KORCH_LOG: return "log";
    case KORCH_TANH: return "tanh";
    case KORCH_SQRT: return "sqrt";
    case KORCH_RSQRT: return "rsqrt";
    case KORCH_RELU: return "relu";
    case KORCH_SQUARE: return "square";
    case KORCH_RECIP: return "recip";
    case KORCH_GELU_TANH: return "gelu_tanh";
    case KORCH_ABS: return "abs";
    case KORCH_IDENTITY: return "identity";
    case KORCH_ADD: return "add";
    case KORCH_SUB: return "sub";
    case KORCH_MUL: return "mul";
    case KORCH_DIV: return "div";
    case KORCH_MAX: return "max";
    case KORCH_MIN: return "min";
    case KORCH_REDUCE_SUM: return "reduce_sum";
    case KORCH_REDUCE_MEAN: return "reduce_mean";
    case KORCH_REDUCE_MAX: return "reduce_max";
    case KORCH_BROADCAST: return "broadcast";
    case KORCH_TRANSPOSE: return "transpose";
    case KORCH_RESHAPE: return "reshape";
    case KORCH_SLICE: return "slice";
    case KORCH_PAD: return "pad";
    case KORCH_CONCAT: return "concat";
    case KORCH_FILL: return "fill";
    case KORCH_MATMUL: return "matmul";
    case KORCH_CONV2D: return "conv2d";
  }
  return "?";
}

static Shape broadcast_shapes(const Shape& a, const Shape& b) {
  size_t r = std::max(a.size(), b.size());
  Shape out(r);
  for (size_t i = 0; i < r; ++i) {
    int64_t x = i + a.size() >= r ? a[i + a.size() - r] : 1;
    int64_t y = i + b.size() >= r ? b[i + b.size() - r] : 1;
    if (x != y && x != 1 && y != 1)
      fail(KORCH_E_SHAPE, "shapes " + shape_str(a) + " and " + shape_str(b) + " do not broadcast");
    out[i] = std::max(x, y);
  }
  return out;
}

int Graph::add_input(int dtype, const Shape& shape) {
  if (finalized) fail(KORCH_E_STATE, "graph is finalized");
  if (dtype < KORCH_F32 || dtype > KORCH_BF16) fail(KORCH_E_ARG, "bad dtype");
  if (shape.size() > KORCH_MAX_RANK) fail(KORCH_E_SHAPE, "rank exceeds 8");
  for (auto d : shape)
    if (d <= 0) fail(KORCH_E_SHAPE, "input dims must be positive");
  Node n;
  n.id = (int)nodes.size();
  n.op = KORCH_INPUT;
  n.shape = shape;
  n.dtype = dtype;
  nodes.push_back(n);
  inputs.push_back(n.id);
  return n.id;
}

int Graph::add_op(int op, const std::vector<int>& in, const korch_attrs* attrs, int dtype) {
  if (finalized) fail(KORCH_E_STATE, "graph is finalized");
  if (dtype < KORCH_F32 || dtype > KORCH_BF16) fail(KORCH_E_ARG, "bad dtype");
  Kind kind = op_kind(op);
  if (kind == Kind::Input) fail(KORCH_E_ARG, "use korch_graph_input for inputs");
  for (int i : in)
    if (i < 0 || i >= (int)nodes.size()) fail(KORCH_E_ARG, "input node id out of range");
  Node n;
  n.id = (int)nodes.size();
  n.op = op;
  n.in = in;
  n.dtype = dtype;
  if (attrs) n.attrs = *attrs;
  const korch_attrs& a = n.attrs;
  auto need = [&](size_t k) {
    if (in.size() != k) fail(KORCH_E_ARG, std::string(op_name(op)) + " takes " + std::to_string(k) + " inputs");
  };
  auto sh = [&](int k) -> const Shape& { return nodes[in[k]].shape; };
  switch (kind) {
    case Kind::Unary:
      need(1);
      n.shape = sh(0);
      break;
    case Kind::Binary:
      if (a.has_scalar) {
        need(1);
        n.shape = sh(0);
      } else {
        need(2);
        n.shape = broadcast_shapes(sh(0), sh(1));
      }
      break;
    case Kind::Reduce: {
      need(1);
      int r = (int)sh(0).size();
      if (r == 0) fail(KORCH_E_SHAPE, "reduce of a scalar");
      int ax = a.axis < 0 ? a.axis + r : a.axis;
      if (ax < 0 || ax >= r) fail(KORCH_E_SHAPE, "reduce axis out of range");
      n.axis = ax;
      n.shape = sh(0);
      if (a.keepdim)
        n.shape[ax] = 1;
      else
        n.shape.erase(n.shape.begin() + ax);
      break;
    }
    case Kind::Broadcast: {
      need(1);
      if (a.rank < 0 || a.rank > KORCH_MAX_RANK) fail(KORCH_E_SHAPE, "bad rank");
      Shape t(a.shape, a.shape + a.rank);
      Shape b = broadcast_shapes(sh(0), t);
      if (b != t) fail(KORCH_E_SHAPE, "broadcast target " + shape_str(t) + " too small for " + shape_str(sh(0)));
      n.shape = t;
      break;
    }
    case Kind::Layout: {
      if (op == KORCH_FILL) {
        need(0);
        if (a.rank < 0 || a.rank > KORCH_MAX_RANK) fail(KORCH_E_SHAPE, "bad rank");
        n.shape.assign(a.shape, a.shape + a.rank);
        for (auto d : n.shape)
          if (d <= 0) fail(KORCH_E_SHAPE, "fill dims must be positive");
        break;
      }
      if (op == KORCH_CONCAT) {
        if (in.size() < 2) fail(KORCH_E_ARG, "concat takes >= 2 inputs");
        int r = (int)sh(0).size();
        int ax = a.axis < 0 ? a.axis + r : a.axis;
        if (ax < 0 || ax >= r) fail(KORCH_E_SHAPE, "concat axis out of range");
        n.axis = ax;
        n.shape = sh(0);
        for (size_t k = 1; k < in.size(); ++k) {
          const Shape& s = sh((int)k);
          if ((int)s.size() != r) fail(KORCH_E_SHAPE, "concat ranks differ");
          for (int d = 0; d < r; ++d)
            if (d != ax && s[d] != n.shape[d]) fail(KORCH_E_SHAPE, "concat dims differ");
          n.shape[ax] += s[ax];
        }
        break;
      }
      need(1);
      const Shape& s = sh(0);
      int r = (int)s.size();
      if (op == KORCH_TRANSPOSE) {
        if (a.rank != r) fail(KORCH_E_SHAPE, "perm rank differs from input rank");
        std::vector<int> seen(r, 0);
        n.shape.resize(r);
        for (int k = 0; k < r; ++k) {
          int p = a.perm[k];
          if (p < 0 || p >= r || seen[p]++) fail(KORCH_E_SHAPE, "perm is not a permutation");
          n.shape[k] = s[p];
        }
      } else if (op == KORCH_RESHAPE) {
        if (a.rank < 0 || a.rank > KORCH_MAX_RANK) fail(KORCH_E_SHAPE, "bad rank");
        Shape t(a.shape, a.shape + a.rank);
        for (auto d : t)
          if (d <= 0) fail(KORCH_E_SHAPE, "reshape dims must be positive");
        if (numel(t) != numel(s)) fail(KORCH_E_SHAPE, "reshape changes the element count");
        n.shape = t;
      } else if (op == KORCH_SLICE) {
        if (a.rank != r) fail(KORCH_E_SHAPE, "slice rank differs");
        n.shape.resize(r);
        for (int k = 0; k < r; ++k) {
          if (a.begin[k] < 0 || a.end[k] > s[k] || a.end[k] <= a.begin[k]) fail(KORCH_E_SHAPE, "bad slice bounds");
          n.shape[k] = a.end[k] - a.begin[k];
        }
      } else if (op == KORCH_PAD) {
        if (a.rank != r) fail(KORCH_E_SHAPE, "pad rank differs");
        n.shape.resize(r);
        for (int k = 0; k < r; ++k) {
          if (a.begin[k] < 0 || a.end[k] < 0) fail(KORCH_E_SHAPE, "negative padding");
          n.shape[k] = s[k] + a.begin[k] + a.end[k];
        }
      }
      break;
    }
    case Kind::Linear: {
      need(2);
      const Shape& x = sh(0);
      const Shape& w = sh(1);
      if (op == KORCH_MATMUL) {
        if (x.size() < 2 || w.size() < 2) fail(KORCH_E_SHAPE, "matmul needs rank >= 2");
        if (x[x.size() - 1] != w[w.size() - 2]) fail(KORCH_E_SHAPE, "matmul contraction sizes differ");
        Shape bx(x.begin(), x.end() - 2), bw(w.begin(), w.end() - 2);
        n.shape = broadcast_shapes(bx, bw);
        n.shape.push_back(x[x.size() - 2]);
        n.shape.push_back(w[w.size() - 1]);
      } else {
        if (x.size() != 3 && x.size() != 4) fail(KORCH_E_SHAPE, "conv2d input must be [H,W,C] or [N,H,W,C]");
        if (w.size() != 4) fail(KORCH_E_SHAPE, "conv2d weight must be [KH,KW,Cin,Cout]");
        if (x.back() != w[2]) fail(KORCH_E_SHAPE, "conv2d channel mismatch");
        int s = a.stride > 0 ? a.stride : 1;
        n.attrs.stride = s;
        int64_t ho = (x[x.size() - 3] + 2 * a.pad - w[0]) / s + 1;
        int64_t wo = (x[x.size() - 2] + 2 * a.pad - w[1]) / s + 1;
        if (ho <= 0 || wo <= 0 || a.pad < 0) fail(KORCH_E_SHAPE, "conv2d output is empty");
        n.shape = Shape(x.begin(), x.end() - 3);
        n.shape.push_back(ho);
        n.shape.push_back(wo);
        n.shape.push_back(w[3]);
      }
      break;
    }
    default:
      fail(KORCH_E_ARG, "bad op");
  }
  if (n.shape.size() > KORCH_MAX_RANK) fail(KORCH_E_SHAPE, "rank exceeds 8");
  nodes.push_back(n);
  return n.id;
}

void Graph::add_output(int node) {
  if (finalized) fail(KORCH_E_STATE, "graph is finalized");
  if (node < 0 || node >= (int)nodes.size()) fail(KORCH_E_ARG, "output node id out of range");
  if (!is_prim(node)) fail(KORCH_E_ARG, "a graph input cannot be a graph output");
  if (std::find(outputs.begin(), outputs.end(), node) != outputs.end())
    fail(KORCH_E_ARG, "node is already an output");
  outputs.push_back(node);
}

bool Graph::is_output(int node) const { return std::find(outputs.begin(), outputs.end(), node) != outputs.end(); }

int Graph::view_root(int node) const {
  while (is_view(node)) node = nodes[node].in[0];
  return node;
}

void Graph::finalize() {
  if (finalized) return;
  if (outputs.empty()) fail(KORCH_E_ARG, "graph has no outputs");
  int n = (int)nodes.size();
  for (int v = 0; v < n; ++v)
    for (int u : nodes[v].in)
      if (u >= v) fail(KORCH_E_CYCLE, "edge does not go forward in creation order");
  consumers.assign(n, {});
  for (int v = 0; v < n; ++v)
    for (int u : nodes[v].in)
      if (std::find(consumers[u].begin(), consumers[u].end(), v) == consumers[u].end()) consumers[u].push_back(v);
  reach.assign(n, Bits(n));
  for (int u = n - 1; u >= 0; --u)
    for (int v : consumers[u]) {
      reach[u].set(v);
      reach[u].or_with(reach[v]);
    }
  finalized = true;
}

// Definition 1: no p1, p2 in P' and q outside P' with p1 ~> q ~> p2.
bool is_convex(const Graph& g, const std::vector<int>& nodes) {
  int n = (int)g.nodes.size();
  Bits in(n);
  for (int v : nodes) in.set(v);
  Bits from_set(n);  // nodes reachable from some member
  for (int v : nodes) from_set.or_with(g.reach[v]);
  for (int q = 0; q < n; ++q) {
    if (in.test(q) || !from_set.test(q)) continue;
    if (g.reach[q].any_and(in)) return false;
  }
  return true;
}

std::vector<int> external_inputs(const Graph& g, const KernelDesc& k) {
  std::set<int> in(k.prims.begin(), k.prims.end()), ext;
  for (int v : k.prims)
    for (int u : g.nodes[v].in)
      if (!in.count(u)) ext.insert(u);
  return std::vector<int>(ext.begin(), ext.end());
}

}  // namespace korch
