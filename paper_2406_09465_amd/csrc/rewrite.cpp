// Primitive-graph transformations (Korch, Section 3: transformations on the
// primitive graph before orchestration).  Each rule preserves the value of
// every graph output in exact arithmetic (sums may be reordered):
//
//  * defer division: (E / s) . V = (E . V) / s when s is constant along the
//    contraction axis (softmax normalization applied after the product);
//  * reduction as product: a sum over the second-to-last axis of X, where the
//    graph also transposes X's last two axes into T, equals the transpose of
//    T . 1 (a ones column); a sum over the last axis of a tensor that is the
//    left operand of a product equals X . 1;
//  * product merge: A . B1 and A . B2 equal two column slices of
//    A . concat(B1, B2) (concatenation along the column axis);
//  * scale folding: a product or convolution scaled (multiplied or divided)
//    by a tensor that varies only along the output-column (output-channel)
//    axis equals the product with that scale applied to the columns of its
//    right operand (the weights), e.g. inference BatchNorm folded into a
//    convolution's weights.
//
// Layout variants (the data-layout extension of the orchestration problem,
// Section 8): every intermediate tensor that a product reads as an operand is
// followed by a pair of mutually inverse transposes of its last two axes, and
// its consumers read the second.  A plan may then materialize the tensor in
// its own layout or in the transposed one (the first transpose), and each
// consuming kernel reads whichever is available; the measured-cost chooser
// picks.  The pair is inserted once, after the other rules, and is not folded.
//
// The graph is rebuilt after every application: a recursive emitter creates
// each needed node after its operands (so the order is topological and dead
// nodes disappear), merges identical nodes, and folds trivial layout chains
// (transposes of transposes, layout of constants, concatenations of adjacent
// slices, full slices).
#include <cstring>
#include <functional>
#include <map>
#include <sstream>

#include "ir.h"

namespace korch {

namespace {

korch_attrs no_attrs() {
  korch_attrs a;
  std::memset(&a, 0, sizeof(a));
  return a;
}

korch_attrs shape_attrs(const Shape& s) {
  korch_attrs a = no_attrs();
  a.rank = (int)s.size();
  for (size_t d = 0; d < s.size(); ++d) a.shape[d] = s[d];
  return a;
}

// The bits of a double, so that two constants merge only when they are the
// same value (a decimal rendering would round them to a few digits).
uint64_t double_bits(double v) {
  uint64_t b;
  std::memcpy(&b, &v, sizeof(b));
  return b;
}

std::string attrs_key(const korch_attrs& a) {
  std::ostringstream o;
  o << a.axis << ',' << a.keepdim << ',' << a.rank << ',' << a.has_scalar << ',' << a.stride << ',' << a.pad << ','
    << double_bits(a.pad_value) << ',' << double_bits(a.scalar);
  for (int d = 0; d < a.rank && d < KORCH_MAX_RANK; ++d)
    o << ';' << a.perm[d] << ':' << a.shape[d] << ':' << a.begin[d] << ':' << a.end[d];
  return o.str();
}

struct Builder;
using Emit = std::function<int(Builder&)>;

struct CycleError {};

// Rebuilds `g` with some nodes replaced by emitters.
struct Builder {
  const Graph& g;
  std::map<int, Emit> subst;
  Graph out;
  std::vector<int> map;
  std::vector<char> state;
  std::map<std::string, int> cse;

  explicit Builder(const Graph& gg) : g(gg), map(gg.nodes.size(), -1), state(gg.nodes.size(), 0) {}

  const Shape& shape(int nid) const { return out.nodes[nid].shape; }

  // New-graph node for old node v.
  int get(int v) {
    if (state[v] == 2) return map[v];
    if (state[v] == 1) throw CycleError{};
    state[v] = 1;
    int r;
    auto it = subst.find(v);
    if (it != subst.end()) {
      r = it->second(*this);
    } else {
      const Node& n = g.nodes[v];
      std::vector<int> in;
      for (int u : n.in) in.push_back(get(u));
      r = add(n.op, in, n.attrs, n.dtype);
    }
    map[v] = r;
    state[v] = 2;
    return r;
  }

  // Adds a node to the new graph after local simplification.
  int add(int op, std::vector<int> in, korch_attrs a, int dtype) {
    if (op == KORCH_TRANSPOSE) {
      const Node& x = out.nodes[in[0]];
      bool ident = true;
      for (int d = 0; d < a.rank; ++d) ident = ident && a.perm[d] == d;
      if (ident) return in[0];
      if (x.op == KORCH_TRANSPOSE) {  // transpose of a transpose: compose
        korch_attrs c = a;
        for (int d = 0; d < a.rank; ++d) c.perm[d] = x.attrs.perm[a.perm[d]];
        return add(KORCH_TRANSPOSE, {x.in[0]}, c, dtype);
      }
      if (x.op == KORCH_FILL) {
        Shape t(a.rank);
        for (int d = 0; d < a.rank; ++d) t[d] = x.shape[a.perm[d]];
        korch_attrs f = shape_attrs(t);
        f.scalar = x.attrs.scalar;
        return add(KORCH_FILL, {}, f, dtype);
      }
    }
    if ((op == KORCH_BROADCAST || op == KORCH_SLICE || op == KORCH_RESHAPE) && out.nodes[in[0]].op == KORCH_FILL) {
      // layout of a constant is a constant of the new shape
      Graph probe;  // shape of the layout node
      const Node& x = out.nodes[in[0]];
      int p = probe.add_input(dtype, x.shape);
      int q = probe.add_op(op, {p}, &a, dtype);
      korch_attrs f = shape_attrs(probe.nodes[q].shape);
      f.scalar = x.attrs.scalar;
      return add(KORCH_FILL, {}, f, dtype);
    }
    if (op == KORCH_SLICE) {
      const Shape& s = out.nodes[in[0]].shape;
      bool full = true;
      for (int d = 0; d < a.rank; ++d) full = full && a.begin[d] == 0 && a.end[d] == s[d];
      if (full) return in[0];
    }
    if (op == KORCH_CONCAT) {
      // adjacent slices of one tensor along the concatenation axis
      int src = -1, ax = -1;
      int64_t lo = 0, hi = 0;
      bool ok = true;
      for (size_t j = 0; j < in.size() && ok; ++j) {
        const Node& x = out.nodes[in[j]];
        if (x.op != KORCH_SLICE) {
          ok = false;
          break;
        }
        const Shape& xs = out.nodes[x.in[0]].shape;
        int r = (int)xs.size();
        int cax = a.axis < 0 ? a.axis + r : a.axis;
        for (int d = 0; d < r && ok; ++d)
          if (d != cax && (x.attrs.begin[d] != 0 || x.attrs.end[d] != xs[d])) ok = false;
        if (j == 0) {
          src = x.in[0];
          ax = cax;
          lo = x.attrs.begin[cax];
          hi = x.attrs.end[cax];
        } else if (x.in[0] != src || x.attrs.begin[cax] != hi) {
          ok = false;
        } else {
          hi = x.attrs.end[cax];
        }
      }
      if (ok && src >= 0) {
        korch_attrs sl = no_attrs();
        const Shape& xs = out.nodes[src].shape;
        sl.rank = (int)xs.size();
        for (int d = 0; d < sl.rank; ++d) {
          sl.begin[d] = d == ax ? lo : 0;
          sl.end[d] = d == ax ? hi : xs[d];
        }
        return add(KORCH_SLICE, {src}, sl, dtype);
      }
    }
    std::ostringstream key;
    key << op << '|' << dtype << '|' << attrs_key(a);
    for (int u : in) key << '|' << u;
    auto f = cse.find(key.str());
    if (f != cse.end()) return f->second;
    int id = out.add_op(op, in, &a, dtype);
    cse[key.str()] = id;
    return id;
  }

  Graph build() {
    for (int i : g.inputs) {
      map[i] = out.add_input(g.nodes[i].dtype, g.nodes[i].shape);
      state[i] = 2;
    }
    for (int o : g.outputs) out.add_output(get(o));
    out.finalize();
    return std::move(out);
  }
};

int matmul(Builder& b, int x, int y, int dtype) { return b.add(KORCH_MATMUL, {x, y}, no_attrs(), dtype); }

int fill(Builder& b, const Shape& s, double v, int dtype) {
  korch_attrs a = shape_attrs(s);
  a.scalar = v;
  return b.add(KORCH_FILL, {}, a, dtype);
}

int transpose_last2(Builder& b, int x, int dtype) {
  int r = (int)b.shape(x).size();
  korch_attrs a = no_attrs();
  a.rank = r;
  for (int d = 0; d < r; ++d) a.perm[d] = d;
  std::swap(a.perm[r - 1], a.perm[r - 2]);
  return b.add(KORCH_TRANSPOSE, {x}, a, dtype);
}

int slice_last(Builder& b, int x, int64_t lo, int64_t hi, int dtype) {
  const Shape& s = b.shape(x);
  korch_attrs a = no_attrs();
  a.rank = (int)s.size();
  for (int d = 0; d < a.rank; ++d) {
    a.begin[d] = 0;
    a.end[d] = s[d];
  }
  a.begin[a.rank - 1] = lo;
  a.end[a.rank - 1] = hi;
  return b.add(KORCH_SLICE, {x}, a, dtype);
}

int reshape(Builder& b, int x, const Shape& t, int dtype) {
  if (b.shape(x) == t) return x;
  return b.add(KORCH_RESHAPE, {x}, shape_attrs(t), dtype);
}

bool swaps_last2(const Node& t) {
  int r = t.attrs.rank;
  if (t.op != KORCH_TRANSPOSE || r < 2) return false;
  for (int d = 0; d < r - 2; ++d)
    if (t.attrs.perm[d] != d) return false;
  return t.attrs.perm[r - 2] == r - 1 && t.attrs.perm[r - 1] == r - 2;
}

Shape batch_of(const Shape& s) { return Shape(s.begin(), s.end() - 2); }

// ---- rules: each returns the substitutions for one application, or none --

using Subst = std::map<int, Emit>;

std::vector<Subst> defer_div(const Graph& g) {
  std::vector<Subst> out;
  for (const Node& o : g.nodes) {
    if (o.op != KORCH_MATMUL) continue;
    const Node& p = g.nodes[o.in[0]];
    if (p.op != KORCH_DIV || p.attrs.has_scalar || p.in.size() != 2) continue;
    const Node& e = g.nodes[p.in[0]];
    const Node& s = g.nodes[p.in[1]];
    if (s.shape.empty() || s.shape.back() != 1 || e.shape.back() == 1 || s.shape.size() > p.shape.size()) continue;
    if (s.shape.size() >= 2 && s.shape[s.shape.size() - 2] != p.shape[p.shape.size() - 2] &&
        s.shape[s.shape.size() - 2] != 1)
      continue;
    int E = p.in[0], S = p.in[1], V = o.in[1], dt = o.dtype, pdt = p.dtype;
    Subst sub;
    sub[o.id] = [=](Builder& b) {
      int ev = matmul(b, b.get(E), b.get(V), dt);
      return b.add(KORCH_DIV, {ev, b.get(S)}, no_attrs(), pdt);
    };
    out.push_back(sub);
  }
  return out;
}

std::vector<Subst> reduce_as_product(const Graph& g) {
  std::vector<Subst> out;
  for (const Node& y : g.nodes) {
    if (y.op != KORCH_REDUCE_SUM) continue;
    const Node& x = g.nodes[y.in[0]];
    int r = (int)x.shape.size();
    if (r < 2) continue;
    int X = x.id, dt = y.dtype;
    Shape yshape = y.shape;
    if (y.axis == r - 2) {
      // a transpose of X's last two axes must already exist (the product merge
      // then shares it): sum_k X[.., k, j] = (T . 1)[.., j, 0]
      int T = -1;
      for (int c : g.consumers[X])
        if (swaps_last2(g.nodes[c])) T = c;
      if (T < 0) continue;
      int64_t n = x.shape[r - 2];
      Subst sub;
      sub[y.id] = [=](Builder& b) {
        int col = matmul(b, b.get(T), fill(b, {n, 1}, 1.0, dt), dt);  // [.., d, 1]
        return reshape(b, transpose_last2(b, col, dt), yshape, dt);
      };
      out.push_back(sub);
    } else if (y.axis == r - 1) {
      // X must also be the left operand of a product (the merge shares it)
      bool left = false;
      for (int c : g.consumers[X])
        if (g.nodes[c].op == KORCH_MATMUL && g.nodes[c].in[0] == X) left = true;
      if (!left) continue;
      int64_t d = x.shape[r - 1];
      Subst sub;
      sub[y.id] = [=](Builder& b) { return reshape(b, matmul(b, b.get(X), fill(b, {d, 1}, 1.0, dt), dt), yshape, dt); };
      out.push_back(sub);
    }
  }
  return out;
}

std::vector<Subst> merge_products(const Graph& g) {
  std::vector<Subst> out;
  for (const Node& m1 : g.nodes) {
    if (m1.op != KORCH_MATMUL) continue;
    for (const Node& m2 : g.nodes) {
      if (m2.op != KORCH_MATMUL || m2.id <= m1.id || m2.in[0] != m1.in[0] || m2.dtype != m1.dtype) continue;
      const Shape& b1 = g.nodes[m1.in[1]].shape;
      const Shape& b2 = g.nodes[m2.in[1]].shape;
      if (b1.size() < 2 || b2.size() < 2 || b1[b1.size() - 2] != b2[b2.size() - 2]) continue;
      if (batch_of(m1.shape) != batch_of(m2.shape)) continue;
      // the operands' batch dims broadcast to the products' batch dims
      Shape bt = batch_of(m1.shape);
      Shape t1 = bt, t2 = bt;
      t1.push_back(b1[b1.size() - 2]);
      t1.push_back(b1.back());
      t2.push_back(b2[b2.size() - 2]);
      t2.push_back(b2.back());
      int A = m1.in[0], B1 = m1.in[1], B2 = m2.in[1], dt = m1.dtype;
      int64_t n1 = b1.back(), n2 = b2.back();
      auto emit_c = std::make_shared<int>(-1);
      auto product = [=](Builder& b) {
        if (*emit_c >= 0) return *emit_c;
        int x1 = b.get(B1), x2 = b.get(B2);
        if (b.shape(x1) != t1) x1 = b.add(KORCH_BROADCAST, {x1}, shape_attrs(t1), dt);
        if (b.shape(x2) != t2) x2 = b.add(KORCH_BROADCAST, {x2}, shape_attrs(t2), dt);
        korch_attrs ca = no_attrs();
        ca.axis = -1;
        int cat = b.add(KORCH_CONCAT, {x1, x2}, ca, dt);
        *emit_c = matmul(b, b.get(A), cat, dt);
        return *emit_c;
      };
      Subst sub;
      sub[m1.id] = [=](Builder& b) { return slice_last(b, product(b), 0, n1, dt); };
      sub[m2.id] = [=](Builder& b) { return slice_last(b, product(b), n1, n1 + n2, dt); };
      out.push_back(sub);
    }
  }
  return out;
}

std::vector<Subst> fold_scale(const Graph& g) {
  std::vector<Subst> out;
  std::vector<char> is_out(g.nodes.size(), 0);
  for (int o : g.outputs) is_out[o] = 1;
  for (const Node& m : g.nodes) {
    if ((m.op != KORCH_MUL && m.op != KORCH_DIV) || m.attrs.has_scalar || m.in.size() != 2) continue;
    for (int side = 0; side < 2; ++side) {
      if (m.op == KORCH_DIV && side == 1) break;  // only (product) / scale
      const Node& lin = g.nodes[m.in[side]];
      if (lin.op != KORCH_MATMUL && lin.op != KORCH_CONV2D) continue;
      if (g.consumers[lin.id].size() != 1 || is_out[lin.id]) continue;
      const Node& sc = g.nodes[m.in[1 - side]];
      const int64_t N = lin.shape.back();
      if (sc.shape.empty() || sc.shape.back() != N || sc.shape.size() > lin.shape.size() || m.shape != lin.shape) continue;
      bool cols_only = true;
      for (size_t d = 0; d + 1 < sc.shape.size(); ++d) cols_only = cols_only && sc.shape[d] == 1;
      if (!cols_only) continue;
      const int A = lin.in[0], B = lin.in[1], S = sc.id, op = m.op, lop = lin.op, mdt = m.dtype;
      const int bdt = g.nodes[B].dtype, sdt = sc.dtype;
      const korch_attrs la = lin.attrs;
      Subst sub;
      sub[m.id] = [=](Builder& b) {
        int s1 = reshape(b, b.get(S), {N}, sdt);
        int bs = b.add(op, {b.get(B), s1}, no_attrs(), bdt);
        return b.add(lop, {b.get(A), bs}, la, mdt);
      };
      out.push_back(sub);
    }
  }
  return out;
}

// Centred values D = X - m, with m the mean of X over a non-last axis, that
// feed both a variance (mean of D^2 over the same axis) and other nodes: the
// square reads m - X instead, a node of its own (the same magnitudes, since
// rounding is symmetric, so the same squares).  D then no longer ties the
// variance chain to its other readers, so one kernel can hold the mean and
// the variance (one pass over X) and export m, from which a later kernel
// recomputes D.  Rows (a last-axis mean) are left alone: one row kernel holds
// the whole normalization (with its rows split too, the MLP block's cheapest
// plan was predicted at 58.63 us against 58.59 for the unsplit graph's).
std::vector<Subst> split_moments(const Graph& g) {
  std::vector<Subst> out;
  for (const Node& q : g.nodes) {
    int D = -1;
    if (q.op == KORCH_SQUARE)
      D = q.in[0];
    else if (q.op == KORCH_MUL && !q.attrs.has_scalar && q.in.size() == 2 && q.in[0] == q.in[1])
      D = q.in[0];
    else
      continue;
    const Node& d = g.nodes[D];
    if (d.op != KORCH_SUB || d.attrs.has_scalar || d.in.size() != 2) continue;
    const Node& m = g.nodes[d.in[1]];
    if (m.op != KORCH_REDUCE_MEAN || m.in[0] != d.in[0]) continue;
    if (m.axis == (int)g.nodes[m.in[0]].shape.size() - 1) continue;
    if (g.consumers[D].size() < 2) continue;
    bool variance = false;
    for (int c : g.consumers[q.id])
      if (g.nodes[c].op == KORCH_REDUCE_MEAN && g.nodes[c].axis == m.axis) variance = true;
    if (!variance) continue;
    const int X = d.in[0], M = m.id, qop = q.op, ddt = d.dtype, qdt = q.dtype;
    const korch_attrs da = d.attrs, qa = q.attrs;
    Subst sub;
    sub[q.id] = [=](Builder& b) {
      int dc = b.add(KORCH_SUB, {b.get(M), b.get(X)}, da, ddt);
      return qop == KORCH_SQUARE ? b.add(KORCH_SQUARE, {dc}, qa, qdt) : b.add(KORCH_MUL, {dc, dc}, qa, qdt);
    };
    out.push_back(sub);
  }
  return out;
}

// The layout-variant graph (see the header comment).  Eligible: a computed
// tensor (not a graph input or output, not a layout node or constant) of rank
// >= 2 whose last two axes both exceed 1 and that some product or convolution
// reads as an operand.
Graph layout_variants(const Graph& g, int* applied) {
  Graph out;
  std::vector<int> map(g.nodes.size(), -1);
  std::vector<char> is_out(g.nodes.size(), 0);
  for (int o : g.outputs) is_out[o] = 1;
  int n = 0;
  for (const Node& v : g.nodes) {
    if (v.op == KORCH_INPUT) {
      map[v.id] = out.add_input(v.dtype, v.shape);
      continue;
    }
    std::vector<int> in;
    for (int u : v.in) in.push_back(map[u]);
    int id = out.add_op(v.op, in, &v.attrs, v.dtype);
    map[v.id] = id;
    const int r = (int)v.shape.size();
    Kind k = op_kind(v.op);
    bool eligible = !is_out[v.id] && r >= 2 && v.shape[r - 1] > 1 && v.shape[r - 2] > 1 && k != Kind::Layout &&
                    v.op != KORCH_FILL;
    bool operand = false;
    for (int c : g.consumers[v.id])
      if (g.nodes[c].op == KORCH_MATMUL || g.nodes[c].op == KORCH_CONV2D) operand = true;
    if (!eligible || !operand) continue;
    korch_attrs t = no_attrs();
    t.rank = r;
    for (int d = 0; d < r; ++d) t.perm[d] = d;
    std::swap(t.perm[r - 1], t.perm[r - 2]);
    int vt = out.add_op(KORCH_TRANSPOSE, {id}, &t, v.dtype);
    map[v.id] = out.add_op(KORCH_TRANSPOSE, {vt}, &t, v.dtype);
    ++n;
  }
  for (int o : g.outputs) out.add_output(map[o]);
  out.finalize();
  if (applied) *applied = n;
  return out;
}

Graph replay(const Graph& g, const Subst& sub) {
  Builder b(g);
  b.subst = sub;
  return b.build();
}

}  // namespace

Graph rewrite_graph(const Graph& g0, uint32_t rules, int* applied) {
  Graph g = replay(g0, {});
  int n = 0;
  using Rule = std::vector<Subst> (*)(const Graph&);
  std::vector<Rule> active;
  if (rules & KORCH_RW_DEFER_DIV) active.push_back(defer_div);
  if (rules & KORCH_RW_REDUCE_AS_PRODUCT) active.push_back(reduce_as_product);
  if (rules & KORCH_RW_MERGE_PRODUCTS) active.push_back(merge_products);
  if (rules & KORCH_RW_FOLD_SCALE) active.push_back(fold_scale);
  if (rules & KORCH_RW_SPLIT_MOMENTS) active.push_back(split_moments);
  for (int iter = 0; iter < 256; ++iter) {
    bool changed = false;
    for (Rule r : active) {
      for (const Subst& s : r(g)) {
        try {
          g = replay(g, s);
        } catch (CycleError&) {
          continue;  // this application would create a cycle
        }
        changed = true;
        ++n;
        break;
      }
      if (changed) break;
    }
    if (!changed) break;
  }
  if (rules & KORCH_RW_LAYOUT_VARIANTS) {
    int m = 0;
    g = layout_variants(g, &m);
    n += m;
  }
  if (applied) *applied = n;
  return g;
}

}  // namespace korch
