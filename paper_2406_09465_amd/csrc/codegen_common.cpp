// Shared code-generation machinery: affine index expressions, elementwise
// expression strings and the per-element emitter that folds broadcast and
// layout primitives (Korch, Section 3: O[x] = I[L(x)]) into load addresses.
#include <cctype>
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <numeric>

#include "codegen.h"

namespace korch {

extern const char* k_device_prelude;

static const int64_t kBigAlign = int64_t(1) << 40;

static int64_t align_of_const(int64_t v) { return v == 0 ? kBigAlign : std::llabs(v); }

Ix Ix::k(int64_t v) {
  Ix r;
  r.b = std::to_string(v);
  r.konst = true;
  r.kv = v;
  r.al = align_of_const(v);
  return r;
}

Ix Ix::var(const std::string& name, int64_t coef, int64_t align) {
  Ix r;
  r.b = name;
  r.konst = false;
  r.c = coef;
  r.al = std::max<int64_t>(1, align);
  return r;
}

std::string Ix::at(const std::string& e) const {
  if (!affine) return b;
  if (c == 0) return b;
  std::string term = c == 1 ? e : "(" + e + "*" + std::to_string(c) + ")";
  if (konst && kv == 0) return term;
  return "(" + b + " + " + term + ")";
}

static Ix nonaffine(const std::string& expr) {
  Ix r;
  r.b = expr;
  r.affine = false;
  r.konst = false;
  r.c = 0;
  r.al = 1;
  return r;
}

Ix ix_add(const Ix& a, const Ix& b) {
  if (!a.affine || !b.affine) return nonaffine("(" + a.at() + " + " + b.at() + ")");
  Ix r;
  r.c = a.c + b.c;
  if (a.konst && b.konst) {
    r.konst = true;
    r.kv = a.kv + b.kv;
    r.b = std::to_string(r.kv);
    r.al = align_of_const(r.kv);
    return r;
  }
  r.konst = false;
  if (a.konst && a.kv == 0)
    r.b = b.b;
  else if (b.konst && b.kv == 0)
    r.b = a.b;
  else
    r.b = "(" + a.b + " + " + b.b + ")";
  r.al = std::gcd(a.al, b.al);
  if (r.al == 0) r.al = 1;
  return r;
}

Ix ix_addk(const Ix& a, int64_t v) { return v == 0 ? a : ix_add(a, Ix::k(v)); }

Ix ix_mulk(const Ix& a, int64_t v, int) {
  if (v == 0) return Ix::k(0);
  if (v == 1) return a;
  if (!a.affine) return nonaffine("(" + a.b + "*" + std::to_string(v) + ")");
  Ix r = a;
  r.c = a.c * v;
  if (a.konst) {
    r.kv = a.kv * v;
    r.b = std::to_string(r.kv);
    r.al = align_of_const(r.kv);
    return r;
  }
  r.b = "(" + a.b + "*" + std::to_string(v) + ")";
  r.al = std::min<int64_t>(kBigAlign, a.al * std::llabs(v));
  return r;
}

Ix ix_divk(const Ix& a, int64_t s, int vec) {
  if (s == 1) return a;
  if (!a.affine) return nonaffine("(" + a.b + "/" + std::to_string(s) + ")");
  int64_t spread = (int64_t)(vec - 1) * a.c;  // largest lane offset
  if (a.c == 0 || spread == 0) {
    if (a.konst) {
      Ix r = Ix::k(a.kv / s);
      return r;
    }
    Ix r = Ix::var("(" + a.b + "/" + std::to_string(s) + ")", 0, a.al % s == 0 ? a.al / s : 1);
    return r;
  }
  if (a.konst) {
    if (a.kv % s + spread < s) return Ix::k(a.kv / s);
    return nonaffine("((" + a.at() + ")/" + std::to_string(s) + ")");
  }
  if (a.al % s == 0 && spread < s) return Ix::var("(" + a.b + "/" + std::to_string(s) + ")", 0, a.al / s);
  if (s % a.al == 0 && spread < a.al) return Ix::var("(" + a.b + "/" + std::to_string(s) + ")", 0, 1);
  return nonaffine("((" + a.at() + ")/" + std::to_string(s) + ")");
}

Ix ix_modk(const Ix& a, int64_t s, int vec) {
  if (s == 1) return Ix::k(0);
  if (!a.affine) return nonaffine("(" + a.b + "%" + std::to_string(s) + ")");
  int64_t spread = (int64_t)(vec - 1) * a.c;
  if (a.c == 0 || spread == 0) {
    if (a.konst) {
      Ix r = Ix::k(a.kv % s);
      r.c = a.c;
      return r;
    }
    Ix r = Ix::var("(" + a.b + "%" + std::to_string(s) + ")", a.c, std::gcd(a.al, s));
    return r;
  }
  if (a.konst) {
    if (a.kv % s + spread < s) {
      Ix r = Ix::k(a.kv % s);
      r.c = a.c;
      return r;
    }
    return nonaffine("((" + a.at() + ")%" + std::to_string(s) + ")");
  }
  if (a.al % s == 0 && spread < s) {
    Ix r = Ix::k(0);
    r.c = a.c;
    return r;
  }
  if (s % a.al == 0 && spread < a.al) return Ix::var("(" + a.b + "%" + std::to_string(s) + ")", a.c, a.al);
  return nonaffine("((" + a.at() + ")%" + std::to_string(s) + ")");
}

std::string ctype(int dtype) {
  switch (dtype) {
    case KORCH_F32: return "float";
    case KORCH_F16: return "f16";
    case KORCH_BF16: return "bf16";
  }
  return "float";
}

std::string flit(double v) {
  if (std::isinf(v)) return v > 0 ? "__builtin_huge_valf()" : "(-__builtin_huge_valf())";
  char buf[64];
  snprintf(buf, sizeof(buf), "%.9g", v);
  std::string s = buf;
  if (s.find_first_of(".eEn") == std::string::npos) s += ".0";
  return "(" + s + "f)";
}

thread_local bool g_fast_math = false;

void set_fast_math(bool on) { g_fast_math = on; }
thread_local int g_reg_relief = 0;
void set_reg_relief(int level) { g_reg_relief = level; }
int reg_relief() { return g_reg_relief; }
bool fast_math() { return g_fast_math; }

std::string unary_expr(int op, const std::string& x) {
  bool f = g_fast_math;
  switch (op) {
    case KORCH_NEG: return "(-" + x + ")";
    case KORCH_EXP: return (f ? "f_exp(" : "expf(") + x + ")";
    case KORCH_LOG: return (f ? "f_log(" : "logf(") + x + ")";
    case KORCH_TANH: return (f ? "f_tanh(" : "tanhf(") + x + ")";
    case KORCH_SQRT: return "sqrtf(" + x + ")";
    case KORCH_RSQRT: return (f ? "f_rsqrt(" : "k_rsqrt(") + x + ")";
    case KORCH_RELU: return "k_relu(" + x + ")";
    case KORCH_SQUARE: return "(" + x + "*" + x + ")";
    case KORCH_RECIP: return f ? "f_div(1.0f, " + x + ")" : "(1.0f/" + x + ")";
    case KORCH_GELU_TANH: return (f ? "f_gelu_tanh(" : "k_gelu_tanh(") + x + ")";
    case KORCH_ABS: return "fabsf(" + x + ")";
    case KORCH_IDENTITY: return x;
  }
  fail(KORCH_E_UNSUPPORTED, std::string("no unary expression for ") + op_name(op));
}

std::string binary_expr(int op, const std::string& x, const std::string& y) {
  switch (op) {
    case KORCH_ADD: return "(" + x + " + " + y + ")";
    case KORCH_SUB: return "(" + x + " - " + y + ")";
    case KORCH_MUL: return "(" + x + " * " + y + ")";
    case KORCH_DIV: return g_fast_math ? "f_div(" + x + ", " + y + ")" : "(" + x + " / " + y + ")";
    case KORCH_MAX: return "k_max(" + x + ", " + y + ")";
    case KORCH_MIN: return "k_min(" + x + ", " + y + ")";
  }
  fail(KORCH_E_UNSUPPORTED, std::string("no binary expression for ") + op_name(op));
}

std::vector<int64_t> strides_of(const Shape& s) {
  std::vector<int64_t> st(s.size(), 1);
  for (int k = (int)s.size() - 2; k >= 0; --k) st[k] = st[k + 1] * s[k + 1];
  return st;
}

std::vector<Ix> broadcast_index(const Shape& shape, const Shape& itshape, const std::vector<Ix>& it) {
  int r = (int)shape.size(), R = (int)itshape.size();
  if (r > R) fail(KORCH_E_UNSUPPORTED, "operand rank exceeds iteration rank");
  std::vector<Ix> out(r);
  for (int k = 0; k < r; ++k) {
    int j = k + R - r;
    if (shape[k] == 1 && itshape[j] != 1)
      out[k] = Ix::k(0);
    else if (shape[k] == itshape[j])
      out[k] = it[j];
    else
      fail(KORCH_E_UNSUPPORTED, "operand shape does not broadcast to iteration shape");
  }
  return out;
}

// Recognizes the fissioned Mish product  Y = B * T,  T = tanh(SP),
// SP = log(E1), E1 = E + 1, E = exp(B)  (all inside the kernel, no
// broadcasting); returns B or -1.
int mish_operand(const Graph& g, const std::set<int>& inset, int node) {
  const Node& y = g.nodes[node];
  if (y.op != KORCH_MUL || y.attrs.has_scalar || y.in.size() != 2) return -1;
  for (int side = 0; side < 2; ++side) {
    int b = y.in[side], t = y.in[1 - side];
    auto is = [&](int v, int op) { return inset.count(v) && g.nodes[v].op == op && g.nodes[v].shape == y.shape; };
    if (g.nodes[b].shape != y.shape || !is(t, KORCH_TANH)) continue;
    int sp = g.nodes[t].in[0];
    if (!is(sp, KORCH_LOG)) continue;
    int e1 = g.nodes[sp].in[0];
    if (!is(e1, KORCH_ADD) || !g.nodes[e1].attrs.has_scalar || g.nodes[e1].attrs.scalar != 1.0) continue;
    int e = g.nodes[e1].in[0];
    if (!is(e, KORCH_EXP) || g.nodes[e].in[0] != b) continue;
    return b;
  }
  return -1;
}

std::string Emitter::key(int node, const std::vector<Ix>& idx) {
  std::string k = std::to_string(node) + "@";
  for (auto& i : idx) k += i.at() + ",";
  return k;
}

// Reshape: map an output index to an input index.  Dimensions are grouped so
// that each group of output dims covers exactly a group of input dims; inside
// a group the linear offset is split with div / mod by constants.
static std::vector<Ix> reshape_index(const Shape& out, const Shape& in, const std::vector<Ix>& idx, int vec) {
  std::vector<Ix> res(in.size());
  size_t i = 0, j = 0;
  while (i < out.size() || j < in.size()) {
    // skip size-1 dims on both sides
    if (i < out.size() && out[i] == 1 && !(j < in.size() && in[j] == 1)) {
      ++i;
      continue;
    }
    if (j < in.size() && in[j] == 1 && !(i < out.size() && out[i] == 1)) {
      res[j++] = Ix::k(0);
      continue;
    }
    if (i < out.size() && j < in.size() && out[i] == 1 && in[j] == 1) {
      res[j++] = Ix::k(0);
      ++i;
      continue;
    }
    size_t i0 = i, j0 = j;
    int64_t po = out[i++], pi = in[j++];
    while (po != pi) {
      if (po < pi) {
        if (i >= out.size()) fail(KORCH_E_SHAPE, "reshape grouping failed");
        po *= out[i++];
      } else {
        if (j >= in.size()) fail(KORCH_E_SHAPE, "reshape grouping failed");
        pi *= in[j++];
      }
    }
    // linear offset inside the group
    Ix lin = Ix::k(0);
    int64_t st = 1;
    for (size_t k = i; k-- > i0;) {
      lin = ix_add(lin, ix_mulk(idx[k], st, vec));
      st *= out[k];
    }
    st = 1;
    std::vector<int64_t> ist(j - j0);
    for (size_t k = j; k-- > j0;) {
      ist[k - j0] = st;
      st *= in[k];
    }
    for (size_t k = j0; k < j; ++k) {
      Ix v = ix_divk(lin, ist[k - j0], vec);
      if (k != j0) v = ix_modk(v, in[k], vec);
      res[k] = v;
    }
  }
  return res;
}

// True if identifier `v` occurs in expression `e` as a whole word.
static bool uses_var(const std::string& e, const std::string& v) {
  auto word = [](char c) { return std::isalnum((unsigned char)c) || c == '_'; };
  for (size_t p = e.find(v); p != std::string::npos; p = e.find(v, p + 1)) {
    bool lo = p == 0 || !word(e[p - 1]);
    bool hi = p + v.size() >= e.size() || !word(e[p + v.size()]);
    if (lo && hi) return true;
  }
  return false;
}

std::string out_store(const Graph& g, int node, const std::string& P, const std::string& off, int V,
                      const std::string& src, bool plain_store) {
  const Node& n = g.nodes[node];
  static const bool plain = getenv("KORCH_OUT_PLAIN") && atoi(getenv("KORCH_OUT_PLAIN")) != 0;  // ablation switch
  const bool big = plain || plain_store || (double)numel(n.shape) * dtype_bytes(n.dtype) >= 2147483648.0;
  if (V == 0) return big ? "st1(" + P + " + " + off + ", " + src + ")" : "st1_out(" + P + ", " + off + ", " + src + ")";
  const std::string v = std::to_string(V);
  return big ? "stv<" + v + ">(" + P + " + " + off + ", " + src + ")" : "stv_out<" + v + ">(" + P + ", " + off + ", " + src + ")";
}

std::string Emitter::load(int node, const std::vector<Ix>& idx) {
  auto it = argslot.find(node);
  if (it == argslot.end()) fail(KORCH_E_UNSUPPORTED, "emitter: node " + std::to_string(node) + " is not available");
  const Node& n = g.nodes[node];
  auto st = strides_of(n.shape);
  Ix off = Ix::k(0);
  for (size_t d = 0; d < n.shape.size(); ++d) off = ix_add(off, ix_mulk(idx[d], st[d], vec));
  std::string T = ctype(n.dtype);
  std::string P = "((const " + T + "*)a.p[" + std::to_string(it->second) + "])";
  bool hoist = guard_depth == 0 && !force_gather;
  std::string gcond;  // conjunction of the enclosing lane-invariant guards
  for (const std::string& c : lane_invariant_guards) gcond += (gcond.empty() ? "" : " && ") + c;
  if (staged && hoist && gcond.empty() && off.affine && (off.c == 0 || (off.c == 1 && vec > 1 && off.al % vec == 0))) {
    bool shared = !slot_var.empty() && !uses_var(off.b, slot_var);
    std::string v = fresh(off.c == 0 ? "su" : "sx");
    std::string ty = off.c == 0 ? T : "vec_t<" + std::to_string(vec) + ", " + T + ">";
    std::string at = shared ? "[st][0]" : "[st][i]";
    stage_decl << "  " << ty << " " << v << "[" << stages << "][" << (shared ? 1 : slots) << "];\n";
    pre << "    " << (shared ? "if (i == 0) " : "") << v << at << " = ";
    if (off.c == 0) {
      ++n_uniform;
      pre << P << "[" << off.b << "];\n";
      return "tof(" + v + at + ")";
    }
    ++n_vector;
    pre << "*(const " << ty << "*)(" << P << " + " << off.b << ");\n";
    return "tof(" + v + at + "[e])";
  }
  bool invariant = hoist && gcond.empty() && off.affine && !varying.empty() &&
                   (off.c == 0 || (off.c == 1 && vec > 1 && off.al % vec == 0));
  for (const std::string& v : varying)
    if (invariant && uses_var(off.b, v)) invariant = false;
  if (invariant) {
    ++n_invariant;
    std::string v = fresh(off.c == 0 ? "iu" : "ix");
    if (off.c == 0) {
      inv << "  float " << v << " = 0.0f;\n  {\n    " << inv_defs << "\n    if (" << inv_guard << ") " << v << " = ld1(" << P
          << " + " << off.b << ");\n  }\n";
      return v;
    }
    const int vb = vec * dtype_bytes(n.dtype);
    if ((vb == 4 || vb == 8 || vb == 16) && (double)numel(n.shape) * dtype_bytes(n.dtype) < 2147483648.0)
      inv << "  float " << v << "[" << vec << "];\n  {\n    " << inv_defs << "\n    ldv_or_zero<" << vec << ">(" << v << ", " << P
          << ", " << off.b << ", " << inv_guard << ");\n  }\n";
    else
      inv << "  float " << v << "[" << vec << "] = {};\n  {\n    " << inv_defs << "\n    if (" << inv_guard << ") ldv<" << vec
          << ">(" << v << ", " << P << " + " << off.b << ");\n  }\n";
    return v + "[e]";
  }
  if (hoist && off.affine && off.c == 0) {
    ++n_uniform;
    std::string v = fresh("u");
    if (gcond.empty())
      pre << "  const float " << v << " = ld1(" << P << " + " << off.b << ");\n";
    else
      pre << "  const float " << v << " = (" << gcond << ") ? ld1(" << P << " + " << off.b << ") : 0.0f;\n";
    return v;
  }
  if (hoist && off.affine && off.c == 1 && vec > 1 && off.al % vec == 0) {
    ++n_vector;
    std::string v = fresh("x");
    if (gcond.empty())
      pre << "  float " << v << "[" << vec << "]; ldv<" << vec << ">(" << v << ", " << P << " + " << off.b << ");\n";
    else if ((vec * dtype_bytes(n.dtype) == 4 || vec * dtype_bytes(n.dtype) == 8 || vec * dtype_bytes(n.dtype) == 16) &&
             (double)numel(n.shape) * dtype_bytes(n.dtype) < 2147483648.0)
      // a branch-free load: a guarded one makes the compiler wait for every
      // load in flight where the branches join
      pre << "  float " << v << "[" << vec << "]; ldv_or_zero<" << vec << ">(" << v << ", " << P << ", " << off.b << ", " << gcond
          << ");\n";
    else
      pre << "  float " << v << "[" << vec << "] = {}; if (" << gcond << ") ldv<" << vec << ">(" << v << ", " << P << " + "
          << off.b << ");\n";
    return v + "[e]";
  }
  ++n_gather;
  std::string v = fresh("g");
  if (!gather_guard.empty()) {
    if ((double)numel(n.shape) * dtype_bytes(n.dtype) < 2147483648.0) {
      body << "    const float " << v << " = ld1_or_zero(" << P << ", " << off.at() << ", " << gather_guard << ");\n";
      return v;
    }
    ++n_guard_fallback;
  }
  body << "    const float " << v << " = ld1(" << P << " + " << off.at() << ");\n";
  return v;
}

std::string Emitter::value(int node, const std::vector<Ix>& idx) {
  std::string k = key(node, idx);
  for (auto s = memo.rbegin(); s != memo.rend(); ++s) {
    auto f = s->find(k);
    if (f != s->end()) return f->second;
  }
  std::string out;
  if (provide && provide(node, idx, &out)) {
    memo.back()[k] = out;
    return out;
  }
  if (!inset.count(node)) {
    out = load(node, idx);
    memo.back()[k] = out;
    return out;
  }
  const Node& n = g.nodes[node];
  Kind kind = op_kind(n.op);
  auto in_shape = [&](int j) -> const Shape& { return g.nodes[n.in[j]].shape; };
  switch (kind) {
    case Kind::Unary: {
      std::string x = value(n.in[0], idx);
      out = fresh("t");
      body << "    const float " << out << " = " << unary_expr(n.op, x) << ";\n";
      break;
    }
    case Kind::Binary: {
      std::string x, y;
      int mb = mish_operand(g, inset, node);
      if (mb >= 0) {
        // B * tanh(log(exp(B) + 1)) evaluated through the exact identity x n / (n + 2)
        x = value(mb, idx);
        out = fresh("t");
        body << "    const float " << out << " = " << (g_fast_math ? "f_mish(" : "k_mish(") << x << ");\n";
        break;
      }
      if (n.attrs.has_scalar) {
        x = value(n.in[0], idx);
        y = flit(n.attrs.scalar);
      } else {
        x = value(n.in[0], broadcast_index(in_shape(0), n.shape, idx));
        y = value(n.in[1], broadcast_index(in_shape(1), n.shape, idx));
      }
      out = fresh("t");
      body << "    const float " << out << " = " << binary_expr(n.op, x, y) << ";\n";
      break;
    }
    case Kind::Broadcast:
      out = value(n.in[0], broadcast_index(in_shape(0), n.shape, idx));
      break;
    case Kind::Layout: {
      if (n.op == KORCH_FILL) {
        out = flit(n.attrs.scalar);
      } else if (n.op == KORCH_TRANSPOSE) {
        std::vector<Ix> src(idx.size());
        for (size_t d = 0; d < idx.size(); ++d) src[n.attrs.perm[d]] = idx[d];
        out = value(n.in[0], src);
      } else if (n.op == KORCH_RESHAPE) {
        out = value(n.in[0], reshape_index(n.shape, in_shape(0), idx, vec));
      } else if (n.op == KORCH_SLICE) {
        std::vector<Ix> src(idx.size());
        for (size_t d = 0; d < idx.size(); ++d) src[d] = ix_addk(idx[d], n.attrs.begin[d]);
        out = value(n.in[0], src);
      } else if (n.op == KORCH_PAD) {
        const Shape& s = in_shape(0);
        std::string cond;
        std::vector<Ix> src(idx.size());
        for (size_t d = 0; d < idx.size(); ++d) {
          src[d] = ix_addk(idx[d], -n.attrs.begin[d]);
          if (n.attrs.begin[d] > 0 || n.attrs.end[d] > 0) {
            std::string ie = idx[d].at();
            if (!cond.empty()) cond += " && ";
            cond += "(" + ie + " >= " + std::to_string(n.attrs.begin[d]) + " && " + ie + " < " +
                    std::to_string(n.attrs.begin[d] + s[d]) + ")";
          }
        }
        // the condition is the same for every lane of a vector when no padded
        // dimension's index moves with the lane
        bool lane_invariant = true;
        for (size_t d = 0; d < idx.size(); ++d)
          if ((n.attrs.begin[d] > 0 || n.attrs.end[d] > 0) && (!idx[d].affine || idx[d].c != 0)) lane_invariant = false;
        if (cond.empty()) {
          out = value(n.in[0], src);
        } else {
          out = fresh("p");
          body << "    float " << out << " = " << flit(n.attrs.pad_value) << ";\n    if (" << cond << ") {\n";
          memo.emplace_back();
          if (lane_invariant)
            lane_invariant_guards.push_back("(" + cond + ")");
          else
            ++guard_depth;
          std::string x = value(n.in[0], src);
          body << "    " << out << " = " << x << ";\n    }\n";
          if (lane_invariant)
            lane_invariant_guards.pop_back();
          else
            --guard_depth;
          memo.pop_back();
        }
      } else if (n.op == KORCH_CONCAT) {
        out = fresh("c");
        body << "    float " << out << ";\n";
        int64_t start = 0;
        int ax = n.axis;
        for (size_t j = 0; j < n.in.size(); ++j) {
          const Shape& s = in_shape((int)j);
          std::vector<Ix> src = idx;
          src[ax] = ix_addk(idx[ax], -start);
          bool last = j + 1 == n.in.size();
          if (j == 0)
            body << "    if (" << idx[ax].at() << " < " << (start + s[ax]) << ") {\n";
          else if (!last)
            body << "    else if (" << idx[ax].at() << " < " << (start + s[ax]) << ") {\n";
          else
            body << "    else {\n";
          memo.emplace_back();
          ++guard_depth;
          std::string x = value(n.in[j], src);
          body << "    " << out << " = " << x << ";\n    }\n";
          --guard_depth;
          memo.pop_back();
          start += s[ax];
        }
      }
      break;
    }
    default:
      fail(KORCH_E_UNSUPPORTED, std::string("emitter cannot evaluate ") + op_name(n.op) + " per element here");
  }
  memo.back()[k] = out;
  return out;
}

std::string source_header(int nargs) {
  return "#define KORCH_NARGS " + std::to_string(nargs) + "\n" + std::string(k_device_prelude) + "\n";
}

}  // namespace korch
