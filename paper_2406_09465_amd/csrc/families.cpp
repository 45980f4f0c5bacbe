// Family matching and the memory-bound families: pointwise chains, row
// programs (last-axis reductions with prologue / broadcast-back epilogue, as
// in softmax and LayerNorm fission) and single column reductions.
//
// A candidate with no linear primitive is memory-intensive and one with a
// linear primitive is compute-intensive (Korch, Section 5.2); here each class
// maps to hand-written gfx950 skeletons instead of a tuner or a vendor library.
#include <algorithm>
#include <cmath>

#include "families.h"

namespace korch {

KInfo::KInfo(const Graph& gg, const KernelDesc& kk) : g(gg), k(kk) {
  in.insert(k.prims.begin(), k.prims.end());
  ext = external_inputs(g, k);
  for (int v : k.prims) {
    Kind kd = op_kind(g.nodes[v].op);
    if (kd == Kind::Linear) linear.push_back(v);
    if (kd == Kind::Reduce) reduces.push_back(v);
    if (kd == Kind::Layout) layouts.push_back(v);
  }
}

bool KInfo::ancestor(int u, int v) const { return g.reach[u].test(v); }

void KInfo::assign_args(GenKernel& gk, std::map<int, int>& slot) const {
  for (int u : ext) {
    slot[u] = (int)gk.args.size();
    ArgRef r;
    r.kind = ArgRef::Tensor;
    r.node = u;
    gk.args.push_back(r);
  }
  for (int o : k.outs) {
    ArgRef r;
    r.kind = ArgRef::Output;
    r.node = o;
    gk.args.push_back(r);
  }
}

int KInfo::out_slot(int o) const {
  auto it = std::find(k.outs.begin(), k.outs.end(), o);
  return (int)ext.size() + (int)(it - k.outs.begin());
}

void KInfo::fill_cost(GenKernel& gk) const {
  double bytes = 0, flops = 0;
  for (int u : ext) bytes += (double)numel(g.nodes[u].shape) * dtype_bytes(g.nodes[u].dtype);
  for (int o : k.outs) bytes += (double)numel(g.nodes[o].shape) * dtype_bytes(g.nodes[o].dtype);
  for (int v : linear) {
    const Node& n = g.nodes[v];
    if (n.op == KORCH_MATMUL) {
      int64_t kdim = g.nodes[n.in[0]].shape.back();
      flops += 2.0 * (double)numel(n.shape) * (double)kdim;
    } else {
      const Shape& w = g.nodes[n.in[1]].shape;
      flops += 2.0 * (double)numel(n.shape) * (double)(w[0] * w[1] * w[2]);
    }
  }
  gk.alg_bytes = bytes;
  gk.alg_flops = flops;
}

static thread_local std::string g_kernel_prefix = "korch_k";
void set_kernel_prefix(const std::string& prefix) { g_kernel_prefix = prefix; }
// Header of a thread's loop over the reduced axis of a column reduction (rows
// l0 + ly, + LY, ... below l1).  When every split holds `chunk` rows and a
// thread's share is a few rows, the loop has a fixed trip count and is
// unrolled, so all of its loads are issued before the first is used; the
// compiler splits a runtime-bounded loop into a first load, a wait, and the rest.
static std::string row_loop(int64_t chunk, int64_t Lr, int64_t LY) {
  std::ostringstream o;
  if (Lr % chunk == 0 && chunk % LY == 0 && chunk / LY <= 8)
    o << "#pragma unroll\n  for (int it_ = 0; it_ < " << chunk / LY << "; ++it_) {\n    const i64 l = l0 + ly + (i64)it_ * " << LY
      << ";\n";
  else
    o << "#pragma unroll 4\n  for (i64 l = l0 + ly; l < l1; l += " << LY << ") {\n";
  return o.str();
}

std::string kernel_name(int index, const char* fam) { return g_kernel_prefix + std::to_string(index) + "_" + fam; }

static int64_t pow2ceil(int64_t x) {
  int64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// ---------------------------------------------------------------------------
// Pointwise family: elementwise, broadcast and layout primitives evaluated per
// output element; layout primitives become load address maps.
// ---------------------------------------------------------------------------

bool match_pointwise(const KInfo& ki, std::string* why) {
  if (!ki.linear.empty() || !ki.reduces.empty()) {
    *why = "pointwise: has linear or reduce primitives";
    return false;
  }
  // outputs must broadcast to the largest output
  const Graph& g = ki.g;
  int big = ki.k.outs[0];
  for (int o : ki.k.outs)
    if (numel(g.nodes[o].shape) > numel(g.nodes[big].shape)) big = o;
  const Shape& IT = g.nodes[big].shape;
  for (int o : ki.k.outs) {
    const Shape& s = g.nodes[o].shape;
    if (s.size() > IT.size()) {
      *why = "pointwise: output ranks differ";
      return false;
    }
    for (size_t d = 0; d < s.size(); ++d) {
      int64_t t = IT[d + IT.size() - s.size()];
      if (s[d] != t && s[d] != 1) {
        *why = "pointwise: outputs do not broadcast to one iteration space";
        return false;
      }
    }
  }
  return true;
}

GenKernel gen_pointwise(const KInfo& ki, int index) {
  const Graph& g = ki.g;
  GenKernel gk;
  gk.family = KORCH_FAM_POINTWISE;
  gk.name = kernel_name(index, "pointwise");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  int big = ki.k.outs[0];
  for (int o : ki.k.outs)
    if (numel(g.nodes[o].shape) > numel(g.nodes[big].shape)) big = o;
  Shape IT = g.nodes[big].shape;
  if (IT.empty()) IT = {1};
  int R = (int)IT.size();
  int maxb = 2;
  for (int o : ki.k.outs) maxb = std::max(maxb, dtype_bytes(g.nodes[o].dtype));
  int vec = 16 / maxb;
  while (vec > 1 && IT.back() % vec) vec /= 2;
  int64_t total = numel(IT);
  int64_t nt = total / vec;
  Emitter em(g);
  em.inset = ki.in;
  em.argslot = slot;
  em.vec = vec;
  std::vector<Ix> it(R);
  for (int d = 0; d < R; ++d)
    it[d] = d == R - 1 ? Ix::var("c" + std::to_string(d), 1, vec) : Ix::var("c" + std::to_string(d), 0, 1);
  std::ostringstream stores, decl, after;
  for (int o : ki.k.outs) {
    const Node& on = g.nodes[o];
    Shape os = on.shape;
    auto idx = broadcast_index(os, IT, it);
    std::string v = em.value(o, idx);
    std::string T = ctype(on.dtype);
    std::string P = "((" + T + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])";
    if (numel(os) == total) {
      std::string arr = "o" + std::to_string(o);
      decl << "  float " << arr << "[" << vec << "];\n";
      em.body << "    " << arr << "[e] = " << v << ";\n";
      after << "  " << out_store(g, o, P, "t * " + std::to_string(vec), vec, arr) << ";\n";
    } else {
      auto st = strides_of(os);
      Ix off = Ix::k(0);
      for (size_t d = 0; d < os.size(); ++d) off = ix_add(off, ix_mulk(idx[d], st[d], vec));
      std::string cond;
      int lead = R - (int)os.size();
      for (int d = 0; d < R; ++d) {
        bool bcast = d < lead || (os[d - lead] == 1 && IT[d] != 1);
        if (!bcast) continue;
        if (!cond.empty()) cond += " && ";
        cond += "(" + it[d].at() + " == 0)";
      }
      em.body << "    if (" << (cond.empty() ? "true" : cond) << ") " << out_store(g, o, P, off.at(), 0, v) << ";\n";
    }
  }
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << "  const i64 t = (i64)blockIdx.x * 256 + threadIdx.x;\n";
  s << "  if (t >= " << nt << "LL) return;\n";
  s << "  i64 r_ = t;\n";
  s << "  const i64 c" << R - 1 << " = (r_ % " << IT[R - 1] / vec << "LL) * " << vec << "; r_ /= " << IT[R - 1] / vec
    << "LL;\n";
  for (int d = R - 2; d >= 0; --d)
    s << "  const i64 c" << d << " = r_ % " << IT[d] << "LL; r_ /= " << IT[d] << "LL;\n";
  s << em.pre.str() << decl.str();
  s << "#pragma unroll\n  for (int e = 0; e < " << vec << "; ++e) {\n" << em.body.str() << "  }\n";
  s << after.str() << "}\n";
  gk.source = s.str();
  gk.grid[0] = (int)((nt + 255) / 256);
  ki.fill_cost(gk);
  return gk;
}

// ---------------------------------------------------------------------------
// Row family: every node is a full row tensor F = [..., L], a keepdim row
// statistic [..., 1] or a no-keepdim statistic [...]; reductions run over the
// last axis.  A group of G lanes holds one row in registers (NC chunks of VEC
// contiguous elements per lane); reductions are lane-butterflies.
// ---------------------------------------------------------------------------

enum RowCls { FULL = 0, STATK = 1, STATN = 2 };

struct RowShape {
  Shape F, FK, FN;
  int64_t L = 0, R = 0;
};

static bool row_shapes(const KInfo& ki, RowShape& rs, std::map<int, int>& cls, std::string* why) {
  const Graph& g = ki.g;
  if (ki.reduces.empty()) {
    *why = "row: no reduction";
    return false;
  }
  for (int r : ki.reduces) {
    const Node& n = g.nodes[r];
    const Shape& s = g.nodes[n.in[0]].shape;
    if (n.axis != (int)s.size() - 1) {
      *why = "row: reduction is not over the last axis";
      return false;
    }
    if (rs.F.empty())
      rs.F = s;
    else if (rs.F != s) {
      *why = "row: reductions over different shapes";
      return false;
    }
  }
  rs.L = rs.F.back();
  if (rs.L < 2) {
    *why = "row: row length < 2";
    return false;
  }
  rs.R = numel(rs.F) / rs.L;
  rs.FK = rs.F;
  rs.FK.back() = 1;
  rs.FN = Shape(rs.F.begin(), rs.F.end() - 1);
  for (int v : ki.k.prims) {
    const Node& n = g.nodes[v];
    Kind kd = op_kind(n.op);
    if (kd != Kind::Unary && kd != Kind::Binary && kd != Kind::Reduce) {
      *why = std::string("row: unsupported primitive ") + op_name(n.op);
      return false;
    }
    if (n.shape == rs.F)
      cls[v] = FULL;
    else if (n.shape == rs.FK)
      cls[v] = STATK;
    else if (n.shape == rs.FN)
      cls[v] = STATN;
    else {
      *why = "row: node shape is neither a row nor a row statistic";
      return false;
    }
    if (kd == Kind::Reduce && cls[v] == FULL) {
      *why = "row: reduce output has full shape";
      return false;
    }
  }
  // in-kernel inputs must be compatible with the consumer's class
  for (int v : ki.k.prims) {
    const Node& n = g.nodes[v];
    for (int u : n.in) {
      if (!ki.in.count(u)) continue;
      int cu = cls[u], cv = cls[v];
      if (op_kind(n.op) == Kind::Reduce) {
        if (cu != FULL) {
          *why = "row: reduce input is not a full row";
          return false;
        }
        continue;
      }
      bool ok = (cv == FULL && (cu == FULL || cu == STATK)) || (cv == STATK && cu == STATK) ||
                (cv == STATN && cu == STATN);
      if (!ok) {
        *why = "row: incompatible operand classes";
        return false;
      }
    }
  }
  return true;
}

bool match_row(const KInfo& ki, std::string* why) {
  if (!ki.linear.empty()) {
    *why = "row: has linear primitives";
    return false;
  }
  RowShape rs;
  std::map<int, int> cls;
  if (!row_shapes(ki, rs, cls, why)) return false;
  return true;
}

// Lanes per row G, elements per vector VEC, chunks per lane NC.
void choose_row_geometry(int64_t L, int elem_bytes, int& G, int& VEC, int& NC) {
  int vmax = 16 / elem_bytes;
  VEC = 1;
  G = 64;
  bool found = false;
  for (int v = vmax; v >= 1; v /= 2) {
    if (L % v) continue;
    int64_t n = L / v;
    if (n >= 64) {
      if (n % 64 == 0) {
        VEC = v;
        G = 64;
        found = true;
        break;
      }
    } else {
      VEC = v;
      G = (int)pow2ceil(n);
      found = true;
      break;
    }
  }
  if (!found) {
    for (int v = vmax; v >= 1; v /= 2)
      if (L % v == 0) {
        VEC = v;
        break;
      }
    G = 64;
  }
  NC = (int)((L / VEC + G - 1) / G);
}

GenKernel gen_row(const KInfo& ki, int index) {
  const Graph& g = ki.g;
  RowShape rs;
  std::map<int, int> cls;
  std::string why;
  if (!row_shapes(ki, rs, cls, &why)) fail(KORCH_E_UNSUPPORTED, why);
  GenKernel gk;
  gk.family = KORCH_FAM_ROW;
  gk.name = kernel_name(index, "row");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  int eb = 2;
  for (int v : ki.k.prims) eb = std::max(eb, dtype_bytes(g.nodes[v].dtype));
  for (int u : ki.ext) eb = std::max(eb, dtype_bytes(g.nodes[u].dtype));
  int G, VEC, NC;
  choose_row_geometry(rs.L, eb, G, VEC, NC);
  if (NC * VEC > 64) fail(KORCH_E_UNSUPPORTED, "row: row too long for one wavefront's registers");
  int RPB = 256 / G;
  int RD = (int)rs.F.size() - 1;  // number of row dims
  bool partial_last = (rs.L / VEC) % G != 0;
  std::vector<Ix> rowc(RD);
  for (int d = 0; d < RD; ++d) rowc[d] = Ix::var("r" + std::to_string(d));

  std::ostringstream loads, comp, stores;
  std::map<std::string, std::string> lmemo;
  int tmp = 0;
  auto chunk_guard = [&](int j) -> std::string {
    if (j == NC - 1 && partial_last) return "cb" + std::to_string(j) + " < " + std::to_string(rs.L) + "LL";
    return "";
  };
  // external tensor read in a full-row context at chunk j; returns an expression valid inside `for e`
  auto ext_full = [&](int u, int j) -> std::string {
    std::string key = std::to_string(u) + "/" + std::to_string(j);
    auto f = lmemo.find(key);
    if (f != lmemo.end()) return f->second;
    std::vector<Ix> idx = rowc;
    idx.push_back(Ix::var("cb" + std::to_string(j), 1, VEC));
    auto bi = broadcast_index(g.nodes[u].shape, rs.F, idx);
    auto st = strides_of(g.nodes[u].shape);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], VEC));
    std::string T = ctype(g.nodes[u].dtype);
    std::string P = "((const " + T + "*)a.p[" + std::to_string(slot.at(u)) + "])";
    std::string name = "x" + std::to_string(tmp++);
    std::string gd = chunk_guard(j);
    std::string res;
    if (off.affine && off.c == 0) {
      loads << "  float " << name << " = 0.0f; " << (gd.empty() ? "" : "if (" + gd + ") ") << name << " = ld1(" << P
            << " + " << off.b << ");\n";
      res = name;
    } else if (off.affine && off.c == 1 && off.al % VEC == 0) {
      loads << "  float " << name << "[" << VEC << "]; " << (gd.empty() ? "" : "if (" + gd + ") ") << "ldv<" << VEC
            << ">(" << name << ", " << P << " + " << off.b << ");\n";
      res = name + "[e]";
    } else {
      res = "ld1(" + P + " + " + off.at() + ")";
    }
    lmemo[key] = res;
    return res;
  };
  auto ext_stat = [&](int u, const Shape& ctx) -> std::string {
    std::string key = std::to_string(u) + "/s" + std::to_string(ctx.size());
    auto f = lmemo.find(key);
    if (f != lmemo.end()) return f->second;
    std::vector<Ix> idx = rowc;
    if (ctx.size() == rs.F.size()) idx.push_back(Ix::k(0));
    auto bi = broadcast_index(g.nodes[u].shape, ctx, idx);
    auto st = strides_of(g.nodes[u].shape);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], 1));
    std::string T = ctype(g.nodes[u].dtype);
    std::string name = "x" + std::to_string(tmp++);
    loads << "  const float " << name << " = ld1((const " << T << "*)a.p[" << slot.at(u) << "] + " << off.at()
          << ");\n";
    lmemo[key] = name;
    return name;
  };
  auto operand = [&](int v, int u, int j) -> std::string {
    // value of input u of node v, in v's context, at chunk j (full context) or as a statistic
    int cv = cls[v];
    if (ki.in.count(u)) {
      if (cls[u] == FULL) return "v" + std::to_string(u) + "[" + std::to_string(j) + "][e]";
      return "s" + std::to_string(u);
    }
    if (cv == FULL || op_kind(g.nodes[v].op) == Kind::Reduce) return ext_full(u, j);
    return ext_stat(u, cv == STATK ? rs.FK : rs.FN);
  };
  for (int v : ki.k.prims) {
    const Node& n = g.nodes[v];
    Kind kd = op_kind(n.op);
    std::string V = std::to_string(v);
    if (kd == Kind::Reduce) {
      bool isMax = n.op == KORCH_REDUCE_MAX;
      comp << "  float s" << V << " = " << (isMax ? "-__builtin_huge_valf()" : "0.0f") << ";\n";
      for (int j = 0; j < NC; ++j) {
        std::string gd = chunk_guard(j);
        comp << "  " << (gd.empty() ? "" : "if (" + gd + ") ") << "{\n#pragma unroll\n  for (int e = 0; e < " << VEC
             << "; ++e) s" << V << " = "
             << (isMax ? "k_max(s" + V + ", " + operand(v, n.in[0], j) + ")"
                       : "s" + V + " + " + operand(v, n.in[0], j))
             << ";\n  }\n";
      }
      comp << "  s" << V << " = " << (isMax ? "group_max<" : "group_sum<") << G << ">(s" << V << ");\n";
      if (n.op == KORCH_REDUCE_MEAN) comp << "  s" << V << " = s" << V << " / " << flit((double)rs.L) << ";\n";
      continue;
    }
    auto expr = [&](int j) {
      if (kd == Kind::Unary) return unary_expr(n.op, operand(v, n.in[0], j));
      if (n.attrs.has_scalar) return binary_expr(n.op, operand(v, n.in[0], j), flit(n.attrs.scalar));
      return binary_expr(n.op, operand(v, n.in[0], j), operand(v, n.in[1], j));
    };
    if (cls[v] == FULL) {
      comp << "  float v" << V << "[" << NC << "][" << VEC << "];\n";
      for (int j = 0; j < NC; ++j) {
        std::string gd = chunk_guard(j);
        comp << "  " << (gd.empty() ? "" : "if (" + gd + ") ") << "{\n#pragma unroll\n  for (int e = 0; e < " << VEC
             << "; ++e) v" << V << "[" << j << "][e] = " << expr(j) << ";\n  }\n";
      }
    } else {
      comp << "  const float s" << V << " = " << expr(0) << ";\n";
    }
  }
  for (int o : ki.k.outs) {
    const Node& on = g.nodes[o];
    std::string T = ctype(on.dtype);
    std::string P = "((" + T + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])";
    if (cls[o] == FULL) {
      for (int j = 0; j < NC; ++j) {
        std::string gd = chunk_guard(j);
        stores << "  if (rv" << (gd.empty() ? "" : " && " + gd) << ") "
               << out_store(g, o, P, "row * " + std::to_string(rs.L) + "LL + cb" + std::to_string(j), VEC,
                            "v" + std::to_string(o) + "[" + std::to_string(j) + "]")
               << ";\n";
      }
    } else {
      stores << "  if (rv && lane == 0) " << out_store(g, o, P, "row", 0, "s" + std::to_string(o)) << ";\n";
    }
  }
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << "  const int lane = threadIdx.x % " << G << ";\n";
  s << "  const i64 row0 = (i64)blockIdx.x * " << RPB << " + threadIdx.x / " << G << ";\n";
  s << "  const bool rv = row0 < " << rs.R << "LL;\n";
  s << "  const i64 row = rv ? row0 : " << rs.R - 1 << "LL;\n";
  s << "  i64 q_ = row;\n";
  for (int d = RD - 1; d >= 0; --d) s << "  const i64 r" << d << " = q_ % " << rs.F[d] << "LL; q_ /= " << rs.F[d] << "LL;\n";
  for (int j = 0; j < NC; ++j)
    s << "  const i64 cb" << j << " = ((i64)" << j << " * " << G << " + lane) * " << VEC << ";\n";
  s << loads.str() << comp.str() << stores.str() << "}\n";
  gk.source = s.str();
  gk.grid[0] = (int)((rs.R + RPB - 1) / RPB);
  ki.fill_cost(gk);
  return gk;
}

// ---------------------------------------------------------------------------
// Column-reduction family: one reduction over a non-last axis, viewed as
// [A, Lr, B]; lanes span B and Lr, partial results combine in LDS in a fixed
// order (deterministic).  Elementwise / layout prologue and epilogue allowed.
// ---------------------------------------------------------------------------

// Column moments: a kernel holding a mean m = mean(X) over a non-last axis, the
// centred values D = X - m (or m - X), their squares and v = mean(D^2) (the variance of a
// normalization fissioned into primitives, Section 3), with X's elementwise or
// layout prologue and an epilogue over the reduced shape.  D and D^2 stay
// inside the kernel (neither is an output nor read by another of its nodes).
struct Moments {
  int r1 = -1, r2 = -1, D = -1, D2 = -1;
};

static bool detect_moments(const KInfo& ki, Moments& mo, std::string* why) {
  const Graph& g = ki.g;
  auto no = [&](const char* m) {
    if (why) *why = std::string("colreduce moments: ") + m;
    return false;
  };
  if (!ki.linear.empty() || ki.reduces.size() != 2) return no("needs two reductions and no linear primitive");
  int a = ki.reduces[0], b = ki.reduces[1];
  if (ki.ancestor(b, a)) std::swap(a, b);
  const Node& na = g.nodes[a];
  const Node& nb = g.nodes[b];
  if (na.op != KORCH_REDUCE_MEAN || nb.op != KORCH_REDUCE_MEAN) return no("both reductions must be means");
  const int X = na.in[0];
  const Shape& S = g.nodes[X].shape;
  if (g.nodes[nb.in[0]].shape != S || na.axis != nb.axis || na.shape != nb.shape) return no("reductions differ in shape");
  if (na.axis == (int)S.size() - 1) return no("last-axis reduction belongs to the row family");
  const int D2 = nb.in[0];
  const Node& n2 = g.nodes[D2];
  int D = -1;
  if (n2.op == KORCH_SQUARE)
    D = n2.in[0];
  else if (n2.op == KORCH_MUL && n2.in.size() == 2 && n2.in[0] == n2.in[1])
    D = n2.in[0];
  else
    return no("the second mean is not over a square");
  const Node& nd = g.nodes[D];
  // X - m, or m - X (the same squares)
  if (nd.op != KORCH_SUB || nd.attrs.has_scalar || nd.in.size() != 2 ||
      !((nd.in[0] == X && nd.in[1] == a) || (nd.in[0] == a && nd.in[1] == X)))
    return no("the squared values are not X minus its mean");
  if (!ki.in.count(D) || !ki.in.count(D2)) return no("centred values computed outside the kernel");
  for (int o : ki.k.outs)
    if (o == D || o == D2) return no("centred values are an output");
  for (int c : g.consumers[D])
    if (ki.in.count(c) && c != D2) return no("centred values read by another node of the kernel");
  for (int c : g.consumers[D2])
    if (ki.in.count(c) && c != b) return no("squares read by another node of the kernel");
  for (int v : ki.k.prims) {
    if (v == a || v == b || v == D || v == D2) continue;
    const bool pro = ki.ancestor(v, a), epi = ki.ancestor(a, v) || ki.ancestor(b, v);
    if (pro && !epi) {
      if (g.nodes[v].shape != S && op_kind(g.nodes[v].op) != Kind::Layout) return no("prologue node shape differs");
      if (std::find(ki.k.outs.begin(), ki.k.outs.end(), v) != ki.k.outs.end()) return no("prologue node is an output");
    } else if (epi && !pro) {
      if (g.nodes[v].shape != na.shape) return no("epilogue node shape differs from the reduced shape");
    } else {
      return no("node unrelated to the reductions");
    }
  }
  mo.r1 = a, mo.r2 = b, mo.D = D, mo.D2 = D2;
  return true;
}

bool match_colreduce(const KInfo& ki, std::string* why) {
  const Graph& g = ki.g;
  if (ki.linear.empty() && ki.reduces.size() == 2) {
    Moments mo;
    return detect_moments(ki, mo, why);
  }
  if (!ki.linear.empty() || ki.reduces.size() != 1) {
    *why = "colreduce: needs exactly one reduction and no linear primitive";
    return false;
  }
  int r = ki.reduces[0];
  const Node& rn = g.nodes[r];
  const Shape& S = g.nodes[rn.in[0]].shape;
  if (rn.axis == (int)S.size() - 1) {
    *why = "colreduce: last-axis reduction belongs to the row family";
    return false;
  }
  for (int v : ki.k.prims) {
    if (v == r) continue;
    bool pro = ki.ancestor(v, r), epi = ki.ancestor(r, v);
    if (!pro && !epi) {
      *why = "colreduce: node unrelated to the reduction";
      return false;
    }
    if (pro && g.nodes[v].shape != S && op_kind(g.nodes[v].op) != Kind::Layout) {
      *why = "colreduce: prologue node shape differs";
      return false;
    }
    if (pro && std::find(ki.k.outs.begin(), ki.k.outs.end(), v) != ki.k.outs.end() && g.nodes[v].shape != S) {
      *why = "colreduce: a prologue output must have the reduced operand's shape";
      return false;
    }
    if (epi && g.nodes[v].shape != rn.shape) {
      *why = "colreduce: epilogue node shape differs from the reduced shape";
      return false;
    }
  }
  return true;
}

// Column reduction: the reduced operand is [A.., L (axis), B..]; out[a][b] =
// combine over l of f(x[a][l][b]).  A workgroup of 256 threads is BB lanes
// along b (VB consecutive b each, vector loads when the innermost dimension
// allows) by LY rows along l.  When the kept columns alone give few
// workgroups, l is split over SPLIT workgroups: each writes fp32 partials, and
// the last to finish (device-scope counter, one release by thread 0, reset by
// that workgroup) sums them in split order (deterministic) and runs the
// epilogue.
// Column moments in one pass over X (the kernel detect_moments accepts).  The
// geometry is the column reduction's (BB lanes along the kept columns, LY rows
// along the reduced axis, SPLIT workgroups along it).  Each thread runs
// Welford's update over its rows, keeping a count n, a mean and M2 (the sum
// of squared deviations from the running mean); triples merge with Chan,
// Golub and LeVeque's pairwise formula
//   n = na + nb,  mean = ma + (mb - ma) nb / n,  M2 = M2a + M2b + (mb - ma)^2 na nb / n,
// always with the lower lane, wave or split as a, in a fixed order (lanes by
// butterflies, then the four waves, then the splits' partials in split
// order), so results are deterministic.  The mean m and v = M2 / L are what
// the graph's two means compute (up to rounding); X is read once.
static GenKernel gen_colmoments(const KInfo& ki, int index, const Moments& mo) {
  const Graph& g = ki.g;
  GenKernel gk;
  gk.family = KORCH_FAM_COLREDUCE;
  gk.name = kernel_name(index, "colreduce");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  const Node& rn = g.nodes[mo.r1];
  const int X = rn.in[0];
  const Shape& S = g.nodes[X].shape;
  const int ax = rn.axis;
  const int R = (int)S.size();
  int64_t A = 1, B = 1, Lr = S[ax];
  for (int d = 0; d < ax; ++d) A *= S[d];
  for (int d = ax + 1; d < R; ++d) B *= S[d];
  const int64_t Bin = S[R - 1];
  const int VB = Bin % 8 == 0 ? 8 : (Bin % 4 == 0 ? 4 : (Bin % 2 == 0 ? 2 : 1));
  const int64_t BV = B / VB;
  const int BB = BV >= 64 ? 64 : (int)pow2ceil(BV);
  const int LY = 256 / BB;
  const int64_t ctiles = (BV + BB - 1) / BB;
  int64_t SPLIT = std::max<int64_t>(1, std::min<int64_t>((256 + ctiles * A - 1) / (ctiles * A), Lr / (4 * LY)));
  const int64_t chunk = (Lr + SPLIT - 1) / SPLIT;
  SPLIT = (Lr + chunk - 1) / chunk;
  std::vector<Ix> xi(S.size());
  for (int d = 0; d < ax; ++d) xi[d] = Ix::var("a" + std::to_string(d));
  xi[ax] = Ix::var("l");
  for (int d = ax + 1; d < R; ++d)
    xi[d] = d == R - 1 ? Ix::var("b" + std::to_string(d), 1, VB) : Ix::var("b" + std::to_string(d));
  Emitter pe(g);
  pe.inset = ki.in;
  pe.argslot = slot;
  pe.vec = VB;
  const std::string xv = pe.value(X, xi);
  std::vector<Ix> ri;
  for (int d = 0; d < ax; ++d) ri.push_back(xi[d]);
  if ((int)rn.shape.size() == R) ri.push_back(Ix::k(0));
  for (int d = ax + 1; d < R; ++d) ri.push_back(xi[d]);
  Emitter ee(g);
  ee.inset = ki.in;
  ee.argslot = slot;
  ee.vec = VB;
  const std::string k1 = Emitter::key(mo.r1, ri), k2 = Emitter::key(mo.r2, ri);
  ee.provide = [&](int node, const std::vector<Ix>& idx, std::string* out) {
    if (node != mo.r1 && node != mo.r2) return false;
    if (Emitter::key(node, idx) != (node == mo.r1 ? k1 : k2))
      fail(KORCH_E_UNSUPPORTED, "colreduce moments: reduction read at another index");
    *out = node == mo.r1 ? "s1_[e]" : "s2_[e]";
    return true;
  };
  for (int o : ki.k.outs) {
    const Node& on = g.nodes[o];
    auto bi = broadcast_index(on.shape, rn.shape, ri);
    std::string v = ee.value(o, bi);
    auto strd = strides_of(on.shape);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], strd[d], VB));
    ee.body << "        "
            << out_store(g, o, "((" + ctype(on.dtype) + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])", off.at(), 0, v)
            << ";\n";
  }
  int scr_slot = -1, cnt_slot = -1;
  if (SPLIT > 1) {
    ArgRef scr;
    scr.kind = ArgRef::Scratch;
    scr.bytes = (size_t)(2 * A * SPLIT * B) * 4;  // mean and M2 planes (a split's count is its row count)
    scr_slot = (int)gk.args.size();
    gk.args.push_back(scr);
    ArgRef cnt;
    cnt.kind = ArgRef::Counter;
    cnt.bytes = (size_t)(A * ctiles) * (SPLIT > 32 ? (SPLIT + 15) / 16 + 1 : 1) * 128;
    cnt_slot = (int)gk.args.size();
    gk.args.push_back(cnt);
  }
  const std::string VBs = std::to_string(VB), BBs = std::to_string(BB);
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << "  __shared__ float red[3 * 256 * " << VB << "];\n";
  if (SPLIT > 1) s << "  __shared__ int last_;\n";
  s << "  const int tid = threadIdx.x, bl = tid % " << BB << ", ly = tid / " << BB << ";\n";
  s << "  const i64 bv0 = (i64)blockIdx.x * " << BB << " + bl;\n";
  s << "  const bool bv = bv0 < " << BV << "LL;\n";
  s << "  const i64 bi = (bv ? bv0 : " << BV - 1 << "LL) * " << VB << ";\n";
  s << "  const i64 ay = blockIdx.y;\n  i64 q_ = ay;\n";
  for (int d = ax - 1; d >= 0; --d) s << "  const i64 a" << d << " = q_ % " << S[d] << "LL; q_ /= " << S[d] << "LL;\n";
  s << "  q_ = bi;\n";
  for (int d = R - 1; d > ax; --d) s << "  const i64 b" << d << " = q_ % " << S[d] << "LL; q_ /= " << S[d] << "LL;\n";
  s << "  const i64 l0 = (i64)blockIdx.z * " << chunk << ", l1 = l0 + " << chunk << " < " << Lr << "LL ? l0 + " << chunk
    << " : " << Lr << "LL;\n";
  // Welford over this thread's rows (one count for its VB columns)
  s << "  float cn_ = 0.0f, mu_[" << VB << "], m2_[" << VB << "];\n";
  s << "#pragma unroll\n  for (int e = 0; e < " << VB << "; ++e) mu_[e] = 0.0f, m2_[e] = 0.0f;\n";
  s << row_loop(chunk, Lr, LY) << pe.pre.str();
  s << "    cn_ += 1.0f;\n    const float inv_ = __builtin_amdgcn_rcpf(cn_);\n";
  s << "#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) {\n" << pe.body.str();
  s << "      const float x_ = " << xv << ";\n";
  s << "      const float d_ = x_ - mu_[e];\n      mu_[e] += d_ * inv_;\n      m2_[e] += d_ * (x_ - mu_[e]);\n    }\n  }\n";
  // merge (na, ma, qa) (the lower) with (nb, mb, qb): f = nb / n, w = na nb / n
  s << "  const int wv_ = tid >> 6, lane_ = tid & 63;\n";
  if (BB < 64) {
    s << "#pragma unroll\n  for (int m_ = " << BB << "; m_ < 64; m_ <<= 1) {\n";
    s << "    const bool lo_ = (lane_ & m_) == 0;\n";
    s << "    const float on_ = __shfl_xor(cn_, m_, 64);\n";
    s << "    const float na_ = lo_ ? cn_ : on_, nb_ = lo_ ? on_ : cn_;\n";
    s << "    const float nt_ = na_ + nb_, f_ = nt_ > 0.0f ? nb_ * __builtin_amdgcn_rcpf(nt_) : 0.0f, w_ = na_ * f_;\n";
    s << "#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) {\n";
    s << "      const float om_ = __shfl_xor(mu_[e], m_, 64), oq_ = __shfl_xor(m2_[e], m_, 64);\n";
    s << "      const float ma_ = lo_ ? mu_[e] : om_, d_ = (lo_ ? om_ : mu_[e]) - ma_;\n";
    s << "      mu_[e] = ma_ + d_ * f_;\n      m2_[e] = m2_[e] + oq_ + d_ * d_ * w_;\n    }\n";
    s << "    cn_ = nt_;\n  }\n";
  }
  // The four waves' triples through LDS; then one thread per column of the
  // tile (TC = BB * VB columns) merges them in wave order, and (with a split
  // reduced axis) stores the column's partial triple.  The column's final mean
  // and M2 end in LDS (cm_, cq_), where the threads of row 0 read them.
  const int TC = BB * VB;
  const std::string PL = std::to_string(4 * TC);  // floats per plane of the wave triples
  s << "  __shared__ float cm_[" << TC << "], cq_[" << TC << "];\n";
  s << "  if (lane_ < " << BB << ") {\n";
  s << "    red[wv_ * " << BB << " + lane_] = cn_;\n";
  s << "#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) {\n";
  s << "      red[" << PL << " + wv_ * " << TC << " + lane_ * " << VB << " + e] = mu_[e];\n";
  s << "      red[2 * " << PL << " + wv_ * " << TC << " + lane_ * " << VB << " + e] = m2_[e];\n    }\n  }\n";
  s << "  __syncthreads();\n";
  if (SPLIT > 1) s << "  float* part = (float*)a.p[" << scr_slot << "];\n";
  s << "  for (int c = tid; c < " << TC << "; c += 256) {\n";
  s << "    float n_ = red[c / " << VB << "], m_ = red[" << PL << " + c], q_ = red[2 * " << PL << " + c];\n";
  s << "#pragma unroll\n    for (int w = 1; w < 4; ++w) {\n";
  s << "      const float nb_ = red[w * " << BB << " + c / " << VB << "], nt_ = n_ + nb_;\n";
  s << "      const float f_ = nt_ > 0.0f ? nb_ * __builtin_amdgcn_rcpf(nt_) : 0.0f;\n";
  s << "      const float d_ = red[" << PL << " + w * " << TC << " + c] - m_;\n";
  s << "      q_ = q_ + red[2 * " << PL << " + w * " << TC << " + c] + d_ * d_ * (n_ * f_);\n";
  s << "      m_ = m_ + d_ * f_;\n      n_ = nt_;\n    }\n";
  if (SPLIT > 1) {
    const std::string PP = std::to_string(A * SPLIT * B);  // floats per partial plane
    s << "    const i64 gc_ = (i64)blockIdx.x * " << TC << " + c;\n";
    s << "    if (gc_ < " << B << "LL) {\n";
    s << "      const i64 o_ = (ay * " << SPLIT << " + blockIdx.z) * " << B << "LL + gc_;\n";
    s << "      coherent_store(&part[o_], m_);\n";
    s << "      coherent_store(&part[" << PP << "LL + o_], q_);\n    }\n";
  } else {
    s << "    cm_[c] = m_;\n    cq_[c] = q_;\n";
  }
  s << "  }\n";
  if (SPLIT > 1) {
    const std::string PP = std::to_string(A * SPLIT * B);
    s << "  __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are performed\n";
    s << "  __syncthreads();\n";
    s << "  const i64 tix = ay * " << ctiles << " + blockIdx.x;\n";
    s << "  if (tid == 0) {\n    int* cnt = (int*)a.p[" << cnt_slot << "];\n";
    if (SPLIT > 32) {
      const int64_t NG = (SPLIT + 15) / 16;
      s << "    const int grp_ = blockIdx.z / 16, gsz_ = " << SPLIT << " - grp_ * 16 < 16 ? " << SPLIT << " - grp_ * 16 : 16;\n";
      s << "    int* c1 = cnt + (tix * " << NG + 1 << " + 1 + grp_) * 32;\n";
      s << "    int* c2 = cnt + tix * " << (NG + 1) * 32 << ";\n";
      s << "    last_ = false;\n";
      s << "    if (__hip_atomic_fetch_add(c1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gsz_ - 1) {\n";
      s << "      __hip_atomic_store(c1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n";
      s << "      last_ = __hip_atomic_fetch_add(c2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == " << NG - 1 << ";\n";
      s << "      if (last_) __hip_atomic_store(c2, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n    }\n  }\n";
    } else {
      s << "    const int old = __hip_atomic_fetch_add(cnt + tix * 32, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n";
      s << "    last_ = (old == " << SPLIT - 1 << ");\n";
      s << "    if (last_) __hip_atomic_store(cnt + tix * 32, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n  }\n";
    }
    s << "  __syncthreads();\n  if (!last_) return;\n";
    // each thread merges one group of splits (z = g, g + G, ...) of one column
    // in split order; then one thread per column merges the groups in order
    const int G = TC <= 256 ? 256 / TC : 1;
    // batches of loads: two per split, within the 63 loads a wave may have in flight
    const int64_t NZ = (SPLIT + G - 1) / G, NBT = std::min<int64_t>(NZ, 31);
    const std::string GT = std::to_string(G * TC);
    s << "  {\n    const i64 cb = (i64)blockIdx.x * " << TC << ";\n";
    s << "    for (int c = tid % " << std::min(TC, 256) << "; c < " << TC << "; c += 256) {\n";
    s << "      const int g = " << (G > 1 ? "tid / " + std::to_string(TC) : std::string("0")) << ";\n";
    s << "      float tn_ = 0.0f, tm_ = 0.0f, tq_ = 0.0f;\n";
    s << "      if (cb + c < " << B << "LL)\n        for (int z0 = g; z0 < " << SPLIT << "; z0 += " << NBT * G << ") {\n";
    s << "          float vn_[" << NBT << "], vm_[" << NBT << "], vq_[" << NBT << "];\n";
    s << "#pragma unroll\n          for (int j = 0; j < " << NBT << "; ++j) {\n";
    s << "            const int z = z0 + j * " << G << ";\n";
    // the address is clamped to a split that exists and the value selected
    // afterwards: a guarded (atomic) load is a branch, and each join waits
    // for every load in flight
    s << "            const i64 o_ = (ay * " << SPLIT << " + (z < " << SPLIT << " ? z : " << SPLIT - 1 << ")) * " << B
      << "LL + cb + c;\n";
    // split z holds rows [z chunk, min((z + 1) chunk, L))
    s << "            vn_[j] = z < " << SPLIT << " ? (float)(" << Lr << "LL - (i64)z * " << chunk << " < " << chunk << " ? " << Lr
      << "LL - (i64)z * " << chunk << " : " << chunk << ") : 0.0f;\n";
    s << "            const float lm_ = coherent_load(&part[o_]), lq_ = coherent_load(&part[" << PP << "LL + o_]);\n";
    s << "            vm_[j] = z < " << SPLIT << " ? lm_ : 0.0f;\n";
    s << "            vq_[j] = z < " << SPLIT << " ? lq_ : 0.0f;\n";
    s << "          }\n";
    // the batch's triples merge as a pairwise tree (j with j + h, h = 1, 2, 4,
    // ...; a fixed order, log-depth dependency chains), then into the running one
    for (int64_t h = 1; h < NBT; h *= 2)
      for (int64_t j = 0; j + h < NBT; j += 2 * h) {
        const std::string a_ = std::to_string(j), b_ = std::to_string(j + h);
        s << "          {\n            const float nt_ = vn_[" << a_ << "] + vn_[" << b_ << "], f_ = nt_ > 0.0f ? vn_[" << b_
          << "] * __builtin_amdgcn_rcpf(nt_) : 0.0f, d_ = vm_[" << b_ << "] - vm_[" << a_ << "];\n";
        s << "            vq_[" << a_ << "] = vq_[" << a_ << "] + vq_[" << b_ << "] + d_ * d_ * (vn_[" << a_ << "] * f_);\n";
        s << "            vm_[" << a_ << "] = vm_[" << a_ << "] + d_ * f_;\n            vn_[" << a_ << "] = nt_;\n          }\n";
      }
    s << "          {\n            const float nt_ = tn_ + vn_[0], f_ = nt_ > 0.0f ? vn_[0] * __builtin_amdgcn_rcpf(nt_) : 0.0f, d_ = vm_[0] - tm_;\n";
    s << "            tq_ = tq_ + vq_[0] + d_ * d_ * (tn_ * f_);\n            tm_ = tm_ + d_ * f_;\n            tn_ = nt_;\n";
    s << "          }\n        }\n";
    s << "      red[g * " << TC << " + c] = tn_;\n";
    s << "      red[" << GT << " + g * " << TC << " + c] = tm_;\n";
    s << "      red[2 * " << GT << " + g * " << TC << " + c] = tq_;\n";
    s << "    }\n  }\n  __syncthreads();\n";
    s << "  for (int c = tid; c < " << TC << "; c += 256) {\n";
    s << "    float n_ = red[c], m_ = red[" << GT << " + c], q_ = red[2 * " << GT << " + c];\n";
    if (G > 1) {
      s << "#pragma unroll\n    for (int g = 1; g < " << G << "; ++g) {\n";
      s << "      const float nb_ = red[g * " << TC << " + c], nt_ = n_ + nb_, f_ = nt_ > 0.0f ? nb_ * __builtin_amdgcn_rcpf(nt_) : 0.0f;\n";
      s << "      const float d_ = red[" << GT << " + g * " << TC << " + c] - m_;\n";
      s << "      q_ = q_ + red[2 * " << GT << " + g * " << TC << " + c] + d_ * d_ * (n_ * f_);\n";
      s << "      m_ = m_ + d_ * f_;\n      n_ = nt_;\n    }\n";
    }
    s << "    cm_[c] = m_;\n    cq_[c] = q_;\n  }\n";
  }
  s << "  __syncthreads();\n";
  s << "  float s1_[" << VB << "], q1_[" << VB << "];\n";
  s << "#pragma unroll\n  for (int e = 0; e < " << VB << "; ++e) s1_[e] = cm_[bl * " << VB << " + e], q1_[e] = cq_[bl * " << VB << " + e];\n";
  s << "  if (ly == 0 && bv) {\n    float s2_[" << VB << "];\n";
  s << "#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) s2_[e] = q1_[e] / " << flit((double)Lr) << ";\n";
  s << "    const i64 l = 0; (void)l;\n" << ee.pre.str() << "#pragma unroll\n    for (int e = 0; e < " << VB
    << "; ++e) {\n" << ee.body.str() << "    }\n  }\n}\n";
  gk.source = s.str();
  gk.grid[0] = (int)ctiles;
  gk.grid[1] = (int)A;
  gk.grid[2] = (int)SPLIT;
  ki.fill_cost(gk);
  return gk;
}

GenKernel gen_colreduce(const KInfo& ki, int index) {
  const Graph& g = ki.g;
  std::string why;
  if (ki.linear.empty() && ki.reduces.size() == 2) {
    Moments mo;
    if (!detect_moments(ki, mo, &why)) fail(KORCH_E_UNSUPPORTED, why);
    return gen_colmoments(ki, index, mo);
  }
  if (!match_colreduce(ki, &why)) fail(KORCH_E_UNSUPPORTED, why);
  GenKernel gk;
  gk.family = KORCH_FAM_COLREDUCE;
  gk.name = kernel_name(index, "colreduce");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  int r = ki.reduces[0];
  const Node& rn = g.nodes[r];
  int X = rn.in[0];
  const Shape& S = g.nodes[X].shape;
  int ax = rn.axis;
  const int R = (int)S.size();
  int64_t A = 1, B = 1, Lr = S[ax];
  for (int d = 0; d < ax; ++d) A *= S[d];
  for (int d = ax + 1; d < R; ++d) B *= S[d];
  const int64_t Bin = S[R - 1];  // innermost kept dimension (ax < R - 1)
  int VB = Bin % 8 == 0 ? 8 : (Bin % 4 == 0 ? 4 : (Bin % 2 == 0 ? 2 : 1));
  const int64_t BV = B / VB;  // vector columns
  int BB = BV >= 64 ? 64 : (int)pow2ceil(BV);
  int LY = 256 / BB;
  const int64_t ctiles = (BV + BB - 1) / BB;
  // split the reduced axis so that about 256 workgroups run, each with at least
  // 8 rows per thread
  int64_t SPLIT = std::max<int64_t>(1, std::min<int64_t>((256 + ctiles * A - 1) / (ctiles * A), Lr / (4 * LY)));
  int64_t chunk = (Lr + SPLIT - 1) / SPLIT;
  SPLIT = (Lr + chunk - 1) / chunk;
  bool isMax = rn.op == KORCH_REDUCE_MAX;
  std::string ident = isMax ? "-__builtin_huge_valf()" : "0.0f";
  auto comb = [&](const std::string& x, const std::string& y) {
    return isMax ? "k_max(" + x + ", " + y + ")" : "(" + x + " + " + y + ")";
  };
  std::vector<Ix> xi(S.size());
  for (int d = 0; d < ax; ++d) xi[d] = Ix::var("a" + std::to_string(d));
  xi[ax] = Ix::var("l");
  for (int d = ax + 1; d < R; ++d)
    xi[d] = d == R - 1 ? Ix::var("b" + std::to_string(d), 1, VB) : Ix::var("b" + std::to_string(d));
  Emitter pe(g);
  pe.inset = ki.in;
  pe.argslot = slot;
  pe.vec = VB;
  std::string xv = pe.value(X, xi);
  // epilogue over the reduced shape
  std::vector<Ix> ri;
  for (int d = 0; d < ax; ++d) ri.push_back(xi[d]);
  if ((int)rn.shape.size() == R) ri.push_back(Ix::k(0));
  for (int d = ax + 1; d < R; ++d) ri.push_back(xi[d]);
  Emitter ee(g);
  ee.inset = ki.in;
  ee.argslot = slot;
  ee.vec = VB;
  std::string rkey = Emitter::key(r, ri);
  ee.provide = [&](int node, const std::vector<Ix>& idx, std::string* out) {
    if (node != r) return false;
    if (Emitter::key(node, idx) != rkey) fail(KORCH_E_UNSUPPORTED, "colreduce: reduction read at another index");
    *out = "s[e]";
    return true;
  };
  // prologue outputs (same shape as the reduced operand) are stored in the loop
  // (one vector store of the VB consecutive elements when they are contiguous)
  std::set<int> pro_out;
  std::ostringstream pdecl, pafter;
  for (int o : ki.k.outs)
    if (o != r && ki.ancestor(o, r)) {
      pro_out.insert(o);
      std::string v = pe.value(o, xi);
      auto strd = strides_of(S);
      Ix off = Ix::k(0);
      for (int d = 0; d < R; ++d) off = ix_add(off, ix_mulk(xi[d], strd[d], VB));
      const std::string T = ctype(g.nodes[o].dtype);
      if (VB > 1 && off.affine && off.c == 1 && off.al % VB == 0) {
        std::string arr = "_po" + std::to_string(o);
        pdecl << "    float " << arr << "[" << VB << "];\n";
        pe.body << "      " << arr << "[e] = " << v << ";\n";
        // prologue values (the operand's shape, e.g. centered inputs) use plain
        // stores: measured 0.4 us faster for instnorm's variance kernel than the
        // write-through policy of the other outputs
        pafter << "    if (bv) "
               << out_store(g, o, "((" + T + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])", off.b, VB, arr, true)
               << ";\n";
      } else {
        pe.body << "      if (bv) "
                << out_store(g, o, "((" + T + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])", off.at(), 0, v, true)
                << ";\n";
      }
    }
  for (int o : ki.k.outs) {
    if (pro_out.count(o)) continue;
    const Node& on = g.nodes[o];
    auto bi = broadcast_index(on.shape, rn.shape, ri);
    std::string v = ee.value(o, bi);
    auto strd = strides_of(on.shape);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], strd[d], VB));
    ee.body << "        "
            << out_store(g, o, "((" + ctype(on.dtype) + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])", off.at(), 0, v)
            << ";\n";
  }
  int scr_slot = -1, cnt_slot = -1;
  if (SPLIT > 1) {
    ArgRef scr;
    scr.kind = ArgRef::Scratch;
    scr.bytes = (size_t)(A * SPLIT * B) * 4;
    scr_slot = (int)gk.args.size();
    gk.args.push_back(scr);
    ArgRef cnt;
    cnt.kind = ArgRef::Counter;
    // one 128-byte line per counter; with more than 32 splits a tile has a
    // counter per group of 16 splits and one for the groups
    cnt.bytes = (size_t)(A * ctiles) * (SPLIT > 32 ? (SPLIT + 15) / 16 + 1 : 1) * 128;
    cnt_slot = (int)gk.args.size();
    gk.args.push_back(cnt);
  }
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << "  __shared__ float red[256 * " << VB << "];\n";
  if (SPLIT > 1) s << "  __shared__ int last_;\n";
  s << "  const int tid = threadIdx.x, bl = tid % " << BB << ", ly = tid / " << BB << ";\n";
  s << "  const i64 bv0 = (i64)blockIdx.x * " << BB << " + bl;\n";
  s << "  const bool bv = bv0 < " << BV << "LL;\n";
  s << "  const i64 bi = (bv ? bv0 : " << BV - 1 << "LL) * " << VB << ";\n";
  s << "  const i64 ay = blockIdx.y;\n  i64 q_ = ay;\n";
  for (int d = ax - 1; d >= 0; --d) s << "  const i64 a" << d << " = q_ % " << S[d] << "LL; q_ /= " << S[d] << "LL;\n";
  s << "  q_ = bi;\n";
  for (int d = R - 1; d > ax; --d) s << "  const i64 b" << d << " = q_ % " << S[d] << "LL; q_ /= " << S[d] << "LL;\n";
  s << "  const i64 l0 = (i64)blockIdx.z * " << chunk << ", l1 = l0 + " << chunk << " < " << Lr << "LL ? l0 + " << chunk
    << " : " << Lr << "LL;\n";
  s << "  float acc[" << VB << "];\n#pragma unroll\n  for (int e = 0; e < " << VB << "; ++e) acc[e] = " << ident << ";\n";
  s << row_loop(chunk, Lr, LY) << pe.pre.str() << pdecl.str()
    << "#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) {\n" << pe.body.str() << "      acc[e] = "
    << comb("acc[e]", xv) << ";\n    }\n" << pafter.str() << "  }\n";
  // combine the LY rows of this workgroup in a fixed order: first the rows of
  // each wave (lanes bl, bl + BB, ... exchanged pairwise), then the four wave
  // results through LDS; s[e] is the result for column bi + e
  s << "  const int wv_ = tid >> 6, lane_ = tid & 63;\n";
  if (BB < 64) {
    s << "#pragma unroll\n  for (int e = 0; e < " << VB << "; ++e) {\n";
    s << "#pragma unroll\n    for (int m = " << BB << "; m < 64; m <<= 1) acc[e] = " << comb("acc[e]", "__shfl_xor(acc[e], m, 64)")
      << ";\n  }\n";
  }
  s << "  if (lane_ < " << BB << ") {\n#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) red[(wv_ * " << VB << " + e) * "
    << BB << " + lane_] = acc[e];\n  }\n  __syncthreads();\n";
  s << "  float s[" << VB << "];\n";
  s << "  if (ly == 0) {\n#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) {\n      s[e] = red[e * " << BB
    << " + bl];\n#pragma unroll\n      for (int w = 1; w < 4; ++w) s[e] = "
    << comb("s[e]", "red[(w * " + std::to_string(VB) + " + e) * " + std::to_string(BB) + " + bl]") << ";\n    }\n  }\n";
  if (SPLIT > 1) {
    s << "  float* part = (float*)a.p[" << scr_slot << "];\n";
    s << "  if (ly == 0 && bv) {\n#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) coherent_store(&part[(ay * " << SPLIT
      << " + blockIdx.z) * " << B << "LL + bi + e], s[e]);\n  }\n";
    // partials stored and read at the device's point of coherence; each wave
    // waits for its stores to complete before the barrier, after which thread
    // 0 counts the workgroup in
    s << "  __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are performed\n";
    s << "  __syncthreads();\n";
    s << "  const i64 tix = ay * " << ctiles << " + blockIdx.x;\n";
    s << "  if (tid == 0) {\n    int* cnt = (int*)a.p[" << cnt_slot << "];\n";
    if (SPLIT > 32) {
      // Two-level arrival: atomics on one line are performed one after another,
      // so the splits count in per group of 16 and the last of each group counts
      // the group in; every split's partials are performed before its first
      // increment, hence before the final one is observed.
      const int64_t NG = (SPLIT + 15) / 16;
      s << "    const int grp_ = blockIdx.z / 16, gsz_ = " << SPLIT << " - grp_ * 16 < 16 ? " << SPLIT << " - grp_ * 16 : 16;\n";
      s << "    int* c1 = cnt + (tix * " << NG + 1 << " + 1 + grp_) * 32;\n";
      s << "    int* c2 = cnt + tix * " << (NG + 1) * 32 << ";\n";
      s << "    last_ = false;\n";
      s << "    if (__hip_atomic_fetch_add(c1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gsz_ - 1) {\n";
      s << "      __hip_atomic_store(c1, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n";
      s << "      last_ = __hip_atomic_fetch_add(c2, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == " << NG - 1 << ";\n";
      s << "      if (last_) __hip_atomic_store(c2, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n    }\n  }\n";
    } else {
      s << "    const int old = __hip_atomic_fetch_add(cnt + tix * 32, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n";
      s << "    last_ = (old == " << SPLIT - 1 << ");\n";
      s << "    if (last_) __hip_atomic_store(cnt + tix * 32, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n  }\n";
    }
    s << "  __syncthreads();\n  if (!last_) return;\n";
    // every thread of the last workgroup sums a group of splits for one column
    // of the tile; the groups are then combined in order (deterministic)
    const int TC = BB * VB;                   // columns of the tile
    const int G = TC <= 256 ? 256 / TC : 1;   // split groups per column
    s << "  {\n    const i64 cb = (i64)blockIdx.x * " << TC << ";\n";
    s << "    for (int c = tid % " << std::min(TC, 256) << "; c < " << TC << "; c += 256) {\n";
    s << "      const int g = " << (G > 1 ? "tid / " + std::to_string(TC) : std::string("0")) << ";\n";
    s << "      float t_ = " << ident << ";\n";
    // the loads of a batch are all issued before the first is combined (one
    // round trip to the point of coherence per batch of up to 32 splits)
    const int64_t NZ = (SPLIT + G - 1) / G, NBT = std::min<int64_t>(NZ, 32);
    s << "      if (cb + c < " << B << "LL)\n        for (int z0 = g; z0 < " << SPLIT << "; z0 += " << NBT * G << ") {\n";
    s << "          float v_[" << NBT << "];\n#pragma unroll\n          for (int j = 0; j < " << NBT << "; ++j) {\n";
    s << "            const int z = z0 + j * " << G << ";\n";
    // clamped address, value selected after the load (no branch around it)
    s << "            const float l_ = coherent_load(&part[(ay * " << SPLIT << " + (z < " << SPLIT << " ? z : " << SPLIT - 1
      << ")) * " << B << "LL + cb + c]);\n";
    s << "            v_[j] = z < " << SPLIT << " ? l_ : " << ident << ";\n          }\n";
    s << "#pragma unroll\n          for (int j = 0; j < " << NBT << "; ++j) t_ = " << comb("t_", "v_[j]") << ";\n        }\n";
    s << "      red[g * " << TC << " + c] = t_;\n    }\n  }\n  __syncthreads();\n";
    s << "  if (ly == 0 && bv) {\n#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) {\n";
    s << "      s[e] = red[bl * " << VB << " + e];\n";
    if (G > 1)
      s << "      for (int g = 1; g < " << G << "; ++g) s[e] = " << comb("s[e]", "red[g * " + std::to_string(TC) + " + bl * " +
                                                                                 std::to_string(VB) + " + e]")
        << ";\n";
    s << "    }\n  }\n";
  }
  s << "  if (ly == 0 && bv) {\n";
  if (rn.op == KORCH_REDUCE_MEAN)
    s << "#pragma unroll\n    for (int e = 0; e < " << VB << "; ++e) s[e] = s[e] / " << flit((double)Lr) << ";\n";
  s << "    const i64 l = 0; (void)l;\n" << ee.pre.str() << "#pragma unroll\n    for (int e = 0; e < " << VB
    << "; ++e) {\n" << ee.body.str() << "    }\n  }\n}\n";
  gk.source = s.str();
  gk.grid[0] = (int)ctiles;
  gk.grid[1] = (int)A;
  gk.grid[2] = (int)SPLIT;
  ki.fill_cost(gk);
  return gk;
}

// ---------------------------------------------------------------------------
// Dispatcher
// ---------------------------------------------------------------------------

// A transpose of a transpose with inverse permutations is the identity.  When
// a kernel computes both (a layout-variant pair, or any such chain) and the
// inner one is not an output, the kernel's nodes that read the outer one read
// the original tensor instead, and transposes left without a reader in the
// kernel (and not outputs) are dropped.  The families then see the kernel
// as if the pair were not there.  g2 differs from g only in those edges, so
// node ids (and the plan's storage) are unchanged.  Returns false when
// nothing collapses.
static bool collapse_identity_layouts(const Graph& g, const KernelDesc& k, Graph& g2, KernelDesc& k2) {
  std::set<int> in(k.prims.begin(), k.prims.end()), outs(k.outs.begin(), k.outs.end());
  std::map<int, int> alias;
  for (int v : k.prims) {
    const Node& n = g.nodes[v];
    if (n.op != KORCH_TRANSPOSE || outs.count(v) || !in.count(n.in[0])) continue;
    const Node& t = g.nodes[n.in[0]];
    if (t.op != KORCH_TRANSPOSE) continue;
    bool ident = true;
    for (int d = 0; d < n.attrs.rank; ++d) ident = ident && t.attrs.perm[n.attrs.perm[d]] == d;
    if (ident) alias[v] = t.in[0];
  }
  if (alias.empty()) return false;
  g2 = g;
  g2.finalized = false;
  for (int v : k.prims)
    for (int& u : g2.nodes[v].in) {
      auto f = alias.find(u);
      if (f != alias.end()) u = f->second;
    }
  g2.finalize();
  std::set<int> keep;
  for (int v : k.prims)
    if (!alias.count(v)) keep.insert(v);
  for (auto& [v, x] : alias) {
    (void)x;
    int t = g.nodes[v].in[0];
    bool read = outs.count(t) > 0;
    for (int c : g2.consumers[t]) read = read || keep.count(c);
    if (!read) keep.erase(t);
  }
  k2.prims.assign(keep.begin(), keep.end());
  k2.outs = k.outs;
  return true;
}

static int match_family_canonical(const Graph& g, const KernelDesc& k, std::string* why);

int match_family(const Graph& g, const KernelDesc& k, std::string* why) {
  Graph g2;
  KernelDesc k2;
  if (collapse_identity_layouts(g, k, g2, k2)) return match_family_canonical(g2, k2, why);
  return match_family_canonical(g, k, why);
}

static int match_family_canonical(const Graph& g, const KernelDesc& k, std::string* why) {
  std::string w;
  if (!why) why = &w;
  try {
    KInfo ki(g, k);
    // A constant tensor is evaluated inline by the pointwise emitter and by
    // product prologues; the row programs take only computed operands.
    bool has_fill = false;
    for (int v : k.prims)
      if (g.nodes[v].op == KORCH_FILL) has_fill = true;
    if (!ki.linear.empty()) {
      if (match_attention(ki, why)) return KORCH_FAM_ATTENTION;
      if (match_conv(ki, why)) return KORCH_FAM_CONV;
      if (match_splitk(ki, why)) return KORCH_FAM_SPLITK;
      if (match_gemm(ki, why)) return KORCH_FAM_GEMM;
      return KORCH_FAM_NONE;
    }
    if (!ki.reduces.empty()) {
      if (has_fill) {
        *why = "row programs do not evaluate constant tensors";
        return KORCH_FAM_NONE;
      }
      if (match_row(ki, why)) return KORCH_FAM_ROW;
      if (match_colreduce(ki, why)) return KORCH_FAM_COLREDUCE;
      return KORCH_FAM_NONE;
    }
    if (match_pointwise(ki, why)) return KORCH_FAM_POINTWISE;
  } catch (Error& e) {
    *why = e.what();
  }
  return KORCH_FAM_NONE;
}

static GenKernel generate_canonical(const Graph& g, const KernelDesc& k, int index);

GenKernel generate_kernel(const Graph& g, const KernelDesc& k, int index) {
  Graph g2;
  KernelDesc k2;
  if (collapse_identity_layouts(g, k, g2, k2)) return generate_canonical(g2, k2, index);
  return generate_canonical(g, k, index);
}

static GenKernel generate_canonical(const Graph& g, const KernelDesc& k, int index) {
  std::string why;
  int fam = match_family_canonical(g, k, &why);
  KInfo ki(g, k);
  bool half_outputs = true;
  for (int o : k.outs)
    if (g.nodes[o].dtype == KORCH_F32) half_outputs = false;
  set_fast_math(half_outputs);
  switch (fam) {
    case KORCH_FAM_POINTWISE: return gen_pointwise(ki, index);
    case KORCH_FAM_ROW: return gen_row(ki, index);
    case KORCH_FAM_COLREDUCE: return gen_colreduce(ki, index);
    case KORCH_FAM_GEMM: return gen_gemm(ki, index);
    case KORCH_FAM_CONV: return gen_gemm(ki, index);
    case KORCH_FAM_SPLITK: return gen_splitk(ki, index);
    case KORCH_FAM_ATTENTION: return gen_attention(ki, index);
  }
  fail(KORCH_E_UNSUPPORTED, "kernel " + std::to_string(index) + ": no family implements it (" + why + ")");
}

}  // namespace korch
