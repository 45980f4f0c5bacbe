// Split-K contraction family: a product whose contraction is long compared
// with its output (M x N small, K large) is split over workgroups along K.
// Each workgroup writes an fp32 partial tile; the last workgroup to finish a
// tile (detected with a device-scope counter) sums the partials in a fixed
// order -- so results are deterministic -- and runs the epilogue.
//
// Besides elementwise epilogues, the epilogue may be a row program over the
// whole output row (reductions over the product's last axis, e.g. a fissioned
// LayerNorm), and the kernel may also produce "side" reductions of the left
// operand over the contraction axis (e.g. the key sums of linear attention),
// accumulated from the operand tiles as they pass through LDS.
#include <algorithm>
#include <cmath>
#include <cstdlib>

#include "gemm_common.h"

namespace korch {

static bool has(const std::vector<int>& v, int x) { return std::find(v.begin(), v.end(), x) != v.end(); }

struct SplitInfo {
  std::vector<int> side_in_a;  // for each side reduction: 1 when it reduces A directly over k
};

static bool analyze_splitk(const KInfo& ki, GemmSpec& sp, SplitInfo& si, std::string* why) {
  const Graph& g = ki.g;
  if (!analyze_gemm(ki, sp, why, true)) return false;
  if (sp.lnf) {
    *why = "splitk: a folded LayerNorm runs in the gemm family";
    return false;
  }
  if (sp.conv || sp.mms.size() != 1) {
    *why = "splitk: needs exactly one matmul";
    return false;
  }
  for (int r : sp.side) {
    const Node& rn = g.nodes[r];
    if (rn.op != KORCH_REDUCE_SUM && rn.op != KORCH_REDUCE_MEAN) {
      *why = "splitk: side reduction must be a sum or mean";
      return false;
    }
    int x = rn.in[0];
    int rx = (int)g.nodes[x].shape.size();
    bool ok = false;
    if (x == sp.A && rn.axis == rx - 1) {
      ok = true;
    } else if (ki.in.count(sp.A)) {
      const Node& an = g.nodes[sp.A];
      int ra = (int)an.shape.size();
      if (an.op == KORCH_TRANSPOSE && an.in[0] == x && rn.axis == rx - 2 && an.attrs.perm[ra - 1] == ra - 2 &&
          an.attrs.perm[ra - 2] == ra - 1) {
        ok = true;
        for (int i = 0; i < ra - 2; ++i)
          if (an.attrs.perm[i] != i) ok = false;
      }
    }
    if (!ok) {
      *why = "splitk: side reduction does not reduce the left operand over the contraction axis";
      return false;
    }
    const Shape& as = g.nodes[sp.A].shape;
    if ((int)as.size() != sp.nb + 2 || !std::equal(as.begin(), as.end() - 2, sp.OUT.begin())) {
      *why = "splitk: side reduction needs unbroadcast batch dims";
      return false;
    }
    for (int c : g.consumers[r])
      if (ki.in.count(c)) {
        *why = "splitk: side reduction feeds the kernel";
        return false;
      }
  }
  if (!sp.rowred.empty()) {
    if (sp.N > 128) {
      *why = "splitk: row epilogue wider than one tile";
      return false;
    }
    Shape FK = sp.OUT;
    FK.back() = 1;
    for (int v : sp.epi) {
      const Node& n = g.nodes[v];
      if (n.shape != sp.OUT && n.shape != FK) {
        *why = "splitk: row epilogue node is neither a row nor a row statistic";
        return false;
      }
      if (op_kind(n.op) == Kind::Reduce && (n.axis != (int)sp.OUT.size() - 1 || !n.attrs.keepdim)) {
        *why = "splitk: row epilogue reductions must be keepdim over the last axis";
        return false;
      }
    }
  }
  if (sp.N > 128) {
    *why = "splitk: output wider than one tile";
    return false;
  }
  int64_t tiles = (sp.M + 63) / 64 * sp.batch;
  bool skinny = tiles <= 64 && sp.K >= 1024;
  if (sp.side.empty() && sp.rowred.empty() && !skinny) {
    *why = "splitk: plain product without a long contraction";
    return false;
  }
  return true;
}

bool match_splitk(const KInfo& ki, std::string* why) {
  GemmSpec sp;
  SplitInfo si;
  return analyze_splitk(ki, sp, si, why);
}

// Row program over the C tile rows in LDS (full rows of N columns).
// With `pre` given and one pass over the tile's rows, the row setup and the
// epilogue's own loads are returned in *pre (the caller emits them ahead of
// the partial loads, so both go to memory together) and the rest, in a scope
// the caller opened, is returned.
static std::string row_epilogue(const KInfo& ki, const GemmSpec& sp, const std::map<int, int>& slot,
                                std::string* pre = nullptr) {
  const Graph& g = ki.g;
  int mm = sp.mms[0];
  Shape F = sp.OUT;
  Shape FK = F;
  FK.back() = 1;
  int64_t L = sp.N;
  int eb = 2;
  for (int v : sp.epi) eb = std::max(eb, dtype_bytes(g.nodes[v].dtype));
  int G, VEC, NC;
  choose_row_geometry(L, eb, G, VEC, NC);
  int RPB = 256 / G;
  int passes = (sp.BM + RPB - 1) / RPB;
  bool partial_last = (L / VEC) % G != 0;
  std::vector<Ix> rowc;
  for (int d = 0; d < sp.nb; ++d) rowc.push_back(Ix::var("z" + std::to_string(d)));
  rowc.push_back(Ix::var("mc"));
  auto cls_full = [&](int v) { return v == mm || g.nodes[v].shape == F; };
  std::ostringstream loads, comp, stores;
  std::map<std::string, std::string> lmemo;
  int tmp = 0;
  auto guard = [&](int j) -> std::string {
    if (j == NC - 1 && partial_last) return "cb" + std::to_string(j) + " < " + std::to_string(L) + "LL";
    return "";
  };
  auto ext = [&](int u, int j, bool full) -> std::string {
    std::string key = std::to_string(u) + "/" + std::to_string(j) + (full ? "f" : "s");
    auto f = lmemo.find(key);
    if (f != lmemo.end()) return f->second;
    std::vector<Ix> idx = rowc;
    idx.push_back(full ? Ix::var("cb" + std::to_string(j), 1, VEC) : Ix::k(0));
    auto bi = broadcast_index(g.nodes[u].shape, full ? F : FK, idx);
    auto st = strides_of(g.nodes[u].shape);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], VEC));
    std::string P = "((const " + ctype(g.nodes[u].dtype) + "*)a.p[" + std::to_string(slot.at(u)) + "])";
    std::string name = "_y" + std::to_string(tmp++);
    std::string gd = full ? guard(j) : "";
    std::string res;
    if (off.affine && off.c == 0) {
      loads << "    float " << name << " = 0.0f; " << (gd.empty() ? "" : "if (" + gd + ") ") << name << " = ld1(" << P
            << " + " << off.b << ");\n";
      res = name;
    } else if (off.affine && off.c == 1 && off.al % VEC == 0) {
      loads << "    float " << name << "[" << VEC << "]; " << (gd.empty() ? "" : "if (" + gd + ") ") << "ldv<" << VEC
            << ">(" << name << ", " << P << " + " << off.b << ");\n";
      res = name + "[e]";
    } else {
      res = "ld1(" + P + " + " + off.at() + ")";
    }
    lmemo[key] = res;
    return res;
  };
  auto operand = [&](int v, int u, int j) -> std::string {
    bool vfull = cls_full(v) || op_kind(g.nodes[v].op) == Kind::Reduce;
    if (u == mm) return "Cs[mlc * " + std::to_string(sp.LDC) + " + cb" + std::to_string(j) + " + e]";
    if (ki.in.count(u)) return cls_full(u) ? "v" + std::to_string(u) + "[" + std::to_string(j) + "][e]" : "s" + std::to_string(u);
    return ext(u, j, vfull);
  };
  for (int v : ki.k.prims) {
    if (!sp.epi.count(v)) continue;
    const Node& n = g.nodes[v];
    Kind kd = op_kind(n.op);
    std::string V = std::to_string(v);
    if (kd == Kind::Reduce) {
      bool isMax = n.op == KORCH_REDUCE_MAX;
      comp << "    float s" << V << " = " << (isMax ? "-__builtin_huge_valf()" : "0.0f") << ";\n";
      for (int j = 0; j < NC; ++j) {
        std::string gd = guard(j);
        comp << "    " << (gd.empty() ? "" : "if (" + gd + ") ") << "{\n#pragma unroll\n    for (int e = 0; e < " << VEC
             << "; ++e) s" << V << " = "
             << (isMax ? "k_max(s" + V + ", " + operand(v, n.in[0], j) + ")" : "s" + V + " + " + operand(v, n.in[0], j))
             << ";\n    }\n";
      }
      comp << "    s" << V << " = " << (isMax ? "group_max<" : "group_sum<") << G << ">(s" << V << ");\n";
      if (n.op == KORCH_REDUCE_MEAN) comp << "    s" << V << " = s" << V << " / " << flit((double)L) << ";\n";
      continue;
    }
    auto expr = [&](int j) {
      if (kd == Kind::Unary) return unary_expr(n.op, operand(v, n.in[0], j));
      if (n.attrs.has_scalar) return binary_expr(n.op, operand(v, n.in[0], j), flit(n.attrs.scalar));
      return binary_expr(n.op, operand(v, n.in[0], j), operand(v, n.in[1], j));
    };
    if (cls_full(v)) {
      comp << "    float v" << V << "[" << NC << "][" << VEC << "];\n";
      for (int j = 0; j < NC; ++j) {
        std::string gd = guard(j);
        comp << "    " << (gd.empty() ? "" : "if (" + gd + ") ") << "{\n#pragma unroll\n    for (int e = 0; e < " << VEC
             << "; ++e) v" << V << "[" << j << "][e] = " << expr(j) << ";\n    }\n";
      }
    } else {
      comp << "    const float s" << V << " = " << expr(0) << ";\n";
    }
  }
  for (int o : ki.k.outs) {
    if (has(sp.side, o)) continue;
    const Node& on = g.nodes[o];
    std::string P = "((" + ctype(on.dtype) + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])";
    if (o == mm || cls_full(o)) {
      for (int j = 0; j < NC; ++j) {
        std::string gd = guard(j);
        std::string src = o == mm ? "_mmv" + std::to_string(j) : "v" + std::to_string(o) + "[" + std::to_string(j) + "]";
        if (o == mm)
          stores << "    float _mmv" << j << "[" << VEC << "];\n#pragma unroll\n    for (int e = 0; e < " << VEC
                 << "; ++e) _mmv" << j << "[e] = Cs[mlc * " << sp.LDC << " + cb" << j << " + e];\n";
        stores << "    if (rv" << (gd.empty() ? "" : " && " + gd) << ") "
               << out_store(g, o, P, "row * " + std::to_string(L) + "LL + cb" + std::to_string(j), VEC, src) << ";\n";
      }
    } else {
      stores << "    if (rv && lane == 0) " << out_store(g, o, P, "row", 0, "s" + std::to_string(o)) << ";\n";
    }
  }
  std::ostringstream s;
  if (pre && passes == 1) {
    std::ostringstream h;
    h << "    const int pass = 0;\n    (void)pass;\n";
    h << "    const int lane = tid % " << G << ";\n";
    h << "    const int ml = tid / " << G << ";\n";
    h << "    const bool rv = ml < " << sp.BM << " && m0 + ml < " << sp.M << "LL;\n";
    h << "    const int mlc = rv ? ml : 0;\n";
    h << "    const i64 mc = rv ? m0 + ml : m0;\n";
    h << "    const i64 row = bz * " << sp.M << "LL + mc;\n";
    for (int j = 0; j < NC; ++j) h << "    const i64 cb" << j << " = ((i64)" << j << " * " << G << " + lane) * " << VEC << ";\n";
    *pre = h.str() + loads.str();
    s << comp.str() << stores.str();
    return s.str();
  }
  if (pre) pre->clear();
  s << "  for (int pass = 0; pass < " << passes << "; ++pass) {\n";
  s << "    const int lane = tid % " << G << ";\n";
  s << "    const int ml = pass * " << RPB << " + tid / " << G << ";\n";
  s << "    const bool rv = ml < " << sp.BM << " && m0 + ml < " << sp.M << "LL;\n";
  s << "    const int mlc = rv ? ml : 0;\n";
  s << "    const i64 mc = rv ? m0 + ml : m0;\n";
  s << "    const i64 row = bz * " << sp.M << "LL + mc;\n";
  for (int j = 0; j < NC; ++j) s << "    const i64 cb" << j << " = ((i64)" << j << " * " << G << " + lane) * " << VEC << ";\n";
  s << loads.str() << comp.str() << stores.str() << "  }\n";
  return s.str();
}

GenKernel gen_splitk(const KInfo& ki, int index) {
  const Graph& g = ki.g;
  GemmSpec sp;
  SplitInfo si;
  std::string why;
  if (!analyze_splitk(ki, sp, si, &why)) fail(KORCH_E_UNSUPPORTED, why);
  choose_tiles(sp, true);
  plan_operands(ki, sp);
  GenKernel gk;
  gk.family = KORCH_FAM_SPLITK;
  gk.name = kernel_name(index, "splitk");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  int64_t mtiles = (sp.M + sp.BM - 1) / sp.BM;
  int64_t KT = (sp.K + sp.BK - 1) / sp.BK;
  int64_t base = mtiles * sp.batch;
  // About KORCH_SPLITK_WGS workgroups in total (default 256, one per compute
  // unit) and at most 16 splits per output tile, so that the last workgroup of
  // a tile sums few partial tiles.  A split count that divides the tile count
  // is preferred (every split then runs the same unrolled loop); each split
  // keeps up to four k-tiles of loads in flight.
  int64_t target = 256;
  if (const char* e = getenv("KORCH_SPLITK_WGS")) target = std::max(1, atoi(e));
  int64_t S = std::max<int64_t>(1, std::min<int64_t>({(target + base - 1) / base, 16, KT}));
  for (int64_t d = S; d >= std::max<int64_t>(1, S / 2); --d)
    if (KT % d == 0) {
      S = d;
      break;
    }
  int64_t ktper = (KT + S - 1) / S;
  S = (KT + ktper - 1) / ktper;
  const bool exact = KT % ktper == 0;
  sp.NS = (int)std::max<int64_t>(2, std::min<int64_t>(4, ktper));
  int64_t tile = (int64_t)sp.BM * sp.BN;
  int nside = (int)sp.side.size();
  // scratch: partial tiles, then side partials; counters: one per output tile
  ArgRef scr;
  scr.kind = ArgRef::Scratch;
  scr.bytes = (size_t)(base * S * tile + base * S * sp.BM * std::max(1, nside)) * 4;
  int scr_slot = (int)gk.args.size();
  gk.args.push_back(scr);
  ArgRef cnt;
  cnt.kind = ArgRef::Counter;
  // Each tile's arrival counter sits on a 128-byte line of its own: device-scope
  // atomics on one line are performed one after another at the point of
  // coherence, and counters packed four bytes apart put every workgroup of the
  // kernel in one queue.
  cnt.bytes = (size_t)base * 128;
  int cnt_slot = (int)gk.args.size();
  gk.args.push_back(cnt);
  std::string T = ctype(sp.mtype);
  std::ostringstream hook;
  // Side sums: every thread adds a fixed segment of one row of each staged A
  // tile (rows over tid % BM, segments over tid / BM); the segments of a row
  // are combined in segment order once the loop is done.
  const int NSEG = sp.BM <= 256 && 256 % sp.BM == 0 && sp.BK % (256 / sp.BM) == 0 ? 256 / sp.BM : 1;
  const int KPS = sp.BK / NSEG;
  if (nside) {
    hook << "      if (tid < " << sp.BM * NSEG << ") {\n        float t_ = 0.0f;\n";
    hook << "        const " << ctype(sp.mtype) << "* Ar = Ab + (tid % " << sp.BM << ") * " << sp.BKP << " + (tid / " << sp.BM
         << ") * " << KPS << ";\n";
    hook << "#pragma unroll\n        for (int k = 0; k < " << KPS << "; ++k) t_ += tof(Ar[k]);\n";
    hook << "        side_acc += t_;\n      }\n";
  }
  size_t smem = gemm_smem_bytes(sp);
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << gemm_prologue_common(sp);
  s << "  __shared__ float side_s[" << sp.BM << "];\n  __shared__ int last_;\n";
  s << "  const int split = blockIdx.x;\n  const i64 mt = blockIdx.y, bz = blockIdx.z;\n";
  s << "  const i64 m0 = mt * " << sp.BM << ", n0 = 0;\n";
  s << "  i64 q_ = bz;\n";
  for (int d = sp.nb - 1; d >= 0; --d) s << "  const i64 z" << d << " = q_ % " << sp.OUT[d] << "LL; q_ /= " << sp.OUT[d] << "LL;\n";
  s << "  const int kt0 = split * " << ktper << ", kt1 = kt0 + " << ktper << " < " << KT << " ? kt0 + " << ktper << " : " << KT << ";\n";
  s << "  float side_acc = 0.0f;\n";
  s << operand_loader(ki, sp, true, slot);
  s << operand_loader(ki, sp, false, slot);
  s << mfma_mainloop(sp, hook.str(), ktper <= 128 ? ktper : 0, exact);
  if (nside && NSEG > 1) {
    s << "  __shared__ float side_r[" << sp.BM * NSEG << "];\n";
    s << "  side_r[tid] = side_acc;\n  __syncthreads();\n";
    s << "  if (tid < " << sp.BM << ") {\n#pragma unroll\n    for (int g_ = 1; g_ < " << NSEG << "; ++g_) side_acc += side_r[g_ * "
      << sp.BM << " + tid];\n  }\n";
  }
  // partial tile -> scratch
  s << "  const i64 tix = bz * " << mtiles << " + mt;\n";
  s << "  float* part = (float*)a.p[" << scr_slot << "];\n";
  s << "  float* sidep = part + " << base * S * tile << "LL;\n";
  // partial tiles move as float4 when rows of the C tile are 16-byte aligned
  // and the tile partials fit a buffer resource's 32-bit offsets
  const bool vec4 = tile % 4 == 0 && sp.BN % 4 == 0 && sp.LDC % 4 == 0 && base * S * tile * 4 < (int64_t(1) << 31);
  if (vec4) {
    s << "  const __amdgpu_buffer_rsrc_t rsP = __builtin_amdgcn_make_buffer_rsrc(part, 0, " << base * S * tile * 4
      << ", 0x00020000);\n";
    s << "#pragma unroll\n  for (int i = tid * 4; i < " << tile << "; i += 1024) coherent_store4(rsP, (unsigned)(((tix * " << S
      << " + split) * " << tile << "LL + i) * 4), *(const float4*)&Cs[(i / " << sp.BN << ") * " << sp.LDC << " + i % " << sp.BN
      << "]);\n";
  } else {
    s << "  for (int i = tid; i < " << tile << "; i += 256) coherent_store(&part[(tix * " << S << " + split) * " << tile
      << "LL + i], Cs[(i / " << sp.BN << ") * " << sp.LDC << " + i % " << sp.BN << "]);\n";
  }
  if (nside)
    s << "  if (tid < " << sp.BM << ") coherent_store(&sidep[(tix * " << S << " + split) * " << sp.BM << " + tid], side_acc);\n";
  // The partials are stored at the device's point of coherence; every wave
  // waits for its stores to complete (a workgroup barrier alone does not wait
  // for global stores), and only after the barrier does thread 0 count the
  // workgroup in.  The last workgroup to arrive reads all partials the same
  // coherent way, so no cache write-back or invalidate is needed.  The counter
  // is reset by the last workgroup for the next launch (ordered before it by
  // the end of the kernel).
  s << "  __builtin_amdgcn_s_waitcnt(0);  // this wave's partial stores are performed\n";
  s << "  __syncthreads();\n";
  s << "  if (tid == 0) {\n    int* cnt = (int*)a.p[" << cnt_slot << "];\n";
  s << "    const int old = __hip_atomic_fetch_add(cnt + tix * 32, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n";
  s << "    last_ = (old == " << S - 1 << ");\n";
  s << "    if (last_) __hip_atomic_store(cnt + tix * 32, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);\n  }\n";
  s << "  __syncthreads();\n  if (!last_) return;\n";
  bool any_tile_out = false;
  for (int o : ki.k.outs)
    if (!has(sp.side, o)) any_tile_out = true;
  // a row-program epilogue's loads go out with the partial loads below
  std::string epi_pre, epi_rest;
  const bool row_epi = any_tile_out && !sp.rowred.empty();
  if (row_epi) {
    epi_rest = row_epilogue(ki, sp, slot, &epi_pre);
    if (!epi_pre.empty()) s << "  {\n" << epi_pre;
  }
  // the side partials' loads go out before the tile's (from a clamped row,
  // the sum kept only for rows of the tile), so both wait on one round trip
  if (nside) {
    s << "  float sv_[" << S << "];\n  {\n    const int ts_ = tid < " << sp.BM << " ? tid : " << sp.BM - 1 << ";\n";
    s << "#pragma unroll\n    for (int p = 0; p < " << S << "; ++p) sv_[p] = coherent_load(&sidep[(tix * " << S << " + p) * "
      << sp.BM << " + ts_]);\n  }\n";
  }
  // deterministic sum of the partials, split 0 first
  if (vec4) {
    // all partial loads of a thread's float4 issued before they are summed
    s << "#pragma unroll\n  for (int i = tid * 4; i < " << tile << "; i += 1024) {\n    float4 v_[" << S << "];\n";
    s << "#pragma unroll\n    for (int p = 0; p < " << S << "; ++p) v_[p] = coherent_load4(rsP, (unsigned)(((tix * " << S
      << " + p) * " << tile << "LL + i) * 4));\n";
    s << "    float4 acc_ = make_float4(0.0f, 0.0f, 0.0f, 0.0f);\n";
    s << "#pragma unroll\n    for (int p = 0; p < " << S << "; ++p) {\n      acc_.x += v_[p].x;\n      acc_.y += v_[p].y;\n"
      << "      acc_.z += v_[p].z;\n      acc_.w += v_[p].w;\n    }\n";
    s << "    *(float4*)&Cs[(i / " << sp.BN << ") * " << sp.LDC << " + i % " << sp.BN << "] = acc_;\n  }\n";
  } else {
    s << "  for (int i = tid; i < " << tile << "; i += 256) {\n    float acc_ = 0.0f;\n";
    s << "    for (int p = 0; p < " << S << "; ++p) acc_ += coherent_load(&part[(tix * " << S << " + p) * " << tile
      << "LL + i]);\n";
    s << "    Cs[(i / " << sp.BN << ") * " << sp.LDC << " + i % " << sp.BN << "] = acc_;\n  }\n";
  }
  if (nside) {
    s << "  if (tid < " << sp.BM << ") {\n    float acc_ = 0.0f;\n";
    s << "#pragma unroll\n    for (int p = 0; p < " << S << "; ++p) acc_ += sv_[p];\n";
    s << "    side_s[tid] = acc_;\n  }\n";
  }
  s << "  __syncthreads();\n";
  for (int r : sp.side) {
    const Node& rn = g.nodes[r];
    if (!has(ki.k.outs, r)) continue;
    std::string val = rn.op == KORCH_REDUCE_MEAN ? "side_s[tid] / " + flit((double)sp.K) : "side_s[tid]";
    s << "  if (tid < " << sp.BM << " && m0 + tid < " << sp.M << "LL) "
      << out_store(g, r, "((" + ctype(rn.dtype) + "*)a.p[" + std::to_string(ki.out_slot(r)) + "])",
                   "bz * " + std::to_string(sp.M) + "LL + m0 + tid", 0, val)
      << ";\n";
  }
  if (any_tile_out) {
    if (!row_epi)
      s << gemm_epilogue(ki, sp, slot, "ml * " + std::to_string(sp.LDC),
                         std::set<int>(sp.side.begin(), sp.side.end()));
    else
      s << epi_rest << (epi_pre.empty() ? "" : "  }\n");
  }
  s << "}\n";
  gk.source = s.str();
  gk.grid[0] = (int)S;
  gk.grid[1] = (int)mtiles;
  gk.grid[2] = (int)sp.batch;
  gk.lds_bytes = (int)smem;
  ki.fill_cost(gk);
  return gk;
}

}  // namespace korch
