// MFMA GEMM family (and implicit-GEMM convolution): C = epi(pro(A) * pro(B)).
//
// Linear-transformation primitives (Korch, Section 3) are the dense
// contractions of a graph; here they run on gfx950 matrix cores
// (v_mfma_f32_16x16x32_{f16,bf16}, v_mfma_f32_16x16x4_f32) with fp32
// accumulation.  Elementwise / broadcast / layout primitives feeding an
// operand are evaluated while the operand tile is staged into LDS (prologue);
// elementwise primitives consuming the product are evaluated on the fp32 tile
// before the single store (epilogue).  Several products that share their left
// operand may run as one kernel, their right operands side by side in the tile.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <regex>

#include "families.h"
#include "gemm_common.h"

namespace korch {

static bool in_vec(const std::vector<int>& v, int x) { return std::find(v.begin(), v.end(), x) != v.end(); }

// The fissioned LayerNorm over the last axis (Korch's operator fission of
// LayerNorm into reduce and elementwise primitives):
//   mu = mean(X), D = X - mu, D2 = D^2, var = mean(D2), ve = var + eps,
//   r = rsqrt(ve), Xh = D r, Yg = Xh gamma, Y = Yg + beta,
// all inside the kernel, Y the product's left operand and its only use, gamma
// and beta vectors along the last axis.  The product is then
//   Y W = r (X diag(gamma) W - mu gamma^T W) + beta^T W   (per row r, mu)
// with var = mean(X^2) - mu^2: the kernel needs only X, the row sums of X
// and X^2, and the column sums gamma^T W and beta^T W, which it accumulates
// from the tiles it stages anyway.
static bool detect_ln_fold(const KInfo& ki, int Y, GemmSpec& sp) {
  const Graph& g = ki.g;
  auto in = [&](int v) { return v >= 0 && ki.in.count(v) > 0; };
  auto nd = [&](int v) -> const Node& { return g.nodes[v]; };
  auto bin = [&](int v, int op) { return in(v) && nd(v).op == op && !nd(v).attrs.has_scalar && nd(v).in.size() == 2; };
  auto last_axis = [&](int v) { return (int)nd(v).axis == (int)nd(nd(v).in[0]).shape.size() - 1 && nd(v).attrs.keepdim; };
  auto vec_k = [&](int v, int64_t K) {
    if (ki.in.count(v)) return false;
    const Shape& sh = nd(v).shape;
    int64_t n = 1;
    for (auto x : sh) n *= x;
    return n == K && !sh.empty() && sh.back() == K;
  };
  if (!bin(Y, KORCH_ADD)) return false;
  for (int s1 = 0; s1 < 2; ++s1) {
    const int Yg = nd(Y).in[s1], beta = nd(Y).in[1 - s1];
    if (!bin(Yg, KORCH_MUL)) continue;
    for (int s2 = 0; s2 < 2; ++s2) {
      const int Xh = nd(Yg).in[s2], gamma = nd(Yg).in[1 - s2];
      if (!bin(Xh, KORCH_MUL)) continue;
      for (int s3 = 0; s3 < 2; ++s3) {
        const int D = nd(Xh).in[s3], r = nd(Xh).in[1 - s3];
        if (!bin(D, KORCH_SUB) || !in(r) || nd(r).op != KORCH_RSQRT) continue;
        const int X = nd(D).in[0], mu = nd(D).in[1];
        if (in(X) || !in(mu) || nd(mu).op != KORCH_REDUCE_MEAN || nd(mu).in[0] != X || !last_axis(mu)) continue;
        const int ve = nd(r).in[0];
        if (!in(ve) || nd(ve).op != KORCH_ADD || !nd(ve).attrs.has_scalar || nd(ve).attrs.scalar < 0) continue;
        const int var = nd(ve).in[0];
        if (!in(var) || nd(var).op != KORCH_REDUCE_MEAN || !last_axis(var)) continue;
        const int D2 = nd(var).in[0];
        if (!in(D2) || nd(D2).op != KORCH_SQUARE || nd(D2).in[0] != D) continue;
        const Shape& xs = nd(X).shape;
        if (xs.size() != 2 || nd(Y).shape != xs || nd(D).shape != xs || nd(Xh).shape != xs) continue;
        const int64_t K = xs.back();
        if (!vec_k(gamma, K) || !vec_k(beta, K)) continue;
        const std::set<int> set = {mu, D, D2, var, ve, r, Xh, Yg, Y};
        // the LayerNorm's values are used only by itself and the product
        bool ok = true;
        for (int v : set) {
          if (std::find(ki.k.outs.begin(), ki.k.outs.end(), v) != ki.k.outs.end()) ok = false;
          for (int c : g.consumers[v])
            if (!set.count(c) && !(v == Y && nd(c).op == KORCH_MATMUL)) ok = false;
        }
        if (!ok || g.consumers[Y].size() != 1) continue;
        sp.lnf = true;
        sp.lnX = X, sp.lng = gamma, sp.lnb = beta, sp.lneps = nd(ve).attrs.scalar;
        sp.lnset = set;
        return true;
      }
    }
  }
  return false;
}

bool analyze_gemm(const KInfo& ki, GemmSpec& sp, std::string* why, bool allow_reduce) {
  const Graph& g = ki.g;
  if (ki.linear.empty()) {
    *why = "gemm: no linear primitive";
    return false;
  }
  const Node& l0 = g.nodes[ki.linear[0]];
  if (l0.op == KORCH_CONV2D) {
    if (ki.linear.size() != 1) {
      *why = "conv: more than one linear primitive";
      return false;
    }
    sp.conv = true;
    sp.mms = {ki.linear[0]};
    sp.A = l0.in[0];
    sp.Bs = {l0.in[1]};
    if (ki.in.count(sp.A)) {
      *why = "conv: the input must be a materialized tensor";
      return false;
    }
    const Shape& x = g.nodes[sp.A].shape;
    const Shape& w = g.nodes[sp.Bs[0]].shape;
    sp.OUT = l0.shape;
    sp.nb = (int)x.size() - 3;
    sp.nmdims = 2;
    sp.H = x[x.size() - 3];
    sp.W = x[x.size() - 2];
    sp.Cin = x.back();
    sp.KH = w[0];
    sp.KW = w[1];
    sp.stride = l0.attrs.stride;
    sp.pad = l0.attrs.pad;
    sp.Ho = sp.OUT[sp.OUT.size() - 3];
    sp.Wo = sp.OUT[sp.OUT.size() - 2];
    sp.M = sp.Ho * sp.Wo;
    sp.N = sp.OUT.back();
    sp.K = sp.KH * sp.KW * sp.Cin;
    sp.Nj = {sp.N};
  } else {
    for (int v : ki.linear)
      if (g.nodes[v].op != KORCH_MATMUL) {
        *why = "gemm: mixed linear primitives";
        return false;
      }
    sp.A = l0.in[0];
    // primary product first: largest N
    std::vector<int> mms = ki.linear;
    std::stable_sort(mms.begin(), mms.end(),
                     [&](int a, int b) { return g.nodes[a].shape.back() > g.nodes[b].shape.back(); });
    sp.mms = mms;
    for (int v : mms) {
      if (g.nodes[v].in[0] != sp.A) {
        *why = "gemm: products do not share their left operand";
        return false;
      }
      sp.Bs.push_back(g.nodes[v].in[1]);
    }
    for (int a : mms)
      for (int b : mms)
        if (a != b && ki.ancestor(a, b)) {
          *why = "gemm: one product feeds another";
          return false;
        }
    sp.OUT = g.nodes[mms[0]].shape;
    sp.nb = (int)sp.OUT.size() - 2;
    sp.nmdims = 1;
    sp.M = sp.OUT[sp.OUT.size() - 2];
    sp.N = sp.OUT.back();
    sp.K = g.nodes[sp.A].shape.back();
    if (mms.size() == 1 && detect_ln_fold(ki, sp.A, sp)) sp.A = sp.lnX;
    for (int v : mms) {
      const Shape& s = g.nodes[v].shape;
      if (!std::equal(s.begin(), s.end() - 1, sp.OUT.begin()) || (s.back() != sp.N && s.back() != 1)) {
        *why = "gemm: products differ in shape";
        return false;
      }
      sp.Nj.push_back(s.back());
    }
  }
  sp.mtype = g.nodes[sp.A].dtype;
  for (int b : sp.Bs)
    if (g.nodes[b].dtype != sp.mtype) {
      *why = "gemm: operand dtypes differ";
      return false;
    }
  int vb = 16 / dtype_bytes(sp.mtype);
  int64_t off = 0;
  for (auto n : sp.Nj) {
    sp.offj.push_back(off);
    off += (n + vb - 1) / vb * vb;
  }
  sp.Ntot = sp.mms.size() == 1 ? sp.N : off;
  sp.batch = 1;
  for (int d = 0; d < sp.nb; ++d) sp.batch *= sp.OUT[d];
  // classify nodes
  std::vector<int> operands = sp.Bs;
  operands.push_back(sp.A);
  for (int v : ki.k.prims) {
    if (in_vec(sp.mms, v) || sp.lnset.count(v)) continue;
    bool pro = false, below = false;
    for (int o : operands)
      if (v == o || ki.ancestor(v, o)) pro = true;
    for (int m : sp.mms)
      if (ki.ancestor(m, v)) below = true;
    const Node& n = g.nodes[v];
    Kind kd = op_kind(n.op);
    if (pro) {
      if (!(kd == Kind::Unary || kd == Kind::Binary || kd == Kind::Broadcast || kd == Kind::Layout)) {
        *why = std::string("gemm: prologue cannot hold ") + op_name(n.op);
        return false;
      }
      if (in_vec(ki.k.outs, v)) {
        *why = "gemm: a prologue node cannot be a kernel output";
        return false;
      }
      sp.pro.insert(v);
    } else if (below) {
      if (kd == Kind::Reduce) {
        if (!allow_reduce) {
          *why = "gemm: reduction in the epilogue";
          return false;
        }
        sp.rowred.push_back(v);
      } else if (!(kd == Kind::Unary || kd == Kind::Binary || kd == Kind::Broadcast)) {
        *why = std::string("gemm: epilogue cannot hold ") + op_name(n.op);
        return false;
      }
      sp.epi.insert(v);
    } else {
      if (!allow_reduce || kd != Kind::Reduce) {
        *why = "gemm: node is neither prologue nor epilogue";
        return false;
      }
      sp.side.push_back(v);
    }
  }
  // prologue nodes may only feed prologue nodes or products
  for (int v : sp.pro)
    for (int c : g.consumers[v])
      if (ki.in.count(c) && !sp.pro.count(c) && !in_vec(sp.mms, c) && !in_vec(sp.side, c)) {
        *why = "gemm: a prologue value is also used after the product";
        return false;
      }
  if (sp.conv && !sp.pro.empty() && !conv_uses_direct(sp, why)) {
    if (why) *why = "conv: a weight prologue needs the direct kernel (" + *why + ")";
    return false;
  }
  // epilogue shapes broadcast to the iteration space
  for (int v : sp.epi) {
    const Shape& s = g.nodes[v].shape;
    if (s.size() > sp.OUT.size()) {
      *why = "gemm: epilogue rank too large";
      return false;
    }
    for (size_t d = 0; d < s.size(); ++d) {
      int64_t t = sp.OUT[d + sp.OUT.size() - s.size()];
      if (s[d] != t && s[d] != 1) {
        *why = "gemm: epilogue shape does not broadcast to the product";
        return false;
      }
    }
    for (int u : g.nodes[v].in)
      if (ki.in.count(u) && !sp.epi.count(u) && !in_vec(sp.mms, u)) {
        *why = "gemm: epilogue reads a prologue value";
        return false;
      }
  }
  for (int o : ki.k.outs) {
    if (sp.pro.count(o)) {
      *why = "gemm: prologue output";
      return false;
    }
    if (sp.epi.count(o) && g.nodes[o].shape != sp.OUT && sp.rowred.empty()) {
      // broadcast-shaped epilogue outputs are stored where broadcast dims are 0
    }
  }
  return true;
}

static size_t gemm_smem_bytes_fwd(const GemmSpec& sp);

// The generator's decisions for a folded LayerNorm, taken on a copy: tiles,
// operand layouts, the register epilogue and direct-to-LDS staging must all
// apply, else the kernel is not supported.
static bool ln_fold_feasible(const KInfo& ki, GemmSpec sp, std::string* why) {
  choose_tiles(sp, false);
  plan_operands(ki, sp);
  sp.acc_t = reg_epilogue_output(ki, sp) >= 0;
  if (sp.acc_t) {
    sp.OSP = sp.BN + 8;
    sp.OSB = sp.BM * sp.OSP * 2;
  }
  plan_dma(ki, sp, false);
  if (!sp.dma || !sp.acc_t || sp.mtype != KORCH_F16 || sp.K % 64 || gemm_smem_bytes_fwd(sp) > 160 * 1024) {
    if (why) *why = "gemm: a folded LayerNorm needs fp16 tiles that divide the problem and the register epilogue";
    return false;
  }
  return true;
}

bool match_gemm(const KInfo& ki, std::string* why) {
  GemmSpec sp;
  if (!analyze_gemm(ki, sp, why, false)) return false;
  if (sp.conv) return false;
  if (sp.lnf && !ln_fold_feasible(ki, sp, why)) return false;
  if (sp.mms.size() > 1 && sp.Ntot > 128) {
    *why = "gemm: combined right operands wider than one tile";
    return false;
  }
  return true;
}

bool match_conv(const KInfo& ki, std::string* why) {
  GemmSpec sp;
  if (!analyze_gemm(ki, sp, why, false)) return false;
  return sp.conv;
}

// ---------------------------------------------------------------------------

void choose_tiles(GemmSpec& sp, bool split) {
  bool f32 = sp.mtype == KORCH_F32;
  sp.kstep = f32 ? 4 : 32;
  if (f32)
    sp.BK = 16;
  else if (sp.K % 64 == 0)
    sp.BK = 64;
  else if (sp.K % 32 == 0 || sp.K < 64)
    sp.BK = 32;
  else
    sp.BK = 64;
  int64_t nt = sp.mms.size() > 1 ? sp.Ntot : sp.N;
  if (nt <= 16)
    sp.BN = 16;
  else if (nt <= 32)
    sp.BN = 32;
  else if (nt <= 64)
    sp.BN = 64;
  else
    sp.BN = 128;
  sp.BM = 128;
  if (!split && nt > 64 && sp.mms.size() == 1) {
    // Tile shape by a throughput model of 256 compute units: tiles run in
    // rounds of 256, each round costs its tile area, and every tile pays for
    // re-reading its operand panels (proportional to 1/BM + 1/BN).  192-wide
    // tiles (half precision, k-tiles of 32 so that two workgroups still share
    // a compute unit's LDS) serve products whose 128-wide tiles would leave a
    // half-filled last round.  256 x 192 tiles (half precision, eight waves of
    // 64 x 96, k-tiles of 64, one workgroup per compute unit) re-read the
    // operand panels least; they are taken when they fill whole rounds.
    double best = 1e300;
    for (int bm : {128, 64, 256}) {
      for (int bn : {128, 96, 64, 192}) {
        if (bn == 96 && sp.N % 96 != 0) continue;
        if (bn == 192 && (sp.N % 192 != 0 || f32 || bm == 64)) continue;
        // register relief 2: no 256-row tiles (eight waves of 64 x 96 accumulators)
        if (bm == 256 && (bn != 192 || (sp.M + 255) / 256 * (sp.N / 192) * sp.batch < 256 || reg_relief() >= 2))
          continue;
        int64_t tiles = (sp.M + bm - 1) / bm * ((sp.N + bn - 1) / bn) * sp.batch;
        double rounds = (double)((tiles + 255) / 256);
        double cost = rounds * bm * bn * (1.0 + 24.0 * (1.0 / bm + 1.0 / bn));
        if (cost < best * (1.0 - 1e-9)) {
          best = cost;
          sp.BM = bm;
          sp.BN = bn;
        }
      }
    }
    if (sp.BN == 192 && sp.BM != 256) sp.BK = std::min(sp.BK, 32);
  } else if (!split) {
    int64_t tiles = (sp.M + 127) / 128 * ((sp.N + sp.BN - 1) / sp.BN) * sp.batch;
    if (tiles < 240 && sp.M > 64) sp.BM = 64;
  }
  // split-K: 32-row tiles, or 16 when that is what brings the workgroup count
  // (tiles times up to 16 splits) toward one per compute unit
  if (split) sp.BM = sp.M <= 16 || (sp.M + 31) / 32 * sp.batch * 16 < 256 ? 16 : 32;
  sp.WN = sp.BN >= 64 ? 2 : 1;
  sp.WM = 4 / sp.WN;
  while (sp.BM / sp.WM < 16) {
    // fewer waves along M; put the rest along N when possible
    if (sp.WN < 4 && sp.BN / (sp.WN * 2) >= 16) {
      sp.WN *= 2;
      sp.WM = 4 / sp.WN;
    } else {
      break;
    }
  }
  if (sp.BM / sp.WM < 16) sp.WM = std::max(1, sp.BM / 16);
  sp.NT = 256;
  if (sp.BM == 256) {
    sp.WM = 4;
    sp.WN = 2;
    sp.NT = 512;
  }
  sp.NS = 2;
  if (const char* e = getenv("KORCH_GEMM_NS")) sp.NS = std::max(2, std::min(8, atoi(e)));
  // Explicit tile override "BM,BN,BK,WM,WN" (tile-configuration sweeps of the
  // profiler); ignored unless it is consistent.
  if (const char* e = getenv("KORCH_GEMM_CFG")) {
    int bm, bn, bk, wm, wn;
    if (!split && sscanf(e, "%d,%d,%d,%d,%d", &bm, &bn, &bk, &wm, &wn) == 5 && (wm * wn == 4 || wm * wn == 8) &&
        bm % (16 * wm) == 0 && bn % (16 * wn) == 0 && bk % sp.kstep == 0 && bk >= sp.kstep &&
        (sp.mms.size() == 1 || bn >= sp.Ntot)) {
      sp.BM = bm;
      sp.BN = bn;
      sp.BK = bk;
      sp.WM = wm;
      sp.WN = wn;
      sp.NT = 64 * wm * wn;
    }
  }
  sp.WTM = sp.BM / sp.WM;
  sp.WTN = sp.BN / sp.WN;
  sp.FM = sp.WTM / 16;
  sp.FN = sp.WTN / 16;
  sp.VA = 16 / dtype_bytes(sp.mtype);
  sp.VB = sp.VA;
  // Row pitch of k-contiguous operand tiles.  A fragment read (16 rows x four
  // consecutive 16-byte slots, one 16-byte vector per lane) is free of bank
  // conflicts on gfx950 when the pitch is an odd multiple of 32 bytes; odd
  // multiples of 16 bytes cost four extra cycles per read (measured).
  sp.BKP = sp.BK + (f32 ? 4 : 16);
  sp.LDC = sp.BN + 4;
}

void plan_operands(const KInfo& ki, GemmSpec& sp) {
  int C = 16 / dtype_bytes(sp.mtype);
  sp.b_kn = sp.Bs.size() == 1 && !ki.in.count(sp.Bs[0]) && sp.N % C == 0;
  // row pitch: 32 extra bytes keep the four rows of one transposing read in distinct banks
  sp.BNP = sp.BN + (sp.mtype == KORCH_F32 ? 4 : 16);
  sp.BSH = 0;
  const char* shift_env = getenv("KORCH_LDS_BANK_SHIFT");  // "0" disables the row shift
  if (sp.b_kn && sp.mtype != KORCH_F32 && !(shift_env && atoi(shift_env) == 0)) {
    // smallest shift (a multiple of 16 bytes) that makes the 32-byte windows of
    // rows {0,1,2,3,8,9,10,11} disjoint modulo the 256 bytes of the 64 banks
    const int P = sp.BNP * 2;
    for (int S = 0; S < 256; S += 16) {
      int w[8], n = 0;
      for (int r : {0, 1, 2, 3, 8, 9, 10, 11}) w[n++] = (r * P + (r >> 3) * S) % 256;
      bool ok = true;
      for (int a = 0; a < 8 && ok; ++a)
        for (int b = a + 1; b < 8 && ok; ++b) {
          int d = (w[b] - w[a] + 256) % 256;
          if (d < 32 || d > 224) ok = false;
        }
      if (ok) {
        sp.BSH = S / 2;
        break;
      }
    }
  }
}

std::string b_row_off(const GemmSpec& sp, const std::string& k) {
  std::string r = "(" + k + ") * " + std::to_string(sp.BNP);
  if (sp.BSH) r += " + ((" + k + ") >> 3) * " + std::to_string(sp.BSH);
  return r;
}

int64_t b_buf_elems(const GemmSpec& sp) {
  return sp.b_kn ? (int64_t)sp.BK * sp.BNP + (int64_t)((sp.BK + 7) / 8) * sp.BSH : (int64_t)sp.BN * sp.BKP;
}

// Raw staging of an operand that is a plain materialized tensor (no prologue):
// the bytes go to LDS unchanged.  A k-contiguous operand ([.., rows, K]) moves
// as 16-byte vectors; a row-contiguous one ([.., K, rows], e.g. a weight
// [K, N]) is read as 4-wide row vectors from KB consecutive k and transposed in
// registers, so every LDS write is a 16-byte vector of KB consecutive k.
// Returns "" when the operand does not qualify.
static std::string raw_loader(const KInfo& ki, const GemmSpec& sp, bool isA, const std::map<int, int>& slot) {
  const Graph& g = ki.g;
  if (sp.conv && isA) return "";
  if (!sp.conv && (!isA && sp.Bs.size() != 1)) return "";
  int node = isA ? sp.A : sp.Bs[0];
  if (ki.in.count(node)) return "";
  bool f32 = sp.mtype == KORCH_F32;
  std::string T = ctype(sp.mtype);
  int rows = isA ? sp.BM : sp.BN;
  int64_t R = isA ? sp.M : sp.N;
  std::string X = isA ? "A" : "B";
  std::string lds = isA ? "As" : "Bs";
  std::string base = isA ? "m0" : "n0";
  std::string P = "((const " + T + "*)a.p[" + std::to_string(slot.at(node)) + "])";
  // batch offset of the operand (broadcast batch dims read index 0)
  std::string boff = "0";
  if (!sp.conv) {
    const Shape& sh = g.nodes[node].shape;
    Shape ob(sp.OUT.begin(), sp.OUT.begin() + sp.nb);
    Shape nbsh(sh.begin(), sh.end() - 2);
    std::vector<Ix> zc;
    for (int d = 0; d < sp.nb; ++d) zc.push_back(Ix::var("z" + std::to_string(d)));
    auto bi = broadcast_index(nbsh, ob, zc);
    auto st = strides_of(sh);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], 1));
    boff = off.at();
  }
  std::ostringstream s;
  if (isA) {
    // A: [.., M, K], k contiguous
    int V = sp.VA;
    if (sp.K % V) return "";
    int kper = sp.BK / V;
    int nslots = rows * kper;
    int per = (nslots + sp.NT - 1) / sp.NT;
    s << "  uint4 r" << X << "[" << sp.NS << "][" << per << "];\n";
    s << "  auto fetch" << X << " = [&](const i64 k0, const int st) {\n#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
    s << "    const int sl = tid + i * " << sp.NT << ";\n";
    if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
    s << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << V << ";\n";
    s << "    const i64 rg = " << base << " + rl, kg = k0 + kl;\n";
    s << "    if (rg < " << R << "LL && kg + " << V << " <= " << sp.K << "LL) r" << X << "[st][i] = *(const uint4*)(" << P
      << " + " << boff << " + rg * " << sp.K << "LL + kg);\n";
    s << "    else {\n      " << T << " t_[" << V << "];\n#pragma unroll\n      for (int e = 0; e < " << V
      << "; ++e) t_[e] = (rg < " << R << "LL && kg + e < " << sp.K << "LL) ? " << P << "[" << boff << " + rg * "
      << sp.K << "LL + kg + e] : fromf<" << T << ">(0.0f);\n      __builtin_memcpy(&r" << X << "[st][i], t_, 16);\n    }\n";
    s << "  }\n  };\n";
    s << "  auto stash" << X << " = [&](const int buf, const int st, const i64 k0_) {\n  (void)k0_;\n#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
    s << "    const int sl = tid + i * " << sp.NT << ";\n";
    if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
    s << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << V << ";\n";
    s << "    *(uint4*)(" << lds << " + buf * " << rows * sp.BKP << " + rl * " << sp.BKP << " + kl) = r" << X << "[st][i];\n";
    s << "  }\n  };\n";
    return s.str();
  }
  // B: [.., K, N] (or conv weights [KH, KW, Cin, Cout] = [K, N]), n contiguous
  if (sp.b_kn) {
    // copied unchanged into LDS as [k][n]; the MFMA reads transpose it
    int C = 16 / dtype_bytes(sp.mtype);
    int cpr = sp.BN / C;
    int nslots = sp.BK * cpr;
    int per = (nslots + sp.NT - 1) / sp.NT;
    s << "  uint4 r" << X << "[" << sp.NS << "][" << per << "];\n";
    s << "  auto fetch" << X << " = [&](const i64 k0, const int st) {\n#pragma unroll\n  for (int i = 0; i < " << per
      << "; ++i) {\n";
    s << "    const int sl = tid + i * " << sp.NT << ";\n";
    if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
    s << "    const int kl = sl / " << cpr << ", nl = (sl % " << cpr << ") * " << C << ";\n";
    s << "    const i64 kg = k0 + kl, ng = " << base << " + nl;\n";
    s << "    if (kg < " << sp.K << "LL && ng + " << C << " <= " << sp.N << "LL) r" << X << "[st][i] = *(const uint4*)(" << P
      << " + " << boff << " + kg * " << sp.N << "LL + ng);\n";
    s << "    else {\n      " << T << " t_[" << C << "];\n#pragma unroll\n      for (int e = 0; e < " << C
      << "; ++e) t_[e] = (kg < " << sp.K << "LL && ng + e < " << sp.N << "LL) ? " << P << "[" << boff << " + kg * "
      << sp.N << "LL + ng + e] : fromf<" << T << ">(0.0f);\n      __builtin_memcpy(&r" << X << "[st][i], t_, 16);\n    }\n";
    s << "  }\n  };\n";
    s << "  auto stash" << X << " = [&](const int buf, const int st, const i64 k0_) {\n  (void)k0_;\n#pragma unroll\n  for (int i = 0; i < " << per
      << "; ++i) {\n";
    s << "    const int sl = tid + i * " << sp.NT << ";\n";
    if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
    s << "    const int kl = sl / " << cpr << ", nl = (sl % " << cpr << ") * " << C << ";\n";
    s << "    *(uint4*)(" << lds << " + buf * " << b_buf_elems(sp) << " + " << b_row_off(sp, "kl") << " + nl) = r" << X
      << "[st][i];\n";
    s << "  }\n  };\n";
    return s.str();
  }
  const int VT = 4;
  int KB = f32 ? 4 : 8;
  if (sp.N % VT) return "";
  int nper = rows / VT;
  int nblocks = (sp.BK / KB) * nper;
  int per = (nblocks + sp.NT - 1) / sp.NT;
  std::string T4 = "vec_t<4, " + T + ">";
  std::string TK = "vec_t<" + std::to_string(KB) + ", " + T + ">";
  s << "  " << T4 << " r" << X << "[" << sp.NS << "][" << per << "][" << KB << "];\n";
  s << "  auto fetch" << X << " = [&](const i64 k0, const int st) {\n#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
  s << "    const int b_ = tid + i * " << sp.NT << ";\n";
  if (nblocks % sp.NT) s << "    if (b_ >= " << nblocks << ") break;\n";
  s << "    const int kb = b_ / " << nper << ", nb = b_ % " << nper << ";\n";
  s << "    const i64 kg = k0 + kb * " << KB << ", ng = " << base << " + nb * " << VT << ";\n";
  s << "#pragma unroll\n    for (int kk = 0; kk < " << KB << "; ++kk) {\n";
  s << "      const i64 k = kg + kk;\n";
  s << "      if (k < " << sp.K << "LL && ng + " << VT << " <= " << sp.N << "LL) r" << X << "[st][i][kk] = *(const " << T4
    << "*)(" << P << " + " << boff << " + k * " << sp.N << "LL + ng);\n";
  s << "      else {\n#pragma unroll\n        for (int j = 0; j < " << VT << "; ++j) r" << X
    << "[st][i][kk][j] = (k < " << sp.K << "LL && ng + j < " << sp.N << "LL) ? " << P << "[" << boff << " + k * " << sp.N
    << "LL + ng + j] : fromf<" << T << ">(0.0f);\n      }\n    }\n  }\n  };\n";
  s << "  auto stash" << X << " = [&](const int buf, const int st, const i64 k0_) {\n  (void)k0_;\n#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
  s << "    const int b_ = tid + i * " << sp.NT << ";\n";
  if (nblocks % sp.NT) s << "    if (b_ >= " << nblocks << ") break;\n";
  s << "    const int kb = b_ / " << nper << ", nb = b_ % " << nper << ";\n";
  s << "#pragma unroll\n    for (int j = 0; j < " << VT << "; ++j) {\n      " << TK << " col;\n";
  s << "#pragma unroll\n      for (int kk = 0; kk < " << KB << "; ++kk) col[kk] = r" << X << "[st][i][kk][j];\n";
  s << "      *(" << TK << "*)(" << lds << " + buf * " << rows * sp.BKP << " + (nb * " << VT << " + j) * " << sp.BKP
    << " + kb * " << KB << ") = col;\n    }\n  }\n  };\n";
  return s.str();
}

// Branch-free staging of plain materialized operands with buffer loads: each
// 16-byte vector's byte offset is replaced by an out-of-range sentinel when the
// vector lies outside the tensor, and the hardware then returns zeros.  With
// no divergent control flow the loads of later k-tiles stay in flight while
// the current tile is multiplied.  Handles the left operand ([.., M, K], k
// contiguous), the implicit-GEMM convolution input, and the right operand
// staged [k][n].  Returns "" when the operand does not qualify (needs
// 16-byte-divisible rows and a tensor below 2 GiB).
static std::string buffer_loader(const KInfo& ki, const GemmSpec& sp, bool isA, const std::map<int, int>& slot) {
  const Graph& g = ki.g;
  int node = isA ? sp.A : sp.Bs[0];
  if (!isA && (sp.Bs.size() != 1 || !sp.b_kn)) return "";
  if (ki.in.count(node)) return "";
  int eb = dtype_bytes(sp.mtype);
  int C = 16 / eb;  // elements per 16-byte vector
  double bytes = (double)numel(g.nodes[node].shape) * eb;
  if (bytes >= 2147483648.0) return "";
  std::string T = ctype(sp.mtype);
  std::string X = isA ? "A" : "B";
  std::string lds = isA ? "As" : "Bs";
  std::string P = "a.p[" + std::to_string(slot.at(node)) + "]";
  std::string boff = "0";
  if (!sp.conv) {
    const Shape& sh = g.nodes[node].shape;
    Shape ob(sp.OUT.begin(), sp.OUT.begin() + sp.nb);
    Shape nbsh(sh.begin(), sh.end() - 2);
    std::vector<Ix> zc;
    for (int d = 0; d < sp.nb; ++d) zc.push_back(Ix::var("z" + std::to_string(d)));
    auto bi = broadcast_index(nbsh, ob, zc);
    auto st = strides_of(sh);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], 1));
    boff = off.at();
  } else if (sp.nb && isA) {
    boff = "z0 * " + std::to_string(sp.H * sp.W * sp.Cin);
  }
  std::ostringstream s;
  int rows, kper, nslots;
  if (isA) {
    if (sp.K % C) return "";
    if (sp.conv && sp.Cin % C) return "";
    kper = sp.BK / C;
    rows = sp.BM;
    nslots = rows * kper;
  } else {
    if (sp.N % C) return "";
    kper = sp.BN / C;  // vectors per k row
    rows = sp.BK;
    nslots = rows * kper;
  }
  int per = (nslots + sp.NT - 1) / sp.NT;
  s << "  const __amdgpu_buffer_rsrc_t rs" << X << " = __builtin_amdgcn_make_buffer_rsrc(" << P << ", 0, "
    << (long long)bytes << ", 0x00020000);\n";
  s << "  uint4 r" << X << "[" << sp.NS << "][" << per << "];\n";
  // per-slot constants
  s << "  int o" << X << "[" << per << "];  // element offset of the slot's vector at k-tile 0\n";
  s << "  bool v" << X << "[" << per << "];  // slot lies inside the tile rows / columns\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
  s << "    const int sl = tid + i * " << sp.NT << ";\n";
  if (isA) {
    s << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << C << ";\n";
    s << "    const i64 rg = m0 + rl;\n";
    if (sp.conv) {
      s << "    o" << X << "[i] = (int)rg;  // output pixel\n";
      s << "    v" << X << "[i] = sl < " << nslots << " && rg < " << sp.M << "LL;\n";
    } else {
      s << "    o" << X << "[i] = (int)(" << boff << " + rg * " << sp.K << "LL + kl);\n";
      s << "    v" << X << "[i] = sl < " << nslots << " && rg < " << sp.M << "LL;\n";
    }
  } else {
    s << "    const int kl = sl / " << kper << ", nl = (sl % " << kper << ") * " << C << ";\n";
    s << "    const i64 ng = n0 + nl;\n";
    s << "    o" << X << "[i] = (int)(" << boff << " + (i64)kl * " << sp.N << "LL + ng);\n";
    s << "    v" << X << "[i] = sl < " << nslots << " && ng < " << sp.N << "LL;\n";
  }
  s << "  }\n";
  s << "  auto fetch" << X << " = [&](const i64 k0, const int st) {\n#pragma unroll\n  for (int i = 0; i < " << per
    << "; ++i) {\n";
  s << "    const int sl = tid + i * " << sp.NT << ";\n";
  if (isA) {
    s << "    const int kl = (sl % " << kper << ") * " << C << ";\n";
    s << "    const int kg = (int)k0 + kl;\n";
    if (sp.conv) {
      s << "    const int p_ = o" << X << "[i];\n";
      s << "    const int oy = p_ / " << sp.Wo << ", ox = p_ % " << sp.Wo << ";\n";
      s << "    const int tap = kg / " << sp.Cin << ", ci = kg % " << sp.Cin << ";\n";
      s << "    const int iy = oy * " << sp.stride << " + tap / " << sp.KW << " - " << sp.pad << ";\n";
      s << "    const int ix = ox * " << sp.stride << " + tap % " << sp.KW << " - " << sp.pad << ";\n";
      s << "    const bool ok = v" << X << "[i] && kg < " << sp.K << " && iy >= 0 && iy < " << sp.H << " && ix >= 0 && ix < "
        << sp.W << ";\n";
      s << "    const int e_ = (int)(" << boff << ") + (iy * " << sp.W << " + ix) * " << sp.Cin << " + ci;\n";
    } else {
      s << "    const bool ok = v" << X << "[i] && kg < " << sp.K << ";\n";
      s << "    const int e_ = o" << X << "[i] + (int)k0;\n";
    }
  } else {
    s << "    const int kl = sl / " << kper << ";\n";
    s << "    const bool ok = v" << X << "[i] && (int)k0 + kl < " << sp.K << ";\n";
    s << "    const int e_ = o" << X << "[i] + (int)k0 * " << sp.N << ";\n";
  }
  s << "    const unsigned off = ok ? (unsigned)e_ * " << eb << "u : 0x80000000u;\n";
  s << "    r" << X << "[st][i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs" << X
    << ", off, 0, 0));\n";
  s << "  }\n  };\n";
  s << "  auto stash" << X << " = [&](const int buf, const int st, const i64 k0_) {\n  (void)k0_;\n#pragma unroll\n  for (int i = 0; i < " << per
    << "; ++i) {\n";
  s << "    const int sl = tid + i * " << sp.NT << ";\n";
  if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
  if (isA) {
    s << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << C << ";\n";
    s << "    *(uint4*)(" << lds << " + buf * " << sp.BM * sp.BKP << " + rl * " << sp.BKP << " + kl) = r" << X << "[st][i];\n";
  } else {
    s << "    const int kl = sl / " << kper << ", nl = (sl % " << kper << ") * " << C << ";\n";
    s << "    *(uint4*)(" << lds << " + buf * " << b_buf_elems(sp) << " + " << b_row_off(sp, "kl") << " + nl) = r" << X
      << "[st][i];\n";
  }
  s << "  }\n  };\n";
  return s.str();
}

// Emits a lambda `fetchX(k0)` that evaluates the operand (with its prologue)
// for this thread's slots of a BM x BK (A) or BN x BK (B) tile into registers,
// and `stashX(buf)` that converts and writes them to LDS in [row][k] layout.
std::string operand_loader(const KInfo& ki, const GemmSpec& sp, bool isA, const std::map<int, int>& slot) {
  {
    std::string buf = buffer_loader(ki, sp, isA, slot);
    if (!buf.empty()) return buf;
  }
  {
    std::string raw = raw_loader(ki, sp, isA, slot);
    if (!raw.empty()) return raw;
  }
  const Graph& g = ki.g;
  int V = isA ? sp.VA : sp.VB;
  int rows = isA ? sp.BM : sp.BN;
  int nslots = rows * sp.BK / V;
  int per = (nslots + sp.NT - 1) / sp.NT;
  std::string X = isA ? "A" : "B";
  std::string T = ctype(sp.mtype);
  std::string lds = isA ? "As" : "Bs";
  std::ostringstream s;
  // batch coordinates of the operand
  auto batch_idx = [&](int node) {
    const Shape& sh = g.nodes[node].shape;
    Shape ob(sp.OUT.begin(), sp.OUT.begin() + sp.nb);
    Shape nbsh(sh.begin(), sh.end() - 2);
    std::vector<Ix> zc;
    for (int d = 0; d < sp.nb; ++d) zc.push_back(Ix::var("z" + std::to_string(d)));
    return broadcast_index(nbsh, ob, zc);
  };
  // Generates loader code for one product operand: value at (row, k) for `node`.
  // axis_k: vector along k (row fixed) else vector along the row.
  auto emit_operand = [&](int node, bool axis_k, bool guarded, const std::string& rowv, const std::string& kv,
                          const std::string& rowlim, int64_t colshift) -> std::string {
    Emitter em(g);
    em.inset = sp.pro;
    em.argslot = slot;
    em.vec = V;
    em.force_gather = guarded;
    std::vector<Ix> idx = batch_idx(node);
    Ix r = axis_k ? Ix::var(rowv, 0, 1) : Ix::var(rowv, 1, V);
    Ix k = axis_k ? Ix::var(kv, 1, V) : Ix::var(kv, 0, 1);
    if (colshift) r = ix_addk(r, -colshift);
    if (isA) {
      idx.push_back(r);
      idx.push_back(k);
    } else {
      idx.push_back(k);
      idx.push_back(r);
    }
    std::string val = em.value(node, idx);
    std::ostringstream o;
    if (!guarded) {
      o << em.pre.str() << "#pragma unroll\n      for (int e = 0; e < " << V << "; ++e) {\n"
        << em.body.str() << "        dst[e] = " << val << ";\n      }\n";
    } else {
      std::string cond = axis_k ? "(" + rowv + " < " + rowlim + " && " + kv + " + e < " + std::to_string(sp.K) + ")"
                                : "(" + rowv + " + e < " + rowlim + " && " + kv + " < " + std::to_string(sp.K) + ")";
      // gathers that read zero out of range are issued without a branch (a
      // guarded load waits for every load in flight at the join); the value
      // is selected afterwards, as the prologue of a zero need not be zero
      Emitter eg(g);
      eg.inset = sp.pro;
      eg.argslot = slot;
      eg.vec = V;
      eg.force_gather = true;
      eg.gather_guard = "ok_";
      std::string gval = eg.value(node, idx);
      if (eg.n_guard_fallback == 0) {
        o << "#pragma unroll\n      for (int e = 0; e < " << V << "; ++e) {\n        const bool ok_ = " << cond << ";\n"
          << eg.pre.str() << eg.body.str() << "        dst[e] = ok_ ? (" << gval << ") : 0.0f;\n      }\n";
      } else {
        o << "#pragma unroll\n      for (int e = 0; e < " << V << "; ++e) {\n        dst[e] = 0.0f;\n        if "
          << cond << " {\n"
          << em.pre.str() << em.body.str() << "        dst[e] = " << val << ";\n        }\n      }\n";
      }
    }
    return o.str();
  };
  auto count_gathers = [&](int node, bool axis_k) {
    Emitter em(g);
    em.inset = sp.pro;
    em.argslot = slot;
    em.vec = V;
    std::vector<Ix> idx = batch_idx(node);
    Ix r = axis_k ? Ix::var("r_", 0, 1) : Ix::var("r_", 1, V);
    Ix k = axis_k ? Ix::var("k_", 1, V) : Ix::var("k_", 0, 1);
    if (isA) {
      idx.push_back(r);
      idx.push_back(k);
    } else {
      idx.push_back(k);
      idx.push_back(r);
    }
    em.value(node, idx);
    return em.n_gather;
  };
  std::vector<int> nodes = isA ? std::vector<int>{sp.A} : sp.Bs;
  bool axis_k = true;
  if (!sp.conv) {
    int gk = 0, gr = 0;
    for (int n : nodes) {
      gk += count_gathers(n, true);
      gr += count_gathers(n, false);
    }
    axis_k = !(gr < gk);
  } else {
    axis_k = isA ? true : false;  // X: channels contiguous; W as [K, N]: N contiguous
  }
  int kper = axis_k ? sp.BK / V : sp.BK;
  // Staged prologue: fetchX only issues the loads of the operand's inputs
  // (uniform and vector loads, into per-stage registers of their own type, at
  // indices clamped into the tensors); stashX evaluates the prologue once the
  // data has arrived, zeroes elements outside the problem and writes LDS.  The
  // loads of a tile then stay in flight while earlier tiles are multiplied.
  if (!sp.conv && nodes.size() == 1) {
    const int64_t R = isA ? sp.M : sp.N;
    if (axis_k ? sp.K % V == 0 : R % V == 0) {
      Emitter em(g);
      em.inset = sp.pro;
      em.argslot = slot;
      em.vec = V;
      em.staged = true;
      em.stages = sp.NS;
      em.slots = per;
      em.tmp = isA ? 0 : 500;  // keep the two operands' register names apart
      // the slots of one thread differ only in their row (axis_k) or only in
      // their k (vector along rows) when the thread count is a multiple of the
      // vectors per row / per k
      if (axis_k ? sp.NT % kper == 0 : sp.NT % (rows / V) == 0) em.slot_var = axis_k ? "rg" : "kg";
      std::vector<Ix> idx = batch_idx(nodes[0]);
      Ix r = axis_k ? Ix::var("rg", 0, 1) : Ix::var("rg", 1, V);
      Ix k = axis_k ? Ix::var("kg", 1, V) : Ix::var("kg", 0, 1);
      if (isA) {
        idx.push_back(r);
        idx.push_back(k);
      } else {
        idx.push_back(k);
        idx.push_back(r);
      }
      std::string val = em.value(nodes[0], idx);
      if (em.n_gather == 0) {
        std::string base = isA ? "m0" : "n0";
        auto slot_coords = [&]() {
          std::ostringstream o;
          o << "    const int sl = tid + i * " << sp.NT << ";\n";
          if (nslots % sp.NT) o << "    if (sl >= " << nslots << ") break;\n";
          if (axis_k)
            o << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << V << ";\n";
          else
            o << "    const int kl = sl / " << rows / V << ", rl = (sl % " << rows / V << ") * " << V << ";\n";
          return o.str();
        };
        s << em.stage_decl.str();
        s << "  auto fetch" << X << " = [&](const i64 k0, const int st) {\n#pragma unroll\n  for (int i = 0; i < " << per
          << "; ++i) {\n";
        s << slot_coords();
        s << "    const i64 rg = " << base << " + rl < " << R - (axis_k ? 1 : V) << "LL ? " << base << " + rl : "
          << R - (axis_k ? 1 : V) << "LL;\n";
        s << "    const i64 kg = k0 + kl < " << sp.K - (axis_k ? V : 1) << "LL ? k0 + kl : " << sp.K - (axis_k ? V : 1)
          << "LL;\n";
        s << em.pre.str() << "  }\n  };\n";
        s << "  auto stash" << X << " = [&](const int buf, const int st, const i64 k0) {\n#pragma unroll\n  for (int i = 0; i < "
          << per << "; ++i) {\n";
        s << slot_coords();
        s << "    const i64 rg = " << base << " + rl, kg = k0 + kl;\n";
        s << "    float dst[" << V << "];\n";
        // a tile-aligned problem has no element outside it
        const bool aligned = R % rows == 0 && sp.K % sp.BK == 0;
        std::string cond = aligned ? "true"
                           : axis_k ? "(rg < " + std::to_string(R) + "LL && kg + e < " + std::to_string(sp.K) + "LL)"
                                    : "(rg + e < " + std::to_string(R) + "LL && kg < " + std::to_string(sp.K) + "LL)";
        s << "#pragma unroll\n    for (int e = 0; e < " << V << "; ++e) {\n" << em.body.str() << "      dst[e] = " << cond
          << " ? (float)(" << val << ") : 0.0f;\n    }\n";
        if (axis_k) {
          s << "    stv<" << V << ">(" << lds << " + buf * " << rows * sp.BKP << " + rl * " << sp.BKP << " + kl, dst);\n";
        } else {
          s << "#pragma unroll\n    for (int e = 0; e < " << V << "; ++e) " << lds << "[buf * " << rows * sp.BKP
            << " + (rl + e) * " << sp.BKP << " + kl] = fromf<" << T << ">(dst[e]);\n";
        }
        s << "  }\n  };\n";
        return s.str();
      }
    }
  }
  // slot s -> (row, k): axis_k: row = s / (BK/V), kk = (s % (BK/V)) * V
  //                     axis_row: kk = s / (rows/V), row = (s % (rows/V)) * V
  s << "  float r" << X << "[" << sp.NS << "][" << per << "][" << V << "];\n";
  s << "  auto fetch" << X << " = [&](const i64 k0, const int st) {\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
  s << "    const int sl = tid + i * " << sp.NT << ";\n";
  if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
  if (axis_k)
    s << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << V << ";\n";
  else
    s << "    const int kl = sl / " << rows / V << ", rl = (sl % " << rows / V << ") * " << V << ";\n";
  std::string base = isA ? "m0" : "n0";
  s << "    const i64 rg = " << base << " + rl, kg = k0 + kl;\n";
  s << "    float* dst = r" << X << "[st][i];\n";
  if (sp.conv && isA) {
    // implicit GEMM: row = output pixel, k = (ky, kx, ci); 32-bit index math
    // (pixel counts and per-image sizes are far below 2^31)
    bool vecok = sp.Cin % V == 0;
    s << "    {\n      const int oy = (int)rg / " << sp.Wo << ", ox = (int)rg % " << sp.Wo << ";\n";
    s << "      const int tap = (int)kg / " << sp.Cin << ", ci = (int)kg % " << sp.Cin << ";\n";
    s << "      const int iy = oy * " << sp.stride << " + tap / " << sp.KW << " - " << sp.pad << ";\n";
    s << "      const int ix = ox * " << sp.stride << " + tap % " << sp.KW << " - " << sp.pad << ";\n";
    std::string P = "((const " + T + "*)a.p[" + std::to_string(slot.at(sp.A)) + "])";
    std::string bofs = sp.nb ? "z0 * " + std::to_string(sp.H * sp.W * sp.Cin) + "LL + " : "";
    s << "      const bool ok = rg < " << sp.M << "LL && kg < " << sp.K << "LL && iy >= 0 && iy < " << sp.H
      << " && ix >= 0 && ix < " << sp.W << ";\n";
    if (vecok) {
      s << "      if (ok) ldv<" << V << ">(dst, " << P << " + " << bofs << "(iy * " << sp.W << " + ix) * " << sp.Cin
        << "LL + ci);\n";
      s << "      else {\n#pragma unroll\n        for (int e = 0; e < " << V << "; ++e) dst[e] = 0.0f;\n      }\n";
    } else {
      s << "#pragma unroll\n      for (int e = 0; e < " << V << "; ++e) {\n";
      s << "        const i64 k2 = kg + e, tap2 = k2 / " << sp.Cin << ", ci2 = k2 % " << sp.Cin << ";\n";
      s << "        const i64 iy2 = oy * " << sp.stride << " + tap2 / " << sp.KW << " - " << sp.pad << ";\n";
      s << "        const i64 ix2 = ox * " << sp.stride << " + tap2 % " << sp.KW << " - " << sp.pad << ";\n";
      s << "        dst[e] = (rg < " << sp.M << "LL && k2 < " << sp.K << "LL && iy2 >= 0 && iy2 < " << sp.H
        << " && ix2 >= 0 && ix2 < " << sp.W << ") ? ld1(" << P << " + " << bofs << "(iy2 * " << sp.W
        << " + ix2) * " << sp.Cin << "LL + ci2) : 0.0f;\n      }\n";
    }
    s << "    }\n";
  } else if (sp.conv && !isA) {
    // weights [KH, KW, Cin, Cout] are a row-major [K, N] matrix
    std::string P = "((const " + T + "*)a.p[" + std::to_string(slot.at(sp.Bs[0])) + "])";
    s << "    if (kg < " << sp.K << "LL && rg + " << V << " <= " << sp.N << "LL) ldv<" << V << ">(dst, " << P
      << " + kg * " << sp.N << "LL + rg);\n";
    s << "    else {\n#pragma unroll\n      for (int e = 0; e < " << V << "; ++e) dst[e] = (kg < " << sp.K
      << "LL && rg + e < " << sp.N << "LL) ? ld1(" << P << " + kg * " << sp.N << "LL + rg + e) : 0.0f;\n    }\n";
  } else {
    // one or several product operands (B columns side by side)
    for (size_t j = 0; j < nodes.size(); ++j) {
      int64_t lo = isA ? 0 : (sp.mms.size() > 1 ? sp.offj[j] : 0);
      int64_t nj = isA ? sp.M : sp.Nj[j];
      std::string rowv = "rg";
      std::string lim = std::to_string(lo + nj);
      if (nodes.size() > 1) {
        int64_t hi = j + 1 < nodes.size() ? sp.offj[j + 1] : (int64_t)1 << 40;
        s << "    " << (j ? "else " : "") << "if (rg < " << hi << "LL) {\n";
      } else {
        s << "    {\n";
      }
      std::string fastc = axis_k ? "(rg < " + lim + "LL && kg + " + std::to_string(V) + " <= " +
                                       std::to_string(sp.K) + "LL)"
                                 : "(rg + " + std::to_string(V) + " <= " + lim + "LL && kg < " +
                                       std::to_string(sp.K) + "LL)";
      // a tile-aligned problem never needs the guarded per-element path
      int64_t R = isA ? sp.M : sp.N;
      bool aligned = nodes.size() == 1 && R % rows == 0 && sp.K % sp.BK == 0;
      if (aligned)
        s << "      {\n" << emit_operand(nodes[j], axis_k, false, rowv, "kg", lim + "LL", lo) << "      }\n    }\n";
      else
        s << "      if " << fastc << " {\n"
          << emit_operand(nodes[j], axis_k, false, rowv, "kg", lim + "LL", lo) << "      } else {\n"
          << emit_operand(nodes[j], axis_k, true, rowv, "kg", lim + "LL", lo) << "      }\n    }\n";
    }
    if (nodes.size() > 1)
      s << "    else {\n#pragma unroll\n      for (int e = 0; e < " << V << "; ++e) dst[e] = 0.0f;\n    }\n";
  }
  s << "  }\n  };\n";
  // stash: fp32 registers -> LDS [row][k] of the MFMA operand type
  s << "  auto stash" << X << " = [&](const int buf, const int st, const i64 k0_) {\n  (void)k0_;\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << per << "; ++i) {\n";
  s << "    const int sl = tid + i * " << sp.NT << ";\n";
  if (nslots % sp.NT) s << "    if (sl >= " << nslots << ") break;\n";
  if (axis_k) {
    s << "    const int rl = sl / " << kper << ", kl = (sl % " << kper << ") * " << V << ";\n";
    s << "    stv<" << V << ">(" << lds << " + buf * " << rows * sp.BKP << " + rl * " << sp.BKP << " + kl, r" << X
      << "[st][i]);\n";
  } else {
    s << "    const int kl = sl / " << rows / V << ", rl = (sl % " << rows / V << ") * " << V << ";\n";
    s << "#pragma unroll\n    for (int e = 0; e < " << V << "; ++e) " << lds << "[buf * " << rows * sp.BKP
      << " + (rl + e) * " << sp.BKP << " + kl] = fromf<" << T << ">(r" << X << "[st][i][e]);\n";
  }
  s << "  }\n  };\n";
  return s.str();
}

// ---------------------------------------------------------------------------
// Direct-to-LDS staging.
//
// A wave's `global_load_lds_dwordx4` moves 16 bytes per lane from global
// memory into 1 KiB of LDS at a wave-uniform address (lane i at +16 i), with
// no register round trip and no LDS write instruction; it is counted by
// vmcnt.  Measured on this part: a stream of LDS writes (ds_write_b128 of
// staged registers) runs at about 75 bytes per clock per compute unit
// whatever the lane-to-address mapping, and competes with the fragment reads;
// the same data staged by direct loads leaves the reads almost undisturbed.
//
// Layouts (16-bit operands, k-tiles of 64, one stage = A then B):
//   A [BM rows][64 k]: row r's 16-byte chunk c at position c ^ (r & 7).  One
//     load covers 8 rows, each lane fetching the chunk its position holds;
//     every 4 lanes still cover one aligned 64-byte segment of a row.  A
//     fragment read (16 rows x 4 chunks, 16 bytes per lane) then touches 16
//     distinct 16-byte bank groups per half-wave pair of lane octets.
//   B [64 k][BN n]: row k's chunk c at c ^ f(k), f chosen below; rows are BN
//     elements apart with no padding, so the stage is contiguous.
// The loads are issued from inline assembly (M0 holds the LDS address; no
// other code in these kernels uses M0): the compiler cannot tell the two
// stages apart and would otherwise wait for the next tile's loads before
// every fragment read of the current tile.  The waits are explicit (see
// dma_mainloop).

// XOR masks of the right operand's chunk index: f keeps every chunk inside its
// row and puts the two 16-byte chunks that each row of a half-wave of
// transposing reads touches (rows {0..3, 8..11} + 4 h of a 16-row block, the
// same chunk pair for all of them) on 16 distinct 16-byte bank groups of the
// 256-byte bank cycle.  f may not use bit 2 of k: the two reads of one
// fragment are 4 rows apart and share f.
static bool dma_b_swizzle(int P, int& x0, int& x1, int& x3) {
  static const int vals[] = {0, 2, 4, 6, 8, 10, 12, 14};
  for (int a : vals)
    for (int b : vals)
      for (int c : vals) {
        auto f = [&](int k) { return a * (k & 1) + b * ((k >> 1) & 1) + c * ((k >> 3) & 1); };
        bool ok = true;
        for (int k = 0; k < 16 && ok; ++k)
          for (int ch = 0; ch < P && ok; ++ch)
            if ((ch ^ f(k)) >= P) ok = false;
        for (int h = 0; h < 2 && ok; ++h)
          for (int c0 = 0; c0 + 1 < P && ok; c0 += 2) {
            bool used[16] = {};
            for (int r : {0, 1, 2, 3, 8, 9, 10, 11}) {
              const int k = r + 4 * h, u = (k * P + (c0 ^ f(k))) % 16;
              for (int d = 0; d < 2 && ok; ++d) {
                const int uu = (u + d) % 16;
                if (used[uu]) ok = false;
                used[uu] = true;
              }
            }
          }
        if (ok) {
          x0 = a, x1 = b, x3 = c;
          return true;
        }
      }
  return false;
}

static std::string dma_fk(const GemmSpec& sp, const std::string& k) {
  std::string r;
  auto term = [&](int x, const std::string& bit) {
    if (!x) return;
    r += std::string(r.empty() ? "" : " + ") + std::to_string(x) + " * " + bit;
  };
  term(sp.dx0, "((" + k + ") & 1)");
  term(sp.dx1, "(((" + k + ") >> 1) & 1)");
  term(sp.dx3, "(((" + k + ") >> 3) & 1)");
  return r.empty() ? "0" : "(" + r + ")";
}

void plan_dma(const KInfo& ki, GemmSpec& sp, bool ksplit) {
  sp.dma = false;
  const char* e = getenv("KORCH_GEMM_DMA");
  if (e && atoi(e) == 0) return;
  if (sp.conv || sp.mms.size() != 1 || sp.Bs.size() != 1 || !sp.b_kn) return;
  // With an intra-workgroup split of K the two groups' stages leave room for
  // the left operand one k-tile ahead only: the MLP block's second product then
  // took 34.0 us after a cache flush against 29.1 with register staging (26.7
  // against 27.3 warm), so the split keeps register staging unless asked.
  if (ksplit && !(getenv("KORCH_GEMM_DMA_KSPLIT") && atoi(getenv("KORCH_GEMM_DMA_KSPLIT")) != 0)) return;
  if (sp.mtype != KORCH_F16 && sp.mtype != KORCH_BF16) return;
  if (ki.in.count(sp.A) || ki.in.count(sp.Bs[0])) return;  // operands computed in the kernel
  if (sp.BK != 64 || sp.K % 64 || sp.M % sp.BM || sp.N % sp.BN || sp.BN % 16) return;
  if (sp.WM * sp.WN * 64 != sp.NT) return;  // every wave multiplies
  const int NW = sp.NT / 64;
  // a third right-operand stage (loaded two k-tiles ahead by wave groups of
  // their own) when it fits and the waves split into the three loading groups
  // an intra-workgroup split of K gives each of its two groups stages of their own
  const size_t lds = ksplit ? 80 * 1024 : 160 * 1024;
  sp.dsb = (size_t)(2 * sp.BM + 3 * sp.BN) * 64 * 2 <= lds && sp.K / 64 >= (ksplit ? 6 : 3) && NW % 4 == 0 &&
                   (sp.BM / 8) % (NW / 2) == 0 && (sp.BN / 8) % (NW / 4) == 0 && !getenv("KORCH_GEMM_DMA_2STAGE")
               ? 3
               : 2;
  if (sp.dsb == 2 && ((sp.BM / 8) % NW || (sp.BN / 8) % NW)) return;  // equal load counts per wave
  // deep staging when asked: S stages of each operand, both loaded S - 1
  // k-tiles ahead by G = S - 1 wave groups per operand (group g loads the
  // k-tiles j with j % G == g); S = 3, or 5 with KORCH_GEMM_DMA_STAGES=5 (one
  // wave per group: slower, 34.2 us warm against 30.0 for the MLP block's
  // second product, the same 37.5 after a cache flush)
  sp.dsa = 2;
  if (sp.dsb == 3 && (sp.want_a3 || (getenv("KORCH_GEMM_DMA_A3") && atoi(getenv("KORCH_GEMM_DMA_A3")) != 0))) {
    const char* se = getenv("KORCH_GEMM_DMA_STAGES");
    for (int S : {3, 5}) {
      if ((se ? atoi(se) : 3) != S) continue;
      const int G = S - 1;
      if (NW % (2 * G)) continue;
      const int per = NW / (2 * G);  // waves per loading group
      if ((size_t)(S * sp.BM + S * sp.BN) * 64 * 2 <= lds && (sp.BM / 8) % per == 0 && (sp.BN / 8) % per == 0) {
        sp.dsa = sp.dsb = S;
        break;
      }
    }
  }
  if ((size_t)(sp.dsa * sp.BM + sp.dsb * sp.BN) * 64 * 2 > lds) return;
  int x0 = 0, x1 = 0, x3 = 0;
  if (!dma_b_swizzle(sp.BN / 8, x0, x1, x3)) return;
  sp.dx0 = x0, sp.dx1 = x1, sp.dx3 = x3;
  sp.dma = true;
}

// LayerNorm fold: LDS byte offset of gamma and beta (K halves each) and the
// column sums gamma^T W, beta^T W (BN floats each), after the operand stages.
static int64_t ln_lds_off(const GemmSpec& sp) { return (int64_t)(sp.dsa * sp.BM + sp.dsb * sp.BN) * 64 * 2; }
static int64_t ln_lds_bytes(const GemmSpec& sp) { return sp.lnf ? 4 * sp.K + 8 * (int64_t)sp.BN : 0; }

// Which waves load what.  With two right-operand stages every wave loads
// blocks of both operands for the next k-tile (wave w: blocks w, w + NW, ...)
// and waits for all its loads before the barrier that ends the tile.  With
// three, the right operand is loaded two k-tiles ahead: waves [0, NW/2) load
// the left operand (one tile ahead), waves [NW/2, 3NW/4) the right operand's
// even k-tiles and waves [3NW/4, NW) its odd ones.  Each wave then waits
// (vmcnt 0) only at the end of a tile whose successor it loaded, when every
// load it has in flight is needed.  Partial waits (vmcnt > 0) are never used:
// direct-to-LDS loads were seen to complete out of issue order (a partial
// wait let a tile be read before its last loads had landed).
struct DmaRoles {
  int NW, ga, gb;   // waves; waves loading A; waves per B parity group
  int PA, PB;       // blocks per loading wave
};
static DmaRoles dma_roles(const GemmSpec& sp) {
  DmaRoles r;
  r.NW = sp.NT / 64;
  if (sp.dsa >= 3) {
    r.ga = r.gb = r.NW / (2 * (sp.dsa - 1));
  } else if (sp.dsb == 3) {
    r.ga = r.NW / 2, r.gb = r.NW / 4;
  } else {
    r.ga = r.NW, r.gb = r.NW;
  }
  r.PA = sp.BM / 8 / r.ga;
  r.PB = sp.BN / 8 / r.gb;
  return r;
}

// Per-wave load offsets and the staging lambdas `dmaA_(kt, st)` and
// `dmaB_(kt, st)` (each called only by the waves that load that operand).
static std::string dma_loader(const KInfo& ki, const GemmSpec& sp, const std::map<int, int>& slot) {
  const Graph& g = ki.g;
  const std::string T = ctype(sp.mtype);
  const DmaRoles R = dma_roles(sp);
  const int P = sp.BN / 8;
  const int64_t SAE = (int64_t)sp.BM * 64, SBE = (int64_t)sp.BN * 64, BOFF = sp.dsa * SAE;
  auto boff = [&](int node) {
    const Shape& sh = g.nodes[node].shape;
    Shape ob(sp.OUT.begin(), sp.OUT.begin() + sp.nb);
    Shape nbsh(sh.begin(), sh.end() - 2);
    std::vector<Ix> zc;
    for (int d = 0; d < sp.nb; ++d) zc.push_back(Ix::var("z" + std::to_string(d)));
    auto bi = broadcast_index(nbsh, ob, zc);
    auto st = strides_of(sh);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], 1));
    return off.at();
  };
  std::ostringstream s;
  s << "  // direct-to-LDS staging: " << sp.BM / 8 << " A blocks and " << sp.BN / 8 << " B blocks of 1 KiB per k-tile, "
    << sp.dsa << " A stages and " << sp.dsb << " B stages\n";
  s << "  const int wv_ = __builtin_amdgcn_readfirstlane(wave);\n";
  if (sp.dsa >= 3) {
    s << "  const int par_ = wv_ / " << R.ga << " % " << sp.dsa - 1 << ", wa_ = wv_ % " << R.ga << ", wb_ = wv_ % " << R.gb
      << ";  // the residue mod " << sp.dsa - 1 << " of the k-tiles the wave's group loads; loader index in the group\n";
  } else if (sp.dsb == 3) {
    s << "  const int wa_ = wv_, wb_ = (wv_ - " << R.ga << ") % " << R.gb << ", par_ = (wv_ - " << R.ga << ") / " << R.gb
      << ";  // A loader index; B loader index and k-tile parity\n";
  } else {
    s << "  const int wa_ = wv_, wb_ = wv_;\n";
  }
  s << "  const unsigned lds0_ = (unsigned)(size_t)(__attribute__((address_space(3))) void*)gsm_;\n";
  s << "  const " << T << "* Ag_ = (const " << T << "*)a.p[" << slot.at(sp.A) << "] + (" << boff(sp.A) << ");\n";
  s << "  const " << T << "* Bg_ = (const " << T << "*)a.p[" << slot.at(sp.Bs[0]) << "] + (" << boff(sp.Bs[0]) << ");\n";
  // element offsets of this lane's chunks at k-tile 0 (32-bit when both
  // operands have fewer than 2^31 elements); with three right-operand stages a
  // wave loads one operand only, and one array holds its offsets
  const bool small = (double)numel(g.nodes[sp.A].shape) < 2147483648.0 && (double)numel(g.nodes[sp.Bs[0]].shape) < 2147483648.0;
  const std::string OT_ = small ? "int" : "i64";
  const std::string aoffs = sp.dsb == 3 ? "doff_" : "doffA_", boffs = sp.dsb == 3 ? "doff_" : "doffB_";
  if (sp.dsb == 3)
    s << "  " << OT_ << " doff_[" << std::max(R.PA, R.PB) << "];\n";
  else
    s << "  " << OT_ << " doffA_[" << R.PA << "], doffB_[" << R.PB << "];\n";
  const int nA = sp.dsa >= 3 ? (sp.dsa - 1) * R.ga : R.ga;  // waves loading A
  if (sp.dsb == 3) s << "  if (wv_ < " << nA << ") {\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << R.PA << "; ++i) {\n";
  s << "    const int r = 8 * (wa_ + i * " << R.ga << ") + (l >> 3);\n";
  s << "    " << aoffs << "[i] = (" << OT_ << ")((m0 + r) * " << sp.K << "LL + (((l & 7) ^ (l >> 3)) * 8));\n  }\n";
  if (sp.dsb == 3) s << "  } else {\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << R.PB << "; ++i) {\n";
  s << "    const int q = (wb_ + i * " << R.gb << ") * 64 + l, k = q / " << P << ", p = q % " << P << ";\n";
  s << "    " << boffs << "[i] = (" << OT_ << ")((i64)k * " << sp.N << "LL + n0 + ((p ^ " << dma_fk(sp, "k") << ") * 8));\n  }\n";
  if (sp.dsb == 3) s << "  }\n";
  const char* ld = "      asm volatile(\"s_mov_b32 m0, %1\\n\\tglobal_load_lds_dwordx4 %0, off\" :: \"v\"(src), \"s\"(la) : \"memory\", \"m0\");\n";
  s << "  auto dmaA_ = [&](const int kt, const int st) {\n#pragma unroll\n    for (int i = 0; i < " << R.PA << "; ++i) {\n";
  s << "      const " << T << "* src = Ag_ + (i64)kt * 64 + " << aoffs << "[i];\n";
  s << "      const unsigned la = lds0_ + (unsigned)((st * " << SAE << " + (wa_ + i * " << R.ga << ") * 512) * 2);\n" << ld;
  s << "    }\n  };\n";
  s << "  auto dmaB_ = [&](const int kt, const int st) {\n#pragma unroll\n    for (int i = 0; i < " << R.PB << "; ++i) {\n";
  s << "      const " << T << "* src = Bg_ + (i64)kt * " << 64 * sp.N << "LL + " << boffs << "[i];\n";
  s << "      const unsigned la = lds0_ + (unsigned)((" << BOFF << " + st * " << SBE << " + (wb_ + i * " << R.gb
    << ") * 512) * 2);\n" << ld;
  s << "    }\n  };\n";
  return s.str();
}

// Main loop over the k-tiles with direct-to-LDS staging.  A tile j + 1 goes to
// the A stage tile j - 1 used and B tile j + dsb - 1 to the B stage tile j - 1
// used; both are issued as tile j's products start.
static std::string dma_mainloop(const GemmSpec& sp, int64_t kconst, bool kconst_exact) {
  std::ostringstream s;
  const std::string T = ctype(sp.mtype);
  const std::string V8 = sp.mtype == KORCH_F16 ? "f16x8" : "bf16x8";
  const std::string fn = sp.mtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16"
                                               : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
  const DmaRoles R = dma_roles(sp);
  const int SB = sp.dsb;
  const int64_t SAE = (int64_t)sp.BM * 64, SBE = (int64_t)sp.BN * 64, BOFF = sp.dsa * SAE;
  const int64_t LNO = ln_lds_off(sp);
  if (sp.lnf) {
    // gamma and beta into LDS once; per-lane row sums of X and X^2 (rows of the
    // lane's A fragments, its quarter of each k-step) and column sums of the
    // B fragments this wave owns (column blocks j with j % WM == wm)
    s << "  const " << T << "* lng_ = (const " << T << "*)(smem + " << LNO << ");\n";
    s << "  const " << T << "* lnb_ = lng_ + " << sp.K << ";\n";
    s << "  for (int t_ = tid; t_ < " << sp.K / 8 << "; t_ += " << sp.NT << ") {\n";
    s << "    *(uint4*)((" << T << "*)lng_ + 8 * t_) = *(const uint4*)((const " << T << "*)a.p[" << sp.lng_slot << "] + 8 * t_);\n";
    s << "    *(uint4*)((" << T << "*)lnb_ + 8 * t_) = *(const uint4*)((const " << T << "*)a.p[" << sp.lnb_slot << "] + 8 * t_);\n";
    s << "  }\n";
    const int TJ = (sp.FN + sp.WM - 1) / sp.WM;  // column blocks per wave
    s << "  float lnsx_[" << sp.FM << "] = {}, lnsq_[" << sp.FM << "] = {}, lncs_[" << TJ << "] = {}, lncc_[" << TJ << "] = {};\n";
    s << "  typedef _Float16 h2_ __attribute__((ext_vector_type(2)));\n";
  }
  s << "  auto compute = [&](const int sa, const int sb, const int kt) {\n";
  s << "    (void)kt;\n";
  s << "    const " << T << "* Ab = (const " << T << "*)gsm_ + sa * " << SAE << ";\n";
  s << "    const " << T << "* Bb = (const " << T << "*)gsm_ + " << BOFF << " + sb * " << SBE << ";\n";
  s << "#pragma unroll\n    for (int kk = 0; kk < 2; ++kk) {\n";
  s << "      " << V8 << " af[" << sp.FM << "], bf[" << sp.FN << "];\n";
  // row & 7 == l & 7: the fragment's rows start at multiples of 16
  s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i) af[i] = *(const " << V8 << "*)(Ab + (wm * " << sp.WTM
    << " + i * 16 + (l & 15)) * 64 + (((kk * 4 + (l >> 4)) ^ (l & 7)) * 8));\n";
  s << "#pragma unroll\n      for (int j = 0; j < " << sp.FN << "; ++j) {\n";
  s << "        const int k_ = kk * 32 + (l >> 4) * 8 + ((l & 15) >> 2), n_ = wn * " << sp.WTN << " + j * 16 + 4 * (l & 3);\n";
  s << "        bf[j] = __builtin_bit_cast(" << V8 << ", lds_tr_k8(Bb + k_ * " << sp.BN << " + (((n_ >> 3) ^ "
    << dma_fk(sp, "k_") << ") * 8) + (n_ & 7), " << sp.BN << "));\n      }\n";
  if (sp.lnf) {
    // the lane's eight k of this k-step: kt * 64 + kk * 32 + 8 (l >> 4) ..
    s << "      const " << V8 << " gs_ = *(const " << V8 << "*)(lng_ + kt * 64 + kk * 32 + 8 * (l >> 4));\n";
    s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i) {\n";
    s << "#pragma unroll\n        for (int h = 0; h < 4; ++h) {\n";
    s << "          const h2_ x2 = {af[i][2 * h], af[i][2 * h + 1]};\n";
    s << "          lnsx_[i] = __builtin_amdgcn_fdot2(x2, h2_{(_Float16)1.0f, (_Float16)1.0f}, lnsx_[i], false);\n";
    s << "          lnsq_[i] = __builtin_amdgcn_fdot2(x2, x2, lnsq_[i], false);\n";
    s << "        }\n";
    s << "        af[i] = af[i] * gs_;\n";
    s << "      }\n";
    s << "      const " << V8 << " bs_ = *(const " << V8 << "*)(lnb_ + kt * 64 + kk * 32 + 8 * (l >> 4));\n";
    // column block j belongs to the wave with wm == j % WM (a uniform branch;
    // the accumulator index j / WM is a constant of the unrolled loop)
    for (int j = 0; j < sp.FN; ++j) {
      const std::string J = std::to_string(j), T_ = std::to_string(j / sp.WM);
      s << "      if (wm == " << j % sp.WM << ") {\n";
      s << "#pragma unroll\n        for (int h = 0; h < 4; ++h) {\n";
      s << "          const h2_ w2 = {bf[" << J << "][2 * h], bf[" << J << "][2 * h + 1]};\n";
      s << "          lncs_[" << T_ << "] = __builtin_amdgcn_fdot2(w2, h2_{gs_[2 * h], gs_[2 * h + 1]}, lncs_[" << T_ << "], false);\n";
      s << "          lncc_[" << T_ << "] = __builtin_amdgcn_fdot2(w2, h2_{bs_[2 * h], bs_[2 * h + 1]}, lncc_[" << T_ << "], false);\n";
      s << "        }\n      }\n";
    }
  }
  s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n      for (int j = 0; j < " << sp.FN
    << "; ++j) acc[i][j] = " << fn << (sp.acc_t ? "(bf[j], af[i]" : "(af[i], bf[j]") << ", acc[i][j], 0, 0, 0);\n";
  s << "    }\n  };\n";
  const std::string W0 = "asm volatile(\"s_waitcnt vmcnt(0)\" ::: \"memory\");";
  s << "  const int nkt_ = kt1 - kt0;\n";
  // a folded LayerNorm's statistics leave too few registers for the unrolled loop
  const bool unrolled = kconst > 0 && kconst <= 128 && !sp.lnf;
  if (sp.dsa >= 3) {
    // 2G loading groups (G = S - 1): A and B, one group per residue of the
    // k-tile index mod G.  Group g loads tiles g, g + G, ...: tile j + G during
    // tile j when j % G == g, and waits at the end of tile j when
    // (j + 1) % G == g, before its tile j + 1 is read (it has issued nothing
    // since that tile, so the full wait waits for that tile only).
    const int S = sp.dsa, G = S - 1;
    const std::string isA = "wv_ < " + std::to_string(G * R.ga), Gs = std::to_string(G), Ss = std::to_string(S);
    s << "  if (par_ < nkt_) {\n    if (" << isA << ") dmaA_(kt0 + par_, par_);\n    else dmaB_(kt0 + par_, par_);\n  }\n";
    s << "  if (par_ == 0) " << W0 << "\n";
    s << "  __syncthreads();\n";
    if (unrolled) s << "#pragma unroll\n  for (int j = 0; j < " << kconst << "; ++j) {\n";
    else s << "  for (int j = 0; j < nkt_; ++j) {\n";
    s << "    if (par_ == j % " << Gs << " && j + " << Gs << " < nkt_) {\n";
    s << "      if (" << isA << ") dmaA_(kt0 + j + " << Gs << ", (j + " << Gs << ") % " << Ss << ");\n";
    s << "      else dmaB_(kt0 + j + " << Gs << ", (j + " << Gs << ") % " << Ss << ");\n    }\n";
    s << "    " << (kconst_exact ? "" : "if (j < nkt_) ") << "compute(j % " << Ss << ", j % " << Ss << ", kt0 + j);\n";
    s << "    if (par_ == (j + 1) % " << Gs << ") " << W0 << "\n";
    s << "    __syncthreads();\n  }\n";
  } else if (SB == 3) {
    const std::string isA = "wv_ < " + std::to_string(R.ga);
    // tiles 0 (A, even B loaders) and 1 (odd B loaders); the loaders of tile 0 wait
    s << "  if (" << isA << ") dmaA_(kt0, 0);\n";
    s << "  else if (par_ < nkt_) dmaB_(kt0 + par_, par_);\n";
    s << "  if (" << isA << " || par_ == 0) " << W0 << "\n";
    s << "  __syncthreads();\n";
    if (unrolled) s << "#pragma unroll\n  for (int j = 0; j < " << kconst << "; ++j) {\n";
    else s << "  for (int j = 0; j < nkt_; ++j) {\n";
    s << "    if (" << isA << ") {\n      if (j + 1 < nkt_) dmaA_(kt0 + j + 1, (j + 1) & 1);\n";
    s << "    } else if (par_ == (j & 1)) {\n      if (j + 2 < nkt_) dmaB_(kt0 + j + 2, (j + 2) % 3);\n    }\n";
    s << "    " << (kconst_exact ? "" : "if (j < nkt_) ") << "compute(j & 1, j % 3, kt0 + j);\n";
    // the A loaders and the loaders of B tile j + 1 wait for everything they issued
    s << "    if (" << isA << " || par_ != (j & 1)) " << W0 << "\n";
    s << "    __syncthreads();\n  }\n";
  } else {
    s << "  dmaA_(kt0, 0);\n  dmaB_(kt0, 0);\n  " << W0 << "\n  __syncthreads();\n";
    if (unrolled) s << "#pragma unroll\n  for (int j = 0; j < " << kconst << "; ++j) {\n";
    else s << "  for (int j = 0; j < nkt_; ++j) {\n";
    s << "    if (j + 1 < nkt_) {\n      dmaA_(kt0 + j + 1, (j + 1) & 1);\n      dmaB_(kt0 + j + 1, (j + 1) & 1);\n    }\n";
    s << "    " << (kconst_exact ? "" : "if (j < nkt_) ") << "compute(j & 1, j & 1, kt0 + j);\n";
    s << "    " << W0 << "\n    __syncthreads();\n  }\n";
  }
  if (sp.lnf) {
    // row statistics: the four lanes of a row (l, l ^ 16, l ^ 32, l ^ 48) hold
    // its four quarters; var = mean(X^2) - mu^2 (clamped at 0)
    s << "  float lnmu_[" << sp.FM << "], lnr_[" << sp.FM << "];\n";
    s << "#pragma unroll\n  for (int i = 0; i < " << sp.FM << "; ++i) {\n";
    s << "    float a_ = lnsx_[i], b_ = lnsq_[i];\n";
    s << "    a_ += __shfl_xor(a_, 16); a_ += __shfl_xor(a_, 32);\n";
    s << "    b_ += __shfl_xor(b_, 16); b_ += __shfl_xor(b_, 32);\n";
    s << "    const float mu_ = a_ * " << flit(1.0 / (double)sp.K) << ";\n";
    s << "    lnmu_[i] = mu_;\n";
    s << "    lnr_[i] = f_rsqrt(k_max(b_ * " << flit(1.0 / (double)sp.K) << " - mu_ * mu_, 0.0f) + " << flit(sp.lneps) << ");\n";
    s << "  }\n";
    // column sums of this wave's column blocks into LDS (after the operand stages)
    s << "  float* lns_ = (float*)(smem + " << LNO + 4 * sp.K << ");\n";
    s << "  float* lnc_ = lns_ + " << sp.BN << ";\n";
    for (int j = 0; j < sp.FN; ++j) {
      const std::string T_ = std::to_string(j / sp.WM);
      s << "  if (wm == " << j % sp.WM << ") {\n";
      s << "    float c0_ = lncs_[" << T_ << "], c1_ = lncc_[" << T_ << "];\n";
      s << "    c0_ += __shfl_xor(c0_, 16); c0_ += __shfl_xor(c0_, 32);\n";
      s << "    c1_ += __shfl_xor(c1_, 16); c1_ += __shfl_xor(c1_, 32);\n";
      s << "    if ((l >> 4) == 0) {\n";
      s << "      lns_[wn * " << sp.WTN << " + " << j * 16 << " + l] = c0_;\n";
      s << "      lnc_[wn * " << sp.WTN << " + " << j * 16 << " + l] = c1_;\n";
      s << "    }\n  }\n";
    }
    s << "  __syncthreads();\n";
  }
  return s.str();
}

// The MFMA main loop over k-tiles [kt0, kt1) of the contraction.
std::string mfma_mainloop(const GemmSpec& sp, const std::string& hook, int64_t kconst, bool kconst_exact, bool ctile) {
  std::ostringstream s;
  bool f32 = sp.mtype == KORCH_F32;
  std::string T = ctype(sp.mtype);
  s << "  f32x4 acc[" << sp.FM << "][" << sp.FN << "];\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n  for (int j = 0; j < " << sp.FN
    << "; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};\n";
  int nw = sp.WM * sp.WN;  // waves that own a sub-tile (the rest only stage operands)
  std::string wguard = nw < sp.NT / 64 ? "if (wave < " + std::to_string(nw) + ") " : "";
  if (sp.dma) {
    s << dma_mainloop(sp, kconst, kconst_exact);
  } else {
  s << "  auto compute = [&](const int buf) {\n";
  s << "    const " << T << "* Ab = As + buf * " << sp.BM * sp.BKP << ";\n";
  int64_t bbuf = b_buf_elems(sp);
  s << "    const " << T << "* Bb = Bs + buf * " << bbuf << ";\n";
  s << "#pragma unroll\n    for (int kk = 0; kk < " << sp.BK / sp.kstep << "; ++kk) {\n";
  if (f32) {
    s << "      float af[" << sp.FM << "], bf[" << sp.FN << "];\n";
    s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i) af[i] = Ab[(wm * " << sp.WTM
      << " + i * 16 + (l & 15)) * " << sp.BKP << " + kk * 4 + (l >> 4)];\n";
    if (sp.b_kn)
      s << "#pragma unroll\n      for (int j = 0; j < " << sp.FN << "; ++j) bf[j] = Bb[(kk * 4 + (l >> 4)) * " << sp.BNP
        << " + wn * " << sp.WTN << " + j * 16 + (l & 15)];\n";
    else
      s << "#pragma unroll\n      for (int j = 0; j < " << sp.FN << "; ++j) bf[j] = Bb[(wn * " << sp.WTN
        << " + j * 16 + (l & 15)) * " << sp.BKP << " + kk * 4 + (l >> 4)];\n";
    s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n      for (int j = 0; j < "
      << sp.FN << "; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bf[j], acc[i][j], 0, 0, 0);\n";
  } else {
    std::string V8 = sp.mtype == KORCH_F16 ? "f16x8" : "bf16x8";
    std::string fn = sp.mtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16"
                                           : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
    s << "      " << V8 << " af[" << sp.FM << "], bf[" << sp.FN << "];\n";
    s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i) af[i] = *(const " << V8 << "*)(Ab + (wm * "
      << sp.WTM << " + i * 16 + (l & 15)) * " << sp.BKP << " + kk * 32 + (l >> 4) * 8);\n";
    if (sp.b_kn)
      s << "#pragma unroll\n      for (int j = 0; j < " << sp.FN << "; ++j) bf[j] = __builtin_bit_cast(" << V8
        << ", lds_tr_k8(Bb + (kk * 32 + (l >> 4) * 8 + ((l & 15) >> 2)) * " << sp.BNP
        << (sp.BSH ? " + (kk * 4 + (l >> 4)) * " + std::to_string(sp.BSH) : std::string()) << " + wn * " << sp.WTN
        << " + j * 16 + 4 * (l & 3), " << sp.BNP << "));\n";
    else
      s << "#pragma unroll\n      for (int j = 0; j < " << sp.FN << "; ++j) bf[j] = *(const " << V8 << "*)(Bb + (wn * "
        << sp.WTN << " + j * 16 + (l & 15)) * " << sp.BKP << " + kk * 32 + (l >> 4) * 8);\n";
    s << "#pragma unroll\n      for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n      for (int j = 0; j < "
      << sp.FN << "; ++j) acc[i][j] = " << fn << (sp.acc_t ? "(bf[j], af[i]" : "(af[i], bf[j]")
      << ", acc[i][j], 0, 0, 0);\n";
  }
  s << "    }\n  };\n";
  // Register pipeline of NS stages over two LDS buffers: while tile t is
  // multiplied from LDS buffer t%2, tiles t+1 .. t+NS-1 are in registers or in
  // flight, and the loads of tile t+NS are issued into the stage tile t
  // occupied (it was staged to LDS before tile t's products).  Fetches are
  // unconditional (tile indices clamped to the last tile) so the compiler counts
  // outstanding loads exactly; with a compile-time tile count the loop is
  // unrolled completely (stage and buffer indices are then constants).
  auto clampk = [&](const std::string& t) {
    return "(i64)((" + t + ") < kt1 ? (" + t + ") : kt1 - 1) * " + std::to_string(sp.BK);
  };
  auto hookat = [&](const std::string& b) {
    if (hook.empty()) return std::string();
    return "    {\n      const " + T + "* Ab = As + (" + b + ") * " + std::to_string(sp.BM * sp.BKP) + ";\n" + hook + "    }\n";
  };
  const bool unrolled = kconst > 0 && kconst <= 128;
  const int NS = unrolled ? sp.NS : 2;
  // Split k-steps across the barrier: the fragments of a tile's last k-step
  // are read before the barrier that publishes the next tile's staging, and
  // that k-step's MFMAs run after it while the next tile's first fragments are
  // read, so no wave waits on LDS reads with the matrix cores idle after the
  // barrier.  Two fragment register sets alternate (even k-steps per tile).
  const int nkk = sp.BK / sp.kstep;
  const bool split_steps = unrolled && !f32 && hook.empty() && nkk >= 2 && nkk % 2 == 0 && sp.split_steps;
  if (split_steps) {
    const std::string V8 = sp.mtype == KORCH_F16 ? "f16x8" : "bf16x8";
    const std::string fn = sp.mtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16"
                                                 : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
    s << "  " << V8 << " af0[" << sp.FM << "], bf0[" << sp.FN << "], af1[" << sp.FM << "], bf1[" << sp.FN << "];\n";
    for (int h = 0; h < 2; ++h) {
      const std::string H = std::to_string(h);
      s << "  auto frag" << H << " = [&](const int buf, const int kk) {\n";
      s << "    const " << T << "* Ab = As + buf * " << sp.BM * sp.BKP << ";\n";
      s << "    const " << T << "* Bb = Bs + buf * " << bbuf << ";\n";
      s << "#pragma unroll\n    for (int i = 0; i < " << sp.FM << "; ++i) af" << H << "[i] = *(const " << V8 << "*)(Ab + (wm * "
        << sp.WTM << " + i * 16 + (l & 15)) * " << sp.BKP << " + kk * 32 + (l >> 4) * 8);\n";
      if (sp.b_kn)
        s << "#pragma unroll\n    for (int j = 0; j < " << sp.FN << "; ++j) bf" << H << "[j] = __builtin_bit_cast(" << V8
          << ", lds_tr_k8(Bb + (kk * 32 + (l >> 4) * 8 + ((l & 15) >> 2)) * " << sp.BNP
          << (sp.BSH ? " + (kk * 4 + (l >> 4)) * " + std::to_string(sp.BSH) : std::string()) << " + wn * " << sp.WTN
          << " + j * 16 + 4 * (l & 3), " << sp.BNP << "));\n";
      else
        s << "#pragma unroll\n    for (int j = 0; j < " << sp.FN << "; ++j) bf" << H << "[j] = *(const " << V8
          << "*)(Bb + (wn * " << sp.WTN << " + j * 16 + (l & 15)) * " << sp.BKP << " + kk * 32 + (l >> 4) * 8);\n";
      s << "  };\n";
      s << "  auto mma" << H << " = [&]() {\n#pragma unroll\n    for (int i = 0; i < " << sp.FM
        << "; ++i)\n#pragma unroll\n    for (int j = 0; j < " << sp.FN << "; ++j) acc[i][j] = " << fn
        << (sp.acc_t ? "(bf" + H + "[j], af" + H + "[i]" : "(af" + H + "[i], bf" + H + "[j]") << ", acc[i][j], 0, 0, 0);\n  };\n";
    }
    for (int st = 0; st < NS; ++st)
      s << "  fetchA(" << clampk("kt0 + " + std::to_string(st)) << ", " << st << "); fetchB("
        << clampk("kt0 + " + std::to_string(st)) << ", " << st << ");\n";
    s << "  stashA(0, 0, " << clampk("kt0") << "); stashB(0, 0, " << clampk("kt0") << ");\n  __syncthreads();\n";
    s << "  " << wguard << "frag0(0, 0);\n";
    std::string live = kconst_exact ? "" : "if (kt < kt1) ";
    s << "#pragma unroll\n  for (int j = 0; j < " << kconst << "; ++j) {\n";
    s << "    const int kt = kt0 + j, b_ = j & 1, s_ = j % " << NS << ", sn_ = (j + 1) % " << NS << ";\n";
    s << "    fetchA(" << clampk("kt + " + std::to_string(NS)) << ", s_); fetchB(" << clampk("kt + " + std::to_string(NS))
      << ", s_);\n";
    s << "    " << live << wguard << "{\n";
    for (int kk = 0; kk + 1 < nkk; ++kk) {
      const int cur = kk % 2, nxt = (kk + 1) % 2;
      s << "      frag" << nxt << "(b_, " << kk + 1 << ");\n      mma" << cur << "();\n";
    }
    s << "    }\n";
    s << "    stashA(1 - b_, sn_, " << clampk("kt + 1") << "); stashB(1 - b_, sn_, " << clampk("kt + 1") << ");\n";
    s << "    __syncthreads();\n";
    // after the barrier: the next tile's first fragments, then this tile's last k-step
    s << "    " << wguard << "{\n";
    s << "      if (j + 1 < " << kconst << ") frag0(1 - b_, 0);\n";
    s << "      " << live << "mma" << (nkk - 1) % 2 << "();\n";
    s << "    }\n";
    s << "  }\n";
  } else {
  for (int st = 0; st < NS; ++st)
    s << "  fetchA(" << clampk("kt0 + " + std::to_string(st)) << ", " << st << "); fetchB("
      << clampk("kt0 + " + std::to_string(st)) << ", " << st << ");\n";
  s << "  stashA(0, 0, " << clampk("kt0") << "); stashB(0, 0, " << clampk("kt0") << ");\n  __syncthreads();\n";
  if (unrolled) {
    // a split shorter than kconst skips the products of its missing tiles
    std::string live = kconst_exact ? "" : "if (kt < kt1) ";
    s << "#pragma unroll\n  for (int j = 0; j < " << kconst << "; ++j) {\n";
    s << "    const int kt = kt0 + j, b_ = j & 1, s_ = j % " << NS << ", sn_ = (j + 1) % " << NS << ";\n";
    s << "    fetchA(" << clampk("kt + " + std::to_string(NS)) << ", s_); fetchB(" << clampk("kt + " + std::to_string(NS))
      << ", s_);\n";
    s << "    " << live << wguard << "compute(b_);\n";
    if (!hook.empty()) s << "    " << live << "{\n" << hookat("b_") << "    }\n";
    s << "    stashA(1 - b_, sn_, " << clampk("kt + 1") << "); stashB(1 - b_, sn_, " << clampk("kt + 1") << ");\n";
    if (sp.sched_w > 0 && !f32 && hook.empty() && sp.BK / sp.kstep >= 2) {
      // Instruction groups for the scheduler: the fragment reads of the first
      // k-step, then its MFMAs each followed by one LDS write (staging of the
      // next k-tile) and one global load (the k-tile after), then the later
      // k-steps' reads and MFMAs.  The writes and loads then issue while the
      // matrix cores work instead of in a block before the barrier (measured:
      // 2-3 % on a 4096 x 768 x 3072 product with two k-steps per tile; no
      // gain with one k-step per tile, where every read precedes the MFMAs).
      const int R = sp.FM + (sp.b_kn ? 2 : 1) * sp.FN, M = sp.FM * sp.FN, nkk = sp.BK / sp.kstep;
      s << "    __builtin_amdgcn_sched_group_barrier(0x100, " << R << ", 0);\n";
      int w = sp.sched_w, gl = sp.sched_g, m = M;
      while (m > 0 && (w > 0 || gl > 0)) {
        s << "    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);\n";
        --m;
        if (w > 0) s << "    __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);\n", --w;
        if (gl > 0) s << "    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);\n", --gl;
      }
      if (m > 0) s << "    __builtin_amdgcn_sched_group_barrier(0x008, " << m << ", 0);\n";
      if (w > 0) s << "    __builtin_amdgcn_sched_group_barrier(0x200, " << w << ", 0);\n";
      if (gl > 0) s << "    __builtin_amdgcn_sched_group_barrier(0x020, " << gl << ", 0);\n";
      for (int kk = 1; kk < nkk; ++kk)
        s << "    __builtin_amdgcn_sched_group_barrier(0x100, " << R << ", 0);\n    __builtin_amdgcn_sched_group_barrier(0x008, "
          << M << ", 0);\n";
    }
    s << "    __syncthreads();\n  }\n";
  } else {
    auto step = [&](const std::string& b, const std::string& kt) {
      std::ostringstream o;
      o << "    fetchA(" << clampk(kt + " + 2") << ", " << b << "); fetchB(" << clampk(kt + " + 2") << ", " << b << ");\n";
      o << "    " << wguard << "compute(" << b << ");\n";
      o << hookat(b);
      o << "    stashA(1 - (" << b << "), 1 - (" << b << "), " << clampk(kt + " + 1") << "); stashB(1 - (" << b << "), 1 - ("
        << b << "), " << clampk(kt + " + 1") << ");\n";
      o << "    __syncthreads();\n";
      return o.str();
    };
    s << "  for (int kt = kt0; kt < kt1; kt += 2) {\n";
    s << step("0", "kt");
    s << "    if (kt + 1 >= kt1) break;\n";
    s << step("1", "(kt + 1)");
    s << "  }\n";
  }
  }
  }
  if (!ctile) return s.str();
  // accumulators -> LDS C tile (fp32)
  s << "  float* Cs = (float*)smem;\n";
  s << "  " << wguard << "{\n#pragma unroll\n  for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n  for (int j = 0; j < " << sp.FN
    << "; ++j)\n#pragma unroll\n  for (int r = 0; r < 4; ++r) Cs[(wm * " << sp.WTM << " + i * 16 + (l >> 4) * 4 + r) * "
    << sp.LDC << " + wn * " << sp.WTN << " + j * 16 + (l & 15)] = acc[i][j][r];\n  }\n";
  s << "  __syncthreads();\n";
  return s.str();
}

static size_t gemm_smem_bytes_fwd(const GemmSpec& sp) { return gemm_smem_bytes(sp); }

size_t gemm_smem_bytes(const GemmSpec& sp) {
  size_t bbuf = (size_t)b_buf_elems(sp);
  size_t ab = (size_t)2 * ((size_t)sp.BM * sp.BKP + bbuf) * dtype_bytes(sp.mtype);
  if (sp.dma) ab = (size_t)(sp.dsa * sp.BM + sp.dsb * sp.BN) * 64 * dtype_bytes(sp.mtype) + (size_t)ln_lds_bytes(sp);
  if (sp.acc_t) return std::max(ab, (size_t)sp.OSB);
  size_t c = (size_t)(sp.CROWS ? sp.CROWS : sp.BM) * sp.LDC * 4;
  return std::max(ab, c);
}

int reg_epilogue_output(const KInfo& ki, const GemmSpec& sp) {
  if (getenv("KORCH_GEMM_NO_REG_EPI") && atoi(getenv("KORCH_GEMM_NO_REG_EPI")) != 0) return -1;
  const Graph& g = ki.g;
  if (sp.conv || sp.mms.size() != 1 || sp.mtype == KORCH_F32 || sp.nmdims != 1 || !sp.rowred.empty() ||
      !sp.side.empty() || (int)sp.OUT.size() != sp.nb + 2 || ki.k.outs.size() != 1)
    return -1;
  const int o = ki.k.outs[0];
  const Node& on = g.nodes[o];
  if (on.shape != sp.OUT || dtype_bytes(on.dtype) != 2 || sp.N % 8 || sp.BN % 8) return -1;
  if (o != sp.mms[0] && !sp.epi.count(o)) return -1;
  // every value the epilogue reads other than the product is the same along
  // the rows (its dimension of the product's M axis is 1 or absent)
  const size_t mdim = (size_t)sp.nb;
  for (int v : sp.epi)
    for (int u : g.nodes[v].in) {
      if (sp.epi.count(u) || in_vec(sp.mms, u)) continue;
      const Shape& s = g.nodes[u].shape;
      const size_t lead = sp.OUT.size() - s.size();
      if (s.size() >= sp.OUT.size() - mdim && s[mdim - lead] != 1) return -1;
    }
  return o;
}

std::string gemm_reg_epilogue(const KInfo& ki, const GemmSpec& sp, const std::map<int, int>& slot, int o) {
  const Graph& g = ki.g;
  const Node& on = g.nodes[o];
  const std::string OT = ctype(on.dtype);
  Emitter em(g);
  em.inset = sp.epi;
  em.inset.insert(sp.mms[0]);
  em.argslot = slot;
  em.vec = 4;
  std::vector<Ix> it;
  for (int d = 0; d < sp.nb; ++d) it.push_back(Ix::var("z" + std::to_string(d)));
  it.push_back(Ix::var("m"));
  it.push_back(Ix::var("n", 1, 4));
  const std::string pkey = Emitter::key(sp.mms[0], broadcast_index(g.nodes[sp.mms[0]].shape, sp.OUT, it));
  em.provide = [&](int node, const std::vector<Ix>& idx, std::string* out) {
    if (node != sp.mms[0]) return false;
    if (Emitter::key(node, idx) != pkey) fail(KORCH_E_UNSUPPORTED, "gemm: epilogue reads the product at another index");
    // folded LayerNorm: r (acc - mu gamma^T W) + beta^T W
    *out = sp.lnf ? "(lnr_[i] * (acc[i][j][e] - lnmu_[i] * lns_[nl + e]) + lnc_[nl + e])" : "acc[i][j][e]";
    return true;
  };
  const std::string v = em.value(o, broadcast_index(on.shape, sp.OUT, it));
  // element offset of (z.., m, n) in the contiguous output
  std::string zoff = "0";
  for (int d = 0; d < sp.nb; ++d) zoff = "(" + zoff + ") * " + std::to_string(sp.OUT[d]) + "LL + z" + std::to_string(d);
  std::ostringstream s;
  s << "  " << OT << "* Os = (" << OT << "*)smem;  // output tile in its storage dtype\n";
  // In phases, one per row of 16x16 fragments (FM of them): a phase evaluates
  // the epilogue of its fragments into Os, waits at a barrier, and stores those
  // 16 rows of every wave row while the next phase computes, so the output
  // stores drain under the epilogue's arithmetic instead of after it (the MLP
  // block's first product with its GELU: 26.5 us against 28.0 warm, the same
  // bytes).  Phases write disjoint rows of Os: no barrier between a phase's
  // stores and the next phase's writes.  KORCH_GEMM_EPI_PHASES=0: one phase.
  const char* pe_env = getenv("KORCH_GEMM_EPI_PHASES");
  const int NPH = pe_env && atoi(pe_env) == 0 ? 1 : sp.FM;
  const int FPH = sp.FM / NPH;  // fragment rows per phase
  // tiles that divide the problem need no bounds checks; without the
  // per-block branch the compiler interleaves the blocks' epilogue chains
  const bool full = sp.M % sp.BM == 0 && sp.N % sp.BN == 0;
  const std::string inb = full ? "true" : "m < " + std::to_string(sp.M) + "LL && n < " + std::to_string(sp.N) + "LL";
  const int vr = sp.BN / 8;  // 16-byte vectors per tile row
  const bool big = (double)numel(on.shape) * 2 >= 2147483648.0 ||
                   (getenv("KORCH_OUT_PLAIN") && atoi(getenv("KORCH_OUT_PLAIN")) != 0);
  std::string P = "((" + OT + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])";
  const int PR = 16 * FPH;  // rows of each wave row per phase
  s << "#pragma unroll\n  for (int h_ = 0; h_ < " << NPH << "; ++h_) {\n";
  // waves beyond WM x WN only stage operands and hold no accumulators
  if (sp.WM * sp.WN < sp.NT / 64) s << "  if (wave < " << sp.WM * sp.WN << ")\n";
  s << "#pragma unroll\n  for (int i = h_ * " << FPH << "; i < (h_ + 1) * " << FPH << "; ++i)\n#pragma unroll\n  for (int j = 0; j < "
    << sp.FN << "; ++j) {\n";
  s << "    const int ml = wm * " << sp.WTM << " + i * 16 + (l & 15), nl = wn * " << sp.WTN << " + j * 16 + 4 * (l >> 4);\n";
  s << "    const i64 m = m0 + ml, n = n0 + nl;\n";
  s << "    float _o[4] = {0.0f, 0.0f, 0.0f, 0.0f};\n";
  s << "    if (" << inb << ") {\n" << em.pre.str();
  s << "#pragma unroll\n      for (int e = 0; e < 4; ++e) {\n" << em.body.str() << "        _o[e] = " << v << ";\n      }\n";
  s << "    }\n";
  s << "    typedef " << OT << " OT4 __attribute__((ext_vector_type(4)));\n";
  s << "    *(OT4*)(Os + ml * " << sp.OSP << " + nl) = OT4{(" << OT << ")_o[0], (" << OT << ")_o[1], (" << OT << ")_o[2], ("
    << OT << ")_o[3]};\n";
  // one block at a time: hoisting every block's chain (no branch separates
  // them) would need more registers than a wave has and spill
  s << "    __builtin_amdgcn_sched_barrier(0);\n";
  s << "  }\n  __syncthreads();\n";
  // this phase's rows: wave row w's rows w * WTM + h_ * PR + [0, PR)
  s << "  for (int s_ = tid; s_ < " << sp.WM * PR * vr << "; s_ += " << sp.NT << ") {\n";
  s << "    const int r_ = s_ / " << vr << ", ml = (r_ / " << PR << ") * " << sp.WTM << " + h_ * " << PR << " + r_ % " << PR
    << ", nl = (s_ % " << vr << ") * 8;\n";
  s << "    const i64 m = m0 + ml, n = n0 + nl;\n";
  s << "    if (" << inb << ") {\n";
  s << "      const uint4 v_ = *(const uint4*)(Os + ml * " << sp.OSP << " + nl);\n";
  s << "      const i64 off = ((" << zoff << ") * " << sp.M << "LL + m) * " << sp.N << "LL + n;\n";
  if (big)
    s << "      *(uint4*)(" << P << " + off) = v_;\n";
  else
    s << "      st16_out(" << P << ", off * 2, v_);\n";
  s << "    }\n  }\n  }\n";
  return s.str();
}

// Pointwise epilogue over the C tile: every kernel output at (batch, m, n).
std::string gemm_epilogue(const KInfo& ki, const GemmSpec& sp, const std::map<int, int>& slot,
                          const std::string& cs_row, const std::set<int>& skip, int conv_tw, int rows,
                          const std::string& row0, std::string* hoisted) {
  const Graph& g = ki.g;
  int maxb = 2;
  for (int o : ki.k.outs) maxb = std::max(maxb, dtype_bytes(g.nodes[o].dtype));
  int VE = 16 / maxb;
  while (VE > 1 && (sp.N % VE || sp.BN % VE)) VE /= 2;
  int cols = (int)std::min<int64_t>(sp.BN, sp.mms.size() > 1 ? sp.N : sp.BN);
  cols = (cols + VE - 1) / VE * VE;
  // every column a tile covers lies inside the product (no check needed)
  const bool n_full = sp.mms.size() > 1 ? cols == sp.N : sp.N % sp.BN == 0;
  Emitter em(g);
  em.inset = sp.epi;
  for (int m : sp.mms) em.inset.insert(m);
  em.argslot = slot;
  em.vec = VE;
  // iteration coordinates of OUT
  std::vector<Ix> it;
  for (int d = 0; d < sp.nb; ++d) it.push_back(Ix::var("z" + std::to_string(d)));
  if (sp.conv) {
    it.push_back(Ix::var("oy"));
    it.push_back(Ix::var("ox"));
  } else {
    it.push_back(Ix::var("m"));
  }
  it.push_back(Ix::var("n", 1, VE));
  if (sp.NT % (cols / VE) == 0) {
    // every element of a thread has the same column vector
    for (size_t d = 0; d + 1 < it.size(); ++d) em.varying.push_back(it[d].b);
    em.inv_defs = "const i64 n = n0 + (i64)((tid % " + std::to_string(cols / VE) + ") * " + std::to_string(VE) + ");";
    em.inv_guard = "n < " + std::to_string(sp.N) + "LL";
  }
  std::map<std::string, std::string> canon;
  // C tile values of a full-width product are read into registers with 16-byte
  // LDS reads before the element loop (rows start 16-byte aligned: LDC and the
  // column offsets are multiples of 4)
  std::ostringstream cvload;
  for (size_t j = 0; j < sp.mms.size(); ++j) {
    int mm = sp.mms[j];
    auto bi = broadcast_index(g.nodes[mm].shape, sp.OUT, it);
    std::string base = cs_row + " + " + std::to_string(sp.mms.size() > 1 ? sp.offj[j] : 0);
    if (sp.Nj[j] == 1 && sp.N != 1) {
      canon[Emitter::key(mm, bi)] = "Cs[" + base + "]";
    } else if (VE % 4 == 0) {
      std::string cv = "_cv" + std::to_string(j);
      cvload << "      float " << cv << "[" << VE << "];\n#pragma unroll\n      for (int q = 0; q < " << VE / 4
             << "; ++q) *(float4*)&" << cv << "[4 * q] = *(const float4*)&Cs[" << base << " + nl + 4 * q];\n";
      canon[Emitter::key(mm, bi)] = cv + "[e]";
    } else {
      canon[Emitter::key(mm, bi)] = "Cs[" + base + " + nl + e]";
    }
  }
  em.provide = [&](int node, const std::vector<Ix>& idx, std::string* out) {
    if (!in_vec(sp.mms, node)) return false;
    auto f = canon.find(Emitter::key(node, idx));
    if (f == canon.end()) fail(KORCH_E_UNSUPPORTED, "gemm: epilogue reads the product at another index");
    *out = f->second;
    return true;
  };
  std::ostringstream decl, after;
  for (int o : ki.k.outs) {
    if (skip.count(o)) continue;
    const Node& on = g.nodes[o];
    auto bi = broadcast_index(on.shape, sp.OUT, it);
    std::string v = em.value(o, bi);
    std::string T = ctype(on.dtype);
    std::string P = "((" + T + "*)a.p[" + std::to_string(ki.out_slot(o)) + "])";
    auto st = strides_of(on.shape);
    Ix off = Ix::k(0);
    for (size_t d = 0; d < bi.size(); ++d) off = ix_add(off, ix_mulk(bi[d], st[d], VE));
    if (on.shape == sp.OUT && off.affine && off.c == 1 && off.al % VE == 0) {
      std::string arr = "_o" + std::to_string(o);
      decl << "      float " << arr << "[" << VE << "];\n";
      em.body << "        " << arr << "[e] = " << v << ";\n";
      after << "      " << out_store(g, o, P, off.b, VE, arr) << ";\n";
    } else {
      std::string cond;
      int lead = (int)sp.OUT.size() - (int)on.shape.size();
      for (int d = 0; d < (int)sp.OUT.size(); ++d) {
        bool bc = d < lead || (on.shape[d - lead] == 1 && sp.OUT[d] != 1);
        if (!bc) continue;
        if (!cond.empty()) cond += " && ";
        cond += "(" + it[d].at() + " == 0)";
      }
      em.body << "        if (" << (cond.empty() ? "true" : cond) << ") " << out_store(g, o, P, off.at(), 0, v) << ";\n";
    }
  }
  std::ostringstream s;
  if (hoisted)
    *hoisted += em.inv.str();
  else
    s << em.inv.str();
  if (rows <= 0) rows = sp.BM;
  // An epilogue that reads tensors per element (a residual, say) runs a
  // fixed-trip unrolled loop when every thread has the same number of vectors:
  // the compiler then issues all of a thread's loads before the first is used
  // (a runtime-bounded loop loads, waits and stores one vector at a time).
  const int nvec_ = rows * (cols / VE);
  if (conv_tw <= 0 && sp.M % sp.BM == 0 && n_full && nvec_ % sp.NT == 0 && nvec_ / sp.NT <= 8 &&
      em.n_vector + em.n_gather > 0) {
    // Every thread stores nvec_ / NT vectors and none is guarded: the loads of
    // all of them (C tile and tensors read per element) are written out first,
    // then the arithmetic and stores of each.  A loop would load, wait and
    // store one vector at a time (the compiler cannot move a load above a store
    // to another tensor), a round trip to memory per vector.
    const int T_ = nvec_ / sp.NT;
    std::string setup = "    const int s_ = tid + IT_ * " + std::to_string(sp.NT) + ";\n    const int mlc = s_ / " +
                        std::to_string(cols / VE) + ", ml = " + row0 + " + mlc, nl = (s_ % " + std::to_string(cols / VE) +
                        ") * " + std::to_string(VE) + ";\n    (void)mlc;\n    const i64 m = m0 + ml, n = n0 + nl;\n    (void)m; (void)n;\n";
    std::string loads = setup + cvload.str() + em.pre.str();
    std::string rest = decl.str() + "#pragma unroll\n      for (int e = 0; e < " + std::to_string(VE) + "; ++e) {\n" +
                       em.body.str() + "      }\n" + after.str();
    // names of one vector's code get the vector's suffix; hoisted (ix / iu)
    // values and everything defined outside are left alone
    static const std::regex id(R"(\b(s_|mlc|ml|nl|m|n|_(?!ix|iu)[a-z]+[0-9]+)\b)");
    auto renamed = [&](const std::string& t, int it) {
      std::string r = std::regex_replace(t, id, "$1_v" + std::to_string(it));
      return std::regex_replace(r, std::regex(R"(\bIT_\b)"), std::to_string(it));
    };
    s << "  {\n";
    for (int it = 0; it < T_; ++it) s << renamed(loads, it);
    for (int it = 0; it < T_; ++it) s << "    {\n" << renamed(rest, it) << "    }\n";
    s << "  }\n";
    return s.str();
  }
  s << "  for (int s_ = tid; s_ < " << nvec_ << "; s_ += " << sp.NT << ") {\n";
  s << "    const int mlc = s_ / " << cols / VE << ", ml = " << row0 << " + mlc, nl = (s_ % " << cols / VE << ") * " << VE
    << ";\n";
  s << "    (void)mlc;\n";
  if (conv_tw > 0) {
    // C tile row ml is pixel (ml / conv_tw, ml % conv_tw) of a 2-D output tile at (ty0, tx0)
    s << "    const i64 oy = ty0 + ml / " << conv_tw << ", ox = tx0 + ml % " << conv_tw << ", n = n0 + nl;\n";
    std::string c;
    if (sp.Ho % (rows / conv_tw)) c += "oy < " + std::to_string(sp.Ho) + "LL";
    if (sp.Wo % conv_tw) c += std::string(c.empty() ? "" : " && ") + "ox < " + std::to_string(sp.Wo) + "LL";
    if (!n_full) c += std::string(c.empty() ? "" : " && ") + "n < " + std::to_string(sp.N) + "LL";
    s << "    if (" << (c.empty() ? "true" : c) << ") {\n";
  } else {
    s << "    const i64 m = m0 + ml, n = n0 + nl;\n";
    std::string c;
    if (sp.M % sp.BM) c += "m < " + std::to_string(sp.M) + "LL";
    if (!n_full) c += std::string(c.empty() ? "" : " && ") + "n < " + std::to_string(sp.N) + "LL";
    s << "    if (" << (c.empty() ? "true" : c) << ") {\n";
    if (sp.conv) s << "      const i64 oy = m / " << sp.Wo << "LL, ox = m % " << sp.Wo << "LL;\n";
  }
  s << cvload.str() << em.pre.str() << decl.str();
  s << "#pragma unroll\n      for (int e = 0; e < " << VE << "; ++e) {\n" << em.body.str() << "      }\n";
  s << after.str() << "    }\n  }\n";
  return s.str();
}

std::string gemm_prologue_common(const GemmSpec& sp) {
  std::ostringstream s;
  std::string T = ctype(sp.mtype);
  s << "  __shared__ __attribute__((aligned(16))) char smem[" << gemm_smem_bytes(sp) << "];\n";
  s << "  " << T << "* As = (" << T << "*)smem;\n";
  s << "  " << T << "* Bs = As + " << 2 * sp.BM * sp.BKP << ";\n";
  s << "  const int tid = threadIdx.x, l = tid & 63, wave = tid >> 6;\n";
  s << "  const int wm = wave / " << sp.WN << ", wn = wave % " << sp.WN << ";\n";
  s << "  (void)wm; (void)wn;\n";
  return s.str();
}

// Eight waves over the whole contraction, both operands staged direct-to-LDS
// three k-tiles deep (loaded two k-tiles ahead), in place of the
// intra-workgroup split of K (whose two groups of stages leave room for the
// left operand one k-tile ahead only); asked for with KORCH_GEMM_DMA8=1.  The
// MLP block's second product (4096 x 768 x 3072, 128 x 96 tiles, waves of
// 32 x 48) alone took 30.0 us warm and 37.6 after a 512 MiB read, against 32.1
// and 40.9 with the split and register staging (33.4 / 46.8 with eight waves
// and two left-operand stages).  Inside the block's flushed step, after the
// first product has written its left operand, it takes 31.0 us against 29.5
// (26.5 against 29.1 warm): the split keeps two groups' loads in flight, twice
// the bytes, while the weights come from HBM.  The split stays the default.
static bool eight_wave_dma(const KInfo& ki, GemmSpec& sp, int64_t tiles, int64_t KT) {
  const char* e = getenv("KORCH_GEMM_DMA8");
  if (!(e && atoi(e) != 0)) return false;
  if (sp.conv || sp.lnf || sp.mms.size() != 1 || tiles > 256 || KT < 16 || sp.NT != 256) return false;
  if (sp.BM % 32 || sp.BN % 32) return false;
  GemmSpec t = sp;
  t.WM = sp.BM / 32;
  t.WN = 2;
  t.NT = 64 * t.WM * t.WN;
  if (t.NT != 512) return false;
  t.WTM = t.BM / t.WM;
  t.WTN = t.BN / t.WN;
  t.FM = t.WTM / 16;
  t.FN = t.WTN / 16;
  t.want_a3 = true;
  plan_dma(ki, t, false);
  if (!t.dma || t.dsa < 3) return false;
  if (t.WM > 1 && !getenv("KORCH_GEMM_FULL_CTILE")) t.CROWS = t.WTM;
  sp = t;
  return true;
}

GenKernel gen_gemm(const KInfo& ki, int index) {
  GemmSpec sp;
  std::string why;
  if (!analyze_gemm(ki, sp, &why, false)) fail(KORCH_E_UNSUPPORTED, why);
  if (sp.conv && conv_uses_direct(sp, nullptr)) return gen_conv_direct(ki, sp, index);
  if (sp.conv && !sp.pro.empty()) fail(KORCH_E_UNSUPPORTED, "conv: a weight prologue needs the direct kernel");
  choose_tiles(sp, false);
  plan_operands(ki, sp);
  if ((sp.K + sp.BK - 1) / sp.BK > 128) sp.NS = 2;  // long contractions use the rolled loop
  if (sp.WM > 1 && !getenv("KORCH_GEMM_FULL_CTILE")) sp.CROWS = sp.WTM;
  GenKernel gk;
  gk.family = sp.conv ? KORCH_FAM_CONV : KORCH_FAM_GEMM;
  gk.name = kernel_name(index, sp.conv ? "conv" : "gemm");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  int64_t ntn = sp.mms.size() > 1 ? 1 : (sp.N + sp.BN - 1) / sp.BN;
  int64_t ntm = (sp.M + sp.BM - 1) / sp.BM;
  int64_t KT = (sp.K + sp.BK - 1) / sp.BK;
  // Intra-workgroup split of the contraction: when the tiles leave at most one
  // workgroup per compute unit (one wave per SIMD, which then waits alone on
  // its loads, LDS traffic and barriers) and K is long, the workgroup runs two
  // groups of four waves, each over half of the k-tiles with operand buffers
  // of its own, and adds the second group's accumulators to the first group's
  // in the C tile (a fixed order).  Eight waves per compute unit then issue
  // MFMAs and loads, one group's waits covered by the other's products.
  const size_t op_bytes = (size_t)2 * ((size_t)sp.BM * sp.BKP + (size_t)b_buf_elems(sp)) * dtype_bytes(sp.mtype);
  const size_t ksplit_lds = std::max(2 * op_bytes, (size_t)sp.BM * sp.LDC * 4);
  const bool dma8 = eight_wave_dma(ki, sp, ntn * ntm * sp.batch, KT);
  const bool ksplit = !dma8 && !sp.conv && !sp.lnf && sp.mms.size() == 1 && ntn * ntm * sp.batch <= 256 && KT >= 16 &&
                      sp.NT == 256 && ksplit_lds <= 160 * 1024 && !getenv("KORCH_GEMM_NO_KSPLIT");
  const int64_t KH = (KT + 1) / 2;
  {
    // register relief 1: a tile's k-steps all before the barrier (one set of
    // fragment registers)
    const char* e = getenv("KORCH_GEMM_SPLIT_STEPS");
    sp.split_steps = !(e && atoi(e) == 0) && reg_relief() < 1;
  }
  const int repi_out = ksplit ? -1 : reg_epilogue_output(ki, sp);
  if (repi_out >= 0) {
    sp.acc_t = true;
    sp.OSP = sp.BN + 8;
    sp.OSB = sp.BM * sp.OSP * 2;
  }
  plan_dma(ki, sp, ksplit);
  // with direct-to-LDS staging each k-group's operand stages take (dsa BM + dsb BN) x 64 elements
  const size_t grp_bytes = sp.dma ? (size_t)(sp.dsa * sp.BM + sp.dsb * sp.BN) * 64 * dtype_bytes(sp.mtype) : op_bytes;
  const size_t ksplit_lds_ = std::max(2 * grp_bytes, (size_t)sp.BM * sp.LDC * 4);
  if (sp.lnf) {
    // the fold needs direct-to-LDS staging (X tiles in their swizzled layout),
    // the register epilogue (each lane holds its rows' statistics) and fp16
    if (!sp.dma || !sp.acc_t || sp.mtype != KORCH_F16 || ksplit || sp.K % 64)
      fail(KORCH_E_UNSUPPORTED, "gemm: a folded LayerNorm needs fp16 tiles that divide the problem and the register epilogue");
    sp.lng_slot = slot.at(sp.lng);
    sp.lnb_slot = slot.at(sp.lnb);
    if (gemm_smem_bytes(sp) > 160 * 1024) fail(KORCH_E_UNSUPPORTED, "gemm: folded LayerNorm exceeds the LDS");
  }
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  if (ksplit) {
    const std::string T = ctype(sp.mtype);
    s << "extern \"C\" __global__ void __launch_bounds__(512) " << gk.name << "(KArgs a) {\n";
    s << "  __shared__ __attribute__((aligned(16))) char smem[" << ksplit_lds_ << "];\n";
    s << "  const int kgrp = threadIdx.x >> 8;  // which half of the k-tiles\n";
    if (sp.dma)
      s << "  char* gsm_ = smem + __builtin_amdgcn_readfirstlane(kgrp) * " << grp_bytes
        << ";  // this group's operand stages (wave-uniform)\n";
    s << "  " << T << "* As = (" << T << "*)(smem + kgrp * " << op_bytes << ");\n";
    s << "  " << T << "* Bs = As + " << 2 * sp.BM * sp.BKP << ";\n";
    s << "  const int tid = threadIdx.x & 255, l = tid & 63, wave = tid >> 6;\n";
    s << "  const int wm = wave / " << sp.WN << ", wn = wave % " << sp.WN << ";\n";
    s << "  (void)wm; (void)wn;\n";
  } else {
    s << "extern \"C\" __global__ void __launch_bounds__(" << sp.NT << ") " << gk.name << "(KArgs a) {\n";
    s << gemm_prologue_common(sp);
    if (sp.dma) s << "  char* gsm_ = smem;  // operand stages\n";
  }
  // Workgroups are dispatched round-robin over the 8 XCDs, each with its own
  // L2.  Renumber them so every XCD owns a contiguous range of tiles, and order
  // tiles in groups of GM row-tiles so the tiles running together on one XCD
  // share their A row-panels and B column-panels in that XCD's L2.
  int64_t total = ntn * ntm * sp.batch;
  int64_t GM = std::min<int64_t>(8, ntm);
  s << "  const int wg = blockIdx.x, xcd = wg % 8, jx = wg / 8;\n";
  s << "  const int q = xcd * " << total / 8 << " + (xcd < " << total % 8 << " ? xcd : " << total % 8 << ") + jx;\n";
  s << "  const int bz_ = q / " << ntm * ntn << ", r_ = q % " << ntm * ntn << ";\n";
  s << "  const int grp = r_ / " << GM * ntn << ", first = grp * " << GM << ";\n";
  s << "  const int gs = " << ntm << " - first < " << GM << " ? " << ntm << " - first : " << GM << ";\n";
  s << "  const int tm = first + (r_ % " << GM * ntn << ") % gs, tn = (r_ % " << GM * ntn << ") / gs;\n";
  s << "  const i64 n0 = (i64)tn * " << sp.BN << ", m0 = (i64)tm * " << sp.BM << ";\n";
  s << "  i64 q_ = bz_;\n";
  for (int d = sp.nb - 1; d >= 0; --d)
    s << "  const i64 z" << d << " = q_ % " << sp.OUT[d] << "LL; q_ /= " << sp.OUT[d] << "LL;\n";
  if (ksplit)
    s << "  const int kt0 = kgrp * " << KH << ", kt1 = kt0 + " << KH << " < " << KT << " ? kt0 + " << KH << " : " << KT
      << ";\n";
  else
    s << "  const int kt0 = 0, kt1 = " << KT << ";\n";
  {
    // scheduling hints when both operands are plain tensors staged by buffer loads
    const bool hints = !getenv("KORCH_GEMM_SCHED") || atoi(getenv("KORCH_GEMM_SCHED")) != 0;
    const int C = 16 / dtype_bytes(sp.mtype);
    if (hints && sp.mtype != KORCH_F32 && !buffer_loader(ki, sp, true, slot).empty() &&
        !buffer_loader(ki, sp, false, slot).empty()) {
      const int perA = (sp.BM * (sp.BK / C) + sp.NT - 1) / sp.NT;
      const int perB = (sp.BK * (sp.BN / C) + sp.NT - 1) / sp.NT;
      sp.sched_w = sp.sched_g = perA + perB;
    }
  }
  if (sp.dma) {
    s << dma_loader(ki, sp, slot);
  } else {
    s << operand_loader(ki, sp, true, slot);
    s << operand_loader(ki, sp, false, slot);
  }
  if (ksplit) {
    s << mfma_mainloop(sp, "", KH, KT % 2 == 0, false);
    s << "  float* Cs = (float*)smem;\n";
    auto ctile = [&](const char* op) {
      std::ostringstream o;
      o << "#pragma unroll\n    for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n    for (int j = 0; j < " << sp.FN
        << "; ++j)\n#pragma unroll\n    for (int r = 0; r < 4; ++r) Cs[(wm * " << sp.WTM << " + i * 16 + (l >> 4) * 4 + r) * "
        << sp.LDC << " + wn * " << sp.WTN << " + j * 16 + (l & 15)] " << op << " acc[i][j][r];\n";
      return o.str();
    };
    s << "  if (kgrp == 0) {\n" << ctile("=") << "  }\n  __syncthreads();\n";
    s << "  if (kgrp == 1) {\n" << ctile("+=") << "  }\n  __syncthreads();\n";
    s << "  {\n  const int tid = threadIdx.x;\n";
    GemmSpec ep = sp;
    ep.NT = 512;
    s << gemm_epilogue(ki, ep, slot, "ml * " + std::to_string(sp.LDC));
    s << "  }\n";
  } else if (sp.acc_t) {
    s << mfma_mainloop(sp, "", KT, true, false);
    s << gemm_reg_epilogue(ki, sp, slot, repi_out);
  } else if (sp.CROWS && sp.CROWS < sp.BM) {
    // The C tile passes through LDS one band of wave rows at a time (waves
    // with wm == p write rows [p*WTM, (p+1)*WTM), then every thread runs the
    // epilogue over them), so the fp32 staging area is WTM rows, not BM: the
    // operand buffers then bound the LDS of a workgroup and more workgroups
    // fit on a compute unit.
    s << mfma_mainloop(sp, "", KT, true, false);
    s << "  float* Cs = (float*)smem;\n";
    s << "  for (int p_ = 0; p_ < " << sp.WM << "; ++p_) {\n";
    s << "    if (p_ > 0) __syncthreads();\n";
    s << "    if (wm == p_) {\n#pragma unroll\n    for (int i = 0; i < " << sp.FM << "; ++i)\n#pragma unroll\n    for (int j = 0; j < "
      << sp.FN << "; ++j)\n#pragma unroll\n    for (int r = 0; r < 4; ++r) Cs[(i * 16 + (l >> 4) * 4 + r) * " << sp.LDC
      << " + wn * " << sp.WTN << " + j * 16 + (l & 15)] = acc[i][j][r];\n    }\n";
    s << "    __syncthreads();\n";
    s << gemm_epilogue(ki, sp, slot, "mlc * " + std::to_string(sp.LDC), {}, 0, sp.CROWS,
                       "p_ * " + std::to_string(sp.CROWS));
    s << "  }\n";
  } else {
    s << mfma_mainloop(sp, "", KT);
    s << gemm_epilogue(ki, sp, slot, "ml * " + std::to_string(sp.LDC));
  }
  s << "}\n";
  gk.source = s.str();
  gk.grid[0] = (int)total;
  gk.block[0] = ksplit ? 512 : sp.NT;
  gk.lds_bytes = ksplit ? (int)ksplit_lds_ : (int)gemm_smem_bytes(sp);
  if (gk.lds_bytes > 160 * 1024) fail(KORCH_E_UNSUPPORTED, "gemm: tiles need more than 160 KiB of LDS");
  ki.fill_cost(gk);
  return gk;
}

}  // namespace korch
