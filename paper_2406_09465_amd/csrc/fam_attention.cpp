// Attention family: S0 = Q K^T, an elementwise score chain (e.g. scaling),
// row softmax (row max, subtract, exp, row sum, divide) and O = P V in one
// kernel, with every key and value of a batch resident in LDS.
//
// Korch admits hand-written attention kernels as a backend for candidates it
// identifies as attention subgraphs (Related Work, hand-optimized kernels);
// this family accepts exactly the fissioned softmax of Section 1 between two
// products.  Scores stay in MFMA accumulator registers; the row reductions are
// butterflies over the 16 lanes that share a row.
#include <algorithm>

#include "families.h"

namespace korch {

struct AttnSpec {
  int s0 = -1, sfinal = -1, m = -1, z = -1, e = -1, s = -1, p = -1, o = -1;
  int kt = -1;               // in-kernel transpose producing K^T (or -1)
  int q = -1, kx = -1, v = -1;  // external tensors
  bool k_is_kt = false;      // kx holds K^T [d, nk] directly
  std::vector<int> chain;    // elementwise score nodes S0 -> ... -> sfinal
  int64_t nq = 0, d = 0, nk = 0, dv = 0, batch = 1;
  int nb = 0;
  Shape bshape;
  int dtype = KORCH_F16;
};

static bool single_in_kernel_input(const KInfo& ki, int v, int* which) {
  const Node& n = ki.g.nodes[v];
  int cnt = 0;
  for (int u : n.in)
    if (ki.in.count(u)) {
      ++cnt;
      *which = u;
    }
  return cnt == 1;
}

static bool analyze_attention(const KInfo& ki, AttnSpec& a, std::string* why) {
  const Graph& g = ki.g;
  auto bad = [&](const char* m) {
    *why = std::string("attention: ") + m;
    return false;
  };
  if (ki.linear.size() != 2) return bad("needs exactly two products");
  for (int v : ki.linear)
    if (g.nodes[v].op != KORCH_MATMUL) return bad("products must be matmuls");
  a.s0 = ki.linear[0];
  a.o = ki.linear[1];
  if (ki.k.outs.size() != 1 || ki.k.outs[0] != a.o) return bad("the only output must be the second product");
  const Node& o = g.nodes[a.o];
  a.p = o.in[0];
  a.v = o.in[1];
  if (!ki.in.count(a.p) || ki.in.count(a.v)) return bad("second product must read P inside and V outside");
  const Node& pn = g.nodes[a.p];
  if (pn.op != KORCH_DIV || pn.attrs.has_scalar) return bad("P must be E / s");
  a.e = pn.in[0];
  a.s = pn.in[1];
  const Node& sn = g.nodes[a.s];
  if (sn.op != KORCH_REDUCE_SUM || sn.in[0] != a.e || !sn.attrs.keepdim) return bad("s must be a keepdim row sum of E");
  const Node& en = g.nodes[a.e];
  if (en.op != KORCH_EXP) return bad("E must be exp(Z)");
  a.z = en.in[0];
  const Node& zn = g.nodes[a.z];
  if (zn.op != KORCH_SUB || zn.attrs.has_scalar) return bad("Z must be S - m");
  a.sfinal = zn.in[0];
  a.m = zn.in[1];
  const Node& mn = g.nodes[a.m];
  if (mn.op != KORCH_REDUCE_MAX || mn.in[0] != a.sfinal || !mn.attrs.keepdim) return bad("m must be a keepdim row max of S");
  // reductions over the last axis
  int r = (int)g.nodes[a.sfinal].shape.size();
  if (sn.axis != r - 1 || mn.axis != r - 1) return bad("softmax must run over the last axis");
  // chain S0 -> ... -> sfinal
  std::vector<int> chain;
  int cur = a.sfinal;
  while (cur != a.s0) {
    if (!ki.in.count(cur)) return bad("score chain leaves the kernel");
    const Node& cn = g.nodes[cur];
    Kind kd = op_kind(cn.op);
    if (kd == Kind::Unary) {
      chain.push_back(cur);
      cur = cn.in[0];
    } else if (kd == Kind::Binary && cn.attrs.has_scalar) {
      chain.push_back(cur);
      cur = cn.in[0];
    } else {
      return bad("score chain must be unary or scalar elementwise primitives");
    }
  }
  std::reverse(chain.begin(), chain.end());
  a.chain = chain;
  const Node& s0 = g.nodes[a.s0];
  a.q = s0.in[0];
  int kop = s0.in[1];
  if (ki.in.count(a.q)) return bad("Q must be a materialized tensor");
  if (ki.in.count(kop)) {
    const Node& kn = g.nodes[kop];
    int rk = (int)kn.shape.size();
    if (kn.op != KORCH_TRANSPOSE || ki.in.count(kn.in[0])) return bad("K^T must be a transpose of a materialized tensor");
    for (int i = 0; i < rk - 2; ++i)
      if (kn.attrs.perm[i] != i) return bad("K^T transpose must swap only the last two dims");
    if (kn.attrs.perm[rk - 2] != rk - 1 || kn.attrs.perm[rk - 1] != rk - 2) return bad("K^T must swap the last two dims");
    a.kt = kop;
    a.kx = kn.in[0];
    a.k_is_kt = false;
  } else {
    a.kx = kop;
    a.k_is_kt = true;
  }
  // every kernel node accounted for
  std::set<int> known = {a.s0, a.m, a.z, a.e, a.s, a.p, a.o};
  if (a.kt >= 0) known.insert(a.kt);
  for (int c : chain) known.insert(c);
  if (known.size() != ki.in.size()) return bad("kernel holds primitives outside the attention pattern");
  for (int v : ki.in)
    if (!known.count(v)) return bad("kernel holds primitives outside the attention pattern");
  // shapes
  const Shape& qs = g.nodes[a.q].shape;
  const Shape& vs = g.nodes[a.v].shape;
  const Shape& os = o.shape;
  a.nb = (int)os.size() - 2;
  a.nq = qs[qs.size() - 2];
  a.d = qs.back();
  a.nk = vs[vs.size() - 2];
  a.dv = vs.back();
  a.bshape = Shape(os.begin(), os.end() - 2);
  a.batch = numel(a.bshape);
  for (int t : {a.q, a.kx, a.v})
    if ((int)g.nodes[t].shape.size() != a.nb + 2 ||
        !std::equal(a.bshape.begin(), a.bshape.end(), g.nodes[t].shape.begin()))
      return bad("batch dims must match exactly");
  a.dtype = g.nodes[a.q].dtype;
  if (g.nodes[a.kx].dtype != a.dtype || g.nodes[a.v].dtype != a.dtype) return bad("operand dtypes differ");
  if (a.nk > 256) return bad("more than 256 keys");
  if (a.dv > 128) return bad("value width above 128");
  if (a.d > 128) return bad("head dim above 128");
  if (a.dtype != KORCH_F32 && a.d % 8) return bad("half-precision needs d % 8 == 0");
  if (a.dtype == KORCH_F32 && a.d % 4) return bad("fp32 needs d % 4 == 0");
  return true;
}

// LDS bytes of the kernel: all keys, all values and one score tile per wave.
// Keys and values read from the same stored tensor with the same [key][dim]
// geometry (attention whose keys and values are one projection, as in
// spatial-reduction attention) are staged into LDS once and read as both.
static bool kv_shared(const AttnSpec& a) {
  bool f32 = a.dtype == KORCH_F32;
  int kstep = f32 ? 4 : 32;
  int64_t dpad = (a.d + kstep - 1) / kstep * kstep, dvp = (a.dv + 15) / 16 * 16;
  return a.kx == a.v && !a.k_is_kt && a.d == a.dv && dpad == dvp && !getenv("KORCH_ATTN_NO_KV_SHARE");
}

static size_t attention_lds_bytes(const AttnSpec& a) {
  bool f32 = a.dtype == KORCH_F32;
  int kstep = f32 ? 4 : 32;
  int64_t dpad = (a.d + kstep - 1) / kstep * kstep;
  int64_t nkp = f32 ? (a.nk + 15) / 16 * 16 : (a.nk + 31) / 32 * 32;
  int64_t KSP = dpad + (f32 ? 4 : 8), NKP = nkp + (f32 ? 4 : 8);
  int64_t dvp = (a.dv + 15) / 16 * 16, VP = dvp + (f32 ? 4 : 8);
  size_t ks = (size_t)(nkp * KSP * dtype_bytes(a.dtype));
  size_t v = kv_shared(a) ? 0 : (size_t)(nkp * VP * dtype_bytes(a.dtype));
  return ks + v + (size_t)(4 * 16 * NKP * dtype_bytes(a.dtype));
}

bool match_attention(const KInfo& ki, std::string* why) {
  AttnSpec a;
  if (!analyze_attention(ki, a, why)) return false;
  if (attention_lds_bytes(a) > 160 * 1024) {
    *why = "attention: keys and values exceed the 160 KiB of LDS";
    return false;
  }
  return true;
}

GenKernel gen_attention(const KInfo& ki, int index) {
  AttnSpec a;
  std::string why;
  if (!analyze_attention(ki, a, &why)) fail(KORCH_E_UNSUPPORTED, why);
  const Graph& g = ki.g;
  GenKernel gk;
  gk.family = KORCH_FAM_ATTENTION;
  gk.name = kernel_name(index, "attention");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  bool f32 = a.dtype == KORCH_F32;
  std::string T = ctype(a.dtype);
  int kstep = f32 ? 4 : 32;
  int64_t dpad = (a.d + kstep - 1) / kstep * kstep;  // contraction of Q K^T padded with zeros
  int64_t nkp = f32 ? (a.nk + 15) / 16 * 16 : (a.nk + 31) / 32 * 32;  // keys padded: zero K/V, -inf scores
  int KSP = (int)dpad + (f32 ? 4 : 8);                // Ks row pitch (elements)
  int NKP = (int)nkp + (f32 ? 4 : 8);                 // Ps / Vt row pitch
  int64_t dvp = (a.dv + 15) / 16 * 16;                // value width padded with zero columns
  int VP = (int)dvp + (f32 ? 4 : 8);                  // V row pitch ([key][dim] in LDS)
  int NF = (int)(nkp / 16), OF = (int)(dvp / 16);
  size_t ks_bytes = (size_t)nkp * KSP * dtype_bytes(a.dtype);
  const bool shareKV = kv_shared(a);  // then VP == KSP and Vs aliases Ks
  size_t v_bytes = shareKV ? 0 : (size_t)nkp * VP * dtype_bytes(a.dtype);
  size_t p_bytes = (size_t)4 * 16 * NKP * dtype_bytes(a.dtype);
  size_t smem = ks_bytes + v_bytes + p_bytes;
  if (smem != attention_lds_bytes(a) || smem > 160 * 1024)
    fail(KORCH_E_UNSUPPORTED, "attention: keys and values exceed the 160 KiB of LDS");
  // Few query rows (fewer than 64 workgroups of 64 rows): split the keys over
  // the four waves instead, one workgroup per 16 query rows.  Each wave scores
  // its quarter of the keys; row maxima and row sums are combined across the
  // waves through LDS, and the four partial P.V products are added in wave
  // order (deterministic).
  const int kalign = f32 ? 16 : 32;  // keys per S fragment / per P.V step
  const int64_t NKW = nkp / 4;
  const size_t red_off = (smem + 15) / 16 * 16, op_off = red_off + 2 * 4 * 16 * 4;
  const size_t smem_split = op_off + (size_t)4 * 16 * dvp * 4;
  const bool ksplit = (a.nq + 63) / 64 * a.batch < 64 && nkp % (4 * kalign) == 0 && smem_split <= 160 * 1024 &&
                      !getenv("KORCH_ATTN_NO_KEY_SPLIT");
  if (ksplit) smem = smem_split;
  std::string Q = "((const " + T + "*)a.p[" + std::to_string(slot.at(a.q)) + "])";
  std::string K = "((const " + T + "*)a.p[" + std::to_string(slot.at(a.kx)) + "])";
  std::string V = "((const " + T + "*)a.p[" + std::to_string(slot.at(a.v)) + "])";
  std::string O = "((" + ctype(g.nodes[a.o].dtype) + "*)a.p[" + std::to_string(ki.out_slot(a.o)) + "])";
  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << "  __shared__ __attribute__((aligned(16))) char smem[" << smem << "];\n";
  s << "  " << T << "* Ks = (" << T << "*)smem;\n";
  if (shareKV)
    s << "  " << T << "* Vs = Ks;  // keys and values are one tensor\n";
  else
    s << "  " << T << "* Vs = (" << T << "*)(smem + " << ks_bytes << ");\n";
  s << "  " << T << "* Ps = (" << T << "*)(smem + " << ks_bytes + v_bytes << ");\n";
  s << "  const int tid = threadIdx.x, l = tid & 63, wave = tid >> 6;\n";
  s << "  const i64 bz = blockIdx.y;\n";
  s << "  const i64 qoff = bz * " << a.nq * a.d << "LL, koff = bz * " << a.nk * a.d << "LL, voff = bz * "
    << a.nk * a.dv << "LL, ooff = bz * " << a.nq * a.dv << "LL;\n";
  // K and V into LDS as [key][dim] (zero-padded), 16-byte vectors along dim
  // when the rows allow (row pitches are multiples of 16 bytes).  When a
  // thread's share is small, all of its loads are issued before the first
  // LDS write (one round trip to memory); the query fragments of the
  // half-precision paths are loaded before them as well.
  const int VL = 16 / dtype_bytes(a.dtype);
  // branch-free (buffer) loads need byte offsets below 2 GiB
  const bool small = (double)a.batch * std::max(a.nq * a.d, a.nk * std::max(a.d, a.dv)) * dtype_bytes(a.dtype) < 2147483648.0;
  const std::string VT = "vec_t<" + std::to_string(VL) + ", " + T + ">";
  const std::string V8 = a.dtype == KORCH_F16 ? "f16x8" : "bf16x8";
  const int64_t QF = f32 ? 0 : dpad / 32;  // query fragments per lane
  const bool qpre = f32 && small;  // fp32 query values loaded up front
  if (qpre) {
    s << "  const i64 qr_ = " << (ksplit ? "(i64)blockIdx.x * 16" : "(i64)blockIdx.x * 64 + wave * 16") << " + (l & 15);\n";
    s << "  float qf_[" << dpad / 4 << "];\n";
    s << "#pragma unroll\n  for (int kk = 0; kk < " << dpad / 4 << "; ++kk) {\n";
    s << "    const int dim = kk * 4 + (l >> 4);\n";
    s << "    qf_[kk] = ld4f_or_zero(" << Q << ", qoff + qr_ * " << a.d << " + dim, qr_ < " << a.nq << "LL && dim < " << a.d
      << ");\n  }\n";
  }
  if (!f32) {
    s << "  const i64 qr_ = " << (ksplit ? "(i64)blockIdx.x * 16" : "(i64)blockIdx.x * 64 + wave * 16") << " + (l & 15);\n";
    s << "  " << V8 << " qa_[" << QF << "];\n";
    s << "#pragma unroll\n  for (int kk = 0; kk < " << QF << "; ++kk) {\n";
    s << "    const int dim = kk * 32 + (l >> 4) * 8;\n";
    if (small && dpad == a.d) {
      s << "    qa_[kk] = __builtin_bit_cast(" << V8 << ", ld16_or_zero(" << Q << ", (qoff + qr_ * " << a.d << " + dim) * 2, qr_ < "
        << a.nq << "LL));\n  }\n";
    } else {
      s << "    if (qr_ < " << a.nq << "LL && dim + 8 <= " << a.d << ") qa_[kk] = *(const " << V8 << "*)(" << Q << " + qoff + qr_ * "
        << a.d << " + dim);\n";
      s << "    else {\n#pragma unroll\n      for (int j = 0; j < 8; ++j) qa_[kk][j] = (qr_ < " << a.nq << "LL && dim + j < " << a.d
        << ") ? " << Q << "[qoff + qr_ * " << a.d << " + dim + j] : fromf<" << T << ">(0.0f);\n    }\n  }\n";
    }
  }
  const bool vecK = !a.k_is_kt && a.d % VL == 0 && dpad % VL == 0;
  const bool vecV = a.dv % VL == 0 && dvp % VL == 0;
  const int64_t NIK = (nkp * dpad / VL + 255) / 256, NIV = shareKV ? 0 : (nkp * dvp / VL + 255) / 256;
  if (vecK && vecV && NIK + NIV <= 24) {
    s << "  " << VT << " kx_[" << NIK << "], vx_[" << std::max<int64_t>(NIV, 1) << "];\n";
    s << "#pragma unroll\n  for (int j = 0; j < " << NIK << "; ++j) {\n";
    s << "    const int i = tid + j * 256, key = i / " << dpad / VL << ", dim = (i % " << dpad / VL << ") * " << VL << ";\n";
    if (small) {
      s << "    kx_[j] = __builtin_bit_cast(" << VT << ", ld16_or_zero(" << K << ", (koff + (i64)key * " << a.d << " + dim) * "
        << dtype_bytes(a.dtype) << ", i < " << nkp * dpad / VL << " && dim < " << a.d << " && key < " << a.nk << "));\n  }\n";
    } else {
      s << "    kx_[j] = " << VT << "{};\n";
      s << "    if (i < " << nkp * dpad / VL << " && dim < " << a.d << " && key < " << a.nk << ") kx_[j] = *(const " << VT << "*)("
        << K << " + koff + (i64)key * " << a.d << " + dim);\n  }\n";
    }
    s << "#pragma unroll\n  for (int j = 0; j < " << NIV << "; ++j) {\n";
    s << "    const int i = tid + j * 256, key = i / " << dvp / VL << ", dim = (i % " << dvp / VL << ") * " << VL << ";\n";
    if (small) {
      s << "    vx_[j] = __builtin_bit_cast(" << VT << ", ld16_or_zero(" << V << ", (voff + (i64)key * " << a.dv << " + dim) * "
        << dtype_bytes(a.dtype) << ", i < " << nkp * dvp / VL << " && key < " << a.nk << " && dim < " << a.dv << "));\n  }\n";
    } else {
      s << "    vx_[j] = " << VT << "{};\n";
      s << "    if (i < " << nkp * dvp / VL << " && key < " << a.nk << " && dim < " << a.dv << ") vx_[j] = *(const " << VT << "*)("
        << V << " + voff + (i64)key * " << a.dv << " + dim);\n  }\n";
    }
    s << "#pragma unroll\n  for (int j = 0; j < " << NIK << "; ++j) {\n";
    s << "    const int i = tid + j * 256, key = i / " << dpad / VL << ", dim = (i % " << dpad / VL << ") * " << VL << ";\n";
    s << "    if (" << ((nkp * dpad / VL) % 256 == 0 ? std::string("true") : "i < " + std::to_string(nkp * dpad / VL)) << ") *(" << VT
      << "*)(Ks + key * " << KSP << " + dim) = kx_[j];\n  }\n";
    s << "#pragma unroll\n  for (int j = 0; j < " << NIV << "; ++j) {\n";
    s << "    const int i = tid + j * 256, key = i / " << dvp / VL << ", dim = (i % " << dvp / VL << ") * " << VL << ";\n";
    s << "    if (" << ((nkp * dvp / VL) % 256 == 0 ? std::string("true") : "i < " + std::to_string(nkp * dvp / VL)) << ") *(" << VT
      << "*)(Vs + key * " << VP << " + dim) = vx_[j];\n  }\n";
  } else {
    if (vecK) {
      s << "#pragma unroll 4\n  for (int i = tid; i < " << nkp * dpad / VL << "; i += 256) {\n";
      s << "    const int key = i / " << dpad / VL << ", dim = (i % " << dpad / VL << ") * " << VL << ";\n";
      s << "    " << VT << " x_ = {};\n";
      s << "    if (dim < " << a.d << " && key < " << a.nk << ") x_ = *(const " << VT << "*)(" << K << " + koff + (i64)key * "
        << a.d << " + dim);\n";
      s << "    *(" << VT << "*)(Ks + key * " << KSP << " + dim) = x_;\n  }\n";
    } else {
      s << "  for (int i = tid; i < " << nkp * dpad << "; i += 256) {\n";
      s << "    const int key = i / " << dpad << ", dim = i % " << dpad << ";\n";
      if (a.k_is_kt)
        s << "    Ks[key * " << KSP << " + dim] = (dim < " << a.d << " && key < " << a.nk << ") ? " << K
          << "[koff + (i64)dim * " << a.nk << " + key] : fromf<" << T << ">(0.0f);\n";
      else
        s << "    Ks[key * " << KSP << " + dim] = (dim < " << a.d << " && key < " << a.nk << ") ? " << K
          << "[koff + (i64)key * " << a.d << " + dim] : fromf<" << T << ">(0.0f);\n";
      s << "  }\n";
    }
    if (shareKV) {
      // the values are the keys already staged
    } else if (vecV) {
      s << "#pragma unroll 4\n  for (int i = tid; i < " << nkp * dvp / VL << "; i += 256) {\n";
      s << "    const int key = i / " << dvp / VL << ", dim = (i % " << dvp / VL << ") * " << VL << ";\n";
      s << "    " << VT << " x_ = {};\n";
      s << "    if (key < " << a.nk << " && dim < " << a.dv << ") x_ = *(const " << VT << "*)(" << V << " + voff + (i64)key * "
        << a.dv << " + dim);\n";
      s << "    *(" << VT << "*)(Vs + key * " << VP << " + dim) = x_;\n  }\n";
    } else {
      s << "  for (int i = tid; i < " << nkp * dvp << "; i += 256) {\n";
      s << "    const int key = i / " << dvp << ", dim = i % " << dvp << ";\n";
      s << "    Vs[key * " << VP << " + dim] = (key < " << a.nk << " && dim < " << a.dv << ") ? " << V << "[voff + (i64)key * "
        << a.dv << " + dim] : fromf<" << T << ">(0.0f);\n";
      s << "  }\n";
    }
  }
  s << "  __syncthreads();\n";
  std::string chain_expr = "x";
  for (int c : a.chain) {
    const Node& cn = g.nodes[c];
    if (op_kind(cn.op) == Kind::Unary)
      chain_expr = unary_expr(cn.op, chain_expr);
    else
      chain_expr = binary_expr(cn.op, chain_expr, flit(cn.attrs.scalar));
  }
  // A score chain that only scales by a positive constant c (the 1/sqrt(d) of
  // attention) commutes with the row maximum, so half-precision kernels take
  // the maximum of the raw scores and evaluate exp(c (x - max)) as one base-2
  // exponential of fma(x, c log2 e, -max c log2 e).
  double fold_c = 0.0;
  if (fast_math() && a.chain.size() == 1) {
    const Node& cn = g.nodes[a.chain[0]];
    if (cn.op == KORCH_MUL && cn.attrs.scalar > 0.0) fold_c = cn.attrs.scalar;
    if (cn.op == KORCH_DIV && cn.attrs.scalar > 0.0) fold_c = 1.0 / cn.attrs.scalar;
  }
  const std::string CL = flit(fold_c * 1.4426950408889634);
  const std::string score_expr = fold_c > 0.0 ? std::string("x") : chain_expr;
  // exponentials of one row block after the maxima: sc[f][i] and sm[i]
  auto exp_stmt = [&]() {
    if (fold_c > 0.0)
      return std::string("    sc[f][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[f][i], ") + CL + ", mcl[i]));\n";
    return "    sc[f][i] = " + unary_expr(KORCH_EXP, "(sc[f][i] - mx[i])") + ";\n";
  };
  auto mcl_stmt = [&]() {
    if (fold_c <= 0.0) return std::string();
    return "  float mcl[4];\n#pragma unroll\n  for (int i = 0; i < 4; ++i) mcl[i] = -mx[i] * " + CL + ";\n";
  };
  if (ksplit) {
    const int NFW = (int)(NKW / 16);
    s << "  const i64 q0 = (i64)blockIdx.x * 16;\n";
    s << "  const i64 qr = q0 + (l & 15);\n";
    s << "  const bool qv = qr < " << a.nq << "LL;\n";
    s << "  const int kb = wave * " << NKW << ";  // this wave's keys [kb, kb + " << NKW << ")\n";
    s << "  f32x4 sc[" << NFW << "];\n";
    s << "#pragma unroll\n  for (int f = 0; f < " << NFW << "; ++f) sc[f] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};\n";
    if (f32) {
      s << "#pragma unroll\n  for (int kk = 0; kk < " << dpad / 4 << "; ++kk) {\n";
      s << "    const int dim = kk * 4 + (l >> 4);\n";
      if (qpre)
        s << "    const float qa = qf_[kk];\n";
      else
        s << "    const float qa = (qv && dim < " << a.d << ") ? " << Q << "[qoff + qr * " << a.d << " + dim] : 0.0f;\n";
      s << "#pragma unroll\n    for (int f = 0; f < " << NFW << "; ++f) sc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa, Ks[(kb + f * 16 + (l & 15)) * "
        << KSP << " + dim], sc[f], 0, 0, 0);\n  }\n";
    } else {
      std::string fn = a.dtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16" : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
      s << "#pragma unroll\n  for (int kk = 0; kk < " << dpad / 32 << "; ++kk) {\n";
      s << "    const int dim = kk * 32 + (l >> 4) * 8;\n";
      s << "    const " << V8 << " qa = qa_[kk];\n";
      s << "#pragma unroll\n    for (int f = 0; f < " << NFW << "; ++f) sc[f] = " << fn << "(qa, *(const " << V8
        << "*)(Ks + (kb + f * 16 + (l & 15)) * " << KSP << " + dim), sc[f], 0, 0, 0);\n  }\n";
    }
    // rows (l>>4)*4 + i of the 16, key kb + f*16 + (l&15)
    s << "  float mx[4], sm[4];\n";
    s << "  float* red = (float*)(smem + " << red_off << ");  // [2][wave][16 rows]\n";
    s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) mx[i] = -__builtin_huge_valf();\n";
    s << "#pragma unroll\n  for (int f = 0; f < " << NFW << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n";
    s << "    const float x = sc[f][i];\n    sc[f][i] = " << score_expr << ";\n";
    if (nkp != a.nk) s << "    if (kb + f * 16 + (l & 15) >= " << a.nk << ") sc[f][i] = -__builtin_huge_valf();\n";
    s << "    mx[i] = k_max(mx[i], sc[f][i]);\n  }\n";
    s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) mx[i] = group_max<16>(mx[i]);\n";
    s << "  if ((l & 15) == 0) {\n#pragma unroll\n    for (int i = 0; i < 4; ++i) red[wave * 16 + (l >> 4) * 4 + i] = mx[i];\n  }\n";
    s << "  __syncthreads();\n";
    s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n    const int r = (l >> 4) * 4 + i;\n";
    s << "    mx[i] = k_max(k_max(red[r], red[16 + r]), k_max(red[32 + r], red[48 + r]));\n    sm[i] = 0.0f;\n  }\n";
    s << mcl_stmt();
    s << "#pragma unroll\n  for (int f = 0; f < " << NFW << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n";
    s << exp_stmt() << "    sm[i] += sc[f][i];\n  }\n";
    s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) sm[i] = group_sum<16>(sm[i]);\n";
    s << "  if ((l & 15) == 0) {\n#pragma unroll\n    for (int i = 0; i < 4; ++i) red[64 + wave * 16 + (l >> 4) * 4 + i] = sm[i];\n  }\n";
    s << "  __syncthreads();\n";
    s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n    const int r = 64 + (l >> 4) * 4 + i;\n";
    s << "    sm[i] = ((red[r] + red[16 + r]) + red[32 + r]) + red[48 + r];\n  }\n";
    s << "  " << T << "* Pw = Ps + wave * " << 16 * NKP << ";  // this wave's probabilities, keys local\n";
    s << "#pragma unroll\n  for (int f = 0; f < " << NFW << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) Pw[((l >> 4) * 4 + i) * "
      << NKP << " + f * 16 + (l & 15)] = fromf<" << T << ">(" << binary_expr(KORCH_DIV, "sc[f][i]", "sm[i]") << ");\n";
    s << "  __syncthreads();\n";
    s << "  f32x4 oc[" << OF << "];\n";
    s << "#pragma unroll\n  for (int f = 0; f < " << OF << "; ++f) oc[f] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};\n";
    if (f32) {
      s << "#pragma unroll\n  for (int kk = 0; kk < " << NKW / 4 << "; ++kk) {\n";
      s << "    const int key = kk * 4 + (l >> 4);\n";
      s << "    const float pa = Pw[(l & 15) * " << NKP << " + key];\n";
      s << "#pragma unroll\n    for (int f = 0; f < " << OF << "; ++f) oc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa, Vs[(kb + key) * " << VP
        << " + f * 16 + (l & 15)], oc[f], 0, 0, 0);\n  }\n";
    } else {
      std::string fn = a.dtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16" : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
      s << "#pragma unroll\n  for (int kk = 0; kk < " << NKW / 32 << "; ++kk) {\n";
      s << "    const int key = kk * 32 + (l >> 4) * 8;\n";
      s << "    const " << V8 << " pa = *(const " << V8 << "*)(Pw + (l & 15) * " << NKP << " + key);\n";
      // V[key][dim] read transposed: lane l gets keys key..key+7 of column f*16 + (l & 15)
      s << "#pragma unroll\n    for (int f = 0; f < " << OF << "; ++f) oc[f] = " << fn << "(pa, __builtin_bit_cast(" << V8
        << ", lds_tr_k8(Vs + (kb + key + ((l & 15) >> 2)) * " << VP << " + f * 16 + 4 * (l & 3), " << VP
        << ")), oc[f], 0, 0, 0);\n  }\n";
    }
    s << "  float* Op = (float*)(smem + " << op_off << ");  // [wave][16 rows][" << dvp << "]\n";
    s << "#pragma unroll\n  for (int f = 0; f < " << OF << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) Op[(wave * 16 + (l >> 4) * 4 + i) * "
      << dvp << " + f * 16 + (l & 15)] = oc[f][i];\n";
    s << "  __syncthreads();\n";
    s << "  for (int t = tid; t < " << 16 * dvp << "; t += 256) {\n";
    s << "    const int row = t / " << dvp << ", col = t % " << dvp << ";\n";
    s << "    const float o_ = ((Op[t] + Op[" << 16 * dvp << " + t]) + Op[" << 32 * dvp << " + t]) + Op[" << 48 * dvp << " + t];\n";
    s << "    if (q0 + row < " << a.nq << "LL && col < " << a.dv << ") "
      << out_store(g, a.o, O, "ooff + (q0 + row) * " + std::to_string(a.dv) + " + col", 0, "o_") << ";\n  }\n";
    s << "}\n";
    gk.source = s.str();
    gk.grid[0] = (int)((a.nq + 15) / 16);
    gk.grid[1] = (int)a.batch;
    gk.lds_bytes = (int)smem;
    ki.fill_cost(gk);
    return gk;
  }
  // this wave's 16 query rows
  s << "  const i64 q0 = (i64)blockIdx.x * 64 + wave * 16;\n";
  s << "  const i64 qr = q0 + (l & 15);\n";
  s << "  const bool qv = qr < " << a.nq << "LL;\n";
  s << "  f32x4 sc[" << NF << "];\n";
  s << "#pragma unroll\n  for (int f = 0; f < " << NF << "; ++f) sc[f] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};\n";
  if (f32) {
    s << "#pragma unroll\n  for (int kk = 0; kk < " << dpad / 4 << "; ++kk) {\n";
    s << "    const int dim = kk * 4 + (l >> 4);\n";
    if (qpre)
      s << "    const float qa = qf_[kk];\n";
    else
      s << "    const float qa = (qv && dim < " << a.d << ") ? " << Q << "[qoff + qr * " << a.d << " + dim] : 0.0f;\n";
    s << "#pragma unroll\n    for (int f = 0; f < " << NF << "; ++f) sc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa, Ks[(f * 16 + (l & 15)) * "
      << KSP << " + dim], sc[f], 0, 0, 0);\n  }\n";
  } else {
    std::string fn = a.dtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16" : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
    s << "#pragma unroll\n  for (int kk = 0; kk < " << dpad / 32 << "; ++kk) {\n";
    s << "    const int dim = kk * 32 + (l >> 4) * 8;\n";
    s << "    const " << V8 << " qa = qa_[kk];\n";
    s << "#pragma unroll\n    for (int f = 0; f < " << NF << "; ++f) sc[f] = " << fn << "(qa, *(const " << V8
      << "*)(Ks + (f * 16 + (l & 15)) * " << KSP << " + dim), sc[f], 0, 0, 0);\n  }\n";
  }
  // score chain, row max, exp, row sum, divide -- rows (l>>4)*4 + i, key f*16 + (l&15)
  s << "  float mx[4], sm[4];\n";
  s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) mx[i] = -__builtin_huge_valf();\n";
  s << "#pragma unroll\n  for (int f = 0; f < " << NF << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n";
  s << "    const float x = sc[f][i];\n    sc[f][i] = " << score_expr << ";\n";
  if (nkp != a.nk) s << "    if (f * 16 + (l & 15) >= " << a.nk << ") sc[f][i] = -__builtin_huge_valf();\n";
  s << "    mx[i] = k_max(mx[i], sc[f][i]);\n  }\n";
  s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) mx[i] = group_max<16>(mx[i]);\n";
  s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) sm[i] = 0.0f;\n";
  s << mcl_stmt();
  s << "#pragma unroll\n  for (int f = 0; f < " << NF << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n";
  s << exp_stmt() << "    sm[i] += sc[f][i];\n  }\n";
  s << "#pragma unroll\n  for (int i = 0; i < 4; ++i) sm[i] = group_sum<16>(sm[i]);\n";
  s << "  " << T << "* Pw = Ps + wave * " << 16 * NKP << ";\n";
  s << "#pragma unroll\n  for (int f = 0; f < " << NF << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) Pw[((l >> 4) * 4 + i) * "
    << NKP << " + f * 16 + (l & 15)] = fromf<" << T << ">(" << binary_expr(KORCH_DIV, "sc[f][i]", "sm[i]") << ");\n";
  s << "  __syncthreads();\n";
  // O = P V
  s << "  f32x4 oc[" << OF << "];\n";
  s << "#pragma unroll\n  for (int f = 0; f < " << OF << "; ++f) oc[f] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};\n";
  if (f32) {
    s << "#pragma unroll\n  for (int kk = 0; kk < " << nkp / 4 << "; ++kk) {\n";
    s << "    const int key = kk * 4 + (l >> 4);\n";
    s << "    const float pa = Pw[(l & 15) * " << NKP << " + key];\n";
    s << "#pragma unroll\n    for (int f = 0; f < " << OF << "; ++f) oc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa, Vs[key * " << VP
      << " + f * 16 + (l & 15)], oc[f], 0, 0, 0);\n  }\n";
  } else {
    std::string fn = a.dtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16" : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
    s << "#pragma unroll\n  for (int kk = 0; kk < " << nkp / 32 << "; ++kk) {\n";
    s << "    const int key = kk * 32 + (l >> 4) * 8;\n";
    s << "    const " << V8 << " pa = *(const " << V8 << "*)(Pw + (l & 15) * " << NKP << " + key);\n";
    // V[key][dim] read transposed: lane l gets keys key..key+7 of column f*16 + (l & 15)
    s << "#pragma unroll\n    for (int f = 0; f < " << OF << "; ++f) oc[f] = " << fn << "(pa, __builtin_bit_cast(" << V8
      << ", lds_tr_k8(Vs + (key + ((l & 15) >> 2)) * " << VP << " + f * 16 + 4 * (l & 3), " << VP << ")), oc[f], 0, 0, 0);\n  }\n";
  }
  s << "#pragma unroll\n  for (int f = 0; f < " << OF << "; ++f)\n#pragma unroll\n  for (int i = 0; i < 4; ++i) {\n";
  s << "    const i64 row = q0 + (l >> 4) * 4 + i;\n";
  s << "    const int col = f * 16 + (l & 15);\n";
  s << "    if (row < " << a.nq << "LL && col < " << a.dv << ") "
    << out_store(g, a.o, O, "ooff + row * " + std::to_string(a.dv) + " + col", 0, "oc[f][i]") << ";\n  }\n";
  s << "}\n";
  gk.source = s.str();
  gk.grid[0] = (int)((a.nq + 63) / 64);
  gk.grid[1] = (int)a.batch;
  gk.lds_bytes = (int)smem;
  ki.fill_cost(gk);
  return gk;
}

}  // namespace korch
