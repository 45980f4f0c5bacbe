// Direct convolution kernel of the conv family (gfx950).
//
// The convolution primitive (Section 3's linear primitives; an NHWC
// cross-correlation with an HWIO weight) with its elementwise epilogue, for
// stride 1 and half precision.  The implicit-GEMM kernel of the GEMM family
// re-reads every input pixel once per filter tap through L2 and runs a short
// pipelined k-loop with a barrier per step; this kernel instead
//
//  * is persistent: a workgroup keeps the weights of its wave's output
//    channels in registers (loaded once through LDS) and loops over output
//    tiles of TH x TW pixels with all output channels;
//  * stages the tile's input halo ((TH + KH - 1) x (TW + KW - 1) pixels, all
//    input channels, zero outside the image) into LDS once, double-buffered:
//    the next tile's halo is loaded into registers while the current tile is
//    multiplied and written back;
//  * forms every tap's MFMA left operand directly from the halo (a pixel shift),
//    so a tile's 9 taps need no k-loop and no barrier between them.
//
// Tiles are spread over the 8 XCDs in contiguous bands, so vertically
// adjacent tiles (which share halo rows) run on one XCD and share its L2.

#include <algorithm>
#include <sstream>

#include "codegen.h"
#include "gemm_common.h"

namespace korch {

namespace {

struct Direct {
  int TH = 0, TW = 0;        // output tile (rows x columns of pixels); TH * TW = 128
  int WM = 0, WN = 0;        // waves along pixels / along output channels
  int FM = 0, FN = 0;        // 16 x 16 fragments per wave along pixels / channels
  int PW = 0, WTN = 0;       // pixels / channels per wave
  int CP = 0, CC = 0;        // input channels padded to 32; 32-channel chunks per tap
  int CPP = 0;               // LDS pitch of one halo pixel (elements)
  int NP = 0, WP = 0, LDC = 0;
  int taps = 0, HR = 0, HC = 0, CV = 0, HV = 0, HPT = 0;
  int64_t halo_bytes = 0, smem = 0;
  int64_t ntx = 0, nty = 0, tiles = 0, G = 0;
};

bool plan_direct(const GemmSpec& sp, Direct& d, std::string* why) {
  auto no = [&](const char* m) {
    if (why) *why = std::string("conv direct: ") + m;
    return false;
  };
  if (!sp.conv) return no("not a convolution");
  if (sp.mtype == KORCH_F32) return no("fp32 operands");
  if (sp.stride != 1) return no("stride is not 1");
  if (sp.nb > 1) return no("more than one batch dimension");
  if (sp.Cin % 8 || sp.N % 8) return no("channels not a multiple of 8");
  if (sp.N > 128) return no("more than 128 output channels");
  if ((double)sp.batch * sp.H * sp.W * sp.Cin * 2 >= 2147483648.0) return no("input of 2 GiB or more");
  d.taps = (int)(sp.KH * sp.KW);
  d.CP = (int)((sp.Cin + 31) / 32 * 32);
  d.CC = d.CP / 32;
  d.NP = (int)((sp.N + 15) / 16 * 16);
  const int fn_all = d.NP / 16;
  // fewest waves along channels that leave each wave at most 2 fragments
  // (fewer waves along pixels re-read the same halo from LDS); else as many as divide
  d.WN = 0;
  for (int wn : {1, 2, 4})
    if (!d.WN && fn_all % wn == 0 && fn_all / wn <= 2) d.WN = wn;
  if (!d.WN) d.WN = fn_all % 4 == 0 ? 4 : fn_all % 2 == 0 ? 2 : 1;
  if (const char* e = getenv("KORCH_CONV_WN")) {  // waves along channels (launch-shape sweeps)
    const int wn = atoi(e);
    if ((wn == 1 || wn == 2 || wn == 4) && fn_all % wn == 0) d.WN = wn;
  }
  d.FN = fn_all / d.WN;
  d.WTN = d.FN * 16;
  d.WM = 4 / d.WN;
  d.PW = 128 / d.WM;
  d.FM = d.PW / 16;
  // weight fragments held per lane: taps x chunks x FN fragments of 4 VGPRs
  if (d.taps * d.CC * d.FN * 4 > 144) return no("weights of a wave exceed 144 registers per lane");
  d.TW = sp.Wo > 16 ? 32 : 16;
  d.TH = 128 / d.TW;
  d.HR = d.TH + (int)sp.KH - 1;
  d.HC = d.TW + (int)sp.KW - 1;
  d.CPP = d.CP + 16;  // pitch an odd multiple of 32 bytes: a 16-byte read of 16 pixels is free of bank conflicts
  d.CV = d.CP / 8;
  d.HV = d.HR * d.HC * d.CV;
  d.HPT = (d.HV + 255) / 256;
  d.WP = d.NP + 16;
  d.LDC = d.NP + 4;
  d.halo_bytes = ((int64_t)d.HR * d.HC * d.CPP * 2 + 15) / 16 * 16;
  const int64_t cs = (int64_t)128 * d.LDC * 4;
  const int64_t stage = (int64_t)d.taps * d.CP * d.WP * 2;
  d.smem = d.halo_bytes + std::max(d.halo_bytes + cs, stage);
  if (d.smem > 80 * 1024) return no("LDS above 80 KiB (two workgroups per compute unit)");
  d.ntx = (sp.Wo + d.TW - 1) / d.TW;
  d.nty = (sp.Ho + d.TH - 1) / d.TH;
  d.tiles = sp.batch * d.ntx * d.nty;
  d.G = d.tiles < 8 ? d.tiles : std::min<int64_t>(512, d.tiles / 8 * 8);
  return true;
}

}  // namespace

bool conv_direct_fits(const GemmSpec& sp, std::string* why) {
  Direct d;
  return plan_direct(sp, d, why);
}

bool conv_uses_direct(const GemmSpec& sp, std::string* why) {
  const char* e = getenv("KORCH_CONV_DIRECT");
  if (e && atoi(e) == 0) {
    if (why) *why = "conv direct: switched off";
    return false;
  }
  return conv_direct_fits(sp, why);
}

GenKernel gen_conv_direct(const KInfo& ki, GemmSpec& sp, int index) {
  Direct d;
  std::string why;
  if (!plan_direct(sp, d, &why)) fail(KORCH_E_UNSUPPORTED, why);
  const Graph& g = ki.g;
  (void)g;
  // the epilogue reads the C tile as a BM x BN product tile
  sp.BM = 128;
  sp.BN = d.NP;
  sp.LDC = d.LDC;
  sp.NT = 256;
  GenKernel gk;
  gk.family = KORCH_FAM_CONV;
  gk.name = kernel_name(index, "conv");
  std::map<int, int> slot;
  ki.assign_args(gk, slot);
  const std::string T = ctype(sp.mtype);
  const std::string V8 = sp.mtype == KORCH_F16 ? "f16x8" : "bf16x8";
  const std::string mfma =
      sp.mtype == KORCH_F16 ? "__builtin_amdgcn_mfma_f32_16x16x32_f16" : "__builtin_amdgcn_mfma_f32_16x16x32_bf16";
  const int64_t H = sp.H, W = sp.W, Cin = sp.Cin, N = sp.N;
  const int64_t HALO = d.halo_bytes / 2;  // elements of one halo buffer
  const std::string X = "a.p[" + std::to_string(slot.at(sp.A)) + "]";
  // the weights as stored (when no prologue computes them)
  const std::string Wt = sp.pro.empty() ? "((const " + T + "*)a.p[" + std::to_string(slot.at(sp.Bs[0])) + "])" : "";
  const int64_t xbytes = sp.batch * H * W * Cin * 2;
  const int64_t per_img = d.ntx * d.nty;

  std::ostringstream s;
  s << source_header((int)gk.args.size());
  s << "extern \"C\" __global__ void __launch_bounds__(256) " << gk.name << "(KArgs a) {\n";
  s << "  __shared__ __attribute__((aligned(16))) char smem[" << d.smem << "];\n";
  s << "  " << T << "* Hs = (" << T << "*)smem;  // two input halo buffers\n";
  s << "  " << T << "* Ws = (" << T << "*)(smem + " << d.halo_bytes << ");  // weight staging (start-up only)\n";
  s << "  float* Cs = (float*)(smem + " << 2 * d.halo_bytes << ");  // fp32 C tile\n";
  s << "  const int tid = threadIdx.x, l = tid & 63, wave = tid >> 6;\n";
  s << "  const int wm = wave / " << d.WN << ", wn = wave % " << d.WN << ";\n";
  s << "  (void)wm; (void)wn;\n";
  s << "  const i64 m0 = 0, n0 = 0;\n  (void)m0;\n";
  // tiles of this workgroup
  if (d.tiles >= 8) {
    s << "  const int xcd = blockIdx.x % 8, jx = blockIdx.x / 8;\n";
    s << "  const int band0 = xcd * " << d.tiles / 8 << " + (xcd < " << d.tiles % 8 << " ? xcd : " << d.tiles % 8
      << ");\n";
    s << "  const int tend = band0 + " << d.tiles / 8 << " + (xcd < " << d.tiles % 8 << " ? 1 : 0);\n";
    s << "  int t = band0 + jx;\n";
    s << "  const int tstep = " << d.G / 8 << ";\n";
  } else {
    s << "  int t = blockIdx.x;\n  const int tend = t + 1, tstep = 1;\n";
  }
  s << "  if (t >= tend) return;\n";
  // per-channel epilogue operands are loaded once per workgroup, first, so that
  // their round trip overlaps the weights' and the first halo's
  std::string inv;
  const std::string epi = gemm_epilogue(ki, sp, slot, "ml * " + std::to_string(d.LDC), {}, d.TW, 0, "0", &inv);
  s << inv;
  // halo slots: vector v of the halo is pixel v / CV (row, column) and channels (v % CV) * 8
  s << "  const __amdgpu_buffer_rsrc_t rsX = __builtin_amdgcn_make_buffer_rsrc(" << X << ", 0, " << xbytes
    << ", 0x00020000);\n";
  s << "  int hsl[" << d.HPT << "], hgo[" << d.HPT << "], hr_[" << d.HPT << "], hc_[" << d.HPT << "];\n";
  s << "  bool hok[" << d.HPT << "];\n";
  s << "#pragma unroll\n  for (int i = 0; i < " << d.HPT << "; ++i) {\n";
  s << "    const int v = tid + i * 256, vv = v < " << d.HV << " ? v : " << d.HV - 1 << ";\n";
  s << "    const int pix = vv / " << d.CV << ", cv = vv % " << d.CV << ";\n";
  s << "    hr_[i] = pix / " << d.HC << "; hc_[i] = pix % " << d.HC << ";\n";
  s << "    hsl[i] = pix * " << d.CPP << " + cv * 8;\n";
  s << "    hgo[i] = (hr_[i] * " << W << " + hc_[i]) * " << Cin << " + cv * 8;\n";
  s << "    hok[i] = v < " << d.HV << " && cv * 8 < " << Cin << ";\n";
  s << "  }\n";
  s << "  uint4 hv[" << d.HPT << "];\n";
  auto origin = [&](const std::string& tv) {
    std::ostringstream o;
    o << "const int z_ = " << tv << " / " << per_img << ", rt_ = " << tv << " % " << per_img << ";\n";
    o << "    const int ty0 = (rt_ / " << d.ntx << ") * " << d.TH << ", tx0 = (rt_ % " << d.ntx << ") * " << d.TW
      << ";\n";
    return o.str();
  };
  s << "  auto fetch_halo = [&](const int tt) {\n    " << origin("tt");
  s << "    const int iy0 = ty0 - " << sp.pad << ", ix0 = tx0 - " << sp.pad << ";\n";
  s << "    const int base = ((z_ * " << H << " + iy0) * " << W << " + ix0) * " << Cin << ";\n";
  s << "#pragma unroll\n    for (int i = 0; i < " << d.HPT << "; ++i) {\n";
  s << "      const int iy = iy0 + hr_[i], ix = ix0 + hc_[i];\n";
  s << "      const bool ok = hok[i] && iy >= 0 && iy < " << H << " && ix >= 0 && ix < " << W << ";\n";
  s << "      const unsigned off = ok ? (unsigned)(base + hgo[i]) * 2u : 0x80000000u;\n";
  s << "      hv[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsX, off, 0, 0));\n";
  s << "    }\n  };\n";
  s << "  auto stash_halo = [&](const int b) {\n#pragma unroll\n    for (int i = 0; i < " << d.HPT << "; ++i)\n";
  s << "      if (" << (d.HV % 256 ? "tid + i * 256 < " + std::to_string(d.HV) : std::string("true")) << ") *(uint4*)(Hs + b * "
    << HALO << " + hsl[i]) = hv[i];\n  };\n";
  // weights: [tap * CP + c][n] in LDS (zero for padded channels and columns),
  // then each wave's fragments into registers with transposing reads
  const int NV = d.NP / 8;
  const int WV = d.taps * d.CP * NV;
  const int WPT = (WV + 255) / 256;
  // When every slot holds a weight vector the loads are unconditional: a
  // guarded load makes the compiler wait for all loads in flight at the join.
  const bool wall = WV % 256 == 0 && Cin == d.CP && N == d.NP;
  const std::string wguard = wall ? std::string("true")
                                  : "v < " + std::to_string(WV) + " && c < " + std::to_string(Cin) + " && nv * 8 < " +
                                        std::to_string(N);
  s << "  {\n    uint4 wv[" << WPT << "];\n";
  s << "#pragma unroll\n    for (int i = 0; i < " << WPT << "; ++i) {\n";
  s << "      const int v = tid + i * 256;\n";
  s << "      const int row = v / " << NV << ", nv = v % " << NV << ", tap = row / " << d.CP << ", c = row % " << d.CP
    << ";\n";
  s << "      wv[i] = uint4{0u, 0u, 0u, 0u};\n";
  if (sp.pro.empty()) {
    s << "      if (" << wguard << ") wv[i] = *(const uint4*)(" << Wt << " + ((i64)tap * " << Cin << " + c) * " << N
      << " + nv * 8);\n";
  } else {
    // the weights are computed by the kernel's prologue (e.g. scaled per
    // output channel): evaluated here, once per workgroup, 8 channels at a time
    Emitter em(ki.g);
    em.inset = sp.pro;
    em.argslot = slot;
    em.vec = 8;
    std::vector<Ix> idx = {Ix::var("ky_"), Ix::var("kx_"), Ix::var("c"), Ix::var("n_", 1, 8)};
    std::string val = em.value(sp.Bs[0], idx);
    s << "      if (" << wguard << ") {\n";
    s << "        const int ky_ = tap / " << sp.KW << ", kx_ = tap % " << sp.KW << ";\n";
    s << "        const i64 n_ = (i64)nv * 8;\n";
    s << "        (void)ky_; (void)kx_; (void)n_;\n";
    s << "        vec_t<8, " << T << "> w_;\n";
    s << em.pre.str();
    s << "#pragma unroll\n        for (int e = 0; e < 8; ++e) {\n" << em.body.str() << "          w_[e] = fromf<" << T
      << ">(" << val << ");\n        }\n";
    s << "        wv[i] = __builtin_bit_cast(uint4, w_);\n      }\n";
  }
  s << "    }\n";
  // the first halo's loads go out behind the weights' (the weights are waited
  // for first, and loads complete in order)
  s << "    fetch_halo(t);\n";
  s << "#pragma unroll\n    for (int i = 0; i < " << WPT << "; ++i) {\n";
  s << "      const int v = tid + i * 256;\n";
  s << "      if (" << (wall ? std::string("true") : "v < " + std::to_string(WV)) << ") *(uint4*)(Ws + (v / " << NV << ") * " << d.WP << " + (v % " << NV << ") * 8) = wv[i];\n";
  s << "    }\n  }\n";
  s << "  __syncthreads();\n";
  s << "  " << V8 << " bfr[" << d.taps << "][" << d.CC << "][" << d.FN << "];\n";
  s << "#pragma unroll\n  for (int tp = 0; tp < " << d.taps << "; ++tp)\n#pragma unroll\n  for (int cc = 0; cc < " << d.CC
    << "; ++cc)\n#pragma unroll\n  for (int j = 0; j < " << d.FN << "; ++j)\n";
  s << "    bfr[tp][cc][j] = __builtin_bit_cast(" << V8 << ", lds_tr_k8(Ws + (tp * " << d.CP
    << " + cc * 32 + (l >> 4) * 8 + ((l & 15) >> 2)) * " << d.WP << " + wn * " << d.WTN << " + j * 16 + 4 * (l & 3), "
    << d.WP << "));\n";
  s << "  __syncthreads();  // the staging area becomes halo buffer 1 and the C tile\n";
  s << "  stash_halo(0);\n  __syncthreads();\n";
  // per-lane part of the halo address of a fragment: pixel column (l & 15), channels (l >> 4) * 8
  s << "  const int lane_off = (l & 15) * " << d.CPP << " + (l >> 4) * 8;\n";
  s << "  int b = 0;\n";
  s << "  for (;;) {\n";
  s << "    const int tn = t + tstep;\n    const bool more = tn < tend;\n";
  s << "    if (more) fetch_halo(tn);\n";
  s << "    f32x4 acc[" << d.FM << "][" << d.FN << "];\n";
  s << "#pragma unroll\n    for (int f = 0; f < " << d.FM << "; ++f)\n#pragma unroll\n    for (int j = 0; j < " << d.FN
    << "; ++j) acc[f][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};\n";
  s << "    const " << T << "* Hb = Hs + b * " << HALO << " + lane_off;\n";
  // The wave's pixels are R rows of TW columns.  Every left-operand fragment
  // (16 pixels of one halo row at a column shift kx) is read from LDS once and
  // used for each of the wave's rows fr it serves (filter row ky = hr - fr), so
  // a wave reads (R + KH - 1) * KW fragments per column block instead of
  // R * KH * KW.  For each output fragment the taps still accumulate in
  // (ky, kx, channel chunk) order.
  const int R = d.PW / d.TW, FC = d.TW / 16;
  s << "    const " << T << "* Hw = Hb + wm * " << R * d.HC * d.CPP << ";\n";
  for (int hr = 0; hr < R + (int)sp.KH - 1; ++hr)
    for (int kx = 0; kx < (int)sp.KW; ++kx)
      for (int fc = 0; fc < FC; ++fc)
        for (int cc = 0; cc < d.CC; ++cc) {
          s << "    {\n      const " << V8 << " af = *(const " << V8 << "*)(Hw + " << ((int64_t)hr * d.HC + fc * 16 + kx) * d.CPP + cc * 32
            << ");\n";
          for (int fr = 0; fr < R; ++fr) {
            const int ky = hr - fr;
            if (ky < 0 || ky >= (int)sp.KH) continue;
            const int f = fr * FC + fc, tp = ky * (int)sp.KW + kx;
            for (int j = 0; j < d.FN; ++j)
              s << "      acc[" << f << "][" << j << "] = " << mfma << "(af, bfr[" << tp << "][" << cc << "][" << j << "], acc[" << f
                << "][" << j << "], 0, 0, 0);\n";
          }
          s << "    }\n";
        }

  s << "#pragma unroll\n    for (int f = 0; f < " << d.FM << "; ++f)\n#pragma unroll\n    for (int j = 0; j < " << d.FN
    << "; ++j)\n#pragma unroll\n    for (int r = 0; r < 4; ++r) Cs[(wm * " << d.PW << " + f * 16 + (l >> 4) * 4 + r) * "
    << d.LDC << " + wn * " << d.WTN << " + j * 16 + (l & 15)] = acc[f][j][r];\n";
  s << "    __syncthreads();\n";
  s << "    {\n    " << origin("t");
  if (sp.nb) s << "    const i64 z0 = z_;\n";
  s << "    (void)z_;\n";
  s << epi;
  s << "    }\n";
  s << "    if (more) stash_halo(b ^ 1);\n";
  s << "    __syncthreads();\n";
  s << "    if (!more) break;\n";
  s << "    t = tn;\n    b ^= 1;\n";
  s << "  }\n";
  s << "}\n";
  gk.source = s.str();
  gk.grid[0] = (int)d.G;
  gk.block[0] = 256;
  gk.lds_bytes = (int)d.smem;
  ki.fill_cost(gk);
  return gk;
}

}  // namespace korch
