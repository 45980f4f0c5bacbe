// Shared pieces of the MFMA product families (GEMM, conv, split-K).
#pragma once

#include <map>
#include <set>
#include <string>
#include <vector>

#include "families.h"

namespace korch {

struct GemmSpec {
  bool conv = false;
  std::vector<int> mms;     // products (primary first)
  int A = -1;               // left operand node (conv: input X)
  std::vector<int> Bs;      // right operand per product (conv: weights W)
  std::set<int> pro, epi;   // prologue / epilogue primitives
  std::vector<int> rowred;  // reductions over the product's last axis (epilogue)
  std::vector<int> side;    // reductions that read the left operand's prologue
  Shape OUT;                // iteration space of the epilogue
  int nb = 0;               // leading batch dims of OUT
  int nmdims = 1;           // dims of OUT that form the M index
  int64_t M = 0, N = 0, K = 0, batch = 1;
  std::vector<int64_t> Nj, offj;
  int64_t Ntot = 0;
  int mtype = KORCH_F16;
  // convolution geometry
  int64_t H = 0, W = 0, Cin = 0, KH = 0, KW = 0, stride = 1, pad = 0, Ho = 0, Wo = 0;
  // tiling
  int BM = 128, BN = 128, BK = 32, BKP = 40, kstep = 32, WM = 2, WN = 2, WTM = 64, WTN = 64, FM = 4, FN = 4;
  int VA = 8, VB = 8, LDC = 132;
  int NT = 256;  // threads per workgroup (64 per wave)
  int NS = 2;    // register pipeline stages (tiles loaded ahead of the one multiplied)
  // Right operand staged raw in LDS as [k][n] (n contiguous, pitch BNP) and
  // read into MFMA fragments with transposing LDS reads (half precision) or
  // plain reads (fp32); otherwise staged as [n][k] with pitch BKP.
  bool b_kn = false;
  int BNP = 0;
  // Each block of 8 rows starts BSH elements after the previous block ends
  // (row k at k * BNP + (k / 8) * BSH): one half-wave of transposing reads
  // covers rows {0..3, 8..11} (+ 16 j), and the relative shift of the second
  // block puts those eight 32-byte windows on distinct LDS banks.
  int BSH = 0;
  // Rows of the fp32 C tile staged in LDS at once for the epilogue (0 = BM).
  int CROWS = 0;
  // Scheduling hints for the unrolled main loop (both operands staged by
  // branch-free buffer loads): LDS writes and global loads per thread and
  // k-tile; 0 leaves the instruction order to the compiler.
  int sched_w = 0, sched_g = 0;
  // Transposed accumulators: the MFMAs take the right operand's fragment as
  // their first source, so lane l of 16 x 16 block (i, j) holds row l % 16 and
  // the four consecutive columns 4 (l / 16) .. + 3 (the register epilogue).
  bool acc_t = false;
  // Main loop with each tile's last k-step after the barrier (see mfma_mainloop).
  bool split_steps = false;
  // Register epilogue: output staging tile in LDS (elements per row; 0 = none).
  int OSP = 0;
  int OSB = 0;  // its bytes
  // Direct-to-LDS staging (plain 16-bit operands, tiles dividing the problem,
  // k-tiles of 64): operand tiles go from global memory straight into LDS, in
  // swizzled layouts, with no register round trip and no LDS write
  // instructions.  The right operand's chunk c of row k is stored at
  // c ^ f(k), f(k) = dx0 (k & 1) + dx1 ((k >> 1) & 1) + dx3 ((k >> 3) & 1).
  bool dma = false;
  int dx0 = 0, dx1 = 0, dx3 = 0;
  int dsb = 2;  // right-operand stages
  int dsa = 2;  // left-operand stages (3: loaded two k-tiles ahead like the right operand)
  bool want_a3 = false;  // ask plan_dma for three left-operand stages
  // LayerNorm folded into the product (see detect_ln_fold): the left operand
  // is LN(X) = (X - mu) r gamma + beta over X's last axis; the kernel stages X,
  // multiplies X gamma by the right operand W, accumulates each row's sum and
  // sum of squares from the staged X and the column sums gamma^T W and
  // beta^T W from the staged W, and provides the product as
  // r (acc - mu gamma^T W) + beta^T W.
  bool lnf = false;
  int lnX = -1, lng = -1, lnb = -1;
  int lng_slot = -1, lnb_slot = -1;  // kernel argument slots of gamma and beta
  double lneps = 0;
  std::set<int> lnset;  // the LayerNorm's primitives (mean ... affine)
};

// Decides direct-to-LDS staging (sets sp.dma) once tiles and the epilogue are known.
void plan_dma(const KInfo& ki, GemmSpec& sp, bool ksplit);

// LDS element offset of row k of the [k][n] right-operand tile.
std::string b_row_off(const GemmSpec& sp, const std::string& k);
// Elements of one LDS buffer of the right operand.
int64_t b_buf_elems(const GemmSpec& sp);

// Decides operand staging layouts once the tiles are chosen.
void plan_operands(const KInfo& ki, GemmSpec& sp);

bool analyze_gemm(const KInfo& ki, GemmSpec& sp, std::string* why, bool allow_reduce);
void choose_tiles(GemmSpec& sp, bool split);
std::string operand_loader(const KInfo& ki, const GemmSpec& sp, bool isA, const std::map<int, int>& slot);
// kconst: number of k-tiles when it is a compile-time constant (the loop is then
// unrolled completely and uses sp.NS register stages), else 0; kconst_exact:
// every workgroup runs exactly kconst tiles (else tiles at or past kt1 are
// skipped).
// ctile: write the accumulators to the fp32 C tile at smem (and synchronize)
// after the loop.
std::string mfma_mainloop(const GemmSpec& sp, const std::string& hook = "", int64_t kconst = 0,
                          bool kconst_exact = true, bool ctile = true);
// Pointwise epilogue over the fp32 C tile `Cs` (row `cs_row`, an expression of
// the local row `mlc` or the tile row `ml`).  It covers `rows` tile rows (0 =
// BM) starting at tile row `row0`.  conv_tw > 0: the tile is a 2-D block of
// output pixels conv_tw wide whose origin is (ty0, tx0), and C tile row ml
// holds pixel (ml / conv_tw, ml % conv_tw).
// Loads that are the same for every element a thread visits (per-column
// vectors such as a BatchNorm scale, when the workgroup's thread count is a
// multiple of the column vectors of a row) are issued once before the element
// loop; with `hoisted` set they are returned there instead, for the caller to
// place before a loop over several tiles of the same columns.
std::string gemm_epilogue(const KInfo& ki, const GemmSpec& sp, const std::map<int, int>& slot,
                          const std::string& cs_row, const std::set<int>& skip = {}, int conv_tw = 0,
                          int rows = 0, const std::string& row0 = "0", std::string* hoisted = nullptr);
// Direct convolution (stride 1, half precision, input halo tile in LDS,
// weights in registers); conv_direct_fits says whether it applies.
bool conv_direct_fits(const GemmSpec& sp, std::string* why);
// conv_direct_fits and not switched off (KORCH_CONV_DIRECT=0 keeps the
// implicit-GEMM kernel, which takes no operand prologue).
bool conv_uses_direct(const GemmSpec& sp, std::string* why);
GenKernel gen_conv_direct(const KInfo& ki, GemmSpec& sp, int index);
std::string gemm_prologue_common(const GemmSpec& sp);
// Register epilogue of a single product whose kernel has one output of the
// product's shape in a 16-bit dtype and whose epilogue reads, besides the
// product, only values that are the same along the product's rows (per-column
// vectors, scalars): the output is evaluated on the accumulators themselves
// (transposed layout), staged once in LDS in its storage dtype and stored as
// 16-byte rows.  Returns the output node, or -1 when the case does not apply.
int reg_epilogue_output(const KInfo& ki, const GemmSpec& sp);
std::string gemm_reg_epilogue(const KInfo& ki, const GemmSpec& sp, const std::map<int, int>& slot, int out);
size_t gemm_smem_bytes(const GemmSpec& sp);

}  // namespace korch
