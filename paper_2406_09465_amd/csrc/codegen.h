// Kernel-family matching and HIP source generation for gfx950.
//
// A kernel (P', O) of a plan is matched to one hand-written kernel family
// (pointwise, row program, column reduction, MFMA GEMM / implicit-GEMM conv,
// split-K contraction, attention).  The family's skeleton is specialized by
// emitting the kernel's own per-element expressions as C++ and compiling the
// result at run time for gfx950.  A kernel no family implements is
// "unsupported", the infinite cost of Korch's profiler (Section 4.1).
#pragma once

#include <functional>
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <vector>

#include "ir.h"

namespace korch {

// One pointer argument of a generated kernel.
struct ArgRef {
  enum Kind { Tensor, Output, Scratch, Counter } kind = Tensor;
  int node = -1;       // Tensor: node whose storage is read; Output: node written
  size_t bytes = 0;    // Scratch / Counter: size
};

struct GenKernel {
  int family = KORCH_FAM_NONE;
  std::string name;
  std::string source;
  int grid[3] = {1, 1, 1};
  int block[3] = {256, 1, 1};
  int lds_bytes = 0;  // static LDS (informational)
  std::vector<ArgRef> args;
  double alg_bytes = 0, alg_flops = 0;
};

// Family matcher only (no source); returns the family or KORCH_FAM_NONE with a reason.
int match_family(const Graph& g, const KernelDesc& k, std::string* why);
// Full specialization; throws Error(KORCH_E_UNSUPPORTED) when no family matches.
GenKernel generate_kernel(const Graph& g, const KernelDesc& k, int index);

// ---------------------------------------------------------------------------
// Shared code-generation machinery (used by the family generators).
// ---------------------------------------------------------------------------

// Integer index expression  base + c*e  where e is the vector-lane variable of
// the current emission (0..VEC-1).  `al` records that base is a multiple of al.
struct Ix {
  std::string b = "0";
  int64_t c = 0;
  int64_t al = 1;
  bool affine = true;
  bool konst = true;
  int64_t kv = 0;
  static Ix k(int64_t v);
  static Ix var(const std::string& name, int64_t coef = 0, int64_t align = 1);
  std::string at(const std::string& e = "e") const;  // full C++ expression
  bool is_zero() const { return konst && kv == 0 && c == 0; }
};

Ix ix_add(const Ix& a, const Ix& b);
Ix ix_addk(const Ix& a, int64_t v);
Ix ix_mulk(const Ix& a, int64_t v, int vec);
Ix ix_divk(const Ix& a, int64_t s, int vec);
Ix ix_modk(const Ix& a, int64_t s, int vec);

std::string ctype(int dtype);                 // "float" / "f16" / "bf16"
std::string flit(double v);                   // float literal
std::string unary_expr(int op, const std::string& x);
std::string binary_expr(int op, const std::string& x, const std::string& y);

// Kernels whose outputs are all fp16 / bf16 use the fast transcendental
// variants (set per generated kernel; thread-local).
void set_fast_math(bool on);
bool fast_math();
// Register relief (thread-local, set while a kernel is regenerated because
// its first code object spilled registers to scratch): families that can
// trade speed for fewer live registers do so at levels 1, 2, ...
void set_reg_relief(int level);
int reg_relief();
constexpr int kMaxRegRelief = 2;
// The fissioned Mish pattern rooted at `node` (a product); returns its input or -1.
int mish_operand(const Graph& g, const std::set<int>& inset, int node);

// Row-major strides of a shape.
std::vector<int64_t> strides_of(const Shape& s);

// Generic per-element emitter.  Produces the fp32 value of a node at an index
// (one Ix per dimension) by walking the kernel's elementwise / broadcast /
// layout nodes down to external tensors (loads) or to values supplied by the
// family skeleton through `provide` (e.g. a matrix-product accumulator).
struct Emitter {
  const Graph& g;
  std::set<int> inset;                 // nodes computed inside this kernel
  std::map<int, int> argslot;          // external storage node -> pointer slot
  int vec = 1;
  std::ostringstream pre;              // statements before the lane loop
  std::ostringstream body;             // statements inside the lane loop
  std::function<bool(int, const std::vector<Ix>&, std::string*)> provide;
  bool force_gather = false;           // all loads per-lane (guarded contexts)
  std::string gather_guard;            // when set, gathers read zero where it is false, without a branch
  int n_guard_fallback = 0;            // gathers of tensors too large for that form
  int tmp = 0;
  int guard_depth = 0;                 // enclosing guards whose condition varies with the vector lane
  // Enclosing guards whose condition is the same for every lane of a vector
  // (e.g. a spatial pad around a channel vector): loads under them are still
  // hoisted as uniform / vector loads, each executed only when the guards hold.
  std::vector<std::string> lane_invariant_guards;
  int n_gather = 0, n_vector = 0, n_uniform = 0;
  std::vector<std::map<std::string, std::string>> memo{1};
  // Staged loads: a hoisted (uniform or vector) load becomes an assignment into
  // an array of the tensor's own type, declared in `stage_decl` with
  // [stages][slots] extents and indexed by the generated variables `st` and
  // `i`; the value is read back (converted to float) where it is used.  The
  // loads can then be issued one pipeline stage ahead of the arithmetic.
  bool staged = false;
  int stages = 2, slots = 1;
  std::ostringstream stage_decl;
  // When set, the only index variable that differs between the slots of one
  // thread: a staged load whose offset does not use it is issued once per stage
  // (slot 0) and shared by all slots.
  std::string slot_var;
  // Loop-invariant loads: when `varying` is set, a hoisted (non-staged) load
  // whose offset uses none of these iteration variables is the same for every
  // element a thread visits.  It goes to `inv` instead of `pre`, as a
  // declaration followed by a block that opens with `inv_defs` (definitions
  // of the invariant variables the offset uses) and loads only when
  // `inv_guard` holds (the value stays 0 otherwise).
  std::vector<std::string> varying;
  std::string inv_defs, inv_guard;
  std::ostringstream inv;
  int n_invariant = 0;

  Emitter(const Graph& gg) : g(gg) {}
  std::string value(int node, const std::vector<Ix>& idx);
  std::string load(int node, const std::vector<Ix>& idx);
  std::string fresh(const char* p) { return "_" + std::string(p) + std::to_string(tmp++); }
  static std::string key(int node, const std::vector<Ix>& idx);
};

// Index of every dimension of `shape` when the tensor is read with numpy-style
// right-aligned broadcasting at iteration index `it` (size-1 dims -> 0).
std::vector<Ix> broadcast_index(const Shape& shape, const Shape& itshape, const std::vector<Ix>& it);

// Common header for generated sources.
std::string source_header(int nargs);

// Store of V consecutive elements of kernel output `node` from the float array
// `src` (V = 0: the one float value `src`) at element offset `off` of its
// storage `P` (a uniform base pointer): written
// through to the device's point of coherence (`stv_out` / `st1_out`) unless the
// tensor is 2 GiB or larger or `plain` asks for ordinary stores.
std::string out_store(const Graph& g, int node, const std::string& P, const std::string& off, int V,
                      const std::string& src, bool plain = false);

}  // namespace korch
