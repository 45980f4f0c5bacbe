// Primitive-graph IR, plan representation and shared host utilities.
//
// A primitive graph G = (P, E) (Korch, Section 4) is stored as nodes in
// creation order; every node's inputs precede it, so creation order is a
// topological order.  Shapes are static and inferred when a node is added.
#pragma once

#include <cstdint>
#include <memory>
#include <stdexcept>
#include <string>
#include <vector>

#include "korch.h"

namespace korch {

// Error carrying a korch_status; converted to a return code at the ABI.
struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};

[[noreturn]] inline void fail(int code, const std::string& msg) { throw Error(code, msg); }

using Shape = std::vector<int64_t>;

int64_t numel(const Shape& s);
std::string shape_str(const Shape& s);
int dtype_bytes(int dtype);
const char* dtype_name(int dtype);

enum class Kind { Input, Unary, Binary, Reduce, Broadcast, Layout, Linear };
Kind op_kind(int op);
const char* op_name(int op);
bool is_elementwise(int op);

struct Node {
  int id = 0;
  int op = KORCH_INPUT;
  std::vector<int> in;
  korch_attrs attrs{};
  Shape shape;
  int dtype = KORCH_F32;
  int axis = 0;  // normalized reduce / concat axis
};

// Dynamic bitset over node ids.
struct Bits {
  std::vector<uint64_t> w;
  explicit Bits(size_t n = 0) : w((n + 63) / 64, 0) {}
  void set(int i) { w[i >> 6] |= (uint64_t(1) << (i & 63)); }
  void reset(int i) { w[i >> 6] &= ~(uint64_t(1) << (i & 63)); }
  bool test(int i) const { return (w[i >> 6] >> (i & 63)) & 1; }
  bool any_and(const Bits& o) const {
    for (size_t k = 0; k < w.size(); ++k)
      if (w[k] & o.w[k]) return true;
    return false;
  }
  void or_with(const Bits& o) {
    for (size_t k = 0; k < w.size(); ++k) w[k] |= o.w[k];
  }
  bool operator==(const Bits& o) const { return w == o.w; }
  bool operator<(const Bits& o) const { return w < o.w; }
  bool subset_of(const Bits& o) const {
    for (size_t k = 0; k < w.size(); ++k)
      if (w[k] & ~o.w[k]) return false;
    return true;
  }
  int count() const {
    int c = 0;
    for (auto x : w) c += __builtin_popcountll(x);
    return c;
  }
};

struct Graph {
  std::vector<Node> nodes;
  std::vector<int> inputs;   // graph input node ids in creation order
  std::vector<int> outputs;  // graph output node ids in korch_graph_output order
  bool finalized = false;
  std::vector<std::vector<int>> consumers;
  std::vector<Bits> reach;  // reach[u]: nodes reachable from u by a non-empty path

  int add_input(int dtype, const Shape& shape);
  int add_op(int op, const std::vector<int>& in, const korch_attrs* attrs, int dtype);
  void add_output(int node);
  void finalize();
  bool is_output(int node) const;
  bool is_prim(int node) const { return nodes[node].op != KORCH_INPUT; }
  // A contiguous reshape is a view: it aliases its input's storage.
  bool is_view(int node) const { return nodes[node].op == KORCH_RESHAPE; }
  // Storage root of a view chain.
  int view_root(int node) const;
};

// One kernel (P', O) of a plan.
struct KernelDesc {
  std::vector<int> prims;  // sorted ascending (topological)
  std::vector<int> outs;   // sorted ascending
};

bool is_convex(const Graph& g, const std::vector<int>& nodes);
std::vector<int> external_inputs(const Graph& g, const KernelDesc& k);

}  // namespace korch
