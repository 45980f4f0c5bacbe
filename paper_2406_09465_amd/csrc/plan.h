// Orchestration plans: validation, workspace planning, compiled kernels.
#pragma once

#include <map>
#include <string>
#include <vector>

#include "codegen.h"
#include "ir.h"

namespace korch {

// Where a tensor lives at execution time.
struct Storage {
  enum Kind { GraphInput, GraphOutput, Workspace, Counters } kind = Workspace;
  int index = 0;        // graph input / output position
  size_t offset = 0;    // byte offset in the workspace or counter buffer
};

struct CompiledKernel {
  KernelDesc desc;
  GenKernel gen;
  std::vector<char> code;        // gfx950 code object
  std::vector<Storage> arg_storage;
  void* module = nullptr;        // hipModule_t
  void* function = nullptr;      // hipFunction_t
  int device = -1;
};

struct Plan {
  Graph g;
  std::vector<KernelDesc> kernels;
  std::vector<CompiledKernel> ck;
  bool compiled = false;
  bool loaded = false;
  size_t ws_bytes = 0;
  size_t counter_bytes = 0;
  void* counters = nullptr;      // device buffer owned by the plan
  int counter_device = -1;
  std::map<int, size_t> ws_offset;  // workspace-resident materialized node -> offset
  std::string name_prefix = "korch_k";  // kernel symbols: <prefix><index>_<family>
};

// Checks a plan against Definitions 1 and 3 and the ordered dependency /
// output constraints; throws Error with the matching status.
void validate_plan(const Graph& g, const std::vector<KernelDesc>& ks, bool strict_single_output);
std::vector<KernelDesc> unfused_plan(const Graph& g);
// Storage node a kernel reads for external node u after kernels [0, k) ran.
int resolve_storage(const Graph& g, const std::vector<KernelDesc>& ks, int k, int u);
void plan_workspace(Plan& p);
void compile_plan(Plan& p);

// Execution states reached by the search of Algorithm 1 (primitive nodes only).
std::vector<Bits> execution_states(const Graph& g, size_t max_states);

}  // namespace korch
