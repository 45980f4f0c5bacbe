// Internal interface between the family dispatcher and the family generators.
#pragma once

#include <map>
#include <set>
#include <string>
#include <vector>

#include "codegen.h"

namespace korch {

// Facts about one kernel (P', O) used by every matcher.
struct KInfo {
  const Graph& g;
  const KernelDesc& k;
  std::set<int> in;           // P'
  std::vector<int> ext;       // external producers read by the kernel (sorted)
  std::vector<int> linear, reduces, layouts;
  KInfo(const Graph& g, const KernelDesc& k);
  bool ancestor(int u, int v) const;  // path u ~> v
  // Pointer slots: external tensors first, then outputs in O order.
  void assign_args(GenKernel& gk, std::map<int, int>& slot) const;
  int out_slot(int o) const;
  void fill_cost(GenKernel& gk) const;
};

std::string kernel_name(int index, const char* fam);
// Prefix of the kernel symbols generated on this thread ("korch_k" for plans).
void set_kernel_prefix(const std::string& prefix);
void choose_row_geometry(int64_t L, int elem_bytes, int& G, int& VEC, int& NC);

bool match_pointwise(const KInfo& ki, std::string* why);
bool match_row(const KInfo& ki, std::string* why);
bool match_colreduce(const KInfo& ki, std::string* why);
bool match_gemm(const KInfo& ki, std::string* why);
bool match_conv(const KInfo& ki, std::string* why);
bool match_splitk(const KInfo& ki, std::string* why);
bool match_attention(const KInfo& ki, std::string* why);

GenKernel gen_pointwise(const KInfo& ki, int index);
GenKernel gen_row(const KInfo& ki, int index);
GenKernel gen_colreduce(const KInfo& ki, int index);
GenKernel gen_gemm(const KInfo& ki, int index);
GenKernel gen_splitk(const KInfo& ki, int index);
GenKernel gen_attention(const KInfo& ki, int index);

}  // namespace korch
