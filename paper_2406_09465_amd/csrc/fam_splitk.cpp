// Split-K contraction family (placeholder until implemented).
#include "gemm_common.h"

namespace korch {

bool match_splitk(const KInfo&, std::string* why) {
  *why = "splitk: not available";
  return false;
}

GenKernel gen_splitk(const KInfo&, int) { fail(KORCH_E_UNSUPPORTED, "splitk: not available"); }

}  // namespace korch
