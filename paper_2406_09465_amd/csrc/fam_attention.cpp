// Attention family (placeholder until implemented).
#include "families.h"

namespace korch {

bool match_attention(const KInfo&, std::string* why) {
  *why = "attention: not available";
  return false;
}

GenKernel gen_attention(const KInfo&, int) { fail(KORCH_E_UNSUPPORTED, "attention: not available"); }

}  // namespace korch
