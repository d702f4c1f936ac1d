// Matrix-core (MFMA) prefill for bfloat16 inputs (not yet enabled).
#include "prefill_mfma.hpp"

namespace sata {

bool plan_prefill_mfma(int, int, int, int, int, int, MfmaPrefillPlan*) { return false; }

hipError_t launch_prefill_mfma(const void*, const void*, const void*, void*, float*, int, int, int, int, int,
                               int, const MfmaPrefillPlan&, void*, hipStream_t) {
  return hipErrorInvalidValue;
}

}  // namespace sata
