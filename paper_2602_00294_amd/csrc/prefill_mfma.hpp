// Matrix-core (MFMA) prefill for bfloat16 inputs.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sata {

struct MfmaPrefillPlan {
  size_t workspace_bytes = 0;
};

// True if a matrix-core kernel covers this shape; fills the plan.
bool plan_prefill_mfma(int BH, int n, int dk, int dv, int P, int chunk, MfmaPrefillPlan* plan);

hipError_t launch_prefill_mfma(const void* q, const void* k, const void* v, void* y, float* S_out, int BH,
                               int n, int dk, int dv, int P, int chunk, const MfmaPrefillPlan& plan,
                               void* workspace, hipStream_t s);

}  // namespace sata
