// Matrix-core (MFMA) prefill for bfloat16 inputs, P = 4: per-block variant.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "prefill_mfma.hpp"

namespace sata {

// True if the per-block kernel covers this shape; fills the plan.
bool plan_prefill_blocks(int BH, int n, int dk, int dv, int P, int chunk, MfmaPrefillPlan* plan);

hipError_t launch_prefill_blocks(const void* q, const void* k, const void* v, void* y, float* S_out, int BH,
                                 int n, int dk, int dv, int P, int chunk, const MfmaPrefillPlan& plan,
                                 void* workspace, hipStream_t s, int qg = 1);

}  // namespace sata
