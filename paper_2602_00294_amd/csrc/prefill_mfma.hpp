// Matrix-core (MFMA) prefill for bfloat16 inputs, P = 4.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sata {

struct MfmaPrefillPlan {
  int dk = 0, dv = 0;
  int nslices = 0;        // workgroups per head
  size_t partial_bytes = 0;
  size_t workspace_bytes = 0;
};

// True if a matrix-core kernel covers this shape; fills the plan.
bool plan_prefill_mfma(int BH, int n, int dk, int dv, int P, int chunk, MfmaPrefillPlan* plan);

hipError_t launch_prefill_mfma(const void* q, const void* k, const void* v, void* y, float* S_out, int BH,
                               int n, int dk, int dv, int P, int chunk, const MfmaPrefillPlan& plan,
                               void* workspace, hipStream_t s, int qg = 1);

}  // namespace sata
