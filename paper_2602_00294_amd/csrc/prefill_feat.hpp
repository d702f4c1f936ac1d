// Matrix-core prefill for any d_k, d_v <= 64 and P >= 2 (64-token chunks):
// features generated directly, state in accumulators.  bfloat16 inputs take
// bfloat16 operands; float32 inputs take split operands (hi + lo bfloat16
// pairs, three products per product).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kernels.hpp"

namespace sata {

struct FeatPrefillPlan {
  int nct = 0;             // column tiles of 16 covering d_v + 1
  bool split = false;      // float32 inputs, split operands
  bool narrow = false;     // slices of 256 features (for few features or few heads)
  int nslices = 0;         // workgroups per head
  int seg_len = 0;         // tokens per segment (partial sums of one segment in the workspace)
  size_t lds_main = 0;
  size_t partial_bytes = 0;
};

// True if the kernel covers this shape (chunk 64, P >= 2, d_k, d_v <= 64);
// split: float32 inputs (else bfloat16).
bool plan_prefill_feat(int64_t D, int BH, int n, int dk, int dv, int P, int chunk, bool split, size_t max_ws_bytes,
                       FeatPrefillPlan* plan);

// S_state: [BH][D][d_v+1] float32, the state after the call (carried between
// segments); partial: plan.partial_bytes.  q holds qg query heads per head.
hipError_t launch_prefill_feat(const void* q, const void* k, const void* v, void* y, int BH, int n, int dk, int dv,
                               int P, const DevTable& t, const FeatPrefillPlan& plan, float* S_state, float* partial,
                               hipStream_t s, int qg = 1);

}  // namespace sata
