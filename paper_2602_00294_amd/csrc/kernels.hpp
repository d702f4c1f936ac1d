// Internal launch interface between the C ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sata {

// Zero entries (degree 0, weight 0) that follow the D features of a device
// table, so that kernels may read whole slices of up to this many features
// past the last one without a bounds check.
constexpr int kTablePad = 4096;
// Features per block of the generation program (table.hpp build_gen_program).
constexpr int kGenBlock = 32;

// One (d, P) feature table resident on a device (see table.hpp for its layout).
struct DevTable {
  const uint64_t* packed = nullptr;  // [D + kTablePad] packed multi-indices
  const float* weight = nullptr;     // [D + kTablePad] feature weights
  const uint32_t* gen = nullptr;     // [D + kTablePad][2] generation program (blocks of kGenBlock)
  int64_t D = 0;
  int d = 0;
  int P = 0;
};

// ---- feature map -------------------------------------------------------------
hipError_t launch_feature_map(const void* x, bool bf16, int64_t rows, const DevTable& t,
                              float* phi, hipStream_t s);

// ---- decode step -------------------------------------------------------------
struct DecodePlan {
  int fps = 0;      // features per workgroup slice
  int nslices = 0;  // slices per head (1: one workgroup streams the whole head)
  int threads = 0;  // workgroup size
  int flat_tu = 0;  // > 0: whole-head float4 streaming kernel with this many threads in use
  size_t flat_lds = 0;
  int flat_nth = 1024;  // threads per workgroup of the flat kernel (256 or 1024)
  int flat_np = 1;      // workgroups (pieces) per head
  int flat_steps = 0;   // float4 steps per thread over a whole head
  int flat_rows = 0;    // state rows a piece touches at most (its feature values in LDS)
  float even_share = 0.5f;  // share of each (even, odd) pair of pieces streamed by the even one
};
DecodePlan plan_decode(int64_t D, int dk, int dv, int BH);
// partial: BH * n * (dv + 1) floats with n = nslices when nslices > 1 and the
// state is not 16-byte aligned, n = flat_np when flat_np > 1; counters: BH
// ints, all zero, when flat_np > 1 (the kernel leaves them zero).
// R (may be null): per head D + (dk + 1) * dv float32 residuals of the
// compensated entries (normaliser column, degree-0 and degree-1 rows); only
// the flat kernel takes them (decode_supports_residuals).
hipError_t launch_decode(float* S, const void* q, const void* k, const void* v, void* y, bool bf16,
                         int BH, int dk, int dv, const DevTable& t, const DecodePlan& plan,
                         float* partial, int* counters, hipStream_t s, float* R = nullptr);
bool decode_supports_residuals(const DecodePlan& plan, const float* S);
// Share of each (even, odd) pair of decode pieces for the even one on the current device.
float xcd_even_share();

// ---- decode step, grouped query heads ------------------------------------------
struct GroupedDecodePlan {
  int tu = 0;      // > 0: supported; threads of the workgroup taking part in the stream
  size_t lds = 0;
  int nth = 1024;  // threads per workgroup (256 or 1024)
  int np = 1;      // workgroups (pieces) per key/value head
  int steps = 0;   // float4 steps per thread over a whole head
  int rows = 0;    // state rows a piece touches at most
  int G = 0;       // query heads per key/value head (2, 4 or 8)
  float even_share = 0.5f;  // share of each (even, odd) pair of pieces streamed by the even one
};
GroupedDecodePlan plan_decode_grouped(int64_t D, int dk, int dv, int BH, int G);
// BH key/value heads; S 16-byte aligned; partial: BH * np * G * (dv + 1)
// floats and counters: BH ints, all zero, when np > 1.
hipError_t launch_decode_grouped(float* S, const void* q, const void* k, const void* v, void* y, bool bf16,
                                 int BH, int dk, int dv, const DevTable& t, const GroupedDecodePlan& plan,
                                 float* partial, int* counters, hipStream_t s);

// ---- prefill, generic float32 path --------------------------------------------
struct PrefillGenericPlan {
  int fs = 0;        // features per slice
  int nslices = 0;   // slices per head
  int seg_len = 0;   // tokens per segment (multiple of the chunk)
  size_t lds_main = 0;
  size_t lds_final = 0;
  size_t partial_bytes = 0;
};
// Returns false if no slice size fits the on-chip memory.
bool plan_prefill_generic(int64_t D, int BH, int n, int dk, int dv, int chunk, size_t max_ws_bytes,
                          PrefillGenericPlan* plan);
hipError_t launch_prefill_generic(const void* q, const void* k, const void* v, void* y, bool bf16,
                                  int BH, int n, int dk, int dv, int chunk, const DevTable& t,
                                  const PrefillGenericPlan& plan, float* S_state, float* partial,
                                  hipStream_t s, int qg = 1);

// One segment of the float32 prefill's main kernel only: the partial readouts
// of tokens [seg0, seg0 + plan.seg_len) against S_state, which it carries from
// the previous segment (first: from zero).
hipError_t launch_prefill_generic_readout(const void* q, const void* k, const void* v, bool bf16, int BH, int n,
                                          int dk, int dv, int chunk, const DevTable& t,
                                          const PrefillGenericPlan& plan, float* S_state, float* partial, int seg0,
                                          int seg_len, bool first, hipStream_t s);

// ---- prefill, matrix cores with generated features (prefill_feat.hip) ---------
// Any d_k, d_v <= 64 and P >= 2 with 64-token chunks; state in accumulators.
struct FeatPrefillPlan {
  int nct = 0;             // column tiles of 16 covering d_v + 1
  bool split = false;      // split operands (hi + lo bfloat16 pairs, three products per product)
  bool narrow = false;     // slices of 256 features (for few features or few heads)
  int nslices = 0;         // workgroups per head
  int seg_len = 0;         // tokens per segment (partial sums of one segment in the workspace)
  int parts = 1;           // parts of a one-segment call that run side by side (states summed first)
  int part_len = 0;        // tokens per part
  size_t part_state_offset = 0;  // workspace bytes before the parts' states
  size_t lds_main = 0;
  size_t partial_bytes = 0;  // the whole workspace: partials, then the parts' states
};

// True if the kernel covers this shape (chunk 64, P >= 2, d_k, d_v <= 64).
bool plan_prefill_feat(int64_t D, int BH, int n, int dk, int dv, int P, int chunk, bool split, size_t max_ws_bytes,
                       FeatPrefillPlan* plan);

// Whole prefill: bf16 inputs with bf16 operands (plan.split false), float32
// inputs with split operands (plan.split true).  S_state: [BH][D][d_v+1]
// float32, the state after the call (carried between segments); partial:
// plan.partial_bytes.  q holds qg query heads per head.
hipError_t launch_prefill_feat(const void* q, const void* k, const void* v, void* y, int BH, int n, int dk, int dv,
                               int P, const DevTable& t, const FeatPrefillPlan& plan, float* S_state, float* partial,
                               hipStream_t s, int qg = 1);

// One segment [seg0, seg0 + plan.seg_len) of the readout only, with split
// operands whatever the input type: the slices' partial readouts, summed into
// slice 0 of partial ([slice][BH][seg_len][d_v+1]), and S_state carried
// (from zero when first).
hipError_t launch_prefill_feat_readout(const void* q, const void* k, const void* v, bool bf16_in, int BH, int n,
                                       int dk, int dv, const DevTable& t, const FeatPrefillPlan& plan,
                                       float* S_state, float* partial, int seg0, bool first, hipStream_t s);

// ---- backward ----------------------------------------------------------------
constexpr int kMaxBackwardDim = 64;
struct BackwardPlan {
  int fs = 0;              // features per slice of the scan kernels
  int nslices = 0;         // slices per head
  int seg_len = 0;         // tokens per segment (multiple of the chunk)
  size_t lds_main = 0, lds_h = 0, lds_fin = 0;
  size_t partial_bytes = 0;  // partial sums of one segment
  size_t h_bytes = 0;        // dL/do for every token, float32 [BH][n][d_v+1]
  size_t state_bytes = 0;    // one float32 state [BH][D][d_v+1]
  bool feat_fwd = false;     // the forward readout of pass 1 on the matrix cores (split operands)
  FeatPrefillPlan feat;      // its plan (seg_len = the backward's)
};
// False if d_k or d_v exceeds kMaxBackwardDim, the chunk is not 16, 32 or 64,
// or no slice fits on chip.  Also fills the forward plan of the first pass.
bool plan_backward(int64_t D, int BH, int n, int dk, int dv, int P, int chunk, size_t max_ws_bytes, BackwardPlan* plan,
                   PrefillGenericPlan* fwd);
hipError_t launch_backward(const void* q, const void* k, const void* v, const void* dy, void* dq, void* dk,
                           void* dv, bool bf16, int BH, int n, int dk_, int dv_, int P, int chunk, const DevTable& t,
                           const BackwardPlan& plan, const PrefillGenericPlan& fwd, float* h, float* state,
                           float* partial, hipStream_t s);

// ---- helpers -----------------------------------------------------------------
hipError_t launch_fill_zero(float* p, int64_t count, hipStream_t s);

}  // namespace sata
