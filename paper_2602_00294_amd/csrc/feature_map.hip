// Feature map phi(x) for rows of coordinates (Sec. 2.4, "Efficient
// Computation"): each output is a monomial's weight times the product of its
// indices' coordinates.  The kernel is bound by the HBM writes of the
// float32 output, D / d times the input.
//
// A workgroup takes kRows rows and 256 consecutive features (one per thread);
// workgroups that write the same rows run on one XCD (see the tile remap).
// Each thread reads its feature's generation-program word once (x offset of
// the last index, the first two other indices, a flag for more, the weight;
// table.hpp build_gen_program), so a row costs three LDS reads, three
// multiplies and one store.  The rows' coordinates sit in LDS transposed,
// [index][row] with a stride of kRows + 1 floats (distinct banks for distinct
// indices), plus an index d held at 1 for features of lower degree, so every
// read of a given index takes an immediate row offset.  Consecutive threads
// write consecutive features of a row.
#include <hip/hip_runtime.h>

#include "device_common.hpp"
#include "kernels.hpp"

namespace sata {

namespace {

constexpr int kRows = 32;       // rows per workgroup
constexpr int kFmThreads = 256;  // features per workgroup
constexpr int kXT = kRows + 1;  // LDS floats per coordinate index

template <typename T>
__global__ void __launch_bounds__(kFmThreads)
feature_map_kernel(const T* __restrict__ x, int64_t rows, int d, const uint32_t* __restrict__ gen,
                   const uint64_t* __restrict__ packed, int64_t D, float* __restrict__ phi) {
  extern __shared__ float xt[];  // [d + 1][kXT]
  // workgroups are dealt to the 8 XCDs in turn by linear index; with more
  // than one feature block per row, the remap gives each XCD a contiguous run
  // of (row block, feature block) tiles, so that the neighbouring feature
  // blocks of a row, which share the cache lines at their edges, are written
  // through the same L2 (one feature block writes whole rows: no remap)
  int64_t rb = blockIdx.y, fb = 0;
  if (gridDim.x > 1) {
    const int64_t nblk = (int64_t)gridDim.x * gridDim.y;
    const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
    const int64_t per_xcd = nblk / 8;
    const int64_t tile = lin < 8 * per_xcd ? (lin % 8) * per_xcd + lin / 8 : lin;
    rb = tile / gridDim.x;
    fb = tile % gridDim.x;
  }
  const int64_t r0 = rb * kRows;
  const int nr = (int)min<int64_t>(kRows, rows - r0);
  const int tid = threadIdx.x;
  for (int i = tid; i < kRows * d; i += kFmThreads) {
    const int r = i / d;
    const int c = i - r * d;
    xt[c * kXT + r] = r < nr ? to_f32(x[(r0 + r) * d + c]) : 0.f;
  }
  for (int r = tid; r < kRows; r += kFmThreads) xt[d * kXT + r] = 1.f;
  __syncthreads();
  const int64_t f = fb * kFmThreads + tid;
  if (f >= D) return;
  const uint32_t w0 = gen[2 * f];
  const float w = __uint_as_float(gen[2 * f + 1]);
  const float* const xl = xt + (int)((w0 & 0x3ffu) >> 2) * kXT;   // last index
  const float* const x0 = xt + (int)((w0 >> 10) & 0xffu) * kXT;   // first other index (or d)
  const float* const x1 = xt + (int)((w0 >> 18) & 0xffu) * kXT;   // second other index (or d)
  // degrees above 3: the further indices come from the packed entry
  uint64_t e = 0;
  int p = 0;
  if ((w0 >> 30) & 1u) {
    e = packed[f];
    p = (int)(e >> 56);
  }
  // all rows' reads first (rows past the end read zeros), then the further
  // factors of high degrees, then the stores
  float v[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) v[r] = w * x0[r] * x1[r] * xl[r];
  for (int j = 2; j < p - 1; ++j) {
    const float* const xj = xt + (int)((e >> (8 * j)) & 0xff) * kXT;
#pragma unroll
    for (int r = 0; r < kRows; ++r) v[r] *= xj[r];
  }
  float* const out = phi + r0 * D + f;
  if (nr == kRows) {
#pragma unroll
    for (int r = 0; r < kRows; ++r) out[(int64_t)r * D] = v[r];
  } else {
#pragma unroll
    for (int r = 0; r < kRows; ++r)
      if (r < nr) out[(int64_t)r * D] = v[r];
  }
}

}  // namespace

hipError_t launch_feature_map(const void* x, bool bf16, int64_t rows, const DevTable& t, float* phi,
                              hipStream_t s) {
  const size_t lds = sizeof(float) * (size_t)(t.d + 1) * kXT;
  const int64_t fblocks = (t.D + kFmThreads - 1) / kFmThreads;
  const int64_t total_rb = (rows + kRows - 1) / kRows;
  // at most 65535 row blocks per launch (the grid's y extent)
  for (int64_t rb = 0; rb < total_rb; rb += 65535) {
    const int64_t nrb = std::min<int64_t>(65535, total_rb - rb);
    const int64_t r0 = rb * kRows;
    const int64_t nrows = std::min<int64_t>(rows - r0, nrb * kRows);
    dim3 grid((unsigned)fblocks, (unsigned)nrb);
    if (bf16)
      hipLaunchKernelGGL(feature_map_kernel<bf16_t>, grid, dim3(kFmThreads), lds, s, (const bf16_t*)x + r0 * t.d,
                         nrows, t.d, t.gen, t.packed, t.D, phi + r0 * t.D);
    else
      hipLaunchKernelGGL(feature_map_kernel<float>, grid, dim3(kFmThreads), lds, s, (const float*)x + r0 * t.d,
                         nrows, t.d, t.gen, t.packed, t.D, phi + r0 * t.D);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sata
