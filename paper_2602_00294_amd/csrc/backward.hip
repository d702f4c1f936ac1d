// Backward pass of causal symmetry-aware Taylor attention: dL/dq, dL/dk and
// dL/dv for a given dL/dy, as chunked scans over the same constant-size states
// as the forward (App. A2), in float32 for both input dtypes.
//
// With o_T = phi(q_T)^T S_T = [N_T | Z_T] (S_T = sum_{t<=T} phi(k_t) (x) [v_t|1]),
// y_T = N_T / Z_T and g_T = dL/dy_T, the loss sees o_T through
//     h_T = dL/do_T = [g_T / Z_T | -(g_T . y_T) / Z_T]          (d_v + 1 values)
// and the chain rule through the linear-attention form gives
//     dL/dq_T = J_phi(q_T)^T (S_T h_T)                          (forward scan)
//     dL/dk_t = J_phi(k_t)^T (U_t [v_t|1]),  dL/dv_t = (U_t^T phi(k_t))[0:d_v]
//     with U_t = sum_{T>=t} phi(q_T) (x) h_T                     (reverse scan)
// where J_phi is the Jacobian of the feature map.  In chunks of C tokens the
// states before (S) or after (U) the chunk give the inter-chunk parts; inside
// a chunk phi(q).phi(k) = f_P(s) and its gradient f_P'(s) k / sqrt(d_k) =
// f_{P-1}(s) k / sqrt(d_k) give the intra-chunk parts directly.
//
// Passes, each over sequence segments whose partial sums fit the workspace:
//   1. the forward readout (the float32 prefill's main kernel) and
//      backward_h_finalize, which forms h_T;
//   2. backward_dq_main: each workgroup keeps one feature slice of S in LDS,
//      per chunk reads it out against h (u = S h) and applies the Jacobian of
//      its features at q, then adds the chunk's keys; backward_dq_finalize adds
//      the slices' partial gradients (in slice order) and the intra-chunk part;
//   3. backward_dkv_main: the reverse scan with U; backward_dkv_finalize.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "device_common.hpp"
#include "kernels.hpp"
#include "table.hpp"

namespace sata {

namespace {

constexpr int kBwThreads = 256;      // finalize kernels
constexpr int kBwScanThreads = 1024;  // scan kernels (four waves per SIMD)
constexpr int kBwPartThreads = 256;  // threads that take the Jacobian: kBwPartThreads / C feature ranges

// Rows of q, k, [v | 1] and h of one chunk into LDS (zero beyond the sequence).
// q and k rows are XS floats apart; with XS > dk, column dk holds 1 (the
// coordinate that degree-0 and lower-degree features read in the generation
// program).
template <typename T>
__device__ void bw_load_chunk(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                              const float* __restrict__ h, int64_t bh, int n, int t0, int cn, int C, int dk, int dv,
                              float* xq, float* xk, float* ve, float* hh, int XS) {
  const int E = dv + 1;
  const int64_t off = (bh * n + t0) * (int64_t)dk;
  for (int i = threadIdx.x; i < C * dk; i += blockDim.x) {
    const int t = i / dk;
    const int c = i - t * dk;
    xq[t * XS + c] = t < cn ? to_f32(q[off + i]) : 0.0f;
    xk[t * XS + c] = t < cn ? to_f32(k[off + i]) : 0.0f;
  }
  if (XS > dk)
    for (int t = threadIdx.x; t < C; t += blockDim.x) {
      xq[t * XS + dk] = 1.0f;
      xk[t * XS + dk] = 1.0f;
    }
  const int64_t voff = (bh * n + t0) * (int64_t)dv;
  const int64_t hoff = (bh * n + t0) * (int64_t)E;
  for (int i = threadIdx.x; i < C * E; i += blockDim.x) {
    const int t = i / E;
    const int j = i - t * E;
    float val = 0.0f, hv = 0.0f;
    if (t < cn) {
      val = (j < dv) ? to_f32(v[voff + (int64_t)t * dv + j]) : 1.0f;
      hv = h[hoff + i];
    }
    ve[i] = val;
    hh[i] = hv;
  }
}

// acc[a] += u * d phi_f(x) / d x[a] for one feature (packed multi-index pk,
// weight w): phi_f = w prod_j x[i_j], so the derivative along x[i_j] of each
// factor is w times the product of the other factors (prefix times suffix).
__device__ __forceinline__ void add_feature_gradient(uint64_t pk, float w, float u, const float* x, float* acc) {
  const int p = (int)(pk >> 56);
  if (p == 0) return;
  float xs[kMaxP];
  int ix[kMaxP];
#pragma unroll
  for (int j = 0; j < kMaxP - 1; ++j) {
    ix[j] = (int)((pk >> (8 * j)) & 0xff);
    xs[j] = (j < p) ? x[ix[j]] : 1.0f;
  }
  float suf[kMaxP];
  suf[kMaxP - 1] = 1.0f;
#pragma unroll
  for (int j = kMaxP - 2; j >= 0; --j) suf[j] = suf[j + 1] * xs[j];
  float pre = w * u;
#pragma unroll
  for (int j = 0; j < kMaxP - 1; ++j) {
    if (j < p) {
      acc[ix[j]] += pre * suf[j + 1];
      pre *= xs[j];
    }
  }
}

// out[t * FS + f] = sum_j A[f * E + j] * B[t * E + j] for t < cn, f < fs
// (A: a feature slice of a state, [fs][E]; B: [C][E] rows, zero past cn),
// each thread taking 4 tokens x 2 features so that a loaded value serves
// several products.
__device__ void bw_rows_dot(const float* A, const float* B, float* out, int fs, int cn, int E, int FS) {
  const int fp_n = (fs + 1) / 2, tq_n = (cn + 3) / 4;
  for (int i = threadIdx.x; i < fp_n * tq_n; i += blockDim.x) {
    const int fp = i % fp_n, tq = i / fp_n;
    const int f0 = 2 * fp, f1 = min(f0 + 1, fs - 1), t0 = 4 * tq;
    float acc[4][2] = {{0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}};
    for (int j = 0; j < E; ++j) {
      const float a0 = A[f0 * E + j], a1 = A[f1 * E + j];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float b = B[(t0 + r) * E + j];
        acc[r][0] += a0 * b;
        acc[r][1] += a1 * b;
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (t0 + r < cn) {
        out[(t0 + r) * FS + f0] = acc[r][0];
        if (f0 + 1 < fs) out[(t0 + r) * FS + f0 + 1] = acc[r][1];
      }
  }
}

// S[f * E + j] += sum_{t < cn} F[t * FS + f] * V[t * E + j] for f < fs, j < E,
// each thread taking 2 features x 4 columns.
__device__ void bw_accumulate_outer(float* S, const float* F, const float* V, int fs, int cn, int E, int FS) {
  const int fp_n = (fs + 1) / 2, jq_n = (E + 3) / 4;
  for (int i = threadIdx.x; i < fp_n * jq_n; i += blockDim.x) {
    const int fp = i % fp_n, jq = i / fp_n;
    const int f0 = 2 * fp, f1 = min(f0 + 1, fs - 1), j0 = 4 * jq;
    float acc[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    for (int t = 0; t < cn; ++t) {
      const float a0 = F[t * FS + f0], a1 = F[t * FS + f1];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float b = V[t * E + min(j0 + c, E - 1)];
        acc[0][c] += a0 * b;
        acc[1][c] += a1 * b;
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (j0 + c < E) {
        S[f0 * E + j0 + c] += acc[0][c];
        if (f0 + 1 < fs) S[f1 * E + j0 + c] += acc[1][c];
      }
  }
}

// out[t * W + j] = sum_{f < fs} U[f * E + j] * F[t * FS + f] for t < cn, j < dv
// (4 tokens x 2 columns per thread).
__device__ void bw_cols_dot(const float* U, const float* F, float* out, int fs, int cn, int E, int dv, int FS, int W) {
  const int jp_n = (dv + 1) / 2, tq_n = (cn + 3) / 4;
  for (int i = threadIdx.x; i < jp_n * tq_n; i += blockDim.x) {
    const int jp = i % jp_n, tq = i / jp_n;
    const int j0 = 2 * jp, j1 = min(j0 + 1, dv - 1), t0 = 4 * tq;
    float acc[4][2] = {{0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}, {0.f, 0.f}};
    for (int f = 0; f < fs; ++f) {
      const float a0 = U[f * E + j0], a1 = U[f * E + j1];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float b = F[(t0 + r) * FS + f];
        acc[r][0] += a0 * b;
        acc[r][1] += a1 * b;
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (t0 + r < cn) {
        out[(t0 + r) * W + j0] = acc[r][0];
        if (j0 + 1 < dv) out[(t0 + r) * W + j0 + 1] = acc[r][1];
      }
  }
}

// Value of one feature from its generation-program words g (table.hpp
// build_gen_program) at the row x (stride with the column d held at 1), the
// packed entry pk supplying any indices past the first two and the last.
__device__ __forceinline__ float gen_feature_value(uint2 g, uint64_t pk, const float* x) {
  float v = __uint_as_float(g.y) * x[(g.x >> 10) & 0xffu] * x[(g.x >> 18) & 0xffu] * x[(g.x & 0x3ffu) >> 2];
  if ((g.x >> 30) & 1u) {
    const int p = (int)(pk >> 56);
    for (int j = 2; j < p - 1; ++j) v *= x[(pk >> (8 * j)) & 0xff];
  }
  return v;
}

// acc[a] += sum over the features f in [lo, hi) of u[f] d phi_f(x) / d x[a],
// in feature order.  For degree <= 3 (indices a0 <= a1 <= c, the missing ones
// being the column d, which acc has room for and nobody reads) the last
// index takes u w x[a0] x[a1] per feature, and the two others take x[a1] and
// x[a0] times the run sum of u w x[c] over consecutive features that share
// (a0, a1), added when the run ends; higher degrees take the full product rule.
__device__ void add_gradient_range(const uint2* gen, const uint64_t* tpk, const float* u, int lo, int hi,
                                   const float* x, float* acc, int d) {
  int ca = d, cb = d;
  float xa = 1.0f, xb = 1.0f, sum = 0.0f;
  for (int f = lo; f < hi; ++f) {
    const uint2 g = gen[f];
    const float uw = u[f] * __uint_as_float(g.y);
    const int a0 = (int)((g.x >> 10) & 0xffu), a1 = (int)((g.x >> 18) & 0xffu);
    if ((g.x >> 30) & 1u) {
      add_feature_gradient(tpk[f], __uint_as_float(g.y), u[f], x, acc);
      continue;
    }
    if (a0 != ca || a1 != cb) {
      acc[ca] += xb * sum;
      acc[cb] += xa * sum;
      sum = 0.0f;
      ca = a0;
      cb = a1;
      xa = x[a0];
      xb = x[a1];
    }
    const int c = (int)((g.x & 0x3ffu) >> 2);
    acc[c] += uw * xa * xb;
    sum += uw * x[c];
  }
  acc[ca] += xb * sum;
  acc[cb] += xa * sum;
}

// Shared LDS layout of the two scan kernels (in floats; the 8-byte table
// entries first, so they stay aligned):
//   tpk [FS] (u64) | tgen [FS] (program words, 2 x u32) | Sl [FS][E] state
//   slice | fb [C][FS] feature values | uu [C][FS] readouts | xq, xk
//   [C][dk+1] | ve, hh [C][E] | jq [parts][C][dk+1] gradient rows
struct BwLds {
  int FS, C, dk, E, parts;
  __host__ __device__ size_t floats() const {
    return (size_t)FS * E + 2 * (size_t)C * FS + 2 * (size_t)C * (dk + 1) + 2 * (size_t)C * E +
           (size_t)parts * C * (dk + 1) + 4 * (size_t)FS;
  }
};

// Pass 2: dL/dq (inter-chunk part), one feature slice of S per workgroup.
template <typename T>
__global__ void __launch_bounds__(kBwScanThreads)
backward_dq_main(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                 const float* __restrict__ h, const uint64_t* __restrict__ packed, const uint32_t* __restrict__ gen,
                 int64_t D, float* __restrict__ S_state, float* __restrict__ part, int BH, int n, int dk, int dv,
                 int C, int FS, int seg0, int seg_len, int first_seg) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  const int parts = kBwPartThreads / C;
  const int XS = dk + 1;
  uint64_t* tpk = (uint64_t*)lds;
  uint2* tgen = (uint2*)(tpk + FS);
  float* Sl = (float*)(tgen + FS);
  float* fb = Sl + FS * E;
  float* uu = fb + C * FS;
  float* xq = uu + C * FS;
  float* xk = xq + C * XS;
  float* ve = xk + C * XS;
  float* hh = ve + C * E;
  float* jq = hh + C * E;
  const int s = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int64_t f0 = (int64_t)s * FS;
  const int fs = (int)min<int64_t>(FS, D - f0);
  float* Sg = S_state + (bh * D + f0) * E;
  for (int i = tid; i < fs * E; i += blockDim.x) Sl[i] = first_seg ? 0.0f : Sg[i];
  for (int f = tid; f < fs; f += blockDim.x) {
    tpk[f] = packed[f0 + f];
    tgen[f] = ((const uint2*)gen)[f0 + f];
  }
  const int seg_end = min(n, seg0 + seg_len);
  for (int t0 = seg0; t0 < seg_end; t0 += C) {
    const int cn = min(C, n - t0);
    __syncthreads();
    bw_load_chunk(q, k, v, h, bh, n, t0, cn, C, dk, dv, xq, xk, ve, hh, XS);
    for (int i = tid; i < parts * C * XS; i += blockDim.x) jq[i] = 0.0f;
    __syncthreads();
    // u_T[f] = S_{c-1}[f, :] . h_T
    bw_rows_dot(Sl, hh, uu, fs, cn, E, FS);
    __syncthreads();
    // dq_T += sum_f u_T[f] d phi_f(q_T) / d q: thread (part, token) takes a
    // contiguous range of the features into its own gradient row
    {
      const int t = tid % C;
      const int pt = tid / C;
      const int per = (fs + parts - 1) / parts;
      if (t < cn && pt < parts)
        add_gradient_range(tgen, tpk, uu + t * FS, pt * per, min(fs, (pt + 1) * per), xq + t * XS,
                           jq + (pt * C + t) * XS, dk);
    }
    __syncthreads();
    float* pout = part + (((int64_t)s * BH + bh) * seg_len + (t0 - seg0)) * dk;
    for (int i = tid; i < cn * dk; i += blockDim.x) {
      const int t = i / dk;
      const int a = i - t * dk;
      float sum = 0.0f;
      for (int pt = 0; pt < parts; ++pt) sum += jq[(pt * C + t) * XS + a];
      pout[i] = sum;
    }
    // S_c = S_{c-1} + phi(K_c)^T [V_c | 1]
    for (int i = tid; i < cn * fs; i += blockDim.x) {
      const int t = i / fs;
      const int f = i - t * fs;
      fb[t * FS + f] = gen_feature_value(tgen[f], tpk[f], xk + t * XS);
    }
    __syncthreads();
    bw_accumulate_outer(Sl, fb, ve, fs, cn, E, FS);
  }
  __syncthreads();
  for (int i = tid; i < fs * E; i += blockDim.x) Sg[i] = Sl[i];
}

// Pass 3: dL/dk and dL/dv (inter-chunk parts), chunks in reverse order, one
// feature slice of U = sum over later tokens of phi(q_T) (x) h_T per workgroup.
template <typename T>
__global__ void __launch_bounds__(kBwScanThreads)
backward_dkv_main(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                  const float* __restrict__ h, const uint64_t* __restrict__ packed, const uint32_t* __restrict__ gen,
                  int64_t D, float* __restrict__ U_state, float* __restrict__ part, int BH, int n, int dk, int dv,
                  int C, int FS, int seg0, int seg_len, int first_seg) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  const int parts = kBwPartThreads / C;
  const int XS = dk + 1;
  uint64_t* tpk = (uint64_t*)lds;
  uint2* tgen = (uint2*)(tpk + FS);
  float* Ul = (float*)(tgen + FS);
  float* fb = Ul + FS * E;
  float* uu = fb + C * FS;
  float* xq = uu + C * FS;
  float* xk = xq + C * XS;
  float* ve = xk + C * XS;
  float* hh = ve + C * E;
  float* jq = hh + C * E;
  const int s = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int64_t f0 = (int64_t)s * FS;
  const int fs = (int)min<int64_t>(FS, D - f0);
  float* Ug = U_state + (bh * D + f0) * E;
  for (int i = tid; i < fs * E; i += blockDim.x) Ul[i] = first_seg ? 0.0f : Ug[i];
  for (int f = tid; f < fs; f += blockDim.x) {
    tpk[f] = packed[f0 + f];
    tgen[f] = ((const uint2*)gen)[f0 + f];
  }
  const int seg_end = min(n, seg0 + seg_len);
  const int PW = dk + dv;  // partial row: dk, then dv
  for (int t0 = seg0 + (seg_end - 1 - seg0) / C * C; t0 >= seg0; t0 -= C) {
    const int cn = min(C, n - t0);
    __syncthreads();
    bw_load_chunk(q, k, v, h, bh, n, t0, cn, C, dk, dv, xq, xk, ve, hh, XS);
    for (int i = tid; i < parts * C * XS; i += blockDim.x) jq[i] = 0.0f;
    __syncthreads();
    // phi(k_t) and r_t[f] = U[f, :] . [v_t | 1]
    for (int i = tid; i < cn * fs; i += blockDim.x) {
      const int t = i / fs;
      const int f = i - t * fs;
      fb[t * FS + f] = gen_feature_value(tgen[f], tpk[f], xk + t * XS);
    }
    bw_rows_dot(Ul, ve, uu, fs, cn, E, FS);
    __syncthreads();
    {
      const int t = tid % C;
      const int pt = tid / C;
      const int per = (fs + parts - 1) / parts;
      if (t < cn && pt < parts)
        add_gradient_range(tgen, tpk, uu + t * FS, pt * per, min(fs, (pt + 1) * per), xk + t * XS,
                           jq + (pt * C + t) * XS, dk);
    }
    __syncthreads();
    float* pout = part + (((int64_t)s * BH + bh) * seg_len + (t0 - seg0)) * PW;
    for (int i = tid; i < cn * dk; i += blockDim.x) {
      const int t = i / dk;
      const int a = i - t * dk;
      float sum = 0.0f;
      for (int pt = 0; pt < parts; ++pt) sum += jq[(pt * C + t) * XS + a];
      pout[t * PW + a] = sum;
    }
    // dv_t[j] = sum_f U[f, j] phi_f(k_t)
    bw_cols_dot(Ul, fb, pout + dk, fs, cn, E, dv, FS, PW);
    __syncthreads();
    // U += phi(Q_c)^T H_c
    for (int i = tid; i < cn * fs; i += blockDim.x) {
      const int t = i / fs;
      const int f = i - t * fs;
      fb[t * FS + f] = gen_feature_value(tgen[f], tpk[f], xq + t * XS);
    }
    __syncthreads();
    bw_accumulate_outer(Ul, fb, hh, fs, cn, E, FS);
  }
  __syncthreads();
  for (int i = tid; i < fs * E; i += blockDim.x) Ug[i] = Ul[i];
}

// Intra-chunk weights of one chunk into LDS: for query row r and key column c
// (c <= r), W[r][c] = f_P(s_rc) and G[r][c] = (h_r . [v_c|1]) f_{P-1}(s_rc) / sqrt(d_k).
// a + p[0] + p[stride] + ... + p[(ns - 1) stride], added in that order, with
// eight of the loads in flight at a time.
__device__ __forceinline__ float add_slices(float a, const float* __restrict__ p, int64_t stride, int ns) {
  int s = 0;
  for (; s + 8 <= ns; s += 8) {
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = p[(s + u) * stride];
#pragma unroll
    for (int u = 0; u < 8; ++u) a += x[u];
  }
  for (; s < ns; ++s) a += p[s * stride];
  return a;
}

// Row stride of the coordinates in the intra-chunk kernels: odd, so that lanes
// that read different key rows at one coordinate hit different LDS banks.
__host__ __device__ constexpr int bw_fin_stride(int dk) { return dk | 1; }

__device__ void bw_intra_weights(const float* xq, const float* xk, const float* ve, const float* hh, int cn, int C,
                                 int dk, int XS, int E, int P, float* W, float* Gm) {
  const float scale = 1.0f / sqrtf((float)dk);
  for (int i = threadIdx.x; i < C * C; i += blockDim.x) {
    const int r = i / C;
    const int c = i - r * C;
    float w = 0.0f, g = 0.0f;
    if (r < cn && c <= r) {
      float dot = 0.0f;
      for (int a = 0; a < dk; ++a) dot += xq[r * XS + a] * xk[c * XS + a];
      const float sc = dot * scale;
      float hv = 0.0f;
      for (int j = 0; j < E; ++j) hv += hh[r * E + j] * ve[c * E + j];
      w = taylor_horner(sc, P);
      g = P > 1 ? hv * taylor_horner(sc, P - 1) * scale : 0.0f;
    }
    W[i] = w;
    Gm[i] = g;
  }
}

// Pass 1 end: h_T from the forward readout partials plus the intra-chunk term.
template <typename T>
__global__ void __launch_bounds__(kBwThreads)
backward_h_finalize(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                    const T* __restrict__ dy, const float* __restrict__ part, float* __restrict__ h, int BH, int n,
                    int dk, int dv, int P, int C, int nslices, int seg0, int seg_len) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  float* xq = lds;
  // odd row stride: the lanes of the Q K^T loop read different key rows
  const int XS = bw_fin_stride(dk);
  float* xk = xq + C * XS;
  float* ve = xk + C * XS;
  float* O = ve + C * E;   // [C][E]
  float* W = O + C * E;    // [C][C]
  const int64_t bh = blockIdx.y;
  const int t0 = seg0 + blockIdx.x * C;
  if (t0 >= n) return;
  const int cn = min(C, n - t0);
  const int tid = threadIdx.x;
  const float scale = 1.0f / sqrtf((float)dk);
  const int64_t off = (bh * n + t0) * (int64_t)dk;
  for (int i = tid; i < C * dk; i += blockDim.x) {
    const int t = i / dk;
    const int a = i - t * dk;
    xq[t * XS + a] = t < cn ? to_f32(q[off + i]) : 0.0f;
    xk[t * XS + a] = t < cn ? to_f32(k[off + i]) : 0.0f;
  }
  for (int i = tid; i < C * E; i += blockDim.x) {
    const int t = i / E;
    const int j = i - t * E;
    ve[i] = t < cn ? ((j < dv) ? to_f32(v[(bh * n + t0 + t) * (int64_t)dv + j]) : 1.0f) : 0.0f;
  }
  __syncthreads();
  for (int i = tid; i < C * C; i += blockDim.x) {
    const int r = i / C;
    const int c = i - r * C;
    float w = 0.0f;
    if (r < cn && c <= r) {
      float dot = 0.0f;
      for (int a = 0; a < dk; ++a) dot += xq[r * XS + a] * xk[c * XS + a];
      w = taylor_horner(dot * scale, P);
    }
    W[i] = w;
  }
  __syncthreads();
  for (int o = tid; o < cn * E; o += blockDim.x) {
    const int r = o / E;
    const int j = o - r * E;
    float acc = 0.0f;
    for (int c = 0; c <= r; ++c) acc += W[r * C + c] * ve[c * E + j];
    acc = add_slices(acc, part + ((int64_t)bh * seg_len + (t0 - seg0) + r) * E + j, (int64_t)BH * seg_len * E, nslices);
    O[o] = acc;
  }
  __syncthreads();
  for (int r = tid; r < cn; r += blockDim.x) {
    const float Z = O[r * E + dv];
    const T* g = dy + (bh * n + t0 + r) * (int64_t)dv;
    float gy = 0.0f;
    for (int j = 0; j < dv; ++j) gy += to_f32(g[j]) * (O[r * E + j] / Z);
    float* hr = h + (bh * n + t0 + r) * (int64_t)E;
    for (int j = 0; j < dv; ++j) hr[j] = to_f32(g[j]) / Z;
    hr[dv] = -gy / Z;
  }
}

// Pass 2 end: dq = sum of the slices' partials + intra-chunk part.
template <typename T>
__global__ void __launch_bounds__(kBwThreads)
backward_dq_finalize(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                     const float* __restrict__ h, const float* __restrict__ part, T* __restrict__ dq, int BH, int n,
                     int dk, int dv, int P, int C, int nslices, int seg0, int seg_len) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  float* xq = lds;
  const int XS = bw_fin_stride(dk);
  float* xk = xq + C * XS;
  float* ve = xk + C * XS;
  float* hh = ve + C * E;
  float* W = hh + C * E;
  float* Gm = W + C * C;
  const int64_t bh = blockIdx.y;
  const int t0 = seg0 + blockIdx.x * C;
  if (t0 >= n) return;
  const int cn = min(C, n - t0);
  bw_load_chunk(q, k, v, h, bh, n, t0, cn, C, dk, dv, xq, xk, ve, hh, XS);
  __syncthreads();
  bw_intra_weights(xq, xk, ve, hh, cn, C, dk, XS, E, P, W, Gm);
  __syncthreads();
  for (int i = threadIdx.x; i < cn * dk; i += blockDim.x) {
    const int r = i / dk;
    const int a = i - r * dk;
    float acc = 0.0f;
    for (int c = 0; c <= r; ++c) acc += Gm[r * C + c] * xk[c * XS + a];
    acc = add_slices(acc, part + ((int64_t)bh * seg_len + (t0 - seg0) + r) * dk + a, (int64_t)BH * seg_len * dk, nslices);
    dq[(bh * n + t0 + r) * (int64_t)dk + a] = from_f32<T>(acc);
  }
}

// Pass 3 end: dk, dv = sum of the slices' partials + intra-chunk parts.
template <typename T>
__global__ void __launch_bounds__(kBwThreads)
backward_dkv_finalize(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                      const float* __restrict__ h, const float* __restrict__ part, T* __restrict__ dk_out,
                      T* __restrict__ dv_out, int BH, int n, int dk, int dv, int P, int C, int nslices, int seg0,
                      int seg_len) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  const int PW = dk + dv;
  float* xq = lds;
  const int XS = bw_fin_stride(dk);
  float* xk = xq + C * XS;
  float* ve = xk + C * XS;
  float* hh = ve + C * E;
  float* W = hh + C * E;
  float* Gm = W + C * C;
  const int64_t bh = blockIdx.y;
  const int t0 = seg0 + blockIdx.x * C;
  if (t0 >= n) return;
  const int cn = min(C, n - t0);
  bw_load_chunk(q, k, v, h, bh, n, t0, cn, C, dk, dv, xq, xk, ve, hh, XS);
  __syncthreads();
  bw_intra_weights(xq, xk, ve, hh, cn, C, dk, XS, E, P, W, Gm);
  __syncthreads();
  for (int i = threadIdx.x; i < cn * PW; i += blockDim.x) {
    const int c = i / PW;
    const int a = i - c * PW;
    float acc = 0.0f;
    if (a < dk) {
      for (int r = c; r < cn; ++r) acc += Gm[r * C + c] * xq[r * XS + a];
    } else {
      for (int r = c; r < cn; ++r) acc += W[r * C + c] * hh[r * E + (a - dk)];
    }
    acc = add_slices(acc, part + ((int64_t)bh * seg_len + (t0 - seg0) + c) * PW + a, (int64_t)BH * seg_len * PW, nslices);
    if (a < dk)
      dk_out[(bh * n + t0 + c) * (int64_t)dk + a] = from_f32<T>(acc);
    else
      dv_out[(bh * n + t0 + c) * (int64_t)dv + (a - dk)] = from_f32<T>(acc);
  }
}

}  // namespace

bool plan_backward(int64_t D, int BH, int n, int dk, int dv, int P, int chunk, size_t max_ws_bytes, BackwardPlan* plan,
                   PrefillGenericPlan* fwd) {
  if (dk > kMaxBackwardDim || dv > kMaxBackwardDim) return false;
  if (chunk != 16 && chunk != 32 && chunk != 64) return false;
  if (!plan_prefill_generic(D, BH, n, dk, dv, chunk, max_ws_bytes, fwd)) return false;
  // the forward readout of pass 1 on the matrix cores (split operands, so
  // float32-accurate for both input types) where its kernel covers the shape
  plan->feat_fwd = plan_prefill_feat(D, BH, std::max(n, 1), dk, dv, P, chunk, true, max_ws_bytes, &plan->feat);
  const int E = dv + 1;
  const int C = chunk;
  BwLds L{0, C, dk, E, kBwPartThreads / C};
  const size_t budget = 150 * 1024;
  const size_t fixed = sizeof(float) * L.floats();
  const size_t per_feature = sizeof(float) * ((size_t)E + 2 * (size_t)C + 4);
  if (fixed + 8 * per_feature > budget) return false;
  int64_t fs = (int64_t)((budget - fixed) / per_feature);
  fs = std::min<int64_t>(fs, 512);
  const int64_t want = (512 + BH - 1) / BH;  // about two workgroups per CU
  fs = std::min<int64_t>(fs, std::max<int64_t>(16, (D + want - 1) / want));
  fs = std::max<int64_t>(1, std::min<int64_t>(fs, D));
  L.FS = (int)fs;
  plan->fs = (int)fs;
  plan->nslices = (int)((D + fs - 1) / fs);
  plan->lds_main = sizeof(float) * L.floats();
  plan->lds_h = sizeof(float) * (2 * (size_t)C * bw_fin_stride(dk) + 2 * (size_t)C * E + (size_t)C * C);
  plan->lds_fin = sizeof(float) * (2 * (size_t)C * bw_fin_stride(dk) + 2 * (size_t)C * E + 2 * (size_t)C * C);
  // partial rows per token: the forward readout (E per forward slice), dq (dk),
  // dk and dv (dk + dv) per backward slice
  const size_t fwd_slices = plan->feat_fwd ? (size_t)plan->feat.nslices : (size_t)fwd->nslices;
  const size_t per_token = sizeof(float) * (size_t)BH *
                           std::max<size_t>(fwd_slices * E, (size_t)plan->nslices * (dk + dv));
  int64_t seg = (int64_t)(max_ws_bytes / per_token) / C * C;
  if (seg < C) seg = C;
  const int64_t n_round = ((int64_t)std::max(n, 1) + C - 1) / C * C;
  plan->seg_len = (int)std::min<int64_t>(seg, n_round);
  plan->partial_bytes = per_token * (size_t)plan->seg_len;
  fwd->seg_len = plan->seg_len;
  plan->feat.seg_len = plan->seg_len;
  plan->feat.parts = 1;  // (the backward's forward readout runs its segments in order)
  plan->feat.part_len = plan->seg_len;
  plan->h_bytes = sizeof(float) * (size_t)BH * n * E;
  plan->state_bytes = sizeof(float) * (size_t)BH * D * E;
  return true;
}

template <typename T>
static hipError_t launch_backward_typed(const T* q, const T* k, const T* v, const T* dy, T* dq, T* dk, T* dv_out,
                                        int BH, int n, int dk_, int dv, int P, int chunk, const DevTable& t,
                                        const BackwardPlan& plan, const PrefillGenericPlan& fwd, float* h,
                                        float* state, float* partial, hipStream_t s) {
  const int C = chunk;
  hipError_t e;
  if ((e = hipFuncSetAttribute((const void*)backward_dq_main<T>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)plan.lds_main)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void*)backward_dkv_main<T>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)plan.lds_main)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void*)backward_h_finalize<T>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)plan.lds_h)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void*)backward_dq_finalize<T>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)plan.lds_fin)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void*)backward_dkv_finalize<T>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)plan.lds_fin)) != hipSuccess)
    return e;
  const int nseg = (n + plan.seg_len - 1) / plan.seg_len;
  // pass 1: the forward readout of each segment, then h
  for (int sg = 0; sg < nseg; ++sg) {
    const int seg0 = sg * plan.seg_len;
    if (plan.feat_fwd)
      e = launch_prefill_feat_readout(q, k, v, std::is_same<T, bf16_t>::value, BH, n, dk_, dv, t, plan.feat, state,
                                      partial, seg0, sg == 0, s);
    else
      e = launch_prefill_generic_readout(q, k, v, std::is_same<T, bf16_t>::value, BH, n, dk_, dv, C, t, fwd, state,
                                         partial, seg0, plan.seg_len, sg == 0, s);
    if (e != hipSuccess) return e;
    const int nchunks = (std::min(plan.seg_len, n - seg0) + C - 1) / C;
    // (the matrix-core readout leaves its slices' sum in slice 0)
    hipLaunchKernelGGL(backward_h_finalize<T>, dim3((unsigned)nchunks, (unsigned)BH), dim3(kBwThreads),
                       plan.lds_h, s, q, k, v, dy, partial, h, BH, n, dk_, dv, P, C,
                       plan.feat_fwd ? 1 : fwd.nslices, seg0, plan.seg_len);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // pass 2: dq
  for (int sg = 0; sg < nseg; ++sg) {
    const int seg0 = sg * plan.seg_len;
    hipLaunchKernelGGL(backward_dq_main<T>, dim3((unsigned)plan.nslices, (unsigned)BH), dim3(kBwScanThreads),
                       plan.lds_main, s, q, k, v, h, t.packed, t.gen, t.D, state, partial, BH, n, dk_, dv, C,
                       plan.fs, seg0, plan.seg_len, sg == 0 ? 1 : 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int nchunks = (std::min(plan.seg_len, n - seg0) + C - 1) / C;
    hipLaunchKernelGGL(backward_dq_finalize<T>, dim3((unsigned)nchunks, (unsigned)BH), dim3(kBwThreads),
                       plan.lds_fin, s, q, k, v, h, partial, dq, BH, n, dk_, dv, P, C, plan.nslices, seg0,
                       plan.seg_len);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // pass 3: dk, dv, segments from the last
  for (int sg = nseg - 1; sg >= 0; --sg) {
    const int seg0 = sg * plan.seg_len;
    hipLaunchKernelGGL(backward_dkv_main<T>, dim3((unsigned)plan.nslices, (unsigned)BH), dim3(kBwScanThreads),
                       plan.lds_main, s, q, k, v, h, t.packed, t.gen, t.D, state, partial, BH, n, dk_, dv, C,
                       plan.fs, seg0, plan.seg_len, sg == nseg - 1 ? 1 : 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int nchunks = (std::min(plan.seg_len, n - seg0) + C - 1) / C;
    hipLaunchKernelGGL(backward_dkv_finalize<T>, dim3((unsigned)nchunks, (unsigned)BH), dim3(kBwThreads),
                       plan.lds_fin, s, q, k, v, h, partial, dk, dv_out, BH, n, dk_, dv, P, C, plan.nslices, seg0,
                       plan.seg_len);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_backward(const void* q, const void* k, const void* v, const void* dy, void* dq, void* dk,
                           void* dv, bool bf16, int BH, int n, int dk_, int dv_, int P, int chunk, const DevTable& t,
                           const BackwardPlan& plan, const PrefillGenericPlan& fwd, float* h, float* state,
                           float* partial, hipStream_t s) {
  if (bf16)
    return launch_backward_typed<bf16_t>((const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, (const bf16_t*)dy,
                                         (bf16_t*)dq, (bf16_t*)dk, (bf16_t*)dv, BH, n, dk_, dv_, P, chunk, t, plan,
                                         fwd, h, state, partial, s);
  return launch_backward_typed<float>((const float*)q, (const float*)k, (const float*)v, (const float*)dy,
                                      (float*)dq, (float*)dk, (float*)dv, BH, n, dk_, dv_, P, chunk, t, plan, fwd, h,
                                      state, partial, s);
}

}  // namespace sata
