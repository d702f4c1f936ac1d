// Generic float32 kernels: feature map, decode step and a chunked prefill that
// works for every supported (d_k, d_v, P, chunk) and both input dtypes.
//
// Prefill follows the linear-attention form of App. A2 in chunks of C tokens:
// for chunk c with query rows Q_c, keys K_c and extended values [V_c | 1],
//     O      = phi(Q_c) S_{c-1}                              (inter-chunk readout)
//            + mask_{t'<=t}(f_P(Q_c K_c^T / sqrt(d_k))) [V_c | 1]   (intra-chunk)
//     S_c    = S_{c-1} + phi(K_c)^T [V_c | 1]                (state update)
//     y      = O[:, :d_v] / O[:, d_v]
// The state is split over workgroups by feature ranges ("slices"); each slice
// keeps its part of S in LDS for the whole sequence and writes its partial
// readout per token; a second kernel adds the slices' partials (in slice
// order, so the result is deterministic), the intra-chunk term, and divides.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <numeric>

#include "device_common.hpp"
#include "kernels.hpp"

namespace sata {

namespace {

constexpr int kThreads = 256;

// ---------------------------------------------------------------- decode step

// Whole-head decode: one workgroup streams all rows of one head's state, so
// the readout needs no cross-workgroup reduction.  Thread t < R*E (R = rows
// per pass) owns column j = t % E of rows t / E + k*R: consecutive threads
// touch consecutive addresses, each element is updated (S += phi_k[f] * [v|1][j])
// and immediately read out (o_j += phi_q[f] * S).  Large heads are split over
// several workgroups instead (decode_slice_kernel + decode_finalize_kernel).
// These row-wise kernels serve states that are not 16-byte aligned; aligned
// ones take the flat float4 stream (decode_flat_kernel).
template <typename T, int NTH>
__device__ __forceinline__ void decode_rows(float* __restrict__ S, const T* __restrict__ q,
                                            const T* __restrict__ k, const T* __restrict__ v,
                                            const uint64_t* __restrict__ packed, const float* __restrict__ weight,
                                            int64_t D, int dk, int dv, int64_t bh, int64_t f0, int nf, float* lds) {
  const int E = dv + 1;
  float* xq = lds;               // [dk]
  float* xk = xq + dk;           // [dk]
  float* ve = xk + dk;           // [E]
  float* fq = ve + E;            // [nf]
  float* fk = fq + nf;           // [nf]
  float* red = fk + nf;          // [NTH]
  const int tid = threadIdx.x;
  for (int i = tid; i < dk; i += NTH) {
    xq[i] = to_f32(q[bh * dk + i]);
    xk[i] = to_f32(k[bh * dk + i]);
  }
  for (int i = tid; i < E; i += NTH) ve[i] = (i < dv) ? to_f32(v[bh * dv + i]) : 1.0f;
  __syncthreads();
  for (int f = tid; f < nf; f += NTH) {
    const uint64_t pk = packed[f0 + f];
    const float w = weight[f0 + f];
    fq[f] = feature_value(pk, w, xq);
    fk[f] = feature_value(pk, w, xk);
  }
  __syncthreads();
  const int R = NTH / E;  // rows per pass
  float acc = 0.0f;
  if (tid < R * E) {
    const int r = tid / E;
    const int j = tid - r * E;
    const float vj = ve[j];
    float* base = S + (bh * D + f0) * E + j;
    int f = r;
    // eight rows in flight per thread
    for (; f + 7 * R < nf; f += 8 * R) {
      float x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = base[(int64_t)(f + u * R) * E];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        x[u] += fk[f + u * R] * vj;
        base[(int64_t)(f + u * R) * E] = x[u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += fq[f + u * R] * x[u];
    }
    for (; f < nf; f += R) {
      const float s0 = base[(int64_t)f * E] + fk[f] * vj;
      base[(int64_t)f * E] = s0;
      acc += fq[f] * s0;
    }
  }
  red[tid] = acc;
  __syncthreads();
  if (tid < E) {
    float o = 0.0f;
    for (int r = 0; r < R; ++r) o += red[r * E + tid];
    red[tid] = o;  // only this thread reads red[r*E + tid] for its own column
  }
  __syncthreads();
}

template <typename T, int NTH>
__global__ void __launch_bounds__(NTH)
decode_head_kernel(float* __restrict__ S, const T* __restrict__ q, const T* __restrict__ k,
                   const T* __restrict__ v, T* __restrict__ y, const uint64_t* __restrict__ packed,
                   const float* __restrict__ weight, int64_t D, int dk, int dv) {
  extern __shared__ float lds[];
  const int64_t bh = blockIdx.x;
  decode_rows<T, NTH>(S, q, k, v, packed, weight, D, dk, dv, bh, 0, (int)D, lds);
  const float* red = lds + 2 * dk + (dv + 1) + 2 * D;
  for (int j = threadIdx.x; j < dv; j += NTH) y[bh * dv + j] = from_f32<T>(red[j] / red[dv]);
}

// Workgroup barrier over LDS data only.  __syncthreads also waits for the
// thread's outstanding global loads; this one lets them stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Whole-head decode as one flat float4 stream.  A head's state is D*E
// contiguous floats (E = d_v + 1).  Of the workgroup's threads, tu (a multiple
// of E / gcd(E, 4)) take part: thread t owns the float4s g = t + tu*m of the
// head's 16-byte aligned part, whose first element is a0 < 4.  A step of tu
// float4s is a whole number of rows, so each of a thread's four lanes keeps
// one value column j for the whole sweep while its row advances by 4 tu / E.
// Each element is updated (S += phi_k[f] [v|1][j]) and read out at once
// (o_j += phi_q[f] S); the per-thread column sums are reduced in a fixed
// order.  The a0 leading and (at most 3) trailing elements are loaded at the
// start by threads of their own and their readout terms added in element
// order at the end, so the result is deterministic.  Loads run two groups of
// kFlatUnroll float4s ahead of the arithmetic.
//
// With npieces > 1 (an even number), each head is streamed by that many
// workgroups (blockIdx = npieces head + piece), piece p taking a thread's
// steps [m(p), m(p+1)).  On MI355X the hardware deals workgroups to the 8 XCDs
// in turn, so even pieces run on even-numbered XCDs and odd pieces on odd
// ones, which stream this pattern about a quarter more slowly: of each (even,
// odd) pair the even piece takes the share `even_share` of the steps (0.557
// there; 0.5 on any other device, where that dispatch pattern is not
// assumed).  Any share gives the same result; it only balances time.  Each piece
// needs the features of its own rows only, kept in LDS from its first row on.
// Each piece stores its E column sums at xpart[npieces head + piece] with
// device-coherent stores and bumps cnt[head]; the last to arrive adds them in
// piece order (so the result does not depend on the order of arrival), writes
// y and sets the counter back to 0.  No device-scope fence is used: one would
// write back the XCD's whole L2, full of freshly written state.
//
// Compensated variant (COMP): R holds, per head, the float32 rounding
// residuals of the entries whose per-token increments are the first to fall
// below half an ulp of a long sum (the normaliser column of every row, and
// the value columns of the degree-0 and degree-1 rows; see comp_index).
// Those entries are updated as an unevaluated float pair (S, R) by exact
// two-sums, and S is renormalised to the rounded pair sum, so S alone keeps
// float32 accuracy however many tokens have been added.  Their residuals are
// loaded with the state, kFlatUnroll steps ahead.
constexpr int kFlatUnroll = 2;
// Share of a head's stream given to the piece on an even-numbered XCD of
// MI355X: their measured streaming times for this pattern are 47 and 59 us
// per head.
constexpr float kMi355EvenShare = 0.557f;

// Residual slot of state entry (row f, column j) of a head, or -1 when the
// entry is not compensated: the normaliser column j = dv of every row at
// [f], the value columns of rows f <= dk (degrees 0 and 1) at [D + f dv + j].
// (Rows and slots fit in 32 bits: D <= 2^26 and dk, dv <= 255.)
__device__ __forceinline__ int comp_index(int f, int j, int D, int dk, int dv) {
  return (j == dv) ? f : ((f <= dk) ? D + f * dv + j : -1);
}

// (s, r) += a for an unevaluated pair s + r: two exact two-sums (Knuth), the
// second folding the residual back so that s is the pair's rounded value.
__device__ __forceinline__ void comp_add(float& s, float& r, float a) {
  const float t = s + a;
  const float tp = t - s;
  const float e = (s - (t - tp)) + (a - tp);  // s + a = t + e exactly
  const float r1 = r + e;
  const float u = t + r1;
  const float up = u - t;
  r = (t - (u - up)) + (r1 - up);  // t + r1 = u + r exactly
  s = u;
}

template <typename T, int NTH, bool COMP>
__global__ void __launch_bounds__(NTH, COMP ? 4 : 8)
decode_flat_kernel(float* __restrict__ S, const T* __restrict__ q, const T* __restrict__ k,
                   const T* __restrict__ v, T* __restrict__ y, const uint64_t* __restrict__ packed,
                   const float* __restrict__ weight, int64_t D, int dk, int dv, int tu, int P, int closed,
                   float xscale, int npieces, int steps, int max_rows, float* __restrict__ xpart,
                   int* __restrict__ cnt, float* __restrict__ R, float even_share) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  const int tid = threadIdx.x;
  const bool split = npieces > 1;
  const int piece = (int)(blockIdx.x % (unsigned)npieces);
  const int64_t bh = (int64_t)(blockIdx.x / (unsigned)npieces);
  // the piece's steps: the first piece starts at 0 and the last runs to the end
  auto step_of = [&](int p) -> int64_t {
    const float w = (float)(p >> 1) + ((p & 1) ? even_share : 0.0f);
    return (int64_t)(w * 2.0f / (float)npieces * (float)steps + 0.5f);
  };
  const int64_t m_lo = (piece == 0) ? 0 : step_of(piece);
  const int64_t m_hi = (piece == npieces - 1) ? ((int64_t)1 << 40) : step_of(piece + 1);
  const int64_t N = D * E;
  float* const Sh = S + bh * N;
  float* const Rh = COMP ? R + bh * (D + (int64_t)(dk + 1) * dv) : nullptr;
  float2* const fkq = (float2*)lds;        // [max_rows] {phi_k, phi_q} of rows row_lo..
  float* const xq = (float*)(fkq + max_rows);  // [dk]
  float* const xk = xq + dk;               // [dk]
  float* const ve = xk + dk;               // [E]
  float* const red = ve + E;               // [4 tu] per-thread column sums
  float* const part = red + 4 * tu;        // [8][E]
  float* const o = part + 8 * E;           // [E]
  float* const lo_val = o + E;             // [8] readout terms of the leftover elements
  int* const lo_col = (int*)(lo_val + 8);  // [8] their columns

  const int a0 = (int)((4 - ((bh * N) & 3)) & 3);
  const int64_t nv = (N - a0) / 4;         // float4s in the aligned part
  const float4* const Sv = (const float4*)(Sh + a0);
  const bool active = tid < tu;
  // leftover elements [0, a0) and [a0 + 4 nv, N): one per thread of the last
  // wave; the first piece takes the leading ones, the last the trailing ones
  const int nlead = (piece == 0) ? (int)min<int64_t>(a0, N) : 0;
  const int ntrail = (piece == npieces - 1) ? (int)(N - (a0 + 4 * nv)) : 0;
  const int nleft = nlead + ntrail;
  const int lt = tid - (NTH - 8);
  const int64_t le = (lt < nlead) ? lt : a0 + 4 * nv + (lt - nlead);
  // the state rows this workgroup touches: its features are kept from row_lo on
  const int64_t row_lo = (piece == 0) ? 0 : min<int64_t>(D - 1, (a0 + 4 * min<int64_t>(nv, (int64_t)tu * m_lo)) / E);
  const int64_t row_hi =
      (piece == npieces - 1) ? D - 1 : max<int64_t>(row_lo, (a0 + 4 * min<int64_t>(nv, (int64_t)tu * m_hi) - 1) / E);
  // q, k, v go to LDS first (in the first wave, which waits for them there),
  // then every wave sends its first state loads, which stay in flight while
  // the features are computed: the barriers below wait for LDS only
  if (tid < dk) {
    xq[tid] = to_f32(q[bh * dk + tid]) * xscale;
    xk[tid] = to_f32(k[bh * dk + tid]) * xscale;
  }
  if (tid < E) ve[tid] = (tid < dv) ? to_f32(v[bh * dv + tid]) : 1.0f;
  // (branch-free: an out-of-range slot reads element 0, which the stream skips)
  const bool lead = lt >= 0 && lt < nleft;
  float lx = Sh[lead ? le : 0];
  float4 cur[kFlatUnroll];
#pragma unroll
  for (int u = 0; u < kFlatUnroll; ++u) {
    const int64_t g = tid + (int64_t)tu * (m_lo + u);
    cur[u] = Sv[(active && g < nv && m_lo + u < m_hi) ? g : 0];
  }
  lx = lead ? lx : 0.0f;
  lds_barrier();
  if (closed) {
    // Features in closed form, no table (LDS holds x~ = x d^(-1/4)).  Work
    // items are (prefix i1 <= i2, block h of up to 8 third indices i3 in
    // [i2 + 8h, i2 + 8h + 8)); tier h holds the prefixes with i2 < d - 8h,
    // numbered i2-major (rank i2 (i2 + 1) / 2 + i1), so an item decodes
    // without a search and none walks more than 8 features.  Tier 0 also
    // writes the degree-2 feature (i1, i2); the last threads write degrees 0
    // and 1.  Rows are the canonical (degree-major, lexicographic) positions;
    // phi_m = prod x~[m_j] / sqrt(prod c!).  Items wholly outside this
    // workgroup's rows are skipped.
    const int npair = dk * (dk + 1) / 2;
    const int base2 = 1 + dk, base3 = 1 + dk + npair;
    const int rlo32 = (int)row_lo, rhi32 = (int)row_hi;  // (a closed-form head has D < 2^31 rows)
    int nitems = 0;
    for (int m = dk; m > 0; m -= 8) nitems += m * (m + 1) / 2;
    for (int it = tid; it < nitems; it += NTH) {
      int h = 0, r = it;
      for (int m = dk; r >= m * (m + 1) / 2; m -= 8) {
        r -= m * (m + 1) / 2;
        ++h;
      }
      // i2 = floor((sqrt(8 r + 1) - 1) / 2), from an estimate and exact corrections
      int i2 = (int)((__builtin_amdgcn_sqrtf(8.0f * (float)r + 1.0f) - 1.0f) * 0.5f);
      while ((i2 + 1) * (i2 + 2) / 2 <= r) ++i2;
      while (i2 * (i2 + 1) / 2 > r) --i2;
      const int i1 = r - i2 * (i2 + 1) / 2;
      const float qa = xq[i1], qb = xq[i2], ka = xk[i1], kb = xk[i2];
      if (h == 0) {
        const int row2 = base2 + i1 * dk - i1 * (i1 - 1) / 2 + (i2 - i1);
        const float w2 = (i1 == i2) ? 0.70710678118654752f : 1.0f;
        if (row2 >= rlo32 && row2 <= rhi32) fkq[row2 - rlo32] = float2{ka * kb * w2, qa * qb * w2};
      }
      // degree-3 tuples before (i1, i2, i2): all with a smaller first index,
      // then first index i1 and second index in [i1, i2)
      const int start3 = base3 + (dk + 2) * (dk + 1) * dk / 6 - (dk - i1 + 2) * (dk - i1 + 1) * (dk - i1) / 6 +
                         (i2 - i1) * dk - (i2 * (i2 - 1) - i1 * (i1 - 1)) / 2;
      const int j0 = i2 + 8 * h;
      // the item's features u = 0..7 (rows rfirst + u) that exist (i3 < d) and
      // fall in this workgroup's rows
      const int rfirst = start3 + (j0 - i2);
      const int ulo = max(0, rlo32 - rfirst);
      const int uhi = min(min(8, dk - j0), rhi32 - rfirst + 1);
      if (ulo >= uhi) continue;
      const float pq = qa * qb, pk = ka * kb;
      // 1 / sqrt(prod c!): three equal indices (1/sqrt(6)) only at i3 = i2 = i1,
      // two (1/sqrt(2)) at i3 = i2 or i1 = i2
      const float wrest = (i1 == i2) ? 0.70710678118654752f : 1.0f;
      const float wfirst = (h > 0) ? wrest : ((i1 == i2) ? 0.40824829046386302f : 0.70710678118654752f);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int i3 = j0 + u;
        const int ic = min(i3, dk - 1);  // in range, so the reads need no guard
        const float xk3 = xk[ic], xq3 = xq[ic];
        const float w3 = (u == 0) ? wfirst : wrest;
        if ((unsigned)(u - ulo) < (unsigned)(uhi - ulo)) fkq[rfirst - rlo32 + u] = float2{pk * xk3 * w3, pq * xq3 * w3};
      }
    }
    const int t1 = NTH - 1 - tid;
    if (t1 <= dk && t1 >= rlo32 && t1 <= rhi32)
      fkq[t1 - rlo32] = (t1 == 0) ? float2{1.0f, 1.0f} : float2{xk[t1 - 1], xq[t1 - 1]};
  } else {
    // the table entries of up to 8 of the rows per thread are loaded together
    for (int64_t fb = row_lo + tid; fb <= row_hi; fb += 8 * NTH) {
      uint64_t pk[8];
      float w[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int64_t f = fb + (int64_t)NTH * u;
        pk[u] = (f <= row_hi) ? packed[f] : 0;
        w[u] = (f <= row_hi) ? weight[f] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int64_t f = fb + (int64_t)NTH * u;
        if (f <= row_hi) fkq[f - row_lo] = float2{feature_value(pk[u], w[u], xk), feature_value(pk[u], w[u], xq)};
      }
    }
  }
  lds_barrier();
  if (lt >= 0 && lt < nleft) {
    const int64_t f = le / E;
    const int j = (int)(le - f * E);
    const float2 fw = fkq[f - row_lo];
    const int ri = COMP ? comp_index((int)f, j, (int)D, dk, dv) : -1;
    if (COMP && ri >= 0) {
      float r = Rh[ri];
      comp_add(lx, r, __fmul_rn(fw.x, ve[j]));
      Rh[ri] = r;
    } else {
      lx += fw.x * ve[j];
    }
    Sh[le] = lx;
    lo_val[lt] = fw.y * lx;
    lo_col[lt] = j;
  }

  // this thread's four lanes: rows fr[c] + rps m (f0[c] + rps m counted from
  // the piece's first row), columns jc[c]
  const int rps = 4 * tu / E;
  int f0[4], jc[4], fr[4];
  float vj[4], acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int e = a0 + 4 * tid + c;
    fr[c] = e / E;
    jc[c] = e - fr[c] * E;
    f0[c] = fr[c] - (int)row_lo;
    vj[c] = ve[jc[c]];
    acc[c] = 0.0f;
  }
  // residuals of the compensated lanes of the first kFlatUnroll steps (COMP only)
  float rc[kFlatUnroll][4];
#pragma unroll
  for (int u = 0; u < kFlatUnroll; ++u) {
    const int64_t g = tid + (int64_t)tu * (m_lo + u);
    const bool ok = active && g < nv && m_lo + u < m_hi;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      rc[u][c] = 0.0f;
      if (COMP) {
        const int ri = comp_index(fr[c] + rps * (int)(m_lo + u), jc[c], (int)D, dk, dv);
        if (ok && ri >= 0) rc[u][c] = Rh[ri];
      }
    }
  }
  float4* const Sw = (float4*)(Sh + a0);
  if (active) {
    for (int64_t m0 = m_lo;; m0 += kFlatUnroll) {
      float4 nxt[kFlatUnroll];
      float rn[kFlatUnroll][4];
#pragma unroll
      for (int u = 0; u < kFlatUnroll; ++u) {
        const int64_t m = m0 + kFlatUnroll + u;
        const int64_t g = tid + (int64_t)tu * m;
        const bool ok = g < nv && m < m_hi;
        nxt[u] = ok ? Sv[g] : float4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          rn[u][c] = 0.0f;
          if (COMP) {
            const int ri = comp_index(fr[c] + rps * (int)m, jc[c], (int)D, dk, dv);
            if (ok && ri >= 0) rn[u][c] = Rh[ri];
          }
        }
      }
      bool more = false;
#pragma unroll
      for (int u = 0; u < kFlatUnroll; ++u) {
        const int64_t m = m0 + u;
        const int64_t g = tid + (int64_t)tu * m;
        if (g < nv && m < m_hi) {
          float x[4] = {cur[u].x, cur[u].y, cur[u].z, cur[u].w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const float2 fw = fkq[f0[c] + rps * m];
            const int ri = COMP ? comp_index(fr[c] + rps * (int)m, jc[c], (int)D, dk, dv) : -1;
            if (COMP && ri >= 0) {
              float r = rc[u][c];
              comp_add(x[c], r, __fmul_rn(fw.x, vj[c]));
              Rh[ri] = r;
            } else {
              x[c] += fw.x * vj[c];
            }
            acc[c] += fw.y * x[c];
          }
          Sw[g] = float4{x[0], x[1], x[2], x[3]};
          more = true;
        }
        cur[u] = nxt[u];
#pragma unroll
        for (int c = 0; c < 4; ++c) rc[u][c] = rn[u][c];
      }
      if (!more) break;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) red[4 * tid + c] = acc[c];
  }
  __syncthreads();
  // column sums: 8 partial sums per column over the entries of that column
  if (tid < 8 * E) {
    const int j = tid % E, pp = tid / E;
    const int p0 = ((j - a0) % E + E) % E;  // red[p] holds column (a0 + p) mod E
    float a = 0.0f;
    for (int p = p0 + E * pp; p < 4 * tu; p += 8 * E) a += red[p];
    part[tid] = a;
  }
  __syncthreads();
  if (tid < E) {
    float a = 0.0f;
#pragma unroll
    for (int pp = 0; pp < 8; ++pp) a += part[pp * E + tid];
    o[tid] = a;
  }
  __syncthreads();
  if (tid == 0)
    for (int i = 0; i < nleft; ++i) o[lo_col[i]] += lo_val[i];  // leftover terms, in element order
  __syncthreads();
  if (split) {
    if (tid < E)
      __hip_atomic_store(xpart + (bh * npieces + piece) * E + tid, o[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);  // the stores have completed before the count goes up
    __syncthreads();
    int* const arrived = (int*)red;  // (the column sums are no longer needed)
    if (tid == 0) arrived[0] = __hip_atomic_fetch_add(cnt + bh, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (arrived[0] != npieces - 1) return;  // a later piece finishes the head
    if (npieces == 2) {  // (a two-term sum does not depend on the order)
      if (tid < E)
        o[tid] += __hip_atomic_load(xpart + (bh * 2 + (piece ^ 1)) * E + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else if (tid < E) {
      // the other pieces' sums, 8 loads in flight at a time, added in piece order
      // (this piece's own from LDS)
      const float* const xp = xpart + bh * npieces * E + tid;
      float a = 0.0f;
      for (int p0 = 0; p0 < npieces; p0 += 8) {
        float w[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          w[u] = (p0 + u < npieces && p0 + u != piece)
                     ? __hip_atomic_load(xp + (p0 + u) * E, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                     : 0.0f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (p0 + u < npieces) a += (p0 + u == piece) ? o[tid] : w[u];
      }
      o[tid] = a;
    }
    if (tid == 0) __hip_atomic_store(cnt + bh, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
  }
  for (int j = tid; j < dv; j += NTH) y[bh * dv + j] = from_f32<T>(o[j] / o[dv]);
}

template <typename T>
__global__ void __launch_bounds__(kThreads)
decode_slice_kernel(float* __restrict__ S, const T* __restrict__ q, const T* __restrict__ k,
                    const T* __restrict__ v, float* __restrict__ partial, const uint64_t* __restrict__ packed,
                    const float* __restrict__ weight, int64_t D, int dk, int dv, int fps, int nslices) {
  extern __shared__ float lds[];
  const int s = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int64_t f0 = (int64_t)s * fps;
  const int nf = (int)min<int64_t>(fps, D - f0);
  decode_rows<T, kThreads>(S, q, k, v, packed, weight, D, dk, dv, bh, f0, nf, lds);
  const float* red = lds + 2 * dk + (dv + 1) + 2 * nf;
  for (int j = threadIdx.x; j < dv + 1; j += kThreads) partial[(bh * nslices + s) * (dv + 1) + j] = red[j];
}

template <typename T>
__global__ void decode_finalize_kernel(const float* __restrict__ partial, T* __restrict__ y, int dv,
                                       int nslices) {
  extern __shared__ float o[];
  const int E = dv + 1;
  const int64_t bh = blockIdx.x;
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    float a = 0.0f;
    for (int s = 0; s < nslices; ++s) a += partial[(bh * nslices + s) * E + j];
    o[j] = a;
  }
  __syncthreads();
  for (int j = threadIdx.x; j < dv; j += blockDim.x) y[bh * dv + j] = from_f32<T>(o[j] / o[dv]);
}

// ---------------------------------------------------------------- generic prefill

// q holds qg query heads per key/value head (head bh's queries at head bh * qg).
template <typename T>
__device__ void load_chunk(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                           int64_t bh, int n, int t0, int cn, int C, int dk, int dv, float* xq, float* xk,
                           float* ve, int qg, int XS) {
  // xq, xk: [C][XS] (XS >= dk); ve: [C][d_v + 1] with the constant-1 column
  const int E = dv + 1;
  const int64_t qoff = (bh * qg * n + t0) * (int64_t)dk;
  const int64_t koff = (bh * n + t0) * (int64_t)dk;
  for (int i = threadIdx.x; i < C * dk; i += kThreads) {
    const int t = i / dk;
    const int c = i - t * dk;
    xq[t * XS + c] = t < cn ? to_f32(q[qoff + i]) : 0.0f;
    xk[t * XS + c] = t < cn ? to_f32(k[koff + i]) : 0.0f;
  }
  const int64_t voff = (bh * n + t0) * (int64_t)dv;
  for (int i = threadIdx.x; i < C * E; i += kThreads) {
    const int t = i / E;
    const int j = i - t * E;
    float val = 0.0f;
    if (t < cn) val = (j < dv) ? to_f32(v[voff + (int64_t)t * dv + j]) : 1.0f;
    ve[i] = val;
  }
}

template <typename T>
__global__ void __launch_bounds__(kThreads)
prefill_generic_main(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                     const uint64_t* __restrict__ packed, const float* __restrict__ weight, int64_t D,
                     float* __restrict__ S_state, float* __restrict__ part, int BH, int n, int dk, int dv,
                     int C, int FS, int seg0, int seg_len, int first_seg, int qg) {
  // FS: features per slice, a multiple of 4 (the last slice may hold fewer, fs)
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  float* Sl = lds;              // [FS][E] this slice of the state
  float* fb = Sl + FS * E;      // [C][FS] feature values of the chunk (q, then k)
  float* xq = fb + C * FS;      // [C][dk]
  float* xk = xq + C * dk;      // [C][dk]
  float* ve = xk + C * dk;      // [C][E]
  uint64_t* tpk = (uint64_t*)(ve + C * E);  // [FS] the slice's table entries
  float* tw = (float*)(tpk + FS);           // [FS]
  const int s = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int64_t f0 = (int64_t)s * FS;
  const int fs = (int)min<int64_t>(FS, D - f0);
  float* Sg = S_state + (bh * D + f0) * E;

  for (int i = tid; i < fs * E; i += kThreads) Sl[i] = first_seg ? 0.0f : Sg[i];
  for (int f = tid; f < fs; f += kThreads) {
    tpk[f] = packed[f0 + f];
    tw[f] = weight[f0 + f];
  }
  const int TQ = C / 4;  // readout tiles: tokens tq + TQ u, u = 0..3

  const int seg_end = min(n, seg0 + seg_len);
  for (int t0 = seg0; t0 < seg_end; t0 += C) {
    const int cn = min(C, n - t0);
    __syncthreads();
    load_chunk(q, k, v, bh, n, t0, cn, C, dk, dv, xq, xk, ve, qg, dk);
    __syncthreads();
    for (int i = tid; i < cn * fs; i += kThreads) {
      const int t = i / fs;
      const int f = i - t * fs;
      fb[t * FS + f] = feature_value(tpk[f], tw[f], xq + t * dk);
    }
    __syncthreads();
    // inter-chunk readout against the state before this chunk: each thread
    // sums 4 tokens x 1 value column, 4 features per step
    float* pout = part + (((int64_t)s * BH + bh) * seg_len + (t0 - seg0)) * E;
    for (int tile = tid; tile < TQ * E; tile += kThreads) {
      const int tq = tile / E;
      const int j = tile - tq * E;
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      int f = 0;
      for (; f + 4 <= fs; f += 4) {
        const float s0 = Sl[f * E + j], s1 = Sl[(f + 1) * E + j], s2 = Sl[(f + 2) * E + j], s3 = Sl[(f + 3) * E + j];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float4 a = *(const float4*)(fb + (tq + TQ * u) * FS + f);
          acc[u] += a.x * s0 + a.y * s1 + a.z * s2 + a.w * s3;
        }
      }
      for (; f < fs; ++f) {
        const float s0 = Sl[f * E + j];
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[u] += fb[(tq + TQ * u) * FS + f] * s0;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (tq + TQ * u < cn) pout[(tq + TQ * u) * E + j] = acc[u];
    }
    __syncthreads();
    for (int i = tid; i < cn * fs; i += kThreads) {
      const int t = i / fs;
      const int f = i - t * fs;
      fb[t * FS + f] = feature_value(tpk[f], tw[f], xk + t * dk);
    }
    __syncthreads();
    // state update with this chunk's keys and values: each thread sums 4
    // features x 1 value column over the chunk's tokens (columns of fb past
    // fs feed only sums that are not stored)
    for (int tile = tid; tile < (FS / 4) * E; tile += kThreads) {
      const int fg = tile / E;
      const int j = tile - fg * E;
      const int f = 4 * fg;
      if (f >= fs) continue;
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int t = 0; t < cn; ++t) {
        const float4 a = *(const float4*)(fb + t * FS + f);
        const float vv = ve[t * E + j];
        acc[0] += a.x * vv;
        acc[1] += a.y * vv;
        acc[2] += a.z * vv;
        acc[3] += a.w * vv;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (f + u < fs) Sl[(f + u) * E + j] += acc[u];
    }
  }
  __syncthreads();
  for (int i = tid; i < fs * E; i += kThreads) Sg[i] = Sl[i];
}

constexpr int kFinRows = 32;
__host__ __device__ constexpr int fin_stride(int dk) { return dk | 1; }

template <typename T>
__global__ void __launch_bounds__(kThreads)
prefill_generic_finalize(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                         const float* __restrict__ part, T* __restrict__ y, int BH, int n, int dk, int dv,
                         int P, int C, int nslices, int seg0, int seg_len, int qg) {
  extern __shared__ float lds[];
  const int E = dv + 1;
  // odd row stride: the lanes of the QK^T loop read different key rows
  const int XS = fin_stride(dk);
  float* xq = lds;                 // [C][XS]
  float* xk = xq + C * XS;         // [C][XS]
  float* ve = xk + C * XS;         // [C][E]
  float* A = ve + C * E;           // [kFinRows][C]
  float* O = A + kFinRows * C;     // [kFinRows][E]
  const int64_t bh = blockIdx.y;
  const int t0 = seg0 + blockIdx.x * C;
  if (t0 >= n) return;
  const int cn = min(C, n - t0);
  const int tid = threadIdx.x;
  const float scale = 1.0f / sqrtf((float)dk);
  load_chunk(q, k, v, bh, n, t0, cn, C, dk, dv, xq, xk, ve, qg, XS);
  __syncthreads();
  for (int rb = 0; rb < cn; rb += kFinRows) {
    const int rn = min(kFinRows, cn - rb);
    for (int i = tid; i < rn * C; i += kThreads) {
      const int r = i / C;
      const int tp = i - r * C;
      const int t = rb + r;
      float a = 0.0f;
      if (tp <= t) {
        float dot = 0.0f;
        for (int c = 0; c < dk; ++c) dot += xq[t * XS + c] * xk[tp * XS + c];
        a = taylor_horner(dot * scale, P);
      }
      A[i] = a;
    }
    __syncthreads();
    for (int o = tid; o < rn * E; o += kThreads) {
      const int r = o / E;
      const int j = o - r * E;
      const int t = rb + r;
      const float* const pr = part + ((int64_t)bh * seg_len + (t0 - seg0) + t) * E + j;
      const int64_t sstride = (int64_t)BH * seg_len * E;
      const float p0 = nslices > 0 ? pr[0] : 0.0f;  // issued before the sum below
      float acc = 0.0f;
      for (int tp = 0; tp <= t; ++tp) acc += A[r * C + tp] * ve[tp * E + j];
      acc += p0;
      for (int s = 1; s < nslices; ++s) acc += pr[s * sstride];
      O[o] = acc;
    }
    __syncthreads();
    for (int o = tid; o < rn * dv; o += kThreads) {
      const int r = o / dv;
      const int j = o - r * dv;
      y[(bh * qg * n + t0 + rb + r) * (int64_t)dv + j] = from_f32<T>(O[r * E + j] / O[r * E + dv]);
    }
    __syncthreads();
  }
}

__global__ void fill_zero_kernel(float* p, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = 0.0f;
}

}  // namespace

// ---------------------------------------------------------------- launchers

bool decode_supports_residuals(const DecodePlan& plan, const float* S) {
  return plan.flat_tu > 0 && ((uintptr_t)S & 15) == 0;
}

hipError_t launch_fill_zero(float* p, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + kThreads - 1) / kThreads, 16384);
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, p, count);
  return hipGetLastError();
}

// Share of each (even, odd) pair of decode pieces given to the even one: the
// MI355X value where the device is one (gfx950 with 256 compute units, whose
// workgroups go to its 8 XCDs in turn), an even split on any other device.
// Looked up once per device.
float xcd_even_share() {
  static std::atomic<int> cache[64];  // 0: unknown, 1: MI355X, 2: other
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0.5f;
  int c = cache[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    hipDeviceProp_t prop;
    c = 2;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess && prop.multiProcessorCount == 256 &&
        std::strncmp(prop.gcnArchName, "gfx950", 6) == 0)
      c = 1;
    cache[dev].store(c, std::memory_order_relaxed);
  }
  return c == 1 ? kMi355EvenShare : 0.5f;
}

DecodePlan plan_decode(int64_t D, int dk, int dv, int BH) {
  const int E = dv + 1;
  DecodePlan p;
  p.even_share = xcd_even_share();
  // Row-wise plans, used when the state is not 16-byte aligned: a head whose
  // feature values fit in LDS is streamed by one workgroup, a larger one in
  // feature slices of about 32K state elements (128 KB of float32) with a
  // second launch adding the slices' sums.
  if (2 * D * (int64_t)sizeof(float) <= 96 * 1024) {
    p.fps = (int)D;
    p.nslices = 1;
    p.threads = D * E > 65536 ? 1024 : 256;
  } else {
    int64_t fps = std::max<int64_t>(kThreads / E, (32768 + E - 1) / E);
    fps = std::min<int64_t>(fps, 4096);
    fps = std::min<int64_t>(fps, D);
    p.fps = (int)fps;
    p.nslices = (int)((D + fps - 1) / fps);
    p.threads = kThreads;
  }
  // The flat float4 stream (decode_flat_kernel).  Heads of at most 256 KB of
  // state take one 256-thread workgroup each (up to 8 stream on a CU at once);
  // larger heads 1024-thread workgroups, an even number of pieces per head:
  // two, or more while the grid has fewer than 512 workgroups and every piece
  // keeps at least 8 steps per thread.
  const int nth = (D * E <= 65536 && 8 * E <= 256 && dk < 256) ? 256 : 1024;
  const int unit = E / std::gcd(E, 4);
  const int tu = (nth / unit) * unit;
  if (tu <= 0 || 8 * E > nth || dk >= nth) return p;
  const int64_t steps = (D * E / 4 + tu - 1) / tu;
  int np = 1;
  if (nth == 1024 && steps >= 4) {
    np = 2;
    while ((int64_t)BH * np < 512 && steps / (2 * np) >= 8 && np < 64) np *= 2;
  }
  // rows a piece touches at most: its steps (the larger share of a pair, plus
  // rounding) times 4 tu elements, and the rows cut at both ends
  int64_t rows = D;
  if (np > 1) {
    const double share = std::max(p.even_share, 1.0f - p.even_share);
    const int64_t piece_steps = (int64_t)(share * 2.0 / np * (double)steps) + 2;
    rows = std::min<int64_t>(D, (4 * tu * piece_steps + 3) / E + 3);
  }
  const size_t lds = sizeof(float2) * (size_t)rows + sizeof(float) * (size_t)(2 * dk + E + 4 * tu + 9 * E + 16);
  if (lds > 150 * 1024) return p;
  p.flat_tu = tu;
  p.flat_lds = lds;
  p.flat_nth = nth;
  p.flat_np = np;
  p.flat_steps = (int)steps;
  p.flat_rows = (int)rows;
  return p;
}

hipError_t launch_decode(float* S, const void* q, const void* k, const void* v, void* y, bool bf16, int BH,
                         int dk, int dv, const DevTable& t, const DecodePlan& plan, float* partial,
                         int* counters, hipStream_t s, float* R) {
  const int E = dv + 1;
  if (R != nullptr && !decode_supports_residuals(plan, S)) return hipErrorInvalidValue;
  if (plan.flat_tu > 0 && ((uintptr_t)S & 15) == 0) {
    hipError_t e;
    if (plan.flat_np > 1 && (partial == nullptr || counters == nullptr)) return hipErrorInvalidValue;
    // Closed-form features for P = 4 when a piece's rows are a large part of
    // the head; the feature table otherwise.  The closed form takes the
    // coordinates already scaled by d^(-1/4) (computed here with the float
    // operations the features would otherwise do per use); the table path
    // scales by itself.
    const int closed = (t.P == 4 && plan.flat_np <= 2) ? 1 : 0;
    const float xscale = closed ? 1.0f / std::sqrt(std::sqrt((float)dk)) : 1.0f;
#define SATA_DECODE_FLAT(TT, NTH, COMP)                                                                   \
  e = hipFuncSetAttribute((const void*)decode_flat_kernel<TT, NTH, COMP>,                                 \
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.flat_lds);                \
  if (e != hipSuccess) return e;                                                                          \
  hipLaunchKernelGGL((decode_flat_kernel<TT, NTH, COMP>), dim3((unsigned)BH * (unsigned)plan.flat_np),         \
                     dim3(NTH), plan.flat_lds, s, S, (const TT*)q, (const TT*)k, (const TT*)v, (TT*)y, t.packed,  \
                     t.weight, t.D, dk, dv, plan.flat_tu, t.P, closed, xscale, plan.flat_np, plan.flat_steps,     \
                     plan.flat_rows, partial, counters, R, plan.even_share)
#define SATA_DECODE_FLAT_C(TT, NTH) \
  if (R) { SATA_DECODE_FLAT(TT, NTH, true); } else { SATA_DECODE_FLAT(TT, NTH, false); }
    if (plan.flat_nth == 256) {
      if (bf16) { SATA_DECODE_FLAT_C(bf16_t, 256); } else { SATA_DECODE_FLAT_C(float, 256); }
    } else {
      if (bf16) { SATA_DECODE_FLAT_C(bf16_t, 1024); } else { SATA_DECODE_FLAT_C(float, 1024); }
    }
#undef SATA_DECODE_FLAT_C
#undef SATA_DECODE_FLAT
    return hipGetLastError();
  }
  if (plan.nslices == 1) {
    // whole head per workgroup: one launch per step
    const size_t lds = sizeof(float) * (2 * dk + E + 2 * (size_t)t.D + plan.threads);
    hipError_t e;
#define SATA_DECODE_HEAD(TT, NTH)                                                                         \
  e = hipFuncSetAttribute((const void*)decode_head_kernel<TT, NTH>, hipFuncAttributeMaxDynamicSharedMemorySize, \
                          (int)lds);                                                                      \
  if (e != hipSuccess) return e;                                                                          \
  hipLaunchKernelGGL((decode_head_kernel<TT, NTH>), dim3((unsigned)BH), dim3(NTH), lds, s, S, (const TT*)q,  \
                     (const TT*)k, (const TT*)v, (TT*)y, t.packed, t.weight, t.D, dk, dv)
    if (plan.threads == 1024) {
      if (bf16) { SATA_DECODE_HEAD(bf16_t, 1024); } else { SATA_DECODE_HEAD(float, 1024); }
    } else {
      if (bf16) { SATA_DECODE_HEAD(bf16_t, 256); } else { SATA_DECODE_HEAD(float, 256); }
    }
#undef SATA_DECODE_HEAD
    return hipGetLastError();
  }
  const size_t lds = sizeof(float) * (2 * dk + E + 2 * plan.fps + kThreads);
  dim3 grid((unsigned)plan.nslices, (unsigned)BH);
  if (bf16)
    hipLaunchKernelGGL(decode_slice_kernel<bf16_t>, grid, dim3(kThreads), lds, s, S, (const bf16_t*)q,
                       (const bf16_t*)k, (const bf16_t*)v, partial, t.packed, t.weight, t.D, dk, dv, plan.fps,
                       plan.nslices);
  else
    hipLaunchKernelGGL(decode_slice_kernel<float>, grid, dim3(kThreads), lds, s, S, (const float*)q,
                       (const float*)k, (const float*)v, partial, t.packed, t.weight, t.D, dk, dv, plan.fps,
                       plan.nslices);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds2 = sizeof(float) * E;
  if (bf16)
    hipLaunchKernelGGL(decode_finalize_kernel<bf16_t>, dim3((unsigned)BH), dim3(64), lds2, s, partial,
                       (bf16_t*)y, dv, plan.nslices);
  else
    hipLaunchKernelGGL(decode_finalize_kernel<float>, dim3((unsigned)BH), dim3(64), lds2, s, partial,
                       (float*)y, dv, plan.nslices);
  return hipGetLastError();
}

// gfx950 offers 160 KB of LDS per workgroup; the generic kernels use up to 128 KB.
static constexpr size_t kLdsBudget = 128 * 1024;

bool plan_prefill_generic(int64_t D, int BH, int n, int dk, int dv, int chunk, size_t max_ws_bytes,
                          PrefillGenericPlan* plan) {
  const int E = dv + 1;
  const int C = chunk;
  const size_t fixed = sizeof(float) * ((size_t)2 * C * dk + (size_t)C * E);
  // per feature: its state row, its column of chunk feature values and its table entry
  const size_t per_feature = sizeof(float) * ((size_t)E + C) + sizeof(uint64_t) + sizeof(float);
  // LDS per workgroup: every slice re-reads the chunk's q, k, v tiles, so
  // slices are as wide as LDS allows when those tiles are large; when they are
  // small, narrower slices let several workgroups share a CU (one per CU
  // leaves the latency of one wave per SIMD exposed)
  const size_t budget = (fixed <= ((size_t)16 << 10)) ? ((size_t)40 << 10)
                        : (fixed <= ((size_t)32 << 10)) ? ((size_t)76 << 10)
                                                         : kLdsBudget;
  if (fixed + 8 * per_feature > budget) return false;
  int64_t fs = (int64_t)((budget - fixed) / per_feature);
  fs = std::min<int64_t>(fs, 512);
  // enough slices for about 4 workgroups per CU, but at least 32 features each
  const int64_t want = (1024 + BH - 1) / BH;
  fs = std::min<int64_t>(fs, std::max<int64_t>(32, (D + want - 1) / want));
  fs = std::min<int64_t>(fs, D);
  fs = std::max<int64_t>(4, fs / 4 * 4);  // a multiple of 4
  plan->fs = (int)fs;
  plan->nslices = (int)((D + fs - 1) / fs);
  plan->lds_main = fixed + per_feature * (size_t)fs;
  plan->lds_final = sizeof(float) * ((size_t)2 * C * fin_stride(dk) + (size_t)C * E + (size_t)kFinRows * C +
                                     (size_t)kFinRows * E);
  if (plan->lds_main > kLdsBudget || plan->lds_final > kLdsBudget) return false;
  // partial readouts for one segment: [nslices][BH][seg_len][E]
  const size_t per_token = sizeof(float) * (size_t)plan->nslices * BH * E;
  int64_t seg = (int64_t)(max_ws_bytes / per_token);
  seg = (seg / C) * C;
  if (seg < C) seg = C;
  const int64_t n_round = ((int64_t)std::max(n, 1) + C - 1) / C * C;
  plan->seg_len = (int)std::min<int64_t>(seg, n_round);
  plan->partial_bytes = per_token * (size_t)plan->seg_len;
  return true;
}

hipError_t launch_prefill_generic(const void* q, const void* k, const void* v, void* y, bool bf16, int BH,
                                  int n, int dk, int dv, int chunk, const DevTable& t,
                                  const PrefillGenericPlan& plan, float* S_state, float* partial,
                                  hipStream_t s, int qg) {
  const int C = chunk;
  hipError_t ea;
  if (bf16) {
    ea = hipFuncSetAttribute((const void*)prefill_generic_main<bf16_t>,
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.lds_main);
    if (ea == hipSuccess)
      ea = hipFuncSetAttribute((const void*)prefill_generic_finalize<bf16_t>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.lds_final);
  } else {
    ea = hipFuncSetAttribute((const void*)prefill_generic_main<float>,
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.lds_main);
    if (ea == hipSuccess)
      ea = hipFuncSetAttribute((const void*)prefill_generic_finalize<float>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.lds_final);
  }
  if (ea != hipSuccess) return ea;
  for (int seg0 = 0; seg0 < n; seg0 += plan.seg_len) {
    const int first = seg0 == 0 ? 1 : 0;
    dim3 g1((unsigned)plan.nslices, (unsigned)BH);
    if (bf16)
      hipLaunchKernelGGL(prefill_generic_main<bf16_t>, g1, dim3(kThreads), plan.lds_main, s,
                         (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, t.packed, t.weight, t.D,
                         S_state, partial, BH, n, dk, dv, C, plan.fs, seg0, plan.seg_len, first, qg);
    else
      hipLaunchKernelGGL(prefill_generic_main<float>, g1, dim3(kThreads), plan.lds_main, s,
                         (const float*)q, (const float*)k, (const float*)v, t.packed, t.weight, t.D, S_state,
                         partial, BH, n, dk, dv, C, plan.fs, seg0, plan.seg_len, first, qg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int seg_tokens = std::min(plan.seg_len, n - seg0);
    dim3 g2((unsigned)((seg_tokens + C - 1) / C), (unsigned)BH);
    if (bf16)
      hipLaunchKernelGGL(prefill_generic_finalize<bf16_t>, g2, dim3(kThreads), plan.lds_final, s,
                         (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, partial, (bf16_t*)y, BH, n,
                         dk, dv, t.P, C, plan.nslices, seg0, plan.seg_len, qg);
    else
      hipLaunchKernelGGL(prefill_generic_finalize<float>, g2, dim3(kThreads), plan.lds_final, s,
                         (const float*)q, (const float*)k, (const float*)v, partial, (float*)y, BH, n, dk,
                         dv, t.P, C, plan.nslices, seg0, plan.seg_len, qg);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_prefill_generic_readout(const void* q, const void* k, const void* v, bool bf16, int BH, int n,
                                          int dk, int dv, int chunk, const DevTable& t,
                                          const PrefillGenericPlan& plan, float* S_state, float* partial, int seg0,
                                          int seg_len, bool first, hipStream_t s) {
  const int C = chunk;
  hipError_t e;
  dim3 g1((unsigned)plan.nslices, (unsigned)BH);
  if (bf16) {
    if ((e = hipFuncSetAttribute((const void*)prefill_generic_main<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)plan.lds_main)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(prefill_generic_main<bf16_t>, g1, dim3(kThreads), plan.lds_main, s, (const bf16_t*)q,
                       (const bf16_t*)k, (const bf16_t*)v, t.packed, t.weight, t.D, S_state, partial, BH, n, dk, dv,
                       C, plan.fs, seg0, seg_len, first ? 1 : 0, 1);
  } else {
    if ((e = hipFuncSetAttribute((const void*)prefill_generic_main<float>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)plan.lds_main)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(prefill_generic_main<float>, g1, dim3(kThreads), plan.lds_main, s, (const float*)q,
                       (const float*)k, (const float*)v, t.packed, t.weight, t.D, S_state, partial, BH, n, dk, dv, C,
                       plan.fs, seg0, seg_len, first ? 1 : 0, 1);
  }
  return hipGetLastError();
}

}  // namespace sata
