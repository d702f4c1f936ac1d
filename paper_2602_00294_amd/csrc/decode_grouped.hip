// Decode step with grouped query heads: one state per key/value head, read
// out for G query heads at once (sharing one key/value head among several
// query heads is among the reuse schemes that a footnote of Sec. 3.3 says
// carry over to this formulation).  For each key/value
// head:  S += phi(k) (x) [v, 1]  once, then for each of its G query heads
// o_g = phi(q_g)^T S  and  y_g = o_g[0:d_v] / o_g[d_v].
//
// The kernel streams the head's state once, as the single-query flat decode
// does (a thread owns float4s t + tu m of the 16-byte aligned part, so each
// of its four lanes keeps one value column), and accumulates G readouts per
// element from that one read: the state traffic per step is that of one
// head, for G query tokens.  Feature values come from the table: phi(k) and
// the G phi(q_g) of the rows a workgroup touches sit in LDS.  Large heads are
// split into an even number of pieces per head; the last piece to arrive adds
// the pieces' sums in piece order, so results do not depend on timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <numeric>

#include "device_common.hpp"
#include "kernels.hpp"

namespace sata {

namespace {

constexpr int kGroupedUnroll = 2;
// The share of a head's stream given to the piece on an even-numbered XCD
// comes from xcd_even_share(): on MI355X the hardware deals workgroups to the
// 8 XCDs in turn and odd ones stream this pattern about a quarter more slowly;
// other devices split evenly.

__device__ __forceinline__ void lds_wait_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int G>
struct GroupRow;  // the G query feature values of one state row
template <>
struct GroupRow<2> {
  float2 a;
  __device__ __forceinline__ float operator[](int g) const { return g == 0 ? a.x : a.y; }
};
template <>
struct GroupRow<4> {
  float4 a;
  __device__ __forceinline__ float operator[](int g) const { return g == 0 ? a.x : g == 1 ? a.y : g == 2 ? a.z : a.w; }
};
template <>
struct GroupRow<8> {
  float4 a, b;
  __device__ __forceinline__ float operator[](int g) const {
    const float4 h = g < 4 ? a : b;
    const int i = g & 3;
    return i == 0 ? h.x : i == 1 ? h.y : i == 2 ? h.z : h.w;
  }
};

// LDS layout (floats): fk [rows4] | fq [rows4][G] | xq [G][dk+1] | xk [dk+1] |
// ve [E] | red [2][4 tu] | part [2][8][E] | o [G][E] | lo_val [G][8] | lo_col [8]
// with rows4 = max_rows rounded up to a multiple of 4 (fq 16-byte aligned).
__host__ __device__ inline size_t grouped_lds_floats(int max_rows, int G, int dk, int E, int tu) {
  const size_t rows4 = ((size_t)max_rows + 3) & ~(size_t)3;
  return rows4 * (1 + G) + (size_t)G * (dk + 1) + (dk + 1) + E + 8 * (size_t)tu + 16 * (size_t)E + (size_t)G * E +
         8 * (size_t)G + 8;
}

template <typename T, int NTH, int G>
__global__ void __launch_bounds__(NTH, (G <= 2 ? 8 : 4))
decode_grouped_kernel(float* __restrict__ S, const T* __restrict__ q, const T* __restrict__ k,
                      const T* __restrict__ v, T* __restrict__ y, const uint64_t* __restrict__ packed,
                      const uint32_t* __restrict__ gen, int64_t D, int dk, int dv, int tu, int npieces, int steps,
                      int max_rows, float* __restrict__ xpart, int* __restrict__ cnt, float even_share) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int E = dv + 1;
  const int tid = threadIdx.x;
  const bool split = npieces > 1;
  const int piece = __builtin_amdgcn_readfirstlane((int)(blockIdx.x % (unsigned)npieces));
  const int64_t bh = __builtin_amdgcn_readfirstlane((int)(blockIdx.x / (unsigned)npieces));  // key/value head
  auto step_of = [&](int p) -> int64_t {
    const float w = (float)(p >> 1) + ((p & 1) ? even_share : 0.0f);
    return (int64_t)(w * 2.0f / (float)npieces * (float)steps + 0.5f);
  };
  const int64_t m_lo = (piece == 0) ? 0 : step_of(piece);
  const int64_t m_hi = (piece == npieces - 1) ? ((int64_t)1 << 40) : step_of(piece + 1);
  const int64_t N = D * E;
  float* const Sh = S + bh * N;
  const int rows4 = (max_rows + 3) & ~3;
  float* const fk = lds;
  float* const fq = fk + rows4;
  float* const xq = fq + (size_t)rows4 * G;
  float* const xk = xq + G * (dk + 1);
  float* const ve = xk + dk + 1;
  float* const red = ve + E;       // [2][4 tu]
  float* const part = red + 8 * tu;  // [2][8][E]
  float* const o = part + 16 * E;
  float* const lo_val = o + G * E;
  int* const lo_col = (int*)(lo_val + 8 * G);

  const int a0 = (int)((4 - ((bh * N) & 3)) & 3);
  const int64_t nv = (N - a0) / 4;
  const float4* const Sv = (const float4*)(Sh + a0);
  const bool active = tid < tu;
  const int nlead = (piece == 0) ? (int)min<int64_t>(a0, N) : 0;
  const int ntrail = (piece == npieces - 1) ? (int)(N - (a0 + 4 * nv)) : 0;
  const int nleft = nlead + ntrail;
  const int lt = tid - (NTH - 8);
  const int64_t le = (lt < nlead) ? lt : a0 + 4 * nv + (lt - nlead);
  const int64_t row_lo = (piece == 0) ? 0 : min<int64_t>(D - 1, (a0 + 4 * min<int64_t>(nv, (int64_t)tu * m_lo)) / E);
  int64_t row_hi =
      (piece == npieces - 1) ? D - 1 : max<int64_t>(row_lo, (a0 + 4 * min<int64_t>(nv, (int64_t)tu * m_hi) - 1) / E);
  row_hi = min<int64_t>(row_hi, row_lo + max_rows - 1);  // never past the LDS rows (the plan bounds them)

  // the G query vectors of this key/value head are rows bh G .. bh G + G - 1
  // coordinates with a column dk held at 1 (read by the generation program
  // for degree-0 features and missing indices)
  for (int i = tid; i < G * (dk + 1); i += NTH) {
    const int g = i / (dk + 1), c = i - g * (dk + 1);
    xq[i] = c < dk ? to_f32(q[(bh * G + g) * dk + c]) : 1.0f;
  }
  for (int i = tid; i <= dk; i += NTH) xk[i] = i < dk ? to_f32(k[bh * dk + i]) : 1.0f;
  for (int i = tid; i < E; i += NTH) ve[i] = (i < dv) ? to_f32(v[bh * dv + i]) : 1.0f;
  const bool lead = lt >= 0 && lt < nleft;
  float lx = Sh[lead ? le : 0];
  float4 cur[kGroupedUnroll];
#pragma unroll
  for (int u = 0; u < kGroupedUnroll; ++u) {
    const int64_t g = tid + (int64_t)tu * (m_lo + u);
    cur[u] = Sv[(active && g < nv && m_lo + u < m_hi) ? g : 0];
  }
  lx = lead ? lx : 0.0f;
  // the first two generation-program entries of this thread's rows load
  // while the coordinates reach LDS (the barrier waits for LDS only)
  uint2 gw[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t f = row_lo + tid + (int64_t)NTH * u;
    gw[u] = (f <= row_hi) ? ((const uint2*)gen)[f] : uint2{0u, 0u};
  }
  lds_wait_barrier();
  // one feature at the G + 1 coordinate rows: weight times the coordinates of
  // the last index and the first two others (the column dk where missing),
  // times any further indices from the packed entry
  auto features = [&](uint2 g2, int64_t f, int64_t r) {
    const float w = __uint_as_float(g2.y);
    const int il = (int)((g2.x & 0x3ffu) >> 2), i0 = (int)((g2.x >> 10) & 0xffu), i1 = (int)((g2.x >> 18) & 0xffu);
    uint64_t e = 0;
    int p = 0;
    if ((g2.x >> 30) & 1u) {
      e = packed[f];
      p = (int)(e >> 56);
    }
    float vk = w * xk[i0] * xk[i1] * xk[il];
    for (int j = 2; j < p - 1; ++j) vk *= xk[(e >> (8 * j)) & 0xff];
    fk[r] = vk;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float* const xg = xq + g * (dk + 1);
      float vq = w * xg[i0] * xg[i1] * xg[il];
      for (int j = 2; j < p - 1; ++j) vq *= xg[(e >> (8 * j)) & 0xff];
      fq[r * G + g] = vq;
    }
  };
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t r = tid + (int64_t)NTH * u;
    if (row_lo + r <= row_hi) features(gw[u], row_lo + r, r);
  }
  for (int64_t f = row_lo + tid + 2 * (int64_t)NTH; f <= row_hi; f += NTH)
    features(((const uint2*)gen)[f], f, f - row_lo);
  lds_wait_barrier();
  if (lead) {
    const int64_t f = le / E;
    const int j = (int)(le - f * E);
    const int64_t r = f - row_lo;
    lx += fk[r] * ve[j];
    Sh[le] = lx;
#pragma unroll
    for (int g = 0; g < G; ++g) lo_val[g * 8 + lt] = fq[r * G + g] * lx;
    lo_col[lt] = j;
  }

  const int rps = 4 * tu / E;
  int f0[4];
  float vj[4];
  float acc[G][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int e = a0 + 4 * tid + c;
    f0[c] = e / E;
    vj[c] = ve[e - f0[c] * E];
    f0[c] -= (int)row_lo;
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g][c] = 0.0f;
  }
  float4* const Sw = (float4*)(Sh + a0);
  if (active) {
    for (int64_t m0 = m_lo;; m0 += kGroupedUnroll) {
      float4 nxt[kGroupedUnroll];
#pragma unroll
      for (int u = 0; u < kGroupedUnroll; ++u) {
        const int64_t m = m0 + kGroupedUnroll + u;
        const int64_t g = tid + (int64_t)tu * m;
        nxt[u] = (g < nv && m < m_hi) ? Sv[g] : float4{0.0f, 0.0f, 0.0f, 0.0f};
      }
      bool more = false;
#pragma unroll
      for (int u = 0; u < kGroupedUnroll; ++u) {
        const int64_t m = m0 + u;
        const int64_t g = tid + (int64_t)tu * m;
        if (g < nv && m < m_hi) {
          float x[4] = {cur[u].x, cur[u].y, cur[u].z, cur[u].w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            const int r = f0[c] + rps * (int)m;
            x[c] += fk[r] * vj[c];
            const GroupRow<G> fr = *(const GroupRow<G>*)(fq + (size_t)r * G);
#pragma unroll
            for (int gq = 0; gq < G; ++gq) acc[gq][c] += fr[gq] * x[c];
          }
          Sw[g] = float4{x[0], x[1], x[2], x[3]};
          more = true;
        }
        cur[u] = nxt[u];
      }
      if (!more) break;
    }
  }
  // column sums, one query head per round through two alternating sets of
  // LDS rows, so that a round needs one barrier: round g stores head g's
  // per-thread sums, then (after the barrier) adds them into 8 partial rows
  // per column and adds up head g-1's partial rows
  const int j8 = tid % E, pp8 = tid / E;
  const int p0 = ((j8 - a0) % E + E) % E;  // red[p] holds column (a0 + p) mod E
#pragma unroll
  for (int g = 0; g <= G; ++g) {
    float* const rb = red + (g & 1) * 4 * tu;
    if (g < G && active) {
#pragma unroll
      for (int c = 0; c < 4; ++c) rb[4 * tid + c] = acc[g < G ? g : 0][c];
    }
    __syncthreads();
    if (g < G && tid < 8 * E) {
      float a = 0.0f;
#pragma unroll 8
      for (int p = p0 + E * pp8; p < 4 * tu; p += 8 * E) a += rb[p];
      part[(g & 1) * 8 * E + tid] = a;
    }
    if (g > 0 && tid < E) {
      const float* const pb = part + ((g - 1) & 1) * 8 * E;
      float a = 0.0f;
#pragma unroll
      for (int pp = 0; pp < 8; ++pp) a += pb[pp * E + tid];
      o[(g - 1) * E + tid] = a;
    }
  }
  __syncthreads();
  if (tid < G) {
    for (int i = 0; i < nleft; ++i) o[tid * E + lo_col[i]] += lo_val[tid * 8 + i];  // leftovers, in element order
  }
  __syncthreads();
  const int GE = G * E;
  if (split) {
    for (int i = tid; i < GE; i += NTH)
      __hip_atomic_store(xpart + (bh * npieces + piece) * GE + i, o[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);  // the stores have completed before the count goes up
    __syncthreads();
    int* const arrived = (int*)red;
    if (tid == 0) arrived[0] = __hip_atomic_fetch_add(cnt + bh, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (arrived[0] != npieces - 1) return;  // a later piece finishes the head
    for (int i = tid; i < GE; i += NTH) {
      // the other pieces' sums, 8 loads in flight at a time, added in piece order
      const float* const xp = xpart + bh * npieces * GE + i;
      float a = 0.0f;
      for (int p0 = 0; p0 < npieces; p0 += 8) {
        float w[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          w[u] = (p0 + u < npieces && p0 + u != piece)
                     ? __hip_atomic_load(xp + (int64_t)(p0 + u) * GE, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                     : 0.0f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (p0 + u < npieces) a += (p0 + u == piece) ? o[i] : w[u];
      }
      o[i] = a;
    }
    if (tid == 0) __hip_atomic_store(cnt + bh, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
  }
  for (int i = tid; i < G * dv; i += NTH) {
    const int g = i / dv, j = i - g * dv;
    y[(bh * G + g) * dv + j] = from_f32<T>(o[g * E + j] / o[g * E + dv]);
  }
}

}  // namespace

GroupedDecodePlan plan_decode_grouped(int64_t D, int dk, int dv, int BH, int G) {
  GroupedDecodePlan p;
  const int E = dv + 1;
  if (G != 2 && G != 4 && G != 8) return p;
  p.even_share = xcd_even_share();
  const int nth = (D * E <= 65536 && 8 * E <= 256) ? 256 : 1024;
  const int unit = E / std::gcd(E, 4);
  const int tu = (nth / unit) * unit;
  if (tu <= 0 || 8 * E > nth) return p;
  const int64_t steps = (D * E / 4 + tu - 1) / tu;
  // pieces per head: at least one 1024-thread workgroup per compute unit (256)
  // while a piece keeps 4 steps per thread, then up to two while it keeps 8
  int np = 1;
  if (nth == 1024 && steps >= 4) {
    np = 2;
    while ((int64_t)BH * np < 256 && steps / (2 * np) >= 4 && np < 64) np *= 2;
    while ((int64_t)BH * np < 512 && steps / (2 * np) >= 8 && np < 64) np *= 2;
  }
  // rows a piece touches at most: its steps (the larger share of a pair, plus
  // rounding) times 4 tu elements, and the rows cut at both ends; more pieces
  // while the pieces' feature values do not fit in LDS
  auto rows_for = [&](int npc) -> int64_t {
    if (npc == 1) return D;
    const double share = std::max(p.even_share, 1.0f - p.even_share);
    const int64_t piece_steps = (int64_t)(share * 2.0 / npc * (double)steps) + 2;
    return std::min<int64_t>(D, (4 * tu * piece_steps + 3) / E + 3);
  };
  int64_t rows = rows_for(np);
  size_t lds = sizeof(float) * grouped_lds_floats((int)rows, G, dk, E, tu);
  while (lds > 150 * 1024 && nth == 1024 && np < 64 && steps / (2 * np) >= 2) {
    np = (np == 1) ? 2 : 2 * np;
    rows = rows_for(np);
    lds = sizeof(float) * grouped_lds_floats((int)rows, G, dk, E, tu);
  }
  if (lds > 150 * 1024) return p;
  p.tu = tu;
  p.lds = lds;
  p.nth = nth;
  p.np = np;
  p.steps = (int)steps;
  p.rows = (int)rows;
  p.G = G;
  return p;
}

hipError_t launch_decode_grouped(float* S, const void* q, const void* k, const void* v, void* y, bool bf16,
                                 int BH, int dk, int dv, const DevTable& t, const GroupedDecodePlan& plan,
                                 float* partial, int* counters, hipStream_t s) {
  if (plan.tu <= 0 || ((uintptr_t)S & 15) != 0) return hipErrorInvalidValue;
  if (plan.np > 1 && (partial == nullptr || counters == nullptr)) return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
#define SATA_DECODE_GROUPED(TT, NTH, GG)                                                                      \
  do {                                                                                                        \
    e = hipFuncSetAttribute((const void*)decode_grouped_kernel<TT, NTH, GG>,                                  \
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)plan.lds);                      \
    if (e != hipSuccess) return e;                                                                            \
    hipLaunchKernelGGL((decode_grouped_kernel<TT, NTH, GG>), dim3((unsigned)BH * (unsigned)plan.np), dim3(NTH), \
                       plan.lds, s, S, (const TT*)q, (const TT*)k, (const TT*)v, (TT*)y, t.packed, t.gen, t.D,   \
                       dk, dv, plan.tu, plan.np, plan.steps, plan.rows, partial, counters, plan.even_share);  \
  } while (0)
#define SATA_DECODE_GROUPED_G(TT, NTH)                  \
  do {                                                  \
    if (plan.G == 2) SATA_DECODE_GROUPED(TT, NTH, 2);   \
    else if (plan.G == 4) SATA_DECODE_GROUPED(TT, NTH, 4); \
    else SATA_DECODE_GROUPED(TT, NTH, 8);               \
  } while (0)
  if (plan.nth == 256) {
    if (bf16) SATA_DECODE_GROUPED_G(bf16_t, 256); else SATA_DECODE_GROUPED_G(float, 256);
  } else {
    if (bf16) SATA_DECODE_GROUPED_G(bf16_t, 1024); else SATA_DECODE_GROUPED_G(float, 1024);
  }
#undef SATA_DECODE_GROUPED_G
#undef SATA_DECODE_GROUPED
  return hipGetLastError();
}

}  // namespace sata
