// Matrix-core causal prefill for bfloat16 inputs and any (d_k, d_v <= 64, P):
// the state contractions of the chunked scan (App. A2),
//     O_c = phi(Q_c) S_{c-1},      S_c = S_{c-1} + phi(K_c)^T [V_c | 1],
// on v_mfma_f32_16x16x32_bf16 with the state in float32 accumulator registers
// for the whole sequence, every feature generated directly from its monomial.
//
// Work split.  A workgroup (8 or 4 waves) owns a contiguous range of features of
// one head ("slice") and all d_v + 1 columns (padded to NCT tiles of 16); each
// wave owns FT tiles of 16 features of it.  Per 64-token chunk a wave walks its
// features in blocks of 32 (two tiles):
//   * generate phi(q_t) and phi(k_t) of the block for the chunk's 64 tokens,
//     one token per lane (each feature is a weight times a product of
//     coordinates; consecutive features that differ in their last index only
//     reuse the product of the others);
//   * read out: O[token tile][column tile] += Phi_Q(16 x 32) * bf16(S block);
//   * update:   S tile += Phi_K^T(16 x 32 tokens) * [V | 1](32 x 16).
// The readout uses the state before the chunk's update, so the inter-chunk
// term is exactly phi(Q_c) S_{c-1}.  The waves' partial readouts are added in
// wave order through LDS and the slice's partial row written per token; the
// float32 prefill's finalize kernel adds the slices' partials in slice order,
// adds the intra-chunk term and divides.
//
// Operand layouts (16 x 16 x 32 bf16): A lane l holds row l % 16 and K entries
// 8 (l / 16) .. +7; B lane l holds column l % 16 and the same K entries; the
// result lane l holds column l % 16, rows 4 (l / 16) .. +3.  A state tile
// (16 features x 16 columns) is an update result; two of them feed the readout
// as B with the K order "features 4h..4h+3 of the first tile, then of the
// second" for lane group h = l / 16, so Phi_Q rows are stored in that order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>
#include <utility>

#include "device_common.hpp"
#include "kernels.hpp"
#include "prefill_feat.hpp"

namespace sata {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr int kCh = 64;        // tokens per chunk
constexpr int kQS = 40;        // bf16 per token row of a wave's Phi_Q block (32 + 8 pad)
constexpr int kKS = 72;        // bf16 per feature row of a wave's Phi_K^T block (64 + 8 pad)
constexpr int kVS = 72;        // bf16 per column row of V^T
constexpr int kWaveLds = kCh * kQS * 2 + 32 * kKS * 2;  // bytes of one wave's feature blocks

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ u16 bf16_bits(float x) {
  const __bf16 b = (__bf16)x;
  return __builtin_bit_cast(u16, b);
}

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ void lds_fence() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// f(integral_constant<int, I>) for I = 0 .. N-1, unrolled, so that register
// arrays indexed by I stay in registers.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Row stride of the float32 coordinates: odd (lanes = tokens hit distinct
// banks) with a column d that holds 1 (degree-0 features and padding read it).
__host__ __device__ constexpr int x_stride(int d) { return (d + 1) | 1; }
constexpr int kXMax = 65;  // x_stride(64): the key rows start at a fixed offset

// LDS map (bytes): region A = x~ of the chunk's queries and keys (float32
// [64][XS] each, 64 * kXMax floats apart) and V^T (bf16 [NCT*16][kVS]); the cross-wave reduction
// buffer (float32 [NW][16][NCT*16]) reuses region A after the generation;
// then the waves' feature blocks.
struct FeatLds {
  int xs, nct, nw, ft;
  __host__ __device__ int region_a() const {
    const int x = 2 * kCh * kXMax * 4 + nct * 16 * kVS * 2;
    const int r = nw * 16 * nct * 16 * 4;
    return ((x > r ? x : r) + 15) & ~15;
  }
  __host__ __device__ int bytes() const { return region_a() + nw * kWaveLds; }
};

// NW waves per workgroup, FT tiles of 16 features per wave, NCT column tiles.
template <int NCT, int FT, int NW>
__global__ void __launch_bounds__(NW * 64, 1)
prefill_feat_main(const u16* __restrict__ q, const u16* __restrict__ k, const u16* __restrict__ v,
                  const uint64_t* __restrict__ packed, const uint32_t* __restrict__ gen, int64_t D,
                  float* __restrict__ S_state, float* __restrict__ part, int BH, int n, int dk, int dv, int seg0,
                  int seg_len, int first_seg, int qg) {
  static_assert(FT % 2 == 0, "feature tiles come in blocks of two");
  static_assert(NW * FT * 16 <= kTablePad, "a slice may end past the last feature by less than the table's padding");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int E = dv + 1;
  const int XS = x_stride(dk);
  const FeatLds L{XS, NCT, NW, FT};
  char* const ra = smem;
  float* const xq = (float*)ra;
  float* const xk = xq + kCh * kXMax;
  u16* const vt = (u16*)(xk + kCh * XS);
  float* const red = (float*)ra;  // after the generation of a chunk
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l15 = lane & 15;
  const int h4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  u16* const phq = (u16*)(ra + L.region_a() + wave * kWaveLds);  // [64][kQS]
  u16* const phk = phq + kCh * kQS;                                 // [32][kKS]
  const int slice = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int fslice = slice * NW * FT * 16;   // (features fit 32 bits: D <= 2^26)
  const int Di = (int)D;
  const int fw0 = fslice + wave * FT * 16;  // this wave's first feature
  // the state tiles: S[t][j] holds features fw0 + 16 t + 4 h4 + r, column 16 j + l15
  f32x4 S[FT][NCT];
#pragma unroll
  for (int t = 0; t < FT; ++t)
#pragma unroll
    for (int j = 0; j < NCT; ++j) {
      f32x4 s = {0.f, 0.f, 0.f, 0.f};
      if (!first_seg) {
        const int c = 16 * j + l15;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int f = fw0 + 16 * t + 4 * h4 + r;
          if (f < Di && c < E) s[r] = S_state[(bh * D + f) * E + c];
        }
      }
      S[t][j] = s;
    }

  const u16* const qh = q + bh * (int64_t)qg * n * dk;
  const u16* const kh = k + bh * (int64_t)n * dk;
  const u16* const vh = v + bh * (int64_t)n * dv;
  const int seg_end = min(n, seg0 + seg_len);
  // The next chunk's q, k and v are fetched into registers (16-byte vectors of
  // eight bf16 of one row) while the current chunk is processed, when every
  // row of the head starts 16-byte aligned; otherwise element by element.
  constexpr int kVec = kCh * 64 / 8 / (NW * 64);  // vectors per thread and tensor at d = 64
  const bool vec = dk % 8 == 0 && dv % 8 == 0 && (((uintptr_t)qh | (uintptr_t)kh | (uintptr_t)vh) & 15) == 0;
  uint4 rq[kVec], rk[kVec], rv[kVec];
  auto fetch = [&](int c0) {
    const int cn = min(kCh, n - c0);
#pragma unroll
    for (int i = 0; i < kVec; ++i) {
      const int idx = tid + i * NW * 64;
      const uint4 z = {0u, 0u, 0u, 0u};
      rq[i] = z;
      rk[i] = z;
      rv[i] = z;
      if (idx < cn * dk / 8) {
        rq[i] = *(const uint4*)(qh + (int64_t)c0 * dk + 8 * idx);
        rk[i] = *(const uint4*)(kh + (int64_t)c0 * dk + 8 * idx);
      }
      if (idx < cn * dv / 8) rv[i] = *(const uint4*)(vh + (int64_t)c0 * dv + 8 * idx);
    }
  };
  if (vec) fetch(seg0);
  for (int t0 = seg0; t0 < seg_end; t0 += kCh) {
    const int cn = min(kCh, n - t0);
    __syncthreads();  // the previous chunk's reduction has read region A
    if (vec) {
      // rows past the sequence arrive as zeros, so their features are finite
      // and their V^T columns (normaliser included) are zero
#pragma unroll
      for (int i = 0; i < kVec; ++i) {
        const int idx = tid + i * NW * 64;
        if (idx < kCh * dk / 8) {
          const int t = idx / (dk / 8);
          const int c = 8 * (idx - t * (dk / 8));
          const uint32_t w[4] = {rq[i].x, rq[i].y, rq[i].z, rq[i].w};
          const uint32_t u[4] = {rk[i].x, rk[i].y, rk[i].z, rk[i].w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            xq[t * XS + c + 2 * j] = __uint_as_float(w[j] << 16);
            xq[t * XS + c + 2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
            xk[t * XS + c + 2 * j] = __uint_as_float(u[j] << 16);
            xk[t * XS + c + 2 * j + 1] = __uint_as_float(u[j] & 0xffff0000u);
          }
        }
        if (idx < kCh * dv / 8) {
          const int t = idx / (dv / 8);
          const int c = 8 * (idx - t * (dv / 8));
          const uint32_t w[4] = {rv[i].x, rv[i].y, rv[i].z, rv[i].w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            vt[(c + 2 * j) * kVS + t] = (u16)(w[j] & 0xffff);
            vt[(c + 2 * j + 1) * kVS + t] = (u16)(w[j] >> 16);
          }
        }
      }
      for (int t = tid; t < kCh; t += NW * 64) {
        xq[t * XS + dk] = 1.f;
        xk[t * XS + dk] = 1.f;
      }
      for (int i = tid; i < (NCT * 16 - dv) * kCh; i += NW * 64) {
        const int c = dv + i / kCh;
        const int t = i - (c - dv) * kCh;
        vt[c * kVS + t] = (c == dv && t < cn) ? (u16)0x3f80 : (u16)0;
      }
      if (t0 + kCh < seg_end) fetch(t0 + kCh);
    } else {
      for (int i = tid; i < kCh * dk; i += NW * 64) {
        const int t = i / dk;
        const int c = i - t * dk;
        float a = 0.f, b = 0.f;
        if (t < cn) {
          a = __uint_as_float((uint32_t)qh[(int64_t)(t0 + t) * dk + c] << 16);
          b = __uint_as_float((uint32_t)kh[(int64_t)(t0 + t) * dk + c] << 16);
        }
        xq[t * XS + c] = a;
        xk[t * XS + c] = b;
      }
      for (int t = tid; t < kCh; t += NW * 64) {
        xq[t * XS + dk] = 1.f;
        xk[t * XS + dk] = 1.f;
      }
      // V^T with the constant-1 normaliser column; tokens past the sequence and
      // padding columns are zero, so they add nothing to the state
      for (int i = tid; i < NCT * 16 * kCh; i += NW * 64) {
        const int c = i / kCh;
        const int t = i - c * kCh;
        u16 b = 0;
        if (t < cn) b = (c < dv) ? vh[(int64_t)(t0 + t) * dv + c] : (c == dv ? (u16)0x3f80 : (u16)0);
        vt[c * kVS + t] = b;
      }
    }
    __syncthreads();
    f32x4 O[4][NCT];
#pragma unroll
    for (int m = 0; m < 4; ++m)
#pragma unroll
      for (int j = 0; j < NCT; ++j) O[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    static_for<FT / 2>([&](auto sbc) {
      constexpr int SB = decltype(sbc)::value;
      const int fb0 = fw0 + 32 * SB;
      asm volatile("" ::: "memory");  // keep each block's table reads inside the block
      if (fb0 < Di) {  // (wave-uniform)
      // ---- generation: lane = token; features fb0 .. fb0 + 31 in groups of
      // eight.  A group's program words (x offset of the last index, flag,
      // weight) are wave-uniform scalar loads; its last-index coordinates are
      // read from LDS together; only a flagged feature (a new product of the
      // other indices: rare, features run through the last index in order)
      // reads its indices and waits on further coordinate reads.
      lds_fence();  // the previous block's operand reads have completed
      {
        const char* const xqt = (const char*)(xq + lane * XS);
        const uint2* const gb = (const uint2*)gen + fb0;
        float pq = 1.f, pk = 1.f;
        for (int g = 0; g < 4; ++g) {
          asm volatile("" ::: "memory");
          uint2 pw[8];
          float xa[8], xb[8];
#pragma unroll
          for (int r = 0; r < 8; ++r) pw[r] = gb[8 * g + r];
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            const uint32_t off = pw[r].x & 0x7fffffffu;
            xa[r] = *(const float*)(xqt + off);
            xb[r] = *(const float*)(xqt + off + kCh * kXMax * 4);
          }
          float vq[8], vk[8];
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            if (pw[r].x >> 31) {
              const uint64_t e = packed[fb0 + 8 * g + r];
              const int p = (int)(e >> 56);
              pq = 1.f;
              pk = 1.f;
              for (int j = 0; j < p - 1; ++j) {
                const int ix = (int)((e >> (8 * j)) & 0xff);
                pq *= xq[lane * XS + ix];
                pk *= xk[lane * XS + ix];
              }
            }
            const float w = __uint_as_float(pw[r].y);
            vq[r] = (pq * w) * xa[r];
            vk[r] = (pk * w) * xb[r];
            phk[(8 * g + r) * kKS + lane] = bf16_bits(vk[r]);  // Phi_K^T row, column = token
          }
          // Phi_Q: feature 8 g + r = 16 T + 4 hh + r' sits in K slot 8 hh + 4 T + r'
          const int T = g >> 1, hh = 2 * (g & 1);
          uint2 w2;
          w2.x = pack2(vq[0], vq[1]);
          w2.y = pack2(vq[2], vq[3]);
          *(uint2*)(phq + lane * kQS + 8 * hh + 4 * T) = w2;
          w2.x = pack2(vq[4], vq[5]);
          w2.y = pack2(vq[6], vq[7]);
          *(uint2*)(phq + lane * kQS + 8 * (hh + 1) + 4 * T) = w2;
        }
      }
      lds_fence();
      // ---- readout of the block against the state before this chunk's update
      bf16x8 bs[NCT];
#pragma unroll
      for (int j = 0; j < NCT; ++j) {
        uint4 w4;
        w4.x = pack2(S[2 * SB][j][0], S[2 * SB][j][1]);
        w4.y = pack2(S[2 * SB][j][2], S[2 * SB][j][3]);
        w4.z = pack2(S[2 * SB + 1][j][0], S[2 * SB + 1][j][1]);
        w4.w = pack2(S[2 * SB + 1][j][2], S[2 * SB + 1][j][3]);
        bs[j] = __builtin_bit_cast(bf16x8, w4);
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const bf16x8 a = *(const bf16x8*)(phq + (16 * m + l15) * kQS + 8 * h4);
#pragma unroll
        for (int j = 0; j < NCT; ++j) O[m][j] = mfma(a, bs[j], O[m][j]);
      }
      // ---- update: S tile += Phi_K^T [V | 1] (the V^T operands are read from
      // LDS per block rather than held, to leave registers to the state)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16x8 a0 = *(const bf16x8*)(phk + l15 * kKS + 32 * s + 8 * h4);
        const bf16x8 a1 = *(const bf16x8*)(phk + (16 + l15) * kKS + 32 * s + 8 * h4);
#pragma unroll
        for (int j = 0; j < NCT; ++j) {
          const bf16x8 b = *(const bf16x8*)(vt + (16 * j + l15) * kVS + 32 * s + 8 * h4);
          S[2 * SB][j] = mfma(a0, b, S[2 * SB][j]);
          S[2 * SB + 1][j] = mfma(a1, b, S[2 * SB + 1][j]);
        }
      }
      }
    });

    // ---- the waves' partial readouts, added in wave order, one token tile at a time
    float* const pout = part + (((int64_t)slice * BH + bh) * seg_len + (t0 - seg0)) * E;
    constexpr int RC = NCT * 16;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      __syncthreads();  // region A is free (generation done / previous tile read)
#pragma unroll
      for (int j = 0; j < NCT; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[(wave * 16 + 4 * h4 + r) * RC + 16 * j + l15] = O[m][j][r];
      __syncthreads();
      for (int i = tid; i < 16 * E; i += NW * 64) {
        const int rr = i / E;
        const int c = i - rr * E;
        float a = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) a += red[(w * 16 + rr) * RC + c];
        const int t = 16 * m + rr;
        if (t < cn) pout[(int64_t)t * E + c] = a;
      }
    }
  }

  // ---- the state after the segment, canonical layout
#pragma unroll
  for (int t = 0; t < FT; ++t)
#pragma unroll
    for (int j = 0; j < NCT; ++j) {
      const int c = 16 * j + l15;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int f = fw0 + 16 * t + 4 * h4 + r;
        if (f < Di && c < E) S_state[(bh * D + f) * E + c] = S[t][j][r];
      }
    }
}

// Slice 0's partial readout of every (head, token, column) of a segment
// becomes the sum of all slices' partials, added in slice order.  One thread
// per element: consecutive threads read consecutive floats of each slice.
__global__ void __launch_bounds__(256) reduce_slices(float* __restrict__ part, int BH, int seg_len, int seg_tokens,
                                                     int E, int nslices) {
  const int64_t per_bh = (int64_t)seg_tokens * E;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per_bh * BH) return;
  const int64_t bh = i / per_bh;
  const int64_t off = bh * seg_len * E + (i - bh * per_bh);
  const int64_t stride = (int64_t)BH * seg_len * E;
  float a = 0.f;
  for (int sl = 0; sl < nslices; ++sl) a += part[sl * stride + off];
  part[off] = a;
}

// Tiles per wave and waves per workgroup for NCT column tiles: the state,
// the readout sums (4 x NCT tiles) and the value operands fit the registers
// of two waves per SIMD up to NCT = 3, of one wave per SIMD beyond.
constexpr int ft_for(int nct) { return nct <= 1 ? 28 : nct == 2 ? 16 : nct == 3 ? 8 : nct == 4 ? 6 : 4; }
constexpr int nw_for(int nct) { return 8; }

template <int NCT>
hipError_t launch_main(const u16* q, const u16* k, const u16* v, const DevTable& t, float* S_state, float* part,
                       int BH, int n, int dk, int dv, int seg0, int seg_len, bool first, int nslices, int qg,
                       hipStream_t s) {
  constexpr int FT = ft_for(NCT), NW = nw_for(NCT);
  const FeatLds L{x_stride(dk), NCT, NW, FT};
  auto kern = prefill_feat_main<NCT, FT, NW>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, L.bytes());
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)nslices, (unsigned)BH), dim3(NW * 64), (size_t)L.bytes(), s, q, k, v,
                     t.packed, t.gen, t.D, S_state, part, BH, n, dk, dv, seg0, seg_len, first ? 1 : 0, qg);
  return hipGetLastError();
}

}  // namespace

bool plan_prefill_feat(int64_t D, int BH, int n, int dk, int dv, int P, int chunk, size_t max_ws_bytes,
                       FeatPrefillPlan* plan) {
  if (chunk != kCh || P < 2 || dk > 64 || dv > 64 || n < 1) return false;
  const int E = dv + 1;
  const int nct = (E + 15) / 16;
  const int fslice = nw_for(nct) * ft_for(nct) * 16;
  plan->nct = nct;
  plan->nslices = (int)((D + fslice - 1) / fslice);
  const FeatLds L{x_stride(dk), nct, nw_for(nct), ft_for(nct)};
  plan->lds_main = (size_t)L.bytes();
  if (plan->lds_main > 160 * 1024) return false;
  const size_t per_token = sizeof(float) * (size_t)plan->nslices * BH * E;
  int64_t seg = (int64_t)(max_ws_bytes / per_token) / kCh * kCh;
  if (seg < kCh) seg = kCh;
  const int64_t n_round = ((int64_t)n + kCh - 1) / kCh * kCh;
  plan->seg_len = (int)std::min<int64_t>(seg, n_round);
  plan->partial_bytes = per_token * (size_t)plan->seg_len;
  return true;
}

hipError_t launch_prefill_feat(const void* q, const void* k, const void* v, void* y, int BH, int n, int dk, int dv,
                               int P, const DevTable& t, const FeatPrefillPlan& plan, float* S_state, float* partial,
                               hipStream_t s, int qg) {
  const u16* qq = (const u16*)q;
  const u16* kk = (const u16*)k;
  const u16* vv = (const u16*)v;
  for (int seg0 = 0; seg0 < n; seg0 += plan.seg_len) {
    const bool first = seg0 == 0;
    hipError_t e;
    switch (plan.nct) {
      case 1: e = launch_main<1>(qq, kk, vv, t, S_state, partial, BH, n, dk, dv, seg0, plan.seg_len, first, plan.nslices, qg, s); break;
      case 2: e = launch_main<2>(qq, kk, vv, t, S_state, partial, BH, n, dk, dv, seg0, plan.seg_len, first, plan.nslices, qg, s); break;
      case 3: e = launch_main<3>(qq, kk, vv, t, S_state, partial, BH, n, dk, dv, seg0, plan.seg_len, first, plan.nslices, qg, s); break;
      case 4: e = launch_main<4>(qq, kk, vv, t, S_state, partial, BH, n, dk, dv, seg0, plan.seg_len, first, plan.nslices, qg, s); break;
      default: e = launch_main<5>(qq, kk, vv, t, S_state, partial, BH, n, dk, dv, seg0, plan.seg_len, first, plan.nslices, qg, s); break;
    }
    if (e != hipSuccess) return e;
    int ns = plan.nslices;
    if (ns > 1) {
      const int seg_tokens = std::min(plan.seg_len, n - seg0);
      const int64_t count = (int64_t)BH * seg_tokens * (dv + 1);
      hipLaunchKernelGGL(reduce_slices, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, partial, BH,
                         plan.seg_len, seg_tokens, dv + 1, ns);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      ns = 1;
    }
    e = launch_prefill_generic_finalize(q, k, v, y, true, BH, n, dk, dv, P, kCh, ns, seg0, plan.seg_len, partial, s,
                                        qg);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace sata
