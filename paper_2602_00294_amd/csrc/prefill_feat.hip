// Matrix-core causal prefill for any (d_k, d_v <= 64, P >= 2) with 64-token
// chunks: the state contractions of the chunked scan (App. A2),
//     O_c = phi(Q_c) S_{c-1},      S_c = S_{c-1} + phi(K_c)^T [V_c | 1],
// on v_mfma_f32_16x16x32_bf16 with the state in float32 accumulator registers
// for the whole sequence, every feature generated directly from its monomial.
//
// Operands.  bfloat16 inputs: each operand is rounded to bfloat16 once.
// float32 inputs ("split" operands): each operand a is carried as a pair of
// bfloat16 numbers hi = bf16(a), lo = bf16(a - hi), which holds a to about
// 2^-16 of its size, and each product as hi*hi + hi*lo + lo*hi (the dropped
// lo*lo is of the same order), three matrix-core products in place of one.
//
// Work split.  A workgroup of 8 waves owns a contiguous range of features of
// one head ("slice") and all d_v + 1 columns (padded to NCT tiles of 16); each
// wave owns FT tiles of 16 features of it.  Per 64-token chunk a wave walks its
// features in blocks of 32 (two tiles):
//   * generate phi(q_t) and phi(k_t) of the block for the chunk's 64 tokens,
//     one token per lane (each feature is a weight times a product of
//     coordinates; consecutive features that differ in their last index only
//     reuse the product of the others);
//   * read out: O[token tile][column tile] += Phi_Q(16 x 32) * S block;
//   * update:   S tile += Phi_K^T(16 x 32 tokens) * [V | 1](32 x 16).
// With split operands the query features are generated, read out, and their
// LDS block then reused for the key features (so the two halves of a pair
// fit).  The readout uses the state before the chunk's update, so the
// inter-chunk term is exactly phi(Q_c) S_{c-1}.  The waves' partial readouts
// are added in wave order through LDS and the slice's partial row written per
// token; a second kernel adds the slices' partials in slice order and a
// finalize kernel (on the float32 matrix-core products) adds the intra-chunk
// term and divides.
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

namespace sata {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

constexpr int kCh = 64;        // tokens per chunk
constexpr int kNW = 8;         // waves per workgroup
constexpr int kQS = 40;        // bf16 per token row of a wave's Phi_Q block (32 + 8 pad)
constexpr int kKS = 72;        // bf16 per feature row of a wave's Phi_K^T block (64 + 8 pad)
constexpr int kVS = 72;        // bf16 per column row of V^T
constexpr int kRS = 20;        // floats per (wave, column) row of the reduction buffer (16 tokens + 4 pad)
constexpr int kQPlane = kCh * kQS * 2;  // bytes of one Phi_Q plane
constexpr int kKPlane = 32 * kKS * 2;   // bytes of one Phi_K^T plane

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

// The part of x that bf16(x) leaves out.
__device__ __forceinline__ float bf16_rest(float x) { return x - (float)(__bf16)x; }

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
// [64][XS] each, 64 * kXMax floats apart) and V^T (PL planes of bf16
// [NCT*16][kVS]), then the waves' feature blocks (Phi_Q and Phi_K^T; with
// split operands one hi and one lo plane, shared by the two).  After a chunk's
// matrix work the reduction buffer (float32 [NW][NCT*16][kRS] per token tile,
// TP tiles at a time) reuses all of it.
template <int NCT, bool X3>
struct FeatLds {
  static constexpr int kPl = X3 ? 2 : 1;
  static constexpr int kWave = X3 ? 2 * kQPlane : kQPlane + kKPlane;
  static constexpr int kRegionA = (2 * kCh * kXMax * 4 + kPl * NCT * 16 * kVS * 2 + 15) & ~15;
  static constexpr int kRedTile = kNW * NCT * 16 * kRS * 4;
  static constexpr int kAll = kRegionA + kNW * kWave;
  static constexpr int kTP = 4 * kRedTile <= kAll ? 4 : 2 * kRedTile <= kAll ? 2 : 1;  // reduction tiles per pass
  static constexpr int kBytes = kAll > kRedTile ? kAll : kRedTile;
};

// Where the parts of a launch (blockIdx.z) start and leave their states, each
// [BH][D][d_v+1] float32.  Part 0 starts from in0, part g >= 1 from
// in + (g - 1) * stride (null: from zero); the last part stores to last, the
// others (and the last, when last is null) to out + g * stride (null: not
// stored).
struct FeatStates {
  const float* in0;
  const float* in;
  float* last;
  float* out;
};

// FT tiles of 16 features per wave, NCT column tiles; X3: split operands;
// T: the input element type (bf16 bits or float); RO: with the readout (else
// the parts' state sums alone).
template <int NCT, int FT, bool X3, typename T, bool RO>
__global__ void __launch_bounds__(kNW * 64, 1)
prefill_feat_main(const void* __restrict__ q_, const void* __restrict__ k_, const void* __restrict__ v_,
                  const uint64_t* __restrict__ packed, const uint32_t* __restrict__ gen, int64_t D,
                  FeatStates st, float* __restrict__ part, int BH, int n, int dk, int dv, int seg0, int seg_len,
                  int part_len, int qg) {
  static_assert(FT % 2 == 0, "feature tiles come in blocks of two");
  static_assert(kNW * FT * 16 <= kTablePad, "a slice may end past the last feature by less than the table's padding");
  using L = FeatLds<NCT, X3>;
  constexpr int kEV = 16 / sizeof(T);  // elements per 16-byte vector
  constexpr int kVPlane = NCT * 16 * kVS;  // bf16 per V^T plane
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int E = dv + 1;
  const int XS = x_stride(dk);
  float* const xq = (float*)smem;
  float* const xk = xq + kCh * kXMax;
  u16* const vt = (u16*)(xk + kCh * kXMax);
  float* const red = (float*)smem;  // after the matrix work of a chunk
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l15 = lane & 15;
  const int h4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  char* const wl = smem + L::kRegionA + wave * L::kWave;
  u16* const phq = (u16*)wl;                                  // [64][kQS] (hi plane; lo plane next)
  u16* const phk = (u16*)(X3 ? wl : wl + kQPlane);            // [32][kKS] (hi plane; lo plane next)
  constexpr int kQLo = X3 ? kQPlane / 2 : 0;                  // u16 from a hi plane to its lo plane
  constexpr int kKLo = X3 ? kQPlane / 2 : 0;
  const int slice = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int fslice = slice * kNW * FT * 16;  // (features fit 32 bits: D <= 2^26)
  const int Di = (int)D;
  const int fw0 = fslice + wave * FT * 16;  // this wave's first feature
  // With split operands the upper half of the waves issue first: of the two
  // waves of a SIMD, the favoured one runs ahead, so that one generates while
  // the other multiplies (about 5% on the float32 sweep; no gain with bf16
  // operands, whose generation is shorter).
  if (X3 && wave >= kNW / 2) __builtin_amdgcn_s_setprio(1);
  // part blockIdx.z of the segment: its tokens, and where its state starts and ends
  const int pz = blockIdx.z;
  const int64_t sstride = (int64_t)BH * D * E;
  const float* const s_in = pz == 0 ? st.in0 : (st.in ? st.in + (pz - 1) * sstride : nullptr);
  float* const s_out = (pz == (int)gridDim.z - 1 && st.last) ? st.last : (st.out ? st.out + pz * sstride : nullptr);
  const int t_begin = seg0 + pz * part_len;

  // the state tiles: S[t][j] holds features fw0 + 16 t + 4 h4 + r, column 16 j + l15
  f32x4 S[FT][NCT];
#pragma unroll
  for (int t = 0; t < FT; ++t)
#pragma unroll
    for (int j = 0; j < NCT; ++j) {
      f32x4 s = {0.f, 0.f, 0.f, 0.f};
      if (s_in) {
        const int c = 16 * j + l15;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int f = fw0 + 16 * t + 4 * h4 + r;
          if (f < Di && c < E) s[r] = s_in[(bh * D + f) * E + c];
        }
      }
      S[t][j] = s;
    }

  const T* const qh = (const T*)q_ + bh * (int64_t)qg * n * dk;
  const T* const kh = (const T*)k_ + bh * (int64_t)n * dk;
  const T* const vh = (const T*)v_ + bh * (int64_t)n * dv;
  const int seg_end = min(min(n, seg0 + seg_len), t_begin + part_len);
  // The next chunk's q, k and v are fetched into registers (16-byte vectors of
  // one row) while the current chunk is processed, when every row of the head
  // starts 16-byte aligned; otherwise element by element.
  constexpr int kVec = kCh * 64 / kEV / (kNW * 64);  // vectors per thread and tensor at d = 64
  const bool vec = dk % kEV == 0 && dv % kEV == 0 && (((uintptr_t)qh | (uintptr_t)kh | (uintptr_t)vh) & 15) == 0;
  uint4 rq[kVec], rk[kVec], rv[kVec];
  auto fetch = [&](int c0) {
    const int cn = min(kCh, n - c0);
#pragma unroll
    for (int i = 0; i < kVec; ++i) {
      const int idx = tid + i * kNW * 64;
      const uint4 z = {0u, 0u, 0u, 0u};
      rq[i] = z;
      rk[i] = z;
      rv[i] = z;
      if (idx < cn * dk / kEV) {
        rq[i] = *(const uint4*)(qh + (int64_t)c0 * dk + kEV * idx);
        rk[i] = *(const uint4*)(kh + (int64_t)c0 * dk + kEV * idx);
      }
      if (idx < cn * dv / kEV) rv[i] = *(const uint4*)(vh + (int64_t)c0 * dv + kEV * idx);
    }
  };
  // element j of a 16-byte vector (j a constant after unrolling)
  constexpr bool kF32In = std::is_same_v<T, float>;
  auto elem = [](const uint4& w, int j) -> T {
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
    if constexpr (kF32In) return __uint_as_float(u[j]);
    else return (u16)(j & 1 ? u[j >> 1] >> 16 : u[j >> 1] & 0xffffu);
  };
  auto to_f32 = [](T x) -> float {
    if constexpr (kF32In) return x;
    else return __uint_as_float((uint32_t)x << 16);
  };
  auto elem_f32 = [&](const uint4& w, int j) -> float { return to_f32(elem(w, j)); };
  // V^T entry (column c, token t) of value x: both planes with split operands
  auto put_v = [&](int c, int t, T x) {
    if constexpr (X3) {
      const float f = to_f32(x);
      vt[c * kVS + t] = bf16_bits(f);
      vt[kVPlane + c * kVS + t] = bf16_bits(bf16_rest(f));
    } else if constexpr (kF32In) {
      vt[c * kVS + t] = bf16_bits(x);
    } else {
      vt[c * kVS + t] = x;
    }
  };
  if (vec) fetch(t_begin);
  for (int t0 = t_begin; t0 < seg_end; t0 += kCh) {
    const int cn = min(kCh, n - t0);
    __syncthreads();  // the previous chunk's reduction has read its buffer
    if (vec) {
      // rows past the sequence arrive as zeros, so their features are finite
      // and their V^T columns (normaliser included) are zero
#pragma unroll
      for (int i = 0; i < kVec; ++i) {
        const int idx = tid + i * kNW * 64;
        if (idx < kCh * dk / kEV) {
          const int t = idx / (dk / kEV);
          const int c = kEV * (idx - t * (dk / kEV));
#pragma unroll
          for (int j = 0; j < kEV; ++j) {
            xq[t * XS + c + j] = elem_f32(rq[i], j);
            xk[t * XS + c + j] = elem_f32(rk[i], j);
          }
        }
        if (idx < kCh * dv / kEV) {
          const int t = idx / (dv / kEV);
          const int c = kEV * (idx - t * (dv / kEV));
#pragma unroll
          for (int j = 0; j < kEV; ++j) put_v(c + j, t, elem(rv[i], j));
        }
      }
      if (t0 + kCh < seg_end) fetch(t0 + kCh);
    } else {
      for (int i = tid; i < kCh * dk; i += kNW * 64) {
        const int t = i / dk;
        const int c = i - t * dk;
        float a = 0.f, b = 0.f;
        if (t < cn) {
          a = to_f32(qh[(int64_t)(t0 + t) * dk + c]);
          b = to_f32(kh[(int64_t)(t0 + t) * dk + c]);
        }
        xq[t * XS + c] = a;
        xk[t * XS + c] = b;
      }
      for (int i = tid; i < dv * kCh; i += kNW * 64) {
        const int c = i / kCh;
        const int t = i - c * kCh;
        put_v(c, t, t < cn ? vh[(int64_t)(t0 + t) * dv + c] : (T)0);
      }
    }
    for (int t = tid; t < kCh; t += kNW * 64) {
      xq[t * XS + dk] = 1.f;
      xk[t * XS + dk] = 1.f;
    }
    // the constant-1 normaliser column (tokens of the sequence only) and the
    // zero padding columns
    for (int i = tid; i < (NCT * 16 - dv) * kCh; i += kNW * 64) {
      const int c = dv + i / kCh;
      const int t = i - (c - dv) * kCh;
      vt[c * kVS + t] = (c == dv && t < cn) ? (u16)0x3f80 : (u16)0;
      if constexpr (X3) vt[kVPlane + c * kVS + t] = 0;
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
      asm volatile("" ::: "memory");  // keep each block's program reads inside the block
      if (fb0 < Di) {  // (wave-uniform)
        // ---- generation: lane = token; features fb0 .. fb0 + 31 in groups of
        // eight.  A group's program words (x offset of the last index, flag,
        // weight) are wave-uniform scalar loads; its last-index coordinates
        // are read from LDS together; only a flagged feature (a new product of
        // the other indices: rare, features run through the last index in
        // order) reads its indices and waits on further coordinate reads.
        // W = 0: query features only, 1: key features only, 2: both.
        auto generate = [&](auto wc) {
          constexpr int W = decltype(wc)::value;
          const char* const xqt = (const char*)(xq + lane * XS);
          const uint2* const gb = (const uint2*)gen + fb0;
          float pq = 1.f, pk = 1.f;
          for (int g = 0; g < 4; ++g) {
            asm volatile("" ::: "memory");
            uint2 pw[8];
            uint64_t pke[8];
            float xa[8], xb[8];
#pragma unroll
            for (int r = 0; r < 8; ++r) pw[r] = gb[8 * g + r];
            // with split operands (the float32 path, whose high-P shapes have
            // many features of degree 4 and up) the group's packed entries,
            // which supply those features' further indices, are loaded with
            // its program words rather than when a feature needs them
            if constexpr (X3) {
#pragma unroll
              for (int r = 0; r < 8; ++r) pke[r] = packed[fb0 + 8 * g + r];
            }
#pragma unroll
            for (int r = 0; r < 8; ++r) {
              const uint32_t off = pw[r].x & 0x3ffu;
              if (W != 1) xa[r] = *(const float*)(xqt + off);
              if (W != 0) xb[r] = *(const float*)(xqt + off + kCh * kXMax * 4);
            }
            float vq[8];
#pragma unroll
            for (int r = 0; r < 8; ++r) {
              if (pw[r].x >> 31) {
                // the product of every index but the last: the first two
                // come with the program word (the column held at 1 where the
                // feature has fewer), any further ones from the packed entry,
                // read two at a time
                const int a0 = (int)((pw[r].x >> 10) & 0xff), a1 = (int)((pw[r].x >> 18) & 0xff);
                if (W != 1) pq = xq[lane * XS + a0] * xq[lane * XS + a1];
                if (W != 0) pk = xk[lane * XS + a0] * xk[lane * XS + a1];
                if ((pw[r].x >> 30) & 1) {
                  uint64_t e;
                  if constexpr (X3) e = pke[r];
                  else e = packed[fb0 + 8 * g + r];
                  const int p = (int)(e >> 56);
                  auto idx = [&](int j) { return j < p - 1 ? (int)((e >> (8 * j)) & 0xff) : dk; };
                  for (int j = 2; j < p - 1; j += 2) {
                    const int i0 = idx(j), i1 = idx(j + 1);
                    if (W != 1) pq *= xq[lane * XS + i0] * xq[lane * XS + i1];
                    if (W != 0) pk *= xk[lane * XS + i0] * xk[lane * XS + i1];
                  }
                }
              }
              const float w = __uint_as_float(pw[r].y);
              if (W != 1) vq[r] = (pq * w) * xa[r];
              if (W != 0) {
                const float vk = (pk * w) * xb[r];
                phk[(8 * g + r) * kKS + lane] = bf16_bits(vk);  // Phi_K^T row, column = token
                if (X3) phk[kKLo + (8 * g + r) * kKS + lane] = bf16_bits(bf16_rest(vk));
              }
            }
            if (W != 1) {
              // Phi_Q: feature 8 g + r = 16 tt + 4 hh + r' sits in K slot 8 hh + 4 tt + r'
              const int tt = g >> 1, hh = 2 * (g & 1);
              u16* const row = phq + lane * kQS + 4 * tt;
              *(uint2*)(row + 8 * hh) = uint2{pack2(vq[0], vq[1]), pack2(vq[2], vq[3])};
              *(uint2*)(row + 8 * (hh + 1)) = uint2{pack2(vq[4], vq[5]), pack2(vq[6], vq[7])};
              if (X3) {
                *(uint2*)(row + kQLo + 8 * hh) = uint2{pack2(bf16_rest(vq[0]), bf16_rest(vq[1])),
                                                       pack2(bf16_rest(vq[2]), bf16_rest(vq[3]))};
                *(uint2*)(row + kQLo + 8 * (hh + 1)) = uint2{pack2(bf16_rest(vq[4]), bf16_rest(vq[5])),
                                                             pack2(bf16_rest(vq[6]), bf16_rest(vq[7]))};
              }
            }
          }
        };
        // ---- readout of the block against the state before this chunk's update
        auto readout = [&]() {
          bf16x8 bs[NCT], bl[NCT];
#pragma unroll
          for (int j = 0; j < NCT; ++j) {
            const f32x4 s0 = S[2 * SB][j], s1 = S[2 * SB + 1][j];
            bs[j] = __builtin_bit_cast(bf16x8, (uint4{pack2(s0[0], s0[1]), pack2(s0[2], s0[3]), pack2(s1[0], s1[1]),
                                                      pack2(s1[2], s1[3])}));
            if (X3)
              bl[j] = __builtin_bit_cast(
                  bf16x8, (uint4{pack2(bf16_rest(s0[0]), bf16_rest(s0[1])), pack2(bf16_rest(s0[2]), bf16_rest(s0[3])),
                                 pack2(bf16_rest(s1[0]), bf16_rest(s1[1])), pack2(bf16_rest(s1[2]), bf16_rest(s1[3]))}));
          }
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            const bf16x8 a = *(const bf16x8*)(phq + (16 * m + l15) * kQS + 8 * h4);
            if (X3) {
              const bf16x8 al = *(const bf16x8*)(phq + kQLo + (16 * m + l15) * kQS + 8 * h4);
#pragma unroll
              for (int j = 0; j < NCT; ++j) O[m][j] = mfma(al, bs[j], mfma(a, bl[j], mfma(a, bs[j], O[m][j])));
            } else {
#pragma unroll
              for (int j = 0; j < NCT; ++j) O[m][j] = mfma(a, bs[j], O[m][j]);
            }
          }
        };
        // ---- update: S tile += Phi_K^T [V | 1] (the V^T operands are read
        // from LDS per block rather than held, to leave registers to the state).
        // With split operands the chunk's 64 tokens are first summed from zero
        // and then added to the state, so that each entry takes one float32
        // rounding per chunk (as the float32 path does) rather than one per
        // 32-token product.
        auto update = [&]() {
          if constexpr (X3) {
#pragma unroll
            for (int j = 0; j < NCT; ++j) {
              f32x4 d0 = {0.f, 0.f, 0.f, 0.f}, d1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
              for (int s = 0; s < 2; ++s) {
                const bf16x8 a0 = *(const bf16x8*)(phk + l15 * kKS + 32 * s + 8 * h4);
                const bf16x8 a1 = *(const bf16x8*)(phk + (16 + l15) * kKS + 32 * s + 8 * h4);
                const bf16x8 a0l = *(const bf16x8*)(phk + kKLo + l15 * kKS + 32 * s + 8 * h4);
                const bf16x8 a1l = *(const bf16x8*)(phk + kKLo + (16 + l15) * kKS + 32 * s + 8 * h4);
                const bf16x8 b = *(const bf16x8*)(vt + (16 * j + l15) * kVS + 32 * s + 8 * h4);
                const bf16x8 bl = *(const bf16x8*)(vt + kVPlane + (16 * j + l15) * kVS + 32 * s + 8 * h4);
                d0 = mfma(a0l, b, mfma(a0, bl, mfma(a0, b, d0)));
                d1 = mfma(a1l, b, mfma(a1, bl, mfma(a1, b, d1)));
              }
              S[2 * SB][j] += d0;
              S[2 * SB + 1][j] += d1;
            }
          } else {
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
        };
        lds_fence();  // the previous block's operand reads have completed
        if constexpr (!RO) {  // the state sum alone
          generate(std::integral_constant<int, 1>{});
          lds_fence();
          update();
        } else if constexpr (X3) {
          generate(std::integral_constant<int, 0>{});
          lds_fence();
          readout();
          lds_fence();  // its operands are in registers: the block is free for the keys
          generate(std::integral_constant<int, 1>{});
          lds_fence();
          update();
        } else {
          generate(std::integral_constant<int, 2>{});
          lds_fence();
          readout();
          update();
        }
      }
    });

    if constexpr (!RO) continue;
    // ---- the waves' partial readouts, added in wave order, TP token tiles at
    // a time; a lane's four rows of a column are one 16-byte store
    float* const pout = part + (((int64_t)slice * BH + bh) * seg_len + (t0 - seg0)) * E;
    constexpr int RC = NCT * 16;
    constexpr int TP = L::kTP;
#pragma unroll
    for (int m0 = 0; m0 < 4; m0 += TP) {
      __syncthreads();  // the matrix work / the previous pass's sums are done
#pragma unroll
      for (int mm = 0; mm < TP; ++mm)
#pragma unroll
        for (int j = 0; j < NCT; ++j)
          *(f32x4*)(red + (((mm * kNW + wave) * RC + 16 * j + l15) * kRS + 4 * h4)) = O[m0 + mm][j];
      __syncthreads();
      for (int i = tid; i < TP * 4 * E; i += kNW * 64) {
        const int mq = i / E;  // token quad of the pass
        const int c = i - mq * E;
        const int mm = mq >> 2, tq = mq & 3;
        f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < kNW; ++w) a += *(const f32x4*)(red + (((mm * kNW + w) * RC + c) * kRS + 4 * tq));
        const int t = 16 * (m0 + mm) + 4 * tq;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (t + r < cn) pout[(int64_t)(t + r) * E + c] = a[r];
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
        if (f < Di && c < E && s_out) s_out[(bh * D + f) * E + c] = S[t][j][r];
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
  // eight loads in flight at a time; the sum still runs in slice order
  float a = 0.f;
  int sl = 0;
  for (; sl + 8 <= nslices; sl += 8) {
    float x[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) x[u] = part[(sl + u) * stride + off];
#pragma unroll
    for (int u = 0; u < 8; ++u) a += x[u];
  }
  for (; sl < nslices; ++sl) a += part[sl * stride + off];
  part[off] = a;
}

// ---- finalize: the intra-chunk term and the division (App. A2: within a
// chunk the causal attention weights are the truncated Taylor polynomial of
// q.k / sqrt(d_k) itself).  One workgroup of 4 waves per (chunk of 64 tokens,
// head); wave w owns query rows 16 w .. 16 w + 15.  Both products run on
// v_mfma_f32_16x16x4_f32 (float32 operands and accumulation):
//   W[t][t'] = f_P(q_t . k_t' / sqrt(d_k)) for t' <= t, else 0   (Q K^T tiles)
//   O = partial + W [V | 1],   y_t = O[t][0:d_v] / O[t][d_v].
// Operand layouts (16 x 16 x 4 f32): A lane l holds row l % 16, K entry l / 16;
// B lane l holds column l % 16, K row l / 16; the result lane l holds column
// l % 16, rows 4 (l / 16) .. +3.  Each wave reads and writes only its own rows
// of W and O, so no barrier separates the steps after the loads.
constexpr int kFinWS = 68;  // floats per row of W (64 + 4: the A reads hit distinct banks)
constexpr int kFinMaxNT = 5;  // column tiles of 16 covering d_v + 1 <= 65
__host__ __device__ constexpr int fin_xq(int dk) { return (dk + 7) / 8 * 8 + 4; }
__host__ __device__ constexpr int fin_ep(int dv) { return (dv + 1 + 15) / 16 * 16; }
__host__ __device__ constexpr int fin_vs(int dv) { return fin_ep(dv) | 16; }
inline size_t fin_lds_bytes(int dk, int dv) {
  return sizeof(float) * ((size_t)2 * kCh * fin_xq(dk) + (size_t)kCh * fin_vs(dv) + (size_t)kCh * kFinWS);
}

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// rows [0, 64) of a chunk (rows of `width` elements, contiguous in src, zero
// past row cn) into float32 LDS rows of `stride`; 16-byte loads where the
// rows allow them
template <typename T>
__device__ __forceinline__ void fin_load_rows(const T* __restrict__ src, int width, int cn, float* dst, int stride,
                                              bool vec) {
  constexpr int kEV = 16 / sizeof(T);
  if (vec) {
    const int per = width / kEV;
    for (int i = threadIdx.x; i < kCh * per; i += 256) {
      const int t = i / per, c = (i - t * per) * kEV;
      uint4 w = {0u, 0u, 0u, 0u};
      if (t < cn) w = *(const uint4*)(src + (int64_t)t * width + c);
      const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int j = 0; j < kEV; ++j) {
        float f;
        if constexpr (sizeof(T) == 4) f = __uint_as_float(u[j]);
        else f = __uint_as_float(j & 1 ? u[j >> 1] & 0xffff0000u : u[j >> 1] << 16);
        dst[t * stride + c + j] = f;
      }
    }
  } else {
    for (int i = threadIdx.x; i < kCh * width; i += 256) {
      const int t = i / width, c = i - t * width;
      dst[t * stride + c] = t < cn ? to_f32(src[(int64_t)t * width + c]) : 0.f;
    }
  }
}

template <typename T>
__global__ void __launch_bounds__(256) feat_finalize(const T* __restrict__ q, const T* __restrict__ k,
                                                     const T* __restrict__ v, const float* __restrict__ part,
                                                     T* __restrict__ y, int n, int dk, int dv, int P, int seg0,
                                                     int seg_len, int qg) {
  extern __shared__ __attribute__((aligned(16))) float flds[];
  const int E = dv + 1;
  const int XQ = fin_xq(dk), EP = fin_ep(dv), VS = fin_vs(dv), NT = EP / 16;
  float* const xq = flds;           // [64][XQ], zero past d_k and past the sequence
  float* const xk = xq + kCh * XQ;  // [64][XQ]
  float* const v1 = xk + kCh * XQ;  // [64][VS]: [V | 1], zero past E and past the sequence
  float* const W = v1 + kCh * VS;   // [64][kFinWS]
  const int64_t bh = blockIdx.y;
  const int t0 = seg0 + blockIdx.x * kCh;
  if (t0 >= n) return;
  const int cn = min(kCh, n - t0);
  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, l4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r0 = 16 * wave;  // this wave's rows
  const T* const qh = q + (bh * qg * n + t0) * (int64_t)dk;
  const T* const kh = k + (bh * n + t0) * (int64_t)dk;
  const T* const vh = v + (bh * n + t0) * (int64_t)dv;
  // the partial sums of this wave's results (rows r0 + 4 l4 + i, column
  // 16 jt + l16), fetched first so that they arrive during the rest
  const float* const pr = part + ((int64_t)bh * seg_len + (t0 - seg0)) * E;
  float pp[kFinMaxNT][4];
#pragma unroll
  for (int jt = 0; jt < kFinMaxNT; ++jt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = r0 + 4 * l4 + i, c = 16 * jt + l16;
      pp[jt][i] = (jt < NT && c < E && t < cn) ? pr[(int64_t)t * E + c] : 0.f;
    }
  constexpr int kEV = 16 / sizeof(T);
  const bool vq = dk % kEV == 0 && (((uintptr_t)qh | (uintptr_t)kh) & 15) == 0;
  const bool vv = dv % kEV == 0 && ((uintptr_t)vh & 15) == 0;
  fin_load_rows(qh, dk, cn, xq, XQ, vq);
  fin_load_rows(kh, dk, cn, xk, XQ, vq);
  fin_load_rows(vh, dv, cn, v1, VS, vv);
  const int dk4 = (dk + 3) & ~3;
  for (int i = tid; i < kCh * (dk4 - dk); i += 256) {  // zero K padding
    const int t = i / (dk4 - dk), c = dk + i - t * (dk4 - dk);
    xq[t * XQ + c] = 0.f;
    xk[t * XQ + c] = 0.f;
  }
  for (int i = tid; i < kCh * (EP - dv); i += 256) {  // the 1 column and zero padding
    const int t = i / (EP - dv), c = dv + i - t * (EP - dv);
    v1[t * VS + c] = (c == dv && t < cn) ? 1.f : 0.f;
  }
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)dk);
  for (int nt = 0; nt <= wave; ++nt) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int kk = 0; kk < dk4; kk += 4)
      acc = mfma4(xq[(r0 + l16) * XQ + kk + l4], xk[(16 * nt + l16) * XQ + kk + l4], acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = r0 + 4 * l4 + i, tp = 16 * nt + l16;
      W[t * kFinWS + tp] = tp <= t ? taylor_horner(acc[i] * scale, P) : 0.f;
    }
  }
  auto out_tile = [&](int jt) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int kk = 0; kk < r0 + 16; kk += 4)
      acc = mfma4(W[(r0 + l16) * kFinWS + kk + l4], v1[(kk + l4) * VS + 16 * jt + l16], acc);
    return acc;
  };
  // the normaliser column first: every lane takes its rows' normalisers from
  // the lane of its row group that holds column d_v
  const int jn = dv >> 4;
  f32x4 accn = out_tile(jn);
  float z[4];
#pragma unroll
  for (int jt = 0; jt < kFinMaxNT; ++jt)
    if (jt == jn)
#pragma unroll
      for (int i = 0; i < 4; ++i) accn[i] += pp[jt][i];
#pragma unroll
  for (int i = 0; i < 4; ++i) z[i] = __shfl(accn[i], 16 * l4 + (dv & 15));
  T* const yh = y + (bh * qg * n + t0) * (int64_t)dv;
#pragma unroll
  for (int jt = 0; jt < kFinMaxNT; ++jt) {
    if (jt >= NT) break;
    f32x4 acc = jt == jn ? accn : out_tile(jt);
    const int c = 16 * jt + l16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = r0 + 4 * l4 + i;
      if (jt != jn) acc[i] += pp[jt][i];
      if (c < dv && t < cn) yh[(int64_t)t * dv + c] = from_f32<T>(acc[i] / z[i]);
    }
  }
}

hipError_t launch_feat_finalize(const void* q, const void* k, const void* v, void* y, bool bf16, int BH, int n,
                                int dk, int dv, int P, int seg0, int seg_len, const float* partial, hipStream_t s,
                                int qg) {
  const size_t lds = fin_lds_bytes(dk, dv);
  const int seg_tokens = std::min(seg_len, n - seg0);
  const dim3 grid((unsigned)((seg_tokens + kCh - 1) / kCh), (unsigned)BH);
  hipError_t e;
  if (bf16) {
    if ((e = hipFuncSetAttribute((const void*)feat_finalize<bf16_t>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)lds)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(feat_finalize<bf16_t>, grid, dim3(256), lds, s, (const bf16_t*)q, (const bf16_t*)k,
                       (const bf16_t*)v, partial, (bf16_t*)y, n, dk, dv, P, seg0, seg_len, qg);
  } else {
    if ((e = hipFuncSetAttribute((const void*)feat_finalize<float>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)lds)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(feat_finalize<float>, grid, dim3(256), lds, s, (const float*)q, (const float*)k,
                       (const float*)v, partial, (float*)y, n, dk, dv, P, seg0, seg_len, qg);
  }
  return hipGetLastError();
}

// Tiles of 16 features per wave for NCT column tiles: the state, the readout
// sums (4 x NCT tiles) and the generation's registers fit two waves per SIMD
// (with bf16 operands, measured: 6 tiles at NCT = 5 spill a few registers yet
// beat 4 (a third fewer slices, so less cross-wave reduction and fewer
// partial rows per feature; 8 spill heavily), and 6 beat 8 and 10 at NCT = 3).
constexpr int ft_for(int nct, bool x3) {
  return x3 ? (nct <= 1 ? 22 : nct == 2 ? 10 : nct == 3 ? 6 : nct == 4 ? 4 : 2)
            : (nct <= 1 ? 28 : nct == 2 ? 16 : nct == 3 ? 6 : nct == 4 ? 6 : 6);
}
// Tiles per wave of the narrow variant: slices of 256 features, for heads
// whose few features would otherwise leave most waves, or most compute
// units, without work.
constexpr int kNarrowFT = 2;
constexpr int lds_for(int nct, bool x3) {
  switch (nct) {
    case 1: return x3 ? FeatLds<1, true>::kBytes : FeatLds<1, false>::kBytes;
    case 2: return x3 ? FeatLds<2, true>::kBytes : FeatLds<2, false>::kBytes;
    case 3: return x3 ? FeatLds<3, true>::kBytes : FeatLds<3, false>::kBytes;
    case 4: return x3 ? FeatLds<4, true>::kBytes : FeatLds<4, false>::kBytes;
    default: return x3 ? FeatLds<5, true>::kBytes : FeatLds<5, false>::kBytes;
  }
}

// One launch over the parts of a segment: `parts` workgroups per (slice,
// head), each taking part_len tokens.
struct FeatLaunch {
  FeatStates st;
  int seg0, seg_len, part_len, parts;
  bool readout;
};

template <int NCT, bool X3, int FT, typename T>
hipError_t launch_main(const void* q, const void* k, const void* v, const DevTable& t, const FeatLaunch& fl,
                       float* part, int BH, int n, int dk, int dv, int nslices, int qg, hipStream_t s) {
  constexpr int bytes = FeatLds<NCT, X3>::kBytes;
  static_assert(bytes <= 160 * 1024, "LDS of one workgroup");
  auto kern = fl.readout ? prefill_feat_main<NCT, FT, X3, T, true> : prefill_feat_main<NCT, FT, X3, T, false>;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)nslices, (unsigned)BH, (unsigned)fl.parts), dim3(kNW * 64), (size_t)bytes, s,
                     q, k, v, t.packed, t.gen, t.D, fl.st, part, BH, n, dk, dv, fl.seg0, fl.seg_len, fl.part_len, qg);
  return hipGetLastError();
}

template <int NCT, bool X3, typename T>
hipError_t launch_main_ft(bool narrow, const void* q, const void* k, const void* v, const DevTable& t,
                          const FeatLaunch& fl, float* part, int BH, int n, int dk, int dv, int nslices, int qg,
                          hipStream_t s) {
  if (narrow) return launch_main<NCT, X3, kNarrowFT, T>(q, k, v, t, fl, part, BH, n, dk, dv, nslices, qg, s);
  return launch_main<NCT, X3, ft_for(NCT, X3), T>(q, k, v, t, fl, part, BH, n, dk, dv, nslices, qg, s);
}

template <bool X3, typename T>
hipError_t launch_main_nct(const FeatPrefillPlan& p, const void* q, const void* k, const void* v, const DevTable& t,
                           const FeatLaunch& fl, float* part, int BH, int n, int dk, int dv, int qg, hipStream_t s) {
  switch (p.nct) {
    case 1: return launch_main_ft<1, X3, T>(p.narrow, q, k, v, t, fl, part, BH, n, dk, dv, p.nslices, qg, s);
    case 2: return launch_main_ft<2, X3, T>(p.narrow, q, k, v, t, fl, part, BH, n, dk, dv, p.nslices, qg, s);
    case 3: return launch_main_ft<3, X3, T>(p.narrow, q, k, v, t, fl, part, BH, n, dk, dv, p.nslices, qg, s);
    case 4: return launch_main_ft<4, X3, T>(p.narrow, q, k, v, t, fl, part, BH, n, dk, dv, p.nslices, qg, s);
    default: return launch_main_ft<5, X3, T>(p.narrow, q, k, v, t, fl, part, BH, n, dk, dv, p.nslices, qg, s);
  }
}

// Sp[g] += Sp[g - 1] for g = 1 .. parts - 2, in order: part g + 1 of the
// readout pass starts from Sp[g], the sum of the state increments of parts 0..g.
__global__ void __launch_bounds__(256) prefix_part_states(float* __restrict__ Sp, int64_t count, int parts) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  float a = Sp[i];
  for (int g = 1; g + 1 < parts; ++g) {
    a += Sp[g * count + i];
    Sp[g * count + i] = a;
  }
}

// The slices' partial readouts of one segment, summed into slice 0.
hipError_t fold_slices(float* partial, const FeatPrefillPlan& plan, int BH, int n, int dv, int seg0, hipStream_t s) {
  if (plan.nslices <= 1) return hipSuccess;
  const int seg_tokens = std::min(plan.seg_len, n - seg0);
  const int64_t count = (int64_t)BH * seg_tokens * (dv + 1);
  hipLaunchKernelGGL(reduce_slices, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, partial, BH, plan.seg_len,
                     seg_tokens, dv + 1, plan.nslices);
  return hipGetLastError();
}

}  // namespace

bool plan_prefill_feat(int64_t D, int BH, int n, int dk, int dv, int P, int chunk, bool split, size_t max_ws_bytes,
                       FeatPrefillPlan* plan) {
  if (chunk != kCh || P < 2 || dk > 64 || dv > 64 || n < 1) return false;
  const int E = dv + 1;
  const int nct = (E + 15) / 16;
  // Wide or narrow slices, by a simple model of the time per chunk: rounds of
  // one workgroup per compute unit (256) times the features of the busiest
  // wave plus a fixed share (loading the chunk, the reduction) worth about 32
  // features.  Narrow slices win where the wide ones leave compute units or
  // waves idle (few heads, few features).
  auto cost = [&](int ft) {
    const int64_t fs = (int64_t)kNW * ft * 16;
    const int64_t rounds = ((D + fs - 1) / fs * BH + 255) / 256;
    return rounds * (32 + std::min<int64_t>((int64_t)ft * 16, D));
  };
  plan->narrow = cost(kNarrowFT) < cost(ft_for(nct, split));
  const int64_t wide = kNW * ft_for(nct, split) * 16, narrow = kNW * kNarrowFT * 16;
  const int64_t fslice = plan->narrow ? narrow : wide;
  plan->nct = nct;
  plan->split = split;
  plan->nslices = (int)((D + fslice - 1) / fslice);
  plan->lds_main = (size_t)lds_for(nct, split);
  const size_t per_token = sizeof(float) * (size_t)plan->nslices * BH * E;
  int64_t seg = (int64_t)(max_ws_bytes / per_token) / kCh * kCh;
  if (seg < kCh) seg = kCh;
  const int64_t n_round = ((int64_t)n + kCh - 1) / kCh * kCh;
  plan->seg_len = (int)std::min<int64_t>(seg, n_round);
  plan->partial_bytes = per_token * (size_t)plan->seg_len;
  // Few workgroups (few heads with few features): a call that fits one
  // segment is cut into parts of at least 1024 tokens that run side by side,
  // up to one workgroup per compute unit.  A first pass sums each part's state
  // increment, and the readout pass starts part g from the sum of the
  // increments of parts 0 .. g-1 (kept after the partials in the workspace).
  plan->parts = 1;
  plan->part_len = plan->seg_len;
  plan->part_state_offset = 0;
  const int64_t wgs = (int64_t)plan->nslices * BH;
  if (plan->seg_len >= n_round) {
    int parts = 1;
    while (parts < 16 && wgs * parts * 2 <= 256 && n_round / (2 * parts) >= 1024) parts *= 2;
    if (parts > 1) {
      const int64_t plen = (n_round / parts + kCh - 1) / kCh * kCh;
      const size_t off = (plan->partial_bytes + 255) / 256 * 256;
      const size_t sbytes = sizeof(float) * (size_t)(parts - 1) * BH * D * E;
      if (off + sbytes <= max_ws_bytes && (parts - 1) * plen < n) {
        plan->parts = parts;
        plan->part_len = (int)plen;
        plan->part_state_offset = off;
        plan->partial_bytes = off + sbytes;
      }
    }
  }
  return true;
}

hipError_t launch_prefill_feat(const void* q, const void* k, const void* v, void* y, int BH, int n, int dk, int dv,
                               int P, const DevTable& t, const FeatPrefillPlan& plan, float* S_state, float* partial,
                               hipStream_t s, int qg) {
  // float32 inputs take split operands, bf16 inputs bf16 operands
  auto launch = [&](const FeatLaunch& fl) {
    return plan.split ? launch_main_nct<true, float>(plan, q, k, v, t, fl, partial, BH, n, dk, dv, qg, s)
                      : launch_main_nct<false, u16>(plan, q, k, v, t, fl, partial, BH, n, dk, dv, qg, s);
  };
  for (int seg0 = 0; seg0 < n; seg0 += plan.seg_len) {
    hipError_t e;
    if (plan.parts > 1) {  // (the call is one segment)
      float* const Sp = (float*)((char*)partial + plan.part_state_offset);
      e = launch(FeatLaunch{{nullptr, nullptr, nullptr, Sp}, seg0, plan.seg_len, plan.part_len, plan.parts - 1, false});
      if (e != hipSuccess) return e;
      if (plan.parts > 2) {
        const int64_t count = (int64_t)BH * t.D * (dv + 1);
        hipLaunchKernelGGL(prefix_part_states, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, Sp, count,
                           plan.parts);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      e = launch(FeatLaunch{{nullptr, Sp, S_state, nullptr}, seg0, plan.seg_len, plan.part_len, plan.parts, true});
    } else {
      const float* in0 = seg0 == 0 ? nullptr : S_state;
      e = launch(FeatLaunch{{in0, nullptr, S_state, nullptr}, seg0, plan.seg_len, plan.seg_len, 1, true});
    }
    if (e != hipSuccess) return e;
    if ((e = fold_slices(partial, plan, BH, n, dv, seg0, s)) != hipSuccess) return e;
    e = launch_feat_finalize(q, k, v, y, !plan.split, BH, n, dk, dv, P, seg0, plan.seg_len, partial, s, qg);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_prefill_feat_readout(const void* q, const void* k, const void* v, bool bf16_in, int BH, int n,
                                       int dk, int dv, const DevTable& t, const FeatPrefillPlan& plan,
                                       float* S_state, float* partial, int seg0, bool first, hipStream_t s) {
  const FeatLaunch fl{{first ? nullptr : S_state, nullptr, S_state, nullptr}, seg0, plan.seg_len, plan.seg_len, 1, true};
  hipError_t e = bf16_in ? launch_main_nct<true, u16>(plan, q, k, v, t, fl, partial, BH, n, dk, dv, 1, s)
                         : launch_main_nct<true, float>(plan, q, k, v, t, fl, partial, BH, n, dk, dv, 1, s);
  if (e != hipSuccess) return e;
  return fold_slices(partial, plan, BH, n, dv, seg0, s);
}

}  // namespace sata
