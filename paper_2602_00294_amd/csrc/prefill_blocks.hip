// Matrix-core (MFMA) causal prefill for bfloat16 q/k/v, P = 4, d_k = d_v in {16, 32},
// any supported chunk: the per-block variant (16 x 16 x 32 tiles, slices of
// consecutive first-index blocks).  The 64-token d = 32 case has a faster kernel.
//
// The method (App. A2) as a chunked scan: for chunk c with queries Q_c, keys
// K_c and values V_c,
//     O_c = phi(Q_c) S_{c-1}  +  mask(f_P(Q_c K_c^T / sqrt d)) [V_c | 1]
//     S_c = S_{c-1} + phi(K_c)^T [V_c | 1],      y = O[:, :d_v] / O[:, d_v].
// Both state contractions run on v_mfma_f32_16x16x32_bf16 with the state held
// in float32 accumulator registers for the whole sequence.  The feature basis
// is used in a factored form so that only the low-degree features are ever
// materialised:
//
//  * Low features (degrees 0..P-2 = 0, 1, 2) are generated per chunk into LDS
//    (bf16) and multiply their rows of S directly.
//  * Every top-degree feature is f = (i1, g) with g a degree-(P-2) feature whose
//    indices are all >= i1 (Sec. 2.4 footnote: a lower-degree monomial times one
//    more coordinate).  Its value is phi_f(x) = x~[i1] phi_g(x) / sqrt(c1), c1 the
//    multiplicity of i1 in f.  For one first index i1 ("block") the readout is
//        O += diag(q~[:, i1]) * (Phi_g(Q)[:, suffix] * (S_block / c1)),
//    an MFMA over already generated degree-(P-2) features followed by one row
//    scale per block, and the update is
//        S_block += Phi_g(K)[:, suffix]^T * (diag(k~[:, i1]) V).
//    The internal state keeps S_int = sqrt(c1) * S for these rows.
//  * The normaliser column is not padded into the value tiles.  Summing over
//    all (i1, g) pairs, sorted or not, gives p times the degree-p term:
//        sum_{i1} sum_{g of degree p-1} x~_q[i1] phi_g(q) x~_k[i1] phi_g(k)
//            = s * s^(p-1)/(p-1)! = p * s^p/p!,   s = q.k/sqrt(d),
//    so one dense matrix Zfull[g][i1] = sum_t phi_g(k_t) k~_t[i1] over the low
//    features g (degree p-1 = deg(g)) yields every degree >= 1 normaliser term
//    with a row weight 1/(deg(g)+1).  Degree 0 contributes the token count.
//
// Features are ordered inside the kernel so that every block's suffix of
// degree-(P-2) features is a prefix of the LDS column order: LDS column c < m1
// holds the degree-2 feature with canonical degree-2 index m1-1-c (reversed
// lexicographic order), columns m1.. hold degree 0 and degree 1.  The state is
// written out in the library's canonical order at the end.
//
// Work split: each head's pairs of 32 state rows ("pairs") are spread over
// several workgroups ("slices"); each slice writes float32 partial readouts
// per token, and a second kernel adds the slices' partials, computes the
// intra-chunk term on the matrix cores, and normalises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <vector>

#include "device_common.hpp"
#include "prefill_blocks.hpp"

namespace sata {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

enum PairKind : int { kEmpty = 0, kLow = 1, kTop = 2, kZmat = 3 };
enum PairFlags : int { kFirstOfRun = 1, kLastOfRun = 2 };

// Host-built description of one pair of 32 state rows.
struct PairMeta {
  int kind;      // PairKind
  int col0;      // first LDS feature column of the pair (a multiple of 32)
  int i1;        // top pairs: first index of the block
  int nrows;     // top pairs: rows that hold a feature of the block
  int rho_from;  // top pairs: rows >= rho_from have first(g) == i1 (32: none)
  int flags;     // top pairs: PairFlags within the owning wave
  int out0;      // top pairs: canonical feature of pair row 0 (rows descend)
  int pad;
};

constexpr int kWaveSize = 64;
constexpr int kGroup = 64;     // tokens per feature-generation group (one per lane)
constexpr int kTS = 68;        // float stride of the transposed [dim][token] LDS tiles

template <int DK>
struct Geo {
  static constexpr int M1 = DK * (DK + 1) / 2;   // degree-2 features
  static constexpr int DL = M1 + DK + 1;         // degrees 0..2
  static constexpr int LW = (DL + 31) / 32 * 32; // LDS feature columns (whole pairs)
  static constexpr int NG = LW / 8;              // groups of 8 columns
  static constexpr int QS = LW * 2 + 16;         // bytes per token row of Phi(Q)
  static constexpr int KS = kGroup * 2 + 16;     // bytes per feature row of Phi(K)
};

// What LDS feature column c holds, as a function of the token's scaled
// coordinates x~ = x * d^(-1/4).
struct ColDesc {
  int kind;  // 0 zero, 1 constant 1, 2 x~[a], 3 x~[a] x~[b], 4 x~[a]^2 / sqrt(2)
  int a, b;
};

template <int DK>
constexpr ColDesc col_desc(int c) {
  constexpr int M1 = DK * (DK + 1) / 2;
  if (c < M1) {
    const int canon = M1 - 1 - c;  // canonical (lexicographic) degree-2 index
    int a = 0, base = 0;
    while (base + (DK - a) <= canon) {
      base += DK - a;
      ++a;
    }
    const int b = a + (canon - base);
    return ColDesc{a == b ? 4 : 3, a, b};
  }
  c -= M1;
  if (c == 0) return ColDesc{1, 0, 0};
  if (c <= DK) return ColDesc{2, c - 1, 0};
  return ColDesc{0, 0, 0};
}

template <int DK, int C>
__device__ __forceinline__ float col_value(const float (&xt)[DK]) {
  constexpr ColDesc cd = col_desc<DK>(C);
  if constexpr (cd.kind == 0) return 0.0f;
  else if constexpr (cd.kind == 1) return 1.0f;
  else if constexpr (cd.kind == 2) return xt[cd.a];
  else if constexpr (cd.kind == 3) return xt[cd.a] * xt[cd.b];
  else return (xt[cd.a] * 0.70710678118654752f) * xt[cd.a];
}

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 pack8(const float (&e)[8]) {
  uint4 w;
  w.x = pack2(e[0], e[1]);
  w.y = pack2(e[2], e[3]);
  w.z = pack2(e[4], e[5]);
  w.w = pack2(e[6], e[7]);
  return __builtin_bit_cast(bf16x8, w);
}

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Feature generation for this lane's token row: groups J, J+NW, J+2NW, ... of
// 8 LDS columns up to the slice's need.  Group indices are compile-time
// constants, so every coordinate index below is a register.
template <int DK, int NW, int J>
__device__ __forceinline__ void gen_q_from(const float (&xt)[DK], char* row, int ngneed) {
  if constexpr (J < Geo<DK>::NG) {
    if (J >= ngneed) return;
    uint4 w;
    w.x = pack2(col_value<DK, 8 * J + 0>(xt), col_value<DK, 8 * J + 1>(xt));
    w.y = pack2(col_value<DK, 8 * J + 2>(xt), col_value<DK, 8 * J + 3>(xt));
    w.z = pack2(col_value<DK, 8 * J + 4>(xt), col_value<DK, 8 * J + 5>(xt));
    w.w = pack2(col_value<DK, 8 * J + 6>(xt), col_value<DK, 8 * J + 7>(xt));
    *(uint4*)(row + 16 * J) = w;  // Phi(Q): [token][column]
    gen_q_from<DK, NW, J + NW>(xt, row, ngneed);
  }
}

template <int DK, int NW, int J>
__device__ __forceinline__ void gen_k_from(const float (&xt)[DK], char* col, int ngneed) {
  if constexpr (J < Geo<DK>::NG) {
    constexpr int KS = Geo<DK>::KS;
    if (J >= ngneed) return;
    const uint32_t w0 = pack2(col_value<DK, 8 * J + 0>(xt), col_value<DK, 8 * J + 1>(xt));
    const uint32_t w1 = pack2(col_value<DK, 8 * J + 2>(xt), col_value<DK, 8 * J + 3>(xt));
    const uint32_t w2 = pack2(col_value<DK, 8 * J + 4>(xt), col_value<DK, 8 * J + 5>(xt));
    const uint32_t w3 = pack2(col_value<DK, 8 * J + 6>(xt), col_value<DK, 8 * J + 7>(xt));
    char* p = col + (8 * J) * KS;  // Phi(K): [column][token]
    *(u16*)(p + 0 * KS) = (u16)w0;
    *(u16*)(p + 1 * KS) = (u16)(w0 >> 16);
    *(u16*)(p + 2 * KS) = (u16)w1;
    *(u16*)(p + 3 * KS) = (u16)(w1 >> 16);
    *(u16*)(p + 4 * KS) = (u16)w2;
    *(u16*)(p + 5 * KS) = (u16)(w2 >> 16);
    *(u16*)(p + 6 * KS) = (u16)w3;
    *(u16*)(p + 7 * KS) = (u16)(w3 >> 16);
    gen_k_from<DK, NW, J + NW>(xt, col, ngneed);
  }
}

template <int DK, int NW, bool IS_Q, int W = 0>
__device__ __forceinline__ void gen_dispatch(const float (&xt)[DK], char* base, int wave, int ngneed) {
  if constexpr (W < NW) {
    if (wave == W) {
      if constexpr (IS_Q) gen_q_from<DK, NW, W>(xt, base, ngneed);
      else gen_k_from<DK, NW, W>(xt, base, ngneed);
      return;
    }
    gen_dispatch<DK, NW, IS_Q, W + 1>(xt, base, wave, ngneed);
  }
}

__device__ __forceinline__ float bf16_to_f32(u16 b) { return __uint_as_float((uint32_t)b << 16); }

// Loads the group's tokens of one input tensor into LDS as [dim][token] float32,
// multiplied by `scale`; tokens at or beyond `ntok` are zero.
// Staging of one tensor's 64-token tile into LDS as [dim][token] float32.
// Each thread moves VEC consecutive bf16 coordinates of one token: first from
// global memory into registers (issued early, so the latency overlaps other
// work), later from registers into LDS.
template <int DIM, int NTHREADS>
struct TileFetch {
  static constexpr int VEC = (DIM * kGroup) / NTHREADS;  // 4 (d = 32, 512 threads) or 2 (d = 16)
  static_assert(VEC == 2 || VEC == 4, "tile fetch width");
  uint32_t w[VEC / 2];
  __device__ __forceinline__ void fetch(const u16* __restrict__ src, int ntok) {
    const int e0 = threadIdx.x * VEC;
    const int tok = e0 / DIM;
    if (tok < ntok) {
      if constexpr (VEC == 4) {
        const uint2 x = *(const uint2*)(src + e0);
        w[0] = x.x;
        w[1] = x.y;
      } else {
        w[0] = *(const uint32_t*)(src + e0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < VEC / 2; ++i) w[i] = 0u;
    }
  }
  __device__ __forceinline__ void stage(float* dst, float scale) const {
    const int e0 = threadIdx.x * VEC;
    const int tok = e0 / DIM;
    const int c0 = e0 - tok * DIM;
#pragma unroll
    for (int i = 0; i < VEC / 2; ++i) {
      dst[(c0 + 2 * i) * kTS + tok] = __uint_as_float(w[i] << 16) * scale;
      dst[(c0 + 2 * i + 1) * kTS + tok] = __uint_as_float(w[i] & 0xffff0000u) * scale;
    }
  }
};

template <int DK, int DV, int NW, int PPW>
struct MainLds {
  static constexpr int kColMeta = 0;
  static constexpr int kZFac = kColMeta + Geo<DK>::LW * 4;   // normaliser row factor 3/(deg+1)
  static constexpr int kRFac = kZFac + Geo<DK>::LW * 4;      // 1/c1 for rows with first(g) == i1
  static constexpr int kPhi = kRFac + Geo<DK>::LW * 4;
  static constexpr int kPhiBytes = (kGroup * Geo<DK>::QS > Geo<DK>::LW * Geo<DK>::KS)
                                       ? kGroup * Geo<DK>::QS
                                       : Geo<DK>::LW * Geo<DK>::KS;
  static constexpr int kQT = kPhi + kPhiBytes;
  static constexpr int kKT = kQT + (DK + 2) * kTS * 4;   // + a row of ones and a row of 1/3
  static constexpr int kVT = kKT + (DK + 2) * kTS * 4;
  static constexpr int kRed = kVT + DV * kTS * 4;
  static constexpr int kMeta = kRed + NW * 32 * (DV + 1) * 4;
  static constexpr int kBytes = kMeta + NW * PPW * 8;
};

// Packed pair description (host-built): see pack_pair().
__device__ __forceinline__ int pk_kind(uint32_t x) { return x & 3; }
__device__ __forceinline__ int pk_flags(uint32_t x) { return (x >> 2) & 3; }
__device__ __forceinline__ bool pk_rowfac(uint32_t x) { return (x >> 4) & 1; }
__device__ __forceinline__ int pk_col0(uint32_t x) { return ((x >> 5) & 127) * 32; }
__device__ __forceinline__ int pk_i1(uint32_t x) { return (x >> 12) & 255; }
__device__ __forceinline__ int pk_nrows(uint32_t x) { return (x >> 20) & 63; }
__device__ __forceinline__ int pk_rho_from(uint32_t x) { return (x >> 26) & 63; }

// DENSE: registers capped for four waves per SIMD (two workgroups per compute
// unit, a few registers spilled), for calls with workgroups to fill both.
template <int DK, int DV, int NW, int PPW, bool DENSE>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(DENSE ? 4 : 1)))
prefill_blocks_main(const u16* __restrict__ q, const u16* __restrict__ k, const u16* __restrict__ v,
                  const uint2* __restrict__ pmeta, const int* __restrict__ slice_ng,
                  const uint32_t* __restrict__ colmeta_g, const int* __restrict__ zmap,
                  float* __restrict__ partial, float* __restrict__ S_out, int BH, int n, int C, int nslices,
                  int qg) {
  static_assert(DK == DV, "matrix-core path assumes d_k == d_v");
  using G = Geo<DK>;
  using L = MainLds<DK, DV, NW, PPW>;
  constexpr int NT = DV / 16;  // N tiles of the value columns (== tiles of the i1 columns)
  constexpr int E = DV + 1;
  constexpr int D = G::DL + (DK * (DK + 1) * (DK + 2)) / 6;  // C(d+3, 3)
  constexpr int NTH = NW * 64;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  uint32_t* colmeta = (uint32_t*)(smem + L::kColMeta);
  float* zfac = (float*)(smem + L::kZFac);
  float* rfac = (float*)(smem + L::kRFac);
  char* phi = smem + L::kPhi;
  float* qT = (float*)(smem + L::kQT);
  float* kT = (float*)(smem + L::kKT);
  float* vT = (float*)(smem + L::kVT);
  float* red = (float*)(smem + L::kRed);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l15 = lane & 15;
  const int g4 = lane >> 4;  // 0..3
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int slice = blockIdx.x;
  const int64_t bh = blockIdx.y;
  const int ngneed = slice_ng[slice];
  const float xscale = 1.0f / sqrtf(sqrtf((float)DK));  // d^(-1/4)

  for (int i = tid; i < G::LW; i += NTH) {
    const uint32_t cm = colmeta_g[i];
    colmeta[i] = cm;
    const int deg = (cm >> 16) & 0xff;
    // the normaliser's 1/(deg+1) relative to the 1/3 folded into its update
    zfac[i] = deg == 2 ? 1.0f : deg == 1 ? 1.5f : deg == 0 ? 3.0f : 0.0f;
    rfac[i] = ((cm >> 8) & 0xff) == 2 ? (1.0f / 3.0f) : 0.5f;  // 1/(1 + count of first index)
  }
  // constant factor rows after the coordinates: row DK = 1 (low pairs),
  // row DK+1 = 1/3 (normaliser pairs, the factor 1/(P-1) of degree-2 rows)
  for (int i = tid; i < kGroup; i += NTH) {
    qT[DK * kTS + i] = 1.0f;
    kT[DK * kTS + i] = 1.0f;
    qT[(DK + 1) * kTS + i] = 1.0f / 3.0f;
    kT[(DK + 1) * kTS + i] = 1.0f / 3.0f;
  }

  // Pair descriptions live in LDS and are re-read where used, which keeps the
  // decoded fields short-lived instead of pinning them in scalar registers.
  uint2* meta = (uint2*)(smem + L::kMeta);
  for (int i = tid; i < NW * PPW; i += NTH) meta[i] = pmeta[(int64_t)slice * NW * PPW + i];
  const uint2* wmeta = meta + wave * PPW;
  auto mxof = [&](int t) -> uint32_t { return __builtin_amdgcn_readfirstlane(wmeta[t].x); };
  __syncthreads();
  bool has_z = false;
#pragma unroll
  for (int t = 0; t < PPW; ++t) has_z = has_z || pk_kind(mxof(t)) == kZmat;

  f32x4 S[PPW][2][NT];
#pragma unroll
  for (int t = 0; t < PPW; ++t)
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int j = 0; j < NT; ++j) S[t][r][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int G_tok = C < kGroup ? C : kGroup;  // tokens per group
  const int ngroups = C / G_tok;
  const u16* qh = q + bh * (int64_t)qg * n * DK;  // qg query heads per key/value head
  const u16* kh = k + bh * (int64_t)n * DK;
  const u16* vh = v + bh * (int64_t)n * DV;

  TileFetch<DK, NTH> fq, fk;
  TileFetch<DV, NTH> fv;
  fq.fetch(qh, min(G_tok, n));

  for (int t0 = 0; t0 < n; t0 += C) {
    // ------------------------------------------------------------ readout
    for (int gi = 0; gi < ngroups; ++gi) {
      const int tg0 = t0 + gi * G_tok;
      if (tg0 >= n) break;
      const int ntok = min(G_tok, n - tg0);
      __syncthreads();
      fq.stage(qT, xscale);
      // prefetch the next staging step: q of the next group, else k and v of this chunk
      if (gi + 1 < ngroups && tg0 + G_tok < n) {
        fq.fetch(qh + (int64_t)(tg0 + G_tok) * DK, min(G_tok, n - tg0 - G_tok));
      } else {
        fk.fetch(kh + (int64_t)t0 * DK, min(G_tok, n - t0));
        fv.fetch(vh + (int64_t)t0 * DV, min(G_tok, n - t0));
      }
      __syncthreads();
      {
        float xt[DK];
#pragma unroll
        for (int i = 0; i < DK; ++i) xt[i] = qT[i * kTS + lane];
        gen_dispatch<DK, NW, true>(xt, phi + lane * G::QS, wave, ngneed);
      }
      __syncthreads();
      for (int h = 0; h * 32 < ntok; ++h) {
        // Readout of 32 tokens (two row tiles) against S_{c-1}.  R accumulates a
        // run of one block (or, in waves that own the normaliser pairs, the
        // normaliser readout; the planner never mixes the two).
        f32x4 O[2][NT], R[2][NT];
        float zp[2][4];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            O[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
            R[m][j] = O[m][j];
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) zp[m][i] = 0.0f;
        }
#pragma unroll
        for (int t = 0; t < PPW; ++t) {
          // Every pair runs the same MFMA code: R += Phi(Q)[:, pair] * S_pair.
          // Empty slots hold a zero state and add nothing.
          const uint32_t x = mxof(t);
          const int col0 = pk_col0(x);
          bf16x8 a[2];
#pragma unroll
          for (int m = 0; m < 2; ++m) {
            const char* p = phi + (32 * h + 16 * m + l15) * G::QS + (col0 + 4 * g4) * 2;
            const uint2 lo = *(const uint2*)p;
            const uint2 hi = *(const uint2*)(p + 32);
            a[m] = __builtin_bit_cast(bf16x8, uint4{lo.x, lo.y, hi.x, hi.y});
          }
          // Row factors, branch-free: rows r >= `from` take the column's factor
          // (normaliser pairs at the low-degree boundary: 3/(deg+1); top pairs:
          // 1/c1 on rows whose g starts with i1), all other rows 1.
          const bool zk = pk_kind(x) == kZmat;
          const float* ftab = zk ? zfac : rfac;
          const int from = pk_rowfac(x) ? (zk ? 0 : pk_rho_from(x)) : 32;
          const f32x4 f0 = *(const f32x4*)(ftab + col0 + 4 * g4);
          const f32x4 f1 = *(const f32x4*)(ftab + col0 + 16 + 4 * g4);
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            float e[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              e[i] = S[t][0][j][i] * (4 * g4 + i >= from ? f0[i] : 1.0f);
              e[4 + i] = S[t][1][j][i] * (16 + 4 * g4 + i >= from ? f1[i] : 1.0f);
            }
            const bf16x8 b = pack8(e);
#pragma unroll
            for (int m = 0; m < 2; ++m) R[m][j] = mfma(a[m], b, R[m][j]);
          }
          // run epilogue: value runs are scaled per token by q~[t][i1] (low runs by
          // the row of ones) and added to O; the normaliser run is reduced into zp
          if (pk_flags(x) & kLastOfRun) {
            if (zk) {
#pragma unroll
              for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                  const f32x4 qv = *(const f32x4*)(qT + (16 * j + l15) * kTS + 32 * h + 16 * m + 4 * g4);
#pragma unroll
                  for (int i = 0; i < 4; ++i) zp[m][i] += qv[i] * R[m][j][i];
                }
            } else {
              const float* qrow = qT + pk_i1(x) * kTS + 32 * h + 4 * g4;
#pragma unroll
              for (int m = 0; m < 2; ++m) {
                const f32x4 qv = *(const f32x4*)(qrow + 16 * m);
#pragma unroll
                for (int j = 0; j < NT; ++j) O[m][j] += qv * R[m][j];
              }
            }
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
              for (int j = 0; j < NT; ++j) R[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
        }
        // normaliser of degrees >= 1: zp holds, per lane, the sum over this lane's
        // i1 columns of q~[t][i1] * R[t][i1]; finish the sum across the 16 lanes
        if (has_z) {
#pragma unroll
          for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              float s = zp[m][i];
              s += __shfl_xor(s, 1, 16);
              s += __shfl_xor(s, 2, 16);
              s += __shfl_xor(s, 4, 16);
              s += __shfl_xor(s, 8, 16);
              zp[m][i] = s;
            }
        }
        float* rw = red + wave * 32 * E;
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int tok = 16 * m + 4 * g4 + i;
#pragma unroll
            for (int j = 0; j < NT; ++j) rw[tok * E + 16 * j + l15] = O[m][j][i];
            if (l15 == 0) rw[tok * E + DV] = zp[m][i];
          }
        __syncthreads();
        const int tbase = tg0 + 32 * h;
        const int tvalid = min(32, n - tbase);
        float* pout = partial + (((int64_t)slice * BH + bh) * n + tbase) * E;
        for (int o = tid; o < tvalid * E; o += NTH) {
          float s = 0.0f;
#pragma unroll
          for (int w = 0; w < NW; ++w) s += red[w * 32 * E + o];
          pout[o] = s;
        }
        __syncthreads();
      }
    }
    // ------------------------------------------------------------ update
    for (int gi = 0; gi < ngroups; ++gi) {
      const int tg0 = t0 + gi * G_tok;
      if (tg0 >= n) break;
      const int ntok = min(G_tok, n - tg0);
      __syncthreads();
      fk.stage(kT, xscale);
      fv.stage(vT, 1.0f);
      // prefetch the next staging step: k, v of the next group, else q of the next chunk
      if (gi + 1 < ngroups && tg0 + G_tok < n) {
        fk.fetch(kh + (int64_t)(tg0 + G_tok) * DK, min(G_tok, n - tg0 - G_tok));
        fv.fetch(vh + (int64_t)(tg0 + G_tok) * DV, min(G_tok, n - tg0 - G_tok));
      } else if (t0 + C < n) {
        fq.fetch(qh + (int64_t)(t0 + C) * DK, min(G_tok, n - t0 - C));
      }
      __syncthreads();
      {
        float xt[DK];
#pragma unroll
        for (int i = 0; i < DK; ++i) xt[i] = kT[i * kTS + lane];
        gen_dispatch<DK, NW, false>(xt, phi + lane * 2, wave, ngneed);
      }
      __syncthreads();
      const int nks = ntok > 32 ? 2 : 1;
      int cur_key = -1;
      bf16x8 B[2][NT];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int j = 0; j < NT; ++j) B[ks][j] = __builtin_bit_cast(bf16x8, uint4{0u, 0u, 0u, 0u});
#pragma unroll
      for (int t = 0; t < PPW; ++t) {
        const uint32_t x = mxof(t);
        const int kind = pk_kind(x);
        // B = src[col][token] * f[token]: values times k~[t][i1] (top), values
        // times 1 (low), keys times 1/3 (normaliser)
        const int frow = kind == kTop ? pk_i1(x) : (kind == kZmat ? DK + 1 : DK);
        const int key = (kind == kZmat ? 1024 : 0) + frow;
        if (key != cur_key) {
          cur_key = key;
          const float* srcb = kind == kZmat ? kT : vT;
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const int tok0 = 32 * ks + 8 * g4;
            const f32x4 f0 = *(const f32x4*)(kT + frow * kTS + tok0);
            const f32x4 f1 = *(const f32x4*)(kT + frow * kTS + tok0 + 4);
#pragma unroll
            for (int j = 0; j < NT; ++j) {
              const float* src = srcb + (16 * j + l15) * kTS + tok0;
              const f32x4 x0 = *(const f32x4*)src;
              const f32x4 x1 = *(const f32x4*)(src + 4);
              float e[8] = {x0[0] * f0[0], x0[1] * f0[1], x0[2] * f0[2], x0[3] * f0[3],
                            x1[0] * f1[0], x1[1] * f1[1], x1[2] * f1[2], x1[3] * f1[3]};
              B[ks][j] = pack8(e);
            }
          }
        }
        const int col0 = pk_col0(x);
        const int nrows = pk_nrows(x);
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int row = 16 * r + l15;
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            if (ks >= nks) break;
            uint4 w = *(const uint4*)(phi + (col0 + row) * G::KS + (32 * ks + 8 * g4) * 2);
            if (nrows < 32 && row >= nrows) w = uint4{0u, 0u, 0u, 0u};
            const bf16x8 a = __builtin_bit_cast(bf16x8, w);
#pragma unroll
            for (int j = 0; j < NT; ++j) S[t][r][j] = mfma(a, B[ks][j], S[t][r][j]);
          }
        }
      }
    }
  }

  // ------------------------------------------------------------ state export
  if (S_out == nullptr) return;
  float* So = S_out + bh * (int64_t)D * E;
#pragma unroll
  for (int t = 0; t < PPW; ++t) {
    const uint32_t x = mxof(t);
    const int kind = pk_kind(x);
    if (kind == kEmpty) continue;
    const int col0 = pk_col0(x);
    const int o0 = __builtin_amdgcn_readfirstlane((int)wmeta[t].y);
#pragma unroll
    for (int r2 = 0; r2 < 2; ++r2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * r2 + 4 * g4 + i;
        const int c = col0 + r;
        const uint32_t cm = colmeta[c];
        const int first = cm & 0xff;
        const int cnt = (cm >> 8) & 0xff;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int col = 16 * j + l15;
          const float val = S[t][r2][j][i];
          if (kind == kLow) {
            if (c < G::DL) {
              const int canon = c < G::M1 ? G::DL - 1 - c : c - G::M1;
              So[(int64_t)canon * E + col] = val;
            }
          } else if (kind == kTop) {
            if (r < pk_nrows(x)) {
              const float sc = r >= pk_rho_from(x) ? rsqrtf((float)(1 + cnt)) : 1.0f;
              So[(int64_t)(o0 - r) * E + col] = val * sc;
            }
          } else {
            if (c < G::DL) {
              const int canon = zmap[c * DK + col];
              if (canon >= 0) {
                // the update carried a factor 1/3; undo it, then the 1/sqrt(c1) weight
                const float sc = 3.0f * (first == col ? rsqrtf((float)(1 + cnt)) : 1.0f);
                So[(int64_t)canon * E + DV] = val * sc;
              }
            }
          }
        }
      }
  }
  if (slice == 0 && tid == 0) So[DV] = (float)n;  // degree 0: the token count
}

// ------------------------------------------------------------ finalize kernel
//
// One workgroup per (chunk, head): intra-chunk term mask(f_P(Q K^T / sqrt d)) [V | 1]
// on the matrix cores, plus the slices' partial inter-chunk readouts, plus the
// degree-0 normaliser (number of earlier tokens), then y = O / Z.

struct FinLayout {
  int qs, ps, vs;             // row strides in bytes
  int oq, ok, op, ov, oz, orow;  // byte offsets
  int bytes;
  __host__ __device__ FinLayout(int DK, int DV, int C) {
    qs = DK * 2 + 16;
    ps = C * 2 + 16;
    vs = C * 2 + 16;
    oq = 0;
    ok = oq + C * qs;
    op = ok + C * qs;
    ov = op + C * ps;
    oz = ov + DV * vs;
    orow = oz + C * 4;
    bytes = orow + C * (C / 16) * 4;
  }
};

template <int DK, int DV>
__global__ void __launch_bounds__(256)
prefill_blocks_finalize(const u16* __restrict__ q, const u16* __restrict__ k, const u16* __restrict__ v,
                      const float* __restrict__ partial, u16* __restrict__ y, int BH, int n, int C, int nslices,
                      int P, int qg) {
  constexpr int E = DV + 1;
  constexpr int NT = DV / 16;
  const FinLayout L(DK, DV, C);
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* Qs = smem + L.oq;
  char* Ks = smem + L.ok;
  char* Pm = smem + L.op;
  char* Vt = smem + L.ov;
  float* Zs = (float*)(smem + L.oz);
  float* rowpart = (float*)(smem + L.orow);  // [query][key tile]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int l15 = lane & 15;
  const int g4 = lane >> 4;
  const int wave = tid >> 6;
  const int64_t bh = blockIdx.y;
  const int t0 = blockIdx.x * C;
  const int cn = min(C, n - t0);
  const float inv_sqrt_d = 1.0f / sqrtf((float)DK);
  const int MT = C / 16;

  // stage Q, K rows and V^T (bf16), 8 coordinates per thread; tokens >= cn are zero
  for (int i = tid; i < C * (DK / 8); i += 256) {
    const int tok = i / (DK / 8);
    const int c8 = (i - tok * (DK / 8)) * 8;
    uint4 qv = {0u, 0u, 0u, 0u}, kv = {0u, 0u, 0u, 0u};
    if (tok < cn) {
      qv = *(const uint4*)(q + (bh * qg * n + t0 + tok) * DK + c8);
      kv = *(const uint4*)(k + (bh * n + t0 + tok) * DK + c8);
    }
    *(uint4*)(Qs + tok * L.qs + c8 * 2) = qv;
    *(uint4*)(Ks + tok * L.qs + c8 * 2) = kv;
  }
  for (int i = tid; i < C * (DV / 8); i += 256) {
    const int tok = i / (DV / 8);
    const int c8 = (i - tok * (DV / 8)) * 8;
    uint4 vv = {0u, 0u, 0u, 0u};
    if (tok < cn) vv = *(const uint4*)(v + (bh * n + t0 + tok) * DV + c8);
    const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      *(u16*)(Vt + (c8 + 2 * e) * L.vs + tok * 2) = (u16)w[e];
      *(u16*)(Vt + (c8 + 2 * e + 1) * L.vs + tok * 2) = (u16)(w[e] >> 16);
    }
  }
  __syncthreads();

  // scores and Taylor weights, one 16x16 tile per step; row sums per tile
  for (int tile = wave; tile < MT * MT; tile += 4) {
    const int mq = tile / MT;
    const int nk = tile - mq * MT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (nk <= mq) {
#pragma unroll
      for (int kk = 0; kk < (DK + 31) / 32; ++kk) {
        uint4 aw = {0u, 0u, 0u, 0u}, bw = {0u, 0u, 0u, 0u};
        if (32 * kk + 8 * g4 < DK) {
          aw = *(const uint4*)(Qs + (16 * mq + l15) * L.qs + (32 * kk + 8 * g4) * 2);
          bw = *(const uint4*)(Ks + (16 * nk + l15) * L.qs + (32 * kk + 8 * g4) * 2);
        }
        acc = mfma(__builtin_bit_cast(bf16x8, aw), __builtin_bit_cast(bf16x8, bw), acc);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qi = 16 * mq + 4 * g4 + i;
      const int ki = 16 * nk + l15;
      float w = 0.0f;
      if (ki <= qi && qi < cn) w = taylor_horner(acc[i] * inv_sqrt_d, P);
      const __bf16 wb = (__bf16)w;
      *(__bf16*)(Pm + qi * L.ps + ki * 2) = wb;
      float rs = (float)wb;  // the normaliser sums the same rounded weights as the numerator
      rs += __shfl_xor(rs, 1, 16);
      rs += __shfl_xor(rs, 2, 16);
      rs += __shfl_xor(rs, 4, 16);
      rs += __shfl_xor(rs, 8, 16);
      if (l15 == 0) rowpart[qi * MT + nk] = rs;
    }
  }
  __syncthreads();

  // normaliser: intra row sums + partials + earlier-token count (degree 0)
  for (int qi = tid; qi < C; qi += 256) {
    float z = (float)t0;
    for (int t = 0; t < MT; ++t) z += rowpart[qi * MT + t];
    if (qi < cn)
      for (int s = 0; s < nslices; ++s) z += partial[(((int64_t)s * BH + bh) * n + t0 + qi) * E + DV];
    Zs[qi] = z;
  }
  __syncthreads();

  // O = P V on the matrix cores, + partials, / Z
  for (int tile = wave; tile < MT * NT; tile += 4) {
    const int mq = tile / NT;
    const int j = tile - mq * NT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks * 32 < C; ++ks) {
      if (32 * ks > 16 * mq + 15) break;  // keys beyond the tile's last query carry zero weight
      const uint4 aw = *(const uint4*)(Pm + (16 * mq + l15) * L.ps + (32 * ks + 8 * g4) * 2);
      const uint4 bw = *(const uint4*)(Vt + (16 * j + l15) * L.vs + (32 * ks + 8 * g4) * 2);
      acc = mfma(__builtin_bit_cast(bf16x8, aw), __builtin_bit_cast(bf16x8, bw), acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int qi = 16 * mq + 4 * g4 + i;
      const int col = 16 * j + l15;
      if (qi < cn) {
        float o = acc[i];
        for (int s = 0; s < nslices; ++s) o += partial[(((int64_t)s * BH + bh) * n + t0 + qi) * E + col];
        y[(bh * qg * n + t0 + qi) * DV + col] = f32_to_bf16(o / Zs[qi]).bits;
      }
    }
  }
}

// ------------------------------------------------------------ host planning

struct DeviceTables {
  uint2* pairs = nullptr;
  int* slice_ng = nullptr;
  uint32_t* colmeta = nullptr;
  int* zmap = nullptr;
  int nslices = 0;
};

std::mutex g_mfma_mu;
std::map<std::pair<int, int>, DeviceTables> g_mfma_tables;  // (device, dk)

constexpr int kNW = 8;

// Pairs per wave.  At d = 16, 6 (measured against 4, 8, 10, 12, 14, 16: fewer
// state registers per wave, so more workgroups resident, outweigh the extra
// slices' partial rows; 16 took 2.26 ms where 6 takes 1.33 ms at B = 8,
// H = 32, n = 8192).
int ppw_for(int dk) { return dk == 16 ? 6 : 8; }

// Canonical index of the degree-2 feature (a, b), a <= b, among degree-2 features.
int idx2(int d, int a, int b) { return a * d - a * (a - 1) / 2 + (b - a); }

// Packs one pair description into two words: word 0 holds kind (2 bits),
// run flags (2), per-row-factor flag (1), col0/32 (7), i1 (8), nrows (6) and
// rho_from (6); word 1 the canonical row of pair row 0 (top pairs).
uint2 pack_pair(const PairMeta& m, int M1) {
  bool rowfac = false;
  if (m.kind == kZmat) rowfac = m.col0 + 32 > M1;  // rows of degree < 2 or padding
  if (m.kind == kTop) rowfac = m.rho_from < 32;
  uint32_t x = (uint32_t)m.kind | ((uint32_t)m.flags << 2) | ((uint32_t)rowfac << 4) |
               ((uint32_t)(m.col0 / 32) << 5) | ((uint32_t)m.i1 << 12) | ((uint32_t)m.nrows << 20) |
               ((uint32_t)m.rho_from << 26);
  return uint2{x, (uint32_t)m.out0};
}

struct HostTables {
  std::vector<PairMeta> pairs;  // [nslices][kNW][ppw]
  std::vector<int> slice_ng;
  std::vector<uint32_t> colmeta;
  std::vector<int> zmap;
  int nslices = 0;
};

HostTables build_tables(int d) {
  HostTables ht;
  const int ppw = ppw_for(d);
  const int M1 = d * (d + 1) / 2;
  const int DL = M1 + d + 1;
  const int LW = (DL + 31) / 32 * 32;
  // column metadata
  ht.colmeta.assign(LW, 0);
  for (int c = 0; c < LW; ++c) {
    int first = 0xff, cnt = 0, deg = 0xff;
    if (c < M1) {
      const int canon = M1 - 1 - c;
      int a = 0, base = 0;
      while (base + (d - a) <= canon) {
        base += d - a;
        ++a;
      }
      const int b = a + (canon - base);
      first = a;
      cnt = 1 + (b == a);
      deg = 2;
    } else if (c == M1) {
      deg = 0;
    } else if (c < DL) {
      first = c - M1 - 1;
      cnt = 1;
      deg = 1;
    }
    ht.colmeta[c] = (uint32_t)first | ((uint32_t)cnt << 8) | ((uint32_t)deg << 16);
  }
  // top blocks: len(i1) = degree-2 features with all indices >= i1
  std::vector<int> len(d), boff(d);
  int acc = 0;
  for (int i1 = 0; i1 < d; ++i1) {
    len[i1] = (d - i1) * (d - i1 + 1) / 2;
    boff[i1] = acc;
    acc += len[i1];
  }
  // normaliser map: canonical feature of (i1, g_c) when min(g_c) >= i1
  ht.zmap.assign((size_t)DL * d, -1);
  for (int c = 0; c < DL; ++c)
    for (int i1 = 0; i1 < d; ++i1) {
      int canon = -1;
      if (c < M1) {
        const int first = (int)(ht.colmeta[c] & 0xff);
        if (first >= i1) canon = DL + boff[i1] + len[i1] - 1 - c;
      } else if (c == M1) {
        canon = 1 + i1;
      } else {
        const int a = c - M1 - 1;
        if (a >= i1) canon = 1 + d + idx2(d, i1, a);
      }
      ht.zmap[(size_t)c * d + i1] = canon;
    }
  // pair list: low, normaliser, then top blocks in order of i1
  std::vector<PairMeta> all;
  // low pairs use i1 = d: the staged factor row of ones
  for (int p = 0; p < LW / 32; ++p) all.push_back(PairMeta{kLow, 32 * p, d, 32, 32, 0, 0, 0});
  for (int p = 0; p < LW / 32; ++p) all.push_back(PairMeta{kZmat, 32 * p, 0, 32, 32, 0, 0, 0});
  for (int i1 = 0; i1 < d; ++i1) {
    const int cnt_first = d - i1;  // degree-2 features (i1, b), b >= i1
    for (int p = 0; 32 * p < len[i1]; ++p) {
      PairMeta m{kTop, 32 * p, i1, std::min(32, len[i1] - 32 * p), 32, 0, 0, 0};
      const int rf = (len[i1] - cnt_first) - 32 * p;
      m.rho_from = std::max(0, std::min(32, rf));
      m.out0 = DL + boff[i1] + len[i1] - 1 - 32 * p;
      all.push_back(m);
    }
  }
  // Pack pairs into waves of at most ppw, starting a new wave where the
  // normaliser pairs end (a wave never mixes normaliser and top pairs), then
  // group NW waves into one slice (workgroup).
  const int npairs = (int)all.size();
  int nslices = (npairs + kNW * ppw - 1) / (kNW * ppw);
  std::vector<std::vector<PairMeta>> waves;
  while (true) {
    waves.clear();
    const int target = (npairs + nslices * kNW - 1) / (nslices * kNW);
    std::vector<PairMeta> cur;
    for (int i = 0; i < npairs; ++i) {
      const PairMeta& m = all[i];
      const bool boundary = !cur.empty() && cur.back().kind == kZmat && m.kind != kZmat;
      if ((int)cur.size() == target || boundary) {
        waves.push_back(cur);
        cur.clear();
      }
      cur.push_back(m);
    }
    if (!cur.empty()) waves.push_back(cur);
    if ((int)waves.size() <= nslices * kNW) break;
    ++nslices;
  }
  waves.resize((size_t)nslices * kNW);
  ht.nslices = nslices;
  // empty slots: zero rows (their state stays zero), no run flags
  ht.pairs.assign((size_t)nslices * kNW * ppw, PairMeta{kEmpty, 0, 0, 0, 32, 0, 0, 0});
  ht.slice_ng.assign(nslices, 0);
  for (int s = 0; s < nslices; ++s) {
    int maxcol = 0;
    for (int w = 0; w < kNW; ++w) {
      const std::vector<PairMeta>& wl = waves[(size_t)s * kNW + w];
      PairMeta* wp = &ht.pairs[((size_t)s * kNW + w) * ppw];
      for (size_t t = 0; t < wl.size(); ++t) {
        wp[t] = wl[t];
        maxcol = std::max(maxcol, wl[t].kind == kTop ? wl[t].col0 + 32 : LW);
      }
      // runs: maximal consecutive pairs of one kind and one i1 within the wave
      for (int t = 0; t < ppw; ++t) {
        if (wp[t].kind == kEmpty) continue;
        auto same = [&](int u) { return wp[u].kind == wp[t].kind && wp[u].i1 == wp[t].i1; };
        const bool first = t == 0 || !same(t - 1);
        const bool last = t == ppw - 1 || !same(t + 1);
        wp[t].flags = (first ? kFirstOfRun : 0) | (last ? kLastOfRun : 0);
      }
    }
    ht.slice_ng[s] = maxcol / 8;
  }
  return ht;
}

hipError_t get_tables(int d, hipStream_t s, DeviceTables* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_mfma_mu);
  auto key = std::make_pair(dev, d);
  auto it = g_mfma_tables.find(key);
  if (it != g_mfma_tables.end()) {
    *out = it->second;
    return hipSuccess;
  }
  HostTables ht = build_tables(d);
  DeviceTables dt;
  dt.nslices = ht.nslices;
  auto upload = [&](void** dst, const void* src, size_t bytes) -> hipError_t {
    hipError_t err = hipMalloc(dst, bytes);
    if (err != hipSuccess) return err;
    return hipMemcpyAsync(*dst, src, bytes, hipMemcpyHostToDevice, s);
  };
  std::vector<uint2> packed(ht.pairs.size());
  const int M1 = d * (d + 1) / 2;
  for (size_t i = 0; i < packed.size(); ++i) packed[i] = pack_pair(ht.pairs[i], M1);
  if ((e = upload((void**)&dt.pairs, packed.data(), packed.size() * sizeof(uint2))) != hipSuccess) return e;
  if ((e = upload((void**)&dt.slice_ng, ht.slice_ng.data(), ht.slice_ng.size() * sizeof(int))) != hipSuccess) return e;
  if ((e = upload((void**)&dt.colmeta, ht.colmeta.data(), ht.colmeta.size() * sizeof(uint32_t))) != hipSuccess)
    return e;
  if ((e = upload((void**)&dt.zmap, ht.zmap.data(), ht.zmap.size() * sizeof(int))) != hipSuccess) return e;
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
  g_mfma_tables[key] = dt;
  *out = dt;
  return hipSuccess;
}

int host_nslices(int d) {
  static std::mutex mu;
  static std::map<int, int> cache;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(d);
  if (it != cache.end()) return it->second;
  const int ns = build_tables(d).nslices;
  cache[d] = ns;
  return ns;
}

template <int DK, int DV, int PPW>
hipError_t launch_typed(const u16* q, const u16* k, const u16* v, u16* y, float* S_out, int BH, int n, int C,
                        const DeviceTables& dt, float* partial, hipStream_t s, int qg) {
  using L = MainLds<DK, DV, kNW, PPW>;
  // two workgroups per compute unit pay where there are workgroups for both
  // (at d = 16, B = 64, H = 32: 2.69 -> 2.02 ms; at 256 heads, one per compute
  // unit, the capped registers cost 5%); only where the LDS lets two share one
  const bool dense = DK == 16 && 2 * L::kBytes <= 160 * 1024 && (int64_t)BH * dt.nslices >= 512;
  auto kmain = dense ? prefill_blocks_main<DK, DV, kNW, PPW, DK == 16> : prefill_blocks_main<DK, DV, kNW, PPW, false>;
  hipError_t e = hipFuncSetAttribute((const void*)kmain, hipFuncAttributeMaxDynamicSharedMemorySize, L::kBytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kmain, dim3((unsigned)dt.nslices, (unsigned)BH), dim3(kNW * 64), L::kBytes, s, q, k, v,
                     dt.pairs, dt.slice_ng, dt.colmeta, dt.zmap, partial, S_out, BH, n, C, dt.nslices, qg);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const FinLayout F(DK, DV, C);
  auto kfin = prefill_blocks_finalize<DK, DV>;
  e = hipFuncSetAttribute((const void*)kfin, hipFuncAttributeMaxDynamicSharedMemorySize, F.bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kfin, dim3((unsigned)((n + C - 1) / C), (unsigned)BH), dim3(256), (size_t)F.bytes, s, q, k,
                     v, partial, y, BH, n, C, dt.nslices, 4, qg);
  return hipGetLastError();
}

}  // namespace

bool plan_prefill_blocks(int BH, int n, int dk, int dv, int P, int chunk, MfmaPrefillPlan* plan) {
  if (P != 4 || dk != dv || (dk != 16 && dk != 32)) return false;
  if (chunk != 32 && chunk != 64 && chunk != 128) return false;
  if (n < 1) return false;
  plan->dk = dk;
  plan->dv = dv;
  plan->nslices = host_nslices(dk);
  plan->partial_bytes = sizeof(float) * (size_t)plan->nslices * BH * n * (dv + 1);
  plan->workspace_bytes = plan->partial_bytes;
  return true;
}

hipError_t launch_prefill_blocks(const void* q, const void* k, const void* v, void* y, float* S_out, int BH,
                               int n, int dk, int dv, int P, int chunk, const MfmaPrefillPlan& plan,
                               void* workspace, hipStream_t s, int qg) {
  (void)P;
  (void)dv;
  DeviceTables dt;
  hipError_t e = get_tables(dk, s, &dt);
  if (e != hipSuccess) return e;
  float* partial = (float*)workspace;
  const u16* qq = (const u16*)q;
  const u16* kk = (const u16*)k;
  const u16* vv = (const u16*)v;
  if (dk == 32) return launch_typed<32, 32, 8>(qq, kk, vv, (u16*)y, S_out, BH, n, chunk, dt, partial, s, qg);
  return launch_typed<16, 16, 6>(qq, kk, vv, (u16*)y, S_out, BH, n, chunk, dt, partial, s, qg);
}

}  // namespace sata
