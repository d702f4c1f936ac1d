// Matrix-core (MFMA) causal prefill for bfloat16 q/k/v, P = 4, d_k = d_v = 32, 64-token chunks.
//
// The method (App. A2) as a chunked scan: for chunk c with queries Q_c, keys
// K_c and values V_c,
//     O_c = phi(Q_c) S_{c-1}  +  mask(f_P(Q_c K_c^T / sqrt d)) [V_c | 1]
//     S_c = S_{c-1} + phi(K_c)^T [V_c | 1],      y = O[:, :d_v] / O[:, d_v].
// Both state contractions run on v_mfma_f32_32x32x16_bf16 with the state in
// float32 accumulator registers for the whole sequence.
//
// Factored basis.  Only the low features (degrees 0, 1, 2) are generated; each
// top-degree feature is f = (i1, g) with g a degree-2 feature whose indices are
// all >= i1 (Sec. 2.4 footnote: a monomial of degree p is one coordinate times
// a monomial of degree p-1), and phi_f(x) = x~[i1] phi_g(x) / sqrt(c1), with
// x~ = x d^(-1/4) and c1 the multiplicity of i1 in f.  State rows are held in
// 32 x 32 blocks ("pairs" of 32 feature rows by the 32 value columns):
//   LOW  pair (cg):      rows = low features of column group cg, B = V;
//   TOP  pair (i1, cg):  rows = degree-2 features g of cg, internal state
//                        sum_t phi_g(k_t) k~_t[i1] v_t (= sqrt(c1) S[f]),
//                        B = diag(k~[:, i1]) V; the readout scales its result
//                        by q~[:, i1] and each row by 1/c1 (0 for g with an
//                        index below i1);
//   ZMAT pair (cg):      rows = low features g' of cg, columns j = 0..d-1,
//                        Z[g'][j] = sum_t phi_g'(k_t) k~_t[j].
// The normaliser needs no padded value column: summing over every (j, g') with
// g' of degree p-1, sorted or not, gives
//     sum_j sum_g' q~[j] phi_g'(q) k~[j] phi_g'(k) = s * s^(p-1)/(p-1)! = p s^p/p!,
// so the ZMAT readout with row weight 1/(deg g' + 1), contracted with q~,
// yields every normaliser term of degree >= 1; degree 0 is the token count.
//
// Column order.  Low features are ordered degree-2 first, by decreasing
// smallest index (so the degree-2 features that pair with first index i1 form
// a prefix), then degree 1, then degree 0.  Column group cg holds 32 of them.
// Inside a group, LDS position = row with bits 2 and 3 swapped, which makes
// both MFMA operand reads single vector loads: the readout reads 8 positions
// of one token, the update reads 4 tokens of 4 rows with the transposing
// ds_read_b64_tr_b16.  Token rows are XOR-swizzled in 16-byte units.
//
// Work split.  The host packs the pairs into slices (workgroups of 8 waves x
// 8 pairs) that each cover a range of at most kMaxNC column groups; a slice
// generates the low features of its range.  Inside a slice, runs of pairs
// that share an epilogue (one kind and i1) are packed whole into waves, so
// that no wave carries many runs.  Each slice writes float32 partial
// readouts per token; a second kernel adds them to the intra-chunk term and
// normalises.
//
// Per chunk, each workgroup runs two phases separated by barriers:
//   U: update of S with phi(K_c) and [V | k~] | generate phi(Q_{c+1}), flush O_c
//   R: readout from phi(Q_{c+1}) and S_c      | generate phi(K_{c+1}), stage k~, v
// In U, waves 0-3 update first and waves 4-7 run the vector work first; R
// has two halves, waves 0-3 reading out in the first and 4-7 in the second,
// so the two waves that share a SIMD overlap matrix and vector work.  Each
// run's readout is scaled into the SIMD's float32 sums in LDS.  Within the
// matrix work, the next pair's operands are read while the current pair's
// MFMAs run.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <type_traits>
#include <vector>

#include "device_common.hpp"
#include "prefill_mfma.hpp"
#include "table.hpp"

namespace sata {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16;

constexpr int kC = 64;        // tokens per chunk
static_assert(kC == 64, "the finalize splits a chunk into 16 score tiles over 4 waves");
constexpr int kNW = 8;        // waves per workgroup
constexpr int kMaxNC = 9;     // column groups per slice
constexpr int kTS = 68;       // floats per row of the transposed float32 tiles
constexpr int kTSb = 72;      // bf16 per row of the transposed bf16 tiles

// Slot descriptor bits.
enum : uint32_t { kNone = 0, kLow = 1, kZmat = 2, kTop = 3 };
constexpr uint32_t kFirst = 1u << 13, kLast = 1u << 14, kFac = 1u << 15;
// An empty slot runs as a LOW pair whose readout is dropped; it is not exported.
constexpr uint32_t kEmpty = 1u << 16;
// Slots with row factors (kFac) index a per-slice table of kMaxFac rows of 32
// factors, held in LDS for the whole kernel.
constexpr int kMaxFac = 32;
__host__ __device__ constexpr uint32_t make_slot(uint32_t kind, int cgl, int i1, uint32_t flags, int fi = 0) {
  return kind | ((uint32_t)cgl << 2) | ((uint32_t)i1 << 6) | flags | ((uint32_t)fi << 17);
}
__device__ __forceinline__ uint32_t s_kind(uint32_t m) { return m & 3u; }
__device__ __forceinline__ int s_cgl(uint32_t m) { return (int)((m >> 2) & 15u); }
__device__ __forceinline__ int s_i1(uint32_t m) { return (int)((m >> 6) & 127u); }
__device__ __forceinline__ int s_fi(uint32_t m) { return (int)((m >> 17) & (kMaxFac - 1)); }

// ------------------------------------------------------------ low features

template <int DK>
struct Low {
  static constexpr int M2 = DK * (DK + 1) / 2;  // degree 2
  static constexpr int NL = M2 + DK + 1;        // degrees 0..2
  static constexpr int NCG = (NL + 31) / 32;    // column groups
  static constexpr int NLP = NCG * 32;
};

struct LowFeat {
  int deg, a, b;  // deg -1: padding; deg 2: a <= b; deg 1: a
};

// Low feature L in the kernel's column order.
template <int DK>
__host__ __device__ constexpr LowFeat low_feat(int L) {
  if (L < Low<DK>::M2) {
    int m = DK - 1, base = 0;
    while (base + (DK - m) <= L) {
      base += DK - m;
      --m;
    }
    return LowFeat{2, m, m + (L - base)};
  }
  L -= Low<DK>::M2;
  if (L < DK) return LowFeat{1, L, 0};
  if (L == DK) return LowFeat{0, 0, 0};
  return LowFeat{-1, 0, 0};
}

__host__ __device__ constexpr int swap23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// Value of low feature L from the unscaled coordinates x: the scale
// d^(-p/4) of a degree-p feature is applied once, to its first factor, so
// features that share a first index share that product.
template <int DK>
struct FeatScale {
  static constexpr float deg1 = (float)(1.0 / 2.378414230005442);  // d^(-1/4) at d = 32
  static constexpr float deg2 = (float)(1.0 / 5.656854249492381);  // d^(-1/2)
  static constexpr float deg2sq = (float)(0.70710678118654752 / 5.656854249492381);  // with 1/sqrt(2!)
};
template <int DK, int L>
__device__ __forceinline__ float low_value(const float (&x)[DK]) {
  static_assert(DK == 32, "scale constants are for d = 32");
  constexpr LowFeat f = low_feat<DK>(L);
  if constexpr (f.deg == 2) {
    if constexpr (f.a == f.b)
      return (x[f.a] * FeatScale<DK>::deg2sq) * x[f.a];
    else
      return (x[f.a] * FeatScale<DK>::deg2) * x[f.b];
  } else if constexpr (f.deg == 1) {
    return x[f.a] * FeatScale<DK>::deg1;
  } else if constexpr (f.deg == 0) {
    return 1.0f;
  } else {
    return 0.0f;
  }
}

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

// One generation unit: LDS positions 8k..8k+7 of column group cg (U = 4 cg + k).
template <int DK, int U>
__device__ __forceinline__ uint4 gen_unit(const float (&x)[DK]) {
  constexpr int base = 32 * (U / 4);
  constexpr int p0 = 8 * (U % 4);
  uint4 r;
  r.x = pack2(low_value<DK, base + swap23(p0 + 0)>(x), low_value<DK, base + swap23(p0 + 1)>(x));
  r.y = pack2(low_value<DK, base + swap23(p0 + 2)>(x), low_value<DK, base + swap23(p0 + 3)>(x));
  r.z = pack2(low_value<DK, base + swap23(p0 + 4)>(x), low_value<DK, base + swap23(p0 + 5)>(x));
  r.w = pack2(low_value<DK, base + swap23(p0 + 6)>(x), low_value<DK, base + swap23(p0 + 7)>(x));
  return r;
}

// Phi tiles: token rows kPhiStride bytes apart (64 mod 256); column group cg
// occupies bytes [64 cg, 64 cg + 64) of a row as four 16-byte units k, and unit
// k of token t is stored at unit k ^ ((t / 4) % 4).  Both MFMA operand reads
// and the generation writes are then free of bank conflicts, and the column-
// group part of every address is the wave-uniform 64 cg.
constexpr int kPhiStride = kMaxNC * 64;
constexpr int kXS = 36;  // floats per token row of the staged x~ tiles
constexpr int kPS = 36;  // floats per token row of the per-SIMD sums and of the slice partials
                         // (value columns, then the normaliser; 16-byte aligned rows)

// A unit whose 8 features are all degree 0 or padding holds the same values
// for every token and chunk: it is written once, not generated.
template <int DK, int U>
__host__ __device__ constexpr bool unit_const() {
  for (int i = 0; i < 8; ++i)
    if (low_feat<DK>(32 * (U / 4) + swap23(8 * (U % 4) + i)).deg > 0) return false;
  return true;
}
template <int DK, int U, int NU>
__device__ __forceinline__ void put_const_units(char* row, int ulo, int uhi, int sw16) {
  if constexpr (U < NU) {
    if constexpr (unit_const<DK, U>()) {
      if (U >= ulo && U < uhi) {
        const float x0[DK] = {};
        *(uint4*)(row + 64 * (U / 4) + ((16 * (U % 4)) ^ sw16)) = gen_unit<DK, U>(x0);
      }
    }
    put_const_units<DK, U + 1, NU>(row, ulo, uhi, sw16);
  }
}

// Generation units of one wave: absolute units U = W, W + kNW, ... inside the
// slice's range [ulo, uhi), constant units excepted.  row points at this lane's token row shifted back
// by the slice's first column group; sw16 = 16 ((t / 4) % 4).
template <int DK, int U, int NU>
__device__ __forceinline__ void gen_chain(const float (&x)[DK], int ulo, int uhi, char* row, int sw16) {
  if constexpr (U < NU) {
    if constexpr (!unit_const<DK, U>())
      if (U >= ulo && U < uhi) *(uint4*)(row + 64 * (U / 4) + ((16 * (U % 4)) ^ sw16)) = gen_unit<DK, U>(x);
    gen_chain<DK, U + kNW, NU>(x, ulo, uhi, row, sw16);
  }
}
// The same with the unit range [ULO, UHI) known at compile time, so that only
// the coordinates the wave's units use are unpacked.
template <int DK, int U, int NU, int ULO, int UHI>
__device__ __forceinline__ void gen_chain_ct(const float (&x)[DK], char* row, int sw16) {
  if constexpr (U < NU) {
    if constexpr (U >= ULO && U < UHI && !unit_const<DK, U>())
      *(uint4*)(row + 64 * (U / 4) + ((16 * (U % 4)) ^ sw16)) = gen_unit<DK, U>(x);
    gen_chain_ct<DK, U + kNW, NU, ULO, UHI>(x, row, sw16);
  }
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int DK>
struct Lds {
  static constexpr int PHIQ = 0;
  static constexpr int PHIK = PHIQ + kC * kPhiStride;
  static constexpr int XQ = PHIK + kC * kPhiStride;  // float [kC][kXS]: q~ of the chunk being read out
  static constexpr int KT = XQ + kC * kXS * 4;       // float [DK][kTS]: k~ transposed
  static constexpr int VT = KT + DK * kTS * 4;       // float [DK][kTS]: v transposed
  static constexpr int KTB = VT + DK * kTS * 4;      // bf16 [DK][kTSb]
  static constexpr int VTB = KTB + DK * kTSb * 2;
  static constexpr int PART = VTB + DK * kTSb * 2;   // 4 x float [kC][kPS]: per-SIMD readout sums
  // raw bf16 tiles of the next chunk, piece-major: the 16-byte piece j (8
  // coordinates) of token t at byte (kC j + t) 16
  static constexpr int RQ = PART + 4 * kC * kPS * 4;  // raw q of the next chunk
  static constexpr int RK = RQ + kC * DK * 2;         // raw k, v of the next chunk
  static constexpr int RV = RK + kC * DK * 2;
  static constexpr int FAC = RV + kC * DK * 2;  // float [kMaxFac][32]: this slice's readout row factors
  static constexpr int BYTES = FAC + kMaxFac * 32 * 4;
};

// ------------------------------------------------------------ main kernel

// The value width equals the MFMA's 32 rows: the readout's M index and the
// update's N index run over the d_v = 32 value columns.
template <int DK, int PPW>
__global__ void __launch_bounds__(kNW * 64, 1)
prefill_mfma_main(const u16* __restrict__ q, const u16* __restrict__ k, const u16* __restrict__ v,
                  const int4* __restrict__ slices, const uint32_t* __restrict__ slots,
                  const float* __restrict__ facs, const int* __restrict__ prep_idx,
                  const float* __restrict__ prep_scale, const int* __restrict__ low_idx,
                  float* __restrict__ partial, float* __restrict__ S_out, int BH, int n, int nslices, int qg) {
  constexpr int DV = DK;
  static_assert(DK == 32, "value columns must fill the 32-row MFMA tile");
  constexpr int E = DV + 1;
  constexpr int EP = kPS;  // per-SIMD sum rows: values, then one normaliser term per lane half
  using L = Lds<DK>;
  static_assert(L::BYTES <= 160 * 1024, "LDS budget");
  constexpr int NU = 4 * Low<DK>::NCG;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* const phiq = smem + L::PHIQ;
  char* const phik = smem + L::PHIK;
  float* const xq = (float*)(smem + L::XQ);
  float* const kt = (float*)(smem + L::KT);
  float* const vt = (float*)(smem + L::VT);
  u16* const ktb = (u16*)(smem + L::KTB);
  u16* const vtb = (u16*)(smem + L::VTB);
  float* const part = (float*)(smem + L::PART);

  const int tid = threadIdx.x;
  const int lane_id = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Slice-major workgroup order: the hardware deals workgroups to the 8 XCDs
  // in turn, so with heads innermost every XCD gets every slice kind (the
  // kinds differ in cost) instead of a fixed one.  The division runs on the
  // vector unit; reading its result back into scalar registers keeps the head
  // offsets and every pointer derived from them scalar, instead of in spilled
  // vector registers.
  const int slice = __builtin_amdgcn_readfirstlane((int)(blockIdx.x / (unsigned)BH));
  const int64_t bh = __builtin_amdgcn_readfirstlane((int)(blockIdx.x - (unsigned)slice * BH));
  const int4 sl = slices[slice];
  const int lo = __builtin_amdgcn_readfirstlane(sl.x);
  const int nc = __builtin_amdgcn_readfirstlane(sl.y);
  const float dscale = 1.0f / sqrtf(sqrtf((float)DK));

  uint32_t meta[PPW];
#pragma unroll
  for (int p = 0; p < PPW; ++p)
    meta[p] = __builtin_amdgcn_readfirstlane(slots[((int64_t)slice * kNW + wave) * PPW + p]);

  const u16* qh_ = q + bh * (int64_t)qg * n * DK;  // qg query heads per key/value head
  const u16* kh_ = k + bh * (int64_t)n * DK;
  const u16* vh_ = v + bh * (int64_t)n * DV;
  const int nch = (n + kC - 1) / kC;

  // prologue: raw q(0); U(-1) loads raw k(0), v(0)
  {
    const int pc0 = tid;  // 256 pieces of 16 bytes
    if (pc0 < kC * DK / 8) {
      const int tok = pc0 / (DK / 8);
      uint4 w = {0u, 0u, 0u, 0u};
      if (tok < n) w = *(const uint4*)(qh_ + (int64_t)tok * DK + (pc0 - tok * (DK / 8)) * 8);
      *(uint4*)(smem + L::RQ + (kC * (pc0 - tok * (DK / 8)) + tok) * 16) = w;
    }
  }
  // this slice's row factors
  if (tid < kMaxFac * 32 / 4)
    ((uint4*)(smem + L::FAC))[tid] = ((const uint4*)(facs + (int64_t)slice * kMaxFac * 32))[tid];
  // U(-1) runs the update on zero operands: clear phi(K), the k~ and v tiles
  // and the partial regions
  for (int i = tid; i < kC * kPhiStride / 16; i += kNW * 64) ((uint4*)phik)[i] = uint4{0u, 0u, 0u, 0u};
  for (int i = tid; i < (L::RQ - L::KT) / 16; i += kNW * 64) ((uint4*)(smem + L::KT))[i] = uint4{0u, 0u, 0u, 0u};
  __syncthreads();
  // the constant feature units of both phi tiles (waves 0 and 1: one token row per lane)
  if (wave < 2)
    put_const_units<DK, 0, NU>((wave == 0 ? phiq : phik) + lane_id * kPhiStride - 64 * lo, 4 * lo, 4 * (lo + nc),
                               16 * ((lane_id >> 2) & 3));

  f32x16 S[PPW];
#pragma unroll
  for (int p = 0; p < PPW; ++p)
#pragma unroll
    for (int j = 0; j < 16; ++j) S[p][j] = 0.0f;
  __syncthreads();

  // Phases in order U(-1), R(0), U(0), R(1), ..., U(nch-1).  The update is
  // straight-line code in every iteration (in U(-1) its operands are zero) so
  // the state accumulators stay in place.  Each vector half loads what it
  // needs from global memory itself; the other wave of its SIMD, in its matrix
  // half meanwhile, covers the latency.
#pragma unroll 1
  for (int c = -1; c < nch; ++c) {
    // Slot descriptors and the factor table pass through an empty asm each
    // iteration so that per-slot addresses and factor loads stay in the loop
    // (hoisted out of it they would not fit in registers).
    uint32_t mt[PPW];
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      mt[p] = meta[p];
      asm volatile("" : "+s"(mt[p]));
    }
    // Each use takes the descriptor through another empty asm, so values
    // derived from it are formed where they are used rather than kept in
    // scalar registers across the iteration.
    auto M = [&](int p) __attribute__((always_inline)) -> uint32_t {
      uint32_t m = mt[p];
      asm volatile("" : "+s"(m));
      return m;
    };
    // The lane index likewise, so per-lane addresses are recomputed each
    // iteration instead of being kept (and spilled) across the loop.
    int lane = lane_id;
    asm volatile("" : "+v"(lane));
    const int l31 = lane & 31;
    const int qh = lane >> 5;  // which 8 of the 16 K slots
    // Next-phase tile loads: one 16-byte piece (8 coordinates of one token) per
    // lane of [0, 32): piece 32 wave + lane of the 64-token tile; zero beyond n.
    auto load_piece = [&](const u16* base, int c, int lid) __attribute__((always_inline)) -> uint4 {
      const int pc = 32 * wave + lid;
      const int tok = pc / (DK / 8);
      const int g = c * kC + tok;
      uint4 r = {0u, 0u, 0u, 0u};
      const u16* const cb = base + (int64_t)c * kC * DK;  // wave-uniform
      if (lid < 32 && pc < kC * DK / 8 && c < nch && g < n) r = *(const uint4*)(cb + (tok * DK + (pc - tok * (DK / 8)) * 8));
      return r;
    };
    auto store_piece = [&](int tile_off, int lid, uint4 w) __attribute__((always_inline)) {
      const int pc = 32 * wave + lid;
      const int tok = pc / (DK / 8);
      if (lid < 32 && pc < kC * DK / 8)
        *(uint4*)(smem + tile_off + (kC * (pc - tok * (DK / 8)) + tok) * 16) = w;
    };
    // the unscaled coordinates of this lane's token from a raw tile
    auto unpack_row = [&](int tile_off, float (&x)[DK]) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < DK / 8; ++i) {
        const uint4 w = *(const uint4*)(smem + tile_off + (kC * i + lane) * 16);
        x[8 * i + 0] = bf_lo(w.x);
        x[8 * i + 1] = bf_hi(w.x);
        x[8 * i + 2] = bf_lo(w.y);
        x[8 * i + 3] = bf_hi(w.y);
        x[8 * i + 4] = bf_lo(w.z);
        x[8 * i + 5] = bf_hi(w.z);
        x[8 * i + 6] = bf_lo(w.w);
        x[8 * i + 7] = bf_hi(w.w);
      }
    };
    // coordinates [4 wave, 4 wave + 4) of this lane's token from a raw tile
    auto quad = [&](int tile_off) __attribute__((always_inline)) -> uint2 {
      return *(const uint2*)(smem + tile_off + (kC * (wave >> 1) + lane) * 16 + 8 * (wave & 1));
    };

    // phi rows of the 64 tokens (lane = token); wave w writes the slice's units w, w + 8, ...
    const int sw16 = 16 * ((lane >> 2) & 3);
    // Slices whose column groups start at 0 or end at the last group (the
    // d = 32 plan has only these) generate with compile-time unit ranges; a
    // slice starting at 0 may write groups past its own, inside its rows.
    constexpr int kLoB = Low<DK>::NCG - kMaxNC;
    const int gen_class = (lo == 0 && nc <= kMaxNC) ? 0 : (lo == kLoB && nc == kMaxNC) ? 1 : 2;
    auto gen_wave = [&](auto W, int tile_off, char* row) __attribute__((always_inline)) {
      constexpr int w = decltype(W)::value;
      float x[DK];
      unpack_row(tile_off, x);
      if (gen_class == 0)
        gen_chain_ct<DK, w, NU, 0, 4 * kMaxNC>(x, row, sw16);
      else if (gen_class == 1)
        gen_chain_ct<DK, w, NU, 4 * kLoB, 4 * (kLoB + kMaxNC)>(x, row, sw16);
      else
        gen_chain<DK, w, NU>(x, 4 * lo, 4 * (lo + nc), row, sw16);
    };
    auto generate = [&](auto lower, int tile_off, char* dst) __attribute__((always_inline)) {
      char* row = dst + lane * kPhiStride - 64 * lo;
      if constexpr (decltype(lower)::value) {
        switch (wave) {
          case 0: gen_wave(std::integral_constant<int, 0>{}, tile_off, row); break;
          case 1: gen_wave(std::integral_constant<int, 1>{}, tile_off, row); break;
          case 2: gen_wave(std::integral_constant<int, 2>{}, tile_off, row); break;
          default: gen_wave(std::integral_constant<int, 3>{}, tile_off, row); break;
        }
      } else {
        switch (wave) {
          case 4: gen_wave(std::integral_constant<int, 4>{}, tile_off, row); break;
          case 5: gen_wave(std::integral_constant<int, 5>{}, tile_off, row); break;
          case 6: gen_wave(std::integral_constant<int, 6>{}, tile_off, row); break;
          default: gen_wave(std::integral_constant<int, 7>{}, tile_off, row); break;
        }
      }
    };

    // Per-lane parts of the operand addresses (the column group adds 64 cg).
    // readout: token 32 t + l31, unit 2 h + qh
    const int rd_base = l31 * kPhiStride;
    const int rd_h0 = 16 * ((0 + qh) ^ ((l31 >> 2) & 3));
    const int rd_h1 = 16 * ((2 + qh) ^ ((l31 >> 2) & 3));
    // update: tokens 16 s + 8 qq + 4 r + j16 / 4, unit 2 hh + (j16 & 1), byte 8 ((j16 >> 1) & 1)
    int up_base[2];
    {
      const int grp = lane >> 4, hh = grp & 1, qq = grp >> 1, j16 = lane & 15;
  #pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int tok = 8 * qq + 4 * r + (j16 >> 2);
        up_base[r] = tok * kPhiStride + 16 * ((2 * hh + (j16 & 1)) ^ ((2 * qq + r) & 3)) + 8 * ((j16 >> 1) & 1);
      }
    }


    // ================= phase U(c): update | phi(Q_{c+1}) and q~(c+1), flush O(c)
    {
      const int t0 = c * kC;
      const int cn = min(kC, n - t0);
      auto vector_u = [&](auto lower) __attribute__((always_inline)) {
        // raw k(c+1) in lanes [0, 32), raw v(c+1) in lanes [32, 64)
        const uint4 pkv = (lane < 32) ? load_piece(kh_, c + 1, lane) : load_piece(vh_, c + 1, lane - 32);
        if (c >= 0) {
          // the four per-SIMD readout sums of chunk c -> this slice's partial
          // (rows of kPS floats: 32 values, the normaliser), clearing them; 8
          // threads per token, 4 value columns each, the first also the normaliser
          // (every lane reads its token's normaliser pair, so that no branch
          // splits the reads; the first lane of the token uses and clears it)
          // (from a laundered thread index, so these offsets are formed here
          // each iteration rather than kept, or spilled, across the loop)
          int ftid = tid;
          asm volatile("" : "+v"(ftid));
          const int tok = ftid >> 3;
          const int cq = 4 * (ftid & 7);
          float4 w[4];
          float2 zz[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float* pr = part + (r * kC + tok) * EP;
            w[r] = *(const float4*)(pr + cq);
            zz[r] = *(const float2*)(pr + DV);
          }
          float4 o = {0.0f, 0.0f, 0.0f, 0.0f};
          float z = 0.0f;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float* pr = part + (r * kC + tok) * EP;
            o.x += w[r].x;
            o.y += w[r].y;
            o.z += w[r].z;
            o.w += w[r].w;
            z += zz[r].x + zz[r].y;
            *(float4*)(pr + cq) = float4{0.0f, 0.0f, 0.0f, 0.0f};
            if (cq == 0) *(float2*)(pr + DV) = float2{0.0f, 0.0f};
          }
          if (tok < cn) {
            // a wave-uniform row base and a 32-bit lane offset
            float* const dst = partial + (((int64_t)slice * BH + bh) * n + t0) * kPS;
            *(float4*)(dst + (tok * kPS + cq)) = o;
            if (cq == 0) dst[tok * kPS + DV] = z;
          }
        }
        // (the flush first: its LDS reads then do not queue behind the feature
        // writes; kept apart so that their registers do not overlap)
        __builtin_amdgcn_sched_barrier(0);
        if (c + 1 < nch) {
          generate(lower, L::RQ, phiq);
          const uint2 qd = quad(L::RQ);
          *(float4*)(xq + lane * kXS + 4 * wave) =
              float4{bf_lo(qd.x) * dscale, bf_hi(qd.x) * dscale, bf_lo(qd.y) * dscale, bf_hi(qd.y) * dscale};
        }
        if (lane < 32)
          store_piece(L::RK, lane, pkv);
        else
          store_piece(L::RV, lane - 32, pkv);
      };
      if (wave >= 4) vector_u(std::false_type{});
      {
        // ---- update: S += phi(K)^T B, 4 key steps of 16 tokens.  Software
        // pipeline over the slots: slot p+1's phi(K) operands are read while
        // slot p's MFMAs run, and a new run's B is built behind them.
        bf16x8 Bk[4];
        auto build_b = [&](uint32_t m, bf16x8 (&Bk)[4]) __attribute__((always_inline)) {
          // one uniform branch on the kind, so that each case is a single block
          // whose LDS reads the scheduler can issue together
          const uint32_t kind = s_kind(m);
          if (kind == kTop) {
            const float* kr = kt + s_i1(m) * kTS + 8 * qh;
            const float* vr = vt + l31 * kTS + 8 * qh;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
              const float4 k0 = *(const float4*)(kr + 16 * s), k1 = *(const float4*)(kr + 16 * s + 4);
              const float4 v0 = *(const float4*)(vr + 16 * s), v1 = *(const float4*)(vr + 16 * s + 4);
              uint4 w;
              w.x = pack2(k0.x * v0.x, k0.y * v0.y);
              w.y = pack2(k0.z * v0.z, k0.w * v0.w);
              w.z = pack2(k1.x * v1.x, k1.y * v1.y);
              w.w = pack2(k1.z * v1.z, k1.w * v1.w);
              Bk[s] = __builtin_bit_cast(bf16x8, w);
            }
          } else {
            const u16* src = ((kind == kLow) ? vtb : ktb) + l31 * kTSb + 8 * qh;
#pragma unroll
            for (int s = 0; s < 4; ++s) Bk[s] = __builtin_bit_cast(bf16x8, *(const uint4*)(src + 16 * s));
          }
        };
        auto load_a = [&](uint32_t m, bf16x8 (&A)[4]) __attribute__((always_inline)) {
          const char* pa = phik + up_base[0] + 64 * s_cgl(m);
          const char* pb = phik + up_base[1] + 64 * s_cgl(m);
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            const bf16x4 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (__attribute__((address_space(3))) bf16x4*)(pa + s * 16 * kPhiStride));
            const bf16x4 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (__attribute__((address_space(3))) bf16x4*)(pb + s * 16 * kPhiStride));
            A[s] = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
          }
        };
        // B of the next run is built two slots ahead (into Bn), so its reads
        // and arithmetic overlap two slots' MFMAs.
        bf16x8 Ac[4], Bn[4];
        load_a(M(0), Ac);
        build_b(M(0), Bk);  // the first slot of a wave always starts a run
        if (PPW > 1 && (M(PPW > 1 ? 1 : 0) & kFirst)) build_b(M(PPW > 1 ? 1 : 0), Bn);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int p = 0; p < PPW; ++p) {
          constexpr int kLastSlot = PPW - 1;
          bf16x8 An[4];
          if (p + 1 < PPW) load_a(M(p + 1 < PPW ? p + 1 : p), An);
#pragma unroll
          for (int s = 0; s < 4; ++s) S[p] = mfma32(Ac[s], Bk[s], S[p]);
          if (p + 1 < PPW) {
            const uint32_t m1 = M(p + 1 < PPW ? p + 1 : kLastSlot);
            if (m1 & kFirst) {
#pragma unroll
              for (int s = 0; s < 4; ++s) Bk[s] = Bn[s];
            }
            if (p + 2 < PPW) {
              const uint32_t m2 = M(p + 2 < PPW ? p + 2 : kLastSlot);
              if (m2 & kFirst) build_b(m2, Bn);
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) Ac[s] = An[s];
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      if (wave < 4) vector_u(std::true_type{});
      __syncthreads();
    }
    if (c + 1 >= nch) break;

    // ================= phase R(c+1): readout | phi(K_{c+1}), k~ and v transposed
    {
      const int cr = c + 1;
      auto vector_r = [&](auto lower) __attribute__((always_inline)) {
        const uint4 pq = load_piece(qh_, cr + 1, lane);  // raw q(c+2), lanes [0, 32)
        generate(lower, L::RK, phik);
        // k~ and v transposed: wave w takes dims [4 w, 4 w + 4) of every token
        const uint2 kd = quad(L::RK);
        const uint2 vd = quad(L::RV);
        const float kx[4] = {bf_lo(kd.x) * dscale, bf_hi(kd.x) * dscale, bf_lo(kd.y) * dscale, bf_hi(kd.y) * dscale};
        const uint32_t vb[4] = {vd.x & 0xffffu, vd.x >> 16, vd.y & 0xffffu, vd.y >> 16};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int dcol = 4 * wave + e;
          kt[dcol * kTS + lane] = kx[e];
          ktb[dcol * kTSb + lane] = f32_to_bf16(kx[e]).bits;
          vt[dcol * kTS + lane] = __uint_as_float(vb[e] << 16);
          vtb[dcol * kTSb + lane] = (u16)vb[e];
        }
        store_piece(L::RQ, lane, pq);
      };
      auto readout = [&]() __attribute__((always_inline)) {
        // O^T (value columns x tokens) = S^T phi(Q)^T per pair for both 32-token
        // tiles; each run's sum is scaled into this SIMD's sums in LDS (which
        // both waves of the SIMD add to, a half apart)
        float* const pr = part + (wave & 3) * kC * EP;
        f32x16 R[2];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int j = 0; j < 16; ++j) R[t][j] = 0.0f;
        // Software pipeline over the slots: while slot p's MFMAs run, slot p+1's
        // phi(Q) operands and row factors are read and its state converted.
        auto load_b = [&](uint32_t m, uint4 (&b)[4]) __attribute__((always_inline)) {
          const char* pq = phiq + rd_base + 64 * s_cgl(m);
          b[0] = *(const uint4*)(pq + rd_h0);
          b[1] = *(const uint4*)(pq + rd_h1);
          b[2] = *(const uint4*)(pq + 32 * kPhiStride + rd_h0);
          b[3] = *(const uint4*)(pq + 32 * kPhiStride + rd_h1);
        };
        auto load_fac = [&](uint32_t m, float4 (&fw)[4]) __attribute__((always_inline)) {
          if (m & kFac) {
            const float* fr = (const float*)(smem + L::FAC) + s_fi(m) * 32 + 4 * qh;
#pragma unroll
            for (int g = 0; g < 4; ++g) fw[g] = *(const float4*)(fr + 8 * g);
          }
        };
        auto convert = [&](const f32x16& Sp, uint32_t m, const float4 (&fw)[4], bf16x8 (&A)[2])
            __attribute__((always_inline)) {
          if (m & kFac) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const float4 fa = fw[2 * h], fb = fw[2 * h + 1];
              uint4 w;
              w.x = pack2(Sp[8 * h + 0] * fa.x, Sp[8 * h + 1] * fa.y);
              w.y = pack2(Sp[8 * h + 2] * fa.z, Sp[8 * h + 3] * fa.w);
              w.z = pack2(Sp[8 * h + 4] * fb.x, Sp[8 * h + 5] * fb.y);
              w.w = pack2(Sp[8 * h + 6] * fb.z, Sp[8 * h + 7] * fb.w);
              A[h] = __builtin_bit_cast(bf16x8, w);
            }
          } else {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              uint4 w;
              w.x = pack2(Sp[8 * h + 0], Sp[8 * h + 1]);
              w.y = pack2(Sp[8 * h + 2], Sp[8 * h + 3]);
              w.z = pack2(Sp[8 * h + 4], Sp[8 * h + 5]);
              w.w = pack2(Sp[8 * h + 6], Sp[8 * h + 7]);
              A[h] = __builtin_bit_cast(bf16x8, w);
            }
          }
        };
        // a zero operand the compiler cannot see through
        bf16x8 zop = {};
        asm volatile("" : "+v"(zop));
        uint4 bc[4];
        bf16x8 Ac[2];
        {
          float4 fw[4];
          load_b(M(0), bc);
          load_fac(M(0), fw);
          convert(S[0], M(0), fw, Ac);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int p = 0; p < PPW; ++p) {
          const uint32_t m = M(p);
          // the next slot's row factors are read before this slot's MFMAs, so
          // that its conversion does not wait for them
          float4 fw[4];
          if (p + 1 < PPW) load_fac(M(p + 1 < PPW ? p + 1 : p), fw);
          R[0] = mfma32(Ac[0], __builtin_bit_cast(bf16x8, bc[0]), R[0]);
          R[0] = mfma32(Ac[1], __builtin_bit_cast(bf16x8, bc[1]), R[0]);
          R[1] = mfma32(Ac[0], __builtin_bit_cast(bf16x8, bc[2]), R[1]);
          R[1] = mfma32(Ac[1], __builtin_bit_cast(bf16x8, bc[3]), R[1]);
          uint4 bn[4];
          bf16x8 An[2];
          if (p + 1 < PPW) load_b(M(p + 1), bn);
          if (m & kLast) {
            // run epilogue into this SIMD's sums: scale by q~[:, i1] (TOP), 1
            // (LOW) or contract with q~ (ZMAT).  Each lane owns its entries.
            // (uniform branches on the kind outside the tile loops, so that each
            // case is one block whose LDS accesses can be issued together)
            const uint32_t kind = s_kind(m);
            if (kind == kZmat) {
#pragma unroll
              for (int t = 0; t < 2; ++t) {
                const float* qrow = xq + (32 * t + l31) * kXS;
                float z = 0.0f;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                  const float4 w = *(const float4*)(qrow + 8 * g + 4 * qh);
                  z += w.x * R[t][4 * g + 0] + w.y * R[t][4 * g + 1] + w.z * R[t][4 * g + 2] + w.w * R[t][4 * g + 3];
                }
                pr[(32 * t + l31) * EP + DV + qh] += z;
              }
            } else if (!(m & kEmpty)) {
              // q~[:, i1] is read for LOW runs too (i1 = 0) and replaced by 1,
              // so that no branch splits the reads; each tile's sums are read
              // together, updated, then written
              const bool top = kind == kTop;
              const int i1 = s_i1(m);
              float sc[2];
#pragma unroll
              for (int t = 0; t < 2; ++t) sc[t] = xq[(32 * t + l31) * kXS + i1];
#pragma unroll
              for (int t = 0; t < 2; ++t) {
                const float f = top ? sc[t] : 1.0f;
                float4* o = (float4*)(pr + (32 * t + l31) * EP + 4 * qh);
                float4 cur[4];
#pragma unroll
                for (int g = 0; g < 4; ++g) cur[g] = o[2 * g];
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                  cur[g].x += f * R[t][4 * g + 0];
                  cur[g].y += f * R[t][4 * g + 1];
                  cur[g].z += f * R[t][4 * g + 2];
                  cur[g].w += f * R[t][4 * g + 3];
                }
#pragma unroll
                for (int g = 0; g < 4; ++g) o[2 * g] = cur[g];
              }
            }
            // restart the sums on the matrix core (a zero product) instead of
            // 16 vector moves
#pragma unroll
            for (int t = 0; t < 2; ++t) R[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(zop, zop, f32x16{}, 0, 0, 0);
          }
          if (p + 1 < PPW) {
            convert(S[p + 1 < PPW ? p + 1 : p], M(p + 1 < PPW ? p + 1 : p), fw, An);
#pragma unroll
            for (int i = 0; i < 4; ++i) bc[i] = bn[i];
            Ac[0] = An[0];
            Ac[1] = An[1];
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      };
      // two halves with a barrier between: waves 0-3 read out first, 4-7 second
      if (wave < 4)
        readout();
      else
        vector_r(std::false_type{});
      __syncthreads();
      if (wave < 4)
        vector_r(std::true_type{});
      else
        readout();
      __syncthreads();
    }
  }

  // ---- state export in the canonical feature order (library layout)
  if (S_out != nullptr) {
    const int l31 = lane_id & 31;
    const int qh = lane_id >> 5;
    constexpr int64_t D = (int64_t)(DK + 1) * (DK + 2) * (DK + 3) / 6;
    float* So = S_out + bh * D * E;
#pragma unroll
    for (int p = 0; p < PPW; ++p) {
      const uint32_t m = meta[p];
      const uint32_t kind = s_kind(m);
      if (m & kEmpty) continue;
      const int Lbase = 32 * (lo + s_cgl(m));
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int row = 8 * (j >> 2) + 4 * qh + (j & 3);
        const int Lf = Lbase + row;
        if (kind == kLow) {
          const int ci = low_idx[Lf];
          if (ci >= 0) So[(int64_t)ci * E + l31] = S[p][j];
        } else if (kind == kTop) {
          const int i1 = s_i1(m);
          const int ci = (Lf < Low<DK>::M2) ? prep_idx[i1 * Low<DK>::NLP + Lf] : -1;
          if (ci >= 0) So[(int64_t)ci * E + l31] = S[p][j] * prep_scale[i1 * Low<DK>::NLP + Lf];
        } else {
          const int ci = prep_idx[l31 * Low<DK>::NLP + Lf];
          if (ci >= 0) So[(int64_t)ci * E + DV] = S[p][j] * prep_scale[l31 * Low<DK>::NLP + Lf];
        }
      }
    }
    if (slice == 0 && tid == 0) So[DV] = (float)n;  // degree 0: the token count
  }
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
    op = 0;  // the weights overwrite Q and K once the scores are in registers
    ov = (C * ps > 2 * C * qs) ? C * ps : 2 * C * qs;
    oz = ov + DV * vs;
    orow = oz + C * 4;
    bytes = orow + C * (C / 16) * 4;
  }
};

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int DK, int DV>
__global__ void __launch_bounds__(256, 8)
prefill_mfma_finalize(const u16* __restrict__ q, const u16* __restrict__ k, const u16* __restrict__ v,
                      const float* __restrict__ partial, u16* __restrict__ y, int BH, int n, int C, int nslices,
                      int P, int PS, int qg) {
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

  // The slices' partials this thread adds in the epilogues are loaded first,
  // so that their latency overlaps the staging and the scores: for each of
  // its two output tiles (computed transposed, so a lane holds 4 consecutive
  // value columns of one query) one float4 per slice, and (threads < C) one
  // normaliser.
  constexpr int kOutTilesPerWave = 2;  // (64 / 16) x (32 / 16) tiles over 4 waves
  static_assert(DV == 32, "two value tiles");
  float4 pre[kOutTilesPerWave];
#pragma unroll
  for (int it = 0; it < kOutTilesPerWave; ++it) {
    const int tile = wave + 4 * it;
    const int mq = tile / NT;
    const int j = tile - mq * NT;
    const int qi = 16 * mq + l15;
    float4 a = {0.0f, 0.0f, 0.0f, 0.0f};
    if (qi < cn)
      for (int s = 0; s < nslices; ++s) {
        const float4 w = *(const float4*)(partial + (((int64_t)s * BH + bh) * n + t0 + qi) * PS + 16 * j + 4 * g4);
        a.x += w.x;
        a.y += w.y;
        a.z += w.z;
        a.w += w.w;
      }
    pre[it] = a;
  }
  float prez = 0.0f;
  if (tid < cn)
    for (int s = 0; s < nslices; ++s) prez += partial[(((int64_t)s * BH + bh) * n + t0 + tid) * PS + DV];

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

  // scores, one 16x16 tile per step, kept in registers; then the Taylor
  // weights (bf16, over the Q and K tiles) and their row sums per tile
  constexpr int kTilesPerWave = 4;  // (64 / 16)^2 tiles over 4 waves
  f32x4 sc[kTilesPerWave];
#pragma unroll
  for (int it = 0; it < kTilesPerWave; ++it) {
    const int tile = wave + 4 * it;
    const int mq = tile / MT;
    const int nk = tile - mq * MT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (tile < MT * MT && nk <= mq) {
#pragma unroll
      for (int kk = 0; kk < (DK + 31) / 32; ++kk) {
        uint4 aw = {0u, 0u, 0u, 0u}, bw = {0u, 0u, 0u, 0u};
        if (32 * kk + 8 * g4 < DK) {
          aw = *(const uint4*)(Qs + (16 * mq + l15) * L.qs + (32 * kk + 8 * g4) * 2);
          bw = *(const uint4*)(Ks + (16 * nk + l15) * L.qs + (32 * kk + 8 * g4) * 2);
        }
        acc = mfma16(__builtin_bit_cast(bf16x8, aw), __builtin_bit_cast(bf16x8, bw), acc);
      }
    }
    sc[it] = acc;
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < kTilesPerWave; ++it) {
    const int tile = wave + 4 * it;
    if (tile >= MT * MT) break;
    const int mq = tile / MT;
    const int nk = tile - mq * MT;
    const f32x4 acc = sc[it];
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
  if (tid < C) {
    float z = (float)t0;
    for (int t = 0; t < MT; ++t) z += rowpart[tid * MT + t];
    Zs[tid] = z + prez;
  }
  __syncthreads();

  // O^T = V^T P^T on the matrix cores, + partials, / Z: lane (l15, g4) ends up
  // with value columns 16 j + 4 g4 + 0..3 of query 16 mq + l15
#pragma unroll
  for (int it = 0; it < kOutTilesPerWave; ++it) {
    const int tile = wave + 4 * it;
    const int mq = tile / NT;
    const int j = tile - mq * NT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks * 32 < C; ++ks) {
      if (32 * ks > 16 * mq + 15) break;  // keys beyond the tile's last query carry zero weight
      const uint4 pw = *(const uint4*)(Pm + (16 * mq + l15) * L.ps + (32 * ks + 8 * g4) * 2);
      const uint4 vw = *(const uint4*)(Vt + (16 * j + l15) * L.vs + (32 * ks + 8 * g4) * 2);
      acc = mfma16(__builtin_bit_cast(bf16x8, vw), __builtin_bit_cast(bf16x8, pw), acc);
    }
    const int qi = 16 * mq + l15;
    if (qi < cn) {
      const float z = Zs[qi];
      uint2 w;
      w.x = (uint32_t)f32_to_bf16((acc[0] + pre[it].x) / z).bits | ((uint32_t)f32_to_bf16((acc[1] + pre[it].y) / z).bits << 16);
      w.y = (uint32_t)f32_to_bf16((acc[2] + pre[it].z) / z).bits | ((uint32_t)f32_to_bf16((acc[3] + pre[it].w) / z).bits << 16);
      *(uint2*)(y + (bh * qg * n + t0 + qi) * DV + 16 * j + 4 * g4) = w;
    }
  }
}

// ------------------------------------------------------------ host planning

struct HostPlan {
  std::vector<int4> slices;       // {first column group, column groups, 0, 0}
  std::vector<uint32_t> slots;    // [slice][wave][slot]
  std::vector<float> facs;        // [slice][kMaxFac][32] readout row factors of the kFac slots
  std::vector<int> prep_idx;      // [j][L]: canonical feature of (j, low feature L), or -1
  std::vector<float> prep_scale;  // [j][L]: 1 / sqrt(multiplicity of j in that feature)
  std::vector<int> low_idx;       // [L]: canonical feature of low feature L, or -1
};

struct PairRef {
  uint32_t kind;
  int cg, i1;
};

template <int DK>
std::vector<int> low_tuple(int L) {
  const LowFeat f = low_feat<DK>(L);
  if (f.deg == 2) return {f.a, f.b};
  if (f.deg == 1) return {f.a};
  return {};
}

// Runs of a wave's slot list: maximal stretches of one kind and i1.  Each run
// costs one readout epilogue and, for TOP, one B build in the update.
inline int count_runs(const std::vector<PairRef>& bin) {
  int r = 0;
  for (size_t i = 0; i < bin.size(); ++i)
    if (i == 0 || bin[i - 1].kind != bin[i].kind || bin[i - 1].i1 != bin[i].i1) ++r;
  return r;
}

// Packs runs (sorted longest first) whole into kNW waves of ppw slots with at
// most max_runs runs each; depth-first with symmetric placements skipped.
inline bool pack_runs(const std::vector<std::vector<PairRef>>& runs, size_t at, int ppw, int max_runs,
                      std::vector<std::vector<PairRef>>& bins, std::vector<int>& nruns, long& budget) {
  if (at == runs.size()) return true;
  if (--budget < 0) return false;
  const int len = (int)runs[at].size();
  for (int w = 0; w < kNW; ++w) {
    const int room = ppw - (int)bins[w].size();
    if (room < len || nruns[w] >= max_runs) continue;
    bool seen = false;  // an earlier wave in the same state was already tried
    for (int u = 0; u < w && !seen; ++u) seen = bins[u].size() == bins[w].size() && nruns[u] == nruns[w];
    if (seen) continue;
    bins[w].insert(bins[w].end(), runs[at].begin(), runs[at].end());
    ++nruns[w];
    if (pack_runs(runs, at + 1, ppw, max_runs, bins, nruns, budget)) return true;
    --nruns[w];
    bins[w].resize(bins[w].size() - len);
  }
  return false;
}

// Wave assignment of a slice's pairs (at most kNW * ppw of them).  Candidates:
// the pairs in order, cut into kNW nearly equal stretches (long runs split
// across neighbouring waves), and, where it exists, a packing of whole runs
// (runs longer than a wave cut into wave-sized pieces first) with fewer runs
// in the busiest wave.  The candidate whose busiest wave has
// the fewest runs wins, then the one with fewer runs in total.
inline std::vector<std::vector<PairRef>> assign_waves(const std::vector<PairRef>& pairs, int ppw) {
  std::vector<std::vector<PairRef>> seq(kNW);
  {
    const int np = (int)pairs.size();
    const int base = np / kNW, extra = np % kNW;
    int at = 0;
    for (int w = 0; w < kNW; ++w) {
      const int cnt = base + (w < extra ? 1 : 0);
      seq[w].assign(pairs.begin() + at, pairs.begin() + at + cnt);
      at += cnt;
    }
  }
  auto score = [](const std::vector<std::vector<PairRef>>& b) {
    int mx = 0, tot = 0;
    for (const auto& x : b) {
      mx = std::max(mx, count_runs(x));
      tot += count_runs(x);
    }
    return std::make_pair(mx, tot);
  };
  std::vector<std::vector<PairRef>> runs;  // runs longer than a wave are cut into wave-sized pieces
  for (size_t i = 0; i < pairs.size(); ++i) {
    if (i == 0 || pairs[i - 1].kind != pairs[i].kind || pairs[i - 1].i1 != pairs[i].i1 ||
        (int)runs.back().size() == ppw)
      runs.emplace_back();
    runs.back().push_back(pairs[i]);
  }
  std::vector<std::vector<PairRef>> best = seq;
  std::stable_sort(runs.begin(), runs.end(),
                   [](const std::vector<PairRef>& a, const std::vector<PairRef>& b) { return a.size() > b.size(); });
  const int lower = ((int)runs.size() + kNW - 1) / kNW;
  for (int mr = lower; mr < score(best).first; ++mr) {
    std::vector<std::vector<PairRef>> bins(kNW);
    std::vector<int> nruns(kNW, 0);
    long budget = 1000000;
    if (pack_runs(runs, 0, ppw, mr, bins, nruns, budget)) {
      if (score(bins) < score(best)) best = bins;
      break;
    }
  }
  return best;
}

template <int DK, int PPW>
HostPlan build_plan() {
  using LW = Low<DK>;
  constexpr int kPPW = PPW;
  constexpr int kSlots = kNW * PPW;
  HostPlan hp;
  // canonical order of the library's state rows (degree-major, lexicographic)
  std::map<uint64_t, int> canon;
  int next = 0;
  for (int p = 0; p < 4; ++p) for_each_tuple(DK, p, [&](const int* t) { canon[pack_feature(p, t)] = next++; });
  auto canon_of = [&](std::vector<int> t) {
    std::sort(t.begin(), t.end());
    return canon.at(pack_feature((int)t.size(), t.data()));
  };
  hp.low_idx.assign(LW::NLP, -1);
  hp.prep_idx.assign((size_t)DK * LW::NLP, -1);
  hp.prep_scale.assign((size_t)DK * LW::NLP, 0.0f);
  for (int L = 0; L < LW::NLP; ++L) {
    const LowFeat f = low_feat<DK>(L);
    if (f.deg < 0) continue;
    hp.low_idx[L] = canon_of(low_tuple<DK>(L));
    const int mn = (f.deg == 0) ? DK : f.a;
    for (int j = 0; j <= std::min(mn, DK - 1); ++j) {
      std::vector<int> t = low_tuple<DK>(L);
      const int mult = 1 + (int)std::count(t.begin(), t.end(), j);
      t.push_back(j);
      hp.prep_idx[(size_t)j * LW::NLP + L] = canon_of(t);
      hp.prep_scale[(size_t)j * LW::NLP + L] = 1.0f / std::sqrt((float)mult);
    }
  }

  // the pair grid: rows LOW, ZMAT, TOP i1 = 0..DK-1; row r covers column groups [0, len(r))
  std::vector<int> maxmin(LW::NCG);
  for (int cg = 0; cg < LW::NCG; ++cg) {
    const LowFeat f = low_feat<DK>(32 * cg);
    maxmin[cg] = (f.deg == 2) ? f.a : -1;
  }
  struct Row {
    uint32_t kind;
    int i1, len;
  };
  std::vector<Row> rows = {{kLow, 0, LW::NCG}, {kZmat, 0, LW::NCG}};
  for (int i1 = 0; i1 < DK; ++i1) {
    int len = 0;
    while (len < LW::NCG && maxmin[len] >= i1) ++len;
    if (len > 0) rows.push_back({kTop, i1, len});
  }

  // slices: column-group blocks of width W, rows split into slices of <= kSlots pairs
  struct Slice {
    int lo, hi;
    std::vector<PairRef> pairs;
  };
  std::vector<Slice> best;
  long best_key = -1;
  for (int W = 1; W <= kMaxNC; ++W) {
    std::vector<Slice> cand;
    for (int lo = 0; lo < LW::NCG; lo += W) {
      const int hi = std::min(LW::NCG, lo + W);
      std::vector<PairRef> seg;
      for (const Row& r : rows)
        for (int cg = lo; cg < std::min(hi, r.len); ++cg) seg.push_back({r.kind, cg, r.i1});
      if (seg.empty()) continue;
      const int ns = ((int)seg.size() + kSlots - 1) / kSlots;
      const int per = ((int)seg.size() + ns - 1) / ns;
      for (size_t s0 = 0; s0 < seg.size(); s0 += per) {
        Slice sl{lo, hi, {}};
        sl.pairs.assign(seg.begin() + s0, seg.begin() + std::min(seg.size(), s0 + per));
        int a = LW::NCG, b = 0;  // tighten the generated range to what the pairs use
        for (const PairRef& pr : sl.pairs) {
          a = std::min(a, pr.cg);
          b = std::max(b, pr.cg + 1);
        }
        sl.lo = a;
        sl.hi = b;
        cand.push_back(sl);
      }
    }
    long gen = 0;
    for (const Slice& sl : cand) gen += sl.hi - sl.lo;
    const long key = (long)cand.size() * 100000 + gen;
    if (best_key < 0 || key < best_key) {
      best_key = key;
      best = cand;
    }
  }

  const int ns = (int)best.size();
  hp.slots.assign((size_t)ns * kSlots, make_slot(kLow, 0, 0, kFirst | kLast | kEmpty));
  hp.facs.assign((size_t)ns * kMaxFac * 32, 0.0f);
  bool fac_overflow = false;
  for (int s = 0; s < ns; ++s) {
    const Slice& sl = best[s];
    const int nc = sl.hi - sl.lo;
    hp.slices.push_back(int4{sl.lo, nc, 0, 0});
    std::vector<std::vector<PairRef>> bins = assign_waves(sl.pairs, kPPW);
    std::vector<int> bin_runs(kNW);
    for (int w = 0; w < kNW; ++w) bin_runs[w] = count_runs(bins[w]);
    std::vector<int> worder(kNW);
    for (int w = 0; w < kNW; ++w) worder[w] = w;
    std::stable_sort(worder.begin(), worder.end(), [&](int a, int b) { return bin_runs[a] > bin_runs[b]; });
    int nfac = 0;
    for (int w = 0; w < kNW; ++w) {
      const std::vector<PairRef>& bin = bins[worder[w]];
      const int cnt = (int)bin.size();
      for (int p = 0; p < cnt; ++p) {
        const PairRef& pr = bin[p];
        uint32_t flags = 0;
        if (p == 0 || bin[p - 1].kind != pr.kind || bin[p - 1].i1 != pr.i1) flags |= kFirst;
        if (p == cnt - 1 || bin[p + 1].kind != pr.kind || bin[p + 1].i1 != pr.i1) flags |= kLast;
        float fr[32];
        bool any = false;
        for (int r = 0; r < 32; ++r) {
          const LowFeat f = low_feat<DK>(32 * pr.cg + r);
          float x = 1.0f;
          if (pr.kind == kTop) {
            x = (f.deg == 2 && f.a >= pr.i1) ? 1.0f / (float)(1 + (f.a == pr.i1) + (f.b == pr.i1)) : 0.0f;
          } else if (pr.kind == kZmat) {
            x = (f.deg >= 0) ? 1.0f / (float)(f.deg + 1) : 0.0f;
          }
          fr[r] = x;
          any = any || (x != 1.0f);
        }
        int fi = 0;
        if (any) {
          flags |= kFac;
          if (nfac < kMaxFac) {
            fi = nfac;
            std::copy(fr, fr + 32, &hp.facs[((size_t)s * kMaxFac + fi) * 32]);
          } else {
            fac_overflow = true;
          }
          ++nfac;
        }
        hp.slots[(size_t)s * kSlots + w * kPPW + p] = make_slot(pr.kind, pr.cg - sl.lo, pr.i1, flags, fi);
      }
    }
  }

  if (fac_overflow) {  // more factor rows than the LDS table holds: unsupported
    hp.slices.clear();
    return hp;
  }
  // every canonical (feature, column) of the exported state must be written exactly once
  {
    const int64_t D = (int64_t)(DK + 1) * (DK + 2) * (DK + 3) / 6;
    std::vector<int> hit((size_t)D * 2, 0);  // [feature][value block, normaliser]
    hit[1] += 1;                              // degree-0 normaliser: the token count
    for (int s = 0; s < ns; ++s)
      for (const PairRef& pr : best[s].pairs)
        for (int r = 0; r < 32; ++r) {
          const int L = 32 * pr.cg + r;
          if (pr.kind == kLow) {
            if (hp.low_idx[L] >= 0) hit[2 * hp.low_idx[L]] += 1;
          } else if (pr.kind == kTop) {
            const int ci = (L < LW::M2) ? hp.prep_idx[(size_t)pr.i1 * LW::NLP + L] : -1;
            if (ci >= 0) hit[2 * ci] += 1;
          } else {
            for (int j = 0; j < DK; ++j) {
              const int ci = hp.prep_idx[(size_t)j * LW::NLP + L];
              if (ci >= 0) hit[2 * ci + 1] += 1;
            }
          }
        }
    for (int64_t i = 0; i < 2 * D; ++i)
      if (hit[i] != 1) {
        hp.slices.clear();  // an incomplete plan is reported as unsupported
        break;
      }
  }
  return hp;
}

struct DeviceTables {
  int4* slices = nullptr;
  uint32_t* slots = nullptr;
  float* facs = nullptr;
  int* prep_idx = nullptr;
  float* prep_scale = nullptr;
  int* low_idx = nullptr;
  int nslices = 0;
};

template <typename T>
hipError_t upload(const std::vector<T>& h, T** d, hipStream_t s) {
  hipError_t e = hipMalloc((void**)d, h.size() * sizeof(T));
  if (e != hipSuccess) return e;
  e = hipMemcpyAsync(*d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(s);
}

std::mutex g_mu;
std::map<std::pair<int, int>, DeviceTables> g_tables;  // (device, d)

// State pairs per wave.
template <int DK>
struct Ppw {
  static constexpr int value = 8;
};

const HostPlan& host_plan() {
  static HostPlan p32 = build_plan<32, Ppw<32>::value>();
  return p32;
}

hipError_t get_tables(int d, hipStream_t s, DeviceTables* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_tables.find({dev, d});
  if (it != g_tables.end()) {
    *out = it->second;
    return hipSuccess;
  }
  const HostPlan& hp = host_plan();
  DeviceTables t;
  t.nslices = (int)hp.slices.size();
  if ((e = upload(hp.slices, &t.slices, s)) != hipSuccess) return e;
  if ((e = upload(hp.slots, &t.slots, s)) != hipSuccess) return e;
  if ((e = upload(hp.facs, &t.facs, s)) != hipSuccess) return e;
  if ((e = upload(hp.prep_idx, &t.prep_idx, s)) != hipSuccess) return e;
  if ((e = upload(hp.prep_scale, &t.prep_scale, s)) != hipSuccess) return e;
  if ((e = upload(hp.low_idx, &t.low_idx, s)) != hipSuccess) return e;
  g_tables[{dev, d}] = t;
  *out = t;
  return hipSuccess;
}

template <int DK>
hipError_t launch_typed(const u16* q, const u16* k, const u16* v, u16* y, float* S_out, int BH, int n,
                        const DeviceTables& dt, float* partial, hipStream_t s, int qg) {
  using L = Lds<DK>;
  auto kmain = prefill_mfma_main<DK, Ppw<DK>::value>;
  hipError_t e = hipFuncSetAttribute((const void*)kmain, hipFuncAttributeMaxDynamicSharedMemorySize, L::BYTES);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kmain, dim3((unsigned)dt.nslices * (unsigned)BH), dim3(kNW * 64), L::BYTES, s, q, k, v,
                     dt.slices, dt.slots, dt.facs, dt.prep_idx, dt.prep_scale, dt.low_idx, partial, S_out, BH, n,
                     dt.nslices, qg);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const FinLayout F(DK, DK, kC);
  auto kfin = prefill_mfma_finalize<DK, DK>;
  e = hipFuncSetAttribute((const void*)kfin, hipFuncAttributeMaxDynamicSharedMemorySize, F.bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kfin, dim3((unsigned)((n + kC - 1) / kC), (unsigned)BH), dim3(256), (size_t)F.bytes, s, q, k,
                     v, partial, y, BH, n, kC, dt.nslices, 4, kPS, qg);
  return hipGetLastError();
}

}  // namespace

bool plan_prefill_mfma(int BH, int n, int dk, int dv, int P, int chunk, MfmaPrefillPlan* plan) {
  if (P != 4 || dk != 32 || dv != 32) return false;
  if (chunk != kC) return false;
  if (n < 1) return false;
  const HostPlan& hp = host_plan();
  if (hp.slices.empty()) return false;
  plan->dk = dk;
  plan->dv = dv;
  plan->nslices = (int)hp.slices.size();
  plan->partial_bytes = sizeof(float) * (size_t)plan->nslices * BH * n * kPS;
  plan->workspace_bytes = plan->partial_bytes;
  return true;
}

hipError_t launch_prefill_mfma(const void* q, const void* k, const void* v, void* y, float* S_out, int BH,
                               int n, int dk, int dv, int P, int chunk, const MfmaPrefillPlan& plan,
                               void* workspace, hipStream_t s, int qg) {
  (void)P;
  (void)dv;
  (void)chunk;
  (void)plan;
  DeviceTables dt;
  hipError_t e = get_tables(dk, s, &dt);
  if (e != hipSuccess) return e;
  float* partial = (float*)workspace;
  const u16* qq = (const u16*)q;
  const u16* kk = (const u16*)k;
  const u16* vv = (const u16*)v;
  return launch_typed<32>(qq, kk, vv, (u16*)y, S_out, BH, n, dt, partial, s, qg);
}

}  // namespace sata
