// Device-side building blocks shared by the quantize and decode kernels.
//
// Cache layout (64-slot tiles, 2048 bytes per tile per tensor):
//   K tile, token-major: 16-byte half c (codes 32c..32c+31) of slot-in-tile r
//        at byte (c*64 + r)*16. One lane per token loads its 32 bytes with two
//        128-bit loads; each wave-wide load covers 1 KiB contiguously. Key word
//        w holds dimensions 8w..8w+7: 3-bit index of dimension 8w+j in bits
//        3j..3j+2, its QJL sign bit in bit 24+j.
//   V tile, dimension-major: 16-byte half c (slots 32c..32c+31) of dimension i
//        at byte (c*64 + i)*16. One lane per dimension loads the 64 codes of its
//        dimension for the whole tile with two 128-bit loads. A value nibble is
//        idx | sign << 3; nibble j of a 32-bit word sits at bits 4j..4j+3.
//   Scalars: 4 x fp16 per slot [n_k, g_k, n_v, g_v] at byte slot*8.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace tq {

constexpr int kDim = 64;
constexpr int kTile = 64;
constexpr int kTileBytes = 2048;   // 64 slots x 32 bytes
constexpr int kPairs = 32;

// Flags (values fixed by the public header).
constexpr uint32_t kVRotate = 1u << 0;
constexpr uint32_t kVQjl = 1u << 1;
constexpr uint32_t kQjlPaper = 1u << 2;
constexpr uint32_t kRopeHalf = 1u << 3;
constexpr uint32_t kInputRotated = 1u << 4;
constexpr uint32_t kOutF32 = 1u << 5;

// sqrt(pi/2) / m with m = 64 projection rows (QJL estimator scale).
constexpr float kQjlAlpha = 0.019583033395554691f;

__device__ __forceinline__ float load_in(const void* p, int64_t i, bool f16) {
  if (f16) return __half2float(reinterpret_cast<const __half*>(p)[i]);
  return reinterpret_cast<const float*>(p)[i];
}

// Norms are stored as fp16 with round-to-nearest-even, saturated at 65504.
__device__ __forceinline__ uint32_t store_norm(float x) {
  x = (x > 65504.0f) ? 65504.0f : x;
  return (uint32_t)__half_as_ushort(__float2half_rn(x));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t bits) {
  return __half2float(__ushort_as_half((unsigned short)(bits & 0xFFFFu)));
}

// Key word of dimensions 8w..8w+7: 3-bit index of dimension 8w+j in bits
// 3j..3j+2, its QJL sign bit in bit 24+j. Value words hold eight 4-bit
// nibbles idx | sign << 3.
__device__ __forceinline__ uint32_t key_code_bits(uint32_t idx, uint32_t sign, int j) {
  return (idx << (3 * j)) | (sign << (24 + j));
}

// Byte offset of 16-byte half c of row r (slot for K, dimension for V) in a tile.
__device__ __forceinline__ int64_t tile_half_offset(int64_t tile, int c, int r) {
  return tile * kTileBytes + (int64_t)(c * kTile + r) * 16;
}

// Fixed-order binary32 steps of the quantizer for one vector held in registers
// (this file is compiled with -ffp-contract=off and correctly rounded sqrtf and
// division, the HIP defaults; fmaf is the only fused operation)
// by one lane: the norm and residual-norm fma chains run over i ascending and
// the projected sign of row i is an fma chain over k ascending, so any kernel
// that calls this on the same x^ produces the same bits.
//   xh[64]   rotated vector (overwritten by the residual r)
//   L        ascending table and its midpoints (0.5f * (c_m + c_{m+1}))
//   S        64 x 64 projection in LDS (row-major); unused unless sign_mode == 1
//   sign_mode 0 none, 1 projected (S r), 2 per element (r), 3 projected with
//            the signs set by the caller (g is computed and stored, no bits)
//   words[8] out: with KEY_WORDS the key word format (index of dimension 8w+j
//            in bits 3j..3j+2, its sign in bit 24+j), else nibble words
//            (idx | sign << 3 in bits 4j..4j+3)
// The eight levels and seven midpoints of one table as named register values.
// Named members (no arrays) keep the level choice a chain of selects between
// registers; an array indexed inside a loop gets folded into an indexed load
// from private memory, which the compiler then spills to LDS or scratch.
struct Levels {
  float c0, c1, c2, c3, c4, c5, c6, c7;
  float t0, t1, t2, t3, t4, t5, t6;
};

__device__ __forceinline__ Levels load_levels(const float* lut) {
  Levels L;
  L.c0 = lut[0]; L.c1 = lut[1]; L.c2 = lut[2]; L.c3 = lut[3];
  L.c4 = lut[4]; L.c5 = lut[5]; L.c6 = lut[6]; L.c7 = lut[7];
  L.t0 = 0.5f * (L.c0 + L.c1); L.t1 = 0.5f * (L.c1 + L.c2); L.t2 = 0.5f * (L.c2 + L.c3);
  L.t3 = 0.5f * (L.c3 + L.c4); L.t4 = 0.5f * (L.c4 + L.c5); L.t5 = 0.5f * (L.c5 + L.c6);
  L.t6 = 0.5f * (L.c6 + L.c7);
  return L;
}

// Strictly ascending levels (false for any NaN level). Kernels skip a
// (layer, head) whose table fails this: the midpoint rule assumes it.
__device__ __forceinline__ bool levels_ascending(const Levels& L) {
  return (L.c0 < L.c1) & (L.c1 < L.c2) & (L.c2 < L.c3) & (L.c3 < L.c4) & (L.c4 < L.c5) &
         (L.c5 < L.c6) & (L.c6 < L.c7);
}

// Nearest level of u by the midpoints (ties go to the lower level): returns
// the level, its index in *idx.
// The levels are passed as separate values, which callers pin in registers
// once (TQ_PIN_LEVELS): the selects then pick between register values, where a
// select between two loads of a table would become one load at a computed
// offset, from private memory.
#define TQ_PIN_LEVELS(L)                                                                  \
  float L##_0 = L.c0, L##_1 = L.c1, L##_2 = L.c2, L##_3 = L.c3, L##_4 = L.c4, L##_5 = L.c5, \
        L##_6 = L.c6, L##_7 = L.c7;                                                       \
  asm volatile("" : "+v"(L##_0), "+v"(L##_1), "+v"(L##_2), "+v"(L##_3), "+v"(L##_4),     \
               "+v"(L##_5), "+v"(L##_6), "+v"(L##_7))
#define TQ_LEVELS(L) L, L##_0, L##_1, L##_2, L##_3, L##_4, L##_5, L##_6, L##_7

__device__ __forceinline__ float nearest_level(float u, const Levels& L, float c0, float c1,
                                               float c2, float c3, float c4, float c5, float c6,
                                               float c7, uint32_t* idx) {
  uint32_t i = 0;
  float lv = c0;
  bool a;
  a = u > L.t0; i += a ? 1u : 0u; lv = a ? c1 : lv;
  a = u > L.t1; i += a ? 1u : 0u; lv = a ? c2 : lv;
  a = u > L.t2; i += a ? 1u : 0u; lv = a ? c3 : lv;
  a = u > L.t3; i += a ? 1u : 0u; lv = a ? c4 : lv;
  a = u > L.t4; i += a ? 1u : 0u; lv = a ? c5 : lv;
  a = u > L.t5; i += a ? 1u : 0u; lv = a ? c6 : lv;
  a = u > L.t6; i += a ? 1u : 0u; lv = a ? c7 : lv;
  *idx = i;
  return lv;
}

// The index alone, #{m : u > t_m} (the same count as nearest_level's), for a
// caller that reads the level itself from a table in LDS. The comparisons
// write VCC only and each is used at once, so no lane mask stays live across
// the elements of a vector (64 unrolled select chains keep so many masks
// live that they spill).
__device__ __forceinline__ uint32_t level_index(float u, const Levels& L, const float* thr_even) {
  // The count is the length of the prefix of thresholds below u (they are
  // non-decreasing), found in three steps: b2 = [t3 < u], b1 =
  // [t(b2 ? 5 : 1) < u] and b0 = [t(4 b2 + 2 b1) < u], each bit added into
  // the count by a carry (a NaN u compares false throughout, like the
  // count). The second threshold is selected in registers (t1 and t5 as
  // vector operands: a select that reads VCC cannot also read a scalar);
  // the third, t(2 i) for i = 2 b2 + b1, is read from thr_even = {t0, t2, t4,
  // t6} in LDS.
  uint32_t i;
  float ta;
  asm("v_cmp_lt_f32 vcc, %2, %5\n\t"
      "v_cndmask_b32_e64 %0, 0, 1, vcc\n\t"
      "v_cndmask_b32 %1, %3, %4, vcc\n\t"
      "v_cmp_lt_f32 vcc, %1, %5\n\t"
      "v_addc_co_u32 %0, vcc, %0, %0, vcc"
      : "=&v"(i), "=&v"(ta)
      : "s"(L.t3), "v"(L.t1), "v"(L.t5), "v"(u)
      : "vcc");
  const float tb = thr_even[i];
  asm("v_cmp_lt_f32 vcc, %1, %2\n\t"
      "v_addc_co_u32 %0, vcc, %0, %0, vcc"
      : "+v"(i)
      : "v"(tb), "v"(u)
      : "vcc");
  return i;
}

struct QuantOut {
  uint32_t n16, g16;
  float g;                 // ||r|| in binary32 (before the fp16 store)
};

template <bool KEY_WORDS>
__device__ __forceinline__ QuantOut quantize_lane(float (&xh)[kDim], const Levels& L, const float* lev,
                                                  const float* thr_even, const float* S, int sign_mode,
                                                  uint32_t (&words)[8]) {
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < kDim; ++i) s = fmaf(xh[i], xh[i], s);
  const float n = sqrtf(s);
  const float inv = (n == 0.0f) ? 0.0f : 8.0f / n;
#pragma unroll
  for (int w = 0; w < 8; ++w) words[w] = 0u;
#pragma unroll
  for (int i = 0; i < kDim; ++i) {
    const float u = xh[i] * inv;
    const uint32_t idx = level_index(u, L, thr_even);
    const float lv = lev[idx];   // the level c[idx], from the table in LDS
    words[i >> 3] |= idx << ((KEY_WORDS ? 3 : 4) * (i & 7));
    xh[i] = u - lv;   // residual r_i
  }
  float gs = 0.0f;
#pragma unroll
  for (int i = 0; i < kDim; ++i) gs = fmaf(xh[i], xh[i], gs);
  const float g = sqrtf(gs);
  uint64_t sbits = 0;
  if (sign_mode == 1) {
    for (int i = 0; i < kDim; ++i) {
      float acc = 0.0f;
      const float4* row = reinterpret_cast<const float4*>(S + i * kDim);
#pragma unroll
      for (int k4 = 0; k4 < kDim / 4; ++k4) {
        const float4 sv = row[k4];
        acc = fmaf(sv.x, xh[4 * k4 + 0], acc);
        acc = fmaf(sv.y, xh[4 * k4 + 1], acc);
        acc = fmaf(sv.z, xh[4 * k4 + 2], acc);
        acc = fmaf(sv.w, xh[4 * k4 + 3], acc);
      }
      sbits |= (uint64_t)((acc < 0.0f) ? 0u : 1u) << i;
    }
  } else if (sign_mode == 2) {
#pragma unroll
    for (int i = 0; i < kDim; ++i) sbits |= (uint64_t)((xh[i] < 0.0f) ? 0u : 1u) << i;
  }
#pragma unroll
  for (int i = 0; i < kDim; ++i)
    words[i >> 3] |= (uint32_t)((sbits >> i) & 1u) << (KEY_WORDS ? 24 + (i & 7) : 4 * (i & 7) + 3);
  QuantOut o;
  o.n16 = store_norm(n);
  o.g16 = (sign_mode == 0) ? 0u : store_norm(g);
  o.g = g;
  return o;
}

// Wave-wide reductions (64 lanes).
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace tq
