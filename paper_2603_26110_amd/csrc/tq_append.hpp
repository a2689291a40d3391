// Wave-per-vector quantizer shared by the append kernel (short decode-step
// appends through tq_quantize_pack) and the decode kernel's step prologue: one
// wave quantizes one key or value vector of a token-head, lane i holding
// element i. Both kernels call these same functions, so a token gets the same
// codes from either (and from the lane-per-token prefill kernel, which keeps
// the same binary32 order; Sec. 3.1 prefill steps 3-4, Sec. 3.3, Sec. 3.4).
#pragma once

#include "tq_device.hpp"

namespace tq {

// Write one dimension-major V nibble group: `mask` selects the nibbles of
// `word` this writer owns. Whole words are stored; partial words are merged
// with atomics so concurrent writers of neighbouring slots do not collide.
__device__ __forceinline__ void store_v_word(uint32_t* addr, uint32_t word, uint32_t mask) {
  if (mask == 0xFFFFFFFFu) {
    *addr = word;
  } else if (mask != 0u) {
    atomicAnd(addr, ~mask);
    atomicOr(addr, word & mask);
  }
}


// Two LDS layouts of a staged 64 x 64 matrix, both read by rows with
// 16-byte reads (lane i reads row i) without bank conflicts:
//   Pitch68  rows 68 floats apart: the 16 lanes served together start on
//            banks 4 apart and cover all 64 banks once (needs 17 KB);
//   Swz16    rows 64 floats apart with the 16-byte chunks of row r permuted
//            (chunk k at position k ^ (r & 15)): the 16 lanes served together
//            read 16 different bank groups. Dense (16 KB), and every 1 KB run
//            of it is whole chunks of four rows, so a direct global-to-LDS
//            copy can fill it (each lane picks the global chunk that belongs
//            at its LDS position).
// chunk(r, k4) is the float4 index of columns 4 k4 .. 4 k4 + 3 of row r.
constexpr int kRowPitch = kDim + 4;

struct Pitch68 {
  __device__ __forceinline__ static int chunk(int r, int k4) { return r * (kRowPitch / 4) + k4; }
};
struct Swz16 {
  __device__ __forceinline__ static int chunk(int r, int k4) { return r * 16 + (k4 ^ (r & 15)); }
  // global chunk held at LDS chunk position c
  __device__ __forceinline__ static int source(int c) { return (c & ~15) | ((c & 15) ^ ((c >> 4) & 15)); }
};

struct VectorSmem {
  float pi[kDim * kRowPitch];   // Pitch68
  float s[kDim * kRowPitch];    // Pitch68
  float x[2][kDim];
  float r[2][kDim];
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Zero, computed after `x`: an offset that makes the reads of a batch wait
// for the chain of the one before, so the compiler cannot hoist them (and
// hold every batch's registers at once).
__device__ __forceinline__ int after(float x) {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z) : "v"(x));
  return z;
}

// Row i of a 64 x 64 matrix staged in `m` (layout LY) times the vector staged
// in `v`: fma chain over k ascending, the order of rotate_lane and
// quantize_lane. The reads are issued in batches of NB chunks of four
// elements, each batch after the chain of the one before (NB = 16: one LDS
// latency for the whole row; smaller batches hold fewer registers). The batch
// size changes no arithmetic.
template <class LY, int NB = 16>
__device__ __forceinline__ float row_dot(const float* m, const float* v, int i) {
  const float4* m4 = reinterpret_cast<const float4*>(m);
  const float4* v4 = reinterpret_cast<const float4*>(v);
  float acc = 0.0f;
#pragma unroll
  for (int b = 0; b < kDim / 4; b += NB) {
    const int z = b > 0 ? after(acc) : 0;
    float4 mr[NB], vv[NB];
#pragma unroll
    for (int k4 = 0; k4 < NB; ++k4) {
      mr[k4] = m4[LY::chunk(i, b + k4) + z];
      vv[k4] = v4[b + k4 + z];
    }
#pragma unroll
    for (int k4 = 0; k4 < NB; ++k4) {
      acc = fmaf(mr[k4].x, vv[k4].x, acc);
      acc = fmaf(mr[k4].y, vv[k4].y, acc);
      acc = fmaf(mr[k4].z, vv[k4].z, acc);
      acc = fmaf(mr[k4].w, vv[k4].w, acc);
    }
  }
  return acc;
}

// fma chain over i ascending of v_i^2 for the vector staged in `v` (every
// lane gets the same value); reads in batches as in row_dot.
template <int NB = 16>
__device__ __forceinline__ float sum_squares(const float* v) {
  const float4* v4 = reinterpret_cast<const float4*>(v);
  float acc = 0.0f;
#pragma unroll
  for (int b = 0; b < kDim / 4; b += NB) {
    const int z = b > 0 ? after(acc) : 0;
    float4 vv[NB];
#pragma unroll
    for (int k4 = 0; k4 < NB; ++k4) vv[k4] = v4[b + k4 + z];
#pragma unroll
    for (int k4 = 0; k4 < NB; ++k4) {
      acc = fmaf(vv[k4].x, vv[k4].x, acc);
      acc = fmaf(vv[k4].y, vv[k4].y, acc);
      acc = fmaf(vv[k4].z, vv[k4].z, acc);
      acc = fmaf(vv[k4].w, vv[k4].w, acc);
    }
  }
  return acc;
}

// Stores columns c .. c+3 of row `row` of a Pitch68-staged matrix.
__device__ __forceinline__ void stage_row4(float* m, int row, int c, float4 v) {
  reinterpret_cast<float4*>(m)[Pitch68::chunk(row, c >> 2)] = v;
}

// Quantize the vector whose element i lane i holds in `xh`; same arithmetic
// order as quantize_lane. Returns the lane's nibble; n16/g16 are uniform.
template <class LY, int NB = 16>
__device__ __forceinline__ uint32_t quantize_wave(float xh, const Levels& L, const float* sm_s,
                                                  int sign_mode, float* xs, float* rs, int i,
                                                  uint32_t* n16, uint32_t* g16) {
  xs[i] = xh;
  wave_sync_lds();
  const float n = sqrtf(sum_squares<NB>(xs));
  const float inv = (n == 0.0f) ? 0.0f : 8.0f / n;
  const float u = xh * inv;
  TQ_PIN_LEVELS(L);
  uint32_t idx;
  const float lv = nearest_level(u, TQ_LEVELS(L), &idx);
  const float r = u - lv;
  rs[i] = r;
  wave_sync_lds();
  const float g = sqrtf(sum_squares<NB>(rs));
  uint32_t bit = 0;
  if (sign_mode == 1) {
    bit = (row_dot<LY, NB>(sm_s, rs, i) < 0.0f) ? 0u : 1u;
  } else if (sign_mode == 2) {
    bit = (r < 0.0f) ? 0u : 1u;
  }
  *n16 = store_norm(n);
  *g16 = (sign_mode == 0) ? 0u : store_norm(g);
  return idx | (bit << 3);
}

// RoPE of a key held one element per lane (pairs (2m, 2m+1), or (m, m+32)
// with half pairing): x'_a = x_a c - x_b s, x'_b = x_a s + x_b c; cs is the
// (cos, sin) of this lane's pair.
__device__ __forceinline__ float rope_wave(float x, float2 cs, bool half, int i) {
  const int partner = half ? (i ^ 32) : (i ^ 1);
  const bool first = half ? (i < 32) : ((i & 1) == 0);
  const float xp = __shfl(x, partner, 64);
  return first ? (x * cs.x - xp * cs.y) : (xp * cs.y + x * cs.x);
}

// What an append wrote for its token: the key word of lane 8w is word w
// (keys), the lane's value nibble (values), and the token's [norm, residual
// norm] fp16 pair, uniform.
struct Appended {
  uint32_t code;
  uint32_t scal;
};

// Rotate (when `rotate`), quantize and store one vector into slot `slot` of
// head lh: keys as token-major key words plus [n_k, g_k], values as
// dimension-major nibbles plus [n_v, g_v]. Pi and S are staged in LDS in
// layout LY; xs and rs are this wave's two 64-float staging vectors; NB as in
// row_dot.
template <class LY, int NB = 16>
__device__ __forceinline__ Appended append_wave(float x, bool is_v, bool rotate, const Levels& L,
                                                const float* pi, const float* s, float* xs, float* rs,
                                                int sign_mode, int64_t slot, int64_t lh, uint8_t* k_codes,
                                                uint8_t* v_codes, uint16_t* scalars, int64_t slots, int i) {
  if (rotate) {
    xs[i] = x;
    wave_sync_lds();
    x = row_dot<LY, NB>(pi, xs, i);
    wave_sync_lds();   // xs is rewritten by quantize_wave
  }
  uint32_t n16, g16;
  const uint32_t nib = quantize_wave<LY, NB>(x, L, s, sign_mode, xs, rs, i, &n16, &g16);
  const uint32_t scal = n16 | (g16 << 16);
  const int64_t tile = slot >> 6;
  const int r = (int)(slot & 63);
  if (!is_v) {
    // key: token-major key words (index bits 3j, sign bit 24 + j); lane 8w
    // ends with word w
    uint32_t word = key_code_bits(nib & 7u, nib >> 3, i & 7);
    word |= __shfl_xor(word, 1, 64);
    word |= __shfl_xor(word, 2, 64);
    word |= __shfl_xor(word, 4, 64);
    uint8_t* kreg = k_codes + lh * slots * 32;
    if ((i & 7) == 0) {
      const int w = i >> 3;
      *reinterpret_cast<uint32_t*>(kreg + tile_half_offset(tile, w >> 2, r) + (w & 3) * 4) = word;
    }
    if (i == 0) reinterpret_cast<uint32_t*>(scalars + (lh * slots + slot) * 4)[0] = scal;
    return Appended{word, scal};
  }
  // value: dimension-major, one nibble of dimension i's word for this slot
  uint8_t* vreg = v_codes + lh * slots * 32;
  const int cc = r >> 5, G4 = (r & 31) >> 3, jj = r & 7;
  uint32_t* addr = reinterpret_cast<uint32_t*>(vreg + tile_half_offset(tile, cc, i) + G4 * 4);
  store_v_word(addr, nib << (4 * jj), 15u << (4 * jj));
  if (i == 0) reinterpret_cast<uint32_t*>(scalars + (lh * slots + slot) * 4)[1] = scal;
  return Appended{nib, scal};
}

}  // namespace tq
