// Wave-per-vector quantizer shared by the append kernel (short decode-step
// appends through tq_quantize_pack) and the decode-step prologue kernel: one
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


// Pi and S are staged row-major in LDS with rows 68 floats apart, so that lane
// i reads row i with sixteen 16-byte reads: at that pitch the 16 lanes served
// together start on banks 4 apart and cover all 64 banks once. The fma chains
// keep k ascending.
constexpr int kRowPitch = kDim + 4;

struct VectorSmem {
  float pi[kDim * kRowPitch];   // pi[i * 68 + k] = Pi[i][k]
  float s[kDim * kRowPitch];    // s[i * 68 + k] = S[i][k]
  float x[2][kDim];
  float r[2][kDim];
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Row i of a 64 x 64 matrix staged in `m` times the vector staged in `v`: fma
// chain over k ascending, the order of rotate_lane and quantize_lane. All 32
// reads are issued before the chain starts (one LDS latency, not one per
// element).
__device__ __forceinline__ float row_dot(const float* m, const float* v, int i) {
  float4 mr[kDim / 4], vv[kDim / 4];
  const float4* row = reinterpret_cast<const float4*>(m + i * kRowPitch);
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) {
    mr[k4] = row[k4];
    vv[k4] = reinterpret_cast<const float4*>(v)[k4];
  }
  float acc = 0.0f;
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) {
    acc = fmaf(mr[k4].x, vv[k4].x, acc);
    acc = fmaf(mr[k4].y, vv[k4].y, acc);
    acc = fmaf(mr[k4].z, vv[k4].z, acc);
    acc = fmaf(mr[k4].w, vv[k4].w, acc);
  }
  return acc;
}

// fma chain over i ascending of v_i^2 for the vector staged in `v` (every
// lane gets the same value); the 16 reads are issued first.
__device__ __forceinline__ float sum_squares(const float* v) {
  float4 vv[kDim / 4];
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) vv[k4] = reinterpret_cast<const float4*>(v)[k4];
  float acc = 0.0f;
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) {
    acc = fmaf(vv[k4].x, vv[k4].x, acc);
    acc = fmaf(vv[k4].y, vv[k4].y, acc);
    acc = fmaf(vv[k4].z, vv[k4].z, acc);
    acc = fmaf(vv[k4].w, vv[k4].w, acc);
  }
  return acc;
}

// Stores columns c .. c+3 of row `row` of a staged matrix.
__device__ __forceinline__ void stage_row4(float* m, int row, int c, float4 v) {
  *reinterpret_cast<float4*>(m + row * kRowPitch + c) = v;
}

// Quantize the vector whose element i lane i holds in `xh`; same arithmetic
// order as quantize_lane. Returns the lane's nibble; n16/g16 are uniform.
__device__ __forceinline__ uint32_t quantize_wave(float xh, const Levels& L,
                                                  const float* sm_s, int sign_mode, float* xs,
                                                  float* rs, int i, uint32_t* n16, uint32_t* g16) {
  xs[i] = xh;
  wave_sync_lds();
  const float n = sqrtf(sum_squares(xs));
  const float inv = (n == 0.0f) ? 0.0f : 8.0f / n;
  const float u = xh * inv;
  TQ_PIN_LEVELS(L);
  uint32_t idx;
  const float lv = nearest_level(u, TQ_LEVELS(L), &idx);
  const float r = u - lv;
  rs[i] = r;
  wave_sync_lds();
  const float g = sqrtf(sum_squares(rs));
  uint32_t bit = 0;
  if (sign_mode == 1) {
    bit = (row_dot(sm_s, rs, i) < 0.0f) ? 0u : 1u;
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

// Rotate (when `rotate`), quantize and store one vector into slot `slot` of
// head lh: keys as token-major key words plus [n_k, g_k], values as
// dimension-major nibbles plus [n_v, g_v]. Pi and S are staged in sm;
// `wave` (0 or 1) picks this wave's staging rows.
__device__ __forceinline__ void append_wave(float x, bool is_v, bool rotate, const Levels& L,
                                            VectorSmem& sm, int sign_mode, int64_t slot,
                                            int64_t lh, uint8_t* k_codes, uint8_t* v_codes,
                                            uint16_t* scalars, int64_t slots, int i, int wave) {
  float* xs = sm.x[wave];
  float* rs = sm.r[wave];
  if (rotate) {
    xs[i] = x;
    wave_sync_lds();
    x = row_dot(sm.pi, xs, i);
    wave_sync_lds();   // xs is rewritten by quantize_wave
  }
  uint32_t n16, g16;
  const uint32_t nib = quantize_wave(x, L, sm.s, sign_mode, xs, rs, i, &n16, &g16);
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
    if (i == 0) reinterpret_cast<uint32_t*>(scalars + (lh * slots + slot) * 4)[0] = n16 | (g16 << 16);
  } else {
    // value: dimension-major, one nibble of dimension i's word for this slot
    uint8_t* vreg = v_codes + lh * slots * 32;
    const int cc = r >> 5, G4 = (r & 31) >> 3, jj = r & 7;
    uint32_t* addr = reinterpret_cast<uint32_t*>(vreg + tile_half_offset(tile, cc, i) + G4 * 4);
    store_v_word(addr, nib << (4 * jj), 15u << (4 * jj));
    if (i == 0) reinterpret_cast<uint32_t*>(scalars + (lh * slots + slot) * 4)[1] = n16 | (g16 << 16);
  }
}

}  // namespace tq
