// Prefill-side quantizer: RoPE -> Pi rotation -> per-vector norm -> 3-bit
// table codes -> residual -> QJL sign bits -> packed cache (TurboESM Sec. 3.1
// prefill steps 1, 3, 4; Sec. 3.3; Sec. 3.4; Sec. 4.2).
//
// Two kernels compute the same bits:
//   quantize_tiles_kernel   one lane per token, 64 tokens per wave, for
//                           prefill-sized T. Pi and S sit in LDS and are read
//                           as wave-wide broadcasts.
//   quantize_vectors_kernel one wave per vector (one lane per dimension; the
//                           key and the value of a token-head in parallel), for
//                           decode-step appends with small T.
// Both evaluate the rotation as an fma chain over k ascending and the
// quantizer steps with the fixed binary32 order of quantize_lane, so a token
// gets the same codes from either kernel.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// ---------------------------------------------------------------- RoPE table
// cs[p][m] = (cos, sin)(p * base^(-2m/64)), fp64 before rounding (Eq. 2).
__global__ void rope_table_kernel(float* cs, int positions, double base) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)positions * kPairs) return;
  const int p = (int)(e / kPairs), m = (int)(e % kPairs);
  const double theta = pow(base, -2.0 * m / (double)kDim);
  const double ang = (double)p * theta;
  cs[2 * e + 0] = (float)cos(ang);
  cs[2 * e + 1] = (float)sin(ang);
}

hipError_t launch_rope_table(float* cs, int positions, double base, hipStream_t st) {
  const int64_t n = (int64_t)positions * kPairs;
  const int threads = 256;
  const int blocks = (int)((n + threads - 1) / threads);
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks), dim3(threads), 0, st, cs, positions, base);
  return hipGetLastError();
}

// ------------------------------------------------------------ shared pieces
// RoPE of one vector held by one lane (pairs (2m, 2m+1), or (m, m+32) with
// half pairing): x'_a = x_a c - x_b s, x'_b = x_a s + x_b c in binary32.
__device__ __forceinline__ void rope_lane(float (&x)[kDim], const float* cs_row, bool half) {
  const float4* cs4 = reinterpret_cast<const float4*>(cs_row);
  float c[kPairs], s[kPairs];
#pragma unroll
  for (int q = 0; q < kPairs / 2; ++q) {
    const float4 v = cs4[q];
    c[2 * q] = v.x; s[2 * q] = v.y; c[2 * q + 1] = v.z; s[2 * q + 1] = v.w;
  }
  if (half) {
#pragma unroll
    for (int m = 0; m < kPairs; ++m) {
      const float xa = x[m], xb = x[m + kPairs];
      x[m] = xa * c[m] - xb * s[m];
      x[m + kPairs] = xa * s[m] + xb * c[m];
    }
  } else {
#pragma unroll
    for (int m = 0; m < kPairs; ++m) {
      const float xa = x[2 * m], xb = x[2 * m + 1];
      x[2 * m] = xa * c[m] - xb * s[m];
      x[2 * m + 1] = xa * s[m] + xb * c[m];
    }
  }
}

// x^_i = fma chain over k ascending of Pi[i][k] x_k; Pi in LDS (row-major),
// read as broadcasts. The per-lane result goes through the lane's own LDS
// column so that the output index stays static.
__device__ __forceinline__ void rotate_lane(float (&x)[kDim], const float* s_pi, float* s_col,
                                            int lane) {
  for (int i = 0; i < kDim; ++i) {
    const float4* row = reinterpret_cast<const float4*>(s_pi + i * kDim);
    float acc = 0.0f;
#pragma unroll
    for (int k4 = 0; k4 < kDim / 4; ++k4) {
      const float4 p = row[k4];
      acc = fmaf(p.x, x[4 * k4 + 0], acc);
      acc = fmaf(p.y, x[4 * k4 + 1], acc);
      acc = fmaf(p.z, x[4 * k4 + 2], acc);
      acc = fmaf(p.w, x[4 * k4 + 3], acc);
    }
    s_col[i * kDim + lane] = acc;
  }
#pragma unroll
  for (int i = 0; i < kDim; ++i) x[i] = s_col[i * kDim + lane];
}

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

// ----------------------------------------------------- lane-per-token kernel
// Block: 2 waves x 64 tokens of one (layer, sequence, head). Grid:
// x = ceil(T/128), y = B*H, z = nlayers. Dynamic LDS (64 KiB): Pi, S and one
// 64 x 64 column buffer per wave.
template <bool F16>
__global__ __launch_bounds__(128) void quantize_tiles_kernel(QuantArgs a) {
  extern __shared__ float smem[];
  float* s_pi = smem;
  float* s_S = smem + kDim * kDim;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float* s_col = smem + 2 * kDim * kDim + wave * kDim * kDim;

  const int h = blockIdx.y % a.H, b = blockIdx.y / a.H, li = blockIdx.z;
  const int l = a.layer0 + li;
  const int64_t lh = (int64_t)l * a.H + h;
  const bool rotated = (a.flags & kInputRotated) != 0;
  const bool paper = (a.flags & kQjlPaper) != 0;
  const int ksign = paper ? 2 : 1;
  const int vsign = (a.flags & kVQjl) ? ksign : 0;

  for (int e = threadIdx.x; e < kDim * kDim; e += blockDim.x) {
    s_pi[e] = a.pi[lh * kDim * kDim + e];
    s_S[e] = a.qjl_s[e];
  }
  const Levels Lk = load_levels(a.lut_k + lh * 8);
  const Levels Lv = load_levels(a.lut_v + lh * 8);
  __syncthreads();

  const int j0 = blockIdx.x * 128 + wave * kTile;
  const int j = j0 + lane;
  const int64_t sbase = a.slot0[b];
  const int pbase = a.pos0[b];
  const int64_t slot = sbase + j;
  const int pos = pbase + j;
  const bool ok = j < a.T && slot >= 0 && slot < a.slots &&
                  (rotated || (pos >= 0 && pos < a.rope_positions));
  const int64_t row = ((((int64_t)li * a.B + b) * a.T + j) * a.H + h) * kDim;

  uint8_t* kreg = a.k_codes + lh * a.slots * 32;
  uint8_t* vreg = a.v_codes + lh * a.slots * 32;

  // ---- K
  float x[kDim];
#pragma unroll
  for (int i = 0; i < kDim; ++i) x[i] = ok ? load_in(a.k, row + i, F16) : 0.0f;
  if (!rotated) {
    if (ok) rope_lane(x, a.rope_cs + (int64_t)pos * 2 * kPairs, (a.flags & kRopeHalf) != 0);
    rotate_lane(x, s_pi, s_col, lane);
  }
  uint32_t kw[8];
  const QuantOut qk = quantize_lane<true>(x, Lk, s_S, ksign, kw);
  if (ok) {
    const int64_t tile = slot >> 6;
    const int r = (int)(slot & 63);
    *reinterpret_cast<uint4*>(kreg + tile_half_offset(tile, 0, r)) = make_uint4(kw[0], kw[1], kw[2], kw[3]);
    *reinterpret_cast<uint4*>(kreg + tile_half_offset(tile, 1, r)) = make_uint4(kw[4], kw[5], kw[6], kw[7]);
  }

  // ---- V (no RoPE)
#pragma unroll
  for (int i = 0; i < kDim; ++i) x[i] = ok ? load_in(a.v, row + i, F16) : 0.0f;
  if (!rotated && (a.flags & kVRotate)) rotate_lane(x, s_pi, s_col, lane);
  uint32_t vw[8];
  const QuantOut qv = quantize_lane<false>(x, Lv, s_S, vsign, vw);
  if (ok) {
    *reinterpret_cast<uint2*>(a.scalars + (lh * a.slots + slot) * 4) =
        make_uint2(qk.n16 | (qk.g16 << 16), qv.n16 | (qv.g16 << 16));
  }

  // V is stored dimension-major: transpose the wave's 64 x 64 nibbles through
  // the lane's LDS column (token-major words in, one dimension per lane out).
  uint32_t* s_w = reinterpret_cast<uint32_t*>(s_col);
#pragma unroll
  for (int w = 0; w < 8; ++w) s_w[lane * 8 + w] = vw[w];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint64_t okmask = __ballot(ok);
  if (okmask != 0) {
    const int i = lane;   // dimension handled by this lane
    const int64_t sA = sbase + j0;           // slot of token j0
    const int64_t g_first = sA >> 3, g_last = (sA + 63) >> 3;
    for (int64_t G = g_first; G <= g_last; ++G) {
      uint32_t word = 0, mask = 0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const int64_t tau = G * 8 + jj - sA;
        if (tau >= 0 && tau < 64 && ((okmask >> tau) & 1ull)) {
          const uint32_t nib = (s_w[tau * 8 + (i >> 3)] >> (4 * (i & 7))) & 15u;
          word |= nib << (4 * jj);
          mask |= 15u << (4 * jj);
        }
      }
      if (mask) {
        const int64_t tile = G >> 3;
        const int c = (int)((G & 7) >> 2);
        uint32_t* addr = reinterpret_cast<uint32_t*>(vreg + tile_half_offset(tile, c, i) + (G & 3) * 4);
        store_v_word(addr, word, mask);
      }
    }
  }
}

// ----------------------------------------------- wave-per-vector kernel
// Block: 2 waves for one (layer, sequence, token, head): wave 0 quantizes the
// key, wave 1 the value; lane = dimension. Pi and S are read with coalesced
// 16-byte loads by the whole block and stored transposed in LDS (rows padded
// to 65 floats), so that lane i walks column i of the transpose, i.e. row i of
// the matrix, with conflict-free reads; the fma chains keep k ascending.
constexpr int kTStride = kDim + 1;

struct VectorSmem {
  float piT[kDim * kTStride];   // piT[k * 65 + i] = Pi[i][k]
  float sT[kDim * kTStride];    // sT[k * 65 + i] = S[i][k]
  float x[2][kDim];
  float r[2][kDim];
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Row i of a 64 x 64 matrix (stored transposed in `mT`) times the vector
// staged in `v`: fma chain over k ascending, the order of rotate_lane and
// quantize_lane.
__device__ __forceinline__ float row_dot_t(const float* mT, const float* v, int i) {
  float acc = 0.0f;
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) {
    const float4 vv = reinterpret_cast<const float4*>(v)[k4];
    acc = fmaf(mT[(4 * k4 + 0) * kTStride + i], vv.x, acc);
    acc = fmaf(mT[(4 * k4 + 1) * kTStride + i], vv.y, acc);
    acc = fmaf(mT[(4 * k4 + 2) * kTStride + i], vv.z, acc);
    acc = fmaf(mT[(4 * k4 + 3) * kTStride + i], vv.w, acc);
  }
  return acc;
}

// Quantize the vector whose element i lane i holds in `xh`; same arithmetic
// order as quantize_lane. Returns the lane's nibble; n16/g16 are uniform.
__device__ __forceinline__ uint32_t quantize_wave(float xh, const Levels& L,
                                                  const float* sT, int sign_mode, float* xs,
                                                  float* rs, int i, uint32_t* n16, uint32_t* g16) {
  xs[i] = xh;
  wave_sync_lds();
  float s = 0.0f;
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) {
    const float4 v = reinterpret_cast<const float4*>(xs)[k4];
    s = fmaf(v.x, v.x, s);
    s = fmaf(v.y, v.y, s);
    s = fmaf(v.z, v.z, s);
    s = fmaf(v.w, v.w, s);
  }
  const float n = sqrtf(s);
  const float inv = (n == 0.0f) ? 0.0f : 8.0f / n;
  const float u = xh * inv;
  TQ_PIN_LEVELS(L);
  uint32_t idx;
  const float lv = nearest_level(u, TQ_LEVELS(L), &idx);
  const float r = u - lv;
  rs[i] = r;
  wave_sync_lds();
  float gs = 0.0f;
#pragma unroll
  for (int k4 = 0; k4 < kDim / 4; ++k4) {
    const float4 v = reinterpret_cast<const float4*>(rs)[k4];
    gs = fmaf(v.x, v.x, gs);
    gs = fmaf(v.y, v.y, gs);
    gs = fmaf(v.z, v.z, gs);
    gs = fmaf(v.w, v.w, gs);
  }
  const float g = sqrtf(gs);
  uint32_t bit = 0;
  if (sign_mode == 1) {
    bit = (row_dot_t(sT, rs, i) < 0.0f) ? 0u : 1u;
  } else if (sign_mode == 2) {
    bit = (r < 0.0f) ? 0u : 1u;
  }
  *n16 = store_norm(n);
  *g16 = (sign_mode == 0) ? 0u : store_norm(g);
  return idx | (bit << 3);
}

// Coalesced copy of a 64 x 64 row-major matrix into its padded transpose, in
// two steps so that the loads can be issued early: thread t holds float4
// number t + 128 j (row e / 16, columns 4 (e % 16) .. 4 (e % 16) + 3).
struct MatrixSlice {
  float4 v[8];
};

__device__ __forceinline__ void load_slice(const float* __restrict__ m, MatrixSlice& sl, int t) {
#pragma unroll
  for (int j = 0; j < 8; ++j) sl.v[j] = reinterpret_cast<const float4*>(m)[t + 128 * j];
}

__device__ __forceinline__ void store_slice_transposed(const MatrixSlice& sl, float* mT, int t) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int e = t + 128 * j, row = e >> 4, col = (e & 15) * 4;
    mT[(col + 0) * kTStride + row] = sl.v[j].x;
    mT[(col + 1) * kTStride + row] = sl.v[j].y;
    mT[(col + 2) * kTStride + row] = sl.v[j].z;
    mT[(col + 3) * kTStride + row] = sl.v[j].w;
  }
}

template <bool F16>
__global__ __launch_bounds__(128) void quantize_vectors_kernel(QuantArgs a, uint32_t total) {
  __shared__ VectorSmem sm;
  const int wave = threadIdx.x >> 6, i = threadIdx.x & 63;
  const uint32_t th = blockIdx.x;   // the host keeps the token-head count below 2^31
  if (th >= total) return;
  const bool is_v = wave == 1;
  const uint32_t h = th % (uint32_t)a.H;
  uint32_t rest = th / (uint32_t)a.H;
  const uint32_t j = rest % (uint32_t)a.T;
  rest /= (uint32_t)a.T;
  const uint32_t b = rest % (uint32_t)a.B;
  const uint32_t li = rest / (uint32_t)a.B;
  const int l = a.layer0 + (int)li;
  const int64_t lh = (int64_t)l * a.H + h;
  const bool rotated = (a.flags & kInputRotated) != 0;
  const bool paper = (a.flags & kQjlPaper) != 0;
  const int ksign = paper ? 2 : 1;
  const int sign_mode = is_v ? ((a.flags & kVQjl) ? ksign : 0) : ksign;
  const bool any_rotate = !rotated;                       // keys rotate unless pre-rotated
  const bool rotate = !rotated && (!is_v || (a.flags & kVRotate));
  const bool any_proj = !paper;                           // keys use the projection unless paper
  const int64_t row = ((((int64_t)li * a.B + b) * a.T + j) * a.H + h) * kDim;

  // ---- loads that do not depend on the slot, issued first
  float x = load_in(is_v ? a.v : a.k, row + i, F16);
  const Levels L = load_levels((is_v ? a.lut_v : a.lut_k) + lh * 8);
  MatrixSlice pi_sl, s_sl;
  if (any_rotate) load_slice(a.pi + lh * kDim * kDim, pi_sl, threadIdx.x);
  if (any_proj) load_slice(a.qjl_s, s_sl, threadIdx.x);
  const int64_t slot = a.slot0[b] + j;
  const int pos = a.pos0[b] + (int)j;
  // block-uniform exits (before any barrier)
  if (slot < 0 || slot >= a.slots) return;
  if (!rotated && (pos < 0 || pos >= a.rope_positions)) return;
  const bool half = (a.flags & kRopeHalf) != 0;
  float2 cs = make_float2(1.0f, 0.0f);
  if (!is_v && !rotated) {
    const int m = half ? (i & 31) : (i >> 1);
    cs = reinterpret_cast<const float2*>(a.rope_cs + (int64_t)pos * 2 * kPairs)[m];
  }
  if (any_rotate) store_slice_transposed(pi_sl, sm.piT, threadIdx.x);
  if (any_proj) store_slice_transposed(s_sl, sm.sT, threadIdx.x);
  __syncthreads();

  // ---- RoPE (keys) and rotation
  if (!is_v && !rotated) {
    const int partner = half ? (i ^ 32) : (i ^ 1);
    const bool first = half ? (i < 32) : ((i & 1) == 0);
    const float xp = __shfl(x, partner, 64);
    // pair (a, b): x'_a = x_a c - x_b s, x'_b = x_a s + x_b c
    x = first ? (x * cs.x - xp * cs.y) : (xp * cs.y + x * cs.x);
  }
  float* xs = sm.x[wave];
  float* rs = sm.r[wave];
  if (rotate) {
    xs[i] = x;
    wave_sync_lds();
    x = row_dot_t(sm.piT, xs, i);
    wave_sync_lds();   // xs is rewritten by quantize_wave
  }

  uint32_t n16, g16;
  const uint32_t nib = quantize_wave(x, L, sm.sT, sign_mode, xs, rs, i, &n16, &g16);
  const int64_t tile = slot >> 6;
  const int r = (int)(slot & 63);
  if (!is_v) {
    // key: token-major key words (index bits 3j, sign bit 24 + j); lane 8w
    // ends with word w
    uint32_t word = key_code_bits(nib & 7u, nib >> 3, i & 7);
    word |= __shfl_xor(word, 1, 64);
    word |= __shfl_xor(word, 2, 64);
    word |= __shfl_xor(word, 4, 64);
    uint8_t* kreg = a.k_codes + lh * a.slots * 32;
    if ((i & 7) == 0) {
      const int w = i >> 3;
      *reinterpret_cast<uint32_t*>(kreg + tile_half_offset(tile, w >> 2, r) + (w & 3) * 4) = word;
    }
    if (i == 0) reinterpret_cast<uint32_t*>(a.scalars + (lh * a.slots + slot) * 4)[0] = n16 | (g16 << 16);
  } else {
    // value: dimension-major, one nibble of dimension i's word for this slot
    uint8_t* vreg = a.v_codes + lh * a.slots * 32;
    const int cc = r >> 5, G4 = (r & 31) >> 3, jj = r & 7;
    uint32_t* addr = reinterpret_cast<uint32_t*>(vreg + tile_half_offset(tile, cc, i) + G4 * 4);
    store_v_word(addr, nib << (4 * jj), 15u << (4 * jj));
    if (i == 0) reinterpret_cast<uint32_t*>(a.scalars + (lh * a.slots + slot) * 4)[1] = n16 | (g16 << 16);
  }
}

hipError_t launch_quantize(const QuantArgs& a, hipStream_t st) {
  const bool f16 = a.f16 && !(a.flags & kInputRotated);
  if (a.T >= 64) {
    dim3 grid((a.T + 127) / 128, a.B * a.H, a.nlayers);
    const size_t lds = (size_t)(2 + 2) * kDim * kDim * sizeof(float);
    if (f16)
      hipLaunchKernelGGL(quantize_tiles_kernel<true>, grid, dim3(128), lds, st, a);
    else
      hipLaunchKernelGGL(quantize_tiles_kernel<false>, grid, dim3(128), lds, st, a);
  } else {
    const uint32_t total = (uint32_t)((int64_t)a.nlayers * a.B * a.T * a.H);
    if (f16)
      hipLaunchKernelGGL(quantize_vectors_kernel<true>, dim3(total), dim3(128), 0, st, a, total);
    else
      hipLaunchKernelGGL(quantize_vectors_kernel<false>, dim3(total), dim3(128), 0, st, a, total);
  }
  return hipGetLastError();
}

}  // namespace tq
