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
#include "tq_append.hpp"
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
// Coalesced copy of a 64 x 64 row-major matrix into its staged form, in two
// steps so that the loads can be issued early: thread t holds float4 number
// t + 128 j (row e / 16, columns 4 (e % 16) .. 4 (e % 16) + 3).
struct MatrixSlice {
  float4 v[8];
};

__device__ __forceinline__ void load_slice(const float* __restrict__ m, MatrixSlice& sl, int t) {
#pragma unroll
  for (int j = 0; j < 8; ++j) sl.v[j] = reinterpret_cast<const float4*>(m)[t + 128 * j];
}

__device__ __forceinline__ void store_slice(const MatrixSlice& sl, float* m, int t) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int e = t + 128 * j;
    stage_row4(m, e >> 4, (e & 15) * 4, sl.v[j]);
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
  if (any_rotate) store_slice(pi_sl, sm.pi, threadIdx.x);
  if (any_proj) store_slice(s_sl, sm.s, threadIdx.x);
  __syncthreads();

  // ---- RoPE (keys), rotation, quantizer, store
  if (!is_v && !rotated) x = rope_wave(x, cs, half, i);
  append_wave<Pitch68>(x, is_v, rotate, L, sm.pi, sm.s, sm.x[wave], sm.r[wave], sign_mode, slot, lh,
                       a.k_codes, a.v_codes, a.scalars, a.slots, i);
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
