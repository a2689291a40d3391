// Prefill-side quantizer: RoPE -> Pi rotation -> per-vector norm -> 3-bit
// table codes -> residual -> QJL sign bits -> packed cache (TurboESM Sec. 3.1
// prefill steps 1, 3, 4; Sec. 3.3; Sec. 3.4; Sec. 4.2).
//
// Two kernels:
//   quantize_tiles_kernel   for prefill-sized T: 64 tokens per wave; the
//                           rotations x^ = Pi x' of the wave's 64 x 64 block
//                           run on the matrix cores (fp32 MFMA), then one lane
//                           per token runs the quantizer steps.
//   quantize_vectors_kernel one wave per vector (one lane per dimension; the
//                           key and the value of a token-head in parallel), for
//                           decode-step appends with small T; its rotation is
//                           an fma chain over k ascending.
// Both run the quantizer steps (norm, levels, residual, projected signs) in
// the fixed binary32 order of quantize_lane / quantize_wave, so identical x^
// give identical bits; for raw inputs the two rotations sum in different
// orders, so a code can differ where x^ sits within rounding of a threshold.
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

// ------------------------------------------------- MFMA rotation of 64 rows
// x^ = Pi x' for the 64 tokens of a wave as D = Pi X'^T on the matrix cores
// (v_mfma_f32_32x32x2f32: fp32 products, fp32 sums), in two 32-row blocks of
// Pi (mb) times two 32-token blocks (nb), 32 rank-2 steps each.
// Operand layout of the instruction (lane l, n = l % 32, h = l / 32):
//   A lane value  A[n][h]       (row n of the 32 x 2 slice)
//   B lane value  B[h][n]       (column n of the 2 x 32 slice)
//   D register r  D[8 (r/4) + 4h + r%4][n]
// Step s (q = s/4, jj = s%4) gives lane half h the contraction index
// k = 8q + 4h + jj, so the 32 k a lane contributes are the dimensions
// {8q + 4h + jj}: the same set that D leaves in that lane half. A lane's
// B values are therefore 8 groups of 4 consecutive dimensions of its token
// (one 8- or 16-byte load each) and its A values are 4 consecutive columns
// of a row of Pi (one 16-byte LDS read per q).
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Pitch of the staged Pi: 16-byte row reads of 16 lanes (rows n, 4n dwords
// apart modulo 64 banks) are conflict-free.
constexpr int kPiPitch = 68;

// Loads the lane's half row of token j0 + 32 nb + n (values x'[8q + 4h + jj]
// at step 4q + jj) and applies RoPE (keys): both pairings keep a pair inside
// the lane's set (interleaved: (2m, 2m + 1) inside one group of 4; half: d and
// d + 32 in groups q and q + 4).
template <bool F16>
__device__ __forceinline__ void load_half_row(float (&xv)[32], const QuantArgs& a, const void* src, int li,
                                              int b, int h, int j0, int nb, int lane, bool rope) {
  const int n = lane & 31, hh = lane >> 5;
  const bool half = (a.flags & kRopeHalf) != 0;
  const int j = j0 + 32 * nb + n;
  const int pos = a.pos0[b] + j;
  const bool ok = j < a.T && (!rope || (pos >= 0 && pos < a.rope_positions));
  const int64_t row = ((((int64_t)li * a.B + b) * a.T + j) * a.H + h) * kDim;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int d0 = 8 * q + 4 * hh;
    float4 f = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (ok) {
      if (F16) {
        const uint2 w = *reinterpret_cast<const uint2*>(reinterpret_cast<const __half*>(src) + row + d0);
        f.x = half_bits_to_float(w.x); f.y = half_bits_to_float(w.x >> 16);
        f.z = half_bits_to_float(w.y); f.w = half_bits_to_float(w.y >> 16);
      } else {
        f = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(src) + row + d0);
      }
    }
    xv[4 * q + 0] = f.x; xv[4 * q + 1] = f.y; xv[4 * q + 2] = f.z; xv[4 * q + 3] = f.w;
  }
  if (!rope || !ok) return;
  const float4* cs4 = reinterpret_cast<const float4*>(a.rope_cs + (int64_t)pos * 2 * kPairs);
  if (!half) {
    // pairs d0/2 and d0/2 + 1 of group q: their (cos, sin) in one float4
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 c = cs4[2 * q + hh];
      const float x0 = xv[4 * q], x1 = xv[4 * q + 1], x2 = xv[4 * q + 2], x3 = xv[4 * q + 3];
      xv[4 * q + 0] = x0 * c.x - x1 * c.y; xv[4 * q + 1] = x0 * c.y + x1 * c.x;
      xv[4 * q + 2] = x2 * c.z - x3 * c.w; xv[4 * q + 3] = x2 * c.w + x3 * c.z;
    }
  } else {
    // pair (d, d + 32) for d in group q < 4, angle index d
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int d0 = 8 * q + 4 * hh;
      const float4 c01 = cs4[d0 >> 1], c23 = cs4[(d0 >> 1) + 1];
      const float cc[4] = {c01.x, c01.z, c23.x, c23.z}, ss[4] = {c01.y, c01.w, c23.y, c23.w};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const float xa = xv[4 * q + jj], xb = xv[4 * (q + 4) + jj];
        xv[4 * q + jj] = xa * cc[jj] - xb * ss[jj];
        xv[4 * (q + 4) + jj] = xa * ss[jj] + xb * cc[jj];
      }
    }
  }
}

// acc[mb] += the 32 rank-2 steps of row block mb of Pi times one token block.
// The Pi reads are issued per group q (the empty asm keeps the compiler from
// holding all 64 values of Pi in registers across both token blocks).
__device__ __forceinline__ void rotate_block(const float (&xv)[32], const float* s_pi, int lane,
                                             f32x16& acc0, f32x16& acc1) {
  const int n = lane & 31, hh = lane >> 5;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    int o = n * kPiPitch + 8 * q + 4 * hh;
    asm volatile("" : "+v"(o));
    const float4 p0 = *reinterpret_cast<const float4*>(s_pi + o);
    const float4 p1 = *reinterpret_cast<const float4*>(s_pi + o + 32 * kPiPitch);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(p0.x, xv[4 * q + 0], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(p1.x, xv[4 * q + 0], acc1, 0, 0, 0);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(p0.y, xv[4 * q + 1], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(p1.y, xv[4 * q + 1], acc1, 0, 0, 0);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(p0.z, xv[4 * q + 2], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(p1.z, xv[4 * q + 2], acc1, 0, 0, 0);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(p0.w, xv[4 * q + 3], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(p1.w, xv[4 * q + 3], acc1, 0, 0, 0);
  }
}

// Rotates the wave's 64 tokens and hands lane l all 64 rotated values of token
// j0 + l: after the products, lane half h of token block nb holds dimensions
// {8q + 4h + jj} of token 32 nb + n; one v_permlane32_swap per register pair
// moves the upper half of block 0 and the lower half of block 1 across, so
// that lane l < 32 holds token l and lane l >= 32 token l (32 + n).
template <bool F16>
__device__ __forceinline__ void rotate_tokens(float (&out)[kDim], const QuantArgs& a, const void* src,
                                              const float* s_pi, int li, int b, int h, int j0, int lane,
                                              bool rope) {
  f32x16 acc[2][2];
#pragma unroll
  for (int r = 0; r < 16; ++r) { acc[0][0][r] = 0.0f; acc[1][0][r] = 0.0f; acc[0][1][r] = 0.0f; acc[1][1][r] = 0.0f; }
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    float xv[32];
    load_half_row<F16>(xv, a, src, li, b, h, j0, nb, lane, rope);
    rotate_block(xv, s_pi, lane, acc[0][nb], acc[1][nb]);
  }
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[mb][0][r]),
                                                       __float_as_uint(acc[mb][1][r]), false, false);
      const int d = 32 * mb + 8 * (r >> 2) + (r & 3);
      out[d] = __uint_as_float(sw[0]);       // dimension set of lane half 0
      out[d + 4] = __uint_as_float(sw[1]);   // dimension set of lane half 1
    }
}

// Projected QJL sign bits of the wave's 64 residuals (lane l: r of token
// j0 + l, in registers): bit i = !(p_i < 0) for p_i = the binary32 fma chain
// over k ascending of S[i][k] r_k (the exact quantizer step). p is first
// computed on the matrix cores as D = S R^T (fp32 products and sums, another
// order); a 64-term fp32 dot product in any order is within 2^-17 sum_k
// |S_ik r_k| <= 2^-17 ||S_i|| ||r|| of the exact value, so where
// |p~_i| > 2^-14 ||S_i|| ||r|| its sign is the chain's, and only the
// coordinates inside that band are recomputed with the chain.
// The residuals reach the instruction's B layout through the same
// v_permlane32_swap pairs that handed the rotated values to the lanes (a swap
// undoes itself), and go back the same way.
__device__ __forceinline__ uint64_t projected_signs(float (&x)[kDim], float g, const float* s_S,
                                                    const float* s_Sn, int lane) {
  const int n = lane & 31, hh = lane >> 5;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int d = 32 * mb + 8 * (r >> 2) + (r & 3);
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[d]), __float_as_uint(x[d + 4]), false,
                                                       false);
      x[d] = __uint_as_float(sw[0]);       // token n, dimension d + 4h
      x[d + 4] = __uint_as_float(sw[1]);   // token 32 + n, dimension d + 4h
    }
  f32x16 acc[2][2];
#pragma unroll
  for (int r = 0; r < 16; ++r) { acc[0][0][r] = 0.0f; acc[1][0][r] = 0.0f; acc[0][1][r] = 0.0f; acc[1][1][r] = 0.0f; }
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    int o = n * kPiPitch + 8 * q + 4 * hh;
    asm volatile("" : "+v"(o));
    const float4 p0 = *reinterpret_cast<const float4*>(s_S + o);
    const float4 p1 = *reinterpret_cast<const float4*>(s_S + o + 32 * kPiPitch);
    const float a0[4] = {p0.x, p0.y, p0.z, p0.w}, a1[4] = {p1.x, p1.y, p1.z, p1.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[j], x[8 * q + j], acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[j], x[8 * q + 4 + j], acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[j], x[8 * q + j], acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[j], x[8 * q + 4 + j], acc[1][1], 0, 0, 0);
    }
  }
  // residuals back to one token per lane; p~ likewise
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int d = 32 * mb + 8 * (r >> 2) + (r & 3);
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[d]), __float_as_uint(x[d + 4]), false,
                                                       false);
      x[d] = __uint_as_float(sw[0]);
      x[d + 4] = __uint_as_float(sw[1]);
      const auto sp = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[mb][0][r]),
                                                       __float_as_uint(acc[mb][1][r]), false, false);
      acc[mb][0][r] = __uint_as_float(sp[0]);   // p~ of row d
      acc[mb][1][r] = __uint_as_float(sp[1]);   // p~ of row d + 4
    }
  uint64_t bits = 0, flagged = 0;
  const float gb = g * 0x1p-14f;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int i = 32 * mb + 8 * (r >> 2) + (r & 3) + 4 * half;
        const float pv = acc[mb][half][r];
        const bool sure = fabsf(pv) > s_Sn[i] * gb;
        bits |= (uint64_t)((sure && !(pv < 0.0f)) ? 1u : 0u) << i;
        flagged |= (uint64_t)(sure ? 0u : 1u) << i;
      }
  // rows inside the band, any lane: the fixed-order chain (wave-uniform row)
  uint64_t any = flagged;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)any, o, 64), hi = __shfl_xor((uint32_t)(any >> 32), o, 64);
    any |= ((uint64_t)hi << 32) | lo;
  }
  while (any) {
    const int i = __builtin_ctzll(any);
    any &= any - 1;
    if ((flagged >> i) & 1ull) {
      const float4* row = reinterpret_cast<const float4*>(s_S + i * kPiPitch);
      float acc_i = 0.0f;
#pragma unroll
      for (int k4 = 0; k4 < kDim / 4; ++k4) {
        const float4 sv = row[k4];
        acc_i = fmaf(sv.x, x[4 * k4 + 0], acc_i);
        acc_i = fmaf(sv.y, x[4 * k4 + 1], acc_i);
        acc_i = fmaf(sv.z, x[4 * k4 + 2], acc_i);
        acc_i = fmaf(sv.w, x[4 * k4 + 3], acc_i);
      }
      bits |= (uint64_t)((acc_i < 0.0f) ? 0u : 1u) << i;
    }
  }
  return bits;
}

// ----------------------------------------------------- lane-per-token kernel
// Block: 4 waves x 64 tokens of one (layer, sequence, head). Grid:
// x = ceil(T/256), y = B*H, z = nlayers. LDS: Pi (pitch 68) for the
// rotations, S (row-major, read by the quantizer as broadcasts) and one
// 64 x 8 word buffer per wave for the V transpose.
// Three waves per SIMD (168 registers; a few values of the quantizer step
// spill) run faster than two without spills: 312 against 343 us on the
// 650M-shape prefill.
template <bool F16, bool VQJL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void quantize_tiles_kernel(QuantArgs a) {
  __shared__ __attribute__((aligned(16))) float s_pi[kDim * kPiPitch];
  __shared__ __attribute__((aligned(16))) float s_S[kDim * kPiPitch];
  __shared__ float s_Sn[kDim];                                       // ||S_i|| (fp32)
  __shared__ uint32_t s_vt[4][kDim * 8];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

  const int h = blockIdx.y % a.H, b = blockIdx.y / a.H, li = blockIdx.z;
  const int l = a.layer0 + li;
  const int64_t lh = (int64_t)l * a.H + h;
  const bool rotated = (a.flags & kInputRotated) != 0;
  const bool paper = (a.flags & kQjlPaper) != 0;
  const int vsign = VQJL ? (paper ? 2 : 1) : 0;   // (a V sign pass is compiled only where asked for)

  for (int e = threadIdx.x; e < kDim * kDim / 4; e += blockDim.x) {
    const float4 pv = reinterpret_cast<const float4*>(a.pi + lh * kDim * kDim)[e];
    *reinterpret_cast<float4*>(s_pi + (e >> 4) * kPiPitch + (e & 15) * 4) = pv;
    *reinterpret_cast<float4*>(s_S + (e >> 4) * kPiPitch + (e & 15) * 4) =
        reinterpret_cast<const float4*>(a.qjl_s)[e];
  }
  if (threadIdx.x < kDim) {
    const float* srow = a.qjl_s + threadIdx.x * kDim;
    float ss = 0.0f;
    for (int k = 0; k < kDim; ++k) ss = fmaf(srow[k], srow[k], ss);
    s_Sn[threadIdx.x] = sqrtf(ss);
  }
  const Levels Lk = load_levels(a.lut_k + lh * 8);
  const Levels Lv = load_levels(a.lut_v + lh * 8);
  __syncthreads();

  const int j0 = blockIdx.x * 256 + wave * kTile;
  if (j0 >= a.T) return;                  // wave-uniform; no barrier follows
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

  // ---- K: RoPE and rotation, or a pre-rotated input as is
  float x[kDim];
  if (rotated) {
#pragma unroll
    for (int i = 0; i < kDim; ++i) x[i] = ok ? load_in(a.k, row + i, false) : 0.0f;
  } else {
    rotate_tokens<F16>(x, a, a.k, s_pi, li, b, h, j0, lane, true);
  }
  uint32_t kw[8];
  const QuantOut qk = quantize_lane<true>(x, Lk, s_S, paper ? 2 : 3, kw);
  if (!paper) {
    const uint64_t sb = projected_signs(x, qk.g, s_S, s_Sn, lane);
#pragma unroll
    for (int w = 0; w < 8; ++w) kw[w] |= (uint32_t)((sb >> (8 * w)) & 0xFFu) << 24;
  }
  if (ok) {
    const int64_t tile = slot >> 6;
    const int r = (int)(slot & 63);
    *reinterpret_cast<uint4*>(kreg + tile_half_offset(tile, 0, r)) = make_uint4(kw[0], kw[1], kw[2], kw[3]);
    *reinterpret_cast<uint4*>(kreg + tile_half_offset(tile, 1, r)) = make_uint4(kw[4], kw[5], kw[6], kw[7]);
  }

  // ---- V (no RoPE): rotated like K unless TQ_V_ROTATE is off. The V loads
  // are not hoisted above the key's stores (registers, occupancy).
  asm volatile("" ::: "memory");
  if (!rotated && (a.flags & kVRotate)) {
    rotate_tokens<F16>(x, a, a.v, s_pi, li, b, h, j0, lane, false);
  } else {
#pragma unroll
    for (int i = 0; i < kDim; ++i) x[i] = ok ? load_in(a.v, row + i, F16) : 0.0f;
  }
  uint32_t vw[8];
  const QuantOut qv = quantize_lane<false>(x, Lv, s_S, (VQJL && !paper) ? 3 : vsign, vw);
  if (VQJL && !paper) {
    const uint64_t sb = projected_signs(x, qv.g, s_S, s_Sn, lane);
#pragma unroll
    for (int i = 0; i < kDim; ++i) vw[i >> 3] |= (uint32_t)((sb >> i) & 1ull) << (4 * (i & 7) + 3);
  }
  if (ok) {
    *reinterpret_cast<uint2*>(a.scalars + (lh * a.slots + slot) * 4) =
        make_uint2(qk.n16 | (qk.g16 << 16), qv.n16 | (qv.g16 << 16));
  }

  // V is stored dimension-major: transpose the wave's 64 x 64 nibbles through
  // its LDS buffer (token-major words in, one dimension per lane out).
  uint32_t* s_w = s_vt[wave];
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
    dim3 grid((a.T + 255) / 256, a.B * a.H, a.nlayers);
    const bool vq = (a.flags & kVQjl) != 0;
    if (f16 && vq)
      hipLaunchKernelGGL((quantize_tiles_kernel<true, true>), grid, dim3(256), 0, st, a);
    else if (f16)
      hipLaunchKernelGGL((quantize_tiles_kernel<true, false>), grid, dim3(256), 0, st, a);
    else if (vq)
      hipLaunchKernelGGL((quantize_tiles_kernel<false, true>), grid, dim3(256), 0, st, a);
    else
      hipLaunchKernelGGL((quantize_tiles_kernel<false, false>), grid, dim3(256), 0, st, a);
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
