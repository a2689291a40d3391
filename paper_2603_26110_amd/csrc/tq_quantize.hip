// Prefill-side quantizer: RoPE -> Pi rotation -> per-vector norm -> 3-bit
// table codes -> residual -> QJL sign bits -> packed cache (TurboESM Sec. 3.1
// prefill steps 1, 3, 4; Sec. 3.3; Sec. 3.4; Sec. 4.2).
//
// Two kernels:
//   quantize_tiles_kernel   for prefill-sized T: 64 tokens per wave; the
//                           rotations x^ = Pi x' of the wave's 64 x 64 block
//                           and the projections S r run on the matrix cores
//                           (fp16 MFMA on hi/lo parts), one lane per token
//                           runs the quantizer steps.
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

// ------------------------------------------- matrix-core products of 64 rows
// Two dense 64 x 64 x 64 products per wave run on the matrix cores: the
// rotation x^ = Pi x' of the wave's 64 tokens and the QJL projection S r of
// their residuals. Both use v_mfma_f32_32x32x16_f16 (fp16 inputs, fp32 sums)
// with each fp32 operand split into fp16 parts hi = fp16(v), lo = fp16(v - hi)
// and three products hi*hi + hi*lo + lo*hi, which carries a product to about
// 2^-21 relative. Each token's vector is first scaled by a power of two
// (exact) so that its largest entry lies in [1, 2), and each row of S
// likewise, which keeps the parts in fp16's range; the results are scaled
// back (exact) or compared with equally scaled bounds.
// Instruction layout (lane l, n = l % 32, h = l / 32; verified on gfx950):
//   A lane values A[n][8h + j], B lane values B[8h + j][n] (j = 0..7),
//   D register r D[8 (r/4) + 4h + r%4][n].
// Step q (0..3) contracts k = 16q + 8h + j: a lane's B values at step q are 8
// consecutive dimensions of its token (one 16-byte load of fp16 input) and
// its A values 8 consecutive columns of a row of the staged matrix (one
// 16-byte LDS read per part). The result leaves lane half h the dimensions
// {8q + 4h + j, j < 4} of its two tokens (32 nb + n, nb = 0, 1); one
// v_permlane32_swap per register pair then hands lane l all 64 values of
// token l.
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));

// Halfs per staged row: the 16-byte reads of 16 rows (36 dwords apart) fall
// on all 64 banks once.
constexpr int kHPitch = 72;

struct SplitOps {
  half8 hi[2][4], lo[2][4];   // [token block nb][step q]
};

__device__ __forceinline__ void split8(const float* v, float sc, half8& hi, half8& lo) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float x = v[j] * sc;
    const _Float16 a = (_Float16)x;
    hi[j] = a;
    lo[j] = (_Float16)(x - (float)a);
  }
}

// 2^(1 - e) for m = f 2^e, f in [0.5, 1): m times it lies in [1, 2); 1 for m = 0.
__device__ __forceinline__ float unit_scale(float m) {
  if (!(m > 0.0f)) return 1.0f;
  int e;
  frexpf(m, &e);
  return ldexpf(1.0f, 1 - e);
}

// acc[mb][nb] = rows 32 mb .. 32 mb + 31 of the staged matrix times the
// wave's token blocks, as hi*hi + hi*lo + lo*hi.
__device__ __forceinline__ void split_products(const SplitOps& b, const _Float16* mh, const _Float16* ml,
                                               int lane, f32x16 (&acc)[2][2]) {
  const int n = lane & 31, hh = lane >> 5;
#pragma unroll
  for (int r = 0; r < 16; ++r) { acc[0][0][r] = 0.0f; acc[1][0][r] = 0.0f; acc[0][1][r] = 0.0f; acc[1][1][r] = 0.0f; }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int o = n * kHPitch + 16 * q + 8 * hh;
    asm volatile("" : "+v"(o));
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const half8 ah = *reinterpret_cast<const half8*>(mh + o + 32 * mb * kHPitch);
      const half8 al = *reinterpret_cast<const half8*>(ml + o + 32 * mb * kHPitch);
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, b.hi[nb][q], acc[mb][nb], 0, 0, 0);
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, b.lo[nb][q], acc[mb][nb], 0, 0, 0);
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al, b.hi[nb][q], acc[mb][nb], 0, 0, 0);
      }
    }
  }
}

// D blocks -> lane l holds all 64 rows for token l (column l of the block pair).
__device__ __forceinline__ void to_lane_per_token(f32x16 (&acc)[2][2], float (&out)[kDim]) {
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[mb][0][r]),
                                                       __float_as_uint(acc[mb][1][r]), false, false);
      const int d = 32 * mb + 8 * (r >> 2) + (r & 3);
      out[d] = __uint_as_float(sw[0]);       // row set of lane half 0
      out[d + 4] = __uint_as_float(sw[1]);   // row set of lane half 1
    }
}

// Loads the lane's values x'[16q + 8h + j] of tokens j0 + n (nb = 0) and
// j0 + 32 + n (nb = 1), applies RoPE (keys; both pairings keep a pair inside
// the lane: (2m, 2m + 1) inside a group of 8, (d, d + 32) in groups q and
// q + 2), scales each token by a power of two and splits it. Returns the
// lane's token scale (of token j0 + lane, for scaling the result back).
template <bool F16>
__device__ __forceinline__ float load_split_rows(SplitOps& ops, const QuantArgs& a, const void* src, int li,
                                                 int b, int h, int j0, int Tb, int lane, bool rope) {
  const int n = lane & 31, hh = lane >> 5;
  const bool half = (a.flags & kRopeHalf) != 0;
  float sc_nb[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int j = j0 + 32 * nb + n;
    const int pos = a.pos0[b] + j;
    const bool ok = j < Tb && (!rope || (pos >= 0 && pos < a.rope_positions));
    const int64_t row = ((((int64_t)li * a.B + b) * a.T + j) * a.H + h) * kDim;
    float xv[32];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int d0 = 16 * q + 8 * hh;
      if (F16) {
        uint4 w = make_uint4(0, 0, 0, 0);
        if (ok) w = *reinterpret_cast<const uint4*>(reinterpret_cast<const __half*>(src) + row + d0);
        const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          xv[8 * q + 2 * p] = half_bits_to_float(ww[p]);
          xv[8 * q + 2 * p + 1] = half_bits_to_float(ww[p] >> 16);
        }
      } else {
        float4 f0 = make_float4(0.0f, 0.0f, 0.0f, 0.0f), f1 = f0;
        if (ok) {
          f0 = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(src) + row + d0);
          f1 = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(src) + row + d0 + 4);
        }
        xv[8 * q + 0] = f0.x; xv[8 * q + 1] = f0.y; xv[8 * q + 2] = f0.z; xv[8 * q + 3] = f0.w;
        xv[8 * q + 4] = f1.x; xv[8 * q + 5] = f1.y; xv[8 * q + 6] = f1.z; xv[8 * q + 7] = f1.w;
      }
    }
    if (rope && ok) {
      const float4* cs4 = reinterpret_cast<const float4*>(a.rope_cs + (int64_t)pos * 2 * kPairs);
      if (!half) {
        // pairs m = (16q + 8h)/2 + p, p = 0..3: (cos, sin) of two pairs per float4
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int pp = 0; pp < 2; ++pp) {
            const float4 c = cs4[(16 * q + 8 * hh) / 4 + pp];
            float* g = &xv[8 * q + 4 * pp];
            const float x0 = g[0], x1 = g[1], x2 = g[2], x3 = g[3];
            g[0] = x0 * c.x - x1 * c.y; g[1] = x0 * c.y + x1 * c.x;
            g[2] = x2 * c.z - x3 * c.w; g[3] = x2 * c.w + x3 * c.z;
          }
      } else {
        // pair (d, d + 32), d = 16q + 8h + j for q < 2, angle index d
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int j4 = 0; j4 < 4; ++j4) {
            const float4 c = cs4[(16 * q + 8 * hh) / 2 + j4];   // (c, s) of d and d + 1
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
              const int jj = 2 * j4 + t2;
              const float cc = t2 ? c.z : c.x, ss = t2 ? c.w : c.y;
              const float xa = xv[8 * q + jj], xb = xv[8 * (q + 2) + jj];
              xv[8 * q + jj] = xa * cc - xb * ss;
              xv[8 * (q + 2) + jj] = xa * ss + xb * cc;
            }
          }
      }
    }
    float m = 0.0f;
#pragma unroll
    for (int k = 0; k < 32; ++k) m = fmaxf(m, fabsf(xv[k]));
    m = fmaxf(m, __shfl_xor(m, 32, 64));   // the token's other 32 values sit in lane l ^ 32
    sc_nb[nb] = unit_scale(m);
#pragma unroll
    for (int q = 0; q < 4; ++q) split8(&xv[8 * q], sc_nb[nb], ops.hi[nb][q], ops.lo[nb][q]);
  }
  return hh ? sc_nb[1] : sc_nb[0];
}

// x^ of token j0 + lane in out[64] (Pi staged as fp16 parts).
template <bool F16>
__device__ __forceinline__ void rotate_tokens(float (&out)[kDim], const QuantArgs& a, const void* src,
                                              const _Float16* pih, const _Float16* pil, int li, int b, int h,
                                              int j0, int Tb, int lane, bool rope) {
  SplitOps ops;
  const float sc = load_split_rows<F16>(ops, a, src, li, b, h, j0, Tb, lane, rope);
  f32x16 acc[2][2];
  split_products(ops, pih, pil, lane, acc);
  to_lane_per_token(acc, out);
  const float inv = 1.0f / sc;   // a power of two: exact
#pragma unroll
  for (int d = 0; d < kDim; ++d) out[d] *= inv;
}

// Projected QJL sign bits of the wave's 64 residuals (lane l: r of token
// j0 + l): bit i = !(p_i < 0) for p_i the binary32 fma chain over k
// ascending of S[i][k] r_k (the exact quantizer step). p~ = (sigma_i S_i) .
// (s r) comes from the matrix cores (sigma_i, s: the row's and the token's
// power-of-two scales). Any evaluation of it there is within
// 2^-17.3 ||sigma_i S_i|| ||s r|| of its exact value (2^-21 per split
// product, the fp16 spacing below the unit-sized entries, and fp32 sums of
// 64 terms) and the chain within 2^-18 of that, so where
// |p~_i| > 2^-14 ||sigma_i S_i|| ||s r|| the signs agree; the coordinates
// inside that band are recomputed with the chain from S in memory.
// The residuals reach the B layout through v_permlane32_swap pairs
// (16q + j, 16q + 8 + j) and go back the same way (a swap undoes itself).
__device__ __forceinline__ uint64_t projected_signs(float (&x)[kDim], float g, const _Float16* sh,
                                                    const _Float16* sl, const float* s_Sn, const float* S,
                                                    int lane) {
  const int n = lane & 31, hh = lane >> 5;
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < kDim; ++k) m = fmaxf(m, fabsf(x[k]));
  const float sc = unit_scale(m);                    // token l's scale
  const float sc_other = __shfl_xor(sc, 32, 64);     // token l ^ 32's
  const float sc0 = hh ? sc_other : sc, sc1 = hh ? sc : sc_other;   // tokens n, 32 + n
  // Step q's operands are built just before its products, from swapped
  // copies (x keeps the lane-per-token layout for the chain below).
  f32x16 acc[2][2];
#pragma unroll
  for (int r = 0; r < 16; ++r) { acc[0][0][r] = 0.0f; acc[1][0][r] = 0.0f; acc[0][1][r] = 0.0f; acc[1][1][r] = 0.0f; }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float b0[8], b1[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[16 * q + j]),
                                                       __float_as_uint(x[16 * q + 8 + j]), false, false);
      b0[j] = __uint_as_float(sw[0]);   // token n, dimension 16q + 8h + j
      b1[j] = __uint_as_float(sw[1]);   // token 32 + n, dimension 16q + 8h + j
    }
    half8 h0, l0, h1, l1;
    split8(b0, sc0, h0, l0);
    split8(b1, sc1, h1, l1);
    int o = n * kHPitch + 16 * q + 8 * hh;
    asm volatile("" : "+v"(o));
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const half8 ah = *reinterpret_cast<const half8*>(sh + o + 32 * mb * kHPitch);
      const half8 al = *reinterpret_cast<const half8*>(sl + o + 32 * mb * kHPitch);
      acc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, h0, acc[mb][0], 0, 0, 0);
      acc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, l0, acc[mb][0], 0, 0, 0);
      acc[mb][0] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al, h0, acc[mb][0], 0, 0, 0);
      acc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, h1, acc[mb][1], 0, 0, 0);
      acc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, l1, acc[mb][1], 0, 0, 0);
      acc[mb][1] = __builtin_amdgcn_mfma_f32_32x32x16_f16(al, h1, acc[mb][1], 0, 0, 0);
    }
  }
  // the result reaches lane l (token l) one register pair at a time and is
  // tested at once (no 64-value copy of it is held)
  uint64_t bits = 0, flagged = 0;
  const float gb = g * sc * 0x1p-14f;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[mb][0][r]),
                                                       __float_as_uint(acc[mb][1][r]), false, false);
      const int d = 32 * mb + 8 * (r >> 2) + (r & 3);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int i = d + 4 * e;
        const float pv = __uint_as_float(sw[e]);
        const bool sure = fabsf(pv) > s_Sn[i] * gb;
        bits |= (uint64_t)((sure && !(pv < 0.0f)) ? 1u : 0u) << i;
        flagged |= (uint64_t)(sure ? 0u : 1u) << i;
      }
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
      const float4* row = reinterpret_cast<const float4*>(S + i * kDim);
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
// Three waves per SIMD (168 registers, no spills for the default flags: the
// key words and the value words wait in LDS while their signs are computed,
// per-lane slot facts are recomputed where used, a level's index is found by
// a three-step search whose comparisons each write VCC only). Asking the
// compiler for four waves per SIMD gives 232 registers (two waves) instead:
// the two rotations' and the projection's 64-value results and their
// operands do not fit in 128.
template <bool F16, bool VQJL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void quantize_tiles_kernel(QuantArgs a) {
  __shared__ __attribute__((aligned(16))) _Float16 s_pih[kDim * kHPitch];   // Pi, fp16 parts
  __shared__ __attribute__((aligned(16))) _Float16 s_pil[kDim * kHPitch];
  __shared__ __attribute__((aligned(16))) _Float16 s_sh[kDim * kHPitch];    // sigma_i S_i, fp16 parts
  __shared__ __attribute__((aligned(16))) _Float16 s_sl[kDim * kHPitch];
  __shared__ float s_Sn[kDim];                                               // ||sigma_i S_i||
  __shared__ uint32_t s_vt[4][kDim * 8];
  __shared__ float s_lev[2][8];                                              // K and V levels
  __shared__ float s_thr[2][4];                                              // their t0, t2, t4, t6
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

  const int h = blockIdx.y % a.H, b = blockIdx.y / a.H, li = blockIdx.z;
  const int l = a.layer0 + li;
  const int64_t lh = (int64_t)l * a.H + h;
  const bool rotated = (a.flags & kInputRotated) != 0;
  const bool paper = (a.flags & kQjlPaper) != 0;
  const int vsign = VQJL ? (paper ? 2 : 1) : 0;   // (a V sign pass is compiled only where asked for)

  // Pi and S staged as fp16 parts, with the rows of S scaled by powers of
  // two sigma_i and their norms: thread t takes row t / 4, columns
  // 16 (t % 4) .. 16 (t % 4) + 15 of both (all eight 16-byte loads issued
  // together); a row's four threads combine their maxima and sums by shuffles.
  {
    const int r = threadIdx.x >> 2, c0 = 16 * (threadIdx.x & 3);
    const float4* pi4 = reinterpret_cast<const float4*>(a.pi + lh * kDim * kDim) + r * 16 + c0 / 4;
    const float4* s4 = reinterpret_cast<const float4*>(a.qjl_s) + r * 16 + c0 / 4;
    float pv[16], sv[16];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 p4 = pi4[u], q4 = s4[u];
      pv[4 * u] = p4.x; pv[4 * u + 1] = p4.y; pv[4 * u + 2] = p4.z; pv[4 * u + 3] = p4.w;
      sv[4 * u] = q4.x; sv[4 * u + 1] = q4.y; sv[4 * u + 2] = q4.z; sv[4 * u + 3] = q4.w;
    }
    float mx = 0.0f;
#pragma unroll
    for (int k = 0; k < 16; ++k) mx = fmaxf(mx, fabsf(sv[k]));
    mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
    const float sig = unit_scale(mx);        // row r's scale (the same in its four threads)
    float ss = 0.0f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float v = sv[k] * sig;
      ss = fmaf(v, v, ss);
    }
    ss += __shfl_xor(ss, 1, 64);
    ss += __shfl_xor(ss, 2, 64);
    if ((threadIdx.x & 3) == 0) s_Sn[r] = sqrtf(ss);   // bounds the guard band only
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float sa = sv[k] * sig;
      const _Float16 ph = (_Float16)pv[k], sh = (_Float16)sa;
      s_pih[r * kHPitch + c0 + k] = ph;
      s_pil[r * kHPitch + c0 + k] = (_Float16)(pv[k] - (float)ph);
      s_sh[r * kHPitch + c0 + k] = sh;
      s_sl[r * kHPitch + c0 + k] = (_Float16)(sa - (float)sh);
    }
    if (threadIdx.x < 16) s_lev[threadIdx.x >> 3][threadIdx.x & 7] =
        ((threadIdx.x >> 3) ? a.lut_v : a.lut_k)[lh * 8 + (threadIdx.x & 7)];
  }
  const Levels Lk = load_levels(a.lut_k + lh * 8);
  const Levels Lv = load_levels(a.lut_v + lh * 8);
  if (threadIdx.x == 0) {
    s_thr[0][0] = Lk.t0; s_thr[0][1] = Lk.t2; s_thr[0][2] = Lk.t4; s_thr[0][3] = Lk.t6;
    s_thr[1][0] = Lv.t0; s_thr[1][1] = Lv.t2; s_thr[1][2] = Lv.t4; s_thr[1][3] = Lv.t6;
  }
  __syncthreads();

  const int j0 = blockIdx.x * 256 + wave * kTile;
  // the sequence's tokens: all T, or its own count in a ragged call
  const int Tb = a.tokens ? min(max(a.tokens[b], 0), a.T) : a.T;
  if (j0 >= Tb) return;                   // wave-uniform; no barrier follows
  // a (layer, head) whose K or V table is not strictly ascending is not written
  if (!levels_ascending(Lk) || !levels_ascending(Lv)) return;
  const int64_t sbase = a.slot0[b];
  const int pbase = a.pos0[b];
  // The lane's token facts (written or not, its slot, its input row) are
  // recomputed where used, from an index the compiler cannot carry over,
  // so that no 64-bit per-lane value stays live through the products.
  auto lane_of = [&]() {
    int ln;
    asm volatile("v_mov_b32 %0, %1" : "=v"(ln) : "v"((int)threadIdx.x));
    return ln & 63;
  };
  auto ok_of = [&](int jl) {
    const int64_t sl = sbase + jl;
    const int ps = pbase + jl;
    return jl < Tb && sl >= 0 && sl < a.slots && (rotated || (ps >= 0 && ps < a.rope_positions));
  };
  auto row_of = [&](int jl) { return ((((int64_t)li * a.B + b) * a.T + jl) * a.H + h) * kDim; };

  uint8_t* kreg = a.k_codes + lh * a.slots * 32;
  uint8_t* vreg = a.v_codes + lh * a.slots * 32;

  // ---- K: RoPE and rotation, or a pre-rotated input as is
  float x[kDim];
  if (rotated) {
    const int jl = j0 + lane;
    const bool okl = ok_of(jl);
    const int64_t row = row_of(jl);
#pragma unroll
    for (int i = 0; i < kDim; ++i) x[i] = okl ? load_in(a.k, row + i, false) : 0.0f;
  } else {
    rotate_tokens<F16>(x, a, a.k, s_pih, s_pil, li, b, h, j0, Tb, lane, true);
  }
  uint32_t kw[8];
  const QuantOut qk = quantize_lane<true>(x, Lk, s_lev[0], s_thr[0], nullptr, paper ? 2 : 3, kw);
  if (!paper) {
    // the key words wait in this wave's transpose buffer while the signs are
    // computed (registers)
    uint32_t* s_k = s_vt[wave];
#pragma unroll
    for (int w = 0; w < 8; ++w) s_k[lane * 8 + w] = kw[w];
    const uint64_t sb = projected_signs(x, qk.g, s_sh, s_sl, s_Sn, a.qjl_s, lane);
    const int lk = lane_of();
#pragma unroll
    for (int w = 0; w < 8; ++w) kw[w] = s_k[lk * 8 + w] | (uint32_t)((sb >> (8 * w)) & 0xFFu) << 24;
  }
  const int jk = j0 + lane_of();
  const int64_t slot = sbase + jk;
  if (ok_of(jk)) {
    const int64_t tile = slot >> 6;
    const int r = (int)(slot & 63);
    *reinterpret_cast<uint4*>(kreg + tile_half_offset(tile, 0, r)) = make_uint4(kw[0], kw[1], kw[2], kw[3]);
    *reinterpret_cast<uint4*>(kreg + tile_half_offset(tile, 1, r)) = make_uint4(kw[4], kw[5], kw[6], kw[7]);
    // [n_k, g_k] now (the V half of the slot's scalars follows), so that
    // nothing of the key stays live through the value's products
    reinterpret_cast<uint32_t*>(a.scalars + (lh * a.slots + slot) * 4)[0] = qk.n16 | (qk.g16 << 16);
  }

  // ---- V (no RoPE): rotated like K unless TQ_V_ROTATE is off. The V loads
  // are not hoisted above the key's stores (registers, occupancy).
  asm volatile("" ::: "memory");
  if (!rotated && (a.flags & kVRotate)) {
    rotate_tokens<F16>(x, a, a.v, s_pih, s_pil, li, b, h, j0, Tb, lane, false);
  } else {
    const int jl = j0 + lane;
    const bool okl = ok_of(jl);
    const int64_t row = row_of(jl);
#pragma unroll
    for (int i = 0; i < kDim; ++i) x[i] = okl ? load_in(a.v, row + i, F16) : 0.0f;
  }
  uint32_t vw[8];
  const QuantOut qv = quantize_lane<false>(x, Lv, s_lev[1], s_thr[1], nullptr, (VQJL && !paper) ? 3 : vsign, vw);
  // V is stored dimension-major: transpose the wave's 64 x 64 nibbles through
  // its LDS buffer (token-major words in, one dimension per lane out). The
  // words go there first; the projected signs of the value residual, where
  // asked for, are merged in there (registers).
  uint32_t* s_w = s_vt[wave];
#pragma unroll
  for (int w = 0; w < 8; ++w) s_w[lane * 8 + w] = vw[w];
  if (VQJL && !paper) {
    const uint64_t sb = projected_signs(x, qv.g, s_sh, s_sl, s_Sn, a.qjl_s, lane);
    const int lv = lane_of();
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      uint32_t add = 0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) add |= (uint32_t)((sb >> (8 * w + jj)) & 1ull) << (4 * jj + 3);
      s_w[lv * 8 + w] |= add;
    }
  }
  const int jv = j0 + lane_of();
  const bool ok = ok_of(jv);
  if (ok) reinterpret_cast<uint32_t*>(a.scalars + (lh * a.slots + sbase + jv) * 4)[1] = qv.n16 | (qv.g16 << 16);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint64_t okmask = __ballot(ok);
  if (okmask == ~0ull && ((sbase + j0) & 7) == 0) {
    // all 64 tokens, starting at a word boundary: eight whole words per
    // dimension, nibble jj of word k from token 8k + jj
    const int i = lane;
    const int wsel = i >> 3, sh = 4 * (i & 7);
    const int64_t g_first = (sbase + j0) >> 3;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      uint32_t word = 0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) word |= ((s_w[(8 * k + jj) * 8 + wsel] >> sh) & 15u) << (4 * jj);
      const int64_t G = g_first + k;
      const int64_t tile = G >> 3;
      const int c = (int)((G & 7) >> 2);
      *reinterpret_cast<uint32_t*>(vreg + tile_half_offset(tile, c, i) + (G & 3) * 4) = word;
    }
  } else if (okmask != 0) {
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
  const Levels Lo = load_levels((is_v ? a.lut_k : a.lut_v) + lh * 8);
  MatrixSlice pi_sl, s_sl;
  if (any_rotate) load_slice(a.pi + lh * kDim * kDim, pi_sl, threadIdx.x);
  if (any_proj) load_slice(a.qjl_s, s_sl, threadIdx.x);
  const int64_t slot = a.slot0[b] + j;
  const int pos = a.pos0[b] + (int)j;
  const int Tb = a.tokens ? min(max(a.tokens[b], 0), a.T) : a.T;
  // block-uniform exits (before any barrier); a (layer, head) whose K or V
  // table is not strictly ascending is not written
  if ((int)j >= Tb) return;               // beyond the sequence's tokens (a ragged call)
  if (slot < 0 || slot >= a.slots) return;
  if (!levels_ascending(L) || !levels_ascending(Lo)) return;
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
