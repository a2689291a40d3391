// Fused decode attention over the packed 3-bit cache (TurboESM Sec. 3.1
// decode steps 1-4; Algorithm 1 of Sec. 4.3).
//
// One block (WAVES waves) handles one (sequence, layer, head) unit, or one
// split of its 64-token tiles. Per block:
//   loads     the first tile of every wave, this thread's slice of Pi (and of
//             S), the query and the tables are requested before any
//             arithmetic, so the prologue runs under the HBM latency.
//   prologue  q' = RoPE(q), q^ = Pi q', u = S q^ (or q^ for the per-element
//             residual form), and a 64 x 16 LDS table
//             T[i][nibble] = (q^_i c_K[nibble & 7], +-u_i)
//             so one table read per code gives both score terms. Rotating the
//             query once replaces the per-key inverse rotation of Algorithm 1
//             (identical by Eq. 4).
//   main loop each wave takes 64-token tiles and keeps the next few in flight.
//             Keys are scored one lane per token:
//             score = n_k/8 (sum_i T_A + coef sum_i T_B), coef = alpha g_k (QJL)
//             or ebar_K. Online softmax in base 2 with a wave-uniform running
//             max that is raised only when a tile max exceeds it by more than
//             2^8 (rescaling is rare). Values are accumulated one lane per
//             dimension from the dimension-major V tile, with the tile's token
//             weights broadcast through LDS.
//   merge     waves merge through LDS; splits of a unit merge through a
//             workspace of (m, l, o) partials written and read with
//             agent-scope atomics: the last split to finish (atomic counter)
//             combines them by log-sum-exp.
//   epilogue  o = Pi^T (o^ / l) (one inverse rotation; Pi staged in LDS), plus
//             the V residual estimate alpha S^T s or ebar_V s when V carries
//             sign bits.
// Work items are dealt so that all splits of a unit land on one XCD (blocks
// go to the 8 XCDs round-robin), keeping that unit's Pi in one L2.
#include <stdlib.h>

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr float kLazyRescale = 8.0f;   // log2 headroom before the max is raised
constexpr int kXcds = 8;
constexpr int kPiPitch = kDim + 1;     // padded LDS row of Pi (conflict-free columns)

template <int WAVES>
struct DecodeSmem {
  float2 ktab[kDim * 16];
  float pi[kDim * kPiPitch];
  float vtab[16];
  float q[kDim];
  float qh[kDim];
  float u[kDim];
  float part[WAVES][kDim];
  float wp[WAVES][kDim];        // per-tile token weights (V accumulate)
  float wg[WAVES][kDim];        // per-tile token weights for the V residual term
  float wo[WAVES][kDim];
  float wsg[WAVES][kDim];
  float wm[WAVES];
  float wl[WAVES];
  float oh[kDim];
  float sh[kDim];
  int last;
};

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// (byte B of x) & m, one VALU op (sub-dword operand select).
template <int B>
__device__ __forceinline__ uint32_t and_byte(uint32_t m, uint32_t x) {
  uint32_t r;
  if constexpr (B == 0) {
    r = x & m;
  } else if constexpr (B == 1) {
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
        : "=v"(r) : "v"(m), "v"(x));
  } else if constexpr (B == 2) {
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
        : "=v"(r) : "v"(m), "v"(x));
  } else {
    asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
        : "=v"(r) : "v"(m), "v"(x));
  }
  return r;
}

// Byte offsets of the 8 nibbles of x into a table with 8-byte entries indexed
// by the nibble: nibble 2b comes from byte b of x << 3, nibble 2b+1 from byte
// b of x >> 1 (each masked with 0x78 = nibble * 8).
__device__ __forceinline__ void nibble_offsets8(uint32_t x, uint32_t (&off)[8]) {
  const uint32_t m = 0x78u;
  const uint32_t lo = x << 3, hi = x >> 1;
  off[0] = and_byte<0>(m, lo); off[1] = and_byte<0>(m, hi);
  off[2] = and_byte<1>(m, lo); off[3] = and_byte<1>(m, hi);
  off[4] = and_byte<2>(m, lo); off[5] = and_byte<2>(m, hi);
  off[6] = and_byte<3>(m, lo); off[7] = and_byte<3>(m, hi);
}

// Byte offsets (nibble & 7) * 4 of the 8 nibbles of x into a float table:
// nibble 2b from byte b of x << 2, nibble 2b+1 from byte b of x >> 2 (0x1C).
__device__ __forceinline__ void nibble_offsets4(uint32_t x, uint32_t (&off)[8]) {
  const uint32_t m = 0x1Cu;
  const uint32_t lo = x << 2, hi = x >> 2;
  off[0] = and_byte<0>(m, lo); off[1] = and_byte<0>(m, hi);
  off[2] = and_byte<1>(m, lo); off[3] = and_byte<1>(m, hi);
  off[4] = and_byte<2>(m, lo); off[5] = and_byte<2>(m, hi);
  off[6] = and_byte<3>(m, lo); off[7] = and_byte<3>(m, hi);
}

// Wave-wide reductions: 16-lane rows through DPP, then the four rows via
// readlane (the result is wave-uniform).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_max_uniform(float v) {
  v = fmaxf(v, dpp<0xB1>(v));    // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp<0x4E>(v));    // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp<0x141>(v));   // row_half_mirror
  v = fmaxf(v, dpp<0x140>(v));   // row_mirror
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}
__device__ __forceinline__ float wave_sum_uniform(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (a + b) + (c + d);
}

__device__ __forceinline__ void store_out(const DecodeArgs& a, int64_t unit, int k, float v) {
  if (a.f16_out)
    reinterpret_cast<__half*>(a.out)[unit * kDim + k] = __float2half_rn(v);
  else
    reinterpret_cast<float*>(a.out)[unit * kDim + k] = v;
}

struct TileRegs {
  uint4 k0, k1, v0, v1;
  uint2 sc;
};

__device__ __forceinline__ void load_tile(TileRegs& r, const uint8_t* kreg, const uint8_t* vreg,
                                          const uint2* sreg, int64_t gt, int64_t s0, int tt,
                                          int lane) {
  r.k0 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 0, lane));
  r.k1 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 1, lane));
  r.v0 = *reinterpret_cast<const uint4*>(vreg + tile_half_offset(gt, 0, lane));
  r.v1 = *reinterpret_cast<const uint4*>(vreg + tile_half_offset(gt, 1, lane));
  r.sc = sreg[s0 + (int64_t)tt * kTile + lane];
}

// Sum of T[i][nibble_i] over the 8 codes of word w (dims 8w..8w+7).
__device__ __forceinline__ void score_word(const float2* ktab_w, uint32_t x, float& A, float& B) {
  uint32_t off[8];
  nibble_offsets8(x, off);
  const char* base = reinterpret_cast<const char*>(ktab_w);
  float2 e[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) e[j] = *reinterpret_cast<const float2*>(base + j * 128 + off[j]);
  A += ((e[0].x + e[1].x) + (e[2].x + e[3].x)) + ((e[4].x + e[5].x) + (e[6].x + e[7].x));
  B += ((e[0].y + e[1].y) + (e[2].y + e[3].y)) + ((e[4].y + e[5].y) + (e[6].y + e[7].y));
}

template <int WAVES, bool VQJL>
__global__ __launch_bounds__(WAVES * 64)
__attribute__((amdgpu_waves_per_eu((WAVES == 8 && !VQJL) ? 6 : 1)))
void decode_kernel(DecodeArgs a, int total_work, int per_xcd) {
  constexpr int NT = WAVES * 64;
  constexpr int COLS = kDim / WAVES;       // columns of Pi / S per thread
  __shared__ DecodeSmem<WAVES> sm;
  const int bid = blockIdx.x;
  const int work = (bid % kXcds) * per_xcd + bid / kXcds;
  if (work >= total_work) return;
  const int unit = work / a.nsplit;
  const int split = work - unit * a.nsplit;
  const int h = unit % a.H;
  const int b = (unit / a.H) % a.B;
  const int li = unit / (a.H * a.B);
  const int l = a.layer0 + li;
  const int lh = l * a.H + h;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);

  const int n = a.seq_len[b];
  const int64_t s0 = a.seq_slot0[b];
  const int qp = a.q_pos[b];
  const bool valid = n >= 0 && n <= a.max_len && s0 >= 0 && (s0 & 63) == 0 &&
                     s0 + n <= a.slots && qp >= 0 && qp < a.rope_positions;
  if (!valid || n == 0) {
    if (split == 0 && t < kDim) store_out(a, unit, t, valid ? 0.0f : __int_as_float(0x7FC00000));
    return;
  }
  const int ntiles = (n + 63) >> 6;
  const int tile_begin = split * a.split_tiles;
  if (tile_begin >= ntiles) return;
  const int tile_end = min(ntiles, tile_begin + a.split_tiles);
  const int participants = (ntiles + a.split_tiles - 1) / a.split_tiles;
  const bool paper = (a.flags & kQjlPaper) != 0;

  // ------------------------------------------------------------------ loads
  const uint8_t* kreg = a.k_codes + (int64_t)lh * a.slots * 32;
  const uint8_t* vreg = a.v_codes + (int64_t)lh * a.slots * 32;
  const uint2* sreg = reinterpret_cast<const uint2*>(a.scalars + (int64_t)lh * a.slots * 4);
  const int64_t tile0 = s0 >> 6;
  const int ri = t & 63, cq = t >> 6;      // row and column group of Pi / S
  const float4* pi_row = reinterpret_cast<const float4*>(a.pi + (int64_t)lh * kDim * kDim + ri * kDim + cq * COLS);
  float4 pr[COLS / 4];
#pragma unroll
  for (int k = 0; k < COLS / 4; ++k) pr[k] = pi_row[k];
  float4 sr[COLS / 4];
  if (!paper) {
    const float4* s_row = reinterpret_cast<const float4*>(a.qjl_s + ri * kDim + cq * COLS);
#pragma unroll
    for (int k = 0; k < COLS / 4; ++k) sr[k] = s_row[k];
  }
  float qv = 0.0f;
  float2 cs = make_float2(1.0f, 0.0f);
  const bool half = (a.flags & kRopeHalf) != 0;
  if (t < kDim) {
    qv = load_in(a.q, (int64_t)unit * kDim + t, a.f16_in != 0);
    const int m = half ? (t & 31) : (t >> 1);
    cs = reinterpret_cast<const float2*>(a.rope_cs + (int64_t)qp * 2 * kPairs)[m];
  }
  const float ck = a.lut_k[lh * 8 + (t & 7)];
  const float cvv = a.lut_v[lh * 8 + (t & 7)];
  const float ebar_k = paper ? a.ebar[lh * 2 + 0] : 0.0f;

  // Tiles are requested after Pi, S and the query (the prologue needs those
  // first). Each wave keeps DEPTH tiles in flight: its first DEPTH tiles are
  // requested now, and every processed tile is replaced by the one DEPTH
  // steps ahead.
  constexpr int DEPTH = (WAVES == 8) ? 1 : 2;
  TileRegs buf[DEPTH];
#pragma unroll
  for (int d = 0; d < DEPTH; ++d) {
    const int tq = tile_begin + wave + d * WAVES;
    if (tq < tile_end) load_tile(buf[d], kreg, vreg, sreg, tile0 + tq, s0, tq, lane);
  }

  // --------------------------------------------------------------- prologue
  if (t < kDim) {
    const int partner = half ? (t ^ 32) : (t ^ 1);
    const bool first = half ? (t < 32) : ((t & 1) == 0);
    const float qpv = __shfl(qv, partner, 64);
    sm.q[t] = first ? (qv * cs.x - qpv * cs.y) : (qpv * cs.y + qv * cs.x);
  }
#pragma unroll
  for (int k = 0; k < COLS / 4; ++k) {
    float* dst = sm.pi + ri * kPiPitch + cq * COLS + 4 * k;
    dst[0] = pr[k].x; dst[1] = pr[k].y; dst[2] = pr[k].z; dst[3] = pr[k].w;
  }
  if (t < 16) sm.vtab[t] = cvv;
  __syncthreads();
  {
    const float* x = sm.q + cq * COLS;
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < COLS / 4; ++k) {
      acc = fmaf(pr[k].x, x[4 * k + 0], acc);
      acc = fmaf(pr[k].y, x[4 * k + 1], acc);
      acc = fmaf(pr[k].z, x[4 * k + 2], acc);
      acc = fmaf(pr[k].w, x[4 * k + 3], acc);
    }
    sm.part[cq][ri] = acc;
  }
  __syncthreads();
  if (t < kDim) {
    float y = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) y += sm.part[w][t];
    sm.qh[t] = y;
  }
  __syncthreads();
  if (!paper) {
    const float* x = sm.qh + cq * COLS;
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < COLS / 4; ++k) {
      acc = fmaf(sr[k].x, x[4 * k + 0], acc);
      acc = fmaf(sr[k].y, x[4 * k + 1], acc);
      acc = fmaf(sr[k].z, x[4 * k + 2], acc);
      acc = fmaf(sr[k].w, x[4 * k + 3], acc);
    }
    sm.part[cq][ri] = acc;
    __syncthreads();
    if (t < kDim) {
      float y = 0.0f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) y += sm.part[w][t];
      sm.u[t] = y;
    }
  } else {
    if (t < kDim) sm.u[t] = sm.qh[t];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 1024 / NT; ++r) {
    const int e = t + NT * r;
    const int d = e >> 4, nib = e & 15;
    const float cknib = __shfl(ck, nib & 7, 64);    // lane j of any wave holds c_K[j & 7]
    sm.ktab[e] = make_float2(sm.qh[d] * cknib, (nib & 8) ? sm.u[d] : -sm.u[d]);
  }
  __syncthreads();

  // -------------------------------------------------------------- main loop
  float m_run = -INFINITY;
  float l_lane = 0.0f;
  float sg = 0.0f;
  float o0 = 0.0f, o1 = 0.0f, o2 = 0.0f, o3 = 0.0f;
  const float lscale = a.logit_scale2;
  const float2* ktab = sm.ktab;
  const char* vtab = reinterpret_cast<const char*>(sm.vtab);

  for (int tb = tile_begin + wave; tb < tile_end; tb += DEPTH * WAVES) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int tt = tb + d * WAVES;
      if (tt >= tile_end) break;
      const TileRegs& cur = buf[d];
      const int tok = tt * kTile + lane;
      const bool tv = tok < n;

      // ---- key score, one lane per token. Two words (16 table reads) in
      // flight at a time: the empty asm pins the partial sums so the compiler
      // does not hoist every table read of the tile (registers, occupancy).
      float A = 0.0f, B = 0.0f;
      score_word(ktab + 0 * 128, cur.k0.x, A, B);
      score_word(ktab + 1 * 128, cur.k0.y, A, B);
      asm volatile("" : "+v"(A), "+v"(B));
      score_word(ktab + 2 * 128, cur.k0.z, A, B);
      score_word(ktab + 3 * 128, cur.k0.w, A, B);
      asm volatile("" : "+v"(A), "+v"(B));
      score_word(ktab + 4 * 128, cur.k1.x, A, B);
      score_word(ktab + 5 * 128, cur.k1.y, A, B);
      asm volatile("" : "+v"(A), "+v"(B));
      score_word(ktab + 6 * 128, cur.k1.z, A, B);
      score_word(ktab + 7 * 128, cur.k1.w, A, B);
      const float nk = half_bits_to_float(cur.sc.x), gk = half_bits_to_float(cur.sc.x >> 16);
      const float nv = half_bits_to_float(cur.sc.y), gv = half_bits_to_float(cur.sc.y >> 16);
      const float coef = paper ? ebar_k : kQjlAlpha * gk;
      float lg = nk * lscale * fmaf(coef, B, A);
      lg = tv ? lg : -INFINITY;

      // ---- online softmax (base 2), lazily rescaled
      const float tmax = wave_max_uniform(lg);
      if (tmax > m_run + kLazyRescale) {
        const float f = __builtin_amdgcn_exp2f(m_run - tmax);
        l_lane *= f;
        sg *= f;
        o0 *= f; o1 *= f; o2 *= f; o3 *= f;
        m_run = tmax;
      }
      const float p = __builtin_amdgcn_exp2f(lg - m_run);
      l_lane += p;
      const float wv = tv ? p * nv * 0.125f : 0.0f;
      sm.wp[wave][lane] = wv;
      if (VQJL) sm.wg[wave][lane] = paper ? wv : wv * gv;
      wave_lds_sync();

      // ---- value accumulate, one lane per dimension
      const uint32_t vw[8] = {cur.v0.x, cur.v0.y, cur.v0.z, cur.v0.w, cur.v1.x, cur.v1.y, cur.v1.z, cur.v1.w};
      const float4* wp4 = reinterpret_cast<const float4*>(sm.wp[wave]);
  #pragma unroll
      for (int w8 = 0; w8 < 8; ++w8) {
        const uint32_t x = vw[w8];
        const float4 wa = wp4[2 * w8], wb = wp4[2 * w8 + 1];
        uint32_t off[8];
        nibble_offsets4(x, off);     // (nibble & 7) * 4: float entries
        o0 = fmaf(wa.x, *reinterpret_cast<const float*>(vtab + off[0]), o0);
        o1 = fmaf(wa.y, *reinterpret_cast<const float*>(vtab + off[1]), o1);
        o2 = fmaf(wa.z, *reinterpret_cast<const float*>(vtab + off[2]), o2);
        o3 = fmaf(wa.w, *reinterpret_cast<const float*>(vtab + off[3]), o3);
        o0 = fmaf(wb.x, *reinterpret_cast<const float*>(vtab + off[4]), o0);
        o1 = fmaf(wb.y, *reinterpret_cast<const float*>(vtab + off[5]), o1);
        o2 = fmaf(wb.z, *reinterpret_cast<const float*>(vtab + off[6]), o2);
        o3 = fmaf(wb.w, *reinterpret_cast<const float*>(vtab + off[7]), o3);
        if (w8 & 1) asm volatile("" : "+v"(o0), "+v"(o1), "+v"(o2), "+v"(o3));
      }
      if (VQJL) {
        const float4* wg4 = reinterpret_cast<const float4*>(sm.wg[wave]);
  #pragma unroll
        for (int w8 = 0; w8 < 8; ++w8) {
          const uint32_t x = vw[w8];
          const float4 ga = wg4[2 * w8], gb = wg4[2 * w8 + 1];
          const float gt8[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
  #pragma unroll
          for (int jj = 0; jj < 8; ++jj) sg += ((x >> (4 * jj + 3)) & 1u) ? gt8[jj] : -gt8[jj];
        }
      }
      wave_lds_sync();   // wp/wg are rewritten by the next tile
      const int tn = tt + DEPTH * WAVES;
      if (tn < tile_end) load_tile(buf[d], kreg, vreg, sreg, tile0 + tn, s0, tn, lane);
    }
  }

  // ------------------------------------------------------ merge the waves
  const float ov = (o0 + o1) + (o2 + o3);
  const float l_wave = wave_sum_uniform(l_lane);
  if (lane == 0) { sm.wm[wave] = m_run; sm.wl[wave] = l_wave; }
  sm.wo[wave][lane] = ov;
  if (VQJL) sm.wsg[wave][lane] = sg;
  __syncthreads();
  float M = -INFINITY, L = 0.0f, O = 0.0f, SG = 0.0f;
  if (t < kDim) {
#pragma unroll
    for (int w = 0; w < WAVES; ++w) M = fmaxf(M, sm.wm[w]);
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float f = __builtin_amdgcn_exp2f(sm.wm[w] - M);
      L += sm.wl[w] * f;
      O += sm.wo[w][t] * f;
      if (VQJL) SG += sm.wsg[w][t] * f;
    }
  }

  if (participants > 1) {
    // Publish this split's partial with agent-scope (coherent) stores and wait
    // until they are performed before counting the split in; the last split
    // reads the partials back with agent-scope loads. No block writes back or
    // invalidates the L2 (which a device-wide fence would do on every block).
    float* part = a.partials + ((int64_t)unit * a.nsplit + split) * kPartialFloats;
    if (t < kDim) {
      __hip_atomic_store(part + 4 + t, O, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (VQJL) __hip_atomic_store(part + 4 + kDim + t, SG, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (t == 0) {
        __hip_atomic_store(part + 0, M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(part + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (t == 0) {
      const uint32_t prev = __hip_atomic_fetch_add(a.counters + unit, 1u, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT);
      sm.last = (prev == (uint32_t)(participants - 1)) ? 1 : 0;
    }
    __syncthreads();
    if (!sm.last) return;
    if (t < kDim) {
      float* base = a.partials + (int64_t)unit * a.nsplit * kPartialFloats;
      M = -INFINITY;
      for (int s = 0; s < participants; ++s)
        M = fmaxf(M, __hip_atomic_load(base + s * kPartialFloats, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      L = 0.0f; O = 0.0f; SG = 0.0f;
      for (int s = 0; s < participants; ++s) {
        float* ps = base + s * kPartialFloats;
        const float f = __builtin_amdgcn_exp2f(__hip_atomic_load(ps, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - M);
        L += __hip_atomic_load(ps + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) * f;
        O += __hip_atomic_load(ps + 4 + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) * f;
        if (VQJL) SG += __hip_atomic_load(ps + 4 + kDim + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) * f;
      }
    }
    // leave the workspace zeroed for the next call
    if (t == 0) __hip_atomic_store(a.counters + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // --------------------------------------------------------------- epilogue
  const float invL = 1.0f / L;
  if (t < kDim) { sm.oh[t] = O * invL; sm.sh[t] = SG * invL; }
  __syncthreads();
  if (VQJL) {
    if (paper) {
      const float ebar_v = a.ebar[lh * 2 + 1];
      if (t < kDim) sm.oh[t] += ebar_v * sm.sh[t];
    } else {
      // o^ += alpha S^T s; thread (k, group) sums COLS rows of column k of S
      const int k = t & 63;
      float acc = 0.0f;
#pragma unroll
      for (int ii = 0; ii < COLS; ++ii) {
        const int i = cq * COLS + ii;
        acc = fmaf(a.qjl_s[i * kDim + k], sm.sh[i], acc);
      }
      sm.part[cq][k] = acc;
      __syncthreads();
      if (t < kDim) {
        float y = 0.0f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) y += sm.part[w][t];
        sm.oh[t] += kQjlAlpha * y;
      }
    }
    __syncthreads();
  }
  if (a.flags & kVRotate) {
    // out_k = sum_i Pi[i][k] o^_i: thread (k, group) sums COLS rows
    const int k = t & 63;
    float acc = 0.0f;
#pragma unroll
    for (int ii = 0; ii < COLS; ++ii) {
      const int i = cq * COLS + ii;
      acc = fmaf(sm.pi[i * kPiPitch + k], sm.oh[i], acc);
    }
    sm.part[cq][k] = acc;
    __syncthreads();
    if (t < kDim) {
      float y = 0.0f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) y += sm.part[w][t];
      store_out(a, unit, t, y);
    }
  } else {
    if (t < kDim) store_out(a, unit, t, sm.oh[t]);
  }
}

void decode_plan(int units, int max_len, int* waves, int* nsplit, int* split_tiles) {
  const int ntiles = max_len > 0 ? (max_len + 63) / 64 : 1;
  int w = ntiles >= 12 ? 8 : 4;
  const char* ew = getenv("TQ_DECODE_WAVES");
  if (ew && (atoi(ew) == 4 || atoi(ew) == 8)) w = atoi(ew);
  int st;
  const char* env = getenv("TQ_DECODE_SPLIT_TILES");
  if (env && atoi(env) > 0) {
    st = atoi(env);
  } else {
    // One block per unit when there are enough units to occupy every CU
    // (a cross-block merge costs more than it balances); otherwise split the
    // tiles so that each wave still gets at least one tile.
    const int target_blocks = 256;
    int ns = (target_blocks + units - 1) / units;
    const int max_ns = (ntiles + w - 1) / w;
    if (ns > max_ns) ns = max_ns;
    if (ns < 1) ns = 1;
    st = (ntiles + ns - 1) / ns;
  }
  if (st > ntiles) st = ntiles;
  *waves = w;
  *split_tiles = st;
  *nsplit = (ntiles + st - 1) / st;
}

hipError_t launch_decode(const DecodeArgs& a, int waves, hipStream_t st) {
  const int64_t units = (int64_t)a.nlayers * a.B * a.H;
  const int64_t total = units * a.nsplit;
  const int64_t per_xcd = (total + kXcds - 1) / kXcds;
  const int64_t blocks = per_xcd * kXcds;
  const bool vq = (a.flags & kVQjl) != 0;
  if (waves == 8) {
    if (vq)
      hipLaunchKernelGGL((decode_kernel<8, true>), dim3((unsigned)blocks), dim3(512), 0, st, a, (int)total, (int)per_xcd);
    else
      hipLaunchKernelGGL((decode_kernel<8, false>), dim3((unsigned)blocks), dim3(512), 0, st, a, (int)total, (int)per_xcd);
  } else {
    if (vq)
      hipLaunchKernelGGL((decode_kernel<4, true>), dim3((unsigned)blocks), dim3(256), 0, st, a, (int)total, (int)per_xcd);
    else
      hipLaunchKernelGGL((decode_kernel<4, false>), dim3((unsigned)blocks), dim3(256), 0, st, a, (int)total, (int)per_xcd);
  }
  return hipGetLastError();
}

}  // namespace tq
