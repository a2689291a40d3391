// Fused decode attention over the packed 3-bit cache (TurboESM Sec. 3.1
// decode steps 1-4; Algorithm 1 of Sec. 4.3).
//
// One block (4 waves) handles one (sequence, layer, head) unit, or one split
// of its 64-token tiles. Per block:
//   prologue  q' = RoPE(q), q^ = Pi q', u = S q^ (or q^ for the per-element
//             residual form), and a 64 x 16 LDS table
//             T[i][nibble] = (q^_i c_K[nibble & 7], +-u_i)
//             so one table read per code gives both score terms. Rotating the
//             query once replaces the per-key inverse rotation of Algorithm 1
//             (identical by Eq. 4).
//   main loop each wave takes 64-token tiles. Keys are scored one lane per
//             token: score = n_k/8 (sum_i T_A + coef sum_i T_B), coef = alpha g_k
//             (QJL) or ebar_K. Online softmax in base 2 with a wave-uniform
//             running max that is raised only when a tile max exceeds it by
//             more than 2^8 (rescaling is rare). Values are accumulated one
//             lane per dimension from the dimension-major V tile, with the
//             tile's token weights broadcast through LDS.
//   merge     waves merge through LDS; splits of a unit merge through a
//             workspace of (m, l, o) partials: the last block of the unit to
//             finish (atomic counter) combines them by log-sum-exp.
//   epilogue  o = Pi^T (o^ / l) (one inverse rotation), plus the V residual
//             estimate alpha S^T s or ebar_V s when V carries sign bits.
// Work items are mapped so that all splits of a unit land on one XCD
// (blocks are dealt to the 8 XCDs round-robin), keeping Pi in that XCD's L2.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr int kWaves = 4;
constexpr float kLazyRescale = 8.0f;   // log2 headroom before the max is raised
constexpr int kXcds = 8;

struct DecodeSmem {
  float2 ktab[kDim * 16];
  float vtab[16];
  float q[kDim];
  float qh[kDim];
  float u[kDim];
  float part[kWaves][kDim];
  float wp[kWaves][kDim];    // per-tile token weights (V accumulate)
  float wg[kWaves][kDim];    // per-tile token weights for the V residual term
  float wo[kWaves][kDim];
  float wsg[kWaves][kDim];
  float wm[kWaves];
  float wl[kWaves];
  float oh[kDim];
  float sh[kDim];
  int last;
};

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// y = M x for a 64 x 64 row-major global matrix, x in LDS; all 256 threads.
// Thread t sums columns 16*(t/64) .. +15 of row t%64; partials go to `part`.
__device__ __forceinline__ float matvec_rows(const float* M, const float* x, DecodeSmem& sm) {
  const int t = threadIdx.x, i = t & 63, q4 = t >> 6;
  const float4* row = reinterpret_cast<const float4*>(M + i * kDim + q4 * 16);
  float acc = 0.0f;
#pragma unroll
  for (int k4 = 0; k4 < 4; ++k4) {
    const float4 m = row[k4];
    acc = fmaf(m.x, x[q4 * 16 + 4 * k4 + 0], acc);
    acc = fmaf(m.y, x[q4 * 16 + 4 * k4 + 1], acc);
    acc = fmaf(m.z, x[q4 * 16 + 4 * k4 + 2], acc);
    acc = fmaf(m.w, x[q4 * 16 + 4 * k4 + 3], acc);
  }
  sm.part[q4][i] = acc;
  __syncthreads();
  float y = 0.0f;
  if (t < kDim) y = (sm.part[0][t] + sm.part[1][t]) + (sm.part[2][t] + sm.part[3][t]);
  __syncthreads();
  return y;   // valid in threads 0..63
}

// y = M^T x (y_k = sum_i M[i][k] x_i); coalesced row reads; all 256 threads.
__device__ __forceinline__ float matvec_cols(const float* M, const float* x, DecodeSmem& sm) {
  const int t = threadIdx.x, k = t & 63, q4 = t >> 6;
  float acc = 0.0f;
#pragma unroll
  for (int ii = 0; ii < 16; ++ii) {
    const int i = q4 * 16 + ii;
    acc = fmaf(M[i * kDim + k], x[i], acc);
  }
  sm.part[q4][k] = acc;
  __syncthreads();
  float y = 0.0f;
  if (t < kDim) y = (sm.part[0][t] + sm.part[1][t]) + (sm.part[2][t] + sm.part[3][t]);
  __syncthreads();
  return y;
}

__device__ __forceinline__ void store_out(const DecodeArgs& a, int64_t unit, int k, float v) {
  if (a.f16_out)
    reinterpret_cast<__half*>(a.out)[unit * kDim + k] = __float2half_rn(v);
  else
    reinterpret_cast<float*>(a.out)[unit * kDim + k] = v;
}

template <bool VQJL>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a, int64_t total_work,
                                                     int64_t per_xcd) {
  __shared__ DecodeSmem sm;
  const int64_t bid = blockIdx.x;
  const int64_t work = (bid % kXcds) * per_xcd + bid / kXcds;
  if (work >= total_work) return;
  const int64_t unit = work / a.nsplit;
  const int split = (int)(work % a.nsplit);
  const int h = (int)(unit % a.H);
  const int b = (int)((unit / a.H) % a.B);
  const int li = (int)(unit / ((int64_t)a.H * a.B));
  const int l = a.layer0 + li;
  const int64_t lh = (int64_t)l * a.H + h;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;

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

  const float* pi_lh = a.pi + lh * kDim * kDim;
  const bool paper = (a.flags & kQjlPaper) != 0;

  // ---------------------------------------------------------------- prologue
  if (t < kDim) {
    const float qv = load_in(a.q, unit * kDim + t, a.f16_in != 0);
    const bool half = (a.flags & kRopeHalf) != 0;
    const int partner = half ? (t ^ 32) : (t ^ 1);
    const bool first = half ? (t < 32) : ((t & 1) == 0);
    const int m = half ? (t & 31) : (t >> 1);
    const float qpv = __shfl(qv, partner, 64);
    const float2 cs = reinterpret_cast<const float2*>(a.rope_cs + (int64_t)qp * 2 * kPairs)[m];
    sm.q[t] = first ? (qv * cs.x - qpv * cs.y) : (qpv * cs.y + qv * cs.x);
  }
  __syncthreads();
  float y = matvec_rows(pi_lh, sm.q, sm);
  if (t < kDim) sm.qh[t] = y;
  __syncthreads();
  if (paper) {
    if (t < kDim) sm.u[t] = sm.qh[t];
  } else {
    y = matvec_rows(a.qjl_s, sm.qh, sm);
    if (t < kDim) sm.u[t] = y;
  }
  __syncthreads();
  const float* lutk = a.lut_k + lh * 8;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int e = t + 256 * r;
    const int d = e >> 4, nib = e & 15;
    sm.ktab[e] = make_float2(sm.qh[d] * lutk[nib & 7], (nib & 8) ? sm.u[d] : -sm.u[d]);
  }
  if (t < 16) sm.vtab[t] = a.lut_v[lh * 8 + (t & 7)];
  const float ebar_k = paper ? a.ebar[lh * 2 + 0] : 0.0f;
  __syncthreads();

  // --------------------------------------------------------------- main loop
  const uint8_t* kreg = a.k_codes + lh * a.slots * 32;
  const uint8_t* vreg = a.v_codes + lh * a.slots * 32;
  const uint2* sreg = reinterpret_cast<const uint2*>(a.scalars + lh * a.slots * 4);
  const int64_t tile0 = s0 >> 6;

  float m_run = -INFINITY;
  float l_lane = 0.0f;
  float o0 = 0.0f, o1 = 0.0f, o2 = 0.0f, o3 = 0.0f;
  float sg = 0.0f;

  for (int tt = tile_begin + wave; tt < tile_end; tt += kWaves) {
    const int64_t gt = tile0 + tt;
    const uint4 kq0 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 0, lane));
    const uint4 kq1 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 1, lane));
    const uint4 vq0 = *reinterpret_cast<const uint4*>(vreg + tile_half_offset(gt, 0, lane));
    const uint4 vq1 = *reinterpret_cast<const uint4*>(vreg + tile_half_offset(gt, 1, lane));
    const int tok = tt * kTile + lane;
    const bool tv = tok < n;
    const uint2 sc = sreg[s0 + tok];

    // ---- key score, one lane per token
    const uint32_t kw[8] = {kq0.x, kq0.y, kq0.z, kq0.w, kq1.x, kq1.y, kq1.z, kq1.w};
    float A0 = 0.0f, A1 = 0.0f, B0 = 0.0f, B1 = 0.0f;
#pragma unroll
    for (int w8 = 0; w8 < 8; ++w8) {
      const uint32_t x = kw[w8];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const float2 e = sm.ktab[(w8 * 8 + jj) * 16 + ((x >> (4 * jj)) & 15u)];
        if (jj & 1) { A1 += e.x; B1 += e.y; } else { A0 += e.x; B0 += e.y; }
      }
    }
    const float nk = half_bits_to_float(sc.x), gk = half_bits_to_float(sc.x >> 16);
    const float nv = half_bits_to_float(sc.y), gv = half_bits_to_float(sc.y >> 16);
    const float coef = paper ? ebar_k : kQjlAlpha * gk;
    float lg = nk * a.logit_scale2 * ((A0 + A1) + coef * (B0 + B1));
    lg = tv ? lg : -INFINITY;

    // ---- online softmax (base 2), lazily rescaled
    const float tmax = wave_max(lg);
    if (tmax > m_run + kLazyRescale) {
      const float f = exp2f(m_run - tmax);
      l_lane *= f;
      o0 *= f; o1 *= f; o2 *= f; o3 *= f;
      sg *= f;
      m_run = tmax;
    }
    const float p = exp2f(lg - m_run);
    l_lane += p;
    const float wv = tv ? p * nv * 0.125f : 0.0f;
    sm.wp[wave][lane] = wv;
    if (VQJL) sm.wg[wave][lane] = paper ? wv : wv * gv;
    wave_lds_sync();

    // ---- value accumulate, one lane per dimension
    const uint32_t vw[8] = {vq0.x, vq0.y, vq0.z, vq0.w, vq1.x, vq1.y, vq1.z, vq1.w};
    const float4* wp4 = reinterpret_cast<const float4*>(sm.wp[wave]);
    const float4* wg4 = reinterpret_cast<const float4*>(sm.wg[wave]);
#pragma unroll
    for (int w8 = 0; w8 < 8; ++w8) {
      const uint32_t x = vw[w8];
      const float4 wa = wp4[2 * w8], wb = wp4[2 * w8 + 1];
      const float wt[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
      o0 = fmaf(wt[0], sm.vtab[(x >> 0) & 7u], o0);
      o1 = fmaf(wt[1], sm.vtab[(x >> 4) & 7u], o1);
      o2 = fmaf(wt[2], sm.vtab[(x >> 8) & 7u], o2);
      o3 = fmaf(wt[3], sm.vtab[(x >> 12) & 7u], o3);
      o0 = fmaf(wt[4], sm.vtab[(x >> 16) & 7u], o0);
      o1 = fmaf(wt[5], sm.vtab[(x >> 20) & 7u], o1);
      o2 = fmaf(wt[6], sm.vtab[(x >> 24) & 7u], o2);
      o3 = fmaf(wt[7], sm.vtab[(x >> 28) & 7u], o3);
      if (VQJL) {
        const float4 ga = wg4[2 * w8], gb = wg4[2 * w8 + 1];
        const float gt8[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) sg += ((x >> (4 * jj + 3)) & 1u) ? gt8[jj] : -gt8[jj];
      }
    }
    wave_lds_sync();   // wp/wg are rewritten by the next tile
  }

  // ------------------------------------------------------- merge the 4 waves
  const float l_wave = wave_sum(l_lane);
  if (lane == 0) { sm.wm[wave] = m_run; sm.wl[wave] = l_wave; }
  sm.wo[wave][lane] = (o0 + o1) + (o2 + o3);
  if (VQJL) sm.wsg[wave][lane] = sg;
  __syncthreads();
  float M = -INFINITY, L = 0.0f, O = 0.0f, SG = 0.0f;
  if (t < kDim) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.wm[w]);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = exp2f(sm.wm[w] - M);
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
    float* part = a.partials + (unit * a.nsplit + split) * kPartialFloats;
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
      float* base = a.partials + unit * a.nsplit * kPartialFloats;
      M = -INFINITY;
      for (int s = 0; s < participants; ++s)
        M = fmaxf(M, __hip_atomic_load(base + s * kPartialFloats, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      L = 0.0f; O = 0.0f; SG = 0.0f;
      for (int s = 0; s < participants; ++s) {
        float* ps = base + s * kPartialFloats;
        const float f = exp2f(__hip_atomic_load(ps, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - M);
        L += __hip_atomic_load(ps + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) * f;
        O += __hip_atomic_load(ps + 4 + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) * f;
        if (VQJL) SG += __hip_atomic_load(ps + 4 + kDim + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) * f;
      }
    }
    // leave the workspace zeroed for the next call
    if (t == 0) __hip_atomic_store(a.counters + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // ---------------------------------------------------------------- epilogue
  const float invL = 1.0f / L;
  if (t < kDim) { sm.oh[t] = O * invL; sm.sh[t] = SG * invL; }
  __syncthreads();
  if (VQJL) {
    if (paper) {
      const float ebar_v = a.ebar[lh * 2 + 1];
      if (t < kDim) sm.oh[t] += ebar_v * sm.sh[t];
    } else {
      y = matvec_cols(a.qjl_s, sm.sh, sm);
      if (t < kDim) sm.oh[t] += kQjlAlpha * y;
    }
    __syncthreads();
  }
  if (a.flags & kVRotate) {
    y = matvec_cols(pi_lh, sm.oh, sm);
    if (t < kDim) store_out(a, unit, t, y);
  } else {
    if (t < kDim) store_out(a, unit, t, sm.oh[t]);
  }
}

void decode_plan(int units, int max_len, int* nsplit, int* split_tiles) {
  const int ntiles = max_len > 0 ? (max_len + 63) / 64 : 1;
  const int target_blocks = 2048;
  int ns = (target_blocks + units - 1) / units;
  const int max_ns = (ntiles + kWaves - 1) / kWaves;   // at least one tile per wave
  if (ns > max_ns) ns = max_ns;
  if (ns < 1) ns = 1;
  int st = (ntiles + ns - 1) / ns;
  ns = (ntiles + st - 1) / st;
  *nsplit = ns;
  *split_tiles = st;
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
  const int64_t units = (int64_t)a.nlayers * a.B * a.H;
  const int64_t total = units * a.nsplit;
  const int64_t per_xcd = (total + kXcds - 1) / kXcds;
  const int64_t blocks = per_xcd * kXcds;
  if (a.flags & kVQjl)
    hipLaunchKernelGGL(decode_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, a, total, per_xcd);
  else
    hipLaunchKernelGGL(decode_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, a, total, per_xcd);
  return hipGetLastError();
}

}  // namespace tq
