// Dequantize the packed cache into fp16 key and value rows: the first step of
// a "dequantize first, then attend" path, the comparison the paper makes for
// its fused kernel (Sec. 5.3, Table 6). The rows are what the fused decode
// reconstructs in registers (Sec. 3.1 decode, Sec. 3.4):
//   k~_j = (n_k/8) (c_K[idx_j] + alpha g_k S^T (2 s_j - 1))
//          (per-element form: ebar_K (2 s_j - 1) in place of alpha g_k S^T (2 s_j - 1))
//   v~_j = (n_v/8) (c_V[idx_j] (+ the same residual estimate with the V signs))
// so that q^ . k~_j is the decode score and v~_j the decoded value.
//
// The residual estimate S^T (2 s_j - 1) of a 64-token tile is a dense
// 64 x 64 x 64 product (+-1 signs times S): it runs on the matrix cores as
// fp16 MFMA (v_mfma_f32_32x32x16_f16, fp32 sums) with S split into
// S_hi = fp16(S) and S_lo = fp16(S - S_hi), so that the +-1 products of both
// halves are exact and the result carries S to about 22 bits; each wave
// computes one 32-token x 32-dimension block, holding its column block of
// S_hi and S_lo in registers for all the tiles the block covers. Everything
// else is a table look-up and a scale. The tile's codes and scalars are staged
// in LDS (the next tile's are loaded while the current one is computed), and
// so are the estimates; a thread then writes 16 dimensions of a key row with
// two 16-byte stores, and the value rows (dimension-major codes) are
// transposed through LDS before their 16-byte stores.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

namespace {

constexpr int kTilesPerBlock = 4;
typedef float f32x16 __attribute__((ext_vector_type(16)));


}  // namespace

// Block: 4 waves; wave w computes tokens 32 (w & 1) .. +31 (mb) and dimensions
// 32 (w >> 1) .. +31 (nb) of each tile. Grid: x = ceil(tiles / 4), y = B*H,
// z = nlayers. Instruction layout (lane l, n = l % 32, h = l / 32): A lane
// values A[n][8h + j], B lane values B[8h + j][n] (j = 0..7), result register
// r D[8 (r/4) + 4h + r%4][n]. Step q contracts sign index i = 16q + 8h + j,
// i.e. the sign byte of key word 2q + h of the lane's token.
typedef _Float16 half8 __attribute__((ext_vector_type(8)));

struct TileCodes {
  uint4 c;      // threads 0..127: K chunk t, 128..255: V chunk t - 128
  uint2 sc;     // threads 0..63: scalars of slot t
};

__device__ __forceinline__ void load_codes(TileCodes& tc, const uint4* kt, const uint4* vt, const uint2* st,
                                           int64_t gt, int t) {
  tc.c = (t < 128) ? kt[gt * 128 + t] : vt[gt * 128 + (t - 128)];
  if (t < 64) tc.sc = st[gt * 64 + t];
}

// +-1 of the 8 sign bits of a byte, as fp16.
__device__ __forceinline__ half8 signs8(uint32_t byte) {
  half8 v;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = ((byte >> j) & 1u) ? (_Float16)1.0f : (_Float16)-1.0f;
  return v;
}

template <bool VQJL>
__global__ __launch_bounds__(256) void dequant_kernel(DequantArgs a) {
  __shared__ __attribute__((aligned(16))) uint4 s_k[128];      // K tile: chunk (c, r) at c*64 + r
  __shared__ __attribute__((aligned(16))) uint4 s_v[128];      // V tile: chunk (c, i) at c*64 + i
  __shared__ __attribute__((aligned(16))) uint2 s_sc[64];      // [n_k | g_k, n_v | g_v] per slot
  __shared__ __attribute__((aligned(16))) float s_ek[64 * 64];                 // key estimates e[t][c]
  __shared__ __attribute__((aligned(16))) float s_ev[VQJL ? 64 * 64 : 1];   // value estimates
  __shared__ __attribute__((aligned(16))) __half s_ov[64 * 64];  // v~ rows of the tile
  __shared__ float s_lk[8], s_lv[8];                             // the tables

  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int n = lane & 31, hh = lane >> 5;
  const int mb = wave & 1, nb = wave >> 1;
  const int h = blockIdx.y % a.H, b = blockIdx.y / a.H, li = blockIdx.z;
  const int l = a.layer0 + li;
  const int64_t lh = (int64_t)l * a.H + h;
  const int len = a.seq_len[b];
  const int64_t s0 = a.seq_slot0[b];
  if (len <= 0 || len > a.max_len || s0 < 0 || (s0 & 63) != 0 || s0 + len > a.slots) return;
  // a (layer, head) whose K or V table is not strictly ascending is skipped
  if (!levels_ascending(load_levels(a.lut_k + lh * 8)) || !levels_ascending(load_levels(a.lut_v + lh * 8)))
    return;
  const int ntiles = (len + 63) >> 6;
  const int tile_first = blockIdx.x * kTilesPerBlock;
  if (tile_first >= ntiles) return;   // block-uniform, before any barrier
  const int tile_last = min(ntiles, tile_first + kTilesPerBlock);

  const uint4* kt = reinterpret_cast<const uint4*>(a.k_codes + lh * a.slots * 32);
  const uint4* vt = reinterpret_cast<const uint4*>(a.v_codes + lh * a.slots * 32);
  const uint2* st = reinterpret_cast<const uint2*>(a.scalars + lh * a.slots * 4);
  TileCodes next;
  load_codes(next, kt, vt, st, (s0 >> 6) + tile_first, t);

  const bool paper = (a.flags & kQjlPaper) != 0;
  constexpr bool vqjl = VQJL;   // (the V sign pass is compiled only where asked for)
  if (t < 8) {
    s_lk[t] = a.lut_k[lh * 8 + t];
    s_lv[t] = a.lut_v[lh * 8 + t];
  }
  const float ebar_k = paper ? a.ebar[lh * 2] : 0.0f;
  const float ebar_v = paper ? a.ebar[lh * 2 + 1] : 0.0f;
  // this lane's B operands: S[16q + 8h + j][32 nb + n] as S_hi + S_lo
  half8 shi[4], slo[4];
  if (!paper) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float sv = a.qjl_s[(16 * q + 8 * hh + j) * kDim + 32 * nb + n];
        const _Float16 hi = (_Float16)sv;
        shi[q][j] = hi;
        slo[q][j] = (_Float16)(sv - (float)hi);
      }
  }

  const int64_t unit = ((int64_t)li * a.B + b) * a.H + h;
  __half* ko = reinterpret_cast<__half*>(a.k_out) + unit * a.max_len * kDim;
  __half* vo = reinterpret_cast<__half*>(a.v_out) + unit * a.max_len * kDim;
  const int c = 32 * nb + n;            // the lane's output dimension
  const int tok = 32 * mb + n;          // the lane's token in the A operand

  for (int tt = tile_first; tt < tile_last; ++tt) {
    if (t < 128) s_k[t] = next.c;
    else s_v[t - 128] = next.c;
    if (t < 64) s_sc[t] = next.sc;
    __syncthreads();
    if (tt + 1 < tile_last) load_codes(next, kt, vt, st, (s0 >> 6) + tt + 1, t);

    // ---- residual estimates e[t][c] = sum_i S[i][c] (2 s_ti - 1) of keys
    // and (with V signs) values, as D blocks in the instruction's layout
    f32x16 ek, ev;
#pragma unroll
    for (int r = 0; r < 16; ++r) { ek[r] = 0.0f; ev[r] = 0.0f; }
    if (!paper) {
      const uint32_t* kw = reinterpret_cast<const uint32_t*>(s_k);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // key word 2q + h of token tok: chunk (2q + h) / 4, word (2q + h) % 4
        const int w = 2 * q + hh;
        const half8 sg = signs8(kw[((w >> 2) * 64 + tok) * 4 + (w & 3)] >> 24);
        ek = __builtin_amdgcn_mfma_f32_32x32x16_f16(sg, shi[q], ek, 0, 0, 0);
        ek = __builtin_amdgcn_mfma_f32_32x32x16_f16(sg, slo[q], ek, 0, 0, 0);
      }
      if (vqjl) {
        // V sign of token tok, dimension i: bit 3 of nibble tok % 8 of word
        // (tok / 8) % 4 of chunk (tok / 32, i)
        const uint32_t* vw = reinterpret_cast<const uint32_t*>(s_v);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t byte = 0;
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const uint32_t w = vw[((tok >> 5) * 64 + 16 * q + 8 * hh + j) * 4 + ((tok >> 3) & 3)];
            byte |= ((w >> (4 * (tok & 7) + 3)) & 1u) << j;
          }
          const half8 sg = signs8(byte);
          ev = __builtin_amdgcn_mfma_f32_32x32x16_f16(sg, shi[q], ev, 0, 0, 0);
          ev = __builtin_amdgcn_mfma_f32_32x32x16_f16(sg, slo[q], ev, 0, 0, 0);
        }
      }
    }

    // ---- the estimates to LDS: register r holds token 32 mb + 8 (r/4) + 4h + r%4,
    // dimension c (consecutive dimensions across a half wave: no conflicts)
    if (!paper) {
      int trb = 32 * mb + 4 * hh;
      asm volatile("" : "+v"(trb));
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int tr = trb + 8 * (r >> 2) + (r & 3);
        s_ek[tr * kDim + c] = ek[r];
        if constexpr (VQJL) s_ev[tr * kDim + c] = ev[r];
      }
    }
    __syncthreads();

    const int rows = min(64, len - 64 * tt);
    // ---- key rows: thread t writes dimensions 16g .. 16g + 15 (g = t % 4) of
    // token t / 4 straight to memory (two 16-byte stores)
    {
      const int tk = t >> 2, g = t & 3;
      const uint2 sc = s_sc[tk];
      const float nk8 = half_bits_to_float(sc.x) * 0.125f, gk = half_bits_to_float(sc.x >> 16);
      const float coef = paper ? ebar_k : kQjlAlpha * gk;
      const uint32_t* kw = reinterpret_cast<const uint32_t*>(s_k);
      uint32_t packed[8];
#pragma unroll
      for (int half16 = 0; half16 < 2; ++half16) {
        const int w = 2 * g + half16;                                  // key word: dims 8w .. 8w + 7
        const uint32_t word = kw[((w >> 2) * 64 + tk) * 4 + (w & 3)];
        const float4 e0 = paper ? make_float4(0.f, 0.f, 0.f, 0.f)
                                : *reinterpret_cast<const float4*>(s_ek + tk * kDim + 8 * w);
        const float4 e1 = paper ? make_float4(0.f, 0.f, 0.f, 0.f)
                                : *reinterpret_cast<const float4*>(s_ek + tk * kDim + 8 * w + 4);
        const float ee[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
          float kv[2];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            const uint32_t idx = (word >> (3 * (j + u))) & 7u;
            const float e = paper ? (((word >> (24 + j + u)) & 1u) ? 1.0f : -1.0f) : ee[j + u];
            kv[u] = (s_lk[idx] + coef * e) * nk8;
          }
          packed[4 * half16 + j / 2] = (uint32_t)__half_as_ushort(__float2half_rn(kv[0])) |
                                       ((uint32_t)__half_as_ushort(__float2half_rn(kv[1])) << 16);
        }
      }
      if (tk < rows) {
        __half* dst = ko + ((int64_t)64 * tt + tk) * kDim + 16 * g;
        reinterpret_cast<uint4*>(dst)[0] = make_uint4(packed[0], packed[1], packed[2], packed[3]);
        reinterpret_cast<uint4*>(dst)[1] = make_uint4(packed[4], packed[5], packed[6], packed[7]);
      }
    }
    // ---- value rows: thread t reads dimension i = t % 64's words of tokens
    // 16 (t / 64) .. + 15 and stages the 16 values in LDS
    {
      const int i = t & 63, tg = t >> 6;
      const uint32_t* vw = reinterpret_cast<const uint32_t*>(s_v);
#pragma unroll
      for (int w2 = 0; w2 < 2; ++w2) {
        const int t0 = 16 * tg + 8 * w2;                               // tokens t0 .. t0 + 7
        const uint32_t word = vw[((t0 >> 5) * 64 + i) * 4 + ((t0 >> 3) & 3)];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int tv = t0 + j;
          const uint32_t nib = (word >> (4 * j)) & 15u;
          const uint2 sc = s_sc[tv];
          float vv = s_lv[nib & 7u];
          if constexpr (VQJL) {
            const float sg = (nib >> 3) ? 1.0f : -1.0f;
            vv += paper ? ebar_v * sg : (kQjlAlpha * half_bits_to_float(sc.y >> 16)) * s_ev[tv * kDim + i];
          }
          s_ov[tv * kDim + i] = __float2half_rn(vv * (half_bits_to_float(sc.y) * 0.125f));
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int e0 = 0; e0 < 512; e0 += 256) {
      const int e = e0 + t, row = e >> 3, col = (e & 7) * 8;
      if (row < rows) {
        const int64_t j = (int64_t)64 * tt + row;
        *reinterpret_cast<uint4*>(vo + j * kDim + col) = *reinterpret_cast<const uint4*>(s_ov + row * kDim + col);
      }
    }
  }
}

hipError_t launch_dequantize(const DequantArgs& a, hipStream_t st) {
  const int ntiles = (a.max_len + 63) / 64;
  dim3 grid((ntiles + kTilesPerBlock - 1) / kTilesPerBlock, a.B * a.H, a.nlayers);
  if (a.flags & kVQjl)
    hipLaunchKernelGGL(dequant_kernel<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(dequant_kernel<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace tq
