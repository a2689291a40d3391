// Dequantize the packed cache into fp16 key and value rows: the first step of
// a "dequantize first, then attend" path, the comparison the paper makes for
// its fused kernel (Sec. 5.4, Table 6). The rows are what the fused decode
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
// in LDS (the next tile's are loaded while the current one is computed), the
// fp16 rows are assembled in LDS and written with 16-byte stores.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

namespace {

constexpr int kTilesPerBlock = 4;
typedef float f32x16 __attribute__((ext_vector_type(16)));

// c[i & 7] by three levels of selects (a register table, never memory).
__device__ __forceinline__ float pick8(const float (&c)[8], uint32_t i) {
  const bool b0 = (i & 1u) != 0, b1 = (i & 2u) != 0, b2 = (i & 4u) != 0;
  const float p01 = b0 ? c[1] : c[0], p23 = b0 ? c[3] : c[2];
  const float p45 = b0 ? c[5] : c[4], p67 = b0 ? c[7] : c[6];
  const float p03 = b1 ? p23 : p01, p47 = b1 ? p67 : p45;
  return b2 ? p47 : p03;
}

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
  __shared__ __attribute__((aligned(16))) __half s_ok[64 * 64];  // k~ rows of the tile
  __shared__ __attribute__((aligned(16))) __half s_ov[64 * 64];  // v~ rows of the tile

  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int n = lane & 31, hh = lane >> 5;
  const int mb = wave & 1, nb = wave >> 1;
  const int h = blockIdx.y % a.H, b = blockIdx.y / a.H, li = blockIdx.z;
  const int l = a.layer0 + li;
  const int64_t lh = (int64_t)l * a.H + h;
  const int len = a.seq_len[b];
  const int64_t s0 = a.seq_slot0[b];
  if (len <= 0 || len > a.max_len || s0 < 0 || (s0 & 63) != 0 || s0 + len > a.slots) return;
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
  float ck[8], cv[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) { ck[m] = a.lut_k[lh * 8 + m]; cv[m] = a.lut_v[lh * 8 + m]; }
  // pinned in registers: a select between elements of a table in an array
  // would otherwise be folded into an indexed load from private memory
  asm volatile("" : "+v"(ck[0]), "+v"(ck[1]), "+v"(ck[2]), "+v"(ck[3]), "+v"(ck[4]), "+v"(ck[5]),
               "+v"(ck[6]), "+v"(ck[7]));
  asm volatile("" : "+v"(cv[0]), "+v"(cv[1]), "+v"(cv[2]), "+v"(cv[3]), "+v"(cv[4]), "+v"(cv[5]),
               "+v"(cv[6]), "+v"(cv[7]));
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

    // ---- rows: register r holds token 32 mb + 8 (r/4) + 4h + r%4, dimension c
    // (the row base is re-derived per tile: the empty asm keeps the compiler
    // from holding every row's addresses across the tile loop)
    const uint32_t* kw = reinterpret_cast<const uint32_t*>(s_k);
    const uint32_t* vw = reinterpret_cast<const uint32_t*>(s_v);
    int trb = 32 * mb + 4 * hh;
    asm volatile("" : "+v"(trb));
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int tr = trb + 8 * (r >> 2) + (r & 3);
      const uint2 sc = s_sc[tr];
      const float nk = half_bits_to_float(sc.x), gk = half_bits_to_float(sc.x >> 16);
      const float nv = half_bits_to_float(sc.y), gv = half_bits_to_float(sc.y >> 16);
      // key word c/8 of token tr: chunk c/32 = nb, word (c/8) % 4
      const uint32_t kword = kw[(nb * 64 + tr) * 4 + ((c >> 3) & 3)];
      const uint32_t kidx = (kword >> (3 * (c & 7))) & 7u;
      const float ksg = ((kword >> (24 + (c & 7))) & 1u) ? 1.0f : -1.0f;
      float kv = pick8(ck, kidx);
      kv += paper ? ebar_k * ksg : (kQjlAlpha * gk) * ek[r];
      // value nibble of token tr, dimension c
      const uint32_t vword = vw[((tr >> 5) * 64 + c) * 4 + ((tr >> 3) & 3)];
      const uint32_t vnib = (vword >> (4 * (tr & 7))) & 15u;
      float vv = pick8(cv, vnib);
      if (vqjl) {
        const float vsg = (vnib >> 3) ? 1.0f : -1.0f;
        vv += paper ? ebar_v * vsg : (kQjlAlpha * gv) * ev[r];
      }
      s_ok[tr * kDim + c] = __float2half_rn(kv * (nk * 0.125f));
      s_ov[tr * kDim + c] = __float2half_rn(vv * (nv * 0.125f));
      if ((r & 3) == 3) asm volatile("" ::: "memory");   // four rows' reads at a time (registers)
    }
    __syncthreads();

    // ---- 16-byte stores of the tile's valid rows (the staging is rewritten
    // only after the next iteration's first barrier)
    const int rows = min(64, len - 64 * tt);
#pragma unroll
    for (int e0 = 0; e0 < 512; e0 += 256) {
      const int e = e0 + t, row = e >> 3, col = (e & 7) * 8;
      if (row < rows) {
        const int64_t j = (int64_t)64 * tt + row;
        *reinterpret_cast<uint4*>(ko + j * kDim + col) = *reinterpret_cast<const uint4*>(s_ok + row * kDim + col);
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
