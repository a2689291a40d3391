// Fused decode attention over the packed 3-bit cache (TurboESM Sec. 3.1
// decode steps 1-4; Algorithm 1 of Sec. 4.3), as two kernels.
//
// decode_prep_kernel (one block per (sequence, layer, head) unit)
//   q^ = Pi RoPE(q) and u = S q^ (u = q^ for the per-element residual form),
//   written to the workspace. Rotating the query once replaces the per-key
//   inverse rotation of Algorithm 1 (identical by Eq. 4). Each row of Pi is
//   shared by 4 contiguous lanes; a lane applies RoPE to its 16-element slice
//   of q in registers and the lanes of a row combine their partial sums with
//   DPP. For a decode step (APPEND) the same block first quantizes the new
//   key and value into the cache (quantize-then-attend), reusing its read of
//   Pi: the wave-per-vector quantizer of the append kernel, on Pi and S
//   staged in LDS.
//
// decode_kernel (one block of WAVES waves per unit, or per split of its tiles)
//   The cache read is bandwidth-bound and, with every block streaming at
//   once, a load issued behind the stream waits for it. So the block's own
//   small inputs (q^ and u, the two tables, the sequence's bounds) come
//   through scalar loads, all issued together before anything else; the
//   block's first tiles are requested after its tables are built, and Pi for
//   the epilogue goes straight into LDS after the last prologue barrier.
//   prologue  two LDS tables per unit: a pair table
//               T_A[p][a + 8 b] = q^_{2p} c_K[a] + q^_{2p+1} c_K[b]
//             (one read scores two dimensions' table terms) and a sign table
//               T_B[w][s] = sum_j u_{8w+j} (2 s_j - 1)
//             over the 8 sign bits s of key word w (one read per word for the
//             QJL term).
//   main loop keys are scored one lane per token from the key words (3-bit
//             indices in bits 0-23, signs in bits 24-31):
//             score = n_k/8 (sum T_A + coef sum T_B), coef = alpha g_k (QJL) or
//             ebar_K. Online softmax in base 2 with a wave-uniform running max
//             raised only when a tile max exceeds it by more than 2^8.
//             Values are accumulated one lane per dimension from the
//             dimension-major V tile; a tile's token weights reach the lanes
//             through DPP row broadcasts.
//   merge     waves merge through LDS; splits of a unit merge through a
//             workspace of (m, l, o) partials written and read with
//             agent-scope atomics: the last split to finish (atomic counter)
//             combines them by log-sum-exp.
//   epilogue  o = Pi^T (o^ / l) (one inverse rotation), plus the V residual
//             estimate alpha S^T s or ebar_V s when V carries sign bits.
// Work items are dealt so that all splits of a unit land on one XCD (blocks
// go to the 8 XCDs round-robin), and each unit's prep block runs on the XCD
// of its decode blocks.
#include <stdlib.h>

#include "tq_append.hpp"
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr float kLazyRescale = 8.0f;   // log2 headroom before the max is raised
constexpr int kXcds = 8;

// Block barrier that orders LDS only. __syncthreads() also waits for every
// outstanding global load of the wave (its release fence covers global
// memory), which would drain the tile prefetch at each prologue barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
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


// (byte 3 of x) << 2, one VALU op (sub-dword operand select).
__device__ __forceinline__ uint32_t byte3_x4(uint32_t x) {
  uint32_t r;
  asm("v_lshlrev_b32_sdwa %0, 2, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
      : "=v"(r) : "v"(x));
  return r;
}

// Score terms of key word W (dimensions 8W..8W+7) from the LDS tables
//   ta[P][f] = q^_{2P} c_K[f & 7] + q^_{2P+1} c_K[f >> 3]   (P: dimension pair)
//   tb[W][s] = sum_j (bit j of s ? u : -u)_{8W+j}            (s: the word's sign byte)
// The four 6-bit index pairs sit at bits 0, 6, 12 and 18 of the word: each is
// brought to bits 2..7 of a byte (4 x index: a float offset) by a shift and
// a byte-selecting AND; the sign byte by one byte-selecting shift.
template <int W>
__device__ __forceinline__ void key_word_score(const float* ta, const float* tb, uint32_t x,
                                               float& A, float& B) {
  const uint32_t m = 0xFCu;
  const uint32_t f0 = and_byte<0>(m, x << 2);    // bits 0..5   -> byte 0 bits 2..7
  const uint32_t f1 = and_byte<1>(m, x << 4);    // bits 6..11  -> byte 1 bits 2..7
  const uint32_t f2 = and_byte<1>(m, x >> 2);    // bits 12..17 -> byte 1 bits 2..7
  const uint32_t f3 = and_byte<2>(m, x);         // bits 18..23 -> byte 2 bits 2..7
  const uint32_t fs = byte3_x4(x);               // sign byte, times 4
  const char* pa = reinterpret_cast<const char*>(ta + (4 * W) * 64);
  const char* pb = reinterpret_cast<const char*>(tb + W * 256);
  const float a0 = *reinterpret_cast<const float*>(pa + f0);
  const float a1 = *reinterpret_cast<const float*>(pa + 256 + f1);
  const float a2 = *reinterpret_cast<const float*>(pa + 512 + f2);
  const float a3 = *reinterpret_cast<const float*>(pa + 768 + f3);
  const float b0 = *reinterpret_cast<const float*>(pb + fs);
  A += (a0 + a1) + (a2 + a3);
  B += b0;
}



// Token weights of a 64-token tile for the lane-per-dimension value loop.
// Lane t holds w_t; two lane swaps give four registers R_j holding tokens
// 16j .. 16j+15 in every 16-lane row (v_permlane32_swap exchanges the upper
// half of one register with the lower half of another, v_permlane16_swap the
// odd rows of one with the even rows of another). An FMA then reads w_{16j+k}
// through a DPP row broadcast of lane k (row_newbcast), so no weight costs an
// instruction of its own.
struct TileWeights {
  float r[4];
};

__device__ __forceinline__ TileWeights spread_weights(float w) {
  const int wi = __float_as_int(w);
  const auto h = __builtin_amdgcn_permlane32_swap(wi, wi, false, false);   // rows 0 1 0 1 | 2 3 2 3
  const auto lo = __builtin_amdgcn_permlane16_swap(h[0], h[0], false, false);   // 0 0 0 0 | 1 1 1 1
  const auto hi = __builtin_amdgcn_permlane16_swap(h[1], h[1], false, false);   // 2 2 2 2 | 3 3 3 3
  TileWeights tw;
  tw.r[0] = __int_as_float(lo[0]);
  tw.r[1] = __int_as_float(lo[1]);
  tw.r[2] = __int_as_float(hi[0]);
  tw.r[3] = __int_as_float(hi[1]);
  return tw;
}

// acc += w_{16j+K} * c, the weight taken from register R_j by a row broadcast.
template <int K>
__device__ __forceinline__ void fma_row_bcast(float& acc, float rj, float c) {
  asm("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
      : "+v"(acc) : "v"(rj), "v"(c), "i"(K));
}

// The 16 tokens 8*W8 .. 8*W8+15 of two value words: acc_{jj & 3} += w_t c_V[code].
// The 16 table reads are issued together (the empty asm makes them complete
// before the first FMA), so the LDS latency is paid once per word pair.
template <int W8>
__device__ __forceinline__ void value_words(const TileWeights& tw, uint32_t x0, uint32_t x1,
                                            const char* vtab, float& o0, float& o1, float& o2,
                                            float& o3) {
  uint32_t off[16];
  nibble_offsets4(x0, *reinterpret_cast<uint32_t(*)[8]>(off));
  nibble_offsets4(x1, *reinterpret_cast<uint32_t(*)[8]>(off + 8));
  float c[16];
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) c[jj] = *reinterpret_cast<const float*>(vtab + off[jj]);
  asm volatile("" : "+v"(c[0]), "+v"(c[1]), "+v"(c[2]), "+v"(c[3]), "+v"(c[4]), "+v"(c[5]),
               "+v"(c[6]), "+v"(c[7]), "+v"(c[8]), "+v"(c[9]), "+v"(c[10]), "+v"(c[11]),
               "+v"(c[12]), "+v"(c[13]), "+v"(c[14]), "+v"(c[15]));
  constexpr int J = W8 / 2;          // W8 is even: both words share R_J
  const float rj = tw.r[J];
  fma_row_bcast<0>(o0, rj, c[0]);
  fma_row_bcast<1>(o1, rj, c[1]);
  fma_row_bcast<2>(o2, rj, c[2]);
  fma_row_bcast<3>(o3, rj, c[3]);
  fma_row_bcast<4>(o0, rj, c[4]);
  fma_row_bcast<5>(o1, rj, c[5]);
  fma_row_bcast<6>(o2, rj, c[6]);
  fma_row_bcast<7>(o3, rj, c[7]);
  fma_row_bcast<8>(o0, rj, c[8]);
  fma_row_bcast<9>(o1, rj, c[9]);
  fma_row_bcast<10>(o2, rj, c[10]);
  fma_row_bcast<11>(o3, rj, c[11]);
  fma_row_bcast<12>(o0, rj, c[12]);
  fma_row_bcast<13>(o1, rj, c[13]);
  fma_row_bcast<14>(o2, rj, c[14]);
  fma_row_bcast<15>(o3, rj, c[15]);
}

// The V residual term of one word: acc += sum_t (+-1 by the sign bit) g_t.
template <int W8>
__device__ __forceinline__ void value_sign_word(const TileWeights& tg, uint32_t x, float& acc) {
  constexpr int J = W8 / 2, K0 = 8 * (W8 & 1);
  const float rj = tg.r[J];
  float sgn[8];
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) sgn[jj] = ((x >> (4 * jj + 3)) & 1u) ? 1.0f : -1.0f;
  fma_row_bcast<K0 + 0>(acc, rj, sgn[0]);
  fma_row_bcast<K0 + 1>(acc, rj, sgn[1]);
  fma_row_bcast<K0 + 2>(acc, rj, sgn[2]);
  fma_row_bcast<K0 + 3>(acc, rj, sgn[3]);
  fma_row_bcast<K0 + 4>(acc, rj, sgn[4]);
  fma_row_bcast<K0 + 5>(acc, rj, sgn[5]);
  fma_row_bcast<K0 + 6>(acc, rj, sgn[6]);
  fma_row_bcast<K0 + 7>(acc, rj, sgn[7]);
}

// N consecutive elements of an fp16 or fp32 vector, in two steps so that all
// prologue loads are in flight before the first wait: load_raw issues the
// 16-byte loads (element e0 is a multiple of 8, so they are aligned) and
// to_float converts after the remaining loads have been issued.
template <int N>
struct RawSlice {
  uint4 w[N / 4];
};

template <int N>
__device__ __forceinline__ void load_raw(const void* p, int64_t e0, bool f16, RawSlice<N>& r) {
  if (f16) {
    const uint4* q = reinterpret_cast<const uint4*>(reinterpret_cast<const __half*>(p) + e0);
#pragma unroll
    for (int j = 0; j < N / 8; ++j) r.w[j] = q[j];
  } else {
    const uint4* q = reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(p) + e0);
#pragma unroll
    for (int j = 0; j < N / 4; ++j) r.w[j] = q[j];
  }
}

template <int N>
__device__ __forceinline__ void to_float(const RawSlice<N>& r, bool f16, float (&x)[N]) {
  if (f16) {
#pragma unroll
    for (int j = 0; j < N / 8; ++j) {
      const uint32_t ws[4] = {r.w[j].x, r.w[j].y, r.w[j].z, r.w[j].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        x[8 * j + 2 * k] = half_bits_to_float(ws[k]);
        x[8 * j + 2 * k + 1] = half_bits_to_float(ws[k] >> 16);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < N / 4; ++j) {
      x[4 * j] = __uint_as_float(r.w[j].x); x[4 * j + 1] = __uint_as_float(r.w[j].y);
      x[4 * j + 2] = __uint_as_float(r.w[j].z); x[4 * j + 3] = __uint_as_float(r.w[j].w);
    }
  }
}


// Pointers into the constant address space (4): same 64-bit addresses, but a
// load through them with a wave-uniform address is always a scalar load.
#define TQ_CONST __attribute__((address_space(4)))
typedef const TQ_CONST float cfloat;
typedef const TQ_CONST int32_t cint32;
typedef const TQ_CONST int64_t cint64;
template <class T>
__device__ __forceinline__ const TQ_CONST T* to_const(const T* p) {
  return (const TQ_CONST T*)p;
}
// Two consecutive floats as one 64-bit scalar load (scalar loads need only
// 4-byte alignment).
typedef uint64_t __attribute__((aligned(4))) u64_a4;
__device__ __forceinline__ uint64_t load_pair(const TQ_CONST float* p) {
  return *(const TQ_CONST u64_a4*)p;
}
__device__ __forceinline__ float2 pair_f2(uint64_t w) {
  return make_float2(__uint_as_float((uint32_t)w), __uint_as_float((uint32_t)(w >> 32)));
}

// Eight table levels held in (scalar) registers; pick() selects one per lane
// by three levels of selects on the index bits, never through memory.
struct Lut8 {
  float c0, c1, c2, c3, c4, c5, c6, c7;
  __device__ __forceinline__ static Lut8 of(const uint64_t (&w)[4]) {
    const float2 a = pair_f2(w[0]), b = pair_f2(w[1]), c = pair_f2(w[2]), d = pair_f2(w[3]);
    return Lut8{a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
  }
  __device__ __forceinline__ float pick(int i) const {
    const bool b0 = (i & 1) != 0, b1 = (i & 2) != 0, b2 = (i & 4) != 0;
    const float p01 = b0 ? c1 : c0, p23 = b0 ? c3 : c2, p45 = b0 ? c5 : c4, p67 = b0 ? c7 : c6;
    const float p03 = b1 ? p23 : p01, p47 = b1 ? p67 : p45;
    return b2 ? p47 : p03;
  }
};

// ------------------------------------------------------------------ prep kernel
// Unit of prep block `bid`: the XCD of a unit's decode blocks is
// (unit * nsplit) / per_xcd; prep blocks are dealt to the same XCD.
// With APPEND (decode step) the block first stages Pi and S in LDS and,
// after q^ and u are written, waves 0 and 1 quantize and append the new key
// and value of the unit with the same functions as the append kernel.
// F16: q, k, v are fp16 (else fp32). HALF: RoPE pairs (m, m + 32).
template <bool APPEND, bool F16, bool HALF>
__global__ __launch_bounds__(256) void decode_prep_kernel(DecodeArgs a, int units, int per_xcd) {
  constexpr int COLS = 16;                 // 4 lanes per row of Pi / S
  __shared__ float s_qh[kDim];
  __shared__ VectorSmem sm;                // APPEND only (the compiler drops it otherwise)
  // Every argument field the block reads, in one batch met by one wait (the
  // asm uses them all), so that no data load waits behind a constant load.
  const int nsplit = a.nsplit, H = a.H, B = a.B, layer0 = a.layer0, rope_positions = a.rope_positions;
  const int len_add = a.len_add, max_len = a.max_len;
  const int64_t slots = a.slots;
  const uint32_t flags = a.flags;
  const float *pi_base = a.pi, *s_base = a.qjl_s, *cs_base = a.rope_cs;
  const void* q_base = a.q;
  const int32_t *qpos_p = a.q_pos, *len_p = a.seq_len;
  const int64_t* s0_p = a.seq_slot0;
  asm volatile("" ::"s"(nsplit), "s"(H), "s"(B), "s"(layer0), "s"(rope_positions), "s"(len_add),
               "s"(max_len), "s"(slots), "s"(flags), "s"(pi_base), "s"(s_base), "s"(cs_base),
               "s"(q_base), "s"(qpos_p), "s"(len_p), "s"(s0_p));
  // (32-bit: the host keeps units * nsplit, and so 8 * per_xcd, below 2^31)
  const unsigned x = blockIdx.x % kXcds, j = blockIdx.x / kXcds;
  const unsigned ns = (unsigned)nsplit, px = (unsigned)per_xcd;
  const unsigned first = (x * px + ns - 1) / ns;
  const unsigned next = ((x + 1) * px + ns - 1) / ns;
  const unsigned unit_u = first + j;
  if (unit_u >= next || unit_u >= (unsigned)units) return;
  const int unit = (int)unit_u;
  const int h = unit % H;
  const int b = (unit / H) % B;
  const int l = layer0 + unit / (H * B);
  const int lh = l * H + h;
  const int t = threadIdx.x;
  const int row = t >> 2, c0 = (t & 3) * COLS;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6), i = t & 63;
  const bool paper = (flags & kQjlPaper) != 0;

  // Loads first, none behind a check: Pi and S row slices, q, and for a step
  // the new key (wave 0) or value (wave 1) with its table levels. Then the
  // sequence's position, length and first slot (scalar loads, one wait), and
  // the RoPE row of the position (clamped into the table, so it is requested
  // as soon as the position arrives, before the checks).
  const float4* pi_row = reinterpret_cast<const float4*>(pi_base + (int64_t)lh * kDim * kDim + row * kDim + c0);
  const float4* s_row = reinterpret_cast<const float4*>(s_base + row * kDim + c0);
  float4 pr[COLS / 4], sr[COLS / 4];
#pragma unroll
  for (int k = 0; k < COLS / 4; ++k) pr[k] = pi_row[k];
#pragma unroll
  for (int k = 0; k < COLS / 4; ++k) sr[k] = s_row[k];
  RawSlice<COLS> qraw, praw;
  load_raw<COLS>(q_base, (int64_t)unit * kDim + c0, F16, qraw);
  if (HALF) load_raw<COLS>(q_base, (int64_t)unit * kDim + (c0 ^ 32), F16, praw);
  float xa = 0.0f;
  Levels La{};
  if (APPEND) {
    xa = load_in(wave == 1 ? a.v_new : a.k_new, (int64_t)unit * kDim + i, F16);
    La = load_levels((wave == 1 ? a.lut_v : a.lut_k) + lh * 8);
  }
  const int qp = to_const(qpos_p)[b];
  const int len = to_const(len_p)[b];
  const int64_t s0 = to_const(s0_p)[b];
  asm volatile("" ::"s"(qp), "s"(len), "s"(s0));
  const int qpc = min(max(qp, 0), rope_positions - 1);
  const float4* cs_row = reinterpret_cast<const float4*>(cs_base + (int64_t)qpc * 2 * kPairs);
  float4 csv[COLS / 2];
  if (HALF) {
#pragma unroll
    for (int k = 0; k < COLS / 2; ++k) csv[k] = cs_row[(c0 & 31) / 2 + k];   // pairs (c0 & 31) ..
  } else {
#pragma unroll
    for (int k = 0; k < COLS / 4; ++k) csv[k] = cs_row[c0 / 4 + k];          // pairs c0/2 ..
  }
  float2 csk = make_float2(1.0f, 0.0f);
  if (APPEND)
    csk = reinterpret_cast<const float2*>(cs_base + (int64_t)qpc * 2 * kPairs)[HALF ? (i & 31) : (i >> 1)];

  const int n = len + len_add;             // tokens attended
  if (qp < 0 || qp >= rope_positions || n <= 0) return;   // the decode kernel writes 0 or NaN
  // the new token goes to slot s0 + len exactly when the decode kernel will
  // accept the sequence (it checks the same bounds for n = len + 1)
  const bool do_append = APPEND && len >= 0 && n <= max_len && s0 >= 0 && (s0 & 63) == 0 &&
                         s0 + n <= slots;
  if (do_append) {
    // Pi and S for the wave-per-vector quantizer: this thread holds columns
    // c0 .. c0 + 15 of row `row`
#pragma unroll
    for (int k = 0; k < COLS / 4; ++k) {
      stage_row4(sm.pi, row, c0 + 4 * k, pr[k]);
      stage_row4(sm.s, row, c0 + 4 * k, sr[k]);
    }
  }

  // q' = RoPE(q) in registers (x'_a = x_a c - x_b s, x'_b = x_a s + x_b c)
  float qx[COLS], qy[COLS], qr[COLS];
  to_float<COLS>(qraw, F16, qx);
  if (HALF) {
    to_float<COLS>(praw, F16, qy);
#pragma unroll
    for (int k = 0; k < COLS; ++k) {
      const float4 v = csv[k / 2];
      const float c = (k & 1) ? v.z : v.x, sn = (k & 1) ? v.w : v.y;
      qr[k] = (c0 + k) < 32 ? (qx[k] * c - qy[k] * sn) : (qy[k] * sn + qx[k] * c);
    }
  } else {
#pragma unroll
    for (int k = 0; k < COLS; k += 2) {
      const float4 v = csv[k / 4];
      const float c = (k & 2) ? v.z : v.x, sn = (k & 2) ? v.w : v.y;
      qr[k] = qx[k] * c - qx[k + 1] * sn;
      qr[k + 1] = qx[k] * sn + qx[k + 1] * c;
    }
  }
  float acc = 0.0f;
#pragma unroll
  for (int k = 0; k < COLS / 4; ++k) {
    acc = fmaf(pr[k].x, qr[4 * k + 0], acc);
    acc = fmaf(pr[k].y, qr[4 * k + 1], acc);
    acc = fmaf(pr[k].z, qr[4 * k + 2], acc);
    acc = fmaf(pr[k].w, qr[4 * k + 3], acc);
  }
  acc += dpp<0xB1>(acc);               // quad_perm [1,0,3,2]
  acc += dpp<0x4E>(acc);               // quad_perm [2,3,0,1]: every lane of the row has q^_row
  const float qh_row = acc;
  float* qu = a.qu + (int64_t)unit * 2 * kDim;
  if ((t & 3) == 0) { s_qh[row] = qh_row; qu[row] = qh_row; }
  float u_row = qh_row;
  if (!paper) {
    lds_barrier();
    float up = 0.0f;
#pragma unroll
    for (int k = 0; k < COLS / 4; ++k) {
      const float4 v = *reinterpret_cast<const float4*>(s_qh + c0 + 4 * k);
      up = fmaf(sr[k].x, v.x, up);
      up = fmaf(sr[k].y, v.y, up);
      up = fmaf(sr[k].z, v.z, up);
      up = fmaf(sr[k].w, v.w, up);
    }
    up += dpp<0xB1>(up);
    up += dpp<0x4E>(up);
    u_row = up;
  }
  if ((t & 3) == 1) qu[kDim + row] = u_row;

  if (do_append) {
    lds_barrier();                     // Pi and S staged
    if (wave < 2) {
      const bool is_v = wave == 1;
      const int ksign = paper ? 2 : 1;
      const int sign_mode = is_v ? ((a.flags & kVQjl) ? ksign : 0) : ksign;
      const bool rotate = !is_v || (a.flags & kVRotate);
      const float xr = is_v ? xa : rope_wave(xa, csk, HALF, i);
      append_wave(xr, is_v, rotate, La, sm, sign_mode, s0 + len, lh, const_cast<uint8_t*>(a.k_codes),
                  const_cast<uint8_t*>(a.v_codes), const_cast<uint16_t*>(a.scalars), a.slots, i, wave);
    }
  }
}


template <int WAVES, bool VQJL>
__global__ __launch_bounds__(WAVES * 64)
__attribute__((amdgpu_waves_per_eu((WAVES == 8 && !VQJL) ? 6 : 1)))
void decode_kernel(DecodeArgs a, int total_work, int per_xcd) {
  constexpr int TAM = 2048 / (WAVES * 64);   // pair-table entries per thread
  constexpr int TBM = 512 / (WAVES * 64);    // groups of 4 sign-table entries per thread
  constexpr int COLS = kDim / WAVES;       // rows of Pi per thread in the epilogue
  constexpr int DEPTH = (WAVES == 8) ? 1 : 2;
  constexpr int NT = WAVES * 64;
  constexpr int PIV = 1024 / NT;          // float4 of Pi per thread
  __shared__ float s_ta[32 * 64];          // pair table of the score's table term
  __shared__ __attribute__((aligned(16))) float s_tb[8 * 256];   // sign-byte table of the QJL term
  __shared__ __attribute__((aligned(16))) float s_pi[kDim * kDim];
  __shared__ float s_vtab[16];
  __shared__ float s_part[WAVES][kDim];
  __shared__ float s_wo[WAVES][kDim];
  __shared__ float s_wsg[VQJL ? WAVES : 1][kDim];
  __shared__ float s_wm[WAVES], s_wl[WAVES];
  __shared__ float s_oh[kDim], s_sh[kDim];
  __shared__ int s_last;
  const int bid = blockIdx.x;
  const int work = (bid % kXcds) * per_xcd + bid / kXcds;
  if (work >= total_work) return;
  // The argument fields the prologue needs, read in one batch and met by one
  // wait (used by the asm), so that no later data load waits on one of them.
  const int nsplit = a.nsplit, H = a.H, B = a.B, layer0 = a.layer0;
  const uint32_t flags = a.flags;
  const float *qu_base = a.qu, *lut_k = a.lut_k, *lut_v = a.lut_v, *ebar = a.ebar;
  const int32_t* seq_len = a.seq_len;
  const int64_t* seq_slot0 = a.seq_slot0;
  const int32_t* q_pos = a.q_pos;
  asm volatile("" ::"s"(nsplit), "s"(H), "s"(B), "s"(layer0), "s"(flags), "s"(qu_base), "s"(lut_k),
               "s"(lut_v), "s"(ebar), "s"(seq_len), "s"(seq_slot0), "s"(q_pos));
  const int unit = work / nsplit;
  const int split = work - unit * nsplit;
  const int h = unit % H;
  const int b = (unit / H) % B;
  const int li = unit / (H * B);
  const int l = layer0 + li;
  const int lh = l * H + h;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);

  const bool paper = (flags & kQjlPaper) != 0;

  // ------------------------------------------------------- prologue loads
  // Everything the prologue reads is the same for a whole wave and is fetched
  // with scalar loads, issued before anything else and before the first store
  // of the kernel (so the compiler may take the scalar path): the scalar cache
  // does not queue behind the tile loads that blocks already running on this
  // compute unit have in its vector memory pipeline, which can hold a late
  // block's first vector load for several microseconds.
  // Table entries built by this thread (NT threads):
  //   ta (2048 entries): e = t + NT m, pair P = e / 64 = wave + NT/64 m, index f = e % 64 = lane
  //   tb (2048 entries in groups of 4): group e = t + NT m of word w = e / 64,
  //      sign bytes 4 (e % 64) .. 4 (e % 64) + 3
  // Read through the constant address space: loads from it with a wave-uniform
  // address always take the scalar path. (Nothing here changes during a launch:
  // q^ and u come from the preceding prep kernel.)
  const cfloat* p_qu = to_const(qu_base);
  const cfloat* p_lk = to_const(lut_k);
  const cfloat* p_lv = to_const(lut_v);
  const cfloat* p_eb = to_const(ebar);
  const cint32* p_len = to_const(seq_len);
  const cint64* p_s0 = to_const(seq_slot0);
  const cint32* p_qp = to_const(q_pos);
  const cfloat* qu = p_qu + (int64_t)unit * 2 * kDim;
  const cfloat* lk = p_lk + lh * 8;
  const cfloat* lv = p_lv + lh * 8;
  // Loaded as 64-bit pairs: one asm operand each (an asm takes at most 30).
  uint64_t qw[TAM], uw[TBM][4], kw[4], vw[4];
#pragma unroll
  for (int m = 0; m < TAM; ++m) qw[m] = load_pair(qu + 2 * (wave + (NT / 64) * m));
#pragma unroll
  for (int m = 0; m < TBM; ++m) {
    const cfloat* e = qu + kDim + 8 * (wave + (NT / 64) * m);
#pragma unroll
    for (int k = 0; k < 4; ++k) uw[m][k] = load_pair(e + 2 * k);
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    kw[k] = load_pair(lk + 2 * k);
    vw[k] = load_pair(lv + 2 * k);
  }
  const float ebar_raw = *(paper ? p_eb + lh * 2 : lk);
  const int n = p_len[b] + a.len_add;
  const int64_t s0 = p_s0[b];
  const int qp = p_qp[b];
  // Every loaded value is used here, before the checks branch: the loads are
  // independent, so they are all issued and met by one wait (a load is
  // otherwise free to sink below the branch, one round trip after the other).
  static_assert(TAM + 4 * TBM + 8 + 4 <= 30, "asm operand limit");
  if constexpr (TBM == 1) {
    asm volatile("" ::"s"(qw[0]), "s"(qw[1]), "s"(qw[2]), "s"(qw[3]), "s"(uw[0][0]), "s"(uw[0][1]),
                 "s"(uw[0][2]), "s"(uw[0][3]), "s"(kw[0]), "s"(kw[1]), "s"(kw[2]), "s"(kw[3]),
                 "s"(vw[0]), "s"(vw[1]), "s"(vw[2]), "s"(vw[3]), "s"(ebar_raw), "s"(n), "s"(s0),
                 "s"(qp));
  } else {
    asm volatile("" ::"s"(qw[0]), "s"(qw[1]), "s"(qw[2]), "s"(qw[3]), "s"(qw[4]), "s"(qw[5]),
                 "s"(qw[6]), "s"(qw[7]), "s"(uw[0][0]), "s"(uw[0][1]), "s"(uw[0][2]),
                 "s"(uw[0][3]), "s"(uw[1][0]), "s"(uw[1][1]), "s"(uw[1][2]), "s"(uw[1][3]),
                 "s"(kw[0]), "s"(kw[1]), "s"(kw[2]), "s"(kw[3]), "s"(vw[0]), "s"(vw[1]),
                 "s"(vw[2]), "s"(vw[3]), "s"(ebar_raw), "s"(n), "s"(s0), "s"(qp));
  }
  float2 qpair[TAM];
#pragma unroll
  for (int m = 0; m < TAM; ++m) qpair[m] = pair_f2(qw[m]);
  float4 ulo[TBM], uhi[TBM];
#pragma unroll
  for (int m = 0; m < TBM; ++m) {
    const float2 a0 = pair_f2(uw[m][0]), a1 = pair_f2(uw[m][1]);
    const float2 a2 = pair_f2(uw[m][2]), a3 = pair_f2(uw[m][3]);
    ulo[m] = make_float4(a0.x, a0.y, a1.x, a1.y);
    uhi[m] = make_float4(a2.x, a2.y, a3.x, a3.y);
  }
  const Lut8 ck = Lut8::of(kw), cvl = Lut8::of(vw);
  const float ebar_k = paper ? ebar_raw : 0.0f;
  const bool valid = (n >= 0) & (n <= a.max_len) & (s0 >= 0) & ((s0 & 63) == 0) &
                     (s0 + n <= a.slots) & (qp >= 0) & (qp < a.rope_positions);
  if (!valid || n == 0) {
    if (split == 0 && t < kDim) store_out(a, unit, t, valid ? 0.0f : __int_as_float(0x7FC00000));
    return;
  }
  const int ntiles = (n + 63) >> 6;
  const int tile_begin = split * a.split_tiles;
  if (tile_begin >= ntiles) return;
  const int tile_end = min(ntiles, tile_begin + a.split_tiles);
  const int participants = (ntiles + a.split_tiles - 1) / a.split_tiles;
  const float ck_lo = ck.pick(lane & 7), ck_hi = ck.pick(lane >> 3);
  const float cv = cvl.pick(t & 7);

  const uint8_t* kreg = a.k_codes + (int64_t)lh * a.slots * 32;
  const uint8_t* vreg = a.v_codes + (int64_t)lh * a.slots * 32;
  const uint2* sreg = reinterpret_cast<const uint2*>(a.scalars + (int64_t)lh * a.slots * 4);
  const int64_t tile0 = s0 >> 6;
  // --------------------------------------------------------------- prologue
#pragma unroll
  for (int m = 0; m < TAM; ++m)
    s_ta[t + NT * m] = fmaf(qpair[m].y, ck_hi, qpair[m].x * ck_lo);
#pragma unroll
  for (int m = 0; m < TBM; ++m) {
    const int e = t + NT * m, k = e & 63;
    const float u[8] = {ulo[m].x, ulo[m].y, ulo[m].z, ulo[m].w, uhi[m].x, uhi[m].y, uhi[m].z, uhi[m].w};
    float base = 0.0f;                 // sign bits 2..7 of the bytes 4k .. 4k+3 are the bits of k
#pragma unroll
    for (int j = 2; j < 8; ++j) base += ((k >> (j - 2)) & 1) ? u[j] : -u[j];
    float4 v;
    v.x = (base - u[0]) - u[1];
    v.y = (base + u[0]) - u[1];
    v.z = (base - u[0]) + u[1];
    v.w = (base + u[0]) + u[1];
    reinterpret_cast<float4*>(s_tb)[e] = v;
  }
  s_vtab[t & 15] = cv;             // every thread: identical values, no branch around the load
  // The first tiles are requested only now: issuing a vector load can stall
  // while this compute unit's memory pipeline is full, and the tables above
  // need nothing from it.
  TileRegs buf[DEPTH];
#pragma unroll
  for (int d = 0; d < DEPTH; ++d) {
    const int tq = min(tile_begin + wave + d * WAVES, tile_end - 1);   // (a wave without tiles re-reads one)
    load_tile(buf[d], kreg, vreg, sreg, tile0 + tq, s0, tq, lane);
  }
  lds_barrier();

  // Pi for the epilogue, straight into LDS (1 KB per wave instruction). Issued
  // after the last barrier before the merge: the compiler makes a barrier wait
  // for transfers into LDS still in flight.
  {
    typedef __attribute__((address_space(3))) void* lds_ptr;
    const float* pig = a.pi + (int64_t)lh * kDim * kDim;
#pragma unroll
    for (int j = 0; j < PIV; ++j) {
      const int chunk = (wave + WAVES * j) * 64;    // first 16-byte chunk of this wave instruction
      __builtin_amdgcn_global_load_lds(pig + (chunk + lane) * 4, (lds_ptr)(s_pi + chunk * 4), 16, 0, 0);
    }
  }

  // -------------------------------------------------------------- main loop
  float m_run = -INFINITY;
  float l_lane = 0.0f;
  float sg = 0.0f;
  float o0 = 0.0f, o1 = 0.0f, o2 = 0.0f, o3 = 0.0f;
  const float lscale = a.logit_scale2;
  const char* vtab = reinterpret_cast<const char*>(s_vtab);

  for (int tb = tile_begin + wave; tb < tile_end; tb += DEPTH * WAVES) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int tt = tb + d * WAVES;
      if (tt >= tile_end) break;
      const TileRegs& cur = buf[d];
      const int tok = tt * kTile + lane;
      const bool tv = tok < n;
      // ---- key score, one lane per token: per key word 4 pair-table reads
      // (table term) and 1 sign-table read (QJL term). The empty asm pins the
      // partial sums half way so the compiler does not hoist every table read
      // of the tile (registers, occupancy).
      float A = 0.0f, B = 0.0f;
      key_word_score<0>(s_ta, s_tb, cur.k0.x, A, B);
      key_word_score<1>(s_ta, s_tb, cur.k0.y, A, B);
      key_word_score<2>(s_ta, s_tb, cur.k0.z, A, B);
      key_word_score<3>(s_ta, s_tb, cur.k0.w, A, B);
      asm volatile("" : "+v"(A), "+v"(B));
      key_word_score<4>(s_ta, s_tb, cur.k1.x, A, B);
      key_word_score<5>(s_ta, s_tb, cur.k1.y, A, B);
      key_word_score<6>(s_ta, s_tb, cur.k1.z, A, B);
      key_word_score<7>(s_ta, s_tb, cur.k1.w, A, B);
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
      const float wg = VQJL ? (paper ? wv : wv * gv) : 0.0f;

      // ---- value accumulate, one lane per dimension; token weights through
      // row broadcasts (spread_weights)
      const uint32_t vw[8] = {cur.v0.x, cur.v0.y, cur.v0.z, cur.v0.w, cur.v1.x, cur.v1.y, cur.v1.z, cur.v1.w};
      const TileWeights tw = spread_weights(wv);
      value_words<0>(tw, vw[0], vw[1], vtab, o0, o1, o2, o3);
      value_words<2>(tw, vw[2], vw[3], vtab, o0, o1, o2, o3);
      value_words<4>(tw, vw[4], vw[5], vtab, o0, o1, o2, o3);
      value_words<6>(tw, vw[6], vw[7], vtab, o0, o1, o2, o3);
      if (VQJL) {
        const TileWeights tg = spread_weights(wg);
        value_sign_word<0>(tg, vw[0], sg);
        value_sign_word<1>(tg, vw[1], sg);
        value_sign_word<2>(tg, vw[2], sg);
        value_sign_word<3>(tg, vw[3], sg);
        value_sign_word<4>(tg, vw[4], sg);
        value_sign_word<5>(tg, vw[5], sg);
        value_sign_word<6>(tg, vw[6], sg);
        value_sign_word<7>(tg, vw[7], sg);
      }
        const int tn = tt + DEPTH * WAVES;
        if (tn < tile_end) load_tile(buf[d], kreg, vreg, sreg, tile0 + tn, s0, tn, lane);
    }
  }

  // ------------------------------------------------------ merge the waves
  // (a full barrier: it also waits for this wave's Pi transfer into LDS)
  const float ov = (o0 + o1) + (o2 + o3);
  const float l_wave = wave_sum_uniform(l_lane);
  if (lane == 0) { s_wm[wave] = m_run; s_wl[wave] = l_wave; }
  s_wo[wave][lane] = ov;
  if (VQJL) s_wsg[wave][lane] = sg;
  __syncthreads();
  float M = -INFINITY, L = 0.0f, O = 0.0f, SG = 0.0f;
  if (t < kDim) {
#pragma unroll
    for (int w = 0; w < WAVES; ++w) M = fmaxf(M, s_wm[w]);
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float f = __builtin_amdgcn_exp2f(s_wm[w] - M);
      L += s_wl[w] * f;
      O += s_wo[w][t] * f;
      if (VQJL) SG += s_wsg[w][t] * f;
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
      s_last = (prev == (uint32_t)(participants - 1)) ? 1 : 0;
    }
    lds_barrier();
    if (!s_last) return;
    if (t < kDim) {
      // Wave 0 merges. Lane p holds split p's (m, l) (64 splits at a time);
      // the o rows are fetched 8 splits per batch with the batch's loads in
      // flight together (a loop that used each load before issuing the next
      // would pay one memory round trip per split).
      const float* base = a.partials + (int64_t)unit * a.nsplit * kPartialFloats;
      float Mw = -INFINITY;
      for (int p0 = 0; p0 < participants; p0 += 64) {
        const int pc = min(p0 + lane, participants - 1);
        Mw = fmaxf(Mw, __hip_atomic_load(base + (int64_t)pc * kPartialFloats, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT));
      }
      M = wave_max_uniform(Mw);
      float Ll = 0.0f;
      O = 0.0f; SG = 0.0f;
      for (int p0 = 0; p0 < participants; p0 += 64) {
        const int cnt = min(64, participants - p0);
        const float* pp = base + (int64_t)min(p0 + lane, participants - 1) * kPartialFloats;
        const float mp = __hip_atomic_load(pp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const float lp = __hip_atomic_load(pp + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const float f = (lane < cnt && mp != -INFINITY) ? __builtin_amdgcn_exp2f(mp - M) : 0.0f;
        Ll = fmaf(f, lp, Ll);
        const int fi = __float_as_int(f);
        for (int q0 = 0; q0 < cnt; q0 += 8) {
          float ov[8], sv[8];
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            const float* pq = base + (int64_t)(p0 + min(q0 + r, cnt - 1)) * kPartialFloats;
            ov[r] = __hip_atomic_load(pq + 4 + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (VQJL) sv[r] = __hip_atomic_load(pq + 4 + kDim + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
#pragma unroll
          for (int r = 0; r < 8; ++r) {
            // weight of split p0 + q0 + r (0 past the last: lanes >= cnt hold f = 0)
            const float fq = __int_as_float(__builtin_amdgcn_readlane(fi, min(q0 + r, 63)));
            O = fmaf(fq, ov[r], O);
            if (VQJL) SG = fmaf(fq, sv[r], SG);
          }
        }
      }
      L = wave_sum_uniform(Ll);
    }
    // leave the workspace zeroed for the next call
    if (t == 0) __hip_atomic_store(a.counters + unit, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // --------------------------------------------------------------- epilogue
  const int cq = t >> 6;                   // row group of the epilogue products
  const float invL = 1.0f / L;
  if (t < kDim) { s_oh[t] = O * invL; s_sh[t] = SG * invL; }
  lds_barrier();
  if (VQJL) {
    if (paper) {
      const float ebar_v = a.ebar[lh * 2 + 1];
      if (t < kDim) s_oh[t] += ebar_v * s_sh[t];
    } else {
      // o^ += alpha S^T s; thread (k, group) sums COLS rows of column k of S
      const int k = t & 63;
      float acc = 0.0f;
#pragma unroll
      for (int ii = 0; ii < COLS; ++ii) {
        const int i = cq * COLS + ii;
        acc = fmaf(a.qjl_s[i * kDim + k], s_sh[i], acc);
      }
      s_part[cq][k] = acc;
      lds_barrier();
      if (t < kDim) {
        float y = 0.0f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) y += s_part[w][t];
        s_oh[t] += kQjlAlpha * y;
      }
    }
    lds_barrier();
  }
  if (a.flags & kVRotate) {
    // out_k = sum_i Pi[i][k] o^_i: thread (k, group) sums COLS rows
    const int k = t & 63;
    float acc = 0.0f;
#pragma unroll
    for (int ii = 0; ii < COLS; ++ii) {
      const int i = cq * COLS + ii;
      acc = fmaf(s_pi[i * kDim + k], s_oh[i], acc);
    }
    s_part[cq][k] = acc;
    lds_barrier();
    if (t < kDim) {
      float y = 0.0f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) y += s_part[w][t];
      store_out(a, unit, t, y);
    }
  } else {
    if (t < kDim) store_out(a, unit, t, s_oh[t]);
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
  // prep blocks: per XCD, the units whose decode blocks run there
  const int64_t prep_per_xcd = (per_xcd + a.nsplit - 1) / a.nsplit + 1;
  {
    const dim3 pg((unsigned)(kXcds * prep_per_xcd)), pb(256);
    const bool f16 = a.f16_in != 0, half = (a.flags & kRopeHalf) != 0;
#define TQ_PREP(AP, F, HF) hipLaunchKernelGGL((decode_prep_kernel<AP, F, HF>), pg, pb, 0, st, a, (int)units, (int)per_xcd)
    if (a.append) {
      if (f16) { if (half) TQ_PREP(true, true, true); else TQ_PREP(true, true, false); }
      else     { if (half) TQ_PREP(true, false, true); else TQ_PREP(true, false, false); }
    } else {
      if (f16) { if (half) TQ_PREP(false, true, true); else TQ_PREP(false, true, false); }
      else     { if (half) TQ_PREP(false, false, true); else TQ_PREP(false, false, false); }
    }
#undef TQ_PREP
  }
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
