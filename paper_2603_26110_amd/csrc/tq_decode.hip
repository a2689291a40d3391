// Fused decode attention over the packed 3-bit cache (TurboESM Sec. 3.1
// decode steps 1-4; Algorithm 1 of Sec. 4.3), one kernel per call.
//
// decode_kernel (one block of WAVES waves per (sequence, layer, head) unit, or
// per split of its tiles)
//   loads     Pi and S are copied straight from global memory into LDS
//             (16-byte direct copies into the Swz16 layout), before anything
//             else; the sequence's bounds and the two tables of levels come
//             through scalar loads.
//   prologue  q^ = Pi RoPE(q) and u = S q^ (u = q^ for the per-element
//             residual form), by all waves: 8 lanes per row of Pi, summed by
//             DPP. Rotating the query once replaces the per-key inverse
//             rotation of Algorithm 1 (identical by Eq. 4). Then two LDS
//             tables per unit: a pair table
//               T_A[p][a + 8 b] = q^_{2p} c_K[a] + q^_{2p+1} c_K[b]
//             (one read scores two dimensions' table terms) and a sign table
//               T_B[w][s] = sum_j u_{8w+j} (2 s_j - 1)
//             over the 8 sign bits s of key word w (one read per word for the
//             QJL term). Only then are the block's tiles requested: a block
//             that starts later on the same compute unit then finds its own
//             Pi copy ahead of them in the memory pipeline.
//   step      for a decode step (quantize-then-attend) waves 1 and 2 then
//             quantize the new key and value into the cache with the append
//             kernel's wave-per-vector quantizer on the staged Pi and S, while
//             the other waves score.
//   last token the tiles cover tokens 0 .. n-2; token n-1 (a step's new one)
//             is scored on its own by wave 3 after its tiles, from the
//             append's codes in LDS (a step) or from registers loaded with
//             its first tile (an attend). With 1024 cached tokens and one new
//             one every wave then takes two tiles, where a 17th one-token
//             tile would cost one wave a third round trip and a full tile of
//             work.
//   main loop keys are scored one lane per token from the key words (3-bit
//             indices in bits 0-23, signs in bits 24-31):
//             score = n_k/8 (sum T_A + coef sum T_B), coef = alpha g_k (QJL) or
//             ebar_K. Online softmax in base 2 with a wave-uniform running max
//             raised only when a tile max exceeds it by more than 2^8.
//             Values are accumulated one lane per dimension from the
//             dimension-major V tile; a tile's token weights reach the lanes
//             through DPP row broadcasts. One tile per wave is in flight
//             (two with 4 waves).
//   blocks    WAVES = 8 for most launches; 16 where the units leave compute
//             units free (one tile round per wave instead of two), 4 for
//             sequences under 12 tiles; decode_plan picks the shape and the
//             splits.
//   merge     waves merge through LDS; splits of a unit merge through a
//             workspace of (m, l, o) partials written and read with
//             agent-scope atomics: the last split to finish (atomic counter)
//             combines them by log-sum-exp.
//   epilogue  o = Pi^T (o^ / l) (one inverse rotation, Pi still in LDS), plus
//             the V residual estimate alpha S^T s or ebar_V s when V carries
//             sign bits.
// Work items are dealt so that all splits of a unit land on one XCD (blocks
// go to the 8 XCDs round-robin), where Pi stays in that XCD's L2.
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

// A tile's loads in the order they are used: the key planes, then the scalars
// (the score needs n_k and g_k), then the value planes, so that the score's
// wait does not include the value planes.
__device__ __forceinline__ void load_tile(TileRegs& r, const uint8_t* kreg, const uint8_t* vreg,
                                          const uint2* sreg, int64_t gt, int64_t s0, int tt,
                                          int lane) {
  r.k0 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 0, lane));
  r.k1 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 1, lane));
  r.sc = sreg[s0 + (int64_t)tt * kTile + lane];
  r.v0 = *reinterpret_cast<const uint4*>(vreg + tile_half_offset(gt, 0, lane));
  r.v1 = *reinterpret_cast<const uint4*>(vreg + tile_half_offset(gt, 1, lane));
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

// Eight table levels held in (scalar) registers, for a step's appends (their
// quantizer compares against them and their midpoints as scalar operands).
struct Lut8 {
  float c0, c1, c2, c3, c4, c5, c6, c7;
  __device__ __forceinline__ static Lut8 of(const uint64_t (&w)[4]) {
    const float2 a = pair_f2(w[0]), b = pair_f2(w[1]), c = pair_f2(w[2]), d = pair_f2(w[3]);
    return Lut8{a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
  }
};


template <int WAVES, bool VQJL>
__global__ __launch_bounds__(WAVES * 64)
__attribute__((amdgpu_waves_per_eu((WAVES == 8 && !VQJL) ? 6 : 1)))
void decode_kernel(DecodeArgs a, int total_work, int per_xcd) {
  // Wave priority 3 from the start: the block's first steps (its indices and
  // the request of Pi) issue ahead of the tile loops of blocks already
  // running on the SIMD.
  __builtin_amdgcn_s_setprio(3);
  constexpr int NT = WAVES * 64;
  constexpr int TAM = 2048 / NT;           // pair-table entries per thread
  constexpr int TBM = (512 + NT - 1) / NT; // groups of 4 sign-table entries per thread (512 groups)
  constexpr int COLS = kDim / WAVES;       // rows of Pi per thread in the epilogue
  // tiles in flight per wave: with 8 or 16 waves one (more only queue ahead of
  // the Pi copies of blocks that start later on the compute unit)
  constexpr int DEPTH = WAVES >= 8 ? 1 : 2;
  constexpr int MCH = 1024 / NT;           // 16-byte chunks of a 64 x 64 matrix per thread
  constexpr int NB = 2;                    // read batch of the append's row products
  __shared__ __attribute__((aligned(16))) float s_pi[kDim * kDim];   // Pi (Swz16)
  // S (Swz16) in the prologue and a step's append; after the main loop the
  // merge's scratch
  __shared__ __attribute__((aligned(16))) float s_ws[kDim * kDim];
  __shared__ __attribute__((aligned(16))) float s_ta[32 * 64];        // pair table of the score's table term
  __shared__ __attribute__((aligned(16))) float s_tb[8 * 256];        // sign-byte table of the QJL term
  // RoPE(q), q^, u, and the staging vectors x, r of the key and value appends
  __shared__ __attribute__((aligned(16))) float s_vec[7][kDim];
  __shared__ uint32_t s_new[2 + 8 + kDim];                           // the appended token's codes
  __shared__ int s_ready;                                            // appends done
  __shared__ int s_fail;                                             // a step's wait gave up
  __shared__ float s_vtab[16];
  __shared__ float s_wm[WAVES], s_wl[WAVES];
  __shared__ int s_last;
  float* const s_wo = s_ws;                        // [WAVES][64] per-wave o
  float* const s_wsg = s_ws + WAVES * kDim;        // [WAVES][64] per-wave V sign sums
  float* const s_part = s_ws + 2 * WAVES * kDim;   // [WAVES][64] epilogue partial products
  float* const s_oh = s_ws + 3 * WAVES * kDim;     // [64]
  float* const s_sh = s_oh + kDim;                 // [64]
  // The argument fields the prologue needs, read in one batch and met by one
  // wait (used by the asm), so that no later data load waits on one of them.
  const int nsplit = a.nsplit, H = a.H, B = a.B, layer0 = a.layer0, len_add = a.len_add;
  const int f16_in = a.f16_in, rope_positions = a.rope_positions;
  const uint32_t flags = a.flags;
  const float *lut_k = a.lut_k, *lut_v = a.lut_v, *ebar = a.ebar, *pi_base = a.pi, *s_base = a.qjl_s;
  const float* rope_cs = a.rope_cs;
  const void *q_in = a.q, *k_in = a.k_new, *v_in = a.v_new;
  const int32_t* seq_len = a.seq_len;
  const int64_t* seq_slot0 = a.seq_slot0;
  const int32_t* q_pos = a.q_pos;
  asm volatile("" ::"s"(total_work), "s"(per_xcd), "s"(nsplit), "s"(H), "s"(B), "s"(layer0), "s"(len_add),
               "s"(f16_in), "s"(rope_positions), "s"(flags), "s"(lut_k), "s"(lut_v), "s"(ebar), "s"(pi_base),
               "s"(s_base), "s"(rope_cs), "s"(q_in), "s"(k_in), "s"(v_in), "s"(seq_len), "s"(seq_slot0),
               "s"(q_pos));
  const int bid = blockIdx.x;
  const int work = (bid % kXcds) * per_xcd + bid / kXcds;
  if (work >= total_work) return;
  // The unit's indices by multiply-high divisions on the scalar unit (an
  // integer division the compiler would expand on the vector unit).
  const int unit = (int)div_magic(work, a.div_ns);
  const int split = work - unit * nsplit;
  const int uh = (int)div_magic(unit, a.div_h);
  const int h = unit - uh * H;
  const int ub = (int)div_magic(uh, a.div_b);
  const int b = uh - ub * B;
  const int l = layer0 + ub;
  const int lh = l * H + h;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const bool paper = (flags & kQjlPaper) != 0;
  const bool use_s = !paper;               // S enters u = S q^ and the keys' sign bits

  // ---------------------------------------------------------- Pi, S -> LDS
  // Each wave instruction fills 1 KB of LDS; a lane fetches the global chunk
  // that belongs at its position.
  {
    typedef __attribute__((address_space(3))) void* lds_ptr;
    const float* pig = pi_base + (int64_t)lh * kDim * kDim;
#pragma unroll
    for (int j = 0; j < MCH; ++j) {
      const int c0 = (wave + WAVES * j) * 64;
      __builtin_amdgcn_global_load_lds(pig + Swz16::source(c0 + lane) * 4, (lds_ptr)(s_pi + c0 * 4), 16, 0, 0);
    }
    if (use_s) {
#pragma unroll
      for (int j = 0; j < MCH; ++j) {
        const int c0 = (wave + WAVES * j) * 64;
        __builtin_amdgcn_global_load_lds(s_base + Swz16::source(c0 + lane) * 4, (lds_ptr)(s_ws + c0 * 4), 16,
                                         0, 0);
      }
    }
  }

  // ------------------------------------------------------ prologue loads
  // Uniform values through the constant address space (a load from it with a
  // wave-uniform address always takes the scalar path; the scalar cache does
  // not queue behind the vector memory pipeline), as 64-bit pairs: one asm
  // operand each.
  const cfloat* lk = to_const(lut_k) + lh * 8;
  const cfloat* lv = to_const(lut_v) + lh * 8;
  uint64_t kw[4], vw[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    kw[k] = load_pair(lk + 2 * k);
    vw[k] = load_pair(lv + 2 * k);
  }
  const float ebar_raw = *(paper ? to_const(ebar) + lh * 2 : lk);
  const int len = to_const(seq_len)[b];
  const int64_t s0 = to_const(seq_slot0)[b];
  const int qp = to_const(q_pos)[b];
  // Every scalar value is used here, before anything branches on them: the
  // loads are independent, so they are all issued and met by one wait.
  asm volatile("" ::"s"(kw[0]), "s"(kw[1]), "s"(kw[2]), "s"(kw[3]), "s"(vw[0]), "s"(vw[1]), "s"(vw[2]),
               "s"(vw[3]), "s"(ebar_raw), "s"(len), "s"(s0), "s"(qp));
  // The vector the wave works on in the prologue, q (wave 0) or a step's
  // new key (wave 1) or value (wave 2), as raw bits (converted where used,
  // so that no wait follows the load), and the RoPE (cos, sin) of the lane's
  // pair at the position, clamped into the table (checked below): both are
  // requested before the checks.
  const bool f16 = f16_in != 0;
  const bool step = a.append != 0;
  const bool half = (flags & kRopeHalf) != 0;
  const bool has_vec = wave == 0 || (step && wave <= 2);
  const void* vsrc = wave == 0 ? q_in : (wave == 1 ? k_in : v_in);
  uint32_t xraw = 0;
  if (has_vec) {
    const int64_t e = (int64_t)unit * kDim + lane;
    xraw = f16 ? (uint32_t)reinterpret_cast<const unsigned short*>(vsrc)[e] : reinterpret_cast<const uint32_t*>(vsrc)[e];
  }
  float2 cs = make_float2(1.0f, 0.0f);
  if (wave <= 1) {
    const int qpc = min(max(qp, 0), rope_positions - 1);
    cs = reinterpret_cast<const float2*>(rope_cs + (int64_t)qpc * 2 * kPairs)[half ? (lane & 31) : (lane >> 1)];
  }
  // Per lane, the levels the tables are built from: c_K[lane & 7],
  // c_K[lane >> 3] and c_V[lane & 7] (vector loads: a per-lane choice among
  // eight scalar values would take seven selects each).
  const float lev_k_lo = lut_k[lh * 8 + (lane & 7)];
  const float lev_k_hi = lut_k[lh * 8 + (lane >> 3)];
  const float lev_v = lut_v[lh * 8 + (lane & 7)];
  const Lut8 ck = Lut8::of(kw), cvl = Lut8::of(vw);
  const float ebar_k = paper ? ebar_raw : 0.0f;
  const int n = len + len_add;             // tokens attended (the step's new one included)
  // a unit whose sequence range or query position is out of bounds, or
  // whose K or V table is not strictly ascending, is not appended to and
  // gets NaN output. Lanes 0..6 compare their level with the next one (a
  // NaN level fails).
  const float next_k = dpp<0x101>(lev_k_lo);   // row_shl:1: lane i + 1
  const float next_v = dpp<0x101>(lev_v);
  const bool lane_asc = (lane & 7) == 7 || (lev_k_lo < next_k && lev_v < next_v);
  const bool asc = (__builtin_amdgcn_ballot_w64(!lane_asc) & 0xFFull) == 0;
  const bool valid = (n >= 0) & (n <= a.max_len) & (s0 >= 0) & ((s0 & 63) == 0) &
                     (s0 + n <= a.slots) & (qp >= 0) & (qp < rope_positions) & asc;
  if (!valid || n == 0) {
    if (split == 0 && t < kDim) store_out(a, unit, t, valid ? 0.0f : __int_as_float(0x7FC00000));
    __builtin_amdgcn_s_waitcnt(0);         // no copy into LDS outlives the block
    return;
  }
  const int ntiles = (n + 63) >> 6;
  const int tile_begin = split * a.split_tiles;
  if (tile_begin >= ntiles) {
    __builtin_amdgcn_s_waitcnt(0);
    return;
  }
  const int tile_end = min(ntiles, tile_begin + a.split_tiles);
  const int participants = (int)div_magic(ntiles + a.split_tiles - 1, a.div_st);
  // Token n - 1 (a step's new one, appended by the block of its tile) is
  // scored on its own by the last wave of that block; the tile loop covers
  // the other n - 1 tokens.
  const int tnew = (n - 1) >> 6, rnew = (n - 1) & 63;
  const bool own_last = tnew >= tile_begin && tnew < tile_end;
  const bool app = step && own_last;
  const int nm = n - 1;
  const int tile_end_main = min(tile_end, (nm + 63) >> 6);

  const uint8_t* kreg = a.k_codes + (int64_t)lh * a.slots * 32;
  const uint8_t* vreg = a.v_codes + (int64_t)lh * a.slots * 32;
  const uint2* sreg = reinterpret_cast<const uint2*>(a.scalars + (int64_t)lh * a.slots * 4);
  const int64_t tile0 = s0 >> 6;

  // Pi and S have arrived (every wave waits for its own copies, then the
  // barrier).
  if (t == 0) { s_ready = 0; s_fail = 0; }
  __builtin_amdgcn_s_waitcnt(0x0F70);      // vmcnt(0)
  lds_barrier();

  // (Wave priority: the start of the block and the prologue, and the merge
  // and epilogue after the tile loop, are chains that gate a block's tile
  // requests or its end; at priority 3 they issue ahead of the tile loops of
  // the other blocks on the same SIMD (3 blocks per compute unit, up to 6
  // waves per SIMD), which are throughput work and run at 0.)
  // -------------------------------------------------------------- prologue
  // q' = RoPE(q) (wave 0, one element per lane), then q^ = Pi q' and u = S q^
  // by all waves: 8 lanes per row, 8 columns each, summed by DPP.
  if (wave == 0) {
    const float xin = f16 ? half_bits_to_float(xraw) : __uint_as_float(xraw);
    s_vec[0][lane] = rope_wave(xin, cs, half, lane);
  }
  lds_barrier();
  const int prow = t >> 3, pc = t & 7;     // NT = 512: rows 0..63; NT = 256: two passes; NT = 1024: waves 8..15 idle
#pragma unroll
  for (int r0 = 0; r0 < kDim; r0 += NT / 8) {
    const int r = r0 + prow;
    if (NT > 512 && r >= kDim) break;      // (16 waves: waves 8..15 have no row)
    const float4* m4 = reinterpret_cast<const float4*>(s_pi);
    const float4* x4 = reinterpret_cast<const float4*>(s_vec[0]);
    const float4 ma = m4[Swz16::chunk(r, 2 * pc)], mb = m4[Swz16::chunk(r, 2 * pc + 1)];
    const float4 xa = x4[2 * pc], xb = x4[2 * pc + 1];
    float acc = ma.x * xa.x;
    acc = fmaf(ma.y, xa.y, acc); acc = fmaf(ma.z, xa.z, acc); acc = fmaf(ma.w, xa.w, acc);
    acc = fmaf(mb.x, xb.x, acc); acc = fmaf(mb.y, xb.y, acc); acc = fmaf(mb.z, xb.z, acc);
    acc = fmaf(mb.w, xb.w, acc);
    acc += dpp<0xB1>(acc);                 // quad_perm [1,0,3,2]
    acc += dpp<0x4E>(acc);                 // quad_perm [2,3,0,1]
    acc += dpp<0x141>(acc);                // row_half_mirror: the 8 lanes of the row
    if (pc == 0) s_vec[1][r] = acc;
  }
  lds_barrier();
#pragma unroll
  for (int r0 = 0; r0 < kDim; r0 += NT / 8) {
    const int r = r0 + prow;
    if (NT > 512 && r >= kDim) break;
    float acc = s_vec[1][r];
    if (use_s) {
      const float4* m4 = reinterpret_cast<const float4*>(s_ws);
      const float4* x4 = reinterpret_cast<const float4*>(s_vec[1]);
      const float4 ma = m4[Swz16::chunk(r, 2 * pc)], mb = m4[Swz16::chunk(r, 2 * pc + 1)];
      const float4 xa = x4[2 * pc], xb = x4[2 * pc + 1];
      acc = ma.x * xa.x;
      acc = fmaf(ma.y, xa.y, acc); acc = fmaf(ma.z, xa.z, acc); acc = fmaf(ma.w, xa.w, acc);
      acc = fmaf(mb.x, xb.x, acc); acc = fmaf(mb.y, xb.y, acc); acc = fmaf(mb.z, xb.z, acc);
      acc = fmaf(mb.w, xb.w, acc);
      acc += dpp<0xB1>(acc);
      acc += dpp<0x4E>(acc);
      acc += dpp<0x141>(acc);
    }
    if (pc == 0) s_vec[2][r] = acc;
  }
  lds_barrier();

  // Table entries built by this thread (NT threads):
  //   ta (2048 entries): e = t + NT m, pair P = e / 64 = wave + WAVES m, index f = e % 64 = lane
  //   tb (2048 entries in groups of 4): group e = t + NT m of word w = e / 64,
  //      sign bytes 4 (e % 64) .. 4 (e % 64) + 3
  {
    const float ck_lo = lev_k_lo, ck_hi = lev_k_hi;
#pragma unroll
    for (int m = 0; m < TAM; ++m) {
      const float2 qq = reinterpret_cast<const float2*>(s_vec[1])[wave + WAVES * m];
      s_ta[t + NT * m] = fmaf(qq.y, ck_hi, qq.x * ck_lo);
    }
#pragma unroll
    for (int m = 0; m < TBM; ++m) {
      const int e = t + NT * m, k = e & 63, w = wave + WAVES * m;
      if (NT > 512 && e >= 512) break;
      const float4 ulo = reinterpret_cast<const float4*>(s_vec[2])[2 * w];
      const float4 uhi = reinterpret_cast<const float4*>(s_vec[2])[2 * w + 1];
      const float u[8] = {ulo.x, ulo.y, ulo.z, ulo.w, uhi.x, uhi.y, uhi.z, uhi.w};
      float base = 0.0f;               // sign bits 2..7 of the bytes 4k .. 4k+3 are the bits of k
#pragma unroll
      for (int j = 2; j < 8; ++j) base += ((k >> (j - 2)) & 1) ? u[j] : -u[j];
      float4 v;
      v.x = (base - u[0]) - u[1];
      v.y = (base + u[0]) - u[1];
      v.z = (base - u[0]) + u[1];
      v.w = (base + u[0]) + u[1];
      reinterpret_cast<float4*>(s_tb)[e] = v;
    }
    if (t < 16) s_vtab[t] = lev_v;       // c_V[t & 7]
  }
  lds_barrier();

  // ------------------------------------------------------------ step append
  // For a decode step, waves 1 and 2 quantize the new key and value into the
  // cache (with the append kernel's quantizer, on the staged Pi and S) while
  // the other waves start scoring; each raises the count in s_ready when its
  // codes are in s_new. Wave 3 waits for both before it scores the new token
  // after its tiles (bounded: the appends never wait on anything).
  if (app && (wave == 1 || wave == 2)) {
    const bool is_v = wave == 2;
    const int ksign = paper ? 2 : 1;
    const int sign_mode = is_v ? ((flags & kVQjl) ? ksign : 0) : ksign;
    const bool rotate = !is_v || (flags & kVRotate);
    const Lut8& c = is_v ? cvl : ck;
    Levels La;
    La.c0 = c.c0; La.c1 = c.c1; La.c2 = c.c2; La.c3 = c.c3;
    La.c4 = c.c4; La.c5 = c.c5; La.c6 = c.c6; La.c7 = c.c7;
    La.t0 = 0.5f * (La.c0 + La.c1); La.t1 = 0.5f * (La.c1 + La.c2); La.t2 = 0.5f * (La.c2 + La.c3);
    La.t3 = 0.5f * (La.c3 + La.c4); La.t4 = 0.5f * (La.c4 + La.c5); La.t5 = 0.5f * (La.c5 + La.c6);
    La.t6 = 0.5f * (La.c6 + La.c7);
    const float xin = f16 ? half_bits_to_float(xraw) : __uint_as_float(xraw);
    const float xr = is_v ? xin : rope_wave(xin, cs, half, lane);
    const Appended ap = append_wave<Swz16, NB>(
        xr, is_v, rotate, La, s_pi, s_ws, s_vec[is_v ? 5 : 3], s_vec[is_v ? 6 : 4], sign_mode, s0 + (n - 1),
        lh, const_cast<uint8_t*>(a.k_codes), const_cast<uint8_t*>(a.v_codes),
        const_cast<uint16_t*>(a.scalars), a.slots, lane);
    if (!is_v) {
      if ((lane & 7) == 0) s_new[2 + (lane >> 3)] = ap.code;
      if (lane == 0) s_new[0] = ap.scal;
    } else {
      s_new[10 + lane] = ap.code;
      if (lane == 0) s_new[1] = ap.scal;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");   // s_new written (LDS only)
    if (lane == 0) __hip_atomic_fetch_add(&s_ready, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  // Tiles are requested only now (the appending waves' registers hold no
  // tiles through the append).
  TileRegs buf[DEPTH];
  if (tile_end_main > tile_begin) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int tq = min(tile_begin + wave + d * WAVES, tile_end_main - 1);   // (a wave without tiles re-reads one)
      load_tile(buf[d], kreg, vreg, sreg, tile0 + tq, s0, tq, lane);
    }
  }
  // An attend's last token: its key words and scalars (every lane the same
  // address) and, per lane, the value word of its dimension that holds the
  // token's nibble, requested after the first tile. (A copy straight into
  // LDS would make the compiler wait for every load before each tile's first
  // LDS read, which stops it from scoring a tile's keys while its values are
  // still arriving.) Wave 3 scores it: it does not append, and with
  // WAVES = 4 it has no more tiles than any other wave.
  const bool lone = own_last && wave == 3;
  TileRegs last{};
  if (lone && !step) {
    const int64_t gt = tile0 + tnew;
    last.k0 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 0, rnew));
    last.k1 = *reinterpret_cast<const uint4*>(kreg + tile_half_offset(gt, 1, rnew));
    last.sc = sreg[s0 + nm];
    last.v0.x = *reinterpret_cast<const uint32_t*>(vreg + tile_half_offset(gt, rnew >> 5, lane) +
                                                   4 * ((rnew & 31) >> 3));
  }

  __builtin_amdgcn_s_setprio(0);
  // -------------------------------------------------------------- main loop
  float m_run = -INFINITY;
  float l_lane = 0.0f;
  float sg = 0.0f;
  float o0 = 0.0f, o1 = 0.0f, o2 = 0.0f, o3 = 0.0f;
  const float lscale = a.logit_scale2;
  const char* vtab = reinterpret_cast<const char*>(s_vtab);

  for (int tb = tile_begin + wave; tb < tile_end_main; tb += DEPTH * WAVES) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      const int tt = tb + d * WAVES;
      if (tt >= tile_end_main) break;
      const TileRegs& cur = buf[d];
      const int tok = tt * kTile + lane;
      const bool tv = tok < nm;
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

      // ---- online softmax (base 2), lazily rescaled: the tile max is formed
      // only when some lane exceeds the running max by the headroom
      if (__builtin_amdgcn_ballot_w64(lg > m_run + kLazyRescale) != 0) {
        const float tmax = wave_max_uniform(lg);
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
      if (tn < tile_end_main) load_tile(buf[d], kreg, vreg, sreg, tile0 + tn, s0, tn, lane);
    }
  }

  __builtin_amdgcn_s_setprio(3);
  // ------------------------------------------------------------ last token
  // Scored with the tile loop's arithmetic (every lane computes the same
  // logit); its value enters lane d's accumulator through dimension d's code.
  if (lone) {
    // key words 0..7 and scalars of the token, and this lane's nibble
    const uint32_t* tok_k;
    uint2 sc;
    uint32_t nib;
    if (step) {
      // bounded wait for the two appends; if it gives up, the unit's output
      // is marked NaN (s_fail) instead of scoring stale codes
      bool got = false;
      for (int i = 0; i < a.wait_limit; ++i) {
        if (__hip_atomic_load(&s_ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= 2) {
          got = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
      if (!got && lane == 0) s_fail = 1;
      tok_k = s_new + 2;
      sc = make_uint2(s_new[0], s_new[1]);
      nib = s_new[10 + lane] & 15u;
    } else {
      tok_k = nullptr;
      sc = last.sc;
      nib = (last.v0.x >> (4 * (rnew & 7))) & 15u;
    }
    if (step) {
      last.k0 = make_uint4(tok_k[0], tok_k[1], tok_k[2], tok_k[3]);
      last.k1 = make_uint4(tok_k[4], tok_k[5], tok_k[6], tok_k[7]);
    }
    float A = 0.0f, B = 0.0f;
    key_word_score<0>(s_ta, s_tb, last.k0.x, A, B);
    key_word_score<1>(s_ta, s_tb, last.k0.y, A, B);
    key_word_score<2>(s_ta, s_tb, last.k0.z, A, B);
    key_word_score<3>(s_ta, s_tb, last.k0.w, A, B);
    key_word_score<4>(s_ta, s_tb, last.k1.x, A, B);
    key_word_score<5>(s_ta, s_tb, last.k1.y, A, B);
    key_word_score<6>(s_ta, s_tb, last.k1.z, A, B);
    key_word_score<7>(s_ta, s_tb, last.k1.w, A, B);
    const float nk = half_bits_to_float(sc.x), gk = half_bits_to_float(sc.x >> 16);
    const float nv = half_bits_to_float(sc.y), gv = half_bits_to_float(sc.y >> 16);
    const float coef = paper ? ebar_k : kQjlAlpha * gk;
    const float lg = nk * lscale * fmaf(coef, B, A);
    if (lg > m_run + kLazyRescale) {
      const float f = __builtin_amdgcn_exp2f(m_run - lg);
      l_lane *= f;
      sg *= f;
      o0 *= f; o1 *= f; o2 *= f; o3 *= f;
      m_run = lg;
    }
    const float p = __builtin_amdgcn_exp2f(lg - m_run);
    if (lane == 0) l_lane += p;
    const float wv = p * nv * 0.125f;
    o0 = fmaf(wv, s_vtab[nib], o0);
    if (VQJL) {
      const float wg = paper ? wv : wv * gv;
      sg = fmaf(wg, (nib & 8u) ? 1.0f : -1.0f, sg);
    }
  }
  // ------------------------------------------------------ merge the waves
  // (s_wo shares its LDS with S, which a step's key append may still be
  // reading until every wave has come here)
  const float ov = (o0 + o1) + (o2 + o3);
  const float l_wave = wave_sum_uniform(l_lane);
  if (lane == 0) { s_wm[wave] = m_run; s_wl[wave] = l_wave; }
  lds_barrier();
  s_wo[wave * kDim + lane] = ov;
  if (VQJL) s_wsg[wave * kDim + lane] = sg;
  __syncthreads();
  float M = -INFINITY, L = 0.0f, O = 0.0f, SG = 0.0f;
  if (t < kDim) {
#pragma unroll
    for (int w = 0; w < WAVES; ++w) M = fmaxf(M, s_wm[w]);
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float f = __builtin_amdgcn_exp2f(s_wm[w] - M);
      L += s_wl[w] * f;
      O += s_wo[w * kDim + t] * f;
      if (VQJL) SG += s_wsg[w * kDim + t] * f;
    }
    // a failed step wait poisons the split's sum of weights: the merged
    // output of the unit is then NaN
    if (s_fail) L = __int_as_float(0x7FC00000);
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
      // Leave the workspace as it was found, all zero: each lane clears what
      // it read (o and s of every partial at its dimension, and the (m, l)
      // of the partials it loaded), after reading it (same addresses, so in
      // program order).
      for (int p = 0; p < participants; ++p) {
        float* pq = a.partials + ((int64_t)unit * a.nsplit + p) * kPartialFloats;
        pq[4 + lane] = 0.0f;
        if (VQJL) pq[4 + kDim + lane] = 0.0f;
      }
      for (int p0 = 0; p0 < participants; p0 += 64) {
        if (p0 + lane < participants) {
          float* pp = a.partials + ((int64_t)unit * a.nsplit + p0 + lane) * kPartialFloats;
          pp[0] = 0.0f;
          pp[1] = 0.0f;
        }
      }
    }
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
      s_part[cq * kDim + k] = acc;
      lds_barrier();
      if (t < kDim) {
        float y = 0.0f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) y += s_part[w * kDim + t];
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
      acc = fmaf(s_pi[Swz16::chunk(i, k >> 2) * 4 + (k & 3)], s_oh[i], acc);
    }
    s_part[cq * kDim + k] = acc;
    lds_barrier();
    if (t < kDim) {
      float y = 0.0f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) y += s_part[w * kDim + t];
      store_out(a, unit, t, y);
    }
  } else {
    if (t < kDim) store_out(a, unit, t, s_oh[t]);
  }
}

void decode_plan(int units, int max_len, int* waves, int* nsplit, int* split_tiles) {
  const int ntiles = max_len > 0 ? (max_len + 63) / 64 : 1;
  // A unit's tiles are split over several blocks, and a block takes 16 waves
  // rather than 8, only where that shortens the longest block: each wave's
  // tiles are serial round trips (about 1.6 us each at low load), and a split
  // adds a merge through the workspace (about 2 us). The blocks of all
  // splits must fit one pass over the 256 compute units (with 16 waves a
  // block fills a compute unit's wave slots). Costs in 0.1 us; the last
  // token is scored apart from the tiles, so a sequence of 64 k + 1 tokens
  // has k tiles to split.
  constexpr int kRound = 16, kMerge = 20, kBlocks = 256;
  const int main_tiles = max_len > 1 ? (max_len - 1 + 63) / 64 : 1;
  int best = -1, bw = ntiles >= 12 ? 8 : 4, bns = 1;
  for (const int w : {4, 8, 16}) {
    if ((w == 4) != (ntiles < 12)) continue;     // 4 waves for short sequences only
    if (w == 16 && units > kBlocks) continue;
    const int max_ns = (ntiles + w - 1) / w;     // every wave keeps a tile
    for (int c = 1; c <= max_ns; ++c) {
      if (c > 1 && (int64_t)units * c > kBlocks) break;
      const int per = (main_tiles + c - 1) / c;
      const int cost = (per + w - 1) / w * kRound + (c > 1 ? kMerge : 0);
      if (best < 0 || cost < best) { best = cost; bw = w; bns = c; }
    }
  }
  int st = (ntiles + bns - 1) / bns;
  if (st > ntiles) st = ntiles;
  *waves = bw;
  *split_tiles = st;
  *nsplit = (ntiles + st - 1) / st;
}

hipError_t launch_decode(const DecodeArgs& a, int waves, hipStream_t st) {
  const int64_t units = (int64_t)a.nlayers * a.B * a.H;
  const int64_t total = units * a.nsplit;
  const int64_t per_xcd = (total + kXcds - 1) / kXcds;
  const int64_t blocks = per_xcd * kXcds;
  const bool vq = (a.flags & kVQjl) != 0;
  if (waves == 16) {
    if (vq)
      hipLaunchKernelGGL((decode_kernel<16, true>), dim3((unsigned)blocks), dim3(1024), 0, st, a, (int)total, (int)per_xcd);
    else
      hipLaunchKernelGGL((decode_kernel<16, false>), dim3((unsigned)blocks), dim3(1024), 0, st, a, (int)total, (int)per_xcd);
  } else if (waves == 8) {
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
