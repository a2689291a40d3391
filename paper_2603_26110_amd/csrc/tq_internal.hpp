// Host/device argument blocks and launchers shared by the C-ABI translation
// unit and the kernel translation units. Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tq {

struct QuantArgs {
  const void* k;
  const void* v;
  int B, T, H, layer0, nlayers;
  int f16;                 // k, v are fp16 (else fp32)
  uint32_t flags;
  const float* rope_cs;
  int rope_positions;
  const int32_t* pos0;
  const int64_t* slot0;
  const float* pi;
  const float* lut_k;
  const float* lut_v;
  const float* qjl_s;
  uint8_t* k_codes;
  uint8_t* v_codes;
  uint16_t* scalars;
  int64_t slots;
  const int32_t* tokens;   // [B] tokens of each sequence (<= T), or null: all T
};

// Division of a nonnegative n < 2^31 by a fixed d >= 1 as
//   q = (umulhi(n, m) + n) >> s,  s = ceil(log2 d),  m = floor(2^32 (2^s - d) / d) + 1
// (the round-up method with a 33-bit multiplier 2^32 + m; umulhi(n, m) + n
// stays below 2^32 for n < 2^31). With d, m and s kernel arguments the
// division runs on the scalar unit.
struct DivMagic {
  uint32_t m;
  uint32_t s;
};

inline DivMagic make_div_magic(uint32_t d) {
  uint32_t s = 0;
  while ((uint64_t(1) << s) < d) ++s;
  const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << s) - d)) / d + 1;
  return DivMagic{(uint32_t)m, s};
}

__device__ __forceinline__ uint32_t div_magic(int n, DivMagic d) {
  return (__umulhi((uint32_t)n, d.m) + (uint32_t)n) >> d.s;
}

struct DecodeArgs {
  const void* q;
  int B, H, layer0, nlayers;
  int f16_in;              // q is fp16
  int f16_out;             // out is fp16
  uint32_t flags;
  float logit_scale2;      // softmax_scale * log2(e) / 8 (applied to n_k * (A + coef B))
  const float* rope_cs;
  int rope_positions;
  const int32_t* q_pos;
  const int64_t* seq_slot0;
  const int32_t* seq_len;
  int max_len;
  const float* pi;
  const float* lut_k;
  const float* lut_v;
  const float* qjl_s;
  const float* ebar;
  const uint8_t* k_codes;
  const uint8_t* v_codes;
  const uint16_t* scalars;
  int64_t slots;
  void* out;
  float* partials;         // [units][nsplit][kPartialFloats]
  uint32_t* counters;      // [units]
  int nsplit;              // splits per unit
  int split_tiles;         // 64-token tiles per split
  // decode step: the kernel also appends one token per sequence (its key and
  // value [nlayers][B][H][64], position q_pos[b], slot seq_slot0[b] +
  // seq_len[b]); the attention then covers seq_len[b] + len_add tokens
  const void* k_new;
  const void* v_new;
  int append;
  int len_add;
  int wait_limit;          // polls of a decode step's wait for its appends before giving up
  DivMagic div_ns, div_h, div_b, div_st;   // by nsplit, H, B and split_tiles
};

// Default bound of that wait (never reached: the appends wait on nothing).
constexpr int kDefaultWaitLimit = 1 << 22;

constexpr int kPartialFloats = 2 * 64 + 4;   // m, l, pad, pad, o[64], s[64]

struct DequantArgs {
  int B, H, layer0, nlayers;
  uint32_t flags;
  const int64_t* seq_slot0;
  const int32_t* seq_len;
  int max_len;             // token stride of the outputs
  const float* lut_k;
  const float* lut_v;
  const float* qjl_s;
  const float* ebar;
  const uint8_t* k_codes;
  const uint8_t* v_codes;
  const uint16_t* scalars;
  int64_t slots;
  void* k_out;             // fp16 [nlayers][B][H][max_len][64]
  void* v_out;
};

// Launchers (return the HIP status of the launch).
hipError_t launch_rope_table(float* cs, int positions, double base, hipStream_t st);
hipError_t launch_quantize(const QuantArgs& a, hipStream_t st);
void decode_plan(int units, int max_len, int* waves, int* nsplit, int* split_tiles);
hipError_t launch_decode(const DecodeArgs& a, int waves, hipStream_t st);
hipError_t launch_dequantize(const DequantArgs& a, hipStream_t st);
// Initial levels of the table calibration (by value: a host array).
struct LutInit {
  float c[8];
};
hipError_t launch_calibrate_lut(const float* x, int nheads, int ncal, const float* pi, const float* init,
                                int max_iter, double tol, float* lut_out, hipStream_t st);
hipError_t launch_calibrate_ebar(const float* x, int nheads, int ncal, const float* pi, const float* lut,
                                 float* ebar_out, int stride, hipStream_t st);
hipError_t launch_calibrate(const float* x, int nheads, int ncal, float* pi_out,
                            float* sing_out, hipStream_t st);

// Streaming read of `bytes` (a multiple of 16) at `data` by `blocks` blocks
// (tq_probe.hip; a measurement, not part of the method).
hipError_t launch_read_probe(const void* data, int64_t bytes, int blocks, uint32_t* sink, hipStream_t st);

}  // namespace tq
