// C ABI of libturboesm: host-side validation and kernel launches. Every
// entry point validates its arguments before launching anything, returns a
// negative tq_status on failure and records a thread-local message.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/turboesm.h"
#include "tq_internal.hpp"

namespace {

thread_local char g_err[512] = "";
std::atomic<int> g_wait_limit{tq::kDefaultWaitLimit};

tq_status fail(tq_status code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

tq_status ok() {
  g_err[0] = '\0';
  return TQ_OK;
}

bool aligned(const void* p, size_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

tq_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(TQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

tq_status check_params(const tq_params* p, bool need_rope) {
  if (!p) return fail(TQ_ERR_ARG, "params is NULL");
  if (p->head_dim != 64) return fail(TQ_ERR_DIM, "head_dim must be 64 (got %d)", p->head_dim);
  if (p->num_layers <= 0 || p->num_heads <= 0)
    return fail(TQ_ERR_ARG, "num_layers and num_heads must be positive");
  if (p->io_dtype != TQ_F16 && p->io_dtype != TQ_F32)
    return fail(TQ_ERR_ARG, "io_dtype must be TQ_F16 or TQ_F32");
  if (p->flags & ~TQ_FLAGS_ALL) return fail(TQ_ERR_ARG, "unknown flag bits 0x%x", p->flags & ~TQ_FLAGS_ALL);
  if (need_rope) {
    if (!p->rope_cs) return fail(TQ_ERR_ARG, "rope_cs is NULL");
    if (!aligned(p->rope_cs, 16)) return fail(TQ_ERR_ALIGN, "rope_cs must be 16-byte aligned");
    if (p->rope_positions <= 0) return fail(TQ_ERR_ARG, "rope_positions must be positive");
  }
  return ok();
}

// ---------------------------------------------------------------- scratch
// The split-K workspace of tq_decode_attend_noalloc: a fixed device array.
// Every GPU the library runs on holds its own copy until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: host
// code reaches the array only through the device address that
// hipGetSymbolAddress returns for the current device, kept per device.
constexpr size_t kScratchBytes = 256 * 1024;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Clears n 32-bit words (a kernel rather than hipMemsetAsync, so that the
// call can be captured into a HIP graph).
__global__ void zero_words_kernel(uint32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

tq_status check_cache(const tq_cache* c) {
  if (!c) return fail(TQ_ERR_ARG, "cache is NULL");
  if (!c->k_codes || !c->v_codes || !c->scalars) return fail(TQ_ERR_ARG, "cache buffer is NULL");
  if (!aligned(c->k_codes, 16) || !aligned(c->v_codes, 16))
    return fail(TQ_ERR_ALIGN, "cache code planes must be 16-byte aligned");
  if (!aligned(c->scalars, 8)) return fail(TQ_ERR_ALIGN, "cache scalars must be 8-byte aligned");
  if (c->slots <= 0 || c->slots % 64 != 0)
    return fail(TQ_ERR_CAPACITY, "slots must be a positive multiple of 64 (got %lld)", (long long)c->slots);
  return ok();
}

}  // namespace

extern "C" {

const char* tq_last_error(void) { return g_err; }

int32_t tq_set_step_wait_limit(int32_t limit) {
  if (limit < 0) limit = tq::kDefaultWaitLimit;
  return g_wait_limit.exchange(limit, std::memory_order_relaxed);
}

const char* tq_version(void) { return "turboesm-gfx950 0.1.0"; }

tq_status tq_read_probe(const void* data, int64_t bytes, int32_t blocks, uint32_t* sink, void* stream) {
  if (bytes == 0) return ok();
  if (!data || !sink) return fail(TQ_ERR_ARG, "tq_read_probe: data and sink must not be NULL");
  if (bytes < 0 || bytes % 16 != 0) return fail(TQ_ERR_ARG, "tq_read_probe: bytes must be a multiple of 16");
  if (!aligned(data, 16) || !aligned(sink, 4)) return fail(TQ_ERR_ALIGN, "tq_read_probe: data must be 16-byte aligned");
  if (blocks < 1 || blocks > 65536) return fail(TQ_ERR_ARG, "tq_read_probe: blocks must be in [1, 65536]");
  return hip_status(tq::launch_read_probe(data, bytes, blocks, sink, (hipStream_t)stream), "tq_read_probe launch");
}

int64_t tq_cache_bytes(int32_t num_layers, int32_t num_heads, int64_t slots) {
  if (num_layers < 0 || num_heads < 0 || slots < 0) return -1;
  return (int64_t)num_layers * num_heads * slots * 72;
}

tq_status tq_rope_table(float* cs, int32_t positions, double base, void* stream) {
  if (!cs) return fail(TQ_ERR_ARG, "cs is NULL");
  if (!aligned(cs, 16)) return fail(TQ_ERR_ALIGN, "cs must be 16-byte aligned");
  if (positions <= 0) return fail(TQ_ERR_ARG, "positions must be positive");
  if (!(base > 0.0) || !std::isfinite(base)) return fail(TQ_ERR_ARG, "base must be positive and finite");
  return hip_status(tq::launch_rope_table(cs, positions, base, (hipStream_t)stream), "tq_rope_table launch");
}

}  // extern "C"

namespace {

// Shared by tq_quantize_pack and tq_quantize_pack_ragged (seq_tokens
// non-NULL: sequence b has its own token count).
tq_status quantize_common(const tq_params* params, const tq_cache* cache, const void* k, const void* v,
                          int32_t B, int32_t T, const int32_t* seq_tokens, int32_t layer0, int32_t nlayers,
                          const int32_t* pos0, const int64_t* slot0, const float* pi, const float* lut_k,
                          const float* lut_v, const float* qjl_s, void* stream) {
  const bool rotated = params && (params->flags & TQ_INPUT_ROTATED);
  tq_status s = check_params(params, !rotated);
  if (s != TQ_OK) return s;
  if ((s = check_cache(cache)) != TQ_OK) return s;
  if (B < 0 || T < 0 || nlayers < 0) return fail(TQ_ERR_ARG, "B, T and nlayers must be >= 0");
  if (layer0 < 0 || layer0 + nlayers > params->num_layers)
    return fail(TQ_ERR_DIM, "layers [%d, %d) outside [0, %d)", layer0, layer0 + nlayers, params->num_layers);
  if ((int64_t)B * T * nlayers == 0) return ok();
  if (!k || !v || !pos0 || !slot0 || !pi || !lut_k || !lut_v || !qjl_s)
    return fail(TQ_ERR_ARG, "a required pointer is NULL");
  if (!aligned(k, 16) || !aligned(v, 16)) return fail(TQ_ERR_ALIGN, "k and v must be 16-byte aligned");
  if (!aligned(pi, 16) || !aligned(qjl_s, 16)) return fail(TQ_ERR_ALIGN, "pi and qjl_s must be 16-byte aligned");
  if ((int64_t)nlayers * B * T * params->num_heads >= ((int64_t)1 << 40))
    return fail(TQ_ERR_ARG, "too many token-heads");
  if ((int64_t)B * params->num_heads > 65535 || nlayers > 65535)
    return fail(TQ_ERR_ARG, "B*H and nlayers must be <= 65535");
  if (T < 64 && (int64_t)nlayers * B * T * params->num_heads >= ((int64_t)1 << 31))
    return fail(TQ_ERR_ARG, "too many token-heads for one call");
  tq::QuantArgs a{};
  a.k = k; a.v = v;
  a.B = B; a.T = T; a.H = params->num_heads; a.layer0 = layer0; a.nlayers = nlayers;
  a.f16 = params->io_dtype == TQ_F16;
  a.flags = params->flags;
  a.rope_cs = params->rope_cs; a.rope_positions = params->rope_positions;
  a.pos0 = pos0; a.slot0 = slot0; a.pi = pi; a.lut_k = lut_k; a.lut_v = lut_v; a.qjl_s = qjl_s;
  a.k_codes = (uint8_t*)cache->k_codes; a.v_codes = (uint8_t*)cache->v_codes;
  a.scalars = (uint16_t*)cache->scalars; a.slots = cache->slots;
  a.tokens = seq_tokens;
  return hip_status(tq::launch_quantize(a, (hipStream_t)stream),
                    seq_tokens ? "tq_quantize_pack_ragged launch" : "tq_quantize_pack launch");
}

}  // namespace

extern "C" {

tq_status tq_quantize_pack(const tq_params* params, const tq_cache* cache, const void* k,
                           const void* v, int32_t B, int32_t T, int32_t layer0, int32_t nlayers,
                           const int32_t* pos0, const int64_t* slot0, const float* pi,
                           const float* lut_k, const float* lut_v, const float* qjl_s,
                           const float* ebar, void* stream) {
  (void)ebar;
  return quantize_common(params, cache, k, v, B, T, nullptr, layer0, nlayers, pos0, slot0, pi, lut_k, lut_v,
                         qjl_s, stream);
}

tq_status tq_quantize_pack_ragged(const tq_params* params, const tq_cache* cache, const void* k,
                                  const void* v, int32_t B, int32_t T, const int32_t* seq_tokens,
                                  int32_t layer0, int32_t nlayers, const int32_t* pos0,
                                  const int64_t* slot0, const float* pi, const float* lut_k,
                                  const float* lut_v, const float* qjl_s, const float* ebar, void* stream) {
  (void)ebar;
  if (!seq_tokens && (int64_t)B * T * nlayers != 0) return fail(TQ_ERR_ARG, "seq_tokens is NULL");
  return quantize_common(params, cache, k, v, B, T, seq_tokens, layer0, nlayers, pos0, slot0, pi, lut_k,
                         lut_v, qjl_s, stream);
}

size_t tq_decode_workspace_bytes(const tq_params* params, int32_t B, int32_t nlayers, int32_t max_len) {
  if (!params || params->num_heads <= 0 || B <= 0 || nlayers <= 0 || max_len < 0) return 0;
  const int64_t units = (int64_t)nlayers * B * params->num_heads;
  int waves, nsplit, split_tiles;
  tq::decode_plan((int)std::min<int64_t>(units, 1 << 30), max_len, &waves, &nsplit, &split_tiles);
  size_t bytes = 0;
  if (nsplit > 1) {
    bytes += align256((size_t)units * nsplit * tq::kPartialFloats * sizeof(float));
    bytes += (size_t)units * sizeof(uint32_t);
  }
  return bytes;
}

}  // extern "C"

namespace {

// Shared by tq_decode_attend and tq_decode_step (k, v non-NULL: append first).
tq_status decode_common(const tq_params* params, const tq_cache* cache, const void* q, const void* k,
                        const void* v, int32_t B, int32_t layer0, int32_t nlayers, const int32_t* q_pos,
                        const int64_t* seq_slot0, const int32_t* seq_len, int32_t max_len,
                        const float* pi, const float* lut_k, const float* lut_v, const float* qjl_s,
                        const float* ebar, void* out, void* workspace, size_t workspace_bytes,
                        void* stream, bool step, bool clear_counters = false) {
  tq_status s = check_params(params, true);
  if (s != TQ_OK) return s;
  if ((s = check_cache(cache)) != TQ_OK) return s;
  if (params->flags & TQ_INPUT_ROTATED) return fail(TQ_ERR_ARG, "TQ_INPUT_ROTATED applies to tq_quantize_pack only");
  if (B < 0 || nlayers < 0 || max_len < 0) return fail(TQ_ERR_ARG, "B, nlayers and max_len must be >= 0");
  if (step && max_len < 1) return fail(TQ_ERR_ARG, "a decode step attends to at least one token (max_len >= 1)");
  if (layer0 < 0 || layer0 + nlayers > params->num_layers)
    return fail(TQ_ERR_DIM, "layers [%d, %d) outside [0, %d)", layer0, layer0 + nlayers, params->num_layers);
  if ((int64_t)B * nlayers == 0) return ok();
  if (!q || !q_pos || !seq_slot0 || !seq_len || !pi || !lut_k || !lut_v || !qjl_s || !out)
    return fail(TQ_ERR_ARG, "a required pointer is NULL");
  if (step && (!k || !v)) return fail(TQ_ERR_ARG, "k and v must not be NULL");
  if ((params->flags & TQ_QJL_PAPER) && !ebar) return fail(TQ_ERR_ARG, "TQ_QJL_PAPER needs ebar");
  if (!aligned(q, 16) || !aligned(out, 16)) return fail(TQ_ERR_ALIGN, "q and out must be 16-byte aligned");
  if (step && (!aligned(k, 16) || !aligned(v, 16))) return fail(TQ_ERR_ALIGN, "k and v must be 16-byte aligned");
  if (!aligned(pi, 16) || !aligned(qjl_s, 16)) return fail(TQ_ERR_ALIGN, "pi and qjl_s must be 16-byte aligned");
  if ((int64_t)max_len > cache->slots) return fail(TQ_ERR_CAPACITY, "max_len exceeds the cache slots");
  const int64_t units = (int64_t)nlayers * B * params->num_heads;
  if (units >= ((int64_t)1 << 31)) return fail(TQ_ERR_ARG, "too many (layer, sequence, head) units");
  int waves, nsplit, split_tiles;
  tq::decode_plan((int)units, max_len, &waves, &nsplit, &split_tiles);
  const size_t need = tq_decode_workspace_bytes(params, B, nlayers, max_len);
  if (need > 0) {
    if (!workspace) return fail(TQ_ERR_CAPACITY, "workspace of %zu bytes required", need);
    if (workspace_bytes < need)
      return fail(TQ_ERR_CAPACITY, "workspace too small: %zu < %zu bytes", workspace_bytes, need);
    if (!aligned(workspace, 16)) return fail(TQ_ERR_ALIGN, "workspace must be 16-byte aligned");
  }
  if (units * nsplit > ((int64_t)1 << 31) - 8) return fail(TQ_ERR_ARG, "grid too large");
  const float scale = params->softmax_scale > 0.0f ? params->softmax_scale : 0.125f;
  tq::DecodeArgs a{};
  a.q = q; a.B = B; a.H = params->num_heads; a.layer0 = layer0; a.nlayers = nlayers;
  a.f16_in = params->io_dtype == TQ_F16;
  a.f16_out = (params->io_dtype == TQ_F16) && !(params->flags & TQ_OUT_FP32);
  a.flags = params->flags;
  a.logit_scale2 = (float)((double)scale * 1.4426950408889634 / 8.0);
  a.rope_cs = params->rope_cs; a.rope_positions = params->rope_positions;
  a.q_pos = q_pos; a.seq_slot0 = seq_slot0; a.seq_len = seq_len; a.max_len = max_len;
  a.pi = pi; a.lut_k = lut_k; a.lut_v = lut_v; a.qjl_s = qjl_s; a.ebar = ebar;
  a.k_codes = (const uint8_t*)cache->k_codes; a.v_codes = (const uint8_t*)cache->v_codes;
  a.scalars = (const uint16_t*)cache->scalars; a.slots = cache->slots;
  a.out = out;
  a.nsplit = nsplit; a.split_tiles = split_tiles;
  a.k_new = k; a.v_new = v; a.append = step ? 1 : 0; a.len_add = step ? 1 : 0;
  a.wait_limit = g_wait_limit.load(std::memory_order_relaxed);
  a.div_ns = tq::make_div_magic((uint32_t)nsplit);
  a.div_h = tq::make_div_magic((uint32_t)a.H);
  a.div_b = tq::make_div_magic((uint32_t)B);
  a.div_st = tq::make_div_magic((uint32_t)split_tiles);
  char* ws = (char*)workspace;
  if (nsplit > 1) {
    a.partials = (float*)ws;
    ws += align256((size_t)units * nsplit * tq::kPartialFloats * sizeof(float));
    a.counters = (uint32_t*)ws;
    if (clear_counters) {
      const int64_t n = units;
      const int threads = 256;
      const int blocks = (int)std::min<int64_t>((n + threads - 1) / threads, 1024);
      hipLaunchKernelGGL(zero_words_kernel, dim3(blocks), dim3(threads), 0, (hipStream_t)stream, a.counters, n);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return fail(TQ_ERR_HIP, "counter clear launch: %s", hipGetErrorString(e));
    }
  }
  return hip_status(tq::launch_decode(a, waves, (hipStream_t)stream),
                    step ? "tq_decode_step launch" : "tq_decode_attend launch");
}

}  // namespace

extern "C" {

tq_status tq_decode_attend(const tq_params* params, const tq_cache* cache, const void* q, int32_t B,
                           int32_t layer0, int32_t nlayers, const int32_t* q_pos,
                           const int64_t* seq_slot0, const int32_t* seq_len, int32_t max_len,
                           const float* pi, const float* lut_k, const float* lut_v,
                           const float* qjl_s, const float* ebar, void* out, void* workspace,
                           size_t workspace_bytes, void* stream) {
  return decode_common(params, cache, q, nullptr, nullptr, B, layer0, nlayers, q_pos, seq_slot0, seq_len,
                       max_len, pi, lut_k, lut_v, qjl_s, ebar, out, workspace, workspace_bytes, stream,
                       false);
}

tq_status tq_decode_attend_noalloc(const tq_params* params, const tq_cache* cache, const void* q, int32_t B,
                                   int32_t layer0, int32_t nlayers, const int32_t* q_pos,
                                   const int64_t* seq_slot0, const int32_t* seq_len, int32_t max_len,
                                   const float* pi, const float* lut_k, const float* lut_v,
                                   const float* qjl_s, const float* ebar, void* out, void* stream) {
  const size_t need = tq_decode_workspace_bytes(params, B, nlayers, max_len);
  void* ws = nullptr;
  if (need > 0) {
    if (need > kScratchBytes)
      return fail(TQ_ERR_CAPACITY, "tq_decode_attend_noalloc: these sizes need %zu bytes of split-K workspace, "
                  "more than its fixed %zu (use tq_decode_attend with a workspace)", need, kScratchBytes);
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(TQ_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return fail(TQ_ERR_HIP, "device index %d out of range", dev);
    {
      std::lock_guard<std::mutex> lock(g_scratch_mu);
      if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
          return fail(TQ_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch_dev[dev] = p;
      }
      ws = g_scratch_dev[dev];
    }
  }
  return decode_common(params, cache, q, nullptr, nullptr, B, layer0, nlayers, q_pos, seq_slot0, seq_len,
                       max_len, pi, lut_k, lut_v, qjl_s, ebar, out, ws, need > 0 ? kScratchBytes : 0, stream,
                       false, true);
}

tq_status tq_decode_step(const tq_params* params, const tq_cache* cache, const void* q, const void* k,
                         const void* v, int32_t B, int32_t layer0, int32_t nlayers, const int32_t* pos,
                         const int64_t* seq_slot0, const int32_t* seq_len, int32_t max_len,
                         const float* pi, const float* lut_k, const float* lut_v, const float* qjl_s,
                         const float* ebar, void* out, void* workspace, size_t workspace_bytes,
                         void* stream) {
  return decode_common(params, cache, q, k, v, B, layer0, nlayers, pos, seq_slot0, seq_len, max_len, pi,
                       lut_k, lut_v, qjl_s, ebar, out, workspace, workspace_bytes, stream, true);
}

tq_status tq_dequantize(const tq_params* params, const tq_cache* cache, int32_t B, int32_t layer0,
                        int32_t nlayers, const int64_t* seq_slot0, const int32_t* seq_len, int32_t max_len,
                        const float* lut_k, const float* lut_v, const float* qjl_s, const float* ebar,
                        void* k_out, void* v_out, void* stream) {
  tq_status s = check_params(params, false);
  if (s != TQ_OK) return s;
  if ((s = check_cache(cache)) != TQ_OK) return s;
  if (params->flags & TQ_INPUT_ROTATED) return fail(TQ_ERR_ARG, "TQ_INPUT_ROTATED applies to tq_quantize_pack only");
  if (B < 0 || nlayers < 0 || max_len < 0) return fail(TQ_ERR_ARG, "B, nlayers and max_len must be >= 0");
  if (layer0 < 0 || layer0 + nlayers > params->num_layers)
    return fail(TQ_ERR_DIM, "layers [%d, %d) outside [0, %d)", layer0, layer0 + nlayers, params->num_layers);
  if ((int64_t)B * nlayers == 0 || max_len == 0) return ok();
  const bool paper = (params->flags & TQ_QJL_PAPER) != 0;
  if (!seq_slot0 || !seq_len || !lut_k || !lut_v || !k_out || !v_out || (!paper && !qjl_s))
    return fail(TQ_ERR_ARG, "a required pointer is NULL");
  if (paper && !ebar) return fail(TQ_ERR_ARG, "TQ_QJL_PAPER needs ebar");
  if (!aligned(k_out, 16) || !aligned(v_out, 16)) return fail(TQ_ERR_ALIGN, "k_out and v_out must be 16-byte aligned");
  if ((int64_t)max_len > cache->slots) return fail(TQ_ERR_CAPACITY, "max_len exceeds the cache slots");
  if ((int64_t)B * params->num_heads > 65535 || nlayers > 65535)
    return fail(TQ_ERR_ARG, "B * num_heads and nlayers must be at most 65535");
  tq::DequantArgs a{};
  a.B = B; a.H = params->num_heads; a.layer0 = layer0; a.nlayers = nlayers; a.flags = params->flags;
  a.seq_slot0 = seq_slot0; a.seq_len = seq_len; a.max_len = max_len;
  a.lut_k = lut_k; a.lut_v = lut_v; a.qjl_s = qjl_s; a.ebar = ebar;
  a.k_codes = (const uint8_t*)cache->k_codes; a.v_codes = (const uint8_t*)cache->v_codes;
  a.scalars = (const uint16_t*)cache->scalars; a.slots = cache->slots;
  a.k_out = k_out; a.v_out = v_out;
  return hip_status(tq::launch_dequantize(a, (hipStream_t)stream), "tq_dequantize launch");
}

tq_status tq_calibrate_rotation(const float* x, int32_t nheads, int32_t ncal, float* pi_out,
                                float* sing_out, void* stream) {
  if (nheads < 0 || ncal < 0) return fail(TQ_ERR_ARG, "nheads and ncal must be >= 0");
  if (nheads == 0) return ok();
  if (!x || !pi_out) return fail(TQ_ERR_ARG, "x and pi_out must not be NULL");
  if (ncal == 0) return fail(TQ_ERR_ARG, "ncal must be positive");
  if (nheads > 65535 * 1024) return fail(TQ_ERR_ARG, "too many heads");
  return hip_status(tq::launch_calibrate(x, nheads, ncal, pi_out, sing_out, (hipStream_t)stream),
                    "tq_calibrate_rotation launch");
}

tq_status tq_calibrate_lut(const float* x, int32_t nheads, int32_t ncal, const float* pi,
                           const float* init, int32_t max_iter, double tol, float* lut_out,
                           void* stream) {
  if (nheads < 0 || ncal < 0) return fail(TQ_ERR_ARG, "nheads and ncal must be >= 0");
  if (!init) return fail(TQ_ERR_ARG, "init must not be NULL");
  for (int m = 0; m < 8; ++m)
    if (!std::isfinite(init[m])) return fail(TQ_ERR_ARG, "init levels must be finite");
  for (int m = 0; m < 7; ++m)
    if (!(init[m] < init[m + 1])) return fail(TQ_ERR_LUT_ORDER, "init levels must be strictly ascending");
  if (max_iter < 1) return fail(TQ_ERR_ARG, "max_iter must be >= 1");
  if (!(tol >= 0.0) || !std::isfinite(tol)) return fail(TQ_ERR_ARG, "tol must be finite and >= 0");
  if (nheads == 0) return ok();
  if (!x || !lut_out) return fail(TQ_ERR_ARG, "x and lut_out must not be NULL");
  if (ncal == 0) return fail(TQ_ERR_ARG, "ncal must be positive");
  if (nheads > 65535 * 1024) return fail(TQ_ERR_ARG, "too many heads");
  return hip_status(tq::launch_calibrate_lut(x, nheads, ncal, pi, init, max_iter, tol, lut_out,
                                             (hipStream_t)stream),
                    "tq_calibrate_lut launch");
}

tq_status tq_calibrate_ebar(const float* x, int32_t nheads, int32_t ncal, const float* pi, const float* lut,
                            float* ebar_out, int32_t stride, void* stream) {
  if (nheads < 0 || ncal < 0) return fail(TQ_ERR_ARG, "nheads and ncal must be >= 0");
  if (stride < 1) return fail(TQ_ERR_ARG, "stride must be >= 1");
  if (nheads == 0) return ok();
  if (!x || !lut || !ebar_out) return fail(TQ_ERR_ARG, "x, lut and ebar_out must not be NULL");
  if (ncal == 0) return fail(TQ_ERR_ARG, "ncal must be positive");
  if (nheads > 65535 * 1024) return fail(TQ_ERR_ARG, "too many heads");
  return hip_status(tq::launch_calibrate_ebar(x, nheads, ncal, pi, lut, ebar_out, stride, (hipStream_t)stream),
                    "tq_calibrate_ebar launch");
}

}  // extern "C"
