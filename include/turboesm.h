/*
 * turboesm.h -- C ABI of the TurboESM 3-bit KV-cache quantizer and fused
 * decode attention for MI355X (gfx950).
 *
 * The method (TurboESM, arXiv 2603.26110) stores the key/value cache of a
 * rotary-position-embedding (RoPE) transformer in 3-bit codes:
 *   prefill  (Sec. 3.1, "operational pipeline", steps 1, 3, 4):
 *       k' = R_{theta,p} k           RoPE first (Eq. 1-2)
 *       k^ = Pi k'                    per-head orthogonal rotation (Eq. 4)
 *       3-bit Lloyd-Max codes of k^   separate K and V tables (Sec. 3.3, Eq. 5)
 *       1-bit QJL residual signs      (Sec. 3.4, Eq. 6-7)
 *   decode   (Sec. 3.1 decode steps 1-4, Algorithm 1 of Sec. 4.3):
 *       one pass over the packed cache: dequantize through the tables in
 *       registers, add the QJL score correction, online softmax, accumulate V.
 * Entry points: tq_quantize_pack (prefill and appends) and
 * tq_quantize_pack_ragged (a prefill of sequences of different lengths), tq_decode_attend,
 * tq_decode_step (append + attend in one launch), tq_dequantize (fp16 rows
 * for a dequantize-then-attend path), tq_calibrate_rotation and
 * tq_calibrate_lut (Sec. 3.2-3.3), tq_calibrate_ebar (Sec. 3.4), tq_rope_table
 * and sizing helpers.
 *
 * Every entry point is asynchronous on the HIP stream it is given and never
 * synchronizes. Device pointers are plain device addresses (hipMalloc or
 * torch allocations on the current device). The library allocates no device
 * memory: the caller owns every buffer, including the cache and workspace.
 * Errors detected on the host are reported before anything is launched:
 * the call returns a negative tq_status and tq_last_error() returns a
 * thread-local message. Device code never traps; per-sequence metadata held
 * in device memory is checked by the kernels, which skip what is out of range
 * as documented per entry point. Tables of levels held in device memory
 * (lut_k, lut_v) must be strictly ascending, since the midpoint rule of the
 * quantizer assumes it; the kernels check each (layer, head)'s pair of tables
 * when they load them: a quantize call does not write a (layer, head) whose
 * K or V table is not strictly ascending (or holds a NaN), tq_dequantize skips
 * it, and decode writes NaN to its output (the host-side equivalent of
 * TQ_ERR_LUT_ORDER, which host tables such as tq_calibrate_lut's init get).
 *
 * Fixed layout facts (head_dim must be 64):
 *   - code words: a token-head vector of 64 codes is 32 bytes, eight 32-bit
 *     little-endian words; word w covers dimensions 8w .. 8w+7. idx is the
 *     3-bit LUT index of a dimension, sign its QJL bit.
 *     Key word: idx of dimension 8w+j at bits 3j .. 3j+2 (bits 0-23), sign of
 *       dimension 8w+j at bit 24+j (bits 24-31).
 *     Value nibbles: dimension-major (below); a nibble is idx | (sign << 3),
 *       sign = 0 unless TQ_V_QJL.
 *   - tiles: slots are grouped in tiles of 64; a tile holds 2048 bytes of
 *     k_codes and 2048 bytes of v_codes. Region (l, h) starts at byte
 *     (l*H + h)*slots*32 of each plane; slot s is in tile t = s/64 at r = s%64.
 *     K plane, token-major: the 16-byte half c (words 4c..4c+3, codes
 *       32c..32c+31) of slot s is at byte t*2048 + (c*64 + r)*16.
 *     V plane, dimension-major: for dimension i, the codes of the tile's 64
 *       slots form 32 bytes; half c (slots 32c..32c+31) is at byte
 *       t*2048 + (c*64 + i)*16, and slot r is nibble r%8 of word (r%32)/8.
 *   - scalars: 4 fp16 values per slot at byte (l*H + h)*slots*8 + s*8:
 *         [0] n_k  = ||k^||,  [1] g_k = ||r_k|| (QJL residual norm),
 *         [2] n_v  = ||v^||,  [3] g_v = ||r_v|| (0 unless TQ_V_QJL).
 *   That is 72 bytes per cached token-head (4.5 bits per element).
 */
#ifndef TURBOESM_H
#define TURBOESM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Every entry point below is exported; everything else in the library is
 * hidden (it is built with -fvisibility=hidden). */
#ifndef TQ_API
#define TQ_API __attribute__((visibility("default")))
#endif

/* ---- status codes ------------------------------------------------------ */
typedef int32_t tq_status;
#define TQ_OK             0
#define TQ_ERR_ARG       -1  /* null pointer, bad count or unknown flag      */
#define TQ_ERR_DIM       -2  /* head_dim != 64 or layer range outside [0, L) */
#define TQ_ERR_ALIGN     -3  /* a pointer misses its documented alignment    */
#define TQ_ERR_LUT_ORDER -4  /* a host table is not strictly ascending       */
#define TQ_ERR_CAPACITY  -5  /* slots not a positive multiple of 64, or a
                                workspace smaller than required              */
#define TQ_ERR_HIP       -6  /* a HIP runtime call or kernel launch failed   */

/* ---- element types of k, v, q and out ---------------------------------- */
#define TQ_F32 0
#define TQ_F16 1

/* ---- behaviour flags (tq_params.flags) ----------------------------------
 * TQ_V_ROTATE      V is stored in the rotated basis v^ = Pi v and decode
 *                  applies one inverse rotation Pi^T to the attention
 *                  output. Without it V is quantized unrotated (Sec. 3.3:
 *                  the value table is calibrated on unrotated values).
 * TQ_V_QJL         V also carries QJL sign bits and a residual norm, and
 *                  decode adds the V residual estimate (Algorithm 1 corrects
 *                  both K and V).
 * TQ_QJL_PAPER     residual signs are taken per element, s_i = sign(r_i),
 *                  and decode adds s_i * ebar with the per-head mean absolute
 *                  residual ebar (Sec. 3.4, Eq. 6-7) instead of the projected
 *                  estimator. Requires `ebar`.
 * TQ_ROPE_HALF     RoPE pairs dimensions (m, m+32) instead of (2m, 2m+1).
 * TQ_INPUT_ROTATED quantize inputs are already x^ (fp32): RoPE and Pi are
 *                  skipped. Used to check the codes bit for bit.
 * TQ_OUT_FP32      decode writes fp32 output even when io_dtype is TQ_F16.
 */
#define TQ_V_ROTATE      (1u << 0)
#define TQ_V_QJL         (1u << 1)
#define TQ_QJL_PAPER     (1u << 2)
#define TQ_ROPE_HALF     (1u << 3)
#define TQ_INPUT_ROTATED (1u << 4)
#define TQ_OUT_FP32      (1u << 5)
#define TQ_FLAGS_ALL     0x3Fu

/* Model-level parameters shared by every call on one cache. */
typedef struct tq_params {
  int32_t head_dim;        /* must be 64                                      */
  int32_t num_layers;      /* L: layers of the cache and of pi / lut arrays   */
  int32_t num_heads;       /* H                                               */
  int32_t io_dtype;        /* TQ_F16 or TQ_F32 for k, v, q and out            */
  uint32_t flags;          /* TQ_* flags above                                */
  float softmax_scale;     /* logit = score * softmax_scale; <= 0 means 1/8   */
  const float* rope_cs;    /* device [rope_positions][32][2] (cos, sin) from
                              tq_rope_table; 16-byte aligned                 */
  int32_t rope_positions;  /* rows of rope_cs; positions must be below it     */
} tq_params;

/* The packed cache. Every (layer, head) owns `slots` consecutive slots. */
typedef struct tq_cache {
  void* k_codes;           /* device, L*H*slots*32 bytes, 16-byte aligned     */
  void* v_codes;           /* device, L*H*slots*32 bytes, 16-byte aligned     */
  void* scalars;           /* device, L*H*slots*8 bytes,  8-byte aligned      */
  int64_t slots;           /* slots per (layer, head), positive multiple of 64 */
} tq_cache;

/* Bytes of k_codes + v_codes + scalars for a cache of L x H x slots
 * (72 bytes per slot per head; the memory accounting of Table 4 in Sec. 5.2
 * counts the same 3-bit codes in 4-bit containers plus 1-bit K signs).
 * Returns -1 for negative arguments. */
TQ_API int64_t tq_cache_bytes(int32_t num_layers, int32_t num_heads, int64_t slots);

/* RoPE cos/sin table (Eq. 2). For position p < positions and pair m < 32:
 *   theta_m = base^(-2m/64),  a = p * theta_m  (both in double precision),
 *   cs[(p*32 + m)*2 + 0] = (float)cos(a),  cs[(p*32 + m)*2 + 1] = (float)sin(a).
 * cs: device, positions*64 floats, 16-byte aligned. base > 0 (10000 for ESM-2). */
TQ_API tq_status tq_rope_table(float* cs, int32_t positions, double base, void* stream);

/* Prefill-side quantizer (Sec. 3.1 prefill steps 1, 3, 4; Sec. 3.3; Sec. 3.4;
 * Sec. 4.2). For every layer l in [layer0, layer0+nlayers), sequence b < B,
 * token j < T and head h < H:
 *   k' = RoPE(k, pos0[b] + j)                          (skipped: TQ_INPUT_ROTATED)
 *   k^ = Pi_{l,h} k'          v^ = Pi_{l,h} v (TQ_V_ROTATE) or v
 *   for x^ in {k^, v^} with its table c (lut_k or lut_v), all in binary32:
 *     n  = sqrt(fma-chain sum_i x^_i^2, i ascending);  inv = n > 0 ? 8/n : 0
 *     u_i = x^_i * inv;   t_m = 0.5*(c_m + c_{m+1});   idx_i = #{m : u_i > t_m}
 *     r_i = u_i - c[idx_i];  g = sqrt(fma-chain sum_i r_i^2)
 *     sign_i = !(p_i < 0), p_i = fma-chain sum_k S[i][k] r_k   (K; V with TQ_V_QJL)
 *            = !(r_i < 0)                                       (TQ_QJL_PAPER)
 *     n, g stored as fp16 (round to nearest even, saturated at 65504)
 *   and writes codes and scalars to slot slot0[b] + j of region (l, h).
 * Codes are bit-identical to a sequential binary32 evaluation of the above
 * whenever x^ is the same (TQ_INPUT_ROTATED makes x^ an input).
 *
 *   k, v   device [nlayers][B][T][H][64] of io_dtype (fp32 when
 *          TQ_INPUT_ROTATED); 16-byte aligned. Layer index is relative to layer0.
 *   pos0   device int32 [B]: RoPE position of token 0 of each sequence.
 *   slot0  device int64 [B]: cache slot of token 0 of each sequence.
 *          Tokens whose slot falls outside [0, slots) or whose position
 *          falls outside [0, rope_positions) are not written.
 *   pi     device [L][H][64][64] fp32, row-major, x^ = pi . x (absolute layer).
 *   lut_k, lut_v  device [L][H][8] fp32, strictly ascending (a (layer, head)
 *          whose pair of tables is not is not written).
 *   qjl_s  device [64][64] fp32 Gaussian projection S (ignored with TQ_QJL_PAPER).
 *   ebar   unused by the quantizer (may be NULL).
 */
TQ_API tq_status tq_quantize_pack(const tq_params* params, const tq_cache* cache,
                           const void* k, const void* v,
                           int32_t B, int32_t T, int32_t layer0, int32_t nlayers,
                           const int32_t* pos0, const int64_t* slot0,
                           const float* pi, const float* lut_k, const float* lut_v,
                           const float* qjl_s, const float* ebar, void* stream);

/* tq_quantize_pack for a batch of sequences of different lengths (the same
 * steps, Sec. 3.1 prefill steps 1, 3, 4), in one call: sequence b has
 *   T_b = min(max(seq_tokens[b], 0), T)
 * tokens, j < T_b; rows j >= T_b of its input are padding and no slot is
 * written for them. Every token gets the bytes tq_quantize_pack gives it.
 *   seq_tokens  device int32 [B] (required).
 *   k, v        device [nlayers][B][T][H][64] as for tq_quantize_pack (T is
 *               the longest sequence; padding rows need not be initialized).
 * Other arguments and errors as for tq_quantize_pack; a NULL seq_tokens is
 * TQ_ERR_ARG. */
TQ_API tq_status tq_quantize_pack_ragged(const tq_params* params, const tq_cache* cache,
                                  const void* k, const void* v,
                                  int32_t B, int32_t T, const int32_t* seq_tokens,
                                  int32_t layer0, int32_t nlayers,
                                  const int32_t* pos0, const int64_t* slot0,
                                  const float* pi, const float* lut_k, const float* lut_v,
                                  const float* qjl_s, const float* ebar, void* stream);

/* Fused decode attention over the packed cache (Sec. 3.1 decode steps 1-4;
 * Algorithm 1 of Sec. 4.3; the query is rotated once instead of rotating
 * every key, which Eq. 4 makes identical). For every layer l in
 * [layer0, layer0+nlayers), sequence b and head h, with n = seq_len[b]
 * cached tokens in slots seq_slot0[b] .. seq_slot0[b]+n-1:
 *   q^ = Pi RoPE(q, q_pos[b]);   u = S q^;   alpha = sqrt(pi/2)/64
 *   score_j = (n_k,j/8) * ( sum_i q^_i c_K[idx_ij] + alpha g_k,j sum_i u_i (2 s_ij - 1) )
 *             (TQ_QJL_PAPER: alpha g_k,j -> ebar_K and u -> q^)
 *   w_j = exp(score_j * softmax_scale - max);   o^ = sum_j w_j v~_j / sum_j w_j
 *   v~_j = (n_v,j/8) * ( c_V[idx^V_j] (+ V residual estimate with TQ_V_QJL) )
 *   out = Pi^T o^ (TQ_V_ROTATE) or o^.   n = 0 gives out = 0.
 *
 *   q       device [nlayers][B][H][64] io_dtype, before RoPE; 16-byte aligned.
 *   q_pos   device int32 [B]: RoPE position of the query.
 *   seq_slot0 device int64 [B]: first slot of each sequence, multiple of 64.
 *   seq_len device int32 [B]: cached tokens, 0 <= seq_len <= max_len.
 *           A sequence whose range or query position is invalid gets NaN
 *           output, and so does a (layer, head) whose lut_k or lut_v is not
 *           strictly ascending.
 *   max_len host bound on every seq_len (sizes the split-K grid), >= 0.
 *   out     device [nlayers][B][H][64]: io_dtype, or fp32 with TQ_OUT_FP32.
 *   workspace device, >= tq_decode_workspace_bytes(...) bytes, 16-byte aligned
 *           (NULL when that is 0). When long sequences are split across
 *           blocks it holds the split partials and one counter per unit; it
 *           must be zero-filled before its first use, and every call that
 *           completes leaves all of it zero again (the split that merges
 *           clears the partials it read and the counter), so one zero-filled
 *           workspace serves later calls of any shape.
 *           Calls that share a workspace must be ordered on one stream.
 */
TQ_API tq_status tq_decode_attend(const tq_params* params, const tq_cache* cache,
                           const void* q, int32_t B, int32_t layer0, int32_t nlayers,
                           const int32_t* q_pos, const int64_t* seq_slot0,
                           const int32_t* seq_len, int32_t max_len,
                           const float* pi, const float* lut_k, const float* lut_v,
                           const float* qjl_s, const float* ebar,
                           void* out, void* workspace, size_t workspace_bytes,
                           void* stream);

/* tq_decode_attend for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and the same kernels, without a workspace
 * argument. When the sizes need a split-K workspace
 * (tq_decode_workspace_bytes > 0), the library uses a fixed device array of
 * 262144 bytes that each GPU it runs on holds until the process ends, and
 * first clears its counters with a small kernel on `stream`; sizes that
 * would need more return TQ_ERR_CAPACITY before anything is launched. The
 * call allocates nothing (no hipMalloc, no allocating library call).
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (other streams, other threads) race, so order them on one stream.
 * `stream` must belong to the current device. Arguments and output as
 * tq_decode_attend. */
TQ_API tq_status tq_decode_attend_noalloc(const tq_params* params, const tq_cache* cache,
                                          const void* q, int32_t B, int32_t layer0, int32_t nlayers,
                                          const int32_t* q_pos, const int64_t* seq_slot0,
                                          const int32_t* seq_len, int32_t max_len,
                                          const float* pi, const float* lut_k, const float* lut_v,
                                          const float* qjl_s, const float* ebar, void* out,
                                          void* stream);

/* One decode step (Sec. 3.1 decode steps: quantize-then-attend): for every
 * layer, sequence b and head, first append the new token exactly as
 * tq_quantize_pack with T = 1, pos0 = pos and slot0 = seq_slot0 + seq_len
 * would (same codes), then attend as tq_decode_attend with q_pos = pos and
 * seq_len[b] + 1 cached tokens (same output). It is one kernel: the block of
 * each (layer, sequence, head) quantizes the new key and value with the Pi it
 * reads for the query, then attends, taking the new token's codes from where
 * it wrote them.
 *
 *   q, k, v device [nlayers][B][H][64] io_dtype, before RoPE; 16-byte aligned.
 *           k and v are the new token's key and value.
 *   pos     device int32 [B]: RoPE position of the new token and of the query.
 *   seq_slot0 device int64 [B]: first slot of each sequence, multiple of 64.
 *   seq_len device int32 [B]: tokens cached BEFORE the step; the new token
 *           goes to slot seq_slot0[b] + seq_len[b] and the step attends over
 *           seq_len[b] + 1 tokens. The caller advances its own lengths.
 *           A sequence that would exceed max_len, its slot range or the RoPE
 *           table is not appended and gets NaN output (as does a (layer,
 *           head) whose lut_k or lut_v is not strictly ascending).
 *           The block's wave that scores the new token waits, bounded, for
 *           the block's own waves that append it (they wait on nothing, so
 *           the bound is never reached in practice); if the wait gives
 *           up, that unit's output is NaN (the appended codes are in the
 *           cache). tq_set_step_wait_limit sets the bound.
 *   max_len host bound on every seq_len[b] + 1, >= 1.
 *   pi, lut_k, lut_v, qjl_s, ebar, out: as tq_decode_attend.
 *   workspace as tq_decode_attend, >= tq_decode_workspace_bytes(params, B,
 *           nlayers, max_len) bytes.
 */
TQ_API tq_status tq_decode_step(const tq_params* params, const tq_cache* cache,
                         const void* q, const void* k, const void* v,
                         int32_t B, int32_t layer0, int32_t nlayers,
                         const int32_t* pos, const int64_t* seq_slot0,
                         const int32_t* seq_len, int32_t max_len,
                         const float* pi, const float* lut_k, const float* lut_v,
                         const float* qjl_s, const float* ebar,
                         void* out, void* workspace, size_t workspace_bytes,
                         void* stream);

/* Dequantize the cache into plain fp16 key and value rows: the first step of
 * a "dequantize first, then attend" path, the comparison the paper makes for
 * its fused kernel (Sec. 5.3, Table 6: unpack to full precision, then
 * attention). For every layer, sequence b and head, token j < seq_len[b]:
 *   k~_j = (n_k,j/8) ( c_K[idx_j] + alpha g_k,j S^T (2 s_j - 1) )
 *          (TQ_QJL_PAPER: ebar_K (2 s_j - 1) in place of alpha g_k,j S^T (2 s_j - 1))
 *   v~_j = (n_v,j/8) ( c_V[idx^V_j] (+ the same residual estimate from the V
 *          signs and g_v,j, or ebar_V, with TQ_V_QJL) )
 * in the basis the cache holds (rotated; values unrotated without
 * TQ_V_ROTATE), so that q^ . k~_j is the score of tq_decode_attend and its
 * o^ is the softmax-weighted mean of the v~_j (before Pi^T).
 *
 *   seq_slot0, seq_len  device [B], as tq_decode_attend; a sequence whose
 *           range is invalid (or seq_len > max_len) is skipped, and so is a
 *           (layer, head) whose lut_k or lut_v is not strictly ascending.
 *   max_len host: the token stride of the outputs, >= every seq_len.
 *   lut_k, lut_v, qjl_s, ebar  as tq_decode_attend (qjl_s may be NULL with
 *           TQ_QJL_PAPER; ebar is needed only then).
 *   k_out, v_out device fp16 [nlayers][B][H][max_len][64], 16-byte aligned;
 *           rows j >= seq_len[b] are not written.
 * params->rope_cs is not used.
 */
TQ_API tq_status tq_dequantize(const tq_params* params, const tq_cache* cache, int32_t B,
                               int32_t layer0, int32_t nlayers, const int64_t* seq_slot0,
                               const int32_t* seq_len, int32_t max_len,
                               const float* lut_k, const float* lut_v, const float* qjl_s,
                               const float* ebar, void* k_out, void* v_out, void* stream);

/* Workspace bytes tq_decode_attend and tq_decode_step need for these sizes:
 * 0 unless sequences are split across blocks (few units, long max_len), and
 * 0 for empty or invalid sizes. */
TQ_API size_t tq_decode_workspace_bytes(const tq_params* params, int32_t B,
                                 int32_t nlayers, int32_t max_len);

/* Head-wise rotation calibration (Sec. 3.2): for each head, X is the
 * [ncal][64] matrix of post-RoPE keys, X = U Sigma V^T, Pi = V^T.
 * Computed as the eigen-decomposition of the fp64 Gram matrix X^T X (cyclic
 * Jacobi, fp64), rows ordered by descending singular value, each row's
 * entry of largest magnitude made positive (lowest index on ties).
 *   x        device [nheads][ncal][64] fp32 (not centered).
 *   pi_out   device [nheads][64][64] fp32.
 *   sing_out device [nheads][64] fp32 singular values, or NULL.
 */
TQ_API tq_status tq_calibrate_rotation(const float* x, int32_t nheads, int32_t ncal,
                                float* pi_out, float* sing_out, void* stream);

/* Calibrated 8-level table per head (Sec. 3.3: calibrated tables, separate
 * for K and V; Eq. 5 fitted to data): the 1-D Lloyd iteration (k-means) on
 * every normalized coordinate u = 8 x^ / ||x^|| of the head's calibration
 * vectors, x^ = Pi x in fp64 (x^ = x when pi is NULL; a zero vector gives
 * zeros, as in the quantizer). Each iteration assigns u to level
 * #{m : u > (c_m + c_{m+1})/2}, replaces every level by the mean of its cell
 * (fp64 sums; an empty cell keeps its level), sorts the levels and stops
 * once the largest level change is below tol, or after max_iter iterations.
 *   x        device [nheads][ncal][64] fp32: post-RoPE keys for the K table,
 *            values for the V table.
 *   pi       device [nheads][64][64] fp32 rotations, or NULL.
 *   init     HOST [8] fp32 starting levels, strictly ascending (for example
 *            the Gaussian Lloyd-Max table).
 *   max_iter >= 1;  tol >= 0 (finite).
 *   lut_out  device [nheads][8] fp32, ascending.
 */
TQ_API tq_status tq_calibrate_lut(const float* x, int32_t nheads, int32_t ncal, const float* pi,
                           const float* init, int32_t max_iter, double tol, float* lut_out,
                           void* stream);

/* Per-head mean absolute residual ebar of the per-element residual form
 * (TQ_QJL_PAPER; Sec. 3.4, Eq. 7: the correction adds sign(r_i) ebar): over
 * every normalized coordinate u = 8 x^ / ||x^|| of the head's calibration
 * vectors (x^ = Pi x in fp64, x^ = x when pi is NULL; a zero vector gives
 * zeros, as in the quantizer),
 *   ebar = mean over vectors and coordinates of |u - c[idx(u)]|,
 *   idx(u) = #{m : u > (c_m + c_{m+1})/2}   (fp64 midpoints),
 * with the head's table c, summed in fp64. Call it once with post-RoPE keys
 * and lut_k for ebar_K and once with values and lut_v for ebar_V.
 *   x        device [nheads][ncal][64] fp32.
 *   pi       device [nheads][64][64] fp32 rotations, or NULL.
 *   lut      device [nheads][8] fp32, strictly ascending (a head whose table
 *            is not gets NaN).
 *   ebar_out device fp32: head h's value goes to element h * stride (stride 2
 *            with ebar_out = ebar or ebar + 1 fills the K or V column of the
 *            [L][H][2] array the decode entry points take).
 *   stride   >= 1. */
TQ_API tq_status tq_calibrate_ebar(const float* x, int32_t nheads, int32_t ncal, const float* pi,
                                   const float* lut, float* ebar_out, int32_t stride, void* stream);

/* Bound, in polls of about 64 clock cycles each, of the wait inside a
 * tq_decode_step block for the two waves that append the new token (default
 * 4194304, restored by a negative limit). For tests of the failure path: a
 * limit of 0 makes every wait give up at once, so every unit of a step whose
 * new token is scored gets NaN output. Process-wide; it applies to launches
 * made after the call. Returns the previous limit. */
TQ_API int32_t tq_set_step_wait_limit(int32_t limit);

/* Measurement helper, not part of the method: a plain streaming read of
 * `bytes` bytes at `data` (device, 16-byte aligned, bytes a multiple of 16)
 * by `blocks` blocks of 256 threads (1..65536), each thread keeping four
 * 16-byte loads in flight. Nothing is written except, in the never-taken case
 * that a block's folded data equals a fixed constant, one word of `sink`
 * (device, >= blocks words). Timing it over a buffer as large as a decode
 * step's bytes gives the read rate the GPU reaches for a transfer of that
 * size, next to which a decode kernel's rate is judged. */
TQ_API tq_status tq_read_probe(const void* data, int64_t bytes, int32_t blocks, uint32_t* sink, void* stream);

/* Message of the last failing call on this thread ("" if none). */
TQ_API const char* tq_last_error(void);

/* Library version string. */
TQ_API const char* tq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TURBOESM_H */
