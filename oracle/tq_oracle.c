/*
 * tq_oracle.c -- plain CPU oracle of the TurboESM KV-cache path.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, obviously-correct
 * reference that the GPU library is checked against. Only the tests, the
 * smoke check and the CPU-baseline leg of the benchmark may load it. It shares
 * no code with the GPU library (no headers, helpers or tables).
 *
 * What it computes (TurboESM, arXiv 2603.26110):
 *   - RoPE (Sec. 2.1, Eq. 1-2) with theta_m = base^(-2m/d).
 *   - RoPE-first rotation k^ = Pi R k (Sec. 3.1, Eq. 4), fp64.
 *   - 3-bit table quantization with a per-vector norm (Sec. 3.3, Eq. 5) and
 *     1-bit residual signs (Sec. 3.4, Eq. 6-7; projected QJL form by default,
 *     the paper's per-element form on request). These steps decide integers
 *     (codes and sign bits), so they are written in binary32 with one fixed
 *     evaluation order: sequential fmaf chains, correctly rounded sqrtf and
 *     division. Build with -ffp-contract=off so nothing else is fused.
 *   - Packing into the cache layout (Sec. 4.2 packs 8 codes per 32-bit word).
 *     Every code is handled as a 4-bit value idx | sign << 3. In a key word
 *     the eight 3-bit indices fill bits 0..23 and the eight sign bits bits
 *     24..31; a value word holds eight such 4-bit nibbles. Key tiles are
 *     token-major, value tiles dimension-major.
 *   - Decode attention (Sec. 3.1 decode steps; Algorithm 1 of Sec. 4.3),
 *     fp64: a streaming online-softmax form and a two-step form that first
 *     materializes the dequantized keys and values.
 * Parity status: every function here is pinned by the CPU tests
 * (closed forms, library routines, brute force, worked examples).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define D 64          /* head dimension */
#define NPAIR 32      /* RoPE pairs */
#define TILE 64       /* slots per tile of the cache layout */

/* ------------------------------------------------------------------------ */
/* fp16 <-> fp32, written from the IEEE 754 binary16 format definition.      */
/* ------------------------------------------------------------------------ */

/* binary16 bits -> float (exact). */
float orc_f16_to_f32(uint16_t h) {
  int sign = (h >> 15) & 1;
  int expo = (h >> 10) & 0x1F;
  int mant = h & 0x3FF;
  double v;
  if (expo == 0) {
    v = ldexp((double)mant, -24);                 /* subnormal: mant * 2^-24 */
  } else if (expo == 31) {
    v = mant ? NAN : INFINITY;
  } else {
    v = ldexp((double)(mant + 1024), expo - 25);  /* (1 + mant/1024) 2^(e-15) */
  }
  return (float)(sign ? -v : v);
}

/* float -> binary16 bits, round to nearest, ties to even. Finite values too
 * large for binary16 become +-inf; NaN becomes a quiet NaN. */
uint16_t orc_f32_to_f16(float f) {
  uint16_t sign = signbit(f) ? 0x8000 : 0;
  double a = fabs((double)f);
  if (isnan(f)) return 0x7E00;
  if (a == 0.0) return sign;
  /* Candidates are multiples of the binary16 spacing at this magnitude. */
  int e;
  frexp(a, &e);                 /* a in [2^(e-1), 2^e) */
  int unbiased = e - 1;         /* a in [2^unbiased, 2^(unbiased+1)) */
  double ulp = unbiased < -14 ? ldexp(1.0, -24) : ldexp(1.0, unbiased - 10);
  double q = a / ulp;           /* exact: power-of-two scaling */
  double fl = floor(q);
  double rem = q - fl;
  double n = fl;
  if (rem > 0.5 || (rem == 0.5 && fmod(fl, 2.0) != 0.0)) n = fl + 1.0;
  double r = n * ulp;           /* rounded magnitude */
  if (r >= 65536.0) return sign | 0x7C00;  /* overflow: max finite is 65504 */
  if (r < ldexp(1.0, -14)) {    /* subnormal (or rounded up to min normal) */
    int m = (int)(r / ldexp(1.0, -24));
    return sign | (uint16_t)m;
  }
  int re;
  double fr = frexp(r, &re);    /* r = fr * 2^re, fr in [0.5, 1) */
  int expo = re - 1 + 15;
  int mant = (int)((fr * 2.0 - 1.0) * 1024.0 + 0.5);
  return sign | (uint16_t)(expo << 10) | (uint16_t)mant;
}

/* Norms are stored as fp16, saturated at the largest finite binary16. */
static uint16_t orc_store_norm(float x) {
  if (x > 65504.0f) x = 65504.0f;
  return orc_f32_to_f16(x);
}

/* ------------------------------------------------------------------------ */
/* RoPE (Sec. 2.1, Eq. 2): block-diagonal 2x2 rotations by p*theta_m.        */
/* ------------------------------------------------------------------------ */

/* cs[(p*32+m)*2 + {0,1}] = (float)cos, (float)sin of p*theta_m,
 * theta_m = base^(-2m/64), everything before the final rounding in fp64. */
void orc_rope_table(int positions, double base, float* cs) {
  for (int p = 0; p < positions; ++p)
    for (int m = 0; m < NPAIR; ++m) {
      double theta = pow(base, -2.0 * m / (double)D);
      double a = (double)p * theta;
      cs[(p * NPAIR + m) * 2 + 0] = (float)cos(a);
      cs[(p * NPAIR + m) * 2 + 1] = (float)sin(a);
    }
}

/* The two dimensions rotated together by pair m. */
static void rope_pair(int m, int half, int* a, int* b) {
  if (half) { *a = m; *b = m + NPAIR; }      /* (m, m + d/2) pairing        */
  else      { *a = 2 * m; *b = 2 * m + 1; }  /* (2m, 2m+1) pairing of Eq. 2 */
}

/* y = R_{theta,p} x in fp64 with the fp32 table entries of row p. */
void orc_rope_apply(const double* x, const float* cs_row, int half, double* y) {
  for (int i = 0; i < D; ++i) y[i] = x[i];
  for (int m = 0; m < NPAIR; ++m) {
    int a, b;
    rope_pair(m, half, &a, &b);
    double c = cs_row[2 * m], s = cs_row[2 * m + 1];
    y[a] = x[a] * c - x[b] * s;
    y[b] = x[a] * s + x[b] * c;
  }
}

/* y = Pi x (Pi row-major [64][64]), fp64. */
static void matvec(const float* pi, const double* x, double* y) {
  for (int i = 0; i < D; ++i) {
    double acc = 0.0;
    for (int k = 0; k < D; ++k) acc += (double)pi[i * D + k] * x[k];
    y[i] = acc;
  }
}

/* y = Pi^T x, fp64. */
static void matvec_t(const float* pi, const double* x, double* y) {
  for (int k = 0; k < D; ++k) {
    double acc = 0.0;
    for (int i = 0; i < D; ++i) acc += (double)pi[i * D + k] * x[i];
    y[k] = acc;
  }
}

/* Rotated input of the quantizer (Sec. 3.1 prefill steps 1 and 3), fp64,
 * rounded to binary32 at the end: keys k^ = Pi R_p k; values v^ = Pi v when
 * rotate_v, else v (values get no RoPE). */
void orc_rotated_input(const float* x, int is_key, int pos, const float* cs,
                       int half, const float* pi, int rotate_v, float* xhat) {
  double in[D], t[D], y[D];
  for (int i = 0; i < D; ++i) in[i] = x[i];
  if (is_key) {
    orc_rope_apply(in, cs + (size_t)pos * NPAIR * 2, half, t);
    matvec(pi, t, y);
  } else if (rotate_v) {
    matvec(pi, in, y);
  } else {
    for (int i = 0; i < D; ++i) y[i] = in[i];
  }
  for (int i = 0; i < D; ++i) xhat[i] = (float)y[i];
}

/* ------------------------------------------------------------------------ */
/* Quantizer (Sec. 3.3, Eq. 5; Sec. 3.4, Eq. 6; Sec. 4.2 fused argmin+sign). */
/* binary32, fixed order: this decides the stored integers.                  */
/* ------------------------------------------------------------------------ */

enum { ORC_SIGN_NONE = 0, ORC_SIGN_PROJECTED = 1, ORC_SIGN_ELEMENT = 2 };

/* Quantize one rotated vector x^ against the ascending 8-level table c.
 *   n = ||x^|| (fmaf chain), u = x^ * (8/n): unit mean-square coordinates,
 *   idx = number of midpoints t_m = (c_m + c_{m+1})/2 strictly below u,
 *   i.e. the nearest level with ties to the lower one,
 *   r = u - c[idx],  g = ||r|| (fmaf chain),
 *   sign bits: projected  !(S r)_i < 0  (fmaf chain over k ascending),
 *              element    !(r_i < 0).
 * nib[i] = idx_i | sign_i << 3. n and g are returned as fp16 bits. */
void orc_quantize_vector(const float* xhat, const float* c, const float* S,
                         int sign_mode, uint8_t* nib, uint16_t* n16,
                         uint16_t* g16) {
  float s = 0.0f;
  for (int i = 0; i < D; ++i) s = fmaf(xhat[i], xhat[i], s);
  float n = sqrtf(s);
  float inv = (n == 0.0f) ? 0.0f : 8.0f / n;
  float t[7];
  for (int m = 0; m < 7; ++m) t[m] = 0.5f * (c[m] + c[m + 1]);
  float u[D], r[D];
  int idx[D];
  for (int i = 0; i < D; ++i) {
    u[i] = xhat[i] * inv;
    int k = 0;
    for (int m = 0; m < 7; ++m) k += (u[i] > t[m]) ? 1 : 0;
    idx[i] = k;
    r[i] = u[i] - c[k];
  }
  float gs = 0.0f;
  for (int i = 0; i < D; ++i) gs = fmaf(r[i], r[i], gs);
  float g = sqrtf(gs);
  for (int i = 0; i < D; ++i) {
    int bit = 0;
    if (sign_mode == ORC_SIGN_PROJECTED) {
      float acc = 0.0f;
      for (int k = 0; k < D; ++k) acc = fmaf(S[i * D + k], r[k], acc);
      bit = !(acc < 0.0f);
    } else if (sign_mode == ORC_SIGN_ELEMENT) {
      bit = !(r[i] < 0.0f);
    }
    nib[i] = (uint8_t)(idx[i] | (bit << 3));
  }
  *n16 = orc_store_norm(n);
  *g16 = (sign_mode == ORC_SIGN_NONE) ? 0 : orc_store_norm(g);
}

/* ------------------------------------------------------------------------ */
/* Cache layout: 8 codes per 32-bit word (Sec. 4.2 packs 8 codes per 32-bit */
/* container); 64-slot tiles, 16-byte halves interleaved by slot.            */
/* ------------------------------------------------------------------------ */

/* K plane, token-major tiles: 16-byte half c (codes 32c..32c+31) of slot s
 * sits at tile*2048 + (c*64 + s%64)*16 inside one (layer, head) region. */
static int64_t k_half_offset(int64_t s, int c) {
  int64_t tile = s / TILE, lane = s % TILE;
  return tile * (TILE * 32) + ((int64_t)c * TILE + lane) * 16;
}

/* K word of dimensions 8w..8w+7: the 3-bit index of dimension 8w+j in bits
 * 3j..3j+2, its sign bit in bit 24+j. */
static uint32_t k_word(const uint8_t* nib8) {
  uint32_t word = 0;
  for (int j = 0; j < 8; ++j) {
    word |= (uint32_t)(nib8[j] & 7) << (3 * j);
    word |= (uint32_t)((nib8[j] >> 3) & 1) << (24 + j);
  }
  return word;
}

/* Write the 64 codes (idx | sign << 3) of one slot of the K plane. */
void orc_pack_slot(uint8_t* region, int64_t s, const uint8_t* nib) {
  for (int w = 0; w < 8; ++w) {
    const uint32_t word = k_word(nib + 8 * w);
    uint8_t* dst = region + k_half_offset(s, w / 4) + (w % 4) * 4;
    dst[0] = (uint8_t)(word & 0xFF);
    dst[1] = (uint8_t)((word >> 8) & 0xFF);
    dst[2] = (uint8_t)((word >> 16) & 0xFF);
    dst[3] = (uint8_t)((word >> 24) & 0xFF);
  }
}

/* Read the 64 codes (idx | sign << 3) of one slot of the K plane. */
void orc_unpack_slot(const uint8_t* region, int64_t s, uint8_t* nib) {
  for (int w = 0; w < 8; ++w) {
    const uint8_t* src = region + k_half_offset(s, w / 4) + (w % 4) * 4;
    uint32_t word = (uint32_t)src[0] | ((uint32_t)src[1] << 8) |
                    ((uint32_t)src[2] << 16) | ((uint32_t)src[3] << 24);
    for (int j = 0; j < 8; ++j)
      nib[w * 8 + j] = (uint8_t)(((word >> (3 * j)) & 7) | (((word >> (24 + j)) & 1) << 3));
  }
}

/* V plane, dimension-major tiles: for dimension i the 64 slots of a tile
 * form 32 bytes; 16-byte half c (slots 32c..32c+31 of the tile) sits at
 * tile*2048 + (c*64 + i)*16, and slot r of the tile is nibble r%8 of 32-bit
 * word (r%32)/8 of that half. Returns the byte holding the nibble and its
 * bit offset inside that byte (0 or 4). */
static int64_t v_nibble_byte(int64_t s, int i, int* shift) {
  int64_t tile = s / TILE;
  int r = (int)(s % TILE);
  int c = r / 32, w = (r % 32) / 8, j = r % 8;
  *shift = (j % 2) * 4;
  return tile * (TILE * 32) + ((int64_t)c * TILE + i) * 16 + w * 4 + j / 2;
}

/* Write the 64 nibbles of one slot of the V plane (other slots untouched). */
void orc_pack_slot_v(uint8_t* region, int64_t s, const uint8_t* nib) {
  for (int i = 0; i < D; ++i) {
    int sh;
    int64_t off = v_nibble_byte(s, i, &sh);
    region[off] = (uint8_t)((region[off] & ~(0xF << sh)) | ((nib[i] & 0xF) << sh));
  }
}

/* Read the 64 nibbles of one slot of the V plane. */
void orc_unpack_slot_v(const uint8_t* region, int64_t s, uint8_t* nib) {
  for (int i = 0; i < D; ++i) {
    int sh;
    int64_t off = v_nibble_byte(s, i, &sh);
    nib[i] = (uint8_t)((region[off] >> sh) & 0xF);
  }
}

/* Flags, spelled as in the library's documentation. */
#define F_V_ROTATE      1u
#define F_V_QJL         2u
#define F_QJL_PAPER     4u
#define F_ROPE_HALF     8u
#define F_INPUT_ROTATED 16u

/* Prefill quantize-and-pack over all tokens (Sec. 3.1 prefill steps 1, 3, 4).
 * k, v: [nl][B][T][H][64] floats (fp16 values already widened, or x^ when
 * F_INPUT_ROTATED). Region (l, h) of the cache starts at (l*H + h)*slots. */
void orc_quantize_pack(int L, int H, int64_t slots, uint32_t flags,
                       const float* cs, int rope_positions,
                       const float* k, const float* v, int B, int T,
                       int layer0, int nl, const int32_t* pos0,
                       const int64_t* slot0, const float* pi,
                       const float* lut_k, const float* lut_v, const float* S,
                       uint8_t* kc, uint8_t* vc, uint16_t* sc) {
  (void)L;
  int half = (flags & F_ROPE_HALF) != 0;
  int ksign = (flags & F_QJL_PAPER) ? ORC_SIGN_ELEMENT : ORC_SIGN_PROJECTED;
  int vsign = (flags & F_V_QJL) ? ksign : ORC_SIGN_NONE;
  for (int li = 0; li < nl; ++li)
    for (int b = 0; b < B; ++b)
      for (int j = 0; j < T; ++j)
        for (int h = 0; h < H; ++h) {
          int l = layer0 + li;
          int64_t s = slot0[b] + j;
          int pos = pos0[b] + j;
          if (s < 0 || s >= slots) continue;
          if (!(flags & F_INPUT_ROTATED) && (pos < 0 || pos >= rope_positions)) continue;
          size_t in_off = ((((size_t)li * B + b) * T + j) * H + h) * D;
          const float* P = pi + ((size_t)l * H + h) * D * D;
          float kh[D], vh[D];
          if (flags & F_INPUT_ROTATED) {
            memcpy(kh, k + in_off, sizeof kh);
            memcpy(vh, v + in_off, sizeof vh);
          } else {
            orc_rotated_input(k + in_off, 1, pos, cs, half, P, 0, kh);
            orc_rotated_input(v + in_off, 0, pos, cs, half, P,
                              (flags & F_V_ROTATE) != 0, vh);
          }
          uint8_t kn[D], vn[D];
          uint16_t nk, gk, nv, gv;
          orc_quantize_vector(kh, lut_k + ((size_t)l * H + h) * 8, S, ksign, kn, &nk, &gk);
          orc_quantize_vector(vh, lut_v + ((size_t)l * H + h) * 8, S, vsign, vn, &nv, &gv);
          int64_t region = ((int64_t)l * H + h) * slots;
          orc_pack_slot(kc + region * 32, s, kn);
          orc_pack_slot_v(vc + region * 32, s, vn);
          uint16_t* dst = sc + (region + s) * 4;
          dst[0] = nk; dst[1] = gk; dst[2] = nv; dst[3] = gv;
        }
}

/* ------------------------------------------------------------------------ */
/* Decode (Sec. 3.1 decode steps 1-4; Algorithm 1), fp64.                   */
/* ------------------------------------------------------------------------ */

/* Everything decode needs for one (sequence, layer, head). */
typedef struct {
  double qhat[D];   /* Pi R q                                   */
  double uq[D];     /* S q^ (projected QJL) or q^ (per element) */
  double ck[8], cv[8];
  double ebar_k, ebar_v;  /* per-head mean |residual| (per-element form) */
} unit_ctx;

static const double ALPHA = 1.2533141373155002512 / 64.0;  /* sqrt(pi/2)/m, m = 64 */

/* Dequantized value vector of one token (rotated basis when V was rotated):
 * v~ = (n_v/8) (c_V[idx] + correction). */
static void dequant_v(const uint8_t* nib, double nv, double gv, const double* cv,
                      uint32_t flags, double ebar_v, const float* S, double* out) {
  for (int i = 0; i < D; ++i) out[i] = cv[nib[i] & 7];
  if (flags & F_V_QJL) {
    if (flags & F_QJL_PAPER) {
      for (int i = 0; i < D; ++i) out[i] += ebar_v * ((nib[i] >> 3) ? 1.0 : -1.0);
    } else {
      /* QJL vector estimate of the residual: alpha g S^T sign(S r). */
      for (int kk = 0; kk < D; ++kk) {
        double acc = 0.0;
        for (int i = 0; i < D; ++i) acc += (double)S[i * D + kk] * ((nib[i] >> 3) ? 1.0 : -1.0);
        out[kk] += ALPHA * gv * acc;
      }
    }
  }
  for (int i = 0; i < D; ++i) out[i] *= nv / 8.0;
}

/* Dequantized key of one token, the form a "dequantize first, then attend"
 * path materializes (Sec. 3.4 applied to a stored key rather than to a
 * score): k~ = (n_k/8) (c_K[idx] + coef e) with e = S^T (2s - 1) and
 * coef = alpha g_k for the projected estimator, or e = 2s - 1 and
 * coef = ebar_K for the per-element form, so that q^ . k~ is key_score. */
static void dequant_k(const uint8_t* nib, double nk, double gk, const double* ck,
                      uint32_t flags, double ebar_k, const float* S, double* out) {
  for (int i = 0; i < D; ++i) out[i] = ck[nib[i] & 7];
  if (flags & F_QJL_PAPER) {
    for (int i = 0; i < D; ++i) out[i] += ebar_k * ((nib[i] >> 3) ? 1.0 : -1.0);
  } else {
    for (int kk = 0; kk < D; ++kk) {
      double acc = 0.0;
      for (int i = 0; i < D; ++i) acc += (double)S[i * D + kk] * ((nib[i] >> 3) ? 1.0 : -1.0);
      out[kk] += ALPHA * gk * acc;
    }
  }
  for (int i = 0; i < D; ++i) out[i] *= nk / 8.0;
}

/* Attention score of one cached key against the rotated query:
 * (n_k/8) ( sum_i q^_i c_K[idx_i] + coef sum_i y_i (2 s_i - 1) ),
 * coef = alpha g_k, y = S q^ (projected QJL), or coef = ebar_K, y = q^. */
static double key_score(const uint8_t* nib, double nk, double gk,
                        const unit_ctx* u, uint32_t flags) {
  double a = 0.0, b = 0.0;
  for (int i = 0; i < D; ++i) {
    a += u->qhat[i] * u->ck[nib[i] & 7];
    b += u->uq[i] * ((nib[i] >> 3) ? 1.0 : -1.0);
  }
  double coef = (flags & F_QJL_PAPER) ? u->ebar_k : ALPHA * gk;
  return nk / 8.0 * (a + coef * b);
}

static void unit_setup(const float* q, int qpos, const float* cs, uint32_t flags,
                       const float* P, const float* S, const float* lk,
                       const float* lv, const float* eb, unit_ctx* u) {
  double in[D], t[D];
  for (int i = 0; i < D; ++i) in[i] = q[i];
  orc_rope_apply(in, cs + (size_t)qpos * NPAIR * 2, (flags & F_ROPE_HALF) != 0, t);
  matvec(P, t, u->qhat);
  if (flags & F_QJL_PAPER) {
    for (int i = 0; i < D; ++i) u->uq[i] = u->qhat[i];
  } else {
    for (int i = 0; i < D; ++i) {
      double acc = 0.0;
      for (int k = 0; k < D; ++k) acc += (double)S[i * D + k] * u->qhat[k];
      u->uq[i] = acc;
    }
  }
  for (int m = 0; m < 8; ++m) { u->ck[m] = lk[m]; u->cv[m] = lv[m]; }
  u->ebar_k = eb ? eb[0] : 0.0;
  u->ebar_v = eb ? eb[1] : 0.0;
}

/* Streaming decode of one unit with an online softmax (Algorithm 1):
 * running max m, running sum l, running weighted value sum o. */
static void decode_unit_streaming(const unit_ctx* u, uint32_t flags, double scale,
                                  const uint8_t* kreg, const uint8_t* vreg,
                                  const uint16_t* screg, int64_t s0, int n,
                                  const float* P, const float* S, double* out) {
  double m = -INFINITY, l = 0.0, o[D];
  for (int i = 0; i < D; ++i) o[i] = 0.0;
  for (int j = 0; j < n; ++j) {
    int64_t s = s0 + j;
    uint8_t kn[D], vn[D];
    orc_unpack_slot(kreg, s, kn);
    orc_unpack_slot_v(vreg, s, vn);
    const uint16_t* sc = screg + s * 4;
    double nk = orc_f16_to_f32(sc[0]), gk = orc_f16_to_f32(sc[1]);
    double nv = orc_f16_to_f32(sc[2]), gv = orc_f16_to_f32(sc[3]);
    double logit = key_score(kn, nk, gk, u, flags) * scale;
    double vt[D];
    dequant_v(vn, nv, gv, u->cv, flags, u->ebar_v, S, vt);
    double mn = logit > m ? logit : m;
    double f = exp(m - mn);           /* rescale of the old state */
    double w = exp(logit - mn);
    l = l * f + w;
    for (int i = 0; i < D; ++i) o[i] = o[i] * f + w * vt[i];
    m = mn;
  }
  double oh[D];
  for (int i = 0; i < D; ++i) oh[i] = (n > 0) ? o[i] / l : 0.0;
  if (flags & F_V_ROTATE) matvec_t(P, oh, out);   /* one inverse rotation */
  else for (int i = 0; i < D; ++i) out[i] = oh[i];
}

/* Two-step decode of one unit: materialize every dequantized key and value
 * (the "dequantize first, then attend" path), then a plain softmax. */
static void decode_unit_twostep(const unit_ctx* u, uint32_t flags, double scale,
                                const uint8_t* kreg, const uint8_t* vreg,
                                const uint16_t* screg, int64_t s0, int n,
                                const float* P, const float* S, double* out) {
  if (n <= 0) { for (int i = 0; i < D; ++i) out[i] = 0.0; return; }
  double* logits = (double*)malloc(sizeof(double) * (size_t)n);
  double* vals = (double*)malloc(sizeof(double) * (size_t)n * D);
  for (int j = 0; j < n; ++j) {
    int64_t s = s0 + j;
    uint8_t kn[D], vn[D];
    orc_unpack_slot(kreg, s, kn);
    orc_unpack_slot_v(vreg, s, vn);
    const uint16_t* sc = screg + s * 4;
    logits[j] = key_score(kn, orc_f16_to_f32(sc[0]), orc_f16_to_f32(sc[1]), u, flags) * scale;
    dequant_v(vn, orc_f16_to_f32(sc[2]), orc_f16_to_f32(sc[3]), u->cv, flags,
              u->ebar_v, S, vals + (size_t)j * D);
  }
  double mx = -INFINITY;
  for (int j = 0; j < n; ++j) if (logits[j] > mx) mx = logits[j];
  double tot = 0.0;
  for (int j = 0; j < n; ++j) tot += exp(logits[j] - mx);
  double oh[D];
  for (int i = 0; i < D; ++i) {
    double acc = 0.0;
    for (int j = 0; j < n; ++j) acc += exp(logits[j] - mx) * vals[(size_t)j * D + i];
    oh[i] = acc / tot;
  }
  if (flags & F_V_ROTATE) matvec_t(P, oh, out);
  else for (int i = 0; i < D; ++i) out[i] = oh[i];
  free(logits);
  free(vals);
}

/* Decode over the units (li, b, h) listed in `units` (count nunits; each unit
 * is the flat index (li*B + b)*H + h), or over all units when units == NULL.
 * q: [nl][B][H][64] floats; out: [nl][B][H][64] doubles (only listed units are
 * written). twostep selects the two-step form. */
/* Threads of the OpenMP loops over units, for timing the oracle (its results
 * do not depend on the count). */
void orc_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
int orc_max_threads(void) { return omp_get_max_threads(); }

void orc_decode(int L, int H, int64_t slots, uint32_t flags, double scale,
                const float* cs, int rope_positions, const float* q, int B,
                int layer0, int nl, const int32_t* qpos, const int64_t* sslot0,
                const int32_t* slen, const float* pi, const float* lut_k,
                const float* lut_v, const float* S, const float* ebar,
                const uint8_t* kc, const uint8_t* vc, const uint16_t* sc,
                const int64_t* units, int64_t nunits, int twostep, double* out) {
  (void)L;
  int64_t total = units ? nunits : (int64_t)nl * B * H;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < total; ++t) {
    int64_t flat = units ? units[t] : t;
    int h = (int)(flat % H);
    int b = (int)((flat / H) % B);
    int li = (int)(flat / ((int64_t)H * B));
    int l = layer0 + li;
    double* o = out + flat * D;
    int n = slen[b];
    int64_t s0 = sslot0[b];
    int qp = qpos[b];
    if (n < 0 || s0 < 0 || s0 % TILE != 0 || s0 + n > slots || qp < 0 ||
        qp >= rope_positions) {
      for (int i = 0; i < D; ++i) o[i] = NAN;
      continue;
    }
    const float* P = pi + ((size_t)l * H + h) * D * D;
    unit_ctx u;
    unit_setup(q + flat * D, qp, cs, flags, P, S, lut_k + ((size_t)l * H + h) * 8,
               lut_v + ((size_t)l * H + h) * 8, ebar ? ebar + ((size_t)l * H + h) * 2 : NULL, &u);
    int64_t region = ((int64_t)l * H + h) * slots;
    if (twostep)
      decode_unit_twostep(&u, flags, scale, kc + region * 32, vc + region * 32,
                          sc + region * 4, s0, n, P, S, o);
    else
      decode_unit_streaming(&u, flags, scale, kc + region * 32, vc + region * 32,
                            sc + region * 4, s0, n, P, S, o);
  }
}

/* Dequantize every cached token of the units (li, b, h): k_out, v_out are
 * [nl][B][H][max_len][64] doubles; rows j < seq_len[b] of a valid sequence
 * are written, the rest are left as they are. */
void orc_dequantize(int L, int H, int64_t slots, uint32_t flags, int B, int layer0, int nl,
                    const int64_t* sslot0, const int32_t* slen, int max_len,
                    const float* lut_k, const float* lut_v, const float* S, const float* ebar,
                    const uint8_t* kc, const uint8_t* vc, const uint16_t* sc,
                    double* k_out, double* v_out) {
  (void)L;
  int64_t total = (int64_t)nl * B * H;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < total; ++t) {
    int h = (int)(t % H);
    int b = (int)((t / H) % B);
    int li = (int)(t / ((int64_t)H * B));
    int l = layer0 + li;
    int n = slen[b];
    int64_t s0 = sslot0[b];
    if (n < 0 || n > max_len || s0 < 0 || s0 % TILE != 0 || s0 + n > slots) continue;
    double ck[8], cv[8];
    for (int m = 0; m < 8; ++m) {
      ck[m] = lut_k[((size_t)l * H + h) * 8 + m];
      cv[m] = lut_v[((size_t)l * H + h) * 8 + m];
    }
    double ebar_k = ebar ? ebar[((size_t)l * H + h) * 2] : 0.0;
    double ebar_v = ebar ? ebar[((size_t)l * H + h) * 2 + 1] : 0.0;
    int64_t region = ((int64_t)l * H + h) * slots;
    for (int j = 0; j < n; ++j) {
      int64_t s = s0 + j;
      uint8_t kn[D], vn[D];
      orc_unpack_slot(kc + region * 32, s, kn);
      orc_unpack_slot_v(vc + region * 32, s, vn);
      const uint16_t* scs = sc + (region + s) * 4;
      double* ko = k_out + ((size_t)t * max_len + j) * D;
      double* vo = v_out + ((size_t)t * max_len + j) * D;
      dequant_k(kn, orc_f16_to_f32(scs[0]), orc_f16_to_f32(scs[1]), ck, flags, ebar_k, S, ko);
      dequant_v(vn, orc_f16_to_f32(scs[2]), orc_f16_to_f32(scs[3]), cv, flags, ebar_v, S, vo);
    }
  }
}
