/*
 * Minima-KV CPU oracle — test infrastructure only.
 *
 * A plain, slow, obviously-correct CPU implementation of what the MI355X hot
 * path computes.  It is linked only by the test-suite, by the smoke check and
 * by the benchmark's CPU-baseline leg; the product library never calls it and
 * shares no source with it.
 *
 * Floating point: fp64 for everything the paper leaves free; fp32 exactly where
 * the FP8 page scales are defined to be fp32.  Build with -ffp-contract=off so
 * that every operation is one IEEE-754 correctly rounded step in the written
 * order.
 *
 * Paper references (arXiv 2608.23834, "Minima-KV"):
 *   Sec. 2.1, Eq. (kv-per-token)    bytes per live token
 *   Sec. 3.1                        tiers z in {R, A, S}; Recent/Anchor FP8,
 *                                   Stale 3-bit rotated scalar quantizer
 *   Alg. 1                          Append / Retier / Promote transitions
 *   Sec. 3.3, Eq. (softmax-merge)   mixed-format partials and their merge
 *   Sec. 4.1                        compact per-format page lists, TQ3 page
 *                                   contents (rotated K codes, FP16 key-norm
 *                                   correction, V codes, FP16 scale/zero)
 *   Sec. 4.3                        FP8 -> TQ3 "normalize-rotate-pack"
 *
 * Readings of the paper where it is silent (each listed in the design notes):
 *   FP8 = OCP E4M3FN, round-to-nearest-even, saturating to +-448.
 *   FP8 scale: one fp32 per (page, KV head, K or V), s = amax/448.
 *   Rotation R = d^-1/2 * H_d * diag(sigma), H_d Sylvester Hadamard.
 *   Codebook: 8 symmetric levels +-{0.25, 0.75, 1.375, 2.25} (E4M3-exact
 *   neighbours of the Lloyd-Max N(0,1) levels), nearest-level decisions.
 *   Key-norm correction gamma = ||k|| / ||mu_c||, stored as fp16.
 *   V: per (page, KV head, channel) asymmetric 3-bit, fp16 scale and zero.
 *   Packed bit layout: the "chunk" layout documented at tq3_bit_pos().
 *
 * parity pinned: every function here is checked by the CPU test-suite against
 * closed forms, library routines or brute force (see tests/test_oracle_*.py).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_PAGE 16
#define TAG_R 0
#define TAG_A 1
#define TAG_S 2
#define TAG_NONE 0xFF

/* ------------------------------------------------------------------------ */
/* FP8 E4M3FN (Sec. 3.1: Recent and Anchor pages are FP8).                   */
/* Value of a code: sign * 2^(e-7) * (1 + m/8) for e >= 1, sign * 2^-6 * m/8  */
/* for e = 0; 0x7F / 0xFF are NaN; there is no infinity.                      */
/* ------------------------------------------------------------------------ */
double orc_e4m3_to_f64(uint8_t b) {
  int s = b >> 7, e = (b >> 3) & 15, m = b & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexp((double)m / 8.0, -6);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return s ? -v : v;
}

/* Round an fp32 to E4M3 by the definition: among the finite E4M3 values pick
 * the nearest; on a tie pick the one with an even mantissa; magnitudes beyond
 * the largest finite value (448) saturate to +-448; NaN maps to 0x7F|sign.
 * The non-negative finite codes 0x00..0x7E are increasing in value, so the
 * neighbours of |x| are found by bisection over their value table (fp64,
 * where every E4M3 value and every midpoint is exact). */
static double E4M3_VALS[127];
static int e4m3_table_ready = 0;
static void e4m3_table(void) {
  if (!e4m3_table_ready) {
    for (int c = 0; c < 127; ++c) E4M3_VALS[c] = orc_e4m3_to_f64((uint8_t)c);
    e4m3_table_ready = 1;
  }
}
static uint8_t e4m3_round(double v) {
  uint8_t sign = 0;
  if (isnan(v)) return signbit(v) ? 0xFF : 0x7F;
  if (signbit(v)) { sign = 0x80; v = -v; }
  if (v >= 448.0) return sign | 0x7E;
  int lo = 0, hi = 126; /* largest c with value(c) <= v */
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (E4M3_VALS[mid] <= v) lo = mid; else hi = mid - 1;
  }
  int best = lo, pick;
  double m = 0.5 * (E4M3_VALS[best] + E4M3_VALS[best + 1]);
  if (v < m) pick = best;
  else if (v > m) pick = best + 1;
  else pick = (best & 1) ? best + 1 : best; /* tie: even mantissa bit */
  return sign | (uint8_t)pick;
}
uint8_t orc_e4m3_from_f32(float xf) {
  e4m3_table();
  return e4m3_round((double)xf);
}

void orc_e4m3_from_f32_array(const float* x, uint8_t* out, int64_t n) {
  e4m3_table();
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = e4m3_round((double)x[i]);
}

/* ------------------------------------------------------------------------ */
/* IEEE binary16 (Sec. 4.1: "FP16" key-norm correction and V scale/zero).     */
/* One round-to-nearest-even from fp64, saturating to +-65504 (the stored     */
/* metadata must stay finite), done by integer manipulation of the fp64       */
/* significand so there is no intermediate rounding.                          */
/* ------------------------------------------------------------------------ */
uint16_t orc_f16_from_f64(double x) {
  uint64_t bits;
  memcpy(&bits, &x, 8);
  uint16_t sign = (uint16_t)((bits >> 48) & 0x8000);
  int e = (int)((bits >> 52) & 0x7FF);
  uint64_t frac = bits & ((1ULL << 52) - 1);
  if (e == 0x7FF) return frac ? (uint16_t)(sign | 0x7E00) : (uint16_t)(sign | 0x7BFF);
  if (e == 0 && frac == 0) return sign;
  /* value = sig * 2^(E) with sig a 53-bit integer */
  uint64_t sig;
  int E;
  if (e == 0) { sig = frac; E = -1074; }
  else { sig = frac | (1ULL << 52); E = e - 1075; }
  /* target: half value = h * 2^(he) where h has <= 11 bits (normal) and
   * he >= -24 (subnormal quantum). Find the quantum exponent q. */
  int msb = 63 - __builtin_clzll(sig);  /* position of leading bit */
  int vexp = E + msb;                   /* floor(log2|x|) */
  int q = vexp - 10;                    /* quantum for a normal half */
  if (q < -24) q = -24;                 /* subnormal range */
  /* h = round(sig * 2^(E - q)) */
  uint64_t h;
  int sh = q - E;
  if (sh <= 0) {
    h = sig << (-sh); /* exact (only when x is tiny-integer-like; safe: <=11 bits) */
  } else if (sh >= 64) {
    h = 0; /* far below half the smallest subnormal */
    if (sh == 64 && sig > (1ULL << 63)) h = 1;
  } else {
    uint64_t keep = sig >> sh;
    uint64_t rem = sig & ((1ULL << sh) - 1);
    uint64_t half = 1ULL << (sh - 1);
    if (rem > half || (rem == half && (keep & 1))) keep += 1;
    h = keep;
  }
  /* h may have become 2^11 after rounding up -> renormalise */
  if (h == 0) return sign;
  int hq = q;
  if (h >= 2048) { h >>= 1; hq += 1; }
  /* encode: value = h * 2^hq */
  if (h < 1024) {
    /* subnormal: hq must be -24 */
    return (uint16_t)(sign | (uint16_t)h);
  }
  int he = hq + 10 + 15; /* biased exponent */
  if (he >= 31) return (uint16_t)(sign | 0x7BFF); /* saturate to 65504 */
  return (uint16_t)(sign | (uint16_t)(he << 10) | (uint16_t)(h - 1024));
}

double orc_f16_to_f64(uint16_t h) {
  int s = h >> 15, e = (h >> 10) & 31, m = h & 1023;
  double v;
  if (e == 31) return m ? NAN : (s ? -INFINITY : INFINITY);
  if (e == 0) v = ldexp((double)m, -24);
  else v = ldexp((double)(m + 1024), e - 25);
  return s ? -v : v;
}

void orc_f16_from_f64_array(const double* x, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_f16_from_f64(x[i]);
}

static double bf16_to_f64(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}
static float bf16_to_f32(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* ------------------------------------------------------------------------ */
/* Rotation (Sec. 3.1 "rotated scalar quantizer"; Sec. 4.3 "rotate").         */
/* Sylvester Hadamard H_ij = (-1)^popcount(i & j), applied by definition.     */
/* ------------------------------------------------------------------------ */
/* y = H * x over int64 (exact), H Sylvester of order n (a power of two),
 * H_ij = (-1)^popcount(i & j).  Computed with the standard radix-2 butterflies
 * (a, b) -> (a + b, a - b), which factor the Sylvester matrix exactly. */
void orc_hadamard_i64(const int64_t* x, int64_t* y, int n) {
  for (int i = 0; i < n; ++i) y[i] = x[i];
  for (int s = 1; s < n; s <<= 1)
    for (int i = 0; i < n; i += 2 * s)
      for (int j = i; j < i + s; ++j) {
        int64_t a = y[j], b = y[j + s];
        y[j] = a + b;
        y[j + s] = a - b;
      }
}
/* Same transform over fp64 (used on sums of codebook levels, which are
 * multiples of 1/8 and therefore exact). */
static void hadamard_f64(double* y, int n) {
  for (int s = 1; s < n; s <<= 1)
    for (int i = 0; i < n; i += 2 * s)
      for (int j = i; j < i + s; ++j) {
        double a = y[j], b = y[j + s];
        y[j] = a + b;
        y[j + s] = a - b;
      }
}

/* ------------------------------------------------------------------------ */
/* TQ3 codebook and decision (Sec. 3.1, Sec. 4.1).                           */
/* ------------------------------------------------------------------------ */
static const double MU[8] = {-2.25, -1.375, -0.75, -0.25, 0.25, 0.75, 1.375, 2.25};
/* 16 * (decision threshold between MU[k] and MU[k+1]) */
static const int64_t TAU16[7] = {-29, -17, -8, 0, 8, 17, 29};
/* 64 * MU[k]^2 */
static const int64_t MU2X64[8] = {324, 121, 36, 4, 4, 36, 121, 324};

double orc_codebook(int k) { return MU[k]; }
int orc_num_threads(void) { return omp_get_max_threads(); }

/* c = #{k : y > T_k * sqrt(n2)}, evaluated exactly with integers; n2 > 0. */
int orc_tq3_decide(int64_t y, int64_t n2) {
  int64_t a = 16 * y;
  int c = 0;
  for (int k = 0; k < 7; ++k) {
    int64_t t = TAU16[k];
    int above;
    if (t == 0) above = a > 0;
    else if (t > 0) above = (a > 0) && (a * a > t * t * n2);
    else above = (a >= 0) || (a * a < t * t * n2);
    c += above;
  }
  return c;
}

/* X_j = E4M3 value * 2^9 (an integer for every finite code). */
static int64_t e4m3_times_512(uint8_t b) {
  double v = orc_e4m3_to_f64(b) * 512.0;
  return (int64_t)v;
}

/* Encode one page-head (all 16 tokens valid) from its FP8 representation.
 *   k8, v8: [16][d] E4M3 codes in logical (token, channel) order
 *   sK, sV: the page-head's fp32 FP8 scales
 * Out (logical): kcode[16][d], gamma[16] (fp16 bits), vcode[16][d] (token,
 * channel), vscale[d], vzero[d] (fp16 bits). */
void orc_tq3_encode(int d, const uint8_t* k8, float sK, const uint8_t* v8, float sV,
                    const int8_t* sigma, uint8_t* kcode, uint16_t* gamma, uint8_t* vcode,
                    uint16_t* vscale, uint16_t* vzero) {
  int64_t* X = (int64_t*)malloc(sizeof(int64_t) * d);
  int64_t* y = (int64_t*)malloc(sizeof(int64_t) * d);
  /* keys: normalize-rotate, then 3-bit codes and the norm correction */
  for (int t = 0; t < ORC_PAGE; ++t) {
    int64_t n2 = 0;
    for (int j = 0; j < d; ++j) {
      X[j] = sigma[j] * e4m3_times_512(k8[t * d + j]);
      n2 += X[j] * X[j]; /* sigma^2 = 1 */
    }
    if (n2 == 0) {
      for (int i = 0; i < d; ++i) kcode[t * d + i] = 3;
      gamma[t] = 0;
      continue;
    }
    orc_hadamard_i64(X, y, d);
    int64_t M = 0;
    for (int i = 0; i < d; ++i) {
      int c = orc_tq3_decide(y[i], n2);
      kcode[t * d + i] = (uint8_t)c;
      M += MU2X64[c];
    }
    /* gamma = ||k|| / ||mu_c|| = sK * 2^-9 * sqrt(n2) / sqrt(M / 64)
     *       = sqrt(n2 / M) * (sK * 2^-6), one rounding per operation */
    double r = (double)n2 / (double)M;
    double s = sqrt(r);
    double g = s * ((double)sK * 0.015625);
    gamma[t] = orc_f16_from_f64(g);
  }
  /* values: per channel asymmetric 3-bit over the page's 16 tokens */
  for (int c = 0; c < d; ++c) {
    double lo = INFINITY, hi = -INFINITY;
    for (int t = 0; t < ORC_PAGE; ++t) {
      double v = (double)sV * orc_e4m3_to_f64(v8[t * d + c]); /* exact */
      if (v < lo) lo = v;
      if (v > hi) hi = v;
    }
    uint16_t z16 = orc_f16_from_f64(lo);
    uint16_t s16 = orc_f16_from_f64((hi - lo) / 7.0);
    vzero[c] = z16;
    vscale[c] = s16;
    double z = orc_f16_to_f64(z16), s = orc_f16_to_f64(s16);
    for (int t = 0; t < ORC_PAGE; ++t) {
      int code = 0;
      if (s != 0.0) {
        double v = (double)sV * orc_e4m3_to_f64(v8[t * d + c]);
        double u = nearbyint((v - z) / s); /* default mode: ties to even */
        if (u < 0) u = 0;
        if (u > 7) u = 7;
        code = (int)u;
      }
      vcode[t * d + c] = (uint8_t)code;
    }
  }
  free(X);
  free(y);
}

/* Reconstruction: k_hat = gamma * R^T mu_c, v_hat = zero + scale * code. */
void orc_tq3_dequant(int d, const uint8_t* kcode, const uint16_t* gamma, const uint8_t* vcode,
                     const uint16_t* vscale, const uint16_t* vzero, const int8_t* sigma,
                     double* khat, double* vhat) {
  double inv = 1.0 / sqrt((double)d);
  double* w = (double*)malloc(sizeof(double) * d);
  for (int t = 0; t < ORC_PAGE; ++t) {
    double g = orc_f16_to_f64(gamma[t]);
    /* R^T mu_c = d^-1/2 diag(sigma) H mu_c  (H symmetric) */
    for (int j = 0; j < d; ++j) w[j] = MU[kcode[t * d + j]];
    hadamard_f64(w, d);
    for (int i = 0; i < d; ++i) khat[t * d + i] = g * sigma[i] * inv * w[i];
    for (int c = 0; c < d; ++c)
      vhat[t * d + c] = orc_f16_to_f64(vzero[c]) + orc_f16_to_f64(vscale[c]) * vcode[t * d + c];
  }
  free(w);
}

/* ------------------------------------------------------------------------ */
/* Physical layouts (Sec. 4.1: codes, scales and metadata stored next to the  */
/* page).  These index functions define the byte layout of both pools.        */
/* ------------------------------------------------------------------------ */
/* FP8 page-head region: 2*16*d bytes. K token-major; V in lane-chunk order. */
int64_t orc_fp8_k_off(int d, int t, int c) { return (int64_t)t * d + c; }
int64_t orc_fp8_v_off(int d, int t, int c) {
  int CL = d / 16, r = c / CL, m = c % CL, g = t / 4, u = t % 4;
  return (int64_t)ORC_PAGE * d + ((int64_t)(r * 4 + g) * CL + m) * 4 + u;
}
int64_t orc_tq3_region_bytes(int d) { return 16LL * d + 32; }
/* A "chunk" holds 16*CL... = d/16 quads of 4 codes in 3d/32 bytes. */
static int chunk_bytes(int d) { return 3 * d / 32; }

/* Bit position (byte index within the chunk, bit within the byte) of bit k of
 * the code at quad q, position b.  With n_dw = chunk_bytes/4 dwords: quads
 * q < 2*n_dw sit in dword q/2, byte b, bits 3*(q%2)+k.  The remaining quads
 * use bits 6-7 of every byte: spare quad e (= q - 2*n_dw) of triple p = e/2
 * takes, for even e, bits 6,7 of dword 3p and bit 6 of dword 3p+1; for odd e,
 * bit 7 of dword 3p+1 and bits 6,7 of dword 3p+2. */
void orc_tq3_bit_pos(int d, int q, int b, int k, int* byte_out, int* bit_out) {
  int n_dw = chunk_bytes(d) / 4;
  int w, bit;
  if (q < 2 * n_dw) {
    w = q / 2;
    bit = 3 * (q % 2) + k;
  } else {
    int e = q - 2 * n_dw, p = e / 2;
    if ((e & 1) == 0) {
      if (k < 2) { w = 3 * p; bit = 6 + k; }
      else { w = 3 * p + 1; bit = 6; }
    } else {
      if (k == 0) { w = 3 * p + 1; bit = 7; }
      else { w = 3 * p + 2; bit = 5 + k; }
    }
  }
  *byte_out = 4 * w + b;
  *bit_out = bit;
}

/* K code of (token t, channel c) -> (chunk byte offset, quad, pos) */
static void kcode_place(int d, int t, int c, int64_t* chunk_off, int* q, int* b) {
  int per = d / 4, g = c / per, cc = c % per;
  *chunk_off = (int64_t)(g * 16 + t) * chunk_bytes(d);
  *q = cc / 4;
  *b = cc % 4;
}
/* V code of (token t, channel c) */
static void vcode_place(int d, int t, int c, int64_t* chunk_off, int* q, int* b) {
  int CL = d / 16, r = c / CL, m = c % CL, g = t / 4, u = t % 4;
  *chunk_off = (int64_t)(g * 16 + r) * chunk_bytes(d);
  *q = m;
  *b = u;
}

static void put_code(uint8_t* chunk, int d, int q, int b, int code) {
  for (int k = 0; k < 3; ++k) {
    int by, bi;
    orc_tq3_bit_pos(d, q, b, k, &by, &bi);
    if ((code >> k) & 1) chunk[by] |= (uint8_t)(1u << bi);
    else chunk[by] &= (uint8_t)~(1u << bi);
  }
}
static int get_code(const uint8_t* chunk, int d, int q, int b) {
  int code = 0;
  for (int k = 0; k < 3; ++k) {
    int by, bi;
    orc_tq3_bit_pos(d, q, b, k, &by, &bi);
    code |= ((chunk[by] >> bi) & 1) << k;
  }
  return code;
}

/* Pack logical codes/metadata into a TQ3 region (16d+32 bytes):
 * [0,6d) K codes, [6d,12d) V codes, [12d,12d+32) gamma fp16[16],
 * then V scale fp16[d], then V zero fp16[d]. */
void orc_tq3_pack(int d, const uint8_t* kcode, const uint16_t* gamma, const uint8_t* vcode,
                  const uint16_t* vscale, const uint16_t* vzero, uint8_t* region) {
  memset(region, 0, (size_t)orc_tq3_region_bytes(d));
  for (int t = 0; t < ORC_PAGE; ++t)
    for (int c = 0; c < d; ++c) {
      int64_t off;
      int q, b;
      kcode_place(d, t, c, &off, &q, &b);
      put_code(region + off, d, q, b, kcode[t * d + c]);
      vcode_place(d, t, c, &off, &q, &b);
      put_code(region + 6 * d + off, d, q, b, vcode[t * d + c]);
    }
  memcpy(region + 12 * d, gamma, 32);
  memcpy(region + 12 * d + 32, vscale, 2 * (size_t)d);
  memcpy(region + 12 * d + 32 + 2 * d, vzero, 2 * (size_t)d);
}

void orc_tq3_unpack(int d, const uint8_t* region, uint8_t* kcode, uint16_t* gamma,
                    uint8_t* vcode, uint16_t* vscale, uint16_t* vzero) {
  for (int t = 0; t < ORC_PAGE; ++t)
    for (int c = 0; c < d; ++c) {
      int64_t off;
      int q, b;
      kcode_place(d, t, c, &off, &q, &b);
      kcode[t * d + c] = (uint8_t)get_code(region + off, d, q, b);
      vcode_place(d, t, c, &off, &q, &b);
      vcode[t * d + c] = (uint8_t)get_code(region + 6 * d + off, d, q, b);
    }
  memcpy(gamma, region + 12 * d, 32);
  memcpy(vscale, region + 12 * d + 32, 2 * (size_t)d);
  memcpy(vzero, region + 12 * d + 32 + 2 * d, 2 * (size_t)d);
}

/* ------------------------------------------------------------------------ */
/* Pool state machine (Alg. 1 Append / Retier / Promote / SealPrefix /      */
/* Finish; Sec. 3.1 tiers; Sec. 4.4 per-kind free lists, reference counts).  */
/* Every mapped page carries a reference count: its block-table entries      */
/* (request references) plus prefix-cache references.  A page with more     */
/* than one reference is shared and immutable: Retier and Promote act on     */
/* request-private pages (count 1) only.                                     */
/* ------------------------------------------------------------------------ */
typedef struct {
  int n_layers, n_kv_heads, d, n_fp8, n_tq3, recent;
  const int8_t* sigma;
  uint8_t* fp8;       /* [L][n_fp8][Hkv][32d] */
  float* fp8_scale;   /* [L][n_fp8][Hkv][2] */
  uint8_t* tq3;       /* [L][n_tq3][Hkv][16d+32] */
  int32_t* fp8_stack; /* ids, valid [0, *fp8_top) */
  int32_t* fp8_top;
  int32_t* tq3_stack;
  int32_t* tq3_top;
  int32_t* rc8;       /* [n_fp8] references to each FP8 page (0: free) */
  int32_t* rc3;       /* [n_tq3] references to each TQ3 page */
} orc_pool;

static uint8_t* fp8_region(const orc_pool* P, int layer, int id, int h) {
  return P->fp8 + (((int64_t)layer * P->n_fp8 + id) * P->n_kv_heads + h) * (int64_t)(32 * P->d);
}
static float* fp8_scales(const orc_pool* P, int layer, int id, int h) {
  return P->fp8_scale + (((int64_t)layer * P->n_fp8 + id) * P->n_kv_heads + h) * 2;
}
static uint8_t* tq3_region(const orc_pool* P, int layer, int id, int h) {
  return P->tq3 + (((int64_t)layer * P->n_tq3 + id) * P->n_kv_heads + h) * orc_tq3_region_bytes(P->d);
}

/* Quantize one page-head of K or V (Sec. 3.1 Recent FP8 append).
 * Slots [0,t0) already hold codes with scale *s; new fp32 values x[t0..t1). */
static void fp8_append_tensor(int d, uint8_t* codes, int is_v, float* s, int t0, int t1,
                              const float* x /*[t1-t0][d]*/) {
  float amax = 0.0f;
  for (int i = 0; i < (t1 - t0) * d; ++i) {
    float a = fabsf(x[i]);
    if (a > amax) amax = a;
  }
  float s_old = (t0 == 0) ? 0.0f : *s;
  float s_new = s_old;
  int requant = 0;
  if (t0 == 0) {
    s_new = amax / 448.0f;
  } else if (!(amax <= 448.0f * s_old)) {
    s_new = amax / 448.0f;
    requant = 1;
  }
#define OFF(t, c) (is_v ? orc_fp8_v_off(d, t, c) - (int64_t)ORC_PAGE * d : orc_fp8_k_off(d, t, c))
  if (requant) {
    for (int t = 0; t < t0; ++t)
      for (int c = 0; c < d; ++c) {
        uint8_t old = codes[OFF(t, c)];
        float deq = (float)orc_e4m3_to_f64(old) * s_old;
        codes[OFF(t, c)] = orc_e4m3_from_f32(deq / s_new);
      }
  }
  for (int t = t0; t < t1; ++t)
    for (int c = 0; c < d; ++c) {
      float v = x[(t - t0) * d + c];
      codes[OFF(t, c)] = (s_new > 0.0f) ? orc_e4m3_from_f32(v / s_new) : 0;
    }
  if (t0 == 0)
    for (int t = t1; t < ORC_PAGE; ++t)
      for (int c = 0; c < d; ++c) codes[OFF(t, c)] = 0;
#undef OFF
  *s = s_new;
}

/* Append(q, p), Alg. 1: allocate request-owned Recent FP8 pages for the new
 * tokens (only where the logical page is unmapped), write KV, publish.
 * layer < 0 writes every layer (k, v: [L][n_new][Hkv][d]); else that layer.
 * Returns 0, or 1 (out of FP8 pages, nothing changed), or 2 (a page that
 * receives tokens is mapped but not Recent FP8, nothing changed). */
int orc_append(orc_pool* P, int layer, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
               const int32_t* seq_before, const int32_t* cu_new, const uint16_t* k,
               const uint16_t* v) {
  int d = P->d, H = P->n_kv_heads;
  int n_new_total = cu_new[n_req];
  /* check first, so a failing call changes nothing */
  int need = 0;
  for (int r = 0; r < n_req; ++r) {
    int n = cu_new[r + 1] - cu_new[r];
    if (n <= 0) continue;
    int p0 = seq_before[r] / ORC_PAGE, p1 = (seq_before[r] + n - 1) / ORC_PAGE;
    if (p1 >= max_pages) return 3;
    for (int p = p0; p <= p1; ++p) {
      int32_t e = bt[(int64_t)r * max_pages + p];
      if (e < 0) need++;
      else if (tags[(int64_t)r * max_pages + p] != TAG_R) return 2;
    }
  }
  if (need > *P->fp8_top) return 1;
  for (int r = 0; r < n_req; ++r) {
    int n = cu_new[r + 1] - cu_new[r];
    if (n <= 0) continue;
    int p0 = seq_before[r] / ORC_PAGE, p1 = (seq_before[r] + n - 1) / ORC_PAGE;
    for (int p = p0; p <= p1; ++p) {
      int64_t i = (int64_t)r * max_pages + p;
      if (bt[i] < 0) {
        *P->fp8_top -= 1;
        bt[i] = P->fp8_stack[*P->fp8_top];
        tags[i] = TAG_R;
        P->rc8[bt[i]] = 1;
      }
    }
  }
  int l0 = layer < 0 ? 0 : layer, l1 = layer < 0 ? P->n_layers : layer + 1;
  /* the page-heads are independent: list them, then quantize each one */
  int64_t n_items = 0;
  for (int r = 0; r < n_req; ++r) {
    int n = cu_new[r + 1] - cu_new[r];
    if (n > 0) n_items += (seq_before[r] + n - 1) / ORC_PAGE - seq_before[r] / ORC_PAGE + 1;
  }
  int32_t* items = (int32_t*)malloc(sizeof(int32_t) * 2 * (n_items + 1));
  int64_t it = 0;
  for (int r = 0; r < n_req; ++r) {
    int n = cu_new[r + 1] - cu_new[r];
    if (n <= 0) continue;
    for (int p = seq_before[r] / ORC_PAGE; p <= (seq_before[r] + n - 1) / ORC_PAGE; ++p) {
      items[2 * it] = r;
      items[2 * it + 1] = p;
      it++;
    }
  }
  int64_t total = n_items * (int64_t)(l1 - l0) * H;
#pragma omp parallel
  {
    float* buf = (float*)malloc(sizeof(float) * ORC_PAGE * d);
#pragma omp for schedule(dynamic, 64)
    for (int64_t w = 0; w < total; ++w) {
      int h = (int)(w % H);
      int64_t rest = w / H;
      int l = l0 + (int)(rest % (l1 - l0));
      int64_t e = rest / (l1 - l0);
      int r = items[2 * e], p = items[2 * e + 1];
      int64_t lbase = (int64_t)(l - l0) * n_new_total * H * d;
      int sb = seq_before[r], n = cu_new[r + 1] - cu_new[r];
      int id = bt[(int64_t)r * max_pages + p];
      int t0 = sb > p * ORC_PAGE ? sb - p * ORC_PAGE : 0;
      int end = sb + n - p * ORC_PAGE;
      int t1 = end < ORC_PAGE ? end : ORC_PAGE;
      uint8_t* reg = fp8_region(P, l, id, h);
      float* sc = fp8_scales(P, l, id, h);
      for (int kv = 0; kv < 2; ++kv) {
        const uint16_t* src = kv ? v : k;
        for (int t = t0; t < t1; ++t) {
          int row = cu_new[r] + (p * ORC_PAGE + t - sb);
          for (int c = 0; c < d; ++c)
            buf[(t - t0) * d + c] = bf16_to_f32(src[lbase + ((int64_t)row * H + h) * d + c]);
        }
        fp8_append_tensor(d, reg + (kv ? (int64_t)ORC_PAGE * d : 0), kv, sc + kv, t0, t1, buf);
      }
    }
    free(buf);
  }
  free(items);
  return 0;
}

/* Tier rule (Sec. 3.1): page p is Recent iff it holds one of the last W
 * tokens, i.e. (p+1)*16 > seq_len - W; otherwise Anchor if in the anchor set;
 * otherwise Stale.  Recent has precedence over Anchor. */
int orc_tier(int p, int seq_len, int W, int is_anchor) {
  if ((p + 1) * ORC_PAGE > seq_len - W) return TAG_R;
  return is_anchor ? TAG_A : TAG_S;
}

/* Retier(p, TQ3), Alg. 1, for every Recent page that has left the window:
 * anchors are re-tagged A and keep their FP8 page; other pages are encoded
 * into a newly allocated TQ3 page (all layers and heads), then the new
 * (tag, id) is published and the FP8 page is released to its free list.
 * Allocation and release follow ascending (request, logical page).
 * Returns the number of migrated pages, or -1 if the TQ3 pool is short
 * (nothing changed). */
int orc_migrate(orc_pool* P, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
                const uint8_t* anchor, const int32_t* seq_lens) {
  int d = P->d, H = P->n_kv_heads;
  int n_mig = 0;
  for (int r = 0; r < n_req; ++r) {
    int np = (seq_lens[r] + ORC_PAGE - 1) / ORC_PAGE;
    for (int p = 0; p < np && p < max_pages; ++p) {
      int64_t i = (int64_t)r * max_pages + p;
      if (tags[i] != TAG_R) continue;
      int is_anchor = anchor ? anchor[i] != 0 : 0;
      if (orc_tier(p, seq_lens[r], P->recent, is_anchor) == TAG_S && P->rc8[bt[i]] == 1) n_mig++;
    }
  }
  if (n_mig > *P->tq3_top) return -1;
  /* 1. tier transitions and id assignment in ascending (request, page) */
  int32_t* mig = (int32_t*)malloc(sizeof(int32_t) * 4 * (n_mig + 1));
  int k_mig = 0;
  for (int r = 0; r < n_req; ++r) {
    int np = (seq_lens[r] + ORC_PAGE - 1) / ORC_PAGE;
    for (int p = 0; p < np && p < max_pages; ++p) {
      int64_t i = (int64_t)r * max_pages + p;
      if (tags[i] != TAG_R) continue;
      int is_anchor = anchor ? anchor[i] != 0 : 0;
      int z = orc_tier(p, seq_lens[r], P->recent, is_anchor);
      if (z == TAG_A) { tags[i] = TAG_A; continue; }
      /* a shared (sealed) page stays as it is until it is private again */
      if (z != TAG_S || P->rc8[bt[i]] != 1) continue;
      *P->tq3_top -= 1;
      mig[4 * k_mig] = r;
      mig[4 * k_mig + 1] = p;
      mig[4 * k_mig + 2] = bt[i];
      mig[4 * k_mig + 3] = P->tq3_stack[*P->tq3_top];
      k_mig++;
    }
  }
  /* 2. normalize-rotate-pack every page-head (independent) */
  int64_t total = (int64_t)n_mig * P->n_layers * H;
#pragma omp parallel
  {
    uint8_t* kcode = (uint8_t*)malloc((size_t)ORC_PAGE * d);
    uint8_t* vcode = (uint8_t*)malloc((size_t)ORC_PAGE * d);
    uint8_t* k8 = (uint8_t*)malloc((size_t)ORC_PAGE * d);
    uint8_t* v8 = (uint8_t*)malloc((size_t)ORC_PAGE * d);
    uint16_t gamma[ORC_PAGE];
    uint16_t* vs = (uint16_t*)malloc(2 * (size_t)d);
    uint16_t* vz = (uint16_t*)malloc(2 * (size_t)d);
#pragma omp for schedule(dynamic, 16)
    for (int64_t w = 0; w < total; ++w) {
      int h = (int)(w % H);
      int l = (int)((w / H) % P->n_layers);
      int e = (int)(w / H / P->n_layers);
      int src = mig[4 * e + 2], dst = mig[4 * e + 3];
      const uint8_t* reg = fp8_region(P, l, src, h);
      const float* sc = fp8_scales(P, l, src, h);
      for (int t = 0; t < ORC_PAGE; ++t)
        for (int c = 0; c < d; ++c) {
          k8[t * d + c] = reg[orc_fp8_k_off(d, t, c)];
          v8[t * d + c] = reg[orc_fp8_v_off(d, t, c)];
        }
      orc_tq3_encode(d, k8, sc[0], v8, sc[1], P->sigma, kcode, gamma, vcode, vs, vz);
      orc_tq3_pack(d, kcode, gamma, vcode, vs, vz, tq3_region(P, l, dst, h));
    }
    free(kcode); free(vcode); free(k8); free(v8); free(vs); free(vz);
  }
  /* 3. publish (tag S, new id) and release the FP8 pages in the same order */
  for (int j = 0; j < n_mig; ++j) {
    int64_t i = (int64_t)mig[4 * j] * max_pages + mig[4 * j + 1];
    bt[i] = mig[4 * j + 3];
    tags[i] = TAG_S;
    P->rc3[mig[4 * j + 3]] = 1;
    P->rc8[mig[4 * j + 2]] = 0;
    P->fp8_stack[*P->fp8_top] = mig[4 * j + 2];
    *P->fp8_top += 1;
  }
  free(mig);
  return n_mig;
}

/* Reconstruction used by Promote, in fp32 with every step fixed:
 *   k_hat_i = gamma * sigma_i * h_i / sqrt(d),  h = H_d mu_c   (Alg. 1 Promote
 *   "reconstruct"; the same k_hat = gamma R^T mu_c as orc_tq3_dequant),
 *   v_hat_c = zero_c + scale_c * code.
 * h_i is a multiple of 1/8 with |h_i| <= 2.25 d, so gamma * sigma_i * h_i is
 * exact in fp64; the division by the correctly rounded sqrt(d) is one fp64
 * rounding (none at d = 256) and the result is rounded once to fp32.  The
 * value is exact in fp64 (two binary16 numbers and a 3-bit integer) and
 * rounded once to fp32.  Out: k32, v32 [16][d] logical order. */
void orc_tq3_reconstruct_f32(int d, const uint8_t* kcode, const uint16_t* gamma,
                             const uint8_t* vcode, const uint16_t* vscale, const uint16_t* vzero,
                             const int8_t* sigma, float* k32, float* v32) {
  double* h = (double*)malloc(sizeof(double) * d);
  double rd = sqrt((double)d);
  for (int t = 0; t < ORC_PAGE; ++t) {
    double g = orc_f16_to_f64(gamma[t]);
    for (int j = 0; j < d; ++j) h[j] = MU[kcode[t * d + j]];
    hadamard_f64(h, d);
    for (int i = 0; i < d; ++i) {
      double a = g * (double)sigma[i] * h[i];
      k32[t * d + i] = (float)(a / rd);
    }
    for (int c = 0; c < d; ++c) {
      double v = orc_f16_to_f64(vzero[c]) + orc_f16_to_f64(vscale[c]) * (double)vcode[t * d + c];
      v32[t * d + c] = (float)v;
    }
  }
  free(h);
}

/* Promote(p), Alg. 1: a Stale page that re-enters the protected budget
 * (Sec. 3.1 Anchor paragraph) is reconstructed (orc_tq3_reconstruct_f32) and
 * quantized into a newly allocated FP8 page with the FP8 rule of a fresh
 * page (per page-head and K/V: s = amax / 448, code = E4M3(x / s)), for every
 * layer and KV head; then (tag Anchor, new FP8 id) is published and the TQ3
 * page is released to its free list.  Pages promoted: tag Stale, promote
 * mask set, logical page below ceil(seq_len / 16); other pages are left
 * alone.  FP8 ids are taken and TQ3 ids released in ascending (request,
 * logical page) order.  Returns the number of promoted pages, or -1 when the
 * FP8 free list is too short (nothing changed). */
int orc_promote(orc_pool* P, int n_req, int32_t* bt, uint8_t* tags, int max_pages,
                const uint8_t* promote, const int32_t* seq_lens) {
  int d = P->d, H = P->n_kv_heads;
  int n_pro = 0;
  for (int r = 0; r < n_req; ++r) {
    int np = (seq_lens[r] + ORC_PAGE - 1) / ORC_PAGE;
    for (int p = 0; p < np && p < max_pages; ++p) {
      int64_t i = (int64_t)r * max_pages + p;
      if (tags[i] == TAG_S && promote[i] && P->rc3[bt[i]] == 1) n_pro++;
    }
  }
  if (n_pro > *P->fp8_top) return -1;
  int32_t* pro = (int32_t*)malloc(sizeof(int32_t) * 4 * (n_pro + 1));
  int k = 0;
  for (int r = 0; r < n_req; ++r) {
    int np = (seq_lens[r] + ORC_PAGE - 1) / ORC_PAGE;
    for (int p = 0; p < np && p < max_pages; ++p) {
      int64_t i = (int64_t)r * max_pages + p;
      if (!(tags[i] == TAG_S && promote[i] && P->rc3[bt[i]] == 1)) continue;
      *P->fp8_top -= 1;
      pro[4 * k] = r;
      pro[4 * k + 1] = p;
      pro[4 * k + 2] = bt[i];
      pro[4 * k + 3] = P->fp8_stack[*P->fp8_top];
      k++;
    }
  }
  int64_t total = (int64_t)n_pro * P->n_layers * H;
#pragma omp parallel
  {
    uint8_t* kc = (uint8_t*)malloc((size_t)ORC_PAGE * d);
    uint8_t* vc = (uint8_t*)malloc((size_t)ORC_PAGE * d);
    uint16_t g[ORC_PAGE];
    uint16_t* vs = (uint16_t*)malloc(2 * (size_t)d);
    uint16_t* vz = (uint16_t*)malloc(2 * (size_t)d);
    float* k32 = (float*)malloc(sizeof(float) * ORC_PAGE * d);
    float* v32 = (float*)malloc(sizeof(float) * ORC_PAGE * d);
#pragma omp for schedule(dynamic, 16)
    for (int64_t w = 0; w < total; ++w) {
      int h = (int)(w % H);
      int l = (int)((w / H) % P->n_layers);
      int e = (int)(w / H / P->n_layers);
      int src = pro[4 * e + 2], dst = pro[4 * e + 3];
      orc_tq3_unpack(d, tq3_region(P, l, src, h), kc, g, vc, vs, vz);
      orc_tq3_reconstruct_f32(d, kc, g, vc, vs, vz, P->sigma, k32, v32);
      uint8_t* reg = fp8_region(P, l, dst, h);
      float* sc = fp8_scales(P, l, dst, h);
      fp8_append_tensor(d, reg, 0, sc, 0, ORC_PAGE, k32);
      fp8_append_tensor(d, reg + (int64_t)ORC_PAGE * d, 1, sc + 1, 0, ORC_PAGE, v32);
    }
    free(kc); free(vc); free(vs); free(vz); free(k32); free(v32);
  }
  for (int j = 0; j < n_pro; ++j) {
    int64_t i = (int64_t)pro[4 * j] * max_pages + pro[4 * j + 1];
    bt[i] = pro[4 * j + 3];
    tags[i] = TAG_A;
    P->rc8[pro[4 * j + 3]] = 1;
    P->rc3[pro[4 * j + 2]] = 0;
    P->tq3_stack[*P->tq3_top] = pro[4 * j + 2];
    *P->tq3_top += 1;
  }
  free(pro);
  return n_pro;
}

/* SealPrefix / prefix attach (Alg. 1 SealPrefix; Sec. 4.4): acquire one
 * reference on each listed page, (id, tag) with tag R/A = FP8, S = TQ3.  Every
 * listed page must be live (count >= 1) and its id in range; otherwise
 * nothing changes and -1 is returned.  Duplicates acquire once each. */
int orc_pages_acquire(orc_pool* P, int n, const int32_t* ids, const uint8_t* tg) {
  for (int k = 0; k < n; ++k) {
    int fp8 = tg[k] == TAG_R || tg[k] == TAG_A;
    if (!fp8 && tg[k] != TAG_S) return -1;
    int lim = fp8 ? P->n_fp8 : P->n_tq3;
    if (ids[k] < 0 || ids[k] >= lim) return -1;
    if ((fp8 ? P->rc8 : P->rc3)[ids[k]] < 1) return -1;
  }
  for (int k = 0; k < n; ++k) {
    int fp8 = tg[k] == TAG_R || tg[k] == TAG_A;
    (fp8 ? P->rc8 : P->rc3)[ids[k]] += 1;
  }
  return 0;
}

/* Release (Alg. 1 Finish / prefix eviction): drop one reference per listed
 * entry, in list order; a page whose count reaches zero returns to the top
 * of its free list at that moment (so a page listed twice is pushed at its
 * second entry).  A page listed more often than it has references, a bad tag
 * or id: nothing changes, -1.  Returns the number of pages freed. */
int orc_pages_release(orc_pool* P, int n, const int32_t* ids, const uint8_t* tg) {
  int32_t* need8 = (int32_t*)calloc((size_t)P->n_fp8 + 1, sizeof(int32_t));
  int32_t* need3 = (int32_t*)calloc((size_t)P->n_tq3 + 1, sizeof(int32_t));
  int bad = 0;
  for (int k = 0; k < n && !bad; ++k) {
    int fp8 = tg[k] == TAG_R || tg[k] == TAG_A;
    if (!fp8 && tg[k] != TAG_S) { bad = 1; break; }
    int lim = fp8 ? P->n_fp8 : P->n_tq3;
    if (ids[k] < 0 || ids[k] >= lim) { bad = 1; break; }
    int32_t* need = fp8 ? need8 : need3;
    if (++need[ids[k]] > (fp8 ? P->rc8 : P->rc3)[ids[k]]) bad = 1;
  }
  free(need8);
  free(need3);
  if (bad) return -1;
  int freed = 0;
  for (int k = 0; k < n; ++k) {
    int fp8 = tg[k] == TAG_R || tg[k] == TAG_A;
    int32_t* rc = fp8 ? P->rc8 : P->rc3;
    if (--rc[ids[k]] == 0) {
      if (fp8) P->fp8_stack[(*P->fp8_top)++] = ids[k];
      else P->tq3_stack[(*P->tq3_top)++] = ids[k];
      freed++;
    }
  }
  return freed;
}

/* Finish(q), Alg. 1: release every request reference of the listed requests'
 * rows (each mapped entry, in ascending (request, page) order, as
 * orc_pages_release), then unmap the rows (id -1, tag 0xFF).  reqs: the
 * request indices, ascending.  Returns the pages freed, or -1 (nothing
 * changed) on an inconsistent table. */
int orc_request_finish(orc_pool* P, int n_fin, const int32_t* reqs, int32_t* bt, uint8_t* tags,
                       int max_pages) {
  int64_t n = 0;
  for (int j = 0; j < n_fin; ++j)
    for (int p = 0; p < max_pages; ++p) n += bt[(int64_t)reqs[j] * max_pages + p] >= 0;
  int32_t* ids = (int32_t*)malloc(sizeof(int32_t) * (n + 1));
  uint8_t* tg = (uint8_t*)malloc((size_t)n + 1);
  int64_t k = 0;
  for (int j = 0; j < n_fin; ++j)
    for (int p = 0; p < max_pages; ++p) {
      int64_t i = (int64_t)reqs[j] * max_pages + p;
      if (bt[i] < 0) continue;
      ids[k] = bt[i];
      tg[k] = tags[i];
      k++;
    }
  int freed = orc_pages_release(P, (int)n, ids, tg);
  if (freed >= 0)
    for (int j = 0; j < n_fin; ++j)
      for (int p = 0; p < max_pages; ++p) {
        int64_t i = (int64_t)reqs[j] * max_pages + p;
        bt[i] = -1;
        tags[i] = TAG_NONE;
      }
  free(ids);
  free(tg);
  return freed;
}

/* Compact per-format page lists (Sec. 4.1): stable partition of the logical
 * pages [0, ceil(seq_len/16)) into FP8 (R or A) and TQ3 (S), logical order kept.
 * out8/out3: [n_req][max_pages][2] (logical index, physical id); counts:
 * [n_req][2]. */
void orc_partition(int n_req, const int32_t* bt, const uint8_t* tags, int max_pages,
                   const int32_t* seq_lens, int32_t* out8, int32_t* out3, int32_t* counts) {
  for (int r = 0; r < n_req; ++r) {
    int np = (seq_lens[r] + ORC_PAGE - 1) / ORC_PAGE;
    int n8 = 0, n3 = 0;
    for (int p = 0; p < np; ++p) {
      int64_t i = (int64_t)r * max_pages + p;
      if (tags[i] == TAG_S) {
        out3[((int64_t)r * max_pages + n3) * 2] = p;
        out3[((int64_t)r * max_pages + n3) * 2 + 1] = bt[i];
        n3++;
      } else {
        out8[((int64_t)r * max_pages + n8) * 2] = p;
        out8[((int64_t)r * max_pages + n8) * 2 + 1] = bt[i];
        n8++;
      }
    }
    counts[r * 2] = n8;
    counts[r * 2 + 1] = n3;
  }
}

/* ------------------------------------------------------------------------ */
/* Reference attention (Sec. 3.3): exact softmax attention, in fp64, over the */
/* codec-reconstructed logical cache; the format partition and the merge of  */
/* Eq. (softmax-merge) are algebraically the same as this single pass.        */
/* ------------------------------------------------------------------------ */
/* Reconstruct K and V of logical tokens [0, n_tok) of request r, KV head h,
 * layer l into khat/vhat [n_tok][d] (fp64). */
void orc_reconstruct(const orc_pool* P, int layer, int r, int h, const int32_t* bt,
                     const uint8_t* tags, int max_pages, int n_tok, double* khat, double* vhat) {
  int d = P->d;
  uint8_t* kc = (uint8_t*)malloc((size_t)ORC_PAGE * d);
  uint8_t* vc = (uint8_t*)malloc((size_t)ORC_PAGE * d);
  uint16_t g[ORC_PAGE];
  uint16_t* vs = (uint16_t*)malloc(2 * (size_t)d);
  uint16_t* vz = (uint16_t*)malloc(2 * (size_t)d);
  double* kh = (double*)malloc(sizeof(double) * ORC_PAGE * d);
  double* vh = (double*)malloc(sizeof(double) * ORC_PAGE * d);
  int np = (n_tok + ORC_PAGE - 1) / ORC_PAGE;
  for (int p = 0; p < np; ++p) {
    int64_t i = (int64_t)r * max_pages + p;
    int id = bt[i];
    int nv = n_tok - p * ORC_PAGE < ORC_PAGE ? n_tok - p * ORC_PAGE : ORC_PAGE;
    if (tags[i] == TAG_S) {
      orc_tq3_unpack(d, tq3_region(P, layer, id, h), kc, g, vc, vs, vz);
      orc_tq3_dequant(d, kc, g, vc, vs, vz, P->sigma, kh, vh);
      for (int t = 0; t < nv; ++t)
        for (int c = 0; c < d; ++c) {
          khat[((int64_t)p * ORC_PAGE + t) * d + c] = kh[t * d + c];
          vhat[((int64_t)p * ORC_PAGE + t) * d + c] = vh[t * d + c];
        }
    } else {
      const uint8_t* reg = fp8_region(P, layer, id, h);
      const float* sc = fp8_scales(P, layer, id, h);
      for (int t = 0; t < nv; ++t)
        for (int c = 0; c < d; ++c) {
          khat[((int64_t)p * ORC_PAGE + t) * d + c] = (double)sc[0] * orc_e4m3_to_f64(reg[orc_fp8_k_off(d, t, c)]);
          vhat[((int64_t)p * ORC_PAGE + t) * d + c] = (double)sc[1] * orc_e4m3_to_f64(reg[orc_fp8_v_off(d, t, c)]);
        }
    }
  }
  free(kc); free(vc); free(vs); free(vz); free(kh); free(vh);
}

/* softmax(q . k_hat / sqrt(d)) v_hat over keys [0, n_keys); out fp64[d] */
static void attend(int d, const double* q, const double* khat, const double* vhat, int n_keys,
                   double* out, double* lse) {
  double scale = 1.0 / sqrt((double)d);
  double* s = (double*)malloc(sizeof(double) * (n_keys > 0 ? n_keys : 1));
  double m = -INFINITY;
  for (int t = 0; t < n_keys; ++t) {
    double acc = 0.0;
    for (int c = 0; c < d; ++c) acc += q[c] * khat[(int64_t)t * d + c];
    s[t] = acc * scale;
    if (s[t] > m) m = s[t];
  }
  double l = 0.0;
  for (int c = 0; c < d; ++c) out[c] = 0.0;
  for (int t = 0; t < n_keys; ++t) {
    double w = exp(s[t] - m);
    l += w;
    for (int c = 0; c < d; ++c) out[c] += w * vhat[(int64_t)t * d + c];
  }
  for (int c = 0; c < d; ++c) out[c] /= l;
  if (lse) *lse = m + log(l);
  free(s);
}

/* Decode: the query of request r sits at position seq_len-1 and sees every
 * logical token t < seq_len.  q: bf16 [n_req][Hq][d]; out fp64 [n_req][Hq][d];
 * lse fp64 [n_req][Hq].  Query head hq uses KV head hq / (Hq/Hkv). */
void orc_decode(const orc_pool* P, int layer, int n_req, int n_q_heads, const uint16_t* q,
                const int32_t* bt, const uint8_t* tags, int max_pages, const int32_t* seq_lens,
                double* out, double* lse) {
  int d = P->d, H = P->n_kv_heads, G = n_q_heads / H;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int r = 0; r < n_req; ++r)
    for (int h = 0; h < H; ++h) {
      int n = seq_lens[r];
      double* kh = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * d);
      double* vh = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * d);
      double* qd = (double*)malloc(sizeof(double) * d);
      orc_reconstruct(P, layer, r, h, bt, tags, max_pages, n, kh, vh);
      for (int j = 0; j < G; ++j) {
        int hq = h * G + j;
        for (int c = 0; c < d; ++c) qd[c] = bf16_to_f64(q[((int64_t)r * n_q_heads + hq) * d + c]);
        attend(d, qd, kh, vh, n, out + ((int64_t)r * n_q_heads + hq) * d,
               lse ? lse + (int64_t)r * n_q_heads + hq : 0);
      }
      free(kh); free(vh); free(qd);
    }
}

/* Attention-score collector (Sec. 3.1, Eqs. score-partial, score-global-weight
 * and attention-score).  For query head h of request r, the globally
 * normalized mass of logical page p is the softmax weight of its tokens,
 *   q_{h,p} = sum_{i in p} exp(s_i - m) / sum_i exp(s_i - m)
 * (the partition form w_j rho_p^{(j)} of the equations is the same quantity
 * for any partition j of the tokens).  The collector conditions on
 * page-addressable mass, q~_{h,p} = q_{h,p} / sum_p' q_{h,p'}, averages it over
 * the sampled heads (head_mask[hq] != 0), r_p = mean_h q~_{h,p}, and updates
 * a_p = beta a_p + (1 - beta) r_p for the request's pages p < ceil(seq_len /
 * 16) in place (other entries unchanged).  qn_out [n_req][max_pages][Hq]
 * (q~, pages past the length left as they are) and r_out [n_req][max_pages]
 * are written when non-null. */
void orc_page_scores(const orc_pool* P, int layer, int n_req, int n_q_heads, const uint16_t* q,
                     const int32_t* bt, const uint8_t* tags, int max_pages, const int32_t* seq_lens,
                     const uint8_t* head_mask, double beta, double* a_inout, double* qn_out,
                     double* r_out) {
  int d = P->d, H = P->n_kv_heads, G = n_q_heads / H;
  int n_sampled = 0;
  for (int hq = 0; hq < n_q_heads; ++hq) n_sampled += head_mask[hq] != 0;
#pragma omp parallel for schedule(dynamic)
  for (int r = 0; r < n_req; ++r) {
    int n = seq_lens[r], np = (n + ORC_PAGE - 1) / ORC_PAGE;
    double* kh = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * d);
    double* vh = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * d);
    double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double* qp = (double*)malloc(sizeof(double) * (size_t)(np > 0 ? np : 1));
    double* racc = (double*)calloc((size_t)(np > 0 ? np : 1), sizeof(double));
    double* qd = (double*)malloc(sizeof(double) * d);
    for (int h = 0; h < H; ++h) {
      orc_reconstruct(P, layer, r, h, bt, tags, max_pages, n, kh, vh);
      for (int j = 0; j < G; ++j) {
        int hq = h * G + j;
        for (int c = 0; c < d; ++c) qd[c] = bf16_to_f64(q[((int64_t)r * n_q_heads + hq) * d + c]);
        double m = -INFINITY;
        for (int t = 0; t < n; ++t) {
          double acc = 0.0;
          for (int c = 0; c < d; ++c) acc += qd[c] * kh[(int64_t)t * d + c];
          s[t] = acc / sqrt((double)d);
          if (s[t] > m) m = s[t];
        }
        double l = 0.0;
        for (int t = 0; t < n; ++t) l += exp(s[t] - m);
        double z = 0.0;
        for (int p = 0; p < np; ++p) {
          double mass = 0.0;
          for (int t = p * ORC_PAGE; t < n && t < (p + 1) * ORC_PAGE; ++t) mass += exp(s[t] - m);
          qp[p] = mass / l;
          z += qp[p];
        }
        for (int p = 0; p < np; ++p) {
          double qn = qp[p] / z;
          if (qn_out) qn_out[((int64_t)r * max_pages + p) * n_q_heads + hq] = qn;
          if (head_mask[hq]) racc[p] += qn;
        }
      }
    }
    for (int p = 0; p < np; ++p) {
      double rp = n_sampled ? racc[p] / n_sampled : 0.0;
      if (r_out) r_out[(int64_t)r * max_pages + p] = rp;
      double* ap = &a_inout[(int64_t)r * max_pages + p];
      *ap = beta * *ap + (1.0 - beta) * rp;
    }
    free(kh); free(vh); free(s); free(qp); free(racc); free(qd);
  }
}

/* Chunk (causal): request r has n_r = cu_q[r+1]-cu_q[r] queries; query i sits
 * at position seq_len - n_r + i and sees keys t <= that position.  The chunk's
 * own KV is read back from the pool (it was appended as FP8 beforehand).
 * q: bf16 [sum n_r][Hq][d]; out fp64 same shape.  strides (NULL: every
 * query): only queries i with i % strides[r] == 0, and each request's last
 * query, are computed; the other rows of out are left as they are. */
void orc_chunk(const orc_pool* P, int layer, int n_req, int n_q_heads, const uint16_t* q,
               const int32_t* cu_q, const int32_t* bt, const uint8_t* tags, int max_pages,
               const int32_t* seq_lens, double* out, const int32_t* strides) {
  int d = P->d, H = P->n_kv_heads, G = n_q_heads / H;
  /* one request at a time: its heads' reconstructed caches, then every
   * sampled (head, query) row in parallel */
  for (int r = 0; r < n_req; ++r) {
    int n = seq_lens[r], nq = cu_q[r + 1] - cu_q[r];
    int64_t stride = strides && strides[r] > 1 ? strides[r] : 1;
    size_t per = (size_t)(n > 0 ? n : 1) * d;
    double* kh = (double*)malloc(sizeof(double) * per * H);
    double* vh = (double*)malloc(sizeof(double) * per * H);
#pragma omp parallel for schedule(static)
    for (int h = 0; h < H; ++h)
      orc_reconstruct(P, layer, r, h, bt, tags, max_pages, n, kh + per * h, vh + per * h);
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int h = 0; h < H; ++h)
      for (int i = 0; i < nq; ++i) {
        if (((int64_t)i % stride) != 0 && i != nq - 1) continue;
        int pos = n - nq + i;
        double* qd = (double*)malloc(sizeof(double) * d);
        for (int j = 0; j < G; ++j) {
          int hq = h * G + j;
          int64_t row = (int64_t)(cu_q[r] + i) * n_q_heads + hq;
          for (int c = 0; c < d; ++c) qd[c] = bf16_to_f64(q[row * d + c]);
          attend(d, qd, kh + per * h, vh + per * h, pos + 1, out + row * d, 0);
        }
        free(qd);
      }
    free(kh);
    free(vh);
  }
}

/* Eq. (softmax-merge), Sec. 3.3: merge partials (m_j, l_j, Obar_j) into O.
 * Empty partials carry l_j = 0 and are skipped. */
void orc_merge(int n_parts, int d, const double* m, const double* l, const double* obar,
               double* out, double* lse) {
  double M = -INFINITY;
  for (int j = 0; j < n_parts; ++j)
    if (l[j] > 0 && m[j] > M) M = m[j];
  double L = 0.0;
  for (int c = 0; c < d; ++c) out[c] = 0.0;
  for (int j = 0; j < n_parts; ++j) {
    if (!(l[j] > 0)) continue;
    double w = exp(m[j] - M) * l[j];
    L += w;
    for (int c = 0; c < d; ++c) out[c] += w * obar[(int64_t)j * d + c];
  }
  for (int c = 0; c < d; ++c) out[c] /= L;
  if (lse) *lse = M + log(L);
}
