/* semkv_oracle.c -- plain, slow CPU oracle of the SemKV hot path.
 *
 * TEST INFRASTRUCTURE ONLY (see semkv_oracle.h).  Written from the paper:
 *   Eq. (4)-(6)  top-K ranking and two-level bit assignment   (Sec. 3.4)
 *   Eq. (7)      per-token quantization of K and V            (Sec. 3.5)
 *   Alg. 2       block-exact deferred quantization            (Sec. 3.7)
 *   Sec. 4.1     affine base, two fp16 parameters, mixed-radix packing
 *   Sec. 4.9     TurboQuant-MSE base, one scalar per row, Lloyd-Max codes
 *   Sec. 4.1/4.9 the affine base under a Hadamard rotation (rotated affine)
 *   Sec. 3.3     token-importance indicators (Eq. 3 and its families)
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -fopenmp (IEEE single on SSE).
 */
#include "semkv_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- fp16 -- */

uint16_t oq_f32_to_f16(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  uint32_t sign = (u >> 16) & 0x8000u;
  uint32_t ex = (u >> 23) & 0xFFu;
  uint32_t man = u & 0x7FFFFFu;
  if (ex == 0xFFu) {                          /* inf or NaN */
    if (man) return (uint16_t)(sign | 0x7E00u | (man >> 13));
    return (uint16_t)(sign | 0x7C00u);
  }
  if (ex == 0) return (uint16_t)sign;         /* f32 zero / subnormal << 2^-25 */
  int32_t e = (int32_t)ex - 127;              /* value = m * 2^(e-23) */
  uint32_t m = man | 0x800000u;
  if (e > 15) return (uint16_t)(sign | 0x7C00u);
  if (e >= -14) {                             /* normal binary16 range */
    uint32_t keep = m >> 13, rest = m & 0x1FFFu;
    if (rest > 0x1000u || (rest == 0x1000u && (keep & 1u))) keep++;
    uint32_t he = (uint32_t)(e + 15);
    if (keep == 0x800u) { keep = 0x400u; he++; }
    if (he >= 31u) return (uint16_t)(sign | 0x7C00u);
    return (uint16_t)(sign | (he << 10) | (keep & 0x3FFu));
  }
  /* subnormal binary16: value = k * 2^-24 with k = m * 2^(e+1) */
  int shift = -(e + 1);
  if (shift > 24) return (uint16_t)sign;
  uint32_t k = m >> shift;
  uint32_t rest = m & ((1u << shift) - 1u), half = 1u << (shift - 1);
  if (rest > half || (rest == half && (k & 1u))) k++;
  return (uint16_t)(sign | k);                /* k == 0x400 is the least normal */
}

float oq_f16_to_f32(uint16_t h) {
  uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
  uint32_t e = ((uint32_t)h >> 10) & 0x1Fu, m = (uint32_t)h & 0x3FFu, u;
  float f;
  if (e == 0) {
    f = ldexpf((float)m, -24);
    return sign ? -f : f;
  }
  if (e == 31) u = sign | 0x7F800000u | (m << 13);
  else u = sign | ((e - 15u + 127u) << 23) | (m << 13);
  memcpy(&f, &u, 4);
  return f;
}

/* ------------------------------------------------------------- counts -- */

int64_t oq_top_count(int64_t T, int64_t r_num, int64_t r_den) {
  return (r_num * T) / r_den;                 /* Eq. (4): floor(r T) */
}

int64_t oq_block_count(int64_t n, int64_t r_num, int64_t r_den) {
  int64_t a = r_num * n, q = a / r_den, rem = a - q * r_den;
  if (2 * rem > r_den || (2 * rem == r_den && (q & 1))) q++;
  return q;                                   /* round(r n), ties to even */
}

/* ------------------------------------------------------------ ranking -- */

static int before(const float* s, int64_t a, int64_t b) {
  float sa = s[a] == 0.0f ? 0.0f : s[a];
  float sb = s[b] == 0.0f ? 0.0f : s[b];
  if (sa != sb) return sa > sb;
  return a < b;
}

static void merge_sort(int64_t* idx, int64_t* tmp, int64_t n, const float* s) {
  if (n < 2) return;
  int64_t h = n / 2;
  merge_sort(idx, tmp, h, s);
  merge_sort(idx + h, tmp, n - h, s);
  int64_t i = 0, j = h, o = 0;
  while (i < h && j < n) tmp[o++] = before(s, idx[j], idx[i]) ? idx[j++] : idx[i++];
  while (i < h) tmp[o++] = idx[i++];
  while (j < n) tmp[o++] = idx[j++];
  memcpy(idx, tmp, (size_t)n * sizeof(int64_t));
}

int oq_rank_k(const float* s, int64_t T, int64_t k, uint8_t* flag) {
  if (T < 0 || k < 0 || k > T) return OQ_EINVAL;
  for (int64_t i = 0; i < T; i++)
    if (isnan(s[i])) return OQ_ENAN;
  int64_t* idx = (int64_t*)malloc((size_t)(T + 1) * sizeof(int64_t));
  int64_t* tmp = (int64_t*)malloc((size_t)(T + 1) * sizeof(int64_t));
  for (int64_t i = 0; i < T; i++) idx[i] = i;
  merge_sort(idx, tmp, T, s);                 /* full sort: TopK of Eq. (4) */
  memset(flag, 0, (size_t)T);
  for (int64_t i = 0; i < k; i++) flag[idx[i]] = 1;
  free(idx);
  free(tmp);
  return OQ_OK;
}

/* ------------------------------------------------------ affine quantizer -- */

/* The two fp16 parameters of a group are finite for finite input (reading
 * R18): an fp16 rounding that overflows to +-inf is stored as +-65504, the
 * largest finite binary16, and the codes are taken against the stored pair
 * (clamped to [0, L-1]).  Only 2 levels can overflow the plain affine scale
 * ((max - min) / 1 may reach 131008); under a rotation the rotated
 * coordinates themselves may exceed 65504. */
static uint16_t sat_f16(uint16_t h) {
  if ((h & 0x7FFFu) == 0x7C00u) return (uint16_t)((h & 0x8000u) | 0x7BFFu);
  return h;
}

int oq_affine_row(const uint16_t* x, int L, int G, uint8_t* codes, uint16_t* meta) {
  if (L < 2 || L > 16 || G <= 0 || 128 % G) return OQ_EINVAL;
  int status = OQ_OK;
  for (int g = 0; g < 128 / G; g++) {
    float mn = INFINITY, mx = -INFINITY;
    for (int j = g * G; j < (g + 1) * G; j++) {
      float f = oq_f16_to_f32(x[j]);
      if (!isfinite(f)) status = OQ_ENAN;
      if (f < mn) mn = f;
      if (f > mx) mx = f;
    }
    float zero = mn + 0.0f;                   /* -0 -> +0 */
    float s32 = (mx - mn) / (float)(L - 1);   /* asymmetric range / (L-1) */
    uint16_t s16 = sat_f16(oq_f32_to_f16(s32));
    float sf = oq_f16_to_f32(s16);
    float inv = sf == 0.0f ? 0.0f : 1.0f / sf;
    meta[2 * g] = s16;
    meta[2 * g + 1] = oq_f32_to_f16(zero);
    for (int j = g * G; j < (g + 1) * G; j++) {
      float t = (oq_f16_to_f32(x[j]) - zero) * inv;
      float c = rintf(t);                      /* nearest, ties to even */
      if (!(c >= 0.0f)) c = 0.0f;
      if (c > (float)(L - 1)) c = (float)(L - 1);
      codes[j] = (uint8_t)c;
    }
  }
  return status;
}

/* ----------------------------------------------------- Lloyd-Max (N(0,1)) -- */

static double phi(double x) { return exp(-0.5 * x * x) / sqrt(2.0 * M_PI); }
static double Phi(double x) { return 0.5 * erfc(-x / sqrt(2.0)); }

int oq_lloyd_max(int L, double* mu, double* tau, double* mse) {
  if (L < 2 || L > 16) return OQ_EINVAL;
  double t[17];
  for (int k = 0; k < L; k++) mu[k] = -2.0 + 4.0 * (k + 0.5) / L;
  for (int it = 0; it < 200000; it++) {
    t[0] = -INFINITY;
    t[L] = INFINITY;
    for (int k = 1; k < L; k++) t[k] = 0.5 * (mu[k - 1] + mu[k]);   /* nearest-neighbour cells */
    double delta = 0.0;
    for (int k = 0; k < L; k++) {             /* centroid of each cell */
      double pa = k == 0 ? 0.0 : phi(t[k]), pb = k == L - 1 ? 0.0 : phi(t[k + 1]);
      double m = (pa - pb) / (Phi(t[k + 1]) - Phi(t[k]));
      delta = fmax(delta, fabs(m - mu[k]));
      mu[k] = m;
    }
    for (int k = 0; k < L / 2; k++) {         /* the Gaussian is symmetric */
      double a = 0.5 * (mu[L - 1 - k] - mu[k]);
      mu[k] = -a;
      mu[L - 1 - k] = a;
    }
    if (L % 2) mu[L / 2] = 0.0;
    if (delta < 1e-17) break;
  }
  for (int k = 1; k < L; k++) tau[k - 1] = 0.5 * (mu[k - 1] + mu[k]);
  if (L % 2 == 0) tau[L / 2 - 1] = 0.0;
  if (mse) {                                  /* E[(X - Q(X))^2] = 1 - sum p_k mu_k^2 */
    double e = 1.0;
    for (int k = 0; k < L; k++) {
      double a = k == 0 ? -INFINITY : tau[k - 1], b = k == L - 1 ? INFINITY : tau[k];
      e -= (Phi(b) - Phi(a)) * mu[k] * mu[k];
    }
    *mse = e;
  }
  return OQ_OK;
}

/* -------------------------------------------------- TurboQuant-MSE base -- */

static int sign_bit(const uint32_t* w, int i) { return (int)((w[i >> 5] >> (i & 31)) & 1u); }

int oq_tq_row(const uint16_t* x, const uint32_t* sign_words, int L, const float* tau32,
              uint8_t* codes, uint16_t* rho) {
  if (L < 2 || L > 16) return OQ_EINVAL;
  int status = OQ_OK;
  float u[128], a[128];
  for (int i = 0; i < 128; i++) {
    float f = oq_f16_to_f32(x[i]);
    if (!isfinite(f)) status = OQ_ENAN;
    u[i] = sign_bit(sign_words, i) ? -f : f;  /* diag(sign) x */
    a[i] = f * f;                              /* exact: 22-bit products */
  }
  for (int h = 1; h < 128; h <<= 1)           /* unnormalized Sylvester WHT */
    for (int i = 0; i < 128; i++)
      if (!(i & h)) {
        float p = u[i], q = u[i + h];
        u[i] = p + q;
        u[i + h] = p - q;
      }
  for (int h = 64; h >= 1; h >>= 1)           /* ||x||^2 by a fixed pairwise tree */
    for (int i = 0; i < h; i++) a[i] = a[i] + a[i + h];
  float r32 = sqrtf(a[0]);
  uint16_t r16 = oq_f32_to_f16(r32);
  if ((r16 & 0x7FFFu) == 0x7C00u) r16 = 0x7BFFu;   /* saturate to 65504 */
  *rho = r16;
  float rf = oq_f16_to_f32(r16);
  for (int j = 0; j < 128; j++) {             /* y/rho is ~N(0,1): count thresholds below */
    int c = 0;
    for (int k = 0; k < L - 1; k++)
      if (u[j] > rf * tau32[k]) c++;
    codes[j] = (uint8_t)c;
  }
  return status;
}

/* ------------------------------------------- affine under a rotation -- */

/* The affine quantizer applied to the rotated row y = H diag(sign) x / 16
 * (Sec. 4.1: integer-level scalar quantization with a Hadamard rotation; Sec.
 * 4.9: the per-row asymmetric affine quantizer under Hadamard rotation).  H is
 * the unnormalized Sylvester matrix, so y is the orthonormal rotation of x
 * scaled by sqrt(128)/16 = 1/sqrt(2): a power of two away from the orthogonal
 * map, which the affine quantizer does not see apart from fp16 range.  The
 * rotation is summed in fp32 in the order of oq_tq_row, then divided by 16
 * (exact).  Per group of G rotated coordinates: zero = fp16(min y) (-0 taken
 * as +0), scale = fp16(max(0, (max y - zero) / (L-1))), both saturated to
 * +-65504 (reading R18: y reaches 128 * 65504 / 16 in magnitude), codes as in
 * oq_affine_row with the stored parameters. */
int oq_rotaffine_row(const uint16_t* x, const uint32_t* sign_words, int L, int G,
                     uint8_t* codes, uint16_t* meta) {
  if (L < 2 || L > 16 || G <= 0 || 128 % G) return OQ_EINVAL;
  int status = OQ_OK;
  float y[128];
  for (int i = 0; i < 128; i++) {
    float f = oq_f16_to_f32(x[i]);
    if (!isfinite(f)) status = OQ_ENAN;
    y[i] = sign_bit(sign_words, i) ? -f : f;
  }
  for (int h = 1; h < 128; h <<= 1)
    for (int i = 0; i < 128; i++)
      if (!(i & h)) {
        float p = y[i], q = y[i + h];
        y[i] = p + q;
        y[i + h] = p - q;
      }
  for (int i = 0; i < 128; i++) y[i] = y[i] / 16.0f;
  for (int g = 0; g < 128 / G; g++) {
    float mn = INFINITY, mx = -INFINITY;
    for (int j = g * G; j < (g + 1) * G; j++) {
      if (y[j] < mn) mn = y[j];
      if (y[j] > mx) mx = y[j];
    }
    uint16_t z16 = sat_f16(oq_f32_to_f16(mn));
    if (z16 == 0x8000u) z16 = 0;
    float zf = oq_f16_to_f32(z16);
    float s32 = (mx - zf) / (float)(L - 1);
    if (!(s32 > 0.0f)) s32 = 0.0f;            /* zero rounded above every value */
    uint16_t s16 = sat_f16(oq_f32_to_f16(s32));
    float sf = oq_f16_to_f32(s16);
    float inv = sf == 0.0f ? 0.0f : 1.0f / sf;
    meta[2 * g] = s16;
    meta[2 * g + 1] = z16;
    for (int j = g * G; j < (g + 1) * G; j++) {
      float c = rintf((y[j] - zf) * inv);
      if (!(c >= 0.0f)) c = 0.0f;
      if (c > (float)(L - 1)) c = (float)(L - 1);
      codes[j] = (uint8_t)c;
    }
  }
  return status;
}

int oq_quantize_rows(const uint16_t* X, int64_t n, int base, int L, int G,
                     const uint32_t* sign_words, const float* tau32,
                     uint8_t* codes, uint16_t* meta) {
  int status = OQ_OK;
  if (base < 0 || base > 2) return OQ_EINVAL;
  int ng = base != 1 ? 128 / G : 1;
  if (base != 1 && (G <= 0 || 128 % G)) return OQ_EINVAL;
#pragma omp parallel for schedule(static) reduction(min : status)
  for (int64_t r = 0; r < n; r++) {
    int st = base == 0 ? oq_affine_row(X + r * 128, L, G, codes + r * 128, meta + r * 2 * ng)
           : base == 1 ? oq_tq_row(X + r * 128, sign_words, L, tau32, codes + r * 128, meta + r)
                       : oq_rotaffine_row(X + r * 128, sign_words, L, G, codes + r * 128, meta + r * 2 * ng);
    if (st < status) status = st;
  }
  return status;
}

/* ---------------------------------------------------- mixed-radix packing -- */

int oq_symbol_digits(int L) {
  switch (L) {
    case 3: return 5;   /* 3^5 = 243 <= 2^8   : 1.600 b/value */
    case 4: return 4;   /* 4^4 = 256  = 2^8   : 2.000 b/value */
    case 5: return 3;   /* 5^3 = 125 <= 2^7   : 2.333 b/value */
    case 6: return 5;   /* 6^5 = 7776 <= 2^13 : 2.600 b/value */
    case 2: return 8;   /* 2^8 = 256          : 1.000 b/value */
    case 7: return 7;   /* 7^7 = 823543 <= 2^20 : 2.857 b/value (the paper gives no 7-level packing) */
    case 8: return 2;   /* 8^2 = 64 = 2^6     : 3.000 b/value */
    case 16: return 2;  /* 16^2 = 256 = 2^8   : 4.000 b/value */
    default: return 0;
  }
}

int oq_symbol_bits(int L, int nd) {
  uint64_t p = 1;
  for (int i = 0; i < nd; i++) p *= (uint64_t)L;
  int w = 0;
  while (((uint64_t)1 << w) < p) w++;
  return w;
}

int64_t oq_line_bits(int L, int nvalues) {
  int n = oq_symbol_digits(L);
  if (!n) return -1;
  int64_t b = (int64_t)(nvalues / n) * oq_symbol_bits(L, n);
  if (nvalues % n) b += oq_symbol_bits(L, nvalues % n);
  return b;
}

int64_t oq_tile_bytes(int L) {
  int64_t kb = 64 * oq_line_bits(L, 128), vb = 128 * oq_line_bits(L, 64);
  int64_t bits = kb > vb ? kb : vb;
  int64_t bytes = (bits + 7) / 8;
  return (bytes + 15) / 16 * 16;
}

static void put_bits(uint8_t* out, int64_t* pos, uint64_t v, int w) {
  for (int b = 0; b < w; b++, (*pos)++)
    if ((v >> b) & 1u) out[*pos >> 3] |= (uint8_t)(1u << (*pos & 7));
}

/* One line of nvalues codes (stride between consecutive codes) as symbols
 * p = 0..S-1; segment j carries the symbols p = j, j+4, j+8, ... */
static void put_segment(uint8_t* out, int64_t* pos, const uint8_t* line, int64_t stride,
                        int nvalues, int L, int j) {
  int n = oq_symbol_digits(L);
  int S = (nvalues + n - 1) / n;
  for (int p = j; p < S; p += 4) {
    int nd = nvalues - n * p < n ? nvalues - n * p : n;
    uint64_t v = 0, w = 1;
    for (int i = 0; i < nd; i++, w *= (uint64_t)L) v += (uint64_t)line[(int64_t)(n * p + i) * stride] * w;
    put_bits(out, pos, v, oq_symbol_bits(L, nd));
  }
}

int oq_pack_tile(const uint8_t* kcodes, const uint8_t* vcodes, int L,
                 uint8_t* kbody, uint8_t* vbody) {
  if (!oq_symbol_digits(L)) return OQ_EINVAL;
  for (int i = 0; i < 64 * 128; i++)
    if (kcodes[i] >= L || vcodes[i] >= L) return OQ_EINVAL;
  int64_t tb = oq_tile_bytes(L);
  memset(kbody, 0, (size_t)tb);
  memset(vbody, 0, (size_t)tb);
  int64_t pos = 0;
  for (int j = 0; j < 4; j++)                 /* K: a line is a token row */
    for (int t = 0; t < 64; t++) put_segment(kbody, &pos, kcodes + t * 128, 1, 128, L, j);
  pos = 0;
  for (int j = 0; j < 4; j++)                 /* V: a line is a channel column */
    for (int c = 0; c < 128; c++) put_segment(vbody, &pos, vcodes + c, 128, 64, L, j);
  return OQ_OK;
}

/* ------------------------------------------------------- dequantization -- */

void oq_affine_dequant_rows(const uint8_t* codes, const uint16_t* meta, int64_t n, int G, float* out) {
  int ng = 128 / G;
  for (int64_t r = 0; r < n; r++)
    for (int j = 0; j < 128; j++) {
      const uint16_t* m = meta + (r * ng + j / G) * 2;
      out[r * 128 + j] = fmaf((float)codes[r * 128 + j], oq_f16_to_f32(m[0]), oq_f16_to_f32(m[1]));
    }
}

void oq_tq_dequant_rows(const uint8_t* codes, const uint16_t* rho, int64_t n,
                        const uint32_t* sign_words, const float* mu32, double* out) {
  for (int64_t r = 0; r < n; r++) {
    double y[128];
    double rf = (double)oq_f16_to_f32(rho[r]);
    for (int i = 0; i < 128; i++) y[i] = rf * (double)mu32[codes[r * 128 + i]];
    for (int h = 1; h < 128; h <<= 1)         /* H is symmetric and H H = 128 I */
      for (int i = 0; i < 128; i++)
        if (!(i & h)) {
          double p = y[i], q = y[i + h];
          y[i] = p + q;
          y[i + h] = p - q;
        }
    for (int i = 0; i < 128; i++) out[r * 128 + i] = (sign_bit(sign_words, i) ? -y[i] : y[i]) / 128.0;
  }
}

/* Inverse of the rotation: x = diag(sign) H (16 y) / 128 = diag(sign) H y / 8,
 * with y = fmaf(c, scale, zero) in fp32 and the transform in double. */
void oq_rotaffine_dequant_rows(const uint8_t* codes, const uint16_t* meta, int64_t n, int G,
                               const uint32_t* sign_words, double* out) {
  int ng = 128 / G;
  for (int64_t r = 0; r < n; r++) {
    double y[128];
    for (int j = 0; j < 128; j++) {
      const uint16_t* m = meta + (r * ng + j / G) * 2;
      y[j] = (double)fmaf((float)codes[r * 128 + j], oq_f16_to_f32(m[0]), oq_f16_to_f32(m[1]));
    }
    for (int h = 1; h < 128; h <<= 1)
      for (int i = 0; i < 128; i++)
        if (!(i & h)) {
          double p = y[i], q = y[i + h];
          y[i] = p + q;
          y[i + h] = p - q;
        }
    for (int i = 0; i < 128; i++) out[r * 128 + i] = (sign_bit(sign_words, i) ? -y[i] : y[i]) / 8.0;
  }
}

/* ----------------------------------------------------------- indicators -- */

static double dot_d(const float* a, const float* b, int d) {
  double s = 0.0;
  for (int j = 0; j < d; j++) s += (double)a[j] * (double)b[j];
  return s;
}

int oq_score_hidden(int indicator, const float* h, int m, int64_t T, int d, double* s) {
  if (indicator < 0 || indicator > 3 || m < 0 || d <= 0 || T < 0) return OQ_EINVAL;
  if ((indicator == 0 || indicator == 3) && m < 1) return OQ_EINVAL;
  int status = OQ_OK;
  for (int64_t t = 0; t < T; t++) {
    const float* last = h + ((int64_t)m * T + t) * d;
    double v = 0.0;
    if (indicator == 0 || indicator == 3) {
      for (int k = 1; k <= m; k++) {
        const float* a = h + ((int64_t)k * T + t) * d;
        const float* b = h + ((int64_t)(k - 1) * T + t) * d;
        if (indicator == 0) {                 /* ||h^(l) - h^(l-1)||_2 */
          double q = 0.0;
          for (int j = 0; j < d; j++) {
            double e = (double)a[j] - (double)b[j];
            q += e * e;
          }
          v += sqrt(q);
        } else {                              /* 1 - cos(h^(l), h^(l-1)) */
          double na = sqrt(dot_d(a, a, d)), nb = sqrt(dot_d(b, b, d));
          double c = (na > 0.0 && nb > 0.0) ? dot_d(a, b, d) / (na * nb) : 0.0;
          v += 1.0 - c;
        }
      }
      v /= m;
    } else if (indicator == 1) {
      v = sqrt(dot_d(last, last, d));
    } else {
      double mean = 0.0;
      for (int j = 0; j < d; j++) mean += last[j];
      mean /= d;
      for (int j = 0; j < d; j++) v += ((double)last[j] - mean) * ((double)last[j] - mean);
      v /= d;
    }
    if (!isfinite(v)) status = OQ_ENAN;
    s[t] = v;
  }
  return status;
}

int oq_score_kv_norm(const float* X, int R, int64_t T, double* s) {
  if (R <= 0 || T < 0) return OQ_EINVAL;
  for (int64_t t = 0; t < T; t++) {
    double q = 0.0;
    for (int r = 0; r < R; r++) q += dot_d(X + ((int64_t)r * T + t) * 128, X + ((int64_t)r * T + t) * 128, 128);
    s[t] = sqrt(q);
  }
  return OQ_OK;
}

void oq_bf16_to_f32_n(const uint16_t* h, int64_t n, float* out) {
  for (int64_t i = 0; i < n; i++) {
    uint32_t u = (uint32_t)h[i] << 16;
    memcpy(&out[i], &u, 4);
  }
}

/* ------------------------------------------------------------ attention -- */

void oq_attention(const double* q, int nq, const double* k, const double* v,
                  int64_t n, int D, double* out) {
#pragma omp parallel for schedule(static)
  for (int h = 0; h < nq; h++) {
    double* lg = (double*)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    double m = -INFINITY, sum = 0.0;
    for (int64_t t = 0; t < n; t++) {
      double d = 0.0;
      for (int c = 0; c < D; c++) d += q[h * D + c] * k[t * D + c];
      lg[t] = d / sqrt((double)D);
      if (lg[t] > m) m = lg[t];
    }
    for (int c = 0; c < D; c++) out[h * D + c] = 0.0;
    for (int64_t t = 0; t < n; t++) {
      double p = exp(lg[t] - m);
      sum += p;
      for (int c = 0; c < D; c++) out[h * D + c] += p * v[t * D + c];
    }
    for (int c = 0; c < D; c++) out[h * D + c] /= sum;
    free(lg);
  }
}

/* Many independent (sequence, layer, kv head) units at once, OpenMP across
 * the units (each unit's heads in one thread): the same arithmetic as
 * oq_attention per unit.  Unit u: q[u] [nq][D], k[u], v[u] [n[u]][D],
 * out[u] [nq][D]. */
void oq_attention_units(int n_units, const double* const* q, int nq, const double* const* k,
                        const double* const* v, const int64_t* n, int D, double* const* out) {
#pragma omp parallel for schedule(dynamic)
  for (int u = 0; u < n_units; u++) oq_attention(q[u], nq, k[u], v[u], n[u], D, out[u]);
}

int oq_max_threads(void) { return omp_get_max_threads(); }

/* ------------------------------------------------- array helpers (tests) -- */

void oq_f32_to_f16_n(const float* x, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; i++) out[i] = oq_f32_to_f16(x[i]);
}

void oq_f16_to_f32_n(const uint16_t* h, int64_t n, float* out) {
  for (int64_t i = 0; i < n; i++) out[i] = oq_f16_to_f32(h[i]);
}

void oq_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
