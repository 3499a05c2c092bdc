/* semkv_oracle.h -- plain, slow CPU oracle of the SemKV hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load this library.  It shares no code,
 * header, table or constant generator with the HIP library.
 *
 * Every function states the passage of the paper (SemKV, arxiv 2608.28911)
 * it follows.  Where the paper is silent the reading taken is named
 * "reading Rn"; the list of readings is kept with the design notes.
 */
#ifndef SEMKV_ORACLE_H
#define SEMKV_ORACLE_H
#include <stdint.h>
#include <stddef.h>

#define OQ_OK 0
#define OQ_EINVAL (-1)
#define OQ_ENAN (-4)

/* IEEE binary16 <-> binary32, round-to-nearest-even, subnormals kept. */
uint16_t oq_f32_to_f16(float x);
float oq_f16_to_f32(uint16_t h);

/* Eq. (4): K = floor(r T) with r = r_num / r_den, in integers. */
int64_t oq_top_count(int64_t T, int64_t r_num, int64_t r_den);
/* Sec. 3.7 / Alg. 2: round(r n), nearest integer, ties to even (reading R3). */
int64_t oq_block_count(int64_t n, int64_t r_num, int64_t r_den);

/* Eq. (4)-(5): flag[i] = 1 iff token i is among the K highest scores.
 * Order: larger score first, equal scores by lower index (reading R4);
 * -0 equals +0.  Returns OQ_ENAN on a NaN score.  Ranks exactly k tokens. */
int oq_rank_k(const float* s, int64_t T, int64_t k, uint8_t* flag);

/* Affine base quantizer (Sec. 4.1): per group of G channels of one 128-dim
 * row, two fp16 parameters.  codes[128] in [0, L-1]; meta[2*(128/G)] =
 * {scale, zero} per group as fp16 bits.  A scale whose fp16 rounding
 * overflows (2 levels, a range above 65504) is stored as 65504 (reading
 * R18), so finite input always gives finite parameters. */
int oq_affine_row(const uint16_t* x, int L, int G, uint8_t* codes, uint16_t* meta);

/* Lloyd-Max codebook of the unit Gaussian with L levels (Sec. 4.9), by the
 * classical Lloyd iteration in double precision.  mu[L], tau[L-1]. */
int oq_lloyd_max(int L, double* mu, double* tau, double* mse);

/* TurboQuant-MSE base (Sec. 4.9): random-sign Hadamard rotation, one fp16
 * scalar (the row norm) per row, Lloyd-Max threshold codes.  sign_words: 4
 * uint32, bit i set = channel i negated.  tau32[L-1]: fp32 thresholds. */
int oq_tq_row(const uint16_t* x, const uint32_t* sign_words, int L, const float* tau32,
              uint8_t* codes, uint16_t* rho);

/* Affine base under a Hadamard rotation (Sec. 4.1, Sec. 4.9): the affine
 * quantizer of y = H diag(sign) x / 16 (H the unnormalized Sylvester matrix),
 * per group of G rotated coordinates; zero = fp16(min y), scale =
 * fp16(max(0, (max y - zero) / (L-1))), each saturated to +-65504 where the
 * fp16 rounding overflows (reading R18).  meta as oq_affine_row. */
int oq_rotaffine_row(const uint16_t* x, const uint32_t* sign_words, int L, int G,
                     uint8_t* codes, uint16_t* meta);

/* Many rows at once (OpenMP across rows).  base 0 affine, 1 tq, 2 rotated
 * affine.  meta: affine [n][128/G][2] fp16 bits; tq [n] fp16 bits. */
int oq_quantize_rows(const uint16_t* X, int64_t n, int base, int L, int G,
                     const uint32_t* sign_words, const float* tau32,
                     uint8_t* codes, uint16_t* meta);

/* Mixed-radix packing (Sec. 4.1). */
int oq_symbol_digits(int L);                 /* codes per full symbol */
int oq_symbol_bits(int L, int ndigits);      /* smallest w with 2^w >= L^ndigits */
int64_t oq_line_bits(int L, int nvalues);    /* bits of one line of nvalues codes */
int64_t oq_tile_bytes(int L);                /* bytes of one packed K or V body */
/* Pack one 64-slot tile.  kcodes, vcodes: [64 slots][128 channels]; unused
 * slots hold code 0.  kbody, vbody: oq_tile_bytes(L) bytes each. */
int oq_pack_tile(const uint8_t* kcodes, const uint8_t* vcodes, int L,
                 uint8_t* kbody, uint8_t* vbody);

/* Dequantization. affine: x = fmaf(c, scale, zero) in fp32.
 * tq: x = (1/128) * diag(sign) * H * (rho * mu[c]) in double. */
void oq_affine_dequant_rows(const uint8_t* codes, const uint16_t* meta, int64_t n, int G, float* out);
void oq_tq_dequant_rows(const uint8_t* codes, const uint16_t* rho, int64_t n,
                        const uint32_t* sign_words, const float* mu32, double* out);

/* rotated affine: x = diag(sign) H y / 8, y = fmaf(c, scale, zero) in fp32,
 * the transform in double. */
void oq_rotaffine_dequant_rows(const uint8_t* codes, const uint16_t* meta, int64_t n, int G,
                               const uint32_t* sign_words, double* out);

/* Token-importance indicators (Sec. 3.3), in double.  Hidden-state family
 * over the states h[k][t][j] of the last m+1 layers (k = 0..m, layer L-m+k;
 * d channels): 0 delta-norm, Eq. (3): (1/m) sum_{k=1..m} ||h_k - h_{k-1}||_2;
 * 1 norm ||h_m||_2; 2 variance (1/d) sum_j (h_m[j] - mean)^2 (population);
 * 3 cosine-delta (1/m) sum_k (1 - cos(h_k, h_{k-1})), cos taken as 0 when a
 * norm is 0.  m >= 1 for 0 and 3, m >= 0 otherwise.  s[T]. */
int oq_score_hidden(int indicator, const float* h, int m, int64_t T, int d, double* s);
/* KV-norm family: s[t] = sqrt(sum_r sum_j X[r][t][j]^2) over R rows of 128
 * channels per token (every layer and kv head of the key or value cache). */
int oq_score_kv_norm(const float* X, int R, int64_t T, double* s);
/* bfloat16 bits -> binary32 (exact) */
void oq_bf16_to_f32_n(const uint16_t* h, int64_t n, float* out);

/* Decode attention (the consumer of the cache, Sec. 3.1 / Alg. 1):
 * out[h] = softmax(q_h . k_t / sqrt(D)) . v over all n tokens, in double. */
void oq_attention(const double* q, int nq, const double* k, const double* v,
                  int64_t n, int D, double* out);

/* oq_attention of many independent units, OpenMP across the units (timing
 * runs on every host core).  Unit u: q[u] [nq][D], k[u], v[u] [n[u]][D]. */
void oq_attention_units(int n_units, const double* const* q, int nq, const double* const* k,
                        const double* const* v, const int64_t* n, int D, double* const* out);

/* OpenMP threads of the row-parallel oracle calls (timing runs), and the
 * number a parallel region uses. */
void oq_set_threads(int n);
int oq_max_threads(void);

/* Array forms of the conversions (used by the pins). */
void oq_f32_to_f16_n(const float* x, int64_t n, uint16_t* out);
void oq_f16_to_f32_n(const uint16_t* h, int64_t n, float* out);

#endif
