/* semkv.h -- C ABI of the SemKV hot path on MI355X (gfx950).
 *
 * SemKV (arxiv 2608.28911) keeps every token of the KV cache and gives each
 * token one of two adjacent fractional precisions by an importance ranking:
 * the top r fraction of tokens gets L_hi levels, the rest L_lo levels
 * (Sec. 3.4, Eq. 4-5); K and V of every layer and KV head of a token share the
 * token's precision (Sec. 3.5, Eq. 7, Fig. 5).  Generated tokens are
 * quantized block-exactly in 64-token blocks (Sec. 3.7, Alg. 2).  Decoding
 * attends over the mixed-precision cache.
 *
 * Conventions for every call:
 *  - Pointers named as device pointers are device memory owned by the caller;
 *    the library never allocates, frees or synchronizes, and enqueues all of
 *    its work on the stream it is given (a hipStream_t).
 *  - Arguments are validated on the host before anything is enqueued; a
 *    failed validation returns a negative status and enqueues nothing.
 *  - Data errors found on the device (a NaN score, a non-finite K/V value) are
 *    OR-ed into the caller's device status word (bit 0: NaN score, bit 1:
 *    non-finite K/V, bit 2: slot index outside [0, T)); read it after the
 *    stream is synchronized.
 *  - A semkv_cache is a plain host struct: configuration, device pointers and
 *    host-side counts.  Calls on one cache must be serialized on one stream.
 *    Calls on different caches are independent.
 *  - fp16 means IEEE binary16 stored as 16-bit words; fp32 is IEEE binary32.
 */
#ifndef SEMKV_H
#define SEMKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SEMKV_OK = 0,
  SEMKV_EINVAL = -1,       /* bad argument: null pointer, bad shape, bad ratio */
  SEMKV_EUNSUPPORTED = -2, /* level count, group or head size not supported   */
  SEMKV_ECAPACITY = -3,    /* pool, prompt or tail capacity would be exceeded */
  SEMKV_ENAN = -4,         /* reserved for status-word reports                */
  SEMKV_EHIP = -5,         /* a HIP runtime call failed                       */
  SEMKV_ESTATE = -6        /* call out of order (e.g. commit before append)   */
};

enum { SEMKV_BASE_AFFINE = 0, SEMKV_BASE_TQ = 1, SEMKV_BASE_ROT_AFFINE = 2 };
enum { SEMKV_STATUS_NAN_SCORE = 1, SEMKV_STATUS_NONFINITE_KV = 2, SEMKV_STATUS_BAD_INDEX = 4 };

/* Configuration of one cache.
 *  base:   SEMKV_BASE_AFFINE -- per group of `group` channels, an asymmetric
 *          affine quantizer with two fp16 parameters (scale, zero) (Sec. 4.1);
 *          L_hi, L_lo in {6, 5} (2.585/2.322 bits) or any two of {3,4,5,6}.
 *          A parameter whose fp16 rounding overflows (the scale at 2 levels
 *          over a range above 65504; zero or scale of the rotated affine base)
 *          is stored as +-65504 and the codes follow the stored pair, so
 *          finite K/V always give finite parameters.
 *          SEMKV_BASE_TQ -- TurboQuant-MSE: random-sign Hadamard rotation and a
 *          Lloyd-Max codebook of the unit Gaussian, one fp16 scalar (the row
 *          norm) per row (Sec. 4.9); L_hi, L_lo in {4, 3} (2.0/1.585 bits).
 *          SEMKV_BASE_ROT_AFFINE -- the affine quantizer of the rotated row
 *          y = H diag(sign) x / 16 (H the unnormalized 128-point Sylvester
 *          Hadamard matrix), the integer-level quantization with a Hadamard
 *          rotation of Sec. 4.1 and Sec. 4.9: per group of `group` rotated
 *          coordinates zero = fp16(min y), scale = fp16((max y - zero)/(L-1))
 *          (at least 0); x is reconstructed as diag(sign) H y_hat / 8.
 *          L_hi, L_lo in {6, 5} or {5, 4}.
 *  group:  affine metadata group in {32, 64, 128}; must be 128 for tq.
 *  r_num/r_den: high-precision fraction r (Eq. 4), 0 <= r <= 1.
 *  block:  deferred block size B of Alg. 2; must be 64.
 *  head_dim must be 128, n_q_heads = 4 * n_kv_heads (GQA group of 4).
 *  max_prompt, max_new: capacity in tokens per sequence (together at most
 *  2^29).  batch * n_layers at most 65535, n_layers at most 128. */
typedef struct semkv_config {
  int32_t n_layers, n_kv_heads, n_q_heads, head_dim, batch;
  int32_t base, L_hi, L_lo, group;
  int32_t r_num, r_den, block;
  int64_t max_prompt, max_new;
} semkv_config;

/* Sizes derived from a configuration (all in bytes unless named otherwise).
 * Storage layout (the packed format):
 *  pools:  [batch][n_layers][n_kv_heads] units of unit_stride bytes; a unit is
 *          cap_hi_tiles high-precision records then cap_lo_tiles
 *          low-precision records.  A record holds 64 token slots:
 *            K body (tile_bytes)  V body (tile_bytes)  K meta  V meta
 *          Bodies hold mixed-radix symbols (Sec. 4.1): a symbol packs n codes
 *          of base L as sum_i c_i L^i in the least number of bits (n = 5, 4,
 *          3, 5 for L = 3, 4, 5, 6: 8, 8, 7, 13 bits).  A K line is one token
 *          row (128 channels), a V line one channel column over the 64 slots;
 *          segment j of a line is its symbols p = j, j+4, j+8, ...; a body is
 *          segment 0 of every line, then segments 1, 2, 3, LSB-first, zero
 *          padded to a multiple of 16 bytes.  Meta: affine and rotated
 *          affine, per group g and slot s, fp16 {scale, zero} at [g][s]; tq,
 *          fp16 rho at [s].
 *          Slots of a pool are in increasing token position, prompt tokens
 *          first, then each closed generation block.
 *  tail:   fp16 [batch][n_layers][n_kv_heads][2 (K,V)][64][128], the
 *          generated tokens not yet quantized (Alg. 2).
 *  tail_scores: fp32 [batch][64].
 *  flags:  uint32 [batch][flag_words]: bit i%32 of word i/32 is 1 iff token i
 *          has the high precision (the 1-bit per-token flag of Sec. 4.1);
 *          then (from word batch*flag_words rounded up to a multiple of 64)
 *          the ranker's scratch for prompts longer than 4096 tokens, per
 *          sequence three histograms of 2048, 2048 and 1024 words, which are
 *          zero again when each semkv_rank call ends, 16 words of selection
 *          state and two counts per 4096-token chunk.  flag_bytes covers both.
 *  workspace: scratch of semkv_decode_attn. */
typedef struct semkv_sizes {
  size_t pool_bytes, tail_bytes, tail_score_bytes, flag_bytes, workspace_bytes;
  int64_t flag_words, cap_hi_tiles, cap_lo_tiles, unit_stride;
  int64_t tile_bytes_hi, tile_bytes_lo, meta_bytes, record_bytes_hi, record_bytes_lo;
} semkv_sizes;

/* One cache.  Filled by semkv_cache_init; the counts are updated by the calls
 * below and may be read (not written) by the caller. */
typedef struct semkv_cache {
  semkv_config cfg;
  semkv_sizes sz;
  uint8_t* pools;             /* device */
  uint16_t* tail;             /* device, fp16 */
  float* tail_scores;         /* device */
  uint32_t* flags;            /* device */
  const uint32_t* signs;      /* device [n_layers][n_kv_heads][4] (bases 1, 2) or NULL */
  int32_t* status;            /* device status word */
  float mu_hi[16], tau_hi[16], mu_lo[16], tau_lo[16];  /* tq codebooks */
  int64_t n_prompt;           /* prompt tokens quantized (same for every sequence) */
  int64_t n_hi, n_lo;         /* rows in the high / low pool of every unit */
  int32_t n_scored;           /* tail rows whose score was committed */
  uint32_t appended[4];       /* layers that appended the current tail row */
} semkv_cache;

/* Message for a status code; never NULL. */
const char* semkv_strerror(int status);

/* Sizes of every buffer for `cfg`; validates the configuration. */
int semkv_cache_sizes(const semkv_config* cfg, semkv_sizes* out);

/* Lloyd-Max codebook of the unit Gaussian with L levels (2 <= L <= 16),
 * computed on the host by bisection on the optimality conditions and rounded
 * to fp32: mu[L] reconstruction points, tau[L-1] thresholds (Sec. 4.9). */
int semkv_tq_codebook(int L, float* mu, float* tau);

/* Initialize `c` over caller buffers sized by semkv_cache_sizes.  The buffers
 * need no clearing except `flags` and `status`, which must be zero.
 * signs: device uint32 [n_layers][n_kv_heads][4]; bit i set = channel i of
 * that head is negated before the Hadamard transform (the rotated bases, tq
 * and rotated affine; NULL for the affine base). */
int semkv_cache_init(semkv_cache* c, const semkv_config* cfg, void* pools, void* tail,
                     float* tail_scores, uint32_t* flags, const uint32_t* signs,
                     int32_t* status);

/* Eq. (4) sizes of the slot lists semkv_rank writes for a prompt of T tokens
 * (1 <= T <= max_prompt): n_hi = floor(r T) high-precision tokens, n_lo =
 * T - n_hi, per sequence.  Pure host arithmetic; enqueues nothing. */
int semkv_rank_sizes(const semkv_cache* c, int64_t T, int64_t* n_hi, int64_t* n_lo);

/* Eq. (4)-(5) for every sequence: K = floor(r T); the K tokens with the
 * highest scores get the high precision, equal scores ordered by lower token
 * index, -0 equal to +0.  scores: device fp32 [batch][T].  Writes the flag
 * bits of tokens [0, T) and the slot lists hi_idx: device int32
 * [batch][K] (ascending), lo_idx: device int32 [batch][T-K] (ascending); a
 * list with no entries may be NULL.
 * A NaN score sets SEMKV_STATUS_NAN_SCORE.  Prompts of up to 4096 tokens take
 * one launch (one workgroup per sequence); longer ones take five, one
 * workgroup per 4096-token chunk, with the scratch at the end of `flags`.
 * Calls that overlap on one cache race. */
int semkv_rank(semkv_cache* c, const float* scores, int64_t T, int32_t* hi_idx,
               int32_t* lo_idx, hipStream_t stream);

/* Eq. (7) for the prompt (Alg. 1): quantize K and V of token hi_idx[b][i]
 * (lo_idx[b][i]) with L_hi (L_lo) levels into slot i of the high (low) pool of
 * every (b, layer, kv head) unit and pack them.  K, V: device fp16; element
 * (b, h, t, d) at b*sB + h*sH + t*sT + d (+ l*sL when layer == -1, which
 * quantizes every layer).  T must be the value given to semkv_rank.
 * Non-finite K/V sets SEMKV_STATUS_NONFINITE_KV. */
int semkv_quantize_pack(semkv_cache* c, int32_t layer, const uint16_t* K, const uint16_t* V,
                        int64_t sL, int64_t sB, int64_t sH, int64_t sT, int64_t T,
                        const int32_t* hi_idx, const int32_t* lo_idx, hipStream_t stream);

/* Alg. 2 (append): store the current generated token's K and V of `layer` at
 * fp16 in the tail.  k_new, v_new: device fp16 [batch][n_kv_heads][128]
 * (with layer == -1: [n_layers][batch][n_kv_heads][128]). */
int semkv_append_kv(semkv_cache* c, int32_t layer, const uint16_t* k_new, const uint16_t* v_new,
                    hipStream_t stream);

/* Alg. 2 (score): record the current token's score (device fp32 [batch]).
 * Every layer must have appended the token.  When 64 scores are held the
 * block closes: in each sequence exactly round(r*64) tokens of the block (the
 * highest scores, ties to the lower index) are quantized with L_hi, the rest
 * with L_lo, and appended to the pools. */
int semkv_append_commit(semkv_cache* c, const float* score_new, hipStream_t stream);

/* Alg. 2 (end of turn): close a partial block of n < 64 scored tokens with
 * round(r*n) high-precision tokens (nearest integer, ties to even). */
int semkv_flush(semkv_cache* c, hipStream_t stream);

/* Empty the cache for a new prompt: clear the flag bitmap (a kernel on
 * `stream`) and every host-side count; pools, tail and status word are left
 * as they are (their contents are rewritten before they are read again).
 * Multi-turn dialogue (Sec. 3.7, Sec. 4.6): each turn resets the cache and
 * applies the prompt procedure to the accumulated conversation (semkv_rank +
 * semkv_quantize_pack), then block-exact generation and semkv_flush at the
 * turn's end. */
int semkv_cache_reset(semkv_cache* c, hipStream_t stream);

/* Bytes of workspace semkv_decode_attn needs for this cache's current counts
 * (semkv_sizes.workspace_bytes bounds it for every count). */
int semkv_workspace_bytes(const semkv_cache* c, size_t* bytes);

/* Decode attention of one layer over the mixed-precision cache: the cache
 * the method builds before decoding is what attention reads at every decoding
 * step (Sec. 3.1, Fig. 1; Alg. 1, last step), every token at its own
 * precision, its K and V of every layer and KV head at the same level (Sec.
 * 3.5, Fig. 5), and the latest partial block of generated tokens at full
 * precision (Alg. 2).  For each sequence b and query head h (KV head h/4),
 * out[b][h] = softmax(q[b][h] . k_t / sqrt(128)) . v_t over every token t of
 * the sequence: both pools (dequantized on the fly) and the fp16 tail rows
 * appended so far, including this layer's current token if appended.
 * q: device fp16 [batch][n_q_heads][128]; out: device fp32, same shape.
 * layer == -1: every layer in one launch, q and out [n_layers][batch]
 * [n_q_heads][128] (for queries known up front, as in a benchmark; a model
 * computes layer l's query from layer l-1's output); every layer must have
 * appended the current token, or none (else SEMKV_ESTATE).
 * workspace: device, ws_bytes >= semkv_workspace_bytes(); it starts with
 * one counter per (layer, sequence, kv head) of the cache -- sized for every
 * layer whichever kind of launch -- that must be zero before the first call
 * (allocate it zeroed); every call leaves them zero again.  One workspace may
 * serve successive calls of either kind on one stream, not concurrent
 * calls. */
int semkv_decode_attn(const semkv_cache* c, int32_t layer, const uint16_t* q, float* out,
                      void* workspace, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): semkv_decode_attn without
 * a workspace, same arguments, semantics and results otherwise.  The split
 * counters and partials live in an 8 MiB device array of the library (1 MiB
 * of counters, one per (layer, sequence, kv head) of the cache on its own
 * 256-byte line: at most 4096; the rest for the partials, 2112 bytes per split
 * of a (layer, sequence, kv head): a launch needs about max(256 compute units,
 * its units) of them, so one layer up to ~3400 (sequence, kv head) units).  A
 * cache or launch beyond either bound returns SEMKV_ECAPACITY before anything
 * is enqueued.  The array is held by each GPU the library runs on until the
 * process ends; the first call on a GPU also enqueues a kernel that clears its
 * counters.  The call allocates and frees nothing.  All calls on one GPU share
 * the array: calls that overlap in time on one GPU (other streams, other
 * threads, not serialized) race and give wrong results; serialize them. */
int semkv_decode_attn_noalloc(const semkv_cache* c, int32_t layer, const uint16_t* q, float* out,
                              hipStream_t stream);

/* Alg. 2, append and attend in one launch: store this layer's K and V of the
 * current generated token in the fp16 tail (exactly as semkv_append_kv with
 * this layer) and compute semkv_decode_attn over the cache including it.
 * k_new, v_new: device fp16 [batch][n_kv_heads][128]; q, out, workspace as
 * for semkv_decode_attn.  SEMKV_ESTATE if this layer already appended the
 * current token or a block of 64 scores awaits its close; SEMKV_ECAPACITY
 * past max_prompt + max_new tokens. */
int semkv_append_decode(semkv_cache* c, int32_t layer, const uint16_t* k_new, const uint16_t* v_new,
                        const uint16_t* q, float* out, void* workspace, size_t ws_bytes,
                        hipStream_t stream);

/* Test and inspection aid: the values decode attention reads from the pools
 * of `layer`, dequantized to fp32 (affine: fmaf(c, scale, zero); rotated
 * affine: sign . H y / 8 of the affine values y; tq: sign . H (rho mu[c]) /
 * 128, the transforms summed in fp32).  k_hat, v_hat: device fp32
 * [batch][n_kv_heads][n_hi + n_lo][128], 16-byte aligned: rows 0 .. n_hi-1
 * are the high pool's slots, then the low pool's, each in slot order
 * (ascending token position, prompt first, then closed blocks; the flag
 * bitmap gives each slot's token).  The fp16 tail is not included. */
int semkv_dequant(const semkv_cache* c, int32_t layer, float* k_hat, float* v_hat, hipStream_t stream);

/* Token-importance indicators (Sec. 3.3): device fp32 scores [batch][T] for
 * semkv_rank (which uses only their order), from tensors the model already
 * computes.  Hidden-state family, over the hidden states of the last m+1
 * layers (state k = layer L-m+k, k = 0..m):
 *   SEMKV_IND_DELTA_NORM    Eq. (3): (1/m) sum_{k=1..m} ||h_k - h_{k-1}||_2 (m >= 1)
 *   SEMKV_IND_NORM          ||h_m||_2
 *   SEMKV_IND_VARIANCE      (1/d) sum_j (h_m[j] - mean)^2 (population variance)
 *   SEMKV_IND_COSINE_DELTA  (1/m) sum_k (1 - cos(h_k, h_{k-1})), cos = 0 when a
 *                           state is all zero (m >= 1)
 * hidden: device, fp16 (SEMKV_DTYPE_F16) or bfloat16 (SEMKV_DTYPE_BF16);
 * element (k, b, t, j) at k*s_state + b*s_batch + t*s_token + j (elements;
 * the norm and variance read state m only, m may be 0).  d_model: a multiple
 * of 8, at most 8192; strides multiples of 8; hidden 16-byte aligned;
 * batch * T below 2^33 (one wave per token).
 * Sums run in fp32 (the score's relative error is below 1e-5 for d <= 8192).
 * A non-finite state gives a non-finite score, which semkv_rank reports. */
enum { SEMKV_IND_DELTA_NORM = 0, SEMKV_IND_NORM = 1, SEMKV_IND_VARIANCE = 2, SEMKV_IND_COSINE_DELTA = 3 };
enum { SEMKV_DTYPE_F16 = 0, SEMKV_DTYPE_BF16 = 1 };
int semkv_score_hidden(int32_t indicator, const void* hidden, int32_t dtype, int32_t m, int32_t batch,
                       int64_t T, int32_t d_model, int64_t s_state, int64_t s_batch, int64_t s_token,
                       float* scores, hipStream_t stream);

/* KV-norm family (Sec. 3.3: key-norm ||K_t||_2, value-norm ||V_t||_2): the
 * norm of token t's rows over every layer and kv head of `c`, from the fp16 K
 * (or V) tensors laid out as for semkv_quantize_pack with layer == -1:
 * element (l, b, h, t, j) at l*sL + b*sB + h*sH + t*sT + j.  scores: device
 * fp32 [batch][T]. */
int semkv_score_kv_norm(const semkv_cache* c, const uint16_t* X, int64_t sL, int64_t sB, int64_t sH,
                        int64_t sT, int64_t T, float* scores, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* SEMKV_H */
