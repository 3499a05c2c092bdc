// semkv_internal.h -- argument blocks and launchers shared by the host API
// (semkv_api.hip) and the kernels (rank.hip, quant.hip, decode.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "semkv_fmt.h"

namespace semkv {

// Per-pool view of the storage of one cache, as kernels need it.
struct PoolGeom {
  uint8_t* pools;          // device base of all units
  int64_t unit_stride;     // bytes per (b, layer, kv head) unit
  int64_t lo_offset;       // byte offset of the low pool inside a unit
  int32_t rec_bytes[2];    // record bytes of the high / low pool
  int32_t tile_bytes[2];   // body bytes of the high / low pool
  int32_t meta_bytes;      // bytes of one K or V metadata block
  int32_t L[2];            // levels of the high / low pool
  int32_t base, G, n_layers, n_kv_heads, batch;
  float tau[2][16];        // tq thresholds of the high / low pool
  const uint32_t* signs;   // tq sign masks [n_layers][n_kv_heads][4]
  int32_t* status;         // device status word
};

__host__ __device__ inline int64_t unit_offset(const PoolGeom& g, int b, int l, int h) {
  return ((int64_t(b) * g.n_layers + l) * g.n_kv_heads + h) * g.unit_stride;
}

struct RankArgs {
  const float* scores; int64_t T, K, ld_s;
  uint32_t* flags; int64_t flag_words;
  int32_t* hi_idx; int32_t* lo_idx;
  int32_t* status;
  uint32_t* scratch; int64_t scratch_words;   // per sequence, zero between calls
};

struct QuantArgs {
  PoolGeom g;
  const uint16_t* K; const uint16_t* V;
  int64_t sL, sB, sH, sT;
  int32_t layer0, n_layers_launched;
  const int32_t* idx[2];   // [batch][n_pool[p]]
  int64_t n_pool[2];
  int64_t T;               // tokens per sequence (slot lists index [0, T))
  int32_t max_tiles;
};

struct CloseArgs {
  PoolGeom g;
  const uint16_t* tail;    // [b][l][h][2][64][128]
  const float* tail_scores;// [b][64]
  int32_t n;               // scored rows in the block (1..64)
  int32_t k_hi;            // rows of the block that take the high precision
  int64_t n0[2];           // rows already in the high / low pool
  uint32_t* flags; int64_t flag_words; int64_t pos0;  // token position of tail row 0
};

struct AppendArgs {
  uint16_t* tail; const uint16_t* k; const uint16_t* v;
  int32_t layer0, n_layers_launched, n_layers, n_kv_heads, batch, slot;
};

struct DecodeArgs {
  PoolGeom g;
  uint16_t* tail;          // fp16 tail base
  const uint16_t* k_new;   // fused append: this layer's new K/V rows [b][kvh][128], or null
  const uint16_t* v_new;
  const uint16_t* q;       // [b][Hq][128]
  float* ws;               // partials [layer of the launch][b][kvh][nsplit][4][132]
  uint32_t* counters;      // [layer of the launch][b][kvh] finished-split counters, zero between calls
  float* out;              // [b][Hq][128]
  int32_t layer;           // first layer of the launch
  int32_t n_layers_launched; // layers of the launch (q, out, partials, counters: [layer][b]...)
  int64_t n_rows[2];       // rows in the high / low pool
  int32_t n_tail;          // fp16 tail rows visible to each layer (taken by the last split)
  int32_t nsplit;          // balanced runs of tiles per unit, one workgroup each
  float mu[2][16];         // tq codebooks
};

struct DequantArgs {
  PoolGeom g;
  int32_t layer;
  int64_t n_rows[2];       // rows in the high / low pool
  float mu[2][16];         // tq codebooks
  float* k_hat;            // [b][kvh][n_rows[0] + n_rows[1]][128]: high pool, then low pool
  float* v_hat;
};

struct HiddenArgs {
  const uint16_t* h;       // state k, sequence b, token t at k*s_state + b*s_batch + t*s_token
  int64_t s_state, s_batch, s_token;
  int32_t indicator, dtype, m, batch, d;
  int64_t T;
  float* scores;           // [batch][T]
};

struct KvNormArgs {
  const uint16_t* X;       // (l, b, h, t, :) at l*sL + b*sB + h*sH + t*sT
  int64_t sL, sB, sH, sT;
  int32_t n_layers, n_kv_heads, batch;
  int64_t T;
  float* scores;           // [batch][T]
};

constexpr int kPartial = 132;  // m, l, 2 pad, o[128]
// dwords between the finished-split counters of two (layer, sequence, kv
// head) units: one counter per 256-byte line, so the workgroups of different
// units do not queue their atomics on one line
constexpr int kCounterStride = 64;
constexpr int kMaxSplits = 256;   // splits per (sequence, kv head)
// buffer descriptor word 3 of a raw buffer of 32-bit elements (gfx9 family)
constexpr int kBufferWord3 = 0x00020000;

// Ranker scratch, per sequence, after the flag bitmaps in the flags buffer
// (zero at cache init and again after every semkv_rank call): three
// histograms (2048, 2048 and 1024 bins), 16 words of selection state, then
// two counts per chunk of kRankChunk tokens.
constexpr int kRankChunk = 4096;
constexpr int kRankH1 = 0, kRankH2 = 2048, kRankH3 = 4096, kRankState = 5120, kRankCounts = 5136;
__host__ __device__ constexpr int64_t rank_chunks(int64_t T) { return (T + kRankChunk - 1) / kRankChunk; }
__host__ __device__ constexpr int64_t rank_scratch_words(int64_t max_prompt) {
  return (kRankCounts + 2 * rank_chunks(max_prompt) + 63) / 64 * 64;
}
__host__ __device__ constexpr int64_t rank_scratch_offset(int64_t batch, int64_t flag_words) {
  return (batch * flag_words + 63) / 64 * 64;
}

int launch_rank(const RankArgs& a, int batch, hipStream_t s);
int launch_quantize(const QuantArgs& a, hipStream_t s);
int launch_append(const AppendArgs& a, hipStream_t s);
int launch_close(const CloseArgs& a, hipStream_t s);
int launch_dequant(const DequantArgs& a, hipStream_t s);
int launch_decode(const DecodeArgs& a, hipStream_t s);
int launch_score_hidden(const HiddenArgs& a, hipStream_t s);
int launch_kv_norm(const KvNormArgs& a, hipStream_t s);
// decode workgroups one compute unit holds at once for this cache's kernel,
// and the waves of one such workgroup (a wave takes every NW-th tile of a run)
int decode_blocks_per_cu(int base, int L_hi, int L_lo, int G);
int decode_waves(int base, int L_hi, int L_lo, int G);

}  // namespace semkv
