// rank.hip -- exact top-K importance ranking (Eq. 4-5) for gfx950.
//
// One 1024-thread workgroup per sequence.  Scores become order-preserving
// 32-bit keys (-0 taken as +0); a 4-pass 8-bit radix select finds the K-th
// largest key theta and how many of the keys equal to it are taken (equal
// keys are taken by increasing token index).  Importance scores are heavily
// tied (integer Zipf draws, peaked accumulated-attention weights), so the
// histogram passes put most keys of a wave in one bin: each wave keeps its
// own histogram and adds its most common bin with a single atomic.  The keys
// of the bin the first pass picks are gathered into LDS when they fit, and
// the remaining passes count only them.  The flag and compaction pass then stages the keys through LDS in segments,
// loaded coalesced, so that each thread owns a contiguous run of 16 tokens:
// block-wide prefix counts give every token its tie rank and its slot in the
// ascending high and low slot lists.
//
// Sequences longer than one chunk of kRankChunk = 4096 tokens are ranked by
// one 256-thread workgroup per chunk instead, in five launches over the same
// grid (chunk, sequence), so that a chunk's scores stay in one L2:
//   1. histogram of key bits [21, 32) of every token;
//   2. the bin b1 holding the K-th largest key, then the histogram of bits
//      [10, 21) of the keys whose top bits are b1;
//   3. the bin b2 of those, then the histogram of bits [0, 10) of the keys
//      with prefix (b1, b2);
//   4. the bin b3: theta = (b1, b2, b3) and the number of keys equal to theta
//      that are taken; each chunk counts its keys above and equal to theta;
//   5. flags and slot lists, each chunk offset by the counts of the chunks
//      before it.
// Each histogram is summed over the chunks with device-scope atomics into
// per-sequence scratch that is zero when the call starts; a later launch of
// the same call clears it again (3 clears the first, 4 the second, 5 the
// third).  Every workgroup of a launch selects the bin itself from the whole
// histogram; chunk 0 also records it for the next launch.
#include "semkv_internal.h"

namespace semkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kRun = 16;                     // tokens per thread in a segment
constexpr int kSeg = kThreads * kRun;        // tokens per LDS segment
constexpr int kBatch = 8;                    // score loads in flight per thread

__device__ inline uint32_t order_key(float v) {
  uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// exclusive prefix sum over the workgroup of one value per thread; returns
// this thread's prefix and the total
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (wave == 0) {
    uint32_t w = lane < kWaves ? wsum[lane] : 0u, s = w;
#pragma unroll
    for (int d = 1; d < kWaves; d <<= 1) {
      const uint32_t y = __shfl_up(s, d);
      if (lane >= d) s += y;
    }
    if (lane < kWaves) wsum[lane] = s - w;
    if (lane == kWaves - 1) wsum[kWaves] = s;
  }
  __syncthreads();
  const uint32_t r = wsum[wave] + x - v;
  *total = wsum[kWaves];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void rank_kernel(RankArgs a) {
  __shared__ uint32_t hist[kWaves][256];
  __shared__ alignas(16) uint32_t keys[kSeg];
  __shared__ uint32_t wsum[kWaves + 1];
  __shared__ uint32_t s_prefix;
  __shared__ int64_t s_krem;
  __shared__ uint32_t s_cand, s_ncand;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* s = a.scores + int64_t(b) * a.ld_s;
  const int64_t T = a.T, K = a.K;

  // ---- radix select of the K-th largest key, 8 bits per pass.  After the
  // first pass only the keys of the chosen bin can still decide theta: when
  // they fit the LDS key buffer they are gathered there once, and the later
  // passes count them alone instead of reading every score again.
  bool nan_seen = false;
  uint32_t prefix = 0, pmask = 0;
  int64_t krem = K;
  if (K > 0) {
    bool staged = false;                     // candidates in keys[0, ncand)
    uint32_t ncand = 0;
    for (int d = 3; d >= 0; --d) {
      for (int i = tid; i < kWaves * 256; i += kThreads) (&hist[0][0])[i] = 0u;
      __syncthreads();
      // add key k (counted when `in`) to this wave's histogram of digit d
      auto count = [&](uint32_t k, bool in) {
        const uint32_t bin = (k >> (8 * d)) & 255u;
        const uint64_t act = __ballot(in);
        if (act != 0) {
          // the wave's first counted key's bin in one atomic, the rest singly
          const int lead = __builtin_ctzll(act);
          const uint32_t b0 = __shfl(bin, lead);
          const uint64_t same = __ballot(in && bin == b0);
          if (lane == lead) atomicAdd(&hist[wave][b0], uint32_t(__popcll(same)));
          if (in && bin != b0) atomicAdd(&hist[wave][bin], 1u);
        }
      };
      if (!staged) {
        for (int64_t i0 = 0; i0 < T; i0 += kBatch * kThreads) {
          float v[kBatch];                   // all loads of the batch in flight at once
#pragma unroll
          for (int j = 0; j < kBatch; ++j) {
            const int64_t i = i0 + j * kThreads + tid;
            v[j] = i < T ? s[i] : 0.0f;
          }
#pragma unroll
          for (int j = 0; j < kBatch; ++j) {
            const int64_t i = i0 + j * kThreads + tid;
            nan_seen |= i < T && isnan(v[j]);
            const uint32_t k = order_key(v[j]);
            count(k, i < T && (k & pmask) == prefix);
          }
        }
      } else {
        for (uint32_t i0 = 0; i0 < ncand; i0 += kThreads) {
          const uint32_t i = i0 + tid;
          const uint32_t k = i < ncand ? keys[i] : 0u;
          count(k, i < ncand && (k & pmask) == prefix);
        }
      }
      __syncthreads();
      // bin counts over the waves, then the bin holding the krem-th largest
      // key: thread t < 256 takes bin 255 - t (descending key order)
      uint32_t cnt = 0;
      if (tid < 256) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) cnt += hist[w][255 - tid];
      }
      uint32_t total;
      const uint32_t above = block_exclusive_scan(cnt, wsum, &total);   // keys in higher bins
      if (tid < 256 && int64_t(above) < krem && int64_t(above) + cnt >= krem) {
        s_prefix = prefix | (uint32_t(255 - tid) << (8 * d));
        s_krem = krem - above;
        s_cand = cnt;
      }
      __syncthreads();
      prefix = s_prefix;
      krem = s_krem;
      pmask |= 255u << (8 * d);
      if (d > 0 && !staged && s_cand <= uint32_t(kSeg)) {
        // gather the chosen bin's keys (exactly s_cand of them) into LDS
        if (tid == 0) s_ncand = 0u;
        __syncthreads();
        for (int64_t i0 = 0; i0 < T; i0 += kBatch * kThreads) {
          float v[kBatch];
#pragma unroll
          for (int j = 0; j < kBatch; ++j) {
            const int64_t i = i0 + j * kThreads + tid;
            v[j] = i < T ? s[i] : 0.0f;
          }
#pragma unroll
          for (int j = 0; j < kBatch; ++j) {
            const int64_t i = i0 + j * kThreads + tid;
            const uint32_t k = order_key(v[j]);
            const bool in = i < T && (k & pmask) == prefix;
            const uint64_t act = __ballot(in);
            if (act != 0) {
              const int lead = __builtin_ctzll(act);
              uint32_t base = 0u;
              if (lane == lead) base = atomicAdd(&s_ncand, uint32_t(__popcll(act)));
              base = __shfl(base, lead);
              if (in) keys[base + uint32_t(__popcll(act & ((uint64_t(1) << lane) - 1u)))] = k;
            }
          }
        }
        __syncthreads();
        ncand = s_ncand;
        staged = true;
      }
      __syncthreads();
    }
  }
  if (nan_seen) atomicOr(a.status, 1);
  // keys above theta are taken, and the first `ties` keys equal to it
  const uint32_t theta = prefix;
  const uint32_t ties = K > 0 ? uint32_t(krem) : 0u;

  // ---- flags and ascending slot lists, one LDS segment of kSeg keys at a time
  int32_t* hi_out = a.hi_idx + int64_t(b) * K;
  int32_t* lo_out = a.lo_idx + int64_t(b) * (T - K);
  uint32_t run_tie = 0, run_hi = 0;          // before this segment (T < 2^29)
  for (int64_t seg0 = 0; seg0 < T; seg0 += kSeg) {
    const int n = T - seg0 < kSeg ? int(T - seg0) : kSeg;
#pragma unroll
    for (int j = 0; j < kRun; ++j) {
      const int i = j * kThreads + tid;
      if (i < n) keys[i] = order_key(s[seg0 + i]);
    }
    __syncthreads();
    // this thread's run of 16 keys, in registers (keys past n are not used)
    const int r0 = tid * kRun, nr = n - r0 < 0 ? 0 : (n - r0 < kRun ? n - r0 : kRun);
    uint32_t kr[kRun];
#pragma unroll
    for (int j = 0; j < kRun / 4; ++j) {
      const uint4 q = reinterpret_cast<const uint4*>(keys + r0)[j];
      kr[4 * j] = q.x;
      kr[4 * j + 1] = q.y;
      kr[4 * j + 2] = q.z;
      kr[4 * j + 3] = q.w;
    }
    uint32_t nt = 0;
#pragma unroll
    for (int j = 0; j < kRun; ++j) nt += (j < nr && kr[j] == theta) ? 1u : 0u;
    uint32_t tot_tie;
    uint32_t tr = run_tie + block_exclusive_scan(nt, wsum, &tot_tie);   // tie rank of the run's first tie
    uint32_t bits = 0, nf = 0;
#pragma unroll
    for (int j = 0; j < kRun; ++j) {
      const uint32_t k = kr[j];
      const bool f = j < nr && K > 0 && (k > theta || (k == theta && tr < ties));
      tr += (j < nr && k == theta) ? 1u : 0u;
      bits |= f ? 1u << j : 0u;
      nf += f ? 1u : 0u;
    }
    // a flag word is the runs of two neighbouring lanes (kRun = 16)
    const uint32_t other = __shfl_xor(bits, 1);
    if ((tid & 1) == 0 && nr > 0) a.flags[int64_t(b) * a.flag_words + ((seg0 + r0) >> 5)] = bits | (other << 16);
    uint32_t tot_hi;
    uint32_t hb = run_hi + block_exclusive_scan(nf, wsum, &tot_hi);
    uint32_t lb = uint32_t(seg0 + r0) - hb;
    for (int j = 0; j < nr; ++j) {
      if ((bits >> j) & 1u) hi_out[hb++] = int32_t(seg0 + r0 + j);
      else lo_out[lb++] = int32_t(seg0 + r0 + j);
    }
    run_tie += tot_tie;
    run_hi += tot_hi;
    __syncthreads();
  }
}

// ------------------------------------------- one workgroup per chunk ----

constexpr int kMT = 256;                     // threads of a chunk's workgroup
constexpr int kMW = kMT / 64;
constexpr int kMRun = kRankChunk / kMT;      // 16 tokens per thread

__device__ uint32_t scan256(uint32_t v, uint32_t* wsum, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kMW; ++w) {
    before += w < wave ? wsum[w] : 0u;
    all += wsum[w];
  }
  *total = all;
  __syncthreads();
  return before + x - v;
}

// the scores of a chunk's tokens as keys, bounded by the sequence's T scores
// (a buffer descriptor: reads past T return 0 and are marked invalid).  RUN:
// thread t holds tokens c0 + 16 t + j (a contiguous run); else c0 + 256 j + t.
// chunk_scores issues the loads; chunk_keys, called after other independent
// loads have been issued, converts (one round trip for both).
template <bool RUN>
__device__ inline void chunk_scores(const RankArgs& a, int b, int c, uint32_t (&v)[kMRun]) {
  const float* s = a.scores + int64_t(b) * a.ld_s;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(s), 0, int(a.T * 4), kBufferWord3);
  const int64_t c0 = int64_t(c) * kRankChunk;
#pragma unroll
  for (int j = 0; j < kMRun; ++j) {
    const int64_t i = c0 + (RUN ? int64_t(kMRun) * threadIdx.x + j : int64_t(j) * kMT + threadIdx.x);
    v[j] = __builtin_amdgcn_raw_buffer_load_b32(rs, int(i * 4), 0, 0);
  }
}

template <bool RUN>
__device__ inline void chunk_keys(const RankArgs& a, int c, uint32_t (&k)[kMRun], uint32_t& valid, bool& nan) {
  const int64_t c0 = int64_t(c) * kRankChunk;
  valid = 0u;
  nan = false;
#pragma unroll
  for (int j = 0; j < kMRun; ++j) {
    const int64_t i = c0 + (RUN ? int64_t(kMRun) * threadIdx.x + j : int64_t(j) * kMT + threadIdx.x);
    const float v = __uint_as_float(k[j]);
    const bool in = i < a.T;
    valid |= in ? 1u << j : 0u;
    nan |= in && isnan(v);
    k[j] = order_key(v);
  }
}

// the bin of G (NB bins, scanned from the top) that holds the krem-th largest
// of the keys G counts: sel[0] = bin, sel[1] = krem less the keys above it
template <int NB>
__device__ inline void bins_of(const uint32_t* G, uint32_t (&c)[NB / kMT]) {
  constexpr int PER = NB / kMT;
#pragma unroll
  for (int i = 0; i < PER; ++i) c[i] = G[NB - 1 - (int(threadIdx.x) * PER + i)];
}

template <int NB>
__device__ void select_bin(const uint32_t (&c)[NB / kMT], uint32_t krem, uint32_t* wsum, uint32_t* sel) {
  constexpr int PER = NB / kMT;
  const int tid = threadIdx.x;
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) sum += c[i];
  uint32_t total;
  const uint32_t above = scan256(sum, wsum, &total);
  if (above < krem && above + sum >= krem) {
    uint32_t acc = above;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      if (acc < krem && acc + c[i] >= krem) {
        sel[0] = uint32_t(NB - 1 - (tid * PER + i));
        sel[1] = krem - acc;
      }
      acc += c[i];
    }
  }
  __syncthreads();
}

// words [0, n) of one of the sequence's histograms cleared, a slice per chunk
__device__ inline void clear_slice(uint32_t* H, int n, int c, int nchunk) {
  const int per = (n + nchunk - 1) / nchunk;
  for (int i = c * per + int(threadIdx.x); i < (c + 1) * per && i < n; i += kMT) H[i] = 0u;
}

// add the counted keys' bins to an LDS histogram: a wave's most common case
// (its first counted key's bin) in one atomic, the others singly
__device__ inline void hist_add(uint32_t* hist, uint32_t bin, bool in) {
  const int lane = threadIdx.x & 63;
  const uint64_t act = __ballot(in);
  if (act != 0) {
    const int lead = __builtin_ctzll(act);
    const uint32_t b0 = __shfl(bin, lead);
    const uint64_t same = __ballot(in && bin == b0);
    if (lane == lead) atomicAdd(&hist[b0], uint32_t(__popcll(same)));
    if (in && bin != b0) atomicAdd(&hist[bin], 1u);
  }
}

// launches 1-3: PASS 1 counts bits [21, 32) of every key, PASS 2 bits
// [10, 21) under the prefix b1, PASS 3 bits [0, 10) under (b1, b2)
template <int PASS>
__global__ __launch_bounds__(kMT) void rank_hist_kernel(RankArgs a) {
  constexpr int NB = PASS == 3 ? 1024 : 2048;
  constexpr int OUT = PASS == 1 ? kRankH1 : PASS == 2 ? kRankH2 : kRankH3;
  __shared__ uint32_t hist[NB];
  __shared__ uint32_t wsum[kMW];
  __shared__ uint32_t sel[2];
  const int c = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, nchunk = gridDim.x;
  uint32_t* S = a.scratch + int64_t(b) * a.scratch_words;
  for (int i = tid; i < NB; i += kMT) hist[i] = 0u;
  if (tid == 0) sel[0] = sel[1] = 0u;
  uint32_t key[kMRun], valid;
  bool nan;
  chunk_scores<false>(a, b, c, key);
  uint32_t pre = 0;
  if constexpr (PASS == 1) {
    chunk_keys<false>(a, c, key, valid, nan);
  } else if constexpr (PASS == 2) {
    uint32_t bins[8];
    bins_of<2048>(S + kRankH1, bins);
    chunk_keys<false>(a, c, key, valid, nan);
    select_bin<2048>(bins, uint32_t(a.K), wsum, sel);
    pre = sel[0];
    if (c == 0 && tid == 0) {
      S[kRankState] = sel[0];
      S[kRankState + 1] = sel[1];
    }
  } else {
    uint32_t bins[8];
    bins_of<2048>(S + kRankH2, bins);
    const uint32_t b1 = S[kRankState], k1 = S[kRankState + 1];
    chunk_keys<false>(a, c, key, valid, nan);
    select_bin<2048>(bins, k1, wsum, sel);
    pre = (b1 << 11) | sel[0];
    if (c == 0 && tid == 0) {
      S[kRankState + 2] = sel[0];
      S[kRankState + 3] = sel[1];
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kMRun; ++j) {
    const uint32_t k = key[j];
    const bool in = ((valid >> j) & 1u) && (PASS == 1 || (k >> (PASS == 2 ? 21 : 10)) == pre);
    hist_add(hist, PASS == 1 ? k >> 21 : PASS == 2 ? (k >> 10) & 2047u : k & 1023u, in);
  }
  __syncthreads();
  for (int i = tid; i < NB; i += kMT)
    if (hist[i] != 0u) __hip_atomic_fetch_add(S + OUT + i, hist[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (PASS == 1 && __syncthreads_or(nan) && tid == 0) atomicOr(a.status, 1);
  if constexpr (PASS == 3) clear_slice(S + kRankH1, 2048, c, nchunk);
}

// launch 4: theta and the ties taken; each chunk's keys above and equal to theta
__global__ __launch_bounds__(kMT) void rank_count_kernel(RankArgs a) {
  __shared__ uint32_t wsum[kMW];
  __shared__ uint32_t sel[2];
  const int c = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, nchunk = gridDim.x;
  uint32_t* S = a.scratch + int64_t(b) * a.scratch_words;
  if (tid == 0) sel[0] = sel[1] = 0u;
  uint32_t key[kMRun], valid;
  bool nan;
  chunk_scores<false>(a, b, c, key);
  uint32_t bins[4];
  bins_of<1024>(S + kRankH3, bins);
  const uint32_t b1 = S[kRankState], b2 = S[kRankState + 2], k2 = S[kRankState + 3];
  chunk_keys<false>(a, c, key, valid, nan);
  select_bin<1024>(bins, k2, wsum, sel);
  const uint32_t theta = (b1 << 21) | (b2 << 10) | sel[0];
  if (c == 0 && tid == 0) {
    S[kRankState + 4] = theta;
    S[kRankState + 5] = sel[1];
  }
  uint32_t gt = 0, eq = 0;
#pragma unroll
  for (int j = 0; j < kMRun; ++j) {
    const bool in = (valid >> j) & 1u;
    gt += in && key[j] > theta ? 1u : 0u;
    eq += in && key[j] == theta ? 1u : 0u;
  }
  uint32_t tgt, teq;
  scan256(gt, wsum, &tgt);
  scan256(eq, wsum, &teq);
  if (tid == 0) {
    S[kRankCounts + 2 * c] = tgt;
    S[kRankCounts + 2 * c + 1] = teq;
  }
  clear_slice(S + kRankH2, 2048, c, nchunk);
}

// launch 5: the flags and the ascending slot lists of the chunk's tokens
__global__ __launch_bounds__(kMT) void rank_final_kernel(RankArgs a) {
  __shared__ uint32_t wsum[kMW];
  const int c = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, nchunk = gridDim.x;
  uint32_t* S = a.scratch + int64_t(b) * a.scratch_words;
  uint32_t key[kMRun], valid;
  bool nan;
  chunk_scores<true>(a, b, c, key);
  const bool any = a.K > 0;
  const uint32_t theta = any ? S[kRankState + 4] : 0u, ties = any ? S[kRankState + 5] : 0u;
  // keys above theta and equal to it in the chunks before this one
  uint32_t gb = 0, eb = 0;
  if (any) {
    for (int i = tid; i < c; i += kMT) {
      gb += S[kRankCounts + 2 * i];
      eb += S[kRankCounts + 2 * i + 1];
    }
  }
  uint32_t gt_before, eq_before;
  scan256(gb, wsum, &gt_before);
  scan256(eb, wsum, &eq_before);
  chunk_keys<true>(a, c, key, valid, nan);
  uint32_t nt = 0;
#pragma unroll
  for (int j = 0; j < kMRun; ++j) nt += ((valid >> j) & 1u) && key[j] == theta ? 1u : 0u;
  uint32_t tot;
  uint32_t tr = eq_before + scan256(nt, wsum, &tot);     // tie rank of the run's first tie
  uint32_t bits = 0, nf = 0;
#pragma unroll
  for (int j = 0; j < kMRun; ++j) {
    const bool in = (valid >> j) & 1u;
    const bool f = in && any && (key[j] > theta || (key[j] == theta && tr < ties));
    tr += in && key[j] == theta ? 1u : 0u;
    bits |= f ? 1u << j : 0u;
    nf += f ? 1u : 0u;
  }
  const int64_t t0 = int64_t(c) * kRankChunk + int64_t(kMRun) * tid;   // first token of the run
  const uint32_t other = __shfl_xor(bits, 1);
  if ((tid & 1) == 0 && valid != 0u) a.flags[int64_t(b) * a.flag_words + (t0 >> 5)] = bits | (other << 16);
  const uint32_t hi_before = gt_before + (eq_before < ties ? eq_before : ties);
  int64_t hb = hi_before + scan256(nf, wsum, &tot);
  int64_t lb = t0 - hb;
  int32_t* hi_out = a.hi_idx + int64_t(b) * a.K;
  int32_t* lo_out = a.lo_idx + int64_t(b) * (a.T - a.K);
#pragma unroll
  for (int j = 0; j < kMRun; ++j) {
    if (!((valid >> j) & 1u)) continue;
    if ((bits >> j) & 1u) hi_out[hb++] = int32_t(t0 + j);
    else lo_out[lb++] = int32_t(t0 + j);
  }
  if (any) clear_slice(S + kRankH3, 1024, c, nchunk);
}

}  // namespace

int launch_rank(const RankArgs& a, int batch, hipStream_t s) {
  if (a.T <= kRankChunk) {
    hipLaunchKernelGGL(rank_kernel, dim3(batch), dim3(kThreads), 0, s, a);
    return hipGetLastError() == hipSuccess ? 0 : -5;
  }
  const dim3 grid(unsigned(rank_chunks(a.T)), unsigned(batch));
  if (a.K > 0) {
    hipLaunchKernelGGL(rank_hist_kernel<1>, grid, dim3(kMT), 0, s, a);
    hipLaunchKernelGGL(rank_hist_kernel<2>, grid, dim3(kMT), 0, s, a);
    hipLaunchKernelGGL(rank_hist_kernel<3>, grid, dim3(kMT), 0, s, a);
    hipLaunchKernelGGL(rank_count_kernel, grid, dim3(kMT), 0, s, a);
  }
  hipLaunchKernelGGL(rank_final_kernel, grid, dim3(kMT), 0, s, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace semkv
