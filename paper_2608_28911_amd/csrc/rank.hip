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

}  // namespace

int launch_rank(const RankArgs& a, int batch, hipStream_t s) {
  hipLaunchKernelGGL(rank_kernel, dim3(batch), dim3(kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace semkv
