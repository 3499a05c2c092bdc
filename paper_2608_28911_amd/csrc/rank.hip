// rank.hip -- exact top-K importance ranking (Eq. 4-5) for gfx950.
//
// One 1024-thread workgroup per sequence.  Scores become order-preserving
// 32-bit keys (-0 taken as +0); a 4-pass 8-bit radix select finds the K-th
// largest key and how many of the keys equal to it are taken; equal keys are
// taken by increasing token index (block-wide prefix counts).  A second scan
// compacts the flagged and unflagged token indices into ascending slot lists.
#include "semkv_internal.h"

namespace semkv {
namespace {

constexpr int kThreads = 1024;

__device__ inline uint32_t order_key(float v) {
  uint32_t u = __float_as_uint(v == 0.0f ? 0.0f : v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// exclusive prefix sum over the workgroup; returns this thread's prefix and
// writes the total to *total
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* wsum, int64_t* total) {
  int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    int64_t y = __shfl_up(x, d);
    if (lane >= d) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      int64_t t = wsum[w];
      wsum[w] = run;
      run += t;
    }
    wsum[kThreads / 64] = run;
  }
  __syncthreads();
  int64_t r = wsum[wave] + x - v;
  *total = wsum[kThreads / 64];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kThreads) void rank_kernel(RankArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_prefix;
  __shared__ int64_t s_krem;
  __shared__ int64_t wsum[kThreads / 64 + 1];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* s = a.scores + int64_t(b) * a.ld_s;
  const int64_t T = a.T, K = a.K;

  bool nan_seen = false;
  uint32_t prefix = 0, pmask = 0;
  int64_t krem = K;
  if (K > 0) {
    for (int d = 3; d >= 0; --d) {
      for (int i = tid; i < 256; i += kThreads) hist[i] = 0;
      __syncthreads();
      for (int64_t i = tid; i < T; i += kThreads) {
        float v = s[i];
        nan_seen |= isnan(v);
        uint32_t k = order_key(v);
        if ((k & pmask) == prefix) atomicAdd(&hist[(k >> (8 * d)) & 255u], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        int64_t cum = 0;
        for (int bin = 255; bin >= 0; --bin) {
          if (cum + hist[bin] >= krem) {
            s_prefix = prefix | (uint32_t(bin) << (8 * d));
            s_krem = krem - cum;
            break;
          }
          cum += hist[bin];
        }
      }
      __syncthreads();
      prefix = s_prefix;
      krem = s_krem;
      pmask |= 255u << (8 * d);
      __syncthreads();
    }
  }
  if (nan_seen) atomicOr(a.status, 1);
  // theta = prefix; keys > theta are taken, and the first krem keys == theta
  const uint32_t theta = prefix;
  const int64_t ties = K > 0 ? krem : 0;
  auto taken = [&](uint32_t k, int64_t tie_rank) {
    return K > 0 && (k > theta || (k == theta && tie_rank < ties));
  };

  // chunks of whole flag words, one per thread, in index order
  const int64_t chunk = ((T + kThreads - 1) / kThreads + 31) / 32 * 32;
  const int64_t lo_i = int64_t(tid) * chunk, hi_i = lo_i + chunk < T ? lo_i + chunk : T;
  int64_t nt = 0;
  for (int64_t i = lo_i; i < hi_i; ++i) nt += order_key(s[i]) == theta ? 1 : 0;
  int64_t tot;
  int64_t tie_base = block_exclusive_scan(nt, wsum, &tot);
  int64_t nflag = 0, tr = tie_base;
  for (int64_t w0 = lo_i; w0 < hi_i; w0 += 32) {
    uint32_t word = 0;
    for (int e = 0; e < 32 && w0 + e < hi_i; ++e) {
      uint32_t k = order_key(s[w0 + e]);
      bool f = taken(k, tr);
      tr += k == theta ? 1 : 0;
      word |= f ? (1u << e) : 0u;
      nflag += f ? 1 : 0;
    }
    a.flags[int64_t(b) * a.flag_words + (w0 >> 5)] = word;
  }
  int64_t hi_base = block_exclusive_scan(nflag, wsum, &tot);
  int64_t lo_base = lo_i - hi_base;
  if (lo_i > T) lo_base = 0;
  tr = tie_base;
  int32_t* hi_out = a.hi_idx + int64_t(b) * K;
  int32_t* lo_out = a.lo_idx + int64_t(b) * (T - K);
  for (int64_t i = lo_i; i < hi_i; ++i) {
    uint32_t k = order_key(s[i]);
    bool f = taken(k, tr);
    tr += k == theta ? 1 : 0;
    if (f) hi_out[hi_base++] = int32_t(i);
    else lo_out[lo_base++] = int32_t(i);
  }
}

}  // namespace

int launch_rank(const RankArgs& a, int batch, hipStream_t s) {
  hipLaunchKernelGGL(rank_kernel, dim3(batch), dim3(kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace semkv
