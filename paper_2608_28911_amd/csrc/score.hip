// score.hip -- token-importance indicators (Sec. 3.3) on gfx950: the scores
// the ranking (Eq. 4-5) consumes, computed from tensors the model already has.
//
// Hidden-state family, one wave per token: each lane holds 8-value chunks
// j = lane + 64 c of a state row (16-byte loads), sums its squares / products
// in fp32, and the wave adds the 64 lane sums by a butterfly of lane
// exchanges.  delta-norm (Eq. 3) and cosine-delta walk the m+1 states once,
// each state read once.  KV-norm family: one 256-thread workgroup per 64
// tokens of a sequence; four lanes per token row of 128 channels, and the
// loop over (layer, kv head) reads one contiguous 16 KB slab per step.
// Both are HBM-bound: a token's states (or rows) are read once, one fp32
// score is written.
#include <hip/hip_fp16.h>

#include "semkv_internal.h"

namespace semkv {
namespace {

template <int DT>
__device__ inline float cvt(uint32_t b16) {
  if constexpr (DT == 0) return __half2float(__ushort_as_half(uint16_t(b16)));
  else return __uint_as_float(b16 << 16);                 // bfloat16: the high half of a binary32
}

// the 8 values of a 16-byte chunk
template <int DT>
__device__ inline void unpack8(const uint4& v, float (&x)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = cvt<DT>(w[e] & 0xFFFFu);
    x[2 * e + 1] = cvt<DT>(w[e] >> 16);
  }
}

__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) x += __shfl_xor(x, s);
  return x;
}

template <int NCH>
__device__ inline void load_row(const uint16_t* row, int lane, int nchunk, uint4 (&v)[NCH]) {
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int j = lane + 64 * c;
    v[c] = j < nchunk ? *reinterpret_cast<const uint4*>(row + 8 * j) : make_uint4(0u, 0u, 0u, 0u);
  }
}

// sum over the lane's chunks of f(a_i, b_i)
template <int DT, int NCH, class F>
__device__ inline float lane_sum2(const uint4 (&a)[NCH], const uint4 (&b)[NCH], F f) {
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    float x[8], y[8];
    unpack8<DT>(a[c], x);
    unpack8<DT>(b[c], y);
#pragma unroll
    for (int i = 0; i < 8; ++i) s += f(x[i], y[i]);
  }
  return s;
}

template <int DT, int NCH>
__global__ __launch_bounds__(256) void score_hidden_kernel(HiddenArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t w = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (w >= int64_t(a.batch) * a.T) return;                 // whole waves leave together
  const int b = int(w / a.T);
  const int64_t t = w - int64_t(b) * a.T;
  const uint16_t* row0 = a.h + b * a.s_batch + t * a.s_token;
  const int nchunk = a.d / 8;
  const float inv_d = 1.0f / float(a.d);
  float s = 0.0f;
  if (a.indicator == 0 || a.indicator == 3) {
    uint4 prev[NCH], cur[NCH];
    load_row<NCH>(row0, lane, nchunk, prev);
    float nprev = 0.0f;
    if (a.indicator == 3) nprev = wave_sum(lane_sum2<DT, NCH>(prev, prev, [](float x, float) { return x * x; }));
    for (int k = 1; k <= a.m; ++k) {
      load_row<NCH>(row0 + k * a.s_state, lane, nchunk, cur);
      if (a.indicator == 0) {                              // ||h^(l) - h^(l-1)||_2
        const float q = wave_sum(lane_sum2<DT, NCH>(cur, prev, [](float x, float y) { return (x - y) * (x - y); }));
        s += sqrtf(q);
      } else {                                             // 1 - cos(h^(l), h^(l-1)); 0-norm: cos = 0
        const float dp = wave_sum(lane_sum2<DT, NCH>(cur, prev, [](float x, float y) { return x * y; }));
        const float ncur = wave_sum(lane_sum2<DT, NCH>(cur, cur, [](float x, float) { return x * x; }));
        const float den = sqrtf(ncur) * sqrtf(nprev);
        s += 1.0f - (den > 0.0f ? dp / den : 0.0f);
        nprev = ncur;
      }
#pragma unroll
      for (int c = 0; c < NCH; ++c) prev[c] = cur[c];
    }
    s /= float(a.m);
  } else {
    uint4 last[NCH];
    load_row<NCH>(row0 + a.m * a.s_state, lane, nchunk, last);
    const float ss = wave_sum(lane_sum2<DT, NCH>(last, last, [](float x, float) { return x * x; }));
    if (a.indicator == 1) {
      s = sqrtf(ss);
    } else {                                               // population variance, two passes in registers
      const float mean = wave_sum(lane_sum2<DT, NCH>(last, last, [](float x, float) { return x; })) * inv_d;
      float v = 0.0f;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        float x[8];
        unpack8<DT>(last[c], x);
        if (lane + 64 * c < nchunk) {
#pragma unroll
          for (int i = 0; i < 8; ++i) v += (x[i] - mean) * (x[i] - mean);
        }
      }
      s = wave_sum(v) * inv_d;
    }
  }
  if (lane == 0) a.scores[int64_t(b) * a.T + t] = s;
}

__global__ __launch_bounds__(256) void kv_norm_kernel(KvNormArgs a) {
  const int tid = threadIdx.x, r = tid >> 2, q = tid & 3;
  const int b = blockIdx.y;
  const int64_t t = int64_t(blockIdx.x) * kSlots + r;
  const bool valid = t < a.T;
  const int64_t tt = valid ? t : 0;
  const int R = a.n_layers * a.n_kv_heads;
  float sum = 0.0f;
#pragma unroll 2
  for (int i = 0; i < R; ++i) {
    const int l = i / a.n_kv_heads, h = i - l * a.n_kv_heads;
    const uint4* p = reinterpret_cast<const uint4*>(a.X + l * a.sL + b * a.sB + h * a.sH + tt * a.sT + 32 * q);
    float part = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float x[8];
      unpack8<0>(p[k], x);
#pragma unroll
      for (int e = 0; e < 8; ++e) part += x[e] * x[e];
    }
    sum += part;
  }
  // the row's four quarters (lanes 4r .. 4r+3)
  sum += __shfl_xor(sum, 1);
  sum += __shfl_xor(sum, 2);
  if (q == 0 && valid) a.scores[int64_t(b) * a.T + t] = sqrtf(sum);
}

template <int DT>
int launch_hidden_dt(const HiddenArgs& a, hipStream_t s) {
  const int64_t waves = int64_t(a.batch) * a.T;
  const dim3 grid(unsigned((waves + 3) / 4));
  const int nch = (a.d / 8 + 63) / 64;
  if (nch <= 1) hipLaunchKernelGGL((score_hidden_kernel<DT, 1>), grid, dim3(256), 0, s, a);
  else if (nch <= 2) hipLaunchKernelGGL((score_hidden_kernel<DT, 2>), grid, dim3(256), 0, s, a);
  else if (nch <= 4) hipLaunchKernelGGL((score_hidden_kernel<DT, 4>), grid, dim3(256), 0, s, a);
  else if (nch <= 8) hipLaunchKernelGGL((score_hidden_kernel<DT, 8>), grid, dim3(256), 0, s, a);
  else if (nch <= 16) hipLaunchKernelGGL((score_hidden_kernel<DT, 16>), grid, dim3(256), 0, s, a);
  else return -2;
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace

int launch_score_hidden(const HiddenArgs& a, hipStream_t s) {
  return a.dtype == 0 ? launch_hidden_dt<0>(a, s) : launch_hidden_dt<1>(a, s);
}

int launch_kv_norm(const KvNormArgs& a, hipStream_t s) {
  const dim3 grid(unsigned((a.T + kSlots - 1) / kSlots), unsigned(a.batch));
  hipLaunchKernelGGL(kv_norm_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace semkv
