// decode.hip -- split-K GQA decode attention over the mixed-precision cache
// (the decoding consumer of SemKV, Sec. 3.1 and Alg. 1), for gfx950.
//
// Grid: (split, kv head, sequence); a split is a run of 64-slot records of one
// pool (so one level count per workgroup) or the fp16 tail of generated
// tokens.  A workgroup is 4 waves; each wave takes every 4th record of the
// split and keeps its own online-softmax state for the 4 query heads of the
// kv head.  Per record:
//   scores  C[16 tokens x 16 cols] += A[16 x 32] B[32 x 16] on MFMA
//           (v_mfma_f32_16x16x32_f16): A holds base-L digits decoded from the
//           packed K symbols as fp16 bit patterns d << 6 (the subnormal
//           d * 2^-18; the matrix core keeps full fp32 accuracy for
//           subnormal inputs only when their leading bit is at or above
//           mantissa bit 5, measured on gfx950),
//           B holds q of head h restricted to group g in column 4h+g.  The
//           affine dequantization x = s c + z is folded out:
//           q.x = s (q.c) + z (sum q) per group.
//   softmax online, base 2; unnormalized p, per-record rescale.
//   values  C[16 channels x 16 cols] += A[16 x 32 tokens] B[32 tokens x 16]
//           with A the V digits (V symbols run along tokens) and B = p * s.
// Waves merge in LDS; the last workgroup of each (sequence, kv head) merges the
// splits (log-sum-exp) and, for the TurboQuant-MSE base, applies the inverse
// random-sign Hadamard rotation.
#include <hip/hip_fp16.h>

#include "semkv_internal.h"

namespace semkv {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef uint32_t uint4v __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kDigitScale = 262144.0f;   // 2^18: digit d is fed as d * 2^-18

// ------------------------------------------------------------ traits ----

template <int BASE, int L>
struct Traits {
  static constexpr int n = sym_digits(L);
  static constexpr int P = (BASE == 1 && L == 4) ? 2 : 1;   // MFMA slots per code
  static constexpr int SPS = n * P;                          // slots per symbol
  static constexpr int SPC = 8 / SPS;                        // symbols per chunk
  static constexpr int SK = num_syms(L, kD), SV = num_syms(L, kSlots);
  static constexpr int NSK = (SK + 3) / 4, NSV = (SV + 3) / 4;
  static constexpr int NCK = (NSK + SPC - 1) / SPC, NCV = (NSV + SPC - 1) / SPC;
  static constexpr int W = width_of(L, n);
  static constexpr int TB = tile_bytes(L);
  static constexpr int KSEGW = (NSK * W + 31) / 32;          // normalized dwords of a K segment
  static constexpr int VSEGW = (NSV * W + 31) / 32;
};

// floor(s / L^i) for every symbol s < L^n as (s*2^8 * M) >> 32 with
// M = ceil(2^24 / L^i): one 24-bit high multiply.
__host__ __device__ constexpr uint32_t magic(int L, int i) {
  uint64_t p = 1;
  for (int k = 0; k < i; ++k) p *= uint64_t(L);
  return uint32_t(((uint64_t(1) << 24) + p - 1) / p);
}

__host__ __device__ constexpr bool magic_exact(int L) {
  int n = sym_digits(L);
  uint64_t top = 1;
  for (int k = 0; k < n; ++k) top *= uint64_t(L);
  for (int i = 1; i < n; ++i) {
    uint64_t p = 1;
    for (int k = 0; k < i; ++k) p *= uint64_t(L);
    for (uint64_t s = 0; s < top; ++s)
      if (((s << 8) * magic(L, i)) >> 32 != s / p) return false;
  }
  return true;
}
static_assert(magic_exact(3) && magic_exact(5) && magic_exact(6), "digit extraction");

__device__ inline uint32_t mulhi24(uint32_t a, uint32_t b) {
  return uint32_t((uint64_t(a & 0xFFFFFFu) * uint64_t(b & 0xFFFFFFu)) >> 32);
}

template <int L, int ND>
__device__ inline void digits_of(uint32_t s, uint32_t d[ND]) {
  if constexpr (L == 4) {
#pragma unroll
    for (int i = 0; i < ND; ++i) d[i] = (s >> (2 * i)) & 3u;
  } else {
    uint32_t s8 = s << 8;
    uint32_t F[ND];
    F[0] = s;
#pragma unroll
    for (int i = 1; i < ND; ++i) F[i] = mulhi24(s8, magic(L, i));
#pragma unroll
    for (int i = 0; i + 1 < ND; ++i) d[i] = F[i] - __umul24(uint32_t(L), F[i + 1]);
    d[ND - 1] = F[ND - 1];
  }
}

// bits [OFF, OFF+W) of a normalized segment
template <int OFF, int W, int NW>
__device__ inline uint32_t field(const uint32_t (&seg)[NW]) {
  constexpr int w = OFF / 32, sh = OFF % 32;
  if constexpr (sh + W <= 32) {
    return (seg[w] >> sh) & ((1u << W) - 1u);
  } else {
    return __builtin_amdgcn_alignbit(seg[w + 1], seg[w], sh) & ((1u << W) - 1u);
  }
}

template <int NW>
__device__ inline void load_segment(const uint8_t* body, int bitoff, uint32_t (&seg)[NW]) {
  const uint32_t* p = reinterpret_cast<const uint32_t*>(body) + (bitoff >> 5);
  uint32_t r[NW + 1];
#pragma unroll
  for (int k = 0; k <= NW; ++k) r[k] = p[k];
  int sh = bitoff & 31;
#pragma unroll
  for (int k = 0; k < NW; ++k) seg[k] = __builtin_amdgcn_alignbit(r[k + 1], r[k], sh);
}

// MFMA slots of symbol K of a segment: its codes (or, with two planes, the
// low and high bit of each 4-level code); packed below as fp16 bit patterns.
template <int BASE, int L, int K, int NW, int NS>
__device__ inline void symbol_slots(const uint32_t (&seg)[NW], const uint32_t (&mask)[NS], uint32_t* slot) {
  using Tr = Traits<BASE, L>;
  if constexpr (K < NS) {
    uint32_t v = field<K * Tr::W, Tr::W, NW>(seg) & mask[K];
    uint32_t d[Tr::n];
    digits_of<L, Tr::n>(v, d);
#pragma unroll
    for (int w = 0; w < Tr::SPS; ++w)
      slot[w] = Tr::P == 1 ? d[w] : (d[w / 2] >> (w % 2)) & 1u;
  } else {
#pragma unroll
    for (int w = 0; w < Tr::SPS; ++w) slot[w] = 0;
  }
}

// MFMA A operand of chunk C of a segment: symbols SPC*C .. SPC*C+SPC-1.
template <int BASE, int L, int C, int NW, int NS>
__device__ inline half8 chunk_operand(const uint32_t (&seg)[NW], const uint32_t (&mask)[NS]) {
  using Tr = Traits<BASE, L>;
  uint32_t slot[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  symbol_slots<BASE, L, Tr::SPC * C, NW, NS>(seg, mask, slot);
  if constexpr (Tr::SPC == 2) symbol_slots<BASE, L, Tr::SPC * C + 1, NW, NS>(seg, mask, slot + Tr::SPS);
  uint4v r;                                   // two codes per dword, each as d << 6
  r.x = (slot[0] | (slot[1] << 16)) << 6;
  r.y = (slot[2] | (slot[3] << 16)) << 6;
  r.z = (slot[4] | (slot[5] << 16)) << 6;
  r.w = (slot[6] | (slot[7] << 16)) << 6;
  return __builtin_bit_cast(half8, r);
}

template <int BASE, int L, int NW, int NS, int NC>
__device__ inline float4v contract(const uint32_t (&seg)[NW], const uint32_t (&mask)[NS],
                                   const half8 (&B)[NC], float4v acc) {
  static_assert(NC <= 11, "chunks");
#define SEMKV_C(C) if constexpr (C < NC) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(chunk_operand<BASE, L, C, NW, NS>(seg, mask), B[C], acc, 0, 0, 0);
  SEMKV_C(0) SEMKV_C(1) SEMKV_C(2) SEMKV_C(3) SEMKV_C(4) SEMKV_C(5)
  SEMKV_C(6) SEMKV_C(7) SEMKV_C(8) SEMKV_C(9) SEMKV_C(10)
#undef SEMKV_C
  return acc;
}

// slot e of chunk c of lane group j -> (line position, plane) or -1
template <int BASE, int L>
__device__ inline int slot_pos(int nvals, int j, int c, int e, int& plane) {
  using Tr = Traits<BASE, L>;
  plane = 0;
  if (e >= Tr::SPC * Tr::SPS) return -1;
  int k = Tr::SPC * c + e / Tr::SPS;
  int w = e % Tr::SPS;
  int dig = w / Tr::P;
  plane = w % Tr::P;
  int p = j + 4 * k;
  int S = (nvals + Tr::n - 1) / Tr::n;
  if (p >= S) return -1;
  int nd = nvals - Tr::n * p < Tr::n ? nvals - Tr::n * p : Tr::n;
  if (dig >= nd) return -1;
  return Tr::n * p + dig;
}

template <int BASE, int L, int NVALS>
__device__ inline void segment_masks(int j, uint32_t* mask, int ns) {
  constexpr int n = sym_digits(L);
  constexpr int S = num_syms(L, NVALS);
  for (int k = 0; k < ns; ++k) {
    int p = j + 4 * k;
    if (p >= S) { mask[k] = 0; continue; }
    int nd = NVALS - n * p < n ? NVALS - n * p : n;
    mask[k] = (1u << width_of(L, nd)) - 1u;
  }
}

__device__ inline int seg_off(int L, int nvals, int nlines, int j, int line) {
  int off = 0;
  for (int i = 0; i < j; ++i) off += nlines * seg_bits(L, nvals, i);
  return off + line * seg_bits(L, nvals, j);
}

struct Shared {
  float q[4][kD];          // query of the 4 heads (rotated for tq)
  float zw[16];            // per column: sum of q over its group (zero-point weight)
  union {
    float pp[4][kSlots][16];           // per wave: p * s_V per (token, column)
    struct {
      float m[4][4], l[4][4];
      float o[4][4][kD];
    } mg;
    struct {
      float lg[4][kSlots];
      float mx[4], sum[4];
      float o[4][kD];
    } tl;
  } u;
};

__device__ inline float hf(uint16_t b) { return __half2float(__ushort_as_half(b)); }

template <int BASE, int L, int G>
__device__ void pool_split(const DecodeArgs& a, Shared& sm, int pool, int t_begin, int t_end,
                           int b, int kvh) {
  using Tr = Traits<BASE, L>;
  const PoolGeom& g = a.g;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int n = lane & 15, r = lane >> 4, kg = r;          // MFMA column / row group
  const int hh = n >> 2, gg = n & 3;                       // head and group of column n
  // score columns: affine, q of head h on group g; tq, high and low fp16 part of q_rot
  constexpr int NG = BASE == 0 ? kD / G : 2;
  // value columns: V group vg of column n; the weight p*s is split into fp16 high
  // and low parts, the low part in the spare columns 4h + NGV + vg when NGV <= 2,
  // else (G = 32) in a second MFMA pass
  constexpr int NGV = BASE == 0 ? kD / G : 1;
  constexpr bool LOPASS = NGV > 2;
  const int vg = gg < NGV ? gg : (!LOPASS && gg < 2 * NGV ? gg - NGV : -1);
  const bool vlo = gg >= NGV;
  // tq: mu = -m, 0, m (L = 3) or -b, -a, a, b (L = 4)
  const float* mu = a.mu[pool];
  const float cS = BASE == 0 ? 1.0f : (L == 3 ? mu[2] / 128.0f : 1.0f / 128.0f);
  const float cZ = BASE == 0 ? 0.0f : (L == 3 ? -mu[2] / 128.0f : -mu[3] / 128.0f);
  const float wP0 = BASE == 0 ? 1.0f : (L == 3 ? 1.0f : mu[3] - mu[2]);
  const float wP1 = BASE == 0 ? 1.0f : (L == 3 ? 1.0f : mu[2] + mu[3]);

  // score B operand: column n = 4h + g, slot -> channel
  half8 Bq[Tr::NCK];
#pragma unroll
  for (int c = 0; c < Tr::NCK; ++c) {
    _Float16 v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      int pl;
      int ch = slot_pos<BASE, L>(kD, kg, c, e, pl);
      float x = 0.0f;
      if (ch >= 0 && gg < NG) {
        if (BASE == 0) {
          x = (ch / G == gg) ? sm.q[hh][ch] : 0.0f;
          v[e] = _Float16(x);
        } else {
          float w = (pl ? wP1 : wP0) * sm.q[hh][ch];
          _Float16 h0 = _Float16(w);
          v[e] = gg == 0 ? h0 : _Float16(w - float(h0));
        }
      } else {
        v[e] = _Float16(0.0f);
      }
    }
    Bq[c] = half8{v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
  }
  uint32_t kmask[Tr::NSK], vmask[Tr::NSV];
  segment_masks<BASE, L, kD>(kg, kmask, Tr::NSK);
  segment_masks<BASE, L, kSlots>(kg, vmask, Tr::NSV);
  const int koff0 = seg_off(L, kD, kSlots, kg, 0), kstep = seg_bits(L, kD, kg);
  const int voff0 = seg_off(L, kSlots, kD, kg, 0), vstep = seg_bits(L, kSlots, kg);
  const float zwn = sm.zw[n];

  float m_run = -INFINITY, l_run = 0.0f, z_run = 0.0f;
  float4v acc_o[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc_o[cb] = float4v{0, 0, 0, 0};

  const uint8_t* unit = g.pools + unit_offset(g, b, a.layer, kvh) + (pool ? g.lo_offset : 0);
  const int64_t nrows = a.n_rows[pool];
  float (*pp)[16] = sm.u.pp[wave];

  for (int tile = t_begin + wave; tile < t_end; tile += 4) {
    const uint8_t* rec = unit + int64_t(tile) * g.rec_bytes[pool];
    const uint8_t* kmeta = rec + 2 * Tr::TB;
    const uint8_t* vmeta = kmeta + g.meta_bytes;
    const int nvalid = nrows - int64_t(tile) * kSlots < kSlots ? int(nrows - int64_t(tile) * kSlots) : kSlots;

    // ---- scores
    float lg[4][4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      uint32_t seg[Tr::KSEGW];
      load_segment<Tr::KSEGW>(rec, koff0 + (16 * blk + n) * kstep, seg);
      float4v acc = contract<BASE, L, Tr::KSEGW, Tr::NSK, Tr::NCK>(seg, kmask, Bq, float4v{0, 0, 0, 0});
      const int t0 = 16 * blk + 4 * r;
      float sk[4], zk[4];
      if (BASE == 0) {
        uint4 mt = gg < NG ? *reinterpret_cast<const uint4*>(kmeta + (gg * kSlots + t0) * 4) : uint4{0, 0, 0, 0};
        uint32_t mm[4] = {mt.x, mt.y, mt.z, mt.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) { sk[i] = hf(mm[i] & 0xFFFFu); zk[i] = hf(mm[i] >> 16); }
      } else {
        uint2 mt = *reinterpret_cast<const uint2*>(kmeta + t0 * 2);
        uint32_t mm[2] = {mt.x, mt.y};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float rho = hf((mm[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
          sk[i] = rho * cS;
          zk[i] = rho * cZ;
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x = acc[i] * kDigitScale * sk[i] + zk[i] * zwn;
        x += __shfl_xor(x, 1);
        x += __shfl_xor(x, 2);
        lg[blk][i] = (t0 + i < nvalid) ? x * (kLog2e * 0.08838834764831845f) : -INFINITY;
      }
    }
    // ---- online softmax (base 2)
    float mt = lg[0][0];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) mt = fmaxf(mt, lg[blk][i]);
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float lsum = 0.0f, zsum = 0.0f;
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      const int t0 = 16 * blk + 4 * r;
      float sv[4], zv[4];
      if (BASE == 0) {
        uint4 mt4 = vg >= 0 ? *reinterpret_cast<const uint4*>(vmeta + (vg * kSlots + t0) * 4) : uint4{0, 0, 0, 0};
        uint32_t mm[4] = {mt4.x, mt4.y, mt4.z, mt4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) { sv[i] = hf(mm[i] & 0xFFFFu); zv[i] = vlo ? 0.0f : hf(mm[i] >> 16); }
      } else {
        uint2 mt2 = *reinterpret_cast<const uint2*>(vmeta + t0 * 2);
        uint32_t mm[2] = {mt2.x, mt2.y};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float rho = hf((mm[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
          sv[i] = vg >= 0 ? rho * cS : 0.0f;
          zv[i] = gg == 0 ? rho * cZ : 0.0f;
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float p = __builtin_amdgcn_exp2f(lg[blk][i] - m_new);
        bool ok = t0 + i < nvalid;
        p = ok ? p : 0.0f;
        lsum += p;
        zsum += p * (ok ? zv[i] : 0.0f);
        pp[t0 + i][n] = p * (ok ? sv[i] : 0.0f);
      }
    }
    l_run = l_run * alpha + lsum;
    z_run = z_run * alpha + zsum;
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) acc_o[cb] *= alpha;
    // p * s_V written by other lanes of this wave is read below
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();

    // ---- values: B = p * s_V over the token slots of each chunk
    half8 Bp[Tr::NCV], Bl[LOPASS ? Tr::NCV : 1];
#pragma unroll
    for (int c = 0; c < Tr::NCV; ++c) {
      _Float16 v[8], w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        int pl;
        int t = slot_pos<BASE, L>(kSlots, kg, c, e, pl);
        float x = 0.0f;
        if (t >= 0 && vg >= 0) x = pp[t][n] * (pl ? wP1 : wP0);
        _Float16 h = _Float16(x);
        _Float16 l = _Float16(x - float(h));
        v[e] = vlo ? l : h;
        w[e] = l;
      }
      Bp[c] = half8{v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
      if constexpr (LOPASS) Bl[c] = half8{w[0], w[1], w[2], w[3], w[4], w[5], w[6], w[7]};
    }
    const uint8_t* vbody = rec + Tr::TB;
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      uint32_t seg[Tr::VSEGW];
      load_segment<Tr::VSEGW>(vbody, voff0 + (16 * cb + n) * vstep, seg);
      acc_o[cb] = contract<BASE, L, Tr::VSEGW, Tr::NSV, Tr::NCV>(seg, vmask, Bp, acc_o[cb]);
      if constexpr (LOPASS) acc_o[cb] = contract<BASE, L, Tr::VSEGW, Tr::NSV, Tr::NCV>(seg, vmask, Bl, acc_o[cb]);
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }

  // ---- wave totals over the 4 row groups, then the workgroup merge
  if constexpr (!LOPASS) {
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc_o[cb][i] += __shfl_xor(acc_o[cb][i], NGV);
  }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  z_run += __shfl_xor(z_run, 16);
  z_run += __shfl_xor(z_run, 32);
  __syncthreads();
  if (r == 0 && gg == 0) {
    sm.u.mg.m[wave][hh] = m_run;
    sm.u.mg.l[wave][hh] = l_run;
  }
#pragma unroll
  for (int cb = 0; cb < 8; ++cb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int ch = 16 * cb + 4 * r + i;
      bool mine = BASE == 0 ? (ch / G == gg) : (gg == 0);
      if (mine) sm.u.mg.o[wave][hh][ch] = acc_o[cb][i] * kDigitScale + z_run;
    }
  __syncthreads();
}

// Partials cross workgroups (and XCDs, whose L2 caches are not coherent with
// each other): they are written and read with agent-scope atomic accesses,
// which go to the coherent level without any cache write-back or invalidate.
__device__ inline void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline float ld_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ void write_partial(const DecodeArgs& a, Shared& sm, int b, int kvh, int split) {
  const int tid = threadIdx.x, h = tid >> 6, c = (tid & 63) * 2;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) M = fmaxf(M, sm.u.mg.m[w][h]);
  float Lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float sc = sm.u.mg.m[w][h] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(sm.u.mg.m[w][h] - M);
    Lsum += sm.u.mg.l[w][h] * sc;
    o0 += sm.u.mg.o[w][h][c] * sc;
    o1 += sm.u.mg.o[w][h][c + 1] * sc;
  }
  float* dst = a.ws + ((int64_t(b) * a.g.n_kv_heads + kvh) * a.nsplit + split) * 4 * kPartial + h * kPartial;
  if ((tid & 63) == 0) {
    st_agent(dst, M);
    st_agent(dst + 1, Lsum);
  }
  st_agent(dst + 4 + c, o0);
  st_agent(dst + 5 + c, o1);
}

// fp16 tail of generated tokens, plain vector arithmetic (at most 64 rows)
template <int BASE>
__device__ void tail_split(const DecodeArgs& a, Shared& sm, float (*qorig)[kD], int b, int kvh) {
  const PoolGeom& g = a.g;
  const int tid = threadIdx.x;
  const int nt = a.n_tail;
  const uint16_t* kt = a.tail + ((((int64_t(b) * g.n_layers + a.layer) * g.n_kv_heads + kvh) * 2) * kSlots) * kD;
  const uint16_t* vt = kt + kSlots * kD;
  if (tid < 4 * nt) {
    int t = tid >> 2, h = tid & 3;
    float d = 0.0f;
    for (int c = 0; c < kD; ++c) d += qorig[h][c] * hf(kt[t * kD + c]);
    sm.u.tl.lg[h][t] = d * (kLog2e * 0.08838834764831845f);
  }
  __syncthreads();
  if (tid < 4) {
    float M = -INFINITY;
    for (int t = 0; t < nt; ++t) M = fmaxf(M, sm.u.tl.lg[tid][t]);
    float s = 0.0f;
    for (int t = 0; t < nt; ++t) {
      float p = __builtin_amdgcn_exp2f(sm.u.tl.lg[tid][t] - M);
      sm.u.tl.lg[tid][t] = p;
      s += p;
    }
    sm.u.tl.mx[tid] = M;
    sm.u.tl.sum[tid] = s;
  }
  __syncthreads();
  {
    int h = tid >> 6, c = (tid & 63) * 2;
    float o0 = 0.0f, o1 = 0.0f;
    for (int t = 0; t < nt; ++t) {
      float p = sm.u.tl.lg[h][t];
      o0 += p * hf(vt[t * kD + c]);
      o1 += p * hf(vt[t * kD + c + 1]);
    }
    if (BASE == 1) {                       // into the rotated domain: H (sign . o) / 128
      const uint32_t* sw = g.signs + (int64_t(a.layer) * g.n_kv_heads + kvh) * 4;
      o0 = ((sw[c >> 5] >> (c & 31)) & 1u) ? -o0 : o0;
      o1 = ((sw[(c + 1) >> 5] >> ((c + 1) & 31)) & 1u) ? -o1 : o1;
    }
    sm.u.tl.o[h][c] = o0;
    sm.u.tl.o[h][c + 1] = o1;
  }
  __syncthreads();
  if (BASE == 1) {
    for (int hs = 1; hs < kD; hs <<= 1) {  // 4 heads x 64 butterflies per stage
      int h = tid >> 6, i = tid & 63;
      int lo = (i / hs) * 2 * hs + (i % hs), hi = lo + hs;
      float x = sm.u.tl.o[h][lo], y = sm.u.tl.o[h][hi];
      __syncthreads();
      sm.u.tl.o[h][lo] = x + y;
      sm.u.tl.o[h][hi] = x - y;
      __syncthreads();
    }
  }
  // the tail partial enters the workgroup merge as wave 0; waves 1-3 are empty
  {
    int h = tid >> 6, c = (tid & 63) * 2;
    float scale = BASE == 1 ? 1.0f / 128.0f : 1.0f;
    float o0 = sm.u.tl.o[h][c] * scale, o1 = sm.u.tl.o[h][c + 1] * scale;
    float M = sm.u.tl.mx[h], S = sm.u.tl.sum[h];
    __syncthreads();                       // tl and mg share storage
    if ((tid & 63) == 0)
      for (int w = 0; w < 4; ++w) {
        sm.u.mg.m[w][h] = w == 0 ? M : -INFINITY;
        sm.u.mg.l[w][h] = w == 0 ? S : 0.0f;
      }
    for (int w = 0; w < 4; ++w) {
      sm.u.mg.o[w][h][c] = w == 0 ? o0 : 0.0f;
      sm.u.mg.o[w][h][c + 1] = w == 0 ? o1 : 0.0f;
    }
  }
  __syncthreads();
}

template <int BASE, int LH, int LL, int G>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a) {
  __shared__ Shared sm;
  __shared__ float qorig[4][kD];
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const PoolGeom& g = a.g;
  {
    const int h = tid >> 6, c = (tid & 63) * 2;
    const uint16_t* qp = a.q + ((int64_t(b) * g.n_kv_heads * 4) + kvh * 4 + h) * kD + c;
    uint32_t w = *reinterpret_cast<const uint32_t*>(qp);
    float x0 = hf(w & 0xFFFFu), x1 = hf(w >> 16);
    qorig[h][c] = x0;
    qorig[h][c + 1] = x1;
    if (BASE == 1) {
      const uint32_t* sw = g.signs + (int64_t(a.layer) * g.n_kv_heads + kvh) * 4;
      x0 = ((sw[c >> 5] >> (c & 31)) & 1u) ? -x0 : x0;
      x1 = ((sw[(c + 1) >> 5] >> ((c + 1) & 31)) & 1u) ? -x1 : x1;
    }
    sm.q[h][c] = x0;
    sm.q[h][c + 1] = x1;
  }
  __syncthreads();
  if (BASE == 1) {
    for (int hs = 1; hs < kD; hs <<= 1) {
      int h = tid >> 6, i = tid & 63;
      int lo = (i / hs) * 2 * hs + (i % hs), hi = lo + hs;
      float x = sm.q[h][lo], y = sm.q[h][hi];
      __syncthreads();
      sm.q[h][lo] = x + y;
      sm.q[h][hi] = x - y;
      __syncthreads();
    }
  }
  if (tid < 16) {
    int h = tid >> 2, gq = tid & 3;
    float s = 0.0f;
    if (BASE == 0) {
      if (gq < kD / G)
        for (int c = gq * G; c < (gq + 1) * G; ++c) s += sm.q[h][c];
    } else if (gq == 0) {
      for (int c = 0; c < kD; ++c) s += sm.q[h][c];
    }
    sm.zw[tid] = s;
  }
  __syncthreads();
  if (split < a.ns[0] + a.ns[1]) {
    const int pool = split < a.ns[0] ? 0 : 1;
    const int s0 = pool ? split - a.ns[0] : split;
    const int ntiles = int((a.n_rows[pool] + kSlots - 1) / kSlots);
    const int t_begin = s0 * a.chunk;
    const int t_end = t_begin + a.chunk < ntiles ? t_begin + a.chunk : ntiles;
    if (pool == 0) pool_split<BASE, LH, G>(a, sm, 0, t_begin, t_end, b, kvh);
    else pool_split<BASE, LL, G>(a, sm, 1, t_begin, t_end, b, kvh);
  } else {
    tail_split<BASE>(a, sm, qorig, b, kvh);
  }
  write_partial(a, sm, b, kvh, split);
  // the last workgroup of this (sequence, kv head) merges the splits: every
  // thread waits for its partial stores (workgroup release), then one counter
  // increment per workgroup at agent scope
  __shared__ int last;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  if (tid == 0) {
    uint32_t* ctr = a.counters + b * g.n_kv_heads + kvh;
    uint32_t old = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = old == uint32_t(a.nsplit - 1);
    if (last) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last) return;
  merge_splits<BASE>(a, sm, b, kvh);
}

// Merge of the splits of one (sequence, kv head), run by the last workgroup
// to finish: log-sum-exp over the partials, then for the tq base the inverse
// rotation o = sign . H o_rot.
template <int BASE>
__device__ void merge_splits(const DecodeArgs& a, Shared& sm, int b, int kvh) {
  const int tid = threadIdx.x, h = tid >> 6, c = (tid & 63) * 2;
  const int ns = a.nsplit;
  const float* unit = a.ws + (int64_t(b) * a.g.n_kv_heads + kvh) * ns * 4 * kPartial;
  float* mm = &sm.u.pp[0][0][0];           // [ns][4] maxima, then [ns][4] sums
  float* ll = mm + kMaxSplits * 4;
  for (int i = tid; i < ns * 4; i += 256) {
    mm[i] = ld_agent(unit + i * kPartial);
    ll[i] = ld_agent(unit + i * kPartial + 1);
  }
  __syncthreads();
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, mm[s * 4 + h]);
  float Lsum = 0.0f, o0 = 0.0f, o1 = 0.0f;
  const float* op = unit + h * kPartial + 4 + c;
  int s = 0;
  for (; s + 4 <= ns; s += 4) {              // four splits' loads in flight
    float x[4][2];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[k][0] = ld_agent(op + (s + k) * 4 * kPartial);
      x[k][1] = ld_agent(op + (s + k) * 4 * kPartial + 1);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float m = mm[(s + k) * 4 + h];
      float sc = m == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m - M);
      Lsum += ll[(s + k) * 4 + h] * sc;
      o0 += x[k][0] * sc;
      o1 += x[k][1] * sc;
    }
  }
  for (; s < ns; ++s) {
    float m = mm[s * 4 + h];
    float sc = m == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(m - M);
    Lsum += ll[s * 4 + h] * sc;
    o0 += ld_agent(op + s * 4 * kPartial) * sc;
    o1 += ld_agent(op + s * 4 * kPartial + 1) * sc;
  }
  o0 /= Lsum;
  o1 /= Lsum;
  if (BASE == 1) {
    __syncthreads();
    sm.q[h][c] = o0;
    sm.q[h][c + 1] = o1;
    __syncthreads();
    for (int hs = 1; hs < kD; hs <<= 1) {
      int i = tid & 63;
      int lo = (i / hs) * 2 * hs + (i % hs), hi = lo + hs;
      float xa = sm.q[h][lo], ya = sm.q[h][hi];
      __syncthreads();
      sm.q[h][lo] = xa + ya;
      sm.q[h][hi] = xa - ya;
      __syncthreads();
    }
    const uint32_t* sw = a.g.signs + (int64_t(a.layer) * a.g.n_kv_heads + kvh) * 4;
    o0 = ((sw[c >> 5] >> (c & 31)) & 1u) ? -sm.q[h][c] : sm.q[h][c];
    o1 = ((sw[(c + 1) >> 5] >> ((c + 1) & 31)) & 1u) ? -sm.q[h][c + 1] : sm.q[h][c + 1];
  }
  float2* dst = reinterpret_cast<float2*>(a.out + ((int64_t(b) * a.g.n_kv_heads + kvh) * 4 + h) * kD + c);
  *dst = make_float2(o0, o1);
}

template <int BASE, int LH, int LL>
int launch_dec(const DecodeArgs& a, hipStream_t st) {
  dim3 grid(a.nsplit, a.g.n_kv_heads, a.g.batch);
  if (BASE == 1 || a.g.G == 128) hipLaunchKernelGGL((decode_kernel<BASE, LH, LL, 128>), grid, dim3(256), 0, st, a);
  else if (a.g.G == 64) hipLaunchKernelGGL((decode_kernel<BASE, LH, LL, 64>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((decode_kernel<BASE, LH, LL, 32>), grid, dim3(256), 0, st, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace

int launch_decode(const DecodeArgs& a, hipStream_t s) {
  const int B = a.g.base, LH = a.g.L[0], LL = a.g.L[1];
  if (B == 0 && LH == 6 && LL == 5) return launch_dec<0, 6, 5>(a, s);
  if (B == 0 && LH == 5 && LL == 4) return launch_dec<0, 5, 4>(a, s);
  if (B == 0 && LH == 6 && LL == 4) return launch_dec<0, 6, 4>(a, s);
  if (B == 0 && LH == 4 && LL == 3) return launch_dec<0, 4, 3>(a, s);
  if (B == 0 && LH == 5 && LL == 3) return launch_dec<0, 5, 3>(a, s);
  if (B == 0 && LH == 6 && LL == 3) return launch_dec<0, 6, 3>(a, s);
  if (B == 1 && LH == 4 && LL == 3) return launch_dec<1, 4, 3>(a, s);
  return -2;
}

}  // namespace semkv
