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

__host__ __device__ constexpr int ipow(int b, int e) {
  int r = 1;
  for (int i = 0; i < e; ++i) r *= b;
  return r;
}

// Chunk layout: 8 MFMA slots per lane group per chunk, filled by SPC symbols
// of STRIDE slots each; slot_digit / slot_plane give the code a slot holds
// (-1: a zero pad slot).  4-level codes of the tq base take two slots, their
// low and high bit (the Lloyd-Max levels are affine in those bits).
template <int BASE, int L>
struct Traits {
  static constexpr int n = sym_digits(L);
  static constexpr int P = (BASE == 1 && L == 4) ? 2 : 1;   // MFMA slots per code
  static constexpr int SPC = (L == 5 || (L == 4 && BASE == 0)) ? 2 : 1;
  static constexpr int STRIDE = 8 / SPC;
  static constexpr int SK = num_syms(L, kD), SV = num_syms(L, kSlots);
  static constexpr int NSK = (SK + 3) / 4, NSV = (SV + 3) / 4;
  static constexpr int NCK = (NSK + SPC - 1) / SPC, NCV = (NSV + SPC - 1) / SPC;
  static constexpr int W = width_of(L, n);
  static constexpr int TB = tile_bytes(L);
  static constexpr int KSEGW = (NSK * W + 31) / 32;          // normalized dwords of a K segment
  static constexpr int VSEGW = (NSV * W + 31) / 32;
  // decode table: symbol -> MFMA operand dwords (codes pre-shifted to d << 6).
  // L = 6 splits a symbol into s mod 216 (3 codes) and s div 216 (2 codes).
  static constexpr int EDW = STRIDE / 2;                     // dwords per table entry
  static constexpr int NENT = L == 6 ? 216 : ipow(L, n);
  static constexpr int LUTDW = L == 6 ? 216 * 2 + 36 : NENT * EDW;
  static constexpr int LUTSTRIDE = (LUTDW + 63) / 64 * 64 + 16;   // replicas start 16 banks apart
};

template <int BASE, int L>
__host__ __device__ constexpr int slot_digit(int w) {
  return (BASE == 1 && L == 4) ? w / 2
       : L == 6 ? (w < 3 ? w : (w == 4 || w == 5) ? w - 1 : -1)
       : L == 5 ? (w < 3 ? w : -1)
       : L == 3 ? (w < 5 ? w : -1)
       : w;                                                  // affine L = 4
}
template <int BASE, int L>
__host__ __device__ constexpr int slot_plane(int w) { return (BASE == 1 && L == 4) ? w % 2 : 0; }

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

// Decode tables in LDS (one replica per lane group), built once per workgroup.
template <int BASE, int L>
__device__ void build_lut(uint32_t* lut) {
  using Tr = Traits<BASE, L>;
  for (int i = threadIdx.x; i < 4 * Tr::LUTDW; i += blockDim.x) {
    const int rep = i / Tr::LUTDW, e = i % Tr::LUTDW;
    uint32_t w = 0;
    if (L == 6) {
      if (e < 432) {                    // table A: s mod 216 -> codes 0, 1, 2
        const int v = e / 2;
        w = e & 1 ? (uint32_t(v / 36) << 6) : (uint32_t(v % 6) << 6) | (uint32_t(v / 6 % 6) << 22);
      } else {                          // table B: s div 216 -> codes 3, 4
        const int v = e - 432;
        w = (uint32_t(v % 6) << 6) | (uint32_t(v / 6) << 22);
      }
    } else {
      const int v = e / Tr::EDW, k = e % Tr::EDW;   // dword k: slots 2k, 2k+1
      uint32_t half[2];
      for (int h = 0; h < 2; ++h) {
        const int wsl = 2 * k + h, dg = slot_digit<BASE, L>(wsl);
        uint32_t d = 0;
        if (dg >= 0) {
          uint32_t c = uint32_t(v);
          for (int t = 0; t < dg; ++t) c /= uint32_t(L);
          c %= uint32_t(L);
          d = slot_plane<BASE, L>(wsl) ? (c >> 1) : (Tr::P == 2 ? (c & 1u) : c);
        }
        half[h] = d << 6;
      }
      w = half[0] | (half[1] << 16);
    }
    lut[rep * Tr::LUTSTRIDE + e] = w;
  }
}

template <int BASE, int L, int K, int NW, int NS>
__device__ inline uint32_t seg_symbol(const uint32_t (&seg)[NW], const uint32_t (&mask)[NS]) {
  using Tr = Traits<BASE, L>;
  if constexpr (K < NS) return field<K * Tr::W, Tr::W, NW>(seg) & mask[K];
  else return 0u;
}

// MFMA operand of chunk C of a segment (symbols SPC*C ..), read from the tables
template <int BASE, int L, int C, int NW, int NS>
__device__ inline half8 chunk_operand(const uint32_t (&seg)[NW], const uint32_t (&mask)[NS], const uint32_t* lut) {
  using Tr = Traits<BASE, L>;
  uint4v r;
  if constexpr (L == 6) {
    const uint32_t v = seg_symbol<BASE, L, C, NW, NS>(seg, mask);
    const uint32_t hi = mulhi24(v << 8, magic(6, 3));      // v div 216
    const uint32_t lo = v - 216u * hi;
    const uint2 a = *reinterpret_cast<const uint2*>(lut + 2 * lo);
    r = uint4v{a.x, a.y, lut[432 + hi], 0u};
  } else if constexpr (Tr::SPC == 2) {
    const uint2 a = *reinterpret_cast<const uint2*>(lut + 2 * seg_symbol<BASE, L, 2 * C, NW, NS>(seg, mask));
    const uint2 b = *reinterpret_cast<const uint2*>(lut + 2 * seg_symbol<BASE, L, 2 * C + 1, NW, NS>(seg, mask));
    r = uint4v{a.x, a.y, b.x, b.y};
  } else {
    const uint4 a = *reinterpret_cast<const uint4*>(lut + 4 * seg_symbol<BASE, L, C, NW, NS>(seg, mask));
    r = uint4v{a.x, a.y, a.z, a.w};
  }
  return __builtin_bit_cast(half8, r);
}

template <int BASE, int L, int NW, int NS, int NC>
__device__ inline float4v contract(const uint32_t (&seg)[NW], const uint32_t (&mask)[NS],
                                   const half8 (&B)[NC], float4v acc, const uint32_t* lut) {
  static_assert(NC <= 11, "chunks");
#define SEMKV_C(C) if constexpr (C < NC) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(chunk_operand<BASE, L, C, NW, NS>(seg, mask, lut), B[C], acc, 0, 0, 0);
  SEMKV_C(0) SEMKV_C(1) SEMKV_C(2) SEMKV_C(3) SEMKV_C(4) SEMKV_C(5)
  SEMKV_C(6) SEMKV_C(7) SEMKV_C(8) SEMKV_C(9) SEMKV_C(10)
#undef SEMKV_C
  return acc;
}

// slot e of chunk c of lane group j -> position in the line (channel or
// token) and plane, or -1 for a pad slot or a position past the line
template <int BASE, int L>
__device__ inline int slot_pos(int nvals, int j, int c, int e, int& plane) {
  using Tr = Traits<BASE, L>;
  const int k = Tr::SPC * c + e / Tr::STRIDE, w = e % Tr::STRIDE;
  const int dig = slot_digit<BASE, L>(w);
  plane = slot_plane<BASE, L>(w);
  if (dig < 0) return -1;
  const int p = j + 4 * k;
  const int S = (nvals + Tr::n - 1) / Tr::n;
  if (p >= S) return -1;
  const int nd = nvals - Tr::n * p < Tr::n ? nvals - Tr::n * p : Tr::n;
  if (dig >= nd) return -1;
  return Tr::n * p + dig;
}

// masks of the symbols of segment j (zero past the line's last symbol)
template <int L, int NVALS, int NLINES, int NS>
__device__ inline void segment_masks(int j, uint32_t (&mask)[NS]) {
  constexpr SegTable<L, NVALS, NLINES> t{};
#pragma unroll
  for (int k = 0; k < NS; ++k)
    mask[k] = pick4(j, (1u << t.width[0][k]) - 1u, (1u << t.width[1][k]) - 1u,
                    (1u << t.width[2][k]) - 1u, (1u << t.width[3][k]) - 1u);
}

// first bit of line `line` in segment j, and the bits one line of it takes
template <int L, int NVALS, int NLINES>
__device__ inline int seg_off(int j, int line) {
  constexpr SegTable<L, NVALS, NLINES> t{};
  return pick4(j, t.start[0], t.start[1], t.start[2], t.start[3]) +
         line * pick4(j, t.bits[0], t.bits[1], t.bits[2], t.bits[3]);
}
template <int L, int NVALS, int NLINES>
__device__ inline int seg_line_bits(int j) {
  constexpr SegTable<L, NVALS, NLINES> t{};
  return pick4(j, t.bits[0], t.bits[1], t.bits[2], t.bits[3]);
}

__device__ inline float hf(uint16_t b) { return __half2float(__ushort_as_half(b)); }

// fp16 weight arrays of one wave: [plane][hi|lo][head][group][80 token slots]
// (slots 64..79 stay zero: chunk slots past the last token read them), then a
// zero block that unused columns read at every plane offset.
constexpr int kPvTok = 80;

template <int BASE, int L, int G>
struct Geo {
  using Tr = Traits<BASE, L>;
  static constexpr int MB = meta_bytes(BASE, G);
  static constexpr int RB = 2 * Tr::TB + 2 * MB;
  static constexpr int NLD = (RB + 1023) / 1024;            // 1 KB staging loads per record
  static constexpr int NG = BASE == 0 ? kD / G : 2;          // score rows per head
  static constexpr int NGV = BASE == 0 ? kD / G : 1;         // value groups
  static constexpr int NPL = Tr::P;                          // value planes (tq, 4 levels: 2)
  static constexpr bool LOPASS = NGV > 2;                    // low part in a second pass
  static constexpr int PLSTRIDE = 2 * 4 * NGV * kPvTok;    // halves per plane
  static constexpr int PV = (2 * NPL - 1) * PLSTRIDE + kPvTok;  // planes + zero block
};

template <int NLD, int PV, int LUT>
struct SharedT {
  alignas(16) uint8_t stage[4][2][NLD * 1024];   // two staged records per wave
  alignas(16) uint32_t lut[4 * LUT];             // decode table, one replica per lane group
  alignas(16) _Float16 pv[4][PV];               // per wave p*s weights, fp16 hi/lo
  float q[4][kD];                                // query of the 4 heads (rotated for tq)
  float zw[16];                                  // per (head, row group): sum of q
  float zc[4][4][4];                             // per wave, head, group: sum p * zero
  union {
    struct { float m[4][4], l[4][4]; float o[4][4][kD]; } mg;
    struct { float lg[4][kSlots]; float mx[4], sum[4]; float o[4][kD]; } tl;
    struct { float mm[kMaxSplits * 4]; float ll[kMaxSplits * 4]; } mr;
  } u;
};

template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
// reductions over the 16 lanes of a row (row_ror 8, 4, 2, 1)
__device__ inline float row_max16(float x) {
  x = fmaxf(x, dpp<0x128>(x));
  x = fmaxf(x, dpp<0x124>(x));
  x = fmaxf(x, dpp<0x122>(x));
  return fmaxf(x, dpp<0x121>(x));
}
__device__ inline float row_sum16(float x) {
  x += dpp<0x128>(x);
  x += dpp<0x124>(x);
  x += dpp<0x122>(x);
  return x + dpp<0x121>(x);
}

// LDS-staged segment: NW dwords starting at bit `bitoff` of an LDS body
template <int NW>
__device__ inline void lds_segment(const uint8_t* body, int bitoff, uint32_t (&seg)[NW]) {
  const uint32_t* p = reinterpret_cast<const uint32_t*>(body) + (bitoff >> 5);
  uint32_t r[NW + 1];
#pragma unroll
  for (int k = 0; k <= NW; ++k) r[k] = p[k];
  const int sh = bitoff & 31;
#pragma unroll
  for (int k = 0; k < NW; ++k) seg[k] = __builtin_amdgcn_alignbit(r[k + 1], r[k], sh);
}

// Copy one record into a wave's LDS buffer with direct global->LDS loads
// (16 bytes per lane per load; the last load may read past the record into
// memory the pool allocation keeps as slack).
template <int NLD>
__device__ inline void stage_record(const uint8_t* rec, uint8_t* lds, int lane) {
#pragma unroll
  for (int j = 0; j < NLD; ++j)
    __builtin_amdgcn_global_load_lds(rec + j * 1024 + lane * 16,
                                     (__attribute__((address_space(3))) void*)(lds + j * 1024), 16, 0, 0);
}

template <int NLD>
__device__ inline void wait_staged(bool one_more_in_flight) {
  // vmcnt(NLD) while the next record's NLD loads are in flight, else vmcnt(0)
  if (one_more_in_flight) __builtin_amdgcn_s_waitcnt(0x0F70 | (NLD & 15) | ((NLD >> 4) << 14));
  else __builtin_amdgcn_s_waitcnt(0x0F70);
  __asm__ volatile("" ::: "memory");   // no LDS read of the record moves above the wait
}

template <int BASE, int L, int G, class SH>
__device__ void pool_split(const DecodeArgs& a, SH& sm, int pool, int t_begin, int t_end,
                           int b, int kvh) {
  using Tr = Traits<BASE, L>;
  using Ge = Geo<BASE, L, G>;
  const PoolGeom& g = a.g;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int n = lane & 15, r = lane >> 4, kg = r;
  // tq: mu = -m, 0, m (L = 3) or -b, -a, a, b (L = 4)
  const float* mu = a.mu[pool];
  const float cS = BASE == 0 ? 1.0f : (L == 3 ? mu[2] / 128.0f : 1.0f / 128.0f);
  const float cZ = BASE == 0 ? 0.0f : (L == 3 ? -mu[2] / 128.0f : -mu[3] / 128.0f);
  const float wP[2] = {BASE == 0 ? 1.0f : (L == 3 ? 1.0f : mu[3] - mu[2]),
                       BASE == 0 ? 1.0f : (L == 3 ? 1.0f : mu[2] + mu[3])};

  // ---- score A operand: row 4h + kq of lane row n; slot -> channel of lane group kg
  half8 Aq[Tr::NCK];
  {
    const int h = n >> 2, kq = n & 3;
#pragma unroll
    for (int c = 0; c < Tr::NCK; ++c) {
      _Float16 v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        int pl;
        const int ch = slot_pos<BASE, L>(kD, kg, c, e, pl);
        v[e] = _Float16(0.0f);
        if (ch >= 0 && kq < Ge::NG) {
          if (BASE == 0) {
            if (ch / G == kq) v[e] = _Float16(sm.q[h][ch]);
          } else {
            const float w = wP[pl] * sm.q[h][ch];
            const _Float16 hi = _Float16(w);
            v[e] = kq == 0 ? hi : _Float16(w - float(hi));
          }
        }
      }
      Aq[c] = half8{v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
    }
  }
  build_lut<BASE, L>(sm.lut);
  __syncthreads();                      // every wave reads all of the tables
  const uint32_t* lut = sm.lut + kg * Tr::LUTSTRIDE;
  uint32_t kmask[Tr::NSK], vmask[Tr::NSV];
  segment_masks<L, kD, kSlots>(kg, kmask);
  segment_masks<L, kSlots, kD>(kg, vmask);
  const int koff0 = seg_off<L, kD, kSlots>(kg, n), kstep = 16 * seg_line_bits<L, kD, kSlots>(kg);
  const int voff0 = seg_off<L, kSlots, kD>(kg, n), vstep = 16 * seg_line_bits<L, kSlots, kD>(kg);
  // softmax lanes: token n of each 16-token block, head r
  const int hs = r;
  float zws[Ge::NG];
#pragma unroll
  for (int i = 0; i < Ge::NG; ++i) zws[i] = sm.zw[hs * 4 + i];
  // value B operand lanes: column n = 4h + gg
  const int hv = n >> 2, gg = n & 3;
  const int vg = gg < Ge::NGV ? gg : (!Ge::LOPASS && gg < 2 * Ge::NGV ? gg - Ge::NGV : -1);
  const bool vlo = gg >= Ge::NGV;
  _Float16* pvw = sm.pv[wave];
  constexpr int PLSTRIDE = Ge::PLSTRIDE;
  const int pvzero = Ge::NPL * PLSTRIDE;
  // base index (plane 0) of this lane's column, token 0 of its lane group's first symbol
  const int pvcol = (vg >= 0 ? (((vlo ? 1 : 0) * 4 + hv) * Ge::NGV + vg) * kPvTok : pvzero) + Tr::n * kg;
  const int pvlo_col = (vg >= 0 ? ((4 + hv) * Ge::NGV + vg) * kPvTok : pvzero) + Tr::n * kg;   // LOPASS
  for (int i = lane; i < Ge::PV; i += 64) pvw[i] = _Float16(0.0f);

  float m_run = -INFINITY, l_run = 0.0f;
  float z_run[Ge::NGV];
#pragma unroll
  for (int i = 0; i < Ge::NGV; ++i) z_run[i] = 0.0f;
  float4v acc_o[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) acc_o[cb] = float4v{0, 0, 0, 0};

  const uint8_t* unit = g.pools + unit_offset(g, b, a.layer, kvh) + (pool ? g.lo_offset : 0);
  const int64_t nrows = a.n_rows[pool];
  uint8_t* buf0 = sm.stage[wave][0];
  uint8_t* buf1 = sm.stage[wave][1];
  const int first = t_begin + wave;
  const int count = first < t_end ? (t_end - first + 3) / 4 : 0;
  if (count > 0) stage_record<Ge::NLD>(unit + int64_t(first) * Ge::RB, buf0, lane);

  for (int it = 0; it < count; ++it) {
    const int tile = first + 4 * it;
    uint8_t* rec = (it & 1) ? buf1 : buf0;
    if (it + 1 < count) {
      __asm__ volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(0xC07F);                  // lgkmcnt(0): last reads of that buffer done
      stage_record<Ge::NLD>(unit + int64_t(tile + 4) * Ge::RB, (it & 1) ? buf0 : buf1, lane);
      wait_staged<Ge::NLD>(true);
    } else {
      wait_staged<Ge::NLD>(false);
    }
    const uint8_t* kmeta = rec + 2 * Tr::TB;
    const uint8_t* vmeta = kmeta + Ge::MB;
    const int nvalid = nrows - int64_t(tile) * kSlots < kSlots ? int(nrows - int64_t(tile) * kSlots) : kSlots;

    // ---- scores: C[(h, kq)][token] = q_h,kq . codes; lane holds token n, head r
    float lg[4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      uint32_t seg[Tr::KSEGW];
      lds_segment<Tr::KSEGW>(rec, koff0 + blk * kstep, seg);
      float4v acc = float4v{0, 0, 0, 0};
#define SEMKV_S(C) if constexpr (C < Tr::NCK) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(Aq[C], chunk_operand<BASE, L, C, Tr::KSEGW, Tr::NSK>(seg, kmask, lut), acc, 0, 0, 0);
      SEMKV_S(0) SEMKV_S(1) SEMKV_S(2) SEMKV_S(3) SEMKV_S(4) SEMKV_S(5) SEMKV_S(6) SEMKV_S(7) SEMKV_S(8) SEMKV_S(9) SEMKV_S(10)
#undef SEMKV_S
      const int t = 16 * blk + n;
      float x = 0.0f;
      if (BASE == 0) {
#pragma unroll
        for (int i = 0; i < Ge::NG; ++i) {
          const uint32_t m = *reinterpret_cast<const uint32_t*>(kmeta + (i * kSlots + t) * 4);
          x += acc[i] * hf(m & 0xFFFFu) + hf(m >> 16) * zws[i] * (1.0f / kDigitScale);
        }
      } else {
        const float rho = hf(*reinterpret_cast<const uint16_t*>(kmeta + t * 2));
        x = (acc[0] + acc[1]) * (rho * cS) + rho * cZ * zws[0] * (1.0f / kDigitScale);
      }
      lg[blk] = t < nvalid ? x * (kDigitScale * kLog2e * 0.08838834764831845f) : -INFINITY;
    }
    // ---- online softmax (base 2) for head r over this record's 64 tokens
    float mt = fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3]));
    mt = row_max16(mt);
    const float m_new = fmaxf(m_run, mt);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float lsum = 0.0f;
#pragma unroll
    for (int i = 0; i < Ge::NGV; ++i) z_run[i] *= alpha;
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      const int t = 16 * blk + n;
      const float p = __builtin_amdgcn_exp2f(lg[blk] - m_new);   // 0 for masked tokens
      lsum += p;
      if (BASE == 0) {
#pragma unroll
        for (int i = 0; i < Ge::NGV; ++i) {
          const uint32_t m = *reinterpret_cast<const uint32_t*>(vmeta + (i * kSlots + t) * 4);
          const float x = p * hf(m & 0xFFFFu);
          const _Float16 hi = _Float16(x);
          pvw[((0 * 4 + hs) * Ge::NGV + i) * kPvTok + t] = hi;
          pvw[((1 * 4 + hs) * Ge::NGV + i) * kPvTok + t] = _Float16(x - float(hi));
          z_run[i] += p * hf(m >> 16);
        }
      } else {
        const float rho = hf(*reinterpret_cast<const uint16_t*>(vmeta + t * 2));
        const float ps = p * rho * cS;
#pragma unroll
        for (int pl = 0; pl < Ge::NPL; ++pl) {
          const float x = ps * wP[pl];
          const _Float16 hi = _Float16(x);
          pvw[pl * PLSTRIDE + (0 * 4 + hs) * kPvTok + t] = hi;
          pvw[pl * PLSTRIDE + (1 * 4 + hs) * kPvTok + t] = _Float16(x - float(hi));
        }
        z_run[0] += p * rho * cZ;
      }
    }
    l_run = l_run * alpha + lsum;
    // acc_o columns belong to head n >> 2: fetch that head's alpha
    {
      const float al[4] = {__builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), 0)),
                           __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), 16)),
                           __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), 32)),
                           __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha), 48))};
      if (al[0] != 1.0f || al[1] != 1.0f || al[2] != 1.0f || al[3] != 1.0f) {
        const float av = al[hv];
#pragma unroll
        for (int cb = 0; cb < 8; ++cb) acc_o[cb] *= av;
      }
    }
    // weights written above by other lanes of this wave are read below
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();

    // ---- values: C[channel][column] += V codes (tokens) x weights
    half8 Bp[Tr::NCV], Bl[Ge::LOPASS ? Tr::NCV : 1];
#pragma unroll
    for (int c = 0; c < Tr::NCV; ++c) {
      _Float16 v[8], w[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // slot e -> token n*(kg + 4k) + digit; slots past the last token land
        // in the zero slots 64..79 (pad slots of the chunk are plain zeros)
        const int k = Tr::SPC * c + e / Tr::STRIDE;
        const int dig = slot_digit<BASE, L>(e % Tr::STRIDE), pl = slot_plane<BASE, L>(e % Tr::STRIDE);
        const bool pad = dig < 0;
        const int toff = Tr::n * 4 * k + (pad ? 0 : dig);
        v[e] = pad ? _Float16(0.0f) : pvw[pl * PLSTRIDE + pvcol + toff];
        if constexpr (Ge::LOPASS) w[e] = pad ? _Float16(0.0f) : pvw[pl * PLSTRIDE + pvlo_col + toff];
      }
      Bp[c] = half8{v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
      if constexpr (Ge::LOPASS) Bl[c] = half8{w[0], w[1], w[2], w[3], w[4], w[5], w[6], w[7]};
    }
    const uint8_t* vbody = rec + Tr::TB;
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      uint32_t seg[Tr::VSEGW];
      lds_segment<Tr::VSEGW>(vbody, voff0 + cb * vstep, seg);
      acc_o[cb] = contract<BASE, L, Tr::VSEGW, Tr::NSV, Tr::NCV>(seg, vmask, Bp, acc_o[cb], lut);
      if constexpr (Ge::LOPASS) acc_o[cb] = contract<BASE, L, Tr::VSEGW, Tr::NSV, Tr::NCV>(seg, vmask, Bl, acc_o[cb], lut);
    }
  }

  // ---- wave totals: sums over the tokens of a row; fold low columns into high ones
  l_run = row_sum16(l_run);
#pragma unroll
  for (int i = 0; i < Ge::NGV; ++i) z_run[i] = row_sum16(z_run[i]);
  if constexpr (!Ge::LOPASS) {
#pragma unroll
    for (int cb = 0; cb < 8; ++cb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        acc_o[cb][i] += Ge::NGV == 1 ? dpp<0xB1>(acc_o[cb][i]) : dpp<0x4E>(acc_o[cb][i]);   // quad xor 1 / xor 2
  }
  if (n == 0) {
#pragma unroll
    for (int i = 0; i < Ge::NGV; ++i) sm.zc[wave][hs][i] = z_run[i];
  }
  __syncthreads();
  if (n == 0) {
    sm.u.mg.m[wave][hs] = m_run;
    sm.u.mg.l[wave][hs] = l_run;
  }
#pragma unroll
  for (int cb = 0; cb < 8; ++cb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ch = 16 * cb + 4 * r + i;
      const bool mine = BASE == 0 ? (ch / G == gg) : (gg == 0);
      if (mine) sm.u.mg.o[wave][hv][ch] = acc_o[cb][i] * kDigitScale + sm.zc[wave][hv][BASE == 0 ? gg : 0];
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

template <class SH>
__device__ void write_partial(const DecodeArgs& a, SH& sm, int b, int kvh, int split) {
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
template <int BASE, class SH>
__device__ void tail_split(const DecodeArgs& a, SH& sm, float (*qorig)[kD], int b, int kvh) {
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
  using GH = Geo<BASE, LH, G>;
  using GL = Geo<BASE, LL, G>;
  constexpr int NLD = GH::NLD > GL::NLD ? GH::NLD : GL::NLD;
  constexpr int PV = GH::PV > GL::PV ? GH::PV : GL::PV;
  constexpr int LUT = Traits<BASE, LH>::LUTSTRIDE > Traits<BASE, LL>::LUTSTRIDE ? Traits<BASE, LH>::LUTSTRIDE
                                                                                 : Traits<BASE, LL>::LUTSTRIDE;
  __shared__ SharedT<NLD, PV, LUT> sm;
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
template <int BASE, class SH>
__device__ void merge_splits(const DecodeArgs& a, SH& sm, int b, int kvh) {
  const int tid = threadIdx.x, h = tid >> 6, c = (tid & 63) * 2;
  const int ns = a.nsplit;
  const float* unit = a.ws + (int64_t(b) * a.g.n_kv_heads + kvh) * ns * 4 * kPartial;
  float* mm = sm.u.mr.mm;                 // [ns][4] maxima
  float* ll = sm.u.mr.ll;                 // [ns][4] sums
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
