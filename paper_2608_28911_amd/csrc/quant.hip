// quant.hip -- quantize + pack of prompt tokens (Alg. 1, Eq. 7), the fp16 tail
// append and the block close of generated tokens (Alg. 2), for gfx950.
//
// One workgroup (256 threads) builds one 64-slot record of one pool of one
// (sequence, layer, kv head) unit.  Four consecutive lanes own one token row:
// lane q holds channels [32q, 32q+32).  Codes go to LDS, then each thread packs
// whole segments (Sec. 4.1 mixed-radix symbols) into the LDS body with atomic
// ORs, and the record is written with 16-byte stores.
#include <hip/hip_fp16.h>

#include "semkv_internal.h"

namespace semkv {
namespace {

constexpr int kPitch = 132;             // LDS row pitch of the code arrays (bytes)
constexpr int kMaxBodyWords = 3072 / 4; // largest body: L = 8

__device__ inline float h2f(uint16_t b) { return __half2float(__ushort_as_half(b)); }
__device__ inline uint16_t f2h(float f) { return __half_as_ushort(__float2half_rn(f)); }
// fp16 bits with +-inf replaced by +-65504, the largest finite binary16: the
// two parameters of a group stay finite for finite input, and the codes are
// taken against the stored (saturated) pair
__device__ inline uint16_t sat16(uint16_t h) {
  return (h & 0x7FFFu) == 0x7C00u ? uint16_t((h & 0x8000u) | 0x7BFFu) : h;
}

// Correctly rounded fp32 square root of a >= 0.  The hardware result is within
// one ulp; the neighbour whose rounding interval holds sqrt(a) is chosen by
// comparing a with the squared interval ends, which are exact in double (a
// 25-bit midpoint squares to at most 50 bits).  sqrt is never exactly halfway
// between two floats, so no tie arises.
__device__ inline float sqrt_rn(float a) {
  float r = __builtin_sqrtf(a);
  if (!(a > 0.0f) || !(a < INFINITY)) return r;
  const double ad = double(a);
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const float dn = __uint_as_float(__float_as_uint(r) - 1u), up = __uint_as_float(__float_as_uint(r) + 1u);
    const double lo = 0.5 * (double(dn) + double(r)), hi = 0.5 * (double(r) + double(up));
    if (ad < lo * lo) r = dn;
    else if (ad >= hi * hi) r = up;
  }
  return r;
}

// A row quarter (32 fp16 values) as fp32, and whether any is inf or NaN (the
// largest magnitude bit pattern, by a packed 16-bit max, reaches 0x7C00).
__device__ inline void load_quarter(const uint16_t* src, float x[32], bool& nonfinite) {
  typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
  const uint4* p = reinterpret_cast<const uint4*>(src);
  u16x2 big = u16x2{0, 0};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint4 w = p[k];
    uint32_t d[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[8 * k + 2 * e] = h2f(uint16_t(d[e] & 0xFFFFu));
      x[8 * k + 2 * e + 1] = h2f(uint16_t(d[e] >> 16));
      big = __builtin_elementwise_max(big, __builtin_bit_cast(u16x2, d[e] & 0x7FFF7FFFu));
    }
  }
  nonfinite |= big.x >= 0x7C00u || big.y >= 0x7C00u;
}

// The value of lane (this lane xor 1), xor 2, or of lane 0 of this lane's
// quad: exact DPP moves within a quad at full VALU rate.  Every lane has a
// source lane, so the move needs no prior value (none to materialize, and the
// compiler may fold the move into the add that uses it).
template <int CTRL>
__device__ inline float quad_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kQuadLane0 = 0x00;

// Asymmetric affine quantizer (Sec. 4.1) of one row quarter; the min/max of a
// group of G channels is combined over the G/32 lanes holding it.  Returns
// {scale, zero} as fp16 bits (low half = scale).
template <int L>
__device__ uint32_t affine_quarter(const float x[32], int G, uint32_t code[8]) {
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    mn = fminf(mn, x[i]);
    mx = fmaxf(mx, x[i]);
  }
  if (G >= 64) {
    mn = fminf(mn, quad_mov<kQuadXor1>(mn));
    mx = fmaxf(mx, quad_mov<kQuadXor1>(mx));
  }
  if (G >= 128) {
    mn = fminf(mn, quad_mov<kQuadXor2>(mn));
    mx = fmaxf(mx, quad_mov<kQuadXor2>(mx));
  }
  float zero = mn + 0.0f;                               // -0 -> +0
  uint16_t s16 = f2h(__fdiv_rn(mx - mn, float(L - 1)));
  // only 2 levels can overflow: (max - min) / 1 reaches 131008, while for
  // L >= 3 the quotient is at most 65504
  if constexpr (L == 2) s16 = sat16(s16);
  float sf = h2f(s16);
  float inv = sf == 0.0f ? 0.0f : __fdiv_rn(1.0f, sf);
  // clamp to [0, L-1] (NaN -> 0), then one convert-and-insert per code: the
  // convert rounds to nearest even, and with integer bounds clamping before
  // rounding gives the code rounding before clamping gives
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t w = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float c = fminf(fmaxf((x[4 * k + e] - zero) * inv, 0.0f), float(L - 1));
      w = __builtin_amdgcn_cvt_pk_u8_f32(c, e, w);
    }
    code[k] = w;
  }
  return uint32_t(s16) | (uint32_t(f2h(zero)) << 16);
}

// H diag(sign) x of one row quarter: sign flip, then the unnormalized
// Walsh-Hadamard transform, stages 1..16 inside the lane and 32, 64 across
// the lanes of the row's quad.
__device__ inline void rotate_quarter(const float x[32], int q, uint32_t sbits, float u[32]) {
#pragma unroll
  for (int i = 0; i < 32; ++i) u[i] = __uint_as_float(__float_as_uint(x[i]) ^ ((sbits << (31 - i)) & 0x80000000u));
#pragma unroll
  for (int h = 1; h < 32; h <<= 1)
#pragma unroll
    for (int i = 0; i < 32; ++i)
      if (!(i & h)) {
        float p = u[i], r = u[i + h];
        u[i] = p + r;
        u[i + h] = p - r;
      }
  // cross-lane stages: the upper lane of a pair takes o - u = o + (-u), the
  // lower u + o = o + u (IEEE addition commutes; -u is a sign flip)
  const uint32_t f1 = (q & 1) ? 0x80000000u : 0u, f2 = (q & 2) ? 0x80000000u : 0u;
#pragma unroll
  for (int i = 0; i < 32; ++i) {                         // h = 32: partner lane q ^ 1
    const float o = quad_mov<kQuadXor1>(u[i]);
    u[i] = o + __uint_as_float(__float_as_uint(u[i]) ^ f1);
  }
#pragma unroll
  for (int i = 0; i < 32; ++i) {                         // h = 64: partner lane q ^ 2
    const float o = quad_mov<kQuadXor2>(u[i]);
    u[i] = o + __uint_as_float(__float_as_uint(u[i]) ^ f2);
  }
}

// TurboQuant-MSE base (Sec. 4.9) of one row quarter: the rotation, the row
// norm by a fixed pairwise tree, one fp16 scalar, and Lloyd-Max threshold
// codes.  Returns rho bits.
template <int L>
__device__ uint16_t tq_quarter(const float x[32], int q, const uint32_t* sw, const float* tau,
                               uint32_t code[8]) {
  float u[32], a[32];
  rotate_quarter(x, q, sw[q], u);
#pragma unroll
  for (int i = 0; i < 32; ++i) a[i] = x[i] * x[i];
#pragma unroll
  for (int i = 0; i < 32; ++i) a[i] = a[i] + quad_mov<kQuadXor2>(a[i]);   // h = 64 (lanes 0,1 keep)
#pragma unroll
  for (int i = 0; i < 32; ++i) a[i] = a[i] + quad_mov<kQuadXor1>(a[i]);   // h = 32 (lane 0 keeps)
#pragma unroll
  for (int h = 16; h >= 1; h >>= 1)
#pragma unroll
    for (int i = 0; i < h; ++i) a[i] = a[i] + a[i + h];
  uint16_t r16 = f2h(sqrt_rn(a[0]));
  if ((r16 & 0x7FFFu) == 0x7C00u) r16 = 0x7BFFu;       // saturate to 65504
  r16 = uint16_t(__float_as_uint(quad_mov<kQuadLane0>(__uint_as_float(uint32_t(r16)))));
  float rf = h2f(r16);
  float thr[L - 1];
#pragma unroll
  for (int k = 0; k < L - 1; ++k) thr[k] = rf * tau[k];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t w = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint32_t c = 0;
#pragma unroll
      for (int t = 0; t < L - 1; ++t) c += u[4 * k + e] > thr[t] ? 1u : 0u;
      w |= c << (8 * e);
    }
    code[k] = w;
  }
  return r16;
}

// Affine quantizer of the rotated row (Sec. 4.1 with its Hadamard rotation):
// y = H diag(sign) x / 16 (the division is exact), then per group of G
// rotated coordinates zero = fp16(min y) (-0 stored as +0) and scale =
// fp16(max(0, (max y - zero) / (L-1))), each saturated at +-65504, codes
// against the stored pair.
// Returns {scale, zero} as fp16 bits (low half = scale).
template <int L>
__device__ uint32_t rot_affine_quarter(const float x[32], int q, const uint32_t* sw, int G, uint32_t code[8]) {
  float y[32];
  rotate_quarter(x, q, sw[q], y);
  float mn = INFINITY, mx = -INFINITY;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    y[i] *= 0.0625f;
    mn = fminf(mn, y[i]);
    mx = fmaxf(mx, y[i]);
  }
  if (G >= 64) {
    mn = fminf(mn, quad_mov<kQuadXor1>(mn));
    mx = fmaxf(mx, quad_mov<kQuadXor1>(mx));
  }
  if (G >= 128) {
    mn = fminf(mn, quad_mov<kQuadXor2>(mn));
    mx = fmaxf(mx, quad_mov<kQuadXor2>(mx));
  }
  // rotated coordinates reach 128 * 65504 / 16 in magnitude: both parameters
  // saturate at +-65504
  uint16_t z16 = sat16(f2h(mn));
  z16 = z16 == 0x8000u ? uint16_t(0) : z16;
  const float zero = h2f(z16);
  const float s32 = __fdiv_rn(mx - zero, float(L - 1));
  const uint16_t s16 = sat16(f2h(s32 > 0.0f ? s32 : 0.0f));
  const float sf = h2f(s16);
  const float inv = sf == 0.0f ? 0.0f : __fdiv_rn(1.0f, sf);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    uint32_t w = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {                         // clamp, then round in the convert
      const float c = fminf(fmaxf((y[4 * k + e] - zero) * inv, 0.0f), float(L - 1));
      w = __builtin_amdgcn_cvt_pk_u8_f32(c, e, w);
    }
    code[k] = w;
  }
  return uint32_t(s16) | (uint32_t(z16) << 16);
}

// Quantize the quarter row held by this lane and write its metadata.
template <int BASE, int L>
__device__ void quantize_quarter(const PoolGeom& g, const float x[32], int q, int layer, int kvh,
                                 const float* tau, uint32_t code[8], uint8_t* meta_dst, int slot,
                                 bool valid) {
  if (BASE != 1) {
    const uint32_t m = BASE == 0 ? affine_quarter<L>(x, g.G, code)
                                 : rot_affine_quarter<L>(x, q, g.signs + (int64_t(layer) * g.n_kv_heads + kvh) * 4,
                                                         g.G, code);
    int per = g.G / 32;
    if (q % per == 0)
      reinterpret_cast<uint32_t*>(meta_dst)[(q / per) * kSlots + slot] = valid ? m : 0u;
  } else {
    const uint32_t* sw = g.signs + (int64_t(layer) * g.n_kv_heads + kvh) * 4;
    uint16_t r = tq_quarter<L>(x, q, sw, tau, code);
    if (q == 0) reinterpret_cast<uint16_t*>(meta_dst)[slot] = valid ? r : uint16_t(0);
  }
}

// OR the bits of one segment into an LDS body.  The segment holds symbols
// p = j, j+4, ... of a line of NV codes: code p*n+i of the line is at
// codes[(p*n+i)*stride].  J is compile-time: the symbols' widths and bit
// positions are constants, the line's offset is applied by one funnel shift
// per word.
template <int L, int NV, int NL, int J>
__device__ __forceinline__ void pack_segment_j(const uint8_t* codes, int stride, int line, uint32_t* body) {
  constexpr int n = sym_digits(L);
  constexpr SegTable<L, NV, NL> t{};
  constexpr int BITS = t.bits[J];
  constexpr int NWD = (BITS + 31) / 32 + 1;             // words, one spare for the shift
  uint32_t w[NWD];
#pragma unroll
  for (int k = 0; k < NWD; ++k) w[k] = 0u;
  int nb = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int wd = t.width[J][k], nd = t.ndig[J][k];
    if (wd > 0) {
      const int p = J + 4 * k;
      uint32_t v = 0;
#pragma unroll
      for (int i = n - 1; i >= 0; --i)
        if (i < nd) v = v * L + codes[(n * p + i) * stride];
      w[nb >> 5] |= v << (nb & 31);
      if ((nb & 31) + wd > 32) w[(nb >> 5) + 1] |= v >> (32 - (nb & 31));
      nb += wd;
    }
  }
  const int off = t.start[J] + line * BITS;
  const int w0 = off >> 5, sh = off & 31;
#pragma unroll
  for (int k = 0; k < NWD; ++k) {
    const uint32_t lo = k ? w[k - 1] : 0u;
    const uint32_t o = sh ? __builtin_amdgcn_alignbit(w[k], lo, 32 - sh) : w[k];
    if (32 * k < sh + BITS && o) atomicOr(&body[w0 + k], o);
  }
}

template <int L, int NV, int NL>
__device__ __forceinline__ void pack_segment(const uint8_t* codes, int stride, int line, int j, uint32_t* body) {
  switch (j) {                                          // j is the same for a whole wave
    case 0: pack_segment_j<L, NV, NL, 0>(codes, stride, line, body); break;
    case 1: pack_segment_j<L, NV, NL, 1>(codes, stride, line, body); break;
    case 2: pack_segment_j<L, NV, NL, 2>(codes, stride, line, body); break;
    default: pack_segment_j<L, NV, NL, 3>(codes, stride, line, body); break;
  }
}

// Decode one segment of an LDS body back into codes (used to extend a
// partially filled record when a generation block closes).
template <int L, int NV, int NL>
__device__ void unpack_segment(const uint32_t* body, int line, int j, uint8_t* codes, int stride) {
  constexpr int n = sym_digits(L);
  constexpr int S = num_syms(L, NV);
  constexpr SegTable<L, NV, NL> t{};
  int off = pick4(j, t.start[0], t.start[1], t.start[2], t.start[3]) +
            line * pick4(j, t.bits[0], t.bits[1], t.bits[2], t.bits[3]);
#pragma unroll
  for (int k = 0; 4 * k < S; ++k) {
    const int p = j + 4 * k;
    const int w = pick4(j, t.width[0][k], t.width[1][k], t.width[2][k], t.width[3][k]);
    const int nd = pick4(j, t.ndig[0][k], t.ndig[1][k], t.ndig[2][k], t.ndig[3][k]);
    if (w > 0) {
      int wd = off >> 5, sh = off & 31;
      uint64_t pair = uint64_t(body[wd]) | (uint64_t(body[wd + 1]) << 32);
      uint32_t v = uint32_t(pair >> sh) & ((1u << w) - 1u);
#pragma unroll
      for (int i = 0; i < n; ++i)
        if (i < nd) {
          codes[(n * p + i) * stride] = uint8_t(v % L);
          v /= L;
        }
      off += w;
    }
  }
}

template <int L>
__device__ __forceinline__ void pack_record(const uint8_t* ck, const uint8_t* cv, uint32_t* bk, uint32_t* bv) {
  int tid = threadIdx.x;
  pack_segment<L, kD, kSlots>(ck + (tid & 63) * kPitch, 1, tid & 63, tid >> 6, bk);
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    int s = tid + 256 * e;
    pack_segment<L, kSlots, kD>(cv + (s & 127), kPitch, s & 127, s >> 7, bv);
  }
}

__device__ void store_bodies(uint8_t* rec, const uint32_t* bk, const uint32_t* bv, int tb) {
  const uint4* sk = reinterpret_cast<const uint4*>(bk);
  const uint4* sv = reinterpret_cast<const uint4*>(bv);
  uint4* dk = reinterpret_cast<uint4*>(rec);
  uint4* dv = reinterpret_cast<uint4*>(rec + tb);
  for (int i = threadIdx.x; i < tb / 16; i += 256) {
    dk[i] = sk[i];
    dv[i] = sv[i];
  }
}

struct Lds {
  alignas(16) uint8_t ck[kSlots * kPitch];
  alignas(16) uint8_t cv[kSlots * kPitch];
  alignas(16) uint32_t bk[kMaxBodyWords + 8];
  alignas(16) uint32_t bv[kMaxBodyWords + 8];
};

template <int BASE, int L>
__device__ void prefill_record(const QuantArgs& a, Lds& s, int pool, int tile, int b, int l, int h) {
  const PoolGeom& g = a.g;
  int tid = threadIdx.x, r = tid >> 2, q = tid & 3;
  int64_t slot = int64_t(tile) * kSlots + r;
  bool valid = slot < a.n_pool[pool];
  int tok = valid ? a.idx[pool][int64_t(b) * a.n_pool[pool] + slot] : 0;
  if (tok < 0 || tok >= a.T) {             // a slot list not produced by semkv_rank
    if (valid) atomicOr(g.status, 4);
    tok = 0;
  }
  constexpr int tb = tile_bytes(L);
  uint8_t* rec = g.pools + unit_offset(g, b, l, h) + (pool ? g.lo_offset : 0) + int64_t(tile) * g.rec_bytes[pool];
  for (int i = tid; i < kMaxBodyWords + 8; i += 256) s.bk[i] = s.bv[i] = 0u;
  bool bad = false;
  const int64_t base_off = int64_t(l) * a.sL + int64_t(b) * a.sB + int64_t(h) * a.sH + int64_t(tok) * a.sT + 32 * q;
  float x[32];
  uint32_t code[8];
#pragma unroll
  for (int kv = 0; kv < 2; ++kv) {
    if (valid) {
      load_quarter((kv ? a.V : a.K) + base_off, x, bad);
    } else {
#pragma unroll
      for (int i = 0; i < 32; ++i) x[i] = 0.0f;
    }
    quantize_quarter<BASE, L>(g, x, q, l, h, g.tau[pool], code, rec + 2 * tb + kv * g.meta_bytes, r, valid);
    uint32_t* dst = reinterpret_cast<uint32_t*>((kv ? s.cv : s.ck) + r * kPitch + 32 * q);
#pragma unroll
    for (int i = 0; i < 8; ++i) dst[i] = valid ? code[i] : 0u;
  }
  if (bad && valid) atomicOr(g.status, 2);
  __syncthreads();
  pack_record<L>(s.ck, s.cv, s.bk, s.bv);
  __syncthreads();
  store_bodies(rec, s.bk, s.bv, tb);
}

template <int BASE, int LH, int LL>
__global__ __launch_bounds__(256) void quantize_pack_kernel(QuantArgs a) {
  __shared__ Lds s;
  int tile = blockIdx.x, pool = blockIdx.y & 1, h = blockIdx.y >> 1;
  int b = blockIdx.z / a.n_layers_launched, l = a.layer0 + blockIdx.z % a.n_layers_launched;
  if (int64_t(tile) * kSlots >= a.n_pool[pool]) return;
  if (pool == 0) prefill_record<BASE, LH>(a, s, 0, tile, b, l, h);
  else prefill_record<BASE, LL>(a, s, 1, tile, b, l, h);
}

// ---------------------------------------------------------------- close --

template <int BASE, int L>
__device__ void close_record(const CloseArgs& a, Lds& s, const int* row_of, int m, int pool,
                             int tile, int b, int l, int h) {
  const PoolGeom& g = a.g;
  int tid = threadIdx.x, r = tid >> 2, q = tid & 3;
  constexpr int tb = tile_bytes(L);
  uint8_t* rec = g.pools + unit_offset(g, b, l, h) + (pool ? g.lo_offset : 0) + int64_t(tile) * g.rec_bytes[pool];
  int64_t first = int64_t(tile) * kSlots;
  int64_t n0 = a.n0[pool];
  // existing rows of this record are unpacked; the rest start at code 0
  for (int i = tid; i < kMaxBodyWords + 8; i += 256) s.bk[i] = s.bv[i] = 0u;
  __syncthreads();
  if (first < n0) {
    const uint32_t* gk = reinterpret_cast<const uint32_t*>(rec);
    const uint32_t* gv = reinterpret_cast<const uint32_t*>(rec + tb);
    for (int i = tid; i < tb / 4; i += 256) {
      s.bk[i] = gk[i];
      s.bv[i] = gv[i];
    }
  }
  __syncthreads();
  unpack_segment<L, kD, kSlots>(s.bk, tid & 63, tid >> 6, s.ck + (tid & 63) * kPitch, 1);
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    int sg = tid + 256 * e;
    unpack_segment<L, kSlots, kD>(s.bv, sg & 127, sg >> 7, s.cv + (sg & 127), kPitch);
  }
  __syncthreads();
  int64_t slot = first + r;
  bool fresh = slot >= n0;                 // slots written by this close
  bool valid = fresh && slot < n0 + m;
  int row = valid ? row_of[slot - n0] : 0;
  bool bad = false;
  if (fresh) {
    const uint16_t* src = a.tail + ((((int64_t(b) * g.n_layers + l) * g.n_kv_heads + h) * 2) * kSlots + row) * kD + 32 * q;
    float x[32];
    uint32_t code[8];
#pragma unroll
    for (int kv = 0; kv < 2; ++kv) {
      if (valid) {
        load_quarter(src + kv * kSlots * kD, x, bad);
      } else {
#pragma unroll
        for (int i = 0; i < 32; ++i) x[i] = 0.0f;
      }
      quantize_quarter<BASE, L>(g, x, q, l, h, g.tau[pool], code, rec + 2 * tb + kv * g.meta_bytes, r, valid);
      uint32_t* dst = reinterpret_cast<uint32_t*>((kv ? s.cv : s.ck) + r * kPitch + 32 * q);
#pragma unroll
      for (int i = 0; i < 8; ++i) dst[i] = valid ? code[i] : 0u;
    }
  }
  if (bad && valid) atomicOr(g.status, 2);
  __syncthreads();
  for (int i = tid; i < kMaxBodyWords + 8; i += 256) s.bk[i] = s.bv[i] = 0u;
  __syncthreads();
  pack_record<L>(s.ck, s.cv, s.bk, s.bv);
  __syncthreads();
  store_bodies(rec, s.bk, s.bv, tb);
}

template <int BASE, int LH, int LL>
__global__ __launch_bounds__(256) void close_kernel(CloseArgs a) {
  __shared__ Lds s;
  __shared__ float sc[kSlots];
  __shared__ int cls[kSlots], row_of[2][kSlots];
  int tid = threadIdx.x;
  int pool = blockIdx.y & 1, h = blockIdx.y >> 1;
  int b = blockIdx.z / a.g.n_layers, l = blockIdx.z % a.g.n_layers;
  if (tid < a.n) {
    float v = a.tail_scores[int64_t(b) * kSlots + tid];
    sc[tid] = v == 0.0f ? 0.0f : v;
    if (isnan(v)) atomicOr(a.g.status, 1);
  }
  __syncthreads();
  if (tid < a.n) {                         // rank inside the block (Alg. 2)
    float v = sc[tid];
    int rank = 0;
    for (int j = 0; j < a.n; ++j) rank += (sc[j] > v || (sc[j] == v && j < tid)) ? 1 : 0;
    cls[tid] = rank < a.k_hi ? 0 : 1;
  }
  __syncthreads();
  if (tid < a.n) {
    int c = cls[tid], pos = 0;
    for (int j = 0; j < tid; ++j) pos += cls[j] == c ? 1 : 0;
    row_of[c][pos] = tid;
    if (c == 0 && pool == 0 && h == 0 && l == 0 && blockIdx.x == 0) {
      int64_t t = a.pos0 + tid;
      atomicOr(&a.flags[int64_t(b) * a.flag_words + (t >> 5)], 1u << (t & 31));
    }
  }
  __syncthreads();
  int m = pool == 0 ? a.k_hi : a.n - a.k_hi;
  int64_t n0 = a.n0[pool];
  int64_t tile = n0 / kSlots + blockIdx.x;
  if (m == 0 || tile > (n0 + m - 1) / kSlots) return;
  if (pool == 0) close_record<BASE, LH>(a, s, row_of[0], m, 0, int(tile), b, l, h);
  else close_record<BASE, LL>(a, s, row_of[1], m, 1, int(tile), b, l, h);
}

// ------------------------------------------------------------ dequant --

// The values one record holds, as decode attention sees them: affine
// x = fmaf(c, scale, zero); rotated affine x = sign . H y / 8 with y the
// affine value; tq x = sign . H (rho mu[c]) / 128.  One workgroup per record:
// the bodies are unpacked into LDS as for a block close, four lanes per slot.
template <int BASE, int L>
__device__ void dequant_record(const DequantArgs& a, Lds& s, int pool, int tile, int b, int h) {
  const PoolGeom& g = a.g;
  const int tid = threadIdx.x, r = tid >> 2, q = tid & 3;
  constexpr int tb = tile_bytes(L);
  const uint8_t* rec = g.pools + unit_offset(g, b, a.layer, h) + (pool ? g.lo_offset : 0) +
                       int64_t(tile) * g.rec_bytes[pool];
  for (int i = tid; i < kMaxBodyWords + 8; i += 256) s.bk[i] = s.bv[i] = 0u;
  __syncthreads();
  const uint32_t* gk = reinterpret_cast<const uint32_t*>(rec);
  const uint32_t* gv = reinterpret_cast<const uint32_t*>(rec + tb);
  for (int i = tid; i < tb / 4; i += 256) {
    s.bk[i] = gk[i];
    s.bv[i] = gv[i];
  }
  __syncthreads();
  unpack_segment<L, kD, kSlots>(s.bk, tid & 63, tid >> 6, s.ck + (tid & 63) * kPitch, 1);
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int sg = tid + 256 * e;
    unpack_segment<L, kSlots, kD>(s.bv, sg & 127, sg >> 7, s.cv + (sg & 127), kPitch);
  }
  __syncthreads();
  const int64_t slot = int64_t(tile) * kSlots + r;
  const bool valid = slot < a.n_rows[pool];
  const int64_t N = a.n_rows[0] + a.n_rows[1];
  const int64_t row = (pool ? a.n_rows[0] : 0) + slot;
  const uint32_t sbits = BASE != 0 ? g.signs[(int64_t(a.layer) * g.n_kv_heads + h) * 4 + q] : 0u;
#pragma unroll
  for (int kv = 0; kv < 2; ++kv) {
    const uint8_t* c = (kv ? s.cv : s.ck) + r * kPitch + 32 * q;
    const uint8_t* meta = rec + 2 * tb + kv * g.meta_bytes;
    float x[32];
    if (BASE != 1) {
      const uint32_t m = reinterpret_cast<const uint32_t*>(meta)[((32 * q) / g.G) * kSlots + r];
      const float sc = h2f(uint16_t(m & 0xFFFFu)), z = h2f(uint16_t(m >> 16));
#pragma unroll
      for (int i = 0; i < 32; ++i) x[i] = fmaf(float(c[i]), sc, z);
    } else {
      const float rho = h2f(reinterpret_cast<const uint16_t*>(meta)[r]);
      const float* mu = a.mu[pool];
#pragma unroll
      for (int i = 0; i < 32; ++i) x[i] = rho * mu[c[i] < L ? c[i] : 0];
    }
    if (BASE != 0) {                       // sign . H x, scaled back
      float u[32];
      rotate_quarter(x, q, 0u, u);
      const float k = BASE == 2 ? 0.125f : 1.0f / 128.0f;
#pragma unroll
      for (int i = 0; i < 32; ++i) x[i] = ((sbits >> i) & 1u) ? -u[i] * k : u[i] * k;
    }
    float* dst = (kv ? a.v_hat : a.k_hat) + ((int64_t(b) * g.n_kv_heads + h) * N + row) * kD + 32 * q;
    if (valid) {
#pragma unroll
      for (int i = 0; i < 32; i += 4) *reinterpret_cast<float4*>(dst + i) = make_float4(x[i], x[i + 1], x[i + 2], x[i + 3]);
    }
  }
}

template <int BASE, int LH, int LL>
__global__ __launch_bounds__(256) void dequant_kernel(DequantArgs a) {
  __shared__ Lds s;
  const int tile = blockIdx.x, pool = blockIdx.y & 1, h = blockIdx.y >> 1, b = blockIdx.z;
  if (int64_t(tile) * kSlots >= a.n_rows[pool]) return;
  if (pool == 0) dequant_record<BASE, LH>(a, s, 0, tile, b, h);
  else dequant_record<BASE, LL>(a, s, 1, tile, b, h);
}

__global__ void append_kernel(AppendArgs a) {
  // one block per (layer, b, kv head); 64 threads copy K and V rows
  int z = blockIdx.x;
  int h = z % a.n_kv_heads;
  int b = (z / a.n_kv_heads) % a.batch;
  int li = z / (a.n_kv_heads * a.batch);
  int l = a.layer0 + li;
  const uint32_t* k = reinterpret_cast<const uint32_t*>(a.k + ((int64_t(li) * a.batch + b) * a.n_kv_heads + h) * kD);
  const uint32_t* v = reinterpret_cast<const uint32_t*>(a.v + ((int64_t(li) * a.batch + b) * a.n_kv_heads + h) * kD);
  uint32_t* dst = reinterpret_cast<uint32_t*>(a.tail + ((((int64_t(b) * a.n_layers + l) * a.n_kv_heads + h) * 2) * kSlots + a.slot) * kD);
  int t = threadIdx.x;
  dst[t] = k[t];
  dst[kSlots * kD / 2 + t] = v[t];
}

template <int BASE, int LH, int LL>
int launch_qp(const QuantArgs& a, hipStream_t st) {
  dim3 grid(a.max_tiles, 2 * a.g.n_kv_heads, a.g.batch * a.n_layers_launched);
  hipLaunchKernelGGL((quantize_pack_kernel<BASE, LH, LL>), grid, dim3(256), 0, st, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

template <int BASE, int LH, int LL>
int launch_dq(const DequantArgs& a, hipStream_t st) {
  const int64_t mt = ((a.n_rows[0] > a.n_rows[1] ? a.n_rows[0] : a.n_rows[1]) + kSlots - 1) / kSlots;
  dim3 grid(unsigned(mt), 2 * a.g.n_kv_heads, a.g.batch);
  hipLaunchKernelGGL((dequant_kernel<BASE, LH, LL>), grid, dim3(256), 0, st, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

template <int BASE, int LH, int LL>
int launch_cl(const CloseArgs& a, hipStream_t st) {
  dim3 grid(2, 2 * a.g.n_kv_heads, a.g.batch * a.g.n_layers);
  hipLaunchKernelGGL((close_kernel<BASE, LH, LL>), grid, dim3(256), 0, st, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace

#define SEMKV_DISPATCH_LEVELS(BASE, LH, LL, FN, ...)                                  \
  if (BASE == 0 && LH == 6 && LL == 5) return FN<0, 6, 5>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 5 && LL == 4) return FN<0, 5, 4>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 6 && LL == 4) return FN<0, 6, 4>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 4 && LL == 3) return FN<0, 4, 3>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 5 && LL == 3) return FN<0, 5, 3>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 6 && LL == 3) return FN<0, 6, 3>(__VA_ARGS__);              \
  if (BASE == 1 && LH == 4 && LL == 3) return FN<1, 4, 3>(__VA_ARGS__);              \
  if (BASE == 2 && LH == 6 && LL == 5) return FN<2, 6, 5>(__VA_ARGS__);              \
  if (BASE == 2 && LH == 5 && LL == 4) return FN<2, 5, 4>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 8 && LL == 7) return FN<0, 8, 7>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 7 && LL == 6) return FN<0, 7, 6>(__VA_ARGS__);              \
  if (BASE == 0 && LH == 3 && LL == 2) return FN<0, 3, 2>(__VA_ARGS__);              \
  if (BASE == 2 && LH == 8 && LL == 7) return FN<2, 8, 7>(__VA_ARGS__);              \
  if (BASE == 2 && LH == 7 && LL == 6) return FN<2, 7, 6>(__VA_ARGS__);              \
  if (BASE == 2 && LH == 3 && LL == 2) return FN<2, 3, 2>(__VA_ARGS__);              \
  return -2;

int launch_quantize(const QuantArgs& a, hipStream_t s) {
  SEMKV_DISPATCH_LEVELS(a.g.base, a.g.L[0], a.g.L[1], launch_qp, a, s)
}

int launch_close(const CloseArgs& a, hipStream_t s) {
  SEMKV_DISPATCH_LEVELS(a.g.base, a.g.L[0], a.g.L[1], launch_cl, a, s)
}

int launch_dequant(const DequantArgs& a, hipStream_t s) {
  SEMKV_DISPATCH_LEVELS(a.g.base, a.g.L[0], a.g.L[1], launch_dq, a, s)
}

int launch_append(const AppendArgs& a, hipStream_t s) {
  dim3 grid(a.n_layers_launched * a.batch * a.n_kv_heads);
  hipLaunchKernelGGL(append_kernel, grid, dim3(64), 0, s, a);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // namespace semkv
