// decode.hip -- split-K GQA decode attention over the mixed-precision cache
// (the decoding consumer of SemKV, Sec. 3.1 and Alg. 1), for gfx950.
//
// Work split: a (sequence, kv head) unit's tiles -- its high pool, then its
// low pool -- are dealt to nsplit workgroups of NW waves (nsplit chosen by the
// host so that the whole grid is resident at once): tile u goes to wave slot
// u mod (nsplit NW), slot v = w nsplit + s being wave w of workgroup s.  Every
// wave thus gets an even share of the (costlier) high-precision tiles, first
// in its sequence, and keeps its own online-softmax state for the 4 query
// heads of the kv head.  Records are staged through registers: the next record's
// 16-byte pieces are loaded while the current one is computed from the wave's
// LDS buffer, then written over it.  Products run on the int8 matrix cores
// (v_mfma_i32_16x16x64_i8), exact in their integer sums.  Per record:
//   scores  C[16 rows (head, byte) x 16 tokens] += A B: A holds the query of
//           head h as a fixed-point integer qi = rint(q 2^e) (|qi| < 2^20, e
//           per head and metadata group) split into three bytes, one per row,
//           restricted to one metadata group; B the base-L digits of 16
//           tokens as bytes, decoded from the packed K symbols through LDS
//           tables (one dword of digit bytes per entry).  The affine
//           dequantization x = s c + z is folded out:
//           q.x = s (q.c) + z (sum q) per group.
//   softmax online, base 2; unnormalized p, rescaled when the maximum moves.
//   values  C[16 rows (head, byte) x 16 channels] += A[16 x 64 tokens]
//           B[64 tokens x 16 channels] with A the weights p * s as 21-bit
//           integers (one power-of-2 scale per head, three bytes in three
//           rows) and B the V digits (V symbols run along tokens).  The
//           integer sums run across records and are folded into float sums
//           only when the running maximum moves or a record's weights would
//           not fit the scale.
// The last run also takes the fp16 tail of generated tokens.  The waves'
// states merge in LDS into one partial per workgroup; the last workgroup of a
// unit to finish merges the partials (log-sum-exp) and, for the rotated bases
// (TurboQuant-MSE, and the affine base under its Hadamard rotation), applies
// the inverse random-sign Hadamard rotation.
// Bases: 0 affine, 1 TurboQuant-MSE, 2 affine of the rotated row.  Bases 0
// and 2 share the affine levels and metadata; bases 1 and 2 score against the
// rotated query H diag(sign) q and accumulate values in the rotated domain.
#include <hip/hip_fp16.h>

#include "semkv_internal.h"

namespace semkv {

// ---- tracing build only (-DSEMKV_TIMELINE, libsemkv_timeline.so): lane 0 of
// every wave of the first kTimelineWGs workgroups of a launch records the
// constant 100 MHz clock at the ends of the kernel's phases (event ids below);
// a later launch overwrites the stamps.  The product library compiles every
// stamp to nothing.
#ifdef SEMKV_TIMELINE
constexpr int kTimelineWGs = 4096, kTimelineWaves = 16, kTimelineEvents = 32;
__device__ unsigned long long g_timeline[kTimelineWGs * kTimelineWaves * kTimelineEvents];
__device__ inline void timeline_stamp(int ev) {
  const int wg = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  if ((threadIdx.x & 63) == 0 && wg < kTimelineWGs)
    g_timeline[(wg * kTimelineWaves + (threadIdx.x >> 6)) * kTimelineEvents + ev] = wall_clock64();
}
// slots 14 and 15 of a wave hold counts, kept in the wave's state and
// written once (a read-modify-write of memory in the record loop would wait
// for the loads in flight)
__device__ inline void timeline_put(int ev, unsigned long long v) {
  const int wg = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  if ((threadIdx.x & 63) == 0 && wg < kTimelineWGs)
    g_timeline[(wg * kTimelineWaves + (threadIdx.x >> 6)) * kTimelineEvents + ev] = v;
}
#define SEMKV_STAMP(ev) timeline_stamp(ev)
#else
#define SEMKV_STAMP(ev) ((void)0)
#endif
// the stamps inside the prologue and the first record (16..21) delay what they
// measure: compiled in only with -DSEMKV_TIMELINE_FINE as well
#if defined(SEMKV_TIMELINE) && defined(SEMKV_TIMELINE_FINE)
#define SEMKV_STAMP_FINE(ev) SEMKV_STAMP(ev)
#else
#define SEMKV_STAMP_FINE(ev) ((void)0)
#endif
// 0 start, 1 tables and query operands built, 2 first record in LDS,
// 3..7 the wave's 1st..5th record done, the next record's data stored in LDS
// (a 6th and later overwrite 7), 8 the first record's arithmetic done (before
// the next record's data is waited for), 16..18 inside the first record: the
// next record's loads issued, scores done, softmax and flush done, 19..21 in
// the prologue: tables written, query value in hand, query runs done,
// 9 the wave's records done, 10 workgroup partial merged, 11 partial stored,
// 12 split counter taken, 13 the last workgroup's merge done; counts: 14 the
// wave's value-sum flushes, 15 its records (both cleared at the wave's start)

namespace {

typedef int32_t int4v __attribute__((ext_vector_type(4)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef uint32_t uint4v __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRsqrtD = 0.08838834764831845f;   // 1 / sqrt(128)
constexpr int kQPad = 160;                         // query rows, zero past channel 127

// ------------------------------------------------------------ traits ----

__host__ __device__ constexpr int ipow(int b, int e) {
  int r = 1;
  for (int i = 0; i < e; ++i) r *= b;
  return r;
}

// Chunk layout: an MFMA operand gives each lane 16 byte slots; a chunk fills
// them with SPC symbols of STRIDE slots each; slot_digit / slot_plane give the
// code a slot holds (-1: a zero pad slot).  4-level codes of the tq base take
// two slots, their low and high bit (the Lloyd-Max levels are affine in those
// bits).
template <int BASE, int L>
struct Traits {
  static constexpr int n = sym_digits(L);
  static constexpr int P = (BASE == 1 && L == 4) ? 2 : 1;   // MFMA slots per code
  static constexpr int STRIDE = (L == 5 || L == 8 || (L == 4 && BASE != 1)) ? 4 : 8;
  static constexpr int SPC = 16 / STRIDE;
  static constexpr int EDW = STRIDE / 4;                     // operand dwords per symbol
  static constexpr int SK = num_syms(L, kD), SV = num_syms(L, kSlots);
  static constexpr int NSK = (SK + 3) / 4, NSV = (SV + 3) / 4;
  static constexpr int NCK = (NSK + SPC - 1) / SPC, NCV = (NSV + SPC - 1) / SPC;
  static constexpr int W = width_of(L, n);
  static constexpr int TB = tile_bytes(L);
  static constexpr int KSEGW = (NSK * W + 31) / 32;          // normalized dwords of a K segment
  static constexpr int VSEGW = (NSV * W + 31) / 32;
  // decode table: symbol -> operand dwords of digit bytes.  L = 6 splits a
  // symbol into s mod 1296 (4 codes, one table dword) and s div 1296 (the
  // fifth code, which is its own operand dword: no table); L = 7 into s mod
  // 2401 (4 codes) and s div 2401 (3 codes), one table dword each.
  static constexpr bool SPLIT = L == 6 || L == 7;
  static constexpr int DIV = L == 6 ? 1296 : L == 7 ? 2401 : 1;  // the split's divisor
  static constexpr int TED = SPLIT ? 1 : EDW;                // dwords per table entry
  static constexpr int NENT = L == 6 ? DIV : SPLIT ? DIV + ipow(L, n) / DIV : ipow(L, n);   // entries
  static constexpr int LUTDW = NENT * TED;                   // dwords of one copy
};

template <int BASE, int L>
__host__ __device__ constexpr int slot_digit(int w) {
  return (BASE == 1 && L == 4) ? w / 2
       : L == 6 ? (w < 5 ? w : -1)
       : L == 5 ? (w < 3 ? w : -1)
       : L == 3 ? (w < 5 ? w : -1)
       : L == 7 ? (w < 7 ? w : -1)
       : L == 8 ? (w < 2 ? w : -1)
       : w;                                                  // affine L = 4, L = 2
}
template <int BASE, int L>
__host__ __device__ constexpr int slot_plane(int w) { return (BASE == 1 && L == 4) ? w % 2 : 0; }
// the slot (within a symbol's STRIDE slots) of code d, plane 0: the inverse
// of slot_digit / slot_plane
template <int BASE, int L>
__host__ __device__ constexpr int digit_slot(int d) {
  return (BASE == 1 && L == 4) ? 2 * d : d;
}
template <int BASE, int L>
__host__ __device__ constexpr bool digit_slot_inverts() {
  for (int d = 0; d < sym_digits(L); ++d) {
    const int w = digit_slot<BASE, L>(d);
    if (w < 0 || w >= 8 || slot_digit<BASE, L>(w) != d || slot_plane<BASE, L>(w) != 0) return false;
  }
  return true;
}
static_assert(digit_slot_inverts<0, 6>() && digit_slot_inverts<0, 5>() && digit_slot_inverts<0, 4>() &&
              digit_slot_inverts<0, 3>() && digit_slot_inverts<1, 4>() && digit_slot_inverts<1, 3>() &&
              digit_slot_inverts<0, 2>() && digit_slot_inverts<0, 7>() && digit_slot_inverts<0, 8>(), "slots");

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
static_assert(magic_exact(6), "digit extraction");

__device__ inline uint32_t mulhi24(uint32_t a, uint32_t b) {
  return uint32_t((uint64_t(a & 0xFFFFFFu) * uint64_t(b & 0xFFFFFFu)) >> 32);
}

// a * b + c on 24-bit signed a, b: one full-rate v_mad_i32_i24 (left to
// itself the compiler widens this to a 64-bit multiply-add)
__device__ inline uint32_t mad_i24(uint32_t a, int b, uint32_t c) {
  uint32_t r;
  __asm__("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(b), "v"(c));
  return r;
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

// ------------------------------------------------------ decode tables ----

// Dword K of table entry E: the digit bytes of operand slots 4K .. 4K+3 of
// symbol value E (L = 6: entry E < 1296 gives the four codes of s mod 1296 ->
// slots 0-3; slot 4 holds s div 1296 itself).
template <int BASE, int L, int K>
__host__ __device__ constexpr uint32_t entry_dword(uint32_t E) {
  using Tr = Traits<BASE, L>;
  if constexpr (L == 6) {
    return (E % 6) | ((E / 6 % 6) << 8) | ((E / 36 % 6) << 16) | ((E / 216) << 24);
  } else if constexpr (L == 7) {                             // s mod 2401: 4 codes; s div 2401: 3 codes
    const bool hi = E >= 2401;
    const uint32_t v = hi ? E - 2401 : E;
    return (v % 7) | ((v / 7 % 7) << 8) | ((v / 49 % 7) << 16) | (hi ? 0u : (v / 343) << 24);
  } else {
    uint32_t w = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int wsl = 4 * K + j, dg = slot_digit<BASE, L>(wsl);
      if (dg >= 0) {
        const uint32_t p = uint32_t(ipow(L, dg)), c = E / p - (E / (p * L)) * L;
        const uint32_t d = slot_plane<BASE, L>(wsl) ? (c >> 1) : (Tr::P == 2 ? (c & 1u) : c);
        w |= d << (8 * j);
      }
    }
    return w;
  }
}

// the digits a table entry gives, checked against plain base-L arithmetic
// (L = 6: the four codes of s mod 1296; L = 7: the entries of both parts,
// which cover every symbol through s mod 2401 and s div 2401)
template <int BASE, int L>
__host__ __device__ constexpr bool entries_match_digits() {
  using Tr = Traits<BASE, L>;
  const int nent = Tr::NENT;
  for (int E = 0; E < nent; ++E) {
    for (int w = 0; w < Tr::STRIDE; ++w) {
      uint32_t byte = 0, want = 0;
      if (L == 6) {
        // entries are s mod 1296: four codes in slots 0-3 (slot 4, the
        // quotient, is not tabled)
        if (w >= 4) continue;
        byte = (entry_dword<BASE, L, 0>(uint32_t(E)) >> (8 * w)) & 0xFFu;
        int c = E;
        for (int t = 0; t < w; ++t) c /= L;
        want = uint32_t(c % L);
      } else if (Tr::SPLIT) {
        // the low part's entry gives the first four digits of base 7 in
        // slots 0-3, the high part's the rest from slot 4 on
        const bool hi = w >= 4;
        if (hi != (E >= Tr::DIV)) continue;
        byte = (entry_dword<BASE, L, 0>(uint32_t(E)) >> (8 * (w % 4))) & 0xFFu;
        const int v = hi ? E - Tr::DIV : E, first = 4;
        const int dg = slot_digit<BASE, L>(w) - (hi ? first : 0);
        if (slot_digit<BASE, L>(w) >= 0) {
          int c = v;
          for (int t = 0; t < dg; ++t) c /= L;
          want = uint32_t(c % L);
        }
      } else {
        const uint32_t dw = w < 4 ? entry_dword<BASE, L, 0>(uint32_t(E)) : entry_dword<BASE, L, 1>(uint32_t(E));
        byte = (dw >> (8 * (w % 4))) & 0xFFu;
        const int dg = slot_digit<BASE, L>(w);
        if (dg >= 0) {
          int c = E;
          for (int t = 0; t < dg; ++t) c /= L;
          c %= L;
          want = slot_plane<BASE, L>(w) ? uint32_t(c >> 1) : (Tr::P == 2 ? uint32_t(c & 1) : uint32_t(c));
        }
      }
      if (byte != want) return false;
    }
  }
  return true;
}
static_assert(entries_match_digits<0, 6>() && entries_match_digits<0, 5>() && entries_match_digits<0, 4>() &&
              entries_match_digits<0, 3>() && entries_match_digits<1, 4>() && entries_match_digits<1, 3>() &&
              entries_match_digits<0, 2>() && entries_match_digits<0, 7>() && entries_match_digits<0, 8>(), "tables");

// 16-byte piece q of the replicated LDS table (entry e of replica r at entry
// slot e R + r; R >= 4, so a piece lies in one entry, repeated)
template <int BASE, int L, int R>
__device__ inline uint4 lut_piece(uint32_t q) {
  using Tr = Traits<BASE, L>;
  static_assert(R >= 4 && (R & (R - 1)) == 0, "replicas");
  if constexpr (Tr::TED == 1) {
    const uint32_t x = entry_dword<BASE, L, 0>((4 * q) / R);
    return make_uint4(x, x, x, x);
  } else {
    const uint32_t E = (2 * q) / R, x = entry_dword<BASE, L, 0>(E), y = entry_dword<BASE, L, 1>(E);
    return make_uint4(x, y, x, y);
  }
}

// Bits [OFF, OFF+W) of a normalized segment moved to bit S; the bits around
// them are junk (the caller masks them off).
template <int OFF, int W, int S, int NW>
__device__ inline uint32_t field_at(const uint32_t (&seg)[NW]) {
  constexpr int w = OFF / 32, sh = OFF % 32;
  if constexpr (sh + W <= 32) {
    if constexpr (sh >= S) return sh == S ? seg[w] : seg[w] >> (sh - S);
    else return seg[w] << (S - sh);
  } else {
    static_assert(sh >= S, "field position");
    return __builtin_amdgcn_alignbit(seg[w + 1], seg[w], sh - S);
  }
}

// (a << s) | c and (a & b) | c as single instructions (the compiler turns the
// OR of disjoint bits into an add and re-associates the table's base address
// into it, which costs an instruction per symbol)
__device__ inline uint32_t lshl_or(uint32_t a, int s, uint32_t c) {
  uint32_t r;
  __asm__("v_lshl_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(s), "v"(c));
  return r;
}
__device__ inline uint32_t and_or(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t r;
  __asm__("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// (symbol K of a segment) << S | lbase; a symbol past the line's last is 0.
// FULL has bit K set when symbol K has the full width in every segment (its
// lane mask is then a constant).
template <int BASE, int L, int S, uint32_t FULL, int K, int NW, int NS>
__device__ inline uint32_t sym_addr(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], uint32_t lbase) {
  using Tr = Traits<BASE, L>;
  if constexpr (K >= NS) {
    return lbase;
  } else {
    constexpr int OFF = K * Tr::W, sh = OFF % 32;
    if constexpr (((FULL >> K) & 1u) && sh + Tr::W <= 32)
      return lshl_or((seg[OFF / 32] >> sh) & ((1u << Tr::W) - 1u), S, lbase);
    else
      return and_or(field_at<OFF, Tr::W, S, NW>(seg), maskS[K], lbase);
  }
}

// bit K set when symbol K of a line of NVALS codes has the full width in all
// four segments
template <int L, int NVALS, int NLINES>
__host__ __device__ constexpr uint32_t full_symbols() {
  constexpr SegTable<L, NVALS, NLINES> t{};
  uint32_t f = 0;
  for (int k = 0; k < 16; ++k) {
    bool all = true;
    for (int j = 0; j < 4; ++j) all = all && t.width[j][k] == width_of(L, sym_digits(L));
    if (all) f |= 1u << k;
  }
  return f;
}

// A lane's view of its pool's LDS tables: entry e of its replica is at byte
// (e << S) + lbase of t; for L = 7 the s div 2401 part starts at hbase.
struct LutRef {
  const uint8_t* t;
  uint32_t lbase, hbase;
};

__host__ __device__ constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// floor(v / 1296) for v < 6^5 as the high word of x * M with x = (v << S) + b,
// b < 2^S a multiple of 4 (the lane's replica offset): the least M above
// 2^(32-S) / 1296 that is exact for every v at both ends of b (x * M does not
// decrease with b), found at compile time.
__host__ __device__ constexpr bool magic1296_ok(int S, uint64_t M) {
  if (M >= (1u << 24) || (7775u << S) + (1u << S) >= (1u << 24)) return false;
  const uint64_t bmax = (1u << S) - 4;
  for (uint64_t v = 0; v < 7776; ++v)
    if (((v << S) * M) >> 32 != v / 1296 || (((v << S) + bmax) * M) >> 32 != v / 1296) return false;
  return true;
}
__host__ __device__ constexpr uint32_t magic1296(int S) {
  const uint64_t m0 = ((uint64_t(1) << (32 - S)) + 1295) / 1296;
  for (uint64_t M = m0; M < m0 + 64; ++M)
    if (magic1296_ok(S, M)) return uint32_t(M);
  return 0u;
}

// floor(v / 2401) for v < 7^7 as the high word of v * 1788825 (v and the
// multiplier fit 24 bits).  floor(v M / 2^32) does not decrease with v, so it
// is exact everywhere when it is exact on both sides of every multiple of 2401.
constexpr uint32_t kMagic2401 = 1788825u;
__host__ __device__ constexpr bool magic2401_exact() {
  if (kMagic2401 >= (1u << 24) || 823542u >= (1u << 24)) return false;
  for (uint64_t k = 1; k <= 343; ++k) {
    const uint64_t below = 2401 * k - 1, at = 2401 * k;
    if ((below * kMagic2401) >> 32 != k - 1) return false;
    if (at < 823543 && (at * kMagic2401) >> 32 != k) return false;
  }
  return true;
}
static_assert(magic2401_exact(), "7-level digit split");

// operand dwords of 7-level symbol K: the s mod 2401 and s div 2401 entries
template <int BASE, int S, uint32_t FULL, int K, int NW, int NS>
__device__ inline uint2 l7_symbol(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], const LutRef& lr) {
  const uint32_t x = sym_addr<BASE, 7, S, FULL, K, NW, NS>(seg, maskS, 0u);   // v << S
  const uint32_t hi = mulhi24(x >> S, kMagic2401);                           // v div 2401
  const uint32_t lo = mad_i24(hi, -(2401 << S), x) + lr.lbase;                // ((v mod 2401) << S) + lbase
  return make_uint2(*reinterpret_cast<const uint32_t*>(lr.t + lo),
                    *reinterpret_cast<const uint32_t*>(lr.t + ((hi << S) + lr.hbase)));
}

// operand dwords of 6-level symbol K: the s mod 1296 entry (codes 0-3) and
// s div 1296 (code 4, a value below 6: its own operand dword)
template <int BASE, int S, uint32_t FULL, int K, int NW, int NS>
__device__ inline uint2 l6_symbol(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], const LutRef& lr) {
  constexpr uint32_t M = magic1296(S);
  static_assert(M != 0, "digit split");
  const uint32_t x = sym_addr<BASE, 6, S, FULL, K, NW, NS>(seg, maskS, lr.lbase);   // (v << S) + lbase
  const uint32_t hi = mulhi24(x, M);                                                // v div 1296
  const uint32_t lo = mad_i24(hi, -(1296 << S), x);                                 // ((v mod 1296) << S) + lbase
  return make_uint2(*reinterpret_cast<const uint32_t*>(lr.t + lo), hi);
}

// Operand dwords of symbol slot K of a segment.  A slot past the longest
// segment (K >= NS, known at compile time) holds no symbol in any lane: its
// digits are zero and no table is read.  Slots of lanes whose segment is one
// symbol shorter read table entry 0 (all digits zero) through a zero mask.
template <int BASE, int L, int S, uint32_t FULL, int K, int NW, int NS>
__device__ inline uint32_t sym_dword(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], const LutRef& lr) {
  if constexpr (K >= NS) return 0u;
  else return *reinterpret_cast<const uint32_t*>(lr.t + sym_addr<BASE, L, S, FULL, K, NW, NS>(seg, maskS, lr.lbase));
}
template <int BASE, int L, int S, uint32_t FULL, int K, int NW, int NS>
__device__ inline uint2 sym_dword2(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], const LutRef& lr) {
  if constexpr (K >= NS) return make_uint2(0u, 0u);
  else return *reinterpret_cast<const uint2*>(lr.t + sym_addr<BASE, L, S, FULL, K, NW, NS>(seg, maskS, lr.lbase));
}

// MFMA operand of chunk C of a segment (symbols SPC*C ..), read from the tables
template <int BASE, int L, int S, uint32_t FULL, int C, int NW, int NS>
__device__ inline int4v chunk_operand(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], const LutRef& lr) {
  using Tr = Traits<BASE, L>;
  uint4v r;
  if constexpr (L == 6 || L == 7) {
    uint2 p0 = make_uint2(0u, 0u), p1 = make_uint2(0u, 0u);
    if constexpr (L == 6) {
      if constexpr (2 * C < NS) p0 = l6_symbol<BASE, S, FULL, 2 * C, NW, NS>(seg, maskS, lr);
      if constexpr (2 * C + 1 < NS) p1 = l6_symbol<BASE, S, FULL, 2 * C + 1, NW, NS>(seg, maskS, lr);
    } else {
      if constexpr (2 * C < NS) p0 = l7_symbol<BASE, S, FULL, 2 * C, NW, NS>(seg, maskS, lr);
      if constexpr (2 * C + 1 < NS) p1 = l7_symbol<BASE, S, FULL, 2 * C + 1, NW, NS>(seg, maskS, lr);
    }
    r = uint4v{p0.x, p0.y, p1.x, p1.y};
  } else if constexpr (Tr::SPC == 4) {
    r = uint4v{sym_dword<BASE, L, S, FULL, 4 * C, NW, NS>(seg, maskS, lr),
               sym_dword<BASE, L, S, FULL, 4 * C + 1, NW, NS>(seg, maskS, lr),
               sym_dword<BASE, L, S, FULL, 4 * C + 2, NW, NS>(seg, maskS, lr),
               sym_dword<BASE, L, S, FULL, 4 * C + 3, NW, NS>(seg, maskS, lr)};
  } else {
    const uint2 a = sym_dword2<BASE, L, S, FULL, 2 * C, NW, NS>(seg, maskS, lr);
    const uint2 b = sym_dword2<BASE, L, S, FULL, 2 * C + 1, NW, NS>(seg, maskS, lr);
    r = uint4v{a.x, a.y, b.x, b.y};
  }
  return __builtin_bit_cast(int4v, r);
}

// MFMA operands of all NC chunks of a segment: every table read is issued
// before the first product needs one (LDS returns them in order)
template <int BASE, int L, int S, uint32_t FULL, int NW, int NS, int NC>
__device__ inline void chunk_operands(const uint32_t (&seg)[NW], const uint32_t (&maskS)[NS], const LutRef& lr,
                                      int4v (&A)[NC]) {
  static_assert(NC <= 4, "chunks");
#define SEMKV_O(C) if constexpr (C < NC) A[C] = chunk_operand<BASE, L, S, FULL, C, NW, NS>(seg, maskS, lr);
  SEMKV_O(0) SEMKV_O(1) SEMKV_O(2) SEMKV_O(3)
#undef SEMKV_O
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

template <int BASE, int L, int G>
struct Geo {
  using Tr = Traits<BASE, L>;
  static constexpr int MB = meta_bytes(BASE, G);
  static constexpr int RB = 2 * Tr::TB + 2 * MB;
  static constexpr int NLD = (RB + 1023) / 1024;            // 1 KB staging pieces per record
  static constexpr int NG = BASE != 1 ? kD / G : 1;          // score products per chunk (query groups)
  static constexpr int NGV = BASE != 1 ? kD / G : 1;         // value groups
  static constexpr int NPL = Tr::P;                          // value planes (tq, 4 levels: 2)
  // int8 weights of one wave and one value group at a time, in value
  // A-operand order: [chunk][lane group][row][16 slots], so a lane reads a
  // chunk's operand at once.  Row 4h + s holds byte s of head h's weights;
  // rows 4h + 3, pad slots and slots past token 63 are never written and
  // stay zero.
  // lane groups 272 bytes apart (16 rows of 16 slots, then 16 bytes of pad):
  // the byte writes of consecutive symbols, which sit in consecutive lane
  // groups, land in different LDS banks rather than all in one
  static constexpr int KGS = 16 * 16 + 16;                   // bytes per lane group
  static constexpr int CHB = 4 * KGS;                        // bytes per chunk
  static constexpr int PV = Tr::NCV * CHB;                   // bytes per wave
  static_assert(RB % 16 == 0, "record pieces");
};

template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
// reductions over the 16 lanes of a row (row_ror 8, 4, 2, 1).  The maximum
// is four DPP maxima written out: fmaxf of a DPP move costs three
// instructions a step (the move, a quieting max of the moved value that the
// IEEE-mode maxNum contract asks of an operand not known to be canonical, the
// max), and the values here are never NaN.  Every DPP read of a register
// written by the VALU instruction just before it needs two wait states, which
// the compiler does not insert around inline assembly: hence the s_nop 1
// before each (and after the last, for a DPP read that may follow).
// Called with the whole wave active.
__device__ inline float row_max16(float x) {
  float r;
  __asm__("s_nop 1\n\t"
          "v_max_f32_dpp %0, %1, %1 row_ror:8 row_mask:0xf bank_mask:0xf\n\t"
          "s_nop 1\n\t"
          "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n\t"
          "s_nop 1\n\t"
          "v_max_f32_dpp %0, %0, %0 row_ror:2 row_mask:0xf bank_mask:0xf\n\t"
          "s_nop 1\n\t"
          "v_max_f32_dpp %0, %0, %0 row_ror:1 row_mask:0xf bank_mask:0xf\n\t"
          "s_nop 1"
          : "=&v"(r) : "v"(x));
  return r;
}
// max of four values that are never NaN (no quieting of operands)
__device__ inline float max4(float a, float b, float c, float d) {
  float r;
  __asm__("v_max3_f32 %0, %1, %2, %3\n\t"
          "v_max_f32 %0, %0, %4"
          : "=&v"(r) : "v"(a), "v"(b), "v"(c), "v"(d));
  return r;
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

// ------------------------------------------------------- kernel layout ----

template <int BASE, int LH, int LL, int G>
struct Plan {
  using GH = Geo<BASE, LH, G>;
  using GL = Geo<BASE, LL, G>;
  static constexpr int NLD = GH::NLD > GL::NLD ? GH::NLD : GL::NLD;
  static constexpr int PV = GH::PV > GL::PV ? GH::PV : GL::PV;
  static constexpr int NGV = GH::NGV;
  static constexpr int NG = GH::NG;
  static constexpr int NCKH = Traits<BASE, LH>::NCK, NCKL = Traits<BASE, LL>::NCK;
  static_assert(GH::NGV == GL::NGV, "pools share the value groups");
  // LDS of a workgroup of nw waves with rh / rl table replicas (the Shared
  // layout below, with margin)
  static constexpr int lds_bytes(int nw, int rh, int rl) {
    return nw * (NLD * 1024 + PV + 256) + (Traits<BASE, LH>::LUTDW * rh + Traits<BASE, LL>::LUTDW * rl) * 4 +
           NG * (NCKH + NCKL) * 64 * 16 + 4 * kQPad * 4 + 4 * kD * 4 + 2080 + 3104 + 512;
  }
  // 8 waves: 2 per SIMD, one workgroup per compute unit.  A level pair whose
  // 8-wave workgroup does not fit is refused by the host.
  static constexpr int NW = lds_bytes(8, 4, 4) <= 160 * 1024 ? 8 : 4;
  static constexpr int NT = 64 * NW;
  // table replicas per pool: the most that fit, the low pool (the larger
  // share of the tokens) first (32 dword replicas: a conflict-free lookup of
  // any entries)
  // (the 7-level tables, 2744 entries, keep 4 replicas: 44 KB; the 6-level
  // table, 1296 entries, at most 8: 41 KB)
  static constexpr int cap(int L) { return L == 7 ? 4 : L == 6 ? 8 : 32; }
  static constexpr int pick_replicas(bool hi) {
    constexpr int opts[8][2] = {{32, 32}, {16, 32}, {8, 32}, {16, 16}, {8, 16}, {8, 8}, {4, 8}, {4, 4}};
    for (const auto& o : opts) {
      const int rh = o[0] < cap(LH) ? o[0] : cap(LH), rl = o[1] < cap(LL) ? o[1] : cap(LL);
      if (lds_bytes(NW, rh, rl) <= 160 * 1024) return hi ? rh : rl;
    }
    return 0;
  }
  static constexpr int RH = pick_replicas(true), RL = pick_replicas(false);
  static_assert(RH >= 4 && RL >= 4, "LDS");
  static constexpr int LUTH = Traits<BASE, LH>::LUTDW * RH;  // dwords of the high-pool tables
  static constexpr int LUTL = Traits<BASE, LL>::LUTDW * RL;
};

struct Fin { float m[4], l[4]; float o[4][kD]; };             // one wave's state, merged form
struct TailScratch { float lg[4][kSlots]; float mx[4], sum[4]; float o[4][kD]; };

template <class PL>
struct Shared {
  // decode tables (high pool, low pool) first: their offsets fit the 16-bit
  // immediate offset of an LDS read, so a lookup needs no base add
  alignas(16) uint32_t lut[PL::LUTH + PL::LUTL];
  alignas(16) uint8_t stage[PL::NW][PL::NLD * 1024];         // per wave: one record, later its Fin
  alignas(16) uint8_t pv[PL::NW][PL::PV];                    // per wave int8 weights
  alignas(16) float qf[4][kQPad];                            // fp32 query, rotated for bases 1, 2
  float qorig[4][kD];                                        // query as given (fp16 tail)
  Fin tfin;                                                  // the fp16 tail's state
  TailScratch ts;
  alignas(16) uint4 aq[PL::NG][PL::NCKH + PL::NCKL][64];     // score A operands, per group, pool and lane
  float zpart[4][4];                                         // per head: sums of q over 32-channel runs
  float qmax[4][4];                                          // per head: max |q| over 32-channel runs
  float zc[PL::NW][4][4];                                    // per wave, head, group: sum p * zero
  int last;
};

template <class PL>
__device__ inline Fin* wave_fin(Shared<PL>& sm, int w) { return reinterpret_cast<Fin*>(sm.stage[w]); }

template <int NGV>
struct WaveState {
  float m, l, z[NGV];
  float qw, qwi;     // scale of the int8 weights (a power of 2) and its inverse
  float of[8];       // flushed value sums, channel 16 cb + n of head r
  int4v cv[8];       // integer value sums since the last flush, rows (head, byte)
#ifdef SEMKV_TIMELINE
  int nrec = 0, nflush = 0;   // tracing build: records and flushes of the wave
#endif
};

// the integer q . codes of one head from its three byte rows
__device__ inline float comb3(const int4v& c) {
  return fmaf(float(c[0]), 16384.0f, fmaf(float(c[1]), 128.0f, float(c[2])));
}
// the same for one product of a score: |row 0| < 2^16, |row 1| < 2^17, so
// the integer sum stays below 2^31
// bits [OFF, OFF+7) of x as one instruction (left to itself the compiler
// emits a shift and a mask).  Its operand must not come straight from a
// matrix instruction: the compiler does not insert the wait states a read of
// an MFMA result needs before inline assembly.
template <int OFF>
__device__ inline uint32_t bits7(uint32_t x) {
  uint32_t r;
  __asm__("v_bfe_u32 %0, %1, %2, 7" : "=v"(r) : "v"(x), "i"(OFF));
  return r;
}
__device__ inline float comb3_score(const int4v& c) {
  // two shift-adds; the empty statement keeps the compiler from re-associating
  // them into two shifts and a three-way add
  int t = (c[0] << 7) + c[1];
  __asm__("" : "+v"(t));
  return float((t << 7) + c[2]);
}

// ---------------------------------------------------------- staging ----

// piece j of lane l is bytes [1024 j + 16 l, +16) of a record, read through a
// buffer descriptor bounded by the record's size: pieces past its end read 0
// without touching memory, so every record takes the same NMAX loads

template <int BASE, int LH, int LL, int G, int NMAX>
__device__ inline void load_tile(const PoolGeom& g, const uint8_t* unit, int tile, int nt0, uint4 (&r)[NMAX], int lane) {
  using PL = Plan<BASE, LH, LL, G>;
  const bool hi = tile < nt0;
  const int rb = hi ? PL::GH::RB : PL::GL::RB;
  const uint8_t* rec = hi ? unit + int64_t(tile) * PL::GH::RB : unit + g.lo_offset + int64_t(tile - nt0) * PL::GL::RB;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(rec), 0, rb, kBufferWord3);
#pragma unroll
  for (int j = 0; j < NMAX; ++j) {
    const uint4v v = __builtin_amdgcn_raw_buffer_load_b128(rs, j * 1024 + lane * 16, 0, 0);
    r[j] = make_uint4(v.x, v.y, v.z, v.w);
  }
}

template <int NMAX>
__device__ inline void store_pieces(const uint4 (&r)[NMAX], uint8_t* lds, int lane) {
#pragma unroll
  for (int j = 0; j < NMAX; ++j) *reinterpret_cast<uint4*>(lds + j * 1024 + lane * 16) = r[j];
}

// Per head, of the query x (affine) or the rotated query (bases 1, 2) held by one
// thread per (head, channel) -- whole waves, 64 channels of one head each:
// sums over aligned runs of 32 channels (the zero-point terms) and the
// largest magnitude of each such run (the fixed-point scale).
template <class PL>
__device__ inline void query_runs(float x, int h, int c, Shared<PL>& sm) {
  const float sx = row_sum16(x), ax = row_max16(fabsf(x));
  const float s0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sx), 0));
  const float s1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sx), 16));
  const float s2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sx), 32));
  const float s3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sx), 48));
  const float a0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ax), 0));
  const float a1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ax), 16));
  const float a2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ax), 32));
  const float a3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ax), 48));
  if ((c & 31) == 0) {
    sm.zpart[h][c / 32] = (c & 32) ? s2 + s3 : s0 + s1;
    sm.qmax[h][c / 32] = (c & 32) ? fmaxf(a2, a3) : fmaxf(a0, a1);
  }
}

// sum of head h's query over query group g, and the exponent e of its fixed-
// point form: the largest magnitude a pool's operands hold (the tq plane
// weights included), times 2^e, lies in [2^19, 2^20)
template <int BASE, int G, class PL>
__device__ inline float query_sum(const Shared<PL>& sm, int h, int g) {
  constexpr int GQ = BASE != 1 ? G : kD;
  float z = 0.0f;
#pragma unroll
  for (int k = 0; k < GQ / 32; ++k) z += sm.zpart[h][g * GQ / 32 + k];
  return z;
}
template <int BASE, int L, int G, class PL>
__device__ inline int query_exp(const Shared<PL>& sm, const float* mu, int h, int g) {
  constexpr int GQ = BASE != 1 ? G : kD;
  float mx = 0.0f;
#pragma unroll
  for (int k = 0; k < GQ / 32; ++k) mx = fmaxf(mx, sm.qmax[h][g * GQ / 32 + k]);
  mx *= BASE != 1 || L == 3 ? 1.0f : mu[2] + mu[3];        // tq, 4 levels: mu2 + mu3 > mu3 - mu2 > 0
  const int E = __builtin_amdgcn_frexp_expf(mx);          // mx = f 2^E, f in [0.5, 1)
  return mx >= 1e-30f ? 20 - E : 0;
}

// Score A operands of one pool for all 64 lane contexts, by the workgroup:
// for query group g, lane (row m = 4h + s, kg) chunk c slot e holds byte s of
// qi = rint(x 2^e) at the channel the slot addresses (zero past channel 127,
// in pad slots, outside group g and in rows 4h + 3), x the query of head h
// (affine), its rotated query (rotated affine) or its plane-weighted rotated
// query (tq), |qi| < 2^20.  qi splits
// as 2^14 b0 + 2^7 b1 + b2 (b0 signed, b1, b2 in [0, 127]), so a product sums
// the exact integer qi . codes in three rows.
// Items are dealt to threads from thread OFF on (the low pool's start where
// the high pool's end), so the two pools' items spread over the workgroup.
template <int BASE, int L, int G, int POOL, int OFF, class PL>
__device__ void build_aq(const DecodeArgs& a, Shared<PL>& sm) {
  using Tr = Traits<BASE, L>;
  using Ge = Geo<BASE, L, G>;
  const float* mu = a.mu[POOL];
  const float wP[2] = {BASE != 1 ? 1.0f : (L == 3 ? 1.0f : mu[3] - mu[2]),
                       BASE != 1 ? 1.0f : (L == 3 ? 1.0f : mu[2] + mu[3])};
  for (int item = (int(threadIdx.x) + PL::NT - OFF % PL::NT) % PL::NT; item < Ge::NG * Tr::NCK * 64; item += PL::NT) {
    const int g = item / (Tr::NCK * 64), c = (item >> 6) % Tr::NCK, ln = item & 63;
    const int m = ln & 15, kg = ln >> 4, h = m >> 2, sp = m & 3;
    const int e = query_exp<BASE, L, G>(sm, mu, h, g);
    // branch free: every slot reads at a clamped channel (all reads in
    // flight together) and keeps the byte only where the slot is real
    const int shift = sp == 0 ? 14 : sp == 1 ? 7 : 0;
    const int bmask = sp == 0 ? 0xFF : 0x7F;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int sl = 0; sl < 16; ++sl) {
      const int k = Tr::SPC * c + sl / Tr::STRIDE, ws = sl % Tr::STRIDE;
      const int dig = slot_digit<BASE, L>(ws), pl = slot_plane<BASE, L>(ws);
      const int ch = kg * Tr::n + Tr::n * 4 * k + (dig < 0 ? 0 : dig);      // >= 128: a pad slot
      const bool ok = dig >= 0 && sp < 3 && ch < kD && (BASE == 1 || ch / G == g);
      const int qi = int(rintf(ldexpf(wP[pl] * sm.qf[h][ch < kD ? ch : 0], e)));
      w[sl >> 2] |= (ok ? uint32_t((qi >> shift) & bmask) : 0u) << (8 * (sl & 3));
    }
    sm.aq[g][(POOL ? PL::NCKH : 0) + c][ln] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// ---------------------------------------------------- one pool's records ----

template <int BASE, int LH, int LL, int G, int POOL, class PL>
__device__ void run_pool(const DecodeArgs& a, Shared<PL>& sm, WaveState<PL::NGV>& st, const uint8_t* unit,
                         int nt0, int first, int stride, int i0, int i1, int count, uint4 (&R)[PL::NLD]) {
  constexpr int L = POOL ? LL : LH;
  using Tr = Traits<BASE, L>;
  using Ge = Geo<BASE, L, G>;
  constexpr int NG = Ge::NG, NGV = Ge::NGV;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int n = lane & 15, r = lane >> 4, kg = r;
  uint8_t* rec = sm.stage[wave];
  // tq: mu = -m, 0, m (L = 3) or -b, -a, a, b (L = 4)
  const float* mu = a.mu[POOL];
  const float cS = BASE != 1 ? 1.0f : (L == 3 ? mu[2] / 128.0f : 1.0f / 128.0f);
  const float cZ = BASE != 1 ? 0.0f : (L == 3 ? -mu[2] / 128.0f : -mu[3] / 128.0f);
  const float wP[2] = {BASE != 1 ? 1.0f : (L == 3 ? 1.0f : mu[3] - mu[2]),
                       BASE != 1 ? 1.0f : (L == 3 ? 1.0f : mu[2] + mu[3])};
  // rotated affine: k = sign . H y / 8 with y = s c + z the affine value of
  // the rotated coordinates, so q . k = (H sign . q) . y / 8, and the values
  // are summed as y / 8 in the rotated domain (powers of 2: exact)
  constexpr float kR = BASE == 2 ? 0.125f : 1.0f;
  constexpr float kScore = kLog2e * kRsqrtD * kR;

  // ---- score A operands (built once per workgroup): in registers for one
  // query group, else read per product
  int4v Aq[NG == 1 ? Tr::NCK : 1];
  if constexpr (NG == 1) {
#pragma unroll
    for (int c = 0; c < Tr::NCK; ++c) {
      const uint4 v = sm.aq[0][(POOL ? PL::NCKH : 0) + c][lane];
      Aq[c] = __builtin_bit_cast(int4v, uint4v{v.x, v.y, v.z, v.w});
    }
  }
  // tables: the lane's replica; entries 2^S bytes apart
  constexpr int NR = POOL ? PL::RL : PL::RH;
  constexpr int S = ilog2(NR * Tr::TED * 4);
  static_assert((1 << S) == NR * Tr::TED * 4, "entry stride");
  constexpr uint32_t KFULL = full_symbols<L, kD, kSlots>(), VFULL = full_symbols<L, kSlots, kD>();
  const uint32_t lb = uint32_t((lane & (NR - 1)) * Tr::TED * 4);
  const LutRef lut{reinterpret_cast<const uint8_t*>(sm.lut + (POOL ? PL::LUTH : 0)), lb, lb + (uint32_t(Tr::DIV) << S)};
  uint32_t kmask[Tr::NSK], vmask[Tr::NSV];
  segment_masks<L, kD, kSlots>(kg, kmask);
  segment_masks<L, kSlots, kD>(kg, vmask);
#pragma unroll
  for (int k = 0; k < Tr::NSK; ++k) kmask[k] <<= S;
#pragma unroll
  for (int k = 0; k < Tr::NSV; ++k) vmask[k] <<= S;
  const int koff0 = seg_off<L, kD, kSlots>(kg, n), kstep = 16 * seg_line_bits<L, kD, kSlots>(kg);
  const int voff0 = seg_off<L, kSlots, kD>(kg, n), vstep = 16 * seg_line_bits<L, kSlots, kD>(kg);
  // softmax lanes: token n of each 16-token block, head r.  Per query group
  // of head r, times the softmax scale: the sum of q (zero-point term) and
  // 2^-e (the fixed-point query's scale); tq folds its level offsets in
  float zwsK[NG], qscK[NG];
#pragma unroll
  for (int i = 0; i < NG; ++i) {
    zwsK[i] = query_sum<BASE, G>(sm, r, i) * (kScore * (BASE != 1 ? 1.0f : cZ));
    qscK[i] = ldexpf(kScore * (BASE != 1 ? 1.0f : cS), -query_exp<BASE, L, G>(sm, mu, r, i));
  }
  // softmax lanes: where token 16 blk + n of each block lands in the weight
  // operands (value group 0, plane 0, row 4r)
  uint8_t* pvw = sm.pv[wave];
  int pvwr[4];
#pragma unroll
  for (int blk = 0; blk < 4; ++blk) {
    const int t = 16 * blk + n, p = t / Tr::n, d = t - p * Tr::n, k = p >> 2;
    pvwr[blk] = (k / Tr::SPC) * Ge::CHB + (p & 3) * Ge::KGS + 64 * r + (k % Tr::SPC) * Tr::STRIDE + digit_slot<BASE, L>(d);
  }
  static_assert(Ge::PV % 16 == 0, "weight array pieces");
  for (int i = lane; i < Ge::PV / 16; i += 64) reinterpret_cast<uint4*>(pvw)[i] = make_uint4(0u, 0u, 0u, 0u);
  const int64_t nrows = a.n_rows[POOL];

  for (int it = i0; it < i1; ++it) {
    const int tile = first + stride * it;
    const bool more = it + 1 < count;
    if (more) load_tile<BASE, LH, LL, G>(a.g, unit, tile + stride, nt0, R, lane);
    if (it == 0) SEMKV_STAMP_FINE(16);
    const int ptile = POOL ? tile - nt0 : tile;
    const uint8_t* kmeta = rec + 2 * Tr::TB;
    const uint8_t* vmeta = kmeta + Ge::MB;
    const int nvalid = nrows - int64_t(ptile) * kSlots < kSlots ? int(nrows - int64_t(ptile) * kSlots) : kSlots;

    // ---- scores: C[(h, byte)][token] = q_h bytes . codes; lane holds token n, head r
    float lg[4];
    // all four K segments and the lane's metadata words in one round trip
    uint32_t kseg[4][Tr::KSEGW];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) lds_segment<Tr::KSEGW>(rec, koff0 + blk * kstep, kseg[blk]);
    constexpr int NKM = BASE != 1 ? NG : 1, NVM = BASE != 1 ? NGV : 1;
    uint32_t km[4][NKM], vm[4][NVM];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      const int t = 16 * blk + n;
#pragma unroll
      for (int i = 0; i < NKM; ++i)
        km[blk][i] = BASE != 1 ? *reinterpret_cast<const uint32_t*>(kmeta + (i * kSlots + t) * 4)
                               : uint32_t(*reinterpret_cast<const uint16_t*>(kmeta + t * 2));
#pragma unroll
      for (int i = 0; i < NVM; ++i)
        vm[blk][i] = BASE != 1 ? *reinterpret_cast<const uint32_t*>(vmeta + (i * kSlots + t) * 4)
                               : uint32_t(*reinterpret_cast<const uint16_t*>(vmeta + t * 2));
    }
    // the score of token 16 blk + n from its products, one per query group,
    // in the softmax's base-2 scale: (q . c) 2^-e s + z (sum q) per group
    // (tq: rho ((q . c) 2^-e cS + cZ sum q)); masked tokens are set apart
    auto score = [&](int blk, const int4v (&acc)[NG]) {
      float x;
      if constexpr (BASE != 1) {
        x = hf(km[blk][0] >> 16) * zwsK[0];
#pragma unroll
        for (int i = 1; i < NG; ++i) x = fmaf(hf(km[blk][i] >> 16), zwsK[i], x);
#pragma unroll
        for (int i = 0; i < NG; ++i) x = fmaf(comb3_score(acc[i]) * qscK[i], hf(km[blk][i] & 0xFFFFu), x);
      } else {
        x = fmaf(comb3_score(acc[0]), qscK[0], zwsK[0]) * hf(uint16_t(km[blk][0]));
      }
      return x;
    };
    // software pipeline: the next block's table reads are in flight during
    // the current block's products
    int4v Bk[2][Tr::NCK];
    chunk_operands<BASE, L, S, KFULL, Tr::KSEGW, Tr::NSK, Tr::NCK>(kseg[0], kmask, lut, Bk[0]);
    constexpr bool DEFER = NG == 1;          // score arithmetic after the value segment reads
    int4v acck[DEFER ? 4 : 1][NG];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      if (blk + 1 < 4) chunk_operands<BASE, L, S, KFULL, Tr::KSEGW, Tr::NSK, Tr::NCK>(kseg[blk + 1], kmask, lut, Bk[(blk + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
      int4v acc[NG];
#pragma unroll
      for (int i = 0; i < NG; ++i) {
        acc[i] = int4v{0, 0, 0, 0};
#pragma unroll
        for (int ch = 0; ch < Tr::NCK; ++ch) {
          int4v A;
          if constexpr (NG == 1) {
            A = Aq[ch];
          } else {
            const uint4 v = sm.aq[i][(POOL ? PL::NCKH : 0) + ch][lane];
            A = __builtin_bit_cast(int4v, uint4v{v.x, v.y, v.z, v.w});
          }
          acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, Bk[blk & 1][ch], acc[i], 0, 0, 0);
        }
      }
      if constexpr (DEFER) {
#pragma unroll
        for (int i = 0; i < NG; ++i) acck[blk][i] = acc[i];
      } else {
        lg[blk] = score(blk, acc);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // the value segments and the first value operands do not depend on the
    // softmax: their LDS round trips overlap it
    const uint8_t* vbody = rec + Tr::TB;
    uint32_t vseg[8][Tr::VSEGW];
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) lds_segment<Tr::VSEGW>(vbody, voff0 + cb * vstep, vseg[cb]);
    int4v Bv[2][Tr::NCV];
    chunk_operands<BASE, L, S, VFULL, Tr::VSEGW, Tr::NSV, Tr::NCV>(vseg[0], vmask, lut, Bv[0]);
    if constexpr (DEFER) {
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) lg[blk] = score(blk, acck[blk]);
    }
    if (nvalid < kSlots) {                   // the pool's last record: slots past its rows
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) lg[blk] = 16 * blk + n < nvalid ? lg[blk] : -INFINITY;
    }
    if (it == 0) SEMKV_STAMP_FINE(17);
    // ---- online softmax (base 2) for head r over this record's 64 tokens,
    // rescaled lazily: the reference maximum st.m moves only when a score
    // passes it by more than 8 (weights up to 2^8 fit the fixed-point range),
    // or on the wave's first record
    const float mt = row_max16(max4(lg[0], lg[1], lg[2], lg[3]));
    const bool grow = !(mt <= st.m + 8.0f);
    const float m_new = grow ? mt : st.m;
    const float alpha = grow ? __builtin_amdgcn_exp2f(st.m - m_new) : 1.0f;
    st.m = m_new;
    float lsum = 0.0f, wmax = 0.0f;
    float wv[4][NGV][Ge::NPL];               // value weights of the lane's tokens
    float zadd[NGV];
#pragma unroll
    for (int i = 0; i < NGV; ++i) zadd[i] = 0.0f;
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      const float p = __builtin_amdgcn_exp2f(lg[blk] - m_new);   // 0 for masked tokens
      lsum += p;
      if constexpr (BASE != 1) {
        const float pr = p * kR;
#pragma unroll
        for (int i = 0; i < NGV; ++i) {
          const uint32_t m = vm[blk][i];
          wv[blk][i][0] = pr * hf(m & 0xFFFFu);
          wmax = fmaxf(wmax, wv[blk][i][0]);
          zadd[i] = fmaf(pr, hf(m >> 16), zadd[i]);
        }
      } else {
        const float rho = hf(uint16_t(vm[blk][0]));
#pragma unroll
        for (int pl = 0; pl < Ge::NPL; ++pl) {
          wv[blk][0][pl] = p * rho * cS * wP[pl];
          wmax = fmaxf(wmax, wv[blk][0][pl]);
        }
        zadd[0] = fmaf(p * rho, cZ, zadd[0]);
      }
    }
    // ---- the integer value sums hold weights of one scale and one reference
    // maximum: fold them into the float sums when the maximum moves or this
    // record's weights would not fit 21 bits (their rounding stays below
    // 2^21 - 1, so the top byte stays below 128), and re-pick the scale
    const bool flush = grow || wmax * st.qw >= 2097151.0f;
#ifdef SEMKV_TIMELINE
    st.nrec += 1;
#endif
    if (__builtin_amdgcn_ballot_w64(flush) != 0) {
#ifdef SEMKV_TIMELINE
      st.nflush += 1;
#endif
      wmax = row_max16(wmax);
      st.l *= alpha;
#pragma unroll
      for (int i = 0; i < NGV; ++i) st.z[i] *= alpha;
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
        st.of[cb] = (st.of[cb] + comb3(st.cv[cb]) * st.qwi) * alpha;
        st.cv[cb] = int4v{0, 0, 0, 0};
      }
      const int E = __builtin_amdgcn_frexp_expf(wmax);          // wmax = f 2^E, f in [0.5, 1)
      const int e = wmax >= 1e-30f ? 19 - E : 100;
      st.qw = ldexpf(1.0f, e);
      st.qwi = ldexpf(1.0f, -e);
    }
    st.l += lsum;
#pragma unroll
    for (int i = 0; i < NGV; ++i) st.z[i] += zadd[i];
    if (it == 0) SEMKV_STAMP_FINE(18);

    // ---- values: C[(h, byte)][channel] += weights (tokens) x V codes, one
    // value group's int8 weights (byte s of rint(w qw) in row 4r + s) at a time
    int4v Aw[Tr::NCV];
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) {
      constexpr int CPG = BASE != 1 ? G / 16 : 8;          // channel blocks per value group
      if (cb % CPG == 0) {
        const int gv = cb / CPG;
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
#pragma unroll
          for (int pl = 0; pl < Ge::NPL; ++pl) {
            // the integer nearest w qw (< 2^21 - 1) in the low mantissa bits
            // of w qw + 1.5 2^23 (one rounding of the exact sum)
            const uint32_t q = __float_as_uint(fmaf(wv[blk][gv][pl], st.qw, 12582912.0f));
            uint8_t* w = pvw + pvwr[blk] + pl;
            w[0] = uint8_t(bits7<14>(q));
            w[16] = uint8_t(bits7<7>(q));
            w[32] = uint8_t(bits7<0>(q));
          }
        // weights written above by other lanes of this wave are read below
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int c = 0; c < Tr::NCV; ++c) {
          const uint4 v = *reinterpret_cast<const uint4*>(pvw + c * Ge::CHB + kg * Ge::KGS + n * 16);
          Aw[c] = __builtin_bit_cast(int4v, uint4v{v.x, v.y, v.z, v.w});
        }
      }
      if (cb + 1 < 8) chunk_operands<BASE, L, S, VFULL, Tr::VSEGW, Tr::NSV, Tr::NCV>(vseg[cb + 1], vmask, lut, Bv[(cb + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < Tr::NCV; ++c) st.cv[cb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(Aw[c], Bv[cb & 1][c], st.cv[cb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // the next record replaces this one in the wave's buffer (LDS serves a
    // wave's accesses in order: the reads above come first)
#ifdef SEMKV_TIMELINE
    if (it == 0) SEMKV_STAMP(8);
#endif
    if (more) store_pieces(R, rec, lane);
    SEMKV_STAMP(3 + (it < 4 ? it : 4));
  }
}

// A wave's state in merged form: sums over the tokens of a row, the integer
// value sums folded in, the zero-point term added.  Lane (n, r) holds head r
// at channels 16 cb + n.
template <int BASE, int G, class PL>
__device__ void wave_finish(Shared<PL>& sm, WaveState<PL::NGV>& st) {
  constexpr int NGV = PL::NGV;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int n = lane & 15, r = lane >> 4;
  st.l = row_sum16(st.l);
#pragma unroll
  for (int i = 0; i < NGV; ++i) st.z[i] = row_sum16(st.z[i]);
  if (n == 0) {
#pragma unroll
    for (int i = 0; i < NGV; ++i) sm.zc[wave][r][i] = st.z[i];
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
  Fin* f = wave_fin(sm, wave);
  if (n == 0) {
    f->m[r] = st.m;
    f->l[r] = st.l;
  }
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
    const int ch = 16 * cb + n;
    f->o[r][ch] = st.of[cb] + comb3(st.cv[cb]) * st.qwi + sm.zc[wave][r][BASE != 1 ? ch / G : 0];
  }
}

// Partials cross workgroups (and XCDs, whose L2 caches are not coherent with
// each other): they are written with agent-scope atomic stores and read with
// the same coherent cache policy (sc1), so neither side needs a cache
// write-back or invalidate.
__device__ inline void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


// The unnormalized Walsh-Hadamard transform H x of the 4 rows of 128 values
// held one per thread by threads 0..511 (thread t: row t >> 7, entry t & 127).
// Stages 1..32 pair lanes of one wave (DPP quad permutes for 1 and 2, lane
// exchanges for the rest); stage 64 pairs the two waves of a row through the
// LDS buffer xch.  Each stage computes the lower entry as lower + upper and the
// upper as lower - upper, the radix-2 butterflies in the usual order.  Every
// thread of the workgroup calls it; xch is free again when it returns.
__device__ inline float fwht_rows(float x, float (*xch)[kD]) {
  const int tid = threadIdx.x, lane = tid & 63;
  float p = dpp<0xB1>(x);                                  // lane ^ 1
  x = (lane & 1) ? p - x : x + p;
  p = dpp<0x4E>(x);                                        // lane ^ 2
  x = (lane & 2) ? p - x : x + p;
#pragma unroll
  for (int hs = 4; hs < 64; hs <<= 1) {
    p = __shfl_xor(x, hs);
    x = (lane & hs) ? p - x : x + p;
  }
  const bool mine = tid < 4 * kD;
  if (mine) xch[tid >> 7][tid & 127] = x;
  __syncthreads();
  if (mine) {
    p = xch[tid >> 7][(tid & 127) ^ 64];
    x = (tid & 64) ? p - x : x + p;
  }
  __syncthreads();
  return x;
}

// fp16 tail of generated tokens (1 to 64 rows): its attention state goes to
// sm.tfin.  Runs after the workgroup's records, when the decode tables and the
// weight arrays are free: the K tail is staged in the table area and the V
// tail in the weight area (both in one round trip), then every thread works:
// 8 threads per row for the scores, one wave per head for the softmax, one
// thread per (head, channel) for the values.
template <int BASE, class PL>
__device__ void tail_split(const DecodeArgs& a, Shared<PL>& sm, int b, int layer, int kvh) {
  static_assert(sizeof(sm.lut) >= kSlots * kD * 2 && sizeof(sm.pv) >= kSlots * kD * 2, "tail staging");
  static_assert(PL::NT == 4 * kD, "one thread per (head, channel)");
  const PoolGeom& g = a.g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nt = a.n_tail;
  TailScratch& ts = sm.ts;
  const uint16_t* kt = a.tail + ((((int64_t(b) * g.n_layers + layer) * g.n_kv_heads + kvh) * 2) * kSlots) * kD;
  const uint16_t* vt = kt + kSlots * kD;
  uint4* kl = reinterpret_cast<uint4*>(sm.lut);             // [64 rows][16 pieces of 8 fp16]
  uint4* vl = reinterpret_cast<uint4*>(&sm.pv[0][0]);
  {
    // piece i (8 channels of row i / 16); the two pieces of a thread: i0, i1
    const int i0 = tid, i1 = tid + PL::NT;
    const bool in0 = (i0 >> 4) < nt, in1 = (i1 >> 4) < nt;
    uint4 ka = make_uint4(0u, 0u, 0u, 0u), kb = ka, va = ka, vb2 = ka;
    if (in0) {
      ka = reinterpret_cast<const uint4*>(kt)[i0];
      va = reinterpret_cast<const uint4*>(vt)[i0];
    }
    if (in1) {
      kb = reinterpret_cast<const uint4*>(kt)[i1];
      vb2 = reinterpret_cast<const uint4*>(vt)[i1];
    }
    if (in0) {
      kl[i0] = ka;
      vl[i0] = va;
    }
    if (in1) {
      kl[i1] = kb;
      vl[i1] = vb2;
    }
  }
  __syncthreads();
  // scores: thread (row t, channel block j of 16) sums its block for the 4
  // heads; the 8 threads of a row are 8 neighbouring lanes (scalars only:
  // small arrays here would be placed in memory)
  {
    const int t = tid >> 3, j = tid & 7;
    uint4 k0 = make_uint4(0u, 0u, 0u, 0u), k1 = k0;
    if (t < nt) {
      k0 = kl[t * 16 + 2 * j];
      k1 = kl[t * 16 + 2 * j + 1];
    }
    auto dot4 = [](const float* q, uint32_t w0, uint32_t w1, float x) {
      const float4 qv = *reinterpret_cast<const float4*>(q);
      x = fmaf(qv.x, hf(uint16_t(w0 & 0xFFFFu)), x);
      x = fmaf(qv.y, hf(uint16_t(w0 >> 16)), x);
      x = fmaf(qv.z, hf(uint16_t(w1 & 0xFFFFu)), x);
      return fmaf(qv.w, hf(uint16_t(w1 >> 16)), x);
    };
    auto dot16 = [&](int h) {
      const float* q = &sm.qorig[h][16 * j];
      float x = dot4(q, k0.x, k0.y, 0.0f);
      x = dot4(q + 4, k0.z, k0.w, x);
      x = dot4(q + 8, k1.x, k1.y, x);
      return dot4(q + 12, k1.z, k1.w, x);
    };
    float d0 = dot16(0), d1 = dot16(1), d2 = dot16(2), d3 = dot16(3);
#pragma unroll
    for (int m = 1; m < 8; m <<= 1) {
      d0 += __shfl_xor(d0, m);
      d1 += __shfl_xor(d1, m);
      d2 += __shfl_xor(d2, m);
      d3 += __shfl_xor(d3, m);
    }
    if (t < nt && j == 0) {
      constexpr float sc = kLog2e * kRsqrtD;
      ts.lg[0][t] = d0 * sc;
      ts.lg[1][t] = d1 * sc;
      ts.lg[2][t] = d2 * sc;
      ts.lg[3][t] = d3 * sc;
    }
  }
  __syncthreads();
  // softmax: wave h takes head h, lane t token t
  if (wave < 4) {
    const float x = lane < nt ? ts.lg[wave][lane] : -INFINITY;
    float M = x;
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) M = fmaxf(M, __shfl_xor(M, m));
    const float p = lane < nt ? __builtin_amdgcn_exp2f(x - M) : 0.0f;
    float ssum = p;
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) ssum += __shfl_xor(ssum, m);
    if (lane < nt) ts.lg[wave][lane] = p;
    if (lane == 0) {
      ts.mx[wave] = M;
      ts.sum[wave] = ssum;
    }
  }
  __syncthreads();
  const int h = tid >> 7, c = tid & 127;
  const uint16_t* vrow = reinterpret_cast<const uint16_t*>(vl);
  float o = 0.0f;
  for (int t = 0; t < nt; ++t) o = fmaf(ts.lg[h][t], hf(vrow[t * kD + c]), o);
  if (BASE != 0) {                           // into the rotated domain: H (sign . o) / 128
    const uint32_t* sw = g.signs + (int64_t(layer) * g.n_kv_heads + kvh) * 4;
    o = ((sw[c >> 5] >> (c & 31)) & 1u) ? -o : o;
    o = fwht_rows(o, ts.o) * (1.0f / 128.0f);
  }
  sm.tfin.o[h][c] = o;
  if (c == 0) {
    sm.tfin.m[h] = ts.mx[h];
    sm.tfin.l[h] = ts.sum[h];
  }
}

// Merge of the partials of one (layer, sequence, kv head), run by the last
// workgroup to finish: log-sum-exp over the partials, then for the rotated
// bases the inverse rotation o = sign . H o_rot.  vb indexes the launch's
// (layer, sequence) pairs: partials, counters, queries and outputs.
template <int BASE, class PL>
__device__ void merge_splits(const DecodeArgs& a, Shared<PL>& sm, int vb, int layer, int kvh) {
  const int tid = threadIdx.x;
  const int ns = a.nsplit;
  const float* unit = a.ws + (int64_t(vb) * a.g.n_kv_heads + kvh) * ns * 4 * kPartial;
  // thread (head h, quarter q, channel quad cq) takes the splits s = q, q+4,
  // ... with 16-byte loads at the coherent level (cache policy sc1, as the
  // agent-scope loads), then the four quarters merge in LDS
  const bool mine = tid < 4 * kD;
  const int h = (tid >> 7) & 3, q = (tid >> 5) & 3, cq = tid & 31;
  // the sign of this thread's output channel (rotated bases), loaded first
  const uint32_t sbits = BASE != 0 && mine ? a.g.signs[(int64_t(layer) * a.g.n_kv_heads + kvh) * 4 + ((tid & 127) >> 5)] : 0u;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(unit), 0, ns * 4 * kPartial * 4, kBufferWord3);
  constexpr int kCoherent = 16;              // sc1
  constexpr int kBatch = 8;
  float M = -INFINITY, Lsum = 0.0f;
  float4v o = float4v{0, 0, 0, 0};
  for (int s0 = q; mine && s0 < ns; s0 += 4 * kBatch) {
    float mv[kBatch], lv[kBatch];
    float4v x[kBatch];
    // all loads issued at once, unconditionally (one round trip): a split
    // past the last reads zeros through the buffer descriptor and is given
    // m = -inf afterwards
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const int sp = s0 + 4 * k;
      const int off = (sp * 4 + h) * kPartial * 4;
      const auto ml = __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, kCoherent);
      mv[k] = __uint_as_float(ml[0]);
      lv[k] = __uint_as_float(ml[1]);
      x[k] = __builtin_bit_cast(float4v, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 + 16 * cq, 0, kCoherent));
    }
#pragma unroll
    for (int k = 0; k < kBatch; ++k) mv[k] = s0 + 4 * k < ns ? mv[k] : -INFINITY;
    float Mn = M;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) Mn = fmaxf(Mn, mv[k]);
    const float keep = M == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(M - Mn);
    Lsum *= keep;
    o *= keep;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float sc = mv[k] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(mv[k] - Mn);
      Lsum += lv[k] * sc;
      o += x[k] * sc;
    }
    M = Mn;
  }
  struct Quarters { float m[4][4], l[4][4]; float4v o[4][4][32]; };
  static_assert(sizeof(Quarters) <= sizeof(sm.stage), "merge scratch");
  Quarters& qs = *reinterpret_cast<Quarters*>(&sm.stage[0][0]);
  if (mine) {
    if (cq == 0) {
      qs.m[h][q] = M;
      qs.l[h][q] = Lsum;
    }
    qs.o[h][q][cq] = o;
  }
  __syncthreads();
  const int hc = tid >> 7, c = tid & 127;
  float r = 0.0f;
  if (mine) {
    float Mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < 4; ++k) Mx = fmaxf(Mx, qs.m[hc][k]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float sc = qs.m[hc][k] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(qs.m[hc][k] - Mx);
      L += qs.l[hc][k] * sc;
      O += qs.o[hc][k][c >> 2][c & 3] * sc;
    }
    r = O / L;
  }
  if (BASE != 0) {
    r = fwht_rows(r, sm.ts.o);
    r = ((sbits >> (c & 31)) & 1u) ? -r : r;
  }
  if (mine) a.out[((int64_t(vb) * a.g.n_kv_heads + kvh) * 4 + hc) * kD + c] = r;
}

template <int BASE, int LH, int LL, int G>
__global__ __launch_bounds__((Plan<BASE, LH, LL, G>::NT)) void decode_kernel(DecodeArgs a) {
  using PL = Plan<BASE, LH, LL, G>;
  constexpr int NW = PL::NW, NT = PL::NT;
  __shared__ Shared<PL> sm;
  static_assert(sizeof(Shared<PL>) <= 160 * 1024, "LDS");
  static_assert(NT >= 4 * kD, "one thread per (head, channel) of the query and the output");
  // blockIdx.z = (layer of the launch) x batch + sequence: an all-layers
  // launch covers n_layers_launched layers from a.layer
  const int split = blockIdx.x, kvh = blockIdx.y, vb = blockIdx.z;
  const int li = vb / a.g.batch, b = vb - li * a.g.batch, layer = a.layer + li;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const PoolGeom& g = a.g;
  SEMKV_STAMP(0);

  // ---- the query first (the longest wait of the prologue); its work takes
  // the first 4 x 128 threads, one per (head, channel) -- with 8 waves every
  // thread, known at compile time, so no branch forces a wait on the load
  const bool qt = NT == 4 * kD || tid < 4 * kD;
  const int h = qt ? tid >> 7 : 0, c = tid & 127;
  const uint16_t qbits = qt ? a.q[((int64_t(vb) * g.n_kv_heads * 4) + kvh * 4 + h) * kD + c] : uint16_t(0);
  // rotated bases: the sign word of this thread's channel, in flight with the query
  const uint32_t qsign = BASE != 0 && qt ? g.signs[(int64_t(layer) * g.n_kv_heads + kvh) * 4 + (c >> 5)] : 0u;

  // ---- fused append (Alg. 2): the workgroup that attends over the fp16 tail
  // first stores this layer's new K/V row in it, as its last row (read back
  // by the same workgroup after the barriers below); placed before the record
  // loads, so that its wait covers the query load only
  if (a.k_new != nullptr && split == a.nsplit - 1 && tid < 2 * kD / 2) {
    const int kv = tid >> 6, w = tid & 63;                // 64 dwords each of K and V
    const uint32_t* src = reinterpret_cast<const uint32_t*>((kv ? a.v_new : a.k_new) + (int64_t(b) * g.n_kv_heads + kvh) * kD);
    uint32_t* dst = reinterpret_cast<uint32_t*>(
        a.tail + ((((int64_t(b) * g.n_layers + layer) * g.n_kv_heads + kvh) * 2 + kv) * kSlots + (a.n_tail - 1)) * kD);
    dst[w] = src[w];
  }

  // ---- this wave's tiles: first, first + stride, ... (high pool first),
  // and the first of them in flight (a wave without records loads tile 0,
  // unused)
  const int nt0 = int((a.n_rows[0] + kSlots - 1) / kSlots), nt1 = int((a.n_rows[1] + kSlots - 1) / kSlots);
  const int nt = nt0 + nt1, stride = a.nsplit * NW;
  const int first = wave * a.nsplit + split;
  const int count = first < nt ? (nt - first + stride - 1) / stride : 0;
  const int nhi = first < nt0 ? (nt0 - first + stride - 1) / stride : 0;
  const uint8_t* unit = g.pools + unit_offset(g, b, layer, kvh);
  uint4 R[PL::NLD];
  load_tile<BASE, LH, LL, G>(g, unit, count > 0 ? first : 0, nt0, R, lane);

  // ---- decode tables (the query and the first record are in flight)
  constexpr int NTH = (PL::LUTH / 4 + NT - 1) / NT, NTL = (PL::LUTL / 4 + NT - 1) / NT;
  uint4 th[NTH], tl[NTL];
#pragma unroll
  for (int k = 0; k < NTH; ++k) th[k] = lut_piece<BASE, LH, PL::RH>(tid + k * NT < PL::LUTH / 4 ? tid + k * NT : 0);
#pragma unroll
  for (int k = 0; k < NTL; ++k) tl[k] = lut_piece<BASE, LL, PL::RL>(tid + k * NT < PL::LUTL / 4 ? tid + k * NT : 0);
  {
    uint4* d = reinterpret_cast<uint4*>(sm.lut);
#pragma unroll
    for (int k = 0; k < NTH; ++k)
      if (tid + k * NT < PL::LUTH / 4) d[tid + k * NT] = th[k];
#pragma unroll
    for (int k = 0; k < NTL; ++k)
      if (tid + k * NT < PL::LUTL / 4) d[PL::LUTH / 4 + tid + k * NT] = tl[k];
  }
  SEMKV_STAMP_FINE(19);
  float xq = 0.0f;
  if (qt) {
    xq = hf(qbits);
    sm.qorig[h][c] = xq;
    if (BASE != 0) xq = ((qsign >> (c & 31)) & 1u) ? -xq : xq;
  }
  SEMKV_STAMP_FINE(20);
  if (BASE != 0) xq = fwht_rows(xq, sm.ts.o);    // rotate: H (sign . q)
  if (qt) {
    sm.qf[h][c] = xq;
    if (c < kQPad - kD) sm.qf[h][kD + c] = 0.0f;
    query_runs(xq, h, c, sm);                   // the query the scores use: its runs
  }
  SEMKV_STAMP_FINE(21);
  __syncthreads();
  build_aq<BASE, LH, G, 0, 0>(a, sm);
  build_aq<BASE, LL, G, 1, PL::GH::NG * PL::NCKH * 64>(a, sm);
  __syncthreads();
  SEMKV_STAMP(1);

  // ---- this wave's records
  WaveState<PL::NGV> st;
  st.m = -INFINITY;
  st.l = 0.0f;
#pragma unroll
  for (int i = 0; i < PL::NGV; ++i) st.z[i] = 0.0f;
  st.qw = st.qwi = 1.0f;
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
    st.of[cb] = 0.0f;
    st.cv[cb] = int4v{0, 0, 0, 0};
  }
  if (count > 0) store_pieces(R, sm.stage[wave], lane);
  SEMKV_STAMP(2);
  if (nhi > 0) run_pool<BASE, LH, LL, G, 0>(a, sm, st, unit, nt0, first, stride, 0, nhi, count, R);
  if (count > nhi) run_pool<BASE, LH, LL, G, 1>(a, sm, st, unit, nt0, first, stride, nhi, count, count, R);
  SEMKV_STAMP(9);
#ifdef SEMKV_TIMELINE
  timeline_put(14, uint32_t(st.nflush));
  timeline_put(15, uint32_t(st.nrec));
#endif
  wave_finish<BASE, G>(sm, st);
  __syncthreads();
  const bool tail = split == a.nsplit - 1 && a.n_tail > 0;
  if (tail) {
    tail_split<BASE>(a, sm, b, layer, kvh);
    __syncthreads();
  }

  // ---- workgroup partial: merge of the waves' (and the tail's) states
  SEMKV_STAMP(10);
  if (qt) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, wave_fin(sm, w)->m[h]);
    if (tail) M = fmaxf(M, sm.tfin.m[h]);
    float Lsum = 0.0f, o = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const Fin* f = wave_fin(sm, w);
      const float sc = f->m[h] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(f->m[h] - M);
      Lsum += f->l[h] * sc;
      o += f->o[h][c] * sc;
    }
    if (tail) {
      const float sc = sm.tfin.m[h] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(sm.tfin.m[h] - M);
      Lsum += sm.tfin.l[h] * sc;
      o += sm.tfin.o[h][c] * sc;
    }
    float* dst = a.ws + ((int64_t(vb) * g.n_kv_heads + kvh) * a.nsplit + split) * 4 * kPartial + h * kPartial;
    if (c == 0) {
      st_agent(dst, M);
      st_agent(dst + 1, Lsum);
    }
    st_agent(dst + 4 + c, o);
  }
  // every thread's partial stores are complete (at the coherent level) before
  // the workgroup's counter increment; the last workgroup reads them after it
  __asm__ volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  SEMKV_STAMP(11);
  if (tid == 0) {
    uint32_t* ctr = a.counters + (vb * g.n_kv_heads + kvh) * kCounterStride;
    const uint32_t old = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sm.last = old == uint32_t(a.nsplit - 1);
    if (sm.last) __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  SEMKV_STAMP(12);
  if (!sm.last) return;
  merge_splits<BASE>(a, sm, vb, layer, kvh);
#ifdef SEMKV_TIMELINE
  __syncthreads();
  SEMKV_STAMP(13);
#endif
}

template <int BASE, int LH, int LL, int G>
int waves_of() { return Plan<BASE, LH, LL, G>::NW; }

// the kernel needs 4 x 128 threads (one per query head and channel): level
// pairs whose 8-wave workgroup does not fit the LDS are not built
template <int BASE, int LH, int LL, int G>
constexpr bool fits() { return Plan<BASE, LH, LL, G>::NT >= 4 * kD; }

template <int BASE, int LH, int LL, int G>
int occupancy() {
  if constexpr (!fits<BASE, LH, LL, G>()) {
    return 0;
  } else {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_kernel<BASE, LH, LL, G>, Plan<BASE, LH, LL, G>::NT, 0) != hipSuccess)
      return 1;
    return n > 0 ? n : 1;
  }
}

template <int BASE, int LH, int LL, int G>
int launch_g(const DecodeArgs& a, hipStream_t st) {
  if constexpr (!fits<BASE, LH, LL, G>()) {
    return -2;
  } else {
    dim3 grid(a.nsplit, a.g.n_kv_heads, a.g.batch * a.n_layers_launched);
    hipLaunchKernelGGL((decode_kernel<BASE, LH, LL, G>), grid, dim3(Plan<BASE, LH, LL, G>::NT), 0, st, a);
    return hipGetLastError() == hipSuccess ? 0 : -5;
  }
}

template <int BASE, int LH, int LL>
int launch_dec(const DecodeArgs& a, hipStream_t st) {
  if constexpr (BASE == 1) {
    return launch_g<BASE, LH, LL, 128>(a, st);
  } else {
    if (a.g.G == 128) return launch_g<BASE, LH, LL, 128>(a, st);
    if (a.g.G == 64) return launch_g<BASE, LH, LL, 64>(a, st);
    return launch_g<BASE, LH, LL, 32>(a, st);
  }
}

template <int BASE, int LH, int LL>
int occ_dec(int G, bool waves) {
  if constexpr (BASE == 1) {
    return waves ? waves_of<BASE, LH, LL, 128>() : occupancy<BASE, LH, LL, 128>();
  } else {
    if (G == 128) return waves ? waves_of<BASE, LH, LL, 128>() : occupancy<BASE, LH, LL, 128>();
    if (G == 64) return waves ? waves_of<BASE, LH, LL, 64>() : occupancy<BASE, LH, LL, 64>();
    return waves ? waves_of<BASE, LH, LL, 32>() : occupancy<BASE, LH, LL, 32>();
  }
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
  if (B == 2 && LH == 6 && LL == 5) return launch_dec<2, 6, 5>(a, s);
  if (B == 2 && LH == 5 && LL == 4) return launch_dec<2, 5, 4>(a, s);
  // the rest of the level grid (uniform sweeps, Sec. 4.2): metadata per row only
  if (a.g.G == 128) {
    if (B == 0 && LH == 8 && LL == 7) return launch_g<0, 8, 7, 128>(a, s);
    if (B == 0 && LH == 7 && LL == 6) return launch_g<0, 7, 6, 128>(a, s);
    if (B == 0 && LH == 3 && LL == 2) return launch_g<0, 3, 2, 128>(a, s);
    if (B == 2 && LH == 8 && LL == 7) return launch_g<2, 8, 7, 128>(a, s);
    if (B == 2 && LH == 7 && LL == 6) return launch_g<2, 7, 6, 128>(a, s);
    if (B == 2 && LH == 3 && LL == 2) return launch_g<2, 3, 2, 128>(a, s);
  }
  return -2;
}

static int decode_query(int base, int LH, int LL, int G, bool waves) {
  if (base == 0 && LH == 6 && LL == 5) return occ_dec<0, 6, 5>(G, waves);
  if (base == 0 && LH == 5 && LL == 4) return occ_dec<0, 5, 4>(G, waves);
  if (base == 0 && LH == 6 && LL == 4) return occ_dec<0, 6, 4>(G, waves);
  if (base == 0 && LH == 4 && LL == 3) return occ_dec<0, 4, 3>(G, waves);
  if (base == 0 && LH == 5 && LL == 3) return occ_dec<0, 5, 3>(G, waves);
  if (base == 0 && LH == 6 && LL == 3) return occ_dec<0, 6, 3>(G, waves);
  if (base == 1 && LH == 4 && LL == 3) return occ_dec<1, 4, 3>(G, waves);
  if (base == 2 && LH == 6 && LL == 5) return occ_dec<2, 6, 5>(G, waves);
  if (base == 2 && LH == 5 && LL == 4) return occ_dec<2, 5, 4>(G, waves);
  if (G == 128) {
    if (base == 0 && LH == 8 && LL == 7) return waves ? waves_of<0, 8, 7, 128>() : occupancy<0, 8, 7, 128>();
    if (base == 0 && LH == 7 && LL == 6) return waves ? waves_of<0, 7, 6, 128>() : occupancy<0, 7, 6, 128>();
    if (base == 0 && LH == 3 && LL == 2) return waves ? waves_of<0, 3, 2, 128>() : occupancy<0, 3, 2, 128>();
    if (base == 2 && LH == 8 && LL == 7) return waves ? waves_of<2, 8, 7, 128>() : occupancy<2, 8, 7, 128>();
    if (base == 2 && LH == 7 && LL == 6) return waves ? waves_of<2, 7, 6, 128>() : occupancy<2, 7, 6, 128>();
    if (base == 2 && LH == 3 && LL == 2) return waves ? waves_of<2, 3, 2, 128>() : occupancy<2, 3, 2, 128>();
  }
  return waves ? 8 : 1;
}

int decode_blocks_per_cu(int base, int LH, int LL, int G) { return decode_query(base, LH, LL, G, false); }
int decode_waves(int base, int LH, int LL, int G) { return decode_query(base, LH, LL, G, true); }

}  // namespace semkv

#ifdef SEMKV_TIMELINE
#include "semkv.h"
#include "semkv_timeline.h"
extern "C" int semkv_timeline_read(void* host, size_t bytes) {
  if (host == nullptr || bytes != sizeof(semkv::g_timeline)) return SEMKV_EINVAL;
  return hipMemcpyFromSymbol(host, HIP_SYMBOL(semkv::g_timeline), bytes) == hipSuccess ? SEMKV_OK : SEMKV_EHIP;
}
#endif
