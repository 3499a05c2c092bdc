// semkv_fmt.h -- the packed storage format, as compile-time arithmetic shared
// by the host API and the gfx950 kernels of this library.
//
// Mixed-radix packing (SemKV, Sec. 4.1): a symbol holds n codes of base L as
// sum_i c_i L^i in the least number of bits.  n is 3 for L = 5 (7 bits, the
// paper's three-in-seven) and 5 for L = 6 (13 bits, five-in-thirteen); the
// TurboQuant-MSE levels of Sec. 4.9 use 4 codes of L = 4 (8 bits) and 5 codes
// of L = 3 (8 bits).  The rest of the integer-level grid swept in Sec. 4.2:
// 8 codes of L = 2 (8 bits), 2 of L = 8 (6 bits) and 7 of L = 7 (20 bits,
// 2.857 bits per value; the paper gives no 7-level packing).  A K line is one token row (128 channels); a V line is one
// channel column over the 64 slots of a tile.  Segment j of a line holds its
// symbols p = j, j+4, j+8, ...; a body is segment 0 of all lines, then
// segments 1, 2, 3, LSB first, zero padded to 16 bytes.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace semkv {

constexpr int kSlots = 64;   // token slots per tile
constexpr int kD = 128;      // head dimension

__host__ __device__ constexpr int sym_digits(int L) {
  return L == 2 ? 8 : L == 3 ? 5 : L == 4 ? 4 : L == 5 ? 3 : L == 6 ? 5 : L == 7 ? 7 : L == 8 ? 2 : 0;
}

__host__ __device__ constexpr int width_of(int L, int nd) {
  uint64_t p = 1;
  for (int i = 0; i < nd; ++i) p *= (uint64_t)L;
  int w = 0;
  while ((uint64_t(1) << w) < p) ++w;
  return w;
}

__host__ __device__ constexpr int num_syms(int L, int nvals) {
  return (nvals + sym_digits(L) - 1) / sym_digits(L);
}

// codes held by symbol p of a line of nvals codes
__host__ __device__ constexpr int sym_ndig(int L, int nvals, int p) {
  return nvals - sym_digits(L) * p < sym_digits(L) ? nvals - sym_digits(L) * p : sym_digits(L);
}

__host__ __device__ constexpr int sym_width(int L, int nvals, int p) {
  return width_of(L, sym_ndig(L, nvals, p));
}

__host__ __device__ constexpr int seg_bits(int L, int nvals, int j) {
  int b = 0;
  for (int p = j; p < num_syms(L, nvals); p += 4) b += sym_width(L, nvals, p);
  return b;
}

__host__ __device__ constexpr int seg_nsym(int L, int nvals, int j) {
  int c = 0;
  for (int p = j; p < num_syms(L, nvals); p += 4) ++c;
  return c;
}

// first bit of segment j (all lines of segments < j come before it)
__host__ __device__ constexpr int seg_start(int L, int nvals, int nlines, int j) {
  int b = 0;
  for (int i = 0; i < j; ++i) b += nlines * seg_bits(L, nvals, i);
  return b;
}

__host__ __device__ constexpr int body_bits_k(int L) { return seg_start(L, kD, kSlots, 4); }
__host__ __device__ constexpr int body_bits_v(int L) { return seg_start(L, kSlots, kD, 4); }

__host__ __device__ constexpr int tile_bytes(int L) {
  int bits = body_bits_k(L) > body_bits_v(L) ? body_bits_k(L) : body_bits_v(L);
  return ((bits + 7) / 8 + 15) / 16 * 16;
}

// bytes of one slot-major metadata block (K or V) of a tile: fp16 {scale,
// zero} per group for the affine bases (0, and 2 under a rotation), one fp16
// rho for TurboQuant-MSE (1)
__host__ __device__ constexpr int meta_bytes(int base, int G) {
  return base != 1 ? (kD / G) * kSlots * 4 : kSlots * 2;
}

__host__ __device__ constexpr int record_bytes(int base, int L, int G) {
  return 2 * tile_bytes(L) + 2 * meta_bytes(base, G);
}

// Per-segment geometry of a body of NL lines of NV codes as compile-time
// tables: kernels that pick a segment by lane read constants rather than
// re-running the loops above.
template <int L, int NV, int NL>
struct SegTable {
  static_assert(num_syms(L, NV) <= 64, "segment symbols");
  int start[4] = {0, 0, 0, 0};   // first bit of segment j
  int bits[4] = {0, 0, 0, 0};    // bits of segment j in one line
  int width[4][16] = {};         // width of the k-th symbol of segment j (0: none)
  int ndig[4][16] = {};          // codes of that symbol
  constexpr SegTable() {
    for (int j = 0; j < 4; ++j) {
      start[j] = seg_start(L, NV, NL, j);
      bits[j] = seg_bits(L, NV, j);
      for (int k = 0; k < 16; ++k) {
        const int p = j + 4 * k;
        width[j][k] = p < num_syms(L, NV) ? sym_width(L, NV, p) : 0;
        ndig[j][k] = p < num_syms(L, NV) ? sym_ndig(L, NV, p) : 0;
      }
    }
  }
};

// value of a 4-entry table at a run-time index, as selects
template <typename T>
__host__ __device__ inline T pick4(int j, T a, T b, T c, T d) {
  return j == 0 ? a : j == 1 ? b : j == 2 ? c : d;
}

}  // namespace semkv
