// Internal declarations shared by the host (host.cpp) and device (kernels.hip)
// halves of libleech.  Not part of the public ABI (include/leech.h).
#pragma once

#include <algorithm>
#include <cstdint>
#include <string>

#include "leech.h"

#ifndef __HIPCC__
#define __host__
#define __device__
#endif

namespace leech {

constexpr int kDim = 24;
constexpr int kMaxLevels = 5;
constexpr int kTableSlots = LEECH_TABLE_SLOTS;
// Classes of the ball Λ24(12) (shells 2..12); the layouts only hold these ids.
constexpr int kBallClasses = 301;
constexpr int kWave = 64;
constexpr int kPadBytes = 16;        // trailing zero bytes after every record stream

// Record widths of the four layouts (bytes).
constexpr int kPlanes14Bytes = 14;
// Planes14: three 32-bit pair words at bits 0, 32, 64, class (9 bits) and
// gain bit from bit 96.  A block's 24 coordinates form the 12 pairs of
// kPairCoords; pair q = 4w + k lies in word w: rotated right by 4k and masked
// with 0x08070807, the word holds the level code (level + 1) of the pair's
// first coordinate in bits 0..2 and its non-negative bit in bit 11, and the
// second coordinate's in bits 16..18 and 27 (the four rotations use each bit
// of the word once).
constexpr int kP14PairWordPos[3] = {0, 32, 64};
constexpr int kP14ClassPos = 96;

// The pairs the GEMV multiplies with the staged activation, in summation
// order: pair q = (kPairCoords[q][0], kPairCoords[q][1]).
constexpr int kPairCoords[12][2] = {{0, 16}, {4, 20}, {8, 12}, {1, 17}, {5, 21}, {9, 13},
                                    {2, 18}, {6, 22}, {10, 14}, {3, 19}, {7, 23}, {11, 15}};

__host__ __device__ inline uint32_t p14_rotl(uint32_t v, int s) {
  s &= 31;
  return s ? (v << s) | (v >> (32 - s)) : v;
}

// Planes14 pair words of a block from each coordinate's level code (1..5) and
// its non-negative bit (bit i of pos).
__host__ __device__ inline void planes14_words(const uint8_t code[24], uint32_t pos,
                                               uint32_t w[3]) {
  w[0] = w[1] = w[2] = 0;
  for (int q = 0; q < 12; ++q) {
    const int a = kPairCoords[q][0], b = kPairCoords[q][1];
    const uint32_t sel = (uint32_t)code[a] | (pos >> a & 1u) << 11 | (uint32_t)code[b] << 16 |
                         (pos >> b & 1u) << 27;
    w[q >> 2] |= p14_rotl(sel, 4 * (q & 3));
  }
}

// The inverse: level codes and the non-negative mask of a block's pair words.
__host__ __device__ inline void planes14_codes(const uint32_t w[3], uint8_t code[24],
                                               uint32_t* pos) {
  uint32_t p = 0;
  for (int q = 0; q < 12; ++q) {
    const uint32_t sel = p14_rotl(w[q >> 2], 32 - 4 * (q & 3)) & 0x08070807u;
    const int a = kPairCoords[q][0], b = kPairCoords[q][1];
    code[a] = (uint8_t)(sel & 7u);
    code[b] = (uint8_t)(sel >> 16 & 7u);
    p |= (sel >> 11 & 1u) << a | (sel >> 27 & 1u) << b;
  }
  *pos = p;
}
constexpr int kPlanes12Bytes = 12;
constexpr int kGolay70Bytes = 9;
constexpr int kSlot32Small = 16;     // ≤ 4 levels
constexpr int kSlot32Large = 20;     // 5 levels
constexpr int kUnitEntryBytes = 16;  // per-unit side entry: u64 bitmap, u32 base, u32 zero

// Planes12x record (96 bits, little-endian from its first byte, words W0, W1,
// W2): bits [0, 12) hold the block's table entry, class | gain << 9, or, for a
// block with five levels, kExcEntry0 + its index in its tile's exception
// list; the other 84 bits hold the 12 pairs of coordinates in the GEMV's
// consumption order, each as one selector word taken straight from the
// record.  Pair q's selector word is (kP12Sel[q]): word w rotated right by s
// (rot = 1), or words w + 1 : w shifted right by s (rot = 0); its bits 0, 1
// hold the level of coordinate kPairCoords[q][0] (bit 0 the low bit), bit
// 8 + k that coordinate's non-negative bit, bits 16, 17 and 24 + l the same
// of kPairCoords[q][1].  Bits of the record no selector names are zero.  A
// five-level block carries only its entry field; its exact Planes14 record is
// in the exception list.
struct P12Sel {
  int rot, word, shift, k, l;
};
constexpr P12Sel kP12Sel[12] = {{0, 0, 12, 0, 0}, {0, 0, 14, 0, 0}, {0, 0, 16, 0, 0},
                                {0, 0, 18, 0, 1}, {1, 1, 12, 0, 1}, {1, 1, 14, 0, 1},
                                {0, 1, 9, 0, 0},  {0, 1, 18, 1, 0}, {0, 1, 23, 1, 1},
                                {1, 2, 11, 0, 1}, {1, 2, 5, 0, 0},  {1, 2, 14, 1, 3}};
// Record bit of bit j (0..31) of pair q's selector word.
__host__ __device__ constexpr int p12_bit(int q, int j) {
  return kP12Sel[q].rot ? 32 * kP12Sel[q].word + (j + kP12Sel[q].shift) % 32
                        : 32 * kP12Sel[q].word + kP12Sel[q].shift + j;
}
// The six record bits of pair q: level bits 0, 1 and the non-negative bit of
// its first coordinate, then of its second.
__host__ __device__ constexpr int p12_pair_bit(int q, int t) {
  return p12_bit(q, t == 0 ? 0 : t == 1 ? 1 : t == 2 ? 8 + kP12Sel[q].k : t == 3 ? 16
                    : t == 4 ? 17 : 24 + kP12Sel[q].l);
}
// Every pair bit is a distinct record bit outside the entry field.
__host__ __device__ constexpr bool p12_layout_ok() {
  for (int q = 0; q < 12; ++q)
    for (int t = 0; t < 6; ++t) {
      const int b = p12_pair_bit(q, t);
      if (b < 12 || b >= 96) return false;
      for (int q2 = 0; q2 < 12; ++q2)
        for (int t2 = 0; t2 < 6; ++t2)
          if ((q2 != q || t2 != t) && p12_pair_bit(q2, t2) == b) return false;
    }
  return true;
}
static_assert(p12_layout_ok(), "Planes12x pair selectors overlap");
// Exceptions of Planes12x and Golay70: a block whose record cannot hold it
// carries only its table entry field, kExcEntry0 + its index in its tile's
// exception list; a list entry is 16 bytes, the block's exact Planes14 record
// (14 bytes, bits [106, 112) zero) with the block's storage slot inside its
// tile in bits [106, 128); lists follow each other in tile order and a u32 per
// tile gives the index of its first entry.
constexpr int kExcEntryBytes = 16;
constexpr int kExcSlotShift = 106;
constexpr int kExcSlotBits = 22;
constexpr uint32_t kExcEntry0 = 1024;        // entry of a tile's first exception
constexpr uint32_t kExcMax = 4096 - 1024;    // exceptions one tile may hold
// Golay70 record (72 bits): table entry field [0, 12) (class | gain << 9, or
// an exception's), codeword message [12, 24), low code plane [24, 48), high
// code plane [48, 72) (bit i of each = coordinate i).
constexpr int kG70MsgPos = 12, kG70C0Pos = 24, kG70C1Pos = 48;

// Device class record: 32 bytes per class id (LEECH_DEVICE_TABLE_BYTES / 512).
//   perm[8]   : byte table read by v_perm_b32: perm[0] = 0x80 (the binary16
//               sign byte), perm[1 + k] = |z| of level k (k < n_levels),
//               then zeros.  Planes records code level k as k + 1.
//   inv_norm  : f32 of 1 / (4 √m)
//   info      : n_levels | parity << 8 | shell << 16 | Golay70 sign bits << 24
//               (bit side·4 + code set when g70[side][code] < 0)
//   g70[2][4] : Golay70 signed values, [side][2-bit code]
//   g70abs[8] : |g70[side][code]| at side·4 + code
struct DevClass {
  uint8_t perm[8];
  float inv_norm;
  uint32_t info;
  int8_t g70[2][4];
  uint8_t g70abs[8];
};
constexpr int kSignByteCode = 0;
__host__ __device__ inline int level_code(int level) { return level + 1; }
static_assert(sizeof(DevClass) == 32, "device class record is 32 bytes");

// Geometry shared by the expansion and the kernels: rows are grouped into
// tiles of R = tile_rows rows; a unit is the R · C (or fewer, at the edges)
// blocks of one tile × C = lane_cols consecutive block columns, stored row by
// row, and a wavefront step decodes one unit with lane r · C + c on block
// (r, c) of it (lanes past R · C hold no block).  Units of a tile are stored in
// column order; tiles in row order.
struct Geometry {
  int64_t M, nb;
  int C;            // lane_cols
  int R;            // tile_rows
  int64_t tiles;    // ceil(M / R)
  int64_t groups;   // units per tile = ceil(nb / C)

  Geometry(int64_t M_, int64_t nb_, int C_, int R_)
      : M(M_), nb(nb_), C(C_), R(R_), tiles((M_ + R_ - 1) / R_), groups((nb_ + C_ - 1) / C_) {}
  int rows_in_tile(int64_t t) const { return (int)std::min<int64_t>(R, M - t * R); }
  int cols_in_group(int64_t g) const { return (int)std::min<int64_t>(C, nb - g * C); }
  // first block index of unit (t, g) in storage order
  int64_t unit_base(int64_t t, int64_t g) const {
    return t * (int64_t)R * nb + g * (int64_t)rows_in_tile(t) * C;
  }
  // storage index of block (r, j)
  int64_t index(int64_t r, int64_t j) const {
    int64_t t = r / R, g = j / C;
    return unit_base(t, g) + (r % R) * cols_in_group(g) + (j % C);
  }
  // sequential unit number (t * groups + g): Slot32/Golay70 side entries
  int64_t unit_id(int64_t t, int64_t g) const { return t * groups + g; }
  int64_t units() const { return tiles * groups; }
};

// A geometry the kernels serve: lane_cols 1, 2, 3, 4, 8 or 16 and tile_rows a
// multiple of 4 with tile_rows · lane_cols ≤ 64 (so every tile starts on a
// 4-byte boundary of each fixed-stride stream).
inline bool geometry_ok(int C, int R) {
  return (C == 1 || C == 2 || C == 3 || C == 4 || C == 8 || C == 16) && R >= 4 && R % 4 == 0 &&
         R * C <= kWave;
}
// The library's geometry for an M × (24 · nb) matrix.
void choose_geometry(int64_t M, int64_t nb, int* C, int* R);

// thread-local error reporting
int set_error(int code, const std::string& msg);
void clear_error();

}  // namespace leech
