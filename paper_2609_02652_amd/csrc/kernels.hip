// Device half of libleech: fused Λ24(12) dequantize + GEMV for gfx950, its
// verification decode, the FP16 GEMV control and the no-weights control.
//
// Paper: §2.3 "The kernel" (a divergence-free read of decoded-field records
// with shifts, masks and a class-table lookup, f32 accumulation, a wavefront
// reduction), §3.2 (the four layouts), §3.3 (the no-weights control).
//
// Geometry (MI355X-specific; the paper's one-warp-per-row geometry is not
// used).  A workgroup owns one tile of tile_rows = 64 / lane_cols rows and
// walks its units: a unit is the ≤ 64 blocks of the tile's rows in lane_cols
// consecutive block columns, stored contiguously, so one wavefront step loads
// one unit with coalesced 128-byte lines (896 bytes of Planes14 records and
// 128 bytes of fp16 scales).  Each wavefront keeps kPrefetch units in flight:
// their loads are issued before the workgroup stages x and the class table in
// LDS, and every step refills the slot it consumed.  Lane (r, c) of a step
// handles block (tile·R + r, g·C + c) and keeps its row's partial sum in a
// register; at the end the C lanes of a row are summed by an xor butterfly and
// the waves through LDS, in a fixed order, so y depends only on
// (M, Kpad, lane_cols), never on the layout.
//
// Decode.  The paper's per-coordinate predicated tree is replaced, since the
// MI355X has about an order of magnitude less VALU issue per HBM byte than the
// paper's GPU: the four 24-bit planes of a block (p0, p1, p2 and the inverted
// sign mask) are transposed 4×4 inside every nibble with eight v_bfi_b32,
// giving one nibble per coordinate; a v_perm_b32 byte lookup in the class's
// 8-byte table then yields two binary16 values at once, each the coordinate's
// magnitude |z| as a subnormal (|z|·2^-24, exact) with the sign in bit 15.
// v_dot2_f32_f16 multiplies them with x exactly and sums in f32; the block's
// factor 2^24 · scale · centroid[gain] / (4√m) is applied once per block.

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <string>

#include "leech_internal.h"

namespace leech {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4a __attribute__((ext_vector_type(4)));

constexpr int kNoWeights = 99;   // layout id of the no-weights control
constexpr int kPrefetch = 8;     // units in flight per wavefront
constexpr float kTwo24 = 16777216.0f;

struct GemvArgs {
  const uint8_t* main;
  const uint8_t* side0;
  const uint8_t* side1;
  const DevClass* table;        // global copy of LEECH_TABLE_DEVICE
  const uint32_t* codewords;    // Golay70 only
  const uint16_t* scale;        // fp16, storage order
  const uint16_t* x;            // fp16 [Kpad]
  float* y;                     // f32 [M]
  float cen0, cen1;
  int64_t M, nb, groups;
  int C, R, waves;
  int64_t tiles;
  uint64_t n_exc;               // exception records (Planes12x, Golay70)
};

// Waves per GEMV workgroup, at most: 8 waves leave each lane up to 256 VGPRs,
// so the eight prefetch slots and the exception-path decode stay in registers.
constexpr int kMaxWaves = 8;
constexpr int kExcLdsBytes = 32 * 1024;   // a tile's exception records staged in LDS

// Where side data comes from: global memory (verification decode, and the
// GEMV's first prefetches) or the workgroup's LDS copies (the GEMV's loop).
struct GlobalSide {
  const GemvArgs* a;
  __device__ __forceinline__ uint32_t p12_base(int tile) const {
    return ((const uint32_t*)a->side1)[tile];
  }
  __device__ __forceinline__ void unit_entry(const uint8_t* side, int unit, uint64_t& bits,
                                             uint32_t& base) const {
    const uint8_t* ent = side + (int64_t)unit * kUnitEntryBytes;
    bits = *(const uint64_t*)ent;
    base = *(const uint32_t*)(ent + 8);
  }
  // four-word window holding exception record ex (exact Planes14 record)
  __device__ __forceinline__ void exc_window(uint64_t ex, uint32_t w[4], uint32_t& sh) const;
};
struct LdsSide {
  const GemvArgs* a;
  const uint8_t* exc;        // LDS copy of exception bytes from global offset exc_start
  uint64_t exc_start;
  bool exc_in_lds;           // false: the tile's records exceed the LDS budget
  const uint8_t* units;      // LDS copy of the tile's unit entries
  int unit0;                 // first unit id of the tile
  uint32_t p12base;          // Planes12x: first exception index of the tile
  __device__ __forceinline__ uint32_t p12_base(int) const { return p12base; }
  __device__ __forceinline__ void unit_entry(const uint8_t*, int unit, uint64_t& bits,
                                             uint32_t& base) const {
    const uint8_t* ent = units + (unit - unit0) * kUnitEntryBytes;
    bits = *(const uint64_t*)ent;
    base = *(const uint32_t*)(ent + 8);
  }
  __device__ __forceinline__ void exc_window(uint64_t ex, uint32_t w[4], uint32_t& sh) const;
};

__device__ __forceinline__ void GlobalSide::exc_window(uint64_t ex, uint32_t w[4],
                                                      uint32_t& sh) const {
  const uint64_t off = ex * kPlanes14Bytes;
  const uint32_t* p = (const uint32_t*)(a->side0 + (off & ~3ull));
  w[0] = p[0]; w[1] = p[1]; w[2] = p[2]; w[3] = p[3];
  sh = (uint32_t)(off & 2) * 8u;
}
__device__ __forceinline__ void LdsSide::exc_window(uint64_t ex, uint32_t w[4], uint32_t& sh) const {
  const uint64_t goff = ex * kPlanes14Bytes;
  if (exc_in_lds) {
    const uint32_t* p = (const uint32_t*)(exc + ((uint32_t)(goff - exc_start) & ~3u));
    w[0] = p[0]; w[1] = p[1]; w[2] = p[2]; w[3] = p[3];
  } else {
    const uint32_t* p = (const uint32_t*)(a->side0 + (goff & ~3ull));
    w[0] = p[0]; w[1] = p[1]; w[2] = p[2]; w[3] = p[3];
  }
  sh = (uint32_t)(goff & 2) * 8u;
}

// Per-(class, gain) entry staged in LDS; e = class | gain << 9.
struct LdsEntry {
  uint32_t tlo, thi;    // v_perm table (DevClass::perm)
  float factor;         // 2^24 · centroid[gain] / (4√m)
  uint32_t nlev;        // level count
};
// Golay70 per-class entry staged in LDS (index = class id).
struct G70Entry {
  uint32_t alo, ahi;    // |value| at side·4 + code
  uint32_t slo, shi;    // 0x80 where that value is negative
};

__device__ __forceinline__ uint32_t align(uint32_t hi, uint32_t lo, uint32_t s) {
  return __builtin_amdgcn_alignbit(hi, lo, s);
}
__device__ __forceinline__ uint32_t perm(uint32_t s0, uint32_t s1, uint32_t sel) {
  return __builtin_amdgcn_perm(s0, s1, sel);
}
__device__ __forceinline__ uint32_t bfi(uint32_t m, uint32_t a, uint32_t b) {
  return (m & a) | (~m & b);
}
// Reinterpret a 32-bit word as two binary16 values.  Takes the word by value:
// applying __builtin_bit_cast directly to an ext_vector element (w.y) reads
// element 0 with this compiler, so vector elements go through this function.
__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// 4×4 bit transpose inside every nibble: on return n[r] bit (4g + q) is bit
// (4g + r) of plane q (q = 0..3), i.e. nibble g of n[r] collects the four
// plane bits of coordinate 4g + r.
__device__ __forceinline__ void nibble_transpose(uint32_t q0, uint32_t q1, uint32_t q2,
                                                 uint32_t q3, uint32_t n[4]) {
  const uint32_t a0 = bfi(0xCCCCCCCCu, q2 << 2, q0);
  const uint32_t a2 = bfi(0x33333333u, q0 >> 2, q2);
  const uint32_t a1 = bfi(0xCCCCCCCCu, q3 << 2, q1);
  const uint32_t a3 = bfi(0x33333333u, q1 >> 2, q3);
  n[0] = bfi(0xAAAAAAAAu, a1 << 1, a0);
  n[1] = bfi(0x55555555u, a0 >> 1, a1);
  n[2] = bfi(0xAAAAAAAAu, a3 << 1, a2);
  n[3] = bfi(0x55555555u, a2 >> 1, a3);
}

// The three selector-source words of nibble register N: each holds the
// nibbles of two coordinates in the low nibbles of bytes 0/1 and 2/3:
//   s[0]: coordinates (r, 16+r)   s[1]: (4+r, 20+r)   s[2]: (8+r, 12+r)
__device__ __forceinline__ void pair_sources(uint32_t N, uint32_t s[3]) {
  const uint32_t R = align(N, N, 4);           // rotate right by one nibble
  s[0] = perm(N, N, 0x02020000u);
  s[1] = perm(R, R, 0x02020000u);
  s[2] = perm(R, N, 0x05050101u);
}

// Planes core: nibble (c0, c1, c2, ¬s) per coordinate, with c = level + 1 the
// level code -> 12 binary16 pairs.  Selector byte for the low half: the code
// (table bytes 1..5 hold |z| of levels 0..4); for the high half: 0 (table
// byte 0 = 0x80) when negative, 8 when not (v_perm's selector 8 replicates
// bit 7 of table byte 1, a magnitude below 0x80, giving 0x00).  Pair 3r + k
// of h[] covers the coordinates listed by pair_sources.
__device__ __forceinline__ void planes_core(uint32_t p0, uint32_t p1, uint32_t p2, uint32_t sm,
                                            uint32_t tlo, uint32_t thi, uint32_t h[12]) {
  uint32_t n[4];
  nibble_transpose(p0, p1, p2, ~sm, n);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    uint32_t s[3];
    pair_sources(n[r], s);
#pragma unroll
    for (int k = 0; k < 3; ++k) h[3 * r + k] = perm(thi, tlo, s[k] & 0x08070807u);
  }
}

// Golay70 core: nibble (c0, c1, side, 0) -> index side·4 + code; the low half
// is |value| from one 8-byte table, the high half its sign byte from another.
__device__ __forceinline__ void golay70_core(uint32_t c0, uint32_t c1, uint32_t side,
                                             const G70Entry& t, uint32_t h[12]) {
  uint32_t n[4];
  nibble_transpose(c0, c1, side, 0u, n);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    uint32_t s[3];
    pair_sources(n[r], s);
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      const uint32_t sel = s[k] & 0x07070707u;
      h[3 * r + k] = bfi(0xFF00FF00u, perm(t.shi, t.slo, sel), perm(t.ahi, t.alo, sel));
    }
  }
}

// Coordinates of pair k of h[] (and of the staged x pairs).
__device__ __forceinline__ void pair_coords(int k, int& c0, int& c1) {
  const int r = k / 3, m = k % 3;
  c0 = m == 0 ? r : (m == 1 ? 4 + r : 8 + r);
  c1 = m == 0 ? 16 + r : (m == 1 ? 20 + r : 12 + r);
}

// ---------------------------------------------------------- per-block reads
// Where a lane's block sits: storage index ubase + ul, with ubase the first
// block of the unit (uniform across the wavefront) and ul the lane's position
// inside the unit.
struct LaneBlock {
  int64_t ubase;     // storage index of the unit's first block (wave-uniform)
  int32_t unit;      // tile·groups + g (wave-uniform)
  int32_t tile;      // (wave-uniform)
  uint32_t ul;       // position inside the unit
  uint32_t loff;     // ul · record stride (fixed-stride layouts)
  bool valid;
  __device__ __forceinline__ uint64_t idx() const { return (uint64_t)ubase + ul; }
};

template <int LAYOUT> struct Stride { static constexpr uint32_t v = 0; };
template <> struct Stride<LEECH_PLANES14> { static constexpr uint32_t v = kPlanes14Bytes; };
template <> struct Stride<LEECH_PLANES12X> { static constexpr uint32_t v = kPlanes12Bytes; };
template <> struct Stride<LEECH_GOLAY70> { static constexpr uint32_t v = kGolay70Bytes; };

// Words a lane prefetches for one block.
struct Pref {
  uint32_t w0, w1, w2, w3, w4;
  uint32_t scale;
  uint32_t sh;       // bit offset of the record inside its first word
};

// Window of n words holding the record of block i at stride `stride` bytes:
// the wave-uniform part of the byte offset goes into the base pointer, the
// lane part stays a 32-bit offset.
template <int STRIDE>
__device__ __forceinline__ const uint32_t* record_window(const uint8_t* base, const LaneBlock& b,
                                                         uint32_t& sh) {
  const uint64_t U = (uint64_t)b.ubase * STRIDE;
  const uint32_t lo = (uint32_t)(U & 3u) + b.loff;
  sh = (lo & 3u) * 8u;
  return (const uint32_t*)(base + (U & ~3ull) + (lo & ~3u));
}

// Loads are issued unconditionally (callers hand in a clamped, in-bounds
// block for lanes or units that do not exist and ignore the data): branches
// around loads would make the compiler's wait counts conservative.
template <int LAYOUT, class SIDE>
__device__ __forceinline__ Pref load_block(const GemvArgs& a, const LaneBlock& b, const SIDE& side) {
  Pref p = {0, 0, 0, 0, 0, 0, 0};
  if constexpr (LAYOUT == LEECH_PLANES14) {
    const u32x4 w = *(const u32x4*)record_window<kPlanes14Bytes>(a.main, b, p.sh);
    p.w0 = w.x; p.w1 = w.y; p.w2 = w.z; p.w3 = w.w;
  } else if constexpr (LAYOUT == LEECH_PLANES12X) {
    const u32x3 w = *(const u32x3*)record_window<kPlanes12Bytes>(a.main, b, p.sh);
    p.w0 = w.x; p.w1 = w.y; p.w2 = w.z;
  } else if constexpr (LAYOUT == LEECH_SLOT32) {
    uint64_t bits;
    uint32_t base;
    side.unit_entry(a.side0, b.unit, bits, base);
    const uint32_t nbelow = (uint32_t)__builtin_popcountll(bits & ((1ull << b.ul) - 1ull));
    const uint32_t* rec = (const uint32_t*)(a.main + (uint64_t)base * 4) +
                          (b.ul * (uint32_t)kSlot32Small + nbelow * (uint32_t)(kSlot32Large - kSlot32Small)) / 4;
    const u32x4 w = *(const u32x4*)rec;
    p.w0 = w.x; p.w1 = w.y; p.w2 = w.z; p.w3 = w.w; p.w4 = rec[4];
  } else if constexpr (LAYOUT == LEECH_GOLAY70) {
    const u32x3 w = *(const u32x3*)record_window<kGolay70Bytes>(a.main, b, p.sh);
    p.w0 = w.x; p.w1 = w.y; p.w2 = w.z;
  }
  if constexpr (LAYOUT != kNoWeights)
    p.scale = *(const uint16_t*)((const uint8_t*)(a.scale + b.ubase) + (uint32_t)(b.ul * 2u));
  return p;
}

// Planes14 fields of the four-word window starting at byte (14·i) & ~3: the
// record begins 0 or 16 bits in (§2.3: a four-word window, shift 0 or 16).
__device__ __forceinline__ void planes14_fields(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                                uint32_t sh, uint32_t& e, uint32_t& p0,
                                                uint32_t& p1, uint32_t& p2, uint32_t& sm) {
  const uint32_t r0 = align(w1, w0, sh), r1 = align(w2, w1, sh), r2 = align(w3, w2, sh);
  const uint32_t r3 = w3 >> sh;
  e = r0 & 1023u;              // class | gain << 9
  sm = align(r1, r0, 10);      // plane bits above 23 are never read
  p0 = r1 >> 2;
  p1 = align(r2, r1, 26);
  p2 = align(r3, r2, 18);
}

// Decode one block into 12 binary16 pairs and its table entry index.
// tab(e) returns the LdsEntry of e and g70(class) the G70Entry of a class
// (from LDS in the GEMV, built from the global table in the verification
// decode); cw(rank) is the Golay codeword of a rank.
template <int LAYOUT, class TAB, class G70, class CW, class SIDE>
__device__ __forceinline__ void decode_block(const GemvArgs& a, const LaneBlock& b, const Pref& p,
                                             TAB tab, G70 g70, CW cw, const SIDE& side,
                                             uint32_t h[12], uint32_t& e) {
  uint32_t p0 = 0, p1 = 0, p2 = 0, sm = 0;
  if constexpr (LAYOUT == LEECH_PLANES14) {
    planes14_fields(p.w0, p.w1, p.w2, p.w3, p.sh, e, p0, p1, p2, sm);
  } else if constexpr (LAYOUT == LEECH_PLANES12X) {
    const uint32_t field = p.w2 >> kP12ExcShift;
    if (field) {      // five-level block: exact Planes14 record from the tile's list
      const uint64_t ex = (uint64_t)(side.p12_base(b.tile) + field - 1);
      uint32_t w[4], sh;
      side.exc_window(ex, w, sh);
      planes14_fields(w[0], w[1], w[2], w[3], sh, e, p0, p1, p2, sm);
    } else {
      // two-plane level (0..3) -> code planes of level + 1, bit-parallel
      e = p.w0 & 1023u;
      sm = align(p.w1, p.w0, 10);
      const uint32_t l0 = p.w1 >> 2, l1 = align(p.w2, p.w1, 26);
      p0 = ~l0;
      p1 = l0 ^ l1;
      p2 = l0 & l1;
    }
  } else if constexpr (LAYOUT == LEECH_SLOT32) {
    // one-hot masks of levels 1..4 -> code planes of level + 1 (codes 1..5)
    e = p.w0 & 1023u;
    const uint32_t L = tab(e).nlev;
    sm = align(p.w1, p.w0, 10);
    const uint32_t m1 = L > 1 ? p.w1 >> 2 : 0u;
    const uint32_t m2 = L > 2 ? align(p.w2, p.w1, 26) : 0u;
    const uint32_t m3 = L > 3 ? align(p.w3, p.w2, 18) : 0u;
    const uint32_t m4 = L > 4 ? align(p.w4, p.w3, 10) : 0u;
    p0 = ~(m1 | m3);
    p1 = m1 | m2;
    p2 = m3 | m4;
  } else if constexpr (LAYOUT == LEECH_GOLAY70) {
    const uint32_t r0 = align(p.w1, p.w0, p.sh), r1 = align(p.w2, p.w1, p.sh), r2 = p.w2 >> p.sh;
    if ((r2 >> 6) & 1u) {   // exception: exact Planes14 record located by the unit entry
      uint64_t bits;
      uint32_t base;
      side.unit_entry(a.side1, b.unit, bits, base);
      const uint64_t ex = base + (uint32_t)__builtin_popcountll(bits & ((1ull << b.ul) - 1ull));
      uint32_t w[4], sh;
      side.exc_window(ex, w, sh);
      planes14_fields(w[0], w[1], w[2], w[3], sh, e, p0, p1, p2, sm);
    } else {
      e = r0 & 1023u;
      const uint32_t side = cw((r0 >> 10) & 0xFFFu);
      golay70_core(align(r1, r0, 22), align(r2, r1, 14), side, g70(e & 511u), h);
      return;
    }
  }
  const LdsEntry t = tab(e);
  planes_core(p0, p1, p2, sm, t.tlo, t.thi, h);
}

__device__ __forceinline__ LaneBlock lane_block(const GemvArgs& a, int64_t tile, int R_t, int64_t g,
                                                int rl, int cl) {
  LaneBlock b;
  const int C_g = (int)min((int64_t)a.C, a.nb - g * a.C);
  b.valid = rl < R_t && cl < C_g;
  b.ul = (uint32_t)(rl * C_g + cl);
  b.loff = b.ul * Stride<LEECH_PLANES14>::v;   // overwritten per layout by the caller
  b.tile = (int32_t)tile;
  b.unit = (int32_t)(tile * a.groups + g);
  b.ubase = tile * a.R * a.nb + g * R_t * a.C;
  return b;
}

// The LDS entries, built from the device table: one 16-byte load per entry.
__device__ __forceinline__ LdsEntry make_entry(const DevClass* tab, uint32_t e, float cen0,
                                               float cen1) {
  const u32x4a d = *(const u32x4a*)&tab[e & 511u];      // perm[8], inv_norm, info
  LdsEntry t;
  t.tlo = d.x;
  t.thi = d.y;
  t.factor = __builtin_bit_cast(float, (uint32_t)d.z) * ((e >> 9) ? cen1 : cen0) * kTwo24;
  t.nlev = d.w & 0xFFu;
  return t;
}

__device__ __forceinline__ G70Entry make_g70(const DevClass* tab, uint32_t c) {
  const u32x4a d = *(const u32x4a*)&tab[c];
  const u32x4a v = *((const u32x4a*)&tab[c] + 1);        // g70[8], g70abs[8]
  G70Entry t;
  t.alo = v.z;
  t.ahi = v.w;
  const uint32_t sg = (uint32_t)d.w >> 24;
  uint32_t slo = 0, shi = 0;
  for (int k = 0; k < 4; ++k) {
    slo |= ((sg >> k) & 1u) << (8 * k + 7);
    shi |= ((sg >> (k + 4)) & 1u) << (8 * k + 7);
  }
  t.slo = slo;
  t.shi = shi;
  return t;
}

// x of block j in the cores' pair order: three 16-byte loads, then pair k
// (coordinates pair_coords(k)) picked by one v_perm_b32 each.
struct XBlock {
  u32x4a v0, v1, v2;
};
__device__ __forceinline__ XBlock load_x_block(const uint16_t* xj) {
  const u32x4a* src = (const u32x4a*)xj;
  return XBlock{src[0], src[1], src[2]};
}
__device__ __forceinline__ void store_x_block(const XBlock& xb, uint32_t* dst) {
  const uint32_t w[12] = {xb.v0.x, xb.v0.y, xb.v0.z, xb.v0.w, xb.v1.x, xb.v1.y,
                          xb.v1.z, xb.v1.w, xb.v2.x, xb.v2.y, xb.v2.z, xb.v2.w};
  uint32_t o[12];
#pragma unroll
  for (int k = 0; k < 12; ++k) {
    int c0, c1;
    pair_coords(k, c0, c1);
    // low half: half c0 % 2 of word c0 / 2 (selector bytes 0..3 pick S1);
    // high half: half c1 % 2 of word c1 / 2 (bytes 4..7 pick S0)
    const uint32_t sel = (c0 & 1 ? 0x0302u : 0x0100u) | (c1 & 1 ? 0x07060000u : 0x05040000u);
    o[k] = perm(w[c1 >> 1], w[c0 >> 1], sel);
  }
  u32x4a* d = (u32x4a*)dst;
  d[0] = u32x4a{o[0], o[1], o[2], o[3]};
  d[1] = u32x4a{o[4], o[5], o[6], o[7]};
  d[2] = u32x4a{o[8], o[9], o[10], o[11]};
}

// ------------------------------------------------------------------- GEMV
template <int LAYOUT>
__global__ __launch_bounds__(kMaxWaves * 64) void gemv_kernel(GemvArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int64_t nb = a.nb;
  uint32_t* xs = (uint32_t*)smem;                                   // nb × 12 x pairs
  const size_t xbytes = (size_t)nb * 48;
  LdsEntry* ts = (LdsEntry*)(smem + xbytes);                         // 1024 entries
  const size_t tbytes = (LAYOUT == kNoWeights) ? 0 : 1024 * sizeof(LdsEntry);
  G70Entry* gs = (G70Entry*)(smem + xbytes + tbytes);                // Golay70: 512 entries
  uint32_t* cws = (uint32_t*)(smem + xbytes + tbytes + 512 * sizeof(G70Entry));  // 4096 words
  const size_t gbytes = (LAYOUT == LEECH_GOLAY70) ? 512 * sizeof(G70Entry) + 4096 * 4 : 0;
  constexpr bool kUnits = LAYOUT == LEECH_SLOT32 || LAYOUT == LEECH_GOLAY70;
  constexpr bool kExc = LAYOUT == LEECH_PLANES12X || LAYOUT == LEECH_GOLAY70;
  uint8_t* units_lds = smem + xbytes + tbytes + gbytes;             // groups × 16 B
  const size_t ubytes = kUnits ? (size_t)a.groups * kUnitEntryBytes : 0;
  uint8_t* exc_lds = units_lds + ubytes;                              // ≤ kExcLdsBytes
  const size_t ebytes = kExc ? kExcLdsBytes : 0;
  float* red = (float*)(exc_lds + ebytes);                          // waves × 64

  const int tid = threadIdx.x, nthr = blockDim.x;
  const int tile = (int)blockIdx.x;
  const int R_t = (int)min((int64_t)a.R, a.M - (int64_t)tile * a.R);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int rl = lane / a.C, cl = lane % a.C;
  const int groups = (int)a.groups, waves = a.waves;     // unit counts fit 32 bits
  // lane constants: position inside a full unit and inside the narrower last
  // one; a lane with no block there takes block 0 (in bounds) and is masked
  const int C_last = (int)(a.nb - (int64_t)(groups - 1) * a.C);
  const bool row_ok = rl < R_t, last_ok = row_ok && cl < C_last;
  const uint32_t ul_f = row_ok ? (uint32_t)(rl * a.C + cl) : 0u;
  const uint32_t ul_l = last_ok ? (uint32_t)(rl * C_last + cl) : 0u;
  const uint32_t lo_f = ul_f * Stride<LAYOUT>::v, lo_l = ul_l * Stride<LAYOUT>::v;
  const int64_t tile_base = (int64_t)tile * a.R * a.nb;
  // the block of this lane in unit g (g wave-uniform); past the last unit an
  // in-bounds stand-in with valid = false
  auto unit_block = [&](int g) -> LaneBlock {
    LaneBlock b;
    const bool beyond = g >= groups;
    g = beyond ? groups - 1 : g;
    const bool last = g == groups - 1;
    b.valid = !beyond && (last ? last_ok : row_ok);
    b.ul = last ? ul_l : ul_f;
    b.loff = last ? lo_l : lo_f;
    b.tile = tile;
    b.unit = tile * groups + g;
    b.ubase = tile_base + (int64_t)g * (R_t * a.C);
    return b;
  };

  // Side data of the tile: its unit entries (Slot32, Golay70) and the range of
  // its exception records (Planes12x, Golay70), copied to LDS below.
  const GlobalSide gside{&a};
  LdsSide side{&a, exc_lds, 0, false, units_lds, tile * groups, 0u};
  uint64_t exc_chunks = 0;
  if constexpr (kExc) {
    uint64_t e0, e1;
    if constexpr (LAYOUT == LEECH_PLANES12X) {
      e0 = ((const uint32_t*)a.side1)[tile];
      e1 = tile + 1 < a.tiles ? ((const uint32_t*)a.side1)[tile + 1] : a.n_exc;
      side.p12base = (uint32_t)e0;
    } else {
      uint64_t bits;
      uint32_t b0, b1 = 0;
      gside.unit_entry(a.side1, tile * groups, bits, b0);
      if (tile + 1 < a.tiles) gside.unit_entry(a.side1, (tile + 1) * groups, bits, b1);
      e0 = b0;
      e1 = tile + 1 < a.tiles ? b1 : a.n_exc;
    }
    side.exc_start = (e0 * kPlanes14Bytes) & ~15ull;
    // the window of record e is 16 bytes from (14·e) & ~3, so the tile's
    // windows end by 14·e1 + 2; rounded up to 16 this stays inside side0's
    // 16 bytes of padding
    const uint64_t end = e1 * kPlanes14Bytes + 2;
    exc_chunks = (end - side.exc_start + 15) / 16;
    side.exc_in_lds = exc_chunks * 16 <= (uint64_t)kExcLdsBytes;
  }

  // Prologue, ordered for the in-order load counter: first the L2-resident
  // staging loads (x blocks, class table, side data), then the units' record
  // loads, then the LDS writes, which wait only for the older staging loads.
  constexpr int kXPer = 2, kTPer = 2;          // staged items per thread held in registers
  constexpr int kEPer = kExcLdsBytes / 16 / 512, kUPer = 2;
  // rare overflow first (nb > kXPer·threads, or fewer threads than table
  // entries / kTPer): loads of unknown count here, before the ordered ones
  for (int64_t j = tid + (int64_t)kXPer * nthr; j < nb; j += nthr)
    store_x_block(load_x_block(a.x + 24 * j), xs + 12 * j);
  if constexpr (LAYOUT != kNoWeights)
    for (int e = tid + kTPer * nthr; e < 1024; e += nthr)
      ts[e] = make_entry(a.table, (uint32_t)e, a.cen0, a.cen1);
  if constexpr (LAYOUT == LEECH_GOLAY70) {
    for (int c = tid; c < 512; c += nthr) gs[c] = make_g70(a.table, (uint32_t)c);
    for (int k = tid; k < 1024; k += nthr) ((u32x4a*)cws)[k] = ((const u32x4a*)a.codewords)[k];
  }
  const uint8_t* side_units = LAYOUT == LEECH_SLOT32 ? a.side0 : a.side1;
  if constexpr (kUnits)
    for (int u = tid + kUPer * nthr; u < groups; u += nthr)
      ((u32x4a*)units_lds)[u] = ((const u32x4a*)side_units)[tile * groups + u];
  if constexpr (kExc)
    if (side.exc_in_lds)
      for (int64_t c = tid + (int64_t)kEPer * nthr; c < (int64_t)exc_chunks; c += nthr)
        ((u32x4a*)exc_lds)[c] = ((const u32x4a*)(a.side0 + side.exc_start))[c];
  XBlock xr[kXPer];
#pragma unroll
  for (int q = 0; q < kXPer; ++q) {
    const int64_t j = min(tid + (int64_t)q * nthr, nb - 1);    // clamped: loads stay unconditional
    xr[q] = load_x_block(a.x + 24 * j);
  }
  u32x4a tr[kTPer];
  if constexpr (LAYOUT != kNoWeights) {
#pragma unroll
    for (int q = 0; q < kTPer; ++q) tr[q] = *(const u32x4a*)&a.table[(tid + q * nthr) & 511];
  }
  u32x4a ur[kUPer], er[kEPer];
  if constexpr (kUnits) {
#pragma unroll
    for (int q = 0; q < kUPer; ++q)
      ur[q] = ((const u32x4a*)side_units)[tile * groups + min(tid + q * nthr, groups - 1)];
  }
  if constexpr (kExc) {
    if (side.exc_in_lds) {
#pragma unroll
      for (int q = 0; q < kEPer; ++q)
        er[q] = ((const u32x4a*)(a.side0 + side.exc_start))[min((int64_t)(tid + q * nthr),
                                                                  (int64_t)exc_chunks - 1)];
    }
  }
  Pref pf[kPrefetch];
#pragma unroll
  for (int d = 0; d < kPrefetch; ++d) {
    pf[d] = load_block<LAYOUT>(a, unit_block(wave + d * waves), gside);
    __builtin_amdgcn_sched_barrier(0);    // keep the slots' loads in slot order
  }
#pragma unroll
  for (int q = 0; q < kXPer; ++q) {
    const int64_t j = tid + (int64_t)q * nthr;
    if (j < nb) store_x_block(xr[q], xs + 12 * j);
  }
  if constexpr (LAYOUT != kNoWeights) {
#pragma unroll
    for (int q = 0; q < kTPer; ++q) {
      const int e = tid + q * nthr;
      if (e < 1024) {
        LdsEntry t;
        t.tlo = tr[q].x;
        t.thi = tr[q].y;
        t.factor = __builtin_bit_cast(float, (uint32_t)tr[q].z) * ((e >> 9) ? a.cen1 : a.cen0) * kTwo24;
        t.nlev = tr[q].w & 0xFFu;
        ts[e] = t;
      }
    }
  }
  if constexpr (kUnits) {
#pragma unroll
    for (int q = 0; q < kUPer; ++q)
      if (tid + q * nthr < groups) ((u32x4a*)units_lds)[tid + q * nthr] = ur[q];
  }
  if constexpr (kExc) {
    if (side.exc_in_lds) {
#pragma unroll
      for (int q = 0; q < kEPer; ++q)
        if (tid + q * nthr < (int64_t)exc_chunks) ((u32x4a*)exc_lds)[tid + q * nthr] = er[q];
    }
  }
  __syncthreads();

  auto tab = [&](uint32_t e) -> LdsEntry { return ts[e]; };
  auto g70 = [&](uint32_t c) -> G70Entry { return gs[c]; };
  auto cw = [&](uint32_t r) -> uint32_t { return cws[r]; };
  float acc = 0.0f;
  // One unit: decode slot pf[d] for unit g and accumulate.
  // Lanes without a block decode their in-bounds stand-in and add 0.
  auto process = [&](const Pref& p, int g) {
    const LaneBlock b = unit_block(g);
    const int j = g * a.C + (b.valid ? cl : 0);
    const u32x4a* xp = (const u32x4a*)(xs + 12 * j);
    const u32x4a x0 = xp[0], x1 = xp[1], x2 = xp[2];
    const uint32_t xw[12] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w,
                             x2.x, x2.y, x2.z, x2.w};
    if constexpr (LAYOUT == kNoWeights) {
      float s = 0.0f;
#pragma unroll
      for (int k = 0; k < 12; ++k) s = __builtin_amdgcn_fdot2(as_h2(0x3C003C00u), as_h2(xw[k]), s, false);
      acc += b.valid ? s : 0.0f;
    } else {
      uint32_t h[12], e;
      decode_block<LAYOUT>(a, b, p, tab, g70, cw, side, h, e);
      float s = 0.0f;
#pragma unroll
      for (int k = 0; k < 12; ++k) s = __builtin_amdgcn_fdot2(as_h2(h[k]), as_h2(xw[k]), s, false);
      const float f = half_bits_to_float(p.scale) * ts[e].factor;
      acc = __builtin_fmaf(s, b.valid ? f : 0.0f, acc);
    }
  };
  const int units = (groups - wave + waves - 1) / waves;   // this wave's units
  int done = 0;
  // Full rounds: consume every slot, refilling each with the unit kPrefetch
  // steps ahead (past the wave's last unit the refill is an in-bounds
  // stand-in).  Decoding before refilling lets the refill reuse the slot's
  // registers: a refill into fresh registers would be moved back at the loop
  // latch, and moving a register with a load in flight waits for every
  // outstanding load.
  for (; units - done > kPrefetch; done += kPrefetch) {
#pragma unroll
    for (int d = 0; d < kPrefetch; ++d) {
      const int g = wave + (done + d) * waves;
      process(pf[d], g);
      pf[d] = load_block<LAYOUT>(a, unit_block(g + kPrefetch * waves), side);
    }
  }
  // the last ≤ kPrefetch units are in flight: straight-line, no refills
#pragma unroll
  for (int d = 0; d < kPrefetch; ++d)
    if (d < units - done) process(pf[d], wave + (done + d) * waves);
  for (int off = 1; off < a.C; off <<= 1) acc += __shfl_xor(acc, off);
  if (cl == 0 && rl < R_t) red[wave * 64 + rl] = acc;
  __syncthreads();
  if (tid < R_t) {
    float y = 0.0f;
    for (int w = 0; w < a.waves; ++w) y += red[w * 64 + tid];
    a.y[(int64_t)tile * a.R + tid] = y;
  }
}

// --------------------------------------------------------- decode export
// One thread per block, with the GEMV's own load and decode functions; the
// binary16 pairs are turned back into integer coordinates (|z| in the low
// byte of each half, the sign in its bit 15).
template <int LAYOUT>
__global__ __launch_bounds__(256) void decode_kernel(GemvArgs a, int8_t* zout, uint16_t* cout,
                                                     uint8_t* gout) {
  const int64_t bi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (bi >= a.M * a.nb) return;
  const int64_t r = bi / a.nb, j = bi % a.nb;
  const int64_t tile = r / a.R, g = j / a.C;
  const int R_t = (int)min((int64_t)a.R, a.M - tile * a.R);
  LaneBlock b = lane_block(a, tile, R_t, g, (int)(r % a.R), (int)(j % a.C));
  b.loff = b.ul * Stride<LAYOUT>::v;
  const GlobalSide side{&a};
  const Pref p = load_block<LAYOUT>(a, b, side);
  auto tab = [&](uint32_t e) -> LdsEntry { return make_entry(a.table, e, 1.0f, 1.0f); };
  auto g70 = [&](uint32_t c) -> G70Entry { return make_g70(a.table, c); };
  auto cw = [&](uint32_t rk) -> uint32_t { return a.codewords[rk]; };
  uint32_t h[12], e;
  decode_block<LAYOUT>(a, b, p, tab, g70, cw, side, h, e);
  int8_t z[kDim];
#pragma unroll
  for (int k = 0; k < 12; ++k) {
    int c0, c1;
    pair_coords(k, c0, c1);
    const int m0 = (int)(h[k] & 0xFFu), m1 = (int)((h[k] >> 16) & 0xFFu);
    z[c0] = (int8_t)(((h[k] >> 15) & 1u) ? -m0 : m0);
    z[c1] = (int8_t)(((h[k] >> 31) & 1u) ? -m1 : m1);
  }
  if (zout) {
    uint32_t* zo = (uint32_t*)(zout + bi * kDim);
#pragma unroll
    for (int q = 0; q < 6; ++q)
      zo[q] = (uint32_t)(uint8_t)z[4 * q] | (uint32_t)(uint8_t)z[4 * q + 1] << 8 |
              (uint32_t)(uint8_t)z[4 * q + 2] << 16 | (uint32_t)(uint8_t)z[4 * q + 3] << 24;
  }
  if (cout) cout[bi] = (uint16_t)(e & 511u);
  if (gout) gout[bi] = (uint8_t)(e >> 9);
}

// ------------------------------------------------------ FP16 GEMV control
// One wavefront per row; lanes stream 16-byte chunks of the row (1 KiB per
// wavefront load); x staged in LDS; f32 accumulation with v_dot2_f32_f16.
__global__ __launch_bounds__(512) void fp16_gemv_kernel(const uint16_t* __restrict__ W,
                                                        const uint16_t* __restrict__ x,
                                                        float* __restrict__ y, int64_t M,
                                                        int64_t K) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int64_t K8 = K / 8;
  u32x4a* xs = (u32x4a*)smem;
  for (int64_t k = threadIdx.x; k < K8; k += blockDim.x) xs[k] = ((const u32x4a*)x)[k];
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x >> 6) + wave;
  if (row >= M) return;
  const u32x4a* wr = (const u32x4a*)(W + row * K);
  float acc = 0.0f;
  for (int64_t c = lane; c < K8; c += 64) {
    u32x4a w = wr[c];
    u32x4a xv = xs[c];
    acc = __builtin_amdgcn_fdot2(as_h2(w.x), as_h2(xv.x), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.y), as_h2(xv.y), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.z), as_h2(xv.z), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.w), as_h2(xv.w), acc, false);
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) y[row] = acc;
}

// ------------------------------------------------------------- launching
static int hip_fail(const char* what, hipError_t e) {
  return set_error(LEECH_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Waves per workgroup: each wave walks every waves-th unit of the tile.  The
// summation order depends on it, so it is a function of the shape only (the
// LEECH_WAVES environment variable overrides the cap, for tuning).
static int waves_for(int64_t groups) {
  static const int cap = [] {
    const char* v = std::getenv("LEECH_WAVES");
    const int w = v ? std::atoi(v) : 0;
    return (w >= 1 && w <= kMaxWaves) ? w : kMaxWaves;
  }();
  return (int)std::max<int64_t>(1, std::min<int64_t>(cap, groups));
}

static int check_desc_device(const leech_layout_desc* d) {
  if (!d) return set_error(LEECH_E_ARG, "desc is NULL");
  if (d->M <= 0 || d->Kpad <= 0 || d->Kpad % kDim || d->nb != d->Kpad / kDim)
    return set_error(LEECH_E_SHAPE, "descriptor shape is not valid");
  if (d->lane_cols != choose_lane_cols(d->M))
    return set_error(LEECH_E_SHAPE, "descriptor lane_cols does not match its M");
  return LEECH_OK;
}

static GemvArgs make_args(const leech_layout_desc* d) {
  GemvArgs a;
  std::memset(&a, 0, sizeof a);
  a.M = d->M;
  a.nb = d->nb;
  a.C = d->lane_cols;
  a.R = kWave / d->lane_cols;
  a.groups = (d->nb + a.C - 1) / a.C;
  a.waves = waves_for(a.groups);
  a.tiles = (d->M + a.R - 1) / a.R;
  a.n_exc = d->n_exceptions;
  return a;
}

template <int LAYOUT>
static size_t gemv_lds_bytes(const GemvArgs& a) {
  const bool units = LAYOUT == LEECH_SLOT32 || LAYOUT == LEECH_GOLAY70;
  const bool exc = LAYOUT == LEECH_PLANES12X || LAYOUT == LEECH_GOLAY70;
  return (size_t)a.nb * 48 + (LAYOUT == kNoWeights ? 0 : 1024 * sizeof(LdsEntry)) +
         (LAYOUT == LEECH_GOLAY70 ? 512 * sizeof(G70Entry) + 4096 * 4 : 0) +
         (units ? (size_t)a.groups * kUnitEntryBytes : 0) + (exc ? kExcLdsBytes : 0) +
         (size_t)a.waves * 64 * 4;
}

template <int LAYOUT>
static int launch_gemv(const GemvArgs& a, hipStream_t st) {
  const size_t shmem = gemv_lds_bytes<LAYOUT>(a);
  if (shmem > 160 * 1024)
    return set_error(LEECH_E_SHAPE, "Kpad too large for the LDS-staged activation");
  if (shmem > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)gemv_kernel<LAYOUT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return hip_fail("hipFuncSetAttribute", e);
  }
  const int64_t tiles = (a.M + a.R - 1) / a.R;
  hipLaunchKernelGGL(gemv_kernel<LAYOUT>, dim3((unsigned)tiles), dim3(64 * a.waves), shmem, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("gemv launch", e);
  return LEECH_OK;
}

template <int LAYOUT>
static int launch_decode(const GemvArgs& a, int8_t* z, uint16_t* c, uint8_t* g, hipStream_t st) {
  const int64_t n = a.M * a.nb;
  hipLaunchKernelGGL(decode_kernel<LAYOUT>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     a, z, c, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("decode launch", e);
  return LEECH_OK;
}

}  // namespace leech

using namespace leech;

extern "C" {

int leech_gemv(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
               const void* d_side1, const void* d_class_table, const void* d_codewords,
               const uint16_t* d_scale, const float centroid[2], const uint16_t* d_x,
               float* d_y, void* stream) {
  clear_error();
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_main || !d_class_table || !d_scale || !centroid || !d_x || !d_y)
    return set_error(LEECH_E_ARG, "NULL argument");
  if ((desc->side_bytes[0] && !d_side0) || (desc->side_bytes[1] && !d_side1))
    return set_error(LEECH_E_ARG, "layout needs its side streams");
  if (desc->layout == LEECH_GOLAY70 && !d_codewords)
    return set_error(LEECH_E_ARG, "GOLAY70 needs the codeword table");
  if (((uintptr_t)d_x & 15) || ((uintptr_t)d_main & 3) || ((uintptr_t)d_class_table & 15) ||
      ((uintptr_t)d_codewords & 15) || ((uintptr_t)d_side0 & 3) || ((uintptr_t)d_side1 & 7))
    return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a = make_args(desc);
  a.main = (const uint8_t*)d_main;
  a.side0 = (const uint8_t*)d_side0;
  a.side1 = (const uint8_t*)d_side1;
  a.table = (const DevClass*)d_class_table;
  a.codewords = (const uint32_t*)d_codewords;
  a.scale = d_scale;
  a.x = d_x;
  a.y = d_y;
  a.cen0 = centroid[0];
  a.cen1 = centroid[1];
  hipStream_t st = (hipStream_t)stream;
  switch (desc->layout) {
    case LEECH_SLOT32: return launch_gemv<LEECH_SLOT32>(a, st);
    case LEECH_PLANES14: return launch_gemv<LEECH_PLANES14>(a, st);
    case LEECH_PLANES12X: return launch_gemv<LEECH_PLANES12X>(a, st);
    case LEECH_GOLAY70: return launch_gemv<LEECH_GOLAY70>(a, st);
    default: return set_error(LEECH_E_LAYOUT, "unknown layout");
  }
}

int leech_decode_blocks(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                        const void* d_side1, const void* d_class_table,
                        const void* d_codewords, int8_t* d_z, uint16_t* d_class_id,
                        uint8_t* d_gain_bit, void* stream) {
  clear_error();
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_main || !d_class_table) return set_error(LEECH_E_ARG, "NULL argument");
  if ((desc->side_bytes[0] && !d_side0) || (desc->side_bytes[1] && !d_side1))
    return set_error(LEECH_E_ARG, "layout needs its side streams");
  if (desc->layout == LEECH_GOLAY70 && !d_codewords)
    return set_error(LEECH_E_ARG, "GOLAY70 needs the codeword table");
  if (((uintptr_t)d_z & 3) || ((uintptr_t)d_main & 3) || ((uintptr_t)d_side1 & 7))
    return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a = make_args(desc);
  a.main = (const uint8_t*)d_main;
  a.side0 = (const uint8_t*)d_side0;
  a.side1 = (const uint8_t*)d_side1;
  a.table = (const DevClass*)d_class_table;
  a.codewords = (const uint32_t*)d_codewords;
  hipStream_t st = (hipStream_t)stream;
  switch (desc->layout) {
    case LEECH_SLOT32: return launch_decode<LEECH_SLOT32>(a, d_z, d_class_id, d_gain_bit, st);
    case LEECH_PLANES14: return launch_decode<LEECH_PLANES14>(a, d_z, d_class_id, d_gain_bit, st);
    case LEECH_PLANES12X: return launch_decode<LEECH_PLANES12X>(a, d_z, d_class_id, d_gain_bit, st);
    case LEECH_GOLAY70: return launch_decode<LEECH_GOLAY70>(a, d_z, d_class_id, d_gain_bit, st);
    default: return set_error(LEECH_E_LAYOUT, "unknown layout");
  }
}

int leech_fp16_gemv_ref(int64_t M, int64_t K, const uint16_t* d_W, const uint16_t* d_x,
                        float* d_y, void* stream) {
  clear_error();
  if (!d_W || !d_x || !d_y) return set_error(LEECH_E_ARG, "NULL argument");
  if (M <= 0 || K <= 0 || K % 8) return set_error(LEECH_E_SHAPE, "need M > 0, K > 0, K % 8 == 0");
  if (((uintptr_t)d_W & 15) || ((uintptr_t)d_x & 15))
    return set_error(LEECH_E_ARG, "W and x must be 16-byte aligned");
  size_t shmem = (size_t)K * 2;
  if (shmem > 160 * 1024) return set_error(LEECH_E_SHAPE, "K too large for the LDS-staged x");
  if (shmem > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)fp16_gemv_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return hip_fail("hipFuncSetAttribute", e);
  }
  const int waves = 8;
  hipLaunchKernelGGL(fp16_gemv_kernel, dim3((unsigned)((M + waves - 1) / waves)), dim3(64 * waves),
                     shmem, (hipStream_t)stream, d_W, d_x, d_y, M, K);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("fp16 gemv launch", e);
  return LEECH_OK;
}

int leech_noweights_ctrl(const leech_layout_desc* desc, const uint16_t* d_x, float* d_y,
                         void* stream) {
  clear_error();
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_x || !d_y) return set_error(LEECH_E_ARG, "NULL argument");
  if ((uintptr_t)d_x & 15) return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a = make_args(desc);
  a.x = d_x;
  a.y = d_y;
  return launch_gemv<kNoWeights>(a, (hipStream_t)stream);
}

}  // extern "C"
