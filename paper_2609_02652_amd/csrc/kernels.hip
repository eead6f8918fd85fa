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
// Addressing.  Records and scales are read with raw buffer loads: the
// workgroup's buffer descriptor starts at its tile, the unit's offset is a
// scalar, and the lane's offset inside the unit is a per-lane constant, so a
// step spends no vector instructions on addresses.  Every unit of a tile but
// the last (narrower) column group is full width, so the pipelined loop uses
// one set of lane constants and needs no per-lane masking: lanes of rows past
// the matrix decode a stand-in and their sums are never written.  The last
// column group is loaded in the prologue and added by one wave at the end,
// with lanes past the last column reading zero x.
//
// Decode.  The paper's per-coordinate predicated tree is replaced, since the
// MI355X has about an order of magnitude less VALU issue per HBM byte than the
// paper's GPU.  Every coordinate's level code (level + 1) and sign become one
// byte-permute selector per pair of coordinates; a v_perm_b32 byte lookup in
// the class's 8-byte table then yields two binary16 values at once, each the
// coordinate's magnitude |z| as a subnormal (|z|·2^-24, exact) with the sign
// in bit 15.  Planes14 records hold the codes and signs already in pair order,
// so a selector is one rotate and one mask of a record word; the layouts that
// hold plain planes (p0, p1, p2 and the inverted sign mask) first transpose
// them 4×4 inside every nibble with eight v_bfi_b32 and gather the pairs.
// v_dot2_f32_f16 multiplies the pairs with x exactly and sums in f32; the
// block's factor 2^24 · scale · centroid[gain] / (4√m) is applied once per
// block.

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <string>
#include <type_traits>

#include "leech_internal.h"

namespace leech {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4a __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2a __attribute__((ext_vector_type(2)));
typedef float f32x4a __attribute__((ext_vector_type(4)));

constexpr int kNoWeights = 99;   // layout id of the no-weights control
// Prologue modes of the GEMV (the host picks one from the units each wave
// streams, measured per shape): every wave keeps kPrefetch units in flight;
// the first pro_first(PRO) of them are requested before the staging barrier
// and the rest one per step of the first round, so that the barrier is not
// held up behind a burst of record requests that the CU's load path can only
// accept one after the other.
//   PRO 0: all 8 before the barrier (long tiles: the deepest early burst);
//   PRO 1: 3 of 8 before it;   PRO 2: 2 of 6 (waves with ≤ 6 units).
__host__ __device__ constexpr int pro_prefetch(int pro) { return pro == 2 ? 6 : 8; }
__host__ __device__ constexpr int pro_first(int pro) { return pro == 0 ? 8 : pro == 1 ? 3 : 2; }
constexpr float kTwo24 = 16777216.0f;
// Waves per GEMV workgroup, at most: 8 waves leave each lane up to 256 VGPRs,
// so the eight prefetch slots and the exception-path decode stay in registers.
constexpr int kMaxWaves = 8;
// Exception entries a thread holds in registers from the prologue
constexpr int kExcPrefetch = 4;
constexpr int kTableBytes = 1024 * 16;    // LDS class-table entries (class | gain << 9)
// Raw buffer descriptor, word 3, for the gfx9 family (32-bit elements, no
// swizzle); loads carry the non-temporal hint: records and scales are read once.
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kStreamed = 2;

template <int LAYOUT> struct Stride { static constexpr uint32_t v = 0; };
template <> struct Stride<LEECH_PLANES14> { static constexpr uint32_t v = kPlanes14Bytes; };
template <> struct Stride<LEECH_PLANES12X> { static constexpr uint32_t v = kPlanes12Bytes; };
template <> struct Stride<LEECH_GOLAY70> { static constexpr uint32_t v = kGolay70Bytes; };

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
  uint64_t main_bytes;
  // row groups with their own gain centroids (0: one group, cen0/cen1)
  int ngroups;
  int64_t grp_end[LEECH_MAX_GROUPS];      // first row past each group
  float grp_cen[LEECH_MAX_GROUPS][2];
  int tab2;                     // 1: some tile holds rows of two groups (second LDS table)
  uint32_t tab_bytes;           // bytes of one LDS table copy: 1024 class entries (Planes12x,
                                // exceptions kept: and the tile's exception entries)
  uint32_t tile_exc_max;        // most exceptions in one tile
  int inline_exc;               // Planes12x, Golay70: 1 = exceptions decoded in the loop
  // batched launches: activation b at x + b·ldx, output b at y + b·ldy, for
  // b < nbatch (≤ the kernel's batch width)
  int64_t ldx, ldy;
  int nbatch;
  // rotated launches: the activation is rotated in the prologue from the raw
  // binary16 xraw [K] and the ±1 signs (NULL: all +1), blocks of 2^rot_k
  const uint16_t* xraw;
  const int8_t* signs;
  int64_t K;
  int rot_k;
  float rot_norm;
  // phase stamps (measurement launches): kPhaseStamps u64 per workgroup
  uint64_t* stamps;
};
// Phase stamps of a measurement launch, per workgroup, in the 100 MHz
// real-time counter: 0 the first wave's start, 1 the first wave past the
// staging barrier, 2 + w wave w's last unit decoded, 10 the first wave's
// last y store issued.
constexpr int kPhaseStamps = 11;

// Where side data comes from: global memory (verification decode, and the
// GEMV prologue before LDS is written), or the tile's copy in LDS.  Slot32
// reads its per-unit side entries (record offsets); Planes12x and Golay70 their
// tiles' exception lists (a u32 first index per tile in side1, 16-byte entries
// in side0).
struct GlobalSide {
  const GemvArgs* a;
  __device__ __forceinline__ uint32_t exc_base(int tile) const {
    return ((const uint32_t*)a->side1)[tile];
  }
  __device__ __forceinline__ void unit_entry(const uint8_t* side, int unit, uint64_t& bits,
                                             uint32_t& base) const {
    const uint8_t* ent = side + (int64_t)unit * kUnitEntryBytes;
    bits = *(const uint64_t*)ent;
    base = *(const uint32_t*)(ent + 8);
  }
  // exception entry ex: the exact Planes14 record in its first 14 bytes
  __device__ __forceinline__ u32x4a exc_entry(uint64_t ex) const {
    return *(const u32x4a*)(a->side0 + ex * kExcEntryBytes);
  }
};
struct LdsSide {
  const GemvArgs* a;
  const uint8_t* units;      // LDS copy of the tile's unit entries (Slot32)
  int unit0;                 // first unit id of the tile
  uint32_t excbase;          // first exception index of the tile
  __device__ __forceinline__ uint32_t exc_base(int) const { return excbase; }
  __device__ __forceinline__ void unit_entry(const uint8_t*, int unit, uint64_t& bits,
                                             uint32_t& base) const {
    const uint8_t* ent = units + (unit - unit0) * kUnitEntryBytes;
    bits = *(const uint64_t*)ent;
    base = *(const uint32_t*)(ent + 8);
  }
  __device__ __forceinline__ u32x4a exc_entry(uint64_t ex) const {
    return *(const u32x4a*)(a->side0 + ex * kExcEntryBytes);
  }
};

// Per-(class, gain) entry staged in LDS at byte (class | gain << 9) · 16.
struct LdsEntry {
  uint32_t tlo, thi;    // v_perm table (DevClass::perm; Planes12x: see p12_core;
                        // Golay70: see golay70_core)
  float factor;         // 2^24 · centroid[gain] / (4√m)
  uint32_t aux;         // Slot32: level count; Planes12x, Golay70: f32 added to the
                        // block's sum × factor (0, or an exception's kept contribution)
};
static_assert(sizeof(LdsEntry) * 1024 == kTableBytes, "table entries are 16 bytes");
// Golay70 in LDS: the generator table, and each class's Planes14 table (for
// an exception's exact record)
constexpr int kG70LdsBytes = 128 * 4 + 512 * 8;

__device__ __forceinline__ uint32_t align(uint32_t hi, uint32_t lo, uint32_t s) {
  return __builtin_amdgcn_alignbit(hi, lo, s);
}
__device__ __forceinline__ uint32_t perm(uint32_t s0, uint32_t s1, uint32_t sel) {
  return __builtin_amdgcn_perm(s0, s1, sel);
}
// (m & a) | (~m & b) as one v_bfi_b32: left to itself the compiler splits the
// nibble transpose's bit-field inserts into and / and_or pairs.
__device__ __forceinline__ uint32_t bfi(uint32_t m, uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "s"(m), "v"(a), "v"(b));
  return r;
}
// (s & m) | c as one v_and_or_b32, m from an SGPR and c from a VGPR: left to
// itself the compiler splits it into a v_and and a v_or with literals (a
// gfx9 VOP3 instruction takes no literal and one SGPR at most).
__device__ __forceinline__ uint32_t and_or(uint32_t s, uint32_t m, uint32_t c) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(s), "s"(m), "v"(c));
  return r;
}
// (a << 4) + b as one v_lshl_add_u32.
__device__ __forceinline__ uint32_t lshl4_add(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_lshl_add_u32 %0, %1, 4, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// Reinterpret a 32-bit word as two binary16 values.  Takes the word by value:
// applying __builtin_bit_cast directly to an ext_vector element (w.y) reads
// element 0 with this compiler, so vector elements go through this function.
__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

__device__ __forceinline__ _Float16 as_half(uint32_t h) {
  return __builtin_bit_cast(_Float16, (uint16_t)h);
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

// Nibble core: the four nibble words of a block (nibble g of n[r] holds the
// level code c = level + 1 of coordinate 4g + r in bits 0..2 and its
// non-negative bit in bit 3) -> 12 binary16 pairs; pair 3r + k of h[] covers
// the coordinates listed by pair_sources.  Selector byte for the low half: the
// code (table bytes 1..5 hold |z| of levels 0..4); for the high half: 0 (table
// byte 0 = 0x80) when negative, 8 when not (v_perm's selector 8 replicates bit
// 7 of table byte 1, a magnitude below 0x80, giving 0x00).
__device__ __forceinline__ void nibble_core(const uint32_t n[4], uint32_t tlo, uint32_t thi,
                                            uint32_t h[12]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    uint32_t s[3];
    pair_sources(n[r], s);
#pragma unroll
    for (int k = 0; k < 3; ++k) h[3 * r + k] = perm(thi, tlo, s[k] & 0x08070807u);
  }
}
// Planes core (Slot32 and Planes12x records): the bit planes of a block (p0,
// p1, p2 the bits of each coordinate's level code, pos its non-negative bit),
// transposed to nibbles -> 12 binary16 pairs.
__device__ __forceinline__ void planes_core(uint32_t p0, uint32_t p1, uint32_t p2, uint32_t pos,
                                            uint32_t tlo, uint32_t thi, uint32_t h[12]) {
  uint32_t n[4];
  nibble_transpose(p0, p1, p2, pos, n);
  nibble_core(n, tlo, thi, h);
}

// Golay70 core: nibble (c0, c1, side, 0) -> index j = side·4 + code of a
// coordinate; the class's 8-byte table holds T[j] = |value| | (value < 0) << 7.
// pair_sources puts each coordinate's nibble in two adjacent selector bytes,
// so one byte permute gives T[j] in both bytes of its binary16 half, and the
// mask 0x807F807F keeps the magnitude in the low byte and the sign in the high.
__device__ __forceinline__ void golay70_core(uint32_t c0, uint32_t c1, uint32_t side,
                                             uint32_t tlo, uint32_t thi, uint32_t h[12]) {
  uint32_t n[4];
  nibble_transpose(c0, c1, side, 0u, n);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    uint32_t s[3];
    pair_sources(n[r], s);
#pragma unroll
    for (int k = 0; k < 3; ++k)
      h[3 * r + k] = perm(thi, tlo, s[k] & 0x07070707u) & 0x807F807Fu;
  }
}
// The Golay70 table of a class from the second half of its device record
// (signed values and magnitudes at side·4 + code).
__device__ __forceinline__ void g70_table(const u32x4a& v, uint32_t& tlo, uint32_t& thi) {
  tlo = (uint32_t)v.z | ((uint32_t)v.x & 0x80808080u);
  thi = (uint32_t)v.w | ((uint32_t)v.y & 0x80808080u);
}

// Coordinates of pair k of h[] (and of the staged x pairs).
__host__ __device__ constexpr void pair_coords(int k, int& c0, int& c1) {
  const int r = k / 3, m = k % 3;
  c0 = m == 0 ? r : (m == 1 ? 4 + r : 8 + r);
  c1 = m == 0 ? 16 + r : (m == 1 ? 20 + r : 12 + r);
}
// The Planes14 record stores its pairs in the host's kPairCoords order, which
// must be this one.
__host__ __device__ constexpr bool pair_order_matches_records() {
  for (int k = 0; k < 12; ++k) {
    int c0 = 0, c1 = 0;
    pair_coords(k, c0, c1);
    if (c0 != kPairCoords[k][0] || c1 != kPairCoords[k][1]) return false;
  }
  return true;
}
static_assert(pair_order_matches_records(), "pair order of the kernels and the records");

// ---------------------------------------------------------- per-block reads
// A lane's place in a unit: its position ul (0 for a lane without a block,
// which then reads block 0 as a stand-in) and, for the fixed-stride layouts,
// the record window: a 4-aligned byte offset from the unit's base and the
// record's bit offset sh inside it.  esh is the funnel-shift amount that brings
// a Planes14 record's class|gain field to bits 4..13 of word 3 (entry · 16).
struct Lane {
  uint32_t ul;
  uint32_t rec;
  uint32_t sh;
  uint32_t esh;
  bool own;         // the lane holds a block of its own (not a stand-in)
};
// u: the unit base's byte offset modulo 4
__device__ __forceinline__ Lane lane_place(uint32_t ul, uint32_t stride, uint32_t u,
                                           bool own = true) {
  const uint32_t off = ul * stride + u;
  const uint32_t sh = (off & 3u) * 8u;
  return Lane{ul, off & ~3u, sh, (sh + 28u) & 31u, own};
}

// Words a lane prefetches for one block.
struct Pref {
  uint32_t w0, w1, w2, w3, w4;
  uint32_t scale;
  uint32_t sh, esh;
};

// Planes14 record in the four-word window whose record starts at bit sh (0
// or 16): each pair word starts on a 32-bit boundary of the record, so one
// funnel shift each gives it; e16 = (class | gain << 9)·16, the entry's LDS
// byte address.  Pair q = 4w + k of word w is its rotation by 4k masked with
// 0x08070807, which is already the byte-permute selector of the pair's two
// binary16 values (the store order of the record): no transpose, no pair
// gathering.
__device__ __forceinline__ void p14_record(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                           uint32_t sh, uint32_t esh, uint32_t W[3],
                                           uint32_t& e16) {
  W[0] = align(w1, w0, sh);
  W[1] = align(w2, w1, sh);
  W[2] = align(w3, w2, sh);
  e16 = align(w3, w3, esh) & 0x3FF0u;
}
__device__ __forceinline__ void p14_core(const uint32_t W[3], uint32_t tlo, uint32_t thi,
                                         uint32_t h[12]) {
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t s = k ? align(W[w], W[w], 4 * k) : W[w];
      h[4 * w + k] = perm(thi, tlo, s & 0x08070807u);
    }
}

// Planes12x core: the 12 pair selector words taken straight from the
// record's words (one funnel shift or rotation each, kP12Sel), each masked to
// its pair's level and non-negative bits and pointed at the table's
// magnitude bytes.  The 8-byte table is 0x80 (the binary16 sign byte), three
// zero bytes, then mags = |z| of levels 0..3: the low half's selector is
// 4 + level, the high half's 0 (negative: 0x80) or 1, 2 or 8 (0x00).
__device__ __forceinline__ void p12_core(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t mags,
                                         uint32_t h[12]) {
  const uint32_t w[4] = {w0, w1, w2, 0u};
#pragma unroll
  for (int q = 0; q < 12; ++q) {
    const P12Sel d = kP12Sel[q];
    const uint32_t s = d.rot ? align(w[d.word], w[d.word], d.shift)
                             : align(w[d.word + 1], w[d.word], d.shift);
    const uint32_t m = 0x00030003u | 1u << (8 + d.k) | 1u << (24 + d.l);
    h[q] = perm(mags, 0x80u, and_or(s, m, 0x00040004u));
  }
}

// Decode one block into 12 binary16 pairs and its table entry's byte address.
// tab(e16) returns the LdsEntry at e16 in the layout's own table arrangement
// and tab14(e16) one whose tlo/thi are the class's Planes14 table (for an
// exception's exact record); cw(message) is the Golay codeword of a message.
// te receives the entry the block's sum is scaled with.
template <int LAYOUT, class TAB, class TAB14, class CW, class SIDE>
__device__ __forceinline__ void decode_block(const Pref& p, int tile, TAB tab, TAB14 tab14, CW cw,
                                             const SIDE& side, uint32_t h[12], uint32_t& e16,
                                             LdsEntry& te) {
  uint32_t p0 = 0, p1 = 0, p2 = 0, pos = 0;
  // a Planes14 record (the layout's own, or an exception's exact record)
  auto planes14 = [&](uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, uint32_t sh,
                      uint32_t esh) {
    uint32_t W[3];
    p14_record(w0, w1, w2, w3, sh, esh, W, e16);
    te = tab14(e16);
    p14_core(W, te.tlo, te.thi, h);
  };
  // an exception of Planes12x or Golay70: the exact Planes14 record of entry
  // ent of the tile's list
  auto exception = [&](uint32_t ent) {
    const u32x4a w = side.exc_entry((uint64_t)side.exc_base(tile) + ent - kExcEntry0);
    planes14(w.x, w.y, w.z, w.w, 0u, 28u);
  };
  if constexpr (LAYOUT == LEECH_PLANES14) {
    planes14(p.w0, p.w1, p.w2, p.w3, p.sh, p.esh);
    return;
  } else if constexpr (LAYOUT == LEECH_PLANES12X) {
    const uint32_t ent = p.w0 & 0xFFFu;
    if (ent >= kExcEntry0) {
      exception(ent);
    } else {
      e16 = ent << 4;
      te = tab(e16);
      p12_core(p.w0, p.w1, p.w2, te.thi, h);
    }
    return;
  } else if constexpr (LAYOUT == LEECH_SLOT32) {
    // one-hot masks of levels 1..4 -> code planes of level + 1 (codes 1..5)
    e16 = (p.w0 << 4) & 0x3FF0u;
    const uint32_t L = tab(e16).aux;
    pos = ~align(p.w1, p.w0, 10);
    const uint32_t m1 = L > 1 ? p.w1 >> 2 : 0u;
    const uint32_t m2 = L > 2 ? align(p.w2, p.w1, 26) : 0u;
    const uint32_t m3 = L > 3 ? align(p.w3, p.w2, 18) : 0u;
    const uint32_t m4 = L > 4 ? align(p.w4, p.w3, 10) : 0u;
    p0 = ~(m1 | m3);
    p1 = m1 | m2;
    p2 = m3 | m4;
  } else if constexpr (LAYOUT == LEECH_GOLAY70) {
    const uint32_t r0 = align(p.w1, p.w0, p.sh), r1 = align(p.w2, p.w1, p.sh), r2 = p.w2 >> p.sh;
    const uint32_t ent = r0 & 0xFFFu;
    if (ent >= kExcEntry0) {
      exception(ent);
    } else {
      e16 = ent << 4;
      te = tab(e16);
      golay70_core(align(r1, r0, kG70C0Pos), align(r2, r1, kG70C1Pos - 32),
                   cw(r0 >> kG70MsgPos & 0xFFFu), te.tlo, te.thi, h);
    }
    return;
  }
  te = tab(e16);
  planes_core(p0, p1, p2, pos, te.tlo, te.thi, h);
}

// Per-workgroup view of the streams: buffer descriptors based at the tile's
// first record and first scale, and the tile's shape.
struct TileCtx {
  __amdgpu_buffer_rsrc_t rec, sc;
  int tile, R_t, C, groups;
};
// A descriptor with no records: every load through it is out of range, returns
// zeros and reaches no memory.  Loads whose data is not needed (stand-in units,
// staging loads of waves with nothing to stage) go through it, so every wave
// issues the same load sequence without the bytes.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t null_rsrc() {
  return __builtin_amdgcn_make_buffer_rsrc(nullptr, 0, 0, kRsrcWord3);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)n, kRsrcWord3);
}

// Loads of unit g for a lane at place L.  EVEN: every unit base of the layout
// is 4-aligned, so L is used as is; otherwise the lane's window is recomputed
// from the unit base's offset modulo 4.  Loads are issued unconditionally:
// branches around loads would make the compiler's wait counts conservative.
// For a unit whose data is not needed (live = false, wave-uniform) the loads go
// through the null descriptor; g must still be a real unit (Slot32 reads its
// record pointer from the unit's side entry).
template <int LAYOUT, bool EVEN, class SIDE>
__device__ __forceinline__ Pref load_unit(const GemvArgs& a, const TileCtx& t, bool live,
                                          const Lane& L, int g, const SIDE& side) {
  Pref p = {0, 0, 0, 0, 0, 0, 0, 0};
  if constexpr (LAYOUT == kNoWeights) {
    return p;
  } else {
    const uint32_t blk = (uint32_t)g * (uint32_t)(t.R_t * t.C);   // blocks before the unit
    if constexpr (LAYOUT == LEECH_SLOT32) {
      uint64_t bits;
      uint32_t base;
      side.unit_entry(a.side0, t.tile * t.groups + g, bits, base);
      const uint32_t nbelow = (uint32_t)__builtin_popcountll(bits & ((1ull << L.ul) - 1ull));
      const uint32_t* rec = (const uint32_t*)(a.main + (uint64_t)base * 4) +
                            (L.ul * (uint32_t)kSlot32Small +
                             nbelow * (uint32_t)(kSlot32Large - kSlot32Small)) / 4;
      const u32x4 w = *(const u32x4*)rec;
      p.w0 = w.x; p.w1 = w.y; p.w2 = w.z; p.w3 = w.w; p.w4 = rec[4];
    } else {
      constexpr uint32_t S = Stride<LAYOUT>::v;
      const uint32_t ub = blk * S;
      Lane l = L;
      if constexpr (!EVEN) l = lane_place(L.ul, S, ub & 3u, L.own);
      const int soff = (int)(ub & ~3u);
      if constexpr (LAYOUT == LEECH_PLANES14) {
        const u32x4a w = __builtin_amdgcn_raw_buffer_load_b128(live ? t.rec : null_rsrc(), (int)l.rec,
                                                               soff, kStreamed);
        p.w0 = w.x; p.w1 = w.y; p.w2 = w.z; p.w3 = w.w;
      } else {
        const u32x3 w = __builtin_amdgcn_raw_buffer_load_b96(live ? t.rec : null_rsrc(), (int)l.rec,
                                                             soff, kStreamed);
        p.w0 = w.x; p.w1 = w.y; p.w2 = w.z;
      }
      p.sh = l.sh;
      p.esh = l.esh;
    }
    p.scale = __builtin_amdgcn_raw_buffer_load_b16(live ? t.sc : null_rsrc(), (int)(L.ul * 2u),
                                                   (int)(blk * 2u), kStreamed);
    return p;
  }
}

// The LDS entries, built from the device table: one 16-byte load per entry.
__device__ __forceinline__ LdsEntry make_entry(const DevClass* tab, uint32_t e, float cen0,
                                               float cen1) {
  const u32x4a d = *(const u32x4a*)&tab[e & 511u];      // perm[8], inv_norm, info
  LdsEntry t;
  t.tlo = d.x;
  t.thi = d.y;
  t.factor = __builtin_bit_cast(float, (uint32_t)d.z) * kTwo24 * ((e >> 9) ? cen1 : cen0);
  t.aux = d.w & 0xFFu;
  return t;
}

// Planes12x entries: tlo holds the Planes14 table's high word (|z| of
// levels 3 and 4), thi the magnitudes p12_core reads (levels 0..3), aux the
// added term (0 for a class).  p12_as14 rebuilds the Planes14 table, for an
// exception's exact record.
__device__ __forceinline__ LdsEntry p12_entry(uint32_t tlo14, uint32_t thi14, float factor) {
  LdsEntry t;
  t.tlo = thi14;
  t.thi = align(thi14, tlo14, 8);
  t.factor = factor;
  t.aux = 0u;
  return t;
}
__device__ __forceinline__ LdsEntry p12_as14(const LdsEntry& t) {
  LdsEntry r = t;
  r.tlo = t.thi << 8 | 0x80u;
  r.thi = t.tlo;
  return r;
}
// The entry in a layout's own arrangement.
template <int LAYOUT>
__device__ __forceinline__ LdsEntry make_entry_as(const DevClass* tab, uint32_t e, float cen0,
                                                  float cen1) {
  LdsEntry t = make_entry(tab, e, cen0, cen1);
  if constexpr (LAYOUT == LEECH_PLANES12X) t = p12_entry(t.tlo, t.thi, t.factor);
  if constexpr (LAYOUT == LEECH_GOLAY70) {
    g70_table(*((const u32x4a*)&tab[e & 511u] + 1), t.tlo, t.thi);
    t.aux = 0u;
  }
  return t;
}

// Golay codeword of a 12-bit message from the 128-entry generator table.
__device__ __forceinline__ uint32_t golay_word(const uint32_t* gen, uint32_t m) {
  return gen[m & 63u] ^ gen[64u + (m >> 6)];
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

// s = Σ_k h[k]·x[k] over the 12 binary16 pairs, f32 accumulation; the first
// product is a v_dot2_f32_f16 with a zero addend, where the compiler would
// otherwise zero a register for the accumulate-in-place form.
__device__ __forceinline__ float dot12(const uint32_t h[12], const uint32_t xw[12]) {
  float s;
  asm("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(s) : "v"(h[0]), "v"(xw[0]));
#pragma unroll
  for (int k = 1; k < 12; ++k) s = __builtin_amdgcn_fdot2(as_h2(h[k]), as_h2(xw[k]), s, false);
  return s;
}

// Sum over the C lanes of a row (C = 1, 2, 4, 8 or 16 adjacent lanes) as an
// xor butterfly, partners 1, 2, 4, 8 apart in that order: within a quad by DPP
// quad permutes, across quads by ds_swizzle's xor mode (no address register,
// no LDS memory).  For C = 3 the row's first lane adds the next two, fetched
// by ds_bpermute: (v0 + v1) + v2.  Only the row's first lane (c = 0) holds the
// row's sum.  Every lane is active here.
__device__ __forceinline__ float row_sum(float v, int C) {
  if (C == 3) {
    const int l = (int)(threadIdx.x & 63u);
    const float v1 = __builtin_bit_cast(
        float, __builtin_amdgcn_ds_bpermute(((l + 1) & 63) << 2, __builtin_bit_cast(int, v)));
    const float v2 = __builtin_bit_cast(
        float, __builtin_amdgcn_ds_bpermute(((l + 2) & 63) << 2, __builtin_bit_cast(int, v)));
    return (v + v1) + v2;
  }
  auto add = [&](int partner) { v += __builtin_bit_cast(float, partner); };
  if (C > 1)
    add(__builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
  if (C > 2)
    add(__builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
  if (C > 4) add(__builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), (4 << 10) | 0x1F));
  if (C > 8) add(__builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), (8 << 10) | 0x1F));
  return v;
}

// Row sum of the column-placed lanes of a matrix-core launch: row r's lanes
// are r + c·R, fetched by ds_bpermute.  For C ≤ 4 lane r (c = 0) gets v0
// (C = 1), v0 + v1, (v0 + v1) + v2 or (v0 + v1) + (v2 + v3); for C = 8 and 16
// (R = 4 or 8, both powers of two) an xor butterfly over the column bits,
// partners R, 2R, 4R, ... apart.  Every lane is active here.
__device__ __forceinline__ float row_sum_cols(float v, int C, int R) {
  const int l = (int)(threadIdx.x & 63u);
  auto at = [&](int c) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_ds_bpermute(((l + c * R) & 63) << 2, __builtin_bit_cast(int, v)));
  };
  if (C >= 8) {
    for (int step = R; step < C * R; step <<= 1)
      v += __builtin_bit_cast(
          float, __builtin_amdgcn_ds_bpermute(((l ^ step) & 63) << 2, __builtin_bit_cast(int, v)));
    return v;
  }
  if (C == 1) return v;
  const float s01 = v + at(1);
  if (C == 2) return s01;
  if (C == 3) return s01 + at(2);
  return s01 + (at(2) + at(3));
}

// Sixteen 4×4×4 binary16 products at once (f32 accumulate): block q = l / 4;
// lane 4q + i holds row i of A_q and column i of B_q (k = 0..3, two pair
// words each); d[i] of lane 4q + j is D_q row i, column j.
typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4a mfma4(uint32_t a0, uint32_t a1, uint32_t b0, uint32_t b1,
                                        f32x4a d) {
  return __builtin_amdgcn_mfma_f32_4x4x4f16(__builtin_bit_cast(half4_t, u32x2a{a0, a1}),
                                            __builtin_bit_cast(half4_t, u32x2a{b0, b1}), d, 0, 0,
                                            0);
}

// ------------------------------------------------------- fused rotation
// The activation rotation (blockwise Walsh–Hadamard, §2.3, §6) done by each
// GEMV workgroup in its prologue, while its first record loads are in flight:
// a thread holds up to kRotG groups of 8 consecutive coordinates (loaded
// first), applies the butterflies of index bits 0..2 in registers, the
// workgroup applies bits 3.. in radix-8 passes over an f32 copy in LDS, and a
// last pass scales by 2^(-k/2), rounds to binary16 (the product is rounded to
// f32 first) and stages the blocks in pair order.  Stage order and arithmetic
// are leech_rotate_x's, so the staged activation equals that call's output.
constexpr int kRotG = 5;      // groups of 8 coordinates per thread: K ≤ 40 · threads

__device__ __forceinline__ int rot_pad(int i) { return i + ((i >> 6) << 3); }

template <int E>
__device__ __forceinline__ void rot_butterflies(float* v) {
#pragma unroll
  for (int st = 1; st < E; st <<= 1)
#pragma unroll
    for (int t = 0; t < E; ++t)
      if (!(t & st)) {
        const float x = v[t], y = v[t | st];
        v[t] = x + y;
        v[t | st] = x - y;
      }
}

// One radix-2^BITS pass over index bits [LO, LO + BITS) of the K coordinates.
// The pass's bits are clear in b0 and the others clear in t << LO, so
// rot_pad(b0 + (t << LO)) = rot_pad(b0) + rot_pad(t << LO): one address per
// group and constant offsets.
template <int LO, int BITS>
__device__ __forceinline__ void rot_pass(float* rb, int K, int tid, int nthr) {
  constexpr int E = 1 << BITS;
  const int ngrp = K >> BITS;
  for (int grp = tid; grp < ngrp; grp += nthr) {
    float* base = rb + rot_pad(((grp >> LO) << (LO + BITS)) | (grp & ((1 << LO) - 1)));
    float v[E];
#pragma unroll
    for (int t = 0; t < E; ++t) v[t] = base[rot_pad(t << LO)];
    rot_butterflies<E>(v);
#pragma unroll
    for (int t = 0; t < E; ++t) base[rot_pad(t << LO)] = v[t];
  }
}

// Passes over index bits 3..k − 1, each after a barrier: (LO, BITS) pairs in
// increasing bit order.
template <int LO, int BITS, int... REST>
__device__ __forceinline__ void rot_passes(float* rb, int K, int tid, int nthr) {
  __syncthreads();
  rot_pass<LO, BITS>(rb, K, tid, nthr);
  if constexpr (sizeof...(REST) > 0) rot_passes<REST...>(rb, K, tid, nthr);
}

// The fewest passes of at most 4 bits each, the bits spread evenly over
// them: a pass costs a barrier and a round trip through LDS per group, so a
// split such as 3 + 3 + 1 (k = 10) would pay a third pass, and one with
// K / 2 groups, for a single bit.
__device__ __forceinline__ void rot_lds_stages(float* rb, int K, int k, int tid, int nthr) {
  switch (k) {
    case 4: rot_passes<3, 1>(rb, K, tid, nthr); break;
    case 5: rot_passes<3, 2>(rb, K, tid, nthr); break;
    case 6: rot_passes<3, 3>(rb, K, tid, nthr); break;
    case 7: rot_passes<3, 4>(rb, K, tid, nthr); break;
    case 8: rot_passes<3, 3, 6, 2>(rb, K, tid, nthr); break;
    case 9: rot_passes<3, 3, 6, 3>(rb, K, tid, nthr); break;
    case 10: rot_passes<3, 4, 7, 3>(rb, K, tid, nthr); break;
    case 11: rot_passes<3, 4, 7, 4>(rb, K, tid, nthr); break;
    case 12: rot_passes<3, 3, 6, 3, 9, 3>(rb, K, tid, nthr); break;
    case 13: rot_passes<3, 4, 7, 3, 10, 3>(rb, K, tid, nthr); break;
    case 14: rot_passes<3, 4, 7, 4, 11, 3>(rb, K, tid, nthr); break;
    case 15: rot_passes<3, 4, 7, 4, 11, 4>(rb, K, tid, nthr); break;
    default: break;     // k ≤ 3: every stage ran in registers
  }
}

// Half-word position (2·pair + half) of coordinate c of a block in pair
// order: the inverse of pair_coords.
__host__ __device__ constexpr int pair_half_of(int c) {
  return c < 4 ? 6 * c : c < 8 ? 6 * (c - 4) + 2 : c < 12 ? 6 * (c - 8) + 4
       : c < 16 ? 6 * (c - 12) + 5 : c < 20 ? 6 * (c - 16) + 1 : 6 * (c - 20) + 3;
}

__host__ __device__ constexpr bool pair_half_inverts() {
  for (int k = 0; k < 12; ++k) {
    int c0 = 0, c1 = 0;
    pair_coords(k, c0, c1);
    if (pair_half_of(c0) != 2 * k || pair_half_of(c1) != 2 * k + 1) return false;
  }
  return true;
}
static_assert(pair_half_inverts(), "pair_half_of inverts pair_coords");

__device__ void rotate_activation(const GemvArgs& a, const u32x4a* rx, const u32x2a* rsg,
                                  float* rb, uint32_t* xs, int xblocks, int tid, int nthr) {
  const int k = a.rot_k;
  const int K = (int)a.K;
#pragma unroll
  for (int q = 0; q < kRotG; ++q) {
    const int e0 = 8 * (tid + q * nthr);
    if (e0 < K) {
      float v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float f = (float)__builtin_bit_cast(_Float16, (uint16_t)(rx[q][t >> 1] >> (16 * (t & 1))));
        // bit 7 of the sign byte set means −1: it becomes the f32 sign bit
        const uint32_t neg = (rsg[q][t >> 2] >> (8 * (t & 3)) << 24) & 0x80000000u;
        v[t] = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, f) ^ neg);
      }
      if (k >= 3) {
        rot_butterflies<8>(v);
      } else if (k == 2) {
        rot_butterflies<4>(v);
        rot_butterflies<4>(v + 4);
      } else if (k == 1) {
#pragma unroll
        for (int t = 0; t < 8; t += 2) rot_butterflies<2>(v + t);
      }
      float* d = rb + rot_pad(e0);
      *reinterpret_cast<f32x4a*>(d) = f32x4a{v[0], v[1], v[2], v[3]};
      *reinterpret_cast<f32x4a*>(d + 4) = f32x4a{v[4], v[5], v[6], v[7]};
    }
  }
  // the entry point admits k ≤ 15
  rot_lds_stages(rb, K, k, tid, nthr);
  __syncthreads();
  // scale, round (to f32, then binary16) and store each coordinate at its
  // place in its block's pair order; zero past K up to the staged blocks' end.
  // A group of 8 is a third of a block: coordinates 0..7 and 16..23 fill the
  // low and the high halves of the same eight words, 8..15 four whole words.
  auto rounded = [&](int e0, uint32_t* h) {
    if (e0 < K) {
      const float* d = rb + rot_pad(e0);
      const f32x4a lo4 = *reinterpret_cast<const f32x4a*>(d);
      const f32x4a hi4 = *reinterpret_cast<const f32x4a*>(d + 4);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        float r = (t < 4 ? lo4[t] : hi4[t - 4]) * a.rot_norm;
        asm("" : "+v"(r));
        h[t] = __builtin_bit_cast(uint16_t, (_Float16)r);
      }
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t) h[t] = 0;
    }
  };
  auto place = [&](int e0, const uint32_t* h) {
    const int g = e0 >> 3, j = g / 3, third = g - 3 * j;
    uint32_t* blk = xs + 12 * j;
    uint16_t* half = reinterpret_cast<uint16_t*>(blk);
    if (third == 1) {
#pragma unroll
      for (int t = 0; t < 4; ++t) blk[pair_half_of(8 + t) >> 1] = h[t] | h[t + 4] << 16;
    } else if (third == 0) {
#pragma unroll
      for (int t = 0; t < 8; ++t) half[pair_half_of(t)] = (uint16_t)h[t];
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t) half[pair_half_of(16 + t)] = (uint16_t)h[t];
    }
  };
  for (int e0 = 8 * tid; e0 < 24 * xblocks; e0 += 8 * nthr) {
    uint32_t h[8];
    rounded(e0, h);
    place(e0, h);
  }
}

// ------------------------------------------------------------------- GEMV
// LDS, all dynamically sized: the class table (entry e at byte e·16, so a
// decoded field is its own address; launches whose tiles may hold rows of two
// row groups keep a second copy, with the second group's centroids, right
// after it), then x for groups·C block columns (zero past nb), the Golay70
// tables, the tile's side data, the cross-wave reduction.
template <int LAYOUT>
__host__ __device__ constexpr bool has_units() {
  return LAYOUT == LEECH_SLOT32;
}
template <int LAYOUT>
__host__ __device__ constexpr bool has_exc() {
  return LAYOUT == LEECH_PLANES12X || LAYOUT == LEECH_GOLAY70;
}

// A batched launch (NB > 1) keeps its cross-wave reduction in the activation
// area, which the loop no longer reads once every wave has finished, when
// each activation's share of it holds that activation's partial sums (64 per
// wave); a single GEMV keeps a separate buffer.
__host__ __device__ constexpr bool red_in_x(int nb_vectors, int xblocks, int waves) {
  return nb_vectors > 1 && xblocks * 48 >= waves * 64 * 4;
}

// NB: batch width (1, 2, 4, 8 or 16).  Each decoded block is multiplied with
// NB activations (NB > 1: Planes14), in the same order as a single GEMV, so
// every output vector is bit-identical to that activation's own GEMV.
// MX (NB > 1): the products go through the matrix cores instead, as the
// 16-block 4×4×4 binary16 MFMA with f32 accumulation.  Lanes are placed by
// column (lane c·R + r holds block (r, c) of the unit, R = tile_rows, a
// multiple of 4), so each block of 4 lanes holds blocks of one column.  In
// block q = lane / 4, lane 4q + i supplies activation 4s + i's four values of
// the column as A row i and four values of its own decoded block as B column
// i; D row i, column j (lane 4q + j, d[i]) is then the dot product of lane
// 4q + j's own block with activation 4s + i.  Six products take a block's 24
// values for four activations; no sum crosses a block, so the block's scale
// and class factor still multiply its f32 dot product.  No operand needs
// zeros: a row past NB, or a stand-in lane past the unit's columns, reads
// some staged activation, and only its own row or column of D sees it, which
// is discarded.  The matrix core sums a block's products in its own order, so
// outputs are within rounding of the single GEMV's; activation b always sits
// in row b mod 4 of product set b / 4, so they are bit-identical across batch
// widths.
// XPER: activation blocks each thread stages through registers in the ordered
// prologue (1 when the workgroup's threads cover every block, else 2; more
// blocks go through the unordered loop first).
// ROT: the activation arrives unrotated and the workgroup rotates it itself
// (Planes14, NB = 1): blockwise Walsh–Hadamard with the caller's signs, the
// stages in the order and arithmetic of leech_rotate_x, so the staged binary16
// activation is bit-identical to that call's output.
// PHASE: a measurement launch that records kPhaseStamps real-time stamps per
// workgroup (lane 0 of the stamping wave, a vector store each); the work is
// the plain launch's.
template <int LAYOUT, bool EVEN, int NB, int XPER, bool ROT, int PRO, bool PHASE, bool MX>
__device__ __forceinline__ void gemv_body(const GemvArgs& a) {
  static_assert(!MX || (NB > 1 && LAYOUT == LEECH_PLANES14 && !ROT && !PHASE),
                "matrix-core products serve batched Planes14 launches");
  constexpr int kPrefetch = pro_prefetch(PRO);        // units in flight per wave
  constexpr int kFirstUnits = pro_first(PRO);         // of them, before the barrier
  constexpr bool kRamp = kFirstUnits < kPrefetch;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  constexpr bool kW = LAYOUT != kNoWeights;
  LdsEntry* ts = (LdsEntry*)smem;                    // one table copy, or two
  uint8_t* const xbase = smem + (kW ? (a.tab2 ? 2 : 1) * a.tab_bytes : 0);
  constexpr bool kUnits = has_units<LAYOUT>();
  constexpr bool kExc = has_exc<LAYOUT>();
  const int64_t nb = a.nb;
  const int groups = (int)a.groups, C = a.C, waves = a.waves;   // unit counts fit 32 bits
  const int xblocks = groups * C;
  uint32_t* xs = (uint32_t*)xbase;                                 // NB × xblocks × 12 x pairs
  uint8_t* p = xbase + (size_t)NB * xblocks * 48;
  uint32_t* cws = (uint32_t*)p;                                    // Golay70: 128 words
  u32x2a* p14t = (u32x2a*)(p + 128 * 4);                           // Golay70: 512 tables
  if constexpr (LAYOUT == LEECH_GOLAY70) p += kG70LdsBytes;
  uint8_t* units_lds = p;                                          // groups × 16 B
  if constexpr (kUnits) p += (size_t)groups * kUnitEntryBytes;
  const bool red_x = red_in_x(NB, xblocks, waves);
  float* red = red_x ? (float*)xbase : (float*)p;                  // NB × waves × 64
  float* rb = (float*)p + NB * waves * 64;                         // ROT (NB = 1): rotation buffer

  const int tid = threadIdx.x, nthr = blockDim.x;
  const int tile = (int)blockIdx.x;
  const int R_t = (int)min((int64_t)a.R, a.M - (int64_t)tile * a.R);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  auto stamp = [&](int k) {
    if constexpr (PHASE) {
      const uint64_t t = __builtin_amdgcn_s_memrealtime();
      if (lane == 0) a.stamps[(uint64_t)blockIdx.x * kPhaseStamps + k] = t;
    }
  };
  if (wave == 0) stamp(0);
  // MX: lanes by column
  const int rl = MX ? lane % a.R : lane / C, cl = MX ? lane / a.R : lane % C;
  const int gf = groups - 1;                      // full-width column groups
  const int C_last = (int)(nb - (int64_t)gf * C);
  const bool row_ok = rl < R_t && (!MX || cl < C), last_ok = row_ok && cl < C_last;
  constexpr uint32_t S = Stride<LAYOUT>::v;
  // 24-bit products: a 64-bit multiply-add chosen for these would read an
  // undefined high half that may sit in a register with a load in flight, and
  // the wait for it drains every outstanding load
  const Lane Lf = lane_place(row_ok ? __umul24(rl, C) + cl : 0u, S, 0u, row_ok);
  const Lane Ll = lane_place(last_ok ? __umul24(rl, C_last) + cl : 0u, S, 0u, last_ok);
  // the pipeline's lane place and its stand-in unit: a full unit when there is
  // one, else the last (then the pipeline processes nothing)
  const Lane Lp = gf > 0 ? Lf : Ll;
  const int g_stand = gf > 0 ? gf - 1 : gf;
  const uint64_t tile_blk = (uint64_t)tile * a.R * (uint64_t)nb;
  const uint64_t tile_rec = tile_blk * S;
  TileCtx t;
  t.rec = make_rsrc(a.main + tile_rec, a.main_bytes - tile_rec);
  t.sc = make_rsrc(a.scale + tile_blk, ((uint64_t)a.M * (uint64_t)nb - tile_blk) * 2);
  t.tile = tile;
  t.R_t = R_t;
  t.C = C;
  t.groups = groups;

  // Side data of the tile: its unit entries (Slot32, copied to LDS below) and
  // the range of its exception entries (Planes12x, Golay70).
  const GlobalSide gside{&a};
  LdsSide side{&a, units_lds, tile * groups, 0u};
  uint32_t exc_first = 0, exc_count = 0;    // the tile's exception entries
  if constexpr (kExc) {
    const uint64_t e0 = ((const uint32_t*)a.side1)[tile];
    const uint64_t e1 = tile + 1 < a.tiles ? ((const uint32_t*)a.side1)[tile + 1] : a.n_exc;
    side.excbase = (uint32_t)e0;
    exc_first = (uint32_t)e0;
    exc_count = (uint32_t)(e1 - e0);
  }

  // Prologue, ordered for the in-order load counter: first the staging loads
  // (x blocks, class table, side data), then the last column group's loads,
  // then the pipeline's record loads, then the LDS writes, which wait only for
  // the older staging loads.
  constexpr int kXPer = XPER;                  // x blocks per thread held in registers
  constexpr int kXChunk = 4;                   // batched: x blocks per thread per round trip
  constexpr int kEPer = kExcPrefetch, kUPer = 2;
  // rare overflow first (xblocks > kXPer·threads, or fewer threads than
  // classes): loads of unknown count here, before the ordered ones.  Only the
  // ball's class ids occur in a layout, so only their entries are staged, both
  // gain entries of a class from one read of its table record.
  if constexpr (NB > 1) {
    // A batched launch stages all its activations here, kXChunk blocks a
    // thread in flight at a time: vector b's blocks follow vector b − 1's,
    // zero past nb and for vectors past nbatch.  (Requested after the first records instead, they return behind
    // them: loads return in order, and the launch is slower.)
    const int total = NB * xblocks;
    for (int j0 = tid; j0 < total; j0 += kXChunk * nthr) {
      XBlock r[kXChunk];
#pragma unroll
      for (int u = 0; u < kXChunk; ++u) {
        const int j = j0 + u * nthr;
        const int b = j / xblocks, jb = j - b * xblocks;
        if (j < total && jb < nb && b < a.nbatch)
          r[u] = load_x_block(a.x + b * a.ldx + 24 * (int64_t)jb);
        else
          r[u].v0 = r[u].v1 = r[u].v2 = u32x4a{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < kXChunk; ++u)
        if (j0 + u * nthr < total) store_x_block(r[u], xs + 12 * (j0 + u * nthr));
    }
  }
  if constexpr (NB == 1 && !ROT)
  for (int j = tid + kXPer * nthr; j < xblocks; j += nthr) {
    if (j < nb) {
      store_x_block(load_x_block(a.x + 24 * (int64_t)j), xs + 12 * j);
    } else {
      u32x4a* d = (u32x4a*)(xs + 12 * j);
      d[0] = d[1] = d[2] = u32x4a{0, 0, 0, 0};
    }
  }
  // the tile's gain centroids: its first row's group's, and where a second
  // group starts inside the tile (row `split` of it), that group's, staged in
  // the second table; each lane reads the table of its own row's group
  float cen0 = a.cen0, cen1 = a.cen1, cen0b = 0.0f, cen1b = 0.0f;
  bool two = false;
  int split = R_t;
  if (a.ngroups > 0) {
    const int64_t row0 = (int64_t)tile * a.R;
    int gi = 0;
    while (gi < a.ngroups - 1 && row0 >= a.grp_end[gi]) ++gi;
    cen0 = a.grp_cen[gi][0];
    cen1 = a.grp_cen[gi][1];
    if (gi < a.ngroups - 1 && a.grp_end[gi] < row0 + R_t) {
      two = true;
      split = (int)(a.grp_end[gi] - row0);
      cen0b = a.grp_cen[gi + 1][0];
      cen1b = a.grp_cen[gi + 1][1];
    }
  }
  const uint32_t toff = two && rl >= split ? a.tab_bytes : 0u;
  if constexpr (kW)
    for (int c = tid + nthr; c < kBallClasses; c += nthr) {
      ts[c] = make_entry_as<LAYOUT>(a.table, (uint32_t)c, cen0, cen1);
      ts[c + 512] = make_entry_as<LAYOUT>(a.table, (uint32_t)c | 512u, cen0, cen1);
      if (two) {
        LdsEntry* t2 = (LdsEntry*)(smem + a.tab_bytes);
        t2[c] = make_entry_as<LAYOUT>(a.table, (uint32_t)c, cen0b, cen1b);
        t2[c + 512] = make_entry_as<LAYOUT>(a.table, (uint32_t)c | 512u, cen0b, cen1b);
      }
      if constexpr (LAYOUT == LEECH_GOLAY70) p14t[c] = *(const u32x2a*)&a.table[c];
    }
  const uint8_t* side_units = LAYOUT == LEECH_SLOT32 ? a.side0 : a.side1;
  if constexpr (kUnits)
    for (int u = tid + kUPer * nthr; u < groups; u += nthr)
      ((u32x4a*)units_lds)[u] = ((const u32x4a*)side_units)[tile * groups + u];
  // x and the class table through buffer descriptors: a wave with no block
  // (no class) to stage loads through the null descriptor, and lanes past nb
  // read zeros, which is the padding past the last column
  const __amdgpu_buffer_rsrc_t rs_x = make_rsrc(a.x, (uint64_t)nb * 48);
  // ROT: the raw activation and its signs, eight coordinates per load
  u32x4a rx[kRotG];
  u32x2a rsg[kRotG];
  if constexpr (ROT) {
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.xraw, (uint64_t)a.K * 2);
    const __amdgpu_buffer_rsrc_t rsn = a.signs ? make_rsrc(a.signs, (uint64_t)a.K) : null_rsrc();
#pragma unroll
    for (int q = 0; q < kRotG; ++q) {
      const bool live = (int64_t)(q * nthr + wave * 64) * 8 < a.K;
      rx[q] = __builtin_amdgcn_raw_buffer_load_b128(live ? rr : null_rsrc(), (tid + q * nthr) * 16,
                                                    0, 0);
      rsg[q] = __builtin_amdgcn_raw_buffer_load_b64(live ? rsn : null_rsrc(), (tid + q * nthr) * 8,
                                                    0, 0);
    }
  }
  XBlock xr[kXPer];
#pragma unroll
  for (int q = 0; q < kXPer; ++q) {
    const bool live = NB == 1 && !ROT && q * nthr + wave * 64 < nb;
    const int off = (tid + q * nthr) * 48;
    if (!live) {      // a wave with no block to stage skips the loads (uniform)
      xr[q].v0 = xr[q].v1 = xr[q].v2 = u32x4a{0, 0, 0, 0};
    } else {
      const __amdgpu_buffer_rsrc_t r = live ? rs_x : null_rsrc();
      xr[q].v0 = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
      xr[q].v1 = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, 0);
      xr[q].v2 = __builtin_amdgcn_raw_buffer_load_b128(r, off + 32, 0, 0);
    }
  }
  u32x4a tr = {0, 0, 0, 0}, tr2 = {0, 0, 0, 0}, gr = {0, 0, 0, 0};
  if constexpr (kW) {
    const bool tlive = wave * 64 < kBallClasses;
    const __amdgpu_buffer_rsrc_t r =
        tlive ? make_rsrc(a.table, kBallClasses * sizeof(DevClass)) : null_rsrc();
    if (tlive)
      tr = __builtin_amdgcn_raw_buffer_load_b128(r, tid * (int)sizeof(DevClass), 0, 0);
    if constexpr (LAYOUT == LEECH_GOLAY70) {
      // the Golay70 value tables (second half of each class record) and the
      // 128-word generator table (wave 0)
      tr2 = __builtin_amdgcn_raw_buffer_load_b128(r, tid * (int)sizeof(DevClass) + 16, 0, 0);
      const __amdgpu_buffer_rsrc_t rg = wave == 0 ? make_rsrc(a.codewords, 512) : null_rsrc();
      gr = __builtin_amdgcn_raw_buffer_load_b128(rg, tid * 16, 0, 0);
    }
  }
  // the tile's unit entries and exception records: descriptors sized to the
  // tile's data, and the null descriptor for a wave with nothing to stage, so
  // that loads past the data reach no memory
  u32x4a ur[kUPer], er[kEPer];
  if constexpr (kUnits) {
    const __amdgpu_buffer_rsrc_t ru =
        make_rsrc(side_units + (uint64_t)tile * groups * kUnitEntryBytes,
                  (uint64_t)groups * kUnitEntryBytes);
#pragma unroll
    for (int q = 0; q < kUPer; ++q) {
      const __amdgpu_buffer_rsrc_t r = q * nthr + wave * 64 < groups ? ru : null_rsrc();
      ur[q] = __builtin_amdgcn_raw_buffer_load_b128(r, (tid + q * nthr) * 16, 0, 0);
    }
  }
  if constexpr (kExc) {
    // the tile's exception entries, for the hoisted decoder
    const uint64_t n_chunks = !a.inline_exc ? exc_count : 0;
    const __amdgpu_buffer_rsrc_t re =
        make_rsrc(a.side0 + (uint64_t)exc_first * kExcEntryBytes, n_chunks * kExcEntryBytes);
#pragma unroll
    for (int q = 0; q < kEPer; ++q) {
      const __amdgpu_buffer_rsrc_t r = (uint64_t)(q * nthr + wave * 64) < n_chunks ? re : null_rsrc();
      er[q] = __builtin_amdgcn_raw_buffer_load_b128(r, (tid + q * nthr) * 16, 0, 0);
    }
  }
  // the last column group: only its wave needs the data
  const int w_last = gf % waves;
  const Pref plast = load_unit<LAYOUT, EVEN>(a, t, wave == w_last, Ll, gf, gside);
  // this wave's full units: wave, wave + waves, ... < gf
  const int units = wave < gf ? (gf - 1 - wave) / waves + 1 : 0;
  Pref pf[kPrefetch];
  auto first_load = [&](int d, auto& sd) {
    pf[d] = load_unit<LAYOUT, EVEN>(a, t, d < units, Lp, min(wave + d * waves, g_stand), sd);
    __builtin_amdgcn_sched_barrier(0);    // keep the slots' loads in slot order
  };
#pragma unroll
  for (int d = 0; d < kFirstUnits; ++d) first_load(d, gside);
  if constexpr (NB == 1 && !ROT) {
#pragma unroll
    for (int q = 0; q < kXPer; ++q) {
      const int j = tid + q * nthr;
      if (j < xblocks) store_x_block(xr[q], xs + 12 * j);
    }
  }
  if constexpr (ROT) rotate_activation(a, rx, rsg, rb, xs, xblocks, tid, nthr);
  if constexpr (kW) {
    if (tid < kBallClasses) {
      LdsEntry e;
      e.tlo = tr.x;
      e.thi = tr.y;
      e.aux = tr.w & 0xFFu;
      if constexpr (LAYOUT == LEECH_PLANES12X) e = p12_entry(tr.x, tr.y, 0.0f);
      if constexpr (LAYOUT == LEECH_GOLAY70) {
        g70_table(tr2, e.tlo, e.thi);
        e.aux = 0u;
        p14t[tid] = u32x2a{tr.x, tr.y};
      }
      const float f = __builtin_bit_cast(float, (uint32_t)tr.z) * kTwo24;
      e.factor = f * cen0;
      ts[tid] = e;
      e.factor = f * cen1;
      ts[tid + 512] = e;
      if (two) {
        LdsEntry* t2 = (LdsEntry*)(smem + a.tab_bytes);
        e.factor = f * cen0b;
        t2[tid] = e;
        e.factor = f * cen1b;
        t2[tid + 512] = e;
      }
    }
    if constexpr (LAYOUT == LEECH_GOLAY70)
      if (tid < 32) ((u32x4a*)cws)[tid] = gr;
  }
  if constexpr (kUnits) {
#pragma unroll
    for (int q = 0; q < kUPer; ++q)
      if (tid + q * nthr < groups) ((u32x4a*)units_lds)[tid + q * nthr] = ur[q];
  }
  __syncthreads();
  if (wave == 0) stamp(1);
#pragma unroll
  for (int d = kFirstUnits; d < kPrefetch; ++d) pf[d] = Pref{0, 0, 0, 0, 0, 0, 0, 0};

  // the entry of a decoded field for this lane's row (the first table copy, or
  // the second at toff), in the layout's arrangement and as a Planes14 table,
  // and the entry at a table byte address
  auto tab_at = [&](uint32_t addr) -> LdsEntry {
    return *(const LdsEntry*)__builtin_assume_aligned(smem + addr, 16);
  };
  auto tab = [&](uint32_t e16) -> LdsEntry {
    // a power-of-two copy size lets the offset be or'ed into the field's mask
    return tab_at(kExc ? e16 + toff : e16 | toff);
  };
  // the entry of a decoded field in the table copy at byte offset off, as a
  // Planes14 table
  auto as14 = [&](uint32_t e16, uint32_t off) -> LdsEntry {
    LdsEntry t = tab_at(kExc ? e16 + off : e16 | off);
    if constexpr (LAYOUT == LEECH_PLANES12X) t = p12_as14(t);
    if constexpr (LAYOUT == LEECH_GOLAY70) {
      const u32x2a pt = p14t[(e16 >> 4) & 511u];
      t.tlo = pt.x;
      t.thi = pt.y;
    }
    return t;
  };
  auto tab14 = [&](uint32_t e16) -> LdsEntry { return as14(e16, toff); };
  auto cw = [&](uint32_t m) -> uint32_t { return golay_word(cws, m); };

  // Hoisted exception decoder (Planes12x, Golay70): each of the tile's
  // exceptions is decoded once, densely, before the loop, into a table entry
  // of its own at the entry number its record holds (in its row's table
  // copy): no table bytes, so the loop's lookups give zeros and its sum is +0,
  // and the exception's contribution dot12 · factor as the added term, so the
  // loop's fma(sum, factor, added) yields that contribution exactly.  Same
  // products, same order as decoding the exact record in the loop: y is
  // unchanged, and the loop has no branch, select or count for exceptions.
  bool hoisted = false;
  if constexpr (kExc) {
    hoisted = !a.inline_exc;
    if (hoisted) {
      auto keep = [&](uint32_t e, const u32x4a& w) {
        // the entry names the block's slot in the tile; units are R_t × C
        // blocks in column order
        const uint32_t slot = w.w >> (kExcSlotShift - 96);
        const int unit = min((int)(slot / (uint32_t)(R_t * C)), gf);
        const uint32_t ul = slot - (uint32_t)(unit * R_t * C);
        const uint32_t cols = unit == gf ? (uint32_t)C_last : (uint32_t)C;
        const uint32_t* xj = xs + 12 * (unit * C + ul % cols);
        uint32_t xw[12];
#pragma unroll
        for (int k = 0; k < 12; ++k) xw[k] = xj[k];
        uint32_t e16, W[3], h[12];
        p14_record(w.x, w.y, w.z, w.w, 0u, 28u, W, e16);
        const uint32_t off = two && (int)(ul / cols) >= split ? a.tab_bytes : 0u;
        const LdsEntry te = as14(e16, off);
        p14_core(W, te.tlo, te.thi, h);
        LdsEntry k;
        k.tlo = 0u;
        k.thi = 0u;
        k.factor = 0.0f;
        k.aux = __builtin_bit_cast(uint32_t, dot12(h, xw) * te.factor);
        *(LdsEntry*)(smem + ((kExcEntry0 + e) << 4) + off) = k;
      };
#pragma unroll
      for (int q = 0; q < kEPer; ++q)
        if (tid + q * nthr < (int)exc_count) keep(tid + q * nthr, er[q]);
      for (uint32_t e = tid + kEPer * nthr; e < exc_count; e += nthr)
        keep(e, gside.exc_entry((uint64_t)exc_first + e));
      __syncthreads();
    }
  }

  const uint8_t* x_lane = (const uint8_t*)xs + __umul24(cl, 48u);
  float acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = 0.0f;
  // MX: the A operand's LDS byte address for product set s is the unit's x
  // offset + x_off[s]: lane 4q + i reads activation 4s + i (the last one past
  // NB) of its column (the unit's first past the columns)
  constexpr int kSets = MX ? (NB + 3) / 4 : 1;
  uint32_t x_off[kSets];
  if constexpr (MX) {
    const uint32_t x0 = (uint32_t)(xbase - smem);
    const int i = min(lane & 3, NB - 1), c = min(cl, C - 1);
#pragma unroll
    for (int s = 0; s < kSets; ++s)
      x_off[s] = x0 + (uint32_t)(((4 * s + i) * xblocks + c) * 48);
  }
  // One unit: decode slot p for unit g and accumulate.  LAST: the last
  // column group, whose stand-in lanes (past the last column) must add zero.
  auto process = [&](const Pref& pr, int g, const Lane& L, auto last) {
    if constexpr (MX) {
      uint32_t h[12], e16;
      LdsEntry te;
      decode_block<LAYOUT>(pr, tile, tab, tab14, cw, side, h, e16, te);
      const float sf = (float)as_half(pr.scale) * te.factor;
      const uint32_t ub = (uint32_t)(g * (C * 48));
#pragma unroll
      for (int s = 0; s < kSets; ++s) {
        const u32x4a* xa = (const u32x4a*)__builtin_assume_aligned(smem + (ub + x_off[s]), 16);
        const u32x4a a0 = xa[0], a1 = xa[1], a2 = xa[2];
        f32x4a d = {0.0f, 0.0f, 0.0f, 0.0f};
        d = mfma4(a0.x, a0.y, h[0], h[1], d);
        d = mfma4(a0.z, a0.w, h[2], h[3], d);
        d = mfma4(a1.x, a1.y, h[4], h[5], d);
        d = mfma4(a1.z, a1.w, h[6], h[7], d);
        d = mfma4(a2.x, a2.y, h[8], h[9], d);
        d = mfma4(a2.z, a2.w, h[10], h[11], d);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * s + i < NB) acc[4 * s + i] = __builtin_fmaf(sf, d[i], acc[4 * s + i]);
      }
      return;
    }
    const u32x4a* xp = (const u32x4a*)(x_lane + g * (C * 48));
    const u32x4a x0 = xp[0], x1 = xp[1], x2 = xp[2];
    const uint32_t xw[12] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w,
                             x2.x, x2.y, x2.z, x2.w};
    if constexpr (LAYOUT == kNoWeights) {
      const uint32_t ones[12] = {0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u,
                                 0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u,
                                 0x3C003C00u, 0x3C003C00u, 0x3C003C00u, 0x3C003C00u};
      acc[0] += dot12(ones, xw);
    } else {
      uint32_t h[12], e16;
      if constexpr (kExc) {
        if (hoisted) {
          // the record's entry field addresses the class's entry or the
          // exception's own (added term = its kept contribution)
          LdsEntry te;
          if constexpr (LAYOUT == LEECH_PLANES12X) {
            te = tab_at(lshl4_add(pr.w0 & 0xFFFu, toff));
            p12_core(pr.w0, pr.w1, pr.w2, te.thi, h);
          } else {
            const uint32_t r0 = align(pr.w1, pr.w0, pr.sh), r1 = align(pr.w2, pr.w1, pr.sh);
            const uint32_t r2 = pr.w2 >> pr.sh;
            te = tab_at(lshl4_add(r0 & 0xFFFu, toff));
            golay70_core(align(r1, r0, kG70C0Pos), align(r2, r1, kG70C1Pos - 32),
                         cw(r0 >> kG70MsgPos & 0xFFFu), te.tlo, te.thi, h);
          }
          float v = __builtin_fmaf(dot12(h, xw), te.factor, __builtin_bit_cast(float, te.aux));
          if constexpr (decltype(last)::value) v = L.own ? v : 0.0f;
          acc[0] = __builtin_fmaf((float)as_half(pr.scale), v, acc[0]);
          return;
        }
      }
      LdsEntry te;
      decode_block<LAYOUT>(pr, tile, tab, tab14, cw, side, h, e16, te);
      const float sc = (float)as_half(pr.scale), f = te.factor;
      acc[0] = __builtin_fmaf(sc, dot12(h, xw) * f, acc[0]);
#pragma unroll
      for (int b = 1; b < NB; ++b) {
        const u32x4a* xq = xp + 3 * b * xblocks;
        const u32x4a y0 = xq[0], y1 = xq[1], y2 = xq[2];
        const uint32_t xv[12] = {y0.x, y0.y, y0.z, y0.w, y1.x, y1.y, y1.z, y1.w,
                                 y2.x, y2.y, y2.z, y2.w};
        acc[b] = __builtin_fmaf(sc, dot12(h, xv) * f, acc[b]);
      }
    }
  };
  int done = 0;
  // Full rounds: consume every slot, refilling each with the unit kPrefetch
  // steps ahead (past the wave's last unit the refill is an in-bounds
  // stand-in).  Decoding before refilling lets the refill reuse the slot's
  // registers: a refill into fresh registers would be moved back at the loop
  // latch, and moving a register with a load in flight waits for every
  // outstanding load.
  auto ramp = [&](int d) {     // the first round requests slot d + kFirstUnits
    if constexpr (kRamp)
      if (d + kFirstUnits < kPrefetch) first_load(d + kFirstUnits, side);
  };
  auto round = [&](auto ramped) {
#pragma unroll
    for (int d = 0; d < kPrefetch; ++d) {
      if constexpr (decltype(ramped)::value) ramp(d);
      const int g = wave + (done + d) * waves;
      process(pf[d], g, Lp, std::false_type{});
      pf[d] = load_unit<LAYOUT, EVEN>(a, t, done + d + kPrefetch < units, Lp,
                                      min(g + kPrefetch * waves, g_stand), side);
    }
  };
  auto tail = [&](auto ramped) {
    // the last ≤ kPrefetch units are in flight: straight-line, no refills
#pragma unroll
    for (int d = 0; d < kPrefetch; ++d) {
      if constexpr (decltype(ramped)::value) ramp(d);
      if (d < units - done) process(pf[d], wave + (done + d) * waves, Lp, std::false_type{});
    }
  };
  if constexpr (kRamp) {
    if (units > kPrefetch) {
      round(std::true_type{});
      done = kPrefetch;
      for (; units - done > kPrefetch; done += kPrefetch) round(std::false_type{});
      tail(std::false_type{});
    } else {
      tail(std::true_type{});
    }
  } else {
    for (; units - done > kPrefetch; done += kPrefetch) round(std::false_type{});
    tail(std::false_type{});
  }
  // the last column group, by the wave next in turn; its lanes past the last
  // column read zero x and add exactly zero
  if (wave == w_last) process(plast, gf, Ll, std::true_type{});
  if constexpr (PHASE) {
    // the wave's sum depends on every unit it decoded: stamp once it exists
    float s0 = acc[0];
    asm volatile("" : "+v"(s0));
    acc[0] = s0;
    stamp(2 + wave);
  }
  if (red_x) __syncthreads();     // every wave is done with the activations
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float v = MX ? row_sum_cols(acc[b], C, a.R) : row_sum(acc[b], C);
    if (cl == 0 && rl < R_t) red[(b * waves + wave) * 64 + rl] = v;
  }
  __syncthreads();
  for (int i = tid; i < NB * 64; i += nthr) {
    const int b = i >> 6, row = i & 63;
    if (row < R_t && b < a.nbatch) {
      float y = 0.0f;
      for (int w = 0; w < waves; ++w) y += red[(b * waves + w) * 64 + row];
      a.y[b * a.ldy + (int64_t)tile * a.R + row] = y;
    }
  }
  if (wave == 0) stamp(10);
}

template <int LAYOUT, bool EVEN, int NB = 1, int XPER = 2, bool ROT = false, int PRO = 0,
          bool PHASE = false, bool MX = false>
__global__ __launch_bounds__(kMaxWaves * 64) void gemv_kernel(GemvArgs a) {
  gemv_body<LAYOUT, EVEN, NB, XPER, ROT, PRO, PHASE, MX>(a);
}

// Matrix-core batches of 2 and 4 activations: held to 128 registers (four
// waves per SIMD), so that two 8-wave workgroups share a CU when there are
// more tiles than CUs.  Wider batches would spill there, and their staged
// activations mostly leave LDS for one workgroup a CU anyway.
template <int LAYOUT, bool EVEN, int NB, int XPER>
__global__ __launch_bounds__(kMaxWaves * 64, 4) void gemv_kernel_mx(GemvArgs a) {
  gemv_body<LAYOUT, EVEN, NB, XPER, false, 0, false, true>(a);
}

// --------------------------------------------------------- decode export
// One thread per block, with the GEMV's decode function and plain loads at
// the block's own byte offset; the binary16 pairs are turned back into integer
// coordinates (|z| in the low byte of each half, the sign in its bit 15).
template <int LAYOUT>
__global__ __launch_bounds__(256) void decode_kernel(GemvArgs a, int8_t* zout, uint16_t* cout,
                                                     uint8_t* gout) {
  const int64_t bi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (bi >= a.M * a.nb) return;
  const int64_t r = bi / a.nb, j = bi % a.nb;
  const int tile = (int)(r / a.R);
  const int g = (int)(j / a.C);
  const int R_t = (int)min((int64_t)a.R, a.M - (int64_t)tile * a.R);
  const int C_g = (int)min((int64_t)a.C, a.nb - (int64_t)g * a.C);
  const uint32_t ul = (uint32_t)((r % a.R) * C_g + (j % a.C));
  const uint64_t blk = (uint64_t)tile * a.R * a.nb + (uint64_t)g * R_t * a.C + ul;
  const GlobalSide side{&a};
  Pref p = {0, 0, 0, 0, 0, 0, 0, 0};
  if constexpr (LAYOUT == LEECH_SLOT32) {
    uint64_t bits;
    uint32_t base;
    side.unit_entry(a.side0, tile * (int)a.groups + g, bits, base);
    const uint32_t nbelow = (uint32_t)__builtin_popcountll(bits & ((1ull << ul) - 1ull));
    const uint32_t* rec = (const uint32_t*)(a.main + (uint64_t)base * 4) +
                          (ul * (uint32_t)kSlot32Small + nbelow * (uint32_t)(kSlot32Large - kSlot32Small)) / 4;
    p.w0 = rec[0]; p.w1 = rec[1]; p.w2 = rec[2]; p.w3 = rec[3]; p.w4 = rec[4];
  } else {
    const uint64_t off = blk * Stride<LAYOUT>::v;
    const uint32_t* w = (const uint32_t*)(a.main + (off & ~3ull));
    p.w0 = w[0]; p.w1 = w[1]; p.w2 = w[2];
    if constexpr (LAYOUT == LEECH_PLANES14) p.w3 = w[3];
    p.sh = (uint32_t)(off & 3u) * 8u;
    p.esh = (p.sh + 28u) & 31u;
  }
  auto tab = [&](uint32_t e16) -> LdsEntry {
    return make_entry_as<LAYOUT>(a.table, e16 >> 4, 1.0f, 1.0f);
  };
  auto tab14 = [&](uint32_t e16) -> LdsEntry { return make_entry(a.table, e16 >> 4, 1.0f, 1.0f); };
  auto cw = [&](uint32_t m) -> uint32_t { return golay_word(a.codewords, m); };
  uint32_t h[12], e16;
  LdsEntry te;
  decode_block<LAYOUT>(p, tile, tab, tab14, cw, side, h, e16, te);
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
  const uint32_t e = e16 >> 4;
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
// How GEMV launches enqueued from now on decode Golay70 exceptions.
static std::atomic<int> g_exc_mode{LEECH_EXC_HOISTED};

static int hip_fail(const char* what, hipError_t e) {
  return set_error(LEECH_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Waves per workgroup: each wave walks every waves-th unit of the tile.  The
// summation order depends on it, so it is a function of the shape only.
static int waves_for(int64_t groups) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(kMaxWaves, groups));
}

static int check_desc_device(const leech_layout_desc* d) {
  if (!d) return set_error(LEECH_E_ARG, "desc is NULL");
  if (d->M <= 0 || d->Kpad <= 0 || d->Kpad % kDim || d->nb != d->Kpad / kDim)
    return set_error(LEECH_E_SHAPE, "descriptor shape is not valid");
  if (!geometry_ok(d->lane_cols, d->tile_rows))
    return set_error(LEECH_E_SHAPE, "descriptor geometry (lane_cols, tile_rows) is not valid");
  // tile offsets (R·nb·20 bytes at most) and unit counts stay within 31 bits
  if (d->M > (1ll << 31) || d->nb > (1ll << 24) ||
      (uint64_t)d->tile_rows * (uint64_t)d->nb * 20u > 0x7FFFFFFFull)
    return set_error(LEECH_E_SHAPE, "matrix too large for 32-bit tile offsets");
  return LEECH_OK;
}

static GemvArgs make_args(const leech_layout_desc* d) {
  GemvArgs a;
  std::memset(&a, 0, sizeof a);
  a.M = d->M;
  a.nb = d->nb;
  a.C = d->lane_cols;
  a.R = d->tile_rows;
  a.groups = (d->nb + a.C - 1) / a.C;
  a.waves = waves_for(a.groups);
  a.inline_exc = g_exc_mode.load(std::memory_order_relaxed) == LEECH_EXC_INLINE;
  a.tiles = (d->M + a.R - 1) / a.R;
  a.n_exc = d->n_exceptions;
  a.main_bytes = d->main_bytes;
  a.nbatch = 1;
  a.tab_bytes = kTableBytes;
  a.tile_exc_max = d->tile_exc_max;
  return a;
}

// Every unit base of a fixed-stride layout is 4-aligned when the last tile's
// units are (tile bases are: tile_rows is a multiple of 4; so are a full
// tile's unit bases, R · C blocks apart).
static bool even_bases(const GemvArgs& a, int layout) {
  const int64_t stride = layout == LEECH_PLANES14 ? kPlanes14Bytes
                         : layout == LEECH_PLANES12X ? kPlanes12Bytes
                         : layout == LEECH_GOLAY70 ? kGolay70Bytes : 0;
  const int64_t rows_last = a.M - (a.tiles - 1) * a.R;
  return (rows_last * a.C * stride) % 4 == 0;
}

template <int LAYOUT, int NB = 1>
static size_t gemv_lds_bytes(const GemvArgs& a) {
  const size_t red = red_in_x(NB, a.groups * a.C, a.waves) ? 0 : (size_t)NB * a.waves * 64 * 4;
  const size_t table = LAYOUT == kNoWeights ? 0 : (a.tab2 ? 2 : 1) * (size_t)a.tab_bytes;
  return table + (size_t)NB * a.groups * a.C * 48 +
         (LAYOUT == LEECH_GOLAY70 ? kG70LdsBytes : 0) +
         (has_units<LAYOUT>() ? (size_t)a.groups * kUnitEntryBytes : 0) +
         red;
}

template <int LAYOUT, bool EVEN, int NB, int XPER, bool ROT = false, int PRO = 0,
          bool PHASE = false, bool MX = false>
static int launch_gemv_kernel(const GemvArgs& a, size_t shmem, hipStream_t st) {
  constexpr bool kCapped = MX && NB <= 4;
  const void* fn;
  if constexpr (kCapped)
    fn = (const void*)gemv_kernel_mx<LAYOUT, EVEN, NB, XPER>;
  else
    fn = (const void*)gemv_kernel<LAYOUT, EVEN, NB, XPER, ROT, PRO, PHASE, MX>;
  if (shmem > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    if (e != hipSuccess) return hip_fail("hipFuncSetAttribute", e);
  }
  if constexpr (kCapped)
    hipLaunchKernelGGL((gemv_kernel_mx<LAYOUT, EVEN, NB, XPER>), dim3((unsigned)a.tiles),
                       dim3(64 * a.waves), shmem, st, a);
  else
    hipLaunchKernelGGL((gemv_kernel<LAYOUT, EVEN, NB, XPER, ROT, PRO, PHASE, MX>),
                       dim3((unsigned)a.tiles), dim3(64 * a.waves), shmem, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail("gemv launch", e);
  return LEECH_OK;
}

// Prologue mode of a single GEMV from the most units a wave streams (the
// tile's full column groups over its waves), by measurement: 4096×4104 (6 a
// wave) 5.17 -> 4.60 µs with mode 2; 5120×5136 (14) 6.89 -> 6.59 µs with
// mode 1; 8192×8208 (22) is fastest with mode 0.
static std::atomic<int> g_pro_mode{LEECH_PROLOGUE_AUTO};

static int prologue_mode(const GemvArgs& a) {
  const int forced = g_pro_mode.load(std::memory_order_relaxed);
  if (forced != LEECH_PROLOGUE_AUTO) return forced;
  const int64_t full = a.groups - 1;
  const int64_t per_wave = full > 0 ? (full + a.waves - 1) / a.waves : 0;
  return per_wave <= 6 ? 2 : per_wave <= 16 ? 1 : 0;
}

template <int LAYOUT, bool EVEN, int NB, int XPER, bool PHASE = false, bool MX = false>
static int launch_gemv_pro(const GemvArgs& a, size_t shmem, hipStream_t st) {
  if constexpr (MX) return launch_gemv_kernel<LAYOUT, EVEN, NB, XPER, false, 0, false, true>(a, shmem, st);
  if constexpr (NB == 1 && EVEN && LAYOUT != kNoWeights) {
    switch (prologue_mode(a)) {
      case 2: return launch_gemv_kernel<LAYOUT, EVEN, NB, XPER, false, 2, PHASE>(a, shmem, st);
      case 1: return launch_gemv_kernel<LAYOUT, EVEN, NB, XPER, false, 1, PHASE>(a, shmem, st);
      default: break;
    }
  }
  return launch_gemv_kernel<LAYOUT, EVEN, NB, XPER, false, 0, PHASE>(a, shmem, st);
}

template <int LAYOUT, bool EVEN, int NB = 1, bool PHASE = false, bool MX = false>
static int launch_gemv_as(const GemvArgs& a, size_t shmem, hipStream_t st) {
  // one activation block per thread when the workgroup's threads cover them
  if (NB > 1 || a.groups * a.C <= 64 * a.waves)
    return launch_gemv_pro<LAYOUT, EVEN, NB, 1, PHASE, MX>(a, shmem, st);
  return launch_gemv_pro<LAYOUT, EVEN, NB, 2, PHASE, MX>(a, shmem, st);
}


template <int LAYOUT, int NB = 1, bool PHASE = false, bool MX = false>
static int launch_gemv(const GemvArgs& a0, hipStream_t st) {
  GemvArgs a = a0;
  if constexpr (has_exc<LAYOUT>()) {
    // the hoisted decoder keeps the tile's exceptions as table entries after
    // the 1024 class entries; where they do not fit in LDS, exceptions are
    // decoded in the loop
    if (!a.inline_exc) {
      a.tab_bytes = (uint32_t)(kExcEntry0 + a.tile_exc_max) * (uint32_t)sizeof(LdsEntry);
      if (gemv_lds_bytes<LAYOUT, NB>(a) > 160 * 1024) {
        a.inline_exc = 1;
        a.tab_bytes = kTableBytes;
      }
    }
  }
  const size_t shmem = gemv_lds_bytes<LAYOUT, NB>(a);
  if (shmem > 160 * 1024)
    return set_error(LEECH_E_SHAPE, "Kpad too large for the LDS-staged activation");
  if (LAYOUT == kNoWeights || even_bases(a, LAYOUT))
    return launch_gemv_as<LAYOUT, true, NB, PHASE, MX>(a, shmem, st);
  return launch_gemv_as<LAYOUT, false, NB, PHASE, MX>(a, shmem, st);
}

// Rotated launches (Planes14): the LDS of a plain launch plus the f32
// rotation buffer.
static size_t rot_lds_bytes(const GemvArgs& a) {
  return gemv_lds_bytes<LEECH_PLANES14>(a) + ((size_t)a.K + (size_t)(a.K >> 6) * 8 + 16) * 4;
}

static int launch_gemv_rotated(const GemvArgs& a, hipStream_t st) {
  const size_t shmem = rot_lds_bytes(a);
  if (shmem > 160 * 1024)
    return set_error(LEECH_E_SHAPE, "K too large for the LDS-staged rotation");
  if (even_bases(a, LEECH_PLANES14))
    return launch_gemv_kernel<LEECH_PLANES14, true, 1, 1, true>(a, shmem, st);
  return launch_gemv_kernel<LEECH_PLANES14, false, 1, 1, true>(a, shmem, st);
}

// Batch width of the next chunk of a batched launch: 2, 4, 8 or 16 (the next
// power of two at or above the vectors left, at most 16; vectors past the
// chunk's count read zero), narrowed until the activations fit in LDS; 1 for
// a single vector left on the dot-product path, or when not even two fit.  On
// the matrix-core path a single vector left still runs 2 wide, so that every
// vector of a batch gets the same arithmetic.
static int batch_width(const GemvArgs& a, int left, bool mx) {
  if (left <= 1 && !mx) return 1;
  for (int w = left > 8 ? 16 : left > 4 ? 8 : left > 2 ? 4 : 2; w >= 2; w >>= 1) {
    const size_t need = w == 16  ? gemv_lds_bytes<LEECH_PLANES14, 16>(a)
                        : w == 8 ? gemv_lds_bytes<LEECH_PLANES14, 8>(a)
                        : w == 4 ? gemv_lds_bytes<LEECH_PLANES14, 4>(a)
                                 : gemv_lds_bytes<LEECH_PLANES14, 2>(a);
    if (need <= 160 * 1024) return w;
  }
  return 1;
}

// Products of batched launches: the 16-block 4×4×4 MFMA form (default) or
// v_dot2 per activation.
static std::atomic<int> g_batch_mode{LEECH_BATCH_AUTO};

template <int NB>
static int launch_batch(const GemvArgs& c, bool mx, hipStream_t st) {
  return mx ? launch_gemv<LEECH_PLANES14, NB, false, true>(c, st)
            : launch_gemv<LEECH_PLANES14, NB>(c, st);
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

// Validation and argument setup shared by the GEMV entry points; the caller
// fills the centroids.
static int gemv_setup(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                      const void* d_side1, const void* d_class_table, const void* d_codewords,
                      const uint16_t* d_scale, const uint16_t* d_x, float* d_y, GemvArgs* out) {
  int rc = check_desc_device(desc);
  if (rc) return rc;
  if (!d_main || !d_class_table || !d_scale || !d_x || !d_y)
    return set_error(LEECH_E_ARG, "NULL argument");
  if ((desc->side_bytes[0] && !d_side0) || (desc->side_bytes[1] && !d_side1))
    return set_error(LEECH_E_ARG, "layout needs its side streams");
  if (desc->layout == LEECH_GOLAY70 && !d_codewords)
    return set_error(LEECH_E_ARG, "GOLAY70 needs the codeword table");
  if (((uintptr_t)d_x & 15) || ((uintptr_t)d_main & 3) || ((uintptr_t)d_class_table & 15) ||
      ((uintptr_t)d_codewords & 15) || ((uintptr_t)d_side0 & 3) || ((uintptr_t)d_side1 & 7) ||
      ((uintptr_t)d_scale & 1))
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
  *out = a;
  return LEECH_OK;
}

static int gemv_dispatch(const leech_layout_desc* desc, const GemvArgs& a, hipStream_t st) {
  switch (desc->layout) {
    case LEECH_SLOT32: return launch_gemv<LEECH_SLOT32>(a, st);
    case LEECH_PLANES14: return launch_gemv<LEECH_PLANES14>(a, st);
    case LEECH_PLANES12X: return launch_gemv<LEECH_PLANES12X>(a, st);
    case LEECH_GOLAY70: return launch_gemv<LEECH_GOLAY70>(a, st);
    default: return set_error(LEECH_E_LAYOUT, "unknown layout");
  }
}
}  // namespace leech

using namespace leech;

extern "C" {

int leech_gemv(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
               const void* d_side1, const void* d_class_table, const void* d_codewords,
               const uint16_t* d_scale, const float centroid[2], const uint16_t* d_x,
               float* d_y, void* stream) {
  clear_error();
  if (!centroid) return set_error(LEECH_E_ARG, "NULL argument");
  GemvArgs a;
  int rc = gemv_setup(desc, d_main, d_side0, d_side1, d_class_table, d_codewords, d_scale, d_x,
                      d_y, &a);
  if (rc) return rc;
  a.cen0 = centroid[0];
  a.cen1 = centroid[1];
  return gemv_dispatch(desc, a, (hipStream_t)stream);
}

int leech_gemv_batch(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                     const void* d_side1, const void* d_class_table, const void* d_codewords,
                     const uint16_t* d_scale, const float centroid[2], int batch,
                     const uint16_t* d_X, int64_t ldx, float* d_Y, int64_t ldy, void* stream) {
  clear_error();
  if (!centroid) return set_error(LEECH_E_ARG, "NULL argument");
  if (batch < 1) return set_error(LEECH_E_ARG, "batch must be at least 1");
  GemvArgs a;
  int rc = gemv_setup(desc, d_main, d_side0, d_side1, d_class_table, d_codewords, d_scale, d_X,
                      d_Y, &a);
  if (rc) return rc;
  if (batch > 1 && desc->layout != LEECH_PLANES14)
    return set_error(LEECH_E_LAYOUT, "batched GEMVs serve the PLANES14 layout");
  if (batch > 1 && (ldx < desc->Kpad || ldx % 8 || ldy < desc->M))
    return set_error(LEECH_E_ARG, "need ldx >= Kpad, ldx a multiple of 8, ldy >= M");
  a.cen0 = centroid[0];
  a.cen1 = centroid[1];
  a.ldx = ldx;
  a.ldy = ldy;
  const hipStream_t st = (hipStream_t)stream;
  const bool mx = batch > 1 && g_batch_mode.load(std::memory_order_relaxed) == LEECH_BATCH_AUTO;
  for (int b0 = 0; b0 < batch;) {
    const int w = batch_width(a, batch - b0, mx);
    GemvArgs c = a;
    c.x = d_X + (int64_t)b0 * ldx;
    c.y = d_Y + (int64_t)b0 * ldy;
    c.nbatch = std::min(w, batch - b0);
    rc = w == 16  ? launch_batch<16>(c, mx, st)
         : w == 8 ? launch_batch<8>(c, mx, st)
         : w == 4 ? launch_batch<4>(c, mx, st)
         : w == 2 ? launch_batch<2>(c, mx, st)
                  : gemv_dispatch(desc, c, st);
    if (rc) return rc;
    b0 += c.nbatch;
  }
  return LEECH_OK;
}

}  // extern "C"

namespace leech {
// Row groups of a grouped launch, validated into the launch arguments.
static int set_groups(const leech_layout_desc* desc, int n_groups, const int64_t* group_rows,
                      const float* group_centroids, GemvArgs& a) {
  if (!group_rows || !group_centroids) return set_error(LEECH_E_ARG, "NULL argument");
  if (n_groups < 1 || n_groups > LEECH_MAX_GROUPS)
    return set_error(LEECH_E_ARG, "n_groups must be 1.." + std::to_string(LEECH_MAX_GROUPS));
  // a tile holds rows of at most two groups: at most one group boundary
  // strictly inside it (a boundary on its first row starts it in a new group)
  int64_t end = 0, straddled = -1;
  a.tab2 = 0;
  for (int g = 0; g < n_groups; ++g) {
    if (group_rows[g] <= 0) return set_error(LEECH_E_SHAPE, "every group needs rows");
    end += group_rows[g];
    if (g + 1 < n_groups && end % a.R) {
      const int64_t t = end / a.R;
      if (t == straddled)
        return set_error(LEECH_E_SHAPE, "a tile of " + std::to_string(a.R) +
                                            " rows would hold rows of three groups (tile " +
                                            std::to_string(t) + ")");
      straddled = t;
      a.tab2 = 1;
    }
    const float c0 = group_centroids[2 * g], c1 = group_centroids[2 * g + 1];
    if (!std::isfinite(c0) || !std::isfinite(c1))
      return set_error(LEECH_E_ARG, "group centroids must be finite");
    a.grp_end[g] = end;
    a.grp_cen[g][0] = c0;
    a.grp_cen[g][1] = c1;
  }
  if (end != desc->M) return set_error(LEECH_E_SHAPE, "group rows do not sum to M");
  a.ngroups = n_groups;
  a.cen0 = a.grp_cen[0][0];
  a.cen1 = a.grp_cen[0][1];
  return LEECH_OK;
}
}  // namespace leech

extern "C" {

int leech_gemv_rotated(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                       const void* d_side1, const void* d_class_table, const void* d_codewords,
                       const uint16_t* d_scale, int n_groups, const int64_t* group_rows,
                       const float* group_centroids, int64_t K, const uint16_t* d_x,
                       const int8_t* d_signs, float* d_y, void* stream) {
  clear_error();
  GemvArgs a;
  // d_x stands in for the staged activation in the shared checks (alignment)
  int rc = gemv_setup(desc, d_main, d_side0, d_side1, d_class_table, d_codewords, d_scale, d_x,
                      d_y, &a);
  if (rc) return rc;
  if (desc->layout != LEECH_PLANES14)
    return set_error(LEECH_E_LAYOUT, "rotated GEMVs serve the PLANES14 layout");
  rc = set_groups(desc, n_groups, group_rows, group_centroids, a);
  if (rc) return rc;
  if (K <= 0 || K > desc->Kpad || K % 8)
    return set_error(LEECH_E_SHAPE, "need 0 < K <= Kpad and K a multiple of 8");
  const int64_t n = K & -K;
  int k = 0;
  while ((int64_t)1 << k < n) ++k;
  if (k > 15) return set_error(LEECH_E_SHAPE, "power-of-two factor of K above 32768");
  if (K > (int64_t)8 * kRotG * 64 * a.waves)
    return set_error(LEECH_E_SHAPE, "K too large for a fused rotation at this shape");
  if ((uintptr_t)d_signs & 7) return set_error(LEECH_E_ARG, "misaligned device pointer");
  a.x = nullptr;
  a.xraw = d_x;
  a.signs = d_signs;
  a.K = K;
  a.rot_k = k;
  a.rot_norm = (float)(1.0 / std::sqrt((double)n));
  return launch_gemv_rotated(a, (hipStream_t)stream);
}

int leech_gemv_grouped(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                       const void* d_side1, const void* d_class_table, const void* d_codewords,
                       const uint16_t* d_scale, int n_groups, const int64_t* group_rows,
                       const float* group_centroids, const uint16_t* d_x, float* d_y,
                       void* stream) {
  clear_error();
  if (!group_rows || !group_centroids) return set_error(LEECH_E_ARG, "NULL argument");
  GemvArgs a;
  int rc = gemv_setup(desc, d_main, d_side0, d_side1, d_class_table, d_codewords, d_scale, d_x,
                      d_y, &a);
  if (rc) return rc;
  rc = set_groups(desc, n_groups, group_rows, group_centroids, a);
  if (rc) return rc;
  return gemv_dispatch(desc, a, (hipStream_t)stream);
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

int leech_set_exception_mode(int mode) {
  clear_error();
  if (mode != LEECH_EXC_HOISTED && mode != LEECH_EXC_INLINE)
    return set_error(LEECH_E_ARG, "exception mode must be LEECH_EXC_HOISTED or LEECH_EXC_INLINE");
  g_exc_mode.store(mode, std::memory_order_relaxed);
  return LEECH_OK;
}

int leech_set_batch_mode(int mode) {
  clear_error();
  if (mode != LEECH_BATCH_AUTO && mode != LEECH_BATCH_DOT2)
    return set_error(LEECH_E_ARG, "batch mode must be LEECH_BATCH_AUTO or LEECH_BATCH_DOT2");
  g_batch_mode.store(mode, std::memory_order_relaxed);
  return LEECH_OK;
}

int leech_set_prologue_mode(int mode) {
  clear_error();
  if (mode != LEECH_PROLOGUE_AUTO && (mode < 0 || mode > 2))
    return set_error(LEECH_E_ARG, "prologue mode must be LEECH_PROLOGUE_AUTO, 0, 1 or 2");
  g_pro_mode.store(mode, std::memory_order_relaxed);
  return LEECH_OK;
}

int leech_gemv_phases(const leech_layout_desc* desc, const void* d_main, const void* d_side0,
                      const void* d_side1, const void* d_class_table, const void* d_codewords,
                      const uint16_t* d_scale, const float centroid[2], const uint16_t* d_x,
                      float* d_y, uint64_t* d_stamps, void* stream) {
  clear_error();
  if (!centroid || !d_stamps) return set_error(LEECH_E_ARG, "NULL argument");
  if ((uintptr_t)d_stamps & 7) return set_error(LEECH_E_ARG, "misaligned device pointer");
  GemvArgs a;
  int rc = gemv_setup(desc, d_main, d_side0, d_side1, d_class_table, d_codewords, d_scale, d_x,
                      d_y, &a);
  if (rc) return rc;
  if (desc->layout != LEECH_PLANES14)
    return set_error(LEECH_E_LAYOUT, "phase stamps are recorded for the PLANES14 layout");
  a.cen0 = centroid[0];
  a.cen1 = centroid[1];
  a.stamps = d_stamps;
  return launch_gemv<LEECH_PLANES14, 1, true>(a, (hipStream_t)stream);
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
