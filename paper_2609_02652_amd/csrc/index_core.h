// Format-v1 block codes (§2.1 "What a Λ24 index is"; §2.2 "Unfolding at load
// time"): the 47-bit direction index of a point of the ball Λ24(12) plus the
// gain bit, and its conversion to and from decoded fields.  Shared by the host
// library (encode, decode) and the GPU transcoder (decode), which read the
// same table.  Not part of the public ABI.
//
// The order (mixed radix, most significant digit first):
//   index = offset(class) + r, classes in id order;
//   even class, support = {i : |x_i| ≡ 2 mod 4} (a codeword of weight w):
//     r = ((((k_cw · A + a_sup) · B + a_off) · 2^f0 + s_off) · 2^f2 + s_sup)
//     k_cw   rank of the support among the weight-w codewords in ascending value
//     a_sup  arrangement of the ≡ 2 (mod 4) magnitudes over the support
//     a_off  arrangement of the ≡ 0 (mod 4) magnitudes over the other coordinates
//     s_off  signs of the f0 nonzero off-support coordinates (bit j: the j-th
//            of them in increasing order, 1 = negative)
//     s_sup  signs of the first f2 = w − 1 support coordinates; the last one
//            takes the sign that makes Σx ≡ 0 (mod 8)
//   odd class: r = k_cw · A + a_all, k_cw the rank of {i : x_i ≡ 3 mod 4}
//     among all codewords in ascending value, a_all the arrangement over all
//     24 coordinates, signs forced by the codeword.
// An arrangement is one digit per level of the side in ascending order: the
// colex rank Σ_j C(q_j, j) of the level's positions, q_1 < … < q_c counted
// among the positions the smaller levels left free, radix C(free, c).
#pragma once

#include <cstdint>

#include "leech_internal.h"

namespace leech {

constexpr int kIndexBits = 47;
constexpr uint64_t kIndexMask = (1ull << kIndexBits) - 1;

struct IdxClass {            // 48 bytes
  uint64_t offset;           // first index of the class
  uint64_t A;                // radix of the support arrangement (odd: all 24 coordinates)
  uint64_t B;                // radix of the off-support arrangement (odd: 1)
  uint8_t parity, w, f0, f2; // w: support weight (even classes)
  uint8_t n_levels;
  uint8_t side;              // bit k: level k lies on the support (odd: every level)
  uint8_t count[kMaxLevels]; // multiplicity of level k
  uint8_t mag[kMaxLevels];   // magnitude of level k
  uint8_t sum8;              // Σ |z_i| mod 8 over the class's multiset
  uint8_t pad[5];
};
static_assert(sizeof(IdxClass) == 48, "index class record is 48 bytes");

struct IdxTable {
  uint64_t n_points;               // N: indices run over [0, N)
  uint32_t n_classes, reserved;
  IdxClass cls[kTableSlots];
  uint32_t cw_value[4096];         // codewords in ascending value
  uint32_t cw_weight[4096];        // codewords by (weight, value)
  uint32_t weight_start[32];       // cw_weight position of the first codeword of weight w
  uint32_t binom[25][32];          // C(n, k) for n, k ≤ 24; zero for k > n
};

__host__ __device__ inline int idx_popc(uint32_t v) { return __builtin_popcount(v); }
__host__ __device__ inline int idx_top(uint32_t v) { return 31 - __builtin_clz(v); }

// bits of s deposited, in order, at the set bits of mask (lowest first)
__host__ __device__ inline uint32_t idx_deposit(uint32_t s, uint32_t mask) {
  uint32_t out = 0;
  for (int j = 0; mask; ++j) {
    const uint32_t low = mask & (0u - mask);
    if (s >> j & 1) out |= low;
    mask ^= low;
  }
  return out;
}

// the bits of v at the set bits of mask, packed (lowest first)
__host__ __device__ inline uint32_t idx_extract(uint32_t v, uint32_t mask) {
  uint32_t out = 0;
  for (int j = 0; mask; ++j) {
    const uint32_t low = mask & (0u - mask);
    if (v & low) out |= 1u << j;
    mask ^= low;
  }
  return out;
}

// q = a / d and a − q·d for a < 2^48 and 0 < d < 2^48: both convert to double
// exactly, the rounded quotient is within one of the true one, and one integer
// correction in each direction makes it exact.  (A 64-bit integer division is
// a long instruction sequence on the GPU; this is a handful.)
__host__ __device__ inline uint64_t idx_divmod(uint64_t a, uint64_t d, uint64_t* rem) {
  uint64_t q = (uint64_t)((double)a / (double)d);
  if (q * d > a) --q;
  else if (a - q * d >= d) ++q;
  *rem = a - q * d;
  return q;
}

__host__ __device__ inline int idx_find_class(const IdxTable& T, uint64_t idx) {
  int lo = 0, hi = (int)T.n_classes - 1;     // largest c with offset(c) ≤ idx
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (T.cls[mid].offset <= idx) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Arrangement a of the levels in `on` over the positions in `pos`: each
// level's positions go into the level-code planes (code = level + 1, bit b in
// planes[b]), into `zero` if its magnitude is 0 and into `mag3` if it is
// ≡ 3 (mod 4).  Loops run over the five level slots so that every array index
// is a constant.
__host__ __device__ inline void idx_place(const IdxTable& T, const IdxClass& c, uint32_t on,
                                          uint32_t pos, uint64_t a, uint32_t planes[3],
                                          uint32_t* zero, uint32_t* mag3) {
  on &= (1u << c.n_levels) - 1;
  if (!on) return;
  uint32_t radix[kMaxLevels], digit[kMaxLevels];
  int left = idx_popc(pos);
#pragma unroll
  for (int k = 0; k < kMaxLevels; ++k) {
    radix[k] = 1;
    if (on >> k & 1) {
      radix[k] = T.binom[left][c.count[k]];
      left -= c.count[k];
    }
  }
#pragma unroll
  for (int k = kMaxLevels - 1; k >= 0; --k) {
    digit[k] = 0;
    if (radix[k] > 1) {
      uint64_t rem;
      a = idx_divmod(a, radix[k], &rem);
      digit[k] = (uint32_t)rem;
    }
  }
  const int last = idx_top(on);
  uint32_t free = pos;
  int nfree = idx_popc(pos);
#pragma unroll
  for (int k = 0; k < kMaxLevels; ++k) {
    if (!(on >> k & 1)) continue;
    uint32_t take = 0;
    if (k == last) {
      take = free;
    } else {
      uint32_t d = digit[k], scan = free;
      for (int j = c.count[k], q = nfree - 1; j > 0; --q) {
        const int p = idx_top(scan);
        const uint32_t b = T.binom[q][j];
        if (b <= d) {
          d -= b;
          take |= 1u << p;
          --j;
        }
        scan &= ~(1u << p);
      }
    }
    const int code = level_code(k);
#pragma unroll
    for (int b = 0; b < 3; ++b)
      if (code >> b & 1) planes[b] |= take;
    if (c.mag[k] == 0) *zero |= take;
    if ((c.mag[k] & 3) == 3) *mag3 |= take;
    free &= ~take;
    nfree -= c.count[k];
  }
}

// Rank of the arrangement of the levels in `on` over the positions in `pos`.
__host__ __device__ inline uint64_t idx_rank(const IdxTable& T, const IdxClass& c, uint32_t on,
                                             uint32_t pos, const uint8_t* level) {
  uint64_t a = 0;
  uint32_t free = pos;
  int nfree = idx_popc(pos);
  for (int k = 0; k < c.n_levels; ++k) {
    if (!(on >> k & 1)) continue;
    uint32_t mine = 0;
    for (uint32_t m = free; m; m &= m - 1) {
      const int p = __builtin_ctz(m);
      if (level[p] == k) mine |= 1u << p;
    }
    uint32_t d = 0;
    int j = 1;
    for (uint32_t m = mine; m; m &= m - 1, ++j) {
      const int p = __builtin_ctz(m);
      d += T.binom[idx_popc(free & ((1u << p) - 1))][j];
    }
    a = a * T.binom[nfree][c.count[k]] + d;
    free &= ~mine;
    nfree -= c.count[k];
  }
  return a;
}

// Decoded fields of a 48-bit code as the three level-code planes (bit i of
// planes[b] = bit b of coordinate i's level + 1) and the sign mask; false if
// the code is not one (bits above 47 set, or an index ≥ N).
__host__ __device__ inline bool idx_decode(const IdxTable& T, uint64_t code, uint16_t* cls,
                                           uint8_t* gain, uint32_t* smask, uint32_t planes[3]) {
  if (code >> 48) return false;
  const uint64_t idx = code & kIndexMask;
  if (idx >= T.n_points) return false;
  const int ci = idx_find_class(T, idx);
  const IdxClass& c = T.cls[ci];
  uint64_t r = idx - c.offset;
  uint32_t zero = 0, mag3 = 0, neg;
  planes[0] = planes[1] = planes[2] = 0;
  const uint32_t all_levels = (1u << c.n_levels) - 1;
  if (c.parity == 0) {
    const uint32_t s_sup = (uint32_t)(r & ((1ull << c.f2) - 1));
    r >>= c.f2;
    const uint32_t s_off = (uint32_t)(r & ((1ull << c.f0) - 1));
    r >>= c.f0;
    uint64_t a_off, a_sup;
    r = idx_divmod(r, c.B, &a_off);
    const uint64_t k_cw = idx_divmod(r, c.A, &a_sup);
    const uint32_t cw = T.cw_weight[T.weight_start[c.w] + (uint32_t)k_cw];
    idx_place(T, c, c.side, cw, a_sup, planes, &zero, &mag3);
    idx_place(T, c, all_levels & ~(uint32_t)c.side, ~cw & 0xFFFFFFu, a_off, planes, &zero, &mag3);
    // flipping an off-support coordinate (|z| ≡ 0 mod 4) moves Σz by a multiple
    // of 8, a support one (|z| ≡ 2 mod 4) by 4: the last support sign is set
    // when Σ|z| + 4·(negative support coordinates) is not ≡ 0 (mod 8)
    const uint32_t top = cw ? 1u << idx_top(cw) : 0u;
    neg = idx_deposit(s_off, ~zero & ~cw & 0xFFFFFFu) | idx_deposit(s_sup, cw & ~top);
    if (top && ((c.sum8 + 4 * idx_popc(neg & cw)) & 7)) neg |= top;
  } else {
    uint64_t a_all;
    const uint64_t k_cw = idx_divmod(r, c.A, &a_all);
    const uint32_t cw = T.cw_value[(uint32_t)k_cw];
    idx_place(T, c, all_levels, 0xFFFFFFu, a_all, planes, &zero, &mag3);
    neg = cw ^ mag3;
  }
  *cls = (uint16_t)ci;
  *gain = (uint8_t)(code >> kIndexBits & 1);
  *smask = neg;
  return true;
}

// 48-bit code of a block given as decoded fields that were already checked to
// form a point of the ball; false if its sign pattern or codeword is not one
// the index can name (not a lattice point).
__host__ __device__ inline bool idx_encode(const IdxTable& T, uint16_t cls, uint8_t gain,
                                           uint32_t smask, const uint8_t* level, uint64_t* code) {
  const IdxClass& c = T.cls[cls];
  uint64_t r;
  if (c.parity == 0) {
    uint32_t cw = 0, nonzero = 0;
    for (int i = 0; i < kDim; ++i) {
      if (c.side >> level[i] & 1) cw |= 1u << i;
      if (c.mag[level[i]]) nonzero |= 1u << i;
    }
    const uint32_t lo = T.weight_start[c.w], hi = T.weight_start[c.w + 1];
    uint32_t a = lo, b = hi;             // binary search for cw among weight-w codewords
    while (a < b) {
      const uint32_t mid = (a + b) >> 1;
      if (T.cw_weight[mid] < cw) a = mid + 1;
      else b = mid;
    }
    if (a >= hi || T.cw_weight[a] != cw) return false;
    const uint32_t top = cw ? 1u << idx_top(cw) : 0u;
    const uint32_t s_off = idx_extract(smask, nonzero & ~cw);
    const uint32_t s_sup = idx_extract(smask, cw & ~top);
    int sum = 0;
    for (int i = 0; i < kDim; ++i) sum += (smask >> i & 1) ? -c.mag[level[i]] : c.mag[level[i]];
    if (sum & 7) return false;
    const uint64_t a_sup = idx_rank(T, c, c.side, cw, level);
    const uint64_t a_off =
        idx_rank(T, c, ~(uint32_t)c.side & ((1u << c.n_levels) - 1), ~cw & 0xFFFFFFu, level);
    r = (a - lo) * c.A + a_sup;
    r = r * c.B + a_off;
    r = (r << c.f0 | s_off) << c.f2 | s_sup;
  } else {
    uint32_t mag3 = 0;
    for (int i = 0; i < kDim; ++i)
      if ((c.mag[level[i]] & 3) == 3) mag3 |= 1u << i;
    const uint32_t cw = (smask ^ mag3) & 0xFFFFFFu;
    uint32_t a = 0, b = 4096;
    while (a < b) {
      const uint32_t mid = (a + b) >> 1;
      if (T.cw_value[mid] < cw) a = mid + 1;
      else b = mid;
    }
    if (a >= 4096 || T.cw_value[a] != cw) return false;
    r = (uint64_t)a * c.A + idx_rank(T, c, c.side, 0xFFFFFFu, level);
  }
  *code = (c.offset + r) | (uint64_t)(gain & 1) << kIndexBits;
  return true;
}

}  // namespace leech
