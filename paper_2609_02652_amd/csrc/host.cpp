// Host half of libleech: the Λ24(12) codebook, decoded fields, the offline
// expansion into the four VRAM layouts, and a host decode for verification.
//
// Paper: §2.1 (the lattice, its ball and classes), §2.2 (the load-time
// transcoder: decoded fields -> byte layouts), §2.3 (the class table),
// §3.2 (the four layouts: Slot32, Planes14, Planes12x, Golay70).

#include <atomic>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <thread>
#include <unordered_map>
#include <vector>

#include "index_core.h"
#include "leech_internal.h"

namespace leech {

// ---------------------------------------------------------------- errors
static thread_local std::string g_error;

int set_error(int code, const std::string& msg) {
  g_error = msg;
  return code;
}
void clear_error() { g_error.clear(); }

static std::string fmt(const char* f, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, f);
  vsnprintf(buf, sizeof buf, f, ap);
  va_end(ap);
  return buf;
}

void choose_geometry(int64_t M, int64_t nb, int* C_out, int* R_out) {
  // A launch runs its tiles on the 256 CUs in L = ceil(tiles / 256) rounds.
  // Each tile's waves (at most 8) split its units; a wave's units follow one
  // another through its prefetch ring, so a round lasts at least the units
  // per wave, and the whole launch at least the unit steps of all tiles over
  // what the CUs retire together.  Cost, in unit steps:
  //     L · 5 + max(L · units per wave, tiles · units per tile / (256 · 7))
  // (5: a tile's staging, ramp and reduction; 7 unit steps in flight per
  // CU), plus, for three to six rounds, 1.5 · (L − tiles / 256) · units per
  // wave for the CUs a partial last round leaves idle (over more rounds the
  // CUs' uneven finishing spreads the last tiles out).  The least cost wins;
  // ties go to more blocks per unit (idle lanes cost issue slots but move no
  // bytes), then to more tiles.
  // A CU holds two workgroups at once.  Where the choice is one round of 9
  // to 17 units per wave, the prefetch ramp is a large part of each wave's
  // time, and two tiles per CU, each half as long, overlap their ramps: the
  // choice then moves to 257..512 tiles of at least 48 blocks per unit with
  // at most half the units per wave (rounded up, plus one) and no more rows
  // per CU, the most blocks per unit first, then the fewest rows per CU,
  // then the most tiles.  Fitted to per-geometry timings of 27 shapes from
  // 2048 to 34816 rows (bench --geometry-sweep --geometry-all): 4096 rows ×
  // 171 blocks take 4 columns × 16 rows; 5120 rows × 214 or 726 blocks 3 × 20
  // (256 tiles, against 160 of 2 × 32: 6.3 against 6.7 µs and 12.9 against
  // 14.7 µs); 8192 × 342 takes 2 × 32; 8192 × 171 and 6144 × 171 take
  // 4 × 16 (512 and 384 tiles: 6.6 against 7.3 µs for 2 × 32 at 8192 rows);
  // 34816 × 214 takes 2 × 28 (1244 tiles in 4.9 rounds, against 1088 of
  // 2 × 32 in 4.25: 23.6 against 24.5 µs); 14336 × 171 and 152064 × 214
  // take 1 × 64.
  constexpr int64_t kCUs = 256;
  constexpr double kTileFixedUnits = 5.0, kUnitsInFlight = 7.0, kIdleTail = 1.5;
  static const int kCols[] = {1, 2, 3, 4, 8, 16};
  auto shape = [&](int C, int R, int64_t& tiles, int64_t& per_wave, int64_t& L) {
    tiles = (M + R - 1) / R;
    const int64_t groups = (nb + C - 1) / C;
    const int64_t waves = std::min<int64_t>(8, groups);
    per_wave = (groups + waves - 1) / waves;
    L = (tiles + kCUs - 1) / kCUs;
    return groups;
  };
  double best_cost = 0.0;
  int64_t best_tiles = 0;
  int best_lanes = 0, bc = 0, br = 0;
  for (int C : kCols)
    for (int R = 4; R * C <= kWave; R += 4) {
      int64_t tiles, per_wave, L;
      const int64_t groups = shape(C, R, tiles, per_wave, L);
      double cost = (double)L * kTileFixedUnits +
                    std::max((double)(L * per_wave),
                             (double)tiles * (double)groups / (kCUs * kUnitsInFlight));
      if (L >= 3 && L <= 6)
        cost += kIdleTail * ((double)L - (double)tiles / kCUs) * (double)per_wave;
      const int lanes = R * C;
      if (bc == 0 || cost < best_cost ||
          (cost == best_cost &&
           (lanes > best_lanes || (lanes == best_lanes && tiles > best_tiles)))) {
        best_cost = cost;
        best_tiles = tiles;
        best_lanes = lanes;
        bc = C;
        br = R;
      }
    }
  int64_t t1, s1, l1;
  shape(bc, br, t1, s1, l1);
  if (l1 == 1 && s1 >= 9 && s1 <= 17) {
    int pc = 0, pr = 0, p_lanes = 0;
    int64_t p_rows = 0, p_tiles = 0;
    for (int C : kCols)
      for (int R = 4; R * C <= kWave; R += 4) {
        int64_t tiles, per_wave, L;
        shape(C, R, tiles, per_wave, L);
        const int lanes = R * C;
        const int64_t rows = L * R;
        if (tiles <= kCUs || tiles > 2 * kCUs || lanes < 48 || per_wave > (s1 + 1) / 2 + 1 ||
            rows > br)
          continue;
        if (pc == 0 || lanes > p_lanes || (lanes == p_lanes && rows < p_rows) ||
            (lanes == p_lanes && rows == p_rows && tiles > p_tiles)) {
          pc = C;
          pr = R;
          p_lanes = lanes;
          p_rows = rows;
          p_tiles = tiles;
        }
      }
    if (pc != 0) {
      bc = pc;
      br = pr;
    }
  }
  *C_out = bc;
  *R_out = br;
}

// ------------------------------------------------------ extended Golay code
// Cyclic [23,12,7] code generated by g(x) = 1 + x^2 + x^4 + x^5 + x^6 + x^10 +
// x^11 (coordinate i = coefficient of x^i), extended by a parity bit at 23.
// Codeword of a 12-bit message m: Σ_k m_k · x^k g(x), then the parity bit.
static uint32_t encode_golay(uint32_t msg) {
  const uint32_t g = (1u << 0) | (1u << 2) | (1u << 4) | (1u << 5) | (1u << 6) | (1u << 10) |
                     (1u << 11);
  uint32_t c = 0;
  for (int k = 0; k < 12; ++k)
    if (msg >> k & 1) c ^= g << k;
  return c | (uint32_t)(__builtin_popcount(c) & 1) << 23;
}

static std::vector<uint32_t> make_codewords() {
  std::vector<uint32_t> words;
  words.reserve(4096);
  for (uint32_t msg = 0; msg < 4096; ++msg) words.push_back(encode_golay(msg));
  std::sort(words.begin(), words.end());
  return words;
}

// The encoding is linear, so the codeword of m is the XOR of the codewords of
// its low and high six bits: gen[m & 63] ^ gen[64 + (m >> 6)].
static std::vector<uint32_t> make_golay_gen() {
  std::vector<uint32_t> gen(128);
  for (uint32_t a = 0; a < 64; ++a) {
    gen[a] = encode_golay(a);
    gen[64 + a] = encode_golay(a << 6);
  }
  return gen;
}

// --------------------------------------------------------------- classes
struct HostClass {
  int shell = 0, parity = 0, n_levels = 0;
  uint8_t levels[kMaxLevels] = {0};
  uint8_t mult[14] = {0};          // multiplicity of each magnitude 0..13
  uint8_t mags_desc[kDim] = {0};
  uint64_t size = 0;
};

// exact binomial in 128 bits
static unsigned __int128 binom(int n, int k) {
  if (k < 0 || k > n) return 0;
  unsigned __int128 r = 1;
  for (int i = 1; i <= k; ++i) r = r * (unsigned)(n - k + i) / (unsigned)i;
  return r;
}

// orderings of a multiset given its multiplicities
static unsigned __int128 arrangements(const std::vector<int>& counts) {
  int n = 0;
  for (int c : counts) n += c;
  unsigned __int128 r = 1;
  for (int c : counts) {
    r *= binom(n, c);
    n -= c;
  }
  return r;
}

// Points with the given magnitude multiplicities (§2.1 membership conditions):
// even — codeword of weight w on the ≡2 (mod 4) coordinates, arrangements on
// and off it, free signs off it, half the sign patterns on it (all or none
// when w = 0, by the sum mod 8); odd — any codeword, any arrangement, signs
// forced, valid iff #{|x| ≡ 3, 5 (mod 8)} is odd.
static uint64_t points_in_multiset(const uint8_t mult[14], int parity,
                                   const int weight_count[25]) {
  unsigned __int128 total;
  if (parity == 0) {
    std::vector<int> two, zero;
    int w = 0, nz0 = 0, n4 = 0;
    for (int a = 0; a <= 13; ++a) {
      if (!mult[a]) continue;
      if (a & 1) return 0;
      if (a % 4 == 2) {
        two.push_back(mult[a]);
        w += mult[a];
      } else {
        zero.push_back(mult[a]);
        if (a) nz0 += mult[a];
        if (a % 8 == 4) n4 += mult[a];
      }
    }
    if (w > 24 || weight_count[w] == 0) return 0;
    unsigned __int128 signs;
    if (w > 0)
      signs = (unsigned __int128)1 << (w - 1);
    else
      signs = (n4 % 2 == 0) ? 1 : 0;
    total = (unsigned __int128)weight_count[w] * arrangements(two) * arrangements(zero) *
            ((unsigned __int128)1 << nz0) * signs;
  } else {
    std::vector<int> all;
    int t = 0;
    for (int a = 0; a <= 13; ++a) {
      if (!mult[a]) continue;
      if (!(a & 1)) return 0;
      all.push_back(mult[a]);
      if (a % 8 == 3 || a % 8 == 5) t += mult[a];
    }
    if (t % 2 == 0) return 0;
    total = (unsigned __int128)4096 * arrangements(all);
  }
  return (uint64_t)total;
}

static void enumerate_multisets(int remaining, int maxa, int parity, int slots, uint8_t* mult,
                                std::vector<std::vector<uint8_t>>& out) {
  if (slots == 0) {
    if (remaining == 0) out.emplace_back(mult, mult + 14);
    return;
  }
  // largest magnitude still allowed, same parity
  for (int a = maxa; a >= 0; --a) {
    if ((a & 1) != parity) continue;
    if (a * a > remaining) continue;
    if (a == 0) {  // all remaining slots are zero
      if (remaining == 0) {
        mult[0] += slots;
        out.emplace_back(mult, mult + 14);
        mult[0] -= slots;
      }
      continue;
    }
    mult[a]++;
    enumerate_multisets(remaining - a * a, a, parity, slots - 1, mult, out);
    mult[a]--;
  }
}

// key of a multiset: Σ count_a · 25^a, a = 1..13 (counts ≤ 24 < 25)
static uint64_t pow25[14];
static std::once_flag pow25_once;
static void init_pow25() {
  std::call_once(pow25_once, [] {
    uint64_t p = 1;
    pow25[0] = 0;
    for (int a = 1; a <= 13; ++a) {
      pow25[a] = p;
      p *= 25;
    }
  });
}

}  // namespace leech

using namespace leech;

struct leech_codebook {
  int ball_m = 12;
  std::vector<HostClass> classes;
  uint64_t n_points = 0;
  std::vector<uint32_t> codewords;
  std::vector<uint32_t> golay_gen;    // LEECH_TABLE_GOLAY_GEN
  std::unordered_map<uint32_t, uint16_t> message_of;   // codeword -> 12-bit message
  std::vector<uint64_t> golay_bits;   // 2^24-bit membership bitmap
  std::unordered_map<uint64_t, int> by_key;
  std::vector<uint8_t> tab_levels;    // LEECH_TABLE_CLASS_LEVELS
  std::vector<uint8_t> tab_device;    // LEECH_TABLE_DEVICE
  std::vector<uint8_t> tab_index;     // LEECH_TABLE_INDEX (balls with N < 2^47)
  int g70_count[kTableSlots][2] = {{0}};

  bool is_codeword(uint32_t m) const { return golay_bits[m >> 6] >> (m & 63) & 1; }
};

namespace leech {

static void build_golay70_values(leech_codebook* cb, int id, DevClass& dc) {
  // Candidates per side with their frequency under uniform sampling:
  // even points: side 1 = |z| ≡ 2 (mod 4) (±a, each half the multiplicity),
  //              side 0 = |z| ≡ 0 (mod 4) (0 once, ±a halves);
  // odd points:  side 1 = z ≡ 3 (mod 4), side 0 = z ≡ 1 (mod 4); the sign of
  //              each magnitude is forced, frequency = its multiplicity.
  // Keep the four most frequent per side (ties: smaller |v|, then v > 0).
  const HostClass& c = cb->classes[id];
  for (int side = 0; side < 2; ++side) {
    struct Cand { int v; int twice_freq; };
    std::vector<Cand> cand;
    for (int k = 0; k < c.n_levels; ++k) {
      int a = c.levels[k];
      int m = c.mult[a];
      if (c.parity == 0) {
        if ((a % 4 == 2) != (side == 1)) continue;
        if (a == 0) cand.push_back({0, 2 * m});
        else {
          cand.push_back({a, m});
          cand.push_back({-a, m});
        }
      } else {
        int want = side ? 3 : 1;
        int v = (a % 4 == want) ? a : -a;
        cand.push_back({v, 2 * m});
      }
    }
    std::stable_sort(cand.begin(), cand.end(), [](const Cand& x, const Cand& y) {
      if (x.twice_freq != y.twice_freq) return x.twice_freq > y.twice_freq;
      if (std::abs(x.v) != std::abs(y.v)) return std::abs(x.v) < std::abs(y.v);
      return x.v > y.v;
    });
    int n = (int)std::min<size_t>(4, cand.size());
    for (int k = 0; k < 4; ++k) dc.g70[side][k] = (int8_t)(k < n ? cand[k].v : 0);
    cb->g70_count[id][side] = n;
  }
}

// Format-v1 index table (§2.1): class offsets and radices, the codewords in
// the two orders the index ranks them by, and binomial coefficients.
static void build_index_table(leech_codebook* cb, const int weight_count[25]) {
  cb->tab_index.assign(sizeof(IdxTable), 0);
  IdxTable& T = *reinterpret_cast<IdxTable*>(cb->tab_index.data());
  T.n_points = cb->n_points;
  T.n_classes = (uint32_t)cb->classes.size();
  for (int n = 0; n <= 24; ++n)
    for (int k = 0; k <= n; ++k) T.binom[n][k] = (uint32_t)binom(n, k);
  std::vector<uint32_t> byw = cb->codewords;
  std::stable_sort(byw.begin(), byw.end(), [](uint32_t a, uint32_t b) {
    return __builtin_popcount(a) < __builtin_popcount(b);
  });
  for (int i = 0; i < 4096; ++i) {
    T.cw_value[i] = cb->codewords[i];
    T.cw_weight[i] = byw[i];
  }
  uint32_t start = 0;
  for (int w = 0; w < 32; ++w) {
    T.weight_start[w] = start;
    if (w <= 24) start += (uint32_t)weight_count[w];
  }
  uint64_t offset = 0;
  for (size_t i = 0; i < cb->classes.size(); ++i) {
    const HostClass& h = cb->classes[i];
    IdxClass& c = T.cls[i];
    c.offset = offset;
    offset += h.size;
    c.parity = (uint8_t)h.parity;
    c.n_levels = (uint8_t)h.n_levels;
    std::vector<int> on, off;
    int f0 = 0;
    for (int k = 0; k < h.n_levels; ++k) {
      const int a = h.levels[k];
      c.mag[k] = (uint8_t)a;
      c.count[k] = h.mult[a];
      const bool support = h.parity ? true : a % 4 == 2;
      if (support) {
        c.side |= (uint8_t)(1u << k);
        on.push_back(h.mult[a]);
      } else {
        off.push_back(h.mult[a]);
        if (a) f0 += h.mult[a];
      }
    }
    int w = 0;
    for (int x : on) w += x;
    c.w = (uint8_t)(h.parity ? 0 : w);
    c.f0 = (uint8_t)(h.parity ? 0 : f0);
    c.f2 = (uint8_t)(h.parity || w == 0 ? 0 : w - 1);
    int sum = 0;
    for (int k = 0; k < h.n_levels; ++k) sum += h.levels[k] * h.mult[h.levels[k]];
    c.sum8 = (uint8_t)(sum & 7);
    c.A = (uint64_t)arrangements(on);
    c.B = (uint64_t)arrangements(off);
  }
}

static int build_codebook(int ball_m, leech_codebook* cb) {
  init_pow25();
  cb->ball_m = ball_m;
  cb->codewords = make_codewords();
  cb->golay_gen = make_golay_gen();
  for (uint32_t m = 0; m < 4096; ++m) cb->message_of[encode_golay(m)] = (uint16_t)m;
  cb->golay_bits.assign((1u << 24) / 64, 0);
  int weight_count[25] = {0};
  for (uint32_t c : cb->codewords) {
    cb->golay_bits[c >> 6] |= 1ull << (c & 63);
    weight_count[__builtin_popcount(c)]++;
  }
  for (int m = 2; m <= ball_m; ++m) {
    for (int parity = 0; parity < 2; ++parity) {
      std::vector<std::vector<uint8_t>> sets;
      uint8_t mult[14] = {0};
      int maxa = (int)std::sqrt((double)(16 * m)) + 1;
      if (maxa > 13) maxa = 13;
      enumerate_multisets(16 * m, maxa, parity, kDim, mult, sets);
      for (auto& s : sets) {
        uint64_t size = points_in_multiset(s.data(), parity, weight_count);
        if (!size) continue;
        HostClass hc;
        hc.shell = m;
        hc.parity = parity;
        hc.size = size;
        int pos = 0;
        for (int a = 13; a >= 0; --a)
          for (int k = 0; k < s[a]; ++k) hc.mags_desc[pos++] = (uint8_t)a;
        for (int a = 0; a <= 13; ++a) {
          hc.mult[a] = s[a];
          if (s[a]) hc.levels[hc.n_levels++] = (uint8_t)a;
        }
        cb->classes.push_back(hc);
      }
    }
  }
  // canonical order: (shell, parity, descending magnitudes lexicographic)
  std::stable_sort(cb->classes.begin(), cb->classes.end(),
                   [](const HostClass& a, const HostClass& b) {
                     if (a.shell != b.shell) return a.shell < b.shell;
                     if (a.parity != b.parity) return a.parity < b.parity;
                     return std::lexicographical_compare(a.mags_desc, a.mags_desc + kDim,
                                                         b.mags_desc, b.mags_desc + kDim);
                   });
  if ((int)cb->classes.size() > kTableSlots)
    return set_error(LEECH_E_CAPACITY, "more classes than table slots");
  cb->n_points = 0;
  for (size_t i = 0; i < cb->classes.size(); ++i) {
    const HostClass& c = cb->classes[i];
    cb->n_points += c.size;
    uint64_t key = 0;
    for (int a = 1; a <= 13; ++a) key += c.mult[a] * pow25[a];
    cb->by_key[key] = (int)i;
  }
  // paper's class table (§2.3): five f32 levels a/(4√m) and a u32 count
  cb->tab_levels.assign(kTableSlots * 24, 0);
  cb->tab_device.assign(LEECH_DEVICE_TABLE_BYTES, 0);
  for (size_t i = 0; i < cb->classes.size(); ++i) {
    const HostClass& c = cb->classes[i];
    double norm = 4.0 * std::sqrt((double)c.shell);
    float lv[kMaxLevels] = {0};
    for (int k = 0; k < c.n_levels; ++k) lv[k] = (float)(c.levels[k] / norm);
    uint32_t cnt = (uint32_t)c.n_levels;
    std::memcpy(&cb->tab_levels[i * 24], lv, sizeof lv);
    std::memcpy(&cb->tab_levels[i * 24 + 20], &cnt, 4);
    DevClass dc;
    std::memset(&dc, 0, sizeof dc);
    for (int k = 0; k < c.n_levels; ++k) dc.perm[level_code(k)] = c.levels[k];
    dc.perm[kSignByteCode] = 0x80;
    dc.inv_norm = (float)(1.0 / norm);
    dc.info = (uint32_t)c.n_levels | (uint32_t)c.parity << 8 | (uint32_t)c.shell << 16;
    build_golay70_values(cb, (int)i, dc);
    for (int k = 0; k < 8; ++k) {
      int v = dc.g70[k >> 2][k & 3];
      dc.g70abs[k] = (uint8_t)(v < 0 ? -v : v);
      if (v < 0) dc.info |= 1u << (24 + k);
    }
    std::memcpy(&cb->tab_device[i * sizeof(DevClass)], &dc, sizeof dc);
  }
  if (cb->n_points <= kIndexMask + 1) build_index_table(cb, weight_count);
  return LEECH_OK;
}

// ------------------------------------------------------- block validation
// Integer point of one block from its fields; returns 0 or a LEECH_E_* code.
static int fields_to_point(const leech_codebook* cb, uint16_t cls, uint32_t smask,
                           const uint8_t* level, int8_t* z, const char** why) {
  if (cls >= cb->classes.size()) {
    *why = "class id out of range";
    return LEECH_E_FIELD;
  }
  if (smask >> kDim) {
    *why = "sign mask has bits above coordinate 23";
    return LEECH_E_FIELD;
  }
  const HostClass& c = cb->classes[cls];
  uint8_t seen[14] = {0};
  for (int i = 0; i < kDim; ++i) {
    if (level[i] >= c.n_levels) {
      *why = "level beyond the class's level count";
      return LEECH_E_FIELD;
    }
    int a = c.levels[level[i]];
    bool neg = smask >> i & 1;
    if (neg && a == 0) {
      *why = "sign bit on a zero coordinate";
      return LEECH_E_FIELD;
    }
    seen[a]++;
    z[i] = (int8_t)(neg ? -a : a);
  }
  if (std::memcmp(seen, c.mult, 14) != 0) {
    *why = "levels do not form the class's magnitude multiset";
    return LEECH_E_FIELD;
  }
  // membership (§2.1): parity shared, residue set a codeword, sum mod 8
  int mu = z[0] & 1;
  uint32_t mask = 0;
  int sum = 0;
  for (int i = 0; i < kDim; ++i) {
    int r = ((z[i] % 4) + 4) % 4;
    if (r == (mu ? 3 : 2)) mask |= 1u << i;
    sum += z[i];
  }
  if (!cb->is_codeword(mask) || (((sum % 8) + 8) % 8) != 4 * mu) {
    *why = "fields decode to a vector outside the lattice";
    return LEECH_E_NOT_LATTICE;
  }
  return LEECH_OK;
}

// ------------------------------------------------------------- bit packing
static inline void put_bits(uint8_t* rec, int pos, uint64_t v, int n) {
  for (int k = 0; k < n; ++k)
    if (v >> k & 1) rec[(pos + k) >> 3] |= (uint8_t)(1u << ((pos + k) & 7));
}
static inline uint64_t get_bits(const uint8_t* rec, int pos, int n) {
  uint64_t v = 0;
  for (int k = 0; k < n; ++k) v |= (uint64_t)(rec[(pos + k) >> 3] >> ((pos + k) & 7) & 1) << k;
  return v;
}

// Planes14 record (§2.3): the three level-code planes and the sign plane (96
// bits) and the 10-bit class|gain entry, in 112 bits.  The 96 plane bits are
// stored in the order the GPU consumes them: three 32-bit pair words, each
// holding four pairs' byte-permute selectors, one per 4-bit rotation
// (leech_internal.h):
//   pair word 0 [0,32) | pair word 1 [32,64) | pair word 2 [64,96) |
//   class [96,105) | gain 105 | zero [106,112)
// The level code is level + 1, so codes run 1..5 and code 0 never occurs (the
// kernels keep the sign byte there).
static void pack_planes14(uint8_t* rec, uint16_t cls, uint8_t g, uint32_t smask,
                          const uint8_t* level) {
  uint8_t code[kDim];
  for (int i = 0; i < kDim; ++i) code[i] = (uint8_t)level_code(level[i]);
  uint32_t w[3];
  planes14_words(code, ~smask & 0xFFFFFFu, w);
  std::memset(rec, 0, kPlanes14Bytes);
  for (int k = 0; k < 3; ++k) put_bits(rec, kP14PairWordPos[k], w[k], 32);
  put_bits(rec, kP14ClassPos, cls, 9);
  put_bits(rec, kP14ClassPos + 9, g, 1);
}

static void unpack_planes14(const leech_codebook* cb, const uint8_t* rec, int8_t* z,
                            uint16_t* cls, uint8_t* g) {
  uint32_t w[3];
  for (int k = 0; k < 3; ++k) w[k] = (uint32_t)get_bits(rec, kP14PairWordPos[k], 32);
  uint8_t code[kDim];
  uint32_t pos;
  planes14_codes(w, code, &pos);
  const uint16_t c = (uint16_t)get_bits(rec, kP14ClassPos, 9);
  const DevClass* dc = (const DevClass*)cb->tab_device.data() + c;
  for (int i = 0; i < kDim; ++i) {
    int a = code[i] == kSignByteCode ? 0 : dc->perm[code[i]];
    z[i] = (int8_t)((pos >> i & 1) ? a : -a);
  }
  *cls = c;
  *g = (uint8_t)get_bits(rec, kP14ClassPos + 9, 1);
}

}  // namespace leech

// =================================================================== C ABI
extern "C" {

const char* leech_last_error(void) { return g_error.c_str(); }

int leech_codebook_build(int ball_m, leech_codebook** out) {
  clear_error();
  if (!out) return set_error(LEECH_E_ARG, "out is NULL");
  if (ball_m != 12 && ball_m != 13)
    return set_error(LEECH_E_ARG, fmt("ball_m must be 12 or 13 (got %d)", ball_m));
  leech_codebook* cb = new leech_codebook();
  int rc = build_codebook(ball_m, cb);
  if (rc) {
    delete cb;
    return rc;
  }
  *out = cb;
  return LEECH_OK;
}

void leech_codebook_free(leech_codebook* cb) { delete cb; }

int leech_codebook_info(const leech_codebook* cb, int* n_classes, uint64_t* n_points,
                        int* index_bits) {
  clear_error();
  if (!cb) return set_error(LEECH_E_ARG, "codebook is NULL");
  if (n_classes) *n_classes = (int)cb->classes.size();
  if (n_points) *n_points = cb->n_points;
  if (index_bits) {
    int b = 0;
    while (b < 64 && (1ull << b) < cb->n_points) ++b;
    *index_bits = b;
  }
  return LEECH_OK;
}

int leech_codebook_class(const leech_codebook* cb, int class_id, int* shell, int* parity,
                         int* n_levels, uint8_t levels[5], uint64_t* size) {
  clear_error();
  if (!cb) return set_error(LEECH_E_ARG, "codebook is NULL");
  if (class_id < 0 || class_id >= (int)cb->classes.size())
    return set_error(LEECH_E_ARG, fmt("class id %d out of range", class_id));
  const HostClass& c = cb->classes[class_id];
  if (shell) *shell = c.shell;
  if (parity) *parity = c.parity;
  if (n_levels) *n_levels = c.n_levels;
  if (levels)
    for (int k = 0; k < kMaxLevels; ++k) levels[k] = k < c.n_levels ? c.levels[k] : 0;
  if (size) *size = c.size;
  return LEECH_OK;
}

int leech_codebook_table(const leech_codebook* cb, int which, const void** host_ptr,
                         size_t* nbytes) {
  clear_error();
  if (!cb || !host_ptr || !nbytes) return set_error(LEECH_E_ARG, "NULL argument");
  switch (which) {
    case LEECH_TABLE_CLASS_LEVELS:
      *host_ptr = cb->tab_levels.data();
      *nbytes = cb->tab_levels.size();
      return LEECH_OK;
    case LEECH_TABLE_CODEWORDS:
      *host_ptr = cb->codewords.data();
      *nbytes = cb->codewords.size() * sizeof(uint32_t);
      return LEECH_OK;
    case LEECH_TABLE_DEVICE:
      if (cb->ball_m != 12)
        return set_error(LEECH_E_ARG, "the device table exists for the ball Λ24(12) only");
      *host_ptr = cb->tab_device.data();
      *nbytes = cb->tab_device.size();
      return LEECH_OK;
    case LEECH_TABLE_GOLAY_GEN:
      *host_ptr = cb->golay_gen.data();
      *nbytes = cb->golay_gen.size() * sizeof(uint32_t);
      return LEECH_OK;
    case LEECH_TABLE_INDEX:
      if (cb->tab_index.empty())
        return set_error(LEECH_E_ARG, "this ball holds 2^47 points or more: no format-v1 index");
      *host_ptr = cb->tab_index.data();
      *nbytes = cb->tab_index.size();
      return LEECH_OK;
    default:
      return set_error(LEECH_E_ARG, fmt("unknown table %d", which));
  }
}

int leech_fields_from_points(const leech_codebook* cb, int64_t n, const int8_t* z,
                             uint16_t* class_id, uint32_t* sign_mask, uint8_t* level) {
  clear_error();
  if (!cb || (n > 0 && (!z || !class_id || !sign_mask || !level)))
    return set_error(LEECH_E_ARG, "NULL argument");
  if (n < 0) return set_error(LEECH_E_ARG, "n < 0");
  std::atomic<int64_t> first_bad{INT64_MAX};
  auto work = [&](int64_t b0, int64_t b1) {
    for (int64_t b = b0; b < b1; ++b) {
      const int8_t* v = z + b * kDim;
      uint64_t key = 0;
      int mu = v[0] & 1, sum = 0;
      uint32_t mask = 0, smask = 0;
      bool ok = true;
      for (int i = 0; i < kDim; ++i) {
        int a = v[i] < 0 ? -v[i] : v[i];
        if (a > 13 || (v[i] & 1) != mu) { ok = false; break; }
        key += pow25[a];
        int r = ((v[i] % 4) + 4) % 4;
        if (r == (mu ? 3 : 2)) mask |= 1u << i;
        if (v[i] < 0) smask |= 1u << i;
        sum += v[i];
      }
      auto it = ok ? cb->by_key.find(key) : cb->by_key.end();
      if (!ok || it == cb->by_key.end() || !cb->is_codeword(mask) ||
          (((sum % 8) + 8) % 8) != 4 * mu) {
        int64_t cur = first_bad.load();
        while (b < cur && !first_bad.compare_exchange_weak(cur, b)) {}
        return;
      }
      const HostClass& c = cb->classes[it->second];
      class_id[b] = (uint16_t)it->second;
      sign_mask[b] = smask;
      for (int i = 0; i < kDim; ++i) {
        int a = v[i] < 0 ? -v[i] : v[i];
        uint8_t lv = 0;
        while (c.levels[lv] != a) ++lv;
        level[b * kDim + i] = lv;
      }
    }
  };
  int nt = (int)std::min<int64_t>(std::max(1u, std::thread::hardware_concurrency()),
                                  std::max<int64_t>(1, n / 65536));
  std::vector<std::thread> th;
  for (int t = 0; t < nt; ++t) th.emplace_back(work, n * t / nt, n * (t + 1) / nt);
  for (auto& t : th) t.join();
  if (first_bad.load() != INT64_MAX)
    return set_error(LEECH_E_NOT_LATTICE,
                     fmt("block %lld is not a point of the ball", (long long)first_bad.load()));
  return LEECH_OK;
}

}  // extern "C"

// ============================================================== layouts
namespace leech {

static inline void put_u32(uint8_t* p, uint32_t v) { std::memcpy(p, &v, 4); }
static inline void put_u64(uint8_t* p, uint64_t v) { std::memcpy(p, &v, 8); }
static inline uint32_t get_u32(const uint8_t* p) { uint32_t v; std::memcpy(&v, p, 4); return v; }
static inline uint64_t get_u64(const uint8_t* p) { uint64_t v; std::memcpy(&v, p, 8); return v; }

// Planes12x record (layout in leech_internal.h): the entry field, then each
// pair's level bits and non-negative bits at its selector word's places.  A
// five-level block (exc_local ≥ 0) carries only its exception entry number.
static void pack_planes12(uint8_t* rec, uint16_t cls, uint8_t g, uint32_t smask,
                          const uint8_t* level, int64_t exc_local) {
  std::memset(rec, 0, kPlanes12Bytes);
  if (exc_local >= 0) {
    put_bits(rec, 0, kExcEntry0 + (uint64_t)exc_local, 12);
    return;
  }
  put_bits(rec, 0, (uint64_t)cls | (uint64_t)g << 9, 12);
  for (int q = 0; q < 12; ++q)
    for (int h = 0; h < 2; ++h) {
      const int c = kPairCoords[q][h];
      put_bits(rec, p12_pair_bit(q, 3 * h), level[c] & 1u, 1);
      put_bits(rec, p12_pair_bit(q, 3 * h + 1), level[c] >> 1 & 1u, 1);
      put_bits(rec, p12_pair_bit(q, 3 * h + 2), (smask >> c & 1u) ^ 1u, 1);
    }
}

// Slot32 record: class [0,9) | gain 9 | sign mask [10,34) | one-hot mask of
// level k at [34 + 24(k−1), 58 + 24(k−1)) for k = 1..L−1; level 0 implicit.
static int pack_slot32(uint8_t* rec, uint16_t cls, uint8_t g, uint32_t smask,
                       const uint8_t* level, int n_levels) {
  int bytes = n_levels == kMaxLevels ? kSlot32Large : kSlot32Small;
  std::memset(rec, 0, bytes);
  put_bits(rec, 0, cls, 9);
  put_bits(rec, 9, g, 1);
  put_bits(rec, 10, smask, 24);
  for (int k = 1; k < n_levels; ++k) {
    uint32_t m = 0;
    for (int i = 0; i < kDim; ++i) m |= (uint32_t)(level[i] == k) << i;
    put_bits(rec, 34 + 24 * (k - 1), m, 24);
  }
  return bytes;
}

// Golay70 (record layout in leech_internal.h): the 2-bit code of coordinate i
// is bit i of the low code plane | bit i of the high one << 1; its side is bit i
// of the codeword; its value is the class's g70[side][code].  The codeword, on
// the coordinates with |z| ≡ 2 (mod 4) (even points) or z ≡ 3 (mod 4) (odd
// points), is stored as its 12-bit message under the code's generator, so a
// decoder rebuilds it from two 64-entry tables.
static bool golay70_codes(const leech_codebook* cb, uint16_t cls, const int8_t* z,
                          uint32_t* rank, uint64_t* codes) {
  const HostClass& c = cb->classes[cls];
  uint32_t word = 0;
  for (int i = 0; i < kDim; ++i) {
    int r = ((z[i] % 4) + 4) % 4;
    if (r == (c.parity ? 3 : 2)) word |= 1u << i;
  }
  *rank = cb->message_of.at(word);
  const DevClass* dc = (const DevClass*)cb->tab_device.data() + cls;
  uint64_t cd = 0;
  bool ok = true;
  for (int i = 0; i < kDim; ++i) {
    int side = word >> i & 1;
    int k = 0, n = cb->g70_count[cls][side];
    while (k < n && dc->g70[side][k] != z[i]) ++k;
    if (k == n) { ok = false; k = 0; }
    cd |= (uint64_t)k << (2 * i);
  }
  *codes = cd;
  return ok;
}

static void pack_golay70(uint8_t* rec, uint16_t cls, uint8_t g, uint32_t rank, uint64_t codes,
                         int64_t exc_local) {
  std::memset(rec, 0, kGolay70Bytes);
  if (exc_local >= 0) {
    put_bits(rec, 0, kExcEntry0 + (uint64_t)exc_local, 12);
    return;
  }
  put_bits(rec, 0, (uint64_t)cls | (uint64_t)g << 9, 12);
  put_bits(rec, kG70MsgPos, rank, 12);
  uint32_t c0 = 0, c1 = 0;
  for (int i = 0; i < kDim; ++i) {
    c0 |= (uint32_t)(codes >> (2 * i) & 1) << i;
    c1 |= (uint32_t)(codes >> (2 * i + 1) & 1) << i;
  }
  put_bits(rec, kG70C0Pos, c0, 24);
  put_bits(rec, kG70C1Pos, c1, 24);
}

struct Fields {
  const uint16_t* cls;
  const uint8_t* gain;
  const uint32_t* smask;
  const uint8_t* level;
};

static void fill_desc(leech_layout_desc* d, int layout, const Geometry& geo, int64_t Kpad) {
  std::memset(d, 0, sizeof *d);
  d->layout = layout;
  d->lane_cols = geo.C;
  d->tile_rows = geo.R;
  d->M = geo.M;
  d->Kpad = Kpad;
  d->nb = geo.nb;
}

static void finish_desc(leech_layout_desc* d) {
  d->served_bytes = d->main_bytes + d->side_bytes[0] + d->side_bytes[1] +
                    2ull * (uint64_t)(d->M * d->nb);
}

template <class F>
static void parallel_rows(int64_t n, F f) {
  int nt = (int)std::min<int64_t>(std::max(1u, std::thread::hardware_concurrency()),
                                  std::max<int64_t>(1, n / 16));
  if (nt <= 1) { f(0, n); return; }
  std::vector<std::thread> th;
  for (int t = 0; t < nt; ++t) th.emplace_back(f, n * t / nt, n * (t + 1) / nt);
  for (auto& t : th) t.join();
}

static int expand(const leech_codebook* cb, int layout, int64_t M, int64_t Kpad, int C, int R,
                  const Fields& in, uint8_t* main_out, uint8_t* side0, uint8_t* side1,
                  leech_layout_desc* desc) {
  const int64_t nb = Kpad / kDim;
  const int64_t n = M * nb;
  Geometry geo(M, nb, C, R);
  leech_layout_desc d;
  fill_desc(&d, layout, geo, Kpad);

  // validate every block, decode to integer points (needed by every layout)
  std::vector<int8_t> z((size_t)n * kDim);
  std::atomic<int64_t> first_bad{INT64_MAX};
  std::atomic<int> bad_code{0};
  const char* bad_why = "";
  std::mutex why_mu;
  parallel_rows(M, [&](int64_t r0, int64_t r1) {
    for (int64_t b = r0 * nb; b < r1 * nb; ++b) {
      const char* why = "";
      int rc = in.gain[b] > 1 ? (why = "gain bit must be 0 or 1", LEECH_E_FIELD)
                              : fields_to_point(cb, in.cls[b], in.smask[b], in.level + b * kDim,
                                                &z[b * kDim], &why);
      if (rc) {
        int64_t cur = first_bad.load();
        while (b < cur && !first_bad.compare_exchange_weak(cur, b)) {}
        std::lock_guard<std::mutex> lk(why_mu);
        if (first_bad.load() == b) { bad_code = rc; bad_why = why; }
        return;
      }
    }
  });
  if (first_bad.load() != INT64_MAX)
    return set_error(bad_code.load(), fmt("block %lld (row %lld, column block %lld): %s",
                                          (long long)first_bad.load(),
                                          (long long)(first_bad.load() / nb),
                                          (long long)(first_bad.load() % nb), bad_why));

  auto nlev = [&](int64_t b) { return cb->classes[in.cls[b]].n_levels; };

  switch (layout) {
    case LEECH_PLANES14: {
      d.main_bytes = (uint64_t)n * kPlanes14Bytes + kPadBytes;
      if (main_out) {
        std::memset(main_out + n * kPlanes14Bytes, 0, kPadBytes);
        parallel_rows(M, [&](int64_t r0, int64_t r1) {
          for (int64_t r = r0; r < r1; ++r)
            for (int64_t j = 0; j < nb; ++j) {
              int64_t b = r * nb + j;
              pack_planes14(main_out + geo.index(r, j) * kPlanes14Bytes, in.cls[b], in.gain[b],
                            in.smask[b], in.level + b * kDim);
            }
        });
      }
      break;
    }
    case LEECH_PLANES12X:
    case LEECH_GOLAY70: {
      // exceptions: five-level blocks (Planes12x), blocks with a value outside
      // their side's four (Golay70); Golay70 keeps every block's message and codes
      const bool g70 = layout == LEECH_GOLAY70;
      const int rec_bytes = g70 ? kGolay70Bytes : kPlanes12Bytes;
      std::vector<uint8_t> flag(n, 0);     // row-major block index
      std::vector<uint32_t> rank(g70 ? n : 0);
      std::vector<uint64_t> codes(g70 ? n : 0);
      parallel_rows(M, [&](int64_t r0, int64_t r1) {
        for (int64_t b = r0 * nb; b < r1 * nb; ++b)
          flag[b] = g70 ? !golay70_codes(cb, in.cls[b], &z[b * kDim], &rank[b], &codes[b])
                        : nlev(b) == kMaxLevels;
      });
      // exception lists per tile, in storage order
      std::vector<uint32_t> tile_count(geo.tiles, 0);
      std::vector<int64_t> local(n, -1);   // by storage index
      for (int64_t t = 0; t < geo.tiles; ++t) {
        int R_t = geo.rows_in_tile(t);
        for (int64_t g = 0; g < geo.groups; ++g) {
          int C_g = geo.cols_in_group(g);
          int64_t base = geo.unit_base(t, g);
          for (int rl = 0; rl < R_t; ++rl)
            for (int cl = 0; cl < C_g; ++cl) {
              int64_t b = (t * geo.R + rl) * nb + g * geo.C + cl;
              if (flag[b]) {
                if (tile_count[t] >= kExcMax)
                  return set_error(LEECH_E_CAPACITY,
                                   fmt("tile %lld holds more than %u exception blocks",
                                       (long long)t, kExcMax));
                local[base + rl * C_g + cl] = tile_count[t]++;
              }
            }
        }
      }
      std::vector<uint32_t> tile_base(geo.tiles, 0);
      uint64_t total = 0;
      for (int64_t t = 0; t < geo.tiles; ++t) {
        tile_base[t] = (uint32_t)total;
        total += tile_count[t];
        d.tile_exc_max = std::max<uint32_t>(d.tile_exc_max, tile_count[t]);
      }
      if (total > 0xFFFFFFFFull) return set_error(LEECH_E_CAPACITY, "too many exceptions");
      if ((uint64_t)geo.R * (uint64_t)nb > (1ull << kExcSlotBits))
        return set_error(LEECH_E_CAPACITY, "tile too large for the exception entries' slot field");
      d.n_exceptions = total;
      d.main_bytes = (uint64_t)n * rec_bytes + kPadBytes;
      d.side_bytes[0] = total * kExcEntryBytes + kPadBytes;
      d.side_bytes[1] = (uint64_t)geo.tiles * 4;
      if (main_out) {
        std::memset(main_out + n * rec_bytes, 0, kPadBytes);
        std::memset(side0 + total * kExcEntryBytes, 0, kPadBytes);
        for (int64_t t = 0; t < geo.tiles; ++t) put_u32(side1 + 4 * t, tile_base[t]);
        parallel_rows(M, [&](int64_t r0, int64_t r1) {
          for (int64_t r = r0; r < r1; ++r)
            for (int64_t j = 0; j < nb; ++j) {
              int64_t b = r * nb + j, s = geo.index(r, j);
              if (g70)
                pack_golay70(main_out + s * kGolay70Bytes, in.cls[b], in.gain[b], rank[b],
                             codes[b], local[s]);
              else
                pack_planes12(main_out + s * kPlanes12Bytes, in.cls[b], in.gain[b], in.smask[b],
                              in.level + b * kDim, local[s]);
              if (local[s] >= 0) {
                uint8_t* ent = side0 + (tile_base[r / geo.R] + local[s]) * kExcEntryBytes;
                pack_planes14(ent, in.cls[b], in.gain[b], in.smask[b], in.level + b * kDim);
                ent[14] = ent[15] = 0;
                put_bits(ent, kExcSlotShift, (uint64_t)(s - (r / geo.R) * geo.R * nb),
                         kExcSlotBits);
              }
            }
        });
      }
      break;
    }
    case LEECH_SLOT32: {
      // per-unit side entries: u64 bitmap of the five-level blocks, u32 word
      // offset of the unit's first record, u32 zero
      std::vector<uint8_t> flag(n, 0);   // by storage index
      parallel_rows(M, [&](int64_t r0, int64_t r1) {
        for (int64_t r = r0; r < r1; ++r)
          for (int64_t j = 0; j < nb; ++j) flag[geo.index(r, j)] = nlev(r * nb + j) == kMaxLevels;
      });
      std::vector<uint64_t> unit_bits(geo.units(), 0);
      std::vector<uint64_t> unit_base(geo.units(), 0);
      uint64_t acc = 0;
      for (int64_t t = 0; t < geo.tiles; ++t)
        for (int64_t g = 0; g < geo.groups; ++g) {
          int64_t u = geo.unit_id(t, g), base = geo.unit_base(t, g);
          int cnt = geo.rows_in_tile(t) * geo.cols_in_group(g);
          unit_base[u] = acc;
          uint64_t bits = 0;
          for (int l = 0; l < cnt; ++l)
            if (flag[base + l]) bits |= 1ull << l;
          unit_bits[u] = bits;
          int nf = __builtin_popcountll(bits);
          acc += (uint64_t)(cnt * kSlot32Small + nf * (kSlot32Large - kSlot32Small)) / 4;
        }
      if (acc > 0xFFFFFFFFull) return set_error(LEECH_E_CAPACITY, "side-table offset overflow");
      d.side_bytes[0] = (uint64_t)geo.units() * kUnitEntryBytes;
      d.main_bytes = acc * 4 + kPadBytes;
      if (main_out) {
        for (int64_t u = 0; u < geo.units(); ++u) {
          put_u64(side0 + u * kUnitEntryBytes, unit_bits[u]);
          put_u32(side0 + u * kUnitEntryBytes + 8, (uint32_t)unit_base[u]);
          put_u32(side0 + u * kUnitEntryBytes + 12, 0);
        }
        std::memset(main_out + d.main_bytes - kPadBytes, 0, kPadBytes);
        parallel_rows(M, [&](int64_t r0, int64_t r1) {
          for (int64_t r = r0; r < r1; ++r)
            for (int64_t j = 0; j < nb; ++j) {
              int64_t b = r * nb + j, s = geo.index(r, j);
              int64_t t = r / geo.R, g = j / geo.C;
              int64_t u = geo.unit_id(t, g);
              int lane = (int)(s - geo.unit_base(t, g));
              int nbelow = __builtin_popcountll(unit_bits[u] & ((1ull << lane) - 1));
              uint64_t off = unit_base[u] * 4 + (uint64_t)lane * kSlot32Small +
                             (uint64_t)nbelow * (kSlot32Large - kSlot32Small);
              pack_slot32(main_out + off, in.cls[b], in.gain[b], in.smask[b],
                          in.level + b * kDim, nlev(b));
            }
        });
      }
      break;
    }
    default:
      return set_error(LEECH_E_LAYOUT, fmt("unknown layout %d", layout));
  }
  finish_desc(&d);
  *desc = d;
  return LEECH_OK;
}

static int check_desc(const leech_layout_desc* d) {
  if (!d) return set_error(LEECH_E_ARG, "desc is NULL");
  if (d->layout < LEECH_SLOT32 || d->layout > LEECH_GOLAY70)
    return set_error(LEECH_E_LAYOUT, fmt("unknown layout %d", d->layout));
  if (d->M <= 0 || d->Kpad <= 0 || d->Kpad % kDim || d->nb != d->Kpad / kDim)
    return set_error(LEECH_E_SHAPE, "descriptor shape is not valid");
  if (!geometry_ok(d->lane_cols, d->tile_rows))
    return set_error(LEECH_E_SHAPE, fmt("descriptor geometry lane_cols = %d, tile_rows = %d is not "
                                        "one the kernels serve", d->lane_cols, d->tile_rows));
  return LEECH_OK;
}

// The geometry an expansion uses: the caller's, validated, or (0, 0) for the
// library's choice.
static int resolve_geometry(int64_t M, int64_t nb, int lane_cols, int tile_rows, int* C, int* R) {
  if (lane_cols == 0 && tile_rows == 0) {
    choose_geometry(M, nb, C, R);
    return LEECH_OK;
  }
  if (!geometry_ok(lane_cols, tile_rows))
    return set_error(LEECH_E_SHAPE,
                     fmt("lane_cols = %d, tile_rows = %d: need lane_cols in {1, 2, 3, 4, 8, 16} "
                         "and tile_rows a positive multiple of 4 with tile_rows * lane_cols <= 64",
                         lane_cols, tile_rows));
  *C = lane_cols;
  *R = tile_rows;
  return LEECH_OK;
}

}  // namespace leech

extern "C" {

int leech_expand_layout_tiled(const leech_codebook* cb, int layout, int64_t M, int64_t Kpad,
                              int32_t lane_cols, int32_t tile_rows, const uint16_t* class_id,
                              const uint8_t* gain_bit, const uint32_t* sign_mask,
                              const uint8_t* level, void* main_out, void* side0_out,
                              void* side1_out, leech_layout_desc* desc) {
  clear_error();
  if (!cb || !desc || !class_id || !gain_bit || !sign_mask || !level)
    return set_error(LEECH_E_ARG, "NULL argument");
  if (cb->ball_m != 12) return set_error(LEECH_E_ARG, "layouts serve the ball Λ24(12) only");
  if (layout < LEECH_SLOT32 || layout > LEECH_GOLAY70)
    return set_error(LEECH_E_LAYOUT, fmt("unknown layout %d", layout));
  if (M <= 0 || Kpad <= 0 || Kpad % kDim)
    return set_error(LEECH_E_SHAPE, fmt("M = %lld, Kpad = %lld: need M > 0, Kpad > 0 and Kpad %% 24 == 0",
                                        (long long)M, (long long)Kpad));
  int C = 0, R = 0;
  int rc = resolve_geometry(M, Kpad / kDim, lane_cols, tile_rows, &C, &R);
  if (rc) return rc;
  const Fields f{class_id, gain_bit, sign_mask, level};
  if (main_out) {
    leech_layout_desc probe;
    rc = expand(cb, layout, M, Kpad, C, R, f, nullptr, nullptr, nullptr, &probe);
    if (rc) return rc;
    if ((probe.side_bytes[0] && !side0_out) || (probe.side_bytes[1] && !side1_out))
      return set_error(LEECH_E_ARG, "a side stream of this layout needs an output buffer");
  }
  return expand(cb, layout, M, Kpad, C, R, f, (uint8_t*)main_out, (uint8_t*)side0_out,
                (uint8_t*)side1_out, desc);
}

int leech_expand_layout(const leech_codebook* cb, int layout, int64_t M, int64_t Kpad,
                        const uint16_t* class_id, const uint8_t* gain_bit,
                        const uint32_t* sign_mask, const uint8_t* level, void* main_out,
                        void* side0_out, void* side1_out, leech_layout_desc* desc) {
  return leech_expand_layout_tiled(cb, layout, M, Kpad, 0, 0, class_id, gain_bit, sign_mask,
                                   level, main_out, side0_out, side1_out, desc);
}

int leech_layout_geometry(int64_t M, int64_t Kpad, int32_t* lane_cols, int32_t* tile_rows) {
  clear_error();
  if (!lane_cols || !tile_rows) return set_error(LEECH_E_ARG, "NULL argument");
  if (M <= 0 || Kpad <= 0 || Kpad % kDim)
    return set_error(LEECH_E_SHAPE, fmt("M = %lld, Kpad = %lld: need M > 0, Kpad > 0 and Kpad %% 24 == 0",
                                        (long long)M, (long long)Kpad));
  int C = 0, R = 0;
  choose_geometry(M, Kpad / kDim, &C, &R);
  *lane_cols = C;
  *tile_rows = R;
  return LEECH_OK;
}

int leech_layout_scales(const leech_layout_desc* desc, const uint16_t* scale_rowmajor,
                        uint16_t* scale_out) {
  clear_error();
  int rc = check_desc(desc);
  if (rc) return rc;
  if (!scale_rowmajor || !scale_out) return set_error(LEECH_E_ARG, "NULL argument");
  Geometry geo(desc->M, desc->nb, desc->lane_cols, desc->tile_rows);
  parallel_rows(desc->M, [&](int64_t r0, int64_t r1) {
    for (int64_t r = r0; r < r1; ++r)
      for (int64_t j = 0; j < desc->nb; ++j)
        scale_out[geo.index(r, j)] = scale_rowmajor[r * desc->nb + j];
  });
  return LEECH_OK;
}

int leech_host_decode_layout(const leech_codebook* cb, const leech_layout_desc* desc,
                             const void* main_, const void* side0_, const void* side1_,
                             int8_t* z, uint16_t* class_id, uint8_t* gain_bit) {
  clear_error();
  int rc = check_desc(desc);
  if (rc) return rc;
  if (!cb || !main_) return set_error(LEECH_E_ARG, "NULL argument");
  const uint8_t* mainp = (const uint8_t*)main_;
  const uint8_t* side0 = (const uint8_t*)side0_;
  const uint8_t* side1 = (const uint8_t*)side1_;
  if ((desc->side_bytes[0] && !side0) || (desc->side_bytes[1] && !side1))
    return set_error(LEECH_E_ARG, "layout needs its side streams");
  Geometry geo(desc->M, desc->nb, desc->lane_cols, desc->tile_rows);
  const int64_t nb = desc->nb;
  std::atomic<bool> bad{false};
  parallel_rows(desc->M, [&](int64_t r0, int64_t r1) {
    int8_t zz[kDim];
    for (int64_t r = r0; r < r1; ++r)
      for (int64_t j = 0; j < nb; ++j) {
        int64_t b = r * nb + j, s = geo.index(r, j);
        int64_t t = r / geo.R, g = j / geo.C;
        uint16_t cls = 0;
        uint8_t gb = 0;
        switch (desc->layout) {
          case LEECH_PLANES14:
            unpack_planes14(cb, mainp + s * kPlanes14Bytes, zz, &cls, &gb);
            break;
          case LEECH_PLANES12X:
          case LEECH_GOLAY70: {
            const bool g70 = desc->layout == LEECH_GOLAY70;
            const uint8_t* rec = mainp + s * (g70 ? kGolay70Bytes : kPlanes12Bytes);
            const uint32_t field = (uint32_t)get_bits(rec, 0, 12);
            if (field >= kExcEntry0) {
              uint32_t base = get_u32(side1 + 4 * t);
              unpack_planes14(cb, side0 + (uint64_t)(base + field - kExcEntry0) * kExcEntryBytes,
                              zz, &cls, &gb);
              break;
            }
            cls = (uint16_t)(field & 511u);
            gb = (uint8_t)(field >> 9 & 1u);
            const DevClass* dc = (const DevClass*)cb->tab_device.data() + cls;
            if (g70) {
              const uint32_t msg = (uint32_t)get_bits(rec, kG70MsgPos, 12);
              const uint32_t word = cb->golay_gen[msg & 63] ^ cb->golay_gen[64 + (msg >> 6)];
              for (int i = 0; i < kDim; ++i)
                zz[i] = dc->g70[word >> i & 1][get_bits(rec, kG70C0Pos + i, 1) |
                                               get_bits(rec, kG70C1Pos + i, 1) << 1];
            } else {
              for (int q = 0; q < 12; ++q)
                for (int h = 0; h < 2; ++h) {
                  const int lev = (int)(get_bits(rec, p12_pair_bit(q, 3 * h), 1) |
                                        get_bits(rec, p12_pair_bit(q, 3 * h + 1), 1) << 1);
                  const int a = dc->perm[level_code(lev)];
                  const bool neg = !get_bits(rec, p12_pair_bit(q, 3 * h + 2), 1);
                  zz[kPairCoords[q][h]] = (int8_t)(neg ? -a : a);
                }
            }
            break;
          }
          case LEECH_SLOT32: {
            int64_t u = geo.unit_id(t, g);
            uint64_t bits = get_u64(side0 + u * kUnitEntryBytes);
            uint32_t base = get_u32(side0 + u * kUnitEntryBytes + 8);
            int lane = (int)(s - geo.unit_base(t, g));
            int nbelow = __builtin_popcountll(bits & ((1ull << lane) - 1));
            const uint8_t* rec = mainp + (uint64_t)base * 4 + (uint64_t)lane * kSlot32Small +
                                 (uint64_t)nbelow * (kSlot32Large - kSlot32Small);
            cls = (uint16_t)get_bits(rec, 0, 9);
            gb = (uint8_t)get_bits(rec, 9, 1);
            uint32_t sm = (uint32_t)get_bits(rec, 10, 24);
            const DevClass* dc = (const DevClass*)cb->tab_device.data() + cls;
            int L = dc->info & 0xFF;
            for (int i = 0; i < kDim; ++i) {
              int code = 0;
              for (int k = 1; k < L; ++k)
                if (get_bits(rec, 34 + 24 * (k - 1) + i, 1)) code = k;
              int a = dc->perm[level_code(code)];
              zz[i] = (int8_t)((sm >> i & 1) ? -a : a);
            }
            break;
          }
        }
        if (cls >= cb->classes.size()) bad = true;
        if (z) std::memcpy(z + b * kDim, zz, kDim);
        if (class_id) class_id[b] = cls;
        if (gain_bit) gain_bit[b] = gb;
      }
  });
  if (bad) return set_error(LEECH_E_FIELD, "a record names a class id out of range");
  return LEECH_OK;
}


// ------------------------------------------------ format-v1 block codes (§2.1)
int leech_index_encode(const leech_codebook* cb, int64_t n, const uint16_t* class_id,
                       const uint8_t* gain_bit, const uint32_t* sign_mask, const uint8_t* level,
                       uint64_t* code) {
  clear_error();
  if (!cb || (n > 0 && (!class_id || !gain_bit || !sign_mask || !level || !code)))
    return set_error(LEECH_E_ARG, "NULL argument");
  if (n < 0) return set_error(LEECH_E_ARG, "n < 0");
  if (cb->tab_index.empty())
    return set_error(LEECH_E_ARG, "this ball holds 2^47 points or more: no format-v1 index");
  const IdxTable& T = *reinterpret_cast<const IdxTable*>(cb->tab_index.data());
  std::atomic<int64_t> first_bad{INT64_MAX};
  std::atomic<int> bad_code{0};
  const char* bad_why = "";
  std::mutex why_mu;
  parallel_rows(n, [&](int64_t b0, int64_t b1) {
    int8_t z[kDim];
    for (int64_t b = b0; b < b1; ++b) {
      const char* why = "";
      int rc = gain_bit[b] > 1 ? (why = "gain bit must be 0 or 1", LEECH_E_FIELD)
                               : fields_to_point(cb, class_id[b], sign_mask[b], level + b * kDim,
                                                 z, &why);
      if (!rc && !idx_encode(T, class_id[b], gain_bit[b], sign_mask[b], level + b * kDim,
                             &code[b])) {
        rc = LEECH_E_NOT_LATTICE;
        why = "fields are not a point the index names";
      }
      if (rc) {
        int64_t cur = first_bad.load();
        while (b < cur && !first_bad.compare_exchange_weak(cur, b)) {}
        std::lock_guard<std::mutex> lk(why_mu);
        if (first_bad.load() == b) { bad_code = rc; bad_why = why; }
        return;
      }
    }
  });
  if (first_bad.load() != INT64_MAX)
    return set_error(bad_code.load(),
                     fmt("block %lld: %s", (long long)first_bad.load(), bad_why));
  return LEECH_OK;
}

int leech_index_decode(const leech_codebook* cb, int64_t n, const uint64_t* code,
                       uint16_t* class_id, uint8_t* gain_bit, uint32_t* sign_mask,
                       uint8_t* level) {
  clear_error();
  if (!cb || (n > 0 && (!code || !class_id || !gain_bit || !sign_mask || !level)))
    return set_error(LEECH_E_ARG, "NULL argument");
  if (n < 0) return set_error(LEECH_E_ARG, "n < 0");
  if (cb->tab_index.empty())
    return set_error(LEECH_E_ARG, "this ball holds 2^47 points or more: no format-v1 index");
  const IdxTable& T = *reinterpret_cast<const IdxTable*>(cb->tab_index.data());
  std::atomic<int64_t> first_bad{INT64_MAX};
  parallel_rows(n, [&](int64_t b0, int64_t b1) {
    for (int64_t b = b0; b < b1; ++b) {
      uint32_t p[3];
      if (!idx_decode(T, code[b], &class_id[b], &gain_bit[b], &sign_mask[b], p)) {
        int64_t cur = first_bad.load();
        while (b < cur && !first_bad.compare_exchange_weak(cur, b)) {}
        return;
      }
      for (int i = 0; i < kDim; ++i)
        level[b * kDim + i] =
            (uint8_t)(((p[0] >> i & 1) | (p[1] >> i & 1) << 1 | (p[2] >> i & 1) << 2) - 1);
    }
  });
  if (first_bad.load() != INT64_MAX)
    return set_error(LEECH_E_FIELD, fmt("code %lld (0x%llx) is not a format-v1 block code",
                                        (long long)first_bad.load(),
                                        (unsigned long long)code[first_bad.load()]));
  return LEECH_OK;
}

int leech_planes14_desc(int64_t M, int64_t Kpad, int32_t lane_cols, int32_t tile_rows,
                        leech_layout_desc* desc) {
  clear_error();
  if (!desc) return set_error(LEECH_E_ARG, "NULL argument");
  if (M <= 0 || Kpad <= 0 || Kpad % kDim)
    return set_error(LEECH_E_SHAPE, fmt("M = %lld, Kpad = %lld: need M > 0, Kpad > 0 and Kpad %% 24 == 0",
                                        (long long)M, (long long)Kpad));
  int C = 0, R = 0;
  int rc = resolve_geometry(M, Kpad / kDim, lane_cols, tile_rows, &C, &R);
  if (rc) return rc;
  Geometry geo(M, Kpad / kDim, C, R);
  fill_desc(desc, LEECH_PLANES14, geo, Kpad);
  desc->main_bytes = (uint64_t)(M * geo.nb) * kPlanes14Bytes + kPadBytes;
  finish_desc(desc);
  return LEECH_OK;
}

}  // extern "C"
