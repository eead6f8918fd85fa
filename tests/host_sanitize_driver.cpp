// Host half of libleech under AddressSanitizer and UndefinedBehaviorSanitizer
// (built with g++ by test_host_sanitizers.py; no GPU code involved).
//
// Reads M, Kpad, the lattice points z[M·nb][24], gain bits and fp16 scales
// from a file written by the test, then runs every host entry point on them:
// fields from points, the expansion into each of the four layouts (sizing call,
// then fill), the host decode of each layout back to points, class ids and gain
// bits, the scale permutation, and the format-v1 index encode and decode.  It
// checks each round trip and the documented error codes of bad inputs, prints
// "ok" and exits 0, or names the first mismatch and exits 1.

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "leech.h"

namespace {

int fail(const char* what) {
  std::printf("FAIL %s: %s\n", what, leech_last_error());
  return 1;
}

template <class T>
bool read_all(FILE* f, std::vector<T>& v, size_t n) {
  v.resize(n);
  return std::fread(v.data(), sizeof(T), n, f) == n;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) return std::printf("usage: driver INPUT\n"), 2;
  FILE* f = std::fopen(argv[1], "rb");
  if (!f) return std::printf("cannot open %s\n", argv[1]), 2;
  int64_t M = 0, Kpad = 0;
  if (std::fread(&M, 8, 1, f) != 1 || std::fread(&Kpad, 8, 1, f) != 1) return 2;
  const int64_t n = M * (Kpad / 24);
  std::vector<int8_t> z;
  std::vector<uint8_t> gain;
  std::vector<uint16_t> scale;
  const bool ok_read = read_all(f, z, (size_t)n * 24) && read_all(f, gain, (size_t)n) &&
                       read_all(f, scale, (size_t)n);
  std::fclose(f);
  if (!ok_read) return std::printf("short input\n"), 2;

  leech_codebook* cb = nullptr;
  if (leech_codebook_build(12, &cb)) return fail("codebook_build");

  std::vector<uint16_t> cls(n);
  std::vector<uint32_t> sm(n);
  std::vector<uint8_t> lv((size_t)n * 24);
  if (leech_fields_from_points(cb, n, z.data(), cls.data(), sm.data(), lv.data()))
    return fail("fields_from_points");

  for (int layout : {LEECH_SLOT32, LEECH_PLANES14, LEECH_PLANES12X, LEECH_GOLAY70}) {
    leech_layout_desc d;
    if (leech_expand_layout(cb, layout, M, Kpad, cls.data(), gain.data(), sm.data(), lv.data(),
                            nullptr, nullptr, nullptr, &d))
      return fail("expand (sizing)");
    std::vector<uint8_t> main_(d.main_bytes), s0(d.side_bytes[0] + 1), s1(d.side_bytes[1] + 1);
    if (leech_expand_layout(cb, layout, M, Kpad, cls.data(), gain.data(), sm.data(), lv.data(),
                            main_.data(), s0.data(), s1.data(), &d))
      return fail("expand (fill)");
    std::vector<int8_t> z2((size_t)n * 24);
    std::vector<uint16_t> c2(n);
    std::vector<uint8_t> g2(n);
    if (leech_host_decode_layout(cb, &d, main_.data(), s0.data(), s1.data(), z2.data(), c2.data(),
                                 g2.data()))
      return fail("host_decode_layout");
    if (z2 != z || c2 != cls || g2 != gain) {
      std::printf("FAIL layout %d does not decode to its points\n", layout);
      return 1;
    }
    std::vector<uint16_t> sc(n);
    if (leech_layout_scales(&d, scale.data(), sc.data())) return fail("layout_scales");
  }

  std::vector<uint64_t> code(n);
  if (leech_index_encode(cb, n, cls.data(), gain.data(), sm.data(), lv.data(), code.data()))
    return fail("index_encode");
  std::vector<uint16_t> c3(n);
  std::vector<uint8_t> g3(n), l3((size_t)n * 24);
  std::vector<uint32_t> s3(n);
  if (leech_index_decode(cb, n, code.data(), c3.data(), g3.data(), s3.data(), l3.data()))
    return fail("index_decode");
  if (c3 != cls || g3 != gain || s3 != sm || l3 != lv) {
    std::printf("FAIL index round trip\n");
    return 1;
  }

  // documented errors: they return a code and leave the process intact
  leech_layout_desc d;
  std::vector<uint16_t> bad = cls;
  bad[n / 2] = 301;                                  // not a class of the ball
  if (leech_expand_layout(cb, LEECH_PLANES14, M, Kpad, bad.data(), gain.data(), sm.data(),
                          lv.data(), nullptr, nullptr, nullptr, &d) != LEECH_E_FIELD)
    return fail("class id 301 accepted");
  if (leech_expand_layout(cb, 7, M, Kpad, cls.data(), gain.data(), sm.data(), lv.data(), nullptr,
                          nullptr, nullptr, &d) != LEECH_E_LAYOUT)
    return fail("unknown layout accepted");
  if (leech_expand_layout(cb, LEECH_PLANES14, M, Kpad + 1, cls.data(), gain.data(), sm.data(),
                          lv.data(), nullptr, nullptr, nullptr, &d) != LEECH_E_SHAPE)
    return fail("Kpad not a multiple of 24 accepted");
  std::vector<int8_t> zbad(z.begin(), z.begin() + 24);
  zbad[0] = (int8_t)(zbad[0] + 1);                   // odd change: off the lattice
  uint16_t c1;
  uint32_t s1;
  uint8_t l1[24];
  if (leech_fields_from_points(cb, 1, zbad.data(), &c1, &s1, l1) == LEECH_OK)
    return fail("non-lattice point accepted");
  uint64_t c64 = code[0] | (1ull << 48);             // bits above 47 set
  if (leech_index_decode(cb, 1, &c64, &c1, l1, &s1, l1) != LEECH_E_FIELD)
    return fail("code with bit 48 accepted");

  leech_codebook_free(cb);
  std::printf("ok %lld blocks\n", (long long)n);
  return 0;
}
