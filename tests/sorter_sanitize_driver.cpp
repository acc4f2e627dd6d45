// Host-only check of the chunk-sorted code form, built with AddressSanitizer
// and UndefinedBehaviorSanitizer on the host code (tests/test_sorter_sanitized.py).
// For every case the sorter's output is checked against the codes it came
// from: the index is consistent, every entry decodes to a code of its row in
// its chunk class, in ascending group order per row, and every code appears
// exactly once.  The codes are read back with a bit reader written here, not
// the sorter's own.  No kernel is launched: the two launch helpers the
// sorter's object refers to are defined below and never called.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <vector>

#include "sorted.h"

namespace aqlm {
hipError_t allow_dynamic_lds(const void*, int) { return hipErrorNotSupported; }
int num_cus() { return 256; }
}  // namespace aqlm

namespace {

uint32_t lcg(uint32_t& s) {
  s = s * 1664525u + 1013904223u;
  return s;
}

struct Case {
  int32_t d_out, d_in, M, B;
  bool packed;
};

// code (row, j, m): unpacked [d_out][G][M] uint16, or one bit string per row
// (code (j, m) at bits [(j M + m) B, + B), least significant bit first,
// 32-bit words)
uint32_t code_at(const std::vector<uint16_t>& u, const std::vector<uint32_t>& w, const Case& c, int64_t words,
                 int32_t row, int32_t j, int32_t m) {
  const int32_t G = c.d_in / 8;
  if (!c.packed) return u[((size_t)row * G + j) * c.M + m] & ((1u << c.B) - 1u);
  const uint64_t bit = ((uint64_t)j * c.M + m) * c.B;
  uint32_t v = 0;
  for (int k = 0; k < c.B; ++k) {
    const uint64_t b = bit + k;
    v |= ((w[(size_t)row * words + b / 32] >> (b % 32)) & 1u) << k;
  }
  return v;
}

bool run(const Case& c) {
  const int32_t G = c.d_in / 8;
  const int K = aqlm::sorted_classes(c.M, c.B);
  const int64_t nb = aqlm::sorted_blocks(c.d_out);
  const int64_t words = ((int64_t)G * c.M * c.B + 31) / 32;
  uint32_t s = 12345u + (uint32_t)(c.d_out * 7 + c.d_in + c.M * 3 + c.B);
  std::vector<uint16_t> u;
  std::vector<uint32_t> w;
  if (c.packed) {
    w.resize((size_t)c.d_out * words);
    for (auto& v : w) v = lcg(s);
  } else {
    u.resize((size_t)c.d_out * G * c.M);
    for (auto& v : u) v = (uint16_t)(lcg(s) >> 16);
  }
  const void* src = c.packed ? static_cast<const void*>(w.data()) : static_cast<const void*>(u.data());
  const int64_t steps = aqlm::sorted_steps(src, c.packed, c.d_out, c.d_in, c.M, c.B);
  std::vector<uint32_t> entries((size_t)steps * 64), index((size_t)K * nb + 1);
  aqlm::sort_codes(src, c.packed, c.d_out, c.d_in, c.M, c.B, entries.data(), steps, index.data());

  if (index[0] != 0 || (int64_t)index.back() != steps) {
    std::printf("case %dx%d %dx%d: index ends %u %u, steps %lld\n", c.d_out, c.d_in, c.M, c.B, index[0],
                index.back(), (long long)steps);
    return false;
  }
  std::vector<uint8_t> seen((size_t)c.d_out * G * c.M, 0);
  const int cpm = 1 << (c.B - aqlm::kChunkBits);  // chunk classes per codebook
  for (int cl = 0; cl < K; ++cl) {
    const int m = cl / cpm;
    const uint32_t chunk = (uint32_t)(cl % cpm);
    for (int64_t b = 0; b < nb; ++b) {
      const uint32_t s0 = index[(size_t)cl * nb + b], s1 = index[(size_t)cl * nb + b + 1];
      if (s1 < s0) {
        std::printf("index decreases at class %d block %lld\n", cl, (long long)b);
        return false;
      }
      for (int i = 0; i < 16; ++i) {
        int32_t last_j = -1;
        bool pad_seen = false;
        for (uint32_t st = s0; st < s1; ++st)
          for (int q = 0; q < 4; ++q) {
            const uint32_t e = entries[(size_t)st * 64 + 16 * q + i];
            if (e == aqlm::kSortedPad) {
              pad_seen = true;
              continue;
            }
            const int32_t row = (int32_t)(16 * b + i), j = (int32_t)(e >> 14);
            if (pad_seen || row >= c.d_out || j >= G || j <= last_j) {
              std::printf("bad entry %08x (class %d block %lld lane row %d)\n", e, cl, (long long)b, i);
              return false;
            }
            last_j = j;
            const uint32_t v = (chunk << aqlm::kChunkBits) | (e & (aqlm::kChunkCodewords - 1));
            if (v != code_at(u, w, c, words, row, j, m)) {
              std::printf("entry %08x decodes to %u, code is %u\n", e, v, code_at(u, w, c, words, row, j, m));
              return false;
            }
            uint8_t& f = seen[((size_t)row * G + j) * c.M + m];
            if (f) {
              std::printf("code (%d, %d, %d) listed twice\n", row, j, m);
              return false;
            }
            f = 1;
          }
      }
    }
  }
  for (uint8_t f : seen)
    if (!f) {
      std::printf("case %dx%d %dx%d: a code is missing\n", c.d_out, c.d_in, c.M, c.B);
      return false;
    }
  return true;
}

}  // namespace

int main() {
  const Case cases[] = {
      {16, 256, 1, 16, false}, {40, 520, 1, 16, false},   {7, 8, 1, 16, false},     {33, 1024, 1, 15, false},
      {48, 512, 2, 16, false}, {21, 136, 2, 15, false},   {21, 136, 2, 15, true},   {40, 1032, 1, 15, true},
      {1, 2048, 2, 16, false}, {1000, 4104, 1, 16, false}, {16400, 64, 1, 16, false},  // 1025 blocks: 16 threads
  };
  for (const Case& c : cases)
    if (!run(c)) return 1;
  std::printf("sorter sanitize ok\n");
  return 0;
}
