// Groups larger than 8 inputs (g = 16, 32 or 64) with 8-bit codes: the
// codebooks-versus-groups settings of the paper's ablation (4x8 with groups
// of 16, 8x8 with 32, 15x8 with 64 - about two bits per weight each).
//
// A code of group j selects a codeword of g values; the kernels see it as
// g / 8 chunks of 8 (chunk p of codeword e of codebook m is the 16 bytes at
// ((m * 256 + e) * (g / 8) + p) * 16 of the codebook tensor), so every code
// is used for g / 8 consecutive 8-input chunks of the row.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace aqlm {

struct GroupLayer {
  const uint8_t* codes;       // [d_out][d_in / g][M]
  const uint16_t* codebooks;  // [M][256][g] fp16
  const uint16_t* scales;     // [d_out] fp16
  int32_t d_out;
  int32_t d_in;
  int32_t M;  // 1 .. 16
  int32_t g;  // 16, 32 or 64
};

constexpr bool groups_supported(int M, int B, int g) {
  return B == 8 && M >= 1 && M <= 16 && (g == 16 || g == 32 || g == 64);
}

// W as fp16 (Eq. 2, bit-exact with the g = 8 rule: fp32 sum of the M
// codewords in ascending m from codeword 0, one fp32 product with the scale,
// one rounding).
hipError_t launch_dequant_groups(const GroupLayer& L, uint16_t* w, hipStream_t s);
// y = fp16(s * sum_chunks <sum_m codeword chunk, x chunk>), fp32 accumulation,
// deterministic.
hipError_t launch_gemv_groups(const GroupLayer& L, const uint16_t* x, uint16_t* y, hipStream_t s);

}  // namespace aqlm
