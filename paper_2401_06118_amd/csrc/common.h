// Shared device helpers for the gfx950 AQLM kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
// 3 and 4 words at a dword-aligned address (global loads of several dwords
// need only dword alignment)
typedef uint32_t u32x3a4_t __attribute__((ext_vector_type(3), aligned(4)));
typedef uint32_t u32x4a4_t __attribute__((ext_vector_type(4), aligned(4)));

namespace aqlm {

constexpr int kWave = 64;

// A compile-time integer passed as an argument, so that one lambda can be
// instantiated per value (register sets and unrolled schedules chosen at
// compile time).
template <int V>
struct IntC {
  static constexpr int value = V;
};

// Code storage: B <= 8 in one byte, 8 < B <= 16 in two (unpacked); a code
// is masked to its B bits before it indexes a codebook of 2^B codewords.
constexpr int code_bytes(int B) { return B > 8 ? 2 : 1; }
constexpr uint32_t code_mask(int B) { return (1u << B) - 1u; }

__device__ __forceinline__ float h2f(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
// Round to fp16 with the hardware conversion (round to nearest even under the
// default MODE; fp16 subnormals are kept).
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
__device__ __forceinline__ h2_t as_h2(uint32_t u) { return __builtin_bit_cast(h2_t, u); }

// <a, b> over the 8 fp16 lanes of two 16-byte vectors, added into four fp32
// partial sums (one per fp16 pair) to keep independent dependency chains.
__device__ __forceinline__ void dot8(const uint4& a, const uint4& b, float& s0, float& s1, float& s2,
                                     float& s3) {
  s0 = __builtin_amdgcn_fdot2(as_h2(a.x), as_h2(b.x), s0, false);
  s1 = __builtin_amdgcn_fdot2(as_h2(a.y), as_h2(b.y), s1, false);
  s2 = __builtin_amdgcn_fdot2(as_h2(a.z), as_h2(b.z), s2, false);
  s3 = __builtin_amdgcn_fdot2(as_h2(a.w), as_h2(b.w), s3, false);
}

// Sum of v over the 64 lanes of the wave, returned to every lane.  Inside a
// row of 16 lanes the sum uses DPP moves (no LDS traffic); the four row sums
// are then combined with readlane.
__device__ __forceinline__ float wave_sum(float v) {
  // quad_perm [1,0,3,2], [2,3,0,1], row_half_mirror, row_mirror
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, true));
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 48));
  return (r0 + r1) + (r2 + r3);
}

// Byte k (0..3) of a 32-bit word.
__device__ __forceinline__ uint32_t byte_of(uint32_t w, int k) { return (w >> (8 * k)) & 0xFFu; }

}  // namespace aqlm
