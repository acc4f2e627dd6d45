// Device helpers shared by the kernels that stream AQLM codes from HBM and
// look codewords up in LDS codebook copies (batch-1 and small-batch
// products).
#pragma once

#include "common.h"

namespace aqlm {

template <int B>
struct GCfg {
  static constexpr int kBpc = code_bytes(B);  // bytes per code
  static constexpr int kCPL = 16 / kBpc;      // codes per lane per item
  static constexpr int kKS = 4 * kCPL;        // codes per row per item
  static constexpr int kXL = (B == 8) ? 4 : 8;  // x staging loads per thread (groups <= kXL * 1024)
};

// Generic (unaligned-pitch) path: byte loads of the valid codes of a lane's
// 16-byte slot, zero past the row end.
template <int B>
__device__ __forceinline__ void load_codes_bytes(const uint8_t* __restrict__ row_ptr, uint32_t pitch, uint32_t off,
                                                 uint32_t (&w)[4]) {
  w[0] = w[1] = w[2] = w[3] = 0;
  const int nbytes = off < pitch ? (int)min(pitch - off, 16u) : 0;
#pragma unroll
  for (int b = 0; b < 16; ++b)
    if (b < nbytes) w[b / 4] |= (uint32_t)row_ptr[off + b] << (8 * (b % 4));
}

typedef __attribute__((address_space(3))) const u32x4_t lds_v4;

// 16-byte LDS load from an LDS byte address (ds_read_b128).
__device__ __forceinline__ uint4 lds_load16(uint32_t byte_addr) {
  const u32x4_t v = *(lds_v4*)(uintptr_t)byte_addr;
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// LDS byte address of codeword `code` of codebook m for this lane's copy.
// With 16 copies and M <= 2 the address is (m << 16) | (code << 8) | (copy << 4),
// built from the code byte with a single v_perm_b32: byte 0 and byte 2 come
// from base_m = (m << 16) | (copy << 4), byte 1 is byte `k` of the code word.
template <int M, int COPIES>
__device__ __forceinline__ uint32_t cw_addr(uint32_t word, int k, uint32_t base_m, uint32_t copy_off, int m) {
  if constexpr (COPIES == 16 && M <= 2) {
    (void)copy_off;
    (void)m;
    return __builtin_amdgcn_perm(word, base_m, 0x0C020000u | ((uint32_t)(4 + k) << 8));
  } else {
    (void)base_m;
    const uint32_t code = (word >> (8 * k)) & 0xFFu;
    return ((uint32_t)(m * 256) + code) * (uint32_t)(COPIES * 16) + copy_off;
  }
}

}  // namespace aqlm
