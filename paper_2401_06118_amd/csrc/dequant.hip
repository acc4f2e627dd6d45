// Dequantization of AQLM weights to fp16 (Eq. 2 with per-output scales,
// Fig. 3 steps i-v), bit-exact by construction:
//   acc = C_0[b_0][k]; acc = acc + C_m[b_m][k] for m = 1..M-1   (fp32, ascending m)
//   w   = fp16_rne(acc * s_i)                                     (one fp32 product)
// Each thread writes one group of 8 weights (16 bytes); consecutive threads
// write consecutive groups, so both the code reads and the fp16 writes are
// fully coalesced.  Bit-packed codes (12 or 15 bits) are cut out of the
// one or two 32-bit words that hold the group.  The kernel is bound by the 16-byte-per-group write
// stream.  For B = 8 the M codebooks (4 KiB each) sit in LDS, and so do the
// two 4096-entry codebooks of 2x12 (128 KiB, k_dequant_lds); wider codes read
// their codebooks (up to 2 x 1 MiB) through L2.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

template <int M, int B>
__device__ __forceinline__ void load_group_codes(const void* __restrict__ codes, uint32_t q, uint32_t (&c)[M]) {
  if constexpr (B > 8) {
    const uint16_t* p = static_cast<const uint16_t*>(codes) + (size_t)q * M;
    if constexpr (M == 2) {
      const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
      c[0] = v & code_mask(B);
      c[1] = (v >> 16) & code_mask(B);
    } else {
      c[0] = p[0] & code_mask(B);
    }
  } else {
    const uint8_t* p = static_cast<const uint8_t*>(codes) + (size_t)q * M;
    if constexpr (M == 2) {
      const uint32_t v = *reinterpret_cast<const uint16_t*>(p);
      c[0] = v & 0xFF;
      c[1] = v >> 8;
    } else if constexpr (M == 4) {
      const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
#pragma unroll
      for (int m = 0; m < 4; ++m) c[m] = byte_of(v, m);
    } else if constexpr (M == 8) {
      const uint2 v = *reinterpret_cast<const uint2*>(p);
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        c[m] = byte_of(v.x, m);
        c[m + 4] = byte_of(v.y, m);
      }
    } else {
#pragma unroll
      for (int m = 0; m < M; ++m) c[m] = p[m];
    }
  }
}

// Codes of group j of a row of bit-packed codes (words: the row's 32-bit
// words): code m is bits [(j*M + m)*B, + B) of the row, at most two words.
template <int M, int B>
__device__ __forceinline__ void load_group_codes_packed(const uint32_t* __restrict__ words, uint32_t j,
                                                        uint32_t (&c)[M]) {
  const uint32_t bit = j * (uint32_t)(M * B);
  const uint32_t w0 = bit >> 5, sh = bit & 31u;
  uint64_t v = words[w0];
  if (sh + (uint32_t)(M * B) > 32u) v |= (uint64_t)words[w0 + 1] << 32;  // (inside the row: the codes end there)
  v >>= sh;
#pragma unroll
  for (int m = 0; m < M; ++m) c[m] = (uint32_t)(v >> (m * B)) & code_mask(B);
}

__device__ __forceinline__ void unpack8(const uint4& v, float (&f)[8]) {
  f[0] = h2f(v.x & 0xFFFF); f[1] = h2f(v.x >> 16);
  f[2] = h2f(v.y & 0xFFFF); f[3] = h2f(v.y >> 16);
  f[4] = h2f(v.z & 0xFFFF); f[5] = h2f(v.z >> 16);
  f[6] = h2f(v.w & 0xFFFF); f[7] = h2f(v.w >> 16);
}

// The 8 weights of one group: fp32 sum of its M codewords in ascending m
// (fetch(m, e): codeword e of codebook m), times the row scale, rounded once.
template <int M, typename Fetch>
__device__ __forceinline__ uint4 group_weights(const uint32_t (&c)[M], float s, Fetch&& fetch) {
#pragma clang fp contract(off)
  float acc[8];
  unpack8(fetch(0, c[0]), acc);
#pragma unroll
  for (int m = 1; m < M; ++m) {
    float v[8];
    unpack8(fetch(m, c[m]), v);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = acc[k] + v[k];
  }
  uint32_t h[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    // The empty asm keeps the fp32 product as its own rounding step: without
    // it the backend folds product and conversion into one v_fma_mixlo_f16,
    // which rounds once (and turns a -0 product into +0).
    float t = acc[k] * s;
    asm volatile("" : "+v"(t));
    h[k] = f2h(t);
  }
  return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
}

template <int M, int B, bool PACKED>
__device__ __forceinline__ void group_codes(const void* __restrict__ codes, uint32_t q, uint32_t row, uint32_t G,
                                            uint32_t pwords, uint32_t (&c)[M]) {
  if constexpr (PACKED)
    load_group_codes_packed<M, B>(static_cast<const uint32_t*>(codes) + (size_t)row * pwords, q - row * G, c);
  else
    load_group_codes<M, B>(codes, q, c);
}

template <int M, int B, bool PACKED>
__global__ __launch_bounds__(256) void k_dequant(const void* __restrict__ codes, const uint4* __restrict__ cb,
                                                 const uint16_t* __restrict__ scales, uint32_t total_groups,
                                                 uint32_t G, uint32_t pwords, uint4* __restrict__ w) {
  constexpr int kLdsEntries = (B == 8) ? M * 256 : 1;
  __shared__ uint4 cb_lds[kLdsEntries];
  if constexpr (B == 8) {
    for (int e = threadIdx.x; e < M * 256; e += 256) cb_lds[e] = cb[e];
    lds_barrier();
  }
  const uint32_t stride = gridDim.x * 256u;
  for (uint32_t q = blockIdx.x * 256u + threadIdx.x; q < total_groups; q += stride) {
    const uint32_t row = q / G;
    uint32_t c[M];
    group_codes<M, B, PACKED>(codes, q, row, G, pwords, c);
    w[q] = group_weights<M>(c, h2f(scales[row]), [&](int m, uint32_t e) {
      return (B == 8) ? cb_lds[m * 256 + e] : cb[((uint32_t)m << B) + e];
    });
  }
}

// Two codebooks of 4096 codewords (2x12): both (128 KiB) fit in LDS, where
// random 16-byte reads from one copy run at about twice the rate of the same
// gathers from L2.  One 1024-thread workgroup per CU copies them once, then
// walks the groups like k_dequant.
constexpr int kDqLdsThreads = 1024;

template <int M, int B, bool PACKED>
__global__ __launch_bounds__(kDqLdsThreads) void k_dequant_lds(const void* __restrict__ codes,
                                                              const uint4* __restrict__ cb,
                                                              const uint16_t* __restrict__ scales,
                                                              uint32_t total_groups, uint32_t G, uint32_t pwords,
                                                              uint4* __restrict__ w) {
  extern __shared__ uint4 cb_lds[];  // [M << B]
  for (int e = threadIdx.x; e < (M << B); e += kDqLdsThreads) cb_lds[e] = cb[e];
  lds_barrier();
  const uint32_t stride = gridDim.x * (uint32_t)kDqLdsThreads;
  for (uint32_t q = blockIdx.x * (uint32_t)kDqLdsThreads + threadIdx.x; q < total_groups; q += stride) {
    const uint32_t row = q / G;
    uint32_t c[M];
    group_codes<M, B, PACKED>(codes, q, row, G, pwords, c);
    w[q] = group_weights<M>(c, h2f(scales[row]),
                            [&](int m, uint32_t e) { return cb_lds[((uint32_t)m << B) + e]; });
  }
}

template <int M, int B, bool PACKED = false>
static hipError_t run_dequant(const Layer& L, uint16_t* w, hipStream_t s) {
  const uint32_t total = (uint32_t)L.d_out * (uint32_t)L.G;
  const uint32_t pwords = PACKED ? (uint32_t)packed_row_words(L.G, M, B) : 0u;
  if constexpr (M == 2 && B == 12) {
    auto kern = k_dequant_lds<M, B, PACKED>;
    const int lds = (M << B) * 16;
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), lds);
    if (e != hipSuccess) return e;
    uint32_t blocks = (total + kDqLdsThreads - 1u) / kDqLdsThreads;
    const uint32_t cap = (uint32_t)num_cus();
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(kDqLdsThreads), lds, s, L.codes,
                       reinterpret_cast<const uint4*>(L.codebooks), L.scales, total, (uint32_t)L.G, pwords,
                       reinterpret_cast<uint4*>(w));
    return hipGetLastError();
  } else {
    uint32_t blocks = (total + 255u) / 256u;
    const uint32_t cap = (uint32_t)num_cus() * 8u;
    if (blocks > cap) blocks = cap;
    hipLaunchKernelGGL((k_dequant<M, B, PACKED>), dim3(blocks), dim3(256), 0, s, L.codes,
                       reinterpret_cast<const uint4*>(L.codebooks), L.scales, total, (uint32_t)L.G, pwords,
                       reinterpret_cast<uint4*>(w));
    return hipGetLastError();
  }
}

hipError_t launch_dequant(const Layer& L, uint16_t* w, hipStream_t s) {
  if (L.packed) {
    if (L.M == 1 && L.B == 15) return run_dequant<1, 15, true>(L, w, s);
    if (L.M == 2 && L.B == 12) return run_dequant<2, 12, true>(L, w, s);
    if (L.M == 2 && L.B == 15) return run_dequant<2, 15, true>(L, w, s);
    return hipErrorInvalidValue;
  }
  if (L.B > 8) {
    if (L.M == 1) return L.B == 16 ? run_dequant<1, 16>(L, w, s) : run_dequant<1, 15>(L, w, s);
    switch (L.B) {
      case 12: return run_dequant<2, 12>(L, w, s);
      case 15: return run_dequant<2, 15>(L, w, s);
      case 16: return run_dequant<2, 16>(L, w, s);
    }
    return hipErrorInvalidValue;
  }
  switch (L.M) {
    case 1: return run_dequant<1, 8>(L, w, s);
    case 2: return run_dequant<2, 8>(L, w, s);
    case 3: return run_dequant<3, 8>(L, w, s);
    case 4: return run_dequant<4, 8>(L, w, s);
    case 5: return run_dequant<5, 8>(L, w, s);
    case 6: return run_dequant<6, 8>(L, w, s);
    case 7: return run_dequant<7, 8>(L, w, s);
    case 8: return run_dequant<8, 8>(L, w, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
