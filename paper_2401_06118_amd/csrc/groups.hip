// Dequantization and the batch-1 product for groups of 16, 32 or 64 inputs
// (8-bit codes, up to 16 codebooks): the codebooks-versus-groups settings of
// the paper's ablation.  Eq. 2 is unchanged; only a codeword now spans g / 8
// chunks of 8 inputs, each chunk a 16-byte slice of the codeword.
//
// These formats have no GPU speed figure in the paper (its GPU kernels cover
// 1x16 and 2x8); the kernels here are plain vector-ALU ones:
//   k_dequant_groups  one thread per 8-input chunk, codeword chunks gathered
//                     from L2 (up to 512 KiB of codebooks), fp32 sums in
//                     ascending m, one product with the scale, one rounding;
//   k_gemv_groups     one wave per output row; each lane adds the M codeword
//                     chunks of its input chunks in fp32 and multiplies them
//                     with x; a fixed-order wave sum, the scale, one rounding.
//                     The codebooks sit in LDS (one copy) when they fit
//                     (up to 128 KiB: 4x8 gs16 32 KiB, 8x8 gs32 128 KiB),
//                     else are gathered from L2 (15x8 gs64, 480 KiB).
#include "common.h"
#include "groups.h"
#include "launch.h"

namespace aqlm {

namespace {

constexpr int kGrpThreads = 1024;
constexpr int kGrpWaves = kGrpThreads / kWave;
constexpr size_t kGrpCbLds = 128 * 1024;

__device__ __forceinline__ void add8(const uint4& v, float (&f)[8]) {
  f[0] += h2f(v.x & 0xFFFF); f[1] += h2f(v.x >> 16);
  f[2] += h2f(v.y & 0xFFFF); f[3] += h2f(v.y >> 16);
  f[4] += h2f(v.z & 0xFFFF); f[5] += h2f(v.z >> 16);
  f[6] += h2f(v.w & 0xFFFF); f[7] += h2f(v.w >> 16);
}

__device__ __forceinline__ void set8(const uint4& v, float (&f)[8]) {
  f[0] = h2f(v.x & 0xFFFF); f[1] = h2f(v.x >> 16);
  f[2] = h2f(v.y & 0xFFFF); f[3] = h2f(v.y >> 16);
  f[4] = h2f(v.z & 0xFFFF); f[5] = h2f(v.z >> 16);
  f[6] = h2f(v.w & 0xFFFF); f[7] = h2f(v.w >> 16);
}

__global__ __launch_bounds__(256) void k_dequant_groups(const GroupLayer L, uint32_t total, uint4* __restrict__ w) {
#pragma clang fp contract(off)
  const uint32_t k = (uint32_t)L.g / 8u;            // chunks per group
  const uint32_t G = (uint32_t)(L.d_in / L.g);      // groups per row
  const uint32_t per_row = (uint32_t)L.d_in / 8u;   // chunks per row
  const uint32_t M = (uint32_t)L.M;
  const uint4* __restrict__ cb = reinterpret_cast<const uint4*>(L.codebooks);
  const uint32_t stride = gridDim.x * 256u;
  for (uint32_t q = blockIdx.x * 256u + threadIdx.x; q < total; q += stride) {
    const uint32_t row = q / per_row;
    const uint32_t c = q - row * per_row;
    const uint32_t j = c / k, p = c - j * k;
    const uint8_t* __restrict__ code = L.codes + ((size_t)row * G + j) * M;
    float acc[8];
    set8(cb[(uint32_t)code[0] * k + p], acc);
    for (uint32_t m = 1; m < M; ++m) add8(cb[((m << 8) + (uint32_t)code[m]) * k + p], acc);
    const float s = h2f(L.scales[row]);
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      // the product keeps its own rounding step (no fused multiply-round)
      float t = acc[e] * s;
      asm volatile("" : "+v"(t));
      h[e] = f2h(t);
    }
    w[q] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
  }
}

template <bool LDS>
__global__ __launch_bounds__(kGrpThreads) void k_gemv_groups(const GroupLayer L, const uint4* __restrict__ x,
                                                             uint16_t* __restrict__ y) {
  extern __shared__ uint4 cb_lds[];
  const uint32_t k = (uint32_t)L.g / 8u;
  const uint32_t G = (uint32_t)(L.d_in / L.g);
  const uint32_t per_row = (uint32_t)L.d_in / 8u;
  const uint32_t M = (uint32_t)L.M;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const uint4* __restrict__ cb = reinterpret_cast<const uint4*>(L.codebooks);
  if constexpr (LDS) {
    const uint32_t entries = M * 256u * k;
    for (uint32_t e = threadIdx.x; e < entries; e += kGrpThreads) cb_lds[e] = cb[e];
    __syncthreads();
  }
  const uint4* src = LDS ? cb_lds : cb;
  for (int32_t row = blockIdx.x * kGrpWaves + wave; row < L.d_out; row += gridDim.x * kGrpWaves) {
    const uint8_t* __restrict__ rc = L.codes + (size_t)row * G * M;
    float acc = 0.f;
    for (uint32_t c = (uint32_t)lane; c < per_row; c += kWave) {
      const uint32_t j = c / k, p = c - j * k;
      const uint8_t* __restrict__ code = rc + (size_t)j * M;
      float u[8];
      set8(src[(uint32_t)code[0] * k + p], u);
      for (uint32_t m = 1; m < M; ++m) add8(src[((m << 8) + (uint32_t)code[m]) * k + p], u);
      const uint4 xv = x[c];
      acc += u[0] * h2f(xv.x & 0xFFFF) + u[1] * h2f(xv.x >> 16) + u[2] * h2f(xv.y & 0xFFFF) +
             u[3] * h2f(xv.y >> 16) + u[4] * h2f(xv.z & 0xFFFF) + u[5] * h2f(xv.z >> 16) +
             u[6] * h2f(xv.w & 0xFFFF) + u[7] * h2f(xv.w >> 16);
    }
    const float sum = wave_sum(acc);
    if (lane == 0) y[row] = f2h(h2f(L.scales[row]) * sum);
  }
}

}  // namespace

hipError_t launch_dequant_groups(const GroupLayer& L, uint16_t* w, hipStream_t s) {
  const uint32_t total = (uint32_t)((int64_t)L.d_out * (L.d_in / 8));
  uint32_t blocks = (total + 255u) / 256u;
  const uint32_t cap = (uint32_t)num_cus() * 8u;
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL(k_dequant_groups, dim3(blocks), dim3(256), 0, s, L, total, reinterpret_cast<uint4*>(w));
  return hipGetLastError();
}

hipError_t launch_gemv_groups(const GroupLayer& L, const uint16_t* x, uint16_t* y, hipStream_t s) {
  const size_t cb_bytes = (size_t)L.M * 256 * (size_t)L.g * 2;
  const int32_t row_blocks = (L.d_out + kGrpWaves - 1) / kGrpWaves;
  int32_t grid = num_cus();
  if (grid > row_blocks) grid = row_blocks;
  const uint4* xv = reinterpret_cast<const uint4*>(x);
  if (cb_bytes <= kGrpCbLds) {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(k_gemv_groups<true>), (int)kGrpCbLds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_gemv_groups<true>, dim3(grid), dim3(kGrpThreads), cb_bytes, s, L, xv, y);
  } else {
    hipLaunchKernelGGL(k_gemv_groups<false>, dim3(grid), dim3(kGrpThreads), 0, s, L, xv, y);
  }
  return hipGetLastError();
}

}  // namespace aqlm
