// Tiled storage of 8-bit codes for the batch-1 product.  The matrix-vector
// kernel reads, per wave and step, the 64-byte K-slice of 16 rows; stored
// row-major those are 16 half-lines a row pitch apart, tiled they are one
// contiguous 1 KiB (layout: tiled_codes_offset in launch.h).  The codes
// themselves, and so Eq. 2's result, are unchanged.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "launch.h"

namespace aqlm {
namespace {

// One thread per 16 destination bytes (a quarter of one row's 64 bytes in a
// tile); source bytes are read one by one (rows need not be 16-byte aligned).
__global__ __launch_bounds__(256) void k_tile_codes(const uint8_t* __restrict__ codes, int64_t d_out,
                                                   int64_t row_bytes, int64_t ks_per_row, int64_t chunks,
                                                   uint8_t* __restrict__ tiled) {
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < chunks;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t tile = q >> 6, within = q & 63;  // 64 chunks of 16 bytes per tile
    const int64_t r = (tile / ks_per_row) * 16 + (within >> 2);
    const int64_t c0 = (tile % ks_per_row) * 64 + (within & 3) * 16;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (r < d_out) {
      const uint8_t* src = codes + r * row_bytes;
#pragma unroll
      for (int b = 0; b < 16; ++b)
        if (c0 + b < row_bytes) w[b >> 2] |= (uint32_t)src[c0 + b] << (8 * (b & 3));
    }
    *reinterpret_cast<uint4*>(tiled + q * 16) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

}  // namespace

hipError_t launch_tile_codes(const uint8_t* codes, int64_t d_out, int64_t row_bytes, uint8_t* tiled, hipStream_t s) {
  if (d_out < 1 || row_bytes < 1) return hipErrorInvalidValue;
  const int64_t ks_per_row = (row_bytes + 63) / 64;
  const int64_t chunks = tiled_codes_bytes(d_out, row_bytes) / 16;
  int64_t blocks = (chunks + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_tile_codes, dim3((unsigned)blocks), dim3(256), 0, s, codes, d_out, row_bytes, ks_per_row,
                     chunks, tiled);
  return hipGetLastError();
}

}  // namespace aqlm
