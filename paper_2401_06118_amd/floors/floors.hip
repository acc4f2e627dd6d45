// Microbenchmarks of the GPU limits that the kernels' designs are measured
// against: the cost of a launch, of one dependent global load, the HBM read
// stream, the matrix-core issue rate, and the gather rates of LDS and L2.
// Measurement only: the product library neither links nor calls them, and
// bench.py --floors times them.  Each entry point launches one kernel on
// `stream` and returns the launch's hipError_t; buffers are the caller's.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Marks a gathered word as used without spending an instruction on it (the
// load stays a full 16-byte load).
__device__ __forceinline__ void consume(u32x4_t v) { asm volatile("" ::"v"(v)); }

__global__ __launch_bounds__(1024) void k_floor_empty() {}

// Thread 0 of each workgroup loads one word (a separate 256-byte line per
// workgroup), the workgroup meets at a barrier, every thread stores.
__global__ __launch_bounds__(1024) void k_floor_dep_load(const uint32_t* __restrict__ src,
                                                         uint32_t* __restrict__ dst) {
  __shared__ uint32_t v;
  if (threadIdx.x == 0) v = src[(size_t)blockIdx.x * 64];
  __syncthreads();
  dst[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = v + threadIdx.x;
}

// Read of n16 16-byte words: each round a workgroup of 256 threads reads a
// contiguous 32 KiB (eight independent loads per thread, each instruction a
// contiguous 4 KiB), and rounds step over the grid.  Indices past the end
// read the last word.  One word per thread is written so that nothing is
// removed.
__global__ __launch_bounds__(256) void k_floor_read(const u32x4_t* __restrict__ p, size_t n16,
                                                    uint32_t* __restrict__ out) {
  uint32_t acc = 0;
  for (size_t base = (size_t)blockIdx.x * 2048; base < n16; base += (size_t)gridDim.x * 2048) {
    u32x4_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const size_t i = base + (size_t)u * 256 + threadIdx.x;
      v[u] = p[i < n16 ? i : n16 - 1];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= (v[u].x + v[u].y) ^ (v[u].z + v[u].w);
  }
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

// Eight independent accumulation chains of v_mfma_f32_16x16x32_f16 per wave.
// The instruction is written out so that each chain keeps its own registers
// (accumulator and result in the same four registers); left to itself the
// register allocator moves the accumulators between register files on every
// round.  The result values are not used, only kept live.
__global__ __launch_bounds__(256) void k_floor_mfma(float* __restrict__ out, int iters) {
  const float t = (float)(threadIdx.x & 63) * 1e-3f;
  h8_t a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (_Float16)(t + 1e-4f * e);
    b[e] = (_Float16)(t - 1e-4f * e);
  }
  f4_t c0 = {t, 0.f, 0.f, 0.f}, c1 = {0.f, t, 0.f, 0.f}, c2 = {0.f, 0.f, t, 0.f}, c3 = {0.f, 0.f, 0.f, t},
       c4 = {2 * t, 0.f, 0.f, 0.f}, c5 = {0.f, 2 * t, 0.f, 0.f}, c6 = {0.f, 0.f, 2 * t, 0.f}, c7 = {0.f, 0.f, 0.f, 2 * t};
#define FLOOR_MFMA(c) asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "v"(b))
  for (int i = 0; i < iters; ++i) {
    FLOOR_MFMA(c0);
    FLOOR_MFMA(c1);
    FLOOR_MFMA(c2);
    FLOOR_MFMA(c3);
    FLOOR_MFMA(c4);
    FLOOR_MFMA(c5);
    FLOOR_MFMA(c6);
    FLOOR_MFMA(c7);
  }
#undef FLOOR_MFMA
  // (the last results are complete before the vector ALU reads them)
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  const f4_t s = ((c0 + c1) + (c2 + c3)) + ((c4 + c5) + (c6 + c7));
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s[0] + s[1] + s[2] + s[3];
}

__device__ __forceinline__ uint32_t xorshift(uint32_t x) {
  x ^= x << 13;
  x ^= x >> 17;
  return x ^ (x << 5);
}

// 16-byte LDS gathers from a table of 256 entries held in 16 copies (entry e,
// copy c at (16 e + c) * 16 bytes); lane l reads copy l % copies of random
// entries (the bytes of a per-lane xorshift word), eight independent gathers
// per round.
__global__ __launch_bounds__(1024) void k_floor_lds_gather(uint32_t* __restrict__ out, int iters, int copies) {
  __shared__ u32x4_t tab[256 * 16];
  for (int i = threadIdx.x; i < 256 * 16; i += 1024) tab[i] = u32x4_t{(uint32_t)i, 3u * i, 5u * i, 7u * i};
  __syncthreads();
  const uint32_t copy = (uint32_t)(threadIdx.x & 63) % (uint32_t)copies;
  uint32_t x = (blockIdx.x * 1024u + threadIdx.x) * 2654435761u + 1u;
  for (int it = 0; it < iters; ++it) {
    x = xorshift(x);
    const uint32_t y = xorshift(x ^ 0x9e3779b9u);
    u32x4_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = tab[(((u < 4 ? x : y) >> (8 * (u & 3))) & 255u) * 16u + copy];
#pragma unroll
    for (int u = 0; u < 8; ++u) consume(v[u]);
  }
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = x;
}

// 16-byte global gathers from a table of (mask + 1) entries (1 MiB: in L2
// after the first pass), eight independent gathers per round.
__global__ __launch_bounds__(1024) void k_floor_l2_gather(const u32x4_t* __restrict__ tab, uint32_t mask,
                                                          uint32_t* __restrict__ out, int iters) {
  uint32_t x = (blockIdx.x * 1024u + threadIdx.x) * 2654435761u + 7u;
  for (int it = 0; it < iters; ++it) {
    const uint32_t y = xorshift(x), z = xorshift(y);
    x = xorshift(z);
    u32x4_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t w = u < 2 ? x : (u < 4 ? y : (u < 6 ? z : (x ^ z)));
      v[u] = tab[(w >> (16 * (u & 1))) & mask];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) consume(v[u]);
  }
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = x;
}

}  // namespace

extern "C" {

// `blocks` workgroups of 1024 threads that do nothing.
int floor_empty(int blocks, hipStream_t stream) {
  if (blocks < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_floor_empty, dim3(blocks), dim3(1024), 0, stream);
  return (int)hipGetLastError();
}

// src: at least blocks * 64 words; dst: blocks * 1024 words.
int floor_dep_load(const uint32_t* src, uint32_t* dst, int blocks, hipStream_t stream) {
  if (!src || !dst || blocks < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_floor_dep_load, dim3(blocks), dim3(1024), 0, stream, src, dst);
  return (int)hipGetLastError();
}

// p: n16 16-byte words; out: blocks * 256 words.
int floor_read(const void* p, size_t n16, uint32_t* out, int blocks, hipStream_t stream) {
  if (!p || !out || blocks < 1) return (int)hipErrorInvalidValue;
  if (n16 == 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_floor_read, dim3(blocks), dim3(256), 0, stream, reinterpret_cast<const u32x4_t*>(p), n16, out);
  return (int)hipGetLastError();
}

// out: blocks * 256 floats; each wave issues 8 * iters MFMAs.
int floor_mfma(float* out, int blocks, int iters, hipStream_t stream) {
  if (!out || blocks < 1 || iters < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_floor_mfma, dim3(blocks), dim3(256), 0, stream, out, iters);
  return (int)hipGetLastError();
}

// out: blocks * 1024 words; each thread makes 8 * iters gathers; copies 1..16.
int floor_lds_gather(uint32_t* out, int blocks, int iters, int copies, hipStream_t stream) {
  if (!out || blocks < 1 || iters < 1 || copies < 1 || copies > 16) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_floor_lds_gather, dim3(blocks), dim3(1024), 0, stream, out, iters, copies);
  return (int)hipGetLastError();
}

// tab: entries 16-byte words, entries a power of two; out: blocks * 1024
// words; each thread makes 8 * iters gathers.
int floor_l2_gather(const void* tab, uint32_t entries, uint32_t* out, int blocks, int iters, hipStream_t stream) {
  if (!tab || !out || blocks < 1 || iters < 1 || entries == 0 || (entries & (entries - 1)) != 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_floor_l2_gather, dim3(blocks), dim3(1024), 0, stream, reinterpret_cast<const u32x4_t*>(tab),
                     entries - 1, out, iters);
  return (int)hipGetLastError();
}

}  // extern "C"
