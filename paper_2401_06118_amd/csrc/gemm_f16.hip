// Dense fp16 product on the matrix cores, second pass of the workspace
// prefill (aqlm_gemm):
//   Y[t][i] = fp16(sum_c X[t][c] W[i][c]),   fp32 accumulation,
// where W [d_out][d_in] is the dequantized weight matrix with the scales
// already applied (Eq. 2, written by k_dequant) and X [n][d_in] the
// activations.  Both operands are contiguous along the reduction dimension,
// which is the layout v_mfma_f32_16x16x32_f16 wants for both of its inputs
// (8 consecutive K values per lane), so no transposition is needed anywhere.
//
// Workgroup: 512 threads (8 waves, 2 along tokens x 4 along rows), a tile of
// BM tokens x BN rows, K-steps of 64.  Each step's X and W rows are copied
// global -> registers -> LDS one step ahead (double-buffered stages), one
// barrier per step.  LDS rows are 128 bytes (eight 16-byte chunks) with the
// chunk index XORed by bits 1..3 of the row, so that the fragment reads of 16
// consecutive rows, and the stores of two consecutive rows, hit 16 different
// bank quads without padding.
#include "common.h"
#include "launch.h"

namespace aqlm {

namespace {

constexpr int kGfThreads = 512;
constexpr int kGfK = 64;  // reduction elements per step (two K32 MFMA halves)

template <int FM, int FN>  // per wave: FM 16-token blocks x FN 16-row blocks
struct GfCfg {
  static constexpr int kBM = 2 * FM * 16;  // tokens per workgroup
  static constexpr int kBN = 4 * FN * 16;  // weight rows per workgroup
  static constexpr int kRows = kBM + kBN;  // LDS rows per stage: tokens, then weight rows
  static constexpr int kStageU4 = kRows * 8;
  static constexpr int kLoads = kRows * 8 / kGfThreads;  // 16-byte loads per thread per step
  static constexpr size_t kLds = 2 * (size_t)kStageU4 * 16;
  static_assert(kBM % 64 == 0 && kBN % 64 == 0, "a load round (64 rows) is all tokens or all weight rows");
};

// LDS position (in 16-byte units) of chunk c of stage row r.
__device__ __forceinline__ int gf_pos(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

struct GemmF16Args {
  const uint4* x;  // [n][K / 8]
  const uint4* w;  // [d_out][K / 8]
  uint16_t* y;     // [n][d_out]
  int32_t n;
  int32_t d_out;
  int32_t K;
  int32_t tok_tiles;
};

template <int FM, int FN>
__global__ __launch_bounds__(kGfThreads) void k_gemm_f16(const GemmF16Args a) {
  using P = GfCfg<FM, FN>;
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15, slot = lane >> 4;
  const int wm = wave & 1, wn = wave >> 1;
  // Workgroup b takes token tile b % tok_tiles: the workgroups are dealt to
  // the 8 XCDs round-robin, so each XCD's L2 keeps its token tiles' X while
  // the weight tiles stream past.
  const int32_t tok0 = (int32_t)(blockIdx.x % (uint32_t)a.tok_tiles) * P::kBM;
  const int32_t row0 = (int32_t)(blockIdx.x / (uint32_t)a.tok_tiles) * P::kBN;
  const int32_t KU = a.K / 8;  // 16-byte chunks per row
  const int ksteps = a.K / kGfK;

  // Load j of this thread: stage row r = tid / 8 + 64 j, chunk tid % 8.  Rows
  // past the end read the last valid row (their results are not stored).
  const int lc = tid & 7;
  const uint4* src[P::kLoads];
  int dst[P::kLoads];
#pragma unroll
  for (int j = 0; j < P::kLoads; ++j) {
    const int r = (tid >> 3) + 64 * j;
    if (r < P::kBM) {
      int32_t t = tok0 + r;
      t = t < a.n ? t : a.n - 1;
      src[j] = a.x + (size_t)t * KU + lc;
    } else {
      int32_t i = row0 + (r - P::kBM);
      i = i < a.d_out ? i : a.d_out - 1;
      src[j] = a.w + (size_t)i * KU + lc;
    }
    dst[j] = gf_pos(r, lc);
  }
  f4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f4_t{0.f, 0.f, 0.f, 0.f};

  // (chunks move as u32x4_t: copies of uint4 from global memory stay in
  // scratch memory instead of registers)
  u32x4_t* lds4 = reinterpret_cast<u32x4_t*>(lds);
  {
    u32x4_t st[P::kLoads];
#pragma unroll
    for (int j = 0; j < P::kLoads; ++j) st[j] = *reinterpret_cast<const u32x4_t*>(src[j]);
#pragma unroll
    for (int j = 0; j < P::kLoads; ++j) lds4[dst[j]] = st[j];
  }
  __syncthreads();
  const int xr0 = wm * FM * 16 + r16;          // this lane's token row in the stage
  const int wr0 = P::kBM + wn * FN * 16 + r16;  // this lane's weight row in the stage
  for (int k = 0; k < ksteps; ++k) {
    // Step k + 1's chunks (past the last step the last one is reloaded, so
    // every load is unconditional and the wait before each store is exact);
    // the scheduling barrier keeps them ahead of this step's multiplies.
    const int kn = (k + 1 < ksteps ? k + 1 : k) * (kGfK / 8);
    u32x4_t st[P::kLoads];
#pragma unroll
    for (int j = 0; j < P::kLoads; ++j) st[j] = *reinterpret_cast<const u32x4_t*>(src[j] + kn);
    __builtin_amdgcn_sched_barrier(0);
    const u32x4_t* stage = lds4 + (k & 1) * P::kStageU4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = h * 4 + slot;  // this lane's 8 K values: chunk c of its rows
      h8_t xf[FM], wf[FN];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) xf[fm] = __builtin_bit_cast(h8_t, stage[gf_pos(xr0 + fm * 16, c)]);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) wf[fn] = __builtin_bit_cast(h8_t, stage[gf_pos(wr0 + fn * 16, c)]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
          acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xf[fm], wf[fn], acc[fm][fn], 0, 0, 0);
    }
    if (k + 1 < ksteps) {  // stage (k+1)&1 was last read before the previous barrier
      u32x4_t* next = lds4 + ((k + 1) & 1) * P::kStageU4;
#pragma unroll
      for (int j = 0; j < P::kLoads; ++j) next[dst[j]] = st[j];
    }
    __syncthreads();
  }

  // D[token][row]: lane holds row r16 of its block and tokens 4 * slot + e.
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int32_t row = row0 + wn * FN * 16 + fn * 16 + r16;
    if (row >= a.d_out) continue;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int32_t t = tok0 + wm * FM * 16 + fm * 16 + 4 * slot + e;
        if (t < a.n) a.y[(size_t)t * a.d_out + row] = f2h(acc[fm][fn][e]);
      }
  }
}

template <int FM, int FN>
hipError_t run_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, int32_t n, int32_t d_out, int32_t K,
                        hipStream_t s) {
  using P = GfCfg<FM, FN>;
  static_assert(P::kLds <= 160 * 1024, "LDS budget");
  auto kern = k_gemm_f16<FM, FN>;
  static bool attr_set = false;  // set once per kernel; a repeated set is harmless
  if (!attr_set) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int64_t row_tiles = (d_out + P::kBN - 1) / P::kBN;
  // token chunks small enough for a one-dimensional grid
  const int64_t chunk = ((int64_t)0x7FFFFFFF / row_tiles) * P::kBM;
  for (int64_t t0 = 0; t0 < n; t0 += chunk) {
    const int32_t nt = (int32_t)(n - t0 < chunk ? n - t0 : chunk);
    const int32_t tok_tiles = (nt + P::kBM - 1) / P::kBM;
    const GemmF16Args a{reinterpret_cast<const uint4*>(x + t0 * K), reinterpret_cast<const uint4*>(w), y + t0 * d_out,
                        nt, d_out, K, tok_tiles};
    hipLaunchKernelGGL(kern, dim3((uint32_t)(row_tiles * tok_tiles)), dim3(kGfThreads), P::kLds, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

bool gemm_f16_supported(int32_t d_in) { return d_in % kGfK == 0; }

// Tile choice: 256 tokens x 128 rows; 128 x 128 when that leaves fewer than
// two tiles per CU.
hipError_t launch_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, int32_t n, int32_t d_out, int32_t K,
                           hipStream_t s) {
  if (K % kGfK != 0 || n < 1 || d_out < 1) return hipErrorInvalidValue;
  const int64_t big = ((n + 255) / 256) * (int64_t)((d_out + 127) / 128);
  if (big >= 2 * num_cus()) return run_gemm_f16<8, 2>(x, w, y, n, d_out, K, s);
  return run_gemm_f16<4, 2>(x, w, y, n, d_out, K, s);
}

}  // namespace aqlm
