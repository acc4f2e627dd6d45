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
// BM tokens x BN rows, K-steps of 64.  Each step's X and W rows are loaded
// into registers two steps ahead and stored into one of two LDS stages
// one step ahead, one barrier per step.  LDS rows are 128 bytes (eight 16-byte chunks) with the
// chunk index XORed by bits 1..3 of the row, so that the fragment reads of 16
// consecutive rows, and the stores of two consecutive rows, hit 16 different
// bank quads without padding.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

namespace {

constexpr int kGfK = 64;  // reduction elements per step (two K32 MFMA halves)

// WM x WN waves; each wave owns FM 16-token blocks x FN 16-row blocks.
template <int WM, int WN, int FM, int FN>
struct GfCfg {
  static constexpr int kThreads = WM * WN * kWave;
  static constexpr int kBM = WM * FM * 16;  // tokens per workgroup
  static constexpr int kBN = WN * FN * 16;  // weight rows per workgroup
  static constexpr int kRows = kBM + kBN;   // LDS rows per stage: tokens, then weight rows
  static constexpr int kStageU4 = kRows * 8;
  static constexpr int kRowsPerLoad = kThreads / 8;  // stage rows one load round covers
  static constexpr int kLoads = kRows / kRowsPerLoad;  // 16-byte loads per thread per step
  static constexpr size_t kLds = 2 * (size_t)kStageU4 * 16;
  static_assert(kBM % kRowsPerLoad == 0 && kBN % kRowsPerLoad == 0,
                "a load round is all tokens or all weight rows");
};

// LDS position (in 16-byte units) of chunk c of stage row r.
__device__ __forceinline__ int gf_pos(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

struct GemmF16Args {
  const uint4* x;  // [n][K / 8]
  const uint4* w;  // [d_out][K / 8]
  uint16_t* y;     // [n][d_out]
  float* part;     // [splits][n][d_out] fp32 partial sums when splits > 1
  int32_t n;
  int32_t d_out;
  int32_t K;
  int32_t tok_tiles;
  int32_t row_tiles;
  int32_t splits;
};

template <int WM, int WN, int FM, int FN>
__global__ __launch_bounds__(WM * WN * kWave) void k_gemm_f16(const GemmF16Args a) {
  using P = GfCfg<WM, WN, FM, FN>;
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15, slot = lane >> 4;
  const int wm = wave % WM, wn = wave / WM;
  // Workgroup b takes token tile b % tok_tiles: the workgroups are dealt to
  // the 8 XCDs round-robin, so each XCD's L2 keeps its token tiles' X while
  // the weight tiles stream past.
  // With splits > 1 (too few tiles to fill the chip) the K-steps are divided
  // among `splits` workgroups per tile, each writing fp32 partial sums that
  // k_splitk_sum adds in a fixed order.
  const uint32_t b = blockIdx.x;
  const int32_t tok0 = (int32_t)(b % (uint32_t)a.tok_tiles) * P::kBM;
  const uint32_t rest = b / (uint32_t)a.tok_tiles;
  const int32_t row0 = (int32_t)(rest % (uint32_t)a.row_tiles) * P::kBN;
  const int split = (int)(rest / (uint32_t)a.row_tiles);
  const int32_t KU = a.K / 8;  // 16-byte chunks per row
  const int kall = a.K / kGfK;
  const int ks0 = (int)((int64_t)kall * split / a.splits);
  const int ksteps = (int)((int64_t)kall * (split + 1) / a.splits) - ks0;

  // Load j of this thread: stage row r = tid / 8 + kRowsPerLoad j, chunk tid % 8.  Rows
  // past the end read the last valid row (their results are not stored).
  const int lc = tid & 7;
  const uint4* src[P::kLoads];
  int dst[P::kLoads];
#pragma unroll
  for (int j = 0; j < P::kLoads; ++j) {
    const int r = (tid >> 3) + P::kRowsPerLoad * j;
    if (r < P::kBM) {
      int32_t t = tok0 + r;
      t = t < a.n ? t : a.n - 1;
      src[j] = a.x + (size_t)t * KU + (size_t)ks0 * (kGfK / 8) + lc;
    } else {
      int32_t i = row0 + (r - P::kBM);
      i = i < a.d_out ? i : a.d_out - 1;
      src[j] = a.w + (size_t)i * KU + (size_t)ks0 * (kGfK / 8) + lc;
    }
    dst[j] = gf_pos(r, lc);
  }
  f4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f4_t{0.f, 0.f, 0.f, 0.f};

  // Chunks move as u32x4_t (copies of uint4 from global memory would stay in
  // scratch memory instead of registers).  Loads run kDepth steps ahead of
  // their store into LDS, in kDepth register sets: set s holds the step j
  // with j % kDepth == s.  A step past the last reloads the last one, so
  // every load is unconditional and the wait before each store counts
  // exactly the loads issued after it.
  constexpr int kDepth = 2;  // three sets measured 2-3 % slower (more registers)
  u32x4_t* lds4 = reinterpret_cast<u32x4_t*>(lds);
  u32x4_t st[kDepth][P::kLoads];
  auto g_load = [&](int k, auto set) {
    constexpr int sidx = decltype(set)::value;
    const int kc = (k < ksteps ? k : ksteps - 1) * (kGfK / 8);
#pragma unroll
    for (int j = 0; j < P::kLoads; ++j) st[sidx][j] = *reinterpret_cast<const u32x4_t*>(src[j] + kc);
  };
  auto l_store = [&](int k, auto set) {
    constexpr int sidx = decltype(set)::value;
    u32x4_t* stage = lds4 + (k & 1) * P::kStageU4;
#pragma unroll
    for (int j = 0; j < P::kLoads; ++j) stage[dst[j]] = st[sidx][j];
  };
  const int xr0 = wm * FM * 16 + r16;          // this lane's token row in the stage
  const int wr0 = P::kBM + wn * FN * 16 + r16;  // this lane's weight row in the stage
  auto compute = [&](int k) {
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
  };
  // Step k (register set of step k + 1: NEXT): multiply stage k & 1, store
  // step k + 1 into the other stage (last read before the previous barrier),
  // then reuse NEXT for the loads of step k + 1 + kDepth.
  auto step = [&](int k, auto next) {
    compute(k);
    if (k + 1 < ksteps) l_store(k + 1, next);
    g_load(k + 1 + kDepth, next);
    lds_barrier();  // (the loads just issued stay in flight)
  };
  if constexpr (kDepth == 3) {
    g_load(0, IntC<0>{});
    g_load(1, IntC<1>{});
    g_load(2, IntC<2>{});
    l_store(0, IntC<0>{});
    g_load(3, IntC<0>{});
    __syncthreads();
    int k = 0;
    for (; k + 3 <= ksteps; k += 3) {
      step(k, IntC<1>{});
      step(k + 1, IntC<2>{});
      step(k + 2, IntC<0>{});
    }
    if (k < ksteps) step(k, IntC<1>{});
    if (k + 1 < ksteps) step(k + 1, IntC<2>{});
  } else {
    static_assert(kDepth == 2, "two or three register sets");
    g_load(0, IntC<0>{});
    g_load(1, IntC<1>{});
    l_store(0, IntC<0>{});
    g_load(2, IntC<0>{});
    __syncthreads();
    int k = 0;
    for (; k + 2 <= ksteps; k += 2) {
      step(k, IntC<1>{});
      step(k + 1, IntC<0>{});
    }
    if (k < ksteps) step(k, IntC<1>{});
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
        if (t >= a.n) continue;
        const size_t o = (size_t)t * a.d_out + row;
        if (a.splits == 1)
          a.y[o] = f2h(acc[fm][fn][e]);
        else
          a.part[(size_t)split * a.n * a.d_out + o] = acc[fm][fn][e];
      }
  }
}

// y = fp16(sum over splits of the partial sums), in split order.
__global__ __launch_bounds__(256) void k_splitk_sum(const float* __restrict__ part, uint16_t* __restrict__ y,
                                                    int64_t count, int32_t splits) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= count) return;
  float v = part[i];
  for (int s = 1; s < splits; ++s) v += part[(size_t)s * count + i];
  y[i] = f2h(v);
}

constexpr int kGfBM = 128, kGfBN = 128;  // the tile launched below

template <int WM, int WN, int FM, int FN>
hipError_t run_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, float* part, int32_t splits, int32_t n,
                        int32_t d_out, int32_t K, hipStream_t s) {
  using P = GfCfg<WM, WN, FM, FN>;
  static_assert(P::kLds <= 160 * 1024, "LDS budget");
  static_assert(P::kBM == kGfBM && P::kBN == kGfBN, "tile size used by gemm_f16_splits");
  auto kern = k_gemm_f16<WM, WN, FM, FN>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), 160 * 1024);
    if (e != hipSuccess) return e;
  }
  const int64_t row_tiles = (d_out + P::kBN - 1) / P::kBN;
  if (splits > 1) {  // one launch (the size query sized the partials for all n tokens)
    const int32_t tok_tiles = (n + P::kBM - 1) / P::kBM;
    const GemmF16Args a{reinterpret_cast<const uint4*>(x), reinterpret_cast<const uint4*>(w), y, part, n, d_out, K,
                        tok_tiles, (int32_t)row_tiles, splits};
    hipLaunchKernelGGL(kern, dim3((uint32_t)(row_tiles * tok_tiles * splits)), dim3(P::kThreads), P::kLds, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t count = (int64_t)n * d_out;
    hipLaunchKernelGGL(k_splitk_sum, dim3((uint32_t)((count + 255) / 256)), dim3(256), 0, s, part, y, count, splits);
    return hipGetLastError();
  }
  // token chunks small enough for a one-dimensional grid
  const int64_t chunk = ((int64_t)0x7FFFFFFF / row_tiles) * P::kBM;
  for (int64_t t0 = 0; t0 < n; t0 += chunk) {
    const int32_t nt = (int32_t)(n - t0 < chunk ? n - t0 : chunk);
    const int32_t tok_tiles = (nt + P::kBM - 1) / P::kBM;
    const GemmF16Args a{reinterpret_cast<const uint4*>(x + t0 * K), reinterpret_cast<const uint4*>(w), y + t0 * d_out,
                        nullptr, nt, d_out, K, tok_tiles, (int32_t)row_tiles, 1};
    hipLaunchKernelGGL(kern, dim3((uint32_t)(row_tiles * tok_tiles)), dim3(P::kThreads), P::kLds, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

bool gemm_f16_supported(int32_t d_in) { return d_in % kGfK == 0; }

// K-splits for a product whose 128 x 128 tiles fill at most half of the CUs:
// doubled while the tiles do not cover the CUs, up to 8 splits and at least
// 8 K-steps per split.  (At 11008 x 4096 x 256 tokens, 172 tiles on 256 CUs,
// two splits were slower than none: the partial sums cost more than the
// idle CUs.)
int32_t gemm_f16_splits(int64_t n, int64_t d_out, int64_t K) {
  const int64_t tiles = ((n + kGfBM - 1) / kGfBM) * ((d_out + kGfBN - 1) / kGfBN);
  const int64_t ksteps = K / kGfK;
  if (2 * tiles > num_cus()) return 1;
  // the grid and the partial-sum offsets stay below 2^31 entries per split
  if (n * d_out >= (int64_t(1) << 31)) return 1;
  int32_t s = 1;
  while (tiles * s < num_cus() && s < 8 && ksteps / (2 * s) >= 8) s *= 2;
  return s;
}

size_t gemm_f16_part_bytes(int64_t n, int64_t d_out, int64_t K) {
  const int32_t s = gemm_f16_splits(n, d_out, K);
  return s > 1 ? (size_t)s * (size_t)n * (size_t)d_out * sizeof(float) : 0;
}

// Tile: 128 tokens x 128 rows (8 waves of 64 x 32, two workgroups per CU).
// Measured at 256 and 2048 x 11008 x 4096: 256 x 128, 128 x 256 and 4-wave
// tiles (64 x 64 per wave) were as fast or slower, and 64 x 128 tiles (more
// workgroups for few tokens) took 88 us against 50 us at 256 tokens.  The
// same tile on v_mfma_f32_32x32x16_f16 (waves of 64 x 32 or 64 x 64) was
// 3-13 % slower at 2048 tokens.
// `part`: gemm_f16_part_bytes(n, d_out, K) bytes (unused when that is 0).
hipError_t launch_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, float* part, int32_t n, int32_t d_out,
                           int32_t K, hipStream_t s) {
  if (K % kGfK != 0 || n < 1 || d_out < 1) return hipErrorInvalidValue;
  const int32_t splits = gemm_f16_splits(n, d_out, K);
  if (splits > 1 && part == nullptr) return hipErrorInvalidValue;
  return run_gemm_f16<2, 4, 4, 2>(x, w, y, part, splits, n, d_out, K, s);
}

}  // namespace aqlm
