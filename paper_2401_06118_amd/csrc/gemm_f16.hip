// Dense fp16 product on the matrix cores, second pass of the workspace
// prefill (aqlm_gemm):
//   Y[t][i] = fp16(sum_c X[t][c] W[i][c]),   fp32 accumulation,
// where W [d_out][d_in] is the dequantized weight matrix with the scales
// already applied (Eq. 2, written by k_dequant) and X [n][d_in] the
// activations.  Both operands are contiguous along the reduction dimension,
// which is the layout v_mfma_f32_16x16x32_f16 wants for both of its inputs
// (8 consecutive K values per lane), so no transposition is needed anywhere.
//
// Workgroup: a tile of BM tokens x BN weight rows, WM x WN waves, each wave
// FM x FN blocks of 16 x 16 outputs.  K runs in steps of 64 through S LDS
// stages.  Operands go from global memory straight into LDS
// (global_load_lds_dwordx4: each lane's 16 bytes land at the instruction's
// LDS address + 16 * lane), so no registers hold them on the way and no LDS
// store instructions are issued; one instruction fills 8 stage rows of 128
// bytes.  Stage rows hold the 16-byte chunk c of row r at chunk position
// c ^ ((r >> 1) & 7), so that the fragment reads of 16 consecutive rows hit
// 16 different bank quads; the loads apply the permutation on the global
// side (lane l of an instruction fetches the chunk that belongs at position
// l % 8).
//
// Each K-step is two halves of 32 (one MFMA K each).  Between two barriers a
// wave issues, in this order: the loads of step k + S - 1 into the stage of
// step k - 1; the first-half fragments of step k; the MFMAs of step k - 1's
// second half (fragments already in registers), which cover those reads'
// latency; the second-half fragments of step k; the MFMAs of step k's first
// half.  Then it waits for its own loads of step k + 1 and its fragment reads
// and meets the others at the barrier.  The matrix cores therefore have work
// queued while a wave waits for LDS, and across the barrier.
#include "common.h"
#include "launch.h"

namespace aqlm {

namespace {

typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kGfK = 64;  // reduction elements per step: one 128-byte stage row

template <int BM, int BN, int WM, int WN, int S>
struct GfCfg {
  static constexpr int kWaves = WM * WN;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int FM = BM / WM / 16;  // 16-token blocks per wave
  static constexpr int FN = BN / WN / 16;  // 16-row blocks per wave
  static constexpr int kRows = BM + BN;    // stage rows: tokens, then weight rows
  static constexpr int kStageU4 = kRows * 8;
  static constexpr int kInsts = kRows / 8;         // load instructions per stage
  static constexpr int kPer = kInsts / kWaves;     // ... per wave
  static constexpr size_t kLds = (size_t)S * kStageU4 * 16;
  static_assert(FM * WM * 16 == BM && FN * WN * 16 == BN, "tile");
  static_assert(kInsts % kWaves == 0 && BM % 8 == 0, "whole load instructions per wave, each all tokens or all rows");
  static_assert(S >= 2 && kPer * (S - 2) < 64, "stages; wait count");
  static_assert(kLds <= 160 * 1024, "LDS budget");
};

// LDS position (in 16-byte units) of chunk c of stage row r.
__device__ __forceinline__ int gf_pos(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

// 16 bytes per lane from global memory into LDS at l + 16 * lane (`l` is
// wave-uniform).  The builtin exists in the device pass only.
__device__ __forceinline__ void load_to_lds(const uint4* g, uint4* l) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_global_load_lds(g, (lds_void_t*)l, 16, 0, 0);
#endif
}

// Waits until at most N of this wave's vector-memory loads are in flight.
template <int N>
__device__ __forceinline__ void wait_loads() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier ordered for the compiler only.  The caller has waited
// for its own loads of the next step and for its own fragment reads of the
// stage that the next loads overwrite; a workgroup memory fence here would
// also wait for the loads still in flight for later steps.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

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

// Fragments of one 32-wide half of a K-step (chunk h * 4 + slot of the
// lane's rows).
template <int FM, int FN>
__device__ __forceinline__ void gf_read_half(const uint4* rd, int h, int xr0, int wr0, int slot, h8_t (&xf)[FM],
                                             h8_t (&wf)[FN]) {
  const int c = h * 4 + slot;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) xf[fm] = __builtin_bit_cast(h8_t, rd[gf_pos(xr0 + fm * 16, c)]);
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) wf[fn] = __builtin_bit_cast(h8_t, rd[gf_pos(wr0 + fn * 16, c)]);
}

template <int FM, int FN>
__device__ __forceinline__ void gf_mfma(const h8_t (&xf)[FM], const h8_t (&wf)[FN], f4_t (&acc)[FM][FN]) {
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      acc[fm][fn] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xf[fm], wf[fn], acc[fm][fn], 0, 0, 0);
}

// One barrier interval (see the top of the file): `rd` is the stage of step
// k, `wr` the stage of step k - 1 (no longer read), `xa`/`wa` step k - 1's
// second-half fragments on entry and step k's on return.  The two stage
// pointers are restrict parameters of an inlined function (the stages are
// different), which tells the compiler's wait-count insertion that the
// fragment reads do not depend on the loads just issued; it would otherwise
// wait for every load in flight before the first read.  Ordering across
// intervals is the explicit waits and the barrier of the caller, and the
// scheduling barriers keep the phases in the order above.
template <int FM, int FN, int PER>
__device__ __forceinline__ void gf_interval(const uint4* __restrict__ rd, uint4* __restrict__ wr,
                                            const uint4* const* src, int kc, int first_inst, int xr0, int wr0,
                                            int slot, f4_t (&acc)[FM][FN], h8_t (&xa)[FM], h8_t (&wa)[FN]) {
#pragma unroll
  for (int i = 0; i < PER; ++i) load_to_lds(src[i] + kc, wr + (first_inst + i) * 64);
  h8_t xb[FM], wb[FN];
  gf_read_half<FM, FN>(rd, 0, xr0, wr0, slot, xb, wb);
  __builtin_amdgcn_sched_barrier(0);
  gf_mfma<FM, FN>(xa, wa, acc);
  __builtin_amdgcn_sched_barrier(0);
  gf_read_half<FM, FN>(rd, 1, xr0, wr0, slot, xa, wa);
  __builtin_amdgcn_sched_barrier(0);
  gf_mfma<FM, FN>(xb, wb, acc);
}

// Waits until none of this wave's LDS reads is in flight.
__device__ __forceinline__ void wait_lds_reads() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8)); }

template <int BM, int BN, int WM, int WN, int S>
__global__ __launch_bounds__(WM * WN * kWave) void k_gemm_f16(const GemmF16Args a) {
  using P = GfCfg<BM, BN, WM, WN, S>;
  constexpr int FM = P::FM, FN = P::FN, PER = P::kPer;
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15, slot = lane >> 4;
  const int wm = wave % WM, wn = wave / WM;
  // Workgroups are dealt to the 8 XCDs round-robin (b % 8); XCD x takes a
  // contiguous range of tiles, token tiles fastest, so the workgroups that
  // share a weight tile share an L2.  With splits > 1 (too few tiles to fill
  // the chip) the K-steps are divided among `splits` workgroups per tile,
  // each writing fp32 partial sums that k_splitk_sum adds in a fixed order.
  uint32_t b = blockIdx.x;
  {
    const uint32_t T = gridDim.x, q = T / 8, r = T % 8, xcd = b % 8;
    b = xcd * q + (xcd < r ? xcd : r) + b / 8;
  }
  const int32_t tok0 = (int32_t)(b % (uint32_t)a.tok_tiles) * BM;
  const uint32_t rest = b / (uint32_t)a.tok_tiles;
  const int32_t row0 = (int32_t)(rest % (uint32_t)a.row_tiles) * BN;
  const int split = (int)(rest / (uint32_t)a.row_tiles);
  const int32_t KU = a.K / 8;  // 16-byte chunks per row
  const int kall = a.K / kGfK;
  const int ks0 = (int)((int64_t)kall * split / a.splits);
  const int ksteps = (int)((int64_t)kall * (split + 1) / a.splits) - ks0;

  // Load instruction i of this wave fills stage rows 8 q .. 8 q + 7
  // (q = wave * PER + i); lane l fetches the chunk of row 8 q + l / 8 that
  // belongs at position l % 8.  Rows past the end read the last valid row
  // (their results are not stored).
  const uint4* src[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int r = (wave * PER + i) * 8 + lane / 8;
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    if (r < BM) {
      int32_t t = tok0 + r;
      t = t < a.n ? t : a.n - 1;
      src[i] = a.x + (size_t)t * KU + (size_t)ks0 * (kGfK / 8) + c;
    } else {
      int32_t row = row0 + (r - BM);
      row = row < a.d_out ? row : a.d_out - 1;
      src[i] = a.w + (size_t)row * KU + (size_t)ks0 * (kGfK / 8) + c;
    }
  }
  f4_t acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = f4_t{0.f, 0.f, 0.f, 0.f};
  const int xr0 = wm * FM * 16 + r16;          // this lane's token row in the stage
  const int wr0 = BM + wn * FN * 16 + r16;     // this lane's weight row in the stage

  // Steps 0 .. S-2 into stages 0 .. S-2.  A step past the last reloads the
  // last one (into a stage that is not read again), so every interval issues
  // the same loads and the wait at its end counts exactly the loads of the
  // S - 2 steps issued after step k + 1's.
#pragma unroll
  for (int s = 0; s < S - 1; ++s) {
    const int kk = s < ksteps ? s : ksteps - 1;
#pragma unroll
    for (int i = 0; i < PER; ++i) load_to_lds(src[i] + kk * (kGfK / 8), lds + s * P::kStageU4 + (wave * PER + i) * 64);
  }
  // (step -1's second half: zero fragments, so the first interval adds 0)
  h8_t xa[FM], wa[FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) xa[fm] = h8_t{};
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) wa[fn] = h8_t{};
  wait_loads<PER * (S - 2)>();
  stage_barrier();
  // (one call site for every interval, so that all share the alias scopes)
  for (int k = 0; k < ksteps; ++k) {
    const int kn = k + S - 1;
    gf_interval<FM, FN, PER>(lds + (k % S) * P::kStageU4, lds + (kn % S) * P::kStageU4, src,
                             (kn < ksteps ? kn : ksteps - 1) * (kGfK / 8), wave * PER, xr0, wr0, slot, acc, xa, wa);
    wait_loads<PER * (S - 2)>();
    wait_lds_reads();
    stage_barrier();
  }
  gf_mfma<FM, FN>(xa, wa, acc);  // the last step's second half
  // (no load may still be writing LDS when the workgroup ends)
  wait_loads<0>();

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

// Tile shapes, each one workgroup per CU (the stages take 112-144 KiB of
// LDS), with their throughput per unit of tile area relative to 128 x 256,
// fitted so that whole rounds of tiles over the CUs pick the fastest shape
// measured at 256-2048 tokens x 4096-11008 rows x 4096-11008 inputs:
//   0: 128 x 128, 8 waves of 64 x 32, 4 stages   (0.80)
//   1: 128 x 256, 16 waves of 64 x 32, 3 stages  (1.00)
//   2: 256 x 192, 8 waves of 64 x 96, 2 stages   (1.05)
//   3: 256 x 256, 8 waves of 128 x 64, 2 stages  (1.10)
struct GfTile {
  int32_t bm, bn, speed;
};
constexpr GfTile kGfTiles[4] = {{128, 128, 80}, {128, 256, 100}, {256, 192, 105}, {256, 256, 110}};

int64_t gf_tiles(const GfTile& t, int64_t n, int64_t d_out) {
  return ((n + t.bm - 1) / t.bm) * ((d_out + t.bn - 1) / t.bn);
}

// The tile shape with the least time by whole rounds of tiles over the CUs
// (rounds x tile area / speed); ties go to the smaller tile.
int gf_choose(int64_t n, int64_t d_out) {
  const int64_t cus = num_cus();
  int best = 0;
  double best_cost = 0.0;
  for (int i = 0; i < 4; ++i) {
    const GfTile& t = kGfTiles[i];
    const int64_t rounds = (gf_tiles(t, n, d_out) + cus - 1) / cus;
    const double cost = (double)rounds * t.bm * t.bn / t.speed;
    if (i == 0 || cost < best_cost) {
      best = i;
      best_cost = cost;
    }
  }
  return best;
}

// K-splits (the 128 x 128 tile only): doubled while the split grid still fits
// one workgroup per CU, up to 8 splits and at least 8 K-steps per split.
int32_t gf_splits(int tile, int64_t n, int64_t d_out, int64_t K) {
  if (tile != 0) return 1;
  // the grid and the partial-sum offsets stay below 2^31 entries per split
  if (n * d_out >= (int64_t(1) << 31)) return 1;
  const int64_t tiles = gf_tiles(kGfTiles[0], n, d_out);
  const int64_t ksteps = K / kGfK;
  int32_t s = 1;
  while (2 * tiles * s <= num_cus() && s < 8 && ksteps / (2 * s) >= 8) s *= 2;
  return s;
}

template <int BM, int BN, int WM, int WN, int S>
hipError_t run_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, float* part, int32_t splits, int32_t n,
                        int32_t d_out, int32_t K, hipStream_t s) {
  using P = GfCfg<BM, BN, WM, WN, S>;
  auto kern = k_gemm_f16<BM, BN, WM, WN, S>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), 160 * 1024);
    if (e != hipSuccess) return e;
  }
  const int64_t row_tiles = (d_out + BN - 1) / BN;
  if (splits > 1) {  // one launch (the size query sized the partials for all n tokens)
    const int32_t tok_tiles = (n + BM - 1) / BM;
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
  const int64_t chunk = ((int64_t)0x7FFFFFFF / row_tiles) * BM;
  for (int64_t t0 = 0; t0 < n; t0 += chunk) {
    const int32_t nt = (int32_t)(n - t0 < chunk ? n - t0 : chunk);
    const int32_t tok_tiles = (nt + BM - 1) / BM;
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

size_t gemm_f16_part_bytes(int64_t n, int64_t d_out, int64_t K) {
  const int32_t s = gf_splits(gf_choose(n, d_out), n, d_out, K);
  return s > 1 ? (size_t)s * (size_t)n * (size_t)d_out * sizeof(float) : 0;
}

// `part`: gemm_f16_part_bytes(n, d_out, K) bytes (unused when that is 0).
// Measured against the previous design (registers staging two K-steps ahead,
// 128 x 128 tiles, two workgroups per CU), same box: 2048 x 11008 x 4096
// 264 -> 165-172 us, 1024 rows 137 -> 83 us, 512 rows 101 -> 51 us,
// 256 rows 44 -> 34 us.
hipError_t launch_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, float* part, int32_t n, int32_t d_out,
                           int32_t K, hipStream_t s) {
  if (K % kGfK != 0 || n < 1 || d_out < 1) return hipErrorInvalidValue;
  const int tile = gf_choose(n, d_out);
  const int32_t splits = gf_splits(tile, n, d_out, K);
  if (splits > 1 && part == nullptr) return hipErrorInvalidValue;
  switch (tile) {
    case 0: return run_gemm_f16<128, 128, 2, 4, 4>(x, w, y, part, splits, n, d_out, K, s);
    case 1: return run_gemm_f16<128, 256, 2, 8, 3>(x, w, y, part, splits, n, d_out, K, s);
    case 2: return run_gemm_f16<256, 192, 4, 2, 2>(x, w, y, part, splits, n, d_out, K, s);
    default: return run_gemm_f16<256, 256, 2, 4, 2>(x, w, y, part, splits, n, d_out, K, s);
  }
}

}  // namespace aqlm
