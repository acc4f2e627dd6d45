// Gradients through Eq. 2: the backward pass of y = x W^T with W in AQLM form,
// for fine-tuning codebooks and scales (Sec. 3, "Phase 2" and "Phase 3";
// App. "End-to-end fine-tuning").
//
// With G[i][c] = sum_t dy[t][i] x[t][c] (the weight gradient) and u[i][c] the
// fp32 sum of the codewords of row i, group c / 8 (Eq. 2 before the scale):
//   dC_m[e][k] += sum over (i, j) with b_ijm = e of s_i * G[i][8j + k]
//   ds_i       += sum_c G[i][c] * u[i][c]
//
// The weight gradient is never stored.  A workgroup computes a 128-row x
// 128-input tile of G on the matrix cores (v_mfma_f32_16x16x32_f16, the
// reduction runs over the tokens), then scatters it straight from the
// accumulators: each value looks its row's codes up (the tile's codes and
// scales are staged in LDS first), adds s_i * G into an
// fp32 copy of dC in LDS (one per workgroup, so LDS atomics take the
// collisions of equal codes) and G * u into the row's dscale partial.  The
// workgroups are persistent (about two per CU) and flush their LDS copy of dC
// into the output with one global atomic add per non-zero entry at the end.
//
// Both operands of the contraction are stored token-major (dy [n][d_out],
// x [n][d_in]), but an MFMA lane needs 8 consecutive tokens of one row: each
// K-step (32 tokens) is loaded with coalesced 16-byte reads of 8 rows of one
// token and written to LDS transposed ([row][token], pitch 40 halfs, so each
// fragment read is one 16-byte LDS read), double-buffered, one barrier per
// step.
//
// Summation order: G is fp32 over tokens in MFMA order; the scatter uses
// atomic adds, so dC and ds agree with the oracle to fp32 accuracy but are not
// bit-reproducible from run to run.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

namespace {

constexpr int kBwThreads = 512;      // 8 waves: 2 along rows x 4 along inputs
constexpr int kBwT = 128;            // rows and inputs per tile
constexpr int kBwK = 32;             // tokens per step
constexpr int kBwP = kBwK + 8;       // LDS pitch of a staged row, in halfs (80 bytes)
constexpr int kBwStage = 2 * kBwT * kBwP;  // halfs of one stage buffer (dy rows, then x rows)

struct BwArgs {
  const uint8_t* codes;  // [d_out][G][M]
  const uint16_t* cb;    // [M][256][8]
  const uint16_t* scales;
  const uint16_t* x;   // [n][d_in]
  const uint16_t* dy;  // [n][d_out]
  float* dcb;          // [M][256][8], accumulated
  float* ds;           // [d_out], accumulated
  int32_t d_out;
  int32_t d_in;
  int32_t n;
  int32_t tiles_c;
  int32_t tiles;
};

template <int M>
constexpr size_t bw_lds_bytes() {
  return (size_t)M * 2048 * 4 + (size_t)M * 2048 * 2 + (size_t)2 * kBwStage * 2 + (size_t)kBwT * 16 * M +
         (size_t)kBwT * 4;
}

template <int M>
__global__ __launch_bounds__(kBwThreads) void k_grad_cb(const BwArgs a) {
  extern __shared__ uint4 lds_u4[];
  float* dcl = reinterpret_cast<float*>(lds_u4);     // [M][256][8] fp32 partial dC
  uint16_t* cbl = reinterpret_cast<uint16_t*>(dcl + M * 2048);  // [M][256][8] fp16 codebooks
  uint16_t* stg = cbl + M * 2048;                    // [2][256][kBwP]: rows 0..127 dy, 128..255 x
  uint8_t* tcodes = reinterpret_cast<uint8_t*>(stg + 2 * kBwStage);  // [128][16 groups][M] codes of the tile
  float* tscales = reinterpret_cast<float*>(tcodes + kBwT * 16 * M);  // [128] scales of the tile
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15, slot = lane >> 4;
  const int wm = wave & 1, wn = wave >> 1;  // rows 64 wm .. + 63, inputs 32 wn .. + 31 of the tile
  const int32_t G = a.d_in / 8;

  for (int e = tid; e < M * 2048; e += kBwThreads) {
    dcl[e] = 0.f;
    cbl[e] = a.cb[e];
  }

  // Loader role: token lt of the step, 8 rows / inputs starting at 8 * lch.
  // The 64 lanes of a wave take 32 tokens of two row chunks, so each of
  // their transposed 2-byte stores hits one of 32 different dwords (two
  // lanes per dword, one half each) in 32 different banks.
  const int lt = tid & 31, lch = tid >> 5;
  const int nsteps = (a.n + kBwK - 1) / kBwK;
  auto load = [&](int step, int32_t i0, int32_t c0, uint4& vd, uint4& vx) {
    const int32_t t = step * kBwK + lt;
    const int32_t i = i0 + 8 * lch, c = c0 + 8 * lch;
    vd = make_uint4(0, 0, 0, 0);
    vx = make_uint4(0, 0, 0, 0);
    if (t < a.n && i < a.d_out) vd = *reinterpret_cast<const uint4*>(a.dy + (size_t)t * a.d_out + i);
    if (t < a.n && c < a.d_in) vx = *reinterpret_cast<const uint4*>(a.x + (size_t)t * a.d_in + c);
  };
  auto store = [&](int buf, const uint4& vd, const uint4& vx) {
    uint16_t* s = stg + buf * kBwStage;
    const uint32_t d[4] = {vd.x, vd.y, vd.z, vd.w}, xx[4] = {vx.x, vx.y, vx.z, vx.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      s[(8 * lch + e) * kBwP + lt] = (uint16_t)(d[e / 2] >> (16 * (e % 2)));
      s[(kBwT + 8 * lch + e) * kBwP + lt] = (uint16_t)(xx[e / 2] >> (16 * (e % 2)));
    }
  };

  for (int tile = blockIdx.x; tile < a.tiles; tile += gridDim.x) {
    const int32_t i0 = (tile / a.tiles_c) * kBwT, c0 = (tile % a.tiles_c) * kBwT;
    f4_t acc[4][2];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int nj = 0; nj < 2; ++nj) acc[mi][nj] = f4_t{0.f, 0.f, 0.f, 0.f};
    uint4 vd, vx;
    load(0, i0, c0, vd, vx);
    // The tile's codes (16 groups x M bytes per row) and scales, for the
    // scatter: loaded now, stored into LDS after the contraction, so their
    // latency hides under it.  Rows whose 16M-byte window is whole and
    // 16-byte aligned take one 16-byte load per thread (M <= 4).
    const int32_t j0 = c0 / 8;
    const bool vec_codes = M <= 4 && (G * M) % 16 == 0 && j0 + 16 <= G;
    constexpr int kCodeU4 = kBwT * M;  // 16-byte chunks of the tile's codes (M <= 4)
    uint4 cv = make_uint4(0, 0, 0, 0);
    float scv = 0.f;
    if (vec_codes && tid < kCodeU4) {
      const int row = tid / M, q = tid % M;
      const int32_t i = i0 + row < a.d_out ? i0 + row : a.d_out - 1;
      cv = *reinterpret_cast<const uint4*>(a.codes + ((size_t)i * G + j0) * M + 16 * q);
    }
    if (tid < kBwT && i0 + tid < a.d_out) scv = h2f(a.scales[i0 + tid]);
    lds_barrier();  // (the previous tile's last reads of stage 0 and of the tile's codes are done)
    store(0, vd, vx);
    lds_barrier();
    for (int step = 0; step < nsteps; ++step) {
      const bool more = step + 1 < nsteps;
      if (more) load(step + 1, i0, c0, vd, vx);
      const uint16_t* s = stg + (step & 1) * kBwStage;
      h8_t af[4], bf[2];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        af[mi] = *reinterpret_cast<const h8_t*>(s + (64 * wm + 16 * mi + r16) * kBwP + 8 * slot);
#pragma unroll
      for (int nj = 0; nj < 2; ++nj)
        bf[nj] = *reinterpret_cast<const h8_t*>(s + (kBwT + 32 * wn + 16 * nj + r16) * kBwP + 8 * slot);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int nj = 0; nj < 2; ++nj)
          acc[mi][nj] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[mi], bf[nj], acc[mi][nj], 0, 0, 0);
      if (more) store((step + 1) & 1, vd, vx);
      lds_barrier();
    }
    if (vec_codes) {
      if (tid < kCodeU4) reinterpret_cast<uint4*>(tcodes)[tid] = cv;
    } else {
      const int gw = (G - j0 < 16 ? G - j0 : 16) * M;  // code bytes of a row inside the tile
#pragma unroll 1
      for (int e = tid; e < kBwT * 16 * M; e += kBwThreads) {
        const int row = e / (16 * M), b = e % (16 * M);
        const int32_t i = i0 + row;
        tcodes[e] = (i < a.d_out && b < gw) ? a.codes[((size_t)i * G + j0) * M + b] : (uint8_t)0;
      }
    }
    if (tid < kBwT) tscales[tid] = scv;
    lds_barrier();

    // Scatter: lane holds G[i][c] for i = i0 + 64 wm + 16 mi + 4 slot + r and
    // c = c0 + 32 wn + 16 nj + r16.
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int il = 64 * wm + 16 * mi + 4 * slot + r;  // row within the tile
        const int32_t i = i0 + il;
        float dsum = 0.f;
        if (i < a.d_out) {
          const float si = tscales[il];
#pragma unroll
          for (int nj = 0; nj < 2; ++nj) {
            const int cl = 32 * wn + 16 * nj + r16;  // input within the tile
            if (c0 + cl < a.d_in) {
              const float gv = acc[mi][nj][r];
              const int k = cl & 7;
              const uint8_t* cp = tcodes + (il * 16 + (cl >> 3)) * M;
              float u = 0.f;
#pragma unroll
              for (int m = 0; m < M; ++m) {
                const int idx = (m * 256 + cp[m]) * 8 + k;
                const float v = h2f(cbl[idx]);
                u = (m == 0) ? v : u + v;
                atomicAdd(&dcl[idx], si * gv);
              }
              dsum += gv * u;
            }
          }
        }
        // the 16 lanes of a DPP row share the row i
        dsum += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, dsum), 0xB1, 0xF, 0xF, true));
        dsum += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, dsum), 0x4E, 0xF, 0xF, true));
        dsum += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, dsum), 0x141, 0xF, 0xF, true));
        dsum += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, dsum), 0x140, 0xF, 0xF, true));
        if (r16 == 0 && i < a.d_out) atomicAdd(&a.ds[i], dsum);
        // one row at a time: hoisting the next rows' lookups would only
        // take registers
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  lds_barrier();
  for (int e = tid; e < M * 2048; e += kBwThreads) {
    const float v = dcl[e];
    if (v != 0.f) atomicAdd(&a.dcb[e], v);
  }
}

template <int M>
hipError_t run_grad(const BwArgs& a, hipStream_t s) {
  constexpr size_t lds = bw_lds_bytes<M>();
  static_assert(lds <= 160 * 1024, "backward LDS budget");
  auto kern = k_grad_cb<M>;
  const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), (int)lds);
  if (e != hipSuccess) return e;
  // persistent workgroups: as many as can be resident at once (registers
  // and LDS), so that none waits for another to finish all of its tiles
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kBwThreads, lds) != hipSuccess || per_cu < 1)
    per_cu = 1;
  int grid = num_cus() * per_cu;
  if (grid > a.tiles) grid = a.tiles;
  hipLaunchKernelGGL(kern, dim3(grid), dim3(kBwThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace

bool backward_supported(const Layer& L) { return L.B == 8 && L.M >= 1 && L.M <= 8 && L.d_out % 8 == 0; }

hipError_t launch_backward(const Layer& L, int32_t n, const uint16_t* x, const uint16_t* dy, float* dcb, float* ds,
                           hipStream_t s) {
  if (!backward_supported(L) || n < 1) return hipErrorInvalidValue;
  BwArgs a{static_cast<const uint8_t*>(L.codes), L.codebooks, L.scales, x, dy, dcb, ds, L.d_out, L.d_in, n,
           (L.d_in + kBwT - 1) / kBwT, 0};
  const int64_t tiles = (int64_t)((L.d_out + kBwT - 1) / kBwT) * a.tiles_c;
  if (tiles >= (int64_t(1) << 31)) return hipErrorInvalidValue;
  a.tiles = (int32_t)tiles;
  switch (L.M) {
    case 1: return run_grad<1>(a, s);
    case 2: return run_grad<2>(a, s);
    case 3: return run_grad<3>(a, s);
    case 4: return run_grad<4>(a, s);
    case 5: return run_grad<5>(a, s);
    case 6: return run_grad<6>(a, s);
    case 7: return run_grad<7>(a, s);
    case 8: return run_grad<8>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
