// Small-batch AQLM product for M = 2 or 4 8-bit codebooks, 2 <= n <= 16
// activation rows:
//   Y[t][i] = fp16(s_i * sum_j sum_m <C_m[b_ijm], X[t, 8j:8j+8]>)   (Eq. 2)
//
// The same matrix-core scheme as the batch-1 kernel (k_gemv_ks): lane (r, s)
// of a wave gathers the codewords of row r for its 16 codes of a 64-code
// K-slice (one A fragment each), and column c of the B operand carries the
// x-slice of token c, so one v_mfma_f32_16x16x32_f16 now does useful work in
// n of its 16 columns instead of one.  The code stream, and hence the time,
// stays that of a single product while n grows to 16.
//
// Work split.  One workgroup of 16 waves per CU owns a range of rows; wave w
// takes K-slices w, w + 16, ... (one per round) of all of its row blocks and
// keeps one accumulator per 16-row block.  x of all n tokens would not fit in
// LDS next to the codebook copies, so it is staged one round (16 K-slices) at
// a time; the next round's x is loaded into registers while the current one
// is consumed.  Code loads run kInFlightNB items ahead of their use, across
// rounds.  At the end the 16 waves' partial tiles are added in a fixed order
// per row block, so results are deterministic.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"
#include "stream_common.h"

namespace aqlm {

namespace {

constexpr int kWavesNB = 16;
constexpr int kThreadsNB = kWavesNB * kWave;
constexpr int kMaxTokNB = 16;  // tokens per launch (the 16 MFMA columns)
// code items requested ahead of their use per wave (at least both items of a
// pair of row blocks); 11008x4096 4x8 at 2 / 4 / 8 / 16 tokens: 12.7 / 14.1
// / 15.9 / 18.2 us with 2, 13.4 / 14.8 / 16.4 / 18.7 with 3, slower with 4
// or 6; 2x8 and other shapes the same with 2 or 3
constexpr int kInFlightNB = 2;
constexpr size_t kLdsLimit = 160 * 1024;

struct GemmNbArgs {
  const uint8_t* codes;
  const uint4* cb;
  const uint16_t* scales;
  const uint4* x;  // [n][G] groups of 8 fp16
  uint16_t* y;     // [n][d_out]
  int32_t d_out;
  int32_t G;
  int32_t n;
  int32_t rows_per_wg;
  int32_t tiled;  // codes in 1 KiB tiles (tiled_codes_offset), not row-major
};

template <int M>
struct NbCfg {
  using C = GCfg<8>;
  static constexpr int kXS = C::kCPL / M;          // x groups per lane per K-slice
  static constexpr int kGS = C::kKS / M;           // groups per K-slice
  static constexpr int kXG = kWavesNB * kGS;       // groups per round
  static constexpr int kXV = kMaxTokNB * kXG / kThreadsNB;  // x staging loads per thread
  static constexpr size_t kPartBytes = (size_t)kWavesNB * 16 * 16 * 4;
};

template <int M, int COPIES, int RB, int D, bool VEC>
__global__ __launch_bounds__(kThreadsNB) void k_gemm_nb(const GemmNbArgs a) {
  using C = GCfg<8>;
  using N = NbCfg<M>;
  constexpr int kXS = N::kXS;
  constexpr int kXG = N::kXG;
  constexpr int kStep = RB >= 5 ? 2 : 4;
  constexpr int kSlots = D * RB;
  // both items of a row-block pair must be in flight when the pair starts
  constexpr int kAheadMin = RB >= 2 ? 2 : 1;
  constexpr int kAheadWant = kInFlightNB > kAheadMin ? kInFlightNB : kAheadMin;
  constexpr int kAhead = kAheadWant < kSlots ? kAheadWant : kSlots;
  static_assert(kAhead >= kAheadMin, "a pair of row blocks needs both items loaded");
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15;
  const int slot = lane >> 4;
  const int n = a.n;

  const int32_t row0 = (int32_t)blockIdx.x * a.rows_per_wg;
  int32_t rows = a.d_out - row0;
  if (rows > a.rows_per_wg) rows = a.rows_per_wg;
  const int32_t G = a.G;
  const uint32_t pitch = (uint32_t)G * M;        // code bytes per row
  const int KS = (int)((pitch + 63u) / 64u);     // 64-byte K-slices per row
  const int R = (KS + kWavesNB - 1) / kWavesNB;  // rounds (the same for every wave)
  const int nks = KS > wave ? (KS - wave + kWavesNB - 1) / kWavesNB : 0;  // rounds with a K-slice for this wave
  // Row-major codes: an item is 16 rows x 64 bytes at the row pitch; tiled
  // codes: the same item is one contiguous 1 KiB tile.
  const bool tiled = a.tiled != 0;
  const uint8_t* __restrict__ wg_codes = tiled ? a.codes : a.codes + (size_t)row0 * pitch;
  const uint32_t k_stride = tiled ? 1024u : 64u;         // bytes from one K-slice to the next
  const uint32_t k_limit = tiled ? 0xFFFFFFFFu : pitch;  // (tiles hold whole K-slices)

  uint4* cb_lds = lds;
  uint4* x_lds = lds + M * 256 * COPIES;                        // [n][kXG]
  float* part = reinterpret_cast<float*>(x_lds + n * kXG);      // [wave][16 rows][16 tokens]

  // 1. small loads first: codebooks, the scales of this thread's epilogue
  // rows (clamped, unconditional), x of round 0.
  uint4 cbv = make_uint4(0, 0, 0, 0);
  if (tid < M * 256) cbv = a.cb[tid];
  uint16_t sc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    int r = rb * 16 + (tid & 15);
    r = r < rows ? r : rows - 1;
    sc[rb] = a.scales[row0 + r];
  }
  uint4 xv[N::kXV];
  auto load_x = [&](int round) {
#pragma unroll
    for (int i = 0; i < N::kXV; ++i) {
      const int e = tid + i * kThreadsNB;
      const int t = e / kXG, g = round * kXG + e % kXG;
      xv[i] = make_uint4(0, 0, 0, 0);
      if (t < n && g < G) xv[i] = a.x[(size_t)t * G + g];
    }
  };
  load_x(0);

  // 2. code loads for the first kAhead items (item j * RB + rb is row block rb
  // of this wave's K-slice of round j; rows past the end repeat the last row).
  const uint32_t slot_off = (uint32_t)slot * 16u;
  int row_off[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    int row = rb * 16 + r16;
    row = row < rows ? row : rows - 1;
    const int grow = row0 + row;
    row_off[rb] = tiled ? (grow >> 4) * KS * 1024 + (grow & 15) * 64 : row * (int)pitch;
  }
  auto issue_rb = [&](int j, int rb, uint32_t (&w)[4]) {
    const uint32_t ks_off = (uint32_t)(wave + j * kWavesNB) * 64u + slot_off;  // in a row-major row
    const uint32_t off = (uint32_t)(wave + j * kWavesNB) * k_stride + slot_off;
    if constexpr (VEC) {
      const uint32_t o = (uint32_t)row_off[rb] + (ks_off < k_limit ? off : 0u);
      const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(wg_codes + o));
      w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
    } else {
      load_codes_bytes<8>(wg_codes + row_off[rb], pitch, off, w);
    }
  };
  uint32_t ring[D][RB][4];
#pragma unroll
  for (int i = 0; i < kAhead; ++i)
    if (i / RB < nks) issue_rb(i / RB, i % RB, ring[i / RB][i % RB]);

  // 3. codebook copies (lane l reads copy l % COPIES).
  if (tid < M * 256) {
#pragma unroll
    for (int k = 0; k < COPIES; ++k) cb_lds[tid * COPIES + ((k + lane) % COPIES)] = cbv;
  }

  const uint32_t copy_off = (uint32_t)(lane % COPIES) * 16u;
  const uint32_t cb_base = (uint32_t)(uintptr_t)cb_lds;
  uint32_t base_m[M];
#pragma unroll
  for (int m = 0; m < M; ++m) base_m[m] = cb_base + ((uint32_t)m << 16) + copy_off;
  f4_t acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = f4_t{0.f, 0.f, 0.f, 0.f};
  f4_t acc_odd = {0.f, 0.f, 0.f, 0.f};
  uint4 xr[kXS];

  // 4. rounds.  Every wave runs every round (the barriers need it); waves
  // without a K-slice in the last round only stage x.
  for (int j0 = 0; j0 < R; j0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int j = j0 + d;
      if (j < R) {
        if (j > 0) lds_barrier();  // round j - 1's x fully read
#pragma unroll
        for (int i = 0; i < N::kXV; ++i) {
          const int e = tid + i * kThreadsNB;
          if (e < n * kXG) x_lds[e] = xv[i];
        }
        if (j + 1 < R) load_x(j + 1);
        lds_barrier();
      }
      const bool live = j < nks;
      if (live) {
        const uint4* xs = x_lds + (r16 < n ? r16 : 0) * kXG + wave * N::kGS + slot * kXS;
#pragma unroll
        for (int s2 = 0; s2 < kXS; ++s2) xr[s2] = r16 < n ? xs[s2] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int rb = 0; rb < RB; rb += 2) {
        const bool pair = rb + 1 < RB;
        if (live) {
#pragma unroll
          for (int t0 = 0; t0 < C::kCPL; t0 += kStep) {
            uint4 av[kStep], bv[kStep];
#pragma unroll
            for (int u = 0; u < kStep; ++u) {
              const int t = t0 + u;
              av[u] = lds_load16(
                  cw_addr<M, COPIES>(ring[d][rb][t / 4], t % 4, base_m[t % M], copy_off + cb_base, t % M));
              if (pair)
                bv[u] = lds_load16(cw_addr<M, COPIES>(ring[d][pair ? rb + 1 : rb][t / 4], t % 4, base_m[t % M],
                                                      copy_off + cb_base, t % M));
            }
#pragma unroll
            for (int u = 0; u < kStep; ++u) {
              const int t = t0 + u;
              const h8_t xh = __builtin_bit_cast(h8_t, xr[t / M]);
              if (pair) {
                acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[u]), xh, acc[rb], 0, 0, 0);
                acc[pair ? rb + 1 : rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                    __builtin_bit_cast(h8_t, bv[u]), xh, acc[pair ? rb + 1 : rb], 0, 0, 0);
              } else {
                f4_t& acc_u = (u % 2 == 0) ? acc[rb] : acc_odd;
                acc_u = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[u]), xh, acc_u, 0, 0, 0);
              }
            }
          }
        }
#pragma unroll
        for (int q = 0; q < (pair ? 2 : 1); ++q) {
          const int target = d * RB + rb + q + kAhead;  // item position relative to round j0
          const int jt = j0 + target / RB;
          if (jt < nks) issue_rb(jt, target % RB, ring[(target % kSlots) / RB][target % RB]);
        }
      }
    }
  }
  if constexpr (RB % 2 == 1) acc[RB - 1] += acc_odd;

  // 5. per row block: every wave stores its 16x16 tile (lane: token r16, rows
  // 4 * slot + i), then (row, token) threads add the 16 waves in order.
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    lds_barrier();  // previous block's sums read (and the last round's x)
#pragma unroll
    for (int i = 0; i < 4; ++i) part[(wave * 16 + 4 * slot + i) * 16 + r16] = acc[rb][i];
    lds_barrier();
    if (tid < 16 * n) {
      const int rr = tid & 15, t = tid >> 4;
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kWavesNB; ++w) s += part[(w * 16 + rr) * 16 + t];
      const int32_t r = rb * 16 + rr;
      if (r < rows) a.y[(size_t)t * a.d_out + row0 + r] = f2h(h2f(sc[rb]) * s);
    }
  }
}

template <int M, int COPIES, int RB, int D, bool VEC>
hipError_t launch_nb(const GemmNbArgs& a, int nwg, size_t lds_bytes, hipStream_t s) {
  auto kern = k_gemm_nb<M, COPIES, RB, D, VEC>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), (int)kLdsLimit);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3(nwg), dim3(kThreadsNB), lds_bytes, s, a);
  return hipGetLastError();
}

// Code-load ring in rounds (as in the batch-1 kernel): about four items, one
// round for M = 2 and two row blocks (its x staging registers leave no room).
template <int M, int COPIES, int RB, bool VEC>
hipError_t launch_nb_d(const GemmNbArgs& a, int nwg, int rounds, size_t lds, hipStream_t s) {
  constexpr int D4 = RB >= 4 ? 1 : (RB == 1 ? 4 : (M == 2 ? 1 : 2));
  if (D4 >= 4 && rounds >= 4) return launch_nb<M, COPIES, RB, (D4 >= 4 ? 4 : 1), VEC>(a, nwg, lds, s);
  if (D4 >= 2 && rounds >= 2) return launch_nb<M, COPIES, RB, (D4 >= 2 ? 2 : 1), VEC>(a, nwg, lds, s);
  return launch_nb<M, COPIES, RB, 1, VEC>(a, nwg, lds, s);
}

// Row blocks per workgroup that fit in registers without spilling.
constexpr int nb_rb_cap(int M) { return M == 2 ? 2 : 4; }

template <int M, int COPIES, bool VEC>
hipError_t launch_nb_rb(const GemmNbArgs& a, int nwg, int rb, int rounds, size_t lds, hipStream_t s) {
  switch (rb) {
    case 1: return launch_nb_d<M, COPIES, 1, VEC>(a, nwg, rounds, lds, s);
    case 2: return launch_nb_d<M, COPIES, 2, VEC>(a, nwg, rounds, lds, s);
  }
  if constexpr (nb_rb_cap(M) >= 4) {
    switch (rb) {
      case 3: return launch_nb_d<M, COPIES, 3, VEC>(a, nwg, rounds, lds, s);
      case 4: return launch_nb_d<M, COPIES, 4, VEC>(a, nwg, rounds, lds, s);
    }
  }
  return hipErrorInvalidValue;
}

template <int M, bool VEC>
hipError_t launch_nb_copies(const GemmNbArgs& a, int nwg, int rb, int rounds, int copies, size_t lds,
                            hipStream_t s) {
  switch (copies) {
    case 16: return launch_nb_rb<M, 16, VEC>(a, nwg, rb, rounds, lds, s);
    case 8: return launch_nb_rb<M, 8, VEC>(a, nwg, rb, rounds, lds, s);
    case 4: return launch_nb_rb<M, 4, VEC>(a, nwg, rb, rounds, lds, s);
    case 2: return launch_nb_rb<M, 2, VEC>(a, nwg, rb, rounds, lds, s);
    case 1: return launch_nb_rb<M, 1, VEC>(a, nwg, rb, rounds, lds, s);
  }
  return hipErrorInvalidValue;
}

template <int M>
size_t nb_fixed_lds(int n) {
  return (size_t)n * NbCfg<M>::kXG * 16 + NbCfg<M>::kPartBytes;
}

size_t nb_fixed_lds_m(int M, int n) {
  switch (M) {
    case 2: return nb_fixed_lds<2>(n);
    case 4: return nb_fixed_lds<4>(n);
  }
  return kLdsLimit + 1;
}

}  // namespace

bool gemm_nb_supported(const Layer& L, int32_t n) {
  if (L.B != 8 || !(L.M == 2 || L.M == 4) || n < 2 || n > kMaxTokNB) return false;
  // at least one codebook copy must fit next to a round of x and the partial tiles
  return nb_fixed_lds_m(L.M, n) + (size_t)L.M * 256 * 16 <= kLdsLimit;
}

hipError_t launch_gemm_nb(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (!gemm_nb_supported(L, n) || (L.tiled && !L.vec_codes)) return hipErrorInvalidValue;
  const int M = L.M;
  const int cus = num_cus();
  // One workgroup per CU when the rows allow it; at most nb_rb_cap(M) row
  // blocks per workgroup (registers), more workgroups if needed.
  const int rb_cap = nb_rb_cap(M);
  const int blocks = (L.d_out + 15) / 16;
  const int waves_of_wgs = (blocks + rb_cap * cus - 1) / (rb_cap * cus);
  const int rows_per_wg = (L.d_out + cus * waves_of_wgs - 1) / (cus * waves_of_wgs);
  const int nwg = (L.d_out + rows_per_wg - 1) / rows_per_wg;
  const int rb = (rows_per_wg + 15) / 16;
  const int KS = (int)(((int64_t)L.G * M + 63) / 64);
  const int rounds = (KS + kWavesNB - 1) / kWavesNB;
  const size_t fixed = nb_fixed_lds_m(M, n);
  const size_t per_copy = (size_t)M * 256 * 16;
  int copies = 16;
  while (copies > 1 && fixed + per_copy * copies > kLdsLimit) copies /= 2;
  const size_t lds = fixed + per_copy * copies;
  GemmNbArgs a{static_cast<const uint8_t*>(L.codes), reinterpret_cast<const uint4*>(L.codebooks), L.scales,
               reinterpret_cast<const uint4*>(x), y, L.d_out, L.G, n, rows_per_wg, L.tiled ? 1 : 0};
  const bool vec = L.vec_codes;
  switch (M) {
    case 2: return vec ? launch_nb_copies<2, true>(a, nwg, rb, rounds, copies, lds, s)
                       : launch_nb_copies<2, false>(a, nwg, rb, rounds, copies, lds, s);
    case 4: return vec ? launch_nb_copies<4, true>(a, nwg, rb, rounds, copies, lds, s)
                       : launch_nb_copies<4, false>(a, nwg, rb, rounds, copies, lds, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
