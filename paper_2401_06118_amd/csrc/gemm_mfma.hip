// AQLM product with several activation rows on the matrix cores:
//   Y[t][i] = fp16(s_i * sum_c W[i][c] X[t][c]),  W from Eq. 2.
//
// The contraction runs on v_mfma_f32_16x16x32_f16.  Its A operand gives each
// lane 8 consecutive K values of one row (lane = row + 16 * K-slot), which is
// exactly one codeword, so a lane builds its A fragment with a single codeword
// lookup and no fp16 rounding of W.  The K axis of one MFMA step is the
// 4 K-slots x 8 values of four codes of the same row; because every code of
// a row contributes <codeword, x-slice of its group>, the codes can be dealt
// to the K-slots in any order as long as the B operand (lane = token + 16 *
// K-slot) carries the x-slice of the group each A lane's code belongs to.
// Lane (r, s) therefore takes 8 consecutive codes of row r per K-tile of 32
// codes, loaded with one 8- or 16-byte load, and the B lanes of slot s read
// the matching x-slices from an LDS tile.  Each A fragment is reused for NB
// blocks of 16 tokens and each B fragment for RB blocks of 16 rows.
//
// Codeword lookups use the same LDS codebook copies as the matrix-vector
// kernel (B = 8), one LDS copy of two 12-bit codebooks (2x12, 128 KiB), or
// 16-byte L2 gathers (other wide codes).  Supported: B = 8 with
// M in {1, 2, 4, 8} (M divides the 32 codes of a K-tile) and the wide-code
// formats with M in {1, 2}.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

namespace {

constexpr int kThreads = 256;
constexpr int kCPL = 8;          // codes per lane per K-tile
constexpr int kQT = 4 * kCPL;    // codes per row per K-tile

template <int M, int B>
struct MfmaCfg {
  static constexpr int kBytesPerCode = code_bytes(B);
  static constexpr int kGT = kQT / M;  // groups (x-slices) per K-tile
  static constexpr int kCopies = (B > 8) ? 0 : (M <= 2 ? 16 : (M <= 4 ? 8 : 4));
  // two 12-bit codebooks (128 KiB) sit whole in LDS, one copy
  static constexpr bool kWideLds = (M == 2 && B == 12);
  static constexpr int kLaneBytes = kCPL * kBytesPerCode;  // 8 or 16
  static constexpr int kWords = kLaneBytes / 4;
};

// Codes k0..k0+7 (code index within the row) of row `row`: zero past the row.
template <int M, int B, bool VEC>
__device__ __forceinline__ void load_codes8(const uint8_t* __restrict__ codes, int32_t row, int32_t d_out,
                                            int64_t codes_per_row, int64_t k0,
                                            uint32_t (&w)[MfmaCfg<M, B>::kWords]) {
  using C = MfmaCfg<M, B>;
#pragma unroll
  for (int i = 0; i < C::kWords; ++i) w[i] = 0;
  if (row >= d_out) return;
  const size_t off = ((size_t)row * codes_per_row + k0) * C::kBytesPerCode;
  if (VEC && k0 + kCPL <= codes_per_row) {
    if constexpr (C::kLaneBytes == 16) {
      const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(codes + off));
      w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
    } else {
      const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(codes + off));
      w[0] = v[0]; w[1] = v[1];
    }
    return;
  }
  int64_t valid = codes_per_row - k0;
  if (valid > kCPL) valid = kCPL;
  const int nbytes = valid > 0 ? (int)valid * C::kBytesPerCode : 0;
#pragma unroll
  for (int b = 0; b < C::kLaneBytes; ++b)
    if (b < nbytes) w[b / 4] |= (uint32_t)codes[off + b] << (8 * (b % 4));
}

template <int B>
__device__ __forceinline__ uint32_t code_k(const uint32_t* w, int k) {
  if constexpr (B > 8) return (w[k / 2] >> (16 * (k % 2))) & code_mask(B);
  return (w[k / 4] >> (8 * (k % 4))) & 0xFFu;
}

// RB: 16-row blocks per wave; NB: 16-token blocks per workgroup; KSPLIT:
// waves that share one row group and split its K-tiles (their partial sums
// are added in a fixed order at the end).
template <int M, int B, bool VEC, int RB, int NB, int KSPLIT>
__global__ __launch_bounds__(kThreads) void k_gemm_mfma(const uint8_t* __restrict__ codes,
                                                         const uint4* __restrict__ cb,
                                                         const uint16_t* __restrict__ scales,
                                                         const uint4* __restrict__ x, uint16_t* __restrict__ y,
                                                         int32_t d_out, int32_t G, int32_t n) {
  using C = MfmaCfg<M, B>;
  constexpr int kWaves = kThreads / kWave;
  constexpr int kRowGroups = kWaves / KSPLIT;
  constexpr int kRowsPerWg = kRowGroups * RB * 16;
  constexpr int kTok = NB * 16;
  constexpr int kPitch = C::kGT + 1;  // uint4 per token row of an x tile (+1 against bank conflicts)
  constexpr int kXTile = kTok * kPitch;
  constexpr int kLdsCb = (B == 8) ? M * 256 * C::kCopies : (C::kWideLds ? (M << B) : 1);
  constexpr int kXLds = KSPLIT * kXTile;
  constexpr int kRedLds = (KSPLIT > 1) ? (KSPLIT - 1) * kRowGroups * RB * NB * kWave : 0;  // f4_t entries
  __shared__ uint4 cb_lds[kLdsCb];
  __shared__ uint4 x_lds[kXLds > kRedLds ? kXLds : kRedLds];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int rgrp = wave / KSPLIT;
  const int kl = wave % KSPLIT;
  const int r16 = lane & 15;
  const int slot = lane >> 4;
  const int32_t row_base = blockIdx.x * kRowsPerWg + rgrp * RB * 16;
  const int32_t tok0 = blockIdx.y * kTok;
  const int64_t codes_per_row = (int64_t)G * M;
  const int32_t n_kt = (int32_t)((codes_per_row + kQT - 1) / kQT);
  const int32_t iters = (n_kt + KSPLIT - 1) / KSPLIT;

  uint32_t cw[RB][C::kWords];
  {
    const int kt = kl;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      load_codes8<M, B, VEC>(codes, row_base + rb * 16 + r16, d_out, codes_per_row, (int64_t)kt * kQT + slot * kCPL,
                             cw[rb]);
  }

  if constexpr (B == 8) {
    constexpr int E = M * 256;
    for (int e = tid; e < E; e += kThreads) {
      const uint4 v = cb[e];
#pragma unroll
      for (int k = 0; k < C::kCopies; ++k) cb_lds[e * C::kCopies + ((k + lane) % C::kCopies)] = v;
    }
  }
  if constexpr (C::kWideLds) {
    // (read before the first x tile's barrier, like the 8-bit copies)
    for (int e = tid; e < kLdsCb; e += kThreads) cb_lds[e] = cb[e];
  }
  const uint32_t copy_off = (B == 8) ? (uint32_t)(lane % (C::kCopies ? C::kCopies : 1)) * 16u : 0u;

  f4_t acc[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[rb][nb] = f4_t{0.f, 0.f, 0.f, 0.f};

  for (int32_t it = 0; it < iters; ++it) {
    lds_barrier();  // previous x tiles fully read
    // Stage the x tiles of K-tiles it*KSPLIT .. it*KSPLIT+KSPLIT-1.
    for (int e = tid; e < KSPLIT * kTok * C::kGT; e += kThreads) {
      const int ks = e / (kTok * C::kGT);
      const int rem = e % (kTok * C::kGT);
      const int t = rem / C::kGT;
      const int jl = rem % C::kGT;
      const int64_t grp = (int64_t)(it * KSPLIT + ks) * C::kGT + jl;
      const int32_t tok = tok0 + t;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (tok < n && grp < G) v = x[(int64_t)tok * G + grp];
      x_lds[ks * kXTile + t * kPitch + jl] = v;
    }
    lds_barrier();

    const int32_t kt = it * KSPLIT + kl;
    uint32_t cur[RB][C::kWords];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < C::kWords; ++i) cur[rb][i] = cw[rb][i];
    if (it + 1 < iters) {
      const int64_t k0 = (int64_t)(kt + KSPLIT) * kQT + slot * kCPL;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        load_codes8<M, B, VEC>(codes, row_base + rb * 16 + r16, d_out, codes_per_row, k0, cw[rb]);
    }
    if (kt >= n_kt) continue;

    const uint4* xt = x_lds + kl * kXTile;
    h8_t bf[NB];
#pragma unroll
    for (int t = 0; t < kCPL; ++t) {
      const int q = slot * kCPL + t;  // code index within the K-tile
      const int m = q % M;
      if (m == 0 || t == 0) {
        const int jl = q / M;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) bf[nb] = __builtin_bit_cast(h8_t, xt[(nb * 16 + r16) * kPitch + jl]);
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const uint32_t code = code_k<B>(cur[rb], t);
        uint4 v;
        if constexpr (B == 8) {
          const uint32_t addr = ((uint32_t)(m * 256) + code) * (uint32_t)(C::kCopies * 16) + copy_off;
          v = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(cb_lds) + addr);
        } else if constexpr (C::kWideLds) {
          v = cb_lds[((uint32_t)m << B) + code];
        } else {
          v = cb[((uint32_t)m << B) + code];
        }
        const h8_t af = __builtin_bit_cast(h8_t, v);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[rb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af, bf[nb], acc[rb][nb], 0, 0, 0);
      }
    }
  }

  if constexpr (KSPLIT > 1) {
    // Waves kl = 1..KSPLIT-1 hand their partial sums to wave kl = 0 of the
    // same row group, which adds them in ascending kl.
    lds_barrier();
    f4_t* red = reinterpret_cast<f4_t*>(x_lds);
    if (kl > 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          red[(((kl - 1) * kRowGroups + rgrp) * RB * NB + rb * NB + nb) * kWave + lane] = acc[rb][nb];
    }
    lds_barrier();
    if (kl != 0) return;
#pragma unroll
    for (int k = 1; k < KSPLIT; ++k)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[rb][nb] += red[(((k - 1) * kRowGroups + rgrp) * RB * NB + rb * NB + nb) * kWave + lane];
  }

  // D layout of the 16x16 MFMA: lane holds column (lane % 16) and rows
  // 4 * (lane / 16) + i, i = 0..3.
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t row = row_base + rb * 16 + 4 * slot + i;
      if (row >= d_out) continue;
      const float s = h2f(scales[row]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int32_t tok = tok0 + nb * 16 + r16;
        if (tok < n) y[(int64_t)tok * d_out + row] = f2h(s * acc[rb][nb][i]);
      }
    }
  }
}

template <int M, int B, bool VEC, int RB, int NB, int KSPLIT>
hipError_t run(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  constexpr int kRowsPerWg = (kThreads / kWave / KSPLIT) * RB * 16;
  const dim3 grid((L.d_out + kRowsPerWg - 1) / kRowsPerWg, (n + NB * 16 - 1) / (NB * 16));
  hipLaunchKernelGGL((k_gemm_mfma<M, B, VEC, RB, NB, KSPLIT>), grid, dim3(kThreads), 0, s,
                     static_cast<const uint8_t*>(L.codes), reinterpret_cast<const uint4*>(L.codebooks), L.scales,
                     reinterpret_cast<const uint4*>(x), y, L.d_out, L.G, n);
  return hipGetLastError();
}

template <int M, int B, bool VEC>
hipError_t run_shape(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  // Up to 16 tokens: one token block, 16-row workgroups whose four waves split
  // K (many workgroups, like the matrix-vector kernel).  More tokens: 128-row
  // by 64-token tiles, each codeword fragment reused for 4 token blocks.
  // 2x12 stages 128 KiB of codebooks per workgroup: 48-row workgroups
  // amortise it and still cover most CUs (11008x4096, n = 4 / 16: 32.0 /
  // 32.4 us, against 34.2 / 35.0 with 64 rows, 36.7 / 37.6 with 80, 59.7 at
  // n = 16 with 16 rows and 45.8 gathering from L2).
  if (n <= 16 && MfmaCfg<M, B>::kWideLds) return run<M, B, VEC, 3, 1, 4>(L, n, x, y, s);
  if (n <= 16) return run<M, B, VEC, 1, 1, 4>(L, n, x, y, s);
  return run<M, B, VEC, 2, 4, 1>(L, n, x, y, s);
}

template <int M, int B>
hipError_t run_vec(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (L.vec_codes) return run_shape<M, B, true>(L, n, x, y, s);
  return run_shape<M, B, false>(L, n, x, y, s);
}

}  // namespace

bool mfma_supported(const Layer& L) {
  if (L.B > 8) return L.M == 1 || L.M == 2;
  return L.M == 1 || L.M == 2 || L.M == 4 || L.M == 8;
}

hipError_t launch_gemm_mfma(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (L.B > 8) {
    if (L.M == 1) return L.B == 16 ? run_vec<1, 16>(L, n, x, y, s) : run_vec<1, 15>(L, n, x, y, s);
    switch (L.B) {
      case 12: return run_vec<2, 12>(L, n, x, y, s);
      case 15: return run_vec<2, 15>(L, n, x, y, s);
      case 16: return run_vec<2, 16>(L, n, x, y, s);
    }
    return hipErrorInvalidValue;
  }
  switch (L.M) {
    case 1: return run_vec<1, 8>(L, n, x, y, s);
    case 2: return run_vec<2, 8>(L, n, x, y, s);
    case 4: return run_vec<4, 8>(L, n, x, y, s);
    case 8: return run_vec<8, 8>(L, n, x, y, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
