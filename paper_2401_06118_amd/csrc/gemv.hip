// Batch-1 AQLM matrix-vector product (the token-generation product the paper
// benchmarks in Sec. 4.3):  y_i = fp16(s_i * sum_j sum_m <C_m[b_ijm], x_j>).
//
// Work split.  A chunk is 64 lanes x GPL consecutive groups of one row.  A
// wave walks a list of (chunk, row) items, keeping the x values of its chunk
// in registers (GPL x 16 bytes per lane) while it streams the rows' codes
// (one 8- or 16-byte load per lane per item).  Each lane looks up its
// codewords, takes fp16 dot products with x into fp32 (v_dot2_f32_f16), the
// wave sums the lanes (DPP), and the per-(row, chunk) partials are added in a
// fixed order at the end, so results are deterministic.
//
// Codewords.  B = 8: the M codebooks (4 KiB each) are copied COPIES times
// into LDS with copy c of codeword e at ((m*256 + e)*COPIES + c)*16 bytes and
// lane l reads copy l % COPIES.  A ds_read_b128 serves 16 lanes per clock
// from 64 banks; with 16 copies every lane of a 16-lane group hits its own
// 16-byte bank quad, so random codeword lookups run conflict-free at the
// full LDS rate (fewer copies for M > 2, where 16 would not fit).  Wider
// codes: the codebooks (2^B codewords each, up to 1 MiB) stay in L2 and each
// lane gathers its codewords with 16-byte global loads.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

constexpr int kMaxPartials = 2048;

template <int M, int B>
struct GemvCfg {
  static constexpr int kBytesPerCode = code_bytes(B);
  static constexpr int GPL = (M * kBytesPerCode <= 2) ? 8 : (M * kBytesPerCode <= 4 ? 4 : 2);
  static constexpr int kCodeBytes = GPL * M * kBytesPerCode;  // per lane per item
  static constexpr int kWords = (kCodeBytes + 3) / 4;
  static constexpr int kCopies = (B > 8) ? 0 : (M <= 2 ? 16 : (M <= 4 ? 8 : 4));
  static constexpr int kChunkGroups = 64 * GPL;
  static constexpr bool kCanVec = (kCodeBytes == 16 || kCodeBytes == 8);
};

// Codes of one lane's GPL groups of row `row` into 32-bit words.
// VEC: the row pitch is a multiple of 16 bytes, so a lane's chunk is either
// whole or entirely past the row end; the load is always issued (from the
// row start when the chunk is past the end; the caller masks those lanes) so
// that the compiler can count outstanding loads exactly.  Otherwise: byte
// loads of the valid groups, zero past G.
template <int M, int B, bool VEC>
__device__ __forceinline__ void load_lane_codes(const uint8_t* __restrict__ codes, int32_t row, int32_t G,
                                                int32_t gbase, uint32_t (&w)[GemvCfg<M, B>::kWords]) {
  using C = GemvCfg<M, B>;
  constexpr int bpg = M * C::kBytesPerCode;  // code bytes per group
  if constexpr (VEC && C::kCanVec) {
    const size_t off = ((size_t)row * G + (gbase < G ? gbase : 0)) * bpg;
    if constexpr (C::kCodeBytes == 16) {
      const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(codes + off));
      w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
    } else {
      const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(codes + off));
      w[0] = v[0]; w[1] = v[1];
    }
    return;
  }
  const size_t off = ((size_t)row * G + gbase) * bpg;
#pragma unroll
  for (int i = 0; i < C::kWords; ++i) w[i] = 0;
  int valid = G - gbase;
  valid = valid < 0 ? 0 : (valid > C::GPL ? C::GPL : valid);
  const int nbytes = valid * bpg;
#pragma unroll
  for (int b = 0; b < C::kCodeBytes; ++b)
    if (b < nbytes) w[b / 4] |= (uint32_t)codes[off + b] << (8 * (b % 4));
}

template <int M, int B>
__device__ __forceinline__ uint32_t code_at(const uint32_t* w, int gi, int m) {
  if constexpr (B > 8) {
    const int k = gi * M + m;
    return (w[k / 2] >> (16 * (k % 2))) & code_mask(B);
  } else {
    const int b = gi * M + m;
    return (w[b / 4] >> (8 * (b % 4))) & 0xFFu;
  }
}

constexpr int kPrefetch = 4;  // code loads in flight per wave

template <int M, int B, bool VEC, int THREADS>
__global__ __launch_bounds__(THREADS) void k_gemv(const uint8_t* __restrict__ codes, const uint4* __restrict__ cb,
                                                  const uint16_t* __restrict__ scales, const uint4* __restrict__ x,
                                                  uint16_t* __restrict__ y, int32_t d_out, int32_t G,
                                                  int32_t rows_per_wg, int32_t nchunks) {
  using C = GemvCfg<M, B>;
  constexpr int WAVES = THREADS / kWave;
  constexpr int kLdsCb = (B == 8) ? M * 256 * C::kCopies : 1;
  __shared__ uint4 cb_lds[kLdsCb];
  __shared__ float part[kMaxPartials];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int32_t row0 = blockIdx.x * rows_per_wg;
  int32_t rows_local = d_out - row0;
  if (rows_local > rows_per_wg) rows_local = rows_per_wg;
  // This wave owns rows wave, wave + WAVES, ... of the workgroup (nr of them)
  // for every chunk.  Items run chunk-major; each chunk's row list is padded
  // to a multiple of kPrefetch with repeats of its last row whose results are
  // dropped, so the unrolled loop below has no data-dependent branches.
  const int nr = rows_local > wave ? (rows_local - wave + WAVES - 1) / WAVES : 0;
  const int nr_pad = (nr + kPrefetch - 1) / kPrefetch * kPrefetch;

  auto issue = [&](int i, uint32_t (&w)[C::kWords]) {
    int c = i / nr_pad, k = i % nr_pad;
    if (c >= nchunks) { c = nchunks - 1; k = nr - 1; }
    if (k >= nr) k = nr - 1;
    load_lane_codes<M, B, VEC>(codes, row0 + wave + k * WAVES, G, c * C::kChunkGroups + lane * C::GPL, w);
  };

  // Start the first code loads before staging the codebooks so that the HBM
  // latency overlaps the LDS fill.
  uint32_t buf[kPrefetch][C::kWords];
  if (nr > 0) {
#pragma unroll
    for (int u = 0; u < kPrefetch; ++u) issue(u, buf[u]);
  }

  if constexpr (B == 8) {
    constexpr int E = M * 256;
    for (int e = tid; e < E; e += THREADS) {
      const uint4 v = cb[e];
#pragma unroll
      for (int k = 0; k < C::kCopies; ++k) cb_lds[e * C::kCopies + ((k + lane) % C::kCopies)] = v;
    }
  }
  lds_barrier();

  const uint32_t copy_off = (B == 8) ? (uint32_t)(lane % (C::kCopies ? C::kCopies : 1)) * 16u : 0u;
  if (nr > 0) {
    for (int c = 0; c < nchunks; ++c) {
      const int gbase = c * C::kChunkGroups + lane * C::GPL;
      // x slices of this lane's groups; zero past G (and the codes of a lane
      // wholly past G are masked to code 0 below).
      uint4 xr[C::GPL];
#pragma unroll
      for (int gi = 0; gi < C::GPL; ++gi) {
        const int grp = gbase + gi;
        const uint32_t keep = grp < G ? 0xFFFFFFFFu : 0u;
        const uint4 v = x[grp < G ? grp : G - 1];
        xr[gi] = make_uint4(v.x & keep, v.y & keep, v.z & keep, v.w & keep);
      }
      const uint32_t lane_keep = gbase < G ? 0xFFFFFFFFu : 0u;
      for (int k0 = 0; k0 < nr_pad; k0 += kPrefetch) {
#pragma unroll
        for (int u = 0; u < kPrefetch; ++u) {
          uint32_t cw[C::kWords];
#pragma unroll
          for (int i = 0; i < C::kWords; ++i) cw[i] = buf[u][i] & lane_keep;
          issue(c * nr_pad + k0 + u + kPrefetch, buf[u]);
          float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
          for (int gi = 0; gi < C::GPL; ++gi) {
#pragma unroll
            for (int m = 0; m < M; ++m) {
              const uint32_t code = code_at<M, B>(cw, gi, m);
              uint4 v;
              if constexpr (B == 8) {
                const uint32_t addr = ((uint32_t)(m * 256) + code) * (uint32_t)(C::kCopies * 16) + copy_off;
                v = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(cb_lds) + addr);
              } else {
                v = cb[((uint32_t)m << B) + code];
              }
              dot8(v, xr[gi], a0, a1, a2, a3);
            }
          }
          const float tot = wave_sum((a0 + a1) + (a2 + a3));
          const int k = k0 + u;
          if (lane == 0 && k < nr) part[(wave + k * WAVES) * nchunks + c] = tot;
        }
      }
    }
  }
  lds_barrier();
  for (int t = tid; t < rows_local; t += THREADS) {
    float s = 0.f;
    for (int c = 0; c < nchunks; ++c) s += part[t * nchunks + c];
    y[row0 + t] = f2h(h2f(scales[row0 + t]) * s);
  }
}

template <int M, int B, bool VEC>
static hipError_t run_gemv(const Layer& L, const uint16_t* x, uint16_t* y, hipStream_t s) {
  using C = GemvCfg<M, B>;
  constexpr int THREADS = (B == 8) ? 512 : 256;
  const int nchunks = (L.G + C::kChunkGroups - 1) / C::kChunkGroups;
  // B = 8 keeps its codebook copies in LDS (up to 128 KiB): one workgroup per
  // CU.  B = 16 uses little LDS and runs several workgroups per CU so that
  // many L2 gathers are in flight.
  int wgs = (B == 8) ? num_cus() : num_cus() * 4;
  int rows_per_wg = (L.d_out + wgs - 1) / wgs;
  if (rows_per_wg * nchunks > kMaxPartials) rows_per_wg = kMaxPartials / nchunks;
  if (rows_per_wg < 1) return hipErrorInvalidValue;
  wgs = (L.d_out + rows_per_wg - 1) / rows_per_wg;
  hipLaunchKernelGGL((k_gemv<M, B, VEC, THREADS>), dim3(wgs), dim3(THREADS), 0, s,
                     static_cast<const uint8_t*>(L.codes), reinterpret_cast<const uint4*>(L.codebooks), L.scales,
                     reinterpret_cast<const uint4*>(x), y, L.d_out, L.G, rows_per_wg, nchunks);
  return hipGetLastError();
}

template <int M, int B>
static hipError_t run_gemv_v(const Layer& L, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (GemvCfg<M, B>::kCanVec && L.vec_codes) return run_gemv<M, B, true>(L, x, y, s);
  return run_gemv<M, B, false>(L, x, y, s);
}

hipError_t launch_gemv(const Layer& L, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (L.B > 8) {
    if (L.M == 1) return L.B == 16 ? run_gemv_v<1, 16>(L, x, y, s) : run_gemv_v<1, 15>(L, x, y, s);
    switch (L.B) {
      case 12: return run_gemv_v<2, 12>(L, x, y, s);
      case 15: return run_gemv_v<2, 15>(L, x, y, s);
      case 16: return run_gemv_v<2, 16>(L, x, y, s);
    }
    return hipErrorInvalidValue;
  }
  switch (L.M) {
    case 1: return run_gemv_v<1, 8>(L, x, y, s);
    case 2: return run_gemv_v<2, 8>(L, x, y, s);
    case 3: return run_gemv_v<3, 8>(L, x, y, s);
    case 4: return run_gemv_v<4, 8>(L, x, y, s);
    case 5: return run_gemv_v<5, 8>(L, x, y, s);
    case 6: return run_gemv_v<6, 8>(L, x, y, s);
    case 7: return run_gemv_v<7, 8>(L, x, y, s);
    case 8: return run_gemv_v<8, 8>(L, x, y, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
