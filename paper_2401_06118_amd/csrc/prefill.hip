// AQLM product with many activation rows (prefill), on the matrix cores:
//   Y[t][i] = fp16(s_i * sum_c W~[i][c] X[t][c]),   W~[i, 8j:8j+8] = fp16(fp32 sum_m C_m[b_ijm])
// (Eq. 2 with the scale taken out of the sum: it multiplies the finished dot
// product instead of every weight).
//
// Unlike the batch-1 and small-batch kernels, which feed one gathered
// codeword per lane straight into an MFMA (M codewords of a group are M
// K-steps there), this kernel first dequantizes a tile of weights into LDS,
// so the matrix cores do exactly the flops of the dense product.
//
// Workgroup: 512 threads, a 128-row x BN-token output tile (BN = 256, or 128
// when there are few tiles).  Waves 0-3 (consumers) each own 64 rows x BN / 2
// tokens = 4 x BN / 32 MFMA tiles of v_mfma_f32_16x16x32_f16 (A = x,
// B = weights, D[token][row]).  Waves 4-7
// (producers) fill the next K-step's tiles while the consumers multiply the
// current ones: a K-step is 64 inputs (8 groups); per step the producers
// dequantize 128 rows x 8 groups of weights (codeword lookups from LDS
// codebook copies for 8-bit codes, 16-byte L2 gathers for wider codes, one
// or two codebooks) and
// copy BN tokens x 64 inputs of x.  Both tiles are double-buffered in LDS
// with a row pitch of 9 x 16 bytes, so the fragment reads of 16 consecutive
// rows hit 16 different bank quads.  Producer global loads run two K-steps
// ahead of their use.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

namespace {

constexpr int kPfThreads = 512;
constexpr int kBM = 128;        // output rows per workgroup
constexpr int kGK = 8;          // groups (of 8 inputs) per K-step
constexpr int kPitchU4 = kGK + 1;  // uint4 per tile row (one of padding)
constexpr int kATileU4 = kBM * kPitchU4;
constexpr size_t kPfLdsLimit = 160 * 1024;

struct PrefillArgs {
  const uint8_t* codes;
  const uint4* cb;
  const uint16_t* scales;
  const uint4* x;  // [n][G]
  uint16_t* y;     // [n][d_out]
  int32_t d_out;
  int32_t G;
  int32_t n;
};

template <int M, int B, int BN>
struct PfCfg {
  static constexpr int kXTileU4 = BN * kPitchU4;
  static constexpr int kTB = BN / 32;  // 16-token blocks per consumer wave = x rows per producer thread
  static constexpr int kBpc = code_bytes(B);
  static constexpr int kCodeBytes = 4 * M * kBpc;  // codes of a producer thread's 4 groups
  static constexpr int kCodeWords = (kCodeBytes + 3) / 4;
  // 32 KiB of codebook copies: the tiles take the rest of the LDS
  static constexpr int kCopies = (B > 8) ? 0 : 8 / M;
  static constexpr size_t kCbBytes = (B > 8) ? 0 : (size_t)M * 256 * 16 * kCopies;
  static constexpr size_t kLds = kCbBytes + 2 * (size_t)(kATileU4 + kXTileU4) * 16;
};

template <int B>
__device__ __forceinline__ uint32_t code_at(const uint32_t* w, int q) {
  if constexpr (B > 8) return (w[q / 2] >> (16 * (q % 2))) & code_mask(B);
  return (w[q / 4] >> (8 * (q % 4))) & 0xFFu;
}

// fp32 sums of fp16 halves with v_fma_mix (fma(a, 1, c) = a + c, rounded once):
// mix_add2<H>: half H of a plus half H of b; mix_add<H>: half H of c plus an
// fp32 value; mix_round2: fp16(c.lo + lo) | fp16(c.hi + hi) << 16, each
// rounded once from the exact sum.
template <int H>
__device__ __forceinline__ float mix_add2(uint32_t a, uint32_t b) {
  float d;
  if constexpr (H == 0)
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,1]" : "=v"(d) : "v"(a), "v"(b));
  else
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,1] op_sel_hi:[1,0,1]" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
template <int H>
__device__ __forceinline__ float mix_add(uint32_t c, float acc) {
  float d;
  if constexpr (H == 0)
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=v"(d) : "v"(c), "v"(acc));
  else
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(d) : "v"(c), "v"(acc));
  return d;
}
__device__ __forceinline__ uint32_t mix_round2(uint32_t c, float lo, float hi) {
  uint32_t d;
  asm("v_fma_mixlo_f16 %0, %1, 1.0, %2 op_sel:[0,0,0] op_sel_hi:[1,0,0]" : "=v"(d) : "v"(c), "v"(lo));
  asm("v_fma_mixhi_f16 %0, %1, 1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "+v"(d) : "v"(c), "v"(hi));
  return d;
}

template <int M, int B, int BN, bool VEC>
__global__ __launch_bounds__(kPfThreads) void k_prefill(const PrefillArgs a, int32_t tok_tiles) {
  using P = PfCfg<M, B, BN>;
  constexpr int kXTileU4 = P::kXTileU4;
  constexpr int kTB = P::kTB;
  extern __shared__ uint4 lds[];
  uint4* cb_lds = lds;
  uint4* a_lds = lds + P::kCbBytes / 16;  // [2][kBM][kPitchU4] dequantized weights
  uint4* x_lds = a_lds + 2 * kATileU4;    // [2][BN][kPitchU4] x

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const bool producer = wave >= 4;
  // Workgroup b takes token tile b % tok_tiles of row tile b / tok_tiles:
  // workgroups are dealt to the 8 XCDs round-robin, so with 8 token tiles
  // each XCD's L2 serves one token tile's x to all of its workgroups.
  const int32_t row0 = (int32_t)(blockIdx.x / (uint32_t)tok_tiles) * kBM;
  const int32_t tok0 = (int32_t)(blockIdx.x % (uint32_t)tok_tiles) * BN;
  const int32_t G = a.G;
  const int ksteps = (G + kGK - 1) / kGK;
  const uint32_t pitch = (uint32_t)G * M * P::kBpc;  // code bytes per row

  // codebook copies (8-bit codes): every thread helps
  if constexpr (B == 8) {
    for (int e = tid; e < M * 256; e += kPfThreads) {
      const uint4 v = a.cb[e];
#pragma unroll
      for (int k = 0; k < P::kCopies; ++k) cb_lds[e * P::kCopies + ((k + lane) % P::kCopies)] = v;
    }
  }

  // The two roles run separate copies of the step loop (their registers never
  // live at the same time); both pass the same sequence of barriers.
  if (producer) {
    // Thread p owns row p / 2, groups 4 * (p % 2) .. + 3 of each K-step, and
    // group p % 8 of tokens p / 8 + 32 i, i = 0..7 (eight lanes read one
    // token's 128 contiguous bytes).  Two register sets, indexed by
    // compile-time constants so that they stay in registers.
    const int p = tid - 4 * kWave;
    const int prow = p >> 1, pg0 = (p & 1) * 4;
    const int32_t grow = row0 + prow;
    const bool row_ok = grow < a.d_out;
    const int xtok = p >> 3, xg = p & 7;
    uint32_t cw[2][P::kCodeWords];
    uint4 xv[2][kTB];
    // Loads of step k (into register set s).  With aligned codes (VEC) every
    // load is unconditional: a step past the last one reloads the last step,
    // and rows, groups and tokens past the end read the last valid ones;
    // p_store zeroes what lies outside.  The count of loads is then the same
    // on every path, so the wait in p_store counts exactly the loads issued
    // after the ones it needs (conditional loads made the compiler wait for
    // all outstanding loads, which cancelled the lookahead).  Measured on
    // 11008x4096: 4x8 6-14 % faster; 1x16 about 1 % faster at 256 tokens
    // and 5 % slower at 2048, where the L2 gathers, not the waits, bound it.
    const int32_t grow_c = row_ok ? grow : a.d_out - 1;
    auto p_load = [&](int k, auto set) {
      constexpr int s = decltype(set)::value;
      const int kc = k < ksteps ? k : ksteps - 1;
      const int g = kc * kGK + pg0;
      if constexpr (VEC) {
        // VEC implies G % 4 == 0, so a 4-group window never crosses the row end
        const int gc = g < G ? g : G - 4;
        const uint8_t* src = a.codes + (size_t)grow_c * pitch + (size_t)gc * M * P::kBpc;
        if constexpr (P::kCodeBytes == 16) {
          const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src));
          cw[s][0] = v[0]; cw[s][1] = v[1]; cw[s][2] = v[2]; cw[s][3] = v[3];
        } else if constexpr (P::kCodeBytes == 8) {
          const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(src));
          cw[s][0] = v[0]; cw[s][1] = v[1];
        } else {
          cw[s][0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(src));
        }
      } else {
#pragma unroll
        for (int i = 0; i < P::kCodeWords; ++i) cw[s][i] = 0;
        if (row_ok && g < G) {
          const uint8_t* src = a.codes + (size_t)grow * pitch + (size_t)g * M * P::kBpc;
          const int nb = (G - g < 4 ? G - g : 4) * M * P::kBpc;
          for (int b = 0; b < nb; ++b) cw[s][b / 4] |= (uint32_t)src[b] << (8 * (b % 4));
        }
      }
      const int gx = kc * kGK + xg;
      const int gxc = gx < G ? gx : G - 1;
#pragma unroll
      for (int i = 0; i < kTB; ++i) {
        const int32_t t = tok0 + xtok + 32 * i;
        const int32_t tc = t < a.n ? t : a.n - 1;
        xv[s][i] = a.x[(size_t)tc * G + gxc];
      }
    };
    // Wide codes: the codewords of step k come from L2 with 16-byte
    // gathers (codebook m's entries start 2^B codewords after codebook
    // m - 1's), issued a step before they are stored.
    uint4 gcw[2][4 * M];
    auto p_gather = [&](auto set) {
      constexpr int s = decltype(set)::value;
#pragma unroll
      for (int q = 0; q < 4 * M; ++q) gcw[s][q] = a.cb[((uint32_t)(q % M) << B) + code_at<B>(cw[s], q)];
    };
    // Dequantize this thread's 4 groups of K-step k (register set s) and
    // store them and its x token row into LDS buffer k % 2.
    auto p_store = [&](int k, auto set) {
      constexpr int s = decltype(set)::value;
      uint4* at = a_lds + (k & 1) * kATileU4 + prow * kPitchU4 + pg0;
      const uint32_t copy_off = (uint32_t)(lane % (P::kCopies > 0 ? P::kCopies : 1)) * 16u;
      const int g = k * kGK + pg0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint4 cwv[M];
#pragma unroll
        for (int m = 0; m < M; ++m) {
          if constexpr (B == 8) {
            const uint32_t code = code_at<B>(cw[s], q * M + m);
            const uint32_t addr = ((uint32_t)(m * 256) + code) * (uint32_t)(P::kCopies * 16) + copy_off;
            cwv[m] = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(cb_lds) + addr);
          } else {
            cwv[m] = gcw[s][q * M + m];  // gathered one step earlier
          }
        }
        // Sum of the M codewords in fp32, ascending m, rounded once to fp16
        // (the scale multiplies the finished dot product).  fp16 partial sums
        // would be cheaper but each would round relative to the partial sum,
        // not to the weight: codewords that cancel would then lose the weight
        // entirely.
        h8_t wsum = __builtin_bit_cast(h8_t, cwv[0]);
        if constexpr (M == 4) {
          // v_fma_mix takes the fp16 halves directly: 6 instructions per
          // pair of weights (the compiler's convert-add-pack form takes 15)
          const uint32_t* c0 = reinterpret_cast<const uint32_t*>(&cwv[0]);
          const uint32_t* c1 = reinterpret_cast<const uint32_t*>(&cwv[1]);
          const uint32_t* c2 = reinterpret_cast<const uint32_t*>(&cwv[2]);
          const uint32_t* c3 = reinterpret_cast<const uint32_t*>(&cwv[3]);
          uint32_t o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float lo = mix_add2<0>(c0[i], c1[i]), hi = mix_add2<1>(c0[i], c1[i]);
            lo = mix_add<0>(c2[i], lo);
            hi = mix_add<1>(c2[i], hi);
            o[i] = mix_round2(c3[i], lo, hi);
          }
          wsum = __builtin_bit_cast(h8_t, make_uint4(o[0], o[1], o[2], o[3]));
        } else if constexpr (M > 1) {
          float f[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) f[e] = (float)wsum[e];
#pragma unroll
          for (int m = 1; m < M; ++m) {
            const h8_t cm = __builtin_bit_cast(h8_t, cwv[m]);
#pragma unroll
            for (int e = 0; e < 8; ++e) f[e] += (float)cm[e];
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) wsum[e] = (_Float16)f[e];
        }
        uint4 w = __builtin_bit_cast(uint4, wsum);
        if (!row_ok || g + q >= G) w = make_uint4(0, 0, 0, 0);
        at[q] = w;
      }
      uint4* xt = x_lds + (k & 1) * kXTileU4 + xtok * kPitchU4 + xg;
      const bool gx_ok = k * kGK + xg < G;
#pragma unroll
      for (int i = 0; i < kTB; ++i) {
        const bool ok = gx_ok && tok0 + xtok + 32 * i < a.n;
        xt[32 * i * kPitchU4] = ok ? xv[s][i] : make_uint4(0, 0, 0, 0);
      }
    };

    // Stage step 0, then step k + 1 while the consumers multiply step k; the
    // loads of step k + 3 go out as soon as a register set is free (and, for
    // 16-bit codes, the gathers of step k + 2 as soon as its codes are in).
    // Two steps per trip, so that the register set of step k is k % 2 at
    // compile time; one barrier per step, as in the consumer loop.
    // Loads and gathers past the last step are issued anyway (see p_load);
    // only stores and barriers depend on the step count.
    auto p_step = [&](int k, auto set_next, auto set_after) {  // while step k is multiplied
      if (k + 1 < ksteps) p_store(k + 1, set_next);
      if constexpr (B > 8) p_gather(set_after);
      p_load(k + 3, set_next);
    };
    p_load(0, IntC<0>{});
    p_load(1, IntC<1>{});
    lds_barrier();  // codebook copies visible
    if constexpr (B > 8) p_gather(IntC<0>{});
    p_store(0, IntC<0>{});
    p_load(2, IntC<0>{});
    if constexpr (B > 8) p_gather(IntC<1>{});
    lds_barrier();
    for (int k = 0; k < ksteps; k += 2) {
      p_step(k, IntC<1>{}, IntC<0>{});
      lds_barrier();
      p_step(k + 1, IntC<0>{}, IntC<1>{});
      if (k + 1 < ksteps) lds_barrier();  // the consumers pass one barrier per step
    }
  } else {
    // Wave c owns tokens BN / 2 * (c % 2) .. (kTB blocks) and rows
    // 64 * (c / 2) .. + 63 (4 blocks).
    const int r16 = lane & 15, slot = lane >> 4;
    const int ctok = (wave & 1) * (BN / 2), crow = (wave >> 1 & 1) * 64;
    f4_t acc[kTB][4];
#pragma unroll
    for (int tb = 0; tb < kTB; ++tb)
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) acc[tb][rb] = f4_t{0.f, 0.f, 0.f, 0.f};
    lds_barrier();
    lds_barrier();
    for (int k = 0; k < ksteps; ++k) {
      const uint4* at = a_lds + (k & 1) * kATileU4;
      const uint4* xt = x_lds + (k & 1) * kXTileU4;
#pragma unroll
      for (int kh = 0; kh < 2; ++kh) {  // two K32 halves of the step
        const int gq = kh * 4 + slot;   // this lane's group within the step
        h8_t wf[4];
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
          wf[rb] = __builtin_bit_cast(h8_t, at[(crow + rb * 16 + r16) * kPitchU4 + gq]);
#pragma unroll
        for (int tb = 0; tb < kTB; ++tb) {
          const h8_t xf = __builtin_bit_cast(h8_t, xt[(ctok + tb * 16 + r16) * kPitchU4 + gq]);
#pragma unroll
          for (int rb = 0; rb < 4; ++rb)
            acc[tb][rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xf, wf[rb], acc[tb][rb], 0, 0, 0);
        }
      }
      lds_barrier();
    }

    // D[token][row]: lane holds row r16 of its block and tokens 4 * slot + i.
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      const int32_t row = row0 + crow + rb * 16 + r16;
      if (row >= a.d_out) continue;
      const float sc = h2f(a.scales[row]);
#pragma unroll
      for (int tb = 0; tb < kTB; ++tb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int32_t t = tok0 + ctok + tb * 16 + 4 * slot + i;
          if (t < a.n) a.y[(size_t)t * a.d_out + row] = f2h(sc * acc[tb][rb][i]);
        }
    }
  }
}

template <int M, int B, int BN>
hipError_t run_prefill_bn(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  using P = PfCfg<M, B, BN>;
  static_assert(P::kLds <= kPfLdsLimit, "prefill LDS budget");
  // 8-byte / 16-byte code loads need every row's code pitch to keep that alignment
  const bool vec = ((int64_t)L.G * M * code_bytes(B)) % P::kCodeBytes == 0;
  auto kern = vec ? k_prefill<M, B, BN, true> : k_prefill<M, B, BN, false>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), (int)kPfLdsLimit);
    if (e != hipSuccess) return e;
  }
  // token chunks small enough for a one-dimensional grid of row x token tiles
  const int64_t row_tiles = (L.d_out + kBM - 1) / kBM;
  const int64_t chunk = ((int64_t)0x7FFFFFFF / row_tiles) * BN;
  for (int64_t t0 = 0; t0 < n; t0 += chunk) {
    const int32_t nt = (int32_t)(n - t0 < chunk ? n - t0 : chunk);
    const int32_t tok_tiles = (nt + BN - 1) / BN;
    const PrefillArgs a{static_cast<const uint8_t*>(L.codes), reinterpret_cast<const uint4*>(L.codebooks), L.scales,
                        reinterpret_cast<const uint4*>(x + t0 * L.d_in), y + t0 * L.d_out, L.d_out, L.G, nt};
    hipLaunchKernelGGL(kern, dim3((uint32_t)(row_tiles * tok_tiles)), dim3(kPfThreads), P::kLds, s, a, tok_tiles);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// 256-token tiles when there are enough of them to fill the chip twice over,
// else 128-token tiles (twice the workgroups, half the reuse of each
// dequantized weight tile).
template <int M, int B>
hipError_t run_prefill(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  const int64_t row_tiles = (L.d_out + kBM - 1) / kBM;
  if (row_tiles * ((n + 255) / 256) >= 2 * num_cus()) return run_prefill_bn<M, B, 256>(L, n, x, y, s);
  return run_prefill_bn<M, B, 128>(L, n, x, y, s);
}

}  // namespace

bool prefill_supported(const Layer& L) {
  if (L.B > 8) return L.M == 1 || L.M == 2;
  return L.M == 1 || L.M == 2 || L.M == 4;
}

hipError_t launch_prefill(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (L.B > 8 && L.M == 2) {
    switch (L.B) {
      case 12: return run_prefill<2, 12>(L, n, x, y, s);
      case 15: return run_prefill<2, 15>(L, n, x, y, s);
      case 16: return run_prefill<2, 16>(L, n, x, y, s);
    }
    return hipErrorInvalidValue;
  }
  if (L.B == 16) return L.M == 1 ? run_prefill<1, 16>(L, n, x, y, s) : hipErrorInvalidValue;
  if (L.B == 15) return L.M == 1 ? run_prefill<1, 15>(L, n, x, y, s) : hipErrorInvalidValue;
  switch (L.M) {
    case 1: return run_prefill<1, 8>(L, n, x, y, s);
    case 2: return run_prefill<2, 8>(L, n, x, y, s);
    case 4: return run_prefill<4, 8>(L, n, x, y, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
