// Batch-1 AQLM product through per-group partial-product tables (2x8).
//
// With x fixed, every code of codebook m in input group j contributes
// <C_m[b], x[8j:8j+8]> to its row, whatever the row.  So the inner products
//   T_m[e][j] = <C_m[e], x_j>        (every codeword e, every group j)
// are computed once per workgroup, and the product of Eq. 2 becomes
//   y_i = fp16(s_i * sum_j sum_m T_m[b_ijm][j])
// - M table reads and adds per group instead of M codeword gathers and
// multiply-adds.  This is the lookup of precomputed inner products that
// search with product and additive codes uses (Sec. 2.2), applied to the
// matrix-vector product.
//
// Tables.  A K-slice is 32 groups (256 inputs).  Its table holds 2 x 256 x
// 32 fp32 entries (64 KiB): entry (e, m, j) at byte e*256 + m*128 + j*4.
// Two tables are double-buffered in LDS: while the workgroup looks codes up
// in the table of slice k, it builds the table of slice k + 1 in the other
// buffer, one barrier per slice.  The build is a dense product on the matrix
// cores: v_mfma_f32_32x32x8_f16 with 32 codewords as A (K = 8 = one group)
// and the x vectors of the slice's 32 groups as B; wave w owns codewords
// 32w .. 32w + 31 of the 512 (both codebooks), so its A operand is loaded
// once.  Entries are fp32: rounding them to fp16 would make each one's error
// relative to <C_m[e], x_j>, which codewords that cancel leave far larger
// than the weight.
//
// Lookups.  A wave load covers 4 rows x one slice (64 bytes per row): lane
// (r, q) holds the 4 code bytes of groups 2q and 2q + 1 of row r.  In slot t
// of a K-slice the lane reads group j = 2q + ((t + r) & 1) and takes the
// codebooks in the order m = t' ^ (r >> 1), so the 64 lanes of every read
// hit 64 different LDS banks (bank = m * 32 + j).  One v_perm_b32 builds the
// address from the code byte (byte 1 = e) and a per-lane constant (byte 0 =
// m * 128 + j * 4, byte 2 = buffer).
//
// Rows.  A workgroup owns rows_per_wg rows (4-row quads dealt round-robin to
// its 16 waves) and all K-slices, so the cost of a table is shared by the
// workgroup's rows.  Writing a table takes about as many LDS instructions as
// 256 rows of lookups in it, so the kernel needs a few hundred rows per
// workgroup to break even (Llama-2-70B gate/up: 224).
// Each lane keeps one fp32 sum per quad; at the end the 16 lanes of a row
// are added with DPP moves in a fixed order, so results are deterministic.
//
// Code loads run through a register ring D K-slices deep.  The x fragments
// of a slice go out right before its code loads: loads retire in issue
// order, so waiting for the fragment of slice k + 1 (needed to build its
// table) never waits for code loads issued after it.  Every load is
// unconditional (past the last slice the last one is reloaded), so each wait
// counts exactly the loads issued after the one it needs.
#include "common.h"
#include "launch.h"
#include "lds_sync.h"

namespace aqlm {

namespace {

constexpr int kLWaves = 16;
constexpr int kLThreads = kLWaves * kWave;
constexpr int kLG = 32;                          // groups per K-slice
constexpr int kLTabFloats = 256 * 2 * kLG;       // one table (16384 fp32, 64 KiB)
constexpr int kLLds = 2 * kLTabFloats * 4;       // two tables

typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) const float lds_f32_t;

__device__ __forceinline__ float lds_f32(uint32_t byte_addr) { return *(lds_f32_t*)(uintptr_t)byte_addr; }

// Sum over the 16 lanes of each DPP row (every lane gets its row's sum).
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, true));
  return v;
}

// D: ring depth in K-slices (even, so that a slice's table buffer is known at
// compile time); Q: 4-row quads per wave at most.
template <int D, int Q>
__global__ __launch_bounds__(kLThreads) void k_gemv_lut(const GemvBatch bt) {
  static_assert(D % 2 == 0, "ring depth must be even");
  extern __shared__ float tab[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);

  int p = 0;
  while (p + 1 < bt.count && bt.p[p + 1].wg_begin <= (int)blockIdx.x) ++p;
  const int32_t rows_per_wg = bt.p[p].rows_per_wg;
  const int32_t row0 = ((int32_t)blockIdx.x - bt.p[p].wg_begin) * rows_per_wg;
  int32_t rows = bt.p[p].d_out - row0;
  if (rows > rows_per_wg) rows = rows_per_wg;
  const int32_t G = bt.p[p].G;
  const int nks = G / kLG;                      // G is a multiple of kLG (launcher)
  const uint32_t pitch = (uint32_t)G * 2u;      // code bytes per row
  const int nquads = (rows + 3) >> 2;
  const int nq = nquads > wave ? (nquads - wave + kLWaves - 1) / kLWaves : 0;  // <= Q
  const int q = lane & 15, r = lane >> 4;
  const uint8_t* __restrict__ codes = bt.p[p].codes + (size_t)row0 * pitch;
  const char* __restrict__ xb = reinterpret_cast<const char*>(bt.p[p].x);

  // 1. small loads first: this wave's codeword fragments and the scales of
  // its rows (clamped rows; the extra ones are never stored).
  const int mw = wave >> 3;        // codebook of the wave's 32 codewords
  const int ew = (wave & 7) * 32;  // first of them
  const int half = lane >> 5;      // which 4 of a group's 8 values the fragments carry
  const int col = lane & 31;       // A: codeword; B: group within the slice
  const h4_t afrag = *reinterpret_cast<const h4_t*>(reinterpret_cast<const char*>(bt.p[p].cb) +
                                                    ((mw * 256 + ew + col) * 16 + half * 8));
  uint32_t roff[Q];
  uint16_t sc[Q];
#pragma unroll
  for (int u = 0; u < Q; ++u) {
    int row = (wave + u * kLWaves) * 4 + r;
    row = row < rows ? row : rows - 1;
    roff[u] = (uint32_t)row * pitch + (uint32_t)q * 4u;
    sc[u] = bt.p[p].scales[row0 + row];
  }

  // 2. x fragments and codes of the first D K-slices.
  h4_t xr[D];
  uint32_t ring[D][Q];
  auto issue = [&](int ks, h4_t& xf, uint32_t (&w)[Q]) {
    const int kc = ks < nks ? ks : nks - 1;
    xf = *reinterpret_cast<const h4_t*>(xb + (size_t)(kc * kLG + col) * 16 + half * 8);
#pragma unroll
    for (int u = 0; u < Q; ++u)
      w[u] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(codes + roff[u] + (uint32_t)kc * 64u));
  };
#pragma unroll
  for (int d = 0; d < D; ++d) issue(d, xr[d], ring[d]);

  // Table build: this wave's 32 codewords x the slice's 32 groups.
  const uint32_t wbase = (uint32_t)(ew + 4 * half) * 64u + (uint32_t)mw * 32u + (uint32_t)col;
  auto build = [&](int buf, const h4_t& xf) {
    const f32x16_t t = __builtin_amdgcn_mfma_f32_32x32x8f16(afrag, xf, f32x16_t{}, 0, 0, 0);
    float* dst = tab + buf * kLTabFloats + wbase;
#pragma unroll
    for (int i = 0; i < 16; ++i) dst[(8 * (i / 4) + (i % 4)) * 64] = t[i];
  };

  // Lookup constants: for slot t and codebook position mm, the codebook
  // m = mm ^ (r >> 1) and group j = 2q + ((t + r) & 1); v_perm takes byte 0
  // (m * 128 + j * 4) and byte 2 (the buffer) from lc, byte 1 from the code
  // word (byte 2 * ((t + r) & 1) + m: group, then codebook), byte 3 = 0.
  uint32_t lc[2][2][2], sel[2][2];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int mm = 0; mm < 2; ++mm) {
      const int m = mm ^ (r >> 1), s = (t + r) & 1, j = 2 * q + s;
      const uint32_t c = (uint32_t)(m * 128 + j * 4);
      lc[0][t][mm] = c;
      lc[1][t][mm] = c | 0x10000u;
      sel[t][mm] = 0x0C020000u | ((uint32_t)(4 + 2 * s + m) << 8);
    }

  float acc[Q];
#pragma unroll
  for (int u = 0; u < Q; ++u) acc[u] = 0.f;

  build(0, xr[0]);
  lds_barrier();

  // 3. K-slices, D per trip: slice ks = j0 + d uses ring slot d and table
  // buffer d & 1; it builds slice ks + 1's table into the other buffer and
  // refills slot d with slice ks + D.
  for (int j0 = 0; j0 < nks; j0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int ks = j0 + d;
      if (ks < nks) {  // (the same for the whole workgroup)
        const int buf = d & 1;
        // lookups of slice ks
        float tv[Q][4];
#pragma unroll
        for (int u = 0; u < Q; ++u) {
          if (u < nq) {
            const uint32_t w = ring[d][u];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int mm = 0; mm < 2; ++mm)
                tv[u][2 * t + mm] = lds_f32(__builtin_amdgcn_perm(w, lc[buf][t][mm], sel[t][mm]));
          }
        }
        // table of slice ks + 1 (past the last slice: a copy of the last
        // one, into the buffer no one reads any more)
        build(buf ^ 1, xr[(d + 1) % D]);
#pragma unroll
        for (int u = 0; u < Q; ++u)
          if (u < nq) acc[u] += (tv[u][0] + tv[u][1]) + (tv[u][2] + tv[u][3]);
        issue(ks + D, xr[d], ring[d]);
        lds_barrier();
      }
    }
  }

  // 4. per row: sum of its 16 lanes, scale, round, store.
#pragma unroll
  for (int u = 0; u < Q; ++u) {
    if (u < nq) {
      const float v = row16_sum(acc[u]);
      const int row = (wave + u * kLWaves) * 4 + r;
      if (q == 0 && row < rows) bt.p[p].y[row0 + row] = f2h(h2f(sc[u]) * v);
    }
  }
}

template <int D, int Q>
hipError_t launch_lut(const GemvBatch& bt, hipStream_t s) {
  auto kern = k_gemv_lut<D, Q>;
  const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), kLLds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(bt.total_wgs), dim3(kLThreads), kLLds, s, bt);
  return hipGetLastError();
}

}  // namespace

// 2x8 layers whose rows can take the table kernel: whole K-slices of 32
// groups (d_in a multiple of 256).
bool gemv_lut_supported(const Layer* Ls, int count) {
  for (int i = 0; i < count; ++i) {
    const Layer& L = Ls[i];
    if (L.M != 2 || L.B != 8 || L.G % kLG != 0) return false;
    if ((reinterpret_cast<uintptr_t>(L.codes) & 3) != 0) return false;
  }
  return count >= 1 && count <= kMaxProblems;
}

hipError_t launch_gemv_lut(const Layer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                           hipStream_t s) {
  if (!gemv_lut_supported(Ls, count)) return hipErrorInvalidValue;
  const int cus = num_cus();
  double total = 0;
  for (int i = 0; i < count; ++i) total += (double)Ls[i].d_out * Ls[i].G;
  // CUs per problem in proportion to its codes, by largest remainders (as
  // the matrix-core kernel), one workgroup per CU (the tables take 128 KiB
  // of LDS), rows per workgroup a multiple of 4, at most 256 (four quads per
  // wave: the most that fit in registers with the code ring); larger layers
  // run more workgroups than CUs.
  int want_of[kMaxProblems];
  {
    double rem[kMaxProblems];
    int sum = 0;
    for (int i = 0; i < count; ++i) {
      const double share = cus * ((double)Ls[i].d_out * Ls[i].G) / total;
      want_of[i] = share < 1.0 ? 1 : (int)share;
      rem[i] = share - (double)want_of[i];
      sum += want_of[i];
    }
    while (sum < cus) {
      int best = 0;
      for (int i = 1; i < count; ++i)
        if (rem[i] > rem[best]) best = i;
      ++want_of[best];
      rem[best] -= 1.0;
      ++sum;
    }
  }
  GemvBatch bt{};
  bt.count = count;
  int wg = 0, rpw_max = 4;
  for (int i = 0; i < count; ++i) {
    const Layer& L = Ls[i];
    int rpw = (L.d_out + want_of[i] - 1) / want_of[i];
    rpw = (rpw + 3) & ~3;
    if (rpw > 4 * 4 * kLWaves) rpw = 4 * 4 * kLWaves;
    const int nwg = (L.d_out + rpw - 1) / rpw;
    GemvProblem& P = bt.p[i];
    P.codes = static_cast<const uint8_t*>(L.codes);
    P.cb = reinterpret_cast<const uint4*>(L.codebooks);
    P.scales = L.scales;
    P.x = reinterpret_cast<const uint4*>(xs[i]);
    P.y = ys[i];
    P.d_out = L.d_out;
    P.G = L.G;
    P.wg_begin = wg;
    P.rows_per_wg = rpw;
    wg += nwg;
    if (rpw > rpw_max) rpw_max = rpw;
  }
  bt.total_wgs = wg;
  bt.xg_max = 0;
  const int quads = (rpw_max / 4 + kLWaves - 1) / kLWaves;  // per wave
  switch (quads) {
    case 1: return launch_lut<8, 1>(bt, s);
    case 2: return launch_lut<8, 2>(bt, s);
    case 3: return launch_lut<6, 3>(bt, s);
    case 4: return launch_lut<6, 4>(bt, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace aqlm
