// Batch-1 AQLM matrix-vector product on the matrix cores (the token
// generation product of Sec. 4.3):  y_i = fp16(s_i * sum_j sum_m <C_m[b_ijm], x_j>).
//
// v_mfma_f32_16x16x32_f16 takes, per lane, 8 consecutive K values of one row
// of A (lane = row + 16 * K-slot) and 8 K values of one column of B (lane =
// column + 16 * K-slot).  A lane's A fragment is one gathered codeword, so the
// matrix core does the multiply-adds that a vector-ALU version would spend
// v_dot2 instructions on, and it also sums over K, so no cross-lane reduction
// is needed.  Only column 0 of B carries x (the other 15 columns read the same
// LDS address and their outputs are ignored).
//
// Work split.  A workgroup (16 waves) owns a range of rows of one problem.  An
// item is 16 rows x one K-slice of 4 x kCPL codes (kCPL = 16 codes, 16 bytes,
// per lane); lane (r, s) streams the codes [s*kCPL, s*kCPL + kCPL) of the
// slice for row r with one 16-byte load.  Three kernels:
//   k_gemv_mfma (codes wider than 8 bits: one codebook in small launches,
//     two codebooks always): items dealt round-robin to the waves, one
//     accumulator per wave, stored to LDS whenever its row block changes;
//     codewords gathered from L2, or from one LDS copy of two 12-bit
//     codebooks (128 KiB);
//   k_gemv_ks (B = 8): each wave owns whole K-slices of all the workgroup's
//     row blocks and keeps one accumulator per block;
//   k_gemv_cb (one codebook of 15- or 16-bit codes, large launches): the
//     k_gemv_ks split with the codes held in registers, run once per 128 KiB
//     codebook chunk staged in LDS.
// k_gemv_mfma and k_gemv_cb also read bit-packed codes (B bits per code, a
// bit string per row): a lane loads the 3 or 5 dwords that hold its slot's 8
// codes and cuts them out with shifts.
// In every case the per-wave partials are added in a fixed order at the end,
// so results are deterministic.
//
// Memory order.  Vector-memory loads retire in issue order, so the small
// loads that must finish first (codebooks, x) are issued before the HBM code
// stream; all NI code loads of a wave are then in flight at once.  While
// they arrive the codebooks are copied COPIES times into LDS (lane l reads
// copy l % COPIES, so 16 lanes hit 16 different 16-byte bank quads) and x is
// staged in LDS, zero-padded to whole K-slices.  Codebooks of wider codes
// (2^B codewords, up to 1 MiB each) either stay in L2 and are gathered with
// 16-byte global loads, or, for a single codebook, pass through LDS chunk by
// chunk (k_gemv_cb).
//
// Several independent problems with the same (M, B) can share one launch
// (e.g. the q, k, v projections of a layer): workgroups are dealt to the
// problems in proportion to their code bytes.
#include "common.h"
#include "launch.h"
#include "stream_common.h"

namespace aqlm {

namespace {

constexpr int kWaves = 16;
constexpr int kThreads = kWaves * kWave;
constexpr int kMaxRB = 8;  // 16-row blocks per workgroup

// PACKED: bit-packed B-bit codes (B = 12 or 15), a slot's 8 codes cut out of
// the 3 (B = 12) or 5 (B = 15) 32-bit words that hold them; a slot of 15-bit
// codes starts 24 * slot % 32 bits into its first word.
template <int M, int B, int COPIES, int PF, bool VEC, bool PACKED = false>
__global__ __launch_bounds__(kThreads) void k_gemv_mfma(const GemvBatch bt) {
  using C = GCfg<B>;
  static_assert(!PACKED || B == 12 || B == 15, "packed codes: 12 or 15 bits");
  constexpr int kW = PACKED ? (B == 12 ? 3 : 5) : 4;  // code words per slot
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  // wave-uniform: lets the item bookkeeping below run on the scalar unit
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15;
  const int slot = lane >> 4;

  int p = 0;
  while (p + 1 < bt.count && bt.p[p + 1].wg_begin <= (int)blockIdx.x) ++p;
  const uint4* __restrict__ cb = bt.p[p].cb;
  const uint4* __restrict__ x = bt.p[p].x;
  const int32_t rows_per_wg = bt.p[p].rows_per_wg;
  const int32_t row0 = ((int32_t)blockIdx.x - bt.p[p].wg_begin) * rows_per_wg;
  int32_t rows = bt.p[p].d_out - row0;
  if (rows > rows_per_wg) rows = rows_per_wg;
  const int RB = (rows + 15) / 16;
  const int32_t G = bt.p[p].G;
  const uint32_t pitch = (uint32_t)G * M * C::kBpc;     // code bytes per row
  const int KS = (int)((pitch + 63u) / 64u);             // 64-byte K-slices per row (4 slots x 16 bytes)
  const int items = RB * KS;
  const int xg = KS * (C::kKS / M);  // x groups staged (zero past G)
  // Items are dealt round-robin: wave w takes items w, w + 16, w + 32, ...
  // (nk of them); item i covers row block i / KS and K-slice i % KS.
  const int nk = items > wave ? (items - wave + kWaves - 1) / kWaves : 0;
  const uint32_t pwords = (uint32_t)bt.p[p].pwords;  // packed: 32-bit words per row
  const uint8_t* __restrict__ wg_codes = bt.p[p].codes + (size_t)row0 * (PACKED ? pwords * 4u : pitch);

  // Wide codes with COPIES = 1: the M codebooks sit whole in LDS, one copy
  // (two 4096-entry codebooks are 128 KiB).
  constexpr bool kWideLds = B > 8 && COPIES > 0;
  static_assert(!kWideLds || (COPIES == 1 && (M << B) * 16 <= 128 * 1024), "wide codebooks: one copy, 128 KiB");
  constexpr int kCbEntries = (B == 8) ? M * 256 * COPIES : (kWideLds ? (M << B) : 0);
  constexpr int kWideLoads = kWideLds ? kCbEntries / kThreads : 1;  // codebook loads per thread
  uint4* cb_lds = lds;
  uint4* x_lds = lds + kCbEntries;
  float* part = reinterpret_cast<float*>(x_lds + bt.xg_max);

  // 1. small loads first (codebooks, x, scales): vector-memory loads retire in issue
  // order, so these complete without waiting for the HBM code stream.
  uint4 cbv = make_uint4(0, 0, 0, 0);
  if constexpr (B == 8) {
    if (tid < M * 256) cbv = cb[tid];
  }
  uint4 cbw[kWideLoads];
  if constexpr (kWideLds) {
#pragma unroll
    for (int i = 0; i < kWideLoads; ++i) cbw[i] = cb[tid + i * kThreads];
  }
  // this thread's output row scale, needed only at the end (an unconditional
  // load of a clamped row, so that nothing waits for it here)
  const uint16_t sc = bt.p[p].scales[row0 + (tid < rows ? tid : rows - 1)];
  uint4 xv[C::kXL];
#pragma unroll
  for (int i = 0; i < C::kXL; ++i) {
    const int grp = tid + i * kThreads;
    xv[i] = make_uint4(0, 0, 0, 0);
    if (grp < G) xv[i] = x[grp];
  }

  // 2. the first PF items of the code stream.  The prefetch cursor stops at
  // the wave's last item, so loads past the end repeat that item (valid
  // memory; their results are never used).
  const uint32_t slot_off = (uint32_t)slot * 16u;
  auto issue = [&](int rb, int ks, uint32_t (&w)[kW]) {
    int row = rb * 16 + r16;
    row = row < rows ? row : rows - 1;
    const uint32_t off = (uint32_t)ks * 64u + slot_off;
    if constexpr (PACKED) {
      // words of codes 8 * (4 ks + slot) .. + 7, as one 12-byte load (B = 12)
      // or a 16-byte and a 4-byte load (B = 15), dword-aligned; at the end
      // of a row the words past its last are clamped to it, one by one (those
      // codes meet x = 0)
      const uint32_t* rw = reinterpret_cast<const uint32_t*>(wg_codes) + (size_t)row * pwords;
      const uint32_t w0 = ((uint32_t)(ks * 4 + slot) * 8u * (uint32_t)B) >> 5;
      if (w0 + (uint32_t)kW <= pwords) {
        if constexpr (B == 12) {
          const u32x3a4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x3a4_t*>(rw + w0));
          w[0] = v[0]; w[1] = v[1]; w[2] = v[2];
        } else {
          const u32x4a4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4a4_t*>(rw + w0));
          w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
          w[4] = __builtin_nontemporal_load(rw + w0 + 4);
        }
      } else {
#pragma unroll
        for (int i = 0; i < kW; ++i) {
          const uint32_t wi = w0 + (uint32_t)i < pwords ? w0 + (uint32_t)i : pwords - 1u;
          w[i] = __builtin_nontemporal_load(rw + wi);
        }
      }
    } else if constexpr (VEC) {
      // a 16-byte slot is wholly inside the row or wholly past its end
      const uint32_t o = (uint32_t)row * pitch + (off < pitch ? off : 0u);
      const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(wg_codes + o));
      w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
    } else {
      load_codes_bytes<B>(wg_codes + (size_t)row * pitch, pitch, off, w);
    }
  };
  auto advance = [&](int& rb, int& ks) {
    ks += kWaves;
    while (ks >= KS) { ks -= KS; ++rb; }
  };
  int f_rb = nk > 0 ? wave / KS : 0, f_ks = nk > 0 ? wave % KS : 0, f_k = 0;
  uint32_t buf[PF][kW];
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    issue(f_rb, f_ks, buf[u]);
    if (f_k + 1 < nk) advance(f_rb, f_ks);
    ++f_k;
  }

  // 3. stage codebook copies, x and zeroed partials in LDS.
  if constexpr (B == 8) {
    if (tid < M * 256) {
#pragma unroll
      for (int k = 0; k < COPIES; ++k) cb_lds[tid * COPIES + ((k + lane) % COPIES)] = cbv;
    }
  }
  if constexpr (kWideLds) {
#pragma unroll
    for (int i = 0; i < kWideLoads; ++i) cb_lds[tid + i * kThreads] = cbw[i];
  }
#pragma unroll
  for (int i = 0; i < C::kXL; ++i) {
    const int grp = tid + i * kThreads;
    if (grp < xg) x_lds[grp] = xv[i];
  }
  for (int e = tid; e < RB * kWaves * 16; e += kThreads) part[e] = 0.f;
  __syncthreads();

  // 4. stream the items: gather codewords (A), x from LDS (B), MFMA.
  const uint32_t copy_off = (uint32_t)(lane % (COPIES > 0 ? COPIES : 1)) * 16u;
  // LDS byte address of the codebook copies (low 32 bits of the flat address
  // of an LDS object are its LDS offset)
  const uint32_t cb_base = (uint32_t)(uintptr_t)cb_lds;
  uint32_t base_m[M];
#pragma unroll
  for (int m = 0; m < M; ++m) base_m[m] = cb_base + ((uint32_t)m << 16) + copy_off;
  f4_t acc = {0.f, 0.f, 0.f, 0.f}, acc2 = {0.f, 0.f, 0.f, 0.f};  // even / odd steps
  // B operand: only column 0 (lanes with r16 == 0) carries x; the other
  // columns keep whatever they hold and their outputs are never read.
  uint4 xb = make_uint4(0, 0, 0, 0);
  int cur_rb = -1;
  int c_rb = nk > 0 ? wave / KS : 0, c_ks = nk > 0 ? wave % KS : 0;
  for (int k0 = 0; k0 < nk; k0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int k = k0 + u;
      // the slot's 8 codes: 16-bit lanes of 4 words, or a packed bit string
      // (shifted to start at bit 0)
      uint32_t cw[4];
      if constexpr (!PACKED) {
#pragma unroll
        for (int i = 0; i < 4; ++i) cw[i] = buf[u][i];
      } else if constexpr (B == 12) {
#pragma unroll
        for (int i = 0; i < 3; ++i) cw[i] = buf[u][i];
        cw[3] = 0;
      } else {
        const uint32_t sh = (24u * (uint32_t)slot) & 31u;
#pragma unroll
        for (int i = 0; i < 4; ++i) cw[i] = __builtin_amdgcn_alignbit(buf[u][i + 1], buf[u][i], sh);
      }
      auto code_of = [&](int t) -> uint32_t {
        if constexpr (PACKED) {
          const int b = t * B, wd = b >> 5, of = b & 31;
          uint32_t v = cw[wd] >> of;
          if (of + B > 32) v |= cw[wd + 1] << (32 - of);
          return v & code_mask(B);
        } else {
          return (cw[t / 2] >> (16 * (t % 2))) & code_mask(B);
        }
      };
      uint4 av[C::kCPL];
      if constexpr (B > 8 && !kWideLds) {
        // L2 gathers go out before the next code load so that waiting for
        // them does not wait for HBM.  Code t of a slot belongs to codebook
        // t % M (2^B codewords of 16 bytes each).
        if (k < nk) {
#pragma unroll
          for (int t = 0; t < C::kCPL; ++t)
            av[t] = *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(cb) +
                                                    ((uint32_t)(t % M) << (B + 4)) + (code_of(t) << 4));
        }
      }
      issue(f_rb, f_ks, buf[u]);
      if (f_k + 1 < nk) advance(f_rb, f_ks);
      ++f_k;
      if (k < nk) {
        if (c_rb != cur_rb) {
          if (cur_rb >= 0 && r16 == 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) part[(cur_rb * kWaves + wave) * 16 + 4 * slot + e] = acc[e] + acc2[e];
          }
          acc = f4_t{0.f, 0.f, 0.f, 0.f};
          acc2 = f4_t{0.f, 0.f, 0.f, 0.f};
          cur_rb = c_rb;
        }
        // x groups of this lane's codes; past the row end x is zero
        const uint4* xs = x_lds + (((uint32_t)c_ks * C::kKS + (uint32_t)slot * C::kCPL) / M);
#pragma unroll
        for (int t0 = 0; t0 < C::kCPL; t0 += 4) {
          if constexpr (B == 8) {
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) {
              const int t = t0 + uu;
              const uint32_t addr = cw_addr<M, COPIES>(cw[t / 4], t % 4, base_m[t % M], copy_off + cb_base, t % M);
              av[t] = lds_load16(addr);
            }
          } else if constexpr (kWideLds) {
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) {
              const int t = t0 + uu;
              av[t] = lds_load16(cb_base + ((uint32_t)(t % M) << (B + 4)) + (code_of(t) << 4));
            }
          }
#pragma unroll
          for (int uu = 0; uu < 4; ++uu) {
            const int t = t0 + uu;
            if (t % M == 0 || uu == 0) {  // codes t .. t+M-1 share the group t/M of the slot
              if (r16 == 0) xb = xs[t / M];
            }
            f4_t& a = (uu % 2 == 0) ? acc : acc2;
            a = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[t]), __builtin_bit_cast(h8_t, xb),
                                                      a, 0, 0, 0);
          }
        }
        advance(c_rb, c_ks);
      }
    }
  }
  if (cur_rb >= 0 && r16 == 0) {
#pragma unroll
    for (int e = 0; e < 4; ++e) part[(cur_rb * kWaves + wave) * 16 + 4 * slot + e] = acc[e] + acc2[e];
  }
  __syncthreads();

  // 5. fixed-order sum over waves, scale, round, store.
  if (tid < rows) {
    const int rb = tid / 16, rr = tid % 16;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += part[(rb * kWaves + w) * 16 + rr];
    bt.p[p].y[row0 + tid] = f2h(h2f(sc) * s);
  }
}

// B = 8 variant, K-slice major.  Wave w owns the K-slices ks = w, w + 16, ...
// of the workgroup's RB row blocks.  For each of its K-slices it reads the
// x slices of its four code slots once into registers (column-0 lanes
// only), then runs the RB items (row blocks) of that slice, each into its own
// accumulator, so no partial sums move until the end.  Code loads run
// through a register ring of D K-slices, a few items ahead of their use.
//
// The body serves two kernels: k_gemv_ks (one launch per grouped product;
// vwg = blockIdx.x) and the persistent decode-step kernel k_gemv_step
// (STEP = true), which runs many such products in a row on a resident grid.
// With STEP, the code, codebook and scale loads of a product go out before
// `wait()` (the level barrier: the previous product's outputs may be this
// one's x), x is read after it with system-scope loads and y written with
// system-scope stores (other workgroups of the same grid read it next, from
// other XCDs); returns false when the wait gave up.
template <int M, int COPIES, int RB, int D, bool VEC, bool STEP, typename Wait>
__device__ __forceinline__ bool ks_body(const GemvBatch& bt, const int vwg, Wait&& wait) {
  using C = GCfg<8>;
  constexpr int kXS = C::kCPL / M;  // x slices per code slot per K-slice
  // codewords gathered per block before their MFMAs (fewer where the
  // accumulators or, for M = 1, the sixteen x slices take the registers)
  constexpr int kStep = (RB >= 5 || M == 1) ? 2 : 4;
  // (the byte-load path of unaligned rows has no registers to spare for it
  // in its largest layouts)
  constexpr bool kPinGathers = VEC || (RB < 7 && D < 4);
  // The wave's items run K-slice major, (j, rb) -> item j * RB + rb, through a
  // ring of kSlots code registers (D K-slices of RB blocks).  Consuming an
  // item starts the load of the item kAhead places later (kAhead <= kSlots,
  // so its slot is free), so kAhead items are in flight.  Row blocks are
  // consumed in pairs, so a load is used at least kAhead - 2 items after it
  // is requested.
  constexpr int kSlots = D * RB;
  // Paired blocks: two items ahead (the next pair is requested as the
  // current one starts).  Fewer code loads in flight per wave let the items
  // that every wave needs next arrive sooner, and 16 waves x 2 items still
  // keep about 8 MiB in flight across the chip.  Measured (same box):
  // Llama-2-70B step 5.38-5.41 ms with two ahead, 5.50-5.51 with three,
  // 5.87-5.90 with four (five or six slower still); 7B step 0.853 / 0.906 /
  // 0.888 ms.  An odd block count ends each K-slice with a lone block, which
  // requests one item, so the next pair's first item would be asked for only
  // one item before its use: three ahead there (tiled codes: Llama-2-70B
  // q/k/v, 3 blocks, 9.2 -> 8.5 us, gate/up, 7 blocks, 29.7 -> 28.8 us; step
  // 5.30-5.32 -> 5.21-5.22 ms, 7B unchanged).  Single blocks: the whole ring
  // (four ahead measured the same).
  constexpr int kAheadWant = RB >= 2 ? (RB % 2 == 1 ? 3 : 2) : 8;
  constexpr int kAhead = kAheadWant < kSlots ? kAheadWant : kSlots;
  static_assert(RB < 2 || kAhead >= 2, "both items of a pair must be requested before the pair starts");
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15;
  const int slot = lane >> 4;

  int p = 0;
  while (p + 1 < bt.count && bt.p[p + 1].wg_begin <= vwg) ++p;
  const uint4* __restrict__ cb = bt.p[p].cb;
  const uint4* __restrict__ x = bt.p[p].x;
  const int32_t rows_per_wg = bt.p[p].rows_per_wg;
  const int32_t row0 = ((int32_t)vwg - bt.p[p].wg_begin) * rows_per_wg;
  int32_t rows = bt.p[p].d_out - row0;
  if (rows > rows_per_wg) rows = rows_per_wg;
  const int32_t G = bt.p[p].G;
  const uint32_t pitch = (uint32_t)G * M;           // code bytes per row
  const int KS = (int)((pitch + 63u) / 64u);        // 64-byte K-slices per row
  const int xg = KS * (C::kKS / M);
  const int nks = KS > wave ? (KS - wave + kWaves - 1) / kWaves : 0;
  // Row-major codes: a wave's item is 16 rows x 64 bytes at the row pitch.
  // Tiled codes: the same item is one contiguous 1 KiB tile.
  const bool tiled = bt.tiled != 0;
  const uint8_t* __restrict__ wg_codes = tiled ? bt.p[p].codes : bt.p[p].codes + (size_t)row0 * pitch;
  const uint32_t k_stride = tiled ? 1024u : 64u;   // bytes from one K-slice to the next
  const uint32_t k_limit = tiled ? 0xFFFFFFFFu : pitch;  // (tiles hold whole K-slices)

  uint4* cb_lds = lds;
  uint4* x_lds = lds + M * 256 * COPIES;
  float* part = reinterpret_cast<float*>(x_lds + bt.xg_max);

  // (a persistent workgroup may still be reading the previous product's
  // partial sums, which this one's staging can overlap)
  if constexpr (STEP) __syncthreads();

  // 1. codebooks, x and scales first (they retire before the code stream).
  uint4 cbv = make_uint4(0, 0, 0, 0);
  if (tid < M * 256) cbv = cb[tid];
  // this thread's output row scale, needed only at the end (an unconditional
  // load of a clamped row, so that nothing waits for it here)
  const uint16_t sc = bt.p[p].scales[row0 + (tid < rows ? tid : rows - 1)];
  uint4 xv[C::kXL];
  auto load_x = [&]() {
#pragma unroll
    for (int i = 0; i < C::kXL; ++i) {
      const int grp = tid + i * kThreads;
      xv[i] = make_uint4(0, 0, 0, 0);
      if (grp < G) {
        if constexpr (STEP) {
          const uint32_t* xw = reinterpret_cast<const uint32_t*>(x + grp);
          xv[i].x = __hip_atomic_load(xw + 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          xv[i].y = __hip_atomic_load(xw + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          xv[i].z = __hip_atomic_load(xw + 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          xv[i].w = __hip_atomic_load(xw + 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        } else {
          xv[i] = x[grp];
        }
      }
    }
  };
  if constexpr (!STEP) load_x();

  // 2. code loads for the first kAhead items (rows past the end repeat the
  // last row; their sums are never stored).
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
    const bool past = j >= nks;  // (wave-uniform)
    const int jj = past ? (nks > 0 ? nks - 1 : 0) : j;
    const uint32_t ks_off = (uint32_t)(wave + jj * kWaves) * 64u + slot_off;  // in a row-major row
    const uint32_t off = (uint32_t)(wave + jj * kWaves) * k_stride + slot_off;
    if constexpr (VEC) {
      const uint32_t o = (uint32_t)row_off[rb] + (ks_off < k_limit ? off : 0u);
      // A load past the wave's last K-slice only keeps the count of loads in
      // flight exact; its value is never used.  It reads the codebook, which
      // every workgroup has just read and L2 holds, not the last K-slice
      // again: that line has been consumed by then, and after a nontemporal
      // read L2 may no longer hold it (8192x28672: 15 % more HBM reads).
      const uint8_t* src =
          past ? reinterpret_cast<const uint8_t*>(cb) + (uint32_t)lane * 16u : wg_codes + o;
      const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src));
      w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
    } else {
      load_codes_bytes<8>(wg_codes + row_off[rb], pitch, off, w);
    }
  };
  uint32_t ring[D][RB][4];
#pragma unroll
  for (int i = 0; i < kAhead; ++i) issue_rb(i / RB, i % RB, ring[i / RB][i % RB]);

  // (the step kernel: codebooks to LDS while waiting, then x)
  auto stage_cb = [&]() {
    constexpr bool kPair = COPIES == 8 && M == 2;
    if (tid < M * 256) {
#pragma unroll
      for (int k = 0; k < COPIES; ++k) {
        const int c = (k + lane) % COPIES;
        cb_lds[kPair ? (tid & 255) * 16 + (tid >> 8) * 8 + c : tid * COPIES + c] = cbv;
      }
    }
  };
  if constexpr (STEP) {
    stage_cb();
    if (!wait()) return false;
    load_x();
  }

  // 3. stage codebook copies and x.  Eight copies of two codebooks (x too
  // large for sixteen) are interleaved per codeword: entry e holds the 8
  // copies of codebook 0, then the 8 of codebook 1 (256 bytes, every 16-byte
  // bank group once).  Lanes 8-15 of each 16-lane group then gather the
  // other code of the group (same x, other codebook) in the same
  // instruction, so the 16 lanes of one LDS pass read 16 different bank
  // groups; each row still gets both codebooks over the pair of MFMAs.
  constexpr bool kPairCb = COPIES == 8 && M == 2;
  if constexpr (!STEP) stage_cb();
#pragma unroll
  for (int i = 0; i < C::kXL; ++i) {
    const int grp = tid + i * kThreads;
    if (grp < xg) x_lds[grp] = xv[i];
  }
  __syncthreads();  // (no zeroing of the partials: every wave writes all of its slots)

  // 4. K-slices of this wave.
  const uint32_t copy_off = (uint32_t)(lane % COPIES) * 16u;
  const uint32_t cb_base = (uint32_t)(uintptr_t)cb_lds;
  uint32_t base_m[M];
#pragma unroll
  for (int m = 0; m < M; ++m) base_m[m] = cb_base + ((uint32_t)m << 16) + copy_off;
  // interleaved layout: address (code * 16 + m * 8 + copy) * 16, with m and
  // the code byte (t ^ flip) flipped on lanes 8-15
  const uint32_t flip = (uint32_t)(r16 >> 3);
  uint32_t pbase[2], psel[4];
#pragma unroll
  for (int tm = 0; tm < 2; ++tm) pbase[tm] = cb_base + ((((uint32_t)tm ^ flip) * 8u + (uint32_t)(lane % 8)) * 16u);
#pragma unroll
  for (int k = 0; k < 4; ++k) psel[k] = 0x0C020000u | ((4u + ((uint32_t)k ^ flip)) << 8);
  auto gaddr = [&](uint32_t word, int t) -> uint32_t {
    if constexpr (kPairCb) return __builtin_amdgcn_perm(word, pbase[t % 2], psel[t % 4]);
    return cw_addr<M, COPIES>(word, t % 4, base_m[t % M], copy_off + cb_base, t % M);
  };
  {
    f4_t acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = f4_t{0.f, 0.f, 0.f, 0.f};
    f4_t acc_odd = {0.f, 0.f, 0.f, 0.f};  // second chain of an unpaired last block
    uint4 xr[kXS];
#pragma unroll
    for (int s2 = 0; s2 < kXS; ++s2) xr[s2] = make_uint4(0, 0, 0, 0);

    // One ring period: D K-slices starting at j0.  Consuming an item loads
    // the item kAhead places later.  ISSUE: 2 = every such item exists (the
    // main loop), 1 = load it if it exists, 0 = the last period (only items
    // inside this period remain).  In the main loop every load is
    // unconditional, so the wait before each use counts exactly the loads
    // issued after it.
    auto period = [&](int j0, auto issue) {
      constexpr int kIssue = decltype(issue)::value;
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int j = j0 + d;
        const bool live = j < nks;
        if (live) {
          const int ks = wave + j * kWaves;
          if (r16 == 0) {
            const uint4* xs = x_lds + (((uint32_t)ks * C::kKS + (uint32_t)slot * C::kCPL) / M);
#pragma unroll
            for (int s2 = 0; s2 < kXS; ++s2) xr[s2] = xs[s2];
          }
        }
        // Row blocks two at a time, their MFMAs interleaved so that two
        // accumulation chains are in flight (a lone block alternates two
        // accumulators).  Blocks past the workgroup's last row read the codes
        // of its last row (their sums are never stored), so the loop has no
        // data-dependent branches.
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
                av[u] = lds_load16(gaddr(ring[d][rb][t / 4], t));
                if (pair) bv[u] = lds_load16(gaddr(ring[d][pair ? rb + 1 : rb][t / 4], t));
              }
              // All the step's gathers go out before its first MFMA.  Left
              // alone, the scheduler pairs each gather with its MFMA, so every
              // MFMA waits a full LDS latency.
              if constexpr (kPinGathers) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int u = 0; u < kStep; ++u) {
                const int t = t0 + u;
                const h8_t xh = __builtin_bit_cast(h8_t, xr[t / M]);
                if (pair) {
                  acc[rb] =
                      __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[u]), xh, acc[rb], 0, 0, 0);
                  acc[pair ? rb + 1 : rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                      __builtin_bit_cast(h8_t, bv[u]), xh, acc[pair ? rb + 1 : rb], 0, 0, 0);
                } else {
                  f4_t& a = (u % 2 == 0) ? acc[rb] : acc_odd;
                  a = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[u]), xh, a, 0, 0, 0);
                }
              }
            }
          }
#pragma unroll
          for (int q = 0; q < (pair ? 2 : 1); ++q) {
            const int target = d * RB + rb + q + kAhead;  // item position relative to K-slice j0
            const int jt = j0 + target / RB;
            // (target is a compile-time constant here, so only ISSUE == 1
            // leaves a run-time test; a target inside the last period is
            // loaded even if past the wave's end: issue_rb repeats the last
            // K-slice.)
            if (kIssue == 2 || (kIssue == 1 && jt < nks) || (kIssue == 0 && target < kSlots))
              issue_rb(jt, target % RB, ring[(target % kSlots) / RB][target % RB]);
          }
          // Keep the loads here: the scheduler would otherwise sink them
          // towards their use, leaving the HBM latency exposed.
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    };
    int j0 = 0;
    for (; j0 + 2 * D <= nks; j0 += D) period(j0, IntC<2>{});
    if (j0 + D < nks) {
      period(j0, IntC<1>{});
      j0 += D;
    }
    if (j0 < nks) period(j0, IntC<0>{});
    if constexpr (RB % 2 == 1) acc[RB - 1] += acc_odd;
    if (r16 == 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int e = 0; e < 4; ++e) part[(rb * kWaves + wave) * 16 + 4 * slot + e] = acc[rb][e];
    }
  }
  __syncthreads();

  // 5. fixed-order sum over waves, scale, round, store.
  if (tid < rows) {
    const int rb = tid / 16, rr = tid % 16;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += part[(rb * kWaves + w) * 16 + rr];
    const uint16_t out = f2h(h2f(sc) * s);
    if constexpr (STEP)
      __hip_atomic_store(bt.p[p].y + row0 + tid, out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    else
      bt.p[p].y[row0 + tid] = out;
  }
  return true;
}


template <int M, int COPIES, int RB, int D, bool VEC>
__global__ __launch_bounds__(kThreads) void k_gemv_ks(const GemvBatch bt) {
  ks_body<M, COPIES, RB, D, VEC, false>(bt, (int)blockIdx.x, [] { return true; });
}

// 1x16 with the codebook in LDS, one 128 KiB chunk (8192 codewords) at a
// time.  The 1 MiB codebook does not fit in LDS, and 16-byte gathers from L2
// run at well under one per clock per CU, so instead the workgroup makes one
// pass over its codes per chunk (8 passes).  A code outside the current chunk
// is sent to a zero codeword that follows the chunk in LDS, so every pass runs
// the same MFMAs and each code adds its product in exactly one pass.  The
// codes themselves are loaded from HBM once: a wave owns NKS K-slices of the
// workgroup's RB row blocks (at most 8 items, 32 registers) and keeps them in
// registers for all passes.  The next chunk is loaded into registers while the
// current one is in use, then written to LDS between passes.
constexpr int kCbChunk = 8192;                  // codewords per LDS chunk
constexpr int cb_passes(int B) { return (1 << B) / kCbChunk; }  // chunks of a 2^B codebook (B >= 13)
constexpr int kCbStage = kCbChunk / kThreads;   // 16-byte chunk loads per thread

// LDS byte addresses of the two codewords of a 32-bit code word in the chunk
// starting at code `first` (both halves hold `first`): a code outside the
// chunk gives the zero codeword at entry kCbChunk.  Packed 16-bit arithmetic
// wraps modulo 2^16, so (code - first) lands in [0, kCbChunk) exactly for the
// codes of the chunk and above it otherwise.
template <int B>
__device__ __forceinline__ void cb_chunk_addr(uint32_t word, uint32_t first2, uint32_t base, uint32_t& a0,
                                              uint32_t& a1) {
  typedef uint16_t u16x2_t __attribute__((ext_vector_type(2)));
  if constexpr (B < 16) word &= code_mask(B) * 0x10001u;
  u16x2_t t = __builtin_bit_cast(u16x2_t, word) - __builtin_bit_cast(u16x2_t, first2);
  t = __builtin_elementwise_min(t, (u16x2_t){(uint16_t)kCbChunk, (uint16_t)kCbChunk});
  const uint32_t tw = __builtin_bit_cast(uint32_t, t);
  // base + 16 * half, one v_mad_u32_u16 per code (op_sel picks the high half;
  // the compiler spends three instructions on each otherwise)
  asm("v_mad_u32_u16 %0, %1, 16, %2" : "=v"(a0) : "v"(tw), "v"(base));
  asm("v_mad_u32_u16 %0, %1, 16, %2 op_sel:[1,0,0,0]" : "=v"(a1) : "v"(tw), "v"(base));
}

// PACKED (B = 15): the codes arrive as row bit strings; each item's 8 codes
// per lane are unpacked once into the 16-bit pairs the passes read.
template <int NKS, int RB, int B, bool PACKED = false>
__global__ __launch_bounds__(kThreads) void k_gemv_cb(const GemvBatch bt) {
  static_assert(!PACKED || B == 15, "packed codes: 15 bits");
  constexpr int kCbPasses = cb_passes(B);
  static_assert(kCbPasses * kCbChunk == (1 << B), "whole chunks");
  constexpr int kItems = NKS * RB;
  constexpr int kXG = NKS * kWaves * 32;        // x groups staged (K-slices of 32 groups), zero past G
  constexpr int kXL = (kXG + kThreads - 1) / kThreads;
  constexpr int kStep = 2;                      // codewords gathered per block before their MFMAs
  static_assert(kItems <= 8, "code items are held in registers");
  extern __shared__ uint4 lds[];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int r16 = lane & 15;
  const int slot = lane >> 4;

  int p = 0;
  while (p + 1 < bt.count && bt.p[p + 1].wg_begin <= (int)blockIdx.x) ++p;
  const uint4* __restrict__ cb = bt.p[p].cb;
  const uint4* __restrict__ x = bt.p[p].x;
  const int32_t rows_per_wg = bt.p[p].rows_per_wg;
  const int32_t row0 = ((int32_t)blockIdx.x - bt.p[p].wg_begin) * rows_per_wg;
  int32_t rows = bt.p[p].d_out - row0;
  if (rows > rows_per_wg) rows = rows_per_wg;
  const int32_t G = bt.p[p].G;
  const uint32_t pitch = (uint32_t)G * 2u;  // code bytes per row (unpacked)
  const uint32_t pwords = (uint32_t)bt.p[p].pwords;  // packed: 32-bit words per row
  const uint8_t* __restrict__ wg_codes = bt.p[p].codes + (size_t)row0 * (PACKED ? pwords * 4u : pitch);

  uint4* x_lds = lds + kCbChunk + 1;  // after the chunk and its zero codeword

  // 1. loads, in the order they are needed: chunk 0, x, the codes, the scale.
  // (16-byte values as vector types: a uint4 copy from global goes through
  // private memory)
  const u32x4_t* __restrict__ cbv = reinterpret_cast<const u32x4_t*>(cb);
  u32x4_t stage[kCbStage];
#pragma unroll
  for (int k = 0; k < kCbStage; ++k) stage[k] = cbv[tid + k * kThreads];
  u32x4_t xv[kXL];
#pragma unroll
  for (int i = 0; i < kXL; ++i) {
    const int grp = tid + i * kThreads;
    xv[i] = u32x4_t{0u, 0u, 0u, 0u};
    if (grp < G) xv[i] = reinterpret_cast<const u32x4_t*>(x)[grp];
  }
  // Item (j, rb): K-slice wave + 16 j of row block rb.  A slot past the row
  // end (or a whole K-slice past it) reads the row's first bytes instead; x is
  // zero there.  Rows past the workgroup's last repeat that row; their sums
  // are never stored.
  uint32_t cw[kItems][4];
  uint32_t raw[PACKED ? kItems : 1][5];  // packed: the 5 words that hold a slot's 120 bits
#pragma unroll
  for (int j = 0; j < NKS; ++j) {
    const uint32_t off = (uint32_t)(wave + j * kWaves) * 64u + (uint32_t)slot * 16u;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int row = rb * 16 + r16 < rows ? rb * 16 + r16 : rows - 1;
      if constexpr (PACKED) {
        // words past the row's last are clamped to it (x is zero there)
        const uint32_t* rw = reinterpret_cast<const uint32_t*>(wg_codes) + (size_t)row * pwords;
        const uint32_t w0 = ((uint32_t)((wave + j * kWaves) * 4 + slot) * 120u) >> 5;
        uint32_t* r = raw[j * RB + rb];
        if (w0 + 5u <= pwords) {
          const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4a4_t*>(rw + w0));
          r[0] = v[0]; r[1] = v[1]; r[2] = v[2]; r[3] = v[3];
          r[4] = __builtin_nontemporal_load(rw + w0 + 4);
        } else {
#pragma unroll
          for (int i = 0; i < 5; ++i) r[i] = __builtin_nontemporal_load(rw + (w0 + i < pwords ? w0 + i : pwords - 1u));
        }
      } else {
        const uint32_t o = (uint32_t)row * pitch + (off < pitch ? off : 0u);
        const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(wg_codes + o));
#pragma unroll
        for (int e = 0; e < 4; ++e) cw[j * RB + rb][e] = v[e];
      }
    }
  }
  const uint16_t sc = bt.p[p].scales[row0 + (tid < rows ? tid : rows - 1)];

  // 2. chunk 0, its zero codeword and x into LDS.
  u32x4_t* lds_v = reinterpret_cast<u32x4_t*>(lds);
#pragma unroll
  for (int k = 0; k < kCbStage; ++k) lds_v[tid + k * kThreads] = stage[k];
  if (tid == 0) lds_v[kCbChunk] = u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < kXL; ++i) {
    const int grp = tid + i * kThreads;
    if (grp < kXG) reinterpret_cast<u32x4_t*>(x_lds)[grp] = xv[i];
  }
  __syncthreads();

  // 3. one pass per chunk.
  const uint32_t base = (uint32_t)(uintptr_t)lds;
  f4_t acc[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) acc[rb] = f4_t{0.f, 0.f, 0.f, 0.f};
  f4_t acc_odd = {0.f, 0.f, 0.f, 0.f};  // second chain of an unpaired last block
  for (int c = 0; c < kCbPasses; ++c) {
    if (c + 1 < kCbPasses) {
#pragma unroll
      for (int k = 0; k < kCbStage; ++k) stage[k] = cbv[(c + 1) * kCbChunk + tid + k * kThreads];
    }
    if constexpr (PACKED) {
      // unpack the codes once, after the next chunk's loads are issued (so
      // that those need not wait for the codes); a slot's bits start
      // 24 * slot % 32 bits into its first word
      if (c == 0) {
        const uint32_t sh = (24u * (uint32_t)slot) & 31u;
#pragma unroll
        for (int it = 0; it < kItems; ++it) {
          uint32_t w[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) w[i] = __builtin_amdgcn_alignbit(raw[it][i + 1], raw[it][i], sh);
          uint32_t code[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const int b = t * 15, wd = b >> 5, of = b & 31;
            uint32_t v = w[wd] >> of;
            if (of + 15 > 32) v |= w[wd + 1] << (32 - of);
            code[t] = v & 0x7FFFu;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) cw[it][e] = code[2 * e] | (code[2 * e + 1] << 16);
        }
      }
    }
    const uint32_t first2 = (uint32_t)(c * kCbChunk) * 0x10001u;
#pragma unroll
    for (int j = 0; j < NKS; ++j) {
      // x group of code t of this lane's slot: K-slice * 32 + slot * 8 + t
      const uint4* xs = x_lds + (wave + j * kWaves) * 32 + slot * 8;
      // x for the whole slice where the registers allow, else per step
      constexpr int kXS = RB <= 2 ? 8 : kStep;
      uint4 xr[kXS];
#pragma unroll
      for (int t0 = 0; t0 < 8; t0 += kStep) {
        if (t0 % kXS == 0) {
#pragma unroll
          for (int u = 0; u < kXS; ++u) xr[u] = xs[t0 + u];
        }
        uint4 xb[kStep];
#pragma unroll
        for (int u = 0; u < kStep; ++u) xb[u] = xr[(t0 + u) % kXS];
#pragma unroll
        for (int rb = 0; rb < RB; rb += 2) {
          const bool pair = rb + 1 < RB;
          uint4 av[kStep], bv[kStep];
#pragma unroll
          for (int u = 0; u < kStep; u += 2) {
            const int t = t0 + u;
            uint32_t a0, a1;
            cb_chunk_addr<B>(cw[j * RB + rb][t / 2], first2, base, a0, a1);
            av[u] = lds_load16(a0);
            av[u + 1] = lds_load16(a1);
            if (pair) {
              cb_chunk_addr<B>(cw[j * RB + (pair ? rb + 1 : rb)][t / 2], first2, base, a0, a1);
              bv[u] = lds_load16(a0);
              bv[u + 1] = lds_load16(a1);
            }
          }
          // all the step's gathers before its first MFMA
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int u = 0; u < kStep; ++u) {
            const h8_t xh = __builtin_bit_cast(h8_t, xb[u]);
            if (pair) {
              acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[u]), xh, acc[rb], 0, 0, 0);
              acc[pair ? rb + 1 : rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                  __builtin_bit_cast(h8_t, bv[u]), xh, acc[pair ? rb + 1 : rb], 0, 0, 0);
            } else {
              f4_t& a = (u % 2 == 0) ? acc[rb] : acc_odd;
              a = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, av[u]), xh, a, 0, 0, 0);
            }
          }
        }
      }
    }
    __syncthreads();  // every wave is done with chunk c
    if (c + 1 < kCbPasses) {
#pragma unroll
      for (int k = 0; k < kCbStage; ++k) lds_v[tid + k * kThreads] = stage[k];
      __syncthreads();
    }
  }
  if constexpr (RB % 2 == 1) acc[RB - 1] += acc_odd;

  // 4. per-wave partials (in the chunk's space, no longer read), then the
  // fixed-order sum over waves, scale, round, store.
  float* part = reinterpret_cast<float*>(lds);
  if (r16 == 0) {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int e = 0; e < 4; ++e) part[(rb * kWaves + wave) * 16 + 4 * slot + e] = acc[rb][e];
  }
  __syncthreads();
  if (tid < rows) {
    const int rb = tid / 16, rr = tid % 16;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += part[(rb * kWaves + w) * 16 + rr];
    bt.p[p].y[row0 + tid] = f2h(h2f(sc) * s);
  }
}

template <int NKS, int RB, int B, bool PACKED>
hipError_t launch_cb(const GemvBatch& bt, hipStream_t s) {
  auto kern = k_gemv_cb<NKS, RB, B, PACKED>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), 160 * 1024);
    if (e != hipSuccess) return e;
  }
  const size_t lds = (size_t)(kCbChunk + 1 + NKS * kWaves * 32) * 16;
  hipLaunchKernelGGL(kern, dim3(bt.total_wgs), dim3(kThreads), lds, s, bt);
  return hipGetLastError();
}

// K-slices per wave (NKS) and row blocks per workgroup the chunked 1x16
// kernel supports: the code items (NKS * RB <= 8) stay in registers, and x
// (NKS * 8 KiB) fits next to the 128 KiB chunk.
constexpr int kCbMaxNks = 3;
constexpr int cb_rb_cap(int nks) { return nks == 1 ? 6 : (nks == 2 ? 4 : 2); }

template <int B, bool PACKED = false>
hipError_t launch_cb_shape(const GemvBatch& bt, int nks, int rb, hipStream_t s) {
  switch (nks * 8 + rb) {
    case 8 + 1: return launch_cb<1, 1, B, PACKED>(bt, s);
    case 8 + 2: return launch_cb<1, 2, B, PACKED>(bt, s);
    case 8 + 3: return launch_cb<1, 3, B, PACKED>(bt, s);
    case 8 + 4: return launch_cb<1, 4, B, PACKED>(bt, s);
    case 8 + 5: return launch_cb<1, 5, B, PACKED>(bt, s);
    case 8 + 6: return launch_cb<1, 6, B, PACKED>(bt, s);
    case 16 + 1: return launch_cb<2, 1, B, PACKED>(bt, s);
    case 16 + 2: return launch_cb<2, 2, B, PACKED>(bt, s);
    case 16 + 3: return launch_cb<2, 3, B, PACKED>(bt, s);
    case 16 + 4: return launch_cb<2, 4, B, PACKED>(bt, s);
    case 24 + 1: return launch_cb<3, 1, B, PACKED>(bt, s);
    case 24 + 2: return launch_cb<3, 2, B, PACKED>(bt, s);
  }
  return hipErrorInvalidValue;
}

template <int M, int COPIES, int RB, int D, bool VEC>
hipError_t launch_ks(const GemvBatch& bt, size_t lds_bytes, hipStream_t s) {
  auto kern = k_gemv_ks<M, COPIES, RB, D, VEC>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), 160 * 1024);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3(bt.total_wgs), dim3(kThreads), lds_bytes, s, bt);
  return hipGetLastError();
}

// Row blocks per workgroup the K-slice kernel keeps in registers without
// spilling (1024 threads: 128 VGPRs per lane); M = 1 holds 16 x slices.
constexpr int ks_rb_cap(int M) { return M == 1 ? 2 : 7; }

// Ring depth in K-slices: up to eight single blocks in flight per wave, no
// more K-slices than a wave owns (extra slots would only repeat its last
// one), and for paired blocks two K-slices at most: with two or three items
// requested ahead a deeper ring only moves K-slices out of the loop's
// unconditional part (Llama-2-70B down, two blocks, seven K-slices per wave:
// tiled step 4.858-4.869 ms with four, 4.837-4.852 with two, same box).
// Three blocks (three items ahead) fill a one-K-slice ring (q/k/v, two
// K-slices per wave: 4.824-4.833 -> 4.803-4.814 ms); two blocks keep two
// K-slices so that both items of the next pair have slots of their own.
template <int M, int COPIES, int RB, bool VEC>
hipError_t launch_ks_d(const GemvBatch& bt, int nks, size_t lds_bytes, hipStream_t s) {
  constexpr int kDMax = (RB >= 5 || RB == 3) ? 1 : (RB >= 2 ? 2 : 8);
  constexpr int kDMin = RB == 2 ? 2 : 1;
  if constexpr (kDMax >= 8) {
    if (nks >= 8) return launch_ks<M, COPIES, RB, 8, VEC>(bt, lds_bytes, s);
  }
  if constexpr (kDMax >= 4) {
    if (nks >= 4) return launch_ks<M, COPIES, RB, 4, VEC>(bt, lds_bytes, s);
  }
  if constexpr (kDMax >= 2) {
    if (nks >= 2 || kDMin == 2) return launch_ks<M, COPIES, RB, 2, VEC>(bt, lds_bytes, s);
  }
  return launch_ks<M, COPIES, RB, kDMin, VEC>(bt, lds_bytes, s);
}

template <int M, int COPIES, bool VEC>
hipError_t launch_ks_rb(const GemvBatch& bt, int rb, int nks, size_t lds_bytes, hipStream_t s) {
  switch (rb) {
    case 1: return launch_ks_d<M, COPIES, 1, VEC>(bt, nks, lds_bytes, s);
    case 2: return launch_ks_d<M, COPIES, 2, VEC>(bt, nks, lds_bytes, s);
  }
  if constexpr (ks_rb_cap(M) >= 7) {
    switch (rb) {
      case 3: return launch_ks_d<M, COPIES, 3, VEC>(bt, nks, lds_bytes, s);
      case 4: return launch_ks_d<M, COPIES, 4, VEC>(bt, nks, lds_bytes, s);
      case 5: return launch_ks_d<M, COPIES, 5, VEC>(bt, nks, lds_bytes, s);
      case 6: return launch_ks_d<M, COPIES, 6, VEC>(bt, nks, lds_bytes, s);
      case 7: return launch_ks_d<M, COPIES, 7, VEC>(bt, nks, lds_bytes, s);
    }
  }
  return hipErrorInvalidValue;
}

template <int M, int B, int COPIES, int PF, bool VEC, bool PACKED = false>
hipError_t launch_pf(const GemvBatch& bt, size_t lds_bytes, hipStream_t s) {
  auto kern = k_gemv_mfma<M, B, COPIES, PF, VEC, PACKED>;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(kern), 160 * 1024);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3(bt.total_wgs), dim3(kThreads), lds_bytes, s, bt);
  return hipGetLastError();
}

template <int M, int B, int COPIES, bool VEC, bool PACKED = false>
hipError_t launch_copies(const GemvBatch& bt, int pf, size_t lds_bytes, hipStream_t s) {
  switch (pf) {
    case 1: return launch_pf<M, B, COPIES, 1, VEC, PACKED>(bt, lds_bytes, s);
    case 2: return launch_pf<M, B, COPIES, 2, VEC, PACKED>(bt, lds_bytes, s);
    case 4: return launch_pf<M, B, COPIES, 4, VEC, PACKED>(bt, lds_bytes, s);
  }
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------- decode step
//
// k_gemv_step runs a list of levels (each a grouped 2x8 product, as one
// k_gemv_ks launch would) on a resident grid of one workgroup per CU.
// Level l + 1 may read what level l wrote, so a workgroup reads level l + 1's
// x only after every workgroup has finished level l: a counter that each
// workgroup bumps after its last product of a level (its y stores completed
// first), polled by one thread.  Everything a product reads apart from x is
// loaded before that wait, so a workgroup that finishes a level early streams
// the next level's first codes while the slowest ones finish.
//
// Every wait is bounded: after `spin` polls it sets the error flag and the
// workgroup stops; a workgroup that sees the flag stops too, so the grid
// always drains.  The last workgroup to leave resets the counters.

// (M = 2, 8-bit codes, 16-byte code rows) body instantiations: (id, copies,
// row blocks, ring depth)
#define AQLM_STEP_VARIANTS(X)                                                                    \
  X(0, 16, 1, 1) X(1, 16, 1, 2) X(2, 16, 1, 4) X(3, 16, 1, 8) X(4, 16, 2, 2) X(6, 16, 3, 1)       \
  X(7, 16, 4, 1) X(8, 16, 4, 2) X(9, 16, 5, 1) X(10, 16, 6, 1) X(11, 16, 7, 1) X(12, 8, 1, 1)      \
  X(13, 8, 1, 2) X(14, 8, 1, 4) X(15, 8, 1, 8) X(16, 8, 2, 2)

int step_variant(int M, int copies, int rb, int d, bool vec) {
  if (M != 2 || !vec) return -1;
#define AQLM_STEP_FIND(ID, C, R, D) \
  if (copies == C && rb == R && d == D) return ID;
  AQLM_STEP_VARIANTS(AQLM_STEP_FIND)
#undef AQLM_STEP_FIND
  return -1;
}

// Thread 0 polls until `target` level signals have arrived; the verdict is
// shared through LDS.  False: timed out here or elsewhere (error flag).
// sync words: [0] level signals, [1] error flag, [2] workgroups that left;
// one 64-bit load reads the counter and the flag together.
__device__ bool step_wait(uint32_t* sync, uint32_t target, uint32_t spin, uint32_t* verdict) {
  if (threadIdx.x == 0) {
    uint32_t ok = 0;
    for (uint32_t it = 0;; ++it) {
      const uint64_t w =
          __hip_atomic_load(reinterpret_cast<uint64_t*>(sync), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      // (the flag first: once any wait has given up, no workgroup starts
      // another level)
      if ((uint32_t)(w >> 32) != 0) break;
      if ((uint32_t)w >= target) {
        ok = 1;
        break;
      }
      if (it >= spin) {
        __hip_atomic_store(sync + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        break;
      }
    }
    *verdict = ok;
  }
  __syncthreads();
  const bool ok = *verdict != 0;
  __syncthreads();
  return ok;
}

// This workgroup is done with the level: its y stores have completed (they
// are system-scope, written through to memory) before the counter moves.
__device__ void step_signal(uint32_t* sync) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(sync, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// (The wait verdict lives in dynamic LDS right after the largest level's
// region: a static __shared__ variable next to the dynamic array lost the
// last word of the partial sums.)
__global__ __launch_bounds__(kThreads) void k_gemv_step(const StepLevel* __restrict__ levels, int32_t nlev,
                                                        uint32_t* sync, uint32_t spin, int32_t lds_bytes) {
  extern __shared__ uint4 lds_all[];
  uint32_t& verdict = *reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(lds_all) + lds_bytes);
  const int nwg = (int)gridDim.x;
  bool ok = true;
  for (int l = 0; l < nlev && ok; ++l) {
    const StepLevel& L = levels[l];
    bool waited = l == 0;
    // every workgroup waits for level l - 1 before it signals level l, so
    // the counter reaches (l + 1) * nwg only once all have finished level l
    auto wait = [&]() -> bool {
      if (waited) return true;
      waited = true;
      return step_wait(sync, (uint32_t)l * (uint32_t)nwg, spin, &verdict);
    };
    const int variant = L.variant;
    const int total = L.bt.total_wgs;
    for (int v = (int)blockIdx.x; ok && v < total; v += nwg) {
      switch (variant) {
#define AQLM_STEP_CASE(ID, C, R, D) \
  case ID: ok = ks_body<2, C, R, D, true, true>(L.bt, v, wait); break;
        AQLM_STEP_VARIANTS(AQLM_STEP_CASE)
#undef AQLM_STEP_CASE
      }
    }
    if (ok) ok = wait();
    if (ok) step_signal(sync);
  }
  // leave: the last workgroup out resets the counters (every other one has
  // stopped reading them)
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t out = __hip_atomic_fetch_add(sync + 2, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    if (out == (uint32_t)nwg - 1u) {
      __hip_atomic_store(sync, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      __hip_atomic_store(sync + 2, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
}

}  // namespace

bool gemv_mfma_supported(int M, int B) {
  if (B > 8) return format_supported(M, B);
  return B == 8 && (M == 1 || M == 2 || M == 4);
}

// Whether x (staged whole in LDS, at most kXL groups per thread) and the
// partial sums fit, next to at least one codebook copy for 8-bit codes.
bool gemv_mfma_fits(const Layer* Ls, int count) {
  for (int i = 0; i < count; ++i) {
    const Layer& L = Ls[i];
    const int kCPL = (L.B == 8) ? 16 : 8, kKS = 4 * kCPL, xl = (L.B == 8) ? 4 : 8;
    const int64_t KS = ((int64_t)L.G * L.M * code_bytes(L.B) + 63) / 64;
    const int64_t xg = KS * (kKS / L.M);
    if (xg > (int64_t)xl * kThreads) return false;
    const size_t need = (size_t)xg * 16 + (size_t)kMaxRB * kWaves * 16 * 4 + (L.B == 8 ? (size_t)L.M * 256 * 16 : 0);
    if (need > 160 * 1024) return false;
  }
  return true;
}

// Deal workgroups to problems, pick rows per workgroup and items per wave,
// size LDS, and launch.  All problems share (M, B) and the code-pitch
// alignment class.
// Ring depth k_gemv_ks runs for RB row blocks and nks K-slices per wave
// (launch_ks_d's choice).
int ks_ring_depth(int rb, int nks) {
  const int dmax = (rb >= 5 || rb == 3) ? 1 : (rb >= 2 ? 2 : 8);
  const int dmin = rb == 2 ? 2 : 1;
  if (dmax >= 8 && nks >= 8) return 8;
  if (dmax >= 4 && nks >= 4) return 4;
  if (dmax >= 2 && (nks >= 2 || dmin == 2)) return 2;
  return dmin;
}

// Plans (and, without `plan`, launches) a grouped product.  With `plan` (the
// decode-step planner, 2x8 only) nothing is launched: the workgroup split and
// the k_gemv_ks variant are recorded, with row blocks per workgroup capped at
// rb_cap_max (when > 0) and LDS at lds_limit.
hipError_t gemv_mfma_impl(const Layer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                          hipStream_t s, StepLevel* plan, int rb_cap_max, size_t lds_limit) {
  if (count < 1 || count > kMaxProblems) return hipErrorInvalidValue;
  const int M = Ls[0].M, B = Ls[0].B;
  const bool packed = Ls[0].packed;
  for (int i = 1; i < count; ++i)
    if (Ls[i].packed != packed || Ls[i].tiled != Ls[0].tiled) return hipErrorInvalidValue;
  // tiled codes: 8-bit, 16-byte aligned, read by k_gemv_ks alone
  if (Ls[0].tiled && (B != 8 || packed || plan || !Ls[0].vec_codes)) return hipErrorInvalidValue;
  const int kCPL = (B == 8) ? 16 : 8, kKS = 4 * kCPL;
  bool vec = true;
  double total_bytes = 0;
  for (int i = 0; i < count; ++i) {
    vec = vec && Ls[i].vec_codes;
    total_bytes += (double)Ls[i].d_out * Ls[i].G * M * code_bytes(B);
  }
  const int cus = num_cus();
  // One codebook of wide codes runs the chunked-codebook kernel where its
  // code items fit in registers and x next to the chunk (NKS K-slices per
  // wave).  Two codebooks gather from L2.
  int cb_nks = 0;
  if (B > 8 && M == 1 && vec) {
    for (int i = 0; i < count; ++i) {
      const int KS = (int)(((int64_t)Ls[i].G * 2 + 63) / 64);
      const int nks = (KS + kWaves - 1) / kWaves;
      if (nks > cb_nks) cb_nks = nks;
    }
    if (cb_nks > kCbMaxNks) cb_nks = 0;
    // Every workgroup streams the whole codebook through its CU (about 14 us
    // at the L2 bandwidth), which pays off only above roughly 28 KiB of codes
    // per CU; smaller launches gather from L2.
    if (total_bytes < 28.0 * 1024 * cus) cb_nks = 0;
  }
  // CUs per problem in proportion to its code bytes, at least one each, by
  // largest remainders so that the shares add up to the CU count: rounding
  // each share on its own could ask for more workgroups than CUs (Llama-2-70B
  // q/k/v: 205 + 26 + 26 = 257), and the one extra workgroup then ran after
  // all the others, doubling the launch.
  int want_of[kMaxProblems];
  {
    double rem[kMaxProblems];
    int sum = 0;
    for (int i = 0; i < count; ++i) {
      const double share = cus * ((double)Ls[i].d_out * Ls[i].G * M * code_bytes(B)) / total_bytes;
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
    // (the one-CU minimum of tiny problems can overshoot: take it back from
    // the largest shares)
    while (sum > cus) {
      int big = 0;
      for (int i = 1; i < count; ++i)
        if (want_of[i] > want_of[big]) big = i;
      if (want_of[big] <= 1) break;
      --want_of[big];
      --sum;
    }
  }
  GemvBatch bt{};
  bt.count = count;
  bt.tiled = Ls[0].tiled ? 1 : 0;
  int wg = 0, ni_max = 1, xg_max = 0, rb_max = 1, nks_min = 1 << 30;
  for (int i = 0; i < count; ++i) {
    const Layer& L = Ls[i];
    const int want = want_of[i];
    const int64_t cpr = (int64_t)L.G * M;
    const int KS = (int)((cpr + kKS - 1) / kKS);
    // At most rb_cap row blocks per workgroup (accumulator registers and
    // partial-sum space).  Larger layers run `rounds` workgroups per CU,
    // split evenly rather than leaving a short last round.
    int rb_cap = (B > 8) ? (cb_nks > 0 ? cb_rb_cap(cb_nks) : kMaxRB) : ks_rb_cap(M);
    if (rb_cap_max > 0 && rb_cap > rb_cap_max) rb_cap = rb_cap_max;
    const int blocks = (L.d_out + 15) / 16;
    const int rounds = (blocks + rb_cap * want - 1) / (rb_cap * want);
    const int rows_per_wg = (L.d_out + want * rounds - 1) / (want * rounds);
    const int nwg = (L.d_out + rows_per_wg - 1) / rows_per_wg;
    const int rb = (rows_per_wg + 15) / 16;
    const int ni = (rb * KS + kWaves - 1) / kWaves;
    GemvProblem& P = bt.p[i];
    P.codes = static_cast<const uint8_t*>(L.codes);
    P.cb = reinterpret_cast<const uint4*>(L.codebooks);
    P.scales = L.scales;
    P.x = reinterpret_cast<const uint4*>(xs[i]);
    P.y = ys[i];
    P.d_out = L.d_out;
    P.G = L.G;
    P.wg_begin = wg;
    P.rows_per_wg = rows_per_wg;
    P.pwords = packed ? packed_row_words(L.G, M, B) : 0;
    wg += nwg;
    if (ni > ni_max) ni_max = ni;
    const int xg = KS * (kKS / M);
    if (xg > xg_max) xg_max = xg;
    if (rb > rb_max) rb_max = rb;
    const int nks = (KS + kWaves - 1) / kWaves;  // K-slices of the busiest wave
    if (nks < nks_min) nks_min = nks;
  }
  bt.total_wgs = wg;
  bt.xg_max = xg_max;
  const int ni = ni_max <= 1 ? 1 : (ni_max == 2 ? 2 : 4);  // prefetch depth
  const int xl = (B == 8) ? 4 : 8;
  if (xg_max > xl * kThreads) return hipErrorInvalidValue;
  const size_t base = (size_t)xg_max * 16 + (size_t)rb_max * kWaves * 16 * 4;
  const size_t limit = lds_limit;
  if (plan && B != 8) return hipErrorInvalidValue;
  if (B > 8 && cb_nks > 0) {
    if (packed) return launch_cb_shape<15, true>(bt, cb_nks, rb_max, s);
    return B == 15 ? launch_cb_shape<15>(bt, cb_nks, rb_max, s) : launch_cb_shape<16>(bt, cb_nks, rb_max, s);
  }
  if (packed) {
    if (base > limit) return hipErrorInvalidValue;
    const size_t wide12 = (size_t)(2 << 12) * 16;
    if (M == 2 && B == 12 && base + wide12 <= limit)
      return launch_copies<2, 12, 1, true, true>(bt, ni, base + wide12, s);
    if (M == 2 && B == 12) return launch_copies<2, 12, 0, true, true>(bt, ni, base, s);
    if (M == 2 && B == 15) return launch_copies<2, 15, 0, true, true>(bt, ni, base, s);
    if (M == 1 && B == 15) return launch_copies<1, 15, 0, true, true>(bt, ni, base, s);
    return hipErrorInvalidValue;
  }
  if (B > 8) {
    if (base > limit) return hipErrorInvalidValue;
#define AQLM_GEMV_L2(MM, BB) \
  return vec ? launch_copies<MM, BB, 0, true>(bt, ni, base, s) : launch_copies<MM, BB, 0, false>(bt, ni, base, s);
    if (M == 1) {
      if (B == 15) AQLM_GEMV_L2(1, 15)
      AQLM_GEMV_L2(1, 16)
    }
    // two 4096-entry codebooks (128 KiB) fit in LDS next to x (d_in up to
    // about 12000) and the partials: gathered from there instead of L2
    const size_t wide12 = (size_t)(2 << 12) * 16;
    if (B == 12 && base + wide12 <= limit)
      return vec ? launch_copies<2, 12, 1, true>(bt, ni, base + wide12, s)
                 : launch_copies<2, 12, 1, false>(bt, ni, base + wide12, s);
    switch (B) {
      case 12: AQLM_GEMV_L2(2, 12)
      case 15: AQLM_GEMV_L2(2, 15)
      case 16: AQLM_GEMV_L2(2, 16)
    }
#undef AQLM_GEMV_L2
    return hipErrorInvalidValue;
  }
  // the most codebook copies that fit next to x and the partials
  const size_t per_copy = (size_t)M * 256 * 16;
  int copies = 16;
  while (copies > 1 && base + per_copy * copies > limit) copies /= 2;
  if (base + per_copy * copies > limit) return hipErrorInvalidValue;
  const size_t lds = base + per_copy * copies;
  if (plan) {
    plan->bt = bt;
    plan->variant = step_variant(M, copies, rb_max, ks_ring_depth(rb_max, nks_min), vec);
    plan->lds_bytes = (int32_t)lds;
    return plan->variant < 0 ? hipErrorInvalidValue : hipSuccess;
  }
#define AQLM_GEMV_COPIES(MM)                                                                     \
  switch (copies) {                                                                              \
    case 16: return vec ? launch_ks_rb<MM, 16, true>(bt, rb_max, nks_min, lds, s)                        \
                        : launch_ks_rb<MM, 16, false>(bt, rb_max, nks_min, lds, s);                      \
    case 8: return vec ? launch_ks_rb<MM, 8, true>(bt, rb_max, nks_min, lds, s)                          \
                       : launch_ks_rb<MM, 8, false>(bt, rb_max, nks_min, lds, s);                        \
    case 4: return vec ? launch_ks_rb<MM, 4, true>(bt, rb_max, nks_min, lds, s)                          \
                       : launch_ks_rb<MM, 4, false>(bt, rb_max, nks_min, lds, s);                        \
    default: return hipErrorInvalidValue;                                                        \
  }
  switch (M) {
    case 1: AQLM_GEMV_COPIES(1)
    case 2: AQLM_GEMV_COPIES(2)
    case 4: AQLM_GEMV_COPIES(4)
  }
#undef AQLM_GEMV_COPIES
  return hipErrorInvalidValue;
}

hipError_t launch_gemv_mfma(const Layer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                            hipStream_t s) {
  return gemv_mfma_impl(Ls, xs, ys, count, s, nullptr, 0, 160 * 1024);
}

hipError_t launch_step(const StepLevel* levels, int32_t nlev, int32_t grid, size_t lds, uint32_t* sync,
                       uint32_t spin, hipStream_t s) {
  if (nlev < 1 || grid < 1 || lds > kStepLdsLimit) return hipErrorInvalidValue;
  {
    const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(k_gemv_step), (int)kStepLdsLimit);
    if (e != hipSuccess) return e;
  }
  // cooperative: the runtime refuses the launch unless every workgroup can
  // be resident at once, which the level barrier needs
  int32_t lds_bytes = (int32_t)lds;
  void* args[] = {(void*)&levels, (void*)&nlev, (void*)&sync, (void*)&spin, (void*)&lds_bytes};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(k_gemv_step), dim3(grid), dim3(kThreads), args,
                                    (unsigned)lds + 16u, s);
}

}  // namespace aqlm
