// Batch-1 product over chunk-sorted wide codes (layout in sorted.h).
//
// Why a second storage: a 2^16-entry codebook is 1 MiB, so with codes in row
// order every code gathers its 16-byte codeword from L2 (one line fill per
// codeword) or every workgroup streams the whole codebook through LDS.  With
// the codes of each 16-row block grouped by 8192-codeword chunk, a workgroup
// stages ONE chunk (128 KiB) in LDS and serves every code of that chunk in
// its rows with one LDS gather.
//
// k_gemv_sorted: workgroup (c, r) = class c, row range r (K * R workgroups,
// at most one per CU; the workgroups of a class share an XCD when K = 8).
//   - stage chunk c of its codebook (plus a zero codeword) and, when it fits,
//     x (plus a zero slice) in LDS;
//   - its blocks' lists of class c are cut into P parts; parts are dealt to
//     the 16 waves; a wave reads 16 steps of entries ahead (64 lanes x 4 B per
//     step, coalesced), and for every entry gathers the codeword and the x
//     slice and adds their inner product (4 v_dot2_f32_f16) to its lane's sum;
//     lanes i, i+16, i+32, i+48 of a step belong to row i of the block, so at
//     the end of a part four lanes are added and written to LDS;
//   - the parts of each row are added in order and the row's class partial
//     is written to the workspace; the last of the K workgroups of a row range
//     (a counter per range) adds the K partials in class order, multiplies by
//     the scale and rounds once to fp16, then resets the counter.
// Every sum has a fixed order: results are deterministic.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "common.h"
#include "launch.h"
#include "lds_sync.h"
#include "sorted.h"

namespace aqlm {

// ------------------------------------------------------------------ host sort

namespace {

struct CodeReader {
  const void* codes;
  bool packed;
  int64_t G;
  int32_t M;
  int32_t B;
  int64_t row_words;
  uint32_t at(int64_t row, int64_t j, int m) const {
    const uint32_t mask = (1u << B) - 1u;
    if (!packed) return static_cast<const uint16_t*>(codes)[(row * G + j) * M + m] & mask;
    const uint32_t* w = static_cast<const uint32_t*>(codes) + row * row_words;
    const uint64_t bit = (uint64_t)(j * M + m) * (uint64_t)B;
    const uint64_t wi = bit >> 5;
    const unsigned sh = (unsigned)(bit & 31u);
    uint64_t v = w[wi];
    if (sh + (unsigned)B > 32u) v |= (uint64_t)w[wi + 1] << 32;
    return (uint32_t)(v >> sh) & mask;
  }
  int cls(uint32_t v, int m) const { return (m << (B - kChunkBits)) + (int)(v >> kChunkBits); }
};

CodeReader reader(const void* codes, bool packed, int32_t d_in, int32_t M, int32_t B) {
  const int64_t G = d_in / 8;
  return CodeReader{codes, packed, G, M, B, (G * M * B + 31) / 32};
}

// Runs fn(b_begin, b_end) over the row blocks [0, nb) split among host
// threads (blocks are independent; each thread writes only its blocks).
template <class F>
void for_blocks(int64_t nb, const F& fn) {
  const unsigned hw = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  const int64_t nt = std::min<int64_t>(hw, std::max<int64_t>(1, nb / 64));
  if (nt <= 1) {
    fn(int64_t(0), nb);
    return;
  }
  std::vector<std::thread> th;
  for (int64_t t = 0; t < nt; ++t) th.emplace_back([&, t] { fn(nb * t / nt, nb * (t + 1) / nt); });
  for (auto& x : th) x.join();
}

// steps[c * nb + b] = S(c, b)
void list_steps(const CodeReader& rd, int32_t d_out, std::vector<uint32_t>& steps) {
  const int K = sorted_classes(rd.M, rd.B);
  const int64_t nb = sorted_blocks(d_out);
  steps.assign((size_t)K * nb, 0);
  for_blocks(nb, [&](int64_t b0, int64_t b1) {
    std::vector<uint32_t> cnt((size_t)K * 16);
    for (int64_t b = b0; b < b1; ++b) {
      std::fill(cnt.begin(), cnt.end(), 0u);
      for (int i = 0; i < 16 && b * 16 + i < d_out; ++i)
        for (int64_t j = 0; j < rd.G; ++j)
          for (int m = 0; m < rd.M; ++m) ++cnt[(size_t)rd.cls(rd.at(b * 16 + i, j, m), m) * 16 + i];
      for (int c = 0; c < K; ++c) {
        uint32_t mx = 0;
        for (int i = 0; i < 16; ++i) mx = std::max(mx, cnt[(size_t)c * 16 + i]);
        steps[(size_t)c * nb + b] = (mx + 3u) / 4u;
      }
    }
  });
}

}  // namespace

int64_t sorted_steps(const void* codes, bool packed, int32_t d_out, int32_t d_in, int32_t M, int32_t B) {
  std::vector<uint32_t> steps;
  list_steps(reader(codes, packed, d_in, M, B), d_out, steps);
  int64_t total = 0;
  for (uint32_t s : steps) total += s;
  return total;
}

void sort_codes(const void* codes, bool packed, int32_t d_out, int32_t d_in, int32_t M, int32_t B, uint32_t* entries,
                int64_t steps, uint32_t* index) {
  const CodeReader rd = reader(codes, packed, d_in, M, B);
  const int K = sorted_classes(M, B);
  const int64_t nb = sorted_blocks(d_out);
  std::vector<uint32_t> s;
  list_steps(rd, d_out, s);
  uint32_t run = 0;
  for (size_t q = 0; q < s.size(); ++q) {
    index[q] = run;
    run += s[q];
  }
  index[s.size()] = run;
  (void)steps;
  for_blocks(nb, [&](int64_t b0, int64_t b1) {
    std::vector<uint32_t> pos((size_t)K);
    for (int64_t b = b0; b < b1; ++b) {
      for (int c = 0; c < K; ++c)
        std::fill(entries + 64ull * index[(size_t)c * nb + b], entries + 64ull * index[(size_t)c * nb + b + 1],
                  kSortedPad);
      for (int i = 0; i < 16 && b * 16 + i < d_out; ++i) {
        std::fill(pos.begin(), pos.end(), 0u);
        for (int64_t j = 0; j < rd.G; ++j)
          for (int m = 0; m < M; ++m) {
            const uint32_t v = rd.at(b * 16 + i, j, m);
            const int c = rd.cls(v, m);
            const uint32_t k = pos[(size_t)c]++;
            const uint64_t e = 64ull * (index[(size_t)c * nb + b] + k / 4u) + 16u * (k % 4u) + (uint64_t)i;
            entries[e] = (v & (kChunkCodewords - 1u)) | ((uint32_t)j << 14);
          }
      }
    }
  });
}

// ------------------------------------------------------------------- kernel

namespace {

constexpr int kSThreads = 1024;
constexpr int kSWaves = kSThreads / kWave;
constexpr int kSChunk = 16;                                    // steps of entries held per wave
constexpr uint32_t kCbLdsBytes = (kChunkCodewords + 1u) * 16u;  // chunk + zero codeword
constexpr uint32_t kLdsMax = 160u * 1024u;
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format
constexpr int kXPer = 2;                      // x in LDS: at most 2048 slices (with the zero one)
constexpr int kMaxBpr = 400;                  // most blocks of a row range (LDS of the segment sums)
constexpr uint32_t kTicket = 16;              // every launch adds 16 to the counter of each of its ranges
constexpr uint32_t kSpin = 1u << 22;          // polls of a missing partial before giving up
constexpr uint16_t kNaNh = 0x7E00;
constexpr int kMaxBoundWgs = 256;

struct SortedProblem {
  const uint32_t* entries;
  const uint32_t* index;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* x;
  uint16_t* y;
  uint64_t* part;  // workspace: [K][d_out] (fp32 bits | launch tag << 32)
  uint32_t entry_bytes;
  uint32_t total_steps;
  int32_t nb;
  int32_t d_out;
  int32_t G;
  int32_t R;            // row ranges
  int32_t wg_begin;     // first workgroup (a multiple of K)
  int32_t range_begin;  // counter of its first range
};

struct SortedBatch {
  SortedProblem p[kMaxProblems];
  uint32_t* counters;  // workspace: one per range of the launch
  int32_t count;
  int32_t B;
  int32_t bpr;       // most blocks of a range over the problems
  uint32_t seg_lds;  // byte offset of the segment sums in LDS (after the chunk and x)
  // every workgroup's steps [first, end), at 2 * blockIdx.x, from the
  // caller's host copies of the indexes (when given for every problem and the
  // launch has at most kMaxBoundWgs workgroups): read with the other
  // arguments, by block index alone, so the first entry loads wait for no
  // other load
  int32_t has_bounds;
  uint32_t wg_bounds[2 * kMaxBoundWgs];
};

__device__ __forceinline__ uint4 ld_lds16(uint32_t byte_addr) {
  typedef __attribute__((address_space(3))) const u32x4_t lds_v4_t;
  const u32x4_t v = *(lds_v4_t*)(uintptr_t)byte_addr;
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// LDS after the codebook chunk (and x):
//   seg[bpr + 16][16] fp32  row sums of each (block, wave) segment, slot b + w
//   blk[bpr + 16]           block of each slot (-1: unused)
//   idx[bpr + 1]            first step of each block's list, then the end
//   ticket                  the workgroup's counter value
//
// Cross-workgroup sum: every workgroup takes a ticket from its range's
// counter when it starts (adding 16 / K, so a launch adds 16 to the counter);
// the counter's index and ticket / 16 tag this launch's partial sums of the
// range, and the workgroup that takes the last ticket of the range sums it.  The others store each row's partial
// with the tag in one 64-bit word and exit; the summing workgroup polls the
// K - 1 other words of a row until their tags match (they are running: they
// took tickets), then adds the K partials in class order.
template <int K, bool XLDS>
__global__ __launch_bounds__(kSThreads) void k_gemv_sorted(const SortedBatch bt) {
  extern __shared__ uint4 lds[];
  // (fixed argument offsets: these loads go out together)
  int pi = 0;
#pragma unroll
  for (int q = 1; q < kMaxProblems; ++q) pi += (q < bt.count && (int)blockIdx.x >= bt.p[q].wg_begin) ? 1 : 0;
  const SortedProblem& a = bt.p[pi];
  const int local = (int)blockIdx.x - a.wg_begin;
  const int c = local % K;
  const int r = local / K;
  const int b_lo = (int)((int64_t)r * a.nb / a.R);
  const int b_hi = (int)((int64_t)(r + 1) * a.nb / a.R);
  const int nblk = b_hi - b_lo;
  const int lane = (int)threadIdx.x & (kWave - 1);
  // (wave-uniform: the loop control below stays in scalar registers)
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x / kWave);
  const uint32_t* __restrict__ gidx = a.index + (size_t)c * a.nb + b_lo;
  const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
  const uint32_t x_lds = lds_base + kCbLdsBytes;
  const int nslot = bt.bpr + kSWaves;
  float* seg = reinterpret_cast<float*>(reinterpret_cast<char*>(lds) + bt.seg_lds);
  int* blk = reinterpret_cast<int*>(seg + nslot * 16);
  uint32_t* idx = reinterpret_cast<uint32_t*>(blk + nslot);
  uint32_t* ticket_lds = idx + bt.bpr + 1;

  const __amdgpu_buffer_rsrc_t rs_e =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(a.entries), (short)0, (int)a.entry_bytes, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.x), (short)0, (int)((uint32_t)a.G * 16u), kRsrcWord3);

  // The range's steps [S0, S1) are split evenly over the waves.
  uint32_t S0, S1;
  if (bt.has_bounds) {
    S0 = min(bt.wg_bounds[2 * blockIdx.x], a.total_steps);
    S1 = max(min(bt.wg_bounds[2 * blockIdx.x + 1], a.total_steps), S0);
  } else {
    S0 = min((uint32_t)__builtin_amdgcn_readfirstlane(gidx[0]), a.total_steps);
    S1 = max(min((uint32_t)__builtin_amdgcn_readfirstlane(gidx[nblk]), a.total_steps), S0);
  }
  const uint32_t w_lo = S0 + (uint32_t)(((uint64_t)(S1 - S0) * (uint32_t)wave) / kSWaves);
  const uint32_t w_hi = S0 + (uint32_t)(((uint64_t)(S1 - S0) * (uint32_t)(wave + 1)) / kSWaves);

  // entries of steps [s, s + n) (n <= kSChunk); the rest read out of range (0)
  auto load = [&](uint32_t (&e)[kSChunk], uint32_t s, uint32_t n) {
#pragma unroll
    for (int k = 0; k < kSChunk; ++k) {
      const uint32_t off = (uint32_t)k < n ? (s + (uint32_t)k) * 256u + (uint32_t)lane * 4u : 0x80000000u;
      e[k] = __builtin_amdgcn_raw_buffer_load_b32(rs_e, (int)off, 0, 0);
    }
  };
  uint32_t eA[kSChunk], eB[kSChunk];
  uint32_t s = w_lo;
  uint32_t ticket;  // (thread 0 only)

  // stage the chunk (+ zero codeword), x (+ zero slice) and the range's
  // index; the wave's first entries are loaded at the same time
  {
    const int cpb = 1 << (bt.B - kChunkBits);
    const uint4* __restrict__ src = reinterpret_cast<const uint4*>(a.codebooks) +
                                    ((size_t)(c / cpb) << bt.B) + (size_t)(c % cpb) * kChunkCodewords;
    constexpr int kPer = (int)(kChunkCodewords / kSThreads);
    const int tid = (int)threadIdx.x;
    uint4 st[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) st[q] = src[tid + q * kSThreads];
    uint4 xst[kXPer];
    if constexpr (XLDS) {
      const uint4* __restrict__ xs = reinterpret_cast<const uint4*>(a.x);
      // (unconditional loads at clamped addresses: no branch, no early wait)
#pragma unroll
      for (int q = 0; q < kXPer; ++q) xst[q] = xs[min(tid + q * kSThreads, a.G - 1)];
    }
    const uint32_t iv = gidx[min(tid, nblk)];
    load(eA, s, min(w_hi - s, (uint32_t)kSChunk));
#pragma unroll
    for (int q = 0; q < kPer; ++q) lds[tid + q * kSThreads] = st[q];
    if (tid == 0) lds[kChunkCodewords] = make_uint4(0u, 0u, 0u, 0u);
    if constexpr (XLDS) {
      uint4* xl = lds + kChunkCodewords + 1;
#pragma unroll
      for (int q = 0; q < kXPer; ++q)
        if (tid + q * kSThreads <= a.G)
          xl[tid + q * kSThreads] = tid + q * kSThreads < a.G ? xst[q] : make_uint4(0u, 0u, 0u, 0u);
    }
    if (tid <= nblk) idx[tid] = min(max(iv, S0), S1);
    for (int q = tid; q < nslot; q += kSThreads) blk[q] = -1;
    // the ticket goes out after the staging and entry loads; its value is
    // read only after the main loop
    if (tid == 0)
      ticket = __hip_atomic_fetch_add(bt.counters + a.range_begin + r, kTicket / (uint32_t)K, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_SYSTEM);
  }
  lds_barrier();

  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
  // block (local) of step s and the end of its list
  // (the blocks after the first whose lists start at or before s, counted
  // 64 at a time)
  int b = 0;
  for (int k0 = 1; k0 < nblk; k0 += kWave) {
    const int k = k0 + lane;
    b += __builtin_popcountll(__ballot(k < nblk && idx[min(k, nblk)] <= s));
  }
  uint32_t bend = idx[b + 1];
  auto flush = [&]() {
    float v = (a0 + a1) + (a2 + a3);
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    const int slot = b + wave;
    if (lane < 16) seg[slot * 16 + lane] = v;
    if (lane == 0) blk[slot] = b;
    a0 = a1 = a2 = a3 = 0.f;
  };
  const uint32_t xg_pad = (uint32_t)a.G;  // zero slice in LDS
  // steps [s, s + n) from e: at each block boundary the sums so far are flushed
  auto process = [&](const uint32_t (&e)[kSChunk], uint32_t n) {
#pragma unroll
    for (int k0 = 0; k0 < kSChunk; k0 += 8) {
      if ((uint32_t)k0 < n) {
        uint4 cw[8], xv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const uint32_t en = (uint32_t)(k0 + k) < n ? e[k0 + k] : kSortedPad;
          const uint32_t code = min(en & 0x3FFFu, kChunkCodewords);
          cw[k] = ld_lds16(lds_base + code * 16u);
          if constexpr (XLDS) {
            xv[k] = ld_lds16(x_lds + min(en >> 14, xg_pad) * 16u);
          } else {
            const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs_x, (int)((en >> 14) << 4), 0, 0);
            xv[k] = make_uint4(v[0], v[1], v[2], v[3]);
          }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          if (s + (uint32_t)(k0 + k) == bend && (uint32_t)(k0 + k) < n) {
            flush();
            while (b + 1 < nblk && idx[b + 1] <= s + (uint32_t)(k0 + k)) ++b;
            bend = idx[b + 1];
          }
          dot8(cw[k], xv[k], a0, a1, a2, a3);
        }
      }
    }
  };
  // one step of the ring: process cur while the next chunk's entries load into nxt
  auto step = [&](uint32_t (&cur)[kSChunk], uint32_t (&nxt)[kSChunk]) -> bool {
    const uint32_t n = min(w_hi - s, (uint32_t)kSChunk);
    const uint32_t s2 = s + n;
    load(nxt, s2, min(w_hi - s2, (uint32_t)kSChunk));
    process(cur, n);
    // every load into cur has returned here on every path (also when part of
    // cur was not used), so the next step may reuse its registers at once
#pragma unroll
    for (int k = 0; k < kSChunk; ++k) asm volatile("" ::"v"(cur[k]));
    s = s2;
    return s < w_hi;
  };
  if (s < w_hi) {
    while (step(eA, eB) && step(eB, eA)) {
    }
    flush();
  }
  if (threadIdx.x == 0) *ticket_lds = ticket;
  lds_barrier();

  // rows of the range: add each block's segments in slot order
  // tag: the counter's index and this launch's count on it (never 0, the
  // value of a zeroed workspace); unique among launches that use the counter
  // (until its count wraps at 2^22 - 1) and among counters
  const uint32_t tk = *ticket_lds;
  const uint32_t tag = ((uint32_t)(a.range_begin + r) << 22) | ((tk / kTicket) % ((1u << 22) - 1u) + 1u);
  const bool summer = (tk % kTicket) / (kTicket / (uint32_t)K) == (uint32_t)(K - 1);
  const int row0 = b_lo * 16;
  const int rows = min(b_hi * 16, a.d_out) - row0;
  for (int i = (int)threadIdx.x; i < rows; i += kSThreads) {
    const int bi = i >> 4, ri = i & 15;
    // the block's segments sit in slots bi .. bi + 15, in wave order: all 32
    // LDS reads go out together, then the matching ones are added in order
    int bq[kSWaves];
    float sq[kSWaves];
#pragma unroll
    for (int k = 0; k < kSWaves; ++k) {
      bq[k] = blk[bi + k];
      sq[k] = seg[(bi + k) * 16 + ri];
    }
    float v = 0.f;
    bool any = false;
#pragma unroll
    for (int k = 0; k < kSWaves; ++k) {
      const bool m = bq[k] == bi;
      v = m ? (any ? v + sq[k] : sq[k]) : v;
      any = any || m;
    }
    uint64_t* __restrict__ slot = a.part + row0 + i;
    if (!summer) {
      __hip_atomic_store(slot + (size_t)c * a.d_out, (uint64_t)__builtin_bit_cast(uint32_t, v) | ((uint64_t)tag << 32),
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      continue;
    }
    uint64_t w[K];
#pragma unroll
    for (int cc = 0; cc < K; ++cc)
      w[cc] = cc == c ? 0u : __hip_atomic_load(slot + (size_t)cc * a.d_out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    bool ok = true;
#pragma unroll
    for (int cc = 0; cc < K; ++cc) {
      if (cc == c) continue;
      uint32_t n = 0;
      while ((uint32_t)(w[cc] >> 32) != tag) {
        if (++n > kSpin) {
          ok = false;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
        w[cc] = __hip_atomic_load(slot + (size_t)cc * a.d_out, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
    }
    float t = 0.f;
#pragma unroll
    for (int cc = 0; cc < K; ++cc) {
      const float pc = cc == c ? v : __builtin_bit_cast(float, (uint32_t)w[cc]);
      t = cc == 0 ? pc : t + pc;
    }
    a.y[row0 + i] = ok ? f2h(h2f(a.scales[row0 + i]) * t) : kNaNh;
  }
}

template <int K>
const void* sorted_kernel(bool xlds) {
  return xlds ? reinterpret_cast<const void*>(k_gemv_sorted<K, true>)
              : reinterpret_cast<const void*>(k_gemv_sorted<K, false>);
}

}  // namespace

bool gemv_sorted_fits(const SortedLayer* Ls, int count) {
  int64_t ranges = 0;
  for (int i = 0; i < count; ++i) ranges += (sorted_blocks(Ls[i].d_out) + kMaxBpr - 1) / kMaxBpr;
  return ranges <= (int64_t)(kSortedCounterBytes / 4);
}

size_t gemv_sorted_workspace_bytes(int64_t d_out, int M, int B) {
  return kSortedCounterBytes + (size_t)sorted_classes(M, B) * (size_t)d_out * 8u;
}

hipError_t launch_gemv_sorted(const SortedLayer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                              void* ws, hipStream_t s) {
  // (SortedBatch is passed by value: it must stay within the kernel argument limit)
  static_assert(sizeof(SortedBatch) <= 4000, "kernel arguments");
  const int M = Ls[0].M, B = Ls[0].B;
  const int K = sorted_classes(M, B);
  const int cus = num_cus();
  // ranges: at least one per problem and enough for kMaxBpr blocks each; the
  // rest of the CUs / K dealt by entries (largest remainders)
  int32_t R[kMaxProblems], nb[kMaxProblems];
  int64_t total = 0;
  int32_t used = 0;
  for (int i = 0; i < count; ++i) {
    nb[i] = (int32_t)sorted_blocks(Ls[i].d_out);
    R[i] = std::max<int32_t>(1, (nb[i] + kMaxBpr - 1) / kMaxBpr);
    used += R[i];
    total += Ls[i].steps;
  }
  const int32_t target = std::max(cus / K, used);
  if (target > used) {
    int32_t extra[kMaxProblems] = {};
    double rem[kMaxProblems];
    int32_t given = 0;
    const int32_t spare = target - used;
    for (int i = 0; i < count; ++i) {
      const double share = (double)spare * (double)Ls[i].steps / (double)std::max<int64_t>(total, 1);
      extra[i] = (int32_t)share;
      rem[i] = share - extra[i];
      given += extra[i];
    }
    while (given < spare) {
      int best = 0;
      for (int i = 1; i < count; ++i)
        if (rem[i] > rem[best]) best = i;
      ++extra[best];
      rem[best] = -1.0;
      ++given;
    }
    for (int i = 0; i < count; ++i) R[i] += extra[i];
  }
  SortedBatch bt = {};
  bt.counters = static_cast<uint32_t*>(ws);
  bt.count = count;
  bt.B = B;
  int32_t bpr = 1, G_max = 0, wgs = 0, ranges = 0;
  uint64_t* part = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + kSortedCounterBytes);
  for (int i = 0; i < count; ++i) {
    R[i] = std::min(R[i], nb[i]);
    bpr = std::max(bpr, (nb[i] + R[i] - 1) / R[i]);
    G_max = std::max(G_max, Ls[i].d_in / 8);
    SortedProblem& p = bt.p[i];
    p.entries = Ls[i].entries;
    p.index = Ls[i].index;
    p.codebooks = Ls[i].codebooks;
    p.scales = Ls[i].scales;
    p.x = xs[i];
    p.y = ys[i];
    p.part = part;
    part += (size_t)K * (size_t)Ls[i].d_out;
    p.entry_bytes = (uint32_t)(Ls[i].steps * 256);
    p.total_steps = (uint32_t)Ls[i].steps;
    p.nb = nb[i];
    p.d_out = Ls[i].d_out;
    p.G = Ls[i].d_in / 8;
    p.R = R[i];
    p.wg_begin = wgs;
    p.range_begin = ranges;
    wgs += K * R[i];
    ranges += R[i];
  }
  if (ranges > (int32_t)(kSortedCounterBytes / 4)) return hipErrorInvalidValue;  // (refused by the caller)
  // every workgroup's steps from the host copies of the indexes
  bt.has_bounds = wgs <= kMaxBoundWgs;
  for (int i = 0; i < count; ++i) bt.has_bounds = bt.has_bounds && Ls[i].index_host != nullptr;
  if (bt.has_bounds)
    for (int i = 0; i < count; ++i) {
      const SortedProblem& p = bt.p[i];
      for (int w = 0; w < K * p.R; ++w) {
        const int c = w % K, r = w / K;
        const int64_t b0 = (int64_t)r * p.nb / p.R, b1 = (int64_t)(r + 1) * p.nb / p.R;
        bt.wg_bounds[2 * (p.wg_begin + w)] = Ls[i].index_host[(size_t)c * p.nb + b0];
        bt.wg_bounds[2 * (p.wg_begin + w) + 1] = Ls[i].index_host[(size_t)c * p.nb + b1];
      }
    }
  bt.bpr = bpr;
  const uint32_t x_bytes = ((uint32_t)G_max + 1u) * 16u;
  const uint32_t tail = (uint32_t)(bpr + kSWaves) * (16u * 4u + 4u) + (uint32_t)(bpr + 1) * 4u + 16u;
  const bool xlds = G_max + 1 <= kXPer * kSThreads && kCbLdsBytes + x_bytes + tail <= kLdsMax;
  bt.seg_lds = kCbLdsBytes + (xlds ? x_bytes : 0u);
  const size_t lds = bt.seg_lds + tail;
  const void* kern = K == 4 ? sorted_kernel<4>(xlds) : K == 8 ? sorted_kernel<8>(xlds) : sorted_kernel<16>(xlds);
  const hipError_t e = allow_dynamic_lds(kern, (int)kLdsMax);
  if (e != hipSuccess) return e;
  void* args[] = {&bt};
  return hipLaunchKernel(kern, dim3(wgs), dim3(kSThreads), args, lds, s);
}

}  // namespace aqlm
