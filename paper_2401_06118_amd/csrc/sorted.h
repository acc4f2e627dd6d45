// Chunk-sorted storage of wide codes for the batch-1 product (one or two
// codebooks of 2^15 or 2^16 codewords, g = 8: the 2- and 4-bit settings of
// the appendix "Experimental Configurations").
//
// Eq. 2 is unchanged; only the order in which a row's codes are stored
// changes.  A codebook of 2^B codewords is cut into chunks of 8192 codewords
// (128 KiB of fp16), and a code (row i, group j, codebook m) of value v
// belongs to chunk class c = m * 2^(B-13) + (v >> 13), one of
// K = M * 2^(B-13) classes.  For every block of 16 rows and every class the
// codes of that class are listed row by row, so that one workgroup holding one
// chunk in LDS can serve all of them:
//   - block b, class c: S(c, b) = ceil(max_i n_i / 4) steps of 64 entries,
//     where n_i is the number of codes of class c in row i of the block;
//   - the k-th code of class c of row i (ascending j) is entry
//     64 * (index[c * nb + b] + k / 4) + 16 * (k % 4) + i;
//   - an entry is (v & 8191) | (j << 14); unused entries hold kSortedPad
//     (codeword 8192 = a zero codeword the kernel appends to the chunk, and a
//     group index past the row, whose x slice the kernel reads as zero);
//   - index [K * nb + 1]: first step of every list, class-major, and the total.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace aqlm {

constexpr int kChunkBits = 13;
constexpr uint32_t kChunkCodewords = 1u << kChunkBits;
constexpr uint32_t kSortedPad = 0xFFFFE000u;
constexpr uint32_t kSortedJMax = (1u << 18) - 2;  // largest group index an entry can hold
constexpr size_t kSortedCounterBytes = 4096;      // one 32-bit counter per row range

constexpr bool sorted_supported(int M, int B) { return (M == 1 || M == 2) && (B == 15 || B == 16); }
constexpr int sorted_classes(int M, int B) { return M << (B - kChunkBits); }
constexpr int64_t sorted_blocks(int64_t d_out) { return (d_out + 15) / 16; }

// Host: codes [d_out][d_in/8][M] (uint16 each, or one bit string per row when
// packed) -> total steps of the sorted form.
int64_t sorted_steps(const void* codes, bool packed, int32_t d_out, int32_t d_in, int32_t M, int32_t B);
// Host: fills entries [steps * 64] and index [K * nb + 1].
void sort_codes(const void* codes, bool packed, int32_t d_out, int32_t d_in, int32_t M, int32_t B, uint32_t* entries,
                int64_t steps, uint32_t* index);

struct SortedLayer {
  const uint32_t* entries;  // device, [steps][64]
  const uint32_t* index;    // device, [K * nb + 1]
  const uint32_t* index_host;  // the same on the host, or nullptr
  int64_t steps;
  const uint16_t* codebooks;  // [M][2^B][8] fp16
  const uint16_t* scales;     // [d_out] fp16
  int32_t d_out;
  int32_t d_in;
  int32_t M;
  int32_t B;
};

// Whether `count` problems fit one launch (at most 1024 row ranges of at most
// 400 blocks).
bool gemv_sorted_fits(const SortedLayer* Ls, int count);
// Row-range counters (4096 bytes), then (fp32 partial, launch tag) pairs
// [K][d_out] as 64-bit words (d_out: the sum over a grouped launch).
size_t gemv_sorted_workspace_bytes(int64_t d_out, int M, int B);
// y = fp16(s_i * sum of the row's codeword-times-x products) for `count`
// (1..8) problems of one format in one launch, fp32 accumulation in a fixed
// order (deterministic).  `ws`: the workspace above, its counters zero before
// the first call (each launch adds 16 to each counter it uses).
hipError_t launch_gemv_sorted(const SortedLayer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                              void* ws, hipStream_t s);

}  // namespace aqlm
