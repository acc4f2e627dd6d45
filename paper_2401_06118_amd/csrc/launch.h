// Internal launchers (C++ linkage) behind the C ABI in include/aqlm.h.
// Arguments are already validated by the caller; every function returns a
// hipError_t from the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace aqlm {

// The (M, B) formats the library runs, all with g = 8: one to eight
// codebooks of 8-bit codes; one codebook of 15- or 16-bit codes; two
// codebooks of 12-, 15- or 16-bit codes (the 2-, 3- and 4-bit settings of the
// appendix "Experimental Configurations").  Codes wider than 8 bits are
// stored one per uint16.
constexpr bool format_supported(int M, int B) {
  return (B == 8 && M >= 1 && M <= 8) || ((B == 15 || B == 16) && M == 1) ||
         ((B == 12 || B == 15 || B == 16) && M == 2);
}

// Bit-packed codes: 12-bit codes of two codebooks, 15-bit codes of one or two.
constexpr bool packed_supported(int M, int B) { return (B == 12 && M == 2) || (B == 15 && (M == 1 || M == 2)); }

struct Layer {
  const void* codes;          // [d_out][G][M] uint8 (B = 8) or uint16 (B > 8)
  const uint16_t* codebooks;  // [M][2^B][8] fp16
  const uint16_t* scales;     // [d_out] fp16
  int32_t d_out;
  int32_t d_in;
  int32_t G;  // d_in / 8
  int32_t M;
  int32_t B;
  bool vec_codes;  // codes base 16-byte aligned and row pitch a multiple of 16 bytes
  bool packed;     // B-bit codes packed into a bit string per row (32-bit words; B = 12, 15)
  bool tiled = false;  // 8-bit codes in 1 KiB tiles (tiled_codes_offset), not row-major
};

// Tiled 8-bit codes: the code bytes of 16 rows x one 64-byte K-slice of a row
// are one 1 KiB tile, row after row; tiles run K-slice after K-slice within a
// 16-row block, then block after block.  Rows past d_out and bytes past a
// row's G * M are zero.  Byte c of row r sits at this offset.
inline int64_t tiled_codes_offset(int64_t r, int64_t c, int64_t ks_per_row) {
  return ((r >> 4) * ks_per_row + (c >> 6)) * 1024 + (r & 15) * 64 + (c & 63);
}
inline int64_t tiled_codes_bytes(int64_t d_out, int64_t row_bytes) {
  return ((d_out + 15) / 16) * ((row_bytes + 63) / 64) * 1024;
}

// 32-bit words of one row of packed codes: G*M codes of B bits, zero-padded.
inline int32_t packed_row_words(int32_t G, int32_t M, int32_t B) {
  return (int32_t)(((int64_t)G * M * B + 31) / 32);
}

constexpr int kMaxProblems = 8;

// One matrix-vector problem of a (possibly grouped) launch and its share of
// the workgroups: workgroups [wg_begin, wg_begin + ceil(d_out / rows_per_wg)).
struct GemvProblem {
  const uint8_t* codes;
  const uint4* cb;
  const uint16_t* scales;
  const uint4* x;  // [G] groups of 8 fp16
  uint16_t* y;
  int32_t d_out;
  int32_t G;
  int32_t wg_begin;
  int32_t rows_per_wg;
  int32_t pwords;  // packed codes: 32-bit words per row (0: unpacked)
};

struct GemvBatch {
  GemvProblem p[kMaxProblems];
  int32_t count;
  int32_t total_wgs;
  int32_t xg_max;  // x groups staged in LDS by the largest problem
  int32_t tiled;   // codes of every problem tiled (k_gemv_ks only)
};

// Decode step (a persistent launch over many grouped 2x8 products): one
// record per level, after a StepHeader, in device memory.
struct StepLevel {
  GemvBatch bt;
  int32_t variant;    // k_gemv_ks body instantiation (an index into the step kernel's table)
  int32_t lds_bytes;  // dynamic LDS this level needs
};
struct StepHeader {
  uint32_t magic;
  int32_t levels;
  int32_t lds_bytes;  // maximum over the levels
  int32_t grid;       // workgroups of the resident grid (CU count at planning time)
};
constexpr uint32_t kStepMagic = 0x50455453u;
// Plans one level (no launch); rb_cap_max > 0 caps the row blocks per
// workgroup, lds_limit the dynamic LDS.
hipError_t gemv_mfma_impl(const Layer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                          hipStream_t s, StepLevel* plan, int rb_cap_max, size_t lds_limit);
// LDS the step kernel leaves to the levels (it keeps a word of its own).
constexpr size_t kStepLdsLimit = 160 * 1024 - 256;
// sync: 3 words (level counter, error flag, exit counter), zero before the
// first launch and left zero by a launch that completes (the error flag
// stays set after a timed-out wait).
hipError_t launch_step(const StepLevel* levels, int32_t nlev, int32_t grid, size_t lds, uint32_t* sync,
                       uint32_t spin, hipStream_t s);

hipError_t launch_dequant(const Layer& L, uint16_t* w, hipStream_t s);
bool gemv_mfma_supported(int M, int B);
bool gemv_mfma_fits(const Layer* Ls, int count);
// Row-major 8-bit codes [d_out][row_bytes] to the tiled layout (csrc/tiled.hip).
hipError_t launch_tile_codes(const uint8_t* codes, int64_t d_out, int64_t row_bytes, uint8_t* tiled, hipStream_t s);

hipError_t launch_gemv_mfma(const Layer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                            hipStream_t s);
hipError_t launch_gemv(const Layer& L, const uint16_t* x, uint16_t* y, hipStream_t s);
// Batch-1 2x8 product through per-group partial-product tables (d_in a
// multiple of 256).
bool gemv_lut_supported(const Layer* Ls, int count);
hipError_t launch_gemv_lut(const Layer* Ls, const uint16_t* const* xs, uint16_t* const* ys, int count,
                           hipStream_t s);
hipError_t launch_gemm_mfma(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s);
bool mfma_supported(const Layer& L);
bool gemm_nb_supported(const Layer& L, int32_t n);
bool prefill_supported(const Layer& L);
hipError_t launch_prefill(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s);
hipError_t launch_gemm_nb(const Layer& L, int32_t n, const uint16_t* x, uint16_t* y, hipStream_t s);
// Dense fp16 product y[t][i] = sum_c x[t][c] w[i][c] (w: dequantized weights).
bool gemm_f16_supported(int32_t d_in);
// fp32 scratch for K-split partial sums (0 when the product is not split).
size_t gemm_f16_part_bytes(int64_t n, int64_t d_out, int64_t K);
hipError_t launch_gemm_f16(const uint16_t* x, const uint16_t* w, uint16_t* y, float* part, int32_t n, int32_t d_out,
                           int32_t K, hipStream_t s);

// Gradients through Eq. 2 (8-bit codes, d_out a multiple of 8): accumulates
// dC and dscales for y = x W^T and an upstream gradient dy.
bool backward_supported(const Layer& L);
hipError_t launch_backward(const Layer& L, int32_t n, const uint16_t* x, const uint16_t* dy, float* dcb, float* ds,
                           hipStream_t s);

// Phase-1 beam search over codes (8-bit codes), one workgroup per row, the
// beam state in LDS.
bool beam_search_fits(int32_t d_in, int32_t M, int32_t beam);
hipError_t launch_beam_search(const float* w, const float* h, uint8_t* codes, const uint16_t* codebooks,
                              const uint16_t* scales, int32_t d_out, int32_t d_in, int32_t M, int32_t beam,
                              int32_t sweeps, float* loss, hipStream_t s);

int num_cus();
// Allows a kernel `bytes` of dynamic LDS on the current device (once per
// kernel, device and size).
hipError_t allow_dynamic_lds(const void* kern, int bytes);

}  // namespace aqlm
