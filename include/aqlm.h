/*
 * aqlm.h - C ABI of the MI355X (gfx950) AQLM inference library.
 *
 * AQLM ("Extreme Compression of Large Language Models via Additive
 * Quantization") stores a weight matrix W [d_out][d_in] as
 *   - codes: for output row i, input group j (g consecutive inputs) and
 *     codebook m, an index b[i][j][m] into codebook m (Sec. 3, Eq. 2);
 *   - codebooks C_m: M tables of 2^B codewords of g fp16 values each;
 *   - scales s_i: one fp16 scale per output unit (Sec. 3.3, Fig. 3 step v).
 * Group j of row i reconstructs as s_i * sum_m C_m[b[i][j][m]] (Eq. 2 and
 * Fig. 3 steps i-v).  The library computes that reconstruction and the
 * product of it with activations, the operation the paper benchmarks for
 * token generation (Sec. 4.3, matrix-vector product on one layer).
 *
 * Types: fp16 values travel as their IEEE-754 binary16 bit patterns in
 * uint16_t.  Every pointer is a DEVICE pointer (HIP memory on the current
 * device) unless stated otherwise.  The caller allocates and owns every
 * buffer; the library allocates nothing and keeps no state between calls
 * beyond its loaded kernels, so calls are reentrant and thread-safe.
 *
 * Layouts (dense, row-major, contiguous):
 *   codes      [d_out][d_in/g][M], m fastest.  uint8_t when B = 8,
 *              uint16_t when B = 12, 15 or 16 (unpacked); value = codeword
 *              index, taken modulo 2^B.
 *   codebooks  [M][2^B][g] fp16 (one codeword = g contiguous values).
 *   scales     [d_out] fp16.
 *   x          [n][d_in] fp16 (n = 1 for the matrix-vector product).
 *   y          [n][d_out] fp16.
 *   w_out      [d_out][d_in] fp16.
 *
 * Supported formats, all with g = 8 (the 2x8 model of Sec. 4.3 and the 2-,
 * 3- and 4-bit settings of the appendix "Experimental Configurations"):
 *   B = 8,  1 <= M <= 8   M codebooks of 256 entries;
 *   B = 15 or 16, M = 1   one codebook of 32768 or 65536 entries (2 bits);
 *   B = 12, M = 2         two codebooks of 4096 entries (3 bits);
 *   B = 15 or 16, M = 2   two codebooks of 32768 or 65536 entries (4 bits).
 * Larger groups (the codebooks-versus-groups settings of the ablation:
 * 4x8 with groups of 16, 8x8 with 32, 15x8 with 64): g = 16, 32 or 64 with
 * B = 8 and 1 <= M <= 16, codebooks [M][256][g].  aqlm_dequantize, aqlm_gemv,
 * aqlm_gemv_grouped (gather path), aqlm_gemm_small_batch (one matrix-vector
 * product per row), aqlm_gemm and aqlm_gemm_noalloc take them (for these the
 * two-pass product has the same workspace rule); every other entry point
 * returns AQLM_ERR_UNSUPPORTED.  Here d_out * d_in / 8 must stay below 2^31.
 * Codes wider than 8 bits are stored one per uint16 by default.  Bit-packed
 * codes (the storage the paper's bits-per-parameter figures count, Sec. 3.3):
 * pass B | AQLM_PACKED for B = 12 (M = 2) or 15 (M = 1 or 2).  Each row of
 * codes is then one bit string of d_in/g * M codes of B bits, code (j, m)
 * at bits [(j*M + m)*B, (j*M + m + 1)*B), least significant bit first,
 * zero-padded to whole little-endian 32-bit words: aqlm_packed_row_words()
 * words per row, rows contiguous.  Only aqlm_dequantize, aqlm_gemv and
 * aqlm_gemv_grouped (gather path) accept packed codes; every other entry
 * point returns AQLM_ERR_UNSUPPORTED for them, as does aqlm_gemv when x
 * does not fit the matrix-core kernel's staging (d_in above 65536).  A
 * packed row must hold fewer than 2^32 bits (else AQLM_ERR_SHAPE).
 * Sizes: d_out * (d_in / g) must stay below 2^31 and d_out, d_in, n below
 * 2^31.
 *
 * Alignment: codes, codebooks, x, y and w_out must be 16-byte aligned and
 * scales 2-byte aligned.  Shapes whose code row pitch (d_in/g * M bytes for
 * 8-bit codes, twice that for wider codes) is a multiple of 16 take
 * the vectorized load path; any other shape takes a slower generic path with
 * the same results.
 *
 * Errors: all argument checks run on the host before anything is launched; on
 * an error nothing is launched and no output is touched.  A HIP launch error
 * is reported as AQLM_ERR_HIP.  Calls are asynchronous on `stream` (a
 * hipStream_t; NULL means the default stream): a device-side fault surfaces at
 * the caller's next synchronisation.  Outputs must not alias inputs.
 */
#ifndef AQLM_MI355X_H
#define AQLM_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum aqlm_status {
  AQLM_OK = 0,
  AQLM_ERR_NULL = 1,        /* a required pointer is NULL */
  AQLM_ERR_SHAPE = 2,       /* non-positive or too large size, or d_in % g != 0 */
  AQLM_ERR_UNSUPPORTED = 3, /* (M, B, g) outside the supported set */
  AQLM_ERR_ALIGN = 4,       /* a pointer breaks the alignment rule above */
  AQLM_ERR_HIP = 5,         /* the HIP runtime reported an error */
  AQLM_ERR_WORKSPACE = 6,   /* aqlm_gemm: workspace smaller than aqlm_gemm_workspace_bytes */
  AQLM_ERR_SCRATCH = 7,     /* aqlm_gemm_noalloc: the product needs more than its fixed scratch */
  AQLM_ERR_TIMEOUT = 8      /* aqlm_gemv_step_status: a level barrier gave up waiting */
};

/* OR into B to pass bit-packed codes (see "Bit-packed codes" above). */
#define AQLM_PACKED 0x100

/* 32-bit words that hold one row of bit-packed codes: ceil(d_in/g * M * B / 32)
 * (B without AQLM_PACKED).  Host function; returns 0 for a non-positive size. */
int64_t aqlm_packed_row_words(int64_t d_in, int32_t M, int32_t B, int32_t g);

/* Dequantize: w_out[i][j*g + k] = fp16(fp32(sum_m C_m[b[i][j][m]][k]) * s_i)
 * (Eq. 2, Fig. 3 steps i-v).  The M codewords are added in fp32 in ascending m,
 * starting from codeword 0, then multiplied by the scale in fp32 and rounded
 * once to fp16 (nearest, ties to even, subnormals kept, overflow to inf).
 * The result is bit-exact and deterministic. */
int aqlm_dequantize(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                    int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                    uint16_t* w_out, void* stream);

/* Matrix-vector product for token generation (Sec. 4.3):
 * y[i] = fp16(s_i * sum_j sum_m <C_m[b[i][j][m]], x[j*g .. j*g+g)>), fp32
 * accumulation.  The reconstructed weights are not rounded to fp16 first, and
 * the summation order differs from a dense product: results agree with
 * fp16(W) x to fp32 accumulation accuracy, not bit for bit.  Deterministic. */
int aqlm_gemv(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
              int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
              const uint16_t* x, uint16_t* y, void* stream);

/* One problem of a grouped matrix-vector launch (all pointers device memory,
 * same layouts and rules as aqlm_gemv). */
typedef struct aqlm_gemv_problem {
  const void* codes;
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* x; /* [d_in] */
  uint16_t* y;       /* [d_out] */
  int64_t d_out;
  int64_t d_in;
} aqlm_gemv_problem;

#define AQLM_MAX_GROUPED 8

/* `count` (1..AQLM_MAX_GROUPED) independent matrix-vector products that share
 * (M, B, g), computed as aqlm_gemv would compute each, in one launch - for
 * layers that read the same activation, such as the q, k and v projections or
 * the gate and up projections of a transformer block (the paper's speed
 * measurement is per layer, Sec. 4.3; grouping only removes launch overhead).
 * `problems` is a HOST array read during the call.  Every problem is
 * validated before anything is launched; the first error is returned.
 * Outputs must not alias any input of any problem.  Deterministic; results
 * may differ from separate aqlm_gemv calls in the last bits because the rows
 * are split over workgroups differently. */
int aqlm_gemv_grouped(const aqlm_gemv_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                      void* stream);

/* Kernel families for the batch-1 product (aqlm_gemv_grouped_path). */
enum aqlm_gemv_path {
  AQLM_PATH_AUTO = 0,   /* the library's choice (what aqlm_gemv / aqlm_gemv_grouped run): the
                           gather family, measured at least as fast on every Llama-2 shape */
  AQLM_PATH_GATHER = 1, /* codeword gathers: each code's codeword is looked up and multiplied
                           with x (matrix-core or vector-ALU kernel, by format and size) */
  AQLM_PATH_TABLE = 2   /* per-group partial-product tables: the inner products
                           <C_m[e], x_j> of every codeword e and input group j are
                           computed once per workgroup (in fp32, on the matrix cores)
                           and each code adds its table entry (the lookup of precomputed
                           inner products of Sec. 2.2 applied to Eq. 2).  2x8 only, with
                           d_in a multiple of 256 */
};

/* aqlm_gemv_grouped with the kernel family chosen by the caller (for
 * measurement, or where the caller knows its shapes better).  Same
 * arguments, results and rules as aqlm_gemv_grouped, plus `path`; a path
 * that cannot take the format or shapes returns AQLM_ERR_UNSUPPORTED before
 * anything is launched.  Both families accumulate in fp32 and meet the same
 * accuracy; their results differ in the last bits.  Deterministic. */
int aqlm_gemv_grouped_path(const aqlm_gemv_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                           int32_t path, void* stream);

/* Tiled storage of 8-bit codes for the batch-1 product (the same codes b_ijm
 * of Eq. 2 in another byte order; Sec. 4.3's token-generation product reads
 * them).  Each wave of the product reads the 64-byte K-slice of 16 rows at a
 * time; row-major, those are 16 separate half-lines, tiled they are one
 * contiguous 1 KiB.  Layout, with row_bytes = (d_in / g) * M and
 * ks = ceil(row_bytes / 64): byte c of row r at
 *   ((r / 16) * ks + c / 64) * 1024 + (r % 16) * 64 + c % 64,
 * rows past d_out and bytes past row_bytes zero.  Formats: B = 8, g = 8,
 * M in {1, 2, 4}; anything else AQLM_ERR_UNSUPPORTED; shapes whose tiled
 * size reaches 2^31 bytes AQLM_ERR_SHAPE. */

/* Bytes of the tiled codes of one layer: 16 * ceil(d_out / 16) * ks * 64;
 * 0 for an unsupported format or shape. */
int64_t aqlm_tiled_codes_bytes(int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g);

/* Writes the tiled copy of row-major codes [d_out][d_in / g][M] (DEVICE,
 * uint8, any alignment) to `tiled` (DEVICE, 16-byte aligned, caller-owned,
 * at least aqlm_tiled_codes_bytes bytes: else AQLM_ERR_WORKSPACE) on
 * `stream`.  NULL pointers AQLM_ERR_NULL.  Byte-exact permutation plus zero
 * padding; allocates nothing. */
int aqlm_tile_codes(const void* codes, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, void* tiled,
                    int64_t tiled_bytes, void* stream);

/* aqlm_gemv_grouped over tiled codes: each problem's `codes` points to what
 * aqlm_tile_codes wrote for that layer (16-byte aligned), everything else as
 * for aqlm_gemv_grouped (same validation order, errors, determinism).  The
 * arithmetic is the gather kernel's on the same rows and workgroup split, so
 * the results equal aqlm_gemv_grouped's on the row-major codes bit for bit.
 * Formats beyond the tiled ones, or x too large for the kernel's on-chip
 * staging (d_in above about 32768 for M = 2), return AQLM_ERR_UNSUPPORTED. */
int aqlm_gemv_grouped_tiled(const aqlm_gemv_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                            void* stream);

/* aqlm_gemm_small_batch over tiled codes (what aqlm_tile_codes wrote for the
 * layer, 16-byte aligned) for 1 to 64 activation rows, the token-generation
 * product of Sec. 4.3 with several sequences: n = 1 as aqlm_gemv; 2 <= n <= 64
 * with M in {2, 4} by the small-batch kernel, up to 16 rows per launch (a
 * last chunk of one row as aqlm_gemv).  Validation, errors and results as
 * aqlm_gemm_small_batch on the row-major codes (bit for bit); n > 64, or
 * M = 1 with n > 1, AQLM_ERR_UNSUPPORTED before anything is launched. */
int aqlm_gemm_small_batch_tiled(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                                int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x,
                                uint16_t* y, void* stream);

/* Product with n activation rows: y[t][i] = fp16(s_i * sum_c W[i][c] x[t][c])
 * with W reconstructed as above, fp32 accumulation, any n >= 1 (the batched
 * and prefill products of a layer; the paper times the single-row case,
 * Sec. 4.3).  n = 1 runs the matrix-vector kernel; 2..16 rows put the rows in
 * the matrix-core (MFMA) columns of the same scheme, and up to 64 rows (32
 * for 1x16) run as chunks of 16; more rows dequantize weight tiles into
 * on-chip memory once per tile of 128 or 256 rows of x and feed them to dense
 * fp16 MFMA products.  Needs no workspace.  Results are
 * within fp32-accumulation accuracy of fp16(W) x, not bit-exact with it.
 * Deterministic. */
int aqlm_gemm_small_batch(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                          int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n,
                          const uint16_t* x, uint16_t* y, void* stream);

/* Device workspace, in bytes, that aqlm_gemm needs for these sizes, 0 when
 * it does not take the two-pass path (it does when n >= 64 and d_in is a
 * multiple of 64): the dequantized weights (d_out * d_in * 2, rounded up to
 * 256) and, when the product has fewer 128 x 128 output tiles than the GPU
 * has compute units and is split along d_in, fp32 partial sums (up to
 * 8 * n * d_out * 4).  Depends on the current device's compute-unit count.
 * Returns 0 for invalid sizes (aqlm_gemm then reports the error). */
size_t aqlm_gemm_workspace_bytes(int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n);

/* The product of aqlm_gemm_small_batch with a caller-provided workspace:
 * for many activation rows the weights are dequantized once into `workspace`
 * exactly as aqlm_dequantize writes them (scales included, Eq. 2), then a
 * dense fp16 MFMA product y[t][i] = fp16(sum_c W[i][c] x[t][c]) with fp32
 * accumulation reads them; this removes the per-tile rebuilding of the
 * weights that aqlm_gemm_small_batch pays.  `workspace` is DEVICE memory of
 * at least aqlm_gemm_workspace_bytes(...) bytes, 16-byte aligned, owned by
 * the caller; its contents are overwritten (its first d_out * d_in * 2 bytes
 * hold W afterwards) and it must not alias any other argument.  A split
 * product adds the partial sums in a fixed order, so results stay
 * deterministic.  When the size query returns 0 the
 * workspace is not used and may be NULL, and the call computes exactly what
 * aqlm_gemm_small_batch computes.  Errors as above, plus AQLM_ERR_NULL for a
 * needed NULL workspace and AQLM_ERR_WORKSPACE for a small one.
 * Deterministic. */
int aqlm_gemm(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
              int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n,
              const uint16_t* x, uint16_t* y, void* workspace, size_t workspace_bytes, void* stream);

/* Gradients through Eq. 2 for fine-tuning codebooks and scales (Sec. 3,
 * "Phase 2: Codebook update" and "Phase 3: Fine-tuning"; App. "End-to-end
 * fine-tuning"): for y = x W^T over n activation rows x [n][d_in] and the
 * upstream gradient dy = dL/dy [n][d_out] (fp16), with
 * G[i][c] = sum_t dy[t][i] x[t][c] and u[i][c] the fp32 sum of the codewords
 * of row i, group c / g (the sum the weights are rounded from; the rounding
 * is not differentiated), ACCUMULATES
 *   dcodebooks[m][e][k] += sum over (i, j) with b[i][j][m] = e of s_i * G[i][j*g + k]
 *   dscales[i]          += sum_c G[i][c] * u[i][c]
 * into fp32 device arrays [M][2^B][g] and [d_out] (zero them for a fresh
 * gradient; leave them to accumulate micro-batches).  G is computed in fp32
 * on the matrix cores and never stored; no workspace.  The additions use
 * atomics, so results agree with an exact computation to fp32 accuracy but
 * may differ in the last bits from run to run.  Supported: B = 8 with
 * 1 <= M <= 8, g = 8, d_out a multiple of 8 (else AQLM_ERR_UNSUPPORTED /
 * AQLM_ERR_SHAPE); x and dy 16-byte aligned, the gradients 4-byte aligned.
 * Other errors as aqlm_gemm_small_batch. */
int aqlm_backward(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                  int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, const uint16_t* dy,
                  float* dcodebooks, float* dscales, void* stream);

/* Phase 1 of AQLM, beam search over the codes (Sec. 3, "Phase 1: Beam search
 * for codes"): for every output row i, with H = X X^T [d_in][d_in] (fp32,
 * symmetric) and the original weights w [d_out][d_in] (fp32), improves the
 * row's codes for the objective
 *   L_i = (w_i - what_i) H (w_i - what_i)^T,  what_i[8j + t] = s_i sum_m C_m[b_ijm][t]
 * (the layer's squared output error over the calibration inputs X, Eq.
 * main_obj; what is the exact reconstruction, not rounded to fp16).  A beam
 * of at most `beam` configurations starts as the row's current codes; each
 * step takes one code position (groups in ascending order, codebooks in
 * ascending order within a group), tries every codeword there for every
 * configuration in the beam, and keeps the `beam` distinct configurations of
 * least loss (ties: earlier beam entry, then smaller code); `sweeps` passes
 * over all positions; the best configuration is written back to `codes`
 * (in place).  Candidate losses are the entry's loss plus a change computed
 * incrementally in fp32 from H r and the H_jj block, as the paper describes
 * (fp32 and exact arithmetic can break near-ties differently).  `loss_out`
 * (fp32 [d_out], may be NULL) receives each row's final loss, recomputed
 * exactly (fp64) from the returned codes.  Rows are searched in parallel (one
 * workgroup per row, the beam state in on-chip memory).
 * Supported: B = 8, 1 <= M <= 8, g = 8, 1 <= beam <= 8, and
 * 8 * beam * d_in + 2 * beam * d_in / 8 * M + 4096 * M bytes of state within
 * about 158 KiB (d_in up to 2048 with beam 8, 4096 with beam 4); otherwise
 * AQLM_ERR_UNSUPPORTED.  w, h and loss_out 4-byte aligned.  Deterministic. */
int aqlm_beam_search(const float* w, const float* h, void* codes, const uint16_t* codebooks, const uint16_t* scales,
                     int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int32_t beam, int32_t sweeps,
                     float* loss_out, void* stream);

/* Bytes of the fixed device scratch buffer of aqlm_gemm_noalloc (128 MiB). */
#define AQLM_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/* aqlm_gemm for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same product, computed by the same kernels as aqlm_gemm, with the workspace
 * taken from a fixed scratch buffer of AQLM_NOALLOC_SCRATCH_BYTES that the
 * library holds on each device it runs on (a static device array, allocated
 * when the library's code is loaded on the device and kept until the process
 * ends).  The call itself allocates nothing.  The caller passes inputs and
 * outputs only.  Results are bit-identical to aqlm_gemm's.
 *   - The scratch needed is aqlm_gemm_workspace_bytes(...); a product that
 *     needs more than AQLM_NOALLOC_SCRATCH_BYTES (e.g. more than 64 M weights)
 *     returns AQLM_ERR_SCRATCH before anything is launched.  When no
 *     workspace is needed the call computes exactly aqlm_gemm_small_batch.
 *   - Every call on one device shares that device's buffer, which keeps the
 *     last call's contents (nothing in it needs to start at zero: each call
 *     writes what it reads).  Calls that overlap on one device - on two
 *     streams, or from two host threads without ordering - RACE and give
 *     undefined results; calls on one stream are ordered and safe.
 * Other errors as aqlm_gemm; deterministic. */
int aqlm_gemm_noalloc(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                      int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, uint16_t* y,
                      void* stream);

/* ---------------------------------------------------------------- decode step
 *
 * The matrix-vector products of a whole decode step in ONE launch (the paper
 * times end-to-end generation with the model's computational graph compiled,
 * App. "End-to-End Inference Speed", Table 13; here the compiled form is a
 * step plan run by a persistent kernel).  A step is a list of levels; a level
 * is 1..AQLM_MAX_GROUPED independent products computed exactly as
 * aqlm_gemv_grouped computes them.  Level l + 1 starts reading its x only
 * after every product of level l has been written, so a level may read what
 * earlier levels wrote (e.g. level l + 1's x is level l's y).  While the last
 * workgroups finish a level, the others already load the next level's codes,
 * codebooks and scales.  2x8 (M = 2, B = 8, g = 8) with d_in a multiple of 64
 * and x within the matrix-core kernel's staging (d_in <= 32768); anything else
 * returns AQLM_ERR_UNSUPPORTED. */
#define AQLM_STEP_MAX_LEVELS 65536
#define AQLM_STEP_SYNC_BYTES 256
#define AQLM_STEP_DEFAULT_SPIN (1u << 20)

/* Bytes a plan of `levels` levels takes (0 if levels is out of range). */
int64_t aqlm_gemv_step_plan_bytes(int32_t levels);

/* Builds a step plan in HOST memory `plan` (plan_bytes >= the size above):
 * `problems` (host array) holds the levels' problems one level after the
 * other, level_sizes[l] of them for level l.  Every problem is validated as
 * aqlm_gemv_grouped validates it; nothing touches the GPU, and the plan holds
 * the problems' device pointers, so those buffers must outlive it.  The
 * caller copies the plan, as bytes, to DEVICE memory (16-byte aligned) for
 * aqlm_gemv_step.  The work split is sized for the current device.  A plan
 * smaller than needed: AQLM_ERR_WORKSPACE. */
int aqlm_gemv_step_plan(const aqlm_gemv_problem* problems, const int32_t* level_sizes, int32_t levels,
                        int32_t M, int32_t B, int32_t g, void* plan, int64_t plan_bytes);

/* Runs a planned step: one cooperative launch of one workgroup per CU on
 * `stream`.  plan_host: the host plan; plan_dev: its device copy.  sync:
 * DEVICE memory of AQLM_STEP_SYNC_BYTES, 16-byte aligned, zero before its
 * first use; the launch leaves it zero again (apart from the error flag after
 * a timeout), so it can be reused by the next launch on the same stream, but
 * launches that overlap must not share it.  Each level barrier polls at most
 * spin_limit times (0: AQLM_STEP_DEFAULT_SPIN, seconds of waiting) and then
 * sets the error flag; from then on every workgroup stops at its next level
 * barrier and the launch ends (outputs of the levels after the barrier that
 * gave up are not written, or only partly).  Asynchronous like the
 * other calls: check the flag with aqlm_gemv_step_status.  Returns
 * AQLM_ERR_SHAPE for a plan made for a device with another CU count, and
 * AQLM_ERR_HIP if the runtime refuses the cooperative launch. */
int aqlm_gemv_step(const void* plan_host, const void* plan_dev, void* sync, uint32_t spin_limit, void* stream);

/* Synchronizes `stream`, then reads and clears sync's error flag:
 * AQLM_ERR_TIMEOUT if a level barrier of an earlier aqlm_gemv_step on it gave
 * up, AQLM_OK otherwise. */
int aqlm_gemv_step_status(void* sync, void* stream);

/* ------------------------------------------------------- chunk-sorted codes
 *
 * A second storage of the codes of the formats with large codebooks - one or
 * two codebooks of 2^15 or 2^16 codewords, g = 8 (the 2- and 4-bit settings
 * of the appendix "Experimental Configurations") - for the matrix-vector
 * product (Sec. 4.3).  Such a codebook (1 MiB for 2^16 fp16 codewords of 8)
 * does not fit on chip, so with row-major codes every code fetches its
 * codeword from the L2 cache.  The sorted form lists, for every block of 16
 * output rows, the block's codes chunk by chunk (a chunk is 8192 consecutive
 * codewords of one codebook, 128 KiB), so that the product can stage one
 * chunk per workgroup on chip and serve each code from there.  Eq. 2 and the
 * product are unchanged; only the order in which codes are read changes.
 *
 * Layout (K = M * 2^(B-13) chunk classes; code (i, j, m) of value v is in
 * class c = m * 2^(B-13) + (v >> 13); nb = ceil(d_out / 16) row blocks):
 *   index    uint32 [K * nb + 1]: index[c * nb + b] = first step of the list
 *            of class c in block b; index[K * nb] = total steps.  The list has
 *            ceil(n / 4) steps, n the largest number of class-c codes of one
 *            row of the block.
 *   entries  uint32 [total steps * 64]: the k-th class-c code (ascending j)
 *            of row 16 b + i is entry 64 * (index[c * nb + b] + k / 4)
 *            + 16 * (k % 4) + i, stored as (v & 8191) | (j << 14); every other
 *            entry is the pad 0xFFFFE000, which adds nothing.
 * The sorted form takes about 2.5 times the bytes of 16-bit codes (4 bytes
 * per code, and pads up to the longest row of each block); the row-major
 * codes stay the input of every other entry point. */

/* Sizes of the sorted form of `codes_host` (HOST memory; layout as for
 * aqlm_gemv, unpacked uint16 or bit-packed with B | AQLM_PACKED):
 * *entry_words = total steps * 64, *index_words = K * nb + 1.  Reads every
 * code.  Supported: M = 1 or 2, B = 15 or 16, g = 8 (else
 * AQLM_ERR_UNSUPPORTED); d_in / 8 at most 262142 and the entries below 2 GiB
 * (else AQLM_ERR_SHAPE). */
int aqlm_sort_codes_size(const void* codes_host, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                         int64_t* entry_words, int64_t* index_words);

/* Writes the sorted form of `codes_host` into HOST arrays entries_host
 * [entry_words] and index_host [index_words] (at least the sizes above, else
 * AQLM_ERR_WORKSPACE).  Runs on the host (once per layer, when it is loaded);
 * the caller copies both arrays to the device for aqlm_gemv_sorted.
 * Deterministic. */
int aqlm_sort_codes(const void* codes_host, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                    uint32_t* entries_host, int64_t entry_words, uint32_t* index_host, int64_t index_words);

/* Device workspace of aqlm_gemv_sorted in bytes: 4096 bytes of counters,
 * then one 8-byte (partial sum, launch tag) word per chunk class and output
 * row (K * d_out * 8); for aqlm_gemv_sorted_grouped pass the sum of the
 * problems' d_out.  0 for an unsupported format or size. */
size_t aqlm_gemv_sorted_workspace_bytes(int64_t d_out, int32_t M, int32_t B);

/* The matrix-vector product of aqlm_gemv over sorted codes (entries, index:
 * DEVICE copies of what aqlm_sort_codes wrote for this layer; entry_words:
 * their count; index_host: the HOST array aqlm_sort_codes wrote, or NULL - when
 * given, the workgroups' first steps travel with the launch arguments instead
 * of being read from the device index first, which saves a memory round trip
 * per launch; it must hold the same values as `index`): y[i] = fp16(s_i * sum_j sum_m <C_m[b[i][j][m]], x[j*8 ..
 * j*8+8)>), fp32 accumulation.  One workgroup per (chunk class, range of row
 * blocks) stages its codebook chunk on chip; the K class sums of a row are
 * added in class order by one workgroup of its range, then scaled and rounded
 * once.  Deterministic; agrees with aqlm_gemv to fp32 accumulation accuracy
 * (the summation order differs).
 *   workspace: DEVICE memory of at least aqlm_gemv_sorted_workspace_bytes
 *   bytes, 16-byte aligned, whose first 4096 bytes (counters) are zero before
 *   its first use.  Every launch adds to the counters it uses and leaves them
 *   consistent, so one workspace, sized for the largest launch, serves any
 *   sequence of calls, for any layers and formats, on one stream; calls that
 *   may overlap (other streams) need their own workspace.  A workspace whose
 *   counters were disturbed can make the summing workgroup give up waiting
 *   for a partial sum (after about 4M polls): the rows it sums are then NaN.
 *   Entries and index are read, never written; an index or entries array that
 *   does not belong to the layer gives wrong results but no access outside
 *   the arrays (entry_words bounds every read).  Supported as for
 *   aqlm_sort_codes, with d_out up to 6553600 (else AQLM_ERR_SHAPE); entries
 *   and index 4-byte aligned, x 16-byte aligned, y 2-byte aligned. */
int aqlm_gemv_sorted(const uint32_t* entries, int64_t entry_words, const uint32_t* index, const uint32_t* index_host,
                     const uint16_t* codebooks, const uint16_t* scales, int64_t d_out, int64_t d_in, int32_t M,
                     int32_t B, int32_t g, const uint16_t* x, uint16_t* y, void* workspace, size_t workspace_bytes,
                     void* stream);

/* One problem of a grouped sorted launch (device pointers; as aqlm_gemv_sorted). */
typedef struct aqlm_sorted_problem {
  const uint32_t* entries;
  int64_t entry_words;
  const uint32_t* index;
  const uint32_t* index_host; /* HOST copy of index, or NULL (see aqlm_gemv_sorted) */
  const uint16_t* codebooks;
  const uint16_t* scales;
  const uint16_t* x; /* [d_in] */
  uint16_t* y;       /* [d_out] */
  int64_t d_out;
  int64_t d_in;
} aqlm_sorted_problem;

/* `count` (1..AQLM_MAX_GROUPED) sorted products of one format in one launch
 * (q, k, v or gate, up projections), each computed as aqlm_gemv_sorted
 * computes it; the workgroups are dealt to the problems by their entries.
 * `problems` is a HOST array read during the call; every problem is validated
 * before anything is launched.  Workspace: aqlm_gemv_sorted_workspace_bytes of
 * the summed d_out.  Deterministic; results may differ from separate calls in
 * the last bits (the row ranges differ). */
int aqlm_gemv_sorted_grouped(const aqlm_sorted_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Static text for a status code (never NULL). */
const char* aqlm_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* AQLM_MI355X_H */
