/*
 * CPU oracle for the AQLM compressed-weight format and its matrix-vector
 * product.  TEST INFRASTRUCTURE ONLY: it exists to check the GPU library.
 * Only the tests, the smoke entry point and the CPU-baseline leg of the
 * benchmark may load it; the product path never links or calls it, and it
 * shares no code, header or table with the GPU library.
 *
 * What it computes (paper: "Extreme Compression of Large Language Models via
 * Additive Quantization", Sec. 3 Eq. 2 and Fig. 3):
 *   - a row i of the weight matrix is split into groups of g consecutive
 *     inputs; group j is the sum over m = 0..M-1 of codeword b[i][j][m] of
 *     codebook C_m (Eq. 2), then the whole row is multiplied by the per-output
 *     scale s_i (Fig. 3, step v; scales per output unit in Sec. 3.3);
 *   - codebooks and scales are stored in half precision (App. "Estimating
 *     model size").
 * Numerical reading fixed here (the paper does not state one):
 *   - the M codewords are added in fp32 in ascending m, the accumulator
 *     starting from codeword 0 (so a -0 component survives when M = 1);
 *   - one fp32 multiply by the scale, then one round-to-nearest-even to fp16,
 *     fp16 subnormals kept, overflow to +-inf;
 *   - the matrix-vector product is taken in fp64, ascending input index.
 * Build with -ffp-contract=off and without -ffast-math so that every fp32
 * operation is a single IEEE operation in the stated order.
 *
 * Layouts (all dense, row-major):
 *   codes      [d_out][d_in/g][M], m fastest; uint8 when B <= 8, else uint16
 *   codebooks  [M][2^B][g] fp16 bit patterns
 *   scales     [d_out] fp16 bit patterns
 *   W          [d_out][d_in] fp16 bit patterns
 *   x          [n][d_in] fp16 bit patterns;  y [n][d_out] double
 *
 * Return values: 0 ok, 1 null pointer, 2 bad shape, 3 unsupported
 * (M, B, g), 4 a code outside [0, 2^B).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_NULL 1
#define ORC_ERR_SHAPE 2
#define ORC_ERR_UNSUPPORTED 3
#define ORC_ERR_CODE 4

/* ---- IEEE-754 binary16 <-> binary32, written from the format definition ---- */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
 * Exponent field 0 encodes zero and subnormals (value = frac * 2^-24),
 * field 31 encodes infinities (frac 0) and NaNs. */
float oracle_f16_to_f32(uint16_t h) {
  uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
  uint32_t exp = ((uint32_t)h >> 10) & 0x1Fu;
  uint32_t frac = (uint32_t)h & 0x3FFu;
  uint32_t bits;
  if (exp == 0) {
    if (frac == 0) {
      bits = sign;
    } else {
      /* subnormal: normalise frac * 2^-24 into binary32 */
      int e = -14;
      while ((frac & 0x400u) == 0) {
        frac <<= 1;
        e -= 1;
      }
      frac &= 0x3FFu;
      bits = sign | ((uint32_t)(e + 127) << 23) | (frac << 13);
    }
  } else if (exp == 31) {
    bits = sign | 0x7F800000u | (frac << 13);
  } else {
    bits = sign | ((exp - 15u + 127u) << 23) | (frac << 13);
  }
  float f;
  memcpy(&f, &bits, sizeof f);
  return f;
}

/* Round a binary32 value to the nearest binary16 value, ties to even.
 * Results below the smallest normal are produced as subnormals; magnitudes
 * that round above the largest finite value become infinity; NaN stays NaN
 * (quiet, sign kept). */
uint16_t oracle_f32_to_f16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  uint32_t sign = (u >> 16) & 0x8000u;
  uint32_t exp = (u >> 23) & 0xFFu;
  uint32_t frac = u & 0x7FFFFFu;
  if (exp == 0xFFu) {
    if (frac != 0) return (uint16_t)(sign | 0x7E00u | (frac >> 13));
    return (uint16_t)(sign | 0x7C00u);
  }
  int e = (int)exp - 127; /* unbiased exponent (fp32 subnormals give -127) */
  if (e > 15) return (uint16_t)(sign | 0x7C00u);
  if (e >= -14) {
    /* normal binary16 range: keep 10 fraction bits, round on the other 13 */
    uint32_t h = ((uint32_t)(e + 15) << 10) | (frac >> 13);
    uint32_t rest = frac & 0x1FFFu;
    if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) h += 1u; /* a carry may reach inf */
    return (uint16_t)(sign | h);
  }
  if (e < -25) return (uint16_t)sign; /* below half the smallest subnormal */
  /* subnormal result: value = sig * 2^(e-23); in units of 2^-24 that is
   * sig >> shift with shift = -(e + 1) in [14, 24] */
  uint32_t sig = frac | 0x800000u;
  int shift = -(e + 1);
  uint32_t q = sig >> shift;
  uint32_t rest = sig & ((1u << shift) - 1u);
  uint32_t half = 1u << (shift - 1);
  if (rest > half || (rest == half && (q & 1u))) q += 1u; /* may become the smallest normal */
  return (uint16_t)(sign | q);
}

void oracle_f32_to_f16_array(const float* in, uint16_t* out, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_f32_to_f16(in[i]);
}

void oracle_f16_to_f32_array(const uint16_t* in, float* out, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_f16_to_f32(in[i]);
}

/* ---- bit-packed codes ----
 * A row of packed B-bit codes is its codes in index order q = j*M + m as one
 * little-endian bit string: code q is bits [q*B, (q+1)*B) of the row, bit b
 * being bit b % 8 of byte b / 8; the row is padded with zero bits to a whole
 * number of 32-bit words, so a row takes ceil(G*M*B / 32) * 4 bytes. */
int64_t oracle_packed_row_bytes(int64_t d_in, int32_t M, int32_t B, int32_t g) {
  const int64_t bits = (d_in / g) * M * B;
  return (bits + 31) / 32 * 4;
}

/* Unpack [d_out] packed rows into codes [d_out][G][M] (uint16). */
int oracle_unpack_codes(const uint8_t* packed, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                        uint16_t* codes) {
  if (!packed || !codes) return ORC_ERR_NULL;
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0) return ORC_ERR_SHAPE;
  if (B < 1 || B > 16 || M < 1) return ORC_ERR_UNSUPPORTED;
  const int64_t n = (d_in / g) * M;
  const int64_t pitch = oracle_packed_row_bytes(d_in, M, B, g);
  for (int64_t i = 0; i < d_out; ++i)
    for (int64_t q = 0; q < n; ++q) {
      uint32_t v = 0;
      for (int32_t b = 0; b < B; ++b) {
        const int64_t bit = q * B + b;
        v |= (uint32_t)((packed[i * pitch + bit / 8] >> (bit % 8)) & 1u) << b;
      }
      codes[i * n + q] = (uint16_t)v;
    }
  return ORC_OK;
}

/* ---- dequantization (Eq. 2 with per-output scales, Fig. 3 steps i-v) ---- */

static int check_args(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                      int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g) {
  if (!codes || !codebooks || !scales) return ORC_ERR_NULL;
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0) return ORC_ERR_SHAPE;
  if (M < 1 || M > 64 || B < 1 || B > 16) return ORC_ERR_UNSUPPORTED;
  return ORC_OK;
}

static inline uint32_t code_at(const void* codes, int32_t B, int64_t idx) {
  if (B <= 8) return ((const uint8_t*)codes)[idx];
  return ((const uint16_t*)codes)[idx];
}

/* One output row i of the dequantized matrix into w_row[0..d_in). */
static int dequant_row(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                       int64_t i, int64_t d_in, int32_t M, int32_t B, int32_t g, uint16_t* w_row) {
  const int64_t groups = d_in / g;
  const int64_t entries = (int64_t)1 << B;
  const float s = oracle_f16_to_f32(scales[i]);
  for (int64_t j = 0; j < groups; ++j) {
    const int64_t code_base = (i * groups + j) * M;
    for (int32_t k = 0; k < g; ++k) {
      float acc = 0.0f;
      for (int32_t m = 0; m < M; ++m) {
        const uint32_t c = code_at(codes, B, code_base + m);
        if ((int64_t)c >= entries) return ORC_ERR_CODE;
        const float v = oracle_f16_to_f32(codebooks[((int64_t)m * entries + c) * g + k]);
        if (m == 0)
          acc = v;
        else
          acc = acc + v;
      }
      const float t = acc * s;
      w_row[j * g + k] = oracle_f32_to_f16(t);
    }
  }
  return ORC_OK;
}

int oracle_dequantize(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                      int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, uint16_t* w_out) {
  int st = check_args(codes, codebooks, scales, d_out, d_in, M, B, g);
  if (st != ORC_OK) return st;
  if (!w_out) return ORC_ERR_NULL;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t i = 0; i < d_out; ++i)
    bad |= dequant_row(codes, codebooks, scales, i, d_in, M, B, g, w_out + i * d_in) != ORC_OK;
  return bad ? ORC_ERR_CODE : ORC_OK;
}

/* Dequantize only the listed rows: w_out is [n_rows][d_in]. */
int oracle_dequantize_rows(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                           int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                           const int64_t* rows, int64_t n_rows, uint16_t* w_out) {
  int st = check_args(codes, codebooks, scales, d_out, d_in, M, B, g);
  if (st != ORC_OK) return st;
  if (!w_out || !rows) return ORC_ERR_NULL;
  for (int64_t r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= d_out) return ORC_ERR_SHAPE;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t r = 0; r < n_rows; ++r)
    bad |= dequant_row(codes, codebooks, scales, rows[r], d_in, M, B, g, w_out + r * d_in) != ORC_OK;
  return bad ? ORC_ERR_CODE : ORC_OK;
}

/* ---- dense products on the dequantized fp16 matrix, in fp64 ---- */

/* y[t][i] = sum over c ascending of W[i][c] * x[t][c], every product and sum in
 * fp64 (the product of two fp16 values is exact in fp64). */
int oracle_matmul_f16(const uint16_t* w, int64_t d_out, int64_t d_in, const uint16_t* x, int64_t n,
                      double* y) {
  if (!w || !x || !y) return ORC_ERR_NULL;
  if (d_out <= 0 || d_in <= 0 || n <= 0) return ORC_ERR_SHAPE;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < d_out; ++i) {
    const uint16_t* wr = w + i * d_in;
    for (int64_t t = 0; t < n; ++t) {
      const uint16_t* xr = x + t * d_in;
      double acc = 0.0;
      for (int64_t c = 0; c < d_in; ++c)
        acc = acc + (double)oracle_f16_to_f32(wr[c]) * (double)oracle_f16_to_f32(xr[c]);
      y[t * d_out + i] = acc;
    }
  }
  return ORC_OK;
}

/* ---- gradients through Eq. 2 (the codebook and scale updates of Sec. 3,
 * "Phase 2" and "Phase 3", and end-to-end fine-tuning) ----
 *
 * For y[t][i] = sum_c W[i][c] x[t][c] with W given by Eq. 2 and the scales
 * (W[i][j*g + k] = s_i * u[i][j*g + k], u the sum over m of codeword
 * b[i][j][m] of codebook m), and an upstream gradient dy = dL/dy, the chain
 * rule gives, with G[i][c] = dL/dW[i][c] = sum_t dy[t][i] x[t][c]:
 *   dL/dC_m[e][k] = sum over (i, j) with b[i][j][m] = e of s_i * G[i][j*g + k]
 *   dL/ds_i       = sum_c G[i][c] * u[i][c]
 * u is the fp32 sum of the codewords in ascending m (the sum the weights are
 * rounded from; the rounding itself is not differentiated).  Everything else
 * is fp64: G sums over t ascending, then i and c ascending.  dcodebooks is
 * [M][2^B][g], dscales [d_out]; both are written (not accumulated). */
int oracle_backward(const void* codes, const uint16_t* codebooks, const uint16_t* scales,
                    int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n,
                    const uint16_t* x, const uint16_t* dy, double* dcodebooks, double* dscales) {
  int st = check_args(codes, codebooks, scales, d_out, d_in, M, B, g);
  if (st != ORC_OK) return st;
  if (!x || !dy || !dcodebooks || !dscales) return ORC_ERR_NULL;
  if (n <= 0) return ORC_ERR_SHAPE;
  const int64_t groups = d_in / g;
  const int64_t entries = (int64_t)1 << B;
  const int64_t ncb = (int64_t)M * entries * g;
  for (int64_t e = 0; e < ncb; ++e) dcodebooks[e] = 0.0;
  for (int64_t i = 0; i < d_out; ++i) {
    const double s = (double)oracle_f16_to_f32(scales[i]);
    double ds = 0.0;
    for (int64_t j = 0; j < groups; ++j) {
      const int64_t code_base = (i * groups + j) * M;
      for (int32_t m = 0; m < M; ++m)
        if ((int64_t)code_at(codes, B, code_base + m) >= entries) return ORC_ERR_CODE;
      for (int32_t k = 0; k < g; ++k) {
        const int64_t c = j * g + k;
        double G = 0.0;
        for (int64_t t = 0; t < n; ++t)
          G = G + (double)oracle_f16_to_f32(dy[t * d_out + i]) * (double)oracle_f16_to_f32(x[t * d_in + c]);
        float u = 0.0f;
        for (int32_t m = 0; m < M; ++m) {
          const uint32_t b = code_at(codes, B, code_base + m);
          const float v = oracle_f16_to_f32(codebooks[((int64_t)m * entries + b) * g + k]);
          u = (m == 0) ? v : u + v;
          dcodebooks[((int64_t)m * entries + b) * g + k] += s * G;
        }
        ds = ds + G * (double)u;
      }
    }
    dscales[i] = ds;
  }
  return ORC_OK;
}

/* ---- Phase 1: beam search over codes (Sec. 3, "Phase 1: Beam search for
 * codes"; the codes step of the algorithm listing) ----
 *
 * Row i's objective is the squared error of Eq. main_obj restricted to that
 * row, written with H = X X^T as in Eq. obj_mrf:
 *   L_i(b) = (w_i - what_i) H (w_i - what_i)^T,
 *   what_i[j*g + t] = s_i * sum_m C_m[b_ijm][t]   (exact, no fp16 rounding).
 * Rows are independent.  A beam of at most k configurations of the row's
 * codes starts as the current codes alone.  One step takes one code position
 * (j, m) - positions are swept group by group, codebooks in ascending order
 * within a group - and tries, for every configuration of the beam, every
 * codeword e of codebook m at that position; the beam becomes the k
 * distinct configurations of least loss among those candidates (ties: the
 * earlier beam entry, then the smaller e).  Setting a position to its current
 * code keeps a configuration, so the best loss never increases.  A
 * candidate's loss is the previous loss plus the change of the terms that
 * involve group j: with r = w - what and delta = s (C_m[e] - C_m[b_ijm]) on
 * group j's g coordinates,
 *   L' = L - 2 delta . (H r)_j + delta H_jj delta^T.
 * H r is recomputed from r for every configuration at every step.  After
 * `sweeps` sweeps the best configuration is the result.  Everything in fp64
 * (W, H, codebooks and scales as given).  codes is read and overwritten;
 * loss_out[i] receives the final loss of row i. */

typedef struct {
  double score;
  int32_t beam;
  int32_t code;
} orc_cand;

static int orc_cand_cmp(const void* pa, const void* pb) {
  const orc_cand* a = (const orc_cand*)pa;
  const orc_cand* b = (const orc_cand*)pb;
  if (a->score < b->score) return -1;
  if (a->score > b->score) return 1;
  if (a->beam != b->beam) return a->beam < b->beam ? -1 : 1;
  return a->code < b->code ? -1 : (a->code > b->code ? 1 : 0);
}

static void set_code(void* codes, int32_t B, int64_t idx, uint32_t v) {
  if (B <= 8)
    ((uint8_t*)codes)[idx] = (uint8_t)v;
  else
    ((uint16_t*)codes)[idx] = (uint16_t)v;
}

/* The loss of row i of the given codes: (w - what) H (w - what)^T in fp64. */
static double row_loss(const float* w_row, const float* h, const void* codes_row, const uint16_t* codebooks,
                       double s, int64_t d_in, int32_t M, int32_t B, int32_t g, double* r) {
  const int64_t groups = d_in / g;
  const int64_t entries = (int64_t)1 << B;
  for (int64_t j = 0; j < groups; ++j)
    for (int32_t t = 0; t < g; ++t) {
      double u = 0.0;
      for (int32_t m = 0; m < M; ++m) {
        const uint32_t b = code_at(codes_row, B, j * M + m);
        u += (double)oracle_f16_to_f32(codebooks[((int64_t)m * entries + b) * g + t]);
      }
      r[j * g + t] = (double)w_row[j * g + t] - s * u;
    }
  double loss = 0.0;
  for (int64_t a = 0; a < d_in; ++a) {
    double hr = 0.0;
    for (int64_t c = 0; c < d_in; ++c) hr += (double)h[a * d_in + c] * r[c];
    loss += r[a] * hr;
  }
  return loss;
}

int oracle_aq_loss(const float* w, const float* h, const void* codes, const uint16_t* codebooks,
                   const uint16_t* scales, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                   double* loss_out) {
  int st = check_args(codes, codebooks, scales, d_out, d_in, M, B, g);
  if (st != ORC_OK) return st;
  if (!w || !h || !loss_out) return ORC_ERR_NULL;
  const int64_t groups = d_in / g;
  int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
  for (int64_t i = 0; i < d_out; ++i) {
    double* r = (double*)malloc(sizeof(double) * d_in);
    if (!r) { bad = 1; continue; }
    const void* row = (B <= 8) ? (const void*)((const uint8_t*)codes + i * groups * M)
                               : (const void*)((const uint16_t*)codes + i * groups * M);
    loss_out[i] = row_loss(w + i * d_in, h, row, codebooks, (double)oracle_f16_to_f32(scales[i]), d_in, M, B, g, r);
    free(r);
  }
  return bad ? ORC_ERR_NULL : ORC_OK;
}

int oracle_beam_search(const float* w, const float* h, void* codes, const uint16_t* codebooks,
                       const uint16_t* scales, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                       int32_t beam, int32_t sweeps, double* loss_out) {
  int st = check_args(codes, codebooks, scales, d_out, d_in, M, B, g);
  if (st != ORC_OK) return st;
  if (!w || !h || !loss_out) return ORC_ERR_NULL;
  if (beam < 1 || sweeps < 0) return ORC_ERR_SHAPE;
  if (g > 64) return ORC_ERR_UNSUPPORTED;
  const int64_t groups = d_in / g;
  const int64_t entries = (int64_t)1 << B;
  const int64_t ncodes = groups * M;
  const size_t cb = (B <= 8) ? 1 : 2;
  for (int64_t e = 0; e < d_out * ncodes; ++e)
    if ((int64_t)code_at(codes, B, e) >= entries) return ORC_ERR_CODE;
  int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
  for (int64_t i = 0; i < d_out; ++i) {
    const double s = (double)oracle_f16_to_f32(scales[i]);
    const float* w_row = w + i * d_in;
    void* out_row = (char*)codes + (size_t)(i * ncodes) * cb;
    /* beam state: codes, residual r = w - what, loss; two generations */
    unsigned char* bc[2];
    double* br[2];
    double* bl[2];
    double* hr = (double*)malloc(sizeof(double) * d_in);
    orc_cand* cand = (orc_cand*)malloc(sizeof(orc_cand) * (size_t)(beam * entries));
    int ok = hr && cand;
    for (int q = 0; q < 2; ++q) {
      bc[q] = (unsigned char*)malloc((size_t)(beam * ncodes) * cb);
      br[q] = (double*)malloc(sizeof(double) * (size_t)(beam * d_in));
      bl[q] = (double*)malloc(sizeof(double) * (size_t)beam);
      ok = ok && bc[q] && br[q] && bl[q];
    }
    if (!ok) {
      bad = 1;
    } else {
      int cur = 0, nb = 1;
      memcpy(bc[0], out_row, (size_t)ncodes * cb);
      bl[0][0] = row_loss(w_row, h, bc[0], codebooks, s, d_in, M, B, g, br[0]);
      for (int32_t sw = 0; sw < sweeps; ++sw)
        for (int64_t j = 0; j < groups; ++j)
          for (int32_t m = 0; m < M; ++m) {
            const int64_t pos = j * M + m;
            int nc = 0;
            for (int b = 0; b < nb; ++b) {
              const unsigned char* cfg = bc[cur] + (size_t)(b * ncodes) * cb;
              const double* r = br[cur] + (size_t)b * d_in;
              for (int32_t t = 0; t < g; ++t) {
                double acc = 0.0;
                for (int64_t c = 0; c < d_in; ++c) acc += (double)h[(j * g + t) * d_in + c] * r[c];
                hr[j * g + t] = acc;
              }
              const uint32_t o = code_at(cfg, B, pos);
              for (int64_t e = 0; e < entries; ++e) {
                double delta[64];
                for (int32_t t = 0; t < g; ++t)
                  delta[t] = s * ((double)oracle_f16_to_f32(codebooks[((int64_t)m * entries + e) * g + t]) -
                                  (double)oracle_f16_to_f32(codebooks[((int64_t)m * entries + o) * g + t]));
                double lin = 0.0, quad = 0.0;
                for (int32_t t = 0; t < g; ++t) {
                  lin += delta[t] * hr[j * g + t];
                  double hd = 0.0;
                  for (int32_t u = 0; u < g; ++u) hd += (double)h[(j * g + t) * d_in + j * g + u] * delta[u];
                  quad += delta[t] * hd;
                }
                cand[nc].score = bl[cur][b] - 2.0 * lin + quad;
                cand[nc].beam = b;
                cand[nc].code = (int32_t)e;
                ++nc;
              }
            }
            qsort(cand, (size_t)nc, sizeof(orc_cand), orc_cand_cmp);
            const int nxt = 1 - cur;
            int nn = 0;
            for (int q = 0; q < nc && nn < beam; ++q) {
              unsigned char* dst = bc[nxt] + (size_t)(nn * ncodes) * cb;
              memcpy(dst, bc[cur] + (size_t)(cand[q].beam * ncodes) * cb, (size_t)ncodes * cb);
              set_code(dst, B, pos, (uint32_t)cand[q].code);
              int dup = 0;
              for (int p2 = 0; p2 < nn && !dup; ++p2)
                dup = memcmp(dst, bc[nxt] + (size_t)(p2 * ncodes) * cb, (size_t)ncodes * cb) == 0;
              if (dup) continue;
              /* residual of the new configuration: only group j changes */
              const double* rsrc = br[cur] + (size_t)cand[q].beam * d_in;
              double* rdst = br[nxt] + (size_t)nn * d_in;
              memcpy(rdst, rsrc, sizeof(double) * (size_t)d_in);
              const uint32_t o = code_at(bc[cur] + (size_t)(cand[q].beam * ncodes) * cb, B, pos);
              for (int32_t t = 0; t < g; ++t)
                rdst[j * g + t] -= s * ((double)oracle_f16_to_f32(codebooks[((int64_t)m * entries + cand[q].code) * g + t]) -
                                        (double)oracle_f16_to_f32(codebooks[((int64_t)m * entries + o) * g + t]));
              bl[nxt][nn] = cand[q].score;
              ++nn;
            }
            cur = nxt;
            nb = nn;
          }
      memcpy(out_row, bc[cur], (size_t)ncodes * cb);
      loss_out[i] = bl[cur][0];
    }
    for (int q = 0; q < 2; ++q) {
      free(bc[q]);
      free(br[q]);
      free(bl[q]);
    }
    free(hr);
    free(cand);
  }
  return bad ? ORC_ERR_NULL : ORC_OK;
}

#ifdef _OPENMP
#include <omp.h>
#endif
/* Threads a parallel region of the loops above actually runs with (1 without
 * OpenMP). */
int oracle_num_threads(void) {
  int n = 1;
#ifdef _OPENMP
#pragma omp parallel
  {
#pragma omp single
    n = omp_get_num_threads();
  }
#endif
  return n;
}

/* Threads for later parallel regions started from the calling thread
 * (n >= 1; ignored without OpenMP). */
void oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
