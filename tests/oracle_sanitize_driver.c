/*
 * Runs every function of the CPU oracle on small random inputs, on its error
 * paths, and on the edge shapes the tests use, so that a build of the oracle
 * with AddressSanitizer and UndefinedBehaviorSanitizer sees every code path
 * (out-of-bounds reads or writes, signed overflow, misaligned or invalid
 * shifts, use of uninitialised heap memory through ASan's poisoning).  It
 * also checks a few cheap identities, but the pins that fix the oracle's
 * values live in test_oracle_pins.py; this program is about memory and UB.
 * Exit status 0: every call behaved; a sanitizer report aborts with non-zero.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

float oracle_f16_to_f32(uint16_t h);
uint16_t oracle_f32_to_f16(float f);
void oracle_f32_to_f16_array(const float* in, uint16_t* out, int64_t n);
void oracle_f16_to_f32_array(const uint16_t* in, float* out, int64_t n);
int64_t oracle_packed_row_bytes(int64_t d_in, int32_t M, int32_t B, int32_t g);
int oracle_unpack_codes(const uint8_t* packed, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                        uint16_t* codes);
int oracle_dequantize(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                      int64_t d_in, int32_t M, int32_t B, int32_t g, uint16_t* w_out);
int oracle_dequantize_rows(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                           int64_t d_in, int32_t M, int32_t B, int32_t g, const int64_t* rows, int64_t n_rows,
                           uint16_t* w_out);
int oracle_matmul_f16(const uint16_t* w, int64_t d_out, int64_t d_in, const uint16_t* x, int64_t n, double* y);
int oracle_backward(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                    int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, const uint16_t* dy,
                    double* dcodebooks, double* dscales);
int oracle_aq_loss(const float* w, const float* h, const void* codes, const uint16_t* codebooks,
                   const uint16_t* scales, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                   double* loss_out);
int oracle_beam_search(const float* w, const float* h, void* codes, const uint16_t* codebooks,
                       const uint16_t* scales, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                       int32_t beam, int32_t sweeps, double* loss_out);
int oracle_num_threads(void);
void oracle_set_threads(int n);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd(void) {
  rng_state = rng_state * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(rng_state >> 33);
}
static float rnd_unit(void) { return (float)(rnd() & 0xFFFFFF) / (float)0x1000000 - 0.5f; }

static int failures = 0;
#define CHECK(cond, ...)                     \
  do {                                       \
    if (!(cond)) {                           \
      fprintf(stderr, "FAILED: " __VA_ARGS__); \
      fprintf(stderr, "\n");                 \
      ++failures;                            \
    }                                        \
  } while (0)

/* Exactly-sized heap buffers, so that ASan catches any access one past them. */
static void* xmalloc(size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p) {
    fprintf(stderr, "out of memory\n");
    exit(2);
  }
  return p;
}

static void fill_codes(void* codes, int64_t count, int32_t B) {
  for (int64_t i = 0; i < count; ++i) {
    const uint32_t v = rnd() & ((1u << B) - 1u);
    if (B <= 8)
      ((uint8_t*)codes)[i] = (uint8_t)v;
    else
      ((uint16_t*)codes)[i] = (uint16_t)v;
  }
}

static void fill_f16(uint16_t* a, int64_t n, float scale) {
  for (int64_t i = 0; i < n; ++i) a[i] = oracle_f32_to_f16(rnd_unit() * scale);
}

/* Bit-packs codes [d_out][G*M] (uint16) the way the library does: a little-
 * endian bit string per row, padded to whole 32-bit words. */
static void pack(const uint16_t* codes, int64_t d_out, int64_t per_row, int32_t B, uint8_t* out, int64_t pitch) {
  memset(out, 0, (size_t)(d_out * pitch));
  for (int64_t r = 0; r < d_out; ++r)
    for (int64_t q = 0; q < per_row; ++q)
      for (int32_t b = 0; b < B; ++b)
        if ((codes[r * per_row + q] >> b) & 1u) {
          const int64_t bit = q * B + b;
          out[r * pitch + bit / 8] |= (uint8_t)(1u << (bit % 8));
        }
}

static void run_format(int32_t M, int32_t B, int32_t g, int64_t d_out, int64_t d_in) {
  const int64_t groups = d_in / g, entries = (int64_t)1 << B, ncodes = d_out * groups * M;
  const size_t cb_bytes = B <= 8 ? 1 : 2;
  void* codes = xmalloc((size_t)ncodes * cb_bytes);
  uint16_t* cbk = xmalloc(sizeof(uint16_t) * (size_t)(M * entries * g));
  uint16_t* sc = xmalloc(sizeof(uint16_t) * (size_t)d_out);
  uint16_t* w = xmalloc(sizeof(uint16_t) * (size_t)(d_out * d_in));
  fill_codes(codes, ncodes, B);
  fill_f16(cbk, M * entries * g, 0.1f);
  fill_f16(sc, d_out, 2.0f);
  CHECK(oracle_dequantize(codes, cbk, sc, d_out, d_in, M, B, g, w) == 0, "dequantize %dx%d g%d", M, B, g);

  /* rows: first, last and a middle one, compared with the full result */
  const int64_t rows[3] = {0, d_out - 1, d_out / 2};
  uint16_t* wr = xmalloc(sizeof(uint16_t) * (size_t)(3 * d_in));
  CHECK(oracle_dequantize_rows(codes, cbk, sc, d_out, d_in, M, B, g, rows, 3, wr) == 0, "rows");
  for (int r = 0; r < 3; ++r)
    CHECK(memcmp(wr + r * d_in, w + rows[r] * d_in, sizeof(uint16_t) * (size_t)d_in) == 0, "rows equal full");
  const int64_t bad_row[1] = {d_out};
  CHECK(oracle_dequantize_rows(codes, cbk, sc, d_out, d_in, M, B, g, bad_row, 1, wr) == 2, "row past end");

  /* products and gradients with n = 3 tokens */
  const int64_t n = 3;
  uint16_t* x = xmalloc(sizeof(uint16_t) * (size_t)(n * d_in));
  uint16_t* dy = xmalloc(sizeof(uint16_t) * (size_t)(n * d_out));
  double* y = xmalloc(sizeof(double) * (size_t)(n * d_out));
  fill_f16(x, n * d_in, 2.0f);
  fill_f16(dy, n * d_out, 2.0f);
  CHECK(oracle_matmul_f16(w, d_out, d_in, x, n, y) == 0, "matmul");
  double* dcb = xmalloc(sizeof(double) * (size_t)(M * entries * g));
  double* ds = xmalloc(sizeof(double) * (size_t)d_out);
  CHECK(oracle_backward(codes, cbk, sc, d_out, d_in, M, B, g, n, x, dy, dcb, ds) == 0, "backward");

  /* objective and beam search (small codebooks only: 2^B candidates per step) */
  float* wf = xmalloc(sizeof(float) * (size_t)(d_out * d_in));
  float* h = xmalloc(sizeof(float) * (size_t)(d_in * d_in));
  for (int64_t i = 0; i < d_out * d_in; ++i) wf[i] = rnd_unit() * 0.1f;
  for (int64_t a = 0; a < d_in; ++a)
    for (int64_t c = 0; c <= a; ++c) h[a * d_in + c] = h[c * d_in + a] = (a == c) ? 2.0f : rnd_unit() * 0.1f;
  double* loss = xmalloc(sizeof(double) * (size_t)d_out);
  double* loss2 = xmalloc(sizeof(double) * (size_t)d_out);
  CHECK(oracle_aq_loss(wf, h, codes, cbk, sc, d_out, d_in, M, B, g, loss) == 0, "aq_loss");
  if (B <= 8 && g <= 64) {
    for (int32_t beam = 1; beam <= 3; ++beam) {
      void* c2 = xmalloc((size_t)ncodes * cb_bytes);
      memcpy(c2, codes, (size_t)ncodes * cb_bytes);
      CHECK(oracle_beam_search(wf, h, c2, cbk, sc, d_out, d_in, M, B, g, beam, 1, loss2) == 0, "beam %d", beam);
      double* exact = xmalloc(sizeof(double) * (size_t)d_out);
      CHECK(oracle_aq_loss(wf, h, c2, cbk, sc, d_out, d_in, M, B, g, exact) == 0, "loss after beam");
      for (int64_t i = 0; i < d_out; ++i)
        CHECK(fabs(exact[i] - loss2[i]) <= 1e-6 * (fabs(exact[i]) + 1.0), "beam loss is the objective");
      free(exact);
      free(c2);
    }
  }

  /* packed codes: round trip through the library's layout (B > 8 formats) */
  if (B > 8) {
    const int64_t pitch = oracle_packed_row_bytes(d_in, M, B, g);
    CHECK(pitch % 4 == 0 && pitch * 8 >= groups * M * B, "packed pitch");
    uint8_t* pk = xmalloc((size_t)(d_out * pitch));
    uint16_t* back = xmalloc(sizeof(uint16_t) * (size_t)ncodes);
    pack((const uint16_t*)codes, d_out, groups * M, B, pk, pitch);
    CHECK(oracle_unpack_codes(pk, d_out, d_in, M, B, g, back) == 0, "unpack");
    CHECK(memcmp(back, codes, sizeof(uint16_t) * (size_t)ncodes) == 0, "packed round trip");
    free(pk);
    free(back);
  }

  /* error paths: out-of-range codes, NULLs, shapes */
  if (B < 16) {
    if (B <= 8)
      ((uint8_t*)codes)[ncodes - 1] = (uint8_t)(entries & 0xFF ? entries : 0xFF);
    else
      ((uint16_t*)codes)[ncodes - 1] = (uint16_t)entries;
    if (B < 8 || B > 8) {
      CHECK(oracle_dequantize(codes, cbk, sc, d_out, d_in, M, B, g, w) == 4, "code out of range");
      CHECK(oracle_backward(codes, cbk, sc, d_out, d_in, M, B, g, n, x, dy, dcb, ds) == 4, "backward code range");
    }
  }
  CHECK(oracle_dequantize(NULL, cbk, sc, d_out, d_in, M, B, g, w) == 1, "null codes");
  CHECK(oracle_dequantize(codes, cbk, sc, d_out, d_in + 1, M, B, g, w) == 2, "ragged d_in");
  CHECK(oracle_matmul_f16(w, d_out, d_in, x, 0, y) == 2, "n = 0");
  CHECK(oracle_beam_search(wf, h, codes, cbk, sc, d_out, d_in, M, B, g, 0, 1, loss2) == 2, "beam 0");

  free(codes);
  free(cbk);
  free(sc);
  free(w);
  free(wr);
  free(x);
  free(dy);
  free(y);
  free(dcb);
  free(ds);
  free(wf);
  free(h);
  free(loss);
  free(loss2);
}

int main(void) {
  /* fp16 conversions over every pattern and a spread of fp32 patterns */
  for (uint32_t hbits = 0; hbits < 0x10000u; ++hbits) {
    const float f = oracle_f16_to_f32((uint16_t)hbits);
    const uint16_t back = oracle_f32_to_f16(f);
    if ((hbits & 0x7C00u) != 0x7C00u || (hbits & 0x3FFu) == 0) CHECK(back == hbits, "f16 round trip %04x", hbits);
  }
  for (uint32_t i = 0; i < (1u << 20); ++i) {
    uint32_t bits = rnd() ^ (i << 12);
    float f;
    memcpy(&f, &bits, sizeof(f));
    (void)oracle_f32_to_f16(f);
  }
  float arr[5] = {0.f, -0.f, 1.f, 65504.f, 1e-8f};
  uint16_t out16[5];
  float back32[5];
  oracle_f32_to_f16_array(arr, out16, 5);
  oracle_f16_to_f32_array(out16, back32, 5);
  CHECK(back32[2] == 1.f && back32[3] == 65504.f, "array conversions");

  oracle_set_threads(1);
  CHECK(oracle_num_threads() >= 1, "threads");

  static const int32_t formats[][2] = {{1, 8}, {2, 8}, {3, 8}, {8, 8}, {2, 4}, {2, 12}, {1, 15}, {2, 15},
                                       {1, 16}, {2, 16}};
  for (size_t f = 0; f < sizeof(formats) / sizeof(formats[0]); ++f) {
    const int32_t M = formats[f][0], B = formats[f][1];
    run_format(M, B, 8, 5, 40);  /* ragged: d_in / 8 = 5 groups */
    run_format(M, B, 8, 1, 8);   /* one group */
    if (B <= 8) run_format(M, B, 4, 3, 12);
  }
  run_format(2, 8, 16, 4, 64);
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("oracle sanitizer run: all checks passed\n");
  return 0;
}
