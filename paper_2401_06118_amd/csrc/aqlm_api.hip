// C ABI of the library (declared in include/aqlm.h): argument validation and
// dispatch.  Every check runs on the host before any launch; on an error
// nothing is launched.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <mutex>
#include <set>
#include <tuple>

#include "../../include/aqlm.h"
#include "groups.h"
#include "launch.h"
#include "sorted.h"

namespace aqlm {

// Compute units of the current device (cached per device; the work split
// of every launch is sized by it).
int num_cus() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cached[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  const bool cacheable = dev >= 0 && dev < kMaxDevices;
  if (cacheable) {
    const int v = cached[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return 256;
  const int v = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
  if (cacheable) cached[dev].store(v, std::memory_order_relaxed);
  return v;
}

// The dynamic-LDS limit is a per-device property of a kernel: raise it once
// per (kernel, device, size), under a lock so that concurrent first calls
// are safe.
hipError_t allow_dynamic_lds(const void* kern, int bytes) {
  int dev = 0;
  const hipError_t d = hipGetDevice(&dev);
  if (d != hipSuccess) return d;
  static std::mutex mu;
  static std::set<std::tuple<const void*, int, int>> done;
  const std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(kern, dev, bytes);
  if (done.count(key)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess) done.insert(key);
  return e;
}

}  // namespace aqlm

namespace {

// Scratch of aqlm_gemm_noalloc: one fixed buffer per device, allocated with
// the library's code object and held until the process ends.  Host code never
// uses the array's name as an address (on the host it is only a stand-in):
// the device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = AQLM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

// Device address of this device's scratch array (nullptr on a HIP error),
// looked up on the first call on each device, with that device current.
void* scratch_ptr() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  static std::mutex mu;
  static void* ptrs[kMaxDevices] = {};
  const std::lock_guard<std::mutex> lock(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return nullptr;
    ptrs[dev] = p;
  }
  return ptrs[dev];
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// allow_packed: the entry point takes bit-packed codes (B | AQLM_PACKED).
int check_layer(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out, int64_t d_in,
                int32_t M, int32_t B, int32_t g, aqlm::Layer* L, bool allow_packed = false) {
  if (!codes || !codebooks || !scales) return AQLM_ERR_NULL;
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0) return AQLM_ERR_SHAPE;
  if (g != 8) return AQLM_ERR_UNSUPPORTED;
  const bool packed = (B & AQLM_PACKED) != 0;
  B &= ~AQLM_PACKED;
  if (packed && (!allow_packed || !aqlm::packed_supported(M, B))) return AQLM_ERR_UNSUPPORTED;
  if (!aqlm::format_supported(M, B)) return AQLM_ERR_UNSUPPORTED;
  const int64_t G = d_in / g;
  // (sizes and offsets are held in 32 bits on the device side)
  if (d_out >= (int64_t(1) << 31) || d_in >= (int64_t(1) << 31) || d_out * G >= (int64_t(1) << 31))
    return AQLM_ERR_SHAPE;
  // (bit offsets within a packed row are held in 32 bits)
  if (packed && G * M * B >= (int64_t(1) << 32)) return AQLM_ERR_SHAPE;
  if (!aligned(codes, 16) || !aligned(codebooks, 16) || !aligned(scales, 2)) return AQLM_ERR_ALIGN;
  L->codes = codes;
  L->codebooks = codebooks;
  L->scales = scales;
  L->d_out = (int32_t)d_out;
  L->d_in = (int32_t)d_in;
  L->G = (int32_t)G;
  L->M = M;
  L->B = B;
  const int64_t pitch = G * M * (B > 8 ? 2 : 1);
  L->packed = packed;
  L->vec_codes = packed || (pitch % 16) == 0;  // (packed rows are read as 32-bit words)
  return AQLM_OK;
}

int status_of(hipError_t e) { return e == hipSuccess ? AQLM_OK : AQLM_ERR_HIP; }

// Groups of 16, 32 or 64 inputs (8-bit codes, up to 16 codebooks): validated
// here and served by the group kernels (csrc/groups.hip).
int check_group_layer(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                      int64_t d_in, int32_t M, int32_t B, int32_t g, aqlm::GroupLayer* L) {
  if (!codes || !codebooks || !scales) return AQLM_ERR_NULL;
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0) return AQLM_ERR_SHAPE;
  if (!aqlm::groups_supported(M, B, g)) return AQLM_ERR_UNSUPPORTED;
  // (8-input chunks of the whole matrix are counted in 32 bits)
  if (d_out >= (int64_t(1) << 31) || d_in >= (int64_t(1) << 31) || d_out * (d_in / 8) >= (int64_t(1) << 31))
    return AQLM_ERR_SHAPE;
  if (!aligned(codes, 16) || !aligned(codebooks, 16) || !aligned(scales, 2)) return AQLM_ERR_ALIGN;
  *L = aqlm::GroupLayer{static_cast<const uint8_t*>(codes), codebooks, scales, (int32_t)d_out, (int32_t)d_in, M, g};
  return AQLM_OK;
}

// A validated layer of either kind: groups of 8 (every kernel) or larger
// groups (the group kernels only).
struct AnyLayer {
  bool big = false;
  aqlm::Layer L{};
  aqlm::GroupLayer GL{};
  int64_t d_out() const { return big ? GL.d_out : L.d_out; }
  int64_t d_in() const { return big ? GL.d_in : L.d_in; }
};

// Above this many tokens the dequantize-then-multiply prefill kernel is used
// (up to kChunkedMax tokens in chunks of kSmallBatchMax when the small-batch
// kernel covers the format: its time barely grows up to 16 tokens, while the
// prefill kernel's is flat from 17 to 256 tokens at about four times that).
constexpr int64_t kSmallBatchMax = 16;
constexpr int64_t kChunkedMax = 64;
// 1x16 takes the general tiled kernel per chunk, whose time grows faster
// with the token count: chunks pay off up to two of them.
constexpr int64_t kChunkedMax16 = 32;

// Rows from which two wide codebooks take the prefill kernel.
constexpr int64_t kPrefillMin2x12 = 192;
constexpr int64_t kPrefillMin2xWide = 96;

// From this many tokens aqlm_gemm dequantizes the whole matrix into the
// caller's workspace once and runs the dense product (when d_in allows it).
constexpr int64_t kTwoPassMin = 64;

bool two_pass(int64_t d_in, int64_t n) { return n >= kTwoPassMin && aqlm::gemm_f16_supported((int32_t)d_in); }

// The dequantized weights, rounded up to 256 bytes so that the partial sums
// that follow them in the workspace stay aligned.
size_t ws_weight_bytes(int64_t d_out, int64_t d_in) {
  return ((size_t)d_out * (size_t)d_in * sizeof(uint16_t) + 255) & ~(size_t)255;
}

int check_tokens(const uint16_t* x, uint16_t* y, int64_t n, int64_t d_in) {
  if (!x || !y) return AQLM_ERR_NULL;
  if (n <= 0 || n >= (int64_t(1) << 31) || n * d_in >= (int64_t(1) << 40)) return AQLM_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(y, 16)) return AQLM_ERR_ALIGN;
  return AQLM_OK;
}

// n = 1: the matrix-core (codeword gather) kernel for M in {1, 2, 4}
// (B = 8) and 1x16 when x fits in its LDS staging (d_in up to 32768 for 8-bit
// codes, 65536 for 16-bit); the vector-ALU kernel otherwise.  The
// partial-product-table kernel is never chosen here: measured on every
// Llama-2-7B and 70B launch and on a 65536 x 8192 layer it was no faster (4-7 %
// slower where a table is shared by 224-256 rows, 1.4-3x slower with fewer),
// so it runs only when a caller asks for it (aqlm_gemv_grouped_path).
hipError_t gemv_dispatch(const aqlm::Layer& L, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (aqlm::gemv_mfma_supported(L.M, L.B) && aqlm::gemv_mfma_fits(&L, 1))
    return aqlm::launch_gemv_mfma(&L, &x, &y, 1, s);
  return aqlm::launch_gemv(L, x, y, s);
}


int gemm_dispatch(const aqlm::Layer& L, int64_t n, const uint16_t* x, uint16_t* y, hipStream_t s);

int check_any(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out, int64_t d_in,
              int32_t M, int32_t B, int32_t g, AnyLayer* A, bool allow_packed = false) {
  if (g != 8 && g > 0 && (B & AQLM_PACKED) == 0 && aqlm::groups_supported(M, B, g)) {
    A->big = true;
    return check_group_layer(codes, codebooks, scales, d_out, d_in, M, B, g, &A->GL);
  }
  A->big = false;
  return check_layer(codes, codebooks, scales, d_out, d_in, M, B, g, &A->L, allow_packed);
}

hipError_t any_dequant(const AnyLayer& A, uint16_t* w, hipStream_t s) {
  return A.big ? aqlm::launch_dequant_groups(A.GL, w, s) : aqlm::launch_dequant(A.L, w, s);
}

// Workspace-free product of n rows: the group kernel once per row for large
// groups (a format with no batched kernel), gemm_dispatch otherwise.
int any_gemm_dispatch(const AnyLayer& A, int64_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (!A.big) return gemm_dispatch(A.L, n, x, y, s);
  for (int64_t t = 0; t < n; ++t) {
    const hipError_t e = aqlm::launch_gemv_groups(A.GL, x + t * A.GL.d_in, y + t * A.GL.d_out, s);
    if (e != hipSuccess) return AQLM_ERR_HIP;
  }
  return AQLM_OK;
}

}  // namespace

extern "C" {

int aqlm_dequantize(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                    int64_t d_in, int32_t M, int32_t B, int32_t g, uint16_t* w_out, void* stream) {
  AnyLayer A;
  const int st = check_any(codes, codebooks, scales, d_out, d_in, M, B, g, &A, true);
  if (st != AQLM_OK) return st;
  if (!w_out) return AQLM_ERR_NULL;
  if (!aligned(w_out, 16)) return AQLM_ERR_ALIGN;
  return status_of(any_dequant(A, w_out, static_cast<hipStream_t>(stream)));
}

int aqlm_gemv(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out, int64_t d_in,
              int32_t M, int32_t B, int32_t g, const uint16_t* x, uint16_t* y, void* stream) {
  AnyLayer A;
  const int st = check_any(codes, codebooks, scales, d_out, d_in, M, B, g, &A, true);
  if (st != AQLM_OK) return st;
  if (!x || !y) return AQLM_ERR_NULL;
  if (!aligned(x, 16) || !aligned(y, 16)) return AQLM_ERR_ALIGN;
  if (A.big) return status_of(aqlm::launch_gemv_groups(A.GL, x, y, static_cast<hipStream_t>(stream)));
  const aqlm::Layer& L = A.L;
  if (L.packed && !aqlm::gemv_mfma_fits(&L, 1)) return AQLM_ERR_UNSUPPORTED;
  return status_of(gemv_dispatch(L, x, y, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace {

// Workspace-free product with n activation rows (arguments validated).
int gemm_dispatch(const aqlm::Layer& L, int64_t n, const uint16_t* x, uint16_t* y, hipStream_t s) {
  const int64_t d_in = L.d_in, d_out = L.d_out;
  if (n == 1) return status_of(gemv_dispatch(L, x, y, s));
  // 2..16 tokens with M = 2 or 4 8-bit codebooks: the matrix-vector kernel's
  // scheme with one MFMA column per token; otherwise the tiled kernel.
  if (aqlm::gemm_nb_supported(L, (int32_t)n)) return status_of(aqlm::launch_gemm_nb(L, (int32_t)n, x, y, s));
  const bool chunk_nb = n <= kChunkedMax && aqlm::gemm_nb_supported(L, (int32_t)kSmallBatchMax);
  const bool chunk_16 = n <= kChunkedMax16 && L.B > 8 && aqlm::mfma_supported(L);
  if (n > kSmallBatchMax && (chunk_nb || chunk_16)) {
    for (int64_t t0 = 0; t0 < n; t0 += kSmallBatchMax) {
      const int64_t nt = n - t0 < kSmallBatchMax ? n - t0 : kSmallBatchMax;
      const int st = gemm_dispatch(L, nt, x + t0 * d_in, y + t0 * d_out, s);
      if (st != AQLM_OK) return st;
    }
    return AQLM_OK;
  }
  // More tokens: dequantized weight tiles feed a dense MFMA product.  Two
  // wide codebooks gather every codeword from L2 there, which pays off only
  // from more rows (11008 x 4096, tiled kernel vs prefill: 2x12 92 vs 134 us
  // at 128 rows, 163 vs 147 at 256, 965 vs 551 at 2048; 2x16 140 vs 153 at
  // 64, 163 vs 154 at 128, 1605 vs 623 at 2048).
  const int64_t prefill_min = (L.M == 2 && L.B > 8) ? (L.B == 12 ? kPrefillMin2x12 : kPrefillMin2xWide) : 0;
  if (n > kSmallBatchMax && n >= prefill_min && aqlm::prefill_supported(L))
    return status_of(aqlm::launch_prefill(L, (int32_t)n, x, y, s));
  if (aqlm::mfma_supported(L)) return status_of(aqlm::launch_gemm_mfma(L, (int32_t)n, x, y, s));
  // Formats the matrix-core kernel does not tile (M = 3, 5, 6, 7): one
  // matrix-vector launch per activation row.
  for (int64_t t = 0; t < n; ++t) {
    const hipError_t e = gemv_dispatch(L, x + t * d_in, y + t * d_out, s);
    if (e != hipSuccess) return AQLM_ERR_HIP;
  }
  return AQLM_OK;
}

}  // namespace

extern "C" {

int aqlm_gemm_small_batch(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                          int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, uint16_t* y,
                          void* stream) {
  AnyLayer A;
  int st = check_any(codes, codebooks, scales, d_out, d_in, M, B, g, &A);
  if (st != AQLM_OK) return st;
  st = check_tokens(x, y, n, d_in);
  if (st != AQLM_OK) return st;
  return any_gemm_dispatch(A, n, x, y, static_cast<hipStream_t>(stream));
}

size_t aqlm_gemm_workspace_bytes(int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n) {
  (void)M;
  (void)B;
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0 || n <= 0) return 0;
  if (!two_pass(d_in, n)) return 0;
  return ws_weight_bytes(d_out, d_in) + aqlm::gemm_f16_part_bytes(n, d_out, d_in);
}

int aqlm_gemm(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out, int64_t d_in,
              int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, uint16_t* y, void* workspace,
              size_t workspace_bytes, void* stream) {
  AnyLayer A;
  int st = check_any(codes, codebooks, scales, d_out, d_in, M, B, g, &A);
  if (st != AQLM_OK) return st;
  st = check_tokens(x, y, n, d_in);
  if (st != AQLM_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!two_pass(d_in, n)) return any_gemm_dispatch(A, n, x, y, s);
  if (!workspace) return AQLM_ERR_NULL;
  const size_t wbytes = ws_weight_bytes(d_out, d_in);
  if (workspace_bytes < wbytes + aqlm::gemm_f16_part_bytes(n, d_out, d_in)) return AQLM_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return AQLM_ERR_ALIGN;
  uint16_t* w = static_cast<uint16_t*>(workspace);
  float* part = reinterpret_cast<float*>(static_cast<char*>(workspace) + wbytes);
  const hipError_t e = any_dequant(A, w, s);
  if (e != hipSuccess) return AQLM_ERR_HIP;
  return status_of(aqlm::launch_gemm_f16(x, w, y, part, (int32_t)n, (int32_t)A.d_out(), (int32_t)A.d_in(), s));
}

int aqlm_backward(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                  int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, const uint16_t* dy,
                  float* dcodebooks, float* dscales, void* stream) {
  aqlm::Layer L;
  int st = check_layer(codes, codebooks, scales, d_out, d_in, M, B, g, &L);
  if (st != AQLM_OK) return st;
  if (!x || !dy || !dcodebooks || !dscales) return AQLM_ERR_NULL;
  if (n <= 0 || n >= (int64_t(1) << 31) || n * d_in >= (int64_t(1) << 40) || n * d_out >= (int64_t(1) << 40))
    return AQLM_ERR_SHAPE;
  if (B != 8) return AQLM_ERR_UNSUPPORTED;
  if (d_out % 8 != 0) return AQLM_ERR_SHAPE;
  if (!aligned(x, 16) || !aligned(dy, 16) || !aligned(dcodebooks, 4) || !aligned(dscales, 4)) return AQLM_ERR_ALIGN;
  return status_of(aqlm::launch_backward(L, (int32_t)n, x, dy, dcodebooks, dscales, static_cast<hipStream_t>(stream)));
}

int aqlm_beam_search(const float* w, const float* h, void* codes, const uint16_t* codebooks, const uint16_t* scales,
                     int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int32_t beam, int32_t sweeps,
                     float* loss_out, void* stream) {
  aqlm::Layer L;
  const int st = check_layer(codes, codebooks, scales, d_out, d_in, M, B, g, &L);
  if (st != AQLM_OK) return st;
  if (!w || !h) return AQLM_ERR_NULL;
  if (beam < 1 || sweeps < 0 || d_in >= (int64_t(1) << 16)) return AQLM_ERR_SHAPE;
  if (B != 8 || !aqlm::beam_search_fits((int32_t)d_in, M, beam)) return AQLM_ERR_UNSUPPORTED;
  if (!aligned(w, 4) || !aligned(h, 4) || (loss_out && !aligned(loss_out, 4))) return AQLM_ERR_ALIGN;
  return status_of(aqlm::launch_beam_search(w, h, static_cast<uint8_t*>(const_cast<void*>(codes)), codebooks, scales,
                                            (int32_t)d_out, (int32_t)d_in, M, beam, sweeps, loss_out,
                                            static_cast<hipStream_t>(stream)));
}

int aqlm_gemm_noalloc(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                      int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x, uint16_t* y,
                      void* stream) {
  AnyLayer A;
  int st = check_any(codes, codebooks, scales, d_out, d_in, M, B, g, &A);
  if (st != AQLM_OK) return st;
  st = check_tokens(x, y, n, d_in);
  if (st != AQLM_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!two_pass(d_in, n)) return any_gemm_dispatch(A, n, x, y, s);
  const size_t wbytes = ws_weight_bytes(d_out, d_in);
  if (wbytes + aqlm::gemm_f16_part_bytes(n, d_out, d_in) > kScratchBytes) return AQLM_ERR_SCRATCH;
  char* base = static_cast<char*>(scratch_ptr());
  if (base == nullptr) return AQLM_ERR_HIP;
  uint16_t* w = reinterpret_cast<uint16_t*>(base);
  float* part = reinterpret_cast<float*>(base + wbytes);
  const hipError_t e = any_dequant(A, w, s);
  if (e != hipSuccess) return AQLM_ERR_HIP;
  return status_of(aqlm::launch_gemm_f16(x, w, y, part, (int32_t)n, (int32_t)A.d_out(), (int32_t)A.d_in(), s));
}

int aqlm_gemv_grouped(const aqlm_gemv_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                      void* stream) {
  return aqlm_gemv_grouped_path(problems, count, M, B, g, AQLM_PATH_AUTO, stream);
}

int aqlm_gemv_grouped_path(const aqlm_gemv_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                           int32_t path, void* stream) {
  if (!problems) return AQLM_ERR_NULL;
  if (path != AQLM_PATH_AUTO && path != AQLM_PATH_GATHER && path != AQLM_PATH_TABLE) return AQLM_ERR_UNSUPPORTED;
  if (count < 1 || count > AQLM_MAX_GROUPED) return AQLM_ERR_SHAPE;
  if (g != 8 && aqlm::groups_supported(M, B, g)) {
    // larger groups: one group-kernel launch per problem (no grouped kernel)
    if (path == AQLM_PATH_TABLE) return AQLM_ERR_UNSUPPORTED;
    aqlm::GroupLayer GLs[AQLM_MAX_GROUPED];
    for (int i = 0; i < count; ++i) {
      const aqlm_gemv_problem& P = problems[i];
      const int st = check_group_layer(P.codes, P.codebooks, P.scales, P.d_out, P.d_in, M, B, g, &GLs[i]);
      if (st != AQLM_OK) return st;
      if (!P.x || !P.y) return AQLM_ERR_NULL;
      if (!aligned(P.x, 16) || !aligned(P.y, 16)) return AQLM_ERR_ALIGN;
    }
    for (int i = 0; i < count; ++i) {
      const hipError_t e = aqlm::launch_gemv_groups(GLs[i], problems[i].x, problems[i].y, static_cast<hipStream_t>(stream));
      if (e != hipSuccess) return AQLM_ERR_HIP;
    }
    return AQLM_OK;
  }
  aqlm::Layer Ls[AQLM_MAX_GROUPED];
  const uint16_t* xs[AQLM_MAX_GROUPED];
  uint16_t* ys[AQLM_MAX_GROUPED];
  for (int i = 0; i < count; ++i) {
    const aqlm_gemv_problem& P = problems[i];
    const int st = check_layer(P.codes, P.codebooks, P.scales, P.d_out, P.d_in, M, B, g, &Ls[i], true);
    if (st != AQLM_OK) return st;
    if (!P.x || !P.y) return AQLM_ERR_NULL;
    if (!aligned(P.x, 16) || !aligned(P.y, 16)) return AQLM_ERR_ALIGN;
    xs[i] = P.x;
    ys[i] = P.y;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (Ls[0].packed) {
    // packed codes: the gather kernel only, all problems in one launch
    if (path == AQLM_PATH_TABLE || !aqlm::gemv_mfma_fits(Ls, count)) return AQLM_ERR_UNSUPPORTED;
    return status_of(aqlm::launch_gemv_mfma(Ls, xs, ys, count, s));
  }
  if (path == AQLM_PATH_TABLE) {
    if (!aqlm::gemv_lut_supported(Ls, count)) return AQLM_ERR_UNSUPPORTED;
    return status_of(aqlm::launch_gemv_lut(Ls, xs, ys, count, s));
  }
  bool same_class = true;
  for (int i = 1; i < count; ++i) same_class = same_class && Ls[i].vec_codes == Ls[0].vec_codes;
  if (aqlm::gemv_mfma_supported(M, B) && same_class && aqlm::gemv_mfma_fits(Ls, count))
    return status_of(aqlm::launch_gemv_mfma(Ls, xs, ys, count, s));
  for (int i = 0; i < count; ++i) {
    const hipError_t e = gemv_dispatch(Ls[i], xs[i], ys[i], s);
    if (e != hipSuccess) return AQLM_ERR_HIP;
  }
  return AQLM_OK;
}

// Tiled 8-bit codes: the format checks of check_layer, plus what the tiled
// product reads (M of 1, 2 or 4; tiled offsets held in 31 bits).
static int check_tiled_format(int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t* bytes) {
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0) return AQLM_ERR_SHAPE;
  if (g != 8 || B != 8 || !aqlm::gemv_mfma_supported(M, B)) return AQLM_ERR_UNSUPPORTED;
  if (d_out >= (int64_t(1) << 31) || d_in >= (int64_t(1) << 31)) return AQLM_ERR_SHAPE;
  *bytes = aqlm::tiled_codes_bytes(d_out, d_in / g * M);
  if (*bytes >= (int64_t(1) << 31)) return AQLM_ERR_SHAPE;
  return AQLM_OK;
}

int64_t aqlm_tiled_codes_bytes(int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g) {
  int64_t bytes = 0;
  return check_tiled_format(d_out, d_in, M, B, g, &bytes) == AQLM_OK ? bytes : 0;
}

int aqlm_tile_codes(const void* codes, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, void* tiled,
                    int64_t tiled_bytes, void* stream) {
  if (!codes || !tiled) return AQLM_ERR_NULL;
  int64_t need = 0;
  const int st = check_tiled_format(d_out, d_in, M, B, g, &need);
  if (st != AQLM_OK) return st;
  if (tiled_bytes < need) return AQLM_ERR_WORKSPACE;
  if (!aligned(tiled, 16)) return AQLM_ERR_ALIGN;
  return status_of(aqlm::launch_tile_codes(static_cast<const uint8_t*>(codes), d_out, d_in / g * M,
                                           static_cast<uint8_t*>(tiled), static_cast<hipStream_t>(stream)));
}

int aqlm_gemv_grouped_tiled(const aqlm_gemv_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                            void* stream) {
  if (!problems) return AQLM_ERR_NULL;
  if (count < 1 || count > AQLM_MAX_GROUPED) return AQLM_ERR_SHAPE;
  aqlm::Layer Ls[AQLM_MAX_GROUPED];
  const uint16_t* xs[AQLM_MAX_GROUPED];
  uint16_t* ys[AQLM_MAX_GROUPED];
  for (int i = 0; i < count; ++i) {
    const aqlm_gemv_problem& P = problems[i];
    int st = check_layer(P.codes, P.codebooks, P.scales, P.d_out, P.d_in, M, B, g, &Ls[i]);
    if (st != AQLM_OK) return st;
    int64_t bytes = 0;  // (the formats and sizes tiled codes take)
    st = check_tiled_format(P.d_out, P.d_in, M, B, g, &bytes);
    if (st != AQLM_OK) return st;
    if (!P.x || !P.y) return AQLM_ERR_NULL;
    if (!aligned(P.x, 16) || !aligned(P.y, 16)) return AQLM_ERR_ALIGN;
    Ls[i].tiled = true;
    Ls[i].vec_codes = true;  // (tiles are whole 64-byte K-slices at 16-byte aligned addresses)
    xs[i] = P.x;
    ys[i] = P.y;
  }
  if (!aqlm::gemv_mfma_fits(Ls, count)) return AQLM_ERR_UNSUPPORTED;
  return status_of(aqlm::launch_gemv_mfma(Ls, xs, ys, count, static_cast<hipStream_t>(stream)));
}

int aqlm_gemm_small_batch_tiled(const void* codes, const uint16_t* codebooks, const uint16_t* scales, int64_t d_out,
                                int64_t d_in, int32_t M, int32_t B, int32_t g, int64_t n, const uint16_t* x,
                                uint16_t* y, void* stream) {
  aqlm::Layer L;
  int st = check_layer(codes, codebooks, scales, d_out, d_in, M, B, g, &L);
  if (st != AQLM_OK) return st;
  st = check_tokens(x, y, n, d_in);
  if (st != AQLM_OK) return st;
  int64_t bytes = 0;
  st = check_tiled_format(d_out, d_in, M, B, g, &bytes);
  if (st != AQLM_OK) return st;
  L.tiled = true;
  L.vec_codes = true;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (n == 1) {
    if (!aqlm::gemv_mfma_fits(&L, 1)) return AQLM_ERR_UNSUPPORTED;
    return status_of(aqlm::launch_gemv_mfma(&L, &x, &y, 1, s));
  }
  // up to 16 rows in one launch, up to 64 as launches of 16 (as the row-major
  // product does)
  if (n > kChunkedMax || !aqlm::gemm_nb_supported(L, (int32_t)(n < kSmallBatchMax ? n : kSmallBatchMax)))
    return AQLM_ERR_UNSUPPORTED;
  if (n % kSmallBatchMax == 1 && !aqlm::gemv_mfma_fits(&L, 1)) return AQLM_ERR_UNSUPPORTED;
  for (int64_t t0 = 0; t0 < n; t0 += kSmallBatchMax) {
    const int64_t nt = n - t0 < kSmallBatchMax ? n - t0 : kSmallBatchMax;
    const uint16_t* xt = x + t0 * d_in;
    uint16_t* yt = y + t0 * d_out;
    // (a last chunk of one row is the matrix-vector product, as in the
    // row-major path)
    const hipError_t e = nt == 1 ? aqlm::launch_gemv_mfma(&L, &xt, &yt, 1, s)
                                 : aqlm::launch_gemm_nb(L, (int32_t)nt, xt, yt, s);
    if (e != hipSuccess) return AQLM_ERR_HIP;
  }
  return AQLM_OK;
}

int64_t aqlm_gemv_step_plan_bytes(int32_t levels) {
  if (levels < 1 || levels > AQLM_STEP_MAX_LEVELS) return 0;
  return (int64_t)sizeof(aqlm::StepHeader) + (int64_t)levels * (int64_t)sizeof(aqlm::StepLevel);
}

int aqlm_gemv_step_plan(const aqlm_gemv_problem* problems, const int32_t* level_sizes, int32_t levels, int32_t M,
                        int32_t B, int32_t g, void* plan, int64_t plan_bytes) {
  if (!problems || !level_sizes || !plan) return AQLM_ERR_NULL;
  if (levels < 1 || levels > AQLM_STEP_MAX_LEVELS) return AQLM_ERR_SHAPE;
  if (plan_bytes < aqlm_gemv_step_plan_bytes(levels)) return AQLM_ERR_WORKSPACE;
  auto* head = static_cast<aqlm::StepHeader*>(plan);
  auto* lv = reinterpret_cast<aqlm::StepLevel*>(static_cast<char*>(plan) + sizeof(aqlm::StepHeader));
  int32_t lds = 0;
  int64_t first = 0;
  for (int32_t l = 0; l < levels; ++l) {
    const int32_t n = level_sizes[l];
    if (n < 1 || n > AQLM_MAX_GROUPED) return AQLM_ERR_SHAPE;
    aqlm::Layer Ls[AQLM_MAX_GROUPED];
    const uint16_t* xs[AQLM_MAX_GROUPED];
    uint16_t* ys[AQLM_MAX_GROUPED];
    for (int32_t i = 0; i < n; ++i) {
      const aqlm_gemv_problem& P = problems[first + i];
      const int st = check_layer(P.codes, P.codebooks, P.scales, P.d_out, P.d_in, M, B, g, &Ls[i]);
      if (st != AQLM_OK) return st;
      if (!P.x || !P.y) return AQLM_ERR_NULL;
      if (!aligned(P.x, 16) || !aligned(P.y, 16)) return AQLM_ERR_ALIGN;
      xs[i] = P.x;
      ys[i] = P.y;
    }
    first += n;
    // the step kernel carries the 2x8 matrix-core kernel with 16-byte code rows
    if (M != 2 || B != 8) return AQLM_ERR_UNSUPPORTED;
    for (int32_t i = 0; i < n; ++i)
      if (!Ls[i].vec_codes) return AQLM_ERR_UNSUPPORTED;
    if (!aqlm::gemv_mfma_fits(Ls, n)) return AQLM_ERR_UNSUPPORTED;
    // as aqlm_gemv_grouped would launch it, or, where that layout is not in
    // the step kernel (eight codebook copies with more than two row blocks),
    // with at most two row blocks per workgroup
    hipError_t e = aqlm::gemv_mfma_impl(Ls, xs, ys, n, nullptr, &lv[l], 0, aqlm::kStepLdsLimit);
    if (e != hipSuccess) e = aqlm::gemv_mfma_impl(Ls, xs, ys, n, nullptr, &lv[l], 2, aqlm::kStepLdsLimit);
    if (e != hipSuccess) return AQLM_ERR_UNSUPPORTED;
    if (lv[l].lds_bytes > lds) lds = lv[l].lds_bytes;
  }
  head->magic = aqlm::kStepMagic;
  head->levels = levels;
  head->lds_bytes = lds;
  head->grid = aqlm::num_cus();
  return AQLM_OK;
}

int aqlm_gemv_step(const void* plan_host, const void* plan_dev, void* sync, uint32_t spin_limit, void* stream) {
  if (!plan_host || !plan_dev || !sync) return AQLM_ERR_NULL;
  const auto* head = static_cast<const aqlm::StepHeader*>(plan_host);
  if (head->magic != aqlm::kStepMagic || head->levels < 1 || head->levels > AQLM_STEP_MAX_LEVELS)
    return AQLM_ERR_SHAPE;
  if (!aligned(plan_dev, 16) || !aligned(sync, 16)) return AQLM_ERR_ALIGN;
  // (the workgroup split is sized for the device the plan was made on)
  if (head->grid != aqlm::num_cus()) return AQLM_ERR_SHAPE;
  const auto* lv = reinterpret_cast<const aqlm::StepLevel*>(static_cast<const char*>(plan_dev) +
                                                             sizeof(aqlm::StepHeader));
  const uint32_t spin = spin_limit ? spin_limit : AQLM_STEP_DEFAULT_SPIN;
  return status_of(aqlm::launch_step(lv, head->levels, head->grid, (size_t)head->lds_bytes,
                                     static_cast<uint32_t*>(sync), spin, static_cast<hipStream_t>(stream)));
}

int aqlm_gemv_step_status(void* sync, void* stream) {
  if (!sync) return AQLM_ERR_NULL;
  if (!aligned(sync, 16)) return AQLM_ERR_ALIGN;
  if (hipStreamSynchronize(static_cast<hipStream_t>(stream)) != hipSuccess) return AQLM_ERR_HIP;
  uint32_t err = 0;
  uint32_t* flag = static_cast<uint32_t*>(sync) + 1;
  if (hipMemcpy(&err, flag, sizeof(err), hipMemcpyDeviceToHost) != hipSuccess) return AQLM_ERR_HIP;
  if (err == 0) return AQLM_OK;
  const uint32_t zero = 0;
  if (hipMemcpy(flag, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return AQLM_ERR_HIP;
  return AQLM_ERR_TIMEOUT;
}

// Chunk-sorted codes: the shape and format rules shared by the sorter and
// the product.
static int check_sorted_shape(int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g) {
  if (d_out <= 0 || d_in <= 0 || g <= 0 || d_in % g != 0) return AQLM_ERR_SHAPE;
  if (g != 8 || !aqlm::sorted_supported(M, B)) return AQLM_ERR_UNSUPPORTED;
  const int64_t G = d_in / g;
  if (d_out >= (int64_t(1) << 31) || d_out * G >= (int64_t(1) << 31) || G > (int64_t)aqlm::kSortedJMax)
    return AQLM_ERR_SHAPE;
  return AQLM_OK;
}

// (entries are addressed in bytes with 32 bits on the device)
static constexpr int64_t kSortedMaxSteps = (int64_t(1) << 31) / 256 - 1;

static int sort_input(const void* codes, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g, bool* packed,
                      int64_t* steps) {
  if (!codes) return AQLM_ERR_NULL;
  *packed = (B & AQLM_PACKED) != 0;
  const int32_t b = B & ~AQLM_PACKED;
  int st = check_sorted_shape(d_out, d_in, M, b, g);
  if (st != AQLM_OK) return st;
  if (*packed && !aqlm::packed_supported(M, b)) return AQLM_ERR_UNSUPPORTED;
  if (*packed && (d_in / g) * M * b >= (int64_t(1) << 32)) return AQLM_ERR_SHAPE;
  *steps = aqlm::sorted_steps(codes, *packed, (int32_t)d_out, (int32_t)d_in, M, b);
  if (*steps > kSortedMaxSteps) return AQLM_ERR_SHAPE;
  return AQLM_OK;
}

int aqlm_sort_codes_size(const void* codes_host, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                         int64_t* entry_words, int64_t* index_words) {
  if (!entry_words || !index_words) return AQLM_ERR_NULL;
  bool packed = false;
  int64_t steps = 0;
  const int st = sort_input(codes_host, d_out, d_in, M, B, g, &packed, &steps);
  if (st != AQLM_OK) return st;
  *entry_words = steps * 64;
  *index_words = (int64_t)aqlm::sorted_classes(M, B & ~AQLM_PACKED) * aqlm::sorted_blocks(d_out) + 1;
  return AQLM_OK;
}

int aqlm_sort_codes(const void* codes_host, int64_t d_out, int64_t d_in, int32_t M, int32_t B, int32_t g,
                    uint32_t* entries_host, int64_t entry_words, uint32_t* index_host, int64_t index_words) {
  if (!entries_host || !index_host) return AQLM_ERR_NULL;
  bool packed = false;
  int64_t steps = 0;
  const int st = sort_input(codes_host, d_out, d_in, M, B, g, &packed, &steps);
  if (st != AQLM_OK) return st;
  const int32_t b = B & ~AQLM_PACKED;
  if (entry_words < steps * 64 ||
      index_words < (int64_t)aqlm::sorted_classes(M, b) * aqlm::sorted_blocks(d_out) + 1)
    return AQLM_ERR_WORKSPACE;
  aqlm::sort_codes(codes_host, packed, (int32_t)d_out, (int32_t)d_in, M, b, entries_host, steps, index_host);
  return AQLM_OK;
}

size_t aqlm_gemv_sorted_workspace_bytes(int64_t d_out, int32_t M, int32_t B) {
  if (d_out <= 0 || d_out >= (int64_t(1) << 31) || !aqlm::sorted_supported(M, B)) return 0;
  return aqlm::gemv_sorted_workspace_bytes(d_out, M, B);
}

static int check_sorted_problem(const aqlm_sorted_problem& P, int32_t M, int32_t B, int32_t g,
                                aqlm::SortedLayer* L) {
  if (!P.entries || !P.index || !P.codebooks || !P.scales || !P.x || !P.y) return AQLM_ERR_NULL;
  const int st = check_sorted_shape(P.d_out, P.d_in, M, B, g);
  if (st != AQLM_OK) return st;
  if (P.entry_words <= 0 || P.entry_words % 64 != 0 || P.entry_words / 64 > kSortedMaxSteps) return AQLM_ERR_SHAPE;
  if (!aligned(P.entries, 4) || !aligned(P.index, 4) || !aligned(P.codebooks, 16) || !aligned(P.scales, 2) ||
      !aligned(P.x, 16) || !aligned(P.y, 2))
    return AQLM_ERR_ALIGN;
  *L = aqlm::SortedLayer{P.entries, P.index, P.index_host, P.entry_words / 64, P.codebooks, P.scales,
                         (int32_t)P.d_out, (int32_t)P.d_in, M, B};
  return AQLM_OK;
}

int aqlm_gemv_sorted_grouped(const aqlm_sorted_problem* problems, int32_t count, int32_t M, int32_t B, int32_t g,
                             void* workspace, size_t workspace_bytes, void* stream) {
  if (!problems || !workspace) return AQLM_ERR_NULL;
  if (count < 1 || count > AQLM_MAX_GROUPED) return AQLM_ERR_SHAPE;
  aqlm::SortedLayer Ls[AQLM_MAX_GROUPED];
  const uint16_t* xs[AQLM_MAX_GROUPED];
  uint16_t* ys[AQLM_MAX_GROUPED];
  int64_t rows = 0;
  for (int32_t i = 0; i < count; ++i) {
    const int st = check_sorted_problem(problems[i], M, B, g, &Ls[i]);
    if (st != AQLM_OK) return st;
    xs[i] = problems[i].x;
    ys[i] = problems[i].y;
    rows += problems[i].d_out;
  }
  if (!aqlm::gemv_sorted_fits(Ls, count)) return AQLM_ERR_SHAPE;
  if (!aligned(workspace, 16)) return AQLM_ERR_ALIGN;
  if (workspace_bytes < aqlm::gemv_sorted_workspace_bytes(rows, M, B)) return AQLM_ERR_WORKSPACE;
  return status_of(aqlm::launch_gemv_sorted(Ls, xs, ys, count, workspace, static_cast<hipStream_t>(stream)));
}

int aqlm_gemv_sorted(const uint32_t* entries, int64_t entry_words, const uint32_t* index, const uint32_t* index_host,
                     const uint16_t* codebooks, const uint16_t* scales, int64_t d_out, int64_t d_in, int32_t M,
                     int32_t B, int32_t g, const uint16_t* x, uint16_t* y, void* workspace, size_t workspace_bytes,
                     void* stream) {
  const aqlm_sorted_problem P{entries, entry_words, index, index_host, codebooks, scales, x, y, d_out, d_in};
  return aqlm_gemv_sorted_grouped(&P, 1, M, B, g, workspace, workspace_bytes, stream);
}

int64_t aqlm_packed_row_words(int64_t d_in, int32_t M, int32_t B, int32_t g) {
  if (d_in <= 0 || M <= 0 || B <= 0 || g <= 0) return 0;
  return ((d_in / g) * M * (int64_t)(B & ~AQLM_PACKED) + 31) / 32;
}

const char* aqlm_status_string(int status) {
  switch (status) {
    case AQLM_OK: return "ok";
    case AQLM_ERR_NULL: return "null pointer argument";
    case AQLM_ERR_SHAPE: return "invalid shape";
    case AQLM_ERR_UNSUPPORTED: return "unsupported (M, B, g)";
    case AQLM_ERR_ALIGN: return "misaligned pointer";
    case AQLM_ERR_HIP: return "HIP runtime error";
    case AQLM_ERR_WORKSPACE: return "workspace too small";
    case AQLM_ERR_SCRATCH: return "needs more scratch than aqlm_gemm_noalloc's fixed buffer holds";
    case AQLM_ERR_TIMEOUT: return "a decode-step level barrier timed out";
  }
  return "unknown status";
}

}  // extern "C"
