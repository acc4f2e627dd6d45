// Phase 1 of AQLM: beam search over the codes (Sec. 3, "Phase 1: Beam search
// for codes").  Each output row is independent (the objective is additive
// over rows), so one workgroup searches one row:
//   L(b) = (w - what) H (w - what)^T,  H = X X^T,
//   what[8j + t] = s * sum_m C_m[b_jm][t]   (exact reconstruction).
// A beam of at most k configurations of the row's codes starts as the row's
// current codes.  A step takes one position (j, m) (groups in order,
// codebooks in order within a group) and scores, for every configuration in
// the beam and every codeword e of codebook m, the configuration with code
// (j, m) set to e; the k distinct configurations of least loss form the next
// beam (ties: earlier beam entry, then smaller e).  The result is the best
// configuration after the given number of sweeps.
//
// Scores are incremental, as the paper describes: with h = H r kept per
// configuration (r = w - what) and delta = s (C_e - C_o) on group j,
//   L' = L - 2 delta . h_j + delta H_jj delta^T
// (delta is exactly zero for e = o, so keeping a code keeps the loss
// exactly).  A new configuration's h is its parent's minus H[:, group j] delta
// (8 multiply-adds per input).
//
// Layout: the beam state (codes and h of every entry, two generations) and
// the codebooks (fp16) live in LDS; H stays in global memory (L2/MALL:
// every workgroup reads the same 8 columns at the same step).  Thread e
// scores codeword e against every beam entry and keeps its best k distinct
// candidates (a 64-bit hash of the configuration tells equal ones apart;
// equal configurations from one codeword can only come from entries that
// differ at position (j, m) alone); k rounds of a workgroup argmin over the
// threads' best then pick the next beam.
#include "common.h"
#include "launch.h"

namespace aqlm {

namespace {

constexpr int kBsThreads = 256;
constexpr int kBsMaxBeam = 8;

struct BeamArgs {
  const float* w;       // [d_out][d_in]
  const float* h;       // [d_in][d_in]
  uint8_t* codes;       // [d_out][G][M], read and overwritten
  const uint16_t* cb;   // [M][256][8]
  const uint16_t* scales;
  float* loss;          // [d_out] (may be null)
  int32_t d_in;
  int32_t G;
  int32_t M;
  int32_t beam;
  int32_t sweeps;
};

__device__ __forceinline__ uint64_t mix64(uint64_t x) {
  // splitmix64 finaliser (Steele, Lea, Flood: "Fast splittable pseudorandom
  // number generators", 2014)
  x ^= x >> 30;
  x *= 0xBF58476D1CE4E5B9ull;
  x ^= x >> 27;
  x *= 0x94D049BB133111EBull;
  x ^= x >> 31;
  return x;
}
__device__ __forceinline__ uint64_t pos_hash(int pos, uint32_t code) {
  return mix64(((uint64_t)(uint32_t)pos << 16) | code);
}

// candidate order: score, then beam entry, then code
__device__ __forceinline__ bool cand_less(float s0, int b0, int e0, float s1, int b1, int e1) {
  if (s0 != s1) return s0 < s1;
  if (b0 != b1) return b0 < b1;
  return e0 < e1;
}

size_t beam_lds_bytes(int d_in, int G, int M, int k) {
  size_t b = 0;
  b += (size_t)2 * k * d_in * 4;       // h per entry, two generations
  b += (size_t)M * 256 * 16;           // codebooks (fp16)
  b += 64 * 4;                         // H_jj
  b += (size_t)k * 8 * 4 * 2;          // h_j and C_o (then delta) per entry
  b += (size_t)k * 4 * 4;              // losses rounded to fp32, spare
  b += (size_t)k * 8 * 2;              // hashes, two generations
  b += (size_t)k * 8 * 2;              // losses (fp64), two generations
  b += 4 * 8;                          // fp64 reduction exchange
  b += (size_t)k * 4 * 2;              // parent, code of each new entry
  b += 16 * 4;                         // argmin exchange
  b += (size_t)2 * k * G * M;          // codes per entry, two generations
  return (b + 15) & ~(size_t)15;
}

__global__ __launch_bounds__(kBsThreads) void k_beam(const BeamArgs a) {
  extern __shared__ uint4 lds_u4[];
  const int k = a.beam, d_in = a.d_in, G = a.G, M = a.M;
  const int ncode = G * M;
  // LDS carve-up (byte offsets in beam_lds_bytes order)
  float* hr = reinterpret_cast<float*>(lds_u4);                    // [2][k][d_in]
  uint16_t* cbl = reinterpret_cast<uint16_t*>(hr + 2 * k * d_in);  // [M][256][8]
  float* hjj = reinterpret_cast<float*>(cbl + M * 256 * 8);        // [8][8]
  float* zb = hjj + 64;                                            // [k][8] h_j of each entry
  float* dl = zb + 8 * k;                                          // [k][8] C_o of each entry, then delta of new entries
  float* lossf = dl + 8 * k;                                       // [k] losses of the current entries, fp32
  float* spare = lossf + k;                                        // [3k]
  uint64_t* hsh = reinterpret_cast<uint64_t*>(spare + 3 * k);      // [2][k] (8-byte aligned: k*20 floats before)
  double* lossb = reinterpret_cast<double*>(hsh + 2 * k);          // [2][k] losses, fp64
  double* xd = lossb + 2 * k;                                      // [4]
  int* par = reinterpret_cast<int*>(xd + 4);                       // [k]
  int* pcode = par + k;                                            // [k]
  float* xs = reinterpret_cast<float*>(pcode + k);                 // [4] scores, [4] ints x 3 (argmin)
  int* xi = reinterpret_cast<int*>(xs + 4);                        // [12]
  uint8_t* cod = reinterpret_cast<uint8_t*>(xi + 12);              // [2][k][ncode]

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int32_t row = blockIdx.x;
  const float s = h2f(a.scales[row]);
  const float* wrow = a.w + (size_t)row * d_in;
  uint8_t* crow = a.codes + (size_t)row * ncode;

  for (int e = tid; e < M * 256 * 8; e += kBsThreads) cbl[e] = a.cb[e];
  for (int e = tid; e < ncode; e += kBsThreads) cod[e] = crow[e];
  __syncthreads();

  // Exact loss of a configuration (its codes in LDS at `cfg`): r = w - what
  // into `rs`, h = H r accumulated in fp64 row by row of H (H is symmetric:
  // row q holds column q, so the workgroup reads each row contiguously;
  // thread tid owns inputs tid + 256 v), written to `hs` as fp32 when given,
  // and the loss r . h in fp64 (summed in a fixed order).
  constexpr int kHv = 16;  // inputs per thread (d_in <= 4096)
  auto exact_loss = [&](const uint8_t* cfg, float* rs, float* hs) -> double {
    for (int c = tid; c < d_in; c += kBsThreads) {
      const int j = c >> 3, t = c & 7;
      float u = 0.f;
      for (int m = 0; m < M; ++m) {
        const float v = h2f(cbl[(m * 256 + cfg[j * M + m]) * 8 + t]);
        u = (m == 0) ? v : u + v;
      }
      rs[c] = wrow[c] - s * u;
    }
    __syncthreads();
    double acc[kHv];
#pragma unroll
    for (int v = 0; v < kHv; ++v) acc[v] = 0.0;
    for (int q = 0; q < d_in; ++q) {
      const double rq = (double)rs[q];
      const float* hrow = a.h + (size_t)q * d_in;
#pragma unroll
      for (int v = 0; v < kHv; ++v) {
        const int c = tid + kBsThreads * v;
        if (c < d_in) acc[v] += (double)hrow[c] * rq;
      }
    }
    double lpart = 0.0;
#pragma unroll
    for (int v = 0; v < kHv; ++v) {
      const int c = tid + kBsThreads * v;
      if (c < d_in) lpart += (double)rs[c] * acc[v];
    }
    if (hs) {
#pragma unroll
      for (int v = 0; v < kHv; ++v) {
        const int c = tid + kBsThreads * v;
        if (c < d_in) hs[c] = (float)acc[v];
      }
    }
    for (int off = 32; off >= 1; off >>= 1) lpart += __shfl_xor(lpart, off);
    if (lane == 0) xd[wave] = lpart;
    __syncthreads();
    const double l = (xd[0] + xd[1]) + (xd[2] + xd[3]);
    __syncthreads();
    return l;
  };

  // the starting configuration: residual in the second generation's h
  // space (free until the first step), h into the first generation
  if (tid == 0) hsh[0] = 0;
  const double l0 = exact_loss(cod, hr + k * d_in, hr);
  uint64_t hpart = 0;
  for (int p = tid; p < ncode; p += kBsThreads) hpart += pos_hash(p, cod[p]);
  atomicAdd(reinterpret_cast<unsigned long long*>(&hsh[0]), (unsigned long long)hpart);
  if (tid == 0) {
    lossb[0] = l0;
    lossf[0] = (float)l0;
  }
  int cur = 0, nb = 1;
  __syncthreads();

  for (int sw = 0; sw < a.sweeps; ++sw) {
    for (int j = 0; j < G; ++j) {
      for (int m = 0; m < M; ++m) {
        const int pos = j * M + m;
        const int nxt = cur ^ 1;
        const float* hcur = hr + cur * k * d_in;
        const uint8_t* ccur = cod + cur * k * ncode;
        // H_jj, then h_j and the current codeword C_o of every entry
        if (tid < 64) hjj[tid] = a.h[(size_t)(8 * j + (tid >> 3)) * d_in + 8 * j + (tid & 7)];
        __syncthreads();
        if (tid < 8 * nb) {
          const int b = tid >> 3, t = tid & 7;
          const int o = ccur[b * ncode + pos];
          zb[b * 8 + t] = hcur[b * d_in + 8 * j + t];
          dl[b * 8 + t] = h2f(cbl[(m * 256 + o) * 8 + t]);
        }
        __syncthreads();
        // thread e: codeword e of codebook m against every entry; local best k
        float ls[kBsMaxBeam], ld[kBsMaxBeam];
        int lb[kBsMaxBeam];
        uint64_t lh[kBsMaxBeam];
        int nl = 0;
        {
          const int e = tid;
          float av[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) av[u] = h2f(cbl[(m * 256 + e) * 8 + u]);
          const uint64_t he = pos_hash(pos, (uint32_t)e);
          for (int b = 0; b < nb; ++b) {
            float dv[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) dv[t] = s * (av[t] - dl[b * 8 + t]);
            float dl_ = 0.f;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
              float hd = 0.f;
#pragma unroll
              for (int u = 0; u < 8; ++u) hd += hjj[t * 8 + u] * dv[u];
              dl_ += dv[t] * (hd - 2.f * zb[b * 8 + t]);
            }
            const float sc = lossf[b] + dl_;
            const int o = ccur[b * ncode + pos];
            const uint64_t hc = hsh[cur * k + b] - pos_hash(pos, (uint32_t)o) + he;
            // an equal configuration already listed (from an earlier entry)?
            bool dup = false;
            for (int l = 0; l < nl; ++l) dup = dup || lh[l] == hc;
            if (dup) continue;  // the earlier entry's candidate stands for it
            // insert in (score, entry) order, keep the best k
            if (nl == k && !cand_less(sc, b, e, ls[nl - 1], lb[nl - 1], e)) continue;
            int p = nl < k ? nl : k - 1;
            while (p > 0 && cand_less(sc, b, e, ls[p - 1], lb[p - 1], e)) {
              ls[p] = ls[p - 1];
              ld[p] = ld[p - 1];
              lb[p] = lb[p - 1];
              lh[p] = lh[p - 1];
              --p;
            }
            ls[p] = sc;
            ld[p] = dl_;
            lb[p] = b;
            lh[p] = hc;
            if (nl < k) ++nl;
          }
        }
        __syncthreads();  // (dl is rewritten below)
        // k rounds of a workgroup argmin over the threads' best remaining
        int head = 0, nn = 0;
        for (int n = 0; n < k; ++n) {
          float bs = head < nl ? ls[head] : __builtin_huge_valf();
          int bb = head < nl ? lb[head] : 0x7fffffff;
          int be = tid;
          for (int off = 32; off >= 1; off >>= 1) {
            const float os = __shfl_xor(bs, off);
            const int ob = __shfl_xor(bb, off), oe = __shfl_xor(be, off);
            if (cand_less(os, ob, oe, bs, bb, be)) {
              bs = os;
              bb = ob;
              be = oe;
            }
          }
          if (lane == 0) {
            xs[wave] = bs;
            xi[wave] = bb;
            xi[4 + wave] = be;
          }
          __syncthreads();
          float ws = xs[0];
          int wb = xi[0], we = xi[4];
          for (int v = 1; v < 4; ++v)
            if (cand_less(xs[v], xi[v], xi[4 + v], ws, wb, we)) {
              ws = xs[v];
              wb = xi[v];
              we = xi[4 + v];
            }
          __syncthreads();
          if (!(ws < __builtin_huge_valf())) break;  // fewer candidates than k
          if (tid == we) {
            par[n] = wb;
            pcode[n] = we;
            lossb[nxt * k + n] = lossb[cur * k + wb] + (double)ld[head];
            hsh[nxt * k + n] = lh[head];
            ++head;
          }
          ++nn;
        }
        __syncthreads();
        // the new entries: codes, delta, h
        uint8_t* cnxt = cod + nxt * k * ncode;
        for (int e = tid; e < nn * ncode; e += kBsThreads) {
          const int n = e / ncode, p = e % ncode;
          cnxt[e] = p == pos ? (uint8_t)pcode[n] : ccur[par[n] * ncode + p];
        }
        if (tid < 8 * nn) {
          const int n = tid >> 3, t = tid & 7;
          const int o = ccur[par[n] * ncode + pos];
          dl[n * 8 + t] = s * (h2f(cbl[(m * 256 + pcode[n]) * 8 + t]) - h2f(cbl[(m * 256 + o) * 8 + t]));
        }
        __syncthreads();
        float* hnxt = hr + nxt * k * d_in;
        for (int c = tid; c < d_in; c += kBsThreads) {
          // H[c][8j + t] = H[8j + t][c]: eight rows of H, read contiguously
          float hc8[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) hc8[t] = a.h[(size_t)(8 * j + t) * d_in + c];
          for (int n = 0; n < nn; ++n) {
            float d = 0.f;
#pragma unroll
            for (int t = 0; t < 8; ++t) d += hc8[t] * dl[n * 8 + t];
            hnxt[n * d_in + c] = hcur[par[n] * d_in + c] - d;
          }
        }
        if (tid < nn) lossf[tid] = (float)lossb[nxt * k + tid];
        __syncthreads();
        cur = nxt;
        nb = nn;
      }
    }
  }
  // The best configuration, and its exact loss: the running losses add one
  // fp32 change per step, each a difference of terms far larger than itself.
  const uint8_t* best = cod + cur * k * ncode;
  for (int e = tid; e < ncode; e += kBsThreads) crow[e] = best[e];
  if (a.loss) {
    const double lf = exact_loss(best, hr + (cur ^ 1) * k * d_in, nullptr);
    if (tid == 0) a.loss[row] = (float)lf;
  }
}

}  // namespace

bool beam_search_fits(int32_t d_in, int32_t M, int32_t beam) {
  if (beam < 1 || beam > kBsMaxBeam || M < 1 || M > 8 || d_in > 4096) return false;
  return beam_lds_bytes(d_in, d_in / 8, M, beam) <= 160 * 1024;
}

hipError_t launch_beam_search(const float* w, const float* h, uint8_t* codes, const uint16_t* codebooks,
                              const uint16_t* scales, int32_t d_out, int32_t d_in, int32_t M, int32_t beam,
                              int32_t sweeps, float* loss, hipStream_t s) {
  if (!beam_search_fits(d_in, M, beam)) return hipErrorInvalidValue;
  const size_t lds = beam_lds_bytes(d_in, d_in / 8, M, beam);
  const hipError_t e = allow_dynamic_lds(reinterpret_cast<const void*>(k_beam), 160 * 1024);
  if (e != hipSuccess) return e;
  const BeamArgs a{w, h, codes, codebooks, scales, loss, d_in, d_in / 8, M, beam, sweeps};
  hipLaunchKernelGGL(k_beam, dim3((uint32_t)d_out), dim3(kBsThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace aqlm
