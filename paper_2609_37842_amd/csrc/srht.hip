// Random second stage, EOGP-R (Appendix B.2, eq. app_srht_definition):
//   x = sqrt(p/k) R H_p D J z,  p = 2^ceil(log2 m),
// with H_p the orthonormal Walsh-Hadamard matrix. With W the unnormalised
// transform in Sylvester order (entry (r, i) = (-1)^popcount(r & i)),
//   x_c = W(D J z)[rows[c]] / sqrt(k).
//
// p <= 32768: one workgroup per row. The row is read once (coalesced),
// multiplied by the random signs and zero-padded into LDS; the butterfly
// stages run in LDS two at a time (radix 4: each thread combines four elements
// h apart), one radix-2 stage first when log2 p is odd; the kept rows are then
// gathered and scaled. Cost: p log2 p additions per row, HBM traffic m + k
// floats per row.
//
// p > 32768 (up to 2^20): W_p = W_p1 (x) W_p2 in Sylvester order (index
// i = i1 p2 + i2, p2 = 32768, p1 = p / p2 <= 32). One workgroup per (row,
// chunk i1) transforms its 32768 entries along i2 in LDS as above and writes
// them to the workspace; the gather then forms each kept coordinate
// r = r1 p2 + r2 as the length-p1 transform along i1 of that column,
//   x_c = sum_j (-1)^popcount(r1 & j) S[j p2 + r2] / sqrt(k).
// Extra HBM traffic: p floats written and k p1 read per row.
#include <cmath>

#include "common.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int kSrhtMaxLog = 15;      // one stage: the padded row fits the LDS (128 KB)
constexpr int kSrhtMaxLogTwo = 20;   // two stages: p1 = p / 2^15 <= 32

// In-LDS unnormalised Walsh-Hadamard transform of L[0 .. 2^logp).
__device__ __forceinline__ void fwht_lds(float* L, int logp) {
  const int tid = threadIdx.x, nt = blockDim.x;
  const int p = 1 << logp;
  int h = 1;
  if (logp & 1) {                                   // one radix-2 stage (h = 1)
    for (int b = tid; b < p / 2; b += nt) {
      const float u = L[2 * b], v = L[2 * b + 1];
      L[2 * b] = u + v;
      L[2 * b + 1] = u - v;
    }
    __syncthreads();
    h = 2;
  }
  for (; h < p; h <<= 2) {                          // stages h and 2h together
    for (int b = tid; b < p / 4; b += nt) {
      // element b of the p/4 groups: low bits below h, then two group bits
      const int lo = b & (h - 1);
      const int base = ((b - lo) << 2) + lo;
      const float a0 = L[base], a1 = L[base + h], a2 = L[base + 2 * h], a3 = L[base + 3 * h];
      const float b0 = a0 + a1, b1 = a0 - a1, b2 = a2 + a3, b3 = a2 - a3;
      L[base] = b0 + b2;
      L[base + h] = b1 + b3;
      L[base + 2 * h] = b0 - b2;
      L[base + 3 * h] = b1 - b3;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(1024) void k_srht(const float* __restrict__ Z, int64_t ldz, int m,
                                               int logp, const int8_t* __restrict__ signs,
                                               const int32_t* __restrict__ rows, int k,
                                               float scale, float* __restrict__ X, int64_t ldx) {
  extern __shared__ float L[];
  const int64_t i = blockIdx.x;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int p = 1 << logp;
  const float* z = Z + i * ldz;
  for (int c = tid; c < p; c += nt) {
    float v = 0.f;
    if (c < m) v = signs[c] < 0 ? -z[c] : z[c];
    L[c] = v;
  }
  __syncthreads();
  fwht_lds(L, logp);
  float* x = X + i * ldx;
  for (int c = tid; c < k; c += nt) {
    const int r = rows[c];
    x[c] = (r >= 0 && r < p) ? L[r] * scale : __builtin_nanf("");
  }
}

// Two-stage form, first stage: grid (p1, N); chunk i1 of row i, signed and
// zero-padded, transformed along i2 into S[i][i1 p2 ..].
__global__ __launch_bounds__(1024) void k_srht_chunk(const float* __restrict__ Z, int64_t ldz,
                                                     int m, const int8_t* __restrict__ signs,
                                                     float* __restrict__ S, int64_t lds_row) {
  extern __shared__ float L[];
  const int64_t i = blockIdx.y;
  const int64_t c0 = (int64_t)blockIdx.x << kSrhtMaxLog;
  const int tid = threadIdx.x, nt = blockDim.x;
  const float* z = Z + i * ldz;
  for (int c = tid; c < (1 << kSrhtMaxLog); c += nt) {
    const int64_t g = c0 + c;
    float v = 0.f;
    if (g < m) v = signs[g] < 0 ? -z[g] : z[g];
    L[c] = v;
  }
  __syncthreads();
  fwht_lds(L, kSrhtMaxLog);
  float* out = S + i * lds_row + c0;
  for (int c = tid; c < (1 << kSrhtMaxLog); c += nt) out[c] = L[c];
}

// Second stage fused with the gather: grid (ceil(k / 256), N).
__global__ __launch_bounds__(256) void k_srht_cross(const float* __restrict__ S, int64_t lds_row,
                                                    int logp, const int32_t* __restrict__ rows,
                                                    int k, float scale, float* __restrict__ X,
                                                    int64_t ldx) {
  const int64_t i = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= k) return;
  const int p = 1 << logp, p1 = 1 << (logp - kSrhtMaxLog);
  const int r = rows[c];
  if (r < 0 || r >= p) {
    X[i * ldx + c] = __builtin_nanf("");
    return;
  }
  const int r1 = r >> kSrhtMaxLog, r2 = r & ((1 << kSrhtMaxLog) - 1);
  const float* col = S + i * lds_row + r2;
  float acc = 0.f;
  for (int j = 0; j < p1; ++j) {
    const float v = col[(int64_t)j << kSrhtMaxLog];
    acc += (__popc(r1 & j) & 1) ? -v : v;
  }
  X[i * ldx + c] = acc * scale;
}

}  // namespace

int srht_max_log() { return kSrhtMaxLogTwo; }

namespace {
int srht_log(int64_t m) {
  int logp = 0;
  while ((int64_t(1) << logp) < m) ++logp;
  return logp;
}
}  // namespace

size_t srht_ws(int64_t N, int64_t m) {
  const int logp = srht_log(m);
  if (logp <= kSrhtMaxLog) return 0;
  return align256((size_t)N * ((size_t)1 << logp) * sizeof(float));
}

eogp_status srht_project(const float* Z, int64_t ldz, int64_t N, int64_t m, const int8_t* signs,
                         const int32_t* rows, int64_t k, float* X, int64_t ldx, void* ws,
                         size_t ws_bytes, hipStream_t s) {
  if (N == 0) return EOGP_OK;
  const int logp = srht_log(m);
  for (const void* fn : {(const void*)k_srht, (const void*)k_srht_chunk}) {
    const eogp_status st = ensure_dynamic_lds(fn, (int)(sizeof(float) << kSrhtMaxLog));
    if (st != EOGP_OK) return st;
  }
  const float scale = (float)(1.0 / std::sqrt((double)k));
  timing::Scope ts(EOGP_KT_SRHT, s);
  if (logp <= kSrhtMaxLog) {
    const int p = 1 << logp;
    const size_t lds = (size_t)p * sizeof(float);
    const int nt = std::max(64, std::min(1024, p / 4));
    for (int64_t r0 = 0; r0 < N; r0 += 0x7FFFFFFF) {
      const int64_t nr = std::min<int64_t>(N - r0, 0x7FFFFFFF);
      hipLaunchKernelGGL(k_srht, dim3((unsigned)nr), dim3(nt), lds, s, Z + r0 * ldz, ldz, (int)m,
                         logp, signs, rows, (int)k, scale, X + r0 * ldx, ldx);
      EOGP_LAUNCH_CHECK("srht_project");
    }
    return EOGP_OK;
  }
  if (ws_bytes < srht_ws(N, m) || !ws) return fail(EOGP_ERR_WORKSPACE, "srht_project: workspace too small");
  float* S = static_cast<float*>(ws);
  const int64_t p = int64_t(1) << logp;
  const int p1 = 1 << (logp - kSrhtMaxLog);
  for (int64_t r0 = 0; r0 < N; r0 += 65535) {
    const int64_t nr = std::min<int64_t>(N - r0, 65535);
    hipLaunchKernelGGL(k_srht_chunk, dim3((unsigned)p1, (unsigned)nr), dim3(1024),
                       sizeof(float) << kSrhtMaxLog, s, Z + r0 * ldz, ldz, (int)m, signs,
                       S + r0 * p, p);
    hipLaunchKernelGGL(k_srht_cross, dim3((unsigned)ceil_div(k, 256), (unsigned)nr), dim3(256), 0,
                       s, S + r0 * p, p, logp, rows, (int)k, scale, X + r0 * ldx, ldx);
    EOGP_LAUNCH_CHECK("srht_project (two stages)");
  }
  return EOGP_OK;
}

}  // namespace eogp
