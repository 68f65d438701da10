// Random second stage, EOGP-R (Appendix B.2, eq. app_srht_definition):
//   x = sqrt(p/k) R H_p D J z,  p = 2^ceil(log2 m),
// with H_p the orthonormal Walsh-Hadamard matrix. With W the unnormalised
// transform in Sylvester order (entry (r, i) = (-1)^popcount(r & i)),
//   x_c = W(D J z)[rows[c]] / sqrt(k).
//
// One workgroup per row. The row is read once (coalesced), multiplied by the
// random signs and zero-padded into LDS; the butterfly stages run in LDS two
// at a time (radix 4: each thread combines four elements h apart), one radix-2
// stage first when log2 p is odd; the kept rows are then gathered and scaled.
// Cost: p log2 p additions per row, HBM traffic m + k floats per row.
#include <cmath>

#include "common.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int kSrhtMaxLog = 15;   // p <= 32768: the padded row fits the LDS (128 KB)

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
  float* x = X + i * ldx;
  for (int c = tid; c < k; c += nt) {
    const int r = rows[c];
    x[c] = (r >= 0 && r < p) ? L[r] * scale : __builtin_nanf("");
  }
}

}  // namespace

int srht_max_log() { return kSrhtMaxLog; }

eogp_status srht_project(const float* Z, int64_t ldz, int64_t N, int64_t m, const int8_t* signs,
                         const int32_t* rows, int64_t k, float* X, int64_t ldx, hipStream_t s) {
  if (N == 0) return EOGP_OK;
  int logp = 0;
  while ((int64_t(1) << logp) < m) ++logp;
  const int p = 1 << logp;
  const size_t lds = (size_t)p * sizeof(float);
  static bool attr_set = false;     // the attribute is per kernel, not per device
  if (!attr_set) {
    EOGP_HIP(hipFuncSetAttribute((const void*)k_srht, hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)(sizeof(float) << kSrhtMaxLog)));
    attr_set = true;
  }
  const int nt = std::max(64, std::min(1024, p / 4));
  const float scale = (float)(1.0 / std::sqrt((double)k));
  timing::Scope ts(EOGP_KT_SRHT, s);
  for (int64_t r0 = 0; r0 < N; r0 += 0x7FFFFFFF) {
    const int64_t nr = std::min<int64_t>(N - r0, 0x7FFFFFFF);
    hipLaunchKernelGGL(k_srht, dim3((unsigned)nr), dim3(nt), lds, s, Z + r0 * ldz, ldz, (int)m,
                       logp, signs, rows, (int)k, scale, X + r0 * ldx, ldx);
    EOGP_LAUNCH_CHECK("srht_project");
  }
  return EOGP_OK;
}

}  // namespace eogp
