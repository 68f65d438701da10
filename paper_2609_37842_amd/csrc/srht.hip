// Random second stage, EOGP-R (Appendix B.2, eq. app_srht_definition):
//   x = sqrt(p/k) R H_p D J z,  p = 2^ceil(log2 m),
// with H_p the orthonormal Walsh-Hadamard matrix. With W the unnormalised
// transform in Sylvester order (entry (r, i) = (-1)^popcount(r & i)),
//   x_c = W(D J z)[rows[c]] / sqrt(k).
//
// 1024 <= p <= 16384: one 256-thread workgroup per row, E = p / 256 values per
// thread in registers. The transform is separable over the bits of the index,
// and each bit's butterflies are applied once: (a) element t + 256 j of the
// signed, zero-padded row is loaded into register j of thread t (coalesced) and
// the bits 8 .. log2 p - 1 (those of j) are transformed in registers; (b) the
// values go to LDS (one pad word per 64, so the next reads are free of bank
// conflicts) and thread t takes elements E t .. E t + E - 1, transforms the low
// log2 E bits in registers and the bits log2 E .. 7 (those of the lane index)
// across lanes (DPP or shuffles); (c) the result goes to LDS once more and the
// kept rows are gathered and scaled. LDS traffic: three row writes/reads and
// the gather, against two per radix-4 stage before.
//
// Other p <= 32768: one workgroup per row, the butterfly stages in LDS two at a time
// (radix 4: each thread combines four elements h apart), one radix-2 stage
// first when log2 p is odd. Cost either way: p log2 p additions per row, HBM
// traffic m + k floats per row.
//
// p > 32768 (up to 2^20): W_p = W_p1 (x) W_p2 in Sylvester order (index
// i = i1 p2 + i2, p2 = 32768, p1 = p / p2 <= 32). One workgroup per (row,
// chunk i1) transforms its 32768 entries along i2 in LDS as above and writes
// them to the workspace; the gather then forms each kept coordinate
// r = r1 p2 + r2 as the length-p1 transform along i1 of that column,
//   x_c = sum_j (-1)^popcount(r1 & j) S[j p2 + r2] / sqrt(k).
// Extra HBM traffic: p floats written and k p1 read per row.
#include <cmath>
#include <type_traits>

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

// Unnormalised Walsh-Hadamard transform of E values in registers (index j).
template <int E>
__device__ __forceinline__ void fwht_regs(float (&v)[E]) {
#pragma unroll
  for (int h = 1; h < E; h <<= 1)
#pragma unroll
    for (int j = 0; j < E; ++j)
      if ((j & h) == 0) {
        const float a = v[j], b = v[j + h];
        v[j] = a + b;
        v[j + h] = a - b;
      }
}

// The value of lane (lane ^ 2^b) (b < 6): DPP within quads for b < 2.
template <int B>
__device__ __forceinline__ float lane_xor(float x) {
  if constexpr (B == 0)
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
  else if constexpr (B == 1)
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));
  else
    return __shfl_xor(x, 1 << B);
}

// LDS slot of element idx: one pad word per 2^SH elements, so the stride-2^SH
// reads of the transposed pass fall into distinct banks.
template <int SH>
__device__ __forceinline__ int srht_pad(int idx) { return idx + (idx >> SH); }

// LT: log2 of the threads per row (8 or 9).
template <int LOGP, int LT>
__global__ __launch_bounds__(1 << LT) void k_srht_reg(const float* __restrict__ Z, int64_t ldz, int m,
                                                  const int8_t* __restrict__ signs,
                                                  const int32_t* __restrict__ rows, int k,
                                                  float scale, float* __restrict__ X, int64_t ldx) {
  constexpr int NT = 1 << LT, P = 1 << LOGP, E = P >> LT, LE = LOGP - LT;
  static_assert(LT == 8 || LT == 9, "256 or 512 threads per row");
  static_assert(LE >= 1 && LT - LE <= 6, "the cross-lane bits (thread bits 0 .. LT - LE - 1) lie inside a wave");
  extern __shared__ float L[];
  const int t = threadIdx.x;
  const int64_t i = blockIdx.x;
  const float* z = Z + i * ldz;
  float v[E];
  // (a) element t + NT j into register j: loads at clamped indices, selected
  // afterwards (no branches, so all of them are in flight at once)
  int8_t sg[E];
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const int idx = min(t + NT * j, m - 1);
    v[j] = z[idx];
    sg[j] = signs[idx];
  }
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const bool in = t + NT * j < m;
    v[j] = in ? (sg[j] < 0 ? -v[j] : v[j]) : 0.f;
  }
  fwht_regs<E>(v);                                  //     bits LT .. LOGP - 1
#pragma unroll
  for (int j = 0; j < E; ++j) L[srht_pad<LE>(t + NT * j)] = v[j];
  __syncthreads();
#pragma unroll
  for (int e = 0; e < E; ++e) v[e] = L[srht_pad<LE>(E * t + e)];   // (b) bits 0 .. LE - 1
  fwht_regs<E>(v);
  auto cross = [&](auto b_c) __attribute__((always_inline)) {  //     bit LE + b, lane bit b
    constexpr int B = decltype(b_c)::value;
    const bool hi = (t >> B) & 1;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float o = lane_xor<B>(v[e]);
      v[e] = hi ? o - v[e] : v[e] + o;
    }
  };
  if constexpr (LT - LE > 0) cross(std::integral_constant<int, 0>{});
  if constexpr (LT - LE > 1) cross(std::integral_constant<int, 1>{});
  if constexpr (LT - LE > 2) cross(std::integral_constant<int, 2>{});
  if constexpr (LT - LE > 3) cross(std::integral_constant<int, 3>{});
  if constexpr (LT - LE > 4) cross(std::integral_constant<int, 4>{});
  if constexpr (LT - LE > 5) cross(std::integral_constant<int, 5>{});
  __syncthreads();                                  // every (b) read is done
#pragma unroll
  for (int e = 0; e < E; ++e) L[srht_pad<LE>(E * t + e)] = v[e];   // (c)
  __syncthreads();
  // gather of the kept rows (k <= p, so at most E per thread): every index
  // requested before the first is used
  float* x = X + i * ldx;
  int r[E];
#pragma unroll
  for (int e = 0; e < E; ++e) r[e] = rows[min(t + NT * e, k - 1)];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int c = t + NT * e;
    if (c < k) x[c] = (r[e] >= 0 && r[e] < P) ? L[srht_pad<LE>(r[e])] * scale : __builtin_nanf("");
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
  if (logp >= 10 && logp <= 14) {
    // 2^10 <= p <= 2^14: one row per workgroup, p / NT values per thread in
    // registers; 512 threads from p = 2^12 (more waves per CU for the same LDS)
    const int lt = logp >= 12 ? 9 : 8;
    const void* fns[5] = {(const void*)k_srht_reg<10, 8>, (const void*)k_srht_reg<11, 8>,
                          (const void*)k_srht_reg<12, 9>, (const void*)k_srht_reg<13, 9>,
                          (const void*)k_srht_reg<14, 9>};
    const int lds = (int)(sizeof(float) * (((size_t)1 << logp) + ((size_t)1 << lt)));   // p + NT slots
    const eogp_status st = ensure_dynamic_lds(fns[logp - 10], lds);
    if (st != EOGP_OK) return st;
    timing::Scope ts(EOGP_KT_SRHT, s);
    for (int64_t r0 = 0; r0 < N; r0 += 0x7FFFFFFF) {
      const int64_t nr = std::min<int64_t>(N - r0, 0x7FFFFFFF);
      const dim3 g((unsigned)nr), b(1u << lt);
      const float* z0 = Z + r0 * ldz;
      float* x0 = X + r0 * ldx;
      switch (logp) {
        case 10: hipLaunchKernelGGL((k_srht_reg<10, 8>), g, b, lds, s, z0, ldz, (int)m, signs, rows, (int)k, scale, x0, ldx); break;
        case 11: hipLaunchKernelGGL((k_srht_reg<11, 8>), g, b, lds, s, z0, ldz, (int)m, signs, rows, (int)k, scale, x0, ldx); break;
        case 12: hipLaunchKernelGGL((k_srht_reg<12, 9>), g, b, lds, s, z0, ldz, (int)m, signs, rows, (int)k, scale, x0, ldx); break;
        case 13: hipLaunchKernelGGL((k_srht_reg<13, 9>), g, b, lds, s, z0, ldz, (int)m, signs, rows, (int)k, scale, x0, ldx); break;
        default: hipLaunchKernelGGL((k_srht_reg<14, 9>), g, b, lds, s, z0, ldz, (int)m, signs, rows, (int)k, scale, x0, ldx); break;
      }
    }
    EOGP_LAUNCH_CHECK("srht_project");
    return EOGP_OK;
  }
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
