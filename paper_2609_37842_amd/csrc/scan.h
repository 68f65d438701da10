// Single-workgroup exclusive prefix sums used by the plan builder and the token
// compaction. The input sizes here are modest (per-block counts, per-example
// token counts, per-tile counts), so one workgroup looping over chunks is
// enough and keeps the result deterministic.
#pragma once
#include "common.h"

namespace eogp {

// In-place exclusive scan of data[0..n); data[n] receives the total.
template <typename T>
__global__ __launch_bounds__(1024) void k_scan_exclusive(T* data, int64_t n) {
  __shared__ T part[1024];
  __shared__ T carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t base = 0; base < n; base += 1024) {
    int64_t i = base + threadIdx.x;
    T v = (i < n) ? data[i] : T(0);
    part[threadIdx.x] = v;
    __syncthreads();
    // Hillis-Steele inclusive scan in LDS.
    for (int off = 1; off < 1024; off <<= 1) {
      T add = (threadIdx.x >= (unsigned)off) ? part[threadIdx.x - off] : T(0);
      __syncthreads();
      part[threadIdx.x] += add;
      __syncthreads();
    }
    T incl = part[threadIdx.x];
    T c = carry;
    if (i < n) data[i] = c + incl - v;
    __syncthreads();
    if (threadIdx.x == 1023) carry = c + incl;
    __syncthreads();
  }
  if (threadIdx.x == 0) data[n] = carry;
}

template <typename T>
inline hipError_t scan_exclusive(T* data, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL((k_scan_exclusive<T>), dim3(1), dim3(1024), 0, s, data, n);
  return hipGetLastError();
}

// Wave-level exclusive prefix count of `pred` among active lanes.
__device__ __forceinline__ int wave_prefix_count(bool pred, uint64_t* mask_out) {
  uint64_t m = __ballot(pred);
  if (mask_out) *mask_out = m;
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
}

}  // namespace eogp
