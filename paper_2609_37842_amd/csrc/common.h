// Internal helpers shared by the EOGP HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string>

#include "eogp.h"

namespace eogp {

// ---- status / error reporting ------------------------------------------------
void set_error(const std::string& msg);
eogp_status fail(eogp_status st, const std::string& msg);
eogp_status check_hip(hipError_t e, const char* what);

#define EOGP_HIP(call)                                        \
  do {                                                        \
    hipError_t e_ = (call);                                   \
    if (e_ != hipSuccess) return ::eogp::check_hip(e_, #call); \
  } while (0)

#define EOGP_LAUNCH_CHECK(what)                                 \
  do {                                                          \
    hipError_t e_ = hipGetLastError();                          \
    if (e_ != hipSuccess) return ::eogp::check_hip(e_, what);   \
  } while (0)

// Raises kernel `fn`'s dynamic-LDS limit to `bytes` on the current device, once
// per (kernel, device); safe to call from several host threads.
eogp_status ensure_dynamic_lds(const void* fn, int bytes);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Bump allocator over a caller workspace (256-byte aligned slices).
struct Carve {
  char* base;
  size_t cap;
  size_t used = 0;
  Carve(void* b, size_t c) : base(static_cast<char*>(b)), cap(c) {}
  template <typename T>
  T* take(size_t count) {
    size_t off = used;
    used = align256(used + count * sizeof(T));
    return reinterpret_cast<T*>(base + off);
  }
  bool ok() const { return used <= cap; }
};

// ---- vector types for MFMA operands ------------------------------------------
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;

constexpr int kWave = 64;
constexpr int kXcds = 8;        // MI355X: 8 accelerator complex dies, 32 CUs each
constexpr int kCus = 256;

// fp64 -> fp16 bit pattern, round to nearest even, overflow -> inf (IEEE).
__device__ __forceinline__ uint16_t f64_to_f16_rne(double x) {
  uint64_t u = __double_as_longlong(x);
  uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
  uint64_t a = u & 0x7FFFFFFFFFFFFFFFull;
  if (a >= 0x7FF0000000000000ull)  // inf or NaN
    return sign | (a > 0x7FF0000000000000ull ? 0x7E00u : 0x7C00u);
  int e = (int)(a >> 52) - 1023;           // unbiased exponent
  uint64_t mant = (a & 0xFFFFFFFFFFFFFull) | (1ull << 52);
  if (e > 15) return sign | 0x7C00u;       // certainly overflows
  int shift;                                // bits dropped from the 53-bit significand
  uint32_t exp16;
  if (e >= -14) {                           // normal fp16 range
    shift = 52 - 10;
    exp16 = (uint32_t)(e + 15);
  } else {                                  // subnormal fp16: value = m * 2^-24
    shift = 52 - 10 + (-14 - e);
    exp16 = 0;
    if (shift > 63) return sign;            // far below half the smallest subnormal
  }
  uint64_t kept = mant >> shift;
  uint64_t rem = mant & ((1ull << shift) - 1);
  uint64_t half = 1ull << (shift - 1);
  if (rem > half || (rem == half && (kept & 1))) kept += 1;
  // kept includes the implicit bit for normals (bit 10); carry may bump exponent.
  uint32_t bits;
  if (exp16 == 0) {
    bits = (uint32_t)kept;                  // subnormal (may round up to min normal)
  } else {
    if (kept >= (1ull << 11)) { kept >>= 1; exp16 += 1; }
    if (exp16 >= 31) return sign | 0x7C00u;
    bits = (exp16 << 10) | (uint32_t)(kept & 0x3FFu);
  }
  return sign | (uint16_t)bits;
}

}  // namespace eogp

namespace eogp {
// 16-bit float conversions (round to nearest even, as the hardware converts).
__device__ __forceinline__ uint16_t to_bf16_bits(float v) {
  __bf16 h = (__bf16)v;
  return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}
__device__ __forceinline__ uint16_t to_f16_bits(float v) {
  _Float16 h = (_Float16)v;
  return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}
}  // namespace eogp
