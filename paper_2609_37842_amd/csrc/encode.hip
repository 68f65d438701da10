// Second stage (eq. second_stage) and one-bit encoding (eq. onebit).
#include <algorithm>

#include "gemm.h"
#include "timing.h"

namespace eogp {
namespace {

// One workgroup (4 waves) per row. A ballot of (x >= 0) over 64 consecutive
// coordinates is exactly 8 bytes of the least-significant-bit-first code;
// wave w takes the 64-coordinate chunks w, w + 4, ..., eight at a time so
// that eight loads are in flight per lane. |x| is summed in fp64 (per lane,
// then a fixed butterfly, then the four waves in order) and the mean is
// rounded once to fp16.
constexpr int kPackUnroll = 8;

//
// Tiled store (TILED): rows in tiles of 32; the 64 bytes of row r in 512-bit
// step s of the row (a module's steps start at step0) go to the 2 KB block
// (tile * steps_row + s), 16-byte piece p (bytes 16p .. 16p+15) at block
// offset (p % 2) * 1024 + ((p / 2) * 32 + r) * 16: the order in which the
// scoring pass's wave lanes take them (k a multiple of 512).
template <bool TILED>
__global__ __launch_bounds__(256) void k_sign_pack(const float* __restrict__ X, int64_t ldx,
                                                   int64_t N, int64_t k,
                                                   uint8_t* __restrict__ codes, int64_t cstride,
                                                   uint16_t* __restrict__ scales,
                                                   int64_t sstride, int word_store, int64_t row0,
                                                   int64_t steps_row, int64_t step0) {
  __shared__ double part[4];
  const int64_t i = blockIdx.x;
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float* x = X + i * ldx;
  uint8_t* c = codes + i * cstride;
  const int64_t grow = row0 + i;   // tiled: the row's place in the store
  uint8_t* tb = codes + ((grow >> 5) * steps_row + step0) * 2048 + (grow & 31) * 16;
  const int64_t nchunk = (k + 63) >> 6;
  double acc = 0.0;
  for (int64_t ch0 = wid; ch0 < nchunk; ch0 += 4 * kPackUnroll) {
    float v[kPackUnroll];
#pragma unroll
    for (int u = 0; u < kPackUnroll; ++u) {
      const int64_t cc = (ch0 + 4 * u) * 64 + lane;
      v[u] = cc < k ? x[cc] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kPackUnroll; ++u) {
      const int64_t ch = ch0 + 4 * u;
      if (ch >= nchunk) break;                     // uniform across the wave
      const int64_t c0 = ch * 64;
      const bool in = c0 + lane < k;
      const uint64_t word = __ballot(in && v[u] >= 0.f);
      acc += fabs((double)v[u]);                   // 0 beyond k
      const int64_t nbytes = std::min<int64_t>(8, (k - c0 + 7) >> 3);
      if constexpr (TILED) {
        // chunk ch = 8 bytes: step ch / 8, piece (ch % 8) / 2, half ch % 2
        const int pc = (int)((ch & 7) >> 1);
        if (lane == 0)
          *reinterpret_cast<uint64_t*>(tb + (ch >> 3) * 2048 + (pc & 1) * 1024 + (pc >> 1) * 512 +
                                       (ch & 1) * 8) = word;
      } else if (word_store && nbytes == 8) {
        if (lane == 0) *reinterpret_cast<uint64_t*>(c + (c0 >> 3)) = word;
      } else if (lane < nbytes) {
        c[(c0 >> 3) + lane] = (uint8_t)(word >> (8 * lane));
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) part[wid] = acc;
  __syncthreads();
  if (threadIdx.x == 0)
    scales[i * sstride] = f64_to_f16_rne(((part[0] + part[1]) + (part[2] + part[3])) / (double)k);
}

// fp32 P (column-major, [k][ldp]) -> bf16 high and low parts [k][ldo].
__global__ void k_split_p(const float* __restrict__ P, int64_t ldp, int64_t m, int64_t k,
                          int64_t ldo, uint16_t* __restrict__ hi, uint16_t* __restrict__ lo) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t col = idx / ldo, r = idx % ldo;
  const float v = (r < m && col < k) ? P[col * ldp + r] : 0.f;   // zero padding
  const uint16_t h = to_bf16_bits(v);
  hi[idx] = h;
  lo[idx] = to_bf16_bits(v - bf16_bits_to_f32(h));
}

}  // namespace

eogp_status sign_pack(const float* X, int64_t ldx, int64_t N, int64_t k, uint8_t* codes,
                      int64_t cstride, uint16_t* scales, int64_t sstride, hipStream_t s) {
  if (N == 0) return EOGP_OK;
  const int word_store = ((uintptr_t)codes % 8 == 0) && (cstride % 8 == 0);
  timing::Scope ts(EOGP_KT_SIGN_PACK, s);
  hipLaunchKernelGGL(k_sign_pack<false>, dim3((unsigned)N), dim3(256), 0, s, X, ldx, N, k,
                     codes, cstride, scales, sstride, word_store, (int64_t)0, (int64_t)0,
                     (int64_t)0);
  EOGP_LAUNCH_CHECK("sign_pack");
  return EOGP_OK;
}

eogp_status sign_pack_tiled(const float* X, int64_t ldx, int64_t N, int64_t k, int64_t row0,
                            uint8_t* codes, int64_t steps_row, int64_t step0, uint16_t* scales,
                            int64_t sstride, hipStream_t s) {
  if (N == 0) return EOGP_OK;
  timing::Scope ts(EOGP_KT_SIGN_PACK, s);
  hipLaunchKernelGGL(k_sign_pack<true>, dim3((unsigned)N), dim3(256), 0, s, X, ldx, N, k, codes,
                     (int64_t)0, scales, sstride, 0, row0, steps_row, step0);
  EOGP_LAUNCH_CHECK("sign_pack (tiled)");
  return EOGP_OK;
}

constexpr int kPcaMaxSplits = 8;

// Workspace: the split copy of an fp32 P (padded panel), then split-K partials.
size_t pca_split_copy_bytes(int64_t m, int64_t k, eogp_dtype p_dtype) {
  if (p_dtype != EOGP_F32) return 0;
  const int64_t ldo = round_up(m, 32), rows = round_up(k, 256);
  return 2 * align256((size_t)rows * ldo * 2);
}

size_t pca_ws(int64_t N, int64_t m, int64_t k, eogp_dtype p_dtype) {
  return pca_split_copy_bytes(m, k, p_dtype) +
         align256(gemm_partial_bytes(N, k, kPcaMaxSplits));
}

eogp_status pca_project(const void* Z, eogp_dtype z_dtype, int64_t ldz, int64_t N, int64_t m,
                        const void* P, eogp_dtype p_dtype, int64_t ldp, int64_t k, float* X,
                        int64_t ldx, bool accurate, void* ws, size_t ws_bytes, hipStream_t s) {
  if (N == 0 || k == 0) return EOGP_OK;
  GemmArgs g;
  g.A = Z;
  g.lda = ldz;
  g.C = X;
  g.ldc = ldx;
  g.M = N;
  g.N = k;
  g.K = m;
  // Units run split by split (each XCD's contiguous range is then one K
  // range), column tile by column tile with the row tiles of a column tile
  // together: each P slice is fetched once and shared by the row tiles, and
  // the Z slices of the K range stay in that XCD's L2.
  g.n_major = true;
  g.split_major = true;
  g.timing_class = EOGP_KT_PCA_GEMM;
  const size_t copy = pca_split_copy_bytes(m, k, p_dtype);
  if (ws_bytes < copy) return fail(EOGP_ERR_WORKSPACE, "pca_project: workspace too small");
  // Split-K scratch is optional: without it the projection runs unsplit.
  if (ws && ws_bytes >= copy + gemm_partial_bytes(N, k, 2)) {
    g.partial = reinterpret_cast<float*>(static_cast<char*>(ws) + copy);
    g.max_splits = (int)std::min<int64_t>(
        kPcaMaxSplits, (int64_t)((ws_bytes - copy) / gemm_partial_bytes(N, k, 1)));
  }
  if (p_dtype == EOGP_F32) {   // (Z is fp32 here)
    const int64_t ldo = round_up(m, 32), rows = round_up(k, 256);
    Carve cv(ws, ws_bytes);
    uint16_t* hi = cv.take<uint16_t>((size_t)rows * ldo);
    uint16_t* lo = cv.take<uint16_t>((size_t)rows * ldo);
    const int64_t total = rows * ldo;
    hipLaunchKernelGGL(k_split_p, dim3((unsigned)ceil_div(total, 256)), dim3(256), 0, s,
                       static_cast<const float*>(P), ldp, m, k, ldo, hi, lo);
    EOGP_LAUNCH_CHECK("pca split");
    g.B_hi = hi;
    g.B_lo = lo;
    g.ldb = ldo;
    g.b_padded = true;
    return gemm_nt(g, AType::F32, accurate ? 2 : 1, accurate ? 2 : 1, false, s);
  }
  g.B_hi = static_cast<const uint16_t*>(P);
  g.ldb = ldp;
  // A caller's P needs no bounds checks when its shape already matches the tiles.
  g.b_padded = (m % 32 == 0) && (k % 256 == 0);
  // 16-bit Z has P's type (checked by the caller): one product on that type's MFMA
  if (z_dtype != EOGP_F32) return gemm_nt(g, AType::B16, 1, 1, p_dtype == EOGP_F16, s);
  return gemm_nt(g, AType::F32, accurate ? 2 : 1, 1, p_dtype == EOGP_F16, s);
}

}  // namespace eogp
