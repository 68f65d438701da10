// MFMA contraction core for gfx950: C = A * B^T, K-contiguous operands.
//
// Tiling: a 256-thread workgroup (4 wave64s in a 2 x 2 grid) owns a 128 x 128
// output tile; each wave computes 64 x 64 with 2 x 2 v_mfma_f32_32x32x16
// blocks. K advances 32 at a time through LDS (rows padded to 40 halves so
// the 16-byte fragment reads of 16 consecutive rows hit distinct banks); the
// next K-slice is fetched into registers while the current one is multiplied.
// fp32 A is converted while it is staged: rounded to the MFMA type, or split
// into high and low parts for the accurate mode, whose cross terms
// (A_lo*B_hi, A_hi*B_lo, A_hi*B_hi) accumulate in the same fp32 registers.
//
// The grid is persistent. Tiles are dealt out in contiguous ranges per XCD
// (workgroup b runs on XCD b % 8), so the workgroups that share an A row-block
// (rotations) or a B column-block (PCA, n_major) run together on one XCD and
// hit the same L2.
#include <algorithm>

#include "gemm.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int BM = 128, BN = 128, BK = 32, LDK = BK + 8;

struct KParams {
  GemmArgs g;
  int a_vec;  // A rows allow 16-byte loads
  int b_vec;  // B rows allow 16-byte loads
};

template <bool F16>
__device__ __forceinline__ uint16_t cvt16(float v) {
  if constexpr (F16) return to_f16_bits(v);
  else return to_bf16_bits(v);
}
template <bool F16>
__device__ __forceinline__ float back16(uint16_t b) {
  if constexpr (F16) return f16_bits_to_f32(b);
  else return bf16_bits_to_f32(b);
}

template <bool F16>
__device__ __forceinline__ f32x16 mfma32(const uint4& a, const uint4& b, f32x16 c) {
  if constexpr (F16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo, uint16_t hi) {
  return (uint32_t)lo | ((uint32_t)hi << 16);
}

template <int AT, int AP, int BP, bool F16>
__global__ __launch_bounds__(256, 2) void k_gemm(KParams kp) {
  const GemmArgs& g = kp.g;
  __shared__ __attribute__((aligned(16))) uint16_t sA[AP][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[BP][BN * LDK];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t M = g.M_dev ? (int64_t)(*g.M_dev) : g.M;
  const int64_t N = g.N, K = g.K;
  const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int64_t n_tiles = tiles_m * tiles_n;
  const int64_t nk = (K + BK - 1) / BK;

  const int G = gridDim.x, b = blockIdx.x;
  int64_t t_begin, t_end, t_step;
  if (G >= kXcds && G % kXcds == 0) {
    const int xcd = b % kXcds;
    const int64_t per = G / kXcds, chunk = (n_tiles + kXcds - 1) / kXcds;
    t_begin = xcd * chunk + b / kXcds;
    t_end = std::min<int64_t>((int64_t)(xcd + 1) * chunk, n_tiles);
    t_step = per;
  } else {
    t_begin = b;
    t_end = n_tiles;
    t_step = G;
  }

  const int ar = tid >> 1, ak = (tid & 1) * 16;   // A staging: row, first k
  const int br = tid >> 1, bk = (tid & 1) * 16;   // B staging
  const int wm = (wid >> 1) * 64, wn = (wid & 1) * 64;

  for (int64_t t = t_begin; t < t_end; t += t_step) {
    int64_t tm, tn;
    if (g.n_major) { tn = t / tiles_m; tm = t % tiles_m; }
    else { tm = t / tiles_n; tn = t % tiles_n; }
    const int64_t m0 = tm * BM, n0 = tn * BN;

    const int64_t arow = m0 + ar;
    const bool a_ok = arow < M;
    int64_t asrc = 0;
    if (a_ok) asrc = g.a_rows ? (int64_t)g.a_rows[arow] : arow;
    const int64_t brow = n0 + br;
    const bool b_ok = brow < N;

    // staging registers
    float ra[AT == 0 ? 16 : 1];
    uint4 ra16[2];
    uint4 rb[BP][2];

    auto load = [&](int64_t kt) {
      const int64_t ka = kt * BK + ak;
      if constexpr (AT == 0) {
        const float* p = static_cast<const float*>(g.A) + asrc * g.lda + ka;
        if (a_ok && kp.a_vec && ka + 16 <= K) {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            float4 x = reinterpret_cast<const float4*>(p)[v];
            ra[4 * v + 0] = x.x; ra[4 * v + 1] = x.y; ra[4 * v + 2] = x.z; ra[4 * v + 3] = x.w;
          }
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) ra[e] = (a_ok && ka + e < K) ? p[e] : 0.f;
        }
      } else {
        const uint16_t* p = static_cast<const uint16_t*>(g.A) + asrc * g.lda + ka;
        if (a_ok && kp.a_vec && ka + 16 <= K) {
          ra16[0] = reinterpret_cast<const uint4*>(p)[0];
          ra16[1] = reinterpret_cast<const uint4*>(p)[1];
        } else {
          uint16_t h[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) h[e] = (a_ok && ka + e < K) ? p[e] : (uint16_t)0;
          ra16[0] = make_uint4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
          ra16[1] = make_uint4(pack2(h[8], h[9]), pack2(h[10], h[11]), pack2(h[12], h[13]), pack2(h[14], h[15]));
        }
      }
      const int64_t kb = kt * BK + bk;
#pragma unroll
      for (int part = 0; part < BP; ++part) {
        const uint16_t* base = part == 0 ? g.B_hi : g.B_lo;
        const uint16_t* p = base + brow * g.ldb + kb;
        if (b_ok && kp.b_vec && kb + 16 <= K) {
          rb[part][0] = reinterpret_cast<const uint4*>(p)[0];
          rb[part][1] = reinterpret_cast<const uint4*>(p)[1];
        } else {
          uint16_t h[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) h[e] = (b_ok && kb + e < K) ? p[e] : (uint16_t)0;
          rb[part][0] = make_uint4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
          rb[part][1] = make_uint4(pack2(h[8], h[9]), pack2(h[10], h[11]), pack2(h[12], h[13]), pack2(h[14], h[15]));
        }
      }
    };

    auto stage = [&]() {
      uint4* dA0 = reinterpret_cast<uint4*>(&sA[0][ar * LDK + ak]);
      if constexpr (AT == 0) {
        uint16_t hi[16], lo[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          hi[e] = cvt16<F16>(ra[e]);
          if constexpr (AP == 2) lo[e] = cvt16<F16>(ra[e] - back16<F16>(hi[e]));
        }
        dA0[0] = make_uint4(pack2(hi[0], hi[1]), pack2(hi[2], hi[3]), pack2(hi[4], hi[5]), pack2(hi[6], hi[7]));
        dA0[1] = make_uint4(pack2(hi[8], hi[9]), pack2(hi[10], hi[11]), pack2(hi[12], hi[13]), pack2(hi[14], hi[15]));
        if constexpr (AP == 2) {
          uint4* dA1 = reinterpret_cast<uint4*>(&sA[AP - 1][ar * LDK + ak]);
          dA1[0] = make_uint4(pack2(lo[0], lo[1]), pack2(lo[2], lo[3]), pack2(lo[4], lo[5]), pack2(lo[6], lo[7]));
          dA1[1] = make_uint4(pack2(lo[8], lo[9]), pack2(lo[10], lo[11]), pack2(lo[12], lo[13]), pack2(lo[14], lo[15]));
        }
      } else {
        dA0[0] = ra16[0];
        dA0[1] = ra16[1];
      }
#pragma unroll
      for (int part = 0; part < BP; ++part) {
        uint4* dB = reinterpret_cast<uint4*>(&sB[part][br * LDK + bk]);
        dB[0] = rb[part][0];
        dB[1] = rb[part][1];
      }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    load(0);
    stage();
    __syncthreads();
    for (int64_t kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) load(kt + 1);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ko = ks * 16 + 8 * (lane >> 5);
        uint4 fa[AP][2], fb[BP][2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int part = 0; part < AP; ++part)
            fa[part][i] = *reinterpret_cast<const uint4*>(&sA[part][(wm + 32 * i + (lane & 31)) * LDK + ko]);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int part = 0; part < BP; ++part)
            fb[part][j] = *reinterpret_cast<const uint4*>(&sB[part][(wn + 32 * j + (lane & 31)) * LDK + ko]);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            if constexpr (AP == 2) acc[i][j] = mfma32<F16>(fa[AP - 1][i], fb[0][j], acc[i][j]);
            if constexpr (BP == 2) acc[i][j] = mfma32<F16>(fa[0][i], fb[BP - 1][j], acc[i][j]);
            acc[i][j] = mfma32<F16>(fa[0][i], fb[0][j], acc[i][j]);
          }
      }
      __syncthreads();
      if (kt + 1 < nk) {
        stage();
        __syncthreads();
      }
    }

    // epilogue: lane holds column (lane & 31), rows 8*(r/4) + 4*(lane/32) + r%4
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int64_t col = n0 + wn + 32 * j + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = m0 + wm + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (row < M && col < N) g.C[row * g.ldc + col] = acc[i][j][r];
        }
      }
  }
}

template <int AT, int AP, int BP, bool F16>
eogp_status launch(const KParams& kp, hipStream_t s) {
  const GemmArgs& g = kp.g;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  if (tiles == 0) return EOGP_OK;
  int64_t grid = std::min<int64_t>(tiles, 2 * kCus);
  if (grid >= kXcds) grid = grid / kXcds * kXcds;
  timing::Scope ts(g.timing_class, s);
  hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16>), dim3((unsigned)grid), dim3(256), 0, s, kp);
  EOGP_LAUNCH_CHECK("gemm launch");
  return EOGP_OK;
}

}  // namespace

eogp_status gemm_nt(const GemmArgs& g, AType a_type, int a_parts, int b_parts, bool f16,
                    hipStream_t s) {
  KParams kp;
  kp.g = g;
  const size_t a_elem = a_type == AType::F32 ? 4 : 2;
  const int a_align = a_type == AType::F32 ? 4 : 8;
  kp.a_vec = (g.lda % a_align == 0) && ((uintptr_t)g.A % 16 == 0);
  kp.b_vec = (g.ldb % 8 == 0) && ((uintptr_t)g.B_hi % 16 == 0) &&
             (g.B_lo == nullptr || (uintptr_t)g.B_lo % 16 == 0);
  (void)a_elem;
  const bool A32 = a_type == AType::F32;
  if (b_parts == 2 && g.B_lo == nullptr) return fail(EOGP_ERR_INVALID, "gemm: missing B low part");
  if (!A32 && a_parts != 1) return fail(EOGP_ERR_INVALID, "gemm: 16-bit A cannot be split");
  if (A32 && a_parts == 1 && b_parts == 1 && !f16) return launch<0, 1, 1, false>(kp, s);
  if (A32 && a_parts == 2 && b_parts == 2 && !f16) return launch<0, 2, 2, false>(kp, s);
  if (A32 && a_parts == 2 && b_parts == 1 && !f16) return launch<0, 2, 1, false>(kp, s);
  if (A32 && a_parts == 1 && b_parts == 1 && f16) return launch<0, 1, 1, true>(kp, s);
  if (A32 && a_parts == 2 && b_parts == 1 && f16) return launch<0, 2, 1, true>(kp, s);
  if (!A32 && b_parts == 1 && !f16) return launch<1, 1, 1, false>(kp, s);
  if (!A32 && b_parts == 2 && !f16) return launch<1, 1, 2, false>(kp, s);
  return fail(EOGP_ERR_UNSUPPORTED, "gemm: unsupported operand combination");
}

}  // namespace eogp
