// MFMA contraction core for gfx950: C = A * B^T, K-contiguous operands.
//
// Two kernels share the staging conventions below.
//
// k_gemm_p (single-pass products on aligned operands: the rotations, and the
// PCA projection with split-K). A workgroup owns a 256 x 256 output tile with
// 8 wave64s (two per SIMD, 128 x 64 each; the kernel also builds with 4 waves
// of 128 x 128) computing with v_mfma_f32_32x32x16 blocks. K advances 32 at a
// time through two LDS stages. One iteration per slice, one block barrier:
// the first half's MFMAs issue, A fragment by A fragment, beside the staging
// of the next slice (B, then A converted while it is written) and the global
// requests for later slices, and each A fragment's register is refilled with
// the second half's fragment as soon as its MFMAs have issued; after the
// barrier the second half's MFMAs issue the same way while the next slice's
// first-half fragments are read. A and B are requested two slices before they
// are staged (two register buffers each). A wave whose columns all lie in the
// padding of the last column tile stages its share and skips its fragment
// reads and MFMAs.
//
// k_gemm (everything else: bf16x3 products, unaligned or bounds-checked
// operands). A 512-thread workgroup (8 waves, two per SIMD)
// owns a 256 x BN tile (BN = 256 or 128, whichever pads N less); each wave
// computes 128 x BN/4. Slice k+1 sits in registers while slice k is multiplied
// from LDS; then it is converted and written to the other stage and slice k+2
// is requested, then one barrier.
//
// Common conventions. LDS rows are 64 bytes (32 halves) without padding; the
// four 16-byte chunks of row r are XOR-swizzled by (r / 4) % 4, which makes the
// MFMA fragment reads (32 consecutive rows, two chunks) and the staging writes
// (whole rows, 4 or 8 lanes per row) free of bank conflicts. Rows beyond M
// read a copy of a valid row (their products land in output rows that are
// never stored, or in fp16 output rows nobody reads), and a ragged last
// K-slice is processed first, by the only bounds-checked load. B operands are
// padded panels (rows to 256, K to a multiple of 32, zero-filled) or, for
// general caller layouts, checked loads.
//
// Precision. fp32 A is converted while it is staged: rounded to the MFMA type,
// or split into high and low parts (accurate mode), whose cross terms
// (A_lo*B_hi, A_hi*B_lo, A_hi*B_hi) accumulate into the same fp32 registers.
//
// Schedule. Grids are persistent, one workgroup per CU. Work units
// (tile, K-split) are dealt out in contiguous ranges per XCD (workgroup b runs
// on XCD b % 8), so workgroups sharing an A row-block (rotations) or a B
// column-block (PCA, n_major) run together on one XCD and hit the same L2.
// k_gemm_p can run two independent products in one launch (the two rotations
// of a module): each XCD's range then holds its share of the first product's
// units followed by its share of the second's, and the XCD's workgroups take
// positions from a per-XCD atomic counter, so the short units of the second
// product fill the last round of the first instead of leaving CUs idle.
// Small-M problems split K; each split writes its own fp32 partial tile and a
// second kernel adds the partials in split order (deterministic).
#include <algorithm>
#include <type_traits>

#include "gemm.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int BM = 256, BK = 32, NTHR = 512;

struct KParams {
  GemmArgs g;
  int64_t kc;       // K per split (multiple of BK)
  int splits;
  // k_gemm_p only: an optional second product in the same launch (one split)
  GemmArgs g2;
  int64_t kc2 = 0;
  int nprob = 1;
};

__global__ void k_zero_sched(int32_t* __restrict__ c) {
  if (threadIdx.x < kXcds) c[threadIdx.x] = 0;
}

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4u mk4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  v4u r;
  r.x = a; r.y = b; r.z = c; r.w = d;
  return r;
}
__device__ __forceinline__ uint32_t pack2(uint32_t lo, uint32_t hi) {
  return (lo & 0xFFFFu) | (hi << 16);
}

template <bool F16>
__device__ __forceinline__ uint16_t cvt16(float v) {
  if constexpr (F16) return to_f16_bits(v);
  else return to_bf16_bits(v);
}
template <bool F16>
__device__ __forceinline__ float back16(uint32_t b) {
  if constexpr (F16) return f16_bits_to_f32((uint16_t)b);
  else return bf16_bits_to_f32((uint16_t)b);
}

template <bool F16>
__device__ __forceinline__ f32x16 mfma32(const v4u& a, const v4u& b, f32x16 c) {
  if constexpr (F16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
}

// Offset (in halves) of 16-byte chunk `c` (0..3) of LDS row `r`. With the key
// (r >> 2) & 3, the 16-byte fragment reads of 32 consecutive rows at one chunk
// are conflict-free (measured with the LDS bank-conflict counter; the key
// (r >> 1) ^ (r >> 3) spent half of the read cycles in conflicts).
__device__ __forceinline__ int swz(int r, int c) {
  return r * BK + ((c ^ ((r >> 2) & 3)) << 3);
}

typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2v __attribute__((ext_vector_type(2)));
typedef float f32x2v __attribute__((ext_vector_type(2)));

// Two fp32 values -> one packed pair of the MFMA type (round to nearest even).
template <bool F16>
__device__ __forceinline__ uint32_t cvt_pair(float a, float b) {
  f32x2v v;
  v.x = a;
  v.y = b;
  if constexpr (F16) return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2v));
  else return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
}
// The two fp32 values a packed pair represents.
template <bool F16>
__device__ __forceinline__ f32x2v uncvt_pair(uint32_t p) {
  if constexpr (F16) {
    return __builtin_convertvector(__builtin_bit_cast(f16x2v, p), f32x2v);
  } else {
    f32x2v r;
    r.x = __uint_as_float(p << 16);
    r.y = __uint_as_float(p & 0xFFFF0000u);
    return r;
  }
}

typedef unsigned int v2u __attribute__((ext_vector_type(2)));

// Epilogue of one wave's WI x WJ blocks of 32 x 32 (rows r0.., columns c0..;
// r0 and c0 multiples of 32). Lane l holds column (l & 31) and rows
// 8 (r / 4) + 4 (l / 32) + r % 4 of each block. fp32 C: bounds-checked stores.
// 16-bit CT (fragment order, see GemmArgs; fp16 or bf16): four consecutive
// rows of one column are 8 contiguous bytes; no checks.
//
// The 16-bit fragment-order part (F16OUT: fp16 entries, else bf16).
// Rows 16p .. 16p+15 of a block are one 16-token group: lanes l < 32 hold
// rows +0..3 (q = 2p) and +8..11 (q = 2p+1), lanes l >= 32 rows +4..7 and
// +12..15. One swap between lane l and lane l + 32 gives lane l tokens 0..7
// and lane l + 32 tokens 8..15 of column l % 32, so each wave store writes
// one whole 1 KB block.
template <int WI, int WJ, bool F16OUT>
__device__ __forceinline__ void store_ct(const GemmArgs& g, int64_t r0, int64_t c0, int lane,
                                         const f32x16 (&acc)[WI][WJ]) {
  const int64_t groups = g.ldct / 16;
  const int half = lane >> 5;
#pragma unroll
  for (int i = 0; i < WI; ++i)
#pragma unroll
    for (int j = 0; j < WJ; ++j) {
      const int64_t cb = (c0 + 32 * j) / 32;
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const f32x16& a = acc[i][j];
        const uint32_t x0 = cvt_pair<F16OUT>(a[8 * p + 0], a[8 * p + 1]);
        const uint32_t x1 = cvt_pair<F16OUT>(a[8 * p + 2], a[8 * p + 3]);
        const uint32_t y0 = cvt_pair<F16OUT>(a[8 * p + 4], a[8 * p + 5]);
        const uint32_t y1 = cvt_pair<F16OUT>(a[8 * p + 6], a[8 * p + 7]);
        const auto s0 = __builtin_amdgcn_permlane32_swap(x0, y0, false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(x1, y1, false, false);
        const int64_t grp = (r0 + 32 * i + 16 * p) / 16;
        uint16_t* dst = g.CT + ((cb * groups + grp) * 32 + (lane & 31)) * 16 + 8 * half;
        // streaming store: the rotated tokens are read once, by a later
        // kernel, so their lines need not stay in L2 beside the token rows
        // that the unit's neighbours re-read
        __builtin_nontemporal_store(mk4(s0[0], s1[0], s0[1], s1[1]), reinterpret_cast<v4u*>(dst));
      }
    }
}

template <int WI, int WJ>
__device__ __forceinline__ void store_tile(const GemmArgs& g, float* C, int64_t ldc, int64_t M,
                                           int64_t N, int64_t r0, int64_t c0, int lane,
                                           const f32x16 (&acc)[WI][WJ]) {
  if (g.CT) {
    // the entry type is chosen once per tile (chosen per value pair, it
    // compiled to a branch around every conversion)
    if (g.ct_bf16) store_ct<WI, WJ, false>(g, r0, c0, lane, acc);
    else store_ct<WI, WJ, true>(g, r0, c0, lane, acc);
    return;
  }
#pragma unroll
  for (int i = 0; i < WI; ++i)
#pragma unroll
    for (int j = 0; j < WJ; ++j) {
      const int64_t col = c0 + 32 * j + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = r0 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (row < M && col < N) C[row * ldc + col] = acc[i][j][r];
      }
    }
}

// AT: 0 = fp32 A, 1 = 16-bit A. AV: A rows allow 16-byte loads (else fp32 A is
// loaded one element per lane, 32 lanes per row). BC: B is bounds-checked.
template <int AT, int AP, int BP, bool F16, int BN, bool AV, bool BC>
__global__ __launch_bounds__(NTHR, 1) void k_gemm(KParams kp) {
  constexpr int WI = 4;                  // 32-high row blocks per wave (128 rows)
  constexpr int WJ = BN / 128;           // 32-wide column blocks per wave (BN/4 columns)
  const GemmArgs& g = kp.g;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][AP][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BP][BN * BK];
  __shared__ int64_t sOff[BM];           // element offset of each A row (clamped to a valid row)

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t M = g.M_dev ? (int64_t)(*g.M_dev) : g.M;
  const int64_t N = g.N, K = g.K;
  const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int64_t n_units = tiles_m * tiles_n * kp.splits;

  const int G = gridDim.x, b = blockIdx.x;
  int64_t t_begin, t_end, t_step;
  if (G >= kXcds && G % kXcds == 0) {
    const int xcd = b % kXcds;
    const int64_t per = G / kXcds, chunk = (n_units + kXcds - 1) / kXcds;
    t_begin = xcd * chunk + b / kXcds;
    t_end = std::min<int64_t>((int64_t)(xcd + 1) * chunk, n_units);
    t_step = per;
  } else {
    t_begin = b;
    t_end = n_units;
    t_step = G;
  }

  const int wm = (wid >> 2) * 128, wn = (wid & 3) * (BN / 4);
  const float a_scale = g.a_scale;
  // Staging maps consecutive lanes to consecutive 16-byte pieces of one row, so
  // a wave-wide 16-byte load covers whole cache lines:
  //   fp32 A:   8 lanes per row (128 bytes), rows (tid >> 3) + 32 q, q = 0..7;
  //   16-bit A: 4 lanes per row (64 bytes),  rows (tid >> 2) + 64 q, q = 0..3;
  //   B:        4 lanes per row per part,    rows (tid >> 2) + 64 q, q < BN/64.
  constexpr int AQ = AT == 0 ? 4 : 2;     // A pieces per thread per slice
  constexpr int BQ = BN / 128;            // B pieces per thread per slice and part
  constexpr int NE = BM / (NTHR / 32);    // element A path: rows per thread
  const int a_r0 = AT == 0 ? (tid >> 3) : (tid >> 2);
  const int a_rs = AT == 0 ? NTHR / 8 : NTHR / 4;
  const int a_pc = AT == 0 ? (tid & 7) : (tid & 3);   // piece index within the row
  const int b_r0 = tid >> 2, b_pc = tid & 3;
  const int sc = tid & 31, sr = tid >> 5;   // element A path: column, first row (rows sr + 16e)

  for (int64_t u = t_begin; u < t_end; u += t_step) {
    int64_t t;
    int split;
    if (g.split_major) {
      split = (int)(u / (tiles_m * tiles_n));
      t = u % (tiles_m * tiles_n);
    } else {
      t = u / kp.splits;
      split = (int)(u % kp.splits);
    }
    int64_t tm, tn;
    if (g.n_major) { tn = t / tiles_m; tm = t % tiles_m; }
    else { tm = t / tiles_n; tn = t % tiles_n; }
    const int64_t m0 = tm * BM, n0 = tn * BN;
    const int64_t kbeg = split * kp.kc;
    const int64_t kend = std::min<int64_t>(K, kbeg + kp.kc);
    const int64_t nk = (kend - kbeg + BK - 1) / BK;
    const bool ragged = ((kend - kbeg) % BK) != 0;

    __syncthreads();                     // previous unit's readers of sOff / stages are done
    if (tid < BM) {
      const int64_t r = m0 + tid;
      const bool ok = r < M;
      const int64_t src = g.a_rows ? (int64_t)g.a_rows[ok ? r : m0] : (ok ? r : m0);
      sOff[tid] = src * g.lda;
    }
    __syncthreads();
    constexpr bool A16B = (AT == 1) || AV;      // 16-byte A path
    int64_t a_off[A16B ? AQ : 1];
    if constexpr (A16B) {
#pragma unroll
      for (int q = 0; q < AQ; ++q) a_off[q] = sOff[a_r0 + a_rs * q];
    }
    // B rows n0 + b_r0 + 64 q; rows beyond N (which feed unstored columns)
    // read row 0 instead.
    int64_t b_off[BQ];
#pragma unroll
    for (int q = 0; q < BQ; ++q) {
      const int64_t brow = n0 + b_r0 + (NTHR / 4) * q;
      b_off[q] = (brow < N ? brow : 0) * g.ldb + 8 * b_pc;
    }

    // Slice order: a ragged last slice first, then the full slices in order.
    auto slice_k0 = [&](int64_t i) -> int64_t {
      const int64_t s = ragged ? (i == 0 ? nk - 1 : i - 1) : i;
      return kbeg + s * BK;
    };

    // Register staging of one slice: A rows (from HBM) and B panel rows (small,
    // L2-resident). On the 16-byte paths A is kept in two buffers, so each A
    // slice is requested two slices before it is staged; B one slice before.
    struct ARegs {
      v4f ra[AT == 0 && AV ? AQ : 1];       // fp32 A (16-byte path)
      float re[AT == 0 && !AV ? NE : 1];    // fp32 A (element path)
      v4u ra16[AT == 0 ? 1 : AQ];           // 16-bit A
    };
    struct BRegs {
      v4u rb[BP][BQ];
    };
    ARegs A0, A1;
    BRegs RB;

    // Full slice, unconditional 16-byte loads.
    auto load_a = [&](int64_t k0, ARegs& R) {
      if constexpr (AT == 0) {
        const float* A = static_cast<const float*>(g.A);
        if constexpr (AV) {
#pragma unroll
          for (int q = 0; q < AQ; ++q) R.ra[q] = *reinterpret_cast<const v4f*>(A + a_off[q] + k0 + 4 * a_pc);
        } else {
#pragma unroll
          for (int e = 0; e < NE; ++e) R.re[e] = A[sOff[sr + (NTHR / 32) * e] + k0 + sc];
        }
      } else {
        const uint16_t* A = static_cast<const uint16_t*>(g.A);
#pragma unroll
        for (int q = 0; q < AQ; ++q) R.ra16[q] = *reinterpret_cast<const v4u*>(A + a_off[q] + k0 + 8 * a_pc);
      }
    };
    auto load_b = [&](int64_t k0, BRegs& R) {
#pragma unroll
      for (int part = 0; part < BP; ++part)
#pragma unroll
        for (int q = 0; q < BQ; ++q) {
          const uint16_t* p = (part == 0 ? g.B_hi : g.B_lo) + b_off[q] + k0;
          if constexpr (!BC) {
            R.rb[part][q] = *(const __attribute__((address_space(1))) v4u*)(p);
          } else {
            const int64_t brow = n0 + b_r0 + (NTHR / 4) * q;
            uint32_t h[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int64_t kk = k0 + 8 * b_pc + e;
              h[e] = (brow < N && kk < kend) ? (uint32_t)p[e] : 0u;
            }
            R.rb[part][q] = mk4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
          }
        }
    };
    // The ragged slice: element-wise, bounds-checked.
    auto load_tail = [&](int64_t k0, ARegs& RA, BRegs& R) {
      if constexpr (AT == 0) {
        const float* A = static_cast<const float*>(g.A);
        if constexpr (AV) {
#pragma unroll
          for (int q = 0; q < AQ; ++q) {
            const int64_t kk = k0 + 4 * a_pc;
            v4f x;
            x.x = (kk + 0 < kend) ? A[a_off[q] + kk + 0] : 0.f;
            x.y = (kk + 1 < kend) ? A[a_off[q] + kk + 1] : 0.f;
            x.z = (kk + 2 < kend) ? A[a_off[q] + kk + 2] : 0.f;
            x.w = (kk + 3 < kend) ? A[a_off[q] + kk + 3] : 0.f;
            RA.ra[q] = x;
          }
        } else {
#pragma unroll
          for (int e = 0; e < NE; ++e)
            RA.re[e] = (k0 + sc < kend) ? A[sOff[sr + (NTHR / 32) * e] + k0 + sc] : 0.f;
        }
      } else {
        const uint16_t* A = static_cast<const uint16_t*>(g.A);
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int64_t kk = k0 + 8 * a_pc + e;
            h[e] = kk < kend ? (uint32_t)A[a_off[q] + kk] : 0u;
          }
          RA.ra16[q] = mk4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
        }
      }
#pragma unroll
      for (int part = 0; part < BP; ++part)
#pragma unroll
        for (int q = 0; q < BQ; ++q) {
          const int64_t brow = n0 + b_r0 + (NTHR / 4) * q;
          const uint16_t* p = (part == 0 ? g.B_hi : g.B_lo) + b_off[q] + k0;
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int64_t kk = k0 + 8 * b_pc + e;
            h[e] = (brow < N && kk < kend) ? (uint32_t)p[e] : 0u;
          }
          R.rb[part][q] = mk4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
        }
    };

    // Registers -> LDS stage `st`. Rows beyond M hold a copy of a valid row:
    // they only feed output rows that are never stored, so they are staged as
    // they are.
    auto stage = [&](int st, const ARegs& RA, const BRegs& R) {
      const v4f* ra = RA.ra;
      const float* re = RA.re;
      const v4u* ra16 = RA.ra16;
      const auto& rb = R.rb;
      if constexpr (AT == 0) {
        if constexpr (AV) {
          // 4 floats = half of a 16-byte chunk of 8 halves
#pragma unroll
          for (int q = 0; q < AQ; ++q) {
            const int r = a_r0 + a_rs * q;
            const int o = swz(r, a_pc >> 1) + 4 * (a_pc & 1);
            v4f x = ra[q];
            if constexpr (F16) x *= a_scale;
            const uint32_t h0 = cvt_pair<F16>(x.x, x.y), h1 = cvt_pair<F16>(x.z, x.w);
            v2u hv;
            hv.x = h0;
            hv.y = h1;
            *reinterpret_cast<v2u*>(&sA[st][0][o]) = hv;
            if constexpr (AP == 2) {
              const f32x2v b0 = uncvt_pair<F16>(h0), b1 = uncvt_pair<F16>(h1);
              v2u lv;
              lv.x = cvt_pair<F16>(x.x - b0.x, x.y - b0.y);
              lv.y = cvt_pair<F16>(x.z - b1.x, x.w - b1.y);
              *reinterpret_cast<v2u*>(&sA[st][AP - 1][o]) = lv;
            }
          }
        } else {
#pragma unroll
          for (int e = 0; e < NE; ++e) {
            const int r = sr + (NTHR / 32) * e;
            const int o = swz(r, sc >> 3) + (sc & 7);
            const float x = F16 ? re[e] * a_scale : re[e];
            const uint16_t h = cvt16<F16>(x);
            sA[st][0][o] = h;
            if constexpr (AP == 2) sA[st][AP - 1][o] = cvt16<F16>(x - back16<F16>(h));
          }
        }
      } else {
#pragma unroll
        for (int q = 0; q < AQ; ++q)
          *reinterpret_cast<v4u*>(&sA[st][0][swz(a_r0 + a_rs * q, a_pc)]) = ra16[q];
      }
#pragma unroll
      for (int part = 0; part < BP; ++part)
#pragma unroll
        for (int q = 0; q < BQ; ++q)
          *reinterpret_cast<v4u*>(&sB[st][part][swz(b_r0 + (NTHR / 4) * q, b_pc)]) = rb[part][q];
    };

    f32x16 acc[WI][WJ];
#pragma unroll
    for (int i = 0; i < WI; ++i)
#pragma unroll
      for (int j = 0; j < WJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Each pass sweeps all WI x WJ accumulators, so consecutive MFMAs never
    // depend on each other's result.
    auto compute = [&](int st) {
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ch = 2 * ks + (lane >> 5);
        v4u fa[AP][WI], fb[BP][WJ];
#pragma unroll
        for (int i = 0; i < WI; ++i)
#pragma unroll
          for (int part = 0; part < AP; ++part)
            fa[part][i] = *reinterpret_cast<const v4u*>(&sA[st][part][swz(wm + 32 * i + (lane & 31), ch)]);
#pragma unroll
        for (int j = 0; j < WJ; ++j)
#pragma unroll
          for (int part = 0; part < BP; ++part)
            fb[part][j] = *reinterpret_cast<const v4u*>(&sB[st][part][swz(wn + 32 * j + (lane & 31), ch)]);
#pragma unroll
        for (int j = 0; j < WJ; ++j)
#pragma unroll
          for (int i = 0; i < WI; ++i) acc[i][j] = mfma32<F16>(fa[0][i], fb[0][j], acc[i][j]);
        if constexpr (BP == 2) {
#pragma unroll
          for (int j = 0; j < WJ; ++j)
#pragma unroll
            for (int i = 0; i < WI; ++i) acc[i][j] = mfma32<F16>(fa[0][i], fb[BP - 1][j], acc[i][j]);
        }
        if constexpr (AP == 2) {
#pragma unroll
          for (int j = 0; j < WJ; ++j)
#pragma unroll
            for (int i = 0; i < WI; ++i) acc[i][j] = mfma32<F16>(fa[AP - 1][i], fb[0][j], acc[i][j]);
        }
      }
    };

    auto clamp = [&](int64_t i) { return slice_k0(std::min<int64_t>(i, nk - 1)); };
    // prologue: slice 0 (possibly the ragged one) staged
    if (ragged) load_tail(slice_k0(0), A0, RB);
    else {
      load_a(slice_k0(0), A0);
      load_b(slice_k0(0), RB);
    }
    stage(0, A0, RB);
    if constexpr (AV || AT == 1) {
      // slice 1 into A1 and RB, slice 2 requested into A0 (with a single
      // slice there is nothing to request: clamp would name the ragged slice)
      if (nk > 1) {
        load_a(clamp(1), A1);
        load_b(clamp(1), RB);
        load_a(clamp(2), A0);
      }
      __syncthreads();
      // Steady state, two slices per trip, branch-free: on entry slice p is in
      // LDS stage 0, slice p+1 in A1 and RB, slice p+2 in flight into A0.
      int64_t p = 0;
      for (; p + 2 < nk; p += 2) {
        compute(0);
        stage(1, A1, RB);                               // slice p+1
        load_a(clamp(p + 3), A1);
        load_b(clamp(p + 2), RB);
        __syncthreads();
        compute(1);
        stage(0, A0, RB);                               // slice p+2
        load_a(clamp(p + 4), A0);
        load_b(clamp(p + 3), RB);
        __syncthreads();
      }
      compute(0);
      if (p + 1 < nk) {
        stage(1, A1, RB);
        __syncthreads();
        compute(1);
      }
    } else {
      // element path: one register slice, requested one slice ahead
      if (nk > 1) {
        load_a(clamp(1), A0);
        load_b(clamp(1), RB);
      }
      __syncthreads();
      for (int64_t kt = 0; kt + 1 < nk; ++kt) {
        const int st = (int)(kt & 1);
        compute(st);
        stage(st ^ 1, A0, RB);                          // slice kt+1
        load_a(clamp(kt + 2), A0);
        load_b(clamp(kt + 2), RB);
        __syncthreads();
      }
      compute((int)((nk - 1) & 1));
    }

    // epilogue: lane holds column (lane & 31), rows 8*(r/4) + 4*(lane/32) + r%4
    float* C = g.C;
    int64_t ldc = g.ldc;
    if (kp.splits > 1) {
      C = g.partial + (int64_t)split * M * N;
      ldc = N;
    }
    store_tile<WI, WJ>(g, C, ldc, M, N, m0 + wm, n0 + wn, lane, acc);
  }
}

// k_gemm_p: waves per workgroup (4: one per SIMD, 128 x 128 each; 8: two per
// SIMD, 128 x 64 each), chosen for every pipelined launch.
constexpr int kPipeWaves = 8;

// The pipelined kernel reads B through a range-checked buffer descriptor when
// the last column tile is padded and the rows fit a 31-bit byte range.
inline bool use_buffer_b(const GemmArgs& g) {
  return g.N % 256 != 0 && (double)g.N * (double)g.ldb * 2.0 < 2147483648.0;
}

// AT: 0 = fp32 A, 1 = 16-bit A used as it is, 2 = bf16 A widened, scaled
// and rounded to fp16 while it is staged (all with 16-byte aligned rows); B is
// a padded panel; one part each; no split-K.
// BB: B through a range-checked buffer descriptor (padding rows skipped);
// else plain loads with padding rows mapped to row 0.
// NWV: waves per workgroup (4 or 8), NWV / 4 per SIMD.
template <int AT, bool F16, bool SC, bool BB, int NWV>
__global__ __launch_bounds__(NWV * 64) __attribute__((amdgpu_waves_per_eu(NWV / 4, NWV / 4)))
void k_gemm_p(KParams kp) {
  static_assert(NWV == 4 || NWV == 8, "4 or 8 waves");
  constexpr int PT = NWV * 64;
  constexpr int BNP = 256;
  constexpr int WI = 4, WJ = NWV == 4 ? 4 : 2;   // 128 x 128 or 128 x 64 per wave
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BNP * BK];
  __shared__ int64_t sOff[BM];
  __shared__ int sPos;

  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index through readfirstlane: the compiler then treats the per-wave
  // branch below as uniform (two separate loops, not one masked after the other)
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Units of each product: tiles x splits (M from the device count when given).
  auto units_of = [&](int pi) -> int64_t {
    const GemmArgs& q = pi ? kp.g2 : kp.g;
    const int64_t Mq = q.M_dev ? (int64_t)(*q.M_dev) : q.M;
    return ((Mq + BM - 1) / BM) * ((q.N + BNP - 1) / BNP) * (pi ? 1 : kp.splits);
  };
  const int64_t nu0 = units_of(0), nu1 = kp.nprob > 1 ? units_of(1) : 0;
  // One queue per XCD (workgroup b runs on XCD b % kXcds): the queue holds a
  // contiguous range of each product's units, the first product's before the
  // second's, so the workgroups of an XCD work on neighbouring tiles (shared
  // operand rows in that XCD's L2). Positions are taken at a fixed stride, or
  // from the XCD's counter when kp.g.sched is given.
  const int G = gridDim.x, b = blockIdx.x;
  const bool xq = G >= kXcds && G % kXcds == 0;
  const int nq = xq ? kXcds : 1, x = xq ? b % kXcds : 0;
  const int64_t c0 = (nu0 + nq - 1) / nq, c1 = (nu1 + nq - 1) / nq;
  const int64_t beg0 = std::min<int64_t>(x * c0, nu0);
  const int64_t len0 = std::min<int64_t>((x + 1) * c0, nu0) - beg0;
  const int64_t beg1 = std::min<int64_t>(x * c1, nu1);
  const int64_t len1 = std::min<int64_t>((x + 1) * c1, nu1) - beg1;
  const int64_t qlen = len0 + len1;
  int32_t* const sched = kp.g.sched;
  int64_t pos = b / nq;
  if (sched) {
    if (tid == 0) sPos = atomicAdd(&sched[x], 1);
    __syncthreads();
    pos = sPos;
  }

  const int wm = NWV == 4 ? (wid >> 1) * 128 : (wid >> 2) * 128;
  const int wn = NWV == 4 ? (wid & 1) * 128 : (wid & 3) * 64;
  // Staging: fp32 A 8 lanes per row (rows (tid >> 3) + PT / 8 q); 16-bit A
  // 4 lanes per row (rows (tid >> 2) + PT / 4 q); B 4 lanes per row (rows
  // (tid >> 2) + PT / 4 q).
  constexpr int AQ = AT == 0 ? BM / (PT / 8) : BM / (PT / 4);
  constexpr int B_RS = PT / 4;
  constexpr int BQ = BNP / B_RS;
  static_assert(AT != 2 || F16, "bf16 A is widened to fp16 for fp16 products only");
  const int a_r0 = AT == 0 ? (tid >> 3) : (tid >> 2);
  constexpr int a_rs = AT == 0 ? PT / 8 : PT / 4;
  const int a_pc = AT == 0 ? (tid & 7) : (tid & 3);
  const int b_r0 = tid >> 2, b_pc = tid & 3;

  while (pos < qlen) {
    const int pi = pos < len0 ? 0 : 1;
    const int64_t u = pi ? beg1 + (pos - len0) : beg0 + pos;
    if (sched) {
      __syncthreads();                   // every thread has read sPos
      if (tid == 0) sPos = atomicAdd(&sched[x], 1);   // next position, fetched ahead
    }
    const GemmArgs& g = pi ? kp.g2 : kp.g;
    const int splits = pi ? 1 : kp.splits;
    const int64_t kc = pi ? kp.kc2 : kp.kc;
    const int64_t M = g.M_dev ? (int64_t)(*g.M_dev) : g.M;
    const int64_t N = g.N, K = g.K;
    const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BNP - 1) / BNP;
    const float a_scale = g.a_scale;
    int64_t t;
    int split;
    if (g.split_major) {
      split = (int)(u / (tiles_m * tiles_n));
      t = u % (tiles_m * tiles_n);
    } else {
      t = u / splits;
      split = (int)(u % splits);
    }
    int64_t tm, tn;
    if (g.n_major) { tn = t / tiles_m; tm = t % tiles_m; }
    else { tm = t / tiles_n; tn = t % tiles_n; }
    const int64_t m0 = tm * BM, n0 = tn * BNP;
    const int64_t kbeg = split * kc;
    const int64_t kend = std::min<int64_t>(K, kbeg + kc);
    const int64_t nk = (kend - kbeg + BK - 1) / BK;
    const bool ragged = ((kend - kbeg) % BK) != 0;

    __syncthreads();                     // previous unit's readers of sOff / stages are done
    if (tid < BM) {
      const int64_t row = m0 + tid;
      const bool ok = row < M;
      const int64_t src = g.a_rows ? (int64_t)g.a_rows[ok ? row : m0] : (ok ? row : m0);
      sOff[tid] = src * g.lda;
    }
    __syncthreads();
    int64_t a_off[AQ];
#pragma unroll
    for (int q = 0; q < AQ; ++q) a_off[q] = sOff[a_r0 + a_rs * q];
    // per-piece base pointers: a slice's load is base + k0
    const float* pa32[AT == 0 ? AQ : 1];
    const uint16_t* pa16[AT == 0 ? 1 : AQ];
#pragma unroll
    for (int q = 0; q < AQ; ++q) {
      if constexpr (AT == 0) pa32[q] = static_cast<const float*>(g.A) + a_off[q] + 4 * a_pc;
      else pa16[q] = static_cast<const uint16_t*>(g.A) + a_off[q] + 8 * a_pc;
    }
    // BB: B through a buffer descriptor covering its first N rows: the rows of
    // the last column tile at or beyond N (padding) read as zeros without a
    // memory access, so the load path carries no padding (their products land
    // in output columns that are never stored or never read). The host uses
    // BB only when N * ldb * 2 < 2^31.
    const uint32_t b_bytes = BB ? (uint32_t)(N * g.ldb * 2) : 0u;
    const __amdgpu_buffer_rsrc_t b_rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)g.B_hi, (short)0, (int)b_bytes, 0x00020000);
    uint32_t b_vo[BQ];   // byte offset of the lane's 16 bytes at k = 0
    int64_t b_off[BQ];
    const uint16_t* pb[BQ];
#pragma unroll
    for (int q = 0; q < BQ; ++q) {
      const int64_t brow = n0 + b_r0 + B_RS * q;
      b_vo[q] = brow < N ? (uint32_t)(2 * (brow * g.ldb + 8 * b_pc)) : b_bytes;
      b_off[q] = (brow < N ? brow : 0) * g.ldb + 8 * b_pc;
      pb[q] = g.B_hi + b_off[q];
    }
    // Slice order: a ragged last slice first, then the full slices in order.
    auto slice_k0 = [&](int64_t i) -> int64_t {
      const int64_t s = ragged ? (i == 0 ? nk - 1 : i - 1) : i;
      return kbeg + s * BK;
    };
    auto clamp = [&](int64_t i) { return slice_k0(std::min<int64_t>(i, nk - 1)); };

    struct ARegs {
      v4f ra[AT == 0 ? AQ : 1];
      v4u ra16[AT == 0 ? 1 : AQ];
    };
    struct BRegs { v4u rb[BQ]; };
    ARegs A0, A1;
    BRegs RB, RB2;
    v4u fa[WI];                 // A fragments of the half slice being multiplied
    v4u fb0[WJ], fb1[WJ];       // B fragments of the first and second half

    auto load_a = [&](int64_t k0, ARegs& R) {
      if constexpr (AT == 0) {
#pragma unroll
        for (int q = 0; q < AQ; ++q) R.ra[q] = *reinterpret_cast<const v4f*>(pa32[q] + k0);
      } else {
#pragma unroll
        for (int q = 0; q < AQ; ++q) R.ra16[q] = *reinterpret_cast<const v4u*>(pa16[q] + k0);
      }
    };
    auto load_b = [&](int64_t k0, BRegs& R) {
#pragma unroll
      for (int q = 0; q < BQ; ++q) {
        if constexpr (BB)
          R.rb[q] = __builtin_bit_cast(
              v4u, __builtin_amdgcn_raw_buffer_load_b128(b_rsrc, b_vo[q] + (uint32_t)(2 * k0), 0, 0));
        else
          R.rb[q] = *(const __attribute__((address_space(1))) v4u*)(pb[q] + k0);
      }
    };
    // The ragged slice: element-wise, bounds-checked (B is a padded panel, so
    // its columns up to round_up(K, 32) are readable and zero beyond K).
    auto load_tail = [&](int64_t k0, ARegs& RA, BRegs& R) {
      if constexpr (AT == 0) {
        const float* A = static_cast<const float*>(g.A);
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          const int64_t kk = k0 + 4 * a_pc;
          v4f x;
          x.x = (kk + 0 < kend) ? A[a_off[q] + kk + 0] : 0.f;
          x.y = (kk + 1 < kend) ? A[a_off[q] + kk + 1] : 0.f;
          x.z = (kk + 2 < kend) ? A[a_off[q] + kk + 2] : 0.f;
          x.w = (kk + 3 < kend) ? A[a_off[q] + kk + 3] : 0.f;
          RA.ra[q] = x;
        }
      } else {
        const uint16_t* A = static_cast<const uint16_t*>(g.A);
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int64_t kk = k0 + 8 * a_pc + e;
            h[e] = kk < kend ? (uint32_t)A[a_off[q] + kk] : 0u;
          }
          RA.ra16[q] = mk4(pack2(h[0], h[1]), pack2(h[2], h[3]), pack2(h[4], h[5]), pack2(h[6], h[7]));
        }
      }
      load_b(k0, R);
    };
    auto stage_a = [&](int st, const ARegs& RA, int q0, int q1) {
      if constexpr (AT == 0) {
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          if (q < q0 || q >= q1) continue;
          const int r = a_r0 + a_rs * q;
          const int o = swz(r, a_pc >> 1) + 4 * (a_pc & 1);
          v4f x = RA.ra[q];
          if constexpr (F16 && SC) x *= a_scale;
          v2u hv;
          hv.x = cvt_pair<F16>(x.x, x.y);
          hv.y = cvt_pair<F16>(x.z, x.w);
          *reinterpret_cast<v2u*>(&sA[st][o]) = hv;
        }
      } else if constexpr (AT == 2) {
        // bf16 pairs -> fp32 (exact) -> times 2^e (exact) -> fp16 pairs, nearest even
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          if (q < q0 || q >= q1) continue;
          const v4u w = RA.ra16[q];
          uint32_t h[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xFFFF0000u);
            if constexpr (SC) {
              lo *= a_scale;
              hi *= a_scale;
            }
            h[e] = cvt_pair<true>(lo, hi);
          }
          *reinterpret_cast<v4u*>(&sA[st][swz(a_r0 + a_rs * q, a_pc)]) = mk4(h[0], h[1], h[2], h[3]);
        }
      } else {
#pragma unroll
        for (int q = 0; q < AQ; ++q)
          if (q >= q0 && q < q1)
            *reinterpret_cast<v4u*>(&sA[st][swz(a_r0 + a_rs * q, a_pc)]) = RA.ra16[q];
      }
    };
    auto stage_b = [&](int st, const BRegs& R) {
#pragma unroll
      for (int q = 0; q < BQ; ++q)
        *reinterpret_cast<v4u*>(&sB[st][swz(b_r0 + B_RS * q, b_pc)]) = R.rb[q];
    };
    auto read_a = [&](int st, int ks, int i) -> v4u {
      const int ch = 2 * ks + (lane >> 5);
      return *reinterpret_cast<const v4u*>(&sA[st][swz(wm + 32 * i + (lane & 31), ch)]);
    };
    auto read_b = [&](int st, int ks, v4u (&fb)[WJ]) {
      const int ch = 2 * ks + (lane >> 5);
#pragma unroll
      for (int j = 0; j < WJ; ++j)
        fb[j] = *reinterpret_cast<const v4u*>(&sB[st][swz(wn + 32 * j + (lane & 31), ch)]);
    };

    f32x16 acc[WI][WJ];
#pragma unroll
    for (int i = 0; i < WI; ++i)
#pragma unroll
      for (int j = 0; j < WJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    // Fragments: fa holds the A fragments of the half slice being multiplied,
    // fb0 and fb1 the B fragments of a slice's first and second half. The
    // MFMAs of a half are issued A fragment by A fragment, so fragment i of
    // the next half is read into fa[i] as soon as its own MFMAs have issued
    // (32 fragment registers instead of two full sets of 48).
    static_assert(WI == 4, "the first half's four segments take one A fragment each");
    auto pair = [&](int i, const v4u (&fb)[WJ]) {
#pragma unroll
      for (int j = 0; j < WJ; ++j) acc[i][j] = mfma32<F16>(fa[i], fb[j], acc[i][j]);
    };
    // Scheduling-group masks: MFMA 0x008, VALU 0x002, global load 0x020,
    // LDS read 0x100, LDS write 0x200.

    // prologue: slice 0 staged; slices 1 and 2 (those that exist) requested in
    // the order the loop issues them (B then A of each slice), so that the
    // load counter holds the same sequence on entry as after every iteration
    if (ragged) load_tail(slice_k0(0), A0, RB);
    else {
      load_a(slice_k0(0), A0);
      load_b(slice_k0(0), RB);
    }
    stage_a(0, A0, 0, AQ);
    stage_b(0, RB);
    if (nk > 1) {
      load_b(clamp(1), RB);
      load_a(clamp(1), A1);
    }
    if (nk > 2) {
      load_b(clamp(2), RB2);
      load_a(clamp(2), A0);
    }
    __syncthreads();

    // One slice i in stage st (fa and fb0 hold its first half; the registers
    // hold slices i+1 and i+2 of A and B; RB is the B buffer holding slice
    // i+1, Anext the A buffer). ACT: the wave has columns below N; a wave whose
    // columns all lie in the padding of the last column tile only stages its
    // share of the operands (its accumulators stay zero).
    auto iter = [&](auto act_c, auto ld_c, int st, int64_t i, ARegs& Anext, BRegs& RB) {
      constexpr bool ACT = decltype(act_c)::value;
      constexpr bool LD = decltype(ld_c)::value;   // slice i+3 exists and is requested
      const int64_t k3 = clamp(i + 3);
      // First half, in four segments of one A fragment each: its MFMAs, then
      // its second-half fragment read into fa[i]; beside them B of slice i+1
      // to LDS and B of slice i+3 requested (segment 0), A of slice i+1
      // converted and written to LDS (segments 1 and 2), A of slice i+3
      // requested (segment 3). B is requested before A, so that a wait for B
      // never waits for the A request behind it.
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (ACT) {
        read_b(st, 1, fb1);
        pair(0, fb0);
        fa[0] = read_a(st, 1, 0);
      }
      stage_b(st ^ 1, RB);
      if constexpr (LD) load_b(k3, RB);
      if constexpr (ACT) {
        __builtin_amdgcn_sched_group_barrier(0x100, WJ, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (ACT) {
        pair(1, fb0);
        fa[1] = read_a(st, 1, 1);
      }
      stage_a(st ^ 1, Anext, 0, (AQ + 1) / 2);
      if constexpr (ACT) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 1);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 1);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 1);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (ACT) {
        pair(2, fb0);
        fa[2] = read_a(st, 1, 2);
      }
      stage_a(st ^ 1, Anext, (AQ + 1) / 2, AQ);
      if constexpr (ACT) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 2);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 2);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 2);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (ACT) {
        pair(3, fb0);
        fa[3] = read_a(st, 1, 3);
      }
      if constexpr (LD) load_a(k3, Anext);
      if constexpr (ACT) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
        __builtin_amdgcn_sched_group_barrier(0x020, 2, 3);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
        __builtin_amdgcn_sched_group_barrier(0x020, 2, 3);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 3);
      }
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      __builtin_amdgcn_sched_barrier(0);
      // Second half (fa, fb1): the next slice's first-half fragments are read
      // from the other stage, fb0 first, then fa[i] behind fragment i's MFMAs.
      if constexpr (ACT) {
        read_b(st ^ 1, 0, fb0);
#pragma unroll
        for (int i2 = 0; i2 < WI; ++i2) {
          pair(i2, fb1);
          fa[i2] = read_a(st ^ 1, 0, i2);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, WJ, 4);
#pragma unroll
        for (int i2 = 0; i2 < WI; ++i2) {
          __builtin_amdgcn_sched_group_barrier(0x008, WJ, 4);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 4);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    auto slices = [&](auto act_c) {
      constexpr bool ACT = decltype(act_c)::value;
      if constexpr (ACT) {
        read_b(0, 0, fb0);
#pragma unroll
        for (int i2 = 0; i2 < WI; ++i2) fa[i2] = read_a(0, 0, i2);
      }
      constexpr std::true_type LD;
      constexpr std::false_type NOLD;
      int64_t p = 0;
      for (; p + 5 <= nk; p += 2) {          // slices p + 3 and p + 4 exist
        iter(act_c, LD, 0, p, A1, RB);
        iter(act_c, LD, 1, p + 1, A0, RB2);
      }
      if (p + 4 == nk) {                     // slice p + 3 is the last to request
        iter(act_c, LD, 0, p, A1, RB);
        iter(act_c, NOLD, 1, p + 1, A0, RB2);
        p += 2;
      }
      // the last one to three slices: everything they stage is requested, so
      // no request runs past the unit's last slice (an odd count ends in
      // stage 0 with one iteration)
      for (; p < nk; p += 2) {
        iter(act_c, NOLD, 0, p, A1, RB);
        if (p + 1 < nk) iter(act_c, NOLD, 1, p + 1, A0, RB2);
      }
    };
    if (n0 + wn < N) slices(std::true_type{});
    else slices(std::false_type{});
    float* C = g.C;
    int64_t ldc = g.ldc;
    if (splits > 1) {
      C = g.partial + (int64_t)split * M * N;
      ldc = N;
    }
    store_tile<WI, WJ>(g, C, ldc, M, N, m0 + wm, n0 + wn, lane, acc);
    if (sched) {
      __syncthreads();                   // sPos (written before the unit's first barrier)
      pos = sPos;
    } else {
      pos += G / nq;
    }
  }
}

// C[row, col] = sum over splits, in split order, of the partial tiles. Four
// consecutive columns per thread (16-byte loads) when N and ldc allow it.
__global__ void k_split_sum(const float* __restrict__ part, int splits, int64_t M, int64_t N,
                            float* __restrict__ C, int64_t ldc) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= M * N) return;
  const int64_t row = idx / N, col = idx % N;
  float s = 0.f;
  for (int p = 0; p < splits; ++p) s += part[(int64_t)p * M * N + idx];
  C[row * ldc + col] = s;
}
__global__ void k_split_sum4(const float* __restrict__ part, int splits, int64_t M, int64_t N,
                             float* __restrict__ C, int64_t ldc) {
  const int64_t idx = 4 * ((int64_t)blockIdx.x * blockDim.x + threadIdx.x);
  if (idx >= M * N) return;
  const int64_t row = idx / N, col = idx % N;
  v4f s = {0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < splits; ++p) s += *reinterpret_cast<const v4f*>(part + (int64_t)p * M * N + idx);
  *reinterpret_cast<v4f*>(C + row * ldc + col) = s;
}
void split_sum(const GemmArgs& g, int splits, hipStream_t s) {
  const int64_t total = g.M * g.N;
  if (g.N % 4 == 0 && g.ldc % 4 == 0 && (uintptr_t)g.C % 16 == 0)
    hipLaunchKernelGGL(k_split_sum4, dim3((unsigned)((total / 4 + 255) / 256)), dim3(256), 0, s,
                       g.partial, splits, g.M, g.N, g.C, g.ldc);
  else
    hipLaunchKernelGGL(k_split_sum, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                       g.partial, splits, g.M, g.N, g.C, g.ldc);
}

template <int AT, int AP, int BP, bool F16, int BN>
void pick(const KParams& kp, bool av, bool bc, unsigned grid, hipStream_t s) {
  if constexpr (AT == 0) {
    if (av && !bc) hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16, BN, true, false>), dim3(grid), dim3(NTHR), 0, s, kp);
    else if (av && bc) hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16, BN, true, true>), dim3(grid), dim3(NTHR), 0, s, kp);
    else if (!bc) hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16, BN, false, false>), dim3(grid), dim3(NTHR), 0, s, kp);
    else hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16, BN, false, true>), dim3(grid), dim3(NTHR), 0, s, kp);
  } else {
    if (!bc) hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16, BN, true, false>), dim3(grid), dim3(NTHR), 0, s, kp);
    else hipLaunchKernelGGL((k_gemm<AT, AP, BP, F16, BN, true, true>), dim3(grid), dim3(NTHR), 0, s, kp);
  }
}

template <int AT, int AP, int BP, bool F16>
eogp_status launch(const GemmArgs& g, bool av, bool bc, hipStream_t s) {
  if (g.M == 0 || g.N == 0) return EOGP_OK;
  const int64_t pad256 = ((g.N + 255) / 256) * 256, pad128 = ((g.N + 127) / 128) * 128;
  const bool wide = pad256 * 10 <= pad128 * 11;      // at most 10% more padding
  const int bn = wide ? 256 : 128;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + bn - 1) / bn);
  KParams kp;
  kp.g = g;
  kp.splits = 1;
  kp.kc = ((g.K + BK - 1) / BK) * BK;
  const int64_t nk_all = (g.K + BK - 1) / BK;
  if (!g.M_dev && g.partial && tiles < kCus) {
    // split K so that there are about two work units per CU, >= 16 slices each
    int sp = (int)std::min<int64_t>((2 * kCus + tiles - 1) / tiles, nk_all / 16);
    sp = std::min(sp, g.max_splits);
    if (sp > 1) {
      kp.kc = ((nk_all + sp - 1) / sp) * BK;
      kp.splits = (int)((nk_all * BK + kp.kc - 1) / kp.kc);
    }
  }
  if constexpr (AP == 1 && BP == 1) {
    if (av && !bc) {
      // single-pass product: the pipelined kernel (kPipeWaves waves), 256 x 256 tiles.
      // Split K (host-known M, scratch given) when that shortens the
      // estimated time: rounds of units x slices per unit, plus the partial
      // sums (one slice of a 256 x 256 tile ~ 1.4 us; partials at ~5 TB/s).
      const int64_t tiles_p = ((g.M + BM - 1) / BM) * ((g.N + 255) / 256);
      KParams kq = kp;
      kq.splits = 1;
      kq.kc = nk_all * BK;
      if (!g.M_dev && g.partial && !g.CT && tiles_p < kCus) {
        double best = 1e30;
        for (int sp = 1; sp <= g.max_splits && sp <= std::max<int64_t>(1, nk_all / 16); ++sp) {
          const int64_t kc = ceil_div(nk_all, sp);
          const int64_t units = tiles_p * ceil_div(nk_all, kc);
          const double t_us = (double)ceil_div(units, kCus) * kc * 1.4 +
                              (sp > 1 ? (double)sp * g.M * g.N * 4 / 5e6 : 0.0);
          if (t_us < best) {
            best = t_us;
            kq.kc = kc * BK;
            kq.splits = (int)ceil_div(nk_all, kc);
          }
        }
      }
      int64_t grid = std::min<int64_t>(tiles_p * kq.splits, kCus);
      if (grid >= kXcds) grid = grid / kXcds * kXcds;
      if (g.sched) hipLaunchKernelGGL(k_zero_sched, dim3(1), dim3(64), 0, s, g.sched);
      timing::Scope ts(g.timing_class, s);
      const bool bb = use_buffer_b(g);
      const dim3 gd((unsigned)grid), bd(kPipeWaves * 64);
      if (F16 && g.a_scale != 1.f) {
        if (bb) hipLaunchKernelGGL((k_gemm_p<AT, F16, true, true, kPipeWaves>), gd, bd, 0, s, kq);
        else hipLaunchKernelGGL((k_gemm_p<AT, F16, true, false, kPipeWaves>), gd, bd, 0, s, kq);
      } else {
        if (bb) hipLaunchKernelGGL((k_gemm_p<AT, F16, false, true, kPipeWaves>), gd, bd, 0, s, kq);
        else hipLaunchKernelGGL((k_gemm_p<AT, F16, false, false, kPipeWaves>), gd, bd, 0, s, kq);
      }
      EOGP_LAUNCH_CHECK("gemm launch");
      if (kq.splits > 1) {
        split_sum(g, kq.splits, s);
        EOGP_LAUNCH_CHECK("gemm split sum");
      }
      return EOGP_OK;
    }
  }
  if constexpr (AT == 2) {
    return fail(EOGP_ERR_UNSUPPORTED, "gemm: bf16 A widened to fp16 needs aligned rows and a padded B panel");
  } else {
  if (g.CT && kp.splits > 1) return fail(EOGP_ERR_UNSUPPORTED, "gemm: fp16 transposed output without split-K only");
  int64_t grid = std::min<int64_t>(tiles * kp.splits, kCus);
  if (grid >= kXcds) grid = grid / kXcds * kXcds;
  timing::Scope ts(g.timing_class, s);
  if (wide) pick<AT, AP, BP, F16, 256>(kp, av, bc, (unsigned)grid, s);
  else pick<AT, AP, BP, F16, 128>(kp, av, bc, (unsigned)grid, s);
  EOGP_LAUNCH_CHECK("gemm launch");
  if (kp.splits > 1) {
    split_sum(g, kp.splits, s);
    EOGP_LAUNCH_CHECK("gemm split sum");
  }
  return EOGP_OK;
  }
}

}  // namespace

size_t gemm_partial_bytes(int64_t M, int64_t N, int max_splits) {
  return (size_t)M * N * 4 * (size_t)std::max(1, max_splits);
}

namespace {
// The pipelined kernel applies: single-pass product, 16-byte aligned A rows,
// B a padded panel on 16-byte boundaries.
bool pipelined(const GemmArgs& g, AType a_type) {
  const int a_align = a_type == AType::F32 ? 4 : 8;
  const bool av = (g.lda % a_align == 0) && ((uintptr_t)g.A % 16 == 0);
  const bool bc = !(g.b_padded && (g.ldb % 8 == 0) && ((uintptr_t)g.B_hi % 16 == 0) &&
                    (g.B_lo == nullptr || (uintptr_t)g.B_lo % 16 == 0));
  return av && !bc && !g.partial;
}
}  // namespace

eogp_status gemm_nt2(const GemmArgs& g1, const GemmArgs& g2, AType a_type, int a_parts,
                     int b_parts, bool f16, hipStream_t s) {
  const bool empty1 = g1.M == 0 || g1.N == 0, empty2 = g2.M == 0 || g2.N == 0;
  if (a_parts != 1 || b_parts != 1 || !g1.sched || empty1 || empty2 || !pipelined(g1, a_type) ||
      !pipelined(g2, a_type) || g1.timing_class != g2.timing_class) {
    const eogp_status st = gemm_nt(g1, a_type, a_parts, b_parts, f16, s);
    if (st != EOGP_OK) return st;
    return gemm_nt(g2, a_type, a_parts, b_parts, f16, s);
  }
  KParams kq;
  kq.g = g1;
  kq.splits = 1;
  kq.kc = round_up(g1.K, BK);
  kq.g2 = g2;
  kq.kc2 = round_up(g2.K, BK);
  kq.nprob = 2;
  const int64_t tiles = ceil_div(g1.M, BM) * ceil_div(g1.N, 256) + ceil_div(g2.M, BM) * ceil_div(g2.N, 256);
  int64_t grid = std::min<int64_t>(tiles, kCus);
  if (grid >= kXcds) grid = grid / kXcds * kXcds;
  const bool sc = f16 && (g1.a_scale != 1.f || g2.a_scale != 1.f);
  hipLaunchKernelGGL(k_zero_sched, dim3(1), dim3(64), 0, s, g1.sched);
  timing::Scope ts(g1.timing_class, s);
  const dim3 gd((unsigned)grid), bd(kPipeWaves * 64);
  const bool bb = use_buffer_b(g1) && use_buffer_b(g2);
#define EOGP_GEMM_P2(AT_, F16_, SC_)                                                               \
  do {                                                                                             \
    if (bb) hipLaunchKernelGGL((k_gemm_p<AT_, F16_, SC_, true, kPipeWaves>), gd, bd, 0, s, kq);    \
    else hipLaunchKernelGGL((k_gemm_p<AT_, F16_, SC_, false, kPipeWaves>), gd, bd, 0, s, kq);      \
  } while (0)
  if (a_type == AType::F32) {
    if (f16 && sc) EOGP_GEMM_P2(0, true, true);
    else if (f16) EOGP_GEMM_P2(0, true, false);
    else EOGP_GEMM_P2(0, false, false);
  } else if (a_type == AType::BF16_AS_F16) {
    if (sc) EOGP_GEMM_P2(2, true, true);
    else EOGP_GEMM_P2(2, true, false);
  } else {
    if (f16) EOGP_GEMM_P2(1, true, false);
    else EOGP_GEMM_P2(1, false, false);
  }
#undef EOGP_GEMM_P2
  EOGP_LAUNCH_CHECK("gemm launch (two products)");
  return EOGP_OK;
}

eogp_status gemm_nt(const GemmArgs& g, AType a_type, int a_parts, int b_parts, bool f16,
                    hipStream_t s) {
  const bool A32 = a_type == AType::F32;
  const int a_align = A32 ? 4 : 8;
  const bool av = (g.lda % a_align == 0) && ((uintptr_t)g.A % 16 == 0);
  if (!A32 && !av) return fail(EOGP_ERR_UNSUPPORTED, "gemm: 16-bit A rows must be 16-byte aligned");
  // B needs no checks when rows are padded to the tile and K to the slice.
  const bool bc = !(g.b_padded && (g.ldb % 8 == 0) && ((uintptr_t)g.B_hi % 16 == 0) &&
                    (g.B_lo == nullptr || (uintptr_t)g.B_lo % 16 == 0));
  if (b_parts == 2 && g.B_lo == nullptr) return fail(EOGP_ERR_INVALID, "gemm: missing B low part");
  if (a_type == AType::BF16_AS_F16) {
    if (a_parts != 1 || b_parts != 1 || !f16)
      return fail(EOGP_ERR_UNSUPPORTED, "gemm: bf16 A widened to fp16 is a single fp16 product");
    return launch<2, 1, 1, true>(g, av, bc, s);
  }
  if (!A32 && a_parts != 1) return fail(EOGP_ERR_INVALID, "gemm: 16-bit A cannot be split");
  if (A32 && a_parts == 1 && b_parts == 1 && !f16) return launch<0, 1, 1, false>(g, av, bc, s);
  if (A32 && a_parts == 2 && b_parts == 2 && !f16) return launch<0, 2, 2, false>(g, av, bc, s);
  if (A32 && a_parts == 2 && b_parts == 1 && !f16) return launch<0, 2, 1, false>(g, av, bc, s);
  if (A32 && a_parts == 1 && b_parts == 1 && f16) return launch<0, 1, 1, true>(g, av, bc, s);
  if (A32 && a_parts == 2 && b_parts == 1 && f16) return launch<0, 2, 1, true>(g, av, bc, s);
  if (!A32 && b_parts == 1 && !f16) return launch<1, 1, 1, false>(g, av, bc, s);
  if (!A32 && b_parts == 2 && !f16) return launch<1, 1, 2, false>(g, av, bc, s);
  if (!A32 && b_parts == 1 && f16) return launch<1, 1, 1, true>(g, av, bc, s);
  return fail(EOGP_ERR_UNSUPPORTED, "gemm: unsupported operand combination");
}

}  // namespace eogp
