// First stage of EOGP (eq. first_stage, eq. app_projection_maps):
//   Z[i, r] = w_r * sum_{valid t} (Q_S[:, j_r] . ds[i, t]) (Q_A[:, k_r] . a[i, t])
//
// 1. Token compaction: the valid tokens of the batch are listed example by
//    example (the loss is token-summed over valid positions), so padded and
//    masked tokens cost nothing and are never read.
// 2. Two MFMA contractions rotate every valid token onto just the eigenvector
//    columns the retained axes use: S~ = DS_valid Q_S[:, J], A~ = A_valid Q_A[:, K].
// 3. Retained products: for every example and every 32 x 32 block of
//    (row, column) pairs that holds retained axes, the block of sums
//    sum_t S~[t, j] A~[t, k] over the example's tokens is formed (MFMA)
//    and the retained entries are written, tile by tile, to a contiguous
//    row; a gather then scales them by w_r into their canonical positions
//    in Z.
//
// Intermediates. FAST and ACCURATE keep S~ and A~ in fp32, token-major, and
// form the sums with exact fp32 products. The fp16 mode stores them as fp16
// in MFMA-fragment order (1 KB blocks of 32 rows x 16 tokens), with every
// example's token run starting at a multiple of 8, and forms the sums with
// fp16 MFMA over 16 tokens at a time: half the bytes written and read, whole
// 1 KB blocks per load, and 16x the MFMA rate. The extra rounding
// of S~ and A~ adds about 1e-4 to the relative error of a row of Z in the
// GPT-2-shaped workload (4.1e-4 -> 5.1e-4, against 1e-3).
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "gemm.h"
#include "plan.h"
#include "scan.h"
#include "timing.h"

namespace eogp {
namespace {

// ---- token compaction ---------------------------------------------------------
// len[i] = valid tokens of example i; cnt[i] = len[i] rounded up to `align`
// (the run length the compacted list reserves; scanned into offsets later).
__global__ __launch_bounds__(256) void k_count_valid(const uint8_t* __restrict__ mask, int64_t N,
                                                     int64_t T, int align, int32_t* __restrict__ cnt,
                                                     int32_t* __restrict__ len) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  int c = 0;
  for (int64_t t = lane; t < T; t += 64) c += mask ? (mask[i * T + t] != 0) : 1;
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
  if (lane == 0) {
    cnt[i] = (c + align - 1) / align * align;
    if (len) len[i] = c;
  }
}

// Token list: example i's valid tokens (global index i * T + t) from off[i]
// on; the run is padded to off[i + 1] with token i * T (a readable row whose
// products land in padding columns that the retained products skip).
__global__ __launch_bounds__(256) void k_write_tokens(const uint8_t* __restrict__ mask, int64_t N,
                                                      int64_t T, const int32_t* __restrict__ off,
                                                      int32_t* __restrict__ tok) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  int32_t pos = off[i];
  for (int64_t t0 = 0; t0 < T; t0 += 64) {
    const int64_t t = t0 + lane;
    const bool v = (t < T) && (mask ? (mask[i * T + t] != 0) : true);
    uint64_t bm;
    const int pre = wave_prefix_count(v, &bm);
    if (v) tok[pos + pre] = (int32_t)(i * T + t);
    pos += __popcll(bm);
  }
  for (int32_t q = pos + lane; q < off[i + 1]; q += 64) tok[q] = (int32_t)(i * T);
}

// ---- retained products --------------------------------------------------------
// One wave per (active block, example); the four waves of a workgroup take
// four consecutive blocks of one example (blocks are listed row block first,
// so they mostly share the S~ columns they read). The block of sums
//   C[jj][kk] = sum_t S~[t, 32 jb + jj] * A~[t, 32 kb + kk]
// is one 32 x 32 fp32 MFMA accumulation over the example's tokens, two tokens
// per v_mfma_f32_32x32x2_f32 (lane l feeds row l % 32 of token l / 32 of each
// operand straight from memory). Products are exact fp32 products, so the
// result matches an fp32 dot product up to the order of the additions.
constexpr int kRetWaves = 4;
constexpr int kRetUnroll = 8;      // MFMAs (token pairs) per loaded group

__global__ __launch_bounds__(256) void k_retained(const float* __restrict__ St, int64_t ldS,
                                                  const float* __restrict__ At, int64_t ldA,
                                                  const int32_t* __restrict__ ex_off,
                                                  const int32_t* __restrict__ tiles, int n_tiles,
                                                  const uint16_t* __restrict__ ent_loc,
                                                  float out_scale, float* __restrict__ Zt,
                                                  int64_t m, int64_t ex0) {
  __shared__ float blk[kRetWaves][32][33];
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int tile = blockIdx.x * kRetWaves + wid;
  if (tile >= n_tiles) return;                 // whole wave leaves; no block barrier below
  const int64_t i = ex0 + blockIdx.y;
  const int jb = tiles[4 * tile + 0], kb = tiles[4 * tile + 1];
  const int e0 = tiles[4 * tile + 2], e1 = tiles[4 * tile + 3];
  const int64_t t0 = ex_off[i], t1 = ex_off[i + 1];
  const int half = lane >> 5, col = lane & 31;
  const float* sp = St + (int64_t)jb * 32 + col;
  const float* ap = At + (int64_t)kb * 32 + col;

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  for (int64_t tb = t0; tb < t1; tb += 2 * kRetUnroll) {
    float sv[kRetUnroll], av[kRetUnroll];
#pragma unroll
    for (int u = 0; u < kRetUnroll; ++u) {
      const int64_t t = tb + 2 * u + half;
      const bool ok = t < t1;
      sv[u] = ok ? sp[t * ldS] : 0.f;
      av[u] = ok ? ap[t * ldA] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kRetUnroll; ++u)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(sv[u], av[u], acc, 0, 0, 0);
  }
  // acc[r] holds C[8 (r / 4) + 4 half + r % 4][col]
#pragma unroll
  for (int r = 0; r < 16; ++r) blk[wid][8 * (r >> 2) + 4 * half + (r & 3)][col] = acc[r];
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  for (int e = e0 + lane; e < e1; e += 64) {
    const int loc = ent_loc[e];
    Zt[i * m + e] = out_scale * blk[wid][loc >> 5][loc & 31];
  }
}

// 16-bit intermediates (fp16, or bf16 with BF): S~ and A~ in MFMA-fragment
// order (for every 32 rows j and 16 tokens t one contiguous 1 KB block, j-major,
// 16 tokens per j; token capacity ldt, at least 16 kRetGUnroll + 16 tokens past
// the last run); example i's tokens are t = off[i] .. off[i] + len[i] - 1,
// off[i] a multiple of 8. One wave per (group of up to kRetGroup active blocks
// that share one operand block, example): SR, the group shares a row block of
// S~ (else a column block of A~). Each v_mfma_f32_32x32x16_f16 takes 16
// tokens: lane l feeds row l % 32 and tokens 8 (l / 32) .. +7 of each operand
// with one 16-byte load (the wave reads one whole 1 KB block, or two halves of
// neighbouring blocks when the run starts at an odd multiple of 8); a 16-token
// step loads the shared block once and the other operand of every member, so
// a group of L blocks loads 1 + L blocks per step instead of 2 L. Batches of
// kRetGUnroll steps: all loads of a batch are issued first (a batch may read
// up to 16 kRetGUnroll + 8 tokens past the run, inside the buffer's slack),
// then the steps that hold tokens of the run are multiplied, the last one with
// the tokens past the run (padding, or the next example) zeroed in both
// operands.
constexpr int kRetGUnroll = 4;

template <bool BF, bool SR>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
void k_retained16g(const uint16_t* __restrict__ St, const uint16_t* __restrict__ At, int64_t ldt,
                   const int32_t* __restrict__ ex_off, const int32_t* __restrict__ ex_len,
                   const int32_t* __restrict__ groups, int n_groups, const int32_t* __restrict__ gtiles,
                   const int32_t* __restrict__ tiles, const uint16_t* __restrict__ ent_loc,
                   float out_scale, float* __restrict__ Zt, int64_t m, int64_t ex0, int64_t nex) {
  typedef unsigned int v4u __attribute__((ext_vector_type(4)));
  __shared__ float blk[kRetWaves][32][33];
  // wave index as a wave-uniform value, so that group data sit in scalar registers
  const int wid = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)), lane = threadIdx.x & 63;
  // Workgroup b runs on XCD b % kXcds: the groups of one example all go to
  // one XCD (examples dealt round-robin over the XCDs), so the example's S~
  // and A~ blocks are fetched into one L2.
  const int gx = (n_groups + kRetWaves - 1) / kRetWaves;
  const int xb = blockIdx.x % kXcds, rb = blockIdx.x / kXcds;
  const int64_t ex_local = xb + (int64_t)kXcds * (rb / gx);
  if (ex_local >= nex) return;                 // whole workgroup leaves; no block barrier below
  const int grp = (rb % gx) * kRetWaves + wid;
  if (grp >= n_groups) return;                 // whole wave leaves
  const int64_t i = ex0 + ex_local;
  const int g0 = groups[4 * grp + 0], gc = groups[4 * grp + 1], shb = groups[4 * grp + 2];
  const int64_t t0 = ex_off[i] + 8 * (lane >> 5);   // this lane's first token
  const int n = ex_len[i];
  const int half = lane >> 5, col = lane & 31;
  const int64_t steps = ldt / 16;
  // element offset of (block b, this lane's row, token t) is b * bstride + lane_off + 512 (t - t0) / 16
  const int64_t bstride = steps * 512;
  const int64_t lane_off = ((t0 >> 4) * 32 + col) * 16 + (t0 & 15);
  const uint16_t* shp = (SR ? St : At) + shb * bstride + lane_off;
  const uint16_t* vbase = (SR ? At : St) + lane_off;
  int vb[kRetGroup];                           // the other operand's block of each member
#pragma unroll
  for (int c = 0; c < kRetGroup; ++c) {
    const int tile = gtiles[g0 + (c < gc ? c : gc - 1)];
    vb[c] = SR ? tiles[4 * tile + 1] : tiles[4 * tile + 0];
  }
  f32x16 acc[kRetGroup];
#pragma unroll
  for (int c = 0; c < kRetGroup; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  for (int t = 0; t < n; t += 16 * kRetGUnroll) {
    v4u a[kRetGUnroll], b[kRetGroup][kRetGUnroll];
#pragma unroll
    for (int u = 0; u < kRetGUnroll; ++u) a[u] = *reinterpret_cast<const v4u*>(shp + (int64_t)(t / 16 + u) * 512);
#pragma unroll
    for (int c = 0; c < kRetGroup; ++c)
      if (c < gc)
#pragma unroll
        for (int u = 0; u < kRetGUnroll; ++u)
          b[c][u] = *reinterpret_cast<const v4u*>(vbase + vb[c] * bstride + (int64_t)(t / 16 + u) * 512);
#pragma unroll
    for (int u = 0; u < kRetGUnroll; ++u) {
      const int tu = t + 16 * u;
      if (tu >= n) break;
      const int rem = n - tu - 8 * half;       // valid tokens among this lane's eight
      if (tu + 16 > n) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const uint32_t keep = (2 * d < rem ? 0x0000FFFFu : 0u) | (2 * d + 1 < rem ? 0xFFFF0000u : 0u);
          a[u][d] &= keep;
#pragma unroll
          for (int c = 0; c < kRetGroup; ++c)
            if (c < gc) b[c][u][d] &= keep;
        }
      }
#pragma unroll
      for (int c = 0; c < kRetGroup; ++c) {
        if (c < gc) {
          const v4u& x = SR ? a[u] : b[c][u];   // S~ operand (rows j)
          const v4u& y = SR ? b[c][u] : a[u];   // A~ operand (columns k)
          if constexpr (BF)
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, x),
                                                             __builtin_bit_cast(bf16x8, y), acc[c], 0, 0, 0);
          else
            acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, x),
                                                            __builtin_bit_cast(f16x8, y), acc[c], 0, 0, 0);
        }
      }
    }
  }
  // acc[c][r] holds block c's C[8 (r / 4) + 4 half + r % 4][col]
#pragma unroll
  for (int c = 0; c < kRetGroup; ++c) {
    if (c >= gc) break;
#pragma unroll
    for (int r = 0; r < 16; ++r) blk[wid][8 * (r >> 2) + 4 * half + (r & 3)][col] = acc[c][r];
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
    const int tile = gtiles[g0 + c];
    const int e0 = tiles[4 * tile + 2], e1 = tiles[4 * tile + 3];
    // unrolled so that several entries' positions are requested before the first
    // is used (2% of this kernel's time against one at a time)
#pragma unroll 4
    for (int e = e0 + lane; e < e1; e += 64) {
      const int loc = ent_loc[e];
      Zt[i * m + e] = out_scale * blk[wid][loc >> 5][loc & 31];
    }
    __builtin_amdgcn_s_waitcnt(0);             // this block's reads of blk are done
    __builtin_amdgcn_wave_barrier();
  }
}

// Coordinates in canonical order: the retained kernels write each example's
// block sums in entry (tile) order, contiguously, to Zt; one workgroup per
// example then gathers them into canonical order and applies the weights:
//   Z[i, r] = w_r * Zt[i, pos(r)].
// (Writing canonical positions straight from the blocks scatters 4-byte
// stores over the whole row, which cost as much as the products themselves.)
// Grid: (coordinate chunks of 2048, examples).
constexpr int kZpermPer = 8;    // coordinates per thread (independent gathers in flight)

// OT: float, or _Float16: the fp32 coordinate rounded to fp16 (nearest even).
// The opaque step keeps the product and the conversion apart (a fused
// multiply-convert would round the exact product once), so an fp16 Z equals
// the fp32 Z converted afterwards.
template <typename OT>
__device__ __forceinline__ OT coord_out(float v) {
  if constexpr (!std::is_same<OT, float>::value) asm("" : "+v"(v));
  return (OT)v;
}

template <typename OT>
__global__ __launch_bounds__(256) void k_zperm(const float* __restrict__ Zt, int64_t m,
                                               const int32_t* __restrict__ ent_pos,
                                               const float* __restrict__ w,
                                               OT* __restrict__ Z, int64_t ldz, int64_t ex0) {
  const int64_t i = ex0 + blockIdx.y;
  const float* src = Zt + i * m;
  const int64_t r0 = (int64_t)blockIdx.x * 256 * kZpermPer + threadIdx.x;
  float v[kZpermPer];
#pragma unroll
  for (int e = 0; e < kZpermPer; ++e) {
    const int64_t r = r0 + 256 * e;
    v[e] = r < m ? src[ent_pos[r]] : 0.f;
  }
#pragma unroll
  for (int e = 0; e < kZpermPer; ++e) {
    const int64_t r = r0 + 256 * e;
    if (r < m) Z[i * ldz + r] = coord_out<OT>(w[r] * v[e]);
  }
}

// Rows of up to kZpermLdsMax coordinates: one workgroup per example copies
// the row of block sums into LDS with 16-byte loads, then gathers from LDS and
// writes Z coalesced (the random reads stay on chip).
constexpr int kZpermLdsMax = 32768;

template <typename OT>
__global__ __launch_bounds__(1024) void k_zperm_lds(const float* __restrict__ Zt, int m,
                                                    const int32_t* __restrict__ ent_pos,
                                                    const float* __restrict__ w,
                                                    OT* __restrict__ Z, int64_t ldz, int64_t ex0) {
  extern __shared__ float L[];
  const int64_t i = ex0 + blockIdx.x;
  const float* src = Zt + i * (int64_t)m;
  const int tid = threadIdx.x, nt = blockDim.x;
  if ((m & 3) == 0) {                          // rows start on 16-byte boundaries
    for (int c = tid; c < m / 4; c += nt)
      reinterpret_cast<float4*>(L)[c] = reinterpret_cast<const float4*>(src)[c];
  } else {
    for (int c = tid; c < m; c += nt) L[c] = src[c];
  }
  __syncthreads();
  OT* dst = Z + i * ldz;
  for (int r = tid; r < m; r += nt) dst[r] = coord_out<OT>(w[r] * L[ent_pos[r]]);
}

struct Work {
  int32_t* cnt;   // [N + 1] per-example run lengths, scanned in place into offsets
  int32_t* len;   // [N] valid tokens per example (aligned runs only)
  int32_t* tok;   // [N*T + 8N] global token index of each listed token
  float* St;      // [N*T][rows_pad] (fp32 intermediates)
  float* At;      // [N*T][cols_pad]
  uint16_t* St16; // rows_pad x ldt entries, MFMA-fragment order (fp16 intermediates)
  uint16_t* At16; // cols_pad x ldt entries
  int64_t ldt = 0;
  float* Zt;      // [N][m] block sums in entry order (retained products only)
  int32_t* sched; // [kXcds] work counters of the rotation launch
};

// Token capacity of the fp16 layout: runs padded to multiples of 8, the
// 256-row output tiles of the rotation, and the up to 16 kRetGUnroll + 8
// tokens a batch of the retained products reads past the last run.
int64_t f16_ldt(int64_t N, int64_t T) { return round_up(N * T + 8 * N + 256, 256); }

size_t token_bytes(int64_t N, int64_t T) {
  return align256((N + 1) * 4) + align256((size_t)N * 4) + align256((size_t)(N * T + 8 * N) * 4);
}

size_t work_bytes(const eogp_plan* p, int64_t N, int64_t T) {
  size_t b = token_bytes(N, T);
  const size_t f32b = align256((size_t)N * T * p->rows_pad * 4) + align256((size_t)N * T * p->cols_pad * 4);
  const int64_t ldt = f16_ldt(N, T);
  const size_t f16b = align256((size_t)ldt * p->rows_pad * 2) + align256((size_t)ldt * p->cols_pad * 2);
  b += std::max(f32b, f16b);
  b += align256((size_t)N * p->m * 4);
  b += align256(kXcds * 4);
  return b;
}

}  // namespace

size_t rotate_retain_ws(const eogp_plan* p, int64_t N, int64_t T) { return work_bytes(p, N, T); }

namespace {

// Step 1: the valid-token list (counts, per-example lengths, token indices)
// at the head of the workspace. t16: runs aligned to 8 tokens (the 16-bit
// fragment-order intermediates), else packed.
eogp_status compact_into(const uint8_t* mask, int64_t N, int64_t T, bool t16, int32_t* cnt,
                         int32_t* len, int32_t* tok, hipStream_t s) {
  const unsigned g4 = (unsigned)ceil_div(N, 4);
  timing::Scope ts(EOGP_KT_COMPACTION, s);
  hipLaunchKernelGGL(k_count_valid, dim3(g4), dim3(256), 0, s, mask, N, T, t16 ? 8 : 1, cnt, len);
  EOGP_HIP(scan_exclusive(cnt, N, s));
  hipLaunchKernelGGL(k_write_tokens, dim3(g4), dim3(256), 0, s, mask, N, T, cnt, tok);
  EOGP_LAUNCH_CHECK("token compaction");
  return EOGP_OK;
}

// Steps 1 and 2: compaction of the valid tokens (unless `compact` is false:
// the list is then already in w) and the two rotations onto the plan's
// eigenvector panels; fills w (carved from ws). t16: fp16 transposed
// intermediates with runs aligned to 8 tokens (else fp32, token-major, runs
// packed).
eogp_status rotate_tokens(const eogp_plan* p, const void* acts, int64_t ld_acts,
                          const void* grads, int64_t ld_grads, bool bf16_in, const uint8_t* mask,
                          int64_t N, int64_t T, int prec, bool t16, bool compact, Work& w,
                          hipStream_t s) {
  // 1. compaction
  if (compact) {
    const eogp_status st = compact_into(mask, N, T, t16, w.cnt, w.len, w.tok, s);
    if (st != EOGP_OK) return st;
  }

  // 2. rotations onto the used eigenvectors (rows = listed tokens; count on device)
  // FAST: bf16 operands; ACCURATE: bf16 high+low splits (three products);
  // F16: inputs scaled by 2^e and rounded once to fp16, fp16 bases.
  const bool accurate = prec == EOGP_PREC_ACCURATE;
  const bool f16 = prec == EOGP_PREC_F16;
  // bf16 inputs in the F16 mode are widened, scaled and rounded to fp16 (exact
  // inside fp16's normal range: bf16 carries 8 significant bits, fp16 11)
  const AType at = bf16_in ? (f16 ? AType::BF16_AS_F16 : AType::B16) : AType::F32;
  const int a_parts = (accurate && !bf16_in) ? 2 : 1;
  const int b_parts = accurate ? 2 : 1;
  GemmArgs gs;
  gs.A = grads;
  gs.lda = ld_grads;
  gs.a_rows = w.tok;
  gs.a_scale = f16 ? std::ldexp(1.f, p->e_grads) : 1.f;
  gs.B_hi = f16 ? p->qs_f16 : p->qs_hi;
  gs.B_lo = p->qs_lo;
  gs.ldb = p->ld_out;
  gs.b_padded = true;
  if (t16) {
    gs.CT = w.St16;
    gs.ldct = w.ldt;
    gs.ct_bf16 = !f16;   // FAST: bf16 intermediates (fp32's range); F16: fp16
  } else {
    gs.C = w.St;
    gs.ldc = p->rows_pad;
  }
  gs.M = t16 ? N * T + 7 * N : N * T;
  gs.M_dev = w.cnt + N;
  // Columns n_rows..rows_pad-1 of S~ are left unwritten (fp32) or hold
  // zeros (fp16, zero panel rows): they only feed block outputs never read.
  gs.N = p->n_rows;
  gs.K = p->d_out;
  GemmArgs ga = gs;
  ga.A = acts;
  ga.lda = ld_acts;
  ga.a_scale = f16 ? std::ldexp(1.f, p->e_acts) : 1.f;
  ga.B_hi = f16 ? p->qa_f16 : p->qa_hi;
  ga.B_lo = p->qa_lo;
  ga.ldb = p->ld_in;
  if (t16) {
    ga.CT = w.At16;
  } else {
    ga.C = w.At;
    ga.ldc = p->cols_pad;
  }
  ga.N = p->n_cols;
  ga.K = p->d_in;
  // One launch for both rotations, the longer contraction first.
  GemmArgs& first = gs.K >= ga.K ? gs : ga;
  GemmArgs& second = gs.K >= ga.K ? ga : gs;
  first.sched = w.sched;
  second.sched = nullptr;
  return gemm_nt2(first, second, at, a_parts, b_parts, f16, s);
}

// The token list heads every first-stage workspace (eogp_compact_tokens
// fills it alone): counts [N + 1], lengths [N], token indices [N T + 8 N].
void carve_tokens(int64_t N, int64_t T, Carve& cv, Work& w) {
  w.cnt = cv.take<int32_t>(N + 1);
  w.len = cv.take<int32_t>(N);
  w.tok = cv.take<int32_t>((size_t)(N * T + 8 * N));
}

Work carve_work(const eogp_plan* p, int64_t N, int64_t T, Carve& cv) {
  Work w;
  carve_tokens(N, T, cv, w);
  // the fp32 and fp16 layouts share one region
  const size_t f32b = align256((size_t)N * T * p->rows_pad * 4) + align256((size_t)N * T * p->cols_pad * 4);
  w.ldt = f16_ldt(N, T);
  const size_t f16b = align256((size_t)w.ldt * p->rows_pad * 2) + align256((size_t)w.ldt * p->cols_pad * 2);
  char* base = cv.take<char>(std::max(f32b, f16b));
  w.St = reinterpret_cast<float*>(base);
  w.At = reinterpret_cast<float*>(base + align256((size_t)N * T * p->rows_pad * 4));
  w.St16 = reinterpret_cast<uint16_t*>(base);
  w.At16 = reinterpret_cast<uint16_t*>(base + align256((size_t)w.ldt * p->rows_pad * 2));
  w.Zt = cv.take<float>((size_t)N * p->m);
  w.sched = cv.take<int32_t>(kXcds);
  return w;
}

}  // namespace

size_t compact_ws(int64_t N, int64_t T) { return token_bytes(N, T); }

eogp_status compact_tokens(const uint8_t* mask, int64_t N, int64_t T, int prec, void* ws,
                           size_t ws_bytes, hipStream_t s) {
  if (ws_bytes < token_bytes(N, T)) return fail(EOGP_ERR_WORKSPACE, "compact_tokens: workspace too small");
  Carve cv(ws, ws_bytes);
  Work w;
  carve_tokens(N, T, cv, w);
  return compact_into(mask, N, T, prec != EOGP_PREC_ACCURATE, w.cnt, w.len, w.tok, s);
}

// compacted: the token list is already at the head of ws (compact_tokens or
// an earlier call with the same mask, sizes and precision class).
eogp_status rotate_retain(const eogp_plan* p, const void* acts, int64_t ld_acts, const void* grads,
                          int64_t ld_grads, bool bf16_in,
                          const uint8_t* mask, int64_t N, int64_t T, void* Z, bool z16,
                          int64_t ldz, int prec, bool compacted, void* ws, size_t ws_bytes,
                          hipStream_t s) {
  if (ws_bytes < work_bytes(p, N, T)) return fail(EOGP_ERR_WORKSPACE, "rotate_retain: workspace too small");
  Carve cv(ws, ws_bytes);
  Work w = carve_work(p, N, T, cv);
  const bool f16 = prec == EOGP_PREC_F16;
  // 16-bit fragment-order intermediates in the F16 (fp16) and FAST (bf16)
  // modes; fp32 token-major ones in the ACCURATE mode
  const bool t16 = prec != EOGP_PREC_ACCURATE;
  eogp_status st = rotate_tokens(p, acts, ld_acts, grads, ld_grads, bf16_in, mask, N, T, prec, t16,
                                 !compacted, w, s);
  if (st != EOGP_OK) return st;

  // 3. retained products, half-whitened, in canonical order
  const float out_scale = f16 ? std::ldexp(1.f, -(p->e_acts + p->e_grads)) : 1.f;
  if (p->m <= kZpermLdsMax) {
    const void* fn = z16 ? (const void*)k_zperm_lds<_Float16> : (const void*)k_zperm_lds<float>;
    const eogp_status st_lds = ensure_dynamic_lds(fn, (int)(sizeof(float) * kZpermLdsMax));
    if (st_lds != EOGP_OK) return st_lds;
  }
  // examples per launch: the 2-D grid's y limit, and the 1-D grid of the fp16
  // kernel (kXcds x ceil(nex / kXcds) x tile groups) below 2^31
  // the fp16 kernels take groups of blocks, the fp32 one single blocks
  const int64_t gx64 = ceil_div(t16 ? p->n_groups : p->n_tiles, (int64_t)kRetWaves);
  const int64_t ex_chunk = std::max<int64_t>(
      kXcds, std::min<int64_t>(65535 / kXcds * kXcds,
                               (((int64_t)1 << 31) - 1) / (kXcds * std::max<int64_t>(1, gx64)) * kXcds));
  for (int64_t ex0 = 0; p->n_tiles > 0 && ex0 < N; ex0 += ex_chunk) {
    const int64_t nex = std::min<int64_t>(ex_chunk, N - ex0);
    timing::Scope ts(EOGP_KT_RETAINED, s);
    const unsigned gx = (unsigned)gx64;
    if (t16) {
      const dim3 grid16((unsigned)(kXcds * ceil_div(nex, kXcds) * gx));
      auto kfn = f16 ? (p->group_rows ? k_retained16g<false, true> : k_retained16g<false, false>)
                     : (p->group_rows ? k_retained16g<true, true> : k_retained16g<true, false>);
      hipLaunchKernelGGL(kfn, grid16, dim3(256), 0, s, w.St16, w.At16, w.ldt, w.cnt, w.len, p->groups,
                         (int)p->n_groups, p->gtiles, p->tiles, p->ent_loc, out_scale, w.Zt, p->m,
                         ex0, nex);
    } else {
      hipLaunchKernelGGL(k_retained, dim3(gx, (unsigned)nex), dim3(256), 0, s,
                         w.St, p->rows_pad, w.At, p->cols_pad, w.cnt, p->tiles, (int)p->n_tiles,
                         p->ent_loc, out_scale, w.Zt, p->m, ex0);
    }
    const dim3 gz((unsigned)ceil_div(p->m, 256 * kZpermPer), (unsigned)nex);
    if (p->m <= kZpermLdsMax && z16) {
      hipLaunchKernelGGL(k_zperm_lds<_Float16>, dim3((unsigned)nex), dim3(1024), (size_t)p->m * 4,
                         s, w.Zt, (int)p->m, p->ent_pos, p->ret_w, static_cast<_Float16*>(Z), ldz,
                         ex0);
    } else if (p->m <= kZpermLdsMax) {
      hipLaunchKernelGGL(k_zperm_lds<float>, dim3((unsigned)nex), dim3(1024), (size_t)p->m * 4, s,
                         w.Zt, (int)p->m, p->ent_pos, p->ret_w, static_cast<float*>(Z), ldz, ex0);
    } else if (z16) {
      hipLaunchKernelGGL(k_zperm<_Float16>, gz, dim3(256), 0, s, w.Zt, p->m, p->ent_pos,
                         p->ret_w, static_cast<_Float16*>(Z), ldz, ex0);
    } else {
      hipLaunchKernelGGL(k_zperm<float>, gz, dim3(256), 0, s, w.Zt, p->m, p->ent_pos, p->ret_w,
                         static_cast<float*>(Z), ldz, ex0);
    }
    EOGP_LAUNCH_CHECK("retained products");
  }
  return EOGP_OK;
}

// ---- EK-FAC corrected eigenvalues ---------------------------------------------
// Lambda[j, k] = mean over examples of (Q_S^T G_i Q_A)[j, k]^2 (Section 2.2,
// eq. ekfac_eigendecompose; corrected eigenvalues over examples from
// sequence-level gradients, Appendix C.2). After the rotations onto every
// eigenvector, the examples are walked in order: the block of sums
// C = sum_t S~[t, j] A~[t, k] over the example's valid tokens is formed with
// MFMA and C * C is added to a running sum of squares in registers, so the
// result does not depend on scheduling. FAST and ACCURATE: fp32 token-major
// intermediates, one wave per 32 x 32 block, fp32 MFMA (exact products).
// fp16 mode: fp16 fragment-order intermediates, fp16 MFMA (k_ekfac_sq16).
namespace {

__global__ __launch_bounds__(256) void k_ekfac_sq(const float* __restrict__ St, int64_t ldS,
                                                  const float* __restrict__ At, int64_t ldA,
                                                  const int32_t* __restrict__ ex_off, int64_t N,
                                                  int nbk, int d_out, int d_in,
                                                  float* __restrict__ sq, int accumulate) {
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int jb = blockIdx.y;
  const int kb = blockIdx.x * 4 + wid;
  if (kb >= nbk) return;
  const int half = lane >> 5, col = lane & 31;
  const float* sp = St + (int64_t)jb * 32 + col;
  const float* ap = At + (int64_t)kb * 32 + col;
  f32x16 acc2;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc2[r] = 0.f;
  for (int64_t i = 0; i < N; ++i) {
    const int64_t t0 = ex_off[i], t1 = ex_off[i + 1];
    f32x16 c;
#pragma unroll
    for (int r = 0; r < 16; ++r) c[r] = 0.f;
    for (int64_t tb = t0; tb < t1; tb += 16) {
      float sv[8], av[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int64_t t = tb + 2 * u + half;
        const bool ok = t < t1;
        sv[u] = ok ? sp[t * ldS] : 0.f;
        av[u] = ok ? ap[t * ldA] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) c = __builtin_amdgcn_mfma_f32_32x32x2f32(sv[u], av[u], c, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) acc2[r] = fmaf(c[r], c[r], acc2[r]);
  }
  // acc2[r] holds block entry (8 (r / 4) + 4 half + r % 4, col)
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int j = jb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
    const int k = kb * 32 + col;
    if (j < d_out && k < d_in) {
      float* o = sq + (int64_t)j * d_in + k;
      *o = accumulate ? *o + acc2[r] : acc2[r];
    }
  }
}

// fp16 mode: S~ and A~ in the fp16 fragment order of the first stage (runs
// aligned to 8 tokens). A wave owns one 32-row block jb and KQ = 4 32-column
// blocks kb .. kb+3 (32 x 128 entries); per 16 tokens it loads one S~ block
// and four A~ blocks (1 KB each) and issues four v_mfma_f32_32x32x16_f16, so
// each loaded block feeds 0.8 MFMAs; the four waves of a
// workgroup take neighbouring row blocks and the same column blocks, whose
// loads they share through the L1. Example by example the block sums C are
// formed over the example's tokens (tokens past its run zeroed) and C * C is
// added to the running sums. Small modules split the examples into ranges
// (grid z) so that the grid still fills the chip; each range writes its own
// partial sums, which k_ekfac_sum adds in range order (deterministic).
constexpr int kSq16Unroll = 4;     // 16-token steps loaded per batch
constexpr int kSq16Cols = 4;       // 32-column blocks per wave (measured best of 1, 2, 4, 8)

template <int KQ>
__global__ __launch_bounds__(256) void k_ekfac_sq16(const uint16_t* __restrict__ St,
                                                    const uint16_t* __restrict__ At, int64_t ldt,
                                                    const int32_t* __restrict__ ex_off,
                                                    const int32_t* __restrict__ ex_len, int64_t N,
                                                    int splits, int d_out, int d_in,
                                                    float* __restrict__ part) {
  typedef unsigned int v4u __attribute__((ext_vector_type(4)));
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int jb = blockIdx.y * 4 + wid;
  const int kb0 = blockIdx.x * KQ;
  if (jb * 32 >= d_out) return;                // whole wave leaves; no block barrier below
  const int split = blockIdx.z;
  const int64_t i_beg = split * N / splits, i_end = (split + 1) * N / splits;
  const int half = lane >> 5, col = lane & 31;
  const int64_t groups = ldt / 16;
  auto at_tok = [&](int64_t b, int64_t t) { return ((b * groups + (t >> 4)) * 32 + col) * 16 + (t & 15); };
  f32x16 acc2[KQ];
#pragma unroll
  for (int q = 0; q < KQ; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc2[q][r] = 0.f;
  for (int64_t i = i_beg; i < i_end; ++i) {
    const int n = ex_len[i];
    if (n == 0) continue;
    const int64_t t0 = ex_off[i] + 8 * half;
    const uint16_t* sp = St + at_tok(jb, t0);
    const uint16_t* ap = At + at_tok(kb0, t0);
    const int64_t bstride = groups * 512;      // elements from one column block to the next
    f32x16 c[KQ];
#pragma unroll
    for (int q = 0; q < KQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) c[q][r] = 0.f;
    for (int t = 0; t < n; t += 16 * kSq16Unroll) {
      v4u a[kSq16Unroll], b[kSq16Unroll][KQ];
#pragma unroll
      for (int u = 0; u < kSq16Unroll; ++u) {
        const int64_t o = (int64_t)(t / 16 + u) * 512;
        a[u] = *reinterpret_cast<const v4u*>(sp + o);
#pragma unroll
        for (int q = 0; q < KQ; ++q) b[u][q] = *reinterpret_cast<const v4u*>(ap + q * bstride + o);
      }
#pragma unroll
      for (int u = 0; u < kSq16Unroll; ++u) {
        const int tu = t + 16 * u;
        if (tu >= n) break;
        if (tu + 16 > n) {
          const int rem = n - tu - 8 * half;     // valid tokens among this lane's eight
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            const uint32_t keep = (2 * d < rem ? 0x0000FFFFu : 0u) | (2 * d + 1 < rem ? 0xFFFF0000u : 0u);
            a[u][d] &= keep;
#pragma unroll
            for (int q = 0; q < KQ; ++q) b[u][q][d] &= keep;
          }
        }
#pragma unroll
        for (int q = 0; q < KQ; ++q)
          c[q] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a[u]),
                                                        __builtin_bit_cast(f16x8, b[u][q]), c[q], 0, 0, 0);
      }
    }
#pragma unroll
    for (int q = 0; q < KQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc2[q][r] = fmaf(c[q][r], c[q][r], acc2[q][r]);
  }
  // acc2[q][r] holds entry (32 jb + 8 (r / 4) + 4 half + r % 4, 32 (kb0 + q) + col)
  float* o = part + (int64_t)split * d_out * d_in;
#pragma unroll
  for (int q = 0; q < KQ; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = jb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      const int k = (kb0 + q) * 32 + col;
      if (j < d_out && k < d_in) o[(int64_t)j * d_in + k] = acc2[q][r];
    }
}

// sq[e] = (accumulate ? sq[e] : 0) + h^2 * sum over ranges, in order, of part[s][e]
// (h = 2^-(e_acts + e_grads) undoes the input scaling of both factors; applied
// twice so that the factor itself neither overflows nor underflows).
__global__ __launch_bounds__(256) void k_ekfac_sum(const float* __restrict__ part, int splits,
                                                   int64_t n, float h, float* __restrict__ sq,
                                                   int accumulate) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= n) return;
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[s * n + e];
  v = (v * h) * h;
  sq[e] = accumulate ? sq[e] + v : v;
}

__global__ __launch_bounds__(256) void k_fill_zero(float* __restrict__ x, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n) x[e] = 0.f;
}

// Example ranges of the fp16 squares: enough workgroups for two per CU, at
// least 4 examples per range, at most 32 ranges.
int sq16_splits(int64_t N, int64_t d_in, int64_t d_out) {
  const int64_t groups = ceil_div(d_in, 32 * kSq16Cols) * ceil_div(d_out, 128);
  int64_t sp = ceil_div(2 * kCus, groups);
  sp = std::min<int64_t>(sp, std::max<int64_t>(1, N / 4));
  return (int)std::max<int64_t>(1, std::min<int64_t>(sp, 32));
}

eogp_plan basis_plan(int64_t d_in, int64_t d_out) {
  eogp_plan q;
  q.d_out = d_out;
  q.d_in = d_in;
  q.n_rows = d_out;
  q.n_cols = d_in;
  q.rows_pad = round_up(d_out, kPanelTile);
  q.cols_pad = round_up(d_in, kPanelTile);
  q.ld_out = round_up(d_out, 32);
  q.ld_in = round_up(d_in, 32);
  return q;
}

size_t panel_bytes(const eogp_plan& q) {
  return 3 * align256((size_t)q.rows_pad * q.ld_out * 2) + 3 * align256((size_t)q.cols_pad * q.ld_in * 2) +
         align256((size_t)std::max(q.d_in, q.d_out) * 4);
}

}  // namespace

size_t ekfac_ws(int64_t N, int64_t T, int64_t d_in, int64_t d_out) {
  const eogp_plan q = basis_plan(d_in, d_out);
  return work_bytes(&q, N, T) + panel_bytes(q) +
         align256((size_t)sq16_splits(N, d_in, d_out) * d_out * d_in * 4);
}

eogp_status ekfac_pass(const void* acts, int64_t ld_acts, const void* grads, int64_t ld_grads,
                       bool bf16_in, const uint8_t* mask, int64_t N, int64_t T, int64_t d_in,
                       int64_t d_out, const float* Q_A, const float* Q_S, int prec,
                       int32_t e_acts, int32_t e_grads, float* sq, int accumulate, void* ws,
                       size_t ws_bytes, hipStream_t s) {
  eogp_plan q = basis_plan(d_in, d_out);
  if (ws_bytes < ekfac_ws(N, T, d_in, d_out)) return fail(EOGP_ERR_WORKSPACE, "ekfac: workspace too small");
  if (N == 0) {                                  // an empty batch adds nothing
    if (!accumulate) {
      hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)ceil_div(d_out * d_in, 256)), dim3(256), 0, s,
                         sq, d_out * d_in);
      EOGP_LAUNCH_CHECK("ekfac (empty batch)");
    }
    return EOGP_OK;
  }
  q.e_acts = e_acts;
  q.e_grads = e_grads;
  Carve cv(ws, ws_bytes);
  Work w = carve_work(&q, N, T, cv);
  q.qs_hi = cv.take<uint16_t>((size_t)q.rows_pad * q.ld_out);
  q.qs_lo = cv.take<uint16_t>((size_t)q.rows_pad * q.ld_out);
  q.qs_f16 = cv.take<uint16_t>((size_t)q.rows_pad * q.ld_out);
  q.qa_hi = cv.take<uint16_t>((size_t)q.cols_pad * q.ld_in);
  q.qa_lo = cv.take<uint16_t>((size_t)q.cols_pad * q.ld_in);
  q.qa_f16 = cv.take<uint16_t>((size_t)q.cols_pad * q.ld_in);
  int* list = cv.take<int>((size_t)std::max(d_in, d_out));
  basis_panels(Q_S, d_out, q.rows_pad, q.ld_out, list, q.qs_hi, q.qs_lo, q.qs_f16, s);
  basis_panels(Q_A, d_in, q.cols_pad, q.ld_in, list, q.qa_hi, q.qa_lo, q.qa_f16, s);
  EOGP_LAUNCH_CHECK("ekfac panels");
  float* part = cv.take<float>((size_t)sq16_splits(N, d_in, d_out) * d_out * d_in);
  const bool f16 = prec == EOGP_PREC_F16;
  eogp_status st = rotate_tokens(&q, acts, ld_acts, grads, ld_grads, bf16_in, mask, N, T, prec, f16,
                                 true, w, s);
  if (st != EOGP_OK) return st;
  timing::Scope ts(EOGP_KT_EKFAC, s);
  if (f16) {
    const int sp = sq16_splits(N, d_in, d_out);
    hipLaunchKernelGGL(k_ekfac_sq16<kSq16Cols>, dim3((unsigned)ceil_div(d_in, 32 * kSq16Cols), (unsigned)ceil_div(d_out, 128),
                                          (unsigned)sp),
                       dim3(256), 0, s, w.St16, w.At16, w.ldt, w.cnt, w.len, N, sp, (int)d_out,
                       (int)d_in, part);
    const int64_t n = d_out * d_in;
    const float h = std::ldexp(1.f, -(e_acts + e_grads));
    hipLaunchKernelGGL(k_ekfac_sum, dim3((unsigned)ceil_div(n, 256)), dim3(256), 0, s, part, sp, n,
                       h, sq, accumulate);
    EOGP_LAUNCH_CHECK("ekfac squares");
    return EOGP_OK;
  }
  const int nbj = (int)ceil_div(d_out, 32), nbk = (int)ceil_div(d_in, 32);
  hipLaunchKernelGGL(k_ekfac_sq, dim3((unsigned)ceil_div(nbk, 4), (unsigned)nbj), dim3(256), 0, s,
                     w.St, q.rows_pad, w.At, q.cols_pad, w.cnt, N, nbk, (int)d_out, (int)d_in, sq,
                     accumulate);
  EOGP_LAUNCH_CHECK("ekfac squares");
  return EOGP_OK;
}

}  // namespace eogp
