// Scoring stored one-bit codes against unquantized query projections
// (eq. onebit_influence, eq. app_stored_influence) with a per-query top-k.
//
// Arithmetic. Each query module vector y is taken in fixed point,
// y_int = rint(y 2^f) with f = 14 - e for max|y| = mu 2^e (|y_int| <= 2^14), and
// split into two int8 planes y_int = 256 h + l (h in [-64, 64], l in
// [-128, 127]). With b in {0, 1} the MFMA computes n1 = sum_{b=1} y_int exactly
// in int32, and <y_int, 2b - 1> = 2 n1 - sum(y_int). Each module term
// s * (2 n1 - sum) * 2^-f is exact in fp64 and the terms are added in module
// order, so the score is reproducible bit for bit.
//
// Data flow. A pass streams every stored code once for a group of 16 queries
// (the 16 columns of v_mfma_i32_16x16x64_i8). A 512-thread workgroup (8
// waves) owns 1024 consecutive examples at a time, each wave 8 tiles of 16
// rows. The pass walks the modules in 512-bit steps; per step the workgroup
// stages the query planes (16 KB) in LDS once for its 1024 rows,
// double-buffered, and each wave multiplies its 128 rows against them (each
// plane fragment read from LDS feeds 8 MFMAs) with its code words for that
// step, which it requested one step earlier (16-byte loads). Bits are
// expanded without reordering the stored layout: the 32-bit code word w
// yields the int8 operand dwords (w >> d) & 0x01010101 (bits d, d+8, d+16,
// d+24), and the query planes are laid out in that same permuted order when
// they are prepared.
// After the last module the workgroup's scores are filtered against a
// per-query threshold into an LDS candidate list (score desc, index asc). A
// list that fills up is pruned to the top-k (bitonic sort) and the entries
// that did not fit are inserted again, so no qualifying row is lost. Finally
// each workgroup writes its top-k per query and a merge kernel reduces them.
#include <algorithm>
#include <vector>

#include "common.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int QB = 16;          // queries per pass
constexpr int NW = 8;           // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int KSTEP = 8;        // MFMA k-steps (64 bits each) per 512-bit step
constexpr int MCAP = 512;       // candidate slots per query in the merge
constexpr int MAX_TOPK = 256;

struct ModInfo {
  int32_t k;       // bits of the module
  int32_t coff;    // first coordinate of the module in a query row
  int32_t boff;    // first byte of the module in a code row
  int32_t ksbase;  // first k-step of the module in the plane buffer
};

__device__ __forceinline__ uint64_t order_key(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double key_value(uint64_t k) {
  uint64_t u = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
  return __longlong_as_double((long long)u);
}
__device__ __forceinline__ bool before(uint64_t ka, uint32_t ia, uint64_t kb, uint32_t ib) {
  return ka > kb || (ka == kb && ia < ib);
}

// ---- query preparation --------------------------------------------------------
// grid (Q, U): per (query, module) the exponent f and sum of y_int.
__global__ __launch_bounds__(256) void k_query_stats(const float* __restrict__ Y, int64_t ldy,
                                                     int U, const ModInfo* __restrict__ mods,
                                                     int32_t* __restrict__ fq,
                                                     int32_t* __restrict__ ysum) {
  __shared__ float smax[4];
  __shared__ int ssum[4];
  const int64_t q = blockIdx.x;
  const int u = blockIdx.y;
  const ModInfo md = mods[u];
  const float* y = Y + q * ldy + md.coff;
  float mx = 0.f;
  for (int c = threadIdx.x; c < md.k; c += 256) mx = fmaxf(mx, fabsf(y[c]));
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if ((threadIdx.x & 63) == 0) smax[threadIdx.x >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(smax[0], smax[1]), fmaxf(smax[2], smax[3]));
  int f = 0;
  if (mx > 0.f) {
    int e;
    (void)frexpf(mx, &e);
    f = 14 - e;
  }
  int s = 0;
  if (mx > 0.f)
    for (int c = threadIdx.x; c < md.k; c += 256) s += (int)rintf(ldexpf(y[c], f));
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if ((threadIdx.x & 63) == 0) ssum[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    fq[q * U + u] = f;
    ysum[q * U + u] = ssum[0] + ssum[1] + ssum[2] + ssum[3];
  }
}

// One thread per plane byte: (group, k-step, lane, slot) -> coordinate c of the
// lane's row/column mapping; writes h and l of y_int (0 outside the module).
__global__ void k_query_planes(const float* __restrict__ Y, int64_t ldy, int64_t Q, int U,
                               const ModInfo* __restrict__ mods, const int32_t* __restrict__ fq,
                               int64_t KS, int64_t n_groups, int8_t* __restrict__ ph,
                               int8_t* __restrict__ pl) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = n_groups * KS * 64 * 16;
  if (idx >= total) return;
  const int slot = (int)(idx & 15);
  const int lane = (int)((idx >> 4) & 63);
  const int64_t K = (idx >> 10) % KS;
  const int64_t grp = (idx >> 10) / KS;
  int u = 0;
  while (u + 1 < U && mods[u + 1].ksbase <= K) ++u;
  const ModInfo md = mods[u];
  const int64_t Ku = K - md.ksbase;
  const int64_t ms = Ku / KSTEP;
  const int s = (int)(Ku % KSTEP);
  const int g = lane >> 4, n = lane & 15;
  const int e = slot >> 2, b = slot & 3;
  const int64_t c = 32 * (16 * ms + 4 * g + (s >> 1)) + 4 * (s & 1) + e + 8 * b;
  const int64_t q = grp * QB + n;
  int yi = 0;
  if (q < Q && c < md.k) yi = (int)rintf(ldexpf(Y[q * ldy + md.coff + c], fq[q * U + u]));
  const int h = (yi + 128) >> 8;   // floor division (arithmetic shift)
  const int l = yi - 256 * h;
  ph[idx] = (int8_t)h;
  pl[idx] = (int8_t)l;
}

// ---- candidate lists in LDS ---------------------------------------------------
template <int CAP>
struct Cand {
  uint64_t key[QB][CAP];
  uint32_t idx[QB][CAP];
  int cnt[QB];
  uint64_t thr[QB];
  int overflow;
};

// Sort list n (all NTH threads), keep its first `topk`, update the threshold.
// Entries past CAP (counted but not stored) are dropped here; their owners
// insert them again.
template <int CAP, int NTH>
__device__ void prune(Cand<CAP>& cd, int n, int topk) {
  const int tid = threadIdx.x;
  const int c = min(cd.cnt[n], CAP);
  for (int i = c + tid; i < CAP; i += NTH) {
    cd.key[n][i] = 0ull;
    cd.idx[n][i] = 0xFFFFFFFFu;
  }
  __syncthreads();
  for (int k = 2; k <= CAP; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < CAP; i += NTH) {
        const int p = i ^ j;
        if (p > i) {
          const uint64_t ka = cd.key[n][i], kb = cd.key[n][p];
          const uint32_t ia = cd.idx[n][i], ib = cd.idx[n][p];
          const bool desc = (i & k) == 0;
          const bool ab = before(ka, ia, kb, ib);
          if (desc ? !ab : ab) {
            cd.key[n][i] = kb; cd.key[n][p] = ka;
            cd.idx[n][i] = ib; cd.idx[n][p] = ia;
          }
        }
      }
      __syncthreads();
    }
  }
  if (tid == 0) {
    cd.thr[n] = (c >= topk) ? cd.key[n][topk - 1] : 0ull;
    cd.cnt[n] = c < topk ? c : topk;
  }
  __syncthreads();
}

// One step of the pass (one or two 512-bit halves of one module): module,
// first code byte of the step within a row, first k-step of its query
// planes, valid code bytes, whether it is the module's last step, and its
// number of halves.
struct Step {
  int32_t u, boff, kbase, bytes, last, halves, pad0, pad1;
};

struct ScoreArgs {
  const uint8_t* codes;
  int64_t cstride;
  const uint16_t* scales;
  int64_t N;
  int U;
  const ModInfo* mods;
  const int8_t* ph;
  const int8_t* pl;
  const Step* steps;
  int n_steps;
  int64_t KS;
  int64_t grp;
  const int32_t* fq;
  const int32_t* ysum;
  int64_t Q;
  int topk;
  float* full;
  uint64_t* ckey;   // [grid][QB][topk]
  uint32_t* cidx;
};

// RT: 16-row tiles per wave (rows per block: NW * RT * 16). MULTI: several
// modules, whose fp64 terms are summed in module order as each ends; else
// one module, whose term is formed after its last step. HS: 512-bit halves per
// step; with HS = 2 a lane reads both 64-byte halves of each 128-byte line of
// its rows in the same step.
template <int CAP, int RT, bool MULTI, int HS>
__global__ __launch_bounds__(NTHR) void k_score(ScoreArgs a) {
  constexpr int ROWS = NW * RT * 16;
  constexpr int PU = 2 * HS * KSTEP * 64;            // plane uint4 per step
  constexpr int PV = PU / NTHR;                      // staged per thread
  __shared__ __attribute__((aligned(16))) uint4 sP[2][2][HS * KSTEP][64];
  __shared__ Cand<CAP> cd;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int n = lane & 15;           // query column of this lane
  const int g = lane >> 4;           // k-group of this lane
  const int64_t q = a.grp * QB + n;
  const bool q_ok = q < a.Q;
  if (tid < QB) {
    cd.cnt[tid] = 0;
    cd.thr[tid] = 0ull;
  }
  if (tid == 0) cd.overflow = 0;
  __syncthreads();
  const int64_t n_blocks = (a.N + ROWS - 1) / ROWS;
  const uint4* phv = reinterpret_cast<const uint4*>(a.ph);
  const uint4* plv = reinterpret_cast<const uint4*>(a.pl);
  const uint32_t M1 = 0x01010101u;
  // plane staging: uint4 number f = tid + NTHR v of the step is (plane,
  // k-step, lane) = (f / (HS KSTEP 64), (f / 64) % (HS KSTEP), f % 64), so
  // consecutive lanes move consecutive 16 bytes; k-steps past the step's
  // valid halves are staged as zero
  auto plane_src = [&](const Step& st, int f) -> uint4 {
    const int plane = f / (HS * KSTEP * 64), ks = (f >> 6) % (HS * KSTEP), ln = f & 63;
    if (ks >= st.halves * KSTEP) return make_uint4(0u, 0u, 0u, 0u);
    const int64_t o = (a.grp * a.KS + st.kbase + ks) * 64 + ln;
    return (plane ? plv : phv)[o];
  };
  auto plane_dst = [&](int buf, int f, const uint4& v) {
    sP[buf][f / (HS * KSTEP * 64)][(f >> 6) % (HS * KSTEP)][f & 63] = v;
  };

  for (int64_t blk = blockIdx.x; blk < n_blocks; blk += gridDim.x) {
    const int64_t row0 = blk * ROWS + (int64_t)wid * (RT * 16);
    // this lane's code row of tile rt is row0 + 16 rt + n; rows past N read
    // row N - 1 and are never reported
    auto load_codes = [&](const Step& st, uint4 (*cw)[HS]) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int64_t row = std::min<int64_t>(row0 + rt * 16 + n, a.N - 1);
        const uint8_t* src = a.codes + row * a.cstride + st.boff + 16 * g;
#pragma unroll
        for (int h = 0; h < HS; ++h) {
          const int have = st.bytes - 64 * h - 16 * g;   // valid bytes of this lane's 16
          uint4 v = make_uint4(0u, 0u, 0u, 0u);
          if (have >= 16) {
            v = *reinterpret_cast<const uint4*>(src + 64 * h);
          } else if (have >= 8) {
            const uint2 hv = *reinterpret_cast<const uint2*>(src + 64 * h);
            v.x = hv.x;
            v.y = hv.y;
          }
          cw[rt][h] = v;
        }
      }
    };

    double sc[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[rt][r] = 0.0;
    i32x4 acc_h[RT], acc_l[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      acc_h[rt] = i32x4{0, 0, 0, 0};
      acc_l[rt] = i32x4{0, 0, 0, 0};
    }

    // module term: s * (2 n1 - sum y_int) * 2^-f, added in module order
    auto fold = [&](int u) {
      const int f = q_ok ? a.fq[q * a.U + u] : 0;
      const int ys = q_ok ? a.ysum[q * a.U + u] : 0;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = row0 + rt * 16 + 4 * g + r;
          const uint16_t s16 = row < a.N ? a.scales[row * a.U + u] : (uint16_t)0;
          const int n1 = 256 * acc_h[rt][r] + acc_l[rt][r];
          const int nn = 2 * n1 - ys;
          sc[rt][r] += ldexp((double)f16_bits_to_f32(s16) * (double)nn, -f);
        }
        acc_h[rt] = i32x4{0, 0, 0, 0};
        acc_l[rt] = i32x4{0, 0, 0, 0};
      }
    };

    // prologue: step 0 staged, its code words in registers
    uint4 cw[RT][HS], cwn[RT][HS];
    {
      const Step st = a.steps[0];
#pragma unroll
      for (int v = 0; v < PV; ++v) plane_dst(0, tid + NTHR * v, plane_src(st, tid + NTHR * v));
      load_codes(st, cw);
    }
    __syncthreads();
    for (int sidx = 0; sidx < a.n_steps; ++sidx) {
      const int buf = sidx & 1;
      const Step st = a.steps[sidx];
      const bool more = sidx + 1 < a.n_steps;
      uint4 pv[PV];
      if (more) {
        const Step nx = a.steps[sidx + 1];
#pragma unroll
        for (int v = 0; v < PV; ++v) pv[v] = plane_src(nx, tid + NTHR * v);
        load_codes(nx, cwn);
      }
#pragma unroll
      for (int h = 0; h < HS; ++h) {
        if (h < st.halves) {                          // uniform
          // plane fragments of k-step s + 1 are read while k-step s multiplies
          i32x4 fbh = __builtin_bit_cast(i32x4, sP[buf][0][h * KSTEP][lane]);
          i32x4 fbl = __builtin_bit_cast(i32x4, sP[buf][1][h * KSTEP][lane]);
#pragma unroll
          for (int s = 0; s < KSTEP; ++s) {
            const i32x4 bh = fbh, bl = fbl;
            if (s + 1 < KSTEP) {
              fbh = __builtin_bit_cast(i32x4, sP[buf][0][h * KSTEP + s + 1][lane]);
              fbl = __builtin_bit_cast(i32x4, sP[buf][1][h * KSTEP + s + 1][lane]);
            }
            const int d0 = 4 * (s & 1);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
              const uint4& c = cw[rt][h];
              const uint32_t w = (s >> 1) == 0 ? c.x : (s >> 1) == 1 ? c.y : (s >> 1) == 2 ? c.z : c.w;
              i32x4 av;
              av[0] = (int)((w >> (d0 + 0)) & M1);
              av[1] = (int)((w >> (d0 + 1)) & M1);
              av[2] = (int)((w >> (d0 + 2)) & M1);
              av[3] = (int)((w >> (d0 + 3)) & M1);
              acc_h[rt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bh, acc_h[rt], 0, 0, 0);
              acc_l[rt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bl, acc_l[rt], 0, 0, 0);
              // expand the next operand while these two multiply
              __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);   // VALU
              __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // MFMA
            }
          }
        }
      }
      if (MULTI && st.last) fold(st.u);
      if (more) {
#pragma unroll
        for (int v = 0; v < PV; ++v) plane_dst(buf ^ 1, tid + NTHR * v, pv[v]);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int h = 0; h < HS; ++h) cw[rt][h] = cwn[rt][h];
      }
      __syncthreads();
    }
    if (!MULTI) fold(0);

    // candidates of this block; a full list is pruned and the entries that
    // did not fit are offered again (the loop condition is uniform)
    uint32_t pend = 0;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = row0 + rt * 16 + 4 * g + r;
        if (row < a.N && q_ok) {
          if (a.full) a.full[q * a.N + row] = (float)sc[rt][r];
          pend |= 1u << (4 * rt + r);
        }
      }
    for (;;) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t bit = 1u << (4 * rt + r);
          if (pend & bit) {
            const uint64_t key = order_key(sc[rt][r]);
            if (key < cd.thr[n]) {
              pend &= ~bit;
            } else {
              const int pos = atomicAdd(&cd.cnt[n], 1);
              if (pos < CAP) {
                cd.key[n][pos] = key;
                cd.idx[n][pos] = (uint32_t)(row0 + rt * 16 + 4 * g + r);
                pend &= ~bit;
              } else {
                cd.overflow = 1;
              }
            }
          }
        }
      __syncthreads();
      const int ov = cd.overflow;
      __syncthreads();
      if (!ov) break;
      for (int qq = 0; qq < QB; ++qq)
        if (cd.cnt[qq] >= CAP) prune<CAP, NTHR>(cd, qq, a.topk);
      if (tid == 0) cd.overflow = 0;
      __syncthreads();
    }
  }
  for (int qq = 0; qq < QB; ++qq) prune<CAP, NTHR>(cd, qq, a.topk);
  for (int i = tid; i < QB * a.topk; i += NTHR) {
    const int qq = i / a.topk, e = i % a.topk;
    const int64_t o = ((int64_t)blockIdx.x * QB + qq) * a.topk + e;
    const bool have = e < cd.cnt[qq];
    a.ckey[o] = have ? cd.key[qq][e] : 0ull;
    a.cidx[o] = have ? cd.idx[qq][e] : 0xFFFFFFFFu;
  }
}

// One workgroup per query of the group: reduce the per-workgroup lists.
__global__ __launch_bounds__(256, 1) void k_merge(const uint64_t* __restrict__ ckey,
                                                  const uint32_t* __restrict__ cidx, int G,
                                                  int64_t grp, int64_t Q, int topk,
                                                  int64_t* __restrict__ out_idx,
                                                  float* __restrict__ out_score) {
  __shared__ Cand<MCAP> cd;   // only list 0 is used
  const int n = blockIdx.x;
  const int64_t q = grp * QB + n;
  if (q >= Q) return;
  const int tid = threadIdx.x;
  if (tid == 0) {
    cd.cnt[0] = 0;
    cd.thr[0] = 0ull;
  }
  __syncthreads();
  const int64_t total = (int64_t)G * topk;
  for (int64_t base = 0; base < total; base += 256) {
    const int64_t e = base + tid;
    if (e < total) {
      const int64_t wg = e / topk, j = e % topk;
      const int64_t o = (wg * QB + n) * topk + j;
      const uint64_t key = ckey[o];
      const uint32_t id = cidx[o];
      if (id != 0xFFFFFFFFu && key >= cd.thr[0]) {
        const int pos = atomicAdd(&cd.cnt[0], 1);
        cd.key[0][pos] = key;
        cd.idx[0][pos] = id;
      }
    }
    __syncthreads();
    if (cd.cnt[0] > MCAP - 256) prune<MCAP, 256>(cd, 0, topk);
  }
  prune<MCAP, 256>(cd, 0, topk);
  for (int e = tid; e < topk; e += 256) {
    const bool have = e < cd.cnt[0];
    out_idx[q * topk + e] = have ? (int64_t)cd.idx[0][e] : -1;
    out_score[q * topk + e] = have ? (float)key_value(cd.key[0][e]) : -__builtin_inff();
  }
}

// Pass configuration: candidate slots per query (256 when that leaves room
// for at least 128 new entries after a prune, else 512), 512-bit halves per
// step (two when the LDS holds both), 16-row tiles per wave and whether
// several modules are summed. One workgroup per CU either way (LDS).
struct PassCfg {
  int cap, hs, rt;
  bool multi;
};
inline PassCfg pass_cfg(int32_t U, int32_t topk) {
  PassCfg c;
  c.cap = topk <= 128 ? 256 : 512;
  c.hs = c.cap == 256 ? 2 : 1;
  c.rt = (c.hs == 1 && U == 1) ? 8 : 4;
  c.multi = U > 1;
  return c;
}

struct Layout {
  int64_t KS = 0;        // k-steps per query group over all modules
  int64_t n_steps = 0;   // 512-bit steps over all modules
  int64_t n_groups = 0;
  int64_t grid = 0;      // workgroups of the scoring pass
  size_t o_mods = 0, o_steps = 0, o_fq = 0, o_ys = 0, o_ph = 0, o_pl = 0, o_ck = 0, o_ci = 0,
         total = 0;
};

Layout layout(int64_t N, int64_t Q, int32_t U, const int64_t* kmod, int32_t topk) {
  Layout L;
  const PassCfg c = pass_cfg(U, topk);
  for (int u = 0; u < U; ++u) {
    const int64_t nms = (kmod[u] + 511) / 512;
    L.KS += KSTEP * nms;
    L.n_steps += (nms + c.hs - 1) / c.hs;
  }
  L.n_groups = (Q + QB - 1) / QB;
  const int64_t rows = (int64_t)NW * c.rt * 16;
  const int64_t n_blocks = (N + rows - 1) / rows;
  L.grid = std::max<int64_t>(1, std::min<int64_t>(n_blocks, kCus));
  size_t b = 0;
  auto add = [&](size_t x) { size_t o = b; b = align256(b + x); return o; };
  L.o_mods = add(sizeof(ModInfo) * U);
  L.o_steps = add(sizeof(Step) * L.n_steps);
  L.o_fq = add(4 * Q * U);
  L.o_ys = add(4 * Q * U);
  L.o_ph = add((size_t)L.n_groups * L.KS * 1024);
  L.o_pl = add((size_t)L.n_groups * L.KS * 1024);
  L.o_ck = add((size_t)L.grid * QB * topk * 8);
  L.o_ci = add((size_t)L.grid * QB * topk * 4);
  L.total = b;
  return L;
}

}  // namespace

int32_t score_max_topk() { return MAX_TOPK; }

size_t score_ws(int64_t N, int64_t Q, int32_t U, const int64_t* kmod, int32_t topk) {
  return layout(N, Q, U, kmod, topk).total;
}

eogp_status score_topk(const uint8_t* codes, int64_t cstride, const uint16_t* scales, int64_t N,
                       int32_t U, const int64_t* kmod, const float* Y, int64_t ldy, int64_t Q,
                       int32_t topk, int64_t* out_idx, float* out_score, float* full, void* ws,
                       size_t ws_bytes, hipStream_t s) {
  const Layout L = layout(N, Q, U, kmod, topk);
  if (ws_bytes < L.total) return fail(EOGP_ERR_WORKSPACE, "score_topk: workspace too small");
  if (Q == 0) return EOGP_OK;
  char* base = static_cast<char*>(ws);
  ModInfo* mods = reinterpret_cast<ModInfo*>(base + L.o_mods);
  int32_t* fq = reinterpret_cast<int32_t*>(base + L.o_fq);
  int32_t* ys = reinterpret_cast<int32_t*>(base + L.o_ys);
  int8_t* ph = reinterpret_cast<int8_t*>(base + L.o_ph);
  int8_t* pl = reinterpret_cast<int8_t*>(base + L.o_pl);
  uint64_t* ck = reinterpret_cast<uint64_t*>(base + L.o_ck);
  uint32_t* ci = reinterpret_cast<uint32_t*>(base + L.o_ci);

  Step* steps = reinterpret_cast<Step*>(base + L.o_steps);
  const PassCfg cfg = pass_cfg(U, topk);
  std::vector<ModInfo> hm(U);
  std::vector<Step> hs;
  hs.reserve(L.n_steps);
  int64_t coff = 0, boff = 0, ks = 0;
  for (int u = 0; u < U; ++u) {
    hm[u].k = (int32_t)kmod[u];
    hm[u].coff = (int32_t)coff;
    hm[u].boff = (int32_t)boff;
    hm[u].ksbase = (int32_t)ks;
    const int64_t nms = (kmod[u] + 511) / 512, mbytes = kmod[u] / 8;
    for (int64_t ms = 0; ms < nms; ms += cfg.hs) {
      Step st{};
      st.u = u;
      st.boff = (int32_t)(boff + 64 * ms);
      st.kbase = (int32_t)(ks + KSTEP * ms);
      st.bytes = (int32_t)std::min<int64_t>(64 * cfg.hs, mbytes - 64 * ms);
      st.halves = (int32_t)std::min<int64_t>(cfg.hs, nms - ms);
      st.last = ms + cfg.hs >= nms;
      hs.push_back(st);
    }
    coff += kmod[u];
    boff += kmod[u] / 8;
    ks += KSTEP * nms;
  }
  // the tables are small; copy them synchronously so the host vectors may go
  EOGP_HIP(hipMemcpyAsync(mods, hm.data(), sizeof(ModInfo) * U, hipMemcpyHostToDevice, s));
  EOGP_HIP(hipMemcpyAsync(steps, hs.data(), sizeof(Step) * hs.size(), hipMemcpyHostToDevice, s));
  EOGP_HIP(hipStreamSynchronize(s));
  timing::Scope tprep(EOGP_KT_SCORE_PREP, s);
  hipLaunchKernelGGL(k_query_stats, dim3((unsigned)Q, (unsigned)U), dim3(256), 0, s, Y, ldy, U,
                     mods, fq, ys);
  const int64_t pbytes = L.n_groups * L.KS * 1024;
  hipLaunchKernelGGL(k_query_planes, dim3((unsigned)ceil_div(pbytes, 256)), dim3(256), 0, s, Y,
                     ldy, Q, U, mods, fq, L.KS, L.n_groups, ph, pl);
  EOGP_LAUNCH_CHECK("query preparation");
  timing::end(tprep.slot, s);
  tprep.slot = -1;
  for (int64_t grp = 0; grp < L.n_groups; ++grp) {
    ScoreArgs a;
    a.codes = codes;
    a.cstride = cstride;
    a.scales = scales;
    a.N = N;
    a.U = U;
    a.mods = mods;
    a.ph = ph;
    a.pl = pl;
    a.steps = steps;
    a.n_steps = (int)L.n_steps;
    a.KS = L.KS;
    a.grp = grp;
    a.fq = fq;
    a.ysum = ys;
    a.Q = Q;
    a.topk = topk;
    a.full = full;
    a.ckey = ck;
    a.cidx = ci;
    {
      timing::Scope tp(EOGP_KT_SCORE_PASS, s);
      const dim3 gd((unsigned)L.grid), bd(NTHR);
      if (cfg.cap == 256) {
        if (cfg.multi) hipLaunchKernelGGL((k_score<256, 4, true, 2>), gd, bd, 0, s, a);
        else hipLaunchKernelGGL((k_score<256, 4, false, 2>), gd, bd, 0, s, a);
      } else {
        if (cfg.multi) hipLaunchKernelGGL((k_score<512, 4, true, 1>), gd, bd, 0, s, a);
        else hipLaunchKernelGGL((k_score<512, 8, false, 1>), gd, bd, 0, s, a);
      }
    }
    timing::Scope tm(EOGP_KT_SCORE_MERGE, s);
    hipLaunchKernelGGL(k_merge, dim3(QB), dim3(256), 0, s, ck, ci, (int)L.grid, grp, Q, topk,
                       out_idx, out_score);
    EOGP_LAUNCH_CHECK("score pass");
  }
  return EOGP_OK;
}

}  // namespace eogp
