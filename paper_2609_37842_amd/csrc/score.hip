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
// (the 16 columns of v_mfma_i32_16x16x64_i8). A 256-thread workgroup owns 256
// consecutive examples at a time (each wave 4 tiles of 16 rows). Per 512-bit
// step of a module, the workgroup stages the query planes (16 KB) in LDS once
// and every wave multiplies its 64 rows against them. Bits are expanded without
// reordering the stored layout: the 32-bit code word w yields the int8 operand
// dwords (w >> d) & 0x01010101 (bits d, d+8, d+16, d+24), and the query planes
// are laid out in that same permuted order when they are prepared.
// After the last module the workgroup's scores are filtered against a per-query
// threshold into an LDS candidate list (score desc, index asc), which is pruned
// to the top-k whenever it could overflow; finally each workgroup writes its
// top-k per query and a merge kernel reduces them.
#include <algorithm>
#include <vector>

#include "common.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int QB = 16;          // queries per pass
constexpr int RT = 4;           // 16-row tiles per wave
constexpr int NW = 4;           // waves per workgroup
constexpr int ROWS = NW * RT * 16;
constexpr int KSTEP = 8;        // MFMA k-steps (64 bits each) per 512-bit step
constexpr int CAP = 512;        // candidate slots per query (power of two)
constexpr int MAX_TOPK = CAP - ROWS;

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
struct Cand {
  uint64_t key[QB][CAP];
  uint32_t idx[QB][CAP];
  int cnt[QB];
  uint64_t thr[QB];
};

// Sort list n (all 256 threads), keep its first `topk`, update the threshold.
__device__ void prune(Cand& cd, int n, int topk) {
  const int tid = threadIdx.x;
  const int c = cd.cnt[n];
  for (int i = c + tid; i < CAP; i += 256) {
    cd.key[n][i] = 0ull;
    cd.idx[n][i] = 0xFFFFFFFFu;
  }
  __syncthreads();
  for (int k = 2; k <= CAP; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < CAP; i += 256) {
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

struct ScoreArgs {
  const uint8_t* codes;
  int64_t cstride;
  const uint16_t* scales;
  int64_t N;
  int U;
  const ModInfo* mods;
  const int8_t* ph;
  const int8_t* pl;
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

__global__ __launch_bounds__(256, 1) void k_score(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint4 sB[2][2][KSTEP][64];
  __shared__ Cand cd;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int n = lane & 15;           // query column of this lane
  const int g = lane >> 4;           // k-group of this lane
  const int64_t q = a.grp * QB + n;
  const bool q_ok = q < a.Q;
  if (tid < QB) {
    cd.cnt[tid] = 0;
    cd.thr[tid] = 0ull;
  }
  __syncthreads();
  const int64_t n_blocks = (a.N + ROWS - 1) / ROWS;
  const uint4* phv = reinterpret_cast<const uint4*>(a.ph);
  const uint4* plv = reinterpret_cast<const uint4*>(a.pl);
  const uint32_t M1 = 0x01010101u;

  for (int64_t blk = blockIdx.x; blk < n_blocks; blk += gridDim.x) {
    const int64_t row0 = blk * ROWS + (int64_t)wid * (RT * 16);
    double sc[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) sc[rt][r] = 0.0;

    for (int u = 0; u < a.U; ++u) {
      const ModInfo md = a.mods[u];
      const int nms = (md.k + 511) / 512;
      const int mbytes = md.k >> 3;
      i32x4 acc_h[RT], acc_l[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        acc_h[rt] = i32x4{0, 0, 0, 0};
        acc_l[rt] = i32x4{0, 0, 0, 0};
      }
      for (int ms = 0; ms < nms; ++ms) {
        const int buf = ms & 1;
        // stage this step's query planes: 2 planes x 8 k-steps x 64 lanes x 16 B
        const int64_t kbase = (a.grp * a.KS + md.ksbase + (int64_t)ms * KSTEP) * 64;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int f = tid * 4 + v;               // 0..1023
          const int plane = f >> 9, ks = (f >> 6) & 7, ln = f & 63;
          sB[buf][plane][ks][ln] = (plane ? plv : phv)[kbase + ks * 64 + ln];
        }
        // this lane's code words for each row tile (two 8-byte halves)
        uint32_t wds[RT][4];
        const int boff = 64 * ms + 16 * g;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const int64_t row = row0 + rt * 16 + n;
          const uint8_t* src = a.codes + row * a.cstride + md.boff + boff;
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            uint2 v2 = make_uint2(0u, 0u);
            if (row < a.N && boff + 8 * hf + 8 <= mbytes)
              v2 = *reinterpret_cast<const uint2*>(src + 8 * hf);
            wds[rt][2 * hf] = v2.x;
            wds[rt][2 * hf + 1] = v2.y;
          }
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < KSTEP; ++s) {
          const i32x4 bh = __builtin_bit_cast(i32x4, sB[buf][0][s][lane]);
          const i32x4 bl = __builtin_bit_cast(i32x4, sB[buf][1][s][lane]);
          const int d0 = 4 * (s & 1);
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            const uint32_t w = wds[rt][s >> 1];
            i32x4 av;
            av[0] = (int)((w >> (d0 + 0)) & M1);
            av[1] = (int)((w >> (d0 + 1)) & M1);
            av[2] = (int)((w >> (d0 + 2)) & M1);
            av[3] = (int)((w >> (d0 + 3)) & M1);
            acc_h[rt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bh, acc_h[rt], 0, 0, 0);
            acc_l[rt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bl, acc_l[rt], 0, 0, 0);
          }
        }
      }
      // module term: s * (2 n1 - sum y_int) * 2^-f, added in module order
      const int f = q_ok ? a.fq[q * a.U + u] : 0;
      const int ys = q_ok ? a.ysum[q * a.U + u] : 0;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = row0 + rt * 16 + 4 * g + r;
          const uint16_t s16 = row < a.N ? a.scales[row * a.U + u] : (uint16_t)0;
          const int n1 = 256 * acc_h[rt][r] + acc_l[rt][r];
          const int nn = 2 * n1 - ys;
          const double t = ldexp((double)f16_bits_to_f32(s16) * (double)nn, -f);
          sc[rt][r] += t;
        }
    }

    // candidates of this block
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = row0 + rt * 16 + 4 * g + r;
        if (row < a.N && q_ok) {
          if (a.full) a.full[q * a.N + row] = (float)sc[rt][r];
          const uint64_t key = order_key(sc[rt][r]);
          if (key >= cd.thr[n]) {
            const int pos = atomicAdd(&cd.cnt[n], 1);
            cd.key[n][pos] = key;
            cd.idx[n][pos] = (uint32_t)row;
          }
        }
      }
    __syncthreads();
    for (int qq = 0; qq < QB; ++qq)
      if (cd.cnt[qq] > CAP - ROWS) prune(cd, qq, a.topk);
  }
  for (int qq = 0; qq < QB; ++qq) prune(cd, qq, a.topk);
  for (int i = tid; i < QB * a.topk; i += 256) {
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
  __shared__ Cand cd;   // only list 0 is used
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
    if (cd.cnt[0] > CAP - 256) prune(cd, 0, topk);
  }
  prune(cd, 0, topk);
  for (int e = tid; e < topk; e += 256) {
    const bool have = e < cd.cnt[0];
    out_idx[q * topk + e] = have ? (int64_t)cd.idx[0][e] : -1;
    out_score[q * topk + e] = have ? (float)key_value(cd.key[0][e]) : -__builtin_inff();
  }
}

struct Layout {
  int64_t KS = 0;        // k-steps per query group over all modules
  int64_t n_groups = 0;
  int64_t grid = 0;      // workgroups of the scoring pass
  size_t o_mods = 0, o_fq = 0, o_ys = 0, o_ph = 0, o_pl = 0, o_ck = 0, o_ci = 0, total = 0;
};

Layout layout(int64_t N, int64_t Q, int32_t U, const int64_t* kmod, int32_t topk) {
  Layout L;
  for (int u = 0; u < U; ++u) L.KS += KSTEP * ((kmod[u] + 511) / 512);
  L.n_groups = (Q + QB - 1) / QB;
  const int64_t n_blocks = (N + ROWS - 1) / ROWS;
  L.grid = std::max<int64_t>(1, std::min<int64_t>(n_blocks, kCus));
  size_t b = 0;
  auto add = [&](size_t x) { size_t o = b; b = align256(b + x); return o; };
  L.o_mods = add(sizeof(ModInfo) * U);
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

  std::vector<ModInfo> hm(U);
  int64_t coff = 0, boff = 0, ks = 0;
  for (int u = 0; u < U; ++u) {
    hm[u].k = (int32_t)kmod[u];
    hm[u].coff = (int32_t)coff;
    hm[u].boff = (int32_t)boff;
    hm[u].ksbase = (int32_t)ks;
    coff += kmod[u];
    boff += kmod[u] / 8;
    ks += KSTEP * ((kmod[u] + 511) / 512);
  }
  EOGP_HIP(hipMemcpyAsync(mods, hm.data(), sizeof(ModInfo) * U, hipMemcpyHostToDevice, s));
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
      hipLaunchKernelGGL(k_score, dim3((unsigned)L.grid), dim3(256), 0, s, a);
    }
    timing::Scope tm(EOGP_KT_SCORE_MERGE, s);
    hipLaunchKernelGGL(k_merge, dim3(QB), dim3(256), 0, s, ck, ci, (int)L.grid, grp, Q, topk,
                       out_idx, out_score);
    EOGP_LAUNCH_CHECK("score pass");
  }
  return EOGP_OK;
}

}  // namespace eogp
