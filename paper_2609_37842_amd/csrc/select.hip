// Plan builder: exact top-m selection of corrected eigenvalues, canonical
// ordering, half-whitening weights, and the gathered eigenvector panels.
//
// Selection follows the first stage of Section 3.2 (eq. sigma_ekfac: the m
// largest corrected eigenvalues give the top-m axes of Sigma_proxy) and
// Algorithm 1's fitting block. The order of the retained axes is
// (Lambda descending, flat index j*d_in + k ascending). Everything runs on the
// device: a 4-pass radix select finds the m-th largest 32-bit key, an ordered
// compaction keeps all larger keys and the first ties in index order, and a
// rank count over the m survivors puts them in canonical order.
#include <algorithm>
#include <numeric>
#include <vector>

#include "plan.h"
#include "scan.h"

namespace eogp {
namespace {

constexpr int kSelBlock = 4096;   // elements per block of the ordered compaction

__device__ __forceinline__ uint32_t key32(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;   // -0.0 and +0.0 are the same eigenvalue
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// Larger key64 <=> earlier in canonical order (Lambda desc, index asc).
__device__ __forceinline__ uint64_t key64(float x, uint32_t f) {
  return ((uint64_t)key32(x) << 32) | (uint64_t)(0xFFFFFFFFu - f);
}

struct SelState {
  uint32_t prefix;
  uint32_t pad0;
  long long remaining;
  unsigned long long nan_count;
  int bad_weight;
  int n_rows;
  int n_cols;
  int pad1;
};

__global__ void k_sel_init(SelState* st, long long m) {
  st->prefix = 0;
  st->remaining = m;
  st->nan_count = 0;
  st->bad_weight = 0;
  st->n_rows = 0;
  st->n_cols = 0;
}

__global__ __launch_bounds__(256) void k_hist(const float* __restrict__ lam, int64_t n,
                                              int pass, SelState* st,
                                              unsigned* __restrict__ hist) {
  __shared__ unsigned h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t prefix = st->prefix;
  const int dshift = 24 - 8 * pass;
  unsigned long long nan_local = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256) {
    float x = lam[i];
    if (pass == 0 && x != x) nan_local++;
    uint32_t k = key32(x);
    bool match = (pass == 0) || ((k >> (dshift + 8)) == prefix);
    if (match) atomicAdd(&h[(k >> dshift) & 255u], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&hist[threadIdx.x], h[threadIdx.x]);
  if (pass == 0 && nan_local) atomicAdd(&st->nan_count, nan_local);
}

// Choose the digit holding the remaining-th largest key; narrow the prefix.
__global__ __launch_bounds__(256) void k_pick(SelState* st, unsigned* hist) {
  if (threadIdx.x == 0) {
    long long rem = st->remaining;
    long long cum = 0;
    int d = 255;
    for (; d > 0; --d) {
      if (cum + (long long)hist[d] >= rem) break;
      cum += hist[d];
    }
    st->prefix = (st->prefix << 8) | (uint32_t)d;
    st->remaining = rem - cum;
  }
  __syncthreads();
  hist[threadIdx.x] = 0;
}

__device__ __forceinline__ int block_sum256(int v, int* scratch) {
  // wave reduction then 4-way LDS reduction
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0) scratch[threadIdx.x >> 6] = v;
  __syncthreads();
  int t = scratch[0] + scratch[1] + scratch[2] + scratch[3];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(256) void k_sel_count(const float* __restrict__ lam, int64_t n,
                                                   const SelState* st, long long* cgt,
                                                   long long* ceq) {
  __shared__ int red[4];
  const uint32_t v = st->prefix;
  const int64_t b0 = (int64_t)blockIdx.x * kSelBlock;
  int gt = 0, eq = 0;
  for (int r = 0; r < kSelBlock / 256; ++r) {
    int64_t i = b0 + r * 256 + threadIdx.x;
    if (i < n) {
      uint32_t k = key32(lam[i]);
      gt += (k > v);
      eq += (k == v);
    }
  }
  int G = block_sum256(gt, red);
  int E = block_sum256(eq, red);
  if (threadIdx.x == 0) {
    cgt[blockIdx.x] = G;
    ceq[blockIdx.x] = E;
  }
}

__global__ __launch_bounds__(256) void k_sel_write(const float* __restrict__ lam, int64_t n,
                                                   const SelState* st, const long long* ogt,
                                                   const long long* oeq, long long m,
                                                   int32_t* __restrict__ sel) {
  __shared__ int wg[4], we[4];
  const uint32_t v = st->prefix;
  const long long need_eq = st->remaining;
  const long long count_gt = m - need_eq;
  long long base_gt = ogt[blockIdx.x];
  long long base_eq = oeq[blockIdx.x];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t b0 = (int64_t)blockIdx.x * kSelBlock;
  for (int r = 0; r < kSelBlock / 256; ++r) {
    int64_t i = b0 + r * 256 + threadIdx.x;
    uint32_t k = (i < n) ? key32(lam[i]) : 0u;
    bool isgt = (i < n) && (k > v);
    bool iseq = (i < n) && (k == v);
    uint64_t mg, me;
    int pg = wave_prefix_count(isgt, &mg);
    int pe = wave_prefix_count(iseq, &me);
    if (lane == 0) {
      wg[wid] = __popcll(mg);
      we[wid] = __popcll(me);
    }
    __syncthreads();
    int og = 0, oe = 0, tg = 0, te = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wid) { og += wg[w]; oe += we[w]; }
      tg += wg[w];
      te += we[w];
    }
    if (isgt) sel[base_gt + og + pg] = (int32_t)i;
    if (iseq) {
      long long e = base_eq + oe + pe;
      if (e < need_eq) sel[count_gt + e] = (int32_t)i;
    }
    base_gt += tg;
    base_eq += te;
    __syncthreads();
  }
}

__global__ void k_make_keys(const float* __restrict__ lam, const int32_t* sel, int64_t m,
                            uint64_t* keys) {
  int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x < m) {
    int32_t f = sel[x];
    keys[x] = key64(lam[f], (uint32_t)f);
  }
}

// rank(x) = #{y : key[y] > key[x]} (keys are distinct), counted in chunks of
// kRankChunk keys: workgroup (bx, by) adds the count over chunks by,
// by + gridDim.y, ... to rank[x] for its 256 keys x (rank zeroed beforehand).
constexpr int kRankChunk = 512;
__global__ __launch_bounds__(256) void k_rank(const uint64_t* __restrict__ keys, int64_t m,
                                              int* __restrict__ rank) {
  __shared__ uint64_t sk[kRankChunk];
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const uint64_t K = (x < m) ? keys[x] : ~0ull;
  int c = 0;
  for (int64_t base = (int64_t)blockIdx.y * kRankChunk; base < m; base += (int64_t)gridDim.y * kRankChunk) {
    __syncthreads();   // the previous chunk's readers are done
    for (int j = threadIdx.x; j < kRankChunk; j += 256) sk[j] = (base + j < m) ? keys[base + j] : 0ull;
    __syncthreads();
    const int cnt = (int)std::min<int64_t>(m - base, kRankChunk);
    for (int j = 0; j < cnt; ++j) c += (sk[j] > K);
  }
  if (x < m && c) atomicAdd(&rank[x], c);
}
// ret[rank(x)] = sel[x]
__global__ void k_rank_place(const int* __restrict__ rank, const int32_t* __restrict__ sel,
                             int64_t m, int32_t* __restrict__ ret) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x < m) ret[rank[x]] = sel[x];
}

__global__ void k_finalize(const float* __restrict__ lam, const int32_t* __restrict__ ret,
                           int64_t m, int64_t d_in, double damping, float* __restrict__ w,
                           int* cnt_j, int* cnt_k, SelState* st) {
  int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= m) return;
  int32_t f = ret[r];
  int64_t j = f / d_in, k = f % d_in;
  double L = (double)lam[f] + damping;
  bool ok = (L > 0.0) && (L < __builtin_inf());
  if (!ok) atomicOr(&st->bad_weight, 1);
  // eq. first_stage: (Lambda_r + lambda)^-1/2, in fp64 then rounded once.
  w[r] = ok ? (float)(1.0 / sqrt(L)) : 0.0f;
  atomicAdd(&cnt_j[j], 1);
  atomicAdd(&cnt_k[k], 1);
}

// Order the used rows (or columns) by (retained count desc, index asc): rows
// holding many retained axes come first, which packs the retained set into
// few 32 x 32 blocks (a staircase when Lambda is close to a product). Ranks
// are counted in chunks as in k_rank (rank zeroed beforehand), then placed.
__global__ __launch_bounds__(256) void k_rank_lines(const int* __restrict__ cnt, int64_t d,
                                                    int* __restrict__ rank) {
  __shared__ int sc[kRankChunk];
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int c = (x < d) ? cnt[x] : 0;
  int r = 0;
  for (int64_t base = (int64_t)blockIdx.y * kRankChunk; base < d; base += (int64_t)gridDim.y * kRankChunk) {
    __syncthreads();   // the previous chunk's readers are done
    for (int j = threadIdx.x; j < kRankChunk; j += 256) sc[j] = (base + j < d) ? cnt[base + j] : 0;
    __syncthreads();
    const int lim = (int)std::min<int64_t>(d - base, kRankChunk);
    for (int j = 0; j < lim; ++j) {
      const int cj = sc[j];
      const int64_t xj = base + j;
      r += (cj > 0) && (cj > c || (cj == c && xj < x));
    }
  }
  if (x < d && c > 0 && r) atomicAdd(&rank[x], r);
}
__global__ void k_place_lines(const int* __restrict__ cnt, const int* __restrict__ rank, int64_t d,
                              int* __restrict__ pos, int* __restrict__ list, int* n_used) {
  const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (x >= d) return;
  if (cnt[x] > 0) {
    pos[x] = rank[x];
    list[rank[x]] = (int)x;
    atomicAdd(n_used, 1);
  } else {
    pos[x] = -1;
  }
}

__global__ void k_tile_count(const int32_t* __restrict__ ret, int64_t m, int64_t d_in,
                             const int* __restrict__ jpos, const int* __restrict__ kpos,
                             int n_kt, int* tcount, int* rtile) {
  int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= m) return;
  int32_t f = ret[r];
  int jp = jpos[f / d_in], kp = kpos[f % d_in];
  int tile = (jp >> 5) * n_kt + (kp >> 5);
  rtile[r] = tile;
  atomicAdd(&tcount[tile], 1);
}

__global__ void k_tile_prep(const int* tcount, int64_t nt, long long* toff, long long* flag) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t < nt) {
    toff[t] = tcount[t];
    flag[t] = tcount[t] > 0;
  }
}

__global__ void k_tile_place(const int32_t* __restrict__ ret, int64_t m, int64_t d_in,
                             const int* __restrict__ jpos, const int* __restrict__ kpos,
                             const int* __restrict__ rtile, const long long* toff, int* cursor,
                             int32_t* ent_r, uint16_t* ent_loc, int32_t* ent_pos) {
  int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= m) return;
  int32_t f = ret[r];
  int jp = jpos[f / d_in], kp = kpos[f % d_in];
  int tile = rtile[r];
  long long p = toff[tile] + atomicAdd(&cursor[tile], 1);
  ent_r[p] = (int32_t)r;
  ent_loc[p] = (uint16_t)(((jp & 31) << 5) | (kp & 31));
  ent_pos[r] = (int32_t)p;
}

__global__ void k_tile_desc(const int* tcount, int64_t nt, int n_kt, const long long* toff,
                            const long long* aoff, int32_t* tiles) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= nt || tcount[t] == 0) return;
  long long a = aoff[t];
  tiles[4 * a + 0] = (int32_t)(t / n_kt);
  tiles[4 * a + 1] = (int32_t)(t % n_kt);
  tiles[4 * a + 2] = (int32_t)toff[t];
  tiles[4 * a + 3] = (int32_t)(toff[t] + tcount[t]);
}

// panel[p][c] = Q[c][list[p]] (eigenvector list[p] stored contiguously),
// split into bf16 high and low parts, and rounded once to fp16; rows >= n_used
// and columns >= d are 0.
__global__ __launch_bounds__(256) void k_gather_panel(const float* __restrict__ Q, int64_t d,
                                                      const int* __restrict__ list, int n_used,
                                                      int64_t rows_pad, int64_t ld,
                                                      uint16_t* __restrict__ hi,
                                                      uint16_t* __restrict__ lo,
                                                      uint16_t* __restrict__ h16) {
  __shared__ float t[32][33];
  const int64_t p0 = (int64_t)blockIdx.x * 32, c0 = (int64_t)blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int cc = ty; cc < 32; cc += 8) {
    int64_t c = c0 + cc, p = p0 + tx;
    float v = 0.f;
    if (p < n_used && c < d) v = Q[c * d + list[p]];
    t[cc][tx] = v;
  }
  __syncthreads();
  for (int pp = ty; pp < 32; pp += 8) {
    int64_t p = p0 + pp, c = c0 + tx;
    if (p < rows_pad && c < ld) {
      float v = t[tx][pp];
      uint16_t h = to_bf16_bits(v);
      hi[p * ld + c] = h;
      lo[p * ld + c] = to_bf16_bits(v - bf16_bits_to_f32(h));
      h16[p * ld + c] = to_f16_bits(v);
    }
  }
}

inline unsigned grid_for(int64_t n, int per) {
  return (unsigned)((n + per - 1) / per);
}

}  // namespace

namespace {
__global__ void k_iota(int* __restrict__ v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) v[i] = (int)i;
}
}  // namespace

void basis_panels(const float* Q, int64_t d, int64_t rows_pad, int64_t ld, int* list,
                  uint16_t* hi, uint16_t* lo, uint16_t* h16, hipStream_t s) {
  hipLaunchKernelGGL(k_iota, dim3(grid_for(d, 256)), dim3(256), 0, s, list, d);
  hipLaunchKernelGGL(k_gather_panel, dim3((unsigned)(rows_pad / 32), grid_for(ld, 32)), dim3(256),
                     0, s, Q, d, list, (int)d, rows_pad, ld, hi, lo, h16);
}

void free_plan(eogp_plan* p) {
  if (!p) return;
  if (p->mem) (void)hipFree(p->mem);
  delete p;
}

eogp_status build_plan(const float* eigvals, int64_t d_out, int64_t d_in, double damping,
                       int64_t m, const float* Q_A, const float* Q_S, hipStream_t s,
                       eogp_plan** out) {
  const int64_t n = d_out * d_in;
  const int64_t nb = ceil_div(n, kSelBlock);
  const int n_jt = (int)ceil_div(d_out, kBlk), n_kt = (int)ceil_div(d_in, kBlk);
  const int64_t nt = (int64_t)n_jt * n_kt;

  // ---- temporaries ---------------------------------------------------------
  size_t tbytes = 0;
  auto add = [&](size_t b) { size_t o = tbytes; tbytes = align256(tbytes + b); return o; };
  size_t o_st = add(sizeof(SelState)), o_hist = add(256 * 4);
  size_t o_cgt = add((nb + 1) * 8), o_ceq = add((nb + 1) * 8);
  size_t o_sel = add(m * 4), o_keys = add(m * 8);
  size_t o_cj = add(d_out * 4), o_ck = add(d_in * 4);
  size_t o_jpos = add(d_out * 4), o_kpos = add(d_in * 4);
  size_t o_jl = add(d_out * 4), o_kl = add(d_in * 4);
  size_t o_tc = add(nt * 4), o_rt = add(m * 4);
  size_t o_rk = add(m * 4), o_rj = add(d_out * 4), o_rkk = add(d_in * 4);   // rank counters
  size_t o_toff = add((nt + 1) * 8), o_flag = add((nt + 1) * 8), o_cur = add(nt * 4);
  size_t o_ret = add(m * 4), o_w = add(m * 4);
  char* tmp = nullptr;
  EOGP_HIP(hipMalloc(&tmp, tbytes));
  struct Guard { char* p; ~Guard() { if (p) (void)hipFree(p); } } guard{tmp};
  SelState* st = (SelState*)(tmp + o_st);
  unsigned* hist = (unsigned*)(tmp + o_hist);
  long long *cgt = (long long*)(tmp + o_cgt), *ceq = (long long*)(tmp + o_ceq);
  int32_t* sel = (int32_t*)(tmp + o_sel);
  uint64_t* keys = (uint64_t*)(tmp + o_keys);
  int *cj = (int*)(tmp + o_cj), *ck = (int*)(tmp + o_ck);
  int *jpos = (int*)(tmp + o_jpos), *kpos = (int*)(tmp + o_kpos);
  int *jl = (int*)(tmp + o_jl), *kl = (int*)(tmp + o_kl);
  int *tc = (int*)(tmp + o_tc), *rt = (int*)(tmp + o_rt), *cur = (int*)(tmp + o_cur);
  int *rk = (int*)(tmp + o_rk), *rj = (int*)(tmp + o_rj), *rkk = (int*)(tmp + o_rkk);
  long long *toff = (long long*)(tmp + o_toff), *flag = (long long*)(tmp + o_flag);
  int32_t* ret = (int32_t*)(tmp + o_ret);
  float* w = (float*)(tmp + o_w);
  EOGP_HIP(hipMemsetAsync(tmp, 0, tbytes, s));

  // ---- radix select of the m-th largest key ----------------------------------
  hipLaunchKernelGGL(k_sel_init, dim3(1), dim3(1), 0, s, st, (long long)m);
  const unsigned hgrid = (unsigned)std::min<int64_t>(grid_for(n, 256), 4096);
  for (int pass = 0; pass < 4; ++pass) {
    hipLaunchKernelGGL(k_hist, dim3(hgrid), dim3(256), 0, s, eigvals, n, pass, st, hist);
    hipLaunchKernelGGL(k_pick, dim3(1), dim3(256), 0, s, st, hist);
  }
  EOGP_LAUNCH_CHECK("selection histogram");
  hipLaunchKernelGGL(k_sel_count, dim3((unsigned)nb), dim3(256), 0, s, eigvals, n, st, cgt, ceq);
  EOGP_HIP(scan_exclusive(cgt, nb, s));
  EOGP_HIP(scan_exclusive(ceq, nb, s));
  hipLaunchKernelGGL(k_sel_write, dim3((unsigned)nb), dim3(256), 0, s, eigvals, n, st, cgt, ceq,
                     (long long)m, sel);
  hipLaunchKernelGGL(k_make_keys, dim3(grid_for(m, 256)), dim3(256), 0, s, eigvals, sel, m, keys);
  hipLaunchKernelGGL(k_rank, dim3(grid_for(m, 256), std::min(grid_for(m, kRankChunk), 65535u)), dim3(256), 0, s, keys,
                     m, rk);
  hipLaunchKernelGGL(k_rank_place, dim3(grid_for(m, 256)), dim3(256), 0, s, rk, sel, m, ret);
  hipLaunchKernelGGL(k_finalize, dim3(grid_for(m, 256)), dim3(256), 0, s, eigvals, ret, m, d_in,
                     damping, w, cj, ck, st);
  hipLaunchKernelGGL(k_rank_lines, dim3(grid_for(d_out, 256), std::min(grid_for(d_out, kRankChunk), 65535u)), dim3(256),
                     0, s, cj, d_out, rj);
  hipLaunchKernelGGL(k_rank_lines, dim3(grid_for(d_in, 256), std::min(grid_for(d_in, kRankChunk), 65535u)), dim3(256),
                     0, s, ck, d_in, rkk);
  hipLaunchKernelGGL(k_place_lines, dim3(grid_for(d_out, 256)), dim3(256), 0, s, cj, rj, d_out, jpos,
                     jl, &st->n_rows);
  hipLaunchKernelGGL(k_place_lines, dim3(grid_for(d_in, 256)), dim3(256), 0, s, ck, rkk, d_in, kpos,
                     kl, &st->n_cols);
  hipLaunchKernelGGL(k_tile_count, dim3(grid_for(m, 256)), dim3(256), 0, s, ret, m, d_in, jpos,
                     kpos, n_kt, tc, rt);
  hipLaunchKernelGGL(k_tile_prep, dim3(grid_for(nt, 256)), dim3(256), 0, s, tc, nt, toff, flag);
  EOGP_HIP(scan_exclusive(toff, nt, s));
  EOGP_HIP(scan_exclusive(flag, nt, s));
  EOGP_LAUNCH_CHECK("selection");

  SelState hst;
  long long n_active = 0;
  EOGP_HIP(hipMemcpyAsync(&hst, st, sizeof(hst), hipMemcpyDeviceToHost, s));
  EOGP_HIP(hipMemcpyAsync(&n_active, flag + nt, sizeof(long long), hipMemcpyDeviceToHost, s));
  EOGP_HIP(hipStreamSynchronize(s));
  if (hst.nan_count)
    return fail(EOGP_ERR_INVALID, "eigvals contains NaN");
  if (hst.bad_weight)
    return fail(EOGP_ERR_INVALID, "a retained Lambda + damping is not positive and finite");

  // ---- the plan's own memory ---------------------------------------------------
  eogp_plan* p = new eogp_plan();
  p->d_out = d_out;
  p->d_in = d_in;
  p->m = m;
  p->damping = damping;
  p->n_rows = hst.n_rows;
  p->n_cols = hst.n_cols;
  p->rows_pad = round_up(std::max<int64_t>(p->n_rows, 1), kPanelTile);
  p->cols_pad = round_up(std::max<int64_t>(p->n_cols, 1), kPanelTile);
  p->ld_out = round_up(d_out, 32);
  p->ld_in = round_up(d_in, 32);
  p->n_tiles = n_active;
  (void)hipGetDevice(&p->device);
  size_t pb = 0;
  auto padd = [&](size_t b) { size_t o = pb; pb = align256(pb + b); return o; };
  size_t q_ret = padd(m * 4), q_w = padd(m * 4), q_tiles = padd(std::max<int64_t>(n_active, 1) * 16);
  size_t q_groups = padd(std::max<int64_t>(n_active, 1) * 16), q_gt = padd(std::max<int64_t>(n_active, 1) * 4);
  size_t q_er = padd(m * 4), q_el = padd(m * 2), q_ep = padd(m * 4);
  size_t q_sh = padd(p->rows_pad * p->ld_out * 2), q_sl = padd(p->rows_pad * p->ld_out * 2);
  size_t q_ah = padd(p->cols_pad * p->ld_in * 2), q_al = padd(p->cols_pad * p->ld_in * 2);
  size_t q_s16 = padd(p->rows_pad * p->ld_out * 2), q_a16 = padd(p->cols_pad * p->ld_in * 2);
  hipError_t e = hipMalloc(&p->mem, pb);
  if (e != hipSuccess) {
    delete p;
    return check_hip(e, "hipMalloc(plan)");
  }
  char* base = (char*)p->mem;
  p->ret_flat = (int32_t*)(base + q_ret);
  p->ret_w = (float*)(base + q_w);
  p->tiles = (int32_t*)(base + q_tiles);
  p->groups = (int32_t*)(base + q_groups);
  p->gtiles = (int32_t*)(base + q_gt);
  p->ent_r = (int32_t*)(base + q_er);
  p->ent_loc = (uint16_t*)(base + q_el);
  p->ent_pos = (int32_t*)(base + q_ep);
  p->qs_hi = (uint16_t*)(base + q_sh);
  p->qs_lo = (uint16_t*)(base + q_sl);
  p->qa_hi = (uint16_t*)(base + q_ah);
  p->qa_lo = (uint16_t*)(base + q_al);
  p->qs_f16 = (uint16_t*)(base + q_s16);
  p->qa_f16 = (uint16_t*)(base + q_a16);

  if (hipMemcpyAsync(p->ret_flat, ret, m * 4, hipMemcpyDeviceToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->ret_w, w, m * 4, hipMemcpyDeviceToDevice, s) != hipSuccess) {
    free_plan(p);
    return fail(EOGP_ERR_DEVICE, "plan build: copy failed");
  }
  hipLaunchKernelGGL(k_tile_place, dim3(grid_for(m, 256)), dim3(256), 0, s, ret, m, d_in, jpos,
                     kpos, rt, toff, cur, p->ent_r, p->ent_loc, p->ent_pos);
  hipLaunchKernelGGL(k_tile_desc, dim3(grid_for(nt, 256)), dim3(256), 0, s, tc, nt, n_kt, toff,
                     flag, p->tiles);
  // Groups of active blocks that share one operand block, at most kRetGroup
  // each: the retained products load a group's shared block once. Blocks are
  // grouped by row block of S~ or by column block of A~, whichever loads fewer
  // blocks in all (a run of L blocks sharing one loads ceil(L / kRetGroup) + L).
  std::vector<int32_t> hgroups, hgt;
  if (n_active > 0) {
    std::vector<int32_t> ht((size_t)n_active * 4);
    e = hipMemcpyAsync(ht.data(), p->tiles, ht.size() * 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      free_plan(p);
      return check_hip(e, "plan build: active blocks");
    }
    std::vector<int32_t> by_row((size_t)n_active), by_col((size_t)n_active);
    std::iota(by_row.begin(), by_row.end(), 0);   // tiles are in (row, column) order
    by_col = by_row;
    std::stable_sort(by_col.begin(), by_col.end(),
                     [&](int32_t a, int32_t b) { return ht[4 * a + 1] < ht[4 * b + 1]; });
    auto loads = [&](const std::vector<int32_t>& ord, int axis) {
      int64_t total = 0;
      for (int64_t a = 0; a < n_active;) {
        int64_t b = a;
        while (b < n_active && ht[4 * ord[b] + axis] == ht[4 * ord[a] + axis]) ++b;
        total += ceil_div(b - a, (int64_t)kRetGroup) + (b - a);
        a = b;
      }
      return total;
    };
    p->group_rows = loads(by_row, 0) <= loads(by_col, 1);
    const int axis = p->group_rows ? 0 : 1;
    hgt = p->group_rows ? by_row : by_col;
    for (int64_t a = 0; a < n_active;) {
      int64_t b = a;
      while (b < n_active && b - a < kRetGroup && ht[4 * hgt[b] + axis] == ht[4 * hgt[a] + axis]) ++b;
      hgroups.insert(hgroups.end(), {(int32_t)a, (int32_t)(b - a), ht[4 * hgt[a] + axis], 0});
      a = b;
    }
    p->n_groups = (int64_t)hgroups.size() / 4;
    e = hipMemcpyAsync(p->groups, hgroups.data(), hgroups.size() * 4, hipMemcpyHostToDevice, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(p->gtiles, hgt.data(), hgt.size() * 4, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) {
      free_plan(p);
      return check_hip(e, "plan build: block groups");
    }
  }
  hipLaunchKernelGGL(k_gather_panel, dim3((unsigned)(p->rows_pad / 32), grid_for(p->ld_out, 32)),
                     dim3(256), 0, s, Q_S, d_out, jl, (int)p->n_rows, p->rows_pad, p->ld_out,
                     p->qs_hi, p->qs_lo, p->qs_f16);
  hipLaunchKernelGGL(k_gather_panel, dim3((unsigned)(p->cols_pad / 32), grid_for(p->ld_in, 32)),
                     dim3(256), 0, s, Q_A, d_in, kl, (int)p->n_cols, p->cols_pad, p->ld_in,
                     p->qa_hi, p->qa_lo, p->qa_f16);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    free_plan(p);
    return check_hip(e, "plan build");
  }
  *out = p;
  return EOGP_OK;
}

}  // namespace eogp
