// Scoring stored one-bit codes against unquantized query projections
// (eq. onebit_influence, eq. app_stored_influence) with a per-query top-k.
//
// Arithmetic. Each query module vector y is taken in fixed point,
// y_int = rint(y 2^f) with f = 14 - e for max|y| = mu 2^e (|y_int| <= 2^14), and
// split into two int8 planes y_int = 256 h + l (h in [-64, 64], l in
// [-128, 127]). With b in {0, 1} the MFMAs compute n1 = sum_{b=1} y_int exactly
// in integers, and <y_int, 2b - 1> = 2 n1 - sum(y_int). Each module term
// s * (2 n1 - sum) * 2^-f is exact in fp64 and the terms are added in module
// order, so the score is reproducible bit for bit.
//
// Data flow. A pass streams every stored code once for a group of 16
// queries. v_mfma_i32_32x32x32_i8 takes the 32 plane rows (16 queries x
// {h, l}) as its A operand and 32 stored rows as B, so one instruction
// serves both planes and each lane ends with 8 queries of one stored row
// (the h and l sums of a query land in the same lane). A 512-thread
// workgroup (8 waves, 2 per SIMD) owns 512 consecutive rows at a time, each
// wave two tiles of 32 rows. The modules are walked in steps of 512 bits;
// per step each lane holds 32 bytes of its row (two 16-byte loads, requested
// D steps ahead in a register ring), the workgroup stages the step's plane
// fragments (16 KB) in LDS once, double-buffered, and every fragment read
// from LDS feeds both tiles.
//
// Bit expansion. The 16 bytes c of a lane feed 8 MFMAs, one per bit
// position t of a byte. The operand of MFMA t is (c >> s) & (0x01010101 <<
// w) with t = s + w, w = t mod NCLS: its bytes are 0 or 2^w, so the MFMA adds
// 2^w times the wanted sum into accumulator class w, and n1 = sum_w acc_w /
// 2^w (exact shifts: every term of acc_w is a multiple of 2^w). One shift
// serves NCLS masks, and one 64-bit shift serves two words, so with NCLS = 2
// expanding 16 bytes for their 8 MFMAs takes 32 ANDs and 6 shifts (a shift
// and an AND per word and MFMA would take 64). The query planes are prepared
// in exactly that order: byte j of lane (M, g) of MFMA (u, t) in step s of a
// module holds coordinate 8 (64 s + 32 g + 16 u + j) + t.
//
// After the last module the workgroup's scores are filtered against a
// per-query threshold into an LDS candidate list (score desc, index asc). A
// list that fills up is pruned to the top-k (bitonic sort) and the entries
// that did not fit are inserted again, so no qualifying row is lost. Finally
// each workgroup writes its top-k per query and a merge kernel reduces them.
#include <algorithm>
#include <mutex>
#include <type_traits>
#include <utility>

#include "common.h"
#include "timing.h"

namespace eogp {
namespace {

constexpr int QB = 16;                 // queries per pass
constexpr int NW = 8;                  // waves per workgroup
constexpr int NTHR = NW * 64;
constexpr int MCAP = 1024;             // candidate slots of the merge's list
constexpr int MRU = 2;                 // candidates per thread per merge round
constexpr int MSPLIT = 16;             // first-level merge workgroups per query
constexpr int MAX_TOPK = 256;

// A step covers SB bytes (8 SB bits) of a module in every row: lane (row,
// g) holds SB / 2 of them as NU = SB / 32 16-byte words, which feed FR = 8 NU
// MFMAs per tile, whose plane fragments take PU = 64 FR 16-byte slots (FR KB).
template <int SB>
struct StepShape {
  static constexpr int NU = SB / 32;
  static constexpr int FR = 8 * NU;
  static constexpr int PU = 64 * FR;
  static constexpr int PV = PU / NTHR;   // plane words staged per thread
};

typedef __attribute__((__vector_size__(16 * sizeof(int)))) int i32x16;
template <typename T>
using cptr = const __attribute__((address_space(4))) T*;   // read-only, scalar loads

struct ModInfo {
  int32_t k;       // bits of the module
  int32_t coff;    // first coordinate of the module in a query row
  int32_t boff;    // first byte of the module in a code row
  int32_t sbase;   // first step of the module
};

// Logical right shift of a register pair by s in one VALU instruction. The
// compiler turns a 64-bit shift whose result is masked to bits that never
// cross the halves back into two 32-bit shifts; here the bits that do cross
// are masked away by the caller, so one instruction serves two words.
__device__ __forceinline__ uint64_t shr_pair(uint64_t x, int s) {
  uint64_t r;
  asm("v_lshrrev_b64 %0, %1, %2" : "=v"(r) : "s"(s), "v"(x));
  return r;
}

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
// grid (16 * groups, U): per (query, module) the exponent f and the sum of
// y_int, stored [group][U][16]; queries past Q get f = 0 and sum 0. The sum is
// carried in 64 bits: |y_int| <= 2^14 and k_u <= 2^22 bound it by 2^36.
__global__ __launch_bounds__(256) void k_query_stats(const float* __restrict__ Y, int64_t ldy,
                                                     int64_t Q, int U,
                                                     const ModInfo* __restrict__ mods,
                                                     int32_t* __restrict__ fq,
                                                     int64_t* __restrict__ ysum) {
  __shared__ float smax[4];
  __shared__ int64_t ssum[4];
  const int64_t q = blockIdx.x;
  const int u = blockIdx.y;
  const int64_t o = ((q / QB) * U + u) * QB + (q % QB);
  if (q >= Q) {
    if (threadIdx.x == 0) {
      fq[o] = 0;
      ysum[o] = 0;
    }
    return;
  }
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
  int64_t s = 0;
  if (mx > 0.f)
    for (int c = threadIdx.x; c < md.k; c += 256) s += (int64_t)rintf(ldexpf(y[c], f));
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if ((threadIdx.x & 63) == 0) ssum[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    fq[o] = f;
    ysum[o] = ssum[0] + ssum[1] + ssum[2] + ssum[3];
  }
}

// Writes entries first .. first + count - 1 of the module table. The table
// travels in the kernel arguments (copied when the launch is enqueued), so
// the call needs no host synchronisation and the host's copy may go at once.
constexpr int MOD_CHUNK = 64;
struct ModChunk {
  ModInfo m[MOD_CHUNK];
  int32_t first, count;
};
__global__ void k_mod_table(ModChunk c, ModInfo* __restrict__ mods) {
  const int i = threadIdx.x;
  if (i < c.count) mods[c.first + i] = c.m[i];
}

// Planes laid out [group][step][MFMA f][lane][j] with f = 8 u + t: lane
// (M, g) = (lane % 32, lane / 32) is plane M / 16 (0: h, 1: l) of query M % 16,
// byte j holds coordinate 8 (sb s + sb / 2 g + 16 u + j) + t of the step's
// module (0 past the module), sb = bytes per row and step. One thread per
// (group, step, u, g, query, t) forms the 16 bytes of both planes of its query:
// eight neighbouring threads (t = 0..7) read eight neighbouring coordinates.
__global__ __launch_bounds__(256) void k_query_planes(const float* __restrict__ Y, int64_t ldy,
                                                      int64_t Q, int U,
                                                      const ModInfo* __restrict__ mods,
                                                      const int32_t* __restrict__ fq,
                                                      int64_t n_steps, int64_t n_groups, int sb,
                                                      int8_t* __restrict__ planes) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nu = sb / 32;                                 // 16-byte words per lane and step
  const int64_t per_step = 256 * (int64_t)nu;             // threads per step
  if (idx >= n_groups * n_steps * per_step) return;
  const int t = (int)(idx & 7);
  const int qn = (int)((idx >> 3) & 15);
  const int g = (int)((idx >> 7) & 1);
  const int uc = (int)((idx >> 8) % nu);
  const int64_t gs = idx / per_step;
  const int64_t step = gs % n_steps;
  const int64_t grp = gs / n_steps;
  int lo = 0, hi = U - 1;                    // last module whose first step <= step
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (mods[mid].sbase <= step) lo = mid; else hi = mid - 1;
  }
  const ModInfo md = mods[lo];
  const int64_t sl = step - md.sbase;
  const int64_t q = grp * QB + qn;
  const int f = q < Q ? fq[(grp * U + lo) * QB + qn] : 0;
  const int64_t c0 = 8 * (sb * sl + (sb / 2) * g + 16 * uc) + t;   // coordinate of byte 0
  const float* y = Y + q * ldy + md.coff;
  uint32_t hw[4] = {0u, 0u, 0u, 0u}, lw[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) {
    const int64_t c = c0 + 8 * jj;
    int yi = 0;
    if (q < Q && c < md.k) yi = (int)rintf(ldexpf(y[c], f));
    const int h = (yi + 128) >> 8;   // floor division (arithmetic shift)
    const int l = yi - 256 * h;
    hw[jj >> 2] |= (uint32_t)(h & 0xFF) << (8 * (jj & 3));
    lw[jj >> 2] |= (uint32_t)(l & 0xFF) << (8 * (jj & 3));
  }
  const int fr = 8 * uc + t;
  int8_t* blk = planes + (gs * (sb / 4) + fr) * 1024;
  const int lane = qn + 32 * g;   // plane h; plane l is lane + 16
  *reinterpret_cast<uint4*>(blk + 16 * lane) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
  *reinterpret_cast<uint4*>(blk + 16 * (lane + 16)) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
}

// Copies a store of n < 16 bytes into a zero-padded 16-byte slot.
__global__ void k_pad16(const uint8_t* __restrict__ src, int n, uint8_t* __restrict__ dst) {
  const int i = threadIdx.x;
  dst[i] = i < n ? src[i] : (uint8_t)0;
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

// Sort a list (all NTH threads of the block; the first power of two of slots
// that holds its entries, padded with empty ones), keep its first `topk`,
// update the threshold. Entries past CAP (counted but not stored) are dropped here;
// their owners insert them again.
template <int CAP, int NTH>
__device__ __forceinline__ void prune_list(uint64_t* key, uint32_t* idx, int* cnt, uint64_t* thr,
                                           int topk) {
  const int tid = threadIdx.x;
  const int c = min(*cnt, CAP);
  int P = 2;                     // sorted length: the least power of two >= c (CAP at most)
  while (P < c) P <<= 1;
  for (int i = c + tid; i < P; i += NTH) {
    key[i] = 0ull;
    idx[i] = 0xFFFFFFFFu;
  }
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < P; i += NTH) {
        const int p = i ^ j;
        if (p > i) {
          const uint64_t ka = key[i], kb = key[p];
          const uint32_t ia = idx[i], ib = idx[p];
          const bool desc = (i & k) == 0;
          const bool ab = before(ka, ia, kb, ib);
          if (desc ? !ab : ab) {
            key[i] = kb; key[p] = ka;
            idx[i] = ib; idx[p] = ia;
          }
        }
      }
      __syncthreads();
    }
  }
  if (tid == 0) {
    *thr = (c >= topk) ? key[topk - 1] : 0ull;
    *cnt = c < topk ? c : topk;
  }
  __syncthreads();
}
template <int CAP, int NTH>
__device__ __forceinline__ void prune(Cand<CAP>& cd, int n, int topk) {
  prune_list<CAP, NTH>(cd.key[n], cd.idx[n], &cd.cnt[n], &cd.thr[n], topk);
}

constexpr int MAX_RNG = 64;   // module ranges of the multi-module pass

struct ScoreArgs {
  const uint8_t* codes;
  int64_t cstride;
  const uint16_t* scales;
  int64_t N;
  int U;
  const ModInfo* mods;
  const uint4* planes;
  int n_steps;
  int64_t grp;
  const int32_t* fq;     // [groups][U][16]
  const int64_t* ysum;   // [groups][U][16]
  int64_t Q;
  int topk;
  float* full;
  uint64_t* ckey;   // [grid][QB][topk]
  uint32_t* cidx;
  // multi-module pass: module ranges (range r = modules rng[r] .. rng[r+1]-1)
  // and the per-(module, query, row) integer dots it writes, [U][QB][N]
  int n_rng;
  int32_t rng[MAX_RNG + 1];
  void* part;
  int64_t n_tiles;   // tiled store: 32-row tiles (ceil(N / 32))
};

// Calls f(integral_constant<I>) for I = 0 .. sizeof...(I) - 1 in order.
template <typename F, int... I>
__device__ __forceinline__ void for_each_index(std::integer_sequence<int, I...>, F&& f) {
  (f(std::integral_constant<int, I>{}), ...);
}

// Walks the steps of the modules in order (uniform, scalar registers).
struct Cursor {
  int u, sl, nst, kbytes, boff;
};

// NCLS: accumulator classes of the bit expansion (1, 2 or 4). D: steps
// requested ahead. MODE 0: one module; its fp64 term is formed after the last
// step and the rows are offered to the per-query candidate lists. MODE 1 / 2:
// several modules; a work unit is (512-row block, range of modules), and at
// the end of each module the exact dot <y_int, 2b - 1> of every (row, query)
// is written to `part` as int32 (MODE 1, every k_u <= 2^16) or int64 (MODE 2);
// k_score_fold then forms the fp64 terms and sums them in module order. CAP:
// candidate slots per query (MODE 0). SB: bytes per row and step. RT: 32-row
// tiles per wave (each plane fragment read from LDS feeds RT MFMAs). TILED:
// the store is in the tiled layout (see eogp_sign_pack_tiled): each wave's
// 32-row tile and step is one 2 KB block whose bytes are already in lane
// order, read as two contiguous 1 KB loads; else rows are row-major.
template <int NCLS, int D, int MODE, int CAP, int SB, int RT, bool TILED>
__global__ __launch_bounds__(NTHR) void k_score(ScoreArgs a) {
  constexpr bool MULTI = MODE != 0;
  static_assert(!TILED || SB == 64, "the tiled layout has 64-byte row pieces per step");
  constexpr int ROWS = NW * RT * 32;   // rows per block
  static_assert(NCLS == 1 || NCLS == 2 || NCLS == 4, "bit-weight classes");
  static_assert(D >= 2 && D <= 8, "ring depth");
  using SS = StepShape<SB>;
  constexpr int NU = SS::NU, FR = SS::FR, PU = SS::PU, PV = SS::PV;
  __shared__ __attribute__((aligned(16))) uint4 sP[2][PU];
  __shared__ Cand<MULTI ? 1 : CAP> cd;
  // the wave index through readfirstlane: wave-uniform for the compiler, so the
  // row and tile arithmetic that depends on it stays scalar
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31, hg = lane >> 5;
  const cptr<int32_t> cmods = (cptr<int32_t>)(a.mods);   // ModInfo fields, 4 per module
  const cptr<int32_t> cfq = (cptr<int32_t>)(a.fq);
  const cptr<int64_t> cys = (cptr<int64_t>)(a.ysum);
  if (!MULTI) {
    if (tid < QB) {
      cd.cnt[tid] = 0;
      cd.thr[tid] = 0ull;
    }
    if (tid == 0) cd.overflow = 0;
    __syncthreads();
  }
  const int64_t n_blocks = (a.N + ROWS - 1) / ROWS;
  const uint32_t M1 = 0x01010101u;

  // Work units. MODE 0: row blocks at a fixed stride. Multi-module: units
  // (range, block) in range-major order, dealt to the XCDs in contiguous
  // chunks (workgroup b runs on XCD b % 8), so the workgroups of one XCD share
  // the plane fragments of few module ranges in their L2.
  const int nrng = MULTI ? a.n_rng : 1;
  const int64_t n_units = n_blocks * nrng;
  const int G = gridDim.x, b = blockIdx.x;
  const bool xq = MULTI && G >= kXcds && G % kXcds == 0;
  const int nq = xq ? kXcds : 1, xcd = xq ? b % kXcds : 0;
  const int64_t chunk = (n_units + nq - 1) / nq;
  const int64_t q_end = std::min<int64_t>((int64_t)(xcd + 1) * chunk, n_units);
  for (int64_t unit = (int64_t)xcd * chunk + b / nq; unit < q_end; unit += G / nq) {
    const int rg = MULTI ? (int)(unit / n_blocks) : 0;
    const int64_t blk = MULTI ? unit % n_blocks : unit;
    const int u_lo = MULTI ? a.rng[rg] : 0;
    const int u_hi = MULTI ? a.rng[rg + 1] : 1;
    const int s_lo = MULTI ? cmods[4 * u_lo + 3] : 0;
    const int s_hi = (MULTI && u_hi < a.U) ? cmods[4 * u_hi + 3] : a.n_steps;
    const int n = s_hi - s_lo;
    const uint4* pl_grp = a.planes + ((int64_t)a.grp * a.n_steps + s_lo) * PU;

  auto start = [&](Cursor& c) __attribute__((always_inline)) {
    const int k = cmods[4 * u_lo];
    c.u = u_lo;
    c.sl = 0;
    c.nst = (k + 8 * SB - 1) / (8 * SB);
    c.kbytes = k >> 3;
    c.boff = cmods[4 * u_lo + 2];
  };
  auto advance = [&](Cursor& c) __attribute__((always_inline)) {
    if (++c.sl == c.nst) {
      c.sl = 0;
      if (++c.u < u_hi) {
        const int k = cmods[4 * c.u];
        c.nst = (k + 8 * SB - 1) / (8 * SB);
        c.kbytes = k >> 3;
        c.boff = cmods[4 * c.u + 2];
      }
    }
  };

    int64_t row[RT], rowc[RT];
    const uint8_t* rowp[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      row[rt] = blk * ROWS + (int64_t)(wid * RT + rt) * 32 + r32;   // this lane's stored row
      rowc[rt] = std::min<int64_t>(row[rt], a.N - 1);                // rows past N: never reported
      if constexpr (TILED) {
        const int64_t tile = std::min<int64_t>(blk * (ROWS / 32) + wid * RT + rt, a.n_tiles - 1);
        rowp[rt] = a.codes + tile * (int64_t)a.n_steps * 2048 + lane * 16;
      } else {
        rowp[rt] = a.codes + rowc[rt] * a.cstride + (SB / 2) * hg;
      }
    }

    i32x16 acc[RT][NCLS];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int w = 0; w < NCLS; ++w)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[rt][w][r] = 0;
    double sc[MULTI ? 1 : RT][8];   // [tile][i]: query 8 (i / 4) + 4 (lane / 32) + i % 4 of the group

    // ring slot: [rt][0, NU) the lane's code words of tile rt, [RT][0, PV)
    // the thread's share of the step's plane fragments
    constexpr int RW = NU > PV ? NU : PV;
    uint4 ring[D][RT + 1][RW];
    uint32_t s16[RT];      // one module: the rows' scales, requested before the codes
    if (!MULTI) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) s16[rt] = a.scales[rowc[rt]];
    }
    Cursor cc, cl;
    start(cc);
    start(cl);

    // plane fragments and code words of step `target` (the load cursor's)
    // into ring slot SL, D steps ahead. Every step issues the same loads in
    // the order they are consumed, so the in-order load counter never makes
    // a step wait for a later step's data, and the number of requests in
    // flight never depends on the step or the lane. In a partial step (the
    // last of a module whose k is not a multiple of 8 SB, or a step past the
    // end) a lane whose 16 bytes are not all inside the module reads 16
    // readable bytes instead: the 8 bytes before its 8 valid ones (the valid
    // half is then the upper one), or the store's first 16 bytes; `fixup`
    // keeps the valid bytes when the step is used.
    int64_t voff[D];
    int vbytes[D];
    auto load_step = [&](auto slot_c, int target) __attribute__((always_inline)) {
      constexpr int SL = decltype(slot_c)::value;
      const bool live = target < n;
      const uint4* psrc = pl_grp + (int64_t)(live ? target : n - 1) * PU + tid;
#pragma unroll
      for (int v = 0; v < PV; ++v) ring[SL][RT][v] = psrc[v * NTHR];
      if constexpr (TILED) {
        // every step of a module is whole (k_u a multiple of 512); a step
        // past the range reads the range's last block again, unused
        const int64_t so = (int64_t)(s_lo + (live ? target : n - 1)) * 2048;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int uc = 0; uc < NU; ++uc)
            ring[SL][rt][uc] = *reinterpret_cast<const uint4*>(rowp[rt] + so + uc * 1024);
        voff[SL] = 0;
        vbytes[SL] = SB;
        return;
      }
      const int64_t off = (int64_t)cl.boff + SB * cl.sl;
      const int valid = live ? min(SB, cl.kbytes - SB * cl.sl) : 0;   // multiple of 8
      voff[SL] = off;
      vbytes[SL] = valid;
      if (valid == SB) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int uc = 0; uc < NU; ++uc)
            ring[SL][rt][uc] = *reinterpret_cast<const uint4*>(rowp[rt] + off + 16 * uc);
      } else {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int uc = 0; uc < NU; ++uc) {
            const int have = valid - (SB / 2) * hg - 16 * uc;
            const int64_t pos = off + (SB / 2) * hg + 16 * uc;   // within the row
            const bool at0 = rowc[rt] == 0 && pos == 0;          // the store's first byte
            const uint8_t* src = rowp[rt] + off + 16 * uc;
            const uint8_t* p = have >= 16 ? src : (have >= 8 && !at0) ? src - 8 : a.codes;
            ring[SL][rt][uc] = *reinterpret_cast<const uint4*>(p);
          }
      }
    };
    // keeps the valid bytes of a partial step (branch-free selects)
    auto fixup = [&](auto slot_c) __attribute__((always_inline)) {
      constexpr int SL = decltype(slot_c)::value;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int uc = 0; uc < NU; ++uc) {
          const int have = vbytes[SL] - (SB / 2) * hg - 16 * uc;
          const bool at0 = rowc[rt] == 0 && voff[SL] + (SB / 2) * hg + 16 * uc == 0;
          const uint4 v = ring[SL][rt][uc];
          const uint32_t full = have >= 16 ? ~0u : 0u;
          const uint32_t half = (have >= 8 && have < 16) ? ~0u : 0u;
          const uint32_t lo0 = at0 ? v.x : v.z, lo1 = at0 ? v.y : v.w;
          ring[SL][rt][uc] = make_uint4((v.x & full) | (lo0 & half), (v.y & full) | (lo1 & half),
                                        v.z & full, v.w & full);
        }
    };

    // end of module u: the exact dot n = 2 n1 - sum y_int of every (row,
    // query); one module: its term s * n * 2^-f; several: n to `part`
    auto fold = [&](int u) __attribute__((always_inline)) {
      const int64_t mo = (a.grp * a.U + u) * QB;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        int H[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int v = acc[rt][0][r];
#pragma unroll
          for (int w = 1; w < NCLS; ++w) v += acc[rt][w][r] >> w;
          H[r] = v;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int i0 = 8 * (i >> 2) + (i & 3);
          const int64_t ys = hg ? cys[mo + i0 + 4] : cys[mo + i0];
          const int64_t n1 = 256 * (int64_t)H[i] + (int64_t)H[i + 8];
          const int64_t nn = 2 * n1 - ys;
          if constexpr (MULTI) {
            if (row[rt] < a.N) {
              const int64_t o = ((int64_t)u * QB + i0 + 4 * hg) * a.N + row[rt];
              if constexpr (MODE == 1) static_cast<int32_t*>(a.part)[o] = (int32_t)nn;
              else static_cast<int64_t*>(a.part)[o] = nn;
            }
          } else {
            const int f = hg ? cfq[mo + i0 + 4] : cfq[mo + i0];
            const double sv = (double)f16_bits_to_f32((uint16_t)s16[rt]);
            sc[rt][i] = ldexp(sv * (double)nn, -f);
          }
        }
#pragma unroll
        for (int w = 0; w < NCLS; ++w)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[rt][w][r] = 0;
      }
    };

    auto step = [&](auto slot_c, int s) __attribute__((always_inline)) {
      constexpr int SL = decltype(slot_c)::value;
      constexpr int NX = (SL + 1) % D;   // slot of step s + 1
      const int buf = s & 1;
      if (vbytes[SL] < SB) fixup(slot_c);
      // fragment f = 8 uc + t of the step, read from LDS two rounds ahead of
      // its use so the LDS latency stays hidden; each feeds the RT tiles
      const uint4* frag = &sP[buf][lane];
      i32x4 fr[3];
      fr[0] = __builtin_bit_cast(i32x4, frag[0]);
      fr[1] = __builtin_bit_cast(i32x4, frag[64]);
#pragma unroll
      for (int f = 0; f < FR; ++f) {
        if (f + 2 < FR) fr[(f + 2) % 3] = __builtin_bit_cast(i32x4, frag[(f + 2) * 64]);
        const int uc = f >> 3, t = f & 7;
        const int w = t % NCLS, sh = t - w;
        const uint32_t mk = M1 << w;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const uint4 c = ring[SL][rt][uc];
          // bits shifted across the halves land at 32 - sh and above, never
          // under the mask (its highest bit is 24 + w, and sh + w <= 7)
          uint64_t p0 = ((uint64_t)c.y << 32) | c.x, p1 = ((uint64_t)c.w << 32) | c.z;
          if (sh) {
            p0 = shr_pair(p0, sh);
            p1 = shr_pair(p1, sh);
          }
          i32x4 av;
          av[0] = (int)((uint32_t)p0 & mk);
          av[1] = (int)((uint32_t)(p0 >> 32) & mk);
          av[2] = (int)((uint32_t)p1 & mk);
          av[3] = (int)((uint32_t)(p1 >> 32) & mk);
          acc[rt][w] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fr[f % 3], av, acc[rt][w], 0, 0, 0);
        }
        // per round: the read two rounds ahead, then each tile's expansion and MFMA
        if (f + 2 < FR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          __builtin_amdgcn_sched_group_barrier(0x002, NCLS == 1 ? 8 : NCLS == 2 ? 6 : 5, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // MFMA
        }
      }
      if (MULTI) {
        if (cc.sl == cc.nst - 1) fold(cc.u);
        advance(cc);
      }
      load_step(slot_c, s + D);
      advance(cl);
#pragma unroll
      for (int v = 0; v < PV; ++v) sP[buf ^ 1][tid + v * NTHR] = ring[NX][RT][v];
      __syncthreads();
    };

    // prologue: the first D steps requested, step 0's planes staged
    for_each_index(std::make_integer_sequence<int, D>{}, [&](auto i_c) __attribute__((always_inline)) {
      load_step(i_c, decltype(i_c)::value);
      advance(cl);
    });
#pragma unroll
    for (int v = 0; v < PV; ++v) sP[0][tid + v * NTHR] = ring[0][RT][v];
    __syncthreads();
    // whole rounds of D steps (every step of a round runs, so the loads in
    // flight are the same on every path around the loop), then the rest
    int s0 = 0;
    for (; s0 + D <= n; s0 += D) {
      for_each_index(std::make_integer_sequence<int, D>{}, [&](auto i_c) __attribute__((always_inline)) {
        step(i_c, s0 + decltype(i_c)::value);
      });
    }
    for_each_index(std::make_integer_sequence<int, D - 1>{}, [&](auto i_c) __attribute__((always_inline)) {
      if (s0 + decltype(i_c)::value < n) step(i_c, s0 + decltype(i_c)::value);
    });

    if constexpr (!MULTI) {
      fold(0);

      // candidates of this block; a full list is pruned and the entries that
      // did not fit are offered again (the loop condition is uniform). The
      // opaque copy of the lane half keeps the list addresses from being
      // computed once before the block loop and held through it.
      int hq = hg;
      asm volatile("" : "+v"(hq));
      auto qsel = [&](int i) { return 8 * (i >> 2) + 4 * hq + (i & 3); };
      uint32_t pend = 0;
  #pragma unroll
      for (int rt = 0; rt < RT; ++rt)
  #pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int64_t q = a.grp * QB + qsel(i);
          if (row[rt] < a.N && q < a.Q) {
            if (a.full) a.full[q * a.N + row[rt]] = (float)sc[rt][i];
            pend |= 1u << (8 * rt + i);
          }
        }
      for (;;) {
  #pragma unroll
        for (int rt = 0; rt < RT; ++rt)
  #pragma unroll
          for (int i = 0; i < 8; ++i) {
            const uint32_t bit = 1u << (8 * rt + i);
            if (pend & bit) {
              const int qn = qsel(i);
              const uint64_t key = order_key(sc[rt][i]);
              if (key < cd.thr[qn]) {
                pend &= ~bit;
              } else {
                const int pos = atomicAdd(&cd.cnt[qn], 1);
                if (pos < CAP) {
                  cd.key[qn][pos] = key;
                  cd.idx[qn][pos] = (uint32_t)row[rt];
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
  }
  if constexpr (!MULTI) {
    // lists of at most topk entries are written as they are (the merge
    // takes candidates in any order)
    for (int qq = 0; qq < QB; ++qq)
      if (cd.cnt[qq] > a.topk) prune<CAP, NTHR>(cd, qq, a.topk);
    for (int i = tid; i < QB * a.topk; i += NTHR) {
      const int qq = i / a.topk, e = i % a.topk;
      const int64_t o = ((int64_t)blockIdx.x * QB + qq) * a.topk + e;
      const bool have = e < cd.cnt[qq];
      a.ckey[o] = have ? cd.key[qq][e] : 0ull;
      a.cidx[o] = have ? cd.idx[qq][e] : 0xFFFFFFFFu;
    }
  }
}

// Multi-module scores from the exact per-module dots: wave w of a workgroup
// takes queries 4w .. 4w+3 of the group for 64 consecutive stored rows (one
// per lane); for u = 0 .. U-1 in order, score += s_{i,u} * n * 2^-f (each
// term exact in fp64), then the rows are offered to the per-query candidate
// lists as in k_score. Workgroups walk blocks of 64 rows at a fixed stride.
struct FoldArgs {
  const void* part;           // [U][QB][N] int32 or int64
  const uint16_t* scales;     // [N][U] fp16 bits
  int64_t N;
  int U;
  const int32_t* fq;          // [groups][U][16]
  int64_t grp;
  int64_t Q;
  int topk;
  float* full;
  uint64_t* ckey;             // [grid][QB][topk]
  uint32_t* cidx;
};
constexpr int FOLD_THR = 256;
constexpr int FOLD_ROWS = 64;
constexpr int FOLD_QW = QB / (FOLD_THR / 64);   // queries per wave

template <int CAP, bool N64>
__global__ __launch_bounds__(FOLD_THR) void k_score_fold(FoldArgs a) {
  __shared__ Cand<CAP> cd;
  const int tid = threadIdx.x, lane = tid & 63;
  const int q0 = __builtin_amdgcn_readfirstlane((tid >> 6) * FOLD_QW);   // wave-uniform
  const cptr<int32_t> cfq = (cptr<int32_t>)(a.fq);
  if (tid < QB) {
    cd.cnt[tid] = 0;
    cd.thr[tid] = 0ull;
  }
  if (tid == 0) cd.overflow = 0;
  __syncthreads();
  const int32_t* p32 = static_cast<const int32_t*>(a.part);
  const int64_t* p64 = static_cast<const int64_t*>(a.part);
  for (int64_t r0 = (int64_t)blockIdx.x * FOLD_ROWS; r0 < a.N;
       r0 += (int64_t)gridDim.x * FOLD_ROWS) {
    const int64_t row = r0 + lane;
    const bool ok = row < a.N;
    const int64_t rowc = ok ? row : a.N - 1;
    double sc[FOLD_QW];
#pragma unroll
    for (int j = 0; j < FOLD_QW; ++j) sc[j] = 0.0;
#pragma unroll 4
    for (int u = 0; u < a.U; ++u) {
      const double sv = (double)f16_bits_to_f32(a.scales[rowc * a.U + u]);
      const int64_t mo = (a.grp * a.U + u) * QB + q0;
#pragma unroll
      for (int j = 0; j < FOLD_QW; ++j) {
        const int64_t o = ((int64_t)u * QB + q0 + j) * a.N + rowc;
        const int64_t nn = N64 ? p64[o] : (int64_t)p32[o];
        sc[j] += ldexp(sv * (double)nn, -cfq[mo + j]);
      }
    }
    uint32_t pend = 0;
#pragma unroll
    for (int j = 0; j < FOLD_QW; ++j) {
      const int64_t qg = a.grp * QB + q0 + j;
      if (ok && qg < a.Q) {
        if (a.full) a.full[qg * a.N + row] = (float)sc[j];
        pend |= 1u << j;
      }
    }
    for (;;) {
#pragma unroll
      for (int j = 0; j < FOLD_QW; ++j) {
        const uint32_t bit = 1u << j;
        const int q = q0 + j;
        if (pend & bit) {
          const uint64_t key = order_key(sc[j]);
          if (key < cd.thr[q]) {
            pend &= ~bit;
          } else {
            const int pos = atomicAdd(&cd.cnt[q], 1);
            if (pos < CAP) {
              cd.key[q][pos] = key;
              cd.idx[q][pos] = (uint32_t)row;
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
        if (cd.cnt[qq] >= CAP) prune<CAP, FOLD_THR>(cd, qq, a.topk);
      if (tid == 0) cd.overflow = 0;
      __syncthreads();
    }
  }
  for (int qq = 0; qq < QB; ++qq)
    if (cd.cnt[qq] > a.topk) prune<CAP, FOLD_THR>(cd, qq, a.topk);
  for (int i = tid; i < QB * a.topk; i += FOLD_THR) {
    const int qq = i / a.topk, e = i % a.topk;
    const int64_t o = ((int64_t)blockIdx.x * QB + qq) * a.topk + e;
    const bool have = e < cd.cnt[qq];
    a.ckey[o] = have ? cd.key[qq][e] : 0ull;
    a.cidx[o] = have ? cd.idx[qq][e] : 0xFFFFFFFFu;
  }
}

// Reduction of the per-workgroup candidate lists ([G][QB][topk] keys and
// indices, empty slots marked by index 0xFFFFFFFF) in two levels: workgroup
// (n, sp) merges lists sp * per .. sp * per + per - 1 of query n of the group
// into one list of the same form (!FINAL, list sp of the output), then one
// workgroup per query merges those into the sorted top-k (FINAL). Each round
// requests MRU candidates per thread before any is used; a list longer than
// MCAP - 256 MRU is pruned before the next round, so a round always fits.
struct MergeList {
  uint64_t key[MCAP];
  uint32_t idx[MCAP];
  int cnt;
  uint64_t thr;
};
template <bool FINAL>
__global__ __launch_bounds__(256, 1) void k_merge(const uint64_t* __restrict__ ckey,
                                                  const uint32_t* __restrict__ cidx, int G, int per,
                                                  int64_t grp, int64_t Q, int topk,
                                                  int64_t* __restrict__ out_idx,
                                                  float* __restrict__ out_score,
                                                  uint64_t* __restrict__ okey,
                                                  uint32_t* __restrict__ oidx) {
  __shared__ MergeList ml;
  const int n = blockIdx.x, sp = blockIdx.y;
  const int64_t q = grp * QB + n;
  if (q >= Q) return;                         // never read by the next level either
  const int tid = threadIdx.x;
  if (tid == 0) {
    ml.cnt = 0;
    ml.thr = 0ull;
  }
  __syncthreads();
  const int64_t l0 = (int64_t)sp * per;
  const int64_t total = std::max<int64_t>(0, std::min<int64_t>(G - l0, per)) * topk;
  for (int64_t base = 0; base < total; base += 256 * MRU) {
    uint64_t key[MRU];
    uint32_t id[MRU];
#pragma unroll
    for (int r = 0; r < MRU; ++r) {
      const int64_t e = base + 256 * r + tid;
      key[r] = 0ull;
      id[r] = 0xFFFFFFFFu;
      if (e < total) {
        const int64_t wg = l0 + e / topk, j = e % topk;
        const int64_t o = (wg * QB + n) * topk + j;
        key[r] = ckey[o];
        id[r] = cidx[o];
      }
    }
    const uint64_t thr = ml.thr;
#pragma unroll
    for (int r = 0; r < MRU; ++r) {
      if (id[r] != 0xFFFFFFFFu && key[r] >= thr) {
        const int pos = atomicAdd(&ml.cnt, 1);
        ml.key[pos] = key[r];
        ml.idx[pos] = id[r];
      }
    }
    __syncthreads();
    if (ml.cnt > MCAP - 256 * MRU) prune_list<MCAP, 256>(ml.key, ml.idx, &ml.cnt, &ml.thr, topk);
  }
  if (FINAL || ml.cnt > topk) prune_list<MCAP, 256>(ml.key, ml.idx, &ml.cnt, &ml.thr, topk);
  for (int e = tid; e < topk; e += 256) {
    const bool have = e < ml.cnt;
    if constexpr (FINAL) {
      out_idx[q * topk + e] = have ? (int64_t)ml.idx[e] : -1;
      out_score[q * topk + e] = have ? (float)key_value(ml.key[e]) : -__builtin_inff();
    } else {
      const int64_t o = ((int64_t)sp * QB + n) * topk + e;
      okey[o] = have ? ml.key[e] : 0ull;
      oidx[o] = have ? ml.idx[e] : 0xFFFFFFFFu;
    }
  }
}

// Pass configuration: candidate slots per query of the multi-module fold (256
// when that leaves room for at least 128 new entries after a prune, else 512;
// the one-module pass always takes 512, with which its first blocks prune less
// often: 0.7% faster per pass than 256 at top-100), bytes per row and
// step, 32-row tiles per wave and steps requested ahead. One workgroup runs
// per CU (LDS).
struct PassCfg {
  int cap, sb, rt, d;
};
inline PassCfg pass_cfg(int32_t topk) {
  PassCfg c;
  c.cap = topk <= 128 ? 256 : 512;
  c.sb = 64;
  c.rt = 2;
  c.d = 3;
  return c;
}

struct Layout {
  int64_t n_steps = 0;   // steps over all modules
  int64_t n_groups = 0;
  int64_t grid = 0;      // workgroups of the scoring pass
  int64_t fold_grid = 0; // workgroups of the multi-module fold (0: one module)
  int64_t step_bytes = 0;
  int n_rng = 1;         // module ranges of the multi-module pass
  bool n64 = false;      // multi-module dots stored in 64 bits
  int merge_split = 1;   // first-level merge workgroups per query
  size_t o_mods = 0, o_fq = 0, o_ys = 0, o_pl = 0, o_ck = 0, o_ci = 0, o_ck2 = 0, o_ci2 = 0,
         o_part = 0, o_pad = 0,
         total = 0;
};

Layout layout(int64_t N, int64_t Q, int32_t U, const int64_t* kmod, int32_t topk) {
  Layout L;
  const PassCfg c = pass_cfg(topk);
  int64_t kmax = 0;
  for (int u = 0; u < U; ++u) {
    L.n_steps += (kmod[u] + 8 * c.sb - 1) / (8 * c.sb);
    kmax = std::max<int64_t>(kmax, kmod[u]);
  }
  L.n_groups = (Q + QB - 1) / QB;
  L.step_bytes = 256 * (int64_t)c.sb;
  const int64_t n_blocks = (N + NW * 32 * c.rt - 1) / (NW * 32 * c.rt);
  int64_t lists = 0;
  if (U == 1) {
    L.grid = std::max<int64_t>(1, std::min<int64_t>(n_blocks, kCus));
    lists = L.grid;
  } else {
    // about four units per CU when the row blocks alone are too few, each
    // range at least one module; ranges are cut by step count
    L.n_rng = (int)std::min<int64_t>({(int64_t)U, (int64_t)MAX_RNG,
                                      std::max<int64_t>(1, ceil_div(4 * kCus, std::max<int64_t>(1, n_blocks)))});
    const int64_t units = std::max<int64_t>(1, n_blocks * L.n_rng);
    L.grid = std::min<int64_t>(units, kCus);
    if (L.grid >= kXcds) L.grid = L.grid / kXcds * kXcds;
    L.fold_grid = std::max<int64_t>(1, std::min<int64_t>(ceil_div(N, FOLD_ROWS), 2 * kCus));
    lists = L.fold_grid;
    L.n64 = kmax > (1 << 16);   // |n| <= k 2^14 fits 32 bits up to k = 2^16
  }
  size_t b = 0;
  auto add = [&](size_t x) { size_t o = b; b = align256(b + x); return o; };
  L.o_mods = add(sizeof(ModInfo) * U);
  L.o_fq = add(4 * (size_t)L.n_groups * U * QB);
  L.o_ys = add(8 * (size_t)L.n_groups * U * QB);
  L.o_pl = add((size_t)(L.n_groups * L.n_steps * L.step_bytes));
  L.o_ck = add((size_t)lists * QB * topk * 8);
  L.o_ci = add((size_t)lists * QB * topk * 4);
  L.merge_split = (int)std::min<int64_t>(MSPLIT, std::max<int64_t>(1, lists / 8));
  L.o_ck2 = add((size_t)L.merge_split * QB * topk * 8);
  L.o_ci2 = add((size_t)L.merge_split * QB * topk * 4);
  L.o_part = add(U > 1 ? (size_t)U * QB * (size_t)N * (L.n64 ? 8 : 4) : 0);
  L.o_pad = add(16);   // a store of fewer than 16 bytes is copied here (see score_topk)
  L.total = b;
  return L;
}

// Module ranges of the multi-module pass: n_rng consecutive ranges of
// roughly equal step counts, each at least one module (one pass over the
// module sizes, no host allocation).
void module_ranges(const int64_t* kmod, int U, int sb, int64_t n_steps, int n_rng, int32_t* rng) {
  auto steps = [&](int u) { return (kmod[u] + 8 * sb - 1) / (8 * sb); };
  rng[0] = 0;
  int v = 1;                   // candidate start of the next range
  int64_t base = steps(0);     // first step of module v
  for (int r = 1; r < n_rng; ++r) {
    if (v <= rng[r - 1]) {     // range r - 1 keeps at least one module
      base += steps(v);
      ++v;
    }
    const int64_t target = (n_steps * r + n_rng / 2) / n_rng;
    const int v_max = U - (n_rng - r);     // leaves a module for each later range
    while (v < v_max && base < target) {
      base += steps(v);
      ++v;
    }
    rng[r] = v;
  }
  rng[n_rng] = U;
}

template <int MODE, int CAP, bool TILED>
eogp_status launch_pass(const PassCfg& c, dim3 gd, const ScoreArgs& a, hipStream_t s) {
#define EOGP_SCORE_CFG(SB, RT, D)                                                           \
  if (c.sb == SB && c.rt == RT && c.d == D) {                                               \
    hipLaunchKernelGGL((k_score<2, D, MODE, CAP, SB, RT, TILED>), gd, dim3(NTHR), 0, s, a);  \
    return EOGP_OK;                                                                         \
  }
  EOGP_SCORE_CFG(64, 2, 3)
#undef EOGP_SCORE_CFG
  return fail(EOGP_ERR_UNSUPPORTED, "score_topk: no kernel for this pass configuration");
}

}  // namespace

int32_t score_max_topk() { return MAX_TOPK; }

size_t score_ws(int64_t N, int64_t Q, int32_t U, const int64_t* kmod, int32_t topk) {
  return layout(N, Q, U, kmod, topk).total;
}

template <bool TILED>
eogp_status score_topk_impl(const uint8_t* codes, int64_t cstride, const uint16_t* scales,
                            int64_t N, int32_t U, const int64_t* kmod, const float* Y, int64_t ldy,
                            int64_t Q, int32_t topk, int64_t* out_idx, float* out_score,
                            float* full, void* ws, size_t ws_bytes, hipStream_t s) {
  const Layout L = layout(N, Q, U, kmod, topk);
  if (ws_bytes < L.total) return fail(EOGP_ERR_WORKSPACE, "score_topk: workspace too small");
  if (Q == 0) return EOGP_OK;
  char* base = static_cast<char*>(ws);
  ModInfo* mods = reinterpret_cast<ModInfo*>(base + L.o_mods);
  int32_t* fq = reinterpret_cast<int32_t*>(base + L.o_fq);
  int64_t* ys = reinterpret_cast<int64_t*>(base + L.o_ys);
  int8_t* planes = reinterpret_cast<int8_t*>(base + L.o_pl);
  uint64_t* ck = reinterpret_cast<uint64_t*>(base + L.o_ck);
  uint32_t* ci = reinterpret_cast<uint32_t*>(base + L.o_ci);
  uint64_t* ck2 = reinterpret_cast<uint64_t*>(base + L.o_ck2);
  uint32_t* ci2 = reinterpret_cast<uint32_t*>(base + L.o_ci2);

  // The pass reads 16 bytes at the store's start in place of bytes past a
  // module's end; a store with fewer readable bytes is copied into a zeroed
  // 16-byte slot of the workspace first.
  int64_t ksum = 0;
  for (int u = 0; u < U; ++u) ksum += kmod[u];
  if (!TILED && N > 0 && (N - 1) * cstride + ksum / 8 < 16) {
    uint8_t* pad = reinterpret_cast<uint8_t*>(base + L.o_pad);
    hipLaunchKernelGGL(k_pad16, dim3(1), dim3(16), 0, s, codes,
                       (int)((N - 1) * cstride + ksum / 8), pad);
    EOGP_LAUNCH_CHECK("small-store copy");
    codes = pad;
  }
  const PassCfg cfg = pass_cfg(topk);
  // the module table, MOD_CHUNK entries per launch (kernel arguments)
  int64_t coff = 0, boff = 0, sbase = 0;
  for (int u0 = 0; u0 < U; u0 += MOD_CHUNK) {
    ModChunk mc;
    mc.first = u0;
    mc.count = std::min(MOD_CHUNK, U - u0);
    for (int i = 0; i < mc.count; ++i) {
      const int64_t k = kmod[u0 + i];
      mc.m[i].k = (int32_t)k;
      mc.m[i].coff = (int32_t)coff;
      mc.m[i].boff = (int32_t)boff;
      mc.m[i].sbase = (int32_t)sbase;
      coff += k;
      boff += k / 8;
      sbase += (k + 8 * cfg.sb - 1) / (8 * cfg.sb);
    }
    hipLaunchKernelGGL(k_mod_table, dim3(1), dim3(MOD_CHUNK), 0, s, mc, mods);
  }
  EOGP_LAUNCH_CHECK("module table");
  timing::Scope tprep(EOGP_KT_SCORE_PREP, s);
  hipLaunchKernelGGL(k_query_stats, dim3((unsigned)(L.n_groups * QB), (unsigned)U), dim3(256), 0,
                     s, Y, ldy, Q, U, mods, fq, ys);
  // one thread per 16 bytes of each of the two planes
  const int64_t pthreads = L.n_groups * L.n_steps * L.step_bytes / 32;
  hipLaunchKernelGGL(k_query_planes, dim3((unsigned)ceil_div(pthreads, 256)), dim3(256), 0, s, Y,
                     ldy, Q, U, mods, fq, L.n_steps, L.n_groups, cfg.sb, planes);
  EOGP_LAUNCH_CHECK("query preparation");
  timing::end(tprep.slot, s);
  tprep.slot = -1;
  ScoreArgs a;
  a.codes = codes;
  a.cstride = cstride;
  a.scales = scales;
  a.N = N;
  a.U = U;
  a.mods = mods;
  a.planes = reinterpret_cast<const uint4*>(planes);
  a.n_steps = (int)L.n_steps;
  a.fq = fq;
  a.ysum = ys;
  a.Q = Q;
  a.topk = topk;
  a.full = full;
  a.ckey = ck;
  a.cidx = ci;
  a.n_rng = L.n_rng;
  a.part = base + L.o_part;
  a.n_tiles = ceil_div(N, 32);
  if (U > 1) module_ranges(kmod, U, cfg.sb, L.n_steps, L.n_rng, a.rng);
  FoldArgs fa;
  fa.part = a.part;
  fa.scales = scales;
  fa.N = N;
  fa.U = U;
  fa.fq = fq;
  fa.Q = Q;
  fa.topk = topk;
  fa.full = full;
  fa.ckey = ck;
  fa.cidx = ci;
  for (int64_t grp = 0; grp < L.n_groups; ++grp) {
    a.grp = grp;
    fa.grp = grp;
    {
      // one pass over the store: the streaming kernel, and for several
      // modules the fold that adds their terms in order
      timing::Scope tp(EOGP_KT_SCORE_PASS, s);
      const dim3 gd((unsigned)L.grid);
      eogp_status st;
      if (U == 1) {
        st = launch_pass<0, 512, TILED>(cfg, gd, a, s);
      } else {
        st = L.n64 ? launch_pass<2, 256, TILED>(cfg, gd, a, s) : launch_pass<1, 256, TILED>(cfg, gd, a, s);
        if (st == EOGP_OK) {
          const dim3 fg((unsigned)L.fold_grid), fb(FOLD_THR);
          if (cfg.cap == 256) {
            if (L.n64) hipLaunchKernelGGL((k_score_fold<256, true>), fg, fb, 0, s, fa);
            else hipLaunchKernelGGL((k_score_fold<256, false>), fg, fb, 0, s, fa);
          } else {
            if (L.n64) hipLaunchKernelGGL((k_score_fold<512, true>), fg, fb, 0, s, fa);
            else hipLaunchKernelGGL((k_score_fold<512, false>), fg, fb, 0, s, fa);
          }
        }
      }
      if (st != EOGP_OK) return st;
    }
    timing::Scope tm(EOGP_KT_SCORE_MERGE, s);
    const int lists = (int)(U == 1 ? L.grid : L.fold_grid);
    const int sp = L.merge_split, per = (int)ceil_div(lists, sp);
    if (sp > 1) {
      hipLaunchKernelGGL(k_merge<false>, dim3(QB, sp), dim3(256), 0, s, ck, ci, lists, per, grp, Q,
                         topk, nullptr, nullptr, ck2, ci2);
      hipLaunchKernelGGL(k_merge<true>, dim3(QB), dim3(256), 0, s, ck2, ci2, sp, sp, grp, Q, topk,
                         out_idx, out_score, nullptr, nullptr);
    } else {
      hipLaunchKernelGGL(k_merge<true>, dim3(QB), dim3(256), 0, s, ck, ci, lists, lists, grp, Q,
                         topk, out_idx, out_score, nullptr, nullptr);
    }
    EOGP_LAUNCH_CHECK("score pass");
  }
  return EOGP_OK;
}

eogp_status score_topk(const uint8_t* codes, int64_t cstride, const uint16_t* scales, int64_t N,
                       int32_t U, const int64_t* kmod, const float* Y, int64_t ldy, int64_t Q,
                       int32_t topk, int64_t* out_idx, float* out_score, float* full, void* ws,
                       size_t ws_bytes, hipStream_t s) {
  return score_topk_impl<false>(codes, cstride, scales, N, U, kmod, Y, ldy, Q, topk, out_idx,
                                out_score, full, ws, ws_bytes, s);
}

eogp_status score_topk_tiled(const uint8_t* codes, const uint16_t* scales, int64_t N, int32_t U,
                             const int64_t* kmod, const float* Y, int64_t ldy, int64_t Q,
                             int32_t topk, int64_t* out_idx, float* out_score, float* full,
                             void* ws, size_t ws_bytes, hipStream_t s) {
  return score_topk_impl<true>(codes, 0, scales, N, U, kmod, Y, ldy, Q, topk, out_idx, out_score,
                               full, ws, ws_bytes, s);
}

// ---- scoring without a caller workspace ---------------------------------------
// For callers that cannot allocate device memory (code under graph capture,
// serving loops): the workspace of a scoring call lives in this file-scope
// array, one copy per GPU, held until the process ends. Its device address is
// looked up once per device, with that device current, and only that address
// is handed to kernels. Every call on one GPU shares the array, so calls that
// overlap on one GPU race; nothing in it has to start at zero (each call
// writes every byte it reads).
namespace {
constexpr size_t kScratchBytes = size_t(128) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

size_t score_scratch_bytes() { return kScratchBytes; }

eogp_status score_scratch(void** out) {
  int dev = 0;
  EOGP_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(EOGP_ERR_UNSUPPORTED, "score_topk_noalloc: device index out of range");
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return check_hip(e, "score_topk_noalloc: scratch address");
    if (!p) return fail(EOGP_ERR_DEVICE, "score_topk_noalloc: no scratch address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return EOGP_OK;
}

}  // namespace eogp
