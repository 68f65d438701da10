// PCA fit of the second stage (appendix on PCA fitting, Proposition
// rayleigh_ritz): the columns of P are the top-k right singular vectors of the
// uncentered first-stage coordinates Z [n, m], recovered from the n x n Gram
// matrix Z Z^T. With Z Z^T v_c = lambda_c v_c (lambda descending, |v_c| = 1):
//   p_c = Z^T v_c / sqrt(lambda_c),   mu_c = lambda_c / n
// (mu_c are the eigenvalues of Z^T Z / n). Each p_c is signed so that its
// largest-magnitude entry (the first such on ties) is positive.
//
// Arithmetic. Both contractions (the Gram matrix and Z^T V) run in fp64 on
// v_mfma_f64_16x16x4_f64 (fp32 inputs are exact in fp64), so the only
// approximation before the final rounding of P to fp32 is the eigensolver's.
// The symmetric eigendecomposition of the Gram matrix is rocSOLVER's, working
// in a slice of the caller's workspace: divide and conquer over the whole
// spectrum (dsyevd) when k > n/4, the top-k index range (dsyevdx) otherwise.
//
// Steps: k_gemm64 (G = Z Z^T, fp64) -> dsyevd/dsyevdx -> k_scale_vectors (reorder to
// descending, divide by sqrt(lambda), mu) -> k_gemm64 (P^T = V_s Z, fp32 out)
// -> k_sign_rule.
#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>

#include "common.h"
#include "pcafit_layout.h"
#include "timing.h"

namespace eogp {
namespace {

typedef double f64x4 __attribute__((ext_vector_type(4)));

// ---- fp64 MFMA contraction ------------------------------------------------------
// C[M][N] = A[M][K] * op(B): BT -> B is [N][K] (C = A B^T), else B is [K][N].
// A and B are row-major with leading dimensions lda, ldb (elements); TA is
// float or double, B is float; TC is the output type. A 256-thread workgroup
// computes a 64 x 64 tile, each wave 32 x 32 as 2 x 2 blocks of 16 x 16; K
// advances 16 at a time through LDS ([k][row] layout, so the 16 lanes that
// read one MFMA operand column touch 16 consecutive doubles). All loads are
// bounds-checked (zeros outside), all stores too.
constexpr int G64_BM = 64, G64_BN = 64, G64_BK = 16;

template <typename TA, bool BT, typename TC>
__global__ __launch_bounds__(256) void k_gemm64(const TA* __restrict__ A, int64_t lda,
                                                const float* __restrict__ B, int64_t ldb,
                                                TC* __restrict__ C, int64_t ldc, int64_t M,
                                                int64_t N, int64_t K) {
  __shared__ double As[G64_BK][G64_BM + 2];
  __shared__ double Bs[G64_BK][G64_BN + 2];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int64_t m0 = (int64_t)blockIdx.y * G64_BM, n0 = (int64_t)blockIdx.x * G64_BN;
  const int wm = (wid >> 1) * 32, wn = (wid & 1) * 32;
  f64x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  for (int64_t k0 = 0; k0 < K; k0 += G64_BK) {
    // A tile: 64 rows x 16 k, 4 consecutive k per thread
    {
      const int r = tid >> 2, kq = 4 * (tid & 3);
      const int64_t row = m0 + r;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t kk = k0 + kq + e;
        As[kq + e][r] = (row < M && kk < K) ? (double)A[row * lda + kk] : 0.0;
      }
    }
    if constexpr (BT) {
      const int r = tid >> 2, kq = 4 * (tid & 3);
      const int64_t col = n0 + r;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t kk = k0 + kq + e;
        Bs[kq + e][r] = (col < N && kk < K) ? (double)B[col * ldb + kk] : 0.0;
      }
    } else {
      const int kr = tid >> 4, cq = 4 * (tid & 15);
      const int64_t kk = k0 + kr;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t col = n0 + cq + e;
        Bs[kr][cq + e] = (kk < K && col < N) ? (double)B[kk * ldb + col] : 0.0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < G64_BK; ks += 4) {
      // operand layout: lane l holds A[row l % 16][k l / 16] and B[k l / 16][col l % 16]
      double a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = As[ks + (lane >> 4)][wm + 16 * i + (lane & 15)];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = Bs[ks + (lane >> 4)][wn + 16 * j + (lane & 15)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  // acc[i][j][r] holds C[l / 16 + 4 r][l % 16] of block (i, j) (rows
  // interleaved by lane group; checked with a layout probe)
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn + 16 * j + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + wm + 16 * i + (lane >> 4) + 4 * r;
        if (row < M && col < N) C[row * ldc + col] = (TC)acc[i][j][r];
      }
    }
}

template <typename TA, bool BT, typename TC>
void gemm64(const TA* A, int64_t lda, const float* B, int64_t ldb, TC* C, int64_t ldc, int64_t M,
            int64_t N, int64_t K, hipStream_t s) {
  const dim3 grid((unsigned)ceil_div(N, G64_BN), (unsigned)ceil_div(M, G64_BM));
  hipLaunchKernelGGL((k_gemm64<TA, BT, TC>), grid, dim3(256), 0, s, A, lda, B, ldb, C, ldc, M, N, K);
}

// V_s[c][i] = V[(top-c) n + i] / sqrt(W[top-c]) (eigenvalues ascending in W),
// mu[c] = W[top-c] / n; bad = 1 if an eigenvalue used is not above 1e-12 of
// the largest (Z is then numerically of rank < k).
// `top` is the position of the largest eigenvalue in W (and of its vector
// among the columns of V): k - 1 for the index-range solver, n - 1 for the
// full one.
__global__ void k_scale_vectors(const double* __restrict__ V, const double* __restrict__ W,
                                int64_t n, int64_t top, double* __restrict__ Vs,
                                float* __restrict__ mu, int* __restrict__ bad) {
  const int64_t c = blockIdx.y;
  const double lam = W[top - c];
  const bool ok = lam > 1e-12 * W[top];
  const double inv = ok ? 1.0 / sqrt(lam) : 0.0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    mu[c] = (float)(lam / (double)n);
    if (!ok) *bad = 1;
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    Vs[c * n + i] = V[(top - c) * n + i] * inv;
}

__global__ void k_zero_ints(int* p, int n) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = 0;
}
__global__ void k_set_int(int* p, int v) { *p = v; }

// Per row c of P^T: the first index of the largest magnitude; negate the row
// if that entry is negative.
__global__ __launch_bounds__(256) void k_sign_rule(float* __restrict__ Pt, int64_t ldp, int64_t m) {
  __shared__ float sv[256];
  __shared__ int64_t si[256];
  float* row = Pt + (int64_t)blockIdx.x * ldp;
  float best = -1.f;
  int64_t bi = 0;
  for (int64_t j = threadIdx.x; j < m; j += 256) {
    const float a = fabsf(row[j]);
    if (a > best) { best = a; bi = j; }        // j increases: keeps the first on ties
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) {
      const float o = sv[threadIdx.x + off];
      const int64_t oi = si[threadIdx.x + off];
      if (o > sv[threadIdx.x] || (o == sv[threadIdx.x] && oi < si[threadIdx.x])) {
        sv[threadIdx.x] = o;
        si[threadIdx.x] = oi;
      }
    }
    __syncthreads();
  }
  const bool flip = row[si[0]] < 0.f;
  __syncthreads();
  if (flip)
    for (int64_t j = threadIdx.x; j < m; j += 256) row[j] = -row[j];
}

// One rocBLAS handle per device (created on first use; the eigensolver's
// workspace is always the caller's, set before each call).
rocblas_handle solver_handle(eogp_status* st) {
  static std::mutex mu;
  static std::map<int, rocblas_handle> handles;
  std::lock_guard<std::mutex> lock(mu);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    *st = fail(EOGP_ERR_DEVICE, "pca_fit: no HIP device");
    return nullptr;
  }
  auto it = handles.find(dev);
  if (it != handles.end()) return it->second;
  rocblas_handle h = nullptr;
  if (rocblas_create_handle(&h) != rocblas_status_success) {
    *st = fail(EOGP_ERR_DEVICE, "pca_fit: rocblas_create_handle failed");
    return nullptr;
  }
  handles[dev] = h;
  return h;
}

// The full divide-and-conquer solver (dsyevd) when many vectors are asked
// for; the index-range solver (dsyevdx) for few.
bool full_solver(int64_t n, int64_t k) { return 4 * k > n; }

// Device memory the eigensolver asks for (query mode: nothing runs; the
// pointers are only checked for being non-null).
eogp_status solver_bytes(int64_t n, int64_t k, size_t* out) {
  eogp_status st = EOGP_OK;
  rocblas_handle h = solver_handle(&st);
  if (!h) return st;
  double* dummy = reinterpret_cast<double*>(alignof(double) * 32);
  rocblas_int* idummy = reinterpret_cast<rocblas_int*>(alignof(double) * 32);
  if (rocblas_start_device_memory_size_query(h) != rocblas_status_success)
    return fail(EOGP_ERR_DEVICE, "pca_fit: workspace query failed");
  if (full_solver(n, k))
    (void)rocsolver_dsyevd(h, rocblas_evect_original, rocblas_fill_lower, (rocblas_int)n, dummy,
                           (rocblas_int)n, dummy, dummy, idummy);
  else
    (void)rocsolver_dsyevdx(h, rocblas_evect_original, rocblas_erange_index, rocblas_fill_lower,
                            (rocblas_int)n, dummy, (rocblas_int)n, 0.0, 0.0, (rocblas_int)(n - k + 1),
                            (rocblas_int)n, idummy, dummy, dummy, (rocblas_int)n, idummy);
  size_t sz = 0;
  if (rocblas_stop_device_memory_size_query(h, &sz) != rocblas_status_success)
    return fail(EOGP_ERR_DEVICE, "pca_fit: workspace query failed");
  *out = sz;
  return EOGP_OK;
}

}  // namespace

size_t pca_fit_ws(int64_t n, int64_t m, int64_t k) {
  (void)m;
  size_t sb = 0;
  if (solver_bytes(n, k, &sb) != EOGP_OK) return 0;
  return fit_layout(n, k, sb).total;
}

eogp_status pca_fit(const float* Z, int64_t ldz, int64_t n, int64_t m, int64_t k, float* Pt,
                    int64_t ldp, float* mu, void* ws, size_t ws_bytes, hipStream_t s) {
  size_t sb = 0;
  eogp_status st = solver_bytes(n, k, &sb);
  if (st != EOGP_OK) return st;
  const FitLayout L = fit_layout(n, k, sb);
  if (ws_bytes < L.total) return fail(EOGP_ERR_WORKSPACE, "pca_fit: workspace too small");
  char* base = static_cast<char*>(ws);
  double* G = reinterpret_cast<double*>(base + L.g);
  double* W = reinterpret_cast<double*>(base + L.w);
  double* V = reinterpret_cast<double*>(base + L.v);
  double* Vs = reinterpret_cast<double*>(base + L.vs);
  int* ints = reinterpret_cast<int*>(base + L.ints);   // nev, info, bad

  {
    timing::Scope ts(EOGP_KT_PCA_FIT, s);
    hipLaunchKernelGGL(k_zero_ints, dim3(1), dim3(64), 0, s, ints, 4);
    gemm64<float, true, double>(Z, ldz, Z, ldz, G, n, n, n, m, s);   // G = Z Z^T
    EOGP_LAUNCH_CHECK("pca_fit gram");
  }
  st = EOGP_OK;
  rocblas_handle h = solver_handle(&st);
  if (!h) return st;
  if (rocblas_set_stream(h, s) != rocblas_status_success ||
      rocblas_set_workspace(h, sb ? base + L.solver : nullptr, sb) != rocblas_status_success)
    return fail(EOGP_ERR_DEVICE, "pca_fit: rocBLAS stream/workspace setup failed");
  // full: eigenvectors overwrite G (all n, ascending), V holds the
  // off-diagonal scratch; index range: the top k vectors land in V
  const bool full = full_solver(n, k);
  const rocblas_status rs =
      full ? rocsolver_dsyevd(h, rocblas_evect_original, rocblas_fill_lower, (rocblas_int)n, G,
                              (rocblas_int)n, W, V, ints + 1)
           : rocsolver_dsyevdx(h, rocblas_evect_original, rocblas_erange_index, rocblas_fill_lower,
                               (rocblas_int)n, G, (rocblas_int)n, 0.0, 0.0,
                               (rocblas_int)(n - k + 1), (rocblas_int)n, ints + 0, W, V,
                               (rocblas_int)n, ints + 1);
  (void)rocblas_set_workspace(h, nullptr, 0);
  if (rs != rocblas_status_success) return fail(EOGP_ERR_DEVICE, "pca_fit: the rocSOLVER call failed");
  {
    timing::Scope ts(EOGP_KT_PCA_FIT, s);
    if (full) hipLaunchKernelGGL(k_set_int, dim3(1), dim3(1), 0, s, ints + 0, (int)k);
    hipLaunchKernelGGL(k_scale_vectors, dim3((unsigned)std::min<int64_t>(ceil_div(n, 256), 64), (unsigned)k),
                       dim3(256), 0, s, full ? G : V, W, n, full ? n - 1 : k - 1, Vs, mu, ints + 2);
    gemm64<double, false, float>(Vs, n, Z, ldz, Pt, ldp, k, m, n, s);   // P^T = V_s Z
    hipLaunchKernelGGL(k_sign_rule, dim3((unsigned)k), dim3(256), 0, s, Pt, ldp, m);
    EOGP_LAUNCH_CHECK("pca_fit projection");
  }
  int hv[4] = {0, 0, 0, 0};
  EOGP_HIP(hipMemcpyAsync(hv, ints, 4 * sizeof(int), hipMemcpyDeviceToHost, s));
  EOGP_HIP(hipStreamSynchronize(s));
  if (hv[1] != 0) return fail(EOGP_ERR_DEVICE, "pca_fit: the eigensolver did not converge");
  // fewer vectors than asked for happens when trailing eigenvalues collapse
  // at zero: Z has fewer than k nonzero principal directions
  if (hv[0] != (int)k || hv[2] != 0)
    return fail(EOGP_ERR_INVALID, "pca_fit: Z has fewer than k nonzero principal directions");
  return EOGP_OK;
}

}  // namespace eogp
