// MFMA contraction C[M, N] = A[M, K] * B[N, K]^T for gfx950 (both operands
// K-contiguous, fp32 accumulation). Used by the Kronecker rotations (A =
// gathered token rows of activations or output-gradients, B = a gathered
// eigenvector panel) and by the PCA projection (A = first-stage coordinates,
// B = the PCA directions).
#pragma once
#include "common.h"

namespace eogp {

// B16: bf16 or fp16 bit patterns used as the MFMA type; BF16_AS_F16: bf16 A
// widened to fp32, scaled by a_scale and rounded to fp16 while it is staged
// (fp16 MFMA; single-pass products on aligned rows only).
enum class AType : int { F32 = 0, B16 = 1, BF16_AS_F16 = 2 };

struct GemmArgs {
  // A: row r of the product reads row (a_rows ? a_rows[r] : r) of A.
  const void* A = nullptr;
  int64_t lda = 0;
  const int32_t* a_rows = nullptr;
  // fp16 operands only: fp32 A is multiplied by a_scale before rounding.
  float a_scale = 1.f;
  // B: [N][ldb] 16-bit; B_lo (optional) is the low part of a split operand.
  const uint16_t* B_hi = nullptr;
  const uint16_t* B_lo = nullptr;
  int64_t ldb = 0;
  // B is a padded panel: at least round_up(N, 256) rows and round_up(K, 32)
  // columns per row are readable, zero beyond N and K.
  bool b_padded = false;
  float* C = nullptr;
  int64_t ldc = 0;
  // Optional fp16 output instead of C, in MFMA-fragment order: product entry
  // (row, col) is stored, rounded to nearest even, at
  //   CT[((col / 32) * (ldct / 16) + row / 16) * 512 + (col % 32) * 16 + row % 16],
  // i.e. for every 32 columns and 16 rows one contiguous 1 KB block holding
  // the 32 x 16 fp16 operand of one v_mfma_*_32x32x16 (columns as MFMA rows,
  // rows as the 16-deep reduction). Every row and column of every output
  // tile is written (no bounds checks), so CT must hold round_up(N, 256)
  // columns of ldct >= round_up(M, 256) rows; ldct is a multiple of 256.
  // Single-pass products without split-K only.
  uint16_t* CT = nullptr;
  int64_t ldct = 0;
  bool ct_bf16 = false;            // CT entries are bf16 (else fp16)
  int64_t M = 0;                   // rows (upper bound if M_dev is set)
  const int32_t* M_dev = nullptr;  // device-side row count (<= M), or null
  int64_t N = 0, K = 0;
  bool n_major = false;            // unit order: N-tiles outer (share B across M)
  // Split-K unit order: splits outermost, then tiles (M or N outer per n_major),
  // so that the units running together share one K range of one operand.
  bool split_major = false;
  // Optional kXcds int32 work counters (device memory; the launch zeroes them):
  // when given, each XCD's workgroups take their units from a shared counter
  // (longest units first) instead of a fixed stride.
  int32_t* sched = nullptr;
  // Split-K scratch (host-known M only): max_splits partial [M][N] fp32 tiles.
  float* partial = nullptr;
  int max_splits = 1;
  int timing_class = EOGP_KT_ROTATION_GEMM;
};

// Launch one contraction. a_type: element type of A; a_parts: 1 = rounded to
// the MFMA type, 2 = split into high+low parts (fp32 A only); b_parts: 1 or 2
// (2 needs B_lo); f16: MFMA operands are fp16 (else bf16).
eogp_status gemm_nt(const GemmArgs& g, AType a_type, int a_parts, int b_parts, bool f16,
                    hipStream_t s);

// Two independent products in one launch (same operand types and timing
// class; put the one with the longer K first): their units share the grid, so
// the second fills the first one's last round. Applies to single-pass products
// on aligned operands without split-K, with g1.sched given (the work
// counters); anything else runs as two ordinary launches.
eogp_status gemm_nt2(const GemmArgs& g1, const GemmArgs& g2, AType a_type, int a_parts,
                     int b_parts, bool f16, hipStream_t s);

// Bytes of split-K scratch for an M x N product with up to max_splits splits.
size_t gemm_partial_bytes(int64_t M, int64_t N, int max_splits);

}  // namespace eogp
