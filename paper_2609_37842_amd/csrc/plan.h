// The retained-axis plan of one module (internal layout).
#pragma once
#include "common.h"

struct eogp_plan {
  int64_t d_out = 0, d_in = 0, m = 0;
  double damping = 0;
  int64_t n_rows = 0;      // |J|
  int64_t n_cols = 0;      // |K|
  int64_t rows_pad = 0;    // |J| rounded up to the GEMM column tile
  int64_t cols_pad = 0;    // |K| rounded up likewise
  int64_t ld_out = 0;      // panel row length for Q_S columns (>= d_out, multiple of 32)
  int64_t ld_in = 0;       // panel row length for Q_A columns (>= d_in, multiple of 32)
  int64_t n_tiles = 0;     // active 32x32 (row, column) blocks
  int64_t n_groups = 0;    // groups of active blocks sharing one operand block
  bool group_rows = true;  // groups share a row block of S~ (else a column block of A~)
  int device = 0;

  // Device arrays, all owned by the plan (one allocation, `mem`).
  void* mem = nullptr;
  int32_t* ret_flat = nullptr;   // [m]   j*d_in + k, canonical order
  float* ret_w = nullptr;        // [m]   (Lambda_r + lambda)^-1/2
  int32_t* tiles = nullptr;      // [n_tiles][4] = {row block, col block, entry begin, entry end}
  int32_t* groups = nullptr;     // [n_groups][4] = {first position in gtiles, count, shared block, 0}
  int32_t* gtiles = nullptr;     // [n_tiles] tile indices, group by group
  int32_t* ent_r = nullptr;      // [m]   retained position of each entry, grouped by tile
  uint16_t* ent_loc = nullptr;   // [m]   (row in block) * 32 + (col in block)
  int32_t* ent_pos = nullptr;    // [m]   entry index of each retained position (inverse of ent_r)
  uint16_t* qs_hi = nullptr;     // [rows_pad][ld_out] bf16: Q_S[:, J[p]] high part
  uint16_t* qs_lo = nullptr;     // [rows_pad][ld_out] bf16: low part
  uint16_t* qa_hi = nullptr;     // [cols_pad][ld_in]  bf16: Q_A[:, K[p]] high part
  uint16_t* qa_lo = nullptr;     // [cols_pad][ld_in]
  uint16_t* qs_f16 = nullptr;    // [rows_pad][ld_out] fp16: Q_S[:, J[p]] rounded once
  uint16_t* qa_f16 = nullptr;    // [cols_pad][ld_in]  fp16: Q_A[:, K[p]] rounded once

  // fp16 mode: inputs are multiplied by 2^e before rounding to fp16, and the
  // coordinates by 2^-(e_acts + e_grads) (exact while nothing overflows).
  int32_t e_acts = 0, e_grads = 0;
};

namespace eogp {
constexpr int kPanelTile = 256;   // widest GEMM column tile; panels are padded to it
constexpr int kBlk = 32;          // retained-product block edge
constexpr int kRetGroup = 2;      // active blocks per group at most

eogp_status build_plan(const float* eigvals, int64_t d_out, int64_t d_in, double damping,
                       int64_t m, const float* Q_A, const float* Q_S, hipStream_t s,
                       eogp_plan** out);
void free_plan(eogp_plan* p);
// Panels of a whole eigenbasis (every column, in order): the rows_pad x ld
// bf16 high/low and fp16 images of Q^T, zero beyond d. `list` is d ints of
// scratch.
void basis_panels(const float* Q, int64_t d, int64_t rows_pad, int64_t ld, int* list,
                  uint16_t* hi, uint16_t* lo, uint16_t* h16, hipStream_t s);
}  // namespace eogp
