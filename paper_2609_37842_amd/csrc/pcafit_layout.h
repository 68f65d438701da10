// Workspace layout of the PCA fit (plain C++, no device code, so that a host
// test can check it): the status words, the eigensolver's own workspace, the
// n x n Gram matrix G, its n eigenvalues W, the n x n eigenvector array V and
// the k selected vectors V_s, each region starting on a 256-byte boundary.
#pragma once
#include <cstddef>
#include <cstdint>

namespace eogp {

struct FitLayout {
  size_t g, w, v, vs, ints, solver, total;
};

// The eigenvector array handed to the solver gets all n columns: rocSOLVER
// documents that the columns of its eigenvector output may serve as internal
// workspace, so an array sized for the k requested vectors could be written
// past its end (over V_s, the status words and the solver workspace).
inline FitLayout fit_layout(int64_t n, int64_t k, size_t solver_bytes) {
  auto align = [](size_t x) { return (x + 255) & ~size_t(255); };
  FitLayout L;
  size_t o = 0;
  auto take = [&](size_t b) { size_t r = o; o = align(o + b); return r; };
  L.ints = take(4 * sizeof(int));
  L.solver = take(solver_bytes);
  L.g = take((size_t)n * n * 8);
  L.w = take((size_t)n * 8);
  L.v = take((size_t)n * n * 8);
  L.vs = take((size_t)n * k * 8);
  L.total = o;
  return L;
}

}  // namespace eogp
