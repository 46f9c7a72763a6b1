// fp64 Cholesky factorisation and solve of the small (ell x ell, ell <= 8) symmetric
// positive-definite systems behind Algorithm 1's minimum-norm coefficients: the Gram
// matrix X X^T (Delta >= ell) or X^T X padded with the identity (Delta < ell) of
// X = R[:, S_i].  Fully unrolled so every index is static and the matrices live in
// registers.  Shared by the coefficient kernels and the PS-side estimate.
#pragma once

#include <hip/hip_runtime.h>

namespace gcx {

// In-place Cholesky factorisation A = L L^T (lower triangle read and written).
template <int ELL>
__device__ __forceinline__ void cholesky(double (&A)[ELL][ELL]) {
#pragma unroll
  for (int c = 0; c < ELL; ++c) {
    double s = A[c][c];
#pragma unroll
    for (int q = 0; q < c; ++q) s -= A[c][q] * A[c][q];
    const double dcc = sqrt(s);
    A[c][c] = dcc;
    const double inv = 1.0 / dcc;
#pragma unroll
    for (int r = c + 1; r < ELL; ++r) {
      double v = A[r][c];
#pragma unroll
      for (int q = 0; q < c; ++q) v -= A[r][q] * A[c][q];
      A[r][c] = v * inv;
    }
  }
}

// Solve (L L^T) z = b in place, L the lower factor from cholesky().
template <int ELL>
__device__ __forceinline__ void chol_solve(const double (&Lf)[ELL][ELL], double (&b)[ELL]) {
#pragma unroll
  for (int r = 0; r < ELL; ++r) {
    double v = b[r];
#pragma unroll
    for (int q = 0; q < r; ++q) v -= Lf[r][q] * b[q];
    b[r] = v / Lf[r][r];
  }
#pragma unroll
  for (int r = ELL - 1; r >= 0; --r) {
    double v = b[r];
#pragma unroll
    for (int q = r + 1; q < ELL; ++q) v -= Lf[q][r] * b[q];
    b[r] = v / Lf[r][r];
  }
}

}  // namespace gcx
