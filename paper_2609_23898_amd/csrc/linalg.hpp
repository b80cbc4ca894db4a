// Small dense fp64 linear algebra for plan construction on the host.
// Matrices are row-major std::vector<double>; sizes here are at most a few
// thousand rows by a few hundred columns.
#pragma once

#include <cstddef>
#include <vector>

namespace cerar {
namespace la {

using Mat = std::vector<double>;

// C (m x n) = A (m x k) * B (k x n)
void matmul(const double *A, const double *B, double *C, int m, int k, int n);

// In-place inverse of the n x n matrix A by LU with partial pivoting.
// Returns false when a pivot is exactly zero or the result is not finite.
bool inverse(double *A, int n);

// Solves A X = B (A n x n, B n x m, row-major); X overwrites B.
bool solve(const double *A, int n, double *B, int m);

// Least squares: X (n x k) = argmin ||A X - B||_F, A m x n with m >= n and
// full column rank, via Householder QR.  Returns false on rank deficiency.
bool lstsq(const double *A, int m, int n, const double *B, int k, double *X);

// Default cap on the sweeps of one-sided Jacobi.
constexpr int kJacobiSweeps = 80;

// Singular values of A (m x n), descending.  Tall inputs are reduced by QR
// first, then one-sided Jacobi (Hestenes) runs on the small factor.  When
// converged is non-null, it is set to false if Jacobi reached max_sweeps
// without converging (and left alone otherwise).
std::vector<double> singular_values(const double *A, int m, int n, int max_sweeps = kJacobiSweeps,
                                    bool *converged = nullptr);

// Full SVD of a square n x n matrix: A = P diag(s) Q^T with s descending,
// P and Q orthogonal (row-major n x n).  One-sided Jacobi.  Returns false if
// it reached max_sweeps without converging.
bool svd_square(const double *A, int n, double *P, double *s, double *Q, int max_sweeps = kJacobiSweeps);

double frobenius2(const double *A, size_t count);

}  // namespace la
}  // namespace cerar
