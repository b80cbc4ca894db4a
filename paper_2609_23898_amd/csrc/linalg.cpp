#include "linalg.hpp"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace cerar {
namespace la {

void matmul(const double *A, const double *B, double *C, int m, int k, int n) {
    std::fill(C, C + (size_t)m * n, 0.0);
    for (int i = 0; i < m; ++i) {
        double *ci = C + (size_t)i * n;
        for (int t = 0; t < k; ++t) {
            const double a = A[(size_t)i * k + t];
            if (a == 0.0) continue;
            const double *bt = B + (size_t)t * n;
            for (int j = 0; j < n; ++j) ci[j] += a * bt[j];
        }
    }
}

double frobenius2(const double *A, size_t count) {
    double s = 0.0;
    for (size_t i = 0; i < count; ++i) s += A[i] * A[i];
    return s;
}

// LU factorisation with partial pivoting, in place; piv[i] = row swapped into i.
static bool lu(double *A, int n, std::vector<int> &piv) {
    piv.resize(n);
    for (int k = 0; k < n; ++k) {
        int p = k;
        double best = std::fabs(A[(size_t)k * n + k]);
        for (int i = k + 1; i < n; ++i) {
            double v = std::fabs(A[(size_t)i * n + k]);
            if (v > best) { best = v; p = i; }
        }
        piv[k] = p;
        if (best == 0.0 || !std::isfinite(best)) return false;
        if (p != k)
            for (int j = 0; j < n; ++j) std::swap(A[(size_t)k * n + j], A[(size_t)p * n + j]);
        const double inv = 1.0 / A[(size_t)k * n + k];
        for (int i = k + 1; i < n; ++i) {
            double f = A[(size_t)i * n + k] * inv;
            A[(size_t)i * n + k] = f;
            if (f == 0.0) continue;
            for (int j = k + 1; j < n; ++j) A[(size_t)i * n + j] -= f * A[(size_t)k * n + j];
        }
    }
    return true;
}

// Solves with an LU factor: B (n x m) overwritten by the solution.
static void lu_solve(const double *LU, int n, const std::vector<int> &piv, double *B, int m) {
    for (int k = 0; k < n; ++k)
        if (piv[k] != k)
            for (int j = 0; j < m; ++j) std::swap(B[(size_t)k * m + j], B[(size_t)piv[k] * m + j]);
    for (int i = 0; i < n; ++i)                 // forward: unit lower
        for (int t = 0; t < i; ++t) {
            const double l = LU[(size_t)i * n + t];
            if (l == 0.0) continue;
            for (int j = 0; j < m; ++j) B[(size_t)i * m + j] -= l * B[(size_t)t * m + j];
        }
    for (int i = n - 1; i >= 0; --i) {          // backward: upper
        for (int t = i + 1; t < n; ++t) {
            const double u = LU[(size_t)i * n + t];
            if (u == 0.0) continue;
            for (int j = 0; j < m; ++j) B[(size_t)i * m + j] -= u * B[(size_t)t * m + j];
        }
        const double inv = 1.0 / LU[(size_t)i * n + i];
        for (int j = 0; j < m; ++j) B[(size_t)i * m + j] *= inv;
    }
}

bool solve(const double *A, int n, double *B, int m) {
    Mat LU(A, A + (size_t)n * n);
    std::vector<int> piv;
    if (!lu(LU.data(), n, piv)) return false;
    lu_solve(LU.data(), n, piv, B, m);
    for (size_t i = 0; i < (size_t)n * m; ++i)
        if (!std::isfinite(B[i])) return false;
    return true;
}

bool inverse(double *A, int n) {
    Mat I((size_t)n * n, 0.0);
    for (int i = 0; i < n; ++i) I[(size_t)i * n + i] = 1.0;
    if (!solve(A, n, I.data(), n)) return false;
    std::copy(I.begin(), I.end(), A);
    return true;
}

// Householder QR of the column-major m x n matrix Q (in place): on return the
// upper triangle holds R, below-diagonal entries and tau describe the
// reflectors H_j = I - tau_j v_j v_j^T with v_j[j] = 1.
static bool householder_qr(double *A, int m, int n, std::vector<double> &tau) {
    tau.assign(n, 0.0);
    for (int j = 0; j < n; ++j) {
        double *col = A + (size_t)j * m;
        double norm = 0.0;
        for (int i = j; i < m; ++i) norm += col[i] * col[i];
        norm = std::sqrt(norm);
        if (norm == 0.0) return false;
        const double alpha = col[j] >= 0 ? -norm : norm;
        const double v0 = col[j] - alpha;
        // v = (col[j..] - alpha e_1) / v0, so v[j] = 1
        for (int i = j + 1; i < m; ++i) col[i] /= v0;
        tau[j] = -v0 / alpha;
        col[j] = alpha;
        for (int k = j + 1; k < n; ++k) {       // apply H_j to the remaining columns
            double *ck = A + (size_t)k * m;
            double s = ck[j];
            for (int i = j + 1; i < m; ++i) s += col[i] * ck[i];
            s *= tau[j];
            ck[j] -= s;
            for (int i = j + 1; i < m; ++i) ck[i] -= s * col[i];
        }
    }
    return true;
}

bool lstsq(const double *A, int m, int n, const double *B, int k, double *X) {
    Mat Ac((size_t)m * n), Bc((size_t)m * k);         // column-major copies
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < n; ++j) Ac[(size_t)j * m + i] = A[(size_t)i * n + j];
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < k; ++j) Bc[(size_t)j * m + i] = B[(size_t)i * k + j];
    std::vector<double> tau;
    if (!householder_qr(Ac.data(), m, n, tau)) return false;
    for (int c = 0; c < k; ++c) {                     // Bc <- Q^T Bc
        double *b = Bc.data() + (size_t)c * m;
        for (int j = 0; j < n; ++j) {
            const double *v = Ac.data() + (size_t)j * m;
            double s = b[j];
            for (int i = j + 1; i < m; ++i) s += v[i] * b[i];
            s *= tau[j];
            b[j] -= s;
            for (int i = j + 1; i < m; ++i) b[i] -= s * v[i];
        }
        for (int j = n - 1; j >= 0; --j) {            // R x = (Q^T b)[0..n)
            double s = b[j];
            for (int t = j + 1; t < n; ++t) s -= Ac[(size_t)t * m + j] * X[(size_t)t * k + c];
            const double r = Ac[(size_t)j * m + j];
            if (r == 0.0) return false;
            X[(size_t)j * k + c] = s / r;
        }
    }
    for (size_t i = 0; i < (size_t)n * k; ++i)
        if (!std::isfinite(X[i])) return false;
    return true;
}

// One-sided Jacobi on the columns of the column-major m x n matrix W (m >= n).
// Columns become mutually orthogonal; V (column-major n x n) accumulates the
// rotations when non-null.  Returns false when a sweep still rotated after
// max_sweeps sweeps (the columns are then not orthogonal to working accuracy).
static bool jacobi_columns(double *W, int m, int n, double *V, int max_sweeps) {
    if (V) {
        std::fill(V, V + (size_t)n * n, 0.0);
        for (int i = 0; i < n; ++i) V[(size_t)i * n + i] = 1.0;
    }
    const double tol = 1e-15;
    for (int sweep = 0; sweep < max_sweeps; ++sweep) {
        bool rotated = false;
        for (int p = 0; p < n - 1; ++p) {
            for (int q = p + 1; q < n; ++q) {
                double *ap = W + (size_t)p * m, *aq = W + (size_t)q * m;
                double alpha = 0, beta = 0, gamma = 0;
                for (int i = 0; i < m; ++i) {
                    alpha += ap[i] * ap[i];
                    beta += aq[i] * aq[i];
                    gamma += ap[i] * aq[i];
                }
                if (gamma == 0.0 || std::fabs(gamma) <= tol * std::sqrt(alpha * beta)) continue;
                rotated = true;
                const double zeta = (beta - alpha) / (2.0 * gamma);
                const double t = (zeta >= 0 ? 1.0 : -1.0) / (std::fabs(zeta) + std::sqrt(1.0 + zeta * zeta));
                const double cs = 1.0 / std::sqrt(1.0 + t * t);
                const double sn = cs * t;
                for (int i = 0; i < m; ++i) {
                    const double x = ap[i], y = aq[i];
                    ap[i] = cs * x - sn * y;
                    aq[i] = sn * x + cs * y;
                }
                if (V) {
                    double *vp = V + (size_t)p * n, *vq = V + (size_t)q * n;
                    for (int i = 0; i < n; ++i) {
                        const double x = vp[i], y = vq[i];
                        vp[i] = cs * x - sn * y;
                        vq[i] = sn * x + cs * y;
                    }
                }
            }
        }
        if (!rotated) return true;
    }
    return n < 2;
}

std::vector<double> singular_values(const double *A, int m, int n, int max_sweeps, bool *converged) {
    // Work on the taller orientation, column-major.
    const bool trans = m < n;
    const int mm = trans ? n : m, nn = trans ? m : n;
    Mat W((size_t)mm * nn);
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < n; ++j) {
            if (!trans) W[(size_t)j * mm + i] = A[(size_t)i * n + j];
            else W[(size_t)i * mm + j] = A[(size_t)i * n + j];
        }
    int rows = mm;
    if (mm > 2 * nn) {                                 // reduce to the n x n R factor
        std::vector<double> tau;
        Mat Rf((size_t)nn * nn, 0.0);
        if (householder_qr(W.data(), mm, nn, tau)) {
            for (int j = 0; j < nn; ++j)
                for (int i = 0; i <= j; ++i) Rf[(size_t)j * nn + i] = W[(size_t)j * mm + i];
            W.swap(Rf);
            rows = nn;
        } else {                                       // exactly rank deficient: plain Jacobi
            W.assign(W.size(), 0.0);
            for (int i = 0; i < m; ++i)
                for (int j = 0; j < n; ++j) {
                    if (!trans) W[(size_t)j * mm + i] = A[(size_t)i * n + j];
                    else W[(size_t)i * mm + j] = A[(size_t)i * n + j];
                }
        }
    }
    const bool ok = jacobi_columns(W.data(), rows, nn, nullptr, max_sweeps);
    if (!ok && converged) *converged = false;
    std::vector<double> s(nn);
    for (int j = 0; j < nn; ++j) s[j] = std::sqrt(frobenius2(W.data() + (size_t)j * rows, rows));
    std::sort(s.begin(), s.end(), std::greater<double>());
    return s;
}

bool svd_square(const double *A, int n, double *P, double *s, double *Q, int max_sweeps) {
    Mat W((size_t)n * n), V((size_t)n * n);
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) W[(size_t)j * n + i] = A[(size_t)i * n + j];
    const bool converged = jacobi_columns(W.data(), n, n, V.data(), max_sweeps);
    std::vector<double> sig(n);
    for (int j = 0; j < n; ++j) sig[j] = std::sqrt(frobenius2(W.data() + (size_t)j * n, n));
    std::vector<int> order(n);
    std::iota(order.begin(), order.end(), 0);
    std::sort(order.begin(), order.end(), [&](int a, int b) { return sig[a] > sig[b]; });
    const double smax = n > 0 ? sig[order[0]] : 0.0;
    // left vectors: normalised columns; complete any null directions by Gram-Schmidt
    Mat Pc((size_t)n * n, 0.0);
    std::vector<char> have(n, 0);
    for (int t = 0; t < n; ++t) {
        const int j = order[t];
        s[t] = sig[j];
        if (sig[j] > 1e-300 && sig[j] > smax * 1e-300) {
            for (int i = 0; i < n; ++i) Pc[(size_t)t * n + i] = W[(size_t)j * n + i] / sig[j];
            have[t] = 1;
        }
        for (int i = 0; i < n; ++i) Q[(size_t)i * n + t] = V[(size_t)j * n + i];
    }
    for (int t = 0; t < n; ++t) {
        if (have[t]) continue;
        for (int e = 0; e < n; ++e) {
            std::vector<double> v(n, 0.0);
            v[e] = 1.0;
            for (int u = 0; u < n; ++u) {
                if (!have[u]) continue;
                double d = 0;
                for (int i = 0; i < n; ++i) d += Pc[(size_t)u * n + i] * v[i];
                for (int i = 0; i < n; ++i) v[i] -= d * Pc[(size_t)u * n + i];
            }
            double nv = std::sqrt(frobenius2(v.data(), n));
            if (nv > 1e-8) {
                for (int i = 0; i < n; ++i) Pc[(size_t)t * n + i] = v[i] / nv;
                have[t] = 1;
                break;
            }
        }
    }
    for (int i = 0; i < n; ++i)
        for (int t = 0; t < n; ++t) P[(size_t)i * n + t] = Pc[(size_t)t * n + i];
    return converged;
}

}  // namespace la
}  // namespace cerar
