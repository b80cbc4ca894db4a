// Host fp64 plan construction for CERAR (Sec. II-B to II-D) and the
// slot-ownership tables of the single-GPU handoff ring.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <memory>
#include <set>
#include <thread>

#include "cerar_internal.hpp"
#include "linalg.hpp"

namespace cerar {

// A fixed buffer, so that recording an error never allocates or throws.
static thread_local char g_last_error[512];

int fail(int status, const char *fmt, ...) noexcept {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

void clear_error() noexcept { g_last_error[0] = 0; }

namespace {

const double kNaN = std::numeric_limits<double>::quiet_NaN();

// ---- seeded base matrix: splitmix64 (Steele, Lea & Flood 2014) + Box-Muller
struct SplitMix64 {
    uint64_t state;
    uint64_t next() {
        uint64_t z = (state += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    double uniform() { return ((double)(next() >> 11) + 0.5) * 0x1.0p-53; }
};

std::vector<double> gaussian_base(uint64_t seed, int N, int c) {
    SplitMix64 g{seed};
    std::vector<double> B((size_t)N * c);
    for (size_t i = 0; i < B.size(); i += 2) {
        const double r = std::sqrt(-2.0 * std::log(g.uniform()));
        const double th = 2.0 * M_PI * g.uniform();
        B[i] = r * std::cos(th);
        if (i + 1 < B.size()) B[i + 1] = r * std::sin(th);
    }
    return B;
}

std::vector<double> chebyshev_nodes(int c) {
    std::vector<double> x(c);
    for (int j = 1; j <= c; ++j) x[j - 1] = std::cos((2.0 * j - 1.0) * M_PI / (2.0 * c));
    return x;
}

// Runs f(k) for k in [0, n) on up to hardware_concurrency threads, thread t
// taking k = t, t + nt, ...  The share of a thread that cannot be started runs
// on the calling thread.  An exception thrown by f on any thread is rethrown
// here, after every thread has been joined.
template <class F>
void parallel_for(int n, F f) {
    const int nt = (int)std::min<unsigned>(std::max(1u, std::thread::hardware_concurrency()), (unsigned)std::max(n, 0));
    if (nt <= 1) {
        for (int k = 0; k < n; ++k) f(k);
        return;
    }
    std::exception_ptr err;
    std::mutex mu;
    auto share = [&](int t) {
        try {
            for (int k = t; k < n; k += nt) f(k);
        } catch (...) {
            std::lock_guard<std::mutex> g(mu);
            if (!err) err = std::current_exception();
        }
    };
    std::vector<std::thread> th;
    th.reserve(nt);
    int started = 0;
    try {
        for (; started < nt; ++started) th.emplace_back(share, started);
    } catch (...) {
    }
    for (int t = started; t < nt; ++t) share(t);
    for (auto &x : th) x.join();
    if (err) std::rethrow_exception(err);
}

// ---- multiplicative perturbation construction (eqs. (8)-(11)) -------------

// a_idx = b_r D^m, idx = r + m N (eq. (8)); Dpow[m + 1] = D^m for m >= -1.
struct Sequence {
    int N, c;
    const std::vector<double> *B;
    std::vector<std::vector<double>> Dpow;
    void row(int idx, double *out) const {
        int m = idx >= 0 ? idx / N : -((-idx + N - 1) / N);
        int r = idx - m * N;
        const std::vector<double> &P = Dpow[m + 1];
        la::matmul(B->data() + (size_t)r * c, P.data(), out, 1, c, c);
    }
};

bool make_sequence(const std::vector<double> &B, const std::vector<double> &D, int N, int c,
                   int max_idx, Sequence &s) {
    s.N = N;
    s.c = c;
    s.B = &B;
    const int mmax = max_idx / N + 1;
    s.Dpow.assign(mmax + 2, std::vector<double>((size_t)c * c, 0.0));
    std::vector<double> Dinv = D;
    if (!la::inverse(Dinv.data(), c)) return false;
    s.Dpow[0] = Dinv;                                            // D^{-1}
    for (int i = 0; i < c; ++i) s.Dpow[1][(size_t)i * c + i] = 1.0;   // D^0
    for (int m = 1; m <= mmax; ++m) la::matmul(s.Dpow[m].data(), D.data(), s.Dpow[m + 1].data(), c, c, c);
    return true;
}

// U_k = A_{N-1-k}^{-1} (eq. (10)), R_i[l,:] = a_{l-i} (eq. (11)).
int mpc_plan(cerar_plan *p) {
    const int N = p->N, c = p->c, L = p->L;
    Sequence s;
    if (!make_sequence(p->B, p->D, N, c, L + N, s))
        return fail(CERAR_E_SINGULAR, "perturbation matrix D is singular");
    p->U.assign((size_t)N * c * c, 0.0);
    p->R.assign((size_t)N * (L + 1) * c, 0.0);
    for (int k = 0; k < N; ++k) {
        double *Uk = p->U.data() + (size_t)k * c * c;
        const int ell = N - 1 - k;
        for (int t = 0; t < c; ++t) s.row(ell + t, Uk + (size_t)t * c);
        if (!la::inverse(Uk, c))
            return fail(CERAR_E_SINGULAR, "window A_%d of the construction is singular", ell);
    }
    for (int i = 0; i < N; ++i)
        for (int l = 0; l <= L; ++l) s.row(l - i, p->R.data() + ((size_t)i * (L + 1) + l) * c);
    return CERAR_OK;
}

// ---- coefficient maps and Phi (eqs. (6), (7)) ------------------------------

// Block r of M_i R_i is U_{i+r} W_{N-1-r}(R_i) (c x c).
void block_product(const cerar_plan *p, const std::vector<double> &U, const std::vector<double> &R,
                   int i, int r, double *out) {
    const int N = p->N, c = p->c, L = p->L;
    const double *Uk = U.data() + (size_t)((i + r) % N) * c * c;
    const double *W = R.data() + ((size_t)i * (L + 1) + (N - 1 - r)) * c;
    la::matmul(Uk, W, out, c, c, c);
}

double phi_of(const cerar_plan *p, const std::vector<double> &U, const std::vector<double> &R) {
    const int N = p->N, c = p->c;
    std::vector<double> blk((size_t)c * c);
    double total = 0.0;
    for (int i = 0; i < N; ++i)
        for (int r = 0; r < N; ++r) {
            block_product(p, U, R, i, r, blk.data());
            for (int a = 0; a < c; ++a) blk[(size_t)a * c + a] -= 1.0;
            total += la::frobenius2(blk.data(), blk.size());
        }
    return total;
}

std::vector<double> coefficient_map(const cerar_plan *p, const std::vector<double> &U, int i) {
    const int N = p->N, c = p->c, L = p->L;
    std::vector<double> M((size_t)N * c * (L + 1), 0.0);
    for (int r = 0; r < N; ++r) {
        const double *Uk = U.data() + (size_t)((i + r) % N) * c * c;
        const int col0 = N - 1 - r;
        for (int a = 0; a < c; ++a)
            for (int b = 0; b < c; ++b) M[((size_t)r * c + a) * (L + 1) + col0 + b] = Uk[(size_t)a * c + b];
    }
    return M;
}

// ---- constrained design (Sec. II-D): U-step, R-step, projection -----------

// U_k (sum_r W_r W_r^T) = sum_r W_r^T with W_r = W_{N-1-r}(R_{k-r}).
bool u_step(const cerar_plan *p, const std::vector<double> &R, std::vector<double> &U) {
    const int N = p->N, c = p->c, L = p->L;
    bool ok = true;
    std::mutex mu;
    parallel_for(N, [&](int k) {
        std::vector<double> gram((size_t)c * c, 0.0), rhsT((size_t)c * c, 0.0);
        for (int r = 0; r < N; ++r) {
            const int owner = ((k - r) % N + N) % N;
            const double *W = R.data() + ((size_t)owner * (L + 1) + (N - 1 - r)) * c;
            for (int a = 0; a < c; ++a)
                for (int b = 0; b < c; ++b) {
                    double s = 0.0;
                    for (int t = 0; t < c; ++t) s += W[(size_t)a * c + t] * W[(size_t)b * c + t];
                    gram[(size_t)a * c + b] += s;
                }
            for (int a = 0; a < c * c; ++a) rhsT[a] += W[a];      // (W^T)^T = W
        }
        // gram^T U_k^T = (sum W^T)^T = sum W ; gram is symmetric
        if (!la::solve(gram.data(), c, rhsT.data(), c)) {
            std::lock_guard<std::mutex> g(mu);
            ok = false;
            return;
        }
        double *Uk = U.data() + (size_t)k * c * c;
        for (int a = 0; a < c; ++a)
            for (int b = 0; b < c; ++b) Uk[(size_t)a * c + b] = rhsT[(size_t)b * c + a];
    });
    return ok;
}

// R_i = argmin ||M_i R - T||_F.
bool r_step(const cerar_plan *p, const std::vector<double> &U, std::vector<double> &R) {
    const int N = p->N, c = p->c, L = p->L;
    std::vector<double> T((size_t)N * c * c, 0.0);
    for (int r = 0; r < N; ++r)
        for (int a = 0; a < c; ++a) T[((size_t)r * c + a) * c + a] = 1.0;
    bool ok = true;
    std::mutex mu;
    parallel_for(N, [&](int i) {
        std::vector<double> M = coefficient_map(p, U, i);
        if (!la::lstsq(M.data(), N * c, L + 1, T.data(), c, R.data() + (size_t)i * (L + 1) * c)) {
            std::lock_guard<std::mutex> g(mu);
            ok = false;
        }
    });
    return ok;
}

// Clip every U_k's singular values into [a0, b0], b0/a0 = kappa_max/sqrt(N),
// geometrically centred on the geometric mean of all singular values.
// Returns false when an SVD did not converge within the plan's sweep cap
// (U is then left unchanged: the clipping would rest on inexact factors).
bool project(const cerar_plan *p, std::vector<double> &U, double kappa_max, double &a0, double &b0) {
    const int N = p->N, c = p->c;
    std::vector<double> P((size_t)N * c * c), S((size_t)N * c), Q((size_t)N * c * c);
    std::vector<char> ok(N, 1);
    parallel_for(N, [&](int k) {
        ok[k] = la::svd_square(U.data() + (size_t)k * c * c, c, P.data() + (size_t)k * c * c,
                               S.data() + (size_t)k * c, Q.data() + (size_t)k * c * c, p->svd_sweeps);
    });
    for (char v : ok)
        if (!v) return false;
    double logsum = 0.0;
    for (double s : S) logsum += std::log(s);
    const double centre = std::exp(logsum / (double)S.size());
    const double half = std::sqrt(kappa_max / std::sqrt((double)N));
    a0 = centre / half;
    b0 = centre * half;
    for (int k = 0; k < N; ++k) {
        const double *Pk = P.data() + (size_t)k * c * c, *Qk = Q.data() + (size_t)k * c * c;
        const double *Sk = S.data() + (size_t)k * c;
        double *Uk = U.data() + (size_t)k * c * c;
        for (int a = 0; a < c; ++a)
            for (int b = 0; b < c; ++b) {
                double v = 0.0;
                for (int t = 0; t < c; ++t)
                    v += Pk[(size_t)a * c + t] * std::min(std::max(Sk[t], a0), b0) * Qk[(size_t)b * c + t];
                Uk[(size_t)a * c + b] = v;
            }
    }
    return true;
}

double kappa_of(const double *A, int m, int n, int sweeps, bool *converged) {
    std::vector<double> s = la::singular_values(A, m, n, sweeps, converged);
    return s.back() > 0 ? s.front() / s.back() : std::numeric_limits<double>::infinity();
}

void fill_info(cerar_plan *p, cerar_construction kind, double param) {
    const int N = p->N, c = p->c, L = p->L;
    cerar_plan_info &I = p->info;
    I.N = N;
    I.c = c;
    I.L = L;
    I.r_star = (c + N - 1) / N - 1;
    I.kind = kind;
    I.param = param;
    I.comm_rate = (double)L / c;
    I.storage_rate = 1.0 + (double)N / c;
    I.phi = phi_of(p, p->U, p->R);
    std::vector<double> kM(N), kU(N), kR(N), nU(N), nR(N);
    std::vector<char> conv(N, 1);
    parallel_for(N, [&](int i) {
        bool ok = true;
        std::vector<double> M = coefficient_map(p, p->U, i);
        kM[i] = kappa_of(M.data(), N * c, L + 1, p->svd_sweeps, &ok);
        std::vector<double> su = la::singular_values(p->U.data() + (size_t)i * c * c, c, c, p->svd_sweeps, &ok);
        kU[i] = su.back() > 0 ? su.front() / su.back() : INFINITY;
        nU[i] = su.front();
        std::vector<double> sr = la::singular_values(p->R.data() + (size_t)i * (L + 1) * c, L + 1, c,
                                                     p->svd_sweeps, &ok);
        kR[i] = sr.back() > 0 ? sr.front() / sr.back() : INFINITY;
        nR[i] = sr.front();
        conv[i] = ok;
    });
    for (char v : conv) p->svd_ok = p->svd_ok && v;
    I.svd_converged = p->svd_ok ? 1 : 0;
    I.kappa_M = *std::max_element(kM.begin(), kM.end());
    I.kappa_U = *std::max_element(kU.begin(), kU.end());
    I.kappa_R = *std::max_element(kR.begin(), kR.end());
    I.amplification = *std::max_element(nU.begin(), nU.end()) * *std::max_element(nR.begin(), nR.end());
    I.fp64_reliable = (I.kappa_U * c * 0x1.0p-53 <= 1e-6) ? 1 : 0;
    if (!p->D.empty()) {
        std::vector<double> E = p->D;
        if (la::inverse(E.data(), c)) {
            for (int a = 0; a < c; ++a) E[(size_t)a * c + a] -= 1.0;
            I.phi_closed_form = N * (N - 1) / 2.0 * la::frobenius2(E.data(), E.size());
        } else {
            I.phi_closed_form = kNaN;
        }
    } else {
        I.phi_closed_form = kNaN;
    }
}

// K^(l)(B, H) of Sec. II-C, c x c row-major: B, BH, ..., BH^(beta-1), then the
// s rows r in E_l = {l, ..., l+s-1} (mod N) of BH^beta, where c = beta N + s.
std::vector<double> k_matrix(const std::vector<double> &B, const std::vector<double> &H, int N, int c, int ell) {
    const int beta = c / N, s = c % N;
    std::vector<double> K((size_t)c * c), P = B, T((size_t)N * c);      // P = B H^j
    for (int j = 0; j < beta; ++j) {
        std::copy(P.begin(), P.end(), K.begin() + (size_t)j * N * c);
        la::matmul(P.data(), H.data(), T.data(), N, c, c);
        P.swap(T);
    }
    for (int t = 0; t < s; ++t) {
        const int r = (ell + t) % N;
        std::copy(P.begin() + (size_t)r * c, P.begin() + (size_t)(r + 1) * c, K.begin() + ((size_t)beta * N + t) * c);
    }
    return K;
}

// gamma = min over l of sigma_min(K^(l)(B, H)); with s = 0 every l gives the same K.
// Clears p->svd_ok if an SVD reached the sweep cap.
double gamma_of(cerar_plan *p, const std::vector<double> &B, const std::vector<double> &H, int N, int c) {
    const int nl = (c % N) ? N : 1;
    std::vector<double> g(nl);
    std::vector<char> conv(nl, 1);
    parallel_for(nl, [&](int ell) {
        bool ok = true;
        std::vector<double> K = k_matrix(B, H, N, c, ell);
        g[ell] = la::singular_values(K.data(), c, c, p->svd_sweeps, &ok).back();
        conv[ell] = ok;
    });
    for (char v : conv) p->svd_ok = p->svd_ok && v;
    return *std::min_element(g.begin(), g.end());
}

int validate(const cerar_plan_desc *d) {
    if (!d) return fail(CERAR_E_INVAL, "desc is NULL");
    if (d->N < 2 || d->N > kMaxN) return fail(CERAR_E_INVAL, "N=%d outside [2, %d] (Algorithm 1 needs N >= 2)", d->N, kMaxN);
    if (d->c < d->N || d->c > kMaxC) return fail(CERAR_E_INVAL, "c=%d outside [N=%d, %d]", d->c, d->N, kMaxC);
    if (!std::isfinite(d->param)) return fail(CERAR_E_INVAL, "param is not finite");
    switch (d->kind) {
        case CERAR_VANDERMONDE:
            if (d->param <= 0) return fail(CERAR_E_INVAL, "Vandermonde tau=%g must be > 0", d->param);
            break;
        case CERAR_O_EPS:
            if (d->param < 0) return fail(CERAR_E_INVAL, "eps=%g must be >= 0", d->param);
            break;
        case CERAR_KAPPA:
            if (d->param < std::sqrt((double)d->N))
                return fail(CERAR_E_INVAL, "kappa_max=%g below sqrt(N)=%g: the projection interval would be empty",
                            d->param, std::sqrt((double)d->N));
            if (d->als_order != 0 && d->als_order != 1)
                return fail(CERAR_E_INVAL, "als_order=%d must be 0 or 1", d->als_order);
            break;
        default:
            return fail(CERAR_E_INVAL, "unknown construction %d", (int)d->kind);
    }
    if (d->svd_sweeps < 0) return fail(CERAR_E_INVAL, "svd_sweeps=%d must be >= 0", d->svd_sweeps);
    if (d->als_restarts < 0 || d->als_restarts > 64)
        return fail(CERAR_E_INVAL, "als_restarts=%d outside [0, 64]", d->als_restarts);
    if (d->als_restarts > 1 && d->base)
        return fail(CERAR_E_INVAL, "als_restarts draw new random bases B: not with a given base");
    if (d->n_node_perms < 0 || d->n_node_perms > kMaxNodePerms)
        return fail(CERAR_E_INVAL, "n_node_perms=%d outside [0, %d]", d->n_node_perms, kMaxNodePerms);
    if (d->n_node_perms > 0) {
        if (!d->node_perms) return fail(CERAR_E_INVAL, "node_perms is NULL with n_node_perms=%d", d->n_node_perms);
        if (d->kind == CERAR_VANDERMONDE)
            return fail(CERAR_E_INVAL, "node_perms apply to the O(eps) and KAPPA constructions only");
        if (d->perturb) return fail(CERAR_E_INVAL, "node_perms and perturb are exclusive");
        std::vector<char> seen(d->c);
        for (int t = 0; t < d->n_node_perms; ++t) {
            std::fill(seen.begin(), seen.end(), 0);
            for (int j = 0; j < d->c; ++j) {
                const int v = d->node_perms[(size_t)t * d->c + j];
                if (v < 0 || v >= d->c || seen[v])
                    return fail(CERAR_E_INVAL, "node_perms row %d is not a permutation of 0..c-1", t);
                seen[v] = 1;
            }
        }
    }
    return CERAR_OK;
}

}  // namespace

std::string build_ring_tables(int N, int c, RingTables &t) {
    const int L = c + N - 2;
    t.N = N;
    t.c = c;
    t.L = L;
    t.enc_copy.assign(N, -1);
    t.rounds.assign((size_t)(L + 1) * N, RoundOp{-1, -1, -1, -1});
    t.state.assign((size_t)(L + 1) * N * (c + N), -1);
    std::vector<std::vector<int>> D(N, std::vector<int>(c)), Bs(N, std::vector<int>(N - 1, -1));
    std::vector<int> X(N, -1), next_pool(N, 0);
    auto pool = [&](int i) { return N * c + i * N + next_pool[i]++; };
    auto snapshot = [&](int k) {
        for (int i = 0; i < N; ++i) {
            int *s = t.state.data() + ((size_t)k * N + i) * (c + N);
            for (int j = 0; j < c; ++j) s[j] = D[i][j];
            for (int j = 0; j < N - 1; ++j) s[c + j] = Bs[i][j];
            s[c + N - 1] = X[i];
        }
    };
    for (int i = 0; i < N; ++i) {
        for (int j = 0; j < c; ++j) D[i][j] = i * c + j;     // delta_{i,j+1}, encoded in place
        X[i] = pool(i);                                      // x_{i,1} = delta_{i,1}, a copy
        t.enc_copy[i] = X[i];
    }
    snapshot(0);
    for (int k = 1; k <= L; ++k) {
        std::vector<int> recv(N);
        for (int i = 0; i < N; ++i) recv[i] = X[(i - 1 + N) % N];   // handoff W_{i-1} -> W_i
        for (int i = 0; i < N; ++i) {
            RoundOp &op = t.rounds[(size_t)k * N + i];
            if (k <= N - 1) {
                Bs[i][k - 1] = recv[i];                      // B_{i,k} <- x_{i-1,k}
                const int s = pool(i);
                op = RoundOp{recv[i], -1, D[i][k], s};       // x_{i,k+1} = x_{i-1,k} + delta_{i,k+1}
                X[i] = s;
            } else {
                const int j = k - N + 1;                     // 1-based
                const int old = D[i][j - 1];
                D[i][j - 1] = recv[i];                       // D_{i,j} <- x_{i-1,k}
                if (k < L) {
                    const int add = (k + 1 <= c) ? D[i][k] : -1;
                    op = RoundOp{recv[i], old, add, old};    // x_{i,k+1} = sigma_{i,k} (+ delta_{i,k+1})
                    X[i] = old;
                } else {
                    X[i] = -1;                               // round L only stores
                }
            }
        }
        snapshot(k);
    }
    t.ycols.assign((size_t)N * (L + 1), -1);
    for (int i = 0; i < N; ++i) {
        for (int j = 0; j < N - 1; ++j) t.ycols[(size_t)i * (L + 1) + j] = Bs[i][j];
        for (int j = 0; j < c; ++j) t.ycols[(size_t)i * (L + 1) + N - 1 + j] = D[i][j];
    }
    // Hazard check per launch: a written slot is read by nobody else, and
    // written once; every slot id is in range.
    const int nslots = N * c + N * N;
    for (int k = 1; k <= L; ++k) {
        std::map<int, int> writer;
        for (int i = 0; i < N; ++i) {
            const RoundOp &op = t.rounds[(size_t)k * N + i];
            if (op.dst < 0) continue;
            if (op.dst >= nslots) return "slot out of range";
            if (writer.count(op.dst)) return "slot written twice in one round";
            writer[op.dst] = i;
        }
        for (int i = 0; i < N; ++i) {
            const RoundOp &op = t.rounds[(size_t)k * N + i];
            if (op.dst < 0) continue;
            for (int s : {op.recv, op.sub, op.add}) {
                if (s < 0) continue;
                if (s >= nslots) return "slot out of range";
                auto it = writer.find(s);
                if (it != writer.end() && !(it->second == i && s == op.dst && s == op.sub))
                    return "round reads a slot another operand writes";
            }
        }
    }
    std::set<int> seen;
    for (int s : t.ycols) {
        if (s < 0 || s >= nslots) return "observation slot out of range";
        if (!seen.insert(s).second) return "two observations share a slot";
    }
    return "";
}

void build_fragments(cerar_plan *p) {
    const int N = p->N, c = p->c, L = p->L;
    p->MT = ceil_div(c, kTileM);
    p->KSe = ceil_div(c, kTileK);
    p->KSd = ceil_div(L + 1, kTileK);
    // A operand of a 16x16x4 fp32 MFMA: lane l holds A[row = l % 16][k = l / 16].
    // Encode computes delta^T = U^T G^T: row = output chunk j, k = input chunk l.
    p->enc_frag.assign((size_t)N * p->MT * p->KSe * kLanes, 0.0f);
    for (int i = 0; i < N; ++i)
        for (int mt = 0; mt < p->MT; ++mt)
            for (int ks = 0; ks < p->KSe; ++ks)
                for (int lane = 0; lane < kLanes; ++lane) {
                    const int j = mt * kTileM + lane % kTileM, l = ks * kTileK + lane / kTileM;
                    float v = 0.0f;
                    if (j < c && l < c) v = (float)p->U[((size_t)i * c + l) * c + j];
                    p->enc_frag[(((size_t)i * p->MT + mt) * p->KSe + ks) * kLanes + lane] = v;
                }
    // Decode computes g_hat^T = R^T Y^T: row = output chunk m, k = observation.
    p->dec_frag.assign((size_t)N * p->MT * p->KSd * kLanes, 0.0f);
    for (int i = 0; i < N; ++i)
        for (int mt = 0; mt < p->MT; ++mt)
            for (int ks = 0; ks < p->KSd; ++ks)
                for (int lane = 0; lane < kLanes; ++lane) {
                    const int m = mt * kTileM + lane % kTileM, k = ks * kTileK + lane / kTileM;
                    float v = 0.0f;
                    if (m < c && k <= L) v = (float)p->R[((size_t)i * (L + 1) + k) * c + m];
                    p->dec_frag[(((size_t)i * p->MT + mt) * p->KSd + ks) * kLanes + lane] = v;
                }
}

}  // namespace cerar

using namespace cerar;

static int finish_plan(cerar_plan *p, cerar_construction kind, double param, cerar_plan **out) {
    std::string err = build_ring_tables(p->N, p->c, p->tab);
    if (!err.empty()) return fail(CERAR_E_INVAL, "ownership table: %s", err.c_str());
    for (double v : p->U)
        if (!std::isfinite(v)) return fail(CERAR_E_SINGULAR, "encoding matrix has non-finite entries");
    for (double v : p->R)
        if (!std::isfinite(v)) return fail(CERAR_E_SINGULAR, "decoding matrix has non-finite entries");
    fill_info(p, kind, param);
    build_fragments(p);
    *out = p;
    return CERAR_OK;
}

static int create_desc(const cerar_plan_desc *desc, cerar_plan **out) {
    if (!out) return fail(CERAR_E_INVAL, "out is NULL");
    *out = nullptr;
    int st = validate(desc);
    if (st) return st;
    const int N = desc->N, c = desc->c;
    std::vector<double> nodes = desc->nodes ? std::vector<double>(desc->nodes, desc->nodes + c) : chebyshev_nodes(c);
    {
        std::vector<double> sorted = nodes;
        std::sort(sorted.begin(), sorted.end());
        for (int j = 0; j < c; ++j)
            if (!std::isfinite(sorted[j]) || (j > 0 && sorted[j] == sorted[j - 1]))
                return fail(CERAR_E_INVAL, "Vandermonde nodes must be distinct finite reals");
    }
    std::vector<double> H((size_t)c * c, 0.0);
    if (desc->perturb) {
        H.assign(desc->perturb, desc->perturb + (size_t)c * c);
    } else {
        for (int j = 0; j < c; ++j) H[(size_t)j * c + j] = nodes[j];
    }
    std::unique_ptr<cerar_plan> holder(new cerar_plan());   // freed on every failure, thrown or returned
    cerar_plan *p = holder.get();
    p->N = N;
    p->c = c;
    p->L = c + N - 2;
    p->info.phi_initial = kNaN;
    p->info.proj_a0 = p->info.proj_b0 = kNaN;
    p->info.gamma = kNaN;
    p->info.h_choice = -1;
    p->info.restart_used = -1;
    if (desc->svd_sweeps > 0) p->svd_sweeps = desc->svd_sweeps;
    int result = CERAR_OK;
    if (desc->kind == CERAR_VANDERMONDE) {
        // z_j = exp(tau xi_j); b_l = [z_j^l], l < N; D = diag(z_j^N)
        p->B.assign((size_t)N * c, 0.0);
        p->D.assign((size_t)c * c, 0.0);
        for (int j = 0; j < c; ++j) {
            const double z = std::exp(desc->param * nodes[j]);
            for (int l = 0; l < N; ++l) p->B[(size_t)l * c + j] = std::pow(z, (double)l);
            p->D[(size_t)j * c + j] = std::pow(z, (double)N);
        }
        result = mpc_plan(p);
    } else {
        const double eps = desc->kind == CERAR_O_EPS ? desc->param : (desc->eps0 > 0 ? desc->eps0 : 0.3);
        if (desc->kind == CERAR_O_EPS && eps > 0) {
            bool ok = true;
            std::vector<double> s = la::singular_values(H.data(), c, c, p->svd_sweeps, &ok);
            p->svd_ok = p->svd_ok && ok;
            if (eps * s.front() >= 1.0)
                return fail(CERAR_E_INVAL, "eps ||H||_2 = %g must be < 1 (Sec. II-C)", eps * s.front());
        }
        // one construction from the seeds seed0, seed0 + 1, ... (a new B after
        // an exactly singular window); KAPPA then runs the ALS from it
        auto design = [&](uint64_t seed0) -> int {
            std::vector<double> Hs = H;
            int result = CERAR_OK;
            const int tries = desc->base ? 1 : 8;
            for (int t = 0; t < tries; ++t) {
                if (desc->base) {
                    p->B.assign(desc->base, desc->base + (size_t)N * c);
                    p->info.seed_used = 0;
                } else {
                    p->B = gaussian_base(seed0 + (uint64_t)t, N, c);
                    p->info.seed_used = seed0 + (uint64_t)t;
                }
                if (desc->n_node_perms > 0) {
                    // the candidate H with the largest gamma for this B (Sec. II-C assumption)
                    double best = -1.0;
                    std::vector<double> Ht((size_t)c * c, 0.0);
                    for (int q = 0; q < desc->n_node_perms; ++q) {
                        const int *perm = desc->node_perms + (size_t)q * c;
                        for (int j = 0; j < c; ++j) Ht[(size_t)j * c + j] = nodes[perm[j]];
                        const double g = gamma_of(p, p->B, Ht, N, c);
                        if (g > best) {
                            best = g;
                            Hs = Ht;
                            p->info.h_choice = q;
                        }
                    }
                    p->info.gamma = best;
                } else {
                    p->info.gamma = gamma_of(p, p->B, Hs, N, c);
                }
                p->D.assign((size_t)c * c, 0.0);
                for (size_t a = 0; a < Hs.size(); ++a) p->D[a] = eps * Hs[a];
                for (int j = 0; j < c; ++j) p->D[(size_t)j * c + j] += 1.0;
                result = mpc_plan(p);
                if (result != CERAR_E_SINGULAR) break;
            }
            if (result == CERAR_OK && desc->kind == CERAR_KAPPA) {
                p->info.phi_initial = phi_of(p, p->U, p->R);
                const int iters = desc->als_iters > 0 ? desc->als_iters : 100;
                double a0 = kNaN, b0 = kNaN;
                const bool project_first = desc->als_order == 1;
                // the kappa guarantee rests on the projection's SVDs: one that
                // did not converge fails the plan instead of weakening it
                auto no_conv = [&] {
                    return fail(CERAR_E_NOCONV, "one-sided Jacobi SVD of an encoder did not converge in %d sweeps "
                                "(projection of Sec. II-D)", p->svd_sweeps);
                };
                for (int it = 0; it < iters && result == CERAR_OK; ++it) {
                    if (!u_step(p, p->R, p->U)) {
                        result = fail(CERAR_E_SINGULAR, "U-step normal equations singular");
                    } else if (project_first) {             // U-step, projection, R-step
                        if (!project(p, p->U, desc->param, a0, b0)) result = no_conv();
                        else if (!r_step(p, p->U, p->R))
                            result = fail(CERAR_E_SINGULAR, "R-step least squares rank deficient");
                    } else {                                // U-step, R-step, projection (Sec. II-D)
                        if (!r_step(p, p->U, p->R)) result = fail(CERAR_E_SINGULAR, "R-step least squares rank deficient");
                        else if (!project(p, p->U, desc->param, a0, b0)) result = no_conv();
                    }
                }
                // the decoders of the final (projected) encoders
                if (result == CERAR_OK && !project_first && !r_step(p, p->U, p->R))
                    result = fail(CERAR_E_SINGULAR, "final R-step rank deficient");
                p->info.proj_a0 = a0;
                p->info.proj_b0 = b0;
                p->D.clear();                                  // no closed form for the designed plan
            }
            return result;
        };
        result = design(desc->seed);
        // KAPPA restarts (Sec. II-D's problem is nonconvex): the ALS from the
        // O(eps0) plans of further random bases B, keeping the least Phi
        const int restarts = desc->kind == CERAR_KAPPA && desc->als_restarts > 1 ? desc->als_restarts : 1;
        if (desc->kind == CERAR_KAPPA && result == CERAR_OK) p->info.restart_used = 0;
        for (int r = 1; r < restarts && result == CERAR_OK; ++r) {
            const double best_phi = phi_of(p, p->U, p->R);
            std::vector<double> bU = p->U, bR = p->R, bB = p->B;
            const cerar_plan_info bI = p->info;
            const int st = design(desc->seed + 8 * (uint64_t)r);
            if (st == CERAR_OK && phi_of(p, p->U, p->R) < best_phi) {
                p->info.restart_used = r;
            } else {                                     // keep the best so far
                p->U.swap(bU);
                p->R.swap(bR);
                p->B.swap(bB);
                p->info = bI;
                clear_error();
            }
            p->D.clear();                                  // a failed restart may leave its O(eps0) D
        }
    }
    if (result == CERAR_OK) result = finish_plan(p, desc->kind, desc->param, out);
    if (result == CERAR_OK) holder.release();
    return result;
}

static int create_explicit(int N, int c, const double *U, const double *R, cerar_plan **out) {
    if (!out) return fail(CERAR_E_INVAL, "out is NULL");
    *out = nullptr;
    if (!U || !R) return fail(CERAR_E_INVAL, "U and R must be non-NULL");
    if (N < 2 || N > kMaxN) return fail(CERAR_E_INVAL, "N=%d outside [2, %d]", N, kMaxN);
    if (c < N || c > kMaxC) return fail(CERAR_E_INVAL, "c=%d outside [N=%d, %d]", c, N, kMaxC);
    std::unique_ptr<cerar_plan> holder(new cerar_plan());
    cerar_plan *p = holder.get();
    p->N = N;
    p->c = c;
    p->L = c + N - 2;
    p->U.assign(U, U + (size_t)N * c * c);
    p->R.assign(R, R + (size_t)N * (p->L + 1) * c);
    p->info.phi_initial = kNaN;
    p->info.proj_a0 = p->info.proj_b0 = kNaN;
    p->info.gamma = kNaN;
    p->info.h_choice = -1;
    p->info.restart_used = -1;
    int result = finish_plan(p, CERAR_EXPLICIT, kNaN, out);
    if (result == CERAR_OK) holder.release();
    return result;
}

extern "C" int cerar_plan_create_desc(const cerar_plan_desc *desc, cerar_plan **out) {
    clear_error();
    const int st = guarded([&] { return create_desc(desc, out); });
    if (st != CERAR_OK && out) *out = nullptr;
    return st;
}

extern "C" int cerar_plan_create(int N, int c, cerar_construction kind, double param, uint64_t seed,
                                 cerar_plan **out) {
    cerar_plan_desc d;
    std::memset(&d, 0, sizeof d);
    d.N = N;
    d.c = c;
    d.kind = kind;
    d.param = param;
    d.seed = seed;
    return cerar_plan_create_desc(&d, out);
}

extern "C" int cerar_plan_create_explicit(int N, int c, const double *U, const double *R, cerar_plan **out) {
    clear_error();
    const int st = guarded([&] { return create_explicit(N, c, U, R, out); });
    if (st != CERAR_OK && out) *out = nullptr;
    return st;
}

extern "C" void cerar_plan_destroy(cerar_plan *plan) {
    if (!plan) return;
    release_device(plan);
    delete plan;
}

extern "C" int cerar_plan_get_info(const cerar_plan *plan, cerar_plan_info *info) {
    clear_error();
    if (!plan || !info) return fail(CERAR_E_INVAL, "plan and info must be non-NULL");
    *info = plan->info;
    return CERAR_OK;
}

extern "C" int cerar_plan_get_matrices(const cerar_plan *plan, double *U, double *R) {
    clear_error();
    if (!plan) return fail(CERAR_E_INVAL, "plan is NULL");
    if (U) std::copy(plan->U.begin(), plan->U.end(), U);
    if (R) std::copy(plan->R.begin(), plan->R.end(), R);
    return CERAR_OK;
}

extern "C" int cerar_chunk_len(const cerar_plan *plan, size_t d, size_t *p, size_t *pool_stride) {
    clear_error();
    if (!plan || !p || !pool_stride) return fail(CERAR_E_INVAL, "NULL argument");
    if (d == 0) return fail(CERAR_E_INVAL, "d must be > 0");
    // ceil(d/c) rounded up to whole 128-byte lines: every chunk row of the
    // gradient and of the output then starts on a line, so no 64-position
    // block straddles a partial line (measured 1.4x faster encode/decode at
    // N=8, c=32 than with rows 32 bytes off a line)
    *p = ((d + plan->c - 1) / plan->c + kChunkAlign - 1) / kChunkAlign * kChunkAlign;
    *pool_stride = (*p + 63) / 64 * 64;
    return CERAR_OK;
}

extern "C" int cerar_workspace_bytes(const cerar_plan *plan, size_t d, size_t *bytes) {
    size_t p, stride;
    int st = cerar_chunk_len(plan, d, &p, &stride);
    if (st) return st;
    if (!bytes) return fail(CERAR_E_INVAL, "bytes is NULL");
    *bytes = (size_t)plan->tab.pool_slots() * stride * sizeof(float);
    return CERAR_OK;
}

extern "C" int cerar_slot_map(const cerar_plan *plan, int step, int *slots) {
    clear_error();
    if (!plan || !slots) return fail(CERAR_E_INVAL, "NULL argument");
    if (step < 0 || step > plan->L) return fail(CERAR_E_INVAL, "step %d outside [0, L=%d]", step, plan->L);
    const size_t n = (size_t)plan->N * (plan->c + plan->N);
    std::copy(plan->tab.state.begin() + (size_t)step * n, plan->tab.state.begin() + (size_t)(step + 1) * n, slots);
    return CERAR_OK;
}

extern "C" const char *cerar_last_error(void) { return cerar::g_last_error; }
