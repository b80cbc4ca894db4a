// Internal structures shared by the host plan code and the HIP launchers.
#pragma once

#include <exception>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/cerar.h"

namespace cerar {

// Build limits (validated by cerar_plan_create*).
constexpr int kMaxN = 64;
constexpr int kMaxC = 128;
constexpr int kMaxNodePerms = 4096;    // candidate H permutations per plan

// The MFMA operand tiling of encode/decode: 16 output rows per M-tile, 4
// reduction rows per K-step, 64 lanes per fragment.
constexpr int kTileM = 16;
constexpr int kTileK = 4;
constexpr int kLanes = 64;

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Chunk length p is ceil(d/c) rounded up to a multiple of this many floats
// (128 bytes); the zero padding of the last chunk absorbs the difference.
constexpr size_t kChunkAlign = 32;

// One round's per-worker slot operands: next message dst = recv - sub + add
// (sub/add = -1 when absent; dst = -1 when the round only relabels).
struct RoundOp {
    int recv, sub, add, dst;
};

// Slot-ownership bookkeeping of the handoff ring for given (N, c).
// Slot s < N*c is chunk s % c of worker s / c in `work`; slot s >= N*c is
// pool slot s - N*c of the workspace (N per worker).
struct RingTables {
    int N = 0, c = 0, L = 0;
    std::vector<int> enc_copy;       // N: pool slot that receives x_{i,1} = delta_{i,1}
    std::vector<RoundOp> rounds;     // (L+1) x N, entry k*N + i for round k (row 0 unused)
    std::vector<int> ycols;          // N x (L+1): slots of Y_i = [B_1..B_{N-1} | D_1..D_c]
    std::vector<int> state;          // (L+1) x N x (c+N): D (c), B (N-1), next message (1)
    int pool_slots() const { return N * N; }
};

// Builds the tables and checks that no launch reads a slot another worker
// writes in the same launch.  Returns an empty string or a diagnostic.
std::string build_ring_tables(int N, int c, RingTables &t);

struct DeviceCopy {
    float *enc_frag = nullptr;       // N x MT x KSe x 64 fp32 fragments of U_i
    float *dec_frag = nullptr;       // N x MT x KSd x 64 fp32 fragments of R_i
    int *ycols = nullptr;            // N x (L+1) slot ids
    RoundOp *rounds = nullptr;       // (L+1) x N
};

}  // namespace cerar

struct cerar_plan {
    int N = 0, c = 0, L = 0;
    cerar_plan_info info{};
    std::vector<double> U;           // N x c x c: U[k][l][j]
    std::vector<double> R;           // N x (L+1) x c: R[i][k][m]
    std::vector<double> B, D;        // MPC base / perturbation (empty for EXPLICIT)
    int svd_sweeps = 80;             // cap on one-sided Jacobi sweeps per SVD (cerar_plan_desc.svd_sweeps)
    bool svd_ok = true;              // every SVD so far converged within svd_sweeps
    cerar::RingTables tab;
    int MT = 0, KSe = 0, KSd = 0;    // M-tiles, encode K-steps, decode K-steps
    std::vector<float> enc_frag, dec_frag;
    mutable std::mutex dev_mu;
    mutable std::map<int, cerar::DeviceCopy> dev;   // per HIP device ordinal
};

namespace cerar {
// Thread-local error text; returns `status` for convenient `return fail(...)`.
int fail(int status, const char *fmt, ...) noexcept;
void clear_error() noexcept;

// Runs the body of a C entry point and turns a C++ exception into a status,
// so that none unwinds through the C ABI: a failed host allocation, or a
// host resource that could not be had, is CERAR_E_NOMEM.
template <class F>
int guarded(F &&body) noexcept {
    try {
        return body();
    } catch (const std::bad_alloc &) {
        return fail(CERAR_E_NOMEM, "out of host memory");
    } catch (const std::exception &e) {
        return fail(CERAR_E_NOMEM, "host resources exhausted: %s", e.what());
    } catch (...) {
        return fail(CERAR_E_NOMEM, "unexpected host exception");
    }
}

// Fills MT/KSe/KSd and the fp32 fragment arrays from U and R.
void build_fragments(cerar_plan *plan);
// Releases device copies (called by cerar_plan_destroy; defined with the kernels).
void release_device(cerar_plan *plan);
}  // namespace cerar
