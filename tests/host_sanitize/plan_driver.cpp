// Host-only driver for the plan builder under AddressSanitizer and
// UndefinedBehaviorSanitizer: every construction over a grid of (N, c), the
// read-out calls, explicit plans and rejected arguments.  No device code.
#include <cstdio>
#include <cstring>
#include <vector>
#include "cerar.h"
#include "cerar_internal.hpp"
namespace cerar { void release_device(cerar_plan *) {} }

static int created = 0, rejected = 0;
static void exercise(cerar_plan *p) {
    cerar_plan_info info;
    cerar_plan_get_info(p, &info);
    std::vector<double> U((size_t)info.N * info.c * info.c), R((size_t)info.N * (info.L + 1) * info.c);
    cerar_plan_get_matrices(p, U.data(), R.data());
    size_t pp, stride, ws;
    for (size_t d : {(size_t)1, (size_t)777, (size_t)info.c * 64 + 3, (size_t)1 << 20}) {
        cerar_chunk_len(p, d, &pp, &stride);
        cerar_workspace_bytes(p, d, &ws);
    }
    std::vector<int> map((size_t)info.N * (info.c + info.N));
    for (int k = 0; k <= info.L; ++k) cerar_slot_map(p, k, map.data());
    cerar_plan *e = nullptr;
    if (cerar_plan_create_explicit(info.N, info.c, U.data(), R.data(), &e) == CERAR_OK) cerar_plan_destroy(e);
}
int main() {
    const int Ns[] = {2, 3, 4, 5, 8, 13, 16};
    for (int N : Ns)
        for (int c : {N, N + 1, 2 * N, 2 * N + 3, 4 * N}) {
            if (c > 128) continue;
            struct { cerar_construction k; double param; } kinds[] = {
                {CERAR_VANDERMONDE, 0.3}, {CERAR_O_EPS, 0.1}, {CERAR_O_EPS, 0.0}, {CERAR_KAPPA, 1e3}};
            for (auto &kd : kinds) {
                cerar_plan_desc desc;
                std::memset(&desc, 0, sizeof desc);
                desc.N = N; desc.c = c; desc.kind = kd.k; desc.param = kd.param; desc.seed = 7;
                desc.als_iters = 5;
                std::vector<int> perms;
                if (kd.k != CERAR_VANDERMONDE) {
                    for (int t = 0; t < 3; ++t)
                        for (int j = 0; j < c; ++j) perms.push_back((j + t) % c);
                    desc.node_perms = perms.data();
                    desc.n_node_perms = 3;
                }
                for (int order = 0; order < 2; ++order) {
                    desc.als_order = order;
                    cerar_plan *p = nullptr;
                    if (cerar_plan_create_desc(&desc, &p) == CERAR_OK) { ++created; exercise(p); cerar_plan_destroy(p); }
                    else ++rejected;
                    if (kd.k != CERAR_KAPPA) break;
                }
            }
        }
    // invalid inputs
    cerar_plan *p = nullptr;
    cerar_plan_create(1, 4, CERAR_O_EPS, 0.1, 1, &p);
    cerar_plan_create(4, 3, CERAR_O_EPS, 0.1, 1, &p);
    cerar_plan_create(4, 200, CERAR_O_EPS, 0.1, 1, &p);
    cerar_plan_create(4, 8, CERAR_KAPPA, 1.0, 1, &p);
    cerar_plan_create_explicit(4, 8, nullptr, nullptr, &p);
    printf("created %d, rejected %d, last error: %s\n", created, rejected, cerar_last_error());
    return 0;
}
