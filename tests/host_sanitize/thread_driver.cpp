// Host-only driver for the plan builder under ThreadSanitizer.  Four threads
// at once:
//  - build plans of every construction, each build itself spreading its
//    per-worker steps over up to hardware_concurrency threads;
//  - read one shared plan through every read-out call, since a plan may be
//    shared by threads once created;
//  - record different errors and check that each thread reads back its own
//    text from cerar_last_error (the text is per thread).
// No device code.
#include <atomic>
#include <cstdio>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "cerar.h"
#include "cerar_internal.hpp"
namespace cerar { void release_device(cerar_plan *) {} }

static std::atomic<int> g_failures{0};

static void check(bool ok, const char *what, int t) {
    if (!ok) {
        std::printf("thread %d: %s\n", t, what);
        g_failures.fetch_add(1);
    }
}

static void read_shared(const cerar_plan *p, int t) {
    cerar_plan_info info;
    check(cerar_plan_get_info(p, &info) == CERAR_OK, "get_info", t);
    std::vector<double> U((size_t)info.N * info.c * info.c), R((size_t)info.N * (info.L + 1) * info.c);
    check(cerar_plan_get_matrices(p, U.data(), R.data()) == CERAR_OK, "get_matrices", t);
    size_t pp, stride, ws;
    check(cerar_chunk_len(p, 12345, &pp, &stride) == CERAR_OK, "chunk_len", t);
    check(cerar_workspace_bytes(p, 12345, &ws) == CERAR_OK, "workspace_bytes", t);
    std::vector<int> map((size_t)info.N * (info.c + info.N));
    for (int k = 0; k <= info.L; ++k) check(cerar_slot_map(p, k, map.data()) == CERAR_OK, "slot_map", t);
}

int main() {
    cerar_plan *shared = nullptr;
    if (cerar_plan_create(4, 10, CERAR_O_EPS, 0.1, 5, &shared) != CERAR_OK) {
        std::printf("shared plan: %s\n", cerar_last_error());
        return 1;
    }
    std::atomic<int> arrived{0};
    std::vector<std::thread> th;
    for (int t = 0; t < 4; ++t)
        th.emplace_back([&, t] {
            const int N = 3 + t, c = 2 * (3 + t) + 1;
            const cerar_construction kinds[] = {CERAR_VANDERMONDE, CERAR_O_EPS, CERAR_KAPPA};
            const double params[] = {0.3, 0.1, 1e3};
            for (int r = 0; r < 2; ++r) {
                for (int q = 0; q < 3; ++q) {
                    cerar_plan_desc d;
                    std::memset(&d, 0, sizeof d);
                    d.N = N;
                    d.c = c;
                    d.kind = kinds[q];
                    d.param = params[q];
                    d.seed = 100 + t;
                    d.als_iters = 3;
                    cerar_plan *p = nullptr;
                    check(cerar_plan_create_desc(&d, &p) == CERAR_OK, "create", t);
                    if (p) {
                        read_shared(p, t);
                        cerar_plan_destroy(p);
                    }
                }
                read_shared(shared, t);
            }
            // a different rejected N per thread; every thread records its error
            // before any reads its own back
            cerar_plan *p = nullptr;
            check(cerar_plan_create(1, 40 + t, CERAR_O_EPS, 0.1, 1, &p) == CERAR_E_INVAL, "reject", t);
            const std::string mine = cerar_last_error();
            arrived.fetch_add(1);
            while (arrived.load() < 4) std::this_thread::yield();
            check(mine == cerar_last_error(), "last error changed by another thread", t);
            check(cerar_plan_create(2, 40 + t, CERAR_O_EPS, 0.1, 1, &p) == CERAR_OK, "create after error", t);
            check(cerar_last_error()[0] == 0, "last error not cleared by a successful call", t);
            cerar_plan_destroy(p);
        });
    for (auto &x : th) x.join();
    cerar_plan_destroy(shared);
    std::printf("threads done, failures %d\n", g_failures.load());
    return g_failures.load() ? 1 : 0;
}
