// Host-only driver: allocation-failure injection into the plan builder.
// Global operator new is replaced so that exactly the k-th allocation after
// arming fails (std::bad_alloc, or nullptr for the nothrow forms), on whichever
// thread makes it.  For every k up to the number of allocations one plan
// construction makes, the construction must return CERAR_OK or
// CERAR_E_NOMEM (with a message and a NULL plan), and the number of live
// allocations must come back to where it was: nothing thrown crosses the C
// ABI, and nothing leaks on the failure paths.  No device code.
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "cerar.h"
#include "cerar_internal.hpp"
namespace cerar { void release_device(cerar_plan *) {} }

static std::atomic<long> g_countdown{0};    // > 0: armed; the allocation that takes it to 0 fails
static std::atomic<long> g_live{0};
static std::atomic<long> g_total{0};

static void *take(std::size_t n, bool nothrow) {
    if (g_countdown.load(std::memory_order_relaxed) > 0 && g_countdown.fetch_sub(1) == 1) {
        if (nothrow) return nullptr;
        throw std::bad_alloc();
    }
    void *q = std::malloc(n ? n : 1);
    if (!q) {
        if (nothrow) return nullptr;
        throw std::bad_alloc();
    }
    g_live.fetch_add(1);
    g_total.fetch_add(1);
    return q;
}
static void give(void *q) {
    if (!q) return;
    g_live.fetch_sub(1);
    std::free(q);
}

void *operator new(std::size_t n) { return take(n, false); }
void *operator new[](std::size_t n) { return take(n, false); }
void *operator new(std::size_t n, const std::nothrow_t &) noexcept { return take(n, true); }
void *operator new[](std::size_t n, const std::nothrow_t &) noexcept { return take(n, true); }
void operator delete(void *q) noexcept { give(q); }
void operator delete[](void *q) noexcept { give(q); }
void operator delete(void *q, std::size_t) noexcept { give(q); }
void operator delete[](void *q, std::size_t) noexcept { give(q); }

struct Case {
    const char *name;
    int N, c;
    cerar_construction kind;
    double param;
    int als_iters, n_perms;
};

// The description and its permutations are built before the countdown is
// armed, so that every counted allocation is the library's.
struct Desc {
    cerar_plan_desc d;
    std::vector<int> perms;
    explicit Desc(const Case &k) {
        std::memset(&d, 0, sizeof d);
        d.N = k.N;
        d.c = k.c;
        d.kind = k.kind;
        d.param = k.param;
        d.seed = 11;
        d.als_iters = k.als_iters;
        for (int t = 0; t < k.n_perms; ++t)
            for (int j = 0; j < k.c; ++j) perms.push_back((j + 3 * t) % k.c);
        if (k.n_perms) {
            d.node_perms = perms.data();
            d.n_node_perms = k.n_perms;
        }
    }
};

int main() {
    const Case cases[] = {
        {"vandermonde", 3, 5, CERAR_VANDERMONDE, 0.3, 0, 0},
        {"o_eps+perms", 4, 9, CERAR_O_EPS, 0.1, 0, 3},
        {"kappa", 4, 8, CERAR_KAPPA, 1e3, 2, 0},
    };
    long points = 0, nomem = 0, ok = 0, leaks = 0, bad = 0;
    for (const Case &k : cases) {
        const Desc desc(k);
        auto make = [&](cerar_plan **out) { return cerar_plan_create_desc(&desc.d, out); };
        cerar_plan *p = nullptr;
        if (make(&p) != CERAR_OK) {             // warm-up: lazily made library state
            std::printf("%s: plain construction failed: %s\n", k.name, cerar_last_error());
            return 1;
        }
        cerar_plan_destroy(p);
        const long base = g_live.load();
        const long t0 = g_total.load();
        if (make(&p) != CERAR_OK) return 1;
        const long per_call = g_total.load() - t0;
        cerar_plan_destroy(p);
        if (g_live.load() != base) {
            std::printf("%s: %ld allocations left by a plain create/destroy\n", k.name, g_live.load() - base);
            return 1;
        }
        // every failure point of the first 400 allocations, then every 7th
        for (long at = 1; at <= per_call; at += at <= 400 ? 1 : 7) {
            p = nullptr;
            g_countdown.store(at);
            const int st = make(&p);
            g_countdown.store(0);
            ++points;
            if (st == CERAR_OK) {
                ++ok;
                cerar_plan_destroy(p);
            } else if (st == CERAR_E_NOMEM && p == nullptr && cerar_last_error()[0] != 0) {
                ++nomem;
            } else {
                ++bad;
                std::printf("%s: failure at allocation %ld gave status %d (%s)\n", k.name, at, st, cerar_last_error());
            }
            if (g_live.load() != base) {
                ++leaks;
                std::printf("%s: failure at allocation %ld left %ld allocations\n", k.name, at, g_live.load() - base);
            }
        }
        // the explicit constructor too, from this plan's matrices
        if (make(&p) != CERAR_OK) return 1;
        cerar_plan_info info;
        cerar_plan_get_info(p, &info);
        std::vector<double> U((size_t)info.N * info.c * info.c), R((size_t)info.N * (info.L + 1) * info.c);
        cerar_plan_get_matrices(p, U.data(), R.data());
        cerar_plan_destroy(p);
        const long base2 = g_live.load();
        const long t1 = g_total.load();
        if (cerar_plan_create_explicit(info.N, info.c, U.data(), R.data(), &p) != CERAR_OK) return 1;
        const long per_explicit = g_total.load() - t1;
        cerar_plan_destroy(p);
        for (long at = 1; at <= per_explicit; ++at) {
            p = nullptr;
            g_countdown.store(at);
            const int st = cerar_plan_create_explicit(info.N, info.c, U.data(), R.data(), &p);
            g_countdown.store(0);
            ++points;
            if (st == CERAR_OK) {
                ++ok;
                cerar_plan_destroy(p);
            } else if (st == CERAR_E_NOMEM && p == nullptr) {
                ++nomem;
            } else {
                ++bad;
            }
            if (g_live.load() != base2) ++leaks;
        }
    }
    std::printf("fault points %ld, nomem %ld, ok %ld, bad %ld, leaks %ld\n", points, nomem, ok, bad, leaks);
    return (bad || leaks || nomem == 0) ? 1 : 0;
}
