// K6: the seeded synthetic gradients of the benchmark workloads, generated on
// the device.  Measurement and test input only: none of the all-reduce's
// arithmetic is here.
//
// Every entry is a pure function of (key, flat index), the same function the
// host generator of the tests computes, so the two give identical bits:
//  * 64 random bits per counter from the splitmix64 finaliser (Steele, Lea &
//    Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014,
//    with its published constants) applied to key + counter * golden gamma,
//    counter = 8 * index + slot + 1;
//  * a standard normal value by the Box-Muller transform (Box & Muller, Ann.
//    Math. Statist. 1958), z = sqrt(-2 ln u1) cos(2 pi u2), with u1 in (0, 1]
//    from the top 53 bits of slot 0 and u2 in [0, 1) from those of slot 1.
//    The logarithm (an exact binary split, then an atanh series) and the
//    cosine (an exact octant reduction, then Taylor series on [0, pi/4]) are
//    IEEE double additions, multiplications and divisions in a fixed order,
//    with fused multiply-adds off, and the square root is correctly rounded,
//    so the host generator's steps give the same bits;
//  * an outlier when the low half of slot 6 is below a threshold, which
//    multiplies the value by a factor (fp64);
//  * the entry is float32(value * scale of its tensor): one fp64 product,
//    one rounding to nearest.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "cerar_internal.hpp"

namespace cerar {
namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kMul1 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kMul2 = 0x94D049BB133111EBull;
constexpr int kSynthThreads = 256;
constexpr int kSynthPerThread = 4;
constexpr int kMaxTensors = 1024;

__device__ inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * kMul1;
    z = (z ^ (z >> 27)) * kMul2;
    return z ^ (z >> 31);
}

__device__ inline uint64_t slot_bits(uint64_t key, uint64_t idx, int slot) {
    return mix64(key + (idx * 8 + (uint64_t)(slot + 1)) * kGolden);
}

constexpr double kLn2 = 0.693147180559945309417;
constexpr double kSqrtHalf = 0.707106781186547524401;
constexpr double kPi4 = 0.785398163397448309616;
constexpr int kAtanhTerms = 11;

// (-1)^k / n!, n = first + 2k, with n! an exact double product (n <= 18).
constexpr double taylor_coefficient(int first, int k) {
    double f = 1.0;
    for (int i = 2; i <= first + 2 * k; ++i) f = f * (double)i;
    return (k % 2 ? -1.0 : 1.0) / f;
}

// ln u for u in (0, 1]: u = m 2^e exactly, m in [sqrt(1/2), sqrt(2)), and
// ln m = 2 atanh(t), t = (m - 1) / (m + 1).
__device__ inline double ln_unit(double u) {
#pragma clang fp contract(off)
    int e;
    double m = frexp(u, &e);
    if (m < kSqrtHalf) {
        m = m * 2.0;
        e = e - 1;
    }
    const double t = (m - 1.0) / (m + 1.0);
    const double t2 = t * t;
    double acc = 1.0 / (double)(2 * kAtanhTerms - 1);
#pragma unroll
    for (int k = kAtanhTerms - 2; k >= 0; --k) acc = acc * t2 + 1.0 / (double)(2 * k + 1);
    return (double)e * kLn2 + 2.0 * (t * acc);
}

// cos(2 pi u) from w8 = 8 u (exact) and its octant o: phi = (f or 1 - f) pi/4.
__device__ inline double cos_2pi(double w8, int o) {
#pragma clang fp contract(off)
    const double f = w8 - (double)o;
    const double a = (o & 1) ? 1.0 - f : f;
    const double phi = a * kPi4;
    const double p2 = phi * phi;
    double c = taylor_coefficient(0, 9);
#pragma unroll
    for (int k = 8; k >= 0; --k) c = c * p2 + taylor_coefficient(0, k);
    double sn = taylor_coefficient(1, 8);
#pragma unroll
    for (int k = 7; k >= 0; --k) sn = sn * p2 + taylor_coefficient(1, k);
    sn = sn * phi;
    const double v = (o == 1 || o == 2 || o == 5 || o == 6) ? sn : c;
    return (o >= 2 && o <= 5) ? -v : v;
}

struct SynthArgs {
    float *out;
    uint64_t n, first, d, key;
    const int64_t *toff;       // ntensors + 1 ascending flat offsets, toff[0] = 0
    const float *tscale;       // ntensors scales
    int ntensors;
    uint32_t threshold;        // outlier when the slot-6 low half is below it (0: none)
    double factor;
};

__device__ inline float entry(const SynthArgs &a, uint64_t idx, const int64_t *soff, const float *sscale,
                              int &t) {
#pragma clang fp contract(off)
    if (idx >= a.d) return 0.0f;                          // the zero pad
    const double u1 = (double)((slot_bits(a.key, idx, 0) >> 11) + 1) * 0x1.0p-53;
    const uint64_t i2 = slot_bits(a.key, idx, 1) >> 11;
    const double w8 = (double)i2 * 0x1.0p-50;
    double v = sqrt(-2.0 * ln_unit(u1)) * cos_2pi(w8, (int)(i2 >> 50));
    if (a.threshold != 0 && (uint32_t)(slot_bits(a.key, idx, 6) & 0xFFFFFFFFull) < a.threshold) v = v * a.factor;
    while (t + 1 < a.ntensors && (uint64_t)soff[t + 1] <= idx) ++t;   // the tensor that holds idx
    return (float)(v * (double)sscale[t]);
}

__global__ __launch_bounds__(kSynthThreads) void k_synth_fill(SynthArgs a) {
    __shared__ int64_t soff[kMaxTensors + 1];
    __shared__ float sscale[kMaxTensors];
    for (int i = threadIdx.x; i <= a.ntensors; i += kSynthThreads) soff[i] = a.toff[i];
    for (int i = threadIdx.x; i < a.ntensors; i += kSynthThreads) sscale[i] = a.tscale[i];
    __syncthreads();
    const uint64_t stride = (uint64_t)gridDim.x * kSynthThreads * kSynthPerThread;
    for (uint64_t i0 = ((uint64_t)blockIdx.x * kSynthThreads + threadIdx.x) * kSynthPerThread; i0 < a.n;
         i0 += stride) {
        const uint64_t idx0 = a.first + i0;
        // the first tensor whose end lies beyond idx0 (binary search), then forward
        int lo = 0, hi = a.ntensors - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) / 2;
            if ((uint64_t)soff[mid] <= idx0) lo = mid;
            else hi = mid - 1;
        }
        int t = lo;
        float v[kSynthPerThread];
#pragma unroll
        for (int q = 0; q < kSynthPerThread; ++q) v[q] = entry(a, idx0 + q, soff, sscale, t);
        float *dst = a.out + i0;
        if (i0 + kSynthPerThread <= a.n && ((uintptr_t)dst & 15) == 0) {
            typedef float v4f __attribute__((ext_vector_type(4)));
            *reinterpret_cast<v4f *>(dst) = v4f{v[0], v[1], v[2], v[3]};
        } else {
            for (int q = 0; q < kSynthPerThread && i0 + q < a.n; ++q) dst[q] = v[q];
        }
    }
}

}  // namespace
}  // namespace cerar

using namespace cerar;

extern "C" int cerar_synth_fill(float *out, size_t n, uint64_t first, uint64_t d, uint64_t key,
                                const int64_t *tensor_off, const float *tensor_scale, int ntensors,
                                uint32_t outlier_threshold, double outlier_factor, cerar_stream stream) {
    clear_error();
    if (n == 0) return CERAR_OK;
    if (!out || !tensor_off || !tensor_scale) return fail(CERAR_E_INVAL, "NULL argument");
    if (ntensors < 1 || ntensors > kMaxTensors)
        return fail(CERAR_E_INVAL, "ntensors=%d outside [1, %d]", ntensors, kMaxTensors);
    if (first > UINT64_MAX - n) return fail(CERAR_E_INVAL, "first + n overflows");
    SynthArgs a{out, n, first, d, key, tensor_off, tensor_scale, ntensors, outlier_threshold, outlier_factor};
    const uint64_t per_wg = (uint64_t)kSynthThreads * kSynthPerThread;
    const uint64_t wgs = std::min<uint64_t>((n + per_wg - 1) / per_wg, 1u << 20);
    hipLaunchKernelGGL(k_synth_fill, dim3((unsigned)wgs), dim3(kSynthThreads), 0,
                       reinterpret_cast<hipStream_t>(stream), a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(CERAR_E_DEVICE, "launch synth fill: %s", hipGetErrorString(e));
    return CERAR_OK;
}
