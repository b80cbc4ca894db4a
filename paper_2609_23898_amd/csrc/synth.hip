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
//  * an approximately standard normal value, the Irwin-Hall sum of the twelve
//    32-bit halves of slots 0..5 minus 6, in exact integer arithmetic and one
//    exact scaling by 2^-32;
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
    if (idx >= a.d) return 0.0f;                          // the zero pad
    int64_t total = 0;
#pragma unroll
    for (int j = 0; j < 6; ++j) {
        const uint64_t h = slot_bits(a.key, idx, j);
        total += (int64_t)(h & 0xFFFFFFFFull) + (int64_t)(h >> 32);
    }
    double v = (double)(total + 6 - 6 * ((int64_t)1 << 32)) * 0x1.0p-32;
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
