/* A C consumer of libcerar: one approximate all-reduce of N workers'
 * gradients on the current GPU through the C ABI and the HIP runtime alone,
 * with no Python.  The inputs come from the library's seeded generator
 * (cerar_synth_fill, Box-Muller normals, |z| <= 8.6).  Two plans:
 *  - exact (c = N, eps = 0, Sec. II-B): every output must be the sum of the
 *    N gradients up to fp32 rounding of the coefficients (1e-5 relative);
 *  - condition-number constrained (c > N, kappa_max = 1e3, Sec. II-D): an
 *    approximation, whose error measured here on the host must agree with
 *    cerar_error_norms.
 * Exit status 0 and the line "c-abi example ok" on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "cerar.h"

#define HIP(x)                                                                   \
    do {                                                                         \
        hipError_t e_ = (x);                                                     \
        if (e_ != hipSuccess) {                                                  \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));              \
            return 1;                                                            \
        }                                                                        \
    } while (0)
#define CER(x)                                                                   \
    do {                                                                         \
        int s_ = (x);                                                            \
        if (s_ != CERAR_OK) {                                                    \
            fprintf(stderr, "%s: status %d: %s\n", #x, s_, cerar_last_error());  \
            return 1;                                                            \
        }                                                                        \
    } while (0)

/* Runs one all-reduce; *host_err is the largest relative l2 error of the
 * outputs against the exact sum computed here, *norm_err the same from
 * cerar_error_norms. */
static int run(int N, int c, cerar_construction kind, double param, size_t d, double *host_err,
               double *norm_err) {
    cerar_plan *plan = NULL;
    CER(cerar_plan_create(N, c, kind, param, 7, &plan));
    CER(cerar_plan_prepare_device(plan));
    size_t p, stride, ws_bytes;
    CER(cerar_chunk_len(plan, d, &p, &stride));
    CER(cerar_workspace_bytes(plan, d, &ws_bytes));
    const size_t ld_work = (size_t)c * p;
    float *hg = malloc((size_t)N * d * sizeof(float));
    float *ho = malloc((size_t)N * d * sizeof(float));
    double *sum = malloc(d * sizeof(double));
    double *hn = malloc((size_t)(N + 1) * sizeof(double));
    if (!hg || !ho || !sum || !hn) return 1;
    float *grads, *work, *out, *scale;
    void *ws;
    double *norms;
    int64_t *toff;
    HIP(hipMalloc((void **)&grads, (size_t)N * d * sizeof(float)));
    HIP(hipMalloc((void **)&work, (size_t)N * ld_work * sizeof(float)));
    HIP(hipMalloc(&ws, ws_bytes));
    HIP(hipMalloc((void **)&out, (size_t)N * d * sizeof(float)));
    HIP(hipMalloc((void **)&norms, (size_t)(N + 1) * sizeof(double)));
    /* inputs: the library's seeded generator, one tensor of scale 1, one stream per worker */
    const int64_t h_off[2] = {0, (int64_t)d};
    const float h_scale = 1.0f;
    HIP(hipMalloc((void **)&toff, sizeof h_off));
    HIP(hipMalloc((void **)&scale, sizeof h_scale));
    HIP(hipMemcpy(toff, h_off, sizeof h_off, hipMemcpyHostToDevice));
    HIP(hipMemcpy(scale, &h_scale, sizeof h_scale, hipMemcpyHostToDevice));
    for (int w = 0; w < N; ++w)
        CER(cerar_synth_fill(grads + (size_t)w * d, d, 0, d, 0x5eed0000u + (uint64_t)w, toff, scale, 1, 0, 1.0, NULL));
    HIP(hipMemcpy(hg, grads, (size_t)N * d * sizeof(float), hipMemcpyDeviceToHost));
    for (size_t e = 0; e < d; ++e) {
        sum[e] = 0.0;
        for (int w = 0; w < N; ++w) sum[e] += hg[(size_t)w * d + e];
    }
    int finite_inputs = 1;
    for (size_t i = 0; i < (size_t)N * d; ++i) finite_inputs &= isfinite(hg[i]) && fabsf(hg[i]) <= 8.6f;
    if (!finite_inputs || sum[0] == 0.0) {
        fprintf(stderr, "generated inputs out of range\n");
        return 1;
    }
    CER(cerar_ring_simulate(plan, d, grads, d, work, ld_work, ws, out, d, NULL));
    CER(cerar_error_norms(N, d, grads, d, out, d, norms, NULL));
    HIP(hipDeviceSynchronize());
    HIP(hipMemcpy(ho, out, (size_t)N * d * sizeof(float), hipMemcpyDeviceToHost));
    HIP(hipMemcpy(hn, norms, (size_t)(N + 1) * sizeof(double), hipMemcpyDeviceToHost));
    double ss = 0.0;
    for (size_t e = 0; e < d; ++e) ss += sum[e] * sum[e];
    *host_err = *norm_err = 0.0;
    for (int i = 0; i < N; ++i) {
        double r = 0.0;
        for (size_t e = 0; e < d; ++e) {
            const double t = ho[(size_t)i * d + e] - sum[e];
            r += t * t;
        }
        const double eh = sqrt(r / ss), en = sqrt(hn[i] / hn[N]);
        if (eh > *host_err) *host_err = eh;
        if (en > *norm_err) *norm_err = en;
    }
    HIP(hipFree(grads));
    HIP(hipFree(work));
    HIP(hipFree(ws));
    HIP(hipFree(out));
    HIP(hipFree(norms));
    HIP(hipFree(toff));
    HIP(hipFree(scale));
    free(hg);
    free(ho);
    free(sum);
    free(hn);
    cerar_plan_destroy(plan);
    return 0;
}

int main(void) {
    double ex_h, ex_n, ka_h, ka_n;
    if (run(4, 4, CERAR_O_EPS, 0.0, 4096 * 3 + 5, &ex_h, &ex_n)) return 1;
    if (run(8, 16, CERAR_KAPPA, 1e3, 16 * 1024 + 7, &ka_h, &ka_n)) return 1;
    printf("exact plan (N=4, c=4): max relative error %.3g (host) %.3g (cerar_error_norms)\n", ex_h, ex_n);
    printf("kappa plan (N=8, c=16): max relative error %.3g (host) %.3g (cerar_error_norms)\n", ka_h, ka_n);
    const int ok = ex_h < 1e-5 && fabs(ex_h - ex_n) < 1e-6 && isfinite(ka_h) && ka_h < 1.0 &&
                   fabs(ka_h - ka_n) <= 1e-6 * (1.0 + ka_h);
    if (!ok) {
        printf("FAIL\n");
        return 1;
    }
    printf("c-abi example ok\n");
    return 0;
}
