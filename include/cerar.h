/*
 * cerar.h - C ABI of libcerar, an MI355X (gfx950) implementation of the
 * data-parallel hot path of CERAR, the communication-efficient approximate
 * ring all-reduce of Munim & Ramamoorthy ("Communication-Efficient
 * Distributed Training via Ring-Based Coded Approximate All-Reduce").
 *
 * The method (Sec. II): each of N workers splits its length-d gradient into
 * c chunks of p floats (zero pad; p = ceil(d/c) rounded up to a multiple of
 * 32, see cerar_chunk_len), encodes them linearly
 * (Delta_i = G_i U_i), runs L = c + N - 2 combine-and-forward rounds on a ring
 * (Algorithm 1, update equations (2)), and decodes its L+1 stored
 * observations linearly (g_hat_i = Y_i R_i) into an approximation of the sum
 * of all N gradients.
 *
 * On one GPU all N workers live in one HBM allocation: worker i's buffers
 * are slices of caller-owned arrays, and a send is a handoff of a p-float
 * slot from W_i to W_{i+1}: no bytes move, only the ownership table changes.
 *
 * Conventions for every call
 *  - Return value: a cerar_status.  Details of the last non-OK status of the
 *    calling thread are in cerar_last_error().
 *  - Pointers named "device" are HIP device memory of the current device,
 *    owned by the caller; the library never frees caller memory.
 *  - Calls taking a stream only validate and enqueue work on that stream
 *    (NULL = the legacy default stream); they never synchronise, with one
 *    exception: the first such call for a plan on a device uploads the
 *    plan's fp32 coefficients and tables to that device (hipMalloc and a
 *    synchronous hipMemcpy, once per plan and device), unless
 *    cerar_plan_prepare_device did so before.  After it, the calls
 *    issue kernel launches only (no allocation, copy or memset), so they can
 *    be recorded into a HIP graph by stream capture.  Work enqueued by calls
 *    that share buffers must be ordered by the caller (one stream does
 *    that).
 *  - Data on the device (gradients, encoded chunks, messages, outputs) is
 *    IEEE fp32.  The encode and decode contractions accumulate in fp32; at
 *    c = 128 their fp32 operands are split exactly into three bf16 terms and
 *    six of the nine term products are summed on the bf16 matrix cores
 *    (within two units of fp32 rounding per product).  A round forms
 *    recv - delta_j + delta_{k+1} in fp64 and rounds the message to fp32
 *    once.  The error norms accumulate in fp64.  Plan construction is host
 *    fp64.
 */
#ifndef CERAR_H
#define CERAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same type as hipStream_t. */
typedef struct ihipStream_t *cerar_stream;

typedef enum {
    CERAR_OK = 0,
    CERAR_E_INVAL = -1,    /* an argument is out of range or NULL */
    CERAR_E_NOMEM = -2,    /* a host or device allocation failed, or another host resource (a thread) */
    CERAR_E_SINGULAR = -3, /* some window A_l of the construction is exactly singular */
    CERAR_E_NOCONV = -4,   /* an iterative host routine did not converge */
    CERAR_E_DEVICE = -5,   /* a HIP call failed; the HIP error text is in cerar_last_error() */
    CERAR_E_STATE = -6     /* cerar_encode_round / cerar_decode called out of order */
} cerar_status;

typedef enum {
    CERAR_VANDERMONDE = 0, /* Sec. II-B: z_j = exp(tau xi_j), b_l = [z_j^l], D = diag(z_j^N); param = tau > 0 */
    CERAR_O_EPS = 1,       /* Sec. II-C: B ~ N(0,1), D = I + eps H; param = eps >= 0 with eps ||H||_2 < 1 */
    CERAR_KAPPA = 2,       /* Sec. II-D, eq. (16): ALS under kappa_2(M_i) <= param = kappa_max >= sqrt(N) */
    CERAR_EXPLICIT = 3     /* caller-supplied U and R (cerar_plan_create_explicit) */
} cerar_construction;

/* Opaque plan: N, c, the fp64 matrices (U_k)_{k<N}, (R_i)_{i<N}, their fp32
 * device copies in the kernels' operand layout, and the slot-ownership
 * tables of the handoff ring.  Immutable after creation; may be shared by
 * threads. */
typedef struct cerar_plan cerar_plan;

/* Full description for cerar_plan_create_desc.  Zero-initialise, then set
 * N, c, kind and param; every other field has a default. */
typedef struct {
    int N;                  /* workers, 2 <= N <= 64 */
    int c;                  /* chunks, N <= c <= 128 (c = N is the exact ring all-reduce) */
    cerar_construction kind;
    double param;           /* tau (VANDERMONDE), eps (O_EPS), kappa_max (KAPPA) */
    uint64_t seed;          /* seeds B when base == NULL (splitmix64 + Box-Muller) */
    const double *base;     /* optional host N x c row-major B (O_EPS, KAPPA) */
    const double *perturb;  /* optional host c x c row-major H (O_EPS, KAPPA); default diag(nodes) */
    const double *nodes;    /* optional host c distinct reals xi; default cos((2j-1) pi / 2c) */
    double eps0;            /* KAPPA: eps of the O(eps) starting plan; <= 0 selects 0.3 */
    int als_iters;          /* KAPPA: ALS iterations; <= 0 selects 100 */
    int als_order;          /* KAPPA: steps of one iteration.  0: U-step, R-step, then the
                             * projection (the order Sec. II-D states; the next U-step
                             * overwrites the projected U, so only the last projection acts).
                             * 1: U-step, projection, R-step, so every R-step fits a projected
                             * U (about half the Phi at N=8, c=32..64).  Both end with a
                             * projection and an R-step, so kappa_2(M_i) <= kappa_max holds. */
    const int *node_perms;  /* O_EPS, KAPPA, with perturb == NULL: n_node_perms candidate
                             * permutations of 0..c-1 (host, row-major n x c).  Candidate t is
                             * H_t = diag(xi[perm_t[0]], ..., xi[perm_t[c-1]]); the plan takes the
                             * one with the largest gamma = min_l sigma_min(K^(l)(B, H_t)), the
                             * constant of the Sec. II-C assumption (the first on ties).  A choice
                             * of H that depends on B, which the same assumption allows.  The
                             * permutations leave ||H||, D's spectrum and so Phi unchanged, but
                             * a small gamma makes the windows A_l, and so M_i, ill-conditioned. */
    int n_node_perms;       /* 0: H as above (perturb, else diag(nodes)); at most 4096 */
    int svd_sweeps;         /* cap on the sweeps of each one-sided Jacobi SVD (the projection,
                             * kappa, gamma and ||H||); 0 selects 80 */
    int als_restarts;       /* KAPPA: ALS runs from the O(eps0) plans of different random bases
                             * B (seeds seed, seed + 8, seed + 16, ...; the problem of
                             * Sec. II-D is nonconvex); the plan with the least Phi is kept.
                             * 0 or 1: one run.  At most 64; needs base == NULL */
} cerar_plan_desc;

/* Plan diagnostics (host fp64). */
typedef struct {
    int N, c, L, r_star;          /* L = c+N-2 (Sec. II); r_star = ceil(c/N)-1 (Sec. II-C) */
    cerar_construction kind;
    double param;
    double phi;                   /* Phi(U,R) = sum_i ||M_i R_i - T||_F^2, eq. (7) */
    double phi_closed_form;       /* N(N-1)/2 ||D^-1 - I||_F^2 (Prop. 2) for MPC plans, else NaN */
    double phi_initial;           /* KAPPA: Phi of the O(eps0) starting plan, else NaN */
    double kappa_M;               /* max_i kappa_2(M_i), the constrained quantity of eq. (16) */
    double kappa_U;               /* max_k kappa_2(U_k) */
    double kappa_R;               /* max_i kappa_2(R_i) */
    double amplification;         /* max_k ||U_k||_2 * max_i ||R_i||_2 */
    double comm_rate;             /* L/c = 1 + (N-2)/c (Sec. II-B) */
    double storage_rate;          /* 1 + N/c (Sec. II-B) */
    double proj_a0, proj_b0;      /* KAPPA: last projection interval, else NaN */
    int fp64_reliable;            /* 0 when kappa_U * c * 2^-53 > 1e-6: fp64 inverses lose digits */
    uint64_t seed_used;           /* seed that produced B (after retries), 0 if B was given */
    double gamma;                 /* O_EPS, KAPPA: min_l sigma_min(K^(l)(B, H)) of the (B, H) used
                                   * (Sec. II-C assumption); NaN otherwise */
    int h_choice;                 /* index of the chosen node permutation, -1 if none was given */
    int svd_converged;            /* 1 when every one-sided Jacobi SVD behind kappa_M, kappa_U,
                                   * kappa_R, amplification, gamma and ||H||_2 converged within the
                                   * sweep cap; 0 when one stopped at the cap (those figures are
                                   * then approximate) */
    int restart_used;             /* KAPPA: index of the ALS restart kept (0 = the first run);
                                   * -1 for other constructions */
} cerar_plan_info;

/* Build a plan on the host in fp64 (Sec. II-B to II-D): B and D (or the
 * nodes) of the chosen construction, then U_k = A_{N-1-k}^{-1} (eq. (10)) and
 * R_i[l,:] = a_{l-i} (eq. (11)); KAPPA then runs the alternating least squares
 * of Sec. II-D from the O(eps0) plan.  Synchronous; touches no device.
 * Errors: E_INVAL (N < 2, N > 64, c < N, c > 128, param out of range,
 * node_perms with perturb, with VANDERMONDE or not permutations,
 * svd_sweeps < 0, out == NULL), E_SINGULAR (a window A_l exactly singular
 * for 8 seeds, or for the given B), E_NOCONV (KAPPA: the SVD of an encoder
 * in the projection did not converge within svd_sweeps, so the kappa bound
 * would not be guaranteed), E_NOMEM. */
int cerar_plan_create(int N, int c, cerar_construction kind, double param,
                      uint64_t seed, cerar_plan **out);
int cerar_plan_create_desc(const cerar_plan_desc *desc, cerar_plan **out);

/* Plan from caller matrices: U is host [N][c][c] with U[k][l][j] the
 * coefficient of chunk l in delta_{k,j+1}; R is host [N][L+1][c] with R[i][k][m]
 * the weight of y_{i,k+1} in output chunk m.  Copied. */
int cerar_plan_create_explicit(int N, int c, const double *U, const double *R,
                               cerar_plan **out);

/* Frees host and device memory of the plan.  No work using it may be pending. */
void cerar_plan_destroy(cerar_plan *plan);

/* Uploads the plan's fp32 coefficient fragments and slot tables to the
 * current device, once per plan and device (hipMalloc and a synchronous
 * hipMemcpy); later calls for that device return at once.  Every enqueueing
 * call does this itself on its first use on a device, except
 * cerar_ring_simulate_noalloc, which needs it done.  It also looks up the
 * current device's address of the no-alloc message pool.  Calling it first
 * lets a caller record the enqueueing calls into a HIP graph by stream
 * capture without an eager call, since after it they issue kernel launches
 * only.  Thread-safe.  Errors: E_INVAL (NULL plan); E_DEVICE (a HIP call
 * failed; nothing is kept for that device). */
int cerar_plan_prepare_device(const cerar_plan *plan);

int cerar_plan_get_info(const cerar_plan *plan, cerar_plan_info *info);

/* Copies the fp64 matrices into host arrays laid out as in
 * cerar_plan_create_explicit (N*c*c and N*(L+1)*c doubles). Either may be NULL. */
int cerar_plan_get_matrices(const cerar_plan *plan, double *U, double *R);

/* Geometry for gradient length d: the chunk and message length p (Sec. II:
 * the gradient is zero-padded to c chunks of p entries, chunk l being entries
 * [l p, (l+1) p)).  p = ceil(d/c) rounded up to a multiple of 32 floats, so
 * that every chunk row starts on a 128-byte line; the extra entries are part
 * of the zero pad of the last chunk, and the output keeps only the first d.
 * pool_stride is the stride of pool slots in the workspace (p rounded up to
 * 64).  Errors: E_INVAL (NULL pointers, d == 0). */
int cerar_chunk_len(const cerar_plan *plan, size_t d, size_t *p, size_t *pool_stride);

/* Device workspace needed for gradient length d: the pool of N*N message
 * slots that the first N sends of every worker need (the other c slots of
 * each worker are its own encoded chunks, overwritten in place). */
int cerar_workspace_bytes(const cerar_plan *plan, size_t d, size_t *bytes);

/* Ownership table after step `step` (0 = encode, k = round 1..L): writes
 * N*(c+N) ints, per worker i: the slots of D_{i,1..c} (c), of B_{i,1..N-1}
 * (N-1), and of the next message x_{i,step+1} (1; -1 after round L-1).
 * Slot s < N*c is chunk (s % c) of worker (s / c) in `work`; slot s >= N*c
 * is pool slot (s - N*c) of the workspace. */
int cerar_slot_map(const cerar_plan *plan, int step, int *slots);

/* One step of the protocol for all N workers on `stream`.
 *  step 0   encode (Sec. II, "Initialization"): for every worker i and
 *           position e < p, delta_{i,j}[e] = sum_l U_i[l][j-1] g_i[l p + e]
 *           (entries at l p + e >= d read as the zero pad), written to
 *           work[i*ld_work + (j-1)*p + e]; the first send x_{i,1} = delta_{i,1}
 *           is also written to worker i's first pool slot.
 *  step k   round k of Algorithm 1 / eq. (2), 1 <= k <= L: W_i takes the
 *           slot holding x_{i-1,k}; rounds k <= N-1 keep it as B_{i,k} and
 *           form x_{i,k+1} = x_{i-1,k} + delta_{i,k+1} in a fresh pool slot;
 *           rounds k >= N keep it as D_{i,j} (j = k-N+1) and, if k < L, form
 *           x_{i,k+1} = (x_{i-1,k} - delta_{i,j}) [+ delta_{i,k+1} if k < c]
 *           in the slot that held delta_{i,j}.  Round L only relabels.
 * grads:  device, N slices of >= d floats at stride ld_grads (read at step 0 only).
 * work:   device, N slices of >= c*p floats at stride ld_work; may equal
 *         grads (in-place encode, the paper's storage discipline) when
 *         ld_work == ld_grads.
 * ws:     device, cerar_workspace_bytes(plan, d); may not overlap grads or
 *         work, and grads may overlap work only by being the same buffer
 *         (E_INVAL otherwise).
 * Steps must run in order 0, 1, .., L on the same (work, ws) with the same
 * d: the library keeps the next expected step and the encode's d per
 * workspace address and returns E_STATE otherwise (step 0 is always accepted
 * and restarts the sequence).  That record, a few dozen bytes per workspace
 * address used with the plan, is kept until cerar_plan_destroy; the order is
 * checked at enqueue time, which is also the order on one stream. */
int cerar_encode_round(const cerar_plan *plan, int step, size_t d,
                       const float *grads, size_t ld_grads,
                       float *work, size_t ld_work, void *ws, cerar_stream stream);

/* Decode (Sec. II-A): g_hat_i = Y_i R_i with Y_i = [B_{i,1..N-1} | D_{i,1..c}]
 * read from the slots the ownership table names after round L.  Writes the
 * first d floats of out[i*ld_out ..] for every worker; nothing beyond d.
 * out must not overlap work or ws.  E_STATE unless rounds 1..L completed
 * on this workspace with the same d. */
int cerar_decode(const cerar_plan *plan, size_t d, const float *work, size_t ld_work,
                 const void *ws, float *out, size_t ld_out, cerar_stream stream);

/* Encode, L rounds and decode for all N workers: the whole approximate
 * all-reduce, enqueued on `stream` (L + 1 kernel launches: round L has none). */
int cerar_ring_simulate(const cerar_plan *plan, size_t d,
                        const float *grads, size_t ld_grads,
                        float *work, size_t ld_work, void *ws,
                        float *out, size_t ld_out, cerar_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * cerar_ring_simulate with no workspace argument.  The N*N message slots live
 * in a static device array of the library, CERAR_NOALLOC_SCRATCH_BYTES per
 * device, held by every device the library's code is loaded on until the
 * process ends.  The call allocates nothing, host or device: the plan must
 * already be on the current device (cerar_plan_prepare_device, which also
 * sets up the array's address there), and it keeps no step record.
 * Arguments, layouts and results are those of cerar_ring_simulate (work may
 * equal grads for the in-place encode).  Nothing in the array needs to start
 * at zero: every slot is written before it is read within one call.  All
 * calls on one device share its array, so two such calls whose work can
 * overlap in time on that device (different streams, or graph replays
 * running concurrently) race; order them.
 * Errors: E_INVAL (as cerar_ring_simulate, or N*N*pool_stride*4 bytes above
 * CERAR_NOALLOC_SCRATCH_BYTES, pool_stride from cerar_chunk_len: at N = 8
 * that is p <= 262144, d <= c * 262144); E_STATE (the plan is not on the
 * current device); E_DEVICE. */
#define CERAR_NOALLOC_SCRATCH_BYTES (64u << 20)
int cerar_ring_simulate_noalloc(const cerar_plan *plan, size_t d,
                                const float *grads, size_t ld_grads,
                                float *work, size_t ld_work,
                                float *out, size_t ld_out, cerar_stream stream);

/* Single-GPU fused variant (not a ring implementation): the same result as
 * cerar_ring_simulate up to rounding order, computed by one kernel that runs
 * the encode, the L rounds of Algorithm 1 and the decode for all N workers
 * on one 64-position block at a time, with the encoded chunks, messages and
 * observations on chip (LDS and registers); only grads are read and only out
 * is written (no work or ws).  It shows what sharing one device allows and is
 * reported beside the ring, never in its place: a real ring must move every
 * message through memory.  For N in {2, 4, 8} the messages pass between
 * lanes with no workgroup barrier per round.
 * Needs c in {16, 32, 48, 64}, N <= 8 (or N <= 16 with c <= 32), at most
 * 160 KiB of LDS (N (c + 6) 256 bytes; for N in {2, 4, 8} also
 * N max(64 c, 256 ceil((c + N - 1) / 4)) 4 bytes), and 16-byte aligned rows
 * (ld % 4 == 0).  Errors: E_INVAL. */
int cerar_ring_simulate_fused(const cerar_plan *plan, size_t d, const float *grads, size_t ld_grads,
                              float *out, size_t ld_out, cerar_stream stream);

/* Bucketed all-reduce (one independent CERAR instance per bucket, the same
 * plan for all): bucket b covers flat entries [bucket_off[b],
 * bucket_off[b] + bucket_len[b]) of every worker's gradient and gets its own
 * p_b (cerar_chunk_len of bucket_len[b]).  work holds, per worker, the buckets' c*p_b
 * slots back to back (stride ld_work >= sum_b c*p_b); ws is
 * cerar_bucketed_workspace_bytes.  Enqueued on `stream`: every bucket's
 * encode, then each round as one launch for up to 64 buckets and all
 * workers, then every bucket's decode.  With c <= 64 and 16-byte aligned
 * rows in every bucket, the encode and the decode are batched as well (up to
 * 32 buckets per launch); otherwise each bucket gets its own launches.
 * bucket_off/bucket_len are host arrays; buckets may not overlap in out.
 * Errors: E_INVAL (NULL plan or buffers, nbuckets < 1, an empty bucket,
 * overlapping buckets, ld_work below the slot total, ld_grads or ld_out below
 * the largest bucket end, out overlapping work or ws, grads overlapping
 * work or ws, work overlapping ws, or a bucket too long for one launch);
 * E_DEVICE. */
int cerar_bucketed_workspace_bytes(const cerar_plan *plan, const size_t *bucket_len,
                                   int nbuckets, size_t *work_floats, size_t *ws_bytes);
int cerar_ring_simulate_bucketed(const cerar_plan *plan, int nbuckets,
                                 const size_t *bucket_off, const size_t *bucket_len,
                                 const float *grads, size_t ld_grads,
                                 float *work, size_t ld_work, void *ws,
                                 float *out, size_t ld_out, cerar_stream stream);

/* Error norms (the metric of Table 3, relative l2 error per worker):
 * norms (device, N+1 doubles) receives sum_e (out_i[e] - S[e])^2 for
 * i = 0..N-1, then sum_e S[e]^2, where S = sum_w grads_w (fp64) over
 * e < d.  Overwrites norms.  Errors: E_INVAL (N outside [1, 64], d == 0,
 * NULL buffers, ld_grads or ld_out < d); E_DEVICE. */
int cerar_error_norms(int N, size_t d, const float *grads, size_t ld_grads,
                      const float *out, size_t ld_out, double *norms,
                      cerar_stream stream);

/* K5's parity term on sampled positions: the relative l2 difference between
 * the device's outputs and an independent computation of them (the fp64
 * CPU implementation of the tests and the bench) at the positions it
 * computed.  For every worker i < N: norms[2i] = sum_t (out[i*ld_out +
 * idx[t]] - ref[i*count + t])^2 and norms[2i+1] = sum_t ref[i*count + t]^2,
 * in fp64.  idx: device int64[count] flat output indices, each in [0, d)
 * (one outside makes that worker's sums NaN); ref: device fp64, N x count;
 * out: device fp32, N rows of stride ld_out; norms: device, 2N doubles,
 * overwritten.  Errors: E_INVAL (N outside [1, 64], count == 0, d == 0,
 * NULL buffers, ld_out < d); E_DEVICE. */
int cerar_sampled_norms(int N, size_t count, size_t d, const int64_t *idx, const double *ref,
                        const float *out, size_t ld_out, double *norms, cerar_stream stream);

/* Measurement helper: dst[0..n) = src[0..n), a plain streaming copy used as
 * the achievable-bandwidth reference and as the known-size kernel that
 * scales the HBM traffic counters.  n == 0 does nothing.  Errors: E_INVAL
 * (NULL or overlapping buffers, a copy too long for one launch); E_DEVICE. */
int cerar_copy_f32(float *dst, const float *src, size_t n, cerar_stream stream);

/* Measurement and test input (not part of the method): the seeded
 * synthetic gradient entries of the benchmark workloads, generated on the
 * device.  out[t] (device, n floats) = entry first + t of the stream `key`:
 * with h_s the splitmix64 hash of key + (8 idx + s + 1) * 0x9E3779B97F4A7C15,
 * the Box-Muller normal z = sqrt(-2 ln u1) cos(2 pi u2) of u1 = ((h_0 >> 11)
 * + 1) 2^-53 and u2 = (h_1 >> 11) 2^-53 (the logarithm and cosine as fixed
 * sequences of IEEE double operations, |z| <= 8.57), times outlier_factor
 * when the low half of h_6 is below outlier_threshold (0: never), times the
 * scale of the tensor that holds idx (one fp64 product), rounded once to
 * fp32; 0 for idx >= d (the zero pad).  Tensor j covers flat
 * indices [tensor_off[j], tensor_off[j+1]); tensor_off (int64, ntensors + 1
 * entries, ascending, tensor_off[0] = 0) and tensor_scale (fp32, ntensors)
 * are device arrays owned by the caller.  The host generator of the tests
 * computes the same function, so both give identical bits.  n == 0 does
 * nothing.  Errors: E_INVAL (NULL pointers, ntensors outside [1, 1024],
 * first + n beyond 2^64); E_DEVICE. */
int cerar_synth_fill(float *out, size_t n, uint64_t first, uint64_t d, uint64_t key,
                     const int64_t *tensor_off, const float *tensor_scale, int ntensors,
                     uint32_t outlier_threshold, double outlier_factor, cerar_stream stream);

/* Text of the calling thread's last non-OK status ("" if none). */
const char *cerar_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CERAR_H */
