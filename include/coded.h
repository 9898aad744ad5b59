/*
 * coded.h -- C ABI of the MI355X (gfx950) library for (n,k) MDS-coded matrix
 * multiplication.
 *
 * Method: K. Lee, M. Lam, R. Pedarsani, D. Papailiopoulos, K. Ramchandran,
 * "Speeding Up Distributed Machine Learning Using Codes", IEEE Trans. Inf.
 * Theory (arXiv 1512.02673), Sec. III.  A data matrix A (q x r) is padded with
 * zero rows to a multiple of k and split into k row-blocks A_1..A_k of qb =
 * ceil(q/k) rows.  An (n,k) MDS code with systematic generator G = [I_k; P]
 * maps them to n coded blocks A'_i = sum_j G[i][j] A_j (A'_i = A_i for i < k).
 * Worker i computes Y_i = A'_i X; the master recovers A X from ANY k of the n
 * results by solving G_S B = Y_S and concatenating B (Sec. III-A); the
 * survivor set S is the k fastest of n workers whose runtimes follow the
 * shifted-exponential model (Sec. III-B, III-C).  Workers are simulated on
 * one GPU: all n products run, and the survivor draw picks whose results the
 * master uses.
 *
 * Conventions shared by every call:
 *  - Worker and block indices are 0-based: workers 0..k-1 hold A_0..A_{k-1}
 *    (the systematic blocks), workers k..n-1 hold the n-k parity blocks.
 *  - Matrices are row-major.  A is q x r with row stride lda >= r elements.
 *    X is r x s with row stride ldx >= s.  out is q x s with row stride ldo.
 *  - The parity buffer holds the n-k parity blocks, each qb x r, dense (row
 *    stride r), in `planes` planes: element (p, t, c) of plane h is at
 *    [h*(n-k)*qb*r + p*qb*r + t*r + c].  With planes == 2 the coded block is
 *    the exact-sum pair hi + lo: hi is the coded value rounded to the storage
 *    dtype and lo the rounded remainder, which gives the parity blocks about
 *    twice the storage precision at (n-k)/n extra bytes.  planes == 1 stores
 *    hi only.  With CODED_PLANES_LO_BF16 (fp32 inputs) the hi plane is fp32
 *    and the lo plane bfloat16: hi as above, then at byte offset
 *    4*(n-k)*qb*r the lo plane's uint16 elements [p*qb*r + t*r + c] (about
 *    32 significant bits in all; 6 instead of 8 bytes per parity element).
 *    For bf16 inputs it is the same layout as planes == 2.
 *  - Y (worker results) is n x qb x s, dense: element (i, t, c) at
 *    [(i*qb + t)*s + c].  Rows t with i*qb + t >= q of systematic blocks are
 *    the zero padding and hold 0.
 *  - Device pointers are HIP device memory of the device current when the
 *    call is made; `stream` is a hipStream_t (NULL = the null stream).
 *  - Every call that takes a stream only enqueues work on it and returns; no
 *    call synchronises the device.  Argument errors are found on the host
 *    before anything is enqueued; they return a status and set a
 *    thread-local message (coded_last_error).  Numerical singularity of a
 *    survivor set is found on the device and reported through `info`.
 *  - The caller owns every device buffer, the code's device copy of G
 *    included (coded_code_bytes gives its size); the library allocates and
 *    frees no device memory.
 *  - Nothing throws across this interface.
 */
#ifndef CODED_H
#define CODED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum coded_status {
    CODED_OK = 0,
    CODED_ERR_ARG = 1,         /* null pointer, bad index, value out of range */
    CODED_ERR_SHAPE = 2,       /* inconsistent sizes or strides */
    CODED_ERR_TOO_FEW = 3,     /* fewer than k survivors */
    CODED_ERR_SINGULAR = 4,    /* reserved: singularity is reported via info */
    CODED_ERR_HIP = 5,         /* a HIP runtime call failed */
    CODED_ERR_UNSUPPORTED = 6  /* valid but not implemented (e.g. non-systematic G) */
} coded_status;

typedef enum coded_dtype {
    CODED_F32 = 0,
    CODED_BF16 = 1,            /* bfloat16 bit patterns (uint16) */
    CODED_F64 = 2
} coded_dtype;

/* Largest n supported (survivor and worker lists travel as kernel arguments). */
#define CODED_MAX_N 128

/* Parity storage with an fp32 hi plane and a bfloat16 lo plane (see above). */
#define CODED_PLANES_LO_BF16 3

/* Opaque (n,k) code: the generator G on host and device. */
typedef struct coded_code coded_code;

/*
 * coded_code_bytes -- bytes of the caller-owned device buffer a code needs:
 * G (n*k doubles) and, when n > k, the parity rows P ((n-k)*k floats) for
 * the matrix-core encode, each starting 256-byte aligned.
 */
coded_status coded_code_bytes(int32_t n, int32_t k, int64_t* bytes);

/*
 * coded_code_create -- make the code used by every other call (Sec. III-A:
 * the (n,k) MDS code applied to the k sub-matrices).
 *   n, k      1 <= k <= n <= CODED_MAX_N.
 *   G         host, n*k doubles, row-major.  Rows 0..k-1 must be I_k exactly
 *             (systematic code); otherwise CODED_ERR_UNSUPPORTED.  The caller
 *             is responsible for G being MDS (every k x k row subset
 *             invertible); a set that is not invertible is reported at
 *             decode time through info.
 *   planes    parity storage: 2 (hi + lo, default recipe), 1 (hi only) or
 *             CODED_PLANES_LO_BF16 (fp32 hi + bfloat16 lo, for the
 *             HBM-bound single-vector product: 6 bytes per parity element).
 *             With that mode fp32 products with s > 1 run the general
 *             vector kernel instead of the matrix cores, and coded_matmul
 *             does not take its single-launch path for small problems;
 *             results keep the same bounds.
 *   device_buf, device_buf_bytes
 *             caller-owned device memory of the current device, 16-byte
 *             aligned, at least coded_code_bytes(n, k) bytes (else
 *             CODED_ERR_ARG).  The call copies G (and P) into it
 *             synchronously; the kernels read it, so it must stay allocated
 *             and unmodified until the code is destroyed.
 *   out       receives the new code (a host object: the host copy of G, and
 *             the straggler runner's streams and events once used); destroy
 *             with coded_code_destroy.  Device work that uses the code must
 *             be finished before destroying it or freeing device_buf.
 */
coded_status coded_code_create(int32_t n, int32_t k, const double* G, int32_t planes, void* device_buf,
                               int64_t device_buf_bytes, coded_code** out);
coded_status coded_code_destroy(coded_code* code);
coded_status coded_code_info(const coded_code* code, int32_t* n, int32_t* k, int32_t* planes);

/*
 * coded_sizes -- bytes of the caller-allocated buffers for an A of q x r,
 * X of r x s, compute dtype dt and worker-result dtype y_dt.
 *   parity_bytes     the parity buffer (planes * (n-k) * qb * r elements of dt;
 *                    CODED_PLANES_LO_BF16 with fp32: 6 * (n-k) * qb * r bytes)
 *   y_bytes          Y (n * qb * s elements of y_dt)
 *   workspace_bytes  workspace of coded_matmul (its Y, in y_dt = F64 for F32
 *                    inputs and F32 for BF16 inputs, followed by the worker
 *                    workspace)
 *   worker_workspace_bytes  workspace of coded_worker_mm: 0 for F32 inputs;
 *                    X transposed (s x r bf16, 256-byte aligned size) for
 *                    BF16 inputs, so that the matrix-core kernel reads X
 *                    along K in 16-byte pieces
 * Any output pointer may be NULL.
 */
coded_status coded_sizes(const coded_code* code, coded_dtype dt, coded_dtype y_dt, int64_t q, int64_t r,
                         int64_t s, int64_t* parity_bytes, int64_t* y_bytes, int64_t* workspace_bytes,
                         int64_t* worker_workspace_bytes);

/*
 * coded_encode -- the n-k parity blocks A'_{k+p} = sum_j P[p][j] A_j
 * (Sec. III-A: the code applied to each element of the sub-matrices; the k
 * systematic blocks are A itself and are not copied).  Rows of A at or beyond
 * q are the zero padding of Sec. III-A's footnote and are never read.
 *   dt        CODED_F32: sums in fp64; CODED_BF16: every P entry must be a
 *             bfloat16 value (else CODED_ERR_ARG), sums in fp32.  For bf16
 *             codes with k = 24, n - k = 8 and two planes, r a multiple of 64
 *             below 2^23, lda a multiple of 8 below 2^25 and A, parity
 *             16-byte aligned, each column's
 *             sum is formed on the matrix cores (exact products, one fp32
 *             result); coded_encode_worker_mm writes the same planes.
 *   A         device, q x r of dt, row stride lda.
 *   parity    device, the parity buffer (layout above), written in full.
 */
coded_status coded_encode(const coded_code* code, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                          void* parity, void* stream);

/*
 * coded_worker_mm -- the n local products Y_i = A'_i X (Sec. III-A: worker i
 * multiplies its stored block by the multicast input).  All workers run
 * unless worker_mask says otherwise.
 *   A, parity  device, as written by coded_encode for the same q, r, dt.
 *   X          device, r x s of dt, row stride ldx (s == 1 requires ldx == 1).
 *   worker_mask host, n bytes or NULL: worker i runs iff mask[i] != 0.
 *              Rows of Y of workers that do not run are left untouched.
 *   Y          device, n x qb x s of y_dt (layout above).
 *   y_dt       CODED_F64 (dt = F32: products accumulate in fp64) or
 *              CODED_F32 (dt = F32: fp64 accumulate, rounded on store;
 *              dt = BF16: fp32 accumulate on the matrix cores).
 *   workspace  device, coded_sizes' worker_workspace_bytes; may be NULL when
 *              that size is 0 (fp32 inputs).  For bf16 inputs NULL selects a
 *              slower vector kernel.
 */
coded_status coded_worker_mm(const coded_code* code, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                             const void* parity, const void* X, int64_t s, int64_t ldx, const uint8_t* worker_mask,
                             void* Y, coded_dtype y_dt, void* workspace, void* stream);

/*
 * coded_encode_worker_mm -- the parity blocks and all n worker products in
 * one call (Sec. III-A: the master encodes the sub-matrices, every worker
 * multiplies its block by the multicast input).  The result equals
 * coded_encode followed by coded_worker_mm for every worker: parity is written
 * exactly as coded_encode writes it, and Y holds every worker's product.  For
 * the bf16 shapes coded_encode forms on the matrix cores, with s = 64 and a
 * 16-byte aligned workspace, A is read from memory once for both (the parity
 * rows feed the products from on-chip memory); other inputs run the two steps
 * one after the other.  Products of one worker may be summed in another order
 * than coded_worker_mm's (fp32 accumulation; equal within rounding).
 *   A, X, s, ldx, Y, y_dt, workspace as for coded_worker_mm (workspace is
 *   required for bf16 inputs); parity as for coded_encode.
 */
coded_status coded_encode_worker_mm(const coded_code* code, coded_dtype dt, const void* A, int64_t q, int64_t r,
                                    int64_t lda, void* parity, const void* X, int64_t s, int64_t ldx, void* Y,
                                    coded_dtype y_dt, void* workspace, void* stream);

/*
 * coded_decode -- dec(indices, results) of Sec. III-A for one survivor set.
 *   survivors  host, `count` worker indices in arrival order; the first k are
 *              used (count < k: CODED_ERR_TOO_FEW; an index outside [0,n) or
 *              a repeat among the first k: CODED_ERR_ARG).  The result does
 *              not depend on their order.
 *   Y          device, n x qb x s of y_dt (CODED_F64 or CODED_F32); only the
 *              survivors' rows are read.
 *   out        device fp32, q x s, row stride ldo >= s.  Padding rows are not
 *              written.  Systematic survivors are copied, the missing blocks
 *              are solved for in fp64 (LU of the survivor sub-matrix of G,
 *              partial pivoting, systematic rows first).
 *   info       device int32[1]: set to 0 on success, or j > 0 when pivot j
 *              of the k x k LU is exactly zero (out is then not written).
 */
coded_status coded_decode(const coded_code* code, const int32_t* survivors, int32_t count, const void* Y,
                          coded_dtype y_dt, int64_t q, int64_t s, float* out, int64_t ldo, int32_t* info,
                          void* stream);

/*
 * coded_decode_batched -- coded_decode for `batch` survivor sets at once (one
 * decode per set, all sharing Y).
 *   sets       device int32, batch x k, any order within a row.  A row with an
 *              index outside [0,n) or a repeat gets info = -1 and no output.
 *   out        device fp32; set b writes q x s at out + b*out_stride, row
 *              stride ldo.
 *   info       device int32[batch] (0, -1, or the zero-pivot index).
 */
coded_status coded_decode_batched(const coded_code* code, const int32_t* sets, int32_t batch, const void* Y,
                                  coded_dtype y_dt, int64_t q, int64_t s, float* out, int64_t ldo,
                                  int64_t out_stride, int32_t* info, void* stream);

/*
 * coded_draw_survivors -- host only.  The k fastest of n workers in draw
 * `draw` (Sec. III-B eq. mds_coded; Sec. III-C).  Worker i's mother-runtime
 * sample is T0 = shift + E/rate, E = -ln U, with U from the 64-bit word
 * u = SplitMix64 output number (4<<56 | draw<<16 | i) of the generator seeded
 * with `seed`, U = ((u >> 11) + 0.5) * 2^-53; its task time is T0 / k.  The k
 * workers with the largest u are the k smallest runtimes (ties to the lower
 * index), so the set is chosen in integer arithmetic.
 *   survivors_out  host int32[k], ascending.
 *   t_overall_out  host, T_(k), the k-th smallest task time (may be NULL).
 * Requires rate > 0, draw < 2^40.
 */
coded_status coded_draw_survivors(int32_t n, int32_t k, uint64_t seed, uint64_t draw, double shift, double rate,
                                  int32_t* survivors_out, double* t_overall_out);

/*
 * coded_draw_survivor_sets -- host only.  `batch` distinct survivor sets with
 * at least min_parity parity workers: draws first_draw, first_draw+1, ... are
 * taken in order; a set is kept if it qualifies and differs from every set
 * kept before.  sets_out: host int32[batch*k], each row ascending.
 * next_draw_out (may be NULL): first draw not consumed.  Fails with
 * CODED_ERR_ARG if min_parity > min(k, n-k), or if batch exceeds the number
 * of distinct qualifying sets, sum over m >= min_parity of C(k,m) C(n-k,m)
 * (checked before any draw, so the call always ends).
 */
coded_status coded_draw_survivor_sets(int32_t n, int32_t k, uint64_t seed, uint64_t first_draw, int32_t batch,
                                      int32_t min_parity, int32_t* sets_out, uint64_t* next_draw_out);

/*
 * coded_matmul -- one coded product (Sec. III-A protocol): encode (unless
 * parity_ready), draw the survivors on the host, run all n worker products
 * into the workspace, decode from the survivors into out.
 *   dt          CODED_F32 (worker results in fp64) or CODED_BF16 (fp32).
 *   parity      device parity buffer; written first when parity_ready == 0.
 *   seed, draw, shift, rate   as coded_draw_survivors.
 *   survivors_out  host int32[k] (may be NULL); t_overall_out may be NULL.
 *   workspace   device, coded_sizes' workspace_bytes; holds every worker's
 *               result Y (n x qb x s) when the call completes.
 *   info        device int32[1], as coded_decode.
 * Small fp32 problems with one column (n <= 16, q*r <= 2^22, r and lda
 * multiples of 4, A, parity and X 16-byte aligned) run as one launch: each
 * block row's parity rows, products and decoded outputs are formed together,
 * since block row t of every step depends on block row t of the data only.
 * The planes written equal coded_encode's; results agree with the separate
 * steps to fp64 summation order.
 */
coded_status coded_matmul(const coded_code* code, coded_dtype dt, const void* A, int64_t q, int64_t r, int64_t lda,
                          void* parity, int32_t parity_ready, const void* X, int64_t s, int64_t ldx, uint64_t seed,
                          uint64_t draw, double shift, double rate, int32_t* survivors_out, double* t_overall_out,
                          float* out, int64_t ldo, void* workspace, int32_t* info, void* stream);

/* Bytes of the device scratch that coded_matmul_noalloc uses on each GPU. */
#define CODED_NOALLOC_SCRATCH_BYTES (64u << 20)

/*
 * coded_matmul_noalloc -- coded_matmul for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments and results as coded_matmul, minus
 * the workspace: the worker results (and, for bf16, X transposed) live in a
 * library-owned static device array of CODED_NOALLOC_SCRATCH_BYTES bytes, one
 * per GPU, held from the library's load until the process ends.  The call
 * allocates and frees nothing.
 *   A problem whose coded_sizes workspace_bytes exceeds
 *   CODED_NOALLOC_SCRATCH_BYTES fails with CODED_ERR_UNSUPPORTED before
 *   anything is enqueued.
 *   Every call on a GPU uses that GPU's one array: calls that overlap on a
 *   GPU (other threads, or other streams without ordering between them) race
 *   on it; serialise them.  The array keeps the last call's worker results;
 *   nothing in a call depends on its earlier contents.
 */
coded_status coded_matmul_noalloc(const coded_code* code, coded_dtype dt, const void* A, int64_t q, int64_t r,
                                  int64_t lda, void* parity, int32_t parity_ready, const void* X, int64_t s,
                                  int64_t ldx, uint64_t seed, uint64_t draw, double shift, double rate,
                                  int32_t* survivors_out, double* t_overall_out, float* out, int64_t ldo,
                                  int32_t* info, void* stream);

/*
 * coded_straggler_matmul -- one coded product with real, timed straggling:
 * the master/worker protocol of Sec. III-A run against the clock, with the
 * worker runtimes of Sec. III-B/C (eq. shifted_exp) as start delays.
 * Worker i's task time T_i = (shift - ln U_i / rate) / k comes from the same
 * SplitMix64 word as coded_draw_survivors.  At T_i * time_unit_us
 * microseconds after the call begins the host enqueues worker i's product
 * (on one of four internal default-priority streams, after the work already
 * on `stream`) and an event behind it.  The host polls the events: the first
 * k products seen complete are the survivors, in arrival order, and the
 * decode is enqueued on `stream` when the k-th arrives.  Then the other
 * workers are started at once (launch_all != 0) or never (launch_all == 0:
 * only the workers started before the k-th arrival compute).  The call
 * returns when the decode has completed, so it blocks the host; work
 * enqueued on `stream` afterwards waits for every product it started.
 *   dt, A, parity, X, s, ldx   as coded_worker_mm; parity must be ready.
 *   Y          device n x qb x s of y_dt (as coded_worker_mm); rows of
 *              workers that do not run are left untouched.
 *   workspace  coded_sizes' worker_workspace_bytes (BF16: required).
 *   out, ldo, info   as coded_decode.
 *   survivors_out  host int32[k] or NULL: the survivors in arrival order.
 *   timeline_out   host double[3 n] or NULL: for worker i, [3i] its start
 *              time, [3i+1] when it was enqueued, [3i+2] when the host saw it
 *              complete, in microseconds from the call's start (-1: not
 *              enqueued, or not seen complete before the decode).
 *   latency_us_out host double or NULL: call start to decode complete.
 * Requires rate > 0, time_unit_us >= 0 and a k-th start time under 60 s.
 * Calls with the same code object must not overlap (the internal streams
 * and events belong to the code).
 */
coded_status coded_straggler_matmul(coded_code* code, coded_dtype dt, const void* A, int64_t q, int64_t r,
                                    int64_t lda, const void* parity, const void* X, int64_t s, int64_t ldx,
                                    uint64_t seed, uint64_t draw, double shift, double rate, double time_unit_us,
                                    int32_t launch_all, void* Y, coded_dtype y_dt, void* workspace, float* out,
                                    int64_t ldo, int32_t* info, int32_t* survivors_out, double* timeline_out,
                                    double* latency_us_out, void* stream);

/*
 * coded_transpose -- AT = A^T for fp32 A (q x r, row stride lda) into AT
 * (r x q, row stride ldat >= q).  This forms the column split of A that the
 * transposed code of coded gradient descent encodes (Sec. III-E: worker i
 * stores the i-th row split of A and the i-th column split).  Device
 * pointers; A and AT must not overlap.
 */
coded_status coded_transpose(const float* A, int64_t q, int64_t r, int64_t lda, float* AT, int64_t ldat,
                             void* stream);

/*
 * coded_gd_sizes -- workspace bytes of coded_gd_step for codes codeA (over
 * the q rows of A) and codeAT (over the r rows of A^T).
 */
coded_status coded_gd_sizes(const coded_code* codeA, const coded_code* codeAT, int64_t q, int64_t r,
                            int64_t* workspace_bytes);

/*
 * coded_gd_step -- one iteration of coded gradient descent for least squares
 * (Sec. III-E, eq. exact_gradient): x <- x - eta * A^T (A x - y), where A x is
 * an (n1,k1)-coded product over the row split of A (code codeA, survivors of
 * draw 2*iteration) and A^T z an (n2,k2)-coded product over the row split of
 * A^T (code codeAT, survivors of draw 2*iteration + 1).  The residual
 * z = A x - y and the update are fused into the two decodes.
 *   A, parityA    device fp32, q x r (row stride lda) and its coded parity
 *                 (coded_encode with codeA).
 *   AT, parityAT  device fp32, r x q (row stride ldat; e.g. from
 *                 coded_transpose) and its coded parity (codeAT).
 *   y             device fp32[q]; x device fp32[r], updated in place.
 *   eta           step size as applied (no normalisation inside).
 *   workspace     device, coded_gd_sizes bytes (worker results of both
 *                 products and z).
 *   info          device int32[2]: decode status of the two products.
 *   survivors_out host int32[k1 + k2] or NULL: both survivor sets, ascending.
 */
coded_status coded_gd_step(const coded_code* codeA, const coded_code* codeAT, const float* A, int64_t lda,
                           const float* parityA, const float* AT, int64_t ldat, const float* parityAT, int64_t q,
                           int64_t r, const float* y, float* x, double eta, uint64_t seed, uint64_t iteration,
                           double shift, double rate, void* workspace, int32_t* info, int32_t* survivors_out,
                           void* stream);

/*
 * coded_simulate_runtimes -- Monte-Carlo of the runtime model of Sec. III-B
 * to III-D.  Draw d (first_draw <= d < first_draw + count) gives worker i the
 * mother-runtime sample T0 = shift - ln(U)/rate from the same SplitMix64 word
 * as coded_draw_survivors, and the overall runtime of one job under:
 *   t_uncoded[d]     n subtasks of T0/n: the slowest (eq. uncoded);
 *   t_repetition[d]  k tasks of T0/k, each replicated on n/k consecutive
 *                    workers: the slowest task's fastest replica (eq.
 *                    rep_coded); requires k | n;
 *   t_mds[d]         (n,k) MDS, tasks of T0/k: the k-th finisher (eq.
 *                    mds_coded; equals coded_draw_survivors' T_(k)).
 * Output pointers are device fp64[count]; any may be NULL to skip a scheme.
 */
coded_status coded_simulate_runtimes(int32_t n, int32_t k, uint64_t seed, uint64_t first_draw, int64_t count,
                                     double shift, double rate, double* t_uncoded, double* t_repetition,
                                     double* t_mds, void* stream);

/*
 * coded_optimal_k -- host only.  Lemma 2 (Sec. III-D): with the shifted-
 * exponential model (shift 1, straggling parameter rate), the expected MDS
 * runtime is minimised by k* = [1 + 1/W_{-1}(-e^{-rate-1})] n, with value
 * T* = -W_{-1}(-e^{-rate-1}) / (rate n), where W_{-1} is the lower branch of
 * Lambert W.  k_best is the integer k in [1, n] minimising the exact expected
 * runtime (1/k)(1 + (H_n - H_{n-k})/rate) (smallest k on ties).  Any output
 * pointer may be NULL.
 */
coded_status coded_optimal_k(int32_t n, double rate, double* k_star, double* t_star, int32_t* k_best);

/* Static text of a status code. */
const char* coded_status_string(coded_status status);
/* Message of the last failing call on this thread ("" if none). */
const char* coded_last_error(void);
/* Library version string. */
const char* coded_version(void);

/* ---------------------------------------------------------------- coded shuffling
 * Sec. IV: before every iteration the q data rows are partitioned at random
 * among n workers (S_i, q/n rows each); worker i's cache C_i holds S_i and
 * s - q/n other rows.  The master multicasts, for every worker group I with
 * |I| >= 2, the sum over i in I of the rows A(S_i cap C~_{I - i}) (C~_J: the
 * rows cached by exactly the workers of J), each list zero-padded to the
 * longest (Algorithm 1); worker i recovers its rows by subtracting the other
 * members' rows, which it caches.  The cache update rule keeps the new S_i
 * and s - q/n rows drawn from the old cache minus S_i.
 * Draws: counter-based SplitMix64 of `seed` -- the partition of iteration t
 * ranks the rows by output number (8<<56 | t<<40 | row) and deals them out
 * q/n at a time; the cache rule of iteration t keeps, for worker i, the rows
 * with the smallest output number (9<<56 | t<<40 | row<<6 | i) (ties: lower
 * row).  The first caches are that rule applied to the whole data set.
 * The state and the plan are host objects; encode and decode run on the
 * device over device copies of the plan's tables.
 */
typedef struct coded_shuffle coded_shuffle;

/* n in [1, 64] workers, q rows (a multiple of n, below 2^31), cache_rows in
 * [q/n, q]; draws the partition and the caches of iteration 0. */
coded_status coded_shuffle_create(int32_t n, int64_t q, int64_t cache_rows, uint64_t seed, coded_shuffle** out);
coded_status coded_shuffle_destroy(coded_shuffle* sh);

/* The current iteration t, partition (host int32[q]: worker of each row) and
 * cache signatures (host uint64[q]: bit i set when worker i caches the row);
 * any output may be NULL. */
coded_status coded_shuffle_state(const coded_shuffle* sh, int64_t* t, int32_t* assign, uint64_t* cache_sig);

/* Draws the partition of iteration t+1 and plans its transmission (replacing
 * a pending plan).  coded_rows: multicast rows (the coded rate of eq. r2 for
 * this draw); terms: rows the workers lack (the uncoded rate of eq. r1).
 * Messages are ordered by group (bit mask, increasing), a group's rows by
 * position j, and a message row's terms by worker. */
coded_status coded_shuffle_plan(coded_shuffle* sh, int64_t* coded_rows, int64_t* terms);

/* The pending plan's tables (host; any may be NULL):
 *   enc_off      int64[coded_rows + 1]: message m's terms are [enc_off[m], enc_off[m+1])
 *   enc_rows     int32[terms]: the data row of each term
 *   term_worker  int32[terms]: the worker that lacks it
 *   term_msg     int32[terms]: the message it belongs to
 *   next_assign  int32[q]: the partition of iteration t+1 */
coded_status coded_shuffle_tables(const coded_shuffle* sh, int64_t* enc_off, int32_t* enc_rows, int32_t* term_worker,
                                  int32_t* term_msg, int32_t* next_assign);

/* Applies the cache update rule for the pending plan and advances to t+1. */
coded_status coded_shuffle_commit(coded_shuffle* sh);

/* Device: M (coded_rows x r, row stride ldm) = the multicast rows, message m
 * being the fp32 sum of the rows of its terms in order.  A is q x r fp32,
 * row stride lda; the tables are device copies of coded_shuffle_tables'.  A
 * message with a table entry out of range is written as NaN. */
coded_status coded_shuffle_encode(const float* A, int64_t q, int64_t r, int64_t lda, const int64_t* enc_off,
                                  const int32_t* enc_rows, int64_t coded_rows, int64_t terms, float* M, int64_t ldm,
                                  void* stream);

/* Device: out (terms x r, row stride ldo): row d is worker term_worker[d]'s
 * copy of data row enc_rows[d], decoded as message term_msg[d] minus the
 * other terms' rows of that message, in order (fp32).  A row whose table
 * entries are out of range is written as NaN. */
coded_status coded_shuffle_decode(const float* A, int64_t q, int64_t r, int64_t lda, const float* M, int64_t ldm,
                                  const int64_t* enc_off, const int32_t* enc_rows, const int32_t* term_msg,
                                  int64_t coded_rows, int64_t terms, float* out, int64_t ldo, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CODED_H */
