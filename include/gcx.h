/*
 * gcx.h -- C ABI of the partial-straggler gradient-coding hot path on MI355X (gfx950).
 *
 * Implements, for one GPU holding all m simulated workers, the data-parallel
 * steps of the gradient-coding protocol of "Leveraging partial stragglers
 * within gradient coding" (Ramamoorthy, Meng, Girimaji):
 *
 *   gc_assign         assignment support and chunk order        (Sec. 1; Sec. 3)
 *   gc_chunk_grads    per-chunk gradients g_{D_i}               (Sec. 1)
 *   gc_sum_chunks     the exact target  sum_i g_{D_i}           (Sec. 1)
 *   gc_decode_coeffs  coverage, decodability and Algorithm 1    (Sec. 2; Sec. 2.1)
 *   gc_encode         each worker's transmitted vector g_beta   (Sec. 2)
 *   gc_reconstruct    the PS combine  sum_j R[k][j] g_j         (Sec. 2.2)
 *   gc_decode_direct  the same estimate without forming g_j     (Sec. 2; Sec. 2.2)
 *   gc_progress, gc_completion_times, gc_original_ls
 *                     the straggler simulations of Sec. 4
 *
 * Conventions (every entry point):
 *   - Row-major arrays, 0-based indices.  Chunk i is the paper's D_{i+1},
 *     worker j is W_{j+1}; positions inside a worker are 0-based (the paper's
 *     ordering matrix O keeps 1-based positions, 0 = not assigned).
 *   - The caller owns every buffer.  Pointers documented "device" must be
 *     device memory of the current HIP device; "host" pointers are host memory.
 *     Nothing is allocated by the library except what a workspace argument
 *     brings in; no handle or global state is kept between calls.
 *   - Device entry points enqueue work on `stream` (0 = the null stream) and
 *     return without synchronising; outputs are valid once the caller has
 *     synchronised the stream.  Calls on one stream are ordered.
 *   - Return value: GC_OK, or a negative status.  Arguments are validated on
 *     the host before anything is launched; a non-OK return from validation
 *     means nothing was enqueued.  Nothing is printed.
 *   - The communication factor ell satisfies 1 <= ell <= GC_MAX_ELL.  A
 *     gradient of length d is cut into ell contiguous blocks of length
 *     L = ceil(d / ell); block k covers entries [k*L, (k+1)*L) of the gradient
 *     zero-padded to length ell*L.
 */
#ifndef GCX_H
#define GCX_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define GC_OK 0
#define GC_EINVAL (-1)  /* bad size, null pointer, bad enum, inconsistent tables  */
#define GC_ELAUNCH (-2) /* the HIP runtime reported an error at launch           */
#define GC_ENOTSUP (-3) /* the current device is not gfx950                      */
#define GC_ESCRATCH (-4) /* the request needs more than the fixed scratch array   */

/* assignment kinds for gc_assign */
#define GC_ASSIGN_CYCLIC 0 /* cyclic scheme, N = m, worker j holds j..j+s (mod N) */
#define GC_ASSIGN_ORDER 1  /* tables derived from a caller-given ordering matrix O */
#define GC_ASSIGN_REGULAR 2 /* optimal ordering of a delta-regular support (Algorithm 2) */

/* losses for gc_chunk_grads */
#define GC_LOSS_LINEAR 0   /* l = (x.w - y)^2 / 2           */
#define GC_LOSS_LOGISTIC 1 /* l = log(1 + e^{x.w}) - y x.w  */

/* storage types of chunk gradients */
#define GC_F32 0
#define GC_BF16 1 /* bfloat16, accumulated in fp32 */

/* values of dec[] written by gc_decode_coeffs */
#define GC_DEC_NO 0      /* some chunk has fewer than ell processed copies    */
#define GC_DEC_YES 1     /* every chunk has at least ell processed copies      */
#define GC_DEC_INVALID 2 /* psi had an entry outside [0, delta_j]; Bc zeroed   */

#define GC_MAX_ELL 8
#define GC_MAX_M 1024     /* workers            */
#define GC_MAX_DELTA 64   /* table widths       */

/* Library version (major * 10000 + minor * 100 + patch). */
int gc_version(void);

/* Short static description of a status code. */
const char *gc_strerror(int status);

/*
 * gc_assign -- host only.  The assignment matrix A (Sec. 1, "Background") is
 * described by its support and the order in which each worker processes its
 * chunks, the ordering matrix O of Sec. 3: O[i*m + j] = 0 if chunk i is not
 * assigned to worker j, else its 1-based position inside worker j.
 *
 * kind = GC_ASSIGN_CYCLIC: requires N == m and 0 <= s < m; worker j holds
 *   chunks j, j+1, ..., j+s (mod N) in that order (the cyclic scheme whose
 *   ordering Sec. 3 states is optimal for exact GC).  Writes O (if non-NULL).
 *   delta and gamma must both equal s + 1.
 * kind = GC_ASSIGN_ORDER: O is an input; every column's non-zero entries must
 *   be 1..delta_j, once each (Sec. 3).  s is ignored.  delta >= max_j delta_j
 *   and gamma >= max_i gamma_i.
 * kind = GC_ASSIGN_REGULAR: O is in/out.  On input its non-zero pattern is the
 *   support of A, which must have N == m and exactly delta non-zeros in every
 *   row and column (e.g. the adjacency matrix of a delta-regular graph); gamma
 *   must equal delta.  Algorithm 2 (Chunk-Ordering, Sec. 3) peels delta perfect
 *   matchings P_1..P_delta off the support (Hopcroft-Karp) and O is
 *   overwritten with sum_i i * P_i, an ordering whose every row sums to
 *   delta(delta+1)/2, the optimum of Q_max.  Orderings are not unique.
 *
 * Outputs (host, int32, -1 padded past a row's length):
 *   order  [m][delta]  chunk at position t of worker j
 *   holder [N][gamma]  u-th worker holding chunk i, ascending worker index
 *   hpos   [N][gamma]  position of chunk i inside worker holder[i][u]
 * Errors: GC_EINVAL for a null table pointer, bad sizes, an O that is not an
 * ordering matrix, or tables too narrow.
 */
int gc_assign(int32_t kind, int32_t N, int32_t m, int32_t s, int32_t *O, int32_t delta,
              int32_t gamma, int32_t *order, int32_t *holder, int32_t *hpos);

/*
 * gc_qmax -- the ordering metric of Sec. 3 (host only).  For an ordering matrix
 * O [N][m] (O[i][j] = 0 if worker j does not hold chunk i, else the 1-based
 * position of chunk i in worker j's order; each worker's positions are
 * 1..delta_j once each), Q_i = the most chunks the cluster can process with no
 * copy of chunk i processed = sum over holders j of (O[i][j] - 1) + sum over the
 * other workers of delta_j; with N = m and all loads and replications equal to
 * delta this is the paper's sum_j O_ij + (m - delta - 1) delta.  Writes
 * Q [N] (may be NULL) and *qmax = max_i Q_i (1 + Q_max chunks guarantee one
 * copy of every chunk).  O, Q, qmax: host.  GC_EINVAL for an invalid O.
 */
int gc_qmax(const int32_t *O, int32_t N, int32_t m, int64_t *Q, int64_t *qmax);

/*
 * gc_chunk_grads -- per-chunk gradients (Sec. 1: g_{D_i} is the sum over the
 * samples of chunk i of the per-sample gradient) at b evaluation points:
 *   G[q][i][:] = X_i^T r,  r = X_i w_q - y_i          (GC_LOSS_LINEAR)
 *                          r = sigmoid(X_i w_q) - y_i (GC_LOSS_LOGISTIC)
 * X [N][n][d], y [N][n], W [b][d], G [b][N][d]: device fp32.  fp32 arithmetic.
 * With b >= 16 points (b % 4 == 0, d % 4 == 0) the two contractions run on the
 * fp32 matrix cores; X, y, W, G and the workspace must then be 16-byte aligned.
 * workspace: device, at least gc_chunk_grads_workspace_size(N, n, d, b) bytes.
 * Errors: GC_EINVAL for sizes < 1, a null pointer, an unknown loss, or a
 * workspace that is too small.
 */
size_t gc_chunk_grads_workspace_size(int32_t N, int32_t n, int64_t d, int32_t b);
int gc_chunk_grads(const float *X, const float *y, const float *W, int32_t N, int32_t n,
                   int64_t d, int32_t b, int32_t loss, float *G, void *workspace,
                   size_t workspace_bytes, hipStream_t stream);

/*
 * gc_sum_chunks -- gsum[x] = sum_i G[i][x], the gradient the PS wants
 * (Sec. 1, grad L = sum_j g_{D_j}).  G [N][d] device in g_dtype; gsum [d]
 * device fp32, accumulated in fp64 and rounded once.
 */
int gc_sum_chunks(const void *G, int32_t g_dtype, int32_t N, int64_t d, float *gsum,
                  hipStream_t stream);

/*
 * gc_decode_coeffs -- for each straggler pattern p (a state vector psi of
 * Sec. 2: worker j has processed the chunks at positions 0..psi[p][j]-1 of
 * its order) compute, independently and in parallel:
 *   cov[p][i]   Delta_i = number of workers that processed chunk i
 *   dec[p]      GC_DEC_YES iff every Delta_i >= ell (the exact-GC condition of
 *               Sec. 2 / Sec. 2.1), GC_DEC_NO otherwise, GC_DEC_INVALID if a
 *               psi[p][j] lies outside [0, delta_j]
 *   coef_err[p] sum_i max(0, ell - Delta_i) (the coefficient-space error of
 *               Sec. 2.1)
 *   Bc[p][j][t][k]  the encoding coefficient B^{(i)}_{j,k} of Algorithm 1 for
 *               chunk i = order[j][t]: with S_i the processed holders of chunk
 *               i and X = R[:, S_i] (ell x Delta_i), the rows of B^{(i)} on
 *               S_i are the minimum-norm least-squares solution pinv(X); zero
 *               for t >= psi[p][j], for padded table slots, and for the whole
 *               pattern when dec[p] = GC_DEC_INVALID.
 * The small solves run in fp64 (Gram matrix and Cholesky factorisation of
 * size min(ell, Delta_i)); Bc is rounded to fp32 once.
 * psi [P][m] int32, order [m][delta], holder/hpos [N][gamma] int32 (as from
 * gc_assign, -1 padded), R [ell][m] fp32, cov [P][N] int32, dec [P] uint8,
 * coef_err [P] int32, Bc [P][m][delta][ell] fp32: all device.
 * Requires 1 <= m <= GC_MAX_M, 1 <= delta, gamma <= GC_MAX_DELTA.
 * P = 0 is a no-op.  Invalid psi values are reported in dec, not by the return
 * value (psi is device data and is not read on the host).
 * Coverage-only mode: Bc = NULL skips the solves (R may then be NULL too);
 * cov may be NULL when only dec and coef_err are wanted.
 */
int gc_decode_coeffs(const int32_t *psi, int64_t P, int32_t N, int32_t m, const int32_t *order,
                     int32_t delta, const int32_t *holder, const int32_t *hpos, int32_t gamma,
                     const float *R, int32_t ell, int32_t *cov, uint8_t *dec, int32_t *coef_err,
                     float *Bc, hipStream_t stream);

/*
 * gc_encode -- what every worker transmits (Sec. 2, worker encode): for each
 * pattern p and worker j,
 *   T[p][j][x] = sum_{t < psi[p][j]} sum_{k < ell} Bc[p][j][t][k] * g_{order[j][t]}[k*L + x]
 * for 0 <= x < L, over the worker's processed prefix only.  A worker with
 * psi[p][j] <= 0 has processed nothing and transmits nothing (a straggler in
 * the sense of Sec. 1): its row T[p][j] is NOT written and keeps whatever it
 * held.  G [N][d] device in g_dtype; psi [P][m], order
 * [m][delta] int32 device; Bc [P][m][delta][ell] fp32 device (as from
 * gc_decode_coeffs); T [P][m][L] fp32 device.  fp32 accumulation.  psi is
 * clamped to [0, delta] and padded order slots are skipped.  G must be finite:
 * where the sums run on the matrix cores (bf16 G past the smallest shapes, fp32 G
 * from delta*ell >= 32 terms), a coefficient past a pattern's prefix or of a chunk
 * the worker does not hold enters as zero (and zero times a non-finite value is
 * not zero).  Accuracy per output, M = sum over its terms of |Bc||g| and
 * u = 2^-24: within u M plus the fp32 accumulation of 3 psi*ell products (bf16
 * G; coefficients split exactly into three bf16 parts), within 8u M plus that of
 * 6 psi*ell products (fp32 G on the matrix cores; G split exactly into three
 * bf16 parts as well), or gamma_{psi*ell} M (fp32 vector path).
 */
int gc_encode(const void *G, int32_t g_dtype, int32_t N, int64_t d, const int32_t *psi,
              const int32_t *order, const float *Bc, int64_t P, int32_t m, int32_t delta,
              int32_t ell, float *T, hipStream_t stream);

/*
 * gc_reconstruct -- the PS combine (Sec. 2.2, last step): block k of the
 * estimate is sum_j R[k][j] T[p][j][:] over the workers that transmitted, i.e.
 *   ghat[p][k*L + x] = sum_{j : psi[p][j] > 0} R[k][j] * T[p][j][x]   for k*L + x < d.
 * psi [P][m] int32 device, required (GC_EINVAL if NULL): it names the workers
 * that transmitted, and rows of T with psi <= 0 are never read, so the T that
 * gc_encode leaves unwritten for stragglers is combined correctly.
 * Equals sum_i g_{D_i} when the pattern is decodable; otherwise it is the
 * least-squares estimate.  If gsum is non-NULL and sqerr non-NULL,
 *   sqerr[p] = sum_x (ghat[p][x] - gsum[x])^2   (fp64 accumulation)
 * ghat may be NULL (error-only mode).  T [P][m][L], R [ell][m], ghat [P][d],
 * gsum [d] fp32, sqerr [P] fp64: device.  workspace: device, at least
 * gc_reconstruct_workspace_size(P, m, d, ell) bytes when sqerr is requested
 * (it holds per-slice partial sums, reduced in a fixed order, so sqerr is
 * deterministic).
 */
size_t gc_reconstruct_workspace_size(int64_t P, int32_t m, int64_t d, int32_t ell);
int gc_reconstruct(const float *T, const float *R, const int32_t *psi, int64_t P, int32_t m,
                   int64_t d, int32_t ell, float *ghat, const float *gsum, double *sqerr,
                   void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * gc_reconstruct_noalloc -- gc_reconstruct for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and the same results, with the squared error's
 * per-piece partial sums in a fixed array the library holds on each device
 * (GC_NOALLOC_SCRATCH_BYTES, kept until the process ends) instead of a caller
 * workspace.  Arguments and outputs as in gc_reconstruct; the caller still owns
 * T, R, psi, ghat, gsum and sqerr.  Returns GC_ESCRATCH, with nothing enqueued,
 * when gc_reconstruct_workspace_size(P, m, d, ell) exceeds
 * GC_NOALLOC_SCRATCH_BYTES (split the patterns into smaller calls).  Calls no
 * allocating routine.  All calls on one device share that device's array:
 * calls that may overlap on one device (different streams, different host
 * threads) race and must be serialised by the caller.
 */
#define GC_NOALLOC_SCRATCH_BYTES (4u << 20)
int gc_reconstruct_noalloc(const float *T, const float *R, const int32_t *psi, int64_t P, int32_t m,
                           int64_t d, int32_t ell, float *ghat, const float *gsum, double *sqerr,
                           hipStream_t stream);

/*
 * gc_decode_direct -- the same estimate as gc_decode_coeffs + gc_encode +
 * gc_reconstruct, computed at the PS without forming what the workers transmit.
 * Putting the worker encode (Sec. 2) into the combine (Sec. 2.2) gives
 *   block k of ghat[p] = sum_i sum_k' M_i[k][k'] * block k' of g_i,
 *   M_i = R[:, S_i] B^(i)[S_i, :] = R[:, S_i] pinv(R[:, S_i]),
 * the identity when Delta_i >= ell, the orthogonal projector onto the range of
 * R[:, S_i] when 0 < Delta_i < ell, and zero when Delta_i = 0 (S_i, Delta_i as
 * in gc_decode_coeffs, Sec. 2.1).  The mixing matrices are formed in fp64 and
 * rounded once to fp32; the sum over chunks is an fp32 matrix-core contraction.
 * A simulation shortcut only: in the protocol the PS never sees the g_i.
 * G [N][d] (g_dtype GC_F32 or GC_BF16 bits), psi [P][m], holder/hpos
 * [N][gamma] (gc_assign), R [ell][m]: device.  Outputs as in gc_reconstruct:
 * ghat [P][d] fp32 (may be NULL), and with gsum [d] non-NULL, sqerr [P] fp64
 * (may be NULL; deterministic), where each difference ghat - gsum, its square
 * and the sum of four neighbouring squares are formed in fp32 and every further
 * sum in fp64, so sqerr[p] is within a relative 6 * 2^-24 of the squared error
 * of the returned ghat.  At least one of ghat, sqerr.  workspace:
 * device, 16-byte aligned, at least gc_decode_direct_workspace_size(P, N, d,
 * ell) bytes.  Rows of psi must be valid (0 <= psi[p][j] <= load of j).
 * Requires N, m <= GC_MAX_M.
 */
size_t gc_decode_direct_workspace_size(int64_t P, int32_t N, int64_t d, int32_t ell);
int gc_decode_direct(const void *G, int32_t g_dtype, int32_t N, int64_t d, const int32_t *psi,
                     int64_t P, int32_t m, int32_t delta, const int32_t *holder,
                     const int32_t *hpos, int32_t gamma, const float *R, int32_t ell,
                     float *ghat, const float *gsum, double *sqerr, void *workspace,
                     size_t workspace_bytes, hipStream_t stream);

/*
 * gc_progress -- the straggler simulation of Sec. 4 at a grid of deadlines:
 * worker j finishes the chunk at position t of its order at time
 * sum_{u <= t} tau[r][j][u] (fp64, summed in position order); failed workers
 * finish nothing.  psi[r][g][j] = number of chunks worker j has finished by T[g],
 * i.e. the state vector the PS would broadcast at that deadline.
 * tau [R][m][delta] fp64, failed [R][m] uint8 (non-zero = failed) or NULL,
 * T [G] fp64, psi [R][G][m] int32: all device.
 */
int gc_progress(const double *tau, const uint8_t *failed, int64_t R, int32_t m, int32_t delta,
                const double *T, int32_t G, int32_t *psi, hipStream_t stream);

/*
 * gc_completion_times -- exact-GC completion time of each trial (Sec. 4, the
 * exact-GC simulation): the first time at which every chunk has been processed
 * at least ell times, i.e. for each chunk the ell-th smallest finish time over
 * its holders, maximised over chunks.
 *   partial[r]   every processed chunk counts (the proposed protocol)
 *   original[r]  only workers that have finished all delta of their chunks
 *                count (original GC)
 * +inf where failures leave some chunk with fewer than ell live holders.
 * Every worker must hold delta chunks (tau [R][m][delta]).  tau fp64,
 * failed [R][m] uint8 or NULL, holder/hpos [N][gamma] int32 (gc_assign),
 * partial/original [R] fp64: all device.
 */
int gc_completion_times(const double *tau, const uint8_t *failed, int64_t R, int32_t N,
                        int32_t m, int32_t delta, const int32_t *holder, const int32_t *hpos,
                        int32_t gamma, int32_t ell, double *partial, double *original,
                        hipStream_t stream);

/*
 * gc_original_ls -- original GC's approximate decoding, the comparison of Sec. 4:
 * with F the workers that have processed all their chunks (psi[p][j] equal to
 * the worker's load), r = argmin ||A_F r - 1||_2 over the 0/1 assignment
 * support A (r_j = 0 outside F), and err[p] = ||A r - 1||^2.  Solved per
 * pattern by CGLS in fp64 from r = 0 (so the minimum-norm solution when A_F is
 * rank deficient), stopping when ||A_F^T (1 - A_F r)|| <= tol times its
 * initial value or after max_iter iterations (iters[p] = iterations used;
 * iters may be NULL).  psi [P][m], order [m][delta], holder [N][gamma] int32,
 * err [P] fp64: all device.  Requires N, m <= GC_MAX_M.
 */
int gc_original_ls(const int32_t *psi, int64_t P, int32_t N, int32_t m, const int32_t *order,
                   int32_t delta, const int32_t *holder, int32_t gamma, int32_t max_iter,
                   double tol, double *err, int32_t *iters, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* GCX_H */
