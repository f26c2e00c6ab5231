/*
 * flashgmm.h - C ABI of the fused diagonal-covariance GMM EM iteration for
 * AMD Instinct MI355X (gfx950).
 *
 * Model (Flash-GMM paper, Sec. 2, with a diagonal covariance in place of the
 * paper's isotropic sigma_k^2 I): K components with weights pi_k, means
 * mu_k in R^D and per-dimension variances var_kd.
 *
 * Conventions shared by every entry point
 *   - Every pointer argument is a DEVICE pointer owned by the caller; the
 *     library never allocates and never frees.  Scratch memory comes from the
 *     caller's workspace `ws` of `ws_bytes` bytes, sized by
 *     gmm_workspace_bytes().  The workspace must be 256-byte aligned.
 *   - Layouts are row-major and contiguous: x[n*d], means/vars/s/q[k*d],
 *     weights/nk[k].  Parameters are fp32, statistics fp64.
 *   - Every call only enqueues work on `stream` and returns; results are
 *     valid once the caller synchronises the stream.  Calls that share a
 *     workspace must be ordered on one stream.  Calls with separate
 *     workspaces (and, for the out-of-core call, separate staging buffers and
 *     copy streams) may run concurrently on different streams: the library
 *     keeps no state between calls apart from the optional phase timer and
 *     the statistics chunk limit.
 *   - Errors: argument checks run on the host before anything is enqueued and
 *     return a negative gmm_status (nothing is enqueued then).  A HIP error
 *     reported at launch returns GMM_ERR_DEVICE.  NaN or Inf in the inputs is
 *     not checked; it propagates into the outputs.
 *   - Limits: 1 <= d <= GMM_MAX_D, 1 <= k <= GMM_MAX_K, n >= 1 (n may exceed
 *     2^31), 1 <= m <= GMM_MAX_M.  Shapes beyond them return
 *     GMM_ERR_UNSUPPORTED.
 *   - Results are bitwise deterministic for a given (n, d, k), inputs and
 *     statistics chunk limit (gmm_set_stats_chunk_limit): every sum runs in a
 *     fixed order.  The assignment kernels append candidates to per-point
 *     lists with LDS atomics; each list is sorted before its terms are
 *     summed, so no result depends on the order of arrival.
 */
#ifndef FLASHGMM_H
#define FLASHGMM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GMM_MAX_D 1024
#define GMM_MAX_K 65535
#define GMM_MAX_M 8

typedef enum {
  GMM_OK = 0,
  GMM_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, bad m/tau */
  GMM_ERR_UNSUPPORTED = -2, /* d, k or m beyond the library's limits */
  GMM_ERR_WORKSPACE = -3,   /* workspace missing, misaligned or too small */
  GMM_ERR_DEVICE = -4,      /* a HIP call or kernel launch failed */
  GMM_ERR_FILL = -5         /* the caller's fill function reported a failure */
} gmm_status;

/* Human-readable name of a status code (static string). */
const char* gmm_status_string(int status);

/*
 * Bytes of workspace needed by gmm_estep_accumulate / gmm_fit (m = 0) or by
 * gmm_assign_topk (m >= 1) for n points in d dimensions and k components.
 * Returns 0 when the shape is unsupported.  The size grows as O(n) (about
 * 110 bytes per point: the fp64 log-normaliser, the stored exact pairs and
 * their bucketed records, a mask of the component blocks the dense
 * statistics take, and flag bytes) plus O(k d) for the parameters and the
 * per-workgroup partial statistics; it never holds an n x k array.
 */
size_t gmm_workspace_bytes(int64_t n, int32_t d, int32_t k, int32_t m);

/*
 * E-step and sufficient statistics of one EM iteration (Sec. 3.1 and
 * Algorithm 1 of the paper, steps 1-2, with the diagonal model): at the
 * parameters (weights, means, vars), for every point i and component k
 *   l_ik   = log pi_k + log N(x_i | mu_k, diag var_k)
 *   log Z_i = log sum_k exp(l_ik),  r_ik = exp(l_ik - log Z_i)
 * and ADDS into the caller's fp64 accumulators
 *   nk[k]     += sum_i r_ik
 *   s[k*d+j]  += sum_i r_ik x_ij
 *   q[k*d+j]  += sum_i r_ik x_ij^2
 *   *loglik   += sum_i log Z_i          (natural log, 2*pi constant included)
 * The caller zeroes them first; adding lets row chunks of one data set, or
 * shards of it, be accumulated into one set of statistics.
 * Components with weight 0 are dead: l_ik = -inf, they receive nothing.
 * The n x k responsibility matrix is never stored.
 *   x        [n*d] fp32 points          weights [k] fp32 (>= 0)
 *   means    [k*d] fp32                 vars    [k*d] fp32 (> 0)
 *   nk       [k] fp64, s/q [k*d] fp64, loglik [1] fp64 (all +=)
 */
int gmm_estep_accumulate(const float* x, int64_t n, int32_t d, int32_t k, const float* weights,
                         const float* means, const float* vars, double* nk, double* s, double* q,
                         double* loglik, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * M-step from the statistics (paper Eqs. Nk, muk, sig and Algorithm 1's
 * final step, per dimension), in fp64, written back as fp32 parameters:
 *   pi_k    = nk[k] / n_total
 *   mu_kj   = s[k*d+j] / nk[k]
 *   var_kj  = max(var_floor, q[k*d+j] / nk[k] - mu_kj^2)
 * A component with nk[k] == 0 exactly keeps its mean and variances and gets
 * weight 0.  weights/means/vars hold the old parameters on entry (needed for
 * that rule) and the new ones on return.  n_total > 0, var_floor >= 0.
 */
int gmm_mstep(const double* nk, const double* s, const double* q, double n_total, int32_t d,
              int32_t k, float var_floor, float* weights, float* means, float* vars,
              hipStream_t stream);

/*
 * n_iters full EM iterations (Algorithm 1 of the paper, repeated; Sec. 2
 * stops on a log-likelihood change or an iteration cap, here the cap alone)
 * from Theta_0 = (weights, means, vars), updated
 * in place to Theta_{n_iters}.  loglik_hist[t] (fp64, device, n_iters
 * entries) receives LL(Theta_t), the log-likelihood computed in iteration
 * t's E-step, before its M-step.  Each iteration is gmm_estep_accumulate
 * followed by gmm_mstep with n_total = n.  Resuming means calling again with
 * the returned parameters.
 */
int gmm_fit(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters, float var_floor,
            float* weights, float* means, float* vars, double* loglik_hist, void* ws,
            size_t ws_bytes, hipStream_t stream);

/*
 * Reduced-precision E-step and fit: the calls above with the log-densities
 * left at the precision of the screening pass, i.e. the expanded form
 * (Sec. 3, the two contractions X (mu/var)^T and X^2 (1/var)^T) on split
 * bf16 matrix products, three bf16 products per fp32 product (fp32 above
 * d = 128), with fp32 accumulation.  The exact calls recompute the few
 * pairs that carry a point's mass in the direct form, in fp64; these calls
 * keep the screened values for them too.  Everything else (arguments,
 * accumulation, workspace, dead and ill-conditioned components, status
 * codes) is as in gmm_estep_accumulate / gmm_fit.
 * Error: a screened log-density is within about 2^-22 log2(e) (S_k + d)
 * log2 units of the exact one, S_k = sum_j mu_kj^2 / var_kj, so a
 * responsibility is within about e = 2 ln(2) 2^-22 log2(e) (S + d) =
 * 2^-21 (S + d) relative (both the pair and log Z_i carry the error), S the
 * largest S_k among the point's significant components: e is about 3e-4 at
 * S + d = 640, the paper-shape workloads.  The variances the M-step forms from these
 * statistics are differences Q/N - mu^2, so a relative error e of the
 * weighted sums becomes about 3 e (mu^2 + var) in a variance.  The stated
 * tolerances of these calls (statistics and the M-step's parameters, against
 * exact fp64 arithmetic; for inputs with S + d up to about 1800) are
 *   N_k |err| <= 2e-3 max(N_k, 1),  mu_kj |err| <= 2e-3 max(|mu_kj|, sigma_kj),
 *   var_kj |err| <= 5e-3 (mu_kj^2 + var_kj) (N_k >= 1),  LL |err| <= 2e-5 |LL|.
 */
int gmm_estep_accumulate_screened(const float* x, int64_t n, int32_t d, int32_t k,
                                  const float* weights, const float* means, const float* vars,
                                  double* nk, double* s, double* q, double* loglik, void* ws,
                                  size_t ws_bytes, hipStream_t stream);
int gmm_fit_screened(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters,
                     float var_floor, float* weights, float* means, float* vars,
                     double* loglik_hist, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Top-m multi-assignment (Sec. 4.2 single assignment, Sec. 4.3 multiple
 * assignment): a fresh E-step at the given parameters; for every point the
 * components ranked by responsibility (ties to the lower index).  Rank 1 is
 * always assigned; rank j > 1 is assigned only if its responsibility is
 * strictly greater than tau (the paper uses m = 2, tau = 1/K).
 *   idx  [n*m] int32: component indices, -1 for an empty slot
 *   resp [n*m] fp32 : their responsibilities, 0 for an empty slot
 * 1 <= m <= GMM_MAX_M and m <= k; 0 <= tau < 1.  The ranking is exact: a
 * screening pass bounds its own error per component, every component that
 * can be among a point's m + 2 largest is recomputed in fp64 and ranked (all
 * k in fp64 when more than 32 qualify).  A responsibility divides the exact
 * term by a normaliser whose part from the other components keeps the
 * screening's error (within 1e-4 of exact in the tests).
 */
int gmm_assign_topk(const float* x, int64_t n, int32_t d, int32_t k, const float* weights,
                    const float* means, const float* vars, int32_t m, float tau, int32_t* idx,
                    float* resp, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Out-of-core E-step (data larger than the GPU's memory, the paper's
 * Limitations section, paragraph Scale: X streamed through the device in
 * chunks accumulating into the same O(KD) statistics).  x_host [n*d] fp32 lives in
 * page-locked host memory that the caller allocated (hipHostMalloc); the
 * rows are uploaded chunk_rows at a time on copy_stream into the two halves
 * of the caller's device staging buffer staging [2*min(chunk_rows, n)*d fp32],
 * while the E-step of the previous chunk runs on `stream`.  The statistics
 * are ADDED exactly as gmm_estep_accumulate adds them when called chunk by
 * chunk, in row order, on device copies of the chunks (the result is the
 * same, bit for bit).  ws is sized by gmm_workspace_bytes(min(chunk_rows, n),
 * d, k, 0).  The first upload waits for the work already enqueued on `stream`
 * (which may still read the staging buffer); `stream` holds the statistics
 * when it completes.  copy_stream and stream may be the same stream (then
 * nothing overlaps).  Returns GMM_ERR_INVALID_ARG for a null pointer or
 * chunk_rows < 1, plus the codes of gmm_estep_accumulate.
 */
int gmm_estep_accumulate_streamed(const float* x_host, int64_t n, int32_t d, int32_t k,
                                  const float* weights, const float* means, const float* vars,
                                  double* nk, double* s, double* q, double* loglik,
                                  int64_t chunk_rows, float* staging, void* ws, size_t ws_bytes,
                                  hipStream_t stream, hipStream_t copy_stream);

/*
 * Source of the rows of an out-of-core E-step: writes rows row0 .. row0 +
 * rows - 1 of X (fp32, d values a row, row-major) to dst [rows*d], a slot of
 * the caller's page-locked ring, and returns 0, or non-zero to stop the call.
 * It runs on the calling thread, in row order, each row exactly once.
 */
typedef int (*gmm_fill_fn)(void* user, int64_t row0, int64_t rows, int32_t d, float* dst);

/*
 * A gmm_fill_fn for X held whole in ordinary (pageable) host memory: user is
 * the address of X [n*d] fp32, and the rows are copied with up to 8 host
 * threads.  Returns 0, or 1 for a null pointer or rows < 0.
 */
int gmm_fill_pageable(void* user, int64_t row0, int64_t rows, int32_t d, float* dst);

/*
 * Out-of-core E-step over a ring of page-locked staging chunks (the paper's
 * Limitations section, paragraph Scale: X streamed through the device in
 * chunks accumulating into the same O(KD) statistics), for X that is not held
 * whole in page-locked memory: in pageable memory (fill = gmm_fill_pageable),
 * in a file, or produced as it is consumed.  For each chunk of chunk_rows rows,
 * in row order, the calling thread has `fill` write the rows into the next of
 * the ring_slots slots of ring [ring_slots*min(chunk_rows, n)*d fp32,
 * page-locked host memory that the caller allocated], the slot is uploaded
 * on copy_stream into one half of staging [2*min(chunk_rows, n)*d fp32,
 * device], and the chunk's E-step is enqueued on `stream`.  A slot is filled
 * again only once its previous upload has completed (the calling thread
 * waits for it), so filling chunk c overlaps the upload of chunk c - 1 and
 * the E-step of chunk c - 2.  Before the first fill the calling thread waits
 * for the work already enqueued on copy_stream (which may still read the
 * ring); the first upload waits for the work already enqueued on `stream`
 * (which may still read the staging buffer).  The statistics are ADDED
 * exactly as gmm_estep_accumulate adds them when called chunk by chunk, in
 * row order, on device copies of the chunks (the same result, bit for bit).
 * ws is sized by gmm_workspace_bytes(min(chunk_rows, n), d, k, 0).  The call
 * returns once every chunk has been filled and enqueued; the ring and the
 * staging buffer are read until `stream` completes.  Returns
 * GMM_ERR_INVALID_ARG for a null pointer, chunk_rows < 1 or ring_slots < 2,
 * GMM_ERR_FILL when `fill` returns non-zero (the chunks enqueued before it
 * have already been added: the accumulators then hold a partial sum), plus
 * the codes of gmm_estep_accumulate.
 */
int gmm_estep_accumulate_ring(gmm_fill_fn fill, void* user, int64_t n, int32_t d, int32_t k,
                              const float* weights, const float* means, const float* vars,
                              double* nk, double* s, double* q, double* loglik,
                              int64_t chunk_rows, float* ring, int32_t ring_slots,
                              float* staging, void* ws, size_t ws_bytes, hipStream_t stream,
                              hipStream_t copy_stream);

/*
 * k-means++ seeding (the initialisation the paper compares against its warm
 * start, Sec. 4.5 and App. C; Arthur and Vassilvitskii 2007): D^2 sampling of k rows of x with the caller's
 * uniforms u[k] (fp64, device, 0 <= u < 1).  Centre 0 is row floor(u_0 n);
 * centre t is the first row whose running sum of D^2 (squared distance to the
 * nearest centre chosen so far) exceeds u_t times the total, the sums taken
 * in a fixed order: D^2 of a row as 16 fp64 partial sums of fused
 * multiply-adds (partial l over the dimensions 4 (l + 16 j) + e, e = 0..3,
 * j = 0, 1, ..., in that order) added pairwise; blocks of 1024 rows, each 64
 * runs of 16 consecutive rows; runs add their rows, blocks their runs, 256
 * consecutive stretches of blocks their blocks, the total the stretches, and
 * the search walks stretches, blocks, runs and rows in order.  Every choice is thus a
 * pure function of (x, u).  When the total is 0 (every row on a centre),
 * centre t is row floor(u_t n).  idx[k] (int64, device) receives the rows,
 * centers[k*d] (fp32, device) their coordinates.  ws: device workspace of
 * gmm_kmeanspp_workspace_bytes(n) bytes, 256-byte aligned.  k rounds of two
 * kernels on `stream`; the same status codes as the calls above.
 */
size_t gmm_kmeanspp_workspace_bytes(int64_t n);

/*
 * k-means warm start (the paper's initialisation, Sec. 4.4 and App. C: k-means
 * iterations, then EM from the result).  means [k*d] holds the initial centres; n_iters
 * Lloyd iterations each assign every row to its nearest centre (squared
 * Euclidean distance, evaluated exactly in the ranking as gmm_assign_topk
 * does with equal weights and unit variances; ties to the lower index) and
 * move every centre to the mean of its rows (fp64 sums, stored fp32; a centre
 * without rows stays).  A last assignment then gives the mixture EM starts
 * from, by the M-step of gmm_mstep with hard responsibilities:
 *   weights[k] = rows / n, means = the rows' means, vars[k*d] = max(var_floor,
 *   the rows' per-dimension variance); a centre without rows keeps its centre,
 *   its vars as given on entry and weight 0.
 * assign[n] (int32, device) receives the last assignment.  ws: the workspace
 * of gmm_workspace_bytes(n, d, k, 1).  Same status codes as gmm_fit.
 */
int gmm_kmeans(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters, float var_floor,
               float* weights, float* means, float* vars, int32_t* assign, void* ws,
               size_t ws_bytes, hipStream_t stream);
int gmm_kmeanspp(const float* x, int64_t n, int32_t d, int32_t k, const double* u, int64_t* idx,
                 float* centers, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * The paper's own model (Sec. 2, Eqs. Nk, muk, sig): isotropic components
 * N(mu_k, var_k I) with ONE variance per component, vars[k] (fp32, device).
 * The same conventions as the diagonal calls above, with
 *   l_ik = log pi_k - D/2 log(2 pi var_k) - ||x_i - mu_k||^2 / (2 var_k)
 * gmm_estep_accumulate_iso ADDS nk[k], s[k*d] as above and the scalar
 *   q[k] += sum_i r_ik ||x_i||^2
 * (it runs the diagonal E-step with var_kd = var_k; its workspace is the one
 * gmm_workspace_bytes(n, d, k, 0) gives).  gmm_mstep_iso writes
 *   pi_k = nk[k] / n_total,  mu_kj = s[k*d+j] / nk[k],
 *   var_k = max(var_floor, (q[k] / nk[k] - ||mu_k||^2) / d)
 * (= sum_i r_ik ||x_i - mu_k||^2 / (d nk[k]) for the new mean), with the same
 * dead-component rule.  gmm_fit_iso runs n_iters isotropic iterations, as
 * gmm_fit does.  Same status codes as the diagonal calls.
 */
int gmm_estep_accumulate_iso(const float* x, int64_t n, int32_t d, int32_t k,
                             const float* weights, const float* means, const float* vars,
                             double* nk, double* s, double* q, double* loglik, void* ws,
                             size_t ws_bytes, hipStream_t stream);
int gmm_mstep_iso(const double* nk, const double* s, const double* q, double n_total, int32_t d,
                  int32_t k, float var_floor, float* weights, float* means, float* vars,
                  hipStream_t stream);
int gmm_fit_iso(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters, float var_floor,
                float* weights, float* means, float* vars, double* loglik_hist, void* ws,
                size_t ws_bytes, hipStream_t stream);

/*
 * gmm_estep_accumulate without a workspace argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments (minus ws / ws_bytes),
 * semantics and status codes as gmm_estep_accumulate; the library's own
 * 64 MiB device array (one per GPU, held until the process ends) serves as
 * the workspace, and the call allocates and frees nothing.  The split counts
 * of the statistics passes shrink until the workspace fits those 64 MiB, so
 * the results can differ from gmm_estep_accumulate's by rounding; shapes
 * whose per-point buffers (about 110 bytes a point) and O(k d) arrays cannot
 * fit return GMM_ERR_WORKSPACE before anything is enqueued: at d = 128,
 * k = 1024 calls of up to 475,776 points fit (larger data sets are
 * accumulated over row chunks); at d = 768, k = 4096 the O(k d) arrays alone
 * exceed the array.  Calls that overlap on one GPU share the array and race:
 * order them on one stream.
 */
int gmm_estep_accumulate_static(const float* x, int64_t n, int32_t d, int32_t k,
                                const float* weights, const float* means, const float* vars,
                                double* nk, double* s, double* q, double* loglik,
                                hipStream_t stream);

/*
 * Chunking of the dense statistics pass, a tuning control (no part of the
 * method).  That pass splits the points into chunks, one workgroup per
 * (64-component block, chunk); a workgroup queues the chunk's points that
 * need its block, sums their statistics on fp32 MFMA and adds the fp32 sums
 * into fp64 partials every 4096 queued points; the partials are summed in
 * chunk order.  The library picks the chunk count from (n, d, k) (about 8192
 * workgroups); max_chunks > 0 caps it, 0 restores the automatic count.
 * Fewer, longer chunks change the results by rounding only (the split of the
 * fp32 runs moves) and never need a larger workspace.  The setting is
 * process-wide and read when a call is made; calls made under different
 * settings agree to rounding, not bit for bit.  Returns GMM_OK, or
 * GMM_ERR_INVALID_ARG for max_chunks < 0.
 */
int gmm_set_stats_chunk_limit(int32_t max_chunks);

/*
 * Phase timing of the E-step, a measurement aid (no part of the method).
 * While enabled, every E-step (gmm_estep_accumulate, each iteration of
 * gmm_fit) records HIP events on its stream between its phases, waits for the
 * last of them and adds each phase's GPU duration to a process-wide total:
 *   0  parameter preparation (k_prep_*)
 *   1  screening, refinement and log Z of every point (k_logz)
 *   2  statistics of the stored exact pairs (k_sparse_*, k_stats_sparse)
 *   3  the list of light components (little mass in their stored pairs) and
 *      the dense statistics of the other well-conditioned components
 *      (k_small_mass, k_small_list, k_stats_well / k_stats_wide)
 *   4  routed and light components in the direct form, and the fixed-order
 *      reductions (k_stats_ill, k_reduce_stats, k_reduce_ll)
 * gmm_timing_enable(on) switches it on (creating the events on the current
 * device at first use) or off, and zeroes the totals.  gmm_timing_read copies
 * the first n_phases totals (ms; phases past GMM_TIMING_PHASES read 0) and the
 * number of timed E-steps.  The waiting makes timed calls synchronous.  Not
 * for concurrent callers.  Returns GMM_OK, GMM_ERR_INVALID_ARG (null pointer,
 * n_phases < 0) or GMM_ERR_DEVICE (event creation failed).
 */
#define GMM_TIMING_PHASES 5
int gmm_timing_enable(int on);
int gmm_timing_read(double* ms, int32_t n_phases, int64_t* calls);

#ifdef __cplusplus
}
#endif

#endif /* FLASHGMM_H */
