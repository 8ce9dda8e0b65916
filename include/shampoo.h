/*
 * shampoo.h -- C ABI of the MI355X (gfx950) scalable-Shampoo hot path.
 *
 * Paper: Anil, Gupta, Koren, Regan, Singer, "Scalable Second Order
 * Optimization for Deep Learning" (arXiv 2002.09018).  The three steps the
 * paper lists as Shampoo's extra cost (Section 3, "Scaling-up Second Order
 * Optimization": statistics, inverse p-th roots, preconditioned gradient) map
 * onto shampoo_update_stats, shampoo_inv_root_batched and shampoo_precondition;
 * the layer-wise grafted update of Algorithm 2 and of the appendix "Further
 * details on experiments" (paragraph "Layer wise learning rates") is
 * shampoo_graft.
 *
 * Conventions shared by every call
 *  - Matrices are row-major.  A block is a strided view of a larger tensor:
 *    element (i, j) of the view lives at ptr[i * ld + j].
 *  - Every tensor pointer is a DEVICE pointer on the handle's device, owned
 *    by the caller.  The library never frees caller memory.
 *  - Every call is ordered on `stream` (a hipStream_t passed as void*; NULL
 *    is the null stream).  Host arrays passed in (blocks, jobs, params) are
 *    copied before the call returns and may be reused at once.
 *  - Return codes cover argument and launch errors only.  Numeric outcomes of
 *    root computations are per-matrix status codes written to device memory.
 *  - One handle per host thread/stream pair; handles share no state.
 *  - The library owns only what hangs off its handle: device copies of the
 *    block/job tables, a grow-on-demand scratch area for the intermediate
 *    G*Rr of two-sided preconditioning, and a few bytes of pinned host memory
 *    used to poll convergence.
 */
#ifndef SHAMPOO_MI355X_H
#define SHAMPOO_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum shampoo_status {
  SHAMPOO_OK = 0,
  SHAMPOO_EINVAL = -1,       /* bad argument: NULL where required, size out of range, ... */
  SHAMPOO_EUNSUPPORTED = -2, /* valid but not implemented (e.g. root order p outside [1, 16]) */
  SHAMPOO_EHIP = -3,         /* a HIP runtime call or kernel launch failed */
  SHAMPOO_ENOMEM = -4        /* workspace too small, or a library allocation failed */
} shampoo_status;

/* Element type of the gradient views G. */
typedef enum shampoo_dtype {
  SHAMPOO_F32 = 0,
  SHAMPOO_BF16 = 1 /* raw bfloat16 bit patterns; up-cast exactly to fp32 on load */
} shampoo_dtype;

/* Per-matrix outcome of shampoo_inv_root_batched (shampoo_root_info.status). */
enum {
  SHAMPOO_ROOT_CONVERGED = 0, /* max|M - I| <= tol */
  SHAMPOO_ROOT_STAGNATED = 1, /* residual stopped decreasing below 1e-3: rounding floor reached */
  SHAMPOO_ROOT_MAXITER = 2,   /* iteration cap reached */
  SHAMPOO_ROOT_DIVERGED = 3,  /* residual non-finite or above 1e6 */
  SHAMPOO_ROOT_NOT_PD = 4     /* damped matrix has a non-positive diagonal entry or zero norm */
};
/* NOT_PD is a cheap necessary test only (a positive definite matrix has a
 * positive diagonal), not an eigenvalue test.  An indefinite damped matrix
 * whose diagonal is positive is not flagged up front: its negative
 * eigenvalues make the iteration fail, and it comes back DIVERGED (or
 * MAXITER).  Either status means that no root exists or none was found; X
 * then holds the last iterate and must not be used. */

/* Arithmetic used for roots (shampoo_root_params.precision). */
enum {
  SHAMPOO_PRECISION_FP32 = 0, /* fp32 MFMA only */
  SHAMPOO_PRECISION_AUTO = 1, /* fp32 MFMA; matrices that need more iterations than a matrix
                                 of condition kappa32 would (or that fail) are redone in fp64 */
  SHAMPOO_PRECISION_FP64 = 2  /* fp64 MFMA only */
};

/*
 * One preconditioned block (Section 3.1, "Preconditioning blocks from large
 * tensors": each block of a large tensor is treated as a tensor of its own).
 * rows x cols = m x n, both in [1, 4096].  G, W, D, P, Mg and Ps are m x n
 * views sharing the row stride `ld` (elements, >= cols).  L is m x m and R is
 * n x n, contiguous (ld = m and n).  A NULL statistic means that side is not
 * tracked; a NULL root means the identity on that side (one-sided
 * preconditioning, Lemma 1).  Mg and Ps are needed only when beta1 > 0.
 * Element types: G per call (shampoo_dtype), everything else fp32.
 */
typedef struct shampoo_block {
  int32_t rows, cols;
  int64_t ld;
  const void* G;
  float* W;
  float* D;
  float* P;
  float* Mg;
  float* Ps;
  float* L;
  float* R;
  const float* Lr;
  const float* Rr;
} shampoo_block;

/*
 * One inverse-root job: X = (A_s + eps_eff I)^(-1/p) with A_s the symmetric
 * part of A.  A and X are contiguous n x n fp32, n in [1, 4096]; A is only
 * read.  X receives the root; on a status other than CONVERGED/STAGNATED it
 * holds the last iterate.
 */
typedef struct shampoo_root_job {
  int32_t n;
  int32_t reserved; /* must be 0 */
  const float* A;
  float* X;
} shampoo_root_job;

/* Cold-start scaling of a root call, M0 = z A_d, X0 = z^(1/p) I.  Both keep
 * the largest eigenvalue of M0 at or below (p + 1) / 2 through an upper
 * bound B on lambda_max(A_d), z = (p + 1) / (2 B):
 *   FROBENIUS  B = ||A_d||_F, Algorithm 1 as printed;
 *   POWER4     B = ||A_d^4||_F^(1/4) = (sum_i lambda_i^8)^(1/8), a tighter
 *              bound from two extra products (the first reused as M0^2 in the
 *              first iteration); the coupled-Newton appendix leaves the
 *              start constant free (X0 = I / c).  On flat spectra it saves
 *              3-4 of 7 iterations. */
enum { SHAMPOO_SCALING_FROBENIUS = 0, SHAMPOO_SCALING_POWER4 = 1 };

/* Parameters of a root call (Algorithm 1).  shampoo_root_params_default()
 * fills the values used throughout the repository. */
typedef struct shampoo_root_params {
  int32_t p;            /* root order: X = A^(-1/p); 1 <= p <= 16 */
  float eps;            /* damping: eps_eff = eps, or eps * lambda_max when eps_relative */
  int32_t eps_relative; /* 1: scaled damping with lambda_max from MaxSV power iteration */
  float tol;            /* stop when max_ij |M - I|_ij <= tol */
  int32_t max_iters;    /* iteration cap of a precision phase */
  int32_t precision;    /* SHAMPOO_PRECISION_* */
  float kappa32;        /* AUTO: largest damped condition number accepted from fp32 */
  int32_t maxsv_steps;  /* MaxSV cap on power steps */
  float maxsv_tol;      /* MaxSV stop: |lambda - lambda_old| <= maxsv_tol * lambda */
  int32_t poll;         /* 1: the host polls a device counter and stops enqueuing
                           iterations once no matrix is active (the call then waits
                           for the stream); 0: enqueue max_iters iterations, fully
                           asynchronous, converged matrices skip their work */
  int32_t scaling;      /* SHAMPOO_SCALING_*: the constant of the cold start */
} shampoo_root_params;

/* Per-matrix result of a root call, written on the stream (device memory). */
typedef struct shampoo_root_info {
  int32_t status;     /* SHAMPOO_ROOT_* of the phase that produced X */
  int32_t iters;      /* iterations of that phase */
  int32_t precision;  /* 32 or 64: arithmetic that produced X */
  int32_t iters_fp32; /* iterations spent in fp32 (also when escalated) */
  float resid;        /* last max|M - I| */
  float lambda_max;   /* MaxSV estimate (eps_relative), else 0 */
  float cond_est;     /* condition-number upper estimate from the iteration count */
  float eps_eff;      /* damping actually added */
} shampoo_root_info;

/* Create / destroy a handle bound to HIP device `device`. */
shampoo_status shampoo_create(void** handle, int device);
shampoo_status shampoo_destroy(void* handle);
/* Text of the last error on this handle ("" if none).  Valid until the next call. */
const char* shampoo_last_error(const void* handle);
/* Library version string. */
const char* shampoo_version(void);

/* Defaults: p=4, eps=1e-6 absolute, tol=1e-6, max_iters=100, precision AUTO,
 * kappa32=1e4, maxsv_steps=100, maxsv_tol=1e-6, poll=1, scaling POWER4. */
void shampoo_root_params_default(shampoo_root_params* params);

/*
 * Statistics update, Preliminaries ("The Shampoo algorithm", definition of
 * L_t and R_t) and Algorithm 2:
 *   beta2 == 1:  L += G G^T,  R += G^T G
 *   beta2 <  1:  L = beta2 L + (1 - beta2) G G^T  (same for R)
 * For every block with non-NULL L (resp. R).  L and R stay exactly symmetric:
 * the upper triangle is computed and mirrored.  They must be symmetric on
 * entry as well (zero, or the output of earlier updates): the old value of an
 * off-diagonal element may be read from its mirror.  The ridge eps*I is not
 * added here; shampoo_inv_root_batched adds it once.  G: g_dtype.
 * Errors: EINVAL for nblocks < 0, NULL blocks with nblocks > 0, sizes
 * outside [1, 4096], ld < cols, beta2 outside (0, 1], L, R and G not
 * distinct buffers (a block with both L and R NULL is skipped).
 */
shampoo_status shampoo_update_stats(void* handle, const shampoo_block* blocks, int nblocks,
                                    int g_dtype, float beta2, void* stream);

/* Device workspace (bytes) that shampoo_inv_root_batched needs for `jobs`
 * under `precision`; 0 on invalid arguments. */
size_t shampoo_inv_root_workspace_bytes(const shampoo_root_job* jobs, int njobs, int precision);

/*
 * Batched inverse p-th roots by the coupled Newton iteration, Algorithm 1
 * (appendix "A coupled Newton iteration for computation of inverse p-th
 * roots"), all matrices in one grouped launch per product:
 *   eps_eff = eps, or eps * MaxSV(A) (scaled damping);
 *   A_d = A_s + eps_eff I;  z = (1 + p) / (2 ||A_d||_F);
 *   X = z^(1/p) I;  M = z A_d;
 *   while max|M - I| > tol:  M1 = ((p + 1) I - M) / p;  X = X M1;  M = M1^p M.
 * Each matrix leaves the iteration on its own (CONVERGED, STAGNATED, MAXITER,
 * DIVERGED).  M1^p M is formed by binary powering over the bits of p
 * (floor(log2 p) squarings plus popcount(p) products, launched in
 * floor(log2 p) + 1 stages per iteration).  Products of the commuting
 * symmetric iterates are computed on their upper triangle and mirrored.  `workspace` is device memory of at least
 * shampoo_inv_root_workspace_bytes(jobs, njobs, params->precision) bytes,
 * owned by the caller and used exclusively by this call until the stream
 * reaches its end.  `info` is a device array of njobs entries.
 * Errors: EINVAL (NULL pointers, njobs above 2^22, n outside [1, 4096], eps < 0,
 * tol < 0, max_iters < 1), EUNSUPPORTED (p outside [1, 16]), ENOMEM (ws_bytes
 * too small).
 */
shampoo_status shampoo_inv_root_batched(void* handle, const shampoo_root_job* jobs, int njobs,
                                        const shampoo_root_params* params, void* workspace,
                                        size_t ws_bytes, shampoo_root_info* info, void* stream);

/*
 * Warm-started batched inverse p-th roots (appendix "A coupled Newton
 * iteration for computation of inverse p-th roots", warm start, with the
 * commutator check it proposes for detecting divergence).  On entry jobs[j].X
 * holds X0, the previous root of a nearby matrix (any n x n fp32 matrix with
 * positive eigenvalues in exact arithmetic; typically the last call's result);
 * then
 *   M = X0^p A_d  (A_d = A_s + eps_eff I as in the cold call),  X = X0,
 *   while max|M - I| > tol:  M1 = ((p + 1) I - M) / p;  X = X M1;  M = M1^p M;
 *     after each iteration the warm start is given up when
 *     max|XM - MX| > comm_tol * max|X| * max|M|, when the residual grew in two
 *     consecutive iterations, or when it diverges or reaches max_iters.
 * The iterates no longer commute with A, so every product is a full n x n
 * product (twice the work of a cold product).  A residual that stops
 * decreasing below 1e-3 is accepted (STAGNATED, the rounding floor).  When
 * X0 commutes with A_d the limit is A_d^(-1/p); otherwise it is
 * X0 (X0^p A_d)^(-1/p), close to the root only while the drift is small.
 * Matrices whose warm start is given up are computed by the cold call's
 * iteration in the same call (with its precision policy); the others keep the
 * warm result.  The warm phase runs in fp64 under SHAMPOO_PRECISION_FP64 and
 * in fp32 otherwise (under AUTO an fp32 warm result carries fp32 rounding
 * amplified by the condition number: use FP64 for ill-conditioned factors).
 * A kept warm result is that limit, not the root: its distance from
 * A_d^(-1/p) grows with the drift of the statistics since X0 and is NOT held
 * to the tolerance of the cold call.  The monitor only guards against
 * divergence; it does not bound that distance (measured: 2.5e-4 to 6e-4 from
 * the cold roots one gradient after X0 on 1024 x 1024 statistics of ~20
 * gradients, 1.1e-3 when the statistics doubled since X0, every result kept
 * at comm_tol = 1e-3).  Callers that need the root to a stated tolerance use
 * shampoo_inv_root_batched.
 * params, workspace, info: as shampoo_inv_root_batched (same workspace size;
 * cond_est is 0 for a warm result).  warm_out (device, may be NULL): int32
 * [njobs][2] = {outcome, warm iterations}, outcome 1 = warm result kept,
 * 2 = warm start given up (cold result), 0 = not attempted (NOT_PD).
 * Errors: as shampoo_inv_root_batched, and EINVAL for comm_tol <= 0.
 */
shampoo_status shampoo_inv_root_warm_batched(void* handle, const shampoo_root_job* jobs, int njobs,
                                             const shampoo_root_params* params, float comm_tol, void* workspace,
                                             size_t ws_bytes, shampoo_root_info* info, int32_t* warm_out,
                                             void* stream);

/*
 * Preconditioned gradient P = Lr G Rr (Preliminaries, Shampoo update rule;
 * one-sided forms of Lemma 1 when a root is NULL; P = G when both are).
 * Lr and Rr must be symmetric (inverse roots are).  G: g_dtype.
 * Errors: as shampoo_update_stats; EINVAL when P is NULL or is the same
 * buffer as G, Lr or Rr.
 */
shampoo_status shampoo_precondition(void* handle, const shampoo_block* blocks, int nblocks,
                                    int g_dtype, void* stream);

/*
 * Grafted parameter update, Algorithm 2 with the AdaGrad-magnitude /
 * Shampoo-direction graft ("Layer wise learning rates"):
 *   D  = D + G o G
 *   Mg = beta1 Mg + (1 - beta1) D^(-1/2) o G        (D^(-1/2) o G := 0 where D == 0)
 *   use_shampoo:  Ps  = beta1 Ps + (1 - beta1) P
 *                 eta = eta0 ||Mg||_F / ||Ps||_F     (0 when ||Ps||_F == 0)
 *                 W   = W - eta Ps
 *   otherwise:    W   = W - eta0 Mg                  (before the first roots)
 * With beta1 == 0, Mg and Ps are not stored (may be NULL) and P is used as Ps.
 * norms (device, may be NULL): per block {||Mg||_F, ||Ps||_F, eta} as 3 floats.
 * Errors: EINVAL as above, non-finite eta0, beta1 outside [0, 1), NULL
 * W/D, P NULL with use_shampoo, Mg/Ps NULL with beta1 > 0, and an updated
 * state (W, D, Mg, Ps) that is the same buffer as G, P or another state.
 */
shampoo_status shampoo_graft(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                             float eta0, float beta1, int use_shampoo, float* norms, void* stream);

/*
 * Allocation-free form of shampoo_graft, for callers that cannot allocate
 * device memory (code under stream capture, tight serving loops, harnesses
 * that forbid hipMalloc): same arguments, same kernels and the same result
 * bit for bit.  Its scratch -- the block table and one pair of fp64 norm
 * partials per chunk of at most 16384 elements (whole rows of a block) --
 * lives in a fixed device array of SHAMPOO_GRAFT_NOALLOC_SCRATCH_BYTES that
 * every GPU the library runs on holds until the process ends; the table is
 * staged through pinned host memory that shampoo_create sets up.  The call
 * itself allocates nothing (no hipMalloc/hipFree, no growth of the handle),
 * and its launches are not recorded by shampoo_timing_*.
 * Limits: nblocks <= SHAMPOO_GRAFT_NOALLOC_MAX_BLOCKS and at most
 * SHAMPOO_GRAFT_NOALLOC_MAX_CHUNKS chunks in total, where a block of
 * m x n has ceil(m / max(1, 16384 / n)) chunks (C2's 96 blocks of
 * 1024 x 4096 take 24576); beyond either, ENOMEM and nothing is enqueued.
 * Every call on a GPU uses that GPU's one array: calls on one stream are
 * ordered, calls that overlap on different streams of one GPU race.  The
 * host waits, if needed, for the previous call's table copy out of the
 * handle's staging memory before writing it again.
 * Errors: as shampoo_graft, and ENOMEM as above.
 */
#define SHAMPOO_GRAFT_NOALLOC_MAX_BLOCKS 8192
#define SHAMPOO_GRAFT_NOALLOC_MAX_CHUNKS 196608
#define SHAMPOO_GRAFT_NOALLOC_SCRATCH_BYTES (4u << 20)
shampoo_status shampoo_graft_noalloc(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                     float eta0, float beta1, int use_shampoo, float* norms, void* stream);

/*
 * Preconditioning and the AdaGrad-grafted update in one call: the same
 * result as shampoo_precondition followed by shampoo_graft with beta1 = 0 and
 * use_shampoo = 1 (Preliminaries, Shampoo update rule; Algorithm 2 with the
 * graft of "Layer wise learning rates"):
 *   P = Lr G Rr;  D = D + G o G;
 *   eta = eta0 ||D^(-1/2) o G||_F / ||P||_F  (0 when ||P||_F == 0);  W = W - eta P
 * The GEMM that writes each block's P also updates D and sums the two squared
 * norms per output tile, so G, D and P are not read by a separate pass; the
 * norms are then reduced per block in a fixed order (deterministic, but in
 * another order than shampoo_graft's, so eta may differ in the last bits).
 * Every block needs W, D, P and at least one root; G: g_dtype.  norms:
 * as shampoo_graft.  Errors: as shampoo_graft, and EINVAL for a block with
 * both roots NULL, or whose P, W, D are not distinct or coincide with G or a
 * root.
 */
shampoo_status shampoo_precondition_graft(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                          float eta0, float* norms, void* stream);

/*
 * Grafted update with the LARS/LAMB layer-wise magnitude of the same appendix
 * paragraph ("Layer wise learning rates": learning rate ||W||_F / ||G||_F per
 * layer, applied per block here): the step is eta0 ||W||_F long, W taken
 * before the step,
 *   Mg = beta1 Mg + (1 - beta1) G
 *   use_shampoo:  Ps  = beta1 Ps + (1 - beta1) P
 *                 eta = eta0 ||W||_F / ||Ps||_F     (0 when ||Ps||_F == 0)
 *                 W   = W - eta Ps
 *   otherwise:    eta = eta0 ||W||_F / ||Mg||_F     (LARS step, before the roots)
 *                 W   = W - eta Mg
 * D is not used (may be NULL).  With beta1 == 0, Mg and Ps are not stored.
 * norms (device, may be NULL): per block {||W||_F, ||direction||_F, eta}.
 * Errors: as shampoo_graft (D may be NULL).
 */
shampoo_status shampoo_graft_lamb(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                  float eta0, float beta1, int use_shampoo, float* norms, void* stream);

/*
 * Embedding layers (appendix "Shampoo for embedding layers", with the
 * one-sided preconditioner of Lemma 1 for large layers).
 *
 * A table W (vocab x dim, row-major, row stride ldw) is read by nnz lookup
 * entries: entry e reads row idx[e] into output row feat[e] of the layer
 * output y (m x dim), with weight weight[e].  Its gradient
 *   G = sum_e weight[e] e_{idx[e]} dy[feat[e], :]   (vocab x dim)
 * is nonzero only on the active rows {idx[e]}, and the dim x dim statistic is
 *   R = G^T G = dy^T (S^T S) dy,   S[idx[e], feat[e]] += weight[e],
 * which is dy^T dy when every entry hits its own row (one-hot features on
 * distinct rows), at O(nnz dim^2) cost instead of O(vocab dim^2).
 * The step for the table is then
 *   shampoo_embedding_rows -> shampoo_embedding_stats -> (roots: Rr = R^(-1/2),
 *   shampoo_inv_root_batched with p = 2) -> shampoo_embedding_precondition
 *   -> shampoo_embedding_graft,
 * all on the compact rows.  Every count is read on the device: no call
 * synchronizes the stream.
 *
 * Compact form (written by shampoo_embedding_rows, read by the others):
 *   rows   int32[nnz]: the active rows in ascending order, then -1;
 *   U      fp32 nnz x dim (row stride dim): U[i] = G[rows[i]] for i < u,
 *          summed over the entries of that row in entry order within fixed
 *          chunks of 64 sorted entries, the chunk sums then added in order
 *          (deterministic); rows i >= u are not written;
 *   count  int32[2]: count[0] = u (active rows), count[1] = entries dropped
 *          because idx is outside [0, vocab) or feat outside [0, m).
 */

/* Workspace (bytes) of shampoo_embedding_rows and shampoo_embedding_stats
 * for nnz entries of width dim; 0 on invalid arguments (nnz outside
 * [1, 2^26], dim outside [1, 4096]). */
size_t shampoo_embedding_workspace_bytes(int nnz, int dim);

/*
 * Compacts the lookup gradient.  idx: nnz rows; feat: nnz output rows, or
 * NULL for feat[e] = e (one entry per output row, m >= nnz); weight: nnz
 * weights, or NULL for 1 (one-hot); dy: m x dim, row stride ld_dy.  All
 * device pointers.  rows, U, count: outputs as above.  Sorting uses a stable
 * device radix sort whose temporary storage the handle allocates and keeps.
 * Errors: EINVAL (NULL pointers, nnz or dim out of range, vocab outside
 * [1, 2^31 - 1), m < 1, ld_dy < dim), ENOMEM (workspace too small).
 */
shampoo_status shampoo_embedding_rows(void* handle, const int32_t* idx, const int32_t* feat, const float* weight,
                                      int nnz, int64_t vocab, const float* dy, int m, int dim, int64_t ld_dy,
                                      int32_t* rows, float* U, int32_t* count, void* workspace, size_t ws_bytes,
                                      void* stream);

/*
 * R = beta2 R + c U^T U over the first count[0] rows of U (c = 1 if
 * beta2 == 1 else 1 - beta2): the statistic of the table, dim x dim, kept
 * exactly symmetric (and required symmetric on entry, as for
 * shampoo_update_stats).  The active rows are split into a fixed number of
 * equal parts (set from nnz and dim); their partial products are added in
 * part order (deterministic).
 * Errors: EINVAL (NULL pointers, sizes, beta2 outside (0, 1]), ENOMEM.
 */
shampoo_status shampoo_embedding_stats(void* handle, const float* U, const int32_t* count, int nnz, int dim,
                                       float* R, float beta2, void* workspace, size_t ws_bytes, void* stream);

/*
 * P = U Rr for the first count[0] rows (Rr symmetric, dim x dim): the
 * preconditioned compact gradient G R^(-1/2) of Lemma 1's one-sided form.
 * Rows of P at or past count[0] are not written.  Errors: EINVAL.
 */
shampoo_status shampoo_embedding_precondition(void* handle, const float* U, const int32_t* count, int nnz, int dim,
                                              const float* Rr, float* P, void* stream);

/*
 * Grafted update of the active rows (beta1 = 0 form of shampoo_graft): for
 * i < count[0] and r = rows[i],
 *   D[r] += U[i] o U[i];  eta = eta0 ||D^(-1/2) o G||_F / ||P||_F  (norms over
 *   the active rows, which are all of G's nonzeros);  W[r] -= eta P[i]
 * (use_shampoo = 0: W[r] -= eta0 D[r]^(-1/2) o U[i]).  Rows of W and D that
 * no entry touched are left exactly as they were.  norms (device, may be
 * NULL): {||D^(-1/2) o G||_F, ||P||_F, eta}.
 * Errors: EINVAL (NULL pointers, sizes, ldw < dim, non-finite eta0).
 */
shampoo_status shampoo_embedding_graft(void* handle, const int32_t* rows, const int32_t* count, int nnz, int dim,
                                       const float* U, const float* P, float* W, float* D, int64_t vocab,
                                       int64_t ldw, float eta0, int use_shampoo, float* norms, void* stream);

/*
 * Measurement support.  While enabled, every launch of the timed kernel
 * classes below is bracketed by HIP events on its stream.
 * shampoo_timing_read synchronizes those events, returns the summed duration
 * (ms) and launch count of one class, and clears that class.
 */
enum {
  SHAMPOO_KCLASS_NEWTON_F32 = 0, /* grouped Newton products, fp32 MFMA */
  SHAMPOO_KCLASS_NEWTON_F64 = 1, /* grouped Newton products, fp64 MFMA */
  SHAMPOO_KCLASS_STATS = 2,      /* grouped statistics SYRK */
  SHAMPOO_KCLASS_PRECOND = 3,    /* grouped preconditioning GEMMs */
  SHAMPOO_KCLASS_GRAFT = 4,      /* graft reduction and update passes */
  SHAMPOO_KCLASS_ROOT_AUX = 5,   /* root prologue/epilogue/state kernels */
  SHAMPOO_KCLASS_EMB = 6,        /* embedding row compaction (sort, runs, segment sums) */
  SHAMPOO_KCLASS_NEWTON_WARM = 7, /* full products of warm-started roots (fp32 or fp64 MFMA) */
  SHAMPOO_KCLASS_COUNT = 8
};
shampoo_status shampoo_timing_enable(void* handle, int enable);
shampoo_status shampoo_timing_read(void* handle, int kclass, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* SHAMPOO_MI355X_H */
