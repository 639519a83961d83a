/*
 * greedylore.h -- C ABI of the MI355X (gfx950) GreedyLore compression step.
 *
 * The method is GreedyLore (arXiv 2507.08784): greedy low-rank compression of
 * the gradients of N data-parallel workers with error feedback and a
 * semi-lazy SVD subspace.  One call of glr_step performs, for every layer
 * matrix X in R^{m x n} (problem (1), Section I):
 *
 *   error feedback       M^(i) = G^(i) + E^(i)                (Section V-A, eq-ef)
 *   worker mean          Mbar  = (1/N) sum_i M^(i)           (All-Reduce of Alg. 3/4)
 *   subspace             t mod tau == 0: U = complete left singular basis of
 *                        Mbar, P = first r columns (eq-SVD-P1);
 *                        otherwise P = r columns of U chosen by Approx-Top-r
 *                        (Algorithm 2, eq:lambda-bar, eq-semi-lazy-svd-3)
 *   projection           Q^(i) = P^T M^(i)                    (eq 8zhb2we09)
 *   residual             E^(i) = M^(i) - P Q^(i)              (Algorithm 4)
 *   average              Rbar  = (1/N) sum_i Q^(i)           (All-Reduce)
 *   reconstruction       Ghat  = P Rbar                       (Algorithm 4)
 *   optimizer            MSGD (eq-msgd) or Adam (eq-adam) on X with Ghat.
 *
 * Orientation (Algorithm 4, Appendix D): d = min(m, n), D = max(m, n).  When
 * m > n the method works on the transposed gradient (right projection); no
 * buffer is physically transposed: every m x n buffer stays in the caller's
 * row-major layout.
 *
 * The N workers are simulated on one GPU: G holds all N gradients of a
 * matrix, and the All-Reduce averages are device-side means in a fixed worker
 * order (deterministic: no floating-point atomics).
 *
 * Memory ownership.  The caller owns every device buffer: the weights X, the
 * gradients G, the state blob and the workspace.  The library never allocates
 * device memory and never frees caller memory; the handle holds host metadata
 * and, with more than one matrix, up to four HIP streams and their events.
 * Device pointers must be 256-byte aligned and must not alias.
 *
 * Streams.  `stream` arguments are hipStream_t values passed as void*; NULL is
 * the default stream.  glr_step orders its work after what is already on the
 * stream and before what the caller enqueues next.  With one matrix it
 * enqueues its kernels on the stream itself.  With several, the matrices are
 * spread over up to four non-blocking streams of the handle (created by
 * glr_create, destroyed by glr_destroy), each with its own host thread inside
 * glr_step, forked from and joined back to `stream` with events; every matrix
 * computes exactly what it computes alone (results are bitwise those of
 * running the matrices in order).  On refresh steps (tau > 1) of several
 * matrices with d <= 2048 and one Jacobi group size, the sweeps of all of them
 * run in shared launches on `stream` itself, with one convergence read per
 * sweep for all matrices; each matrix still computes exactly what it computes
 * alone.  GLR_JAC_JOINT=0, read by glr_create, turns this off.  Likewise a
 * selection step of several matrices that all have d <= 2048, the same side
 * (m > n or not) and the same rank r < d, r <= 128, launches each of its
 * kernels once for all matrices on `stream`, after uploading that step's table
 * of matrix views from pinned host memory the handle owns; GLR_GROUPED=0 turns
 * this off.
 * While profiling is enabled the matrices run in order on `stream`.  The
 * environment variable GLR_LANES, read by glr_create, lowers the stream count.
 * Tuning switches of the refresh, also read by glr_create (defaults in
 * brackets; other values change the floating-point path): GLR_JAC_FLOOR=k
 * sets the convergence measure's floor f = 2^-k max_k |w_k| [10];
 * GLR_JAC_SORT=0|1|2 reorders the rows by descending norm never, before
 * every sweep or before the first only [1]; GLR_JAC_INNER=1..16 sets the
 * cyclic sweeps of each group solve [1]; GLR_SUB_ITERS sets the cap of the
 * tau = 1 block iterations after a warm start [4].  GLR_GROUP_PARTS and
 * GLR_GROUP_SPLIT=0 set the parts of a grouped selection step [2 when there
 * are streams for them] (same results).
 *
 * glr_step only enqueues: it never waits for the device (refresh steps
 * included).  A refresh enqueues a budget of Jacobi sweeps; the sweeps after
 * convergence return at once on the device.  The budget is max_sweeps until a
 * refresh of that matrix has been seen converged, then the most sweeps a
 * converged refresh of it took plus half of that (at least four), capped at
 * max_sweeps; the sweep counts come back through
 * pinned host memory the handle owns, read only once their copy has completed.
 * A refresh that ends its budget above tol reports GLR_ERR_NOT_CONVERGED and
 * the next one gets max_sweeps again.  (Grouped selection steps reuse a
 * two-slot pinned ring: the host waits only if it runs two such steps ahead
 * of the device.)
 *
 * Errors.  Every function returns a glr_status and never throws or aborts
 * across the ABI.  Argument and shape errors are detected before anything is
 * enqueued and leave the state untouched.  A HIP error returns GLR_ERR_DEVICE
 * (text via glr_last_error).  Device-side conditions are latched in a status
 * word in the state blob and reported by glr_sync_status: a non-finite
 * gradient (with GLR_CHECK_FINITE), a refresh that did not converge, and an
 * orthonormalisation breakdown of the tau = 1 refresh.
 *
 * Threading.  A handle is not thread-safe; one glr_step may be in flight per
 * handle; kernels of different handles may share a stream.
 */
#ifndef GREEDYLORE_H
#define GREEDYLORE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GLR_OK = 0,
  GLR_ERR_INVALID_ARG = 1,      /* null / misaligned pointer, bad enum, bad hyper-parameter */
  GLR_ERR_SHAPE = 2,            /* non-positive or too large dimensions */
  GLR_ERR_BUFFER_TOO_SMALL = 3, /* state or workspace smaller than glr_workspace_bytes says */
  GLR_ERR_STATE = 4,            /* t out of order, or a handle whose state is suspect */
  GLR_ERR_DEVICE = 5,           /* a HIP call failed */
  GLR_ERR_NONFINITE = 6,        /* a gradient held NaN/Inf (only with GLR_CHECK_FINITE) */
  GLR_ERR_NOT_CONVERGED = 7,    /* a refresh ended above its tolerance (informational) */
  GLR_ERR_BREAKDOWN = 8         /* tau = 1 refresh: dependent rows survived the repair pass */
} glr_status;

/* Optimizers: MSGD (eq-msgd) and Adam (eq-adam) on the full m x n state, or
 * GALORE_ADAM, the distributed Adam-type GaLore of Algorithm 5 (Appendix E,
 * a baseline of the paper): Lazy-SVD projection (P kept between refreshes,
 * as GLR_SELECT_LAZY), no error feedback (as GLR_NO_EF), Adam moments kept
 * in the r x D subspace (S1 = M, S2 = V, the first r D floats of each, row
 * major, oriented) and restarted from zero at every refresh, and the step
 * X -= lr P (M / (sqrt(V) + eps)) (transposed back iff m > n); Rbar then
 * holds that direction M / (sqrt(V) + eps) after the step.  Algorithm 5's
 * printed moment updates exchange beta and 1 - beta and apply lr twice; the
 * main text's Adam with one lr is used.  Requires GLR_REFRESH_COMPRESSED. */
typedef enum { GLR_MSGD = 0, GLR_ADAM = 1, GLR_GALORE_ADAM = 2 } glr_opt;

/* Refresh-step semantics.  COMPRESSED follows Algorithm 4 ("the complete
 * procedure"): refresh steps compress like every other step.  FULL follows
 * Algorithm 3: at a refresh step Ghat = Mbar (uncompressed) and E^(i) = 0. */
typedef enum { GLR_REFRESH_COMPRESSED = 0, GLR_REFRESH_FULL = 1 } glr_refresh;

/* Non-refresh selection.  APPROX is Approx-Top-r (Algorithm 2): scores
 * lambdabar_j^2 with lambdabar_j = u_j^T Mbar v_j and v_j ~ N(0, I_D).
 * EXACT scores ||u_j^T Mbar||^2 (eq-semi-lazy-svd-2).  APPROX_BF16 is
 * Approx-Top-r with the products of u_j and Mbar taken on their bf16
 * roundings (round to nearest even; v_j and the sums stay fp32): a mixed
 * precision mode for the ranking only (a score carries ~2^-8 relative error
 * per term), on the bf16 matrix cores; everything else stays fp32.  LAZY is
 * the Lazy-SVD operator of the basic framework (Section IV, Algorithm 1, a
 * baseline of the paper): P_t = P_{t-1} between refreshes (J and U kept, no
 * scores).  Algorithm 1 itself is LAZY with GLR_NO_EF and
 * GLR_REFRESH_FULL. */
typedef enum {
  GLR_SELECT_APPROX = 0,
  GLR_SELECT_EXACT = 1,
  GLR_SELECT_APPROX_BF16 = 2,
  GLR_SELECT_LAZY = 3
} glr_select;

#define GLR_CHECK_FINITE 0x1u  /* scan G for NaN/Inf during the worker mean */
#define GLR_COLD_START   0x2u  /* start every refresh from U = I instead of the previous U */
#define GLR_NO_EF        0x4u  /* no error feedback: M^(i) = G^(i), E^(i) and Ebar stay zero */
/* Mixed-precision storage (the paper fixes no precision): the gradients G^(i)
 * and the error buffers E^(i) are bfloat16 (the upper half of an IEEE
 * binary32), halving the bytes of the streaming passes.  Each G element is
 * widened exactly; the residual M^(i) - P Q^(i) is formed in fp32 and stored
 * rounded to nearest even; Ebar is the mean of the stored E^(i), so the next
 * step's M^(i) and Mbar are those of the stored buffers.  U, Q, Rbar, X and
 * the optimizer state stay fp32.  Steps run through glr_step_bf16.  MSGD and
 * Adam only (GLR_ERR_INVALID_ARG with GLR_GALORE_ADAM). */
#define GLR_STORE_BF16   0x8u

typedef struct {
  int64_t m, n;                /* layer matrix shape, caller's row-major layout;
                                  m n < 2^30 and min(m, n) <= 8192 (GLR_ERR_SHAPE) */
} glr_shape;

typedef struct {
  int32_t num_mats;            /* number of layer matrices, >= 1 */
  const glr_shape* shapes;     /* host array of num_mats shapes; copied by glr_create */
  int32_t num_workers;         /* N >= 1 simulated workers */
  int32_t rank;                /* r >= 1; r >= min(m, n) keeps every direction (E = 0) */
  int32_t tau;                 /* refresh period >= 1: refresh iff t mod tau == 0 */
  int32_t opt;                 /* glr_opt */
  float lr;                    /* gamma > 0 */
  float beta1;                 /* MSGD momentum beta / Adam beta1, in [0, 1) */
  float beta2;                 /* Adam beta2 in [0, 1) (ignored for MSGD) */
  float eps;                   /* Adam epsilon > 0 (ignored for MSGD) */
  int32_t refresh;             /* glr_refresh */
  int32_t select;              /* glr_select */
  uint64_t seed;               /* Philox4x32-10 key of the random vectors v_j */
  int32_t max_sweeps;          /* bound on Jacobi sweeps per refresh, >= 1 */
  float tol;                   /* Jacobi stop, in (0, 1): every pair of rows of W = U^T Mbar has
                                  |w_p.w_q| <= tol max(|w_p||w_q|, ||w_p|^2 - |w_q|^2|, f^2),
                                  f = 2^-10 max_k |w_k| (cosine and rotation angle below tol) */
  uint32_t flags;              /* GLR_CHECK_FINITE | GLR_COLD_START | GLR_NO_EF | GLR_STORE_BF16 */
} glr_config;

/* Byte offsets into the state blob for one matrix (all 256-byte aligned). */
typedef struct {
  int64_t m, n, d, D;
  int32_t right;               /* 1 iff m > n (the method works on G^T) */
  int32_t r;                   /* effective rank min(rank, d) */
  uint64_t off_E;              /* N x m x n fp32 (bf16 with GLR_STORE_BF16): error buffers
                                  E^(i), worker-major */
  uint64_t off_Ebar;           /* m x n fp32: mean over workers of E^(i) */
  uint64_t off_U;              /* d x d fp32: row j holds u_j, the j-th column of U */
  uint64_t off_sigma;          /* d fp32: singular values of Mbar at the last refresh, descending */
  uint64_t off_J;              /* r int32: selected columns of U, ascending */
  uint64_t off_score;          /* d fp32: last selection scores (lambdabar^2 or ||u_j^T Mbar||^2) */
  uint64_t off_S1;             /* m x n fp32: MSGD buffer M, or Adam first moment M (GaLore: r x D) */
  uint64_t off_S2;             /* m x n fp32: Adam second moment V (GaLore: r x D; 0 for MSGD: absent) */
  uint64_t off_Rbar;           /* r x D fp32: mean over workers of Q^(i) = P^T M^(i) (oriented) */
  uint64_t off_info;           /* 64 int32: [0] sweeps of the last refresh, [1] converged flag,
                                  [2 + s] float bits of sweep s's largest pair off-norm (s < 60);
                                  tau = 1 refresh: [62] block iterations, [63] float bits of
                                  the last iteration's relative gain of the energy ||P^T Mbar||^2
                                  of the oversampled block */
} glr_mat_layout;

typedef struct glr_handle glr_handle;

/* Checks a configuration; pure host, no device call. */
glr_status glr_validate_config(const glr_config* cfg);

/* Bytes of caller-owned device memory a configuration needs; pure host.
 * state_bytes: persistent across steps (error buffers, U, optimizer state).
 * ws_bytes: scratch reused by every step: one region per matrix, sized by
 * that matrix. */
glr_status glr_workspace_bytes(const glr_config* cfg, size_t* state_bytes, size_t* ws_bytes);

/* Layout of matrix `mat` inside the state blob; pure host. */
glr_status glr_state_layout(const glr_config* cfg, int32_t mat, glr_mat_layout* out);

/* Creates a handle over caller-owned device buffers d_state (state_bytes) and
 * d_ws (ws_bytes) on the current HIP device, and enqueues on `stream` the
 * initial state of Algorithm 3: E^(i) = 0, optimizer state 0, U = I.
 * The first step to run is t = 0.  *out receives the handle. */
glr_status glr_create(const glr_config* cfg, void* d_state, size_t state_bytes,
                      void* d_ws, size_t ws_bytes, void* stream, glr_handle** out);

/* glr_create for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * workspace is a static device array of GLR_STATIC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends; the caller
 * still owns the state blob, X and G.  Creating, stepping and destroying such
 * a handle calls no hipMalloc, hipFree, hipHostMalloc nor stream or event
 * creation (profiling, if enabled, creates events).  Such a handle runs every
 * matrix on `stream`, without grouped selection steps, and enqueues
 * max_sweeps sweeps per refresh (no sweep counts come back to the host).
 * GLR_ERR_BUFFER_TOO_SMALL when the configuration's workspace
 * (glr_workspace_bytes) exceeds the array.  The array is shared by the handle
 * and keeps its contents between handles (creation clears what must start
 * at zero), so only one such handle may live per device at a time
 * (GLR_ERR_STATE otherwise): calls of two handles on one device would race. */
#define GLR_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
glr_status glr_create_static(const glr_config* cfg, void* d_state, size_t state_bytes, void* stream,
                             glr_handle** out);

/* Runs step t on every matrix.  X: host array of num_mats device pointers to
 * the m x n fp32 weights, updated in place.  G: host array of num_mats device
 * pointers, each to N contiguous m x n fp32 gradients (worker-major), read
 * only.  t must be the handle's next step (0, 1, 2, ...). */
glr_status glr_step(glr_handle* h, float* const* X, const float* const* G,
                    int64_t t, void* stream);

/* glr_step for a handle created with GLR_STORE_BF16: each G[l] points to N
 * contiguous m x n bfloat16 gradients (the bit patterns, worker-major), read
 * only; X stays fp32.  GLR_ERR_INVALID_ARG on a handle without the flag (and
 * glr_step on one with it). */
glr_status glr_step_bf16(glr_handle* h, float* const* X, const uint16_t* const* G,
                         int64_t t, void* stream);

/* Waits for `stream`, reads and clears the device status word (every step
 * since the last call).  Returns, in this order of precedence:
 *   GLR_ERR_NONFINITE      a gradient held NaN/Inf (GLR_CHECK_FINITE); the
 *                          state is marked suspect;
 *   GLR_ERR_BREAKDOWN      a tau = 1 refresh could not orthonormalise its block
 *                          (rows still dependent after the repair pass that
 *                          replaces dependent rows by Gaussian ones); suspect;
 *   GLR_ERR_NOT_CONVERGED  a refresh ended above its tolerance: Jacobi sweeps
 *                          (budget or max_sweeps) above tol, or a tau = 1
 *                          refresh whose block iteration reached its cap (4
 *                          from the previous block, 8 from a cold start) with
 *                          the leading r rows still moving by more than 10 tol
 *                          and the oversampled block still raising the energy
 *                          ||P^T Mbar||^2 it captures by more than 10 tol
 *                          relative.  (The block
 *                          iteration runs at least 2 times, and more only while
 *                          the previous refresh's Ritz values show a relative
 *                          gap (sigma_r^2 - sigma_{r+1}^2) / sigma_1^2 of at
 *                          least 1e-3: with the gap closed the top-r subspace is
 *                          not determined by the data, and the Rayleigh-Ritz
 *                          step keeps the directions of largest energy.)
 *                          Informational: the basis is orthonormal and the
 *                          handle stays usable.
 *   GLR_OK                 otherwise. */
glr_status glr_sync_status(glr_handle* h, void* stream);

/* Declares the caller-owned state valid again after the caller wrote it
 * (resume from a saved blob, or a hand-off) and sets the next step to t. */
glr_status glr_resume(glr_handle* h, int64_t next_t);

/* Buffers for one matrix's state (glr_read_state / glr_write_state): host or
 * device pointers, any mix; a NULL member is skipped.  Each part has the size
 * and layout glr_mat_layout gives it: E N x m x n (fp32, or bf16 with
 * GLR_STORE_BF16), Ebar / S1 / S2 m x n (fp32,
 * the caller's layout), Ut d x d (row j = u_j), sigma and score d fp32, J r
 * int32, Rbar r x D fp32, info 64 int32.  S2 exists for Adam only. */
typedef struct {
  void* E;
  void* Ebar;
  void* Ut;
  void* sigma;
  void* J;
  void* score;
  void* S1;
  void* S2;
  void* Rbar;
  void* info;
} glr_state_view;

/* Enqueues on `stream` copies of matrix `mat`'s state parts into the non-NULL
 * members of *dst (stream-ordered: the copies see every step enqueued before
 * and are complete when the stream is; pageable host destinations may make
 * the call wait).  GLR_ERR_INVALID_ARG for a bad index or an S2 request
 * without Adam. */
glr_status glr_read_state(glr_handle* h, int32_t mat, const glr_state_view* dst, void* stream);

/* Enqueues on `stream` copies from the non-NULL members of *src into matrix
 * `mat`'s state (a hand-off, or a restore), and marks the state valid again
 * (as glr_resume does, without changing the next step). */
glr_status glr_write_state(glr_handle* h, int32_t mat, const glr_state_view* src, void* stream);

/* Next step the handle expects. */
glr_status glr_next_step(const glr_handle* h, int64_t* next_t);

/* Frees the handle (host memory only). */
glr_status glr_destroy(glr_handle* h);

/* Optional timing of the launch groups of glr_step with HIP events recorded on
 * the step's stream (off by default; recording adds two events per group).
 * Groups: see glr_prof_group.  glr_profile_query waits for the last recorded
 * event and returns the summed milliseconds and the number of timed launches
 * of one group since the last reset. */
typedef enum {
  GLR_PROF_EF_MEAN = 0,      /* worker mean with error feedback */
  GLR_PROF_SELECT = 1,       /* Approx-Top-r (or exact) scores */
  GLR_PROF_TOPR = 2,         /* argtop_r */
  GLR_PROF_PROJ = 3,         /* Q^(i) = P^T M^(i) */
  GLR_PROF_RBAR = 4,         /* Rbar = mean Q^(i) */
  GLR_PROF_RESID_OPT = 5,    /* residual + mean + reconstruction + optimizer */
  GLR_PROF_FULL_REFRESH = 6, /* Algorithm 3 refresh update */
  GLR_PROF_JAC_INIT = 7,     /* refresh: warm-start product and the fp64 Gram */
  GLR_PROF_JAC_UPDATE = 8,   /* refresh: two-sided update of the fp64 Gram in one Jacobi round */
  GLR_PROF_JAC_FINISH = 9,   /* refresh: sigma, sort, permutation, re-orthonormalisation */
  GLR_PROF_REFRESH = 10,     /* refresh: whole basis computation */
  GLR_PROF_SUB_ITER = 11,    /* tau = 1 refresh: one subspace iteration (all its launches) */
  GLR_PROF_JAC_SOLVE = 12,   /* refresh: pair eigensolves of one round, with the previous round's
                                rotation of U^T rows in the same launch */
  GLR_PROF_RR_UPDATE = 13,   /* tau = 1 Rayleigh-Ritz Jacobi (K x K Gram): Gram update */
  GLR_PROF_RR_SOLVE = 14,    /* tau = 1 Rayleigh-Ritz Jacobi: pair eigensolves and rotations */
  GLR_PROF_SUB_Z = 15,       /* tau = 1: Z = P^T Mo (K x D product) */
  GLR_PROF_SUB_P = 16,       /* tau = 1: Z Mo^T (K x d split-K product, before its reduction) */
  GLR_PROF_SUB_ORTH = 17,    /* tau = 1: CholeskyQR2 orthonormalisations (all their launches) */
  GLR_PROF_SUB_CHOL = 18,    /* tau = 1: K x K Cholesky factor and inverse */
  GLR_PROF_COUNT = 19
} glr_prof_group;

glr_status glr_profile_enable(glr_handle* h, int32_t on);
glr_status glr_profile_reset(glr_handle* h);
glr_status glr_profile_query(glr_handle* h, int32_t group, double* total_ms, int64_t* launches);

const char* glr_status_string(glr_status s);

/* Text of the last error on this handle ("" if none); NULL handle gives the
 * last error of a failed glr_create on this thread. */
const char* glr_last_error(const glr_handle* h);

#ifdef __cplusplus
}
#endif

#endif /* GREEDYLORE_H */
