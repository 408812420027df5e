/*
 * baco_gp.h — C-ABI of a gfx950 library for batched Gaussian-process scoring of
 * candidate configurations in a mixed real / integer / ordinal / categorical /
 * permutation search space, as used by the BaCO autotuner (Hellsten et al.,
 * "BaCO: A Fast and Portable Bayesian Compiler Optimization Framework",
 * arXiv 2212.11142).
 *
 * The two main calls are
 *   gp_fit   — GP value model (Sec. 3.2): Gram matrix of the feasible observations
 *              with Matern-5/2 over the mixed distance of Sec. 4.1, its fp64 Cholesky
 *              factor, L^-1, alpha = K^-1 y and K^-1; plus, optionally, the feasibility
 *              classifier used to weight EI (Sec. 4.2, hidden constraints).
 *   gp_score — for M candidates: posterior mean mu and standard deviation sigma of
 *              the latent objective, expected improvement (Sec. 3.3, noise-free EI,
 *              minimisation), probability of feasibility p and the acquisition value
 *              acq = EI * p where p > eps_f and the candidate is allowed by the known
 *              constraint mask, else 0 (Sec. 4.2).
 *
 * Conventions shared by every entry point:
 *  - Ownership: the library never allocates or frees device memory. Every device
 *    buffer (inputs, outputs, workspaces) belongs to the caller and must stay alive
 *    for as long as the call (gp_score, debug calls) or the model (gp_fit workspace)
 *    uses it. A gp_model is a small host-side handle; gp_model_free releases it only.
 *  - Streams: `stream` is a hipStream_t passed as void* (NULL = the null stream). All
 *    device work of gp_score and the debug calls is enqueued on it, asynchronously.
 *    gp_fit synchronises the stream (it reads back pivot status and the classifier's
 *    Newton convergence); it runs the value model on a library-owned side stream of
 *    default priority concurrently with the classifier and joins it before returning.
 *  - Errors: every call returns a gp_status; no C++ exception crosses the ABI.
 *    gp_last_error() returns a thread-local message for the last failure on the
 *    calling thread (for GP_E_NOT_SPD it names the failing pivot).
 *  - Pointers documented as "device" must be device (or managed) memory on the current
 *    HIP device; pointers documented as "host" are ordinary host memory.
 *  - Candidate results are deterministic: the same inputs give bit-identical outputs.
 */
#ifndef BACO_GP_H
#define BACO_GP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GP_OK = 0,
  GP_E_INVALID = 1,       /* bad argument: null pointer, size, range, malformed space */
  GP_E_NOT_SPD = 2,       /* a Cholesky pivot was not positive (gp_last_error names it) */
  GP_E_HIP = 3,           /* a HIP runtime call failed */
  GP_E_UNSUPPORTED = 4,   /* outside the supported envelope (d > 64, perm m > 8, ...) */
  GP_E_WORKSPACE = 5,     /* workspace missing, too small or misaligned (256 B) */
  GP_E_NOT_CONVERGED = 6  /* classifier Newton iteration did not converge */
} gp_status;

/* Parameter types of Sec. 4.1: Real, Integer, Ordinal, Categorical, Permutation. */
typedef enum { GP_REAL = 0, GP_INT = 1, GP_ORD = 2, GP_CAT = 3, GP_PERM = 4 } gp_ptype;

/* Permutation semimetrics of Sec. 4.1 (Spearman is BaCO's default); NAIVE treats the
 * whole permutation as one categorical value (the ablation of Sec. 5.3). */
typedef enum {
  GP_PERM_SPEARMAN = 0,
  GP_PERM_KENDALL = 1,
  GP_PERM_HAMMING = 2,
  GP_PERM_NAIVE = 3
} gp_permdist;

/* Search-space descriptor (all host memory, read during the call only).
 *  d            number of parameters, 1..64
 *  type[d]      gp_ptype
 *  log2[d]      nonzero: distance on log2(value) (Sec. 4.2, exponential parameters);
 *               REAL/INT/ORD only, values must be > 0. NULL = no log transform.
 *  n_levels[d]  CAT: number of levels (2..65536); ORD: number of values (1..4096);
 *               PERM: number of items m (2..8); ignored for REAL/INT.
 *  perm_dist[d] gp_permdist for PERM parameters. NULL = Spearman.
 *  lo[d], hi[d] REAL/INT declared range (inclusive), lo <= hi. Ignored otherwise.
 *  ord_values[d] ORD: pointer to n_levels[p] strictly ascending values. */
typedef struct {
  int32_t d;
  const int32_t *type;
  const int32_t *log2;
  const int32_t *n_levels;
  const int32_t *perm_dist;
  const double *lo;
  const double *hi;
  const double *const *ord_values;
} gp_space;

/* Kernel hyperparameters (host memory). Sec. 3.2: lengthscale l_i per parameter,
 * output scale sigma (a variance multiplier) and observation-noise variance. */
typedef struct {
  const double *lengthscale;  /* [d], each > 0 */
  double signal_var;          /* > 0 */
  double noise_var;           /* >= 0 (value model); ignored for the classifier */
} gp_hyper;

typedef struct gp_model gp_model; /* opaque host-side handle */

/* Raw parameter columns ("cols"): a host array of d device pointers, one per
 * parameter, each holding `count` entries:
 *   GP_REAL: double[count]            the value
 *   GP_INT:  int32_t[count]           the value, lo..hi
 *   GP_ORD:  int32_t[count]           index into ord_values, 0..n_levels-1
 *   GP_CAT:  int32_t[count]           level, 0..n_levels-1
 *   GP_PERM: int32_t[count * m]       row-major; row c is the position vector pi with
 *                                     pi[i] = 0-based position of item i in the new
 *                                     order (the convention of Sec. 4.1's loop example)
 * A configuration with an out-of-range INT/ORD/CAT entry, a non-finite REAL or a PERM
 * row that is not a permutation of 0..m-1 is invalid: gp_fit rejects it with
 * GP_E_INVALID; gp_score returns NaN mu/sigma/ei, p_feas = 0 and acq = 0 for it. */

/* ---------------------------------------------------------------- fitting */

/* Bytes of device workspace gp_fit needs for n observations (0 on invalid input).
 * with_classifier: nonzero if gp_fit will be given a classifier hyperparameter set. */
size_t gp_fit_workspace_bytes(const gp_space *space, int32_t n, int32_t with_classifier);

/* Fit the value model and, if cls != NULL, the feasibility classifier.
 *  X_cols     host array of d device pointers (raw columns, n entries each)
 *  n          number of observations, 1..4096
 *  y          device double[n], objective (lower is better; typically standardised
 *             log runtime). Entries of infeasible observations are never read.
 *  feasible   device uint8[n] (nonzero = feasible) or NULL (all feasible). The value
 *             model uses the feasible observations only (Sec. 4.2); at least one is
 *             required. The classifier uses all n, label +1 feasible / -1 infeasible.
 *  reg        value-model hyperparameters (noise_var is added to the Gram diagonal)
 *  cls        classifier hyperparameters, or NULL: then p_feas = 1 for every
 *             candidate. The classifier's kernel shares the value model's distance:
 *             cls->lengthscale must be NULL or equal to reg->lengthscale element by
 *             element (else GP_E_UNSUPPORTED); cls->signal_var is its own output
 *             scale; cls->noise_var is ignored
 *  workspace  device memory of >= gp_fit_workspace_bytes(...) bytes, 256-B aligned;
 *             owned by the caller, used by the model until gp_model_free
 *  out        receives the model handle on GP_OK
 * Errors: GP_E_INVALID (arguments, invalid configuration, no feasible observation),
 * GP_E_NOT_SPD (no automatic jitter: retry with a larger noise_var),
 * GP_E_NOT_CONVERGED, GP_E_WORKSPACE, GP_E_UNSUPPORTED, GP_E_HIP.
 * Synchronises `stream`. */
gp_status gp_fit(const gp_space *space, const void *const *X_cols, int32_t n,
                 const double *y, const uint8_t *feasible, const gp_hyper *reg,
                 const gp_hyper *cls, void *workspace, size_t ws_bytes, void *stream,
                 gp_model **out);

/* Summary of a fitted model (host struct filled by gp_model_info). */
typedef struct {
  int32_t n;              /* observations */
  int32_t n_feasible;     /* observations in the value model */
  int32_t d;              /* parameters */
  int32_t has_classifier;
  int32_t cls_iterations; /* Newton iterations used by the classifier fit */
  int32_t code_words;     /* 32-bit code words per encoded configuration */
  double fstar;           /* best (lowest) feasible y */
  double signal_var, noise_var, cls_signal_var;
} gp_model_info_t;

gp_status gp_model_info(const gp_model *model, gp_model_info_t *info);

/* Export a fitted quantity to host memory (synchronous copy).
 * Row-major matrices over the value model's feasible observations, in the order of
 * the `feasible_index` field (original observation indices, feasible ones in
 * ascending order), or over all observations (feasible first, then infeasible,
 * each ascending) for the classifier fields.
 *  GP_FIELD_K        n_f*n_f  Gram matrix incl. noise
 *  GP_FIELD_L        n_f*n_f  lower Cholesky factor (upper part zero)
 *  GP_FIELD_LINV     n_f*n_f  L^-1 (lower)
 *  GP_FIELD_KINV     n_f*n_f  K^-1
 *  GP_FIELD_ALPHA    n_f      K^-1 y
 *  GP_FIELD_FEASIBLE_INDEX n  original index of each model row (as double)
 *  GP_FIELD_CLS_F    n        classifier latent mode f_hat
 *  GP_FIELD_CLS_GRAD n        d log p(t|f)/df at f_hat
 *  GP_FIELD_CLS_SQRTW n       sqrt(W) at f_hat
 *  GP_FIELD_CLS_L    n*n      Cholesky factor of B = I + W^1/2 K_c W^1/2
 * `count` is the number of doubles at host_dst; must equal the field's size. */
typedef enum {
  GP_FIELD_K = 0, GP_FIELD_L = 1, GP_FIELD_LINV = 2, GP_FIELD_KINV = 3,
  GP_FIELD_ALPHA = 4, GP_FIELD_FEASIBLE_INDEX = 5, GP_FIELD_CLS_F = 6,
  GP_FIELD_CLS_GRAD = 7, GP_FIELD_CLS_SQRTW = 8, GP_FIELD_CLS_L = 9
} gp_field;

gp_status gp_model_export(const gp_model *model, int32_t field, double *host_dst,
                          size_t count);

/* Release the host handle (the fit workspace stays the caller's). NULL is a no-op. */
void gp_model_free(gp_model *model);

/* ---------------------------------------------------------------- scoring */

/* Bytes of device workspace gp_score needs for M candidates (0 on invalid input). */
size_t gp_score_workspace_bytes(const gp_model *model, int64_t M);

/* Score M candidates (the hot path; asynchronous on `stream`).
 *  C_cols     host array of d device pointers, raw columns with M entries each
 *  M          0..2^31-1 candidates (M = 0 is a no-op returning GP_OK)
 *  mask       device uint8[M], nonzero = allowed by the known constraints, or NULL
 *  eps_f      minimum probability of feasibility (Sec. 4.2), in [0, 1]
 *  mu, sigma, ei, acq   device float[M] outputs (required)
 *  p_feas     device float[M] output or NULL
 *  argmax     device int64[1] output or NULL: index of the largest acq (lowest index
 *             on ties; 0 when every acq is 0)
 *  workspace  device memory of >= gp_score_workspace_bytes(model, M) bytes, 256-B
 *             aligned, not shared with any concurrently running call
 * Outputs: mu = k*^T K^-1 y_f, sigma = sqrt(max(s - k*^T K^-1 k*, 0)) (latent, no
 * noise), ei = E[max(f* - f, 0)], p_feas = Phi(fbar / sqrt(1 + V)) of the Laplace probit
 * classifier (1 without one), acq = ei * p_feas if mask allows and p_feas > eps_f,
 * else 0. Computed in fp32 with an fp64 recomputation of candidates whose variance
 * or mean is ill-conditioned in fp32. */
gp_status gp_score(const gp_model *model, const void *const *C_cols, int64_t M,
                   const uint8_t *mask, float eps_f, float *mu, float *sigma, float *ei,
                   float *p_feas, float *acq, int64_t *argmax, void *workspace,
                   size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------- fit fused with scoring */

/* Bytes of device workspace gp_fit_score needs for n observations and M candidates
 * (0 on invalid input): the fit's workspace (gp_fit_workspace_bytes rounded up to a
 * multiple of 256) followed by the scoring buffers. */
/* For callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that must not call hipMalloc): gp_score with its scoring buffers in a
 * fixed device array of GP_NOALLOC_SCRATCH_BYTES (64 MiB) that the library holds on
 * every GPU it runs on until the process ends, instead of a caller workspace. Same
 * kernels, same results as gp_score; allocates nothing (no hipMalloc, hipFree or
 * allocating library call). The caller still passes the candidates and the outputs.
 * M above gp_score_noalloc_max_candidates(model) (about 29,000 candidates at n = 512,
 * 3,000 at n = 4096) is rejected with GP_E_WORKSPACE. All calls on one GPU share its
 * array: calls that overlap on that GPU (on different streams or threads) race, so the
 * caller orders them, e.g. on one stream. Asynchronous on `stream`. */
#define GP_NOALLOC_SCRATCH_BYTES (64u << 20)
gp_status gp_score_noalloc(const gp_model *model, const void *const *C_cols, int64_t M,
                           const uint8_t *mask, float eps_f, float *mu, float *sigma,
                           float *ei, float *p_feas, float *acq, int64_t *argmax, void *stream);
/* Largest M gp_score_noalloc accepts for this model (0 for a NULL model). */
size_t gp_score_noalloc_max_candidates(const gp_model *model);

size_t gp_fit_score_workspace_bytes(const gp_space *space, int32_t n, int32_t with_classifier,
                                    int64_t M);

/* One optimisation step's model and scores: gp_fit, then gp_score of M candidates with
 * the fitted model (the surrogate refit and the acquisition over a candidate batch that
 * follow every new observation, Sec. 3.2 and Sec. 4.2), with the same arguments,
 * results and errors as those two calls. The two overlap on the device: the value
 * model, candidate encoding and cross-kernel run beside the classifier's Newton
 * iterations, on streams that each hold a fixed share of the compute units (library
 * owned, default priority, ordered after earlier work on `stream`); the contraction
 * and the rest of scoring follow on `stream`. Returns once the classifier has
 * converged and the remaining scoring work is enqueued on `stream`.
 *  workspace  >= gp_fit_score_workspace_bytes(space, n, cls != NULL, M) bytes, 256-B
 *             aligned; the model lives in it (as with gp_fit) and the scoring buffers
 *             are free again once the scoring work on `stream` has completed.
 * On an error nothing is scored, *out is NULL and no work is left in flight. */
gp_status gp_fit_score(const gp_space *space, const void *const *X_cols, int32_t n,
                       const double *y, const uint8_t *feasible, const gp_hyper *reg,
                       const gp_hyper *cls, const void *const *C_cols, int64_t M,
                       const uint8_t *mask, float eps_f, float *mu, float *sigma, float *ei,
                       float *p_feas, float *acq, int64_t *argmax, void *workspace,
                       size_t ws_bytes, void *stream, gp_model **out);

/* ---------------------------------------------------------------- acquisition optimiser */

/* Bytes of device workspace gp_local_search needs (0 on invalid input). */
size_t gp_local_search_workspace_bytes(const gp_model *model, int64_t M, int32_t n_starts);

/* Multi-start local search of the acquisition function (Sec. 3.3: the best of many
 * sampled configurations are starting points; neighbours are the configurations that
 * differ in a single parameter). Scores the M candidates C_cols as gp_score does
 * (mask, eps_f as there), takes the min(n_starts, M) of largest acq (lower index first
 * on ties) as starts, and moves each start to its best neighbour (largest acq, first in
 * the order below on ties) while that acq is strictly larger than its own, at most
 * max_steps times. Neighbours, parameter by parameter in space order: REAL the value
 * moved by -/+ 1/16 of its transformed range (in log2 if flagged); INT value -/+ 1;
 * ORD index -/+ 1; CAT every other level, ascending; PERM every exchange of the
 * positions of two items i < j, (i, j) ascending; a move leaving the declared range is
 * skipped. The mask applies to the M candidates only: neighbours are checked against
 * the declared ranges alone. Moves are decided on the fp32 acq of gp_score.
 *  n_starts   1..64        max_steps  >= 0
 *  out_cols   host array of d device pointers, raw columns (formats above) with
 *             min(n_starts, M) entries: each start's final configuration, starts in
 *             order of their initial acq
 *  out_acq    device float[]: final acq;  out_steps  device int32[]: moves taken
 *  out_start  device int64[]: index of each start in C_cols
 *  workspace  device memory of >= gp_local_search_workspace_bytes(model, M, n_starts)
 *             bytes, 256-B aligned
 * Synchronous: returns when every start has stopped (it checks with the host every few
 * moves). Errors as gp_score. */
gp_status gp_local_search(const gp_model *model, const void *const *C_cols, int64_t M,
                          const uint8_t *mask, float eps_f, int32_t n_starts, int32_t max_steps,
                          void *const *out_cols, float *out_acq, int32_t *out_steps,
                          int64_t *out_start, void *workspace, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------- hyperparameters */

/* Gamma prior on every lengthscale (Sec. 3.2, GP hyperparameter optimisation): density
 * rate^shape l^(shape-1) exp(-rate l) / Gamma(shape) in l itself; shape, rate > 0. The
 * inputs are normalised to [0, 1], so one prior serves every parameter. */
typedef struct {
  double shape;
  double rate;
} gp_gamma_prior;

/* A hyperparameter setting is a double[d + 2] row
 *   theta = (log l_1 .. log l_d, log signal_var, t),  noise_var = noise_floor + e^t,
 * (positivity without bounds; the floor keeps the kernel matrix away from singular
 * when the data are nearly noise free). The objective of a setting is
 *   log p(y_f | theta) + sum_p log Gamma(l_p; shape, rate)      (prior optional)
 * with p(y_f | theta) the GP marginal likelihood of the feasible observations (zero
 * prior mean, the kernel of gp_fit), and -inf where the kernel matrix is not finite and
 * positive definite or the value or gradient overflows. */

/* Bytes of device workspace for a call on n observations with n_settings settings:
 * gp_log_posterior: n_keep = 0, n_settings = count; gp_hyperfit: n_settings = n_samples,
 * n_keep as there. 0 on invalid input. Dominated by 3 fp64 matrices of
 * round_up(n, 32)^2 per setting of a batch (at most 64 settings per batch) and the
 * d n^2 fp64 pair terms. */
size_t gp_hyper_workspace_bytes(const gp_space *space, int32_t n, int32_t n_settings,
                                int32_t n_keep);

/* Objective and gradient of `count` settings (Sec. 3.2):
 *  X_cols, n, y, feasible   the observations, as for gp_fit (infeasible ones and their
 *                           y are ignored; at least one feasible)
 *  theta      device double[count][d + 2] settings
 *  prior      host struct or NULL (no prior);  noise_floor >= 0
 *  value      device double[count] output: the objective (-inf: not a kernel)
 *  grad       device double[count][d + 2] output (d objective / d theta) or NULL;
 *             left unwritten for settings whose value is -inf
 * The gradient is the trace formula 1/2 tr((a a^T - K^-1) dK/dtheta) + d prior/dtheta,
 * a = K^-1 y_f. Computed in fp64 (batched blocked Cholesky and triangular inverse).
 * Synchronous. */
gp_status gp_log_posterior(const gp_space *space, const void *const *X_cols, int32_t n,
                           const double *y, const uint8_t *feasible, const double *theta,
                           int32_t count, const gp_gamma_prior *prior, double noise_floor,
                           double *value, double *grad, void *workspace, size_t ws_bytes,
                           void *stream);

/* Multistart fit of the hyperparameters (Sec. 3.2): evaluates the objective at the
 * n_samples caller-drawn settings theta0 (device double[n_samples][d + 2]; the paper
 * samples them uniformly), keeps the n_keep (1..min(64, n_samples)) of largest
 * objective (lower index first on ties) and runs L-BFGS from each: memory of 10 pairs,
 * two-loop recursion with H0 = (s'y / y'y) I, first step along the normalised
 * gradient, step halving from 1 until the Armijo condition (c1 = 1e-4) holds (30
 * halvings at most; -inf counts as a failed trial), pairs with s'y <= 1e-10 y'y not
 * stored, restart on a non-ascent direction. A start stops when max |grad| <= gtol,
 * when the objective changes by <= ftol * max(|old|, |new|, 1), after max_iter
 * accepted steps or when its line search fails.
 *  theta_out   device double[n_keep][d + 2]: final setting of each kept start
 *  value_out   device double[n_keep]: its objective
 *  value0_out  device double[n_samples] (objective of every sample) or NULL
 *  keep_out    device int32[n_keep] (index of each start in theta0) or NULL
 *  iters_out   device int32[n_keep] (accepted steps) or NULL
 *  status_out  device int32[n_keep] or NULL: 1 gradient tolerance, 2 objective change,
 *              3 iteration limit, 4 line search failed, 5 start not a kernel
 * Starts are in the order of their sample objective. Synchronous: the host checks the
 * running starts every few batched evaluations. */
gp_status gp_hyperfit(const gp_space *space, const void *const *X_cols, int32_t n,
                      const double *y, const uint8_t *feasible, const double *theta0,
                      int32_t n_samples, int32_t n_keep, const gp_gamma_prior *prior,
                      double noise_floor, int32_t max_iter, double gtol, double ftol,
                      double *theta_out, double *value_out, double *value0_out,
                      int32_t *keep_out, int32_t *iters_out, int32_t *status_out,
                      void *workspace, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------- known constraints */

/* Chain-of-Trees (Sec. 4.2, known constraints): the parameters that constraints link
 * form trees (one level per parameter, one node per value); a tree's leaves are its
 * feasible partial configurations. Parameters of different trees are independent, so
 * the chain holds exactly the feasible configurations. Opaque, host-side handle whose
 * tables live in the caller's workspace. */
typedef struct gp_cot gp_cot;

/* Bytes of device workspace of a chain (0 on invalid input); arguments as for
 * gp_cot_create. */
size_t gp_cot_workspace_bytes(const gp_space *space, int32_t n_trees, const int32_t *tree_size,
                              const int32_t *tree_params, const int64_t *n_leaves);

/* Build a chain (synchronous).
 *  n_trees      0..64
 *  tree_size    host int32[n_trees]: parameters of each tree (>= 1)
 *  tree_params  host int32[sum tree_size]: the trees' parameters, tree after tree, each
 *               tree's in level order; INT, ORD and CAT parameters only, each in at most
 *               one tree; a tree's value indices, each in ceil(log2(count)) bits,
 *               must fit 64 bits
 *  n_leaves     host int64[n_trees] (>= 1)
 *  leaves       host array of n_trees device pointers: tree t's leaves as int32
 *               [n_leaves[t]][tree_size[t]] value indices (INT: value - lo, ORD: index,
 *               CAT: level), in strictly increasing lexicographic order (the order of a
 *               depth-first walk that takes children in ascending value order); only
 *               read during the call
 *  workspace    >= gp_cot_workspace_bytes bytes, 256-B aligned; holds the chain's
 *               tables (8 bytes per leaf) and must outlive the handle
 * GP_E_INVALID names the first leaf out of range or out of order. */
gp_status gp_cot_create(const gp_space *space, int32_t n_trees, const int32_t *tree_size,
                        const int32_t *tree_params, const int64_t *n_leaves,
                        const int32_t *const *leaves, void *workspace, size_t ws_bytes,
                        void *stream, gp_cot **out);

/* Draw M configurations (asynchronous): for each tree a leaf uniformly over its
 * leaves (not child by child: Sec. 4.2); parameters outside every tree uniformly over
 * their domain (INT/ORD/CAT values, REAL lo + (hi - lo) x with x uniform in [0, 1) on a
 * 2^-53 grid, PERM a uniform permutation by Fisher-Yates). Random words: Philox4x64-10
 * (Salmon et al., SC 2011) with key (seed, 0) and counter (offset + j, b, 0, 0) for
 * the b-th block of four words of configuration j, used in order: one per tree, then
 * per free parameter in space order one word (m - 1 for PERM, for i = m-1 .. 1); an
 * index uniform in [0, c) is floor(u c / 2^64). Configuration j thus depends only on
 * (seed, offset + j): batches drawn with consecutive offsets concatenate.
 *  out_cols   host array of d device pointers, raw columns (formats of gp_fit) with M
 *             entries each */
gp_status gp_cot_sample(const gp_cot *chain, int64_t M, uint64_t seed, uint64_t offset,
                        void *const *out_cols, void *stream);

/* mask[j] = 1 if configuration j (raw columns; only the trees' parameters are read,
 * the others may be NULL) is in the chain, i.e. satisfies the known constraints, else
 * 0 (also for a value outside its parameter's range). Asynchronous. */
gp_status gp_cot_member(const gp_cot *chain, const void *const *cols, int64_t M,
                        uint8_t *mask, void *stream);

void gp_cot_free(gp_cot *chain);

/* ---------------------------------------------------------------- hidden constraints */

/* Random-forest feasibility model (Sec. 4.2, hidden constraints: a random forest fitted
 * to the feasible / infeasible outcomes predicts the probability of feasibility that
 * multiplies the expected improvement). Opaque handle; its trees live in the caller's
 * workspace. Features: REAL and INT values, ORD index, CAT level, one per PERM item
 * (its position), at most 120. Trees: CART with Gini impurity on a bootstrap sample of
 * the n observations, mtry = floor(sqrt(F)) features tried per node; the best split
 * minimises pos_L neg_L / c_L + pos_R neg_R / c_R (exact rational comparison; ties: the
 * lower feature, then the lower threshold), x_f <= threshold goes left, the threshold
 * being the largest value sent left; a node is a leaf if pure, smaller than min_split,
 * at max_depth, without a candidate threshold or without a strict improvement over its
 * own pos neg / c, and predicts pos / c. Random choices: Philox4x64-10 with key
 * (seed, 0), counter (tree, stream, block, 3); stream 0: bootstrap index i from word i
 * as floor(u n / 2^64); stream k + 1: node k's features, word q choosing position
 * q + floor(u (F - q) / 2^64) of a partial Fisher-Yates shuffle of 0..F-1 (nodes
 * numbered breadth first, children in order). */
typedef struct gp_forest gp_forest;

size_t gp_forest_workspace_bytes(const gp_space *space, int32_t n, int32_t n_trees);

/* Fit n_trees (1..4096) trees on the n (1..4096) observations X_cols with labels
 * feasible (device uint8[n], nonzero = feasible); max_depth >= 0, min_split >= 1.
 * Synchronous; GP_E_INVALID for an invalid observation. */
gp_status gp_forest_fit(const gp_space *space, const void *const *X_cols, int32_t n,
                        const uint8_t *feasible, int32_t n_trees, int32_t max_depth,
                        int32_t min_split, uint64_t seed, void *workspace, size_t ws_bytes,
                        void *stream, gp_forest **out);

/* p_feas[j] = fl32(mean over trees of the leaf value of configuration j), the sum in
 * tree order in fp64 (device float[M]); with acq (device float[M], needs ei): acq =
 * ei * p_feas if mask (NULL = all) allows j and p_feas > eps_f, else 0 (as gp_score
 * forms it with the GP classifier). Asynchronous. */
gp_status gp_forest_predict(const gp_forest *forest, const void *const *C_cols, int64_t M,
                            const float *ei, const uint8_t *mask, float eps_f, float *p_feas,
                            float *acq, void *stream);

/* Inspection: tree `tree` as host arrays of `capacity` entries (2 n suffices) in
 * breadth-first node order: feature (-1 leaf), left child (right = left + 1), value
 * (threshold of an internal node, pos / c of a leaf). Synchronous. */
gp_status gp_forest_tree(const gp_forest *forest, int32_t tree, int32_t capacity,
                         int32_t *n_nodes, int32_t *feature, int32_t *left, double *value,
                         void *stream);

void gp_forest_free(gp_forest *forest);

/* ---------------------------------------------------------------- inspection */

/* Bytes of workspace needed by the debug calls below for `count` configurations. */
size_t gp_debug_workspace_bytes(const gp_space *space, const gp_model *model,
                                int64_t count);

/* Normalised numeric codes of `count` configurations (Sec. 3.2 normalisation,
 * Sec. 4.2 log transform): device float out[count * n_numeric] (row-major, numeric
 * parameters REAL/INT/ORD in space order), u = fl32((t(v) - t_lo) / (t_hi - t_lo))
 * with t = identity or log2 and every step one IEEE fp64 operation. Also writes
 * device uint8 valid[count] (1 = valid configuration) if valid != NULL. */
gp_status gp_debug_encode(const gp_space *space, const void *const *cols, int64_t count,
                          float *out, uint8_t *valid, void *workspace, size_t ws_bytes,
                          void *stream);

/* Per-parameter distance terms between `count` configurations and the model's
 * observations (model order, feasible first), Sec. 4.1: device float
 * terms[count][n][d]: REAL/INT/ORD -> fl32(u_c - u_x); CAT -> 1[c != x];
 * PERM -> the integer semimetric (Kendall discordant pairs, Spearman sum of squared
 * position changes, Hamming moved items, naive 0/1). */
gp_status gp_debug_terms(const gp_model *model, const void *const *cols, int64_t count,
                         float *terms, void *workspace, size_t ws_bytes, void *stream);

/* The fp32 cross-kernel the scorer builds: device float Kstar[count][n] (model order)
 * = signal_var * Matern52(r), r^2 = sum_i d_i^2 / l_i^2 (Sec. 3.2). */
gp_status gp_debug_xkernel(const gp_model *model, const void *const *cols, int64_t count,
                           float *Kstar, void *workspace, size_t ws_bytes, void *stream);

/* Inspection of the production cross-kernel pass itself (its instantiation that also
 * stores what each pair's kernel value is computed from), Sec. 4.1 distances and the
 * Sec. 3.2 kernel: device float r2[count][n] (model order) = the fp32 squared distance
 * sum_p w_p s_p the pass feeds to the Matern function, and device int32
 * counts[count][n][W] = the exact integer sum of each integer word: a BITS word gives
 * popcount(c XOR x) (2 per differing categorical of the one-hot fields it holds, the
 * Kendall discordant-pair count, or the bits of a Hamming permutation's one-hot
 * positions, which span two words: their sum is 2 x moved items), an EQ word gives
 * [c != x], a Spearman permutation gives S2 - pi.pi' = half its sum of squared position
 * changes. Host outputs (optional): n_words = W = BITS + EQ words + Spearman
 * permutations, and word_params[W] = bit mask of the space parameters behind each
 * word. Workspace: gp_debug_workspace_bytes(NULL, model, count). Asynchronous. */
gp_status gp_debug_pairs(const gp_model *model, const void *const *cols, int64_t count,
                         float *r2, int32_t *counts, uint64_t *word_params, int32_t *n_words,
                         void *workspace, size_t ws_bytes, void *stream);

/* Thresholds of the fp64 recomputation inside gp_score: a candidate is recomputed in
 * fp64 when its fp32 variance is below var_frac * signal_var or the fp32 rounding bound
 * of its mean exceeds sens * max(|mu|, 1). Defaults 1e-2 and 300. var_frac = INFINITY
 * or sens < 0 sends every valid candidate through the fp64 path (used by tests of that
 * path); var_frac = 0 with sens = INFINITY sends none. Host call, no device work;
 * applies to later gp_score calls with this model. GP_E_INVALID for NULL model or
 * NaN thresholds. */
gp_status gp_debug_set_refine(gp_model *model, double var_frac, double sens);

/* ---------------------------------------------------------------- profiling */

/* Stage timing of gp_score and of the scoring inside gp_fit_score, with HIP events
 * recorded on the streams the stages run on. The contract stage of a gp_fit_score call
 * is the sum of its two contraction launches (value tiles on the value model's stream,
 * the other tiles on `stream`); its encode stage runs on `stream` beside the value
 * model's fit. */
typedef enum {
  GP_STAGE_ENCODE = 0, GP_STAGE_XKERNEL = 1, GP_STAGE_CONTRACT = 2,
  GP_STAGE_EPILOGUE = 3, GP_STAGE_REFINE = 4, GP_STAGE_ARGMAX = 5, GP_STAGE_COUNT = 6
} gp_stage;

/* Start recording (clears previous totals). Calls made while recording each record
 * up to GP_STAGE_COUNT+5 events; at most 4096 calls are recorded. */
gp_status gp_profile_start(void);
/* Stop, wait for the recorded events and return per-stage totals in milliseconds
 * (host double[GP_STAGE_COUNT]) and the number of recorded scoring calls. */
gp_status gp_profile_stop(double *stage_ms, int64_t *calls);

/* Number of candidates that the most recent gp_score using `workspace` (with this
 * model and M) handed to the fp64 recomputation. Synchronises `stream`; host int64
 * out. Valid until the next gp_score with the same workspace. */
gp_status gp_score_refined_count(const gp_model *model, const void *workspace,
                                 int64_t M, void *stream, int64_t *count);

/* Releases what the library itself allocated: the streams it created per device (for
 * the concurrent parts of gp_fit and gp_fit_score), the pinned host buffers of every host
 * thread (fit status ring, readback and staging; local-search flags) and the profiling
 * events. Each stream is synchronised before it is destroyed. Not a method step: it lets
 * a process end with nothing of the library still registered with the HIP runtime (the
 * Python binding calls it at interpreter exit). Call it only when no library call is
 * running on any thread; a later call recreates what it needs on demand. Models,
 * forests and chains are untouched (they live in caller-owned workspaces). Returns
 * GP_E_HIP with the first failing runtime call in gp_last_error. */
gp_status gp_release(void);

/* Thread-local description of the last error on this thread ("" if none). */
const char *gp_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int32_t gp_version(void);

#ifdef __cplusplus
}
#endif
#endif /* BACO_GP_H */
