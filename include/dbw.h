/*
 * dbw.h -- C ABI of the Dynamic Backup Workers (DBW) hot path on one MI355X.
 *
 * The library simulates a synchronous parameter server (PS) with n logical
 * workers on one GPU (Xu, Neglia, Sebastianelli, "Dynamic Backup Workers for
 * Parallel Machine Learning", Sect. 2 and Sect. 3):
 *   - every worker computes a minibatch gradient at the same w_t (Eq. gradient);
 *   - the PS averages only the k_t fastest gradients (Eq. grad_bw) and updates
 *     w (Eq. update);
 *   - DBW picks k_t = n - b_t from end-of-iteration gradient statistics
 *     (Eqs. sumvariancekt, normsquarekt, estimateL and their D-window means,
 *     Eq. gain) and from an estimate of the order-statistic arrival times
 *     (Eq. quadratic_opt), maximising gain per unit of time (Eqs. greedy,
 *     greedy2).
 *
 * Conventions for every entry point:
 *   - Pointers named as DEVICE are device memory owned by the caller; they are
 *     read or written asynchronously on the context's HIP stream and must stay
 *     valid until the stream has passed the call.  HOST pointers are read or
 *     written before the call returns.
 *   - Arrays are dense and row-major; float is IEEE fp32, double fp64.
 *   - Model parameters w have P = dbw_param_count(cfg) floats:
 *       softmax regression: W [d][C] (no bias), P = d*C;
 *       MLP d-H-C with ReLU: [W1 (d x H) | b1 (H) | W2 (H x C) | b2 (C)];
 *       CNN: [W1 (800 x H) | b1 (H) | W2 (H x C) | b2 (C) | Wc1 (20 x 1 x 5 x 5) |
 *       bc1 (20) | Wc2 (50 x 20 x 5 x 5) | bc2 (50)], P = 800 H + H + H C + C + 25570.
 *     Gradients use the same layout.
 *   - Every call returns a dbw_status; nothing throws across the ABI.  Argument
 *     errors are detected on the host before any work is queued (DBW_EINVAL,
 *     DBW_ERANGE).  Errors only the kernels can see (a minibatch row index
 *     outside the dataset, k larger than the number of workers that ever
 *     arrive) raise a device error flag that dbw_sync() reports.  HIP failures
 *     return DBW_EHIP.  dbw_last_error() gives a text for the last failure.
 *   - A context is not thread-safe; distinct contexts are independent.
 */
#ifndef DBW_H
#define DBW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DBW_OK = 0,
  DBW_EINVAL = -1,      /* bad argument: NULL pointer, shape, config        */
  DBW_ERANGE = -2,      /* k outside [1, n] or beyond the workers that arrive,
                           row index outside the dataset                     */
  DBW_EHIP = -3,        /* a HIP runtime call failed                         */
  DBW_ESTATE = -4,      /* call does not fit the context's state             */
  DBW_EUNSUPPORTED = -5 /* shape the kernels do not handle                   */
} dbw_status;

/* DBW_CNN: the MNIST network shape of Sect. 4 (two 5 x 5 convolutions and
 * two fully connected layers) on 28 x 28 single-channel images (d = 784):
 * conv 1 -> 20 channels, 2 x 2 max pooling, ReLU, conv 20 -> 50, 2 x 2 max
 * pooling, ReLU, the 800 features (channel, row, column), FC 800 -> H with
 * ReLU, FC H -> C.  Convolutions are valid, stride 1; a pooling window passes
 * (and back-propagates to) its first largest entry in row-major order. */
typedef enum { DBW_SOFTMAX = 0, DBW_MLP = 1, DBW_CNN = 2 } dbw_model;

/* Virtual clock of the simulated cluster (Sect. 2, the synchronisation
 * variants; Sect. 3.2).  FRESH: every worker starts each iteration at its
 * beginning, so a worker's arrival offset is its round-trip time and all n
 * arrivals are samples.  PSW (Push & Wait): the PS pushes w_{t+1} once it
 * holds k_t gradients of w_t; a worker still computing a gradient of an older
 * vector finishes it, then takes the most recent vector; with s_t the start
 * of iteration t and b_i the time worker i becomes free, worker i computes
 * w_t iff b_i <= s_t or b_i < s_{t+1}, its offset is
 * max(s_t, b_i) - s_t + tau_i, and a worker still busy at s_{t+1} skips w_t
 * (no sample: the estimate's data are censored).  PSI (Push & Interrupt):
 * the PS pushes w_{t+1} once it holds k_t gradients of w_t and every worker
 * drops the gradient it is computing to start on w_{t+1}; offsets are the
 * round-trip times as under FRESH, but only the first k_t arrivals in
 * (offset, worker index) order complete, so only they are samples. */
typedef enum { DBW_CLOCK_FRESH = 0, DBW_CLOCK_PSW = 1, DBW_CLOCK_PSI = 2 } dbw_clock;

/* How k_t is chosen (Sect. 3.3; the settings compared in Sect. 4).
 * DBW: Eqs. gain, greedy, greedy2.  STATIC: k_t = k_static at every
 * iteration (a fixed number of backup workers); the objective is still
 * computed as under DBW.  BLIND (B-DBW): the gain G_k is replaced by k and
 * the rest of the rule is unchanged (k_t = n before the first smoothness
 * estimate, the largest k among equal objectives, the loss guard). */
typedef enum { DBW_POLICY_DBW = 0, DBW_POLICY_STATIC = 1, DBW_POLICY_BLIND = 2 } dbw_policy;

/* Time estimate T_hat_k (Sect. 3.2).  ISOTONIC: from the solution of Eq.
 * quadratic_opt (see dbw_time_estimate).  NAIVE: the empirical mean of the
 * samples of cell (k,k), the first approach the section sets aside; NaN (k
 * not eligible) while that cell holds no sample. */
typedef enum { DBW_ESTIMATOR_ISOTONIC = 0, DBW_ESTIMATOR_NAIVE = 1 } dbw_estimator;

/* Rows of the worker-gradient buffer that dbw_step writes (the PS only uses
 * the k_t fastest gradients, Eq. grad_bw).  ALL: every worker's row (the
 * aggregation then reads the selected ones back).  SELECTED: only the
 * selected workers' rows; NONE: no row.  With SELECTED or NONE, wherever the
 * softmax gradient kernel splits a worker's minibatch into several row slabs,
 * one kernel sums the selected workers' slab partials and aggregates them
 * directly, so the unselected rows are never formed and no row is read back;
 * g_t, the updated w, the losses, k and the mask are bitwise those of ALL,
 * the statistics equal up to the order of their fp64 and fp32 partial sums.
 * Where the gradients come from per-worker GEMM tiles (softmax with more
 * than 16 classes under SELECTED or NONE, the MLP and the CNN under
 * SELECTED), the choice and the selection run before the gradient kernels,
 * which compute every worker's gradient but store only the selected rows;
 * k, the mask, g_t, w, the losses and the statistics are bitwise those of
 * ALL.  Rows not written hold unspecified values after dbw_step.
 * dbw_worker_grads always writes every row. */
typedef enum { DBW_G_ROWS_ALL = 0, DBW_G_ROWS_SELECTED = 1, DBW_G_ROWS_NONE = 2 } dbw_g_rows;

#define DBW_MAX_N 1024 /* logical workers per context                       */
#define DBW_MAX_D 64   /* length of the estimator averaging window D          */

/* Problem description.  n workers, minibatch B per worker, d input features,
 * C classes, H hidden units (MLP only), learning rate eta (constant for all
 * k), window D of the estimator averages, loss guard factor beta >= 1
 * (Eq. greedy2), virtual clock (dbw_clock; 0 = fresh start), rule of the
 * choice of k (dbw_policy; 0 = DBW) and time estimate (dbw_estimator; 0 =
 * isotonic), rows of G that dbw_step writes (dbw_g_rows; 0 = all).
 * Zero-initialised fields give the method as defined.  S > 0 declares
 * a resident dataset of S rows that minibatches may index (see
 * dbw_worker_grads); S = 0 means minibatches are passed materialised. */
typedef struct {
  int32_t model; /* dbw_model */
  int32_t n, B, d, C, H;
  int32_t D;
  int32_t clock;     /* dbw_clock */
  int32_t policy;    /* dbw_policy */
  int32_t k_static;  /* k of DBW_POLICY_STATIC, in [1, n]; ignored otherwise */
  int32_t estimator; /* dbw_estimator */
  int32_t g_rows;    /* dbw_g_rows */
  double eta, beta;
  int64_t S;
} dbw_config;

/* End-of-iteration statistics over the k received gradients (Sect. 3.1):
 * gnorm2 = ||g_t||^2; V_plus = Eq. sumvariancekt (for k = 1 the current
 * D-window mean of past V_plus, 0 without history); N_plus = Eq.
 * normsquarekt; F_hat = mean minibatch loss of the received workers. */
typedef struct {
  double gnorm2, V_plus, N_plus, F_hat;
} dbw_iter_stats;

/* DBW estimator state carried between iterations (Sect. 3.1, 3.3).  Histories
 * are oldest first; only the last D entries are kept.  hL holds the
 * smoothness estimates L_plus (Eq. estimateL), pushed from the second
 * iteration on when their denominator is positive.  F_prev, F_prev2 are
 * F_hat of the two previous iterations (nF of them valid). */
typedef struct {
  int64_t t;      /* iterations completed                                   */
  int32_t k_prev; /* k_{t-1}; n before the first iteration                  */
  int32_t nV;     /* valid entries of hV and hN                              */
  int32_t nL;     /* valid entries of hL                                     */
  int32_t nF;     /* valid entries among F_prev, F_prev2 (0..2)              */
  double F_prev, F_prev2;
  double hV[DBW_MAX_D], hN[DBW_MAX_D], hL[DBW_MAX_D];
} dbw_estimator_state;

typedef struct dbw_ctx dbw_ctx;

/* P for a configuration; -1 if the configuration is invalid. */
int64_t dbw_param_count(const dbw_config* cfg);

/* Create a context bound to HIP stream `stream` (a hipStream_t, NULL for the
 * default stream) on the current device.  Validates cfg (n in [1, DBW_MAX_N],
 * B, d, C >= 1, C <= 4096, H >= 1 for the MLP and the CNN, d = 784 for the
 * CNN, D in [1, DBW_MAX_D], eta > 0,
 * beta >= 1, S >= 0), allocates all device workspace (no allocation happens in
 * later calls) and sets the estimator state to its initial value.  Returns
 * DBW_EUNSUPPORTED when one array the kernels address (P floats, the n*B*d
 * minibatch floats, the S*d dataset floats, n*B*C or n*B*H activations)
 * would reach 2 GiB. */
dbw_status dbw_create(const dbw_config* cfg, void* stream, dbw_ctx** out);
void dbw_destroy(dbw_ctx* ctx);
/* Text of the last failure on ctx; with ctx NULL, of the last failed
 * context-free call (dbw_grad_stats_static) on the calling thread. */
const char* dbw_last_error(const dbw_ctx* ctx);

/* Waits for the context's stream and reports device-side errors raised since
 * the last dbw_sync (then clears them): DBW_ERANGE for a row index outside
 * [0, S) or k beyond the number of workers whose tick is below INT64_MAX. */
dbw_status dbw_sync(dbw_ctx* ctx);

/* Worker gradients (Sect. 2, Eq. gradient).  For each worker i, at the common
 * parameters w (DEVICE float [P]):
 *   G[i] = (1/B) sum_b grad f(x_{i,b}, w)   (DEVICE float [n][P], out)
 *   loss[i] = (1/B) sum_b f(x_{i,b}, w)      (DEVICE float [n], out)
 * with f the natural-log cross-entropy of the softmax of the model output.
 * Minibatches: if rows == NULL, X is DEVICE float [n][B][d] and y DEVICE int32
 * [n][B]; else X is the resident dataset DEVICE float [S][d], y its labels
 * DEVICE int32 [S], and rows DEVICE int32 [n][B] lists each worker's row
 * indices into it.  Labels must lie in [0, C).  w, X and G must be 16-byte
 * aligned (DBW_EINVAL otherwise). */
dbw_status dbw_worker_grads(dbw_ctx* ctx, const float* w, const float* X, const int32_t* y,
                            const int32_t* rows, float* G, float* loss);

/* Fastest-k aggregation (Sect. 2, Eq. grad_bw).  ticks (DEVICE int64 [n]) are
 * the round-trip times of the n workers in integer ticks; arrival order is the
 * order of (tick, worker index).  Writes mask (DEVICE uint8 [n]): 1 for the k
 * first arrivals, else 0; and g (DEVICE float [P]) = (1/k) sum of their rows
 * of G (DEVICE float [n][P]).  k (host) must lie in [1, n]. */
dbw_status dbw_aggregate_fastest(dbw_ctx* ctx, const float* G, const int64_t* ticks, int32_t k,
                                 float* g, uint8_t* mask);

/* Gradient statistics over the workers with mask[j] = 1 (Sect. 3.1,
 * Eqs. sumvariancekt, normsquarekt, loss estimate).  G DEVICE float [n][P],
 * mask DEVICE uint8 [n] with exactly k ones, g DEVICE float [P] their mean,
 * loss DEVICE float [n].  Writes sqnorm (DEVICE float [n]) = ||G[j]||^2 for
 * selected j, 0 otherwise, and *stats (DEVICE dbw_iter_stats).  For k = 1
 * V_plus is the context's current D-window mean of V_plus. */
dbw_status dbw_grad_stats(dbw_ctx* ctx, const float* G, const uint8_t* mask, int32_t k,
                          const float* g, const float* loss, float* sqnorm,
                          dbw_iter_stats* stats);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * statistics of dbw_grad_stats with no context, computed by the same kernels
 * on the stream `stream` (a hipStream_t, NULL for the default stream) of the
 * current device.  The call allocates nothing: its scratch (n*ceil(P/256)
 * per-row float and 2*ceil(P/256) per-tile double partial sums, each part
 * rounded up to 256 bytes) lives in one file-scope device array of
 * DBW_STATIC_SCRATCH_BYTES per GPU, held until the process ends.  G DEVICE
 * float [n][P], mask DEVICE uint8 [n], g DEVICE float [P], loss DEVICE float
 * [n]; writes sqnorm (DEVICE float [n]) and *stats (DEVICE dbw_iter_stats) as
 * dbw_grad_stats does, except that for k = 1 V_plus is V_window (HOST, the
 * caller's D-window mean of past V_plus).  A mask that does not hold exactly
 * k ones yields NaN statistics.  Errors: DBW_EINVAL (n outside [1,
 * DBW_MAX_N], P < 1, a NULL pointer, V_window not finite), DBW_ERANGE (k
 * outside [1, n]), DBW_EUNSUPPORTED (P above 2^29, or a scratch need above
 * DBW_STATIC_SCRATCH_BYTES), DBW_EHIP; dbw_last_error(NULL) then gives the
 * text, per calling thread.  Every call on one GPU uses the same array: calls
 * that overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller.  No part of the array needs clearing between calls
 * (each value a call reads was written earlier in that call). */
#define DBW_STATIC_SCRATCH_BYTES (8u * 1024u * 1024u)
dbw_status dbw_grad_stats_static(int32_t n, int64_t P, const float* G, const uint8_t* mask, int32_t k,
                                 const float* g, const float* loss, double V_window, float* sqnorm,
                                 dbw_iter_stats* stats, void* stream);

/* Choice of k_t = n - b_t from the context's estimator state (Sect. 3.3,
 * Eqs. gain, greedy, greedy2).  T_hat (DEVICE double [n]) holds the time
 * estimates T_hat_k for k = 1..n; an entry that is not finite and positive
 * makes that k ineligible.  Writes k_out, b_out (DEVICE int32) and, if not
 * NULL, objective (DEVICE double [n]) = G_hat_k / T_hat_k (NaN before the
 * first smoothness estimate exists, and for ineligible k).  The state is not
 * modified. */
dbw_status dbw_choose_b(dbw_ctx* ctx, const double* T_hat, int32_t* k_out, int32_t* b_out,
                        double* objective);

/* One full DBW iteration t: estimate T_hat from the arrival times recorded so
 * far (host, Eq. quadratic_opt), choose k_t, compute all n worker gradients,
 * aggregate the k_t first arrivals, compute the statistics, update
 * w <- w - eta g_t (w DEVICE float [P], 16-byte aligned, in place), and push the estimator
 * state.  X, y, rows as in dbw_worker_grads.  ticks_host (HOST int64 [n],
 * >= 0) are the round-trip ticks tau_i of the gradient each worker computes
 * next; the context's clock turns them into arrival offsets (equal to them
 * under DBW_CLOCK_FRESH; under DBW_CLOCK_PSW the call first waits for k_{t-1}
 * and the offsets must stay below 2^48).  The k_t smallest offsets (ties to
 * the lower worker index) are aggregated; once k_t is known the offsets of
 * the workers that compute w_t are recorded, in arrival order, as samples of
 * row h = k_{t-1}, and the virtual clock advances by the k_t-th smallest
 * offset.  If k_host is not NULL the call waits for the iteration's choice and
 * stores k_t there; otherwise it returns as soon as the work is queued. */
dbw_status dbw_step(dbw_ctx* ctx, float* w, const float* X, const int32_t* y,
                    const int32_t* rows, const int64_t* ticks_host, int32_t* k_host);

/* Device views of the buffers the last dbw_step wrote (valid until the next
 * dbw_step on this context): G [n][P], loss [n], g [P], mask [n], sqnorm [n],
 * stats, T_hat [n], objective [n], k, b. */
typedef struct {
  const float* G;
  const float* loss;
  const float* g;
  const uint8_t* mask;
  const float* sqnorm;
  const dbw_iter_stats* stats;
  const double* T_hat;
  const double* objective;
  const int32_t* k;
  const int32_t* b;
} dbw_step_buffers;
dbw_status dbw_step_outputs(dbw_ctx* ctx, dbw_step_buffers* out);

/* Estimate of E[T_{k,k}] for k = 1..n (Sect. 3.2, Eq. quadratic_opt); pure
 * host computation.  cnt and tsum (HOST int64 [n][n], index [h-1][k-1]) are
 * the number and sum (in ticks) of arrival-time samples of the k-th arrival
 * when the previous iteration waited for h gradients.  The estimates solve the
 * constrained least-squares problem exactly; since unsampled cells leave the
 * solution non-unique, T_hat_k (HOST double [n], out) is the smallest value
 * x_{k,k} takes in a feasible completion of the optimum (equal to x*_{k,k}
 * when cell (k,k) was sampled), and NaN when no sampled cell lies below
 * (k,k).  Returns DBW_EINVAL for n outside [1, DBW_MAX_N], negative counts or
 * sums, or a sum on a cell with zero count. */
dbw_status dbw_time_estimate(int32_t n, const int64_t* cnt, const int64_t* tsum, double* T_hat);

/* The same estimate kept across calls (pure host computation).  A caller that
 * re-estimates after adding a few samples per call (one iteration's arrivals)
 * gets the exact result of dbw_time_estimate at a fraction of the cost: the
 * previous solution is re-certified against the new samples and only the
 * parts that stop being optimal are re-solved.  dbw_step uses one of these
 * inside every context.  Same arguments and errors as dbw_time_estimate. */
typedef struct dbw_time_estimator dbw_time_estimator;
dbw_status dbw_time_estimator_create(dbw_time_estimator** out);
void dbw_time_estimator_destroy(dbw_time_estimator* est);
dbw_status dbw_time_estimator_solve(dbw_time_estimator* est, int32_t n, const int64_t* cnt,
                                    const int64_t* tsum, double* T_hat);
/* How the estimator's solves so far were obtained (diagnostics; HOST int64
 * outs, each may be NULL): fast = exact per-column fits that satisfied every
 * other relation of Eq. quadratic_opt, warm = re-certified and repaired
 * previous solutions, full = solves from scratch.  A solve with no sampled
 * cell counts in none of them.  DBW_EINVAL for a NULL estimator. */
dbw_status dbw_time_estimator_stats(const dbw_time_estimator* est, int64_t* fast, int64_t* warm, int64_t* full);

/* Estimator state transfer (resume, lockstep testing).  HOST structs; both
 * calls synchronise the context's stream. */
dbw_status dbw_state_export(dbw_ctx* ctx, dbw_estimator_state* out);
dbw_status dbw_state_import(dbw_ctx* ctx, const dbw_estimator_state* in);

/* Arrival-time samples (HOST int64 [n][n] each, as in dbw_time_estimate) and
 * the virtual clock (HOST int64, ticks).  Export first folds in every
 * iteration whose row is known (it synchronises the stream).  Import also
 * marks every worker idle at the imported clock (DBW_CLOCK_PSW). */
dbw_status dbw_samples_export(dbw_ctx* ctx, int64_t* cnt, int64_t* tsum, int64_t* clock);
dbw_status dbw_samples_import(dbw_ctx* ctx, const int64_t* cnt, const int64_t* tsum,
                              int64_t clock);

/* Push & Wait clock: the time each worker becomes free (HOST int64 [n],
 * ticks on the virtual clock).  Export folds like dbw_samples_export; import
 * replaces the times (each >= 0; DBW_EINVAL otherwise).  Resume and lockstep
 * testing. */
dbw_status dbw_busy_export(dbw_ctx* ctx, int64_t* busy);
dbw_status dbw_busy_import(dbw_ctx* ctx, const int64_t* busy);

/* Kernel timing with HIP events on the streams the kernels run on.  With
 * dbw_profile_enable(ctx, 1) every launch of the device groups is bracketed
 * by events and the host groups accumulate wall-clock host time (steady
 * clock); with 2 only the host groups are kept (no events are recorded, so
 * the host timings are not inflated by them); 0 turns both off.
 * dbw_kernel_time synchronises and returns the summed milliseconds and the
 * count since the last reset.  Host groups: the time-estimate solve, the
 * whole dbw_step call, the part of it spent waiting for the estimate worker,
 * and the part spent queueing GPU work. */
typedef enum {
  DBW_KT_GRADS = 0,
  DBW_KT_AGGREGATE = 1,
  DBW_KT_CHOOSE = 2,
  DBW_KT_HOST_ESTIMATE = 3,
  DBW_KT_HOST_STEP = 4,
  DBW_KT_HOST_WAIT = 5,
  DBW_KT_HOST_QUEUE = 6,
  DBW_KT_COUNT = 7
} dbw_kernel_group;
dbw_status dbw_profile_enable(dbw_ctx* ctx, int32_t mode);
dbw_status dbw_kernel_time(dbw_ctx* ctx, int32_t group, double* total_ms, int64_t* launches);
dbw_status dbw_profile_reset(dbw_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* DBW_H */
