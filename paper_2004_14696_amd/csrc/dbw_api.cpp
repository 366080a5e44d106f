// C ABI of the DBW library: context, argument checks, workspace, the
// one-iteration pipeline and the host bookkeeping of arrival times.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <initializer_list>
#include <limits>
#include <mutex>
#include <new>
#include <optional>
#include <string>
#include <thread>
#include <utility>
#include <vector>

#include "dbw.h"
#include "dbw_buffer.h"
#include "dbw_internal.h"

#define DBW_API extern "C" __attribute__((visibility("default")))

namespace {

constexpr int kSlots = 4;          // in-flight iterations of the host pipeline
constexpr int kProfilePairs = 8192;

struct Span {
  size_t off = 0;
  size_t bytes = 0;
};

struct ProfileGroup {
  std::vector<hipEvent_t> start, stop;
  int used = 0;
  double done_ms = 0.0;
  int64_t done_launches = 0;
};

}  // namespace

struct dbw_ctx {
  dbw_config cfg{};
  int64_t P = 0;
  hipStream_t stream = nullptr;
  hipEvent_t ev_fin = nullptr;    // end of a step (recorded when the caller waits)
  int device = 0;
  std::string last_error;
  dbw::SoftmaxPlan splan;
  dbw::MlpPlan mplan;
  int64_t agg_nblocks = 0;
  // dbw_step aggregates the slab partials directly (g_rows not ALL, softmax
  // single pass with several slabs per worker): source and column tiles
  int slab_src = 0;
  int64_t slab_nblocks = 0;

  char* pool = nullptr;
  // device buffers (carved from pool)
  float* G = nullptr;
  float* loss = nullptr;         // [2][n]: steps alternate halves
  float* loss_last = nullptr;    // half written by the last step
  float* g = nullptr;
  uint8_t* mask = nullptr;
  float* sqnorm = nullptr;
  dbw_iter_stats* stats = nullptr;
  double* T_hat = nullptr;
  double* objective = nullptr;
  int32_t* k = nullptr;
  int32_t* b = nullptr;
  int32_t* sel = nullptr;
  int64_t* ticks = nullptr;
  dbw_estimator_state* st = nullptr;
  int32_t* err = nullptr;
  float* Gp = nullptr;
  float* lossp = nullptr;
  float* Z = nullptr;
  float* ce = nullptr;
  float* sqpart = nullptr;
  double* part = nullptr;
  float* Hh = nullptr;
  float* dA = nullptr;
  // CNN workspace
  float* cH1 = nullptr;
  uint8_t* cCode1 = nullptr;
  float* cF = nullptr;
  uint8_t* cCode2 = nullptr;
  int32_t* cYlab = nullptr;
  float* cdP2 = nullptr;
  float* cdP1 = nullptr;
  float* cPart1 = nullptr;
  float* cPart2 = nullptr;

  // pinned host staging (coherent; kernels read and write it in place)
  double* h_T = nullptr;        // [kSlots][n]
  int64_t* h_ticks = nullptr;   // [kSlots][n]
  int32_t* h_order = nullptr;   // [kSlots][n] workers by (tick, index)
  int32_t* h_k = nullptr;       // [kSlots]
  double* d_T = nullptr;        // device-side addresses of the three above
  int64_t* d_ticks = nullptr;
  int32_t* d_order = nullptr;
  int32_t* d_k = nullptr;
  int32_t* h_err = nullptr;     // [1]
  hipEvent_t ev_k[kSlots]{};    // (unused by dbw_step: k is polled in h_k)

  // host bookkeeping of arrival times
  int64_t t = 0;                // next iteration index (== device state t once drained)
  int64_t base = 0;             // first iteration issued since create/import
  int32_t k_prev_base = 0;      // k_{base-1}
  int64_t recorded = 0;         // iterations whose samples are in the grid
  int64_t clocked = 0;          // iterations whose k-th arrival advanced the clock
  std::vector<int64_t> sorted[kSlots];  // arrival offsets of the slot's iteration, ascending
  std::vector<int64_t> offs[kSlots];    // the same by worker (Push & Wait)
  std::vector<int64_t> cnt, tsum;
  int64_t clock = 0;                    // start of the next iteration to fold
  std::vector<int64_t> busy;            // Push & Wait: time each worker becomes free
  std::vector<int64_t> psw_samples;     // scratch
  std::vector<double> T_scratch;
  dbw::IsoSolver solver;
  std::vector<int> pending_rows;  // grid rows changed since the solver's last call

  // Estimate worker.  T_hat_{t+1} depends on k_{t-1} only, so it is solved on
  // a host thread of its own while the GPU runs iterations t-1 and t; the
  // launching thread then only queues kernels.  While a job is posted the
  // worker owns the grid, the clock, the solver and the pinned T slots.
  std::thread worker;
  std::mutex mu;
  std::condition_variable cv;
  bool quit = false;
  int64_t job_u = -1;               // iteration whose T_hat the job solves
  std::atomic<int> job_state{0};    // 0 none, 1 posted, 2 finished
  dbw_status job_status = DBW_OK;
  std::string job_error;

  bool profiling = false;      // host timers
  bool prof_events = false;    // device events
  ProfileGroup prof[DBW_KT_COUNT];
};

namespace {

thread_local bool t_in_worker = false;  // errors of a job go to job_error

dbw_status fail(dbw_ctx* c, dbw_status s, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    (t_in_worker ? c->job_error : c->last_error) = buf;
  }
  return s;
}

#define HIP_TRY(ctx, expr)                                                               \
  do {                                                                                   \
    hipError_t e_ = (expr);                                                              \
    if (e_ != hipSuccess)                                                                \
      return fail((ctx), DBW_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));       \
  } while (0)

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && prev != dev) (void)hipSetDevice(dev);
    else prev = -1;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

bool config_ok(const dbw_config* c, std::string* why) {
  if (!c) {
    *why = "config is NULL";
    return false;
  }
  if (c->model != DBW_SOFTMAX && c->model != DBW_MLP && c->model != DBW_CNN)
    *why = "model must be DBW_SOFTMAX, DBW_MLP or DBW_CNN";
  else if (c->n < 1 || c->n > DBW_MAX_N) *why = "n outside [1, DBW_MAX_N]";
  else if (c->B < 1 || c->d < 1) *why = "B and d must be >= 1";
  else if (c->C < 2 || c->C > 4096) *why = "C outside [2, 4096]";
  else if (c->model == DBW_MLP && (c->H < 1 || c->H > 65536)) *why = "H outside [1, 65536]";
  else if (c->model == DBW_CNN && c->d != dbw::CNN_IMG * dbw::CNN_IMG) *why = "the CNN takes d = 784 (28 x 28 images)";
  else if (c->model == DBW_CNN && (c->H < 1 || c->H > 65536)) *why = "H outside [1, 65536]";
  else if (c->D < 1 || c->D > DBW_MAX_D) *why = "D outside [1, DBW_MAX_D]";
  else if (!(c->eta > 0.0) || !std::isfinite(c->eta)) *why = "eta must be finite and > 0";
  else if (!(c->beta >= 1.0) || !std::isfinite(c->beta)) *why = "beta must be finite and >= 1";
  else if (c->S < 0 || c->S > (int64_t{1} << 31)) *why = "S outside [0, 2^31]";
  else if ((int64_t)c->n * c->B > (int64_t{1} << 30)) *why = "n*B too large";
  else if (c->clock != DBW_CLOCK_FRESH && c->clock != DBW_CLOCK_PSW && c->clock != DBW_CLOCK_PSI)
    *why = "clock must be DBW_CLOCK_FRESH, DBW_CLOCK_PSW or DBW_CLOCK_PSI";
  else if (c->policy != DBW_POLICY_DBW && c->policy != DBW_POLICY_STATIC && c->policy != DBW_POLICY_BLIND)
    *why = "policy must be DBW_POLICY_DBW, DBW_POLICY_STATIC or DBW_POLICY_BLIND";
  else if (c->policy == DBW_POLICY_STATIC && (c->k_static < 1 || c->k_static > c->n))
    *why = "k_static outside [1, n] under DBW_POLICY_STATIC";
  else if (c->estimator != DBW_ESTIMATOR_ISOTONIC && c->estimator != DBW_ESTIMATOR_NAIVE)
    *why = "estimator must be DBW_ESTIMATOR_ISOTONIC or DBW_ESTIMATOR_NAIVE";
  else if (c->g_rows != DBW_G_ROWS_ALL && c->g_rows != DBW_G_ROWS_SELECTED && c->g_rows != DBW_G_ROWS_NONE)
    *why = "g_rows must be DBW_G_ROWS_ALL, DBW_G_ROWS_SELECTED or DBW_G_ROWS_NONE";
  else return true;
  return false;
}

int64_t param_count(const dbw_config& c) {
  if (c.model == DBW_SOFTMAX) return (int64_t)c.d * c.C;
  if (c.model == DBW_CNN)
    return (int64_t)dbw::CNN_FEAT * c.H + c.H + (int64_t)c.H * c.C + c.C + dbw::CNN_CONV_PARAMS;
  return (int64_t)c.d * c.H + c.H + (int64_t)c.H * c.C + c.C;
}

void reset_host_pipeline(dbw_ctx* c, int64_t t, int32_t k_prev) {
  c->t = c->base = c->recorded = c->clocked = t;
  c->k_prev_base = k_prev;
}

// k_u for an issued iteration u (waits for the iteration's choice).
dbw_status known_k(dbw_ctx* c, int64_t u, int32_t* k) {
  if (u < c->base) {
    if (u == c->base - 1) {
      *k = c->k_prev_base;
      return DBW_OK;
    }
    return fail(c, DBW_ESTATE, "iteration %lld precedes the context's history", (long long)u);
  }
  // the PS kernel of u writes k_u into its pinned slot (0 until then) early
  // in its run; polling it keeps an event out of the stream and lets the
  // host go on before the kernel ends.  Seeing it also proves the stream has
  // finished every earlier kernel.  A HIP error, or a stream that drained
  // without the value, ends the wait.
  const int slot = static_cast<int>(u % kSlots);
  for (int64_t spin = 0;; ++spin) {
    const int32_t v = __atomic_load_n(c->h_k + slot, __ATOMIC_ACQUIRE);
    if (v != 0) {
      *k = v;
      break;
    }
    if (spin % 4096 == 4095) {
      const hipError_t q = hipStreamQuery(c->stream);
      if (q == hipSuccess && __atomic_load_n(c->h_k + slot, __ATOMIC_ACQUIRE) == 0)
        return fail(c, DBW_ESTATE, "choice of iteration %lld did not complete", (long long)u);
      if (q != hipSuccess && q != hipErrorNotReady)
        return fail(c, DBW_EHIP, "waiting for the choice of iteration %lld: %s", (long long)u, hipGetErrorString(q));
      std::this_thread::yield();
    } else {
      __builtin_ia32_pause();
    }
  }
  if (*k < 1 || *k > c->cfg.n)
    return fail(c, DBW_ESTATE, "choice of iteration %lld did not complete (k=%d)", (long long)u, *k);
  return DBW_OK;
}

// Fold into the grid every iteration u < upto whose row k_{u-1} is known, and
// into the clock every iteration u < clock_upto.  Under Push & Wait and Push
// & Interrupt the samples of iteration u depend on k_u (who computed w_u, who
// completed before the push), so both advance together up to
// max(upto, clock_upto).
dbw_status fold(dbw_ctx* c, int64_t upto, int64_t clock_upto) {
  const int n = c->cfg.n;
  if (c->cfg.clock != DBW_CLOCK_FRESH) {
    const int64_t end = std::max(upto, clock_upto);
    while (c->recorded < end) {
      const int64_t u = c->recorded;
      int32_t h, k;
      dbw_status s = known_k(c, u - 1, &h);
      if (s == DBW_OK) s = known_k(c, u, &k);
      if (s != DBW_OK) return s;
      const std::vector<int64_t>& o = c->offs[u % kSlots];
      const std::vector<int64_t>& srt = c->sorted[u % kSlots];
      const int64_t s_next = c->clock + srt[k - 1];
      std::vector<int64_t>& smp = c->psw_samples;
      smp.clear();
      if (c->cfg.clock == DBW_CLOCK_PSW) {
        for (int i = 0; i < n; ++i)
          if (c->busy[i] <= c->clock || c->busy[i] < s_next) {   // computed w_u
            smp.push_back(o[i]);
            c->busy[i] = c->clock + o[i];
          }
        std::sort(smp.begin(), smp.end());
      } else {
        smp.assign(srt.begin(), srt.begin() + k);   // the first k_u arrivals complete
      }
      c->pending_rows.push_back(h);
      for (size_t r = 0; r < smp.size(); ++r) {
        c->cnt[(size_t)(h - 1) * n + r] += 1;
        c->tsum[(size_t)(h - 1) * n + r] += smp[r];
      }
      c->clock = s_next;
      c->recorded++;
      c->clocked++;
    }
    return DBW_OK;
  }
  while (c->recorded < upto) {
    const int64_t u = c->recorded;
    int32_t h;
    dbw_status s = known_k(c, u - 1, &h);
    if (s != DBW_OK) return s;
    const std::vector<int64_t>& srt = c->sorted[u % kSlots];
    c->pending_rows.push_back(h);
    for (int i = 0; i < n; ++i) {
      c->cnt[(size_t)(h - 1) * n + i] += 1;
      c->tsum[(size_t)(h - 1) * n + i] += srt[i];
    }
    c->recorded++;
  }
  while (c->clocked < clock_upto) {
    const int64_t u = c->clocked;
    int32_t k;
    dbw_status s = known_k(c, u, &k);
    if (s != DBW_OK) return s;
    c->clock += c->sorted[u % kSlots][k - 1];
    c->clocked++;
  }
  return DBW_OK;
}

struct HostScope {
  dbw_ctx* c;
  int g;
  std::chrono::steady_clock::time_point t0;
  HostScope(dbw_ctx* ctx, int group) : c(ctx), g(group), t0(std::chrono::steady_clock::now()) {}
  ~HostScope() {
    if (!c->profiling) return;
    ProfileGroup& pg = c->prof[g];
    pg.done_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    pg.done_launches += 1;
  }
};

// T_hat_u into the pinned slot of iteration u: fold the arrivals of iteration
// u-1 into row k_{u-2} and the clock through iteration u-2, then solve.  The
// slot's previous reader, the choice kernel of iteration u-4, precedes the
// choice of iteration u-2 that the fold waits for.
dbw_status estimate(dbw_ctx* c, int64_t u) {
  // under Push & Wait and Push & Interrupt the samples of iteration u-1 need
  // k_{u-1} (and under Push & Wait the offsets of iteration u the busy times
  // after it), so the fold goes through u-1, waiting for k_{u-1}
  const int64_t clock_upto = c->cfg.clock != DBW_CLOCK_FRESH ? u : std::max<int64_t>(c->clocked, u - 1);
  if (dbw_status s = fold(c, u, clock_upto); s != DBW_OK) return s;
  HostScope hs(c, DBW_KT_HOST_ESTIMATE);
  std::string why;
  double* hT = c->h_T + (size_t)(u % kSlots) * c->cfg.n;
  if (c->cfg.estimator == DBW_ESTIMATOR_NAIVE) {
    const int n = c->cfg.n;
    // the mean of cell (k,k), correctly rounded (sums up to 2^52 convert exactly)
    for (int k = 0; k < n; ++k) {
      const int64_t m = c->cnt[(size_t)k * n + k], sum = c->tsum[(size_t)k * n + k];
      if (sum > (int64_t{1} << 52)) return fail(c, DBW_ESTATE, "time estimate: a cell sum reaches beyond 2^52");
      hT[k] = m > 0 ? static_cast<double>(sum) / static_cast<double>(m) : std::numeric_limits<double>::quiet_NaN();
    }
  } else if (c->solver.solve(c->cfg.n, c->cnt.data(), c->tsum.data(), hT, &why, &c->pending_rows) != 0) {
    return fail(c, DBW_ESTATE, "time estimate: %s", why.c_str());
  }
  c->pending_rows.clear();
  return DBW_OK;
}

void worker_main(dbw_ctx* c) {
  t_in_worker = true;
  (void)hipSetDevice(c->device);
  for (;;) {
    // a job usually follows within one step: spin briefly (a sleeping
    // thread's wake-up costs tens of microseconds), then sleep
    for (int spin = 0; spin < 20000 && c->job_state.load(std::memory_order_acquire) != 1; ++spin)
      __builtin_ia32_pause();
    int64_t u;
    {
      std::unique_lock<std::mutex> lk(c->mu);
      c->cv.wait(lk, [c] { return c->quit || c->job_state.load(std::memory_order_relaxed) == 1; });
      if (c->quit) return;
      u = c->job_u;
    }
    dbw_status st = DBW_ESTATE;
    try {
      st = estimate(c, u);
    } catch (...) {
      c->job_error = "time estimate: out of memory";
    }
    c->job_status = st;
    c->job_state.store(2, std::memory_order_release);
  }
}

void post_estimate(dbw_ctx* c, int64_t u) {
  {
    std::lock_guard<std::mutex> lk(c->mu);
    c->job_u = u;
    c->job_status = DBW_OK;
    c->job_state.store(1, std::memory_order_relaxed);
  }
  c->cv.notify_one();
}

// Wait for the posted job, if any; returns its status.  The wait is short
// (the job only waits for kernels already queued), so it spins.
dbw_status join_estimate(dbw_ctx* c) {
  if (c->job_state.load(std::memory_order_acquire) == 0) return DBW_OK;
  for (int spin = 0; c->job_state.load(std::memory_order_acquire) != 2; ++spin) {
    if (spin < 4096) __builtin_ia32_pause();
    else std::this_thread::yield();
  }
  c->job_state.store(0, std::memory_order_relaxed);
  if (c->job_status != DBW_OK) {
    c->last_error = c->job_error;
    return c->job_status;
  }
  return DBW_OK;
}

dbw_status check_device_ptrs(dbw_ctx* c, std::initializer_list<std::pair<const void*, const char*>> ps) {
  for (auto& p : ps)
    if (!p.first) return fail(c, DBW_EINVAL, "%s is NULL", p.second);
  return DBW_OK;
}

struct ProfScope {
  dbw_ctx* c;
  int g;
  hipStream_t s;
  bool on;
  ProfScope(dbw_ctx* ctx, int group, hipStream_t stream = nullptr)
      : c(ctx), g(group), s(stream ? stream : ctx->stream) {
    ProfileGroup& pg = c->prof[g];
    on = c->prof_events && pg.used < static_cast<int>(pg.start.size());
    if (on) (void)hipEventRecord(pg.start[pg.used], s);
  }
  ~ProfScope() {
    if (on) {
      ProfileGroup& pg = c->prof[g];
      (void)hipEventRecord(pg.stop[pg.used], s);
      pg.used++;
    }
  }
};

dbw_status sync_all(dbw_ctx* c) {
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return DBW_OK;
}

dbw_status launch_grads(dbw_ctx* c, const float* w, const float* X, const int32_t* y, const int32_t* rows,
                        float* G, float* loss, bool keep_slabs = false, const uint8_t* row_mask = nullptr) {
  ProfScope ps(c, DBW_KT_GRADS);
  const dbw_config& cf = c->cfg;
  hipError_t e;
  if (cf.model == DBW_SOFTMAX) {
    dbw::SoftmaxArgs a{};
    a.W = w; a.X = X; a.y = y; a.rows = rows; a.S = cf.S;
    a.n = cf.n; a.B = cf.B; a.d = cf.d; a.C = cf.C;
    a.G = G; a.loss = loss;
    a.Gp = c->Gp; a.lossp = c->lossp; a.Z = c->Z; a.ce = c->ce;
    a.err = c->err;
    a.keep_slabs = keep_slabs ? 1 : 0;
    a.row_mask = row_mask;
    e = dbw::launch_softmax_grads(c->splan, a, c->stream);
  } else if (cf.model == DBW_CNN) {
    dbw::CnnArgs a{};
    a.w = w; a.X = X; a.y = y; a.rows = rows; a.S = cf.S;
    a.n = cf.n; a.B = cf.B; a.H = cf.H; a.C = cf.C;
    a.P = c->P; a.off_c1 = c->P - dbw::CNN_CONV_PARAMS; a.off_c2 = a.off_c1 + dbw::CNN_C1 * 25 + dbw::CNN_C1;
    a.G = G; a.loss = loss;
    a.H1 = c->cH1; a.code1 = c->cCode1; a.F = c->cF; a.code2 = c->cCode2; a.ylab = c->cYlab;
    a.dP2 = c->cdP2; a.dP1 = c->cdP1; a.part1 = c->cPart1; a.part2 = c->cPart2; a.chunk = dbw::kCnnChunk;
    a.Hh = c->Hh; a.dA = c->dA; a.Gp = c->Gp; a.lossp = c->lossp; a.err = c->err; a.row_mask = row_mask;
    e = dbw::launch_cnn_grads(c->mplan, a, c->stream);
  } else {
    dbw::MlpArgs a{};
    a.w = w; a.X = X; a.y = y; a.rows = rows; a.S = cf.S;
    a.n = cf.n; a.B = cf.B; a.d = cf.d; a.H = cf.H; a.C = cf.C;
    a.G = G; a.loss = loss;
    a.Hh = c->Hh; a.dA = c->dA; a.Gp = c->Gp; a.lossp = c->lossp; a.err = c->err; a.row_mask = row_mask;
    e = dbw::launch_mlp_grads(c->mplan, a, c->stream);
  }
  if (e != hipSuccess) return fail(c, DBW_EHIP, "gradient kernels: %s", hipGetErrorString(e));
  return DBW_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

dbw_status check_batch(dbw_ctx* c, const float* X, const int32_t* y, const int32_t* rows) {
  if (!X || !y) return fail(c, DBW_EINVAL, "X and y must be non-NULL");
  if (!aligned16(X)) return fail(c, DBW_EINVAL, "X must be 16-byte aligned");
  if (rows && c->cfg.S <= 0) return fail(c, DBW_EINVAL, "row indices need a dataset: create the context with S > 0");
  return DBW_OK;
}

}  // namespace

// ===========================================================================
DBW_API int64_t dbw_param_count(const dbw_config* cfg) {
  std::string why;
  if (!config_ok(cfg, &why)) return -1;
  return param_count(*cfg);
}

namespace {
thread_local std::string t_free_error = "no error";   // context-free calls of this thread
}  // namespace

dbw_status dbw::set_free_error(dbw_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_free_error = buf;
  return s;
}

DBW_API const char* dbw_last_error(const dbw_ctx* ctx) { return ctx ? ctx->last_error.c_str() : t_free_error.c_str(); }

DBW_API dbw_status dbw_create(const dbw_config* cfg, void* stream, dbw_ctx** out) {
  if (!out) return DBW_EINVAL;
  *out = nullptr;
  std::string why;
  if (!config_ok(cfg, &why)) return DBW_EINVAL;
  {
    // every array a kernel addresses through one buffer resource must stay
    // below 2 GiB
    const int64_t P = param_count(*cfg);
    const int64_t lim = dbw::kMaxBufferBytes;
    if (P * 4 > lim || (int64_t)cfg->n * cfg->B * cfg->d * 4 > lim || cfg->S * cfg->d * 4 > lim ||
        (int64_t)cfg->n * cfg->B * cfg->C * 4 > lim ||
        (cfg->model != DBW_SOFTMAX && (int64_t)cfg->n * cfg->B * cfg->H * 4 > lim) ||
        (cfg->model == DBW_CNN && (int64_t)cfg->n * cfg->B * dbw::CNN_C1 * 144 * 4 > lim))
      return DBW_EUNSUPPORTED;
  }
  dbw_ctx* c = new (std::nothrow) dbw_ctx();
  if (!c) return DBW_EINVAL;
  c->cfg = *cfg;
  c->P = param_count(*cfg);
  c->stream = static_cast<hipStream_t>(stream);
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return DBW_EHIP;
  }
  const dbw_config& cf = c->cfg;
  const int64_t n = cf.n, P = c->P, rowsN = (int64_t)cf.n * cf.B;
  if (cf.model == DBW_SOFTMAX) {
    c->splan = dbw::softmax_plan(cf.n, cf.B, cf.d, cf.C);
  } else {
    // the CNN's fully connected part is the MLP on its 800 features
    c->mplan = dbw::mlp_plan(cf.n, cf.B, cf.model == DBW_CNN ? dbw::CNN_FEAT : cf.d, cf.H, cf.C);
    if (!c->mplan.ok) {
      delete c;
      return DBW_EUNSUPPORTED;
    }
  }
  c->agg_nblocks = dbw::agg_blocks(P);
  if (cf.g_rows != DBW_G_ROWS_ALL && cf.model == DBW_SOFTMAX && c->splan.fused && c->splan.slabs > 1 &&
      c->splan.part % 4 == 0 && dbw::agg_blocks(c->splan.part) <= dbw::kStepPsMaxBlocks) {
    c->slab_src = c->splan.fused == 2 ? dbw::SRC_SLAB_TILES : dbw::SRC_SLABS;
    c->slab_nblocks = dbw::agg_blocks(c->splan.part);
  }
  const int64_t part_blocks = std::max(c->agg_nblocks, c->slab_nblocks);

  // workspace layout
  std::vector<Span> spans;
  size_t total = 0;
  auto take = [&](size_t bytes) {
    Span s;
    s.off = total;
    s.bytes = bytes;
    total += (bytes + 255) / 256 * 256;
    return s;
  };
  Span sG = take(sizeof(float) * n * P), sLoss = take(sizeof(float) * 2 * n), sg = take(sizeof(float) * P),
       sMask = take(n), sSq = take(sizeof(float) * n), sStats = take(sizeof(dbw_iter_stats)),
       sT = take(sizeof(double) * n), sObj = take(sizeof(double) * n), sK = take(4), sB = take(4),
       sSel = take(sizeof(int32_t) * n), sTicks = take(sizeof(int64_t) * n),
       sSt = take(sizeof(dbw_estimator_state)), sErr = take(4),
       sSqp = take(sizeof(float) * n * part_blocks), sPart = take(sizeof(double) * 2 * part_blocks);
  Span sGp, sLp, sZ, sCe, sH, sdA, sH1, sC1, sF, sC2, sYl, sdP2, sdP1, sPa1, sPa2;
  if (cf.model == DBW_SOFTMAX) {
    if (c->splan.fused) {
      if (c->splan.slabs > 1) {
        sGp = take(sizeof(float) * n * c->splan.slabs * c->splan.part);
        sLp = take(sizeof(float) * n * c->splan.slabs);
      }
    } else {
      sZ = take(sizeof(float) * rowsN * cf.C);
      sCe = take(sizeof(float) * rowsN);
    }
  } else {
    sH = take(sizeof(float) * rowsN * cf.H);
    sdA = take(sizeof(float) * rowsN * cf.H);
    sGp = take(sizeof(float) * n * c->mplan.slabs * c->mplan.tail);
    sLp = take(sizeof(float) * n * c->mplan.slabs);
    if (cf.model == DBW_CNN) {
      const int64_t h1 = rowsN * dbw::CNN_C1 * 144, ch = dbw::cnn_chunks(cf.B);
      sH1 = take(sizeof(float) * h1);
      sC1 = take(h1);
      sF = take(sizeof(float) * rowsN * dbw::CNN_FEAT);
      sC2 = take(rowsN * dbw::CNN_FEAT);
      sYl = take(sizeof(int32_t) * rowsN);
      sdP2 = take(sizeof(float) * rowsN * dbw::CNN_FEAT);
      sdP1 = take(sizeof(float) * h1);
      sPa1 = take(sizeof(float) * n * ch * (dbw::CNN_C1 * 25 + dbw::CNN_C1));
      sPa2 = take(sizeof(float) * n * ch * (dbw::CNN_C2 * dbw::CNN_C1 * 25 + dbw::CNN_C2));
    }
  }
  if (hipMalloc(&c->pool, total) != hipSuccess) {
    delete c;
    return DBW_EHIP;
  }
  auto at = [&](const Span& s) -> void* { return s.bytes ? c->pool + s.off : nullptr; };
  c->G = (float*)at(sG); c->loss = (float*)at(sLoss); c->loss_last = c->loss; c->g = (float*)at(sg); c->mask = (uint8_t*)at(sMask);
  c->sqnorm = (float*)at(sSq); c->stats = (dbw_iter_stats*)at(sStats); c->T_hat = (double*)at(sT);
  c->objective = (double*)at(sObj); c->k = (int32_t*)at(sK); c->b = (int32_t*)at(sB);
  c->sel = (int32_t*)at(sSel); c->ticks = (int64_t*)at(sTicks); c->st = (dbw_estimator_state*)at(sSt);
  c->err = (int32_t*)at(sErr); c->sqpart = (float*)at(sSqp); c->part = (double*)at(sPart);
  c->Gp = (float*)at(sGp); c->lossp = (float*)at(sLp);
  c->Z = (float*)at(sZ); c->ce = (float*)at(sCe); c->Hh = (float*)at(sH); c->dA = (float*)at(sdA);
  c->cH1 = (float*)at(sH1); c->cCode1 = (uint8_t*)at(sC1); c->cF = (float*)at(sF); c->cCode2 = (uint8_t*)at(sC2);
  c->cYlab = (int32_t*)at(sYl); c->cdP2 = (float*)at(sdP2); c->cdP1 = (float*)at(sdP1);
  c->cPart1 = (float*)at(sPa1); c->cPart2 = (float*)at(sPa2);

  bool ok = hipMemset(c->pool, 0, total) == hipSuccess;
  const unsigned pin = hipHostMallocMapped | hipHostMallocCoherent;
  ok = ok && hipHostMalloc((void**)&c->h_T, sizeof(double) * kSlots * n, pin) == hipSuccess;
  ok = ok && hipHostMalloc((void**)&c->h_ticks, sizeof(int64_t) * kSlots * n, pin) == hipSuccess;
  ok = ok && hipHostMalloc((void**)&c->h_order, sizeof(int32_t) * kSlots * n, pin) == hipSuccess;
  ok = ok && hipHostMalloc((void**)&c->h_k, sizeof(int32_t) * kSlots, pin) == hipSuccess;
  ok = ok && hipHostGetDevicePointer((void**)&c->d_T, c->h_T, 0) == hipSuccess;
  ok = ok && hipHostGetDevicePointer((void**)&c->d_ticks, c->h_ticks, 0) == hipSuccess;
  ok = ok && hipHostGetDevicePointer((void**)&c->d_order, c->h_order, 0) == hipSuccess;
  ok = ok && hipHostGetDevicePointer((void**)&c->d_k, c->h_k, 0) == hipSuccess;
  if (ok) std::memset(c->h_k, 0, sizeof(int32_t) * kSlots);
  ok = ok && hipHostMalloc((void**)&c->h_err, sizeof(int32_t), hipHostMallocDefault) == hipSuccess;
  ok = ok && hipEventCreateWithFlags(&c->ev_fin, hipEventDisableTiming) == hipSuccess;
  for (int s = 0; s < kSlots && ok; ++s) {
    ok = ok && hipEventCreateWithFlags(&c->ev_k[s], hipEventDisableTiming) == hipSuccess;
  }
  if (!ok) {
    dbw_destroy(c);
    return DBW_EHIP;
  }
  dbw_estimator_state init{};
  init.t = 0;
  init.k_prev = cf.n;
  ok = hipMemcpy(c->st, &init, sizeof init, hipMemcpyHostToDevice) == hipSuccess;
  ok = ok && hipDeviceSynchronize() == hipSuccess;
  if (!ok) {
    dbw_destroy(c);
    return DBW_EHIP;
  }
  c->cnt.assign((size_t)n * n, 0);
  c->tsum.assign((size_t)n * n, 0);
  c->busy.assign(n, 0);
  for (auto& v : c->offs) v.assign(n, 0);
  for (auto& v : c->sorted) v.assign(n, 0);
  c->T_scratch.assign(n, 0.0);
  reset_host_pipeline(c, 0, cf.n);
  try {
    c->worker = std::thread(worker_main, c);
  } catch (...) {
    dbw_destroy(c);
    return DBW_EINVAL;
  }
  *out = c;
  return DBW_OK;
}

DBW_API void dbw_destroy(dbw_ctx* c) {
  if (!c) return;
  DeviceGuard g(c->device);
  if (c->worker.joinable()) {
    (void)join_estimate(c);
    {
      std::lock_guard<std::mutex> lk(c->mu);
      c->quit = true;
    }
    c->cv.notify_one();
    c->worker.join();
  }
  if (c->stream || c->pool) (void)hipStreamSynchronize(c->stream);
  if (c->ev_fin) (void)hipEventDestroy(c->ev_fin);
  for (auto& ev : c->ev_k)
    if (ev) (void)hipEventDestroy(ev);
  for (auto& pg : c->prof) {
    for (auto e : pg.start) (void)hipEventDestroy(e);
    for (auto e : pg.stop) (void)hipEventDestroy(e);
  }
  if (c->h_T) (void)hipHostFree(c->h_T);
  if (c->h_ticks) (void)hipHostFree(c->h_ticks);
  if (c->h_order) (void)hipHostFree(c->h_order);
  if (c->h_k) (void)hipHostFree(c->h_k);
  if (c->h_err) (void)hipHostFree(c->h_err);
  if (c->pool) (void)hipFree(c->pool);
  delete c;
}

DBW_API dbw_status dbw_sync(dbw_ctx* c) {
  if (!c) return DBW_EINVAL;
  DeviceGuard g(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  HIP_TRY(c, hipMemcpy(c->h_err, c->err, sizeof(int32_t), hipMemcpyDeviceToHost));
  const int32_t e = *c->h_err;
  if (e) {
    *c->h_err = 0;
    HIP_TRY(c, hipMemcpy(c->err, c->h_err, sizeof(int32_t), hipMemcpyHostToDevice));
    std::string msg = "device reported:";
    if (e & dbw::ERR_ROW_RANGE) msg += " row index outside [0, S);";
    if (e & dbw::ERR_K_RANGE) msg += " k exceeds the workers that arrive;";
    if (e & dbw::ERR_LABEL_RANGE) msg += " label outside [0, C);";
    if (e & dbw::ERR_MASK_COUNT) msg += " mask does not hold k ones;";
    return fail(c, (e & (dbw::ERR_LABEL_RANGE | dbw::ERR_MASK_COUNT)) && !(e & (dbw::ERR_ROW_RANGE | dbw::ERR_K_RANGE))
                       ? DBW_EINVAL : DBW_ERANGE, "%s", msg.c_str());
  }
  return DBW_OK;
}

DBW_API dbw_status dbw_worker_grads(dbw_ctx* c, const float* w, const float* X, const int32_t* y,
                                    const int32_t* rows, float* G, float* loss) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = check_device_ptrs(c, {{w, "w"}, {G, "G"}, {loss, "loss"}}); s != DBW_OK) return s;
  if (!aligned16(w) || !aligned16(G)) return fail(c, DBW_EINVAL, "w and G must be 16-byte aligned");
  if (dbw_status s = check_batch(c, X, y, rows); s != DBW_OK) return s;
  DeviceGuard g(c->device);
  return launch_grads(c, w, X, y, rows, G, loss);
}

DBW_API dbw_status dbw_aggregate_fastest(dbw_ctx* c, const float* G, const int64_t* ticks, int32_t k, float* g,
                                         uint8_t* mask) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = check_device_ptrs(c, {{G, "G"}, {ticks, "ticks"}, {g, "g"}, {mask, "mask"}}); s != DBW_OK)
    return s;
  if (k < 1 || k > c->cfg.n) return fail(c, DBW_ERANGE, "k=%d outside [1, %d]", k, c->cfg.n);
  DeviceGuard dg(c->device);
  ProfScope ps(c, DBW_KT_AGGREGATE);
  // one launch: every aggregation block ranks the n ticks itself and block 0
  // writes the mask
  dbw::AggArgs aa{};
  aa.G = G; aa.P = c->P; aa.n = c->cfg.n; aa.ticks_sel = ticks; aa.mask_out = mask; aa.err = c->err;
  aa.k_imm = k; aa.g_out = g; aa.sqpart = c->sqpart; aa.part = c->part; aa.mode = dbw::AGG_MEAN;
  HIP_TRY(c, dbw::launch_aggregate(aa, c->stream));
  return DBW_OK;
}

DBW_API dbw_status dbw_grad_stats(dbw_ctx* c, const float* G, const uint8_t* mask, int32_t k, const float* g,
                                  const float* loss, float* sqnorm, dbw_iter_stats* stats) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = check_device_ptrs(
          c, {{G, "G"}, {mask, "mask"}, {g, "g"}, {loss, "loss"}, {sqnorm, "sqnorm"}, {stats, "stats"}});
      s != DBW_OK)
    return s;
  if (k < 1 || k > c->cfg.n) return fail(c, DBW_ERANGE, "k=%d outside [1, %d]", k, c->cfg.n);
  DeviceGuard dg(c->device);
  ProfScope ps(c, DBW_KT_AGGREGATE);
  dbw::AggArgs aa{};
  aa.G = G; aa.P = c->P; aa.n = c->cfg.n; aa.sel_mask = mask; aa.k_imm = k; aa.g_in = g;
  aa.sqpart = c->sqpart; aa.part = c->part; aa.mode = dbw::AGG_STATS_GIVEN_MEAN;
  HIP_TRY(c, dbw::launch_aggregate(aa, c->stream));
  dbw::FinalizeArgs fa{};
  fa.sqpart = c->sqpart; fa.part = c->part; fa.nblocks = c->agg_nblocks; fa.mask = mask; fa.k_imm = k;
  fa.loss = loss; fa.n = c->cfg.n; fa.sqnorm = sqnorm; fa.stats = stats; fa.st = c->st;
  fa.eta = c->cfg.eta; fa.D = c->cfg.D; fa.bookkeeping = 0; fa.err = c->err;
  HIP_TRY(c, dbw::launch_finalize(fa, c->stream));
  return DBW_OK;
}

DBW_API dbw_status dbw_choose_b(dbw_ctx* c, const double* T_hat, int32_t* k_out, int32_t* b_out,
                                double* objective) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = check_device_ptrs(c, {{T_hat, "T_hat"}, {k_out, "k_out"}, {b_out, "b_out"}}); s != DBW_OK)
    return s;
  DeviceGuard dg(c->device);
  ProfScope ps(c, DBW_KT_CHOOSE);
  dbw::ChooseArgs ca{};
  ca.st = c->st; ca.T_src = T_hat; ca.n = c->cfg.n; ca.eta = c->cfg.eta; ca.beta = c->cfg.beta;
  ca.policy = c->cfg.policy; ca.k_static = c->cfg.k_static;
  ca.do_choose = 1; ca.do_select = 0; ca.k_out = k_out; ca.b_out = b_out; ca.objective = objective;
  ca.err = c->err;
  HIP_TRY(c, dbw::launch_choose_select(ca, c->stream));
  return DBW_OK;
}

DBW_API dbw_status dbw_step(dbw_ctx* c, float* w, const float* X, const int32_t* y, const int32_t* rows,
                            const int64_t* ticks_host, int32_t* k_host) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = check_device_ptrs(c, {{w, "w"}}); s != DBW_OK) return s;
  if (!aligned16(w)) return fail(c, DBW_EINVAL, "w must be 16-byte aligned");
  if (dbw_status s = check_batch(c, X, y, rows); s != DBW_OK) return s;
  if (!ticks_host) return fail(c, DBW_EINVAL, "ticks_host is NULL");
  const int n = c->cfg.n;
  for (int i = 0; i < n; ++i)
    if (ticks_host[i] < 0) return fail(c, DBW_EINVAL, "tick of worker %d is negative", i);
  DeviceGuard dg(c->device);
  HostScope hs_step(c, DBW_KT_HOST_STEP);
  const int64_t t = c->t;
  const int slot = static_cast<int>(t % kSlots);
  // loss alternates halves by step parity (the statistics of step t-1 may
  // still read the other half)
  float* loss = c->loss + (size_t)(t & 1) * n;
  //    With a slab source the partials stay for the PS kernel.
  const bool slab = c->slab_src != 0;
  // Rows of G that nothing reads are skipped where the softmax gradients
  // come from per-worker GEMM tiles (no slab source) and the choice is a
  // kernel of its own: the choice and the selection then run first, and the
  // gradient kernels store only the selected workers' rows (every gradient
  // is still computed).  Otherwise the gradients go first: they need neither
  // the time estimate nor the choice, and keep the GPU busy while the host
  // waits for T_hat_t.  (The MLP and CNN kernels take the same row mask, but
  // on their workloads the earlier choice cost more than the skipped rows
  // saved, so their steps keep the gradients-first order.)
  const bool mask_first = c->cfg.g_rows != DBW_G_ROWS_ALL && !slab && c->agg_nblocks > dbw::kStepPsMaxBlocks &&
                          (c->cfg.model == DBW_SOFTMAX || c->cfg.g_rows == DBW_G_ROWS_SELECTED);
  // 0. worker gradients first (see above)
  if (!mask_first)
    if (dbw_status s = launch_grads(c, w, X, y, rows, c->G, loss, slab); s != DBW_OK) return s;
  // 1. T_hat_t in the pinned slot: solved by the worker since k_{t-2} became
  //    known, or here when no job was posted (first step of a history)
  {
    HostScope hw(c, DBW_KT_HOST_WAIT);
    const bool posted = c->job_state.load(std::memory_order_acquire) != 0;
    if (dbw_status s = posted ? join_estimate(c) : estimate(c, t); s != DBW_OK) return s;
  }
  HostScope hq(c, DBW_KT_HOST_QUEUE);
  // 2. this iteration's arrival offsets and order (workers by (offset,
  //    index)) into the pinned slot (its previous reader, the PS kernel of
  //    t-4, precedes the one of t-2 the estimate waited for).  Under Push &
  //    Wait the estimate just joined has folded iteration t-1, so the clock
  //    and the busy times are those at the start of iteration t.
  int64_t* hk = c->h_ticks + (size_t)slot * n;
  std::vector<int64_t>& off = c->offs[slot];
  if (c->cfg.clock == DBW_CLOCK_PSW) {
    if (c->recorded != t) return fail(c, DBW_ESTATE, "iteration %lld not folded before its offsets", (long long)t);
    for (int i = 0; i < n; ++i) {
      const int64_t wait = std::max<int64_t>(c->busy[i], c->clock) - c->clock;
      if (ticks_host[i] >= (int64_t{1} << 48) - wait)
        return fail(c, DBW_ERANGE, "arrival offset of worker %d reaches 2^48", i);
      off[i] = wait + ticks_host[i];
    }
  } else {
    std::memcpy(off.data(), ticks_host, sizeof(int64_t) * n);
  }
  std::memcpy(hk, off.data(), sizeof(int64_t) * n);
  int32_t* ho = c->h_order + (size_t)slot * n;
  for (int i = 0; i < n; ++i) ho[i] = i;
  std::stable_sort(ho, ho + n, [&](int32_t a, int32_t b) { return off[a] < off[b]; });
  std::vector<int64_t>& srt = c->sorted[slot];
  srt.resize(n);
  for (int r = 0; r < n; ++r) srt[r] = off[ho[r]];
  // 3. one PS kernel: the choice of k_t (T_hat read from the pinned slot, k_t
  //    written back into it), the first k_t arrivals, the aggregate and the
  //    update; then the statistics and the estimator bookkeeping (all on the
  //    context stream: the gradient kernel fills every CU, so nothing would
  //    run beside it)
  {
    // with the choice first, its kernel is timed apart from the aggregation
    std::optional<ProfScope> ps;
    ps.emplace(c, mask_first ? DBW_KT_CHOOSE : DBW_KT_AGGREGATE);
    // k_t's pinned slot reads 0 until the PS kernel writes k_t (its previous
    // value, k_{t-4}, was read before the estimate of t-2)
    __atomic_store_n(c->h_k + slot, 0, __ATOMIC_RELEASE);
    dbw::ChooseArgs ca{};
    ca.st = c->st; ca.T_src = c->d_T + (size_t)slot * n; ca.ticks_src = c->d_ticks + (size_t)slot * n;
    ca.order_src = c->d_order + (size_t)slot * n;
    ca.T_hat = c->T_hat; ca.ticks = c->ticks; ca.k_host = c->d_k + slot; ca.n = n; ca.eta = c->cfg.eta;
    ca.beta = c->cfg.beta; ca.policy = c->cfg.policy; ca.k_static = c->cfg.k_static;
    ca.do_choose = 1; ca.do_select = 1; ca.k_out = c->k; ca.b_out = c->b;
    ca.objective = c->objective; ca.sel = c->sel; ca.mask = c->mask; ca.err = c->err;
    dbw::AggArgs aa{};
    aa.G = c->G; aa.P = c->P; aa.n = n; aa.sel = c->sel; aa.k_dev = c->k; aa.g_out = c->g; aa.w = w;
    aa.eta = static_cast<float>(c->cfg.eta); aa.sqpart = c->sqpart; aa.part = c->part; aa.mode = dbw::AGG_FUSED;
    if (slab) {
      aa.src = c->slab_src; aa.Gp = c->Gp; aa.slabs = c->splan.slabs; aa.slab_len = c->splan.part;
      aa.d = c->cfg.d; aa.C = c->cfg.C; aa.B = c->cfg.B; aa.lossp = c->lossp; aa.loss = loss;
      aa.G_rows = c->cfg.g_rows == DBW_G_ROWS_SELECTED ? c->G : nullptr;
    }
    // every block of the fused kernel repeats the choice; beyond about two
    // blocks per CU the separate choice kernel is cheaper (the slab source
    // is only taken within that bound)
    const bool fused = slab || c->agg_nblocks <= dbw::kStepPsMaxBlocks;
    if (fused) {
      // small n: T_hat_t, the ticks and the order travel in the kernel
      // arguments
      dbw::StepInline inl;
      inl.n_inline = 0;
      if (n <= dbw::kInlineN) {
        std::memcpy(inl.T, c->h_T + (size_t)slot * n, sizeof(double) * n);
        std::memcpy(inl.ticks, hk, sizeof(int64_t) * n);
        std::memcpy(inl.order, ho, sizeof(int32_t) * n);
        inl.n_inline = n;
      }
      HIP_TRY(c, dbw::launch_step_ps(ca, aa, inl, c->stream));
    } else {
      HIP_TRY(c, dbw::launch_choose_select(ca, c->stream));
    }
    if (mask_first) {
      // the selection is on the device: gradients with only the selected
      // rows stored
      ps.reset();
      if (dbw_status s = launch_grads(c, w, X, y, rows, c->G, loss, false, c->mask); s != DBW_OK) return s;
      ps.emplace(c, DBW_KT_AGGREGATE);
    }
    if (!fused) HIP_TRY(c, dbw::launch_aggregate(aa, c->stream));
    // T_hat_{t+1} on the worker now (it needs this iteration's ticks, stored
    // above, and k_{t-1}); the rest of the queueing overlaps its solve
    c->t = t + 1;
    post_estimate(c, t + 1);
    dbw::FinalizeArgs fa{};
    fa.sqpart = c->sqpart; fa.part = c->part; fa.nblocks = slab ? c->slab_nblocks : c->agg_nblocks;
    fa.mask = c->mask; fa.k_dev = c->k;
    fa.loss = loss; fa.n = n; fa.sqnorm = c->sqnorm; fa.stats = c->stats; fa.st = c->st;
    fa.eta = c->cfg.eta; fa.D = c->cfg.D; fa.bookkeeping = 1; fa.err = c->err;
    HIP_TRY(c, dbw::launch_finalize(fa, c->stream));
  }
  c->loss_last = loss;
  if (k_host) {
    HIP_TRY(c, hipEventRecord(c->ev_fin, c->stream));
    HIP_TRY(c, hipEventSynchronize(c->ev_fin));
    *k_host = c->h_k[slot];
  }
  return DBW_OK;
}

DBW_API dbw_status dbw_step_outputs(dbw_ctx* c, dbw_step_buffers* out) {
  if (!c || !out) return DBW_EINVAL;
  DeviceGuard dg(c->device);
  out->G = c->G; out->loss = c->loss_last; out->g = c->g; out->mask = c->mask; out->sqnorm = c->sqnorm;
  out->stats = c->stats; out->T_hat = c->T_hat; out->objective = c->objective; out->k = c->k; out->b = c->b;
  return DBW_OK;
}

DBW_API dbw_status dbw_time_estimate(int32_t n, const int64_t* cnt, const int64_t* tsum, double* T_hat) {
  if (!cnt || !tsum || !T_hat) return DBW_EINVAL;
  std::string why;
  return dbw::time_estimate(n, cnt, tsum, T_hat, &why) == 0 ? DBW_OK : DBW_EINVAL;
}

struct dbw_time_estimator {
  dbw::IsoSolver solver;
};

DBW_API dbw_status dbw_time_estimator_create(dbw_time_estimator** out) {
  if (!out) return DBW_EINVAL;
  *out = new (std::nothrow) dbw_time_estimator();
  return *out ? DBW_OK : DBW_EINVAL;
}

DBW_API void dbw_time_estimator_destroy(dbw_time_estimator* est) { delete est; }

DBW_API dbw_status dbw_time_estimator_solve(dbw_time_estimator* est, int32_t n, const int64_t* cnt,
                                            const int64_t* tsum, double* T_hat) {
  if (!est || !cnt || !tsum || !T_hat) return DBW_EINVAL;
  std::string why;
  return est->solver.solve(n, cnt, tsum, T_hat, &why) == 0 ? DBW_OK : DBW_EINVAL;
}

DBW_API dbw_status dbw_time_estimator_stats(const dbw_time_estimator* est, int64_t* fast, int64_t* warm,
                                            int64_t* full) {
  if (!est) return DBW_EINVAL;
  if (fast) *fast = est->solver.fast_solves();
  if (warm) *warm = est->solver.warm_solves();
  if (full) *full = est->solver.full_solves();
  return DBW_OK;
}

DBW_API dbw_status dbw_state_export(dbw_ctx* c, dbw_estimator_state* out) {
  if (!c || !out) return DBW_EINVAL;
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  HIP_TRY(c, hipMemcpy(out, c->st, sizeof *out, hipMemcpyDeviceToHost));
  return DBW_OK;
}

DBW_API dbw_status dbw_state_import(dbw_ctx* c, const dbw_estimator_state* in) {
  if (!c || !in) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  const dbw_config& cf = c->cfg;
  if (in->t < 0 || in->k_prev < 1 || in->k_prev > cf.n || in->nV < 0 || in->nV > cf.D || in->nL < 0 ||
      in->nL > cf.D || in->nF < 0 || in->nF > 2)
    return fail(c, DBW_EINVAL, "estimator state out of range for this configuration");
  if ((in->t == 0) != (in->nV == 0) || in->nF > in->t || in->nV > in->t)
    return fail(c, DBW_EINVAL, "estimator state histories do not match t");
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  // fold what is known before the history restarts
  if (dbw_status s = fold(c, c->t, c->t); s != DBW_OK) return s;
  HIP_TRY(c, hipMemcpy(c->st, in, sizeof *in, hipMemcpyHostToDevice));
  reset_host_pipeline(c, in->t, in->k_prev);
  return DBW_OK;
}

DBW_API dbw_status dbw_samples_export(dbw_ctx* c, int64_t* cnt, int64_t* tsum, int64_t* clock) {
  if (!c || !cnt || !tsum || !clock) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  if (dbw_status s = fold(c, c->t, c->t); s != DBW_OK) return s;
  std::memcpy(cnt, c->cnt.data(), sizeof(int64_t) * c->cnt.size());
  std::memcpy(tsum, c->tsum.data(), sizeof(int64_t) * c->tsum.size());
  *clock = c->clock;
  return DBW_OK;
}

DBW_API dbw_status dbw_samples_import(dbw_ctx* c, const int64_t* cnt, const int64_t* tsum, int64_t clock) {
  if (!c || !cnt || !tsum) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  const int n = c->cfg.n;
  std::vector<double> probe(n);
  std::string why;
  if (dbw::time_estimate(n, cnt, tsum, probe.data(), &why) != 0)
    return fail(c, DBW_EINVAL, "samples: %s", why.c_str());
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  if (dbw_status s = fold(c, c->t, c->t); s != DBW_OK) return s;
  std::memcpy(c->cnt.data(), cnt, sizeof(int64_t) * c->cnt.size());
  std::memcpy(c->tsum.data(), tsum, sizeof(int64_t) * c->tsum.size());
  c->clock = clock;
  std::fill(c->busy.begin(), c->busy.end(), clock);
  c->solver.reset();
  return DBW_OK;
}

DBW_API dbw_status dbw_busy_export(dbw_ctx* c, int64_t* busy) {
  if (!c || !busy) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  if (dbw_status s = fold(c, c->t, c->t); s != DBW_OK) return s;
  std::memcpy(busy, c->busy.data(), sizeof(int64_t) * c->busy.size());
  return DBW_OK;
}

DBW_API dbw_status dbw_busy_import(dbw_ctx* c, const int64_t* busy) {
  if (!c || !busy) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  for (int i = 0; i < c->cfg.n; ++i)
    if (busy[i] < 0) return fail(c, DBW_EINVAL, "busy time of worker %d is negative", i);
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  if (dbw_status s = fold(c, c->t, c->t); s != DBW_OK) return s;
  std::memcpy(c->busy.data(), busy, sizeof(int64_t) * c->busy.size());
  return DBW_OK;
}

DBW_API dbw_status dbw_profile_enable(dbw_ctx* c, int32_t mode) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  DeviceGuard dg(c->device);
  if (mode < 0 || mode > 2) return fail(c, DBW_EINVAL, "profile mode must be 0, 1 or 2");
  if (mode == 1) {
    for (int g = 0; g < DBW_KT_HOST_ESTIMATE; ++g)
      for (auto& pg = c->prof[g]; static_cast<int>(pg.start.size()) < kProfilePairs;) {
        hipEvent_t a, b;
        HIP_TRY(c, hipEventCreate(&a));
        HIP_TRY(c, hipEventCreate(&b));
        pg.start.push_back(a);
        pg.stop.push_back(b);
      }
  }
  c->profiling = mode != 0;
  c->prof_events = mode == 1;
  return DBW_OK;
}

DBW_API dbw_status dbw_kernel_time(dbw_ctx* c, int32_t group, double* total_ms, int64_t* launches) {
  if (!c || !total_ms || !launches || group < 0 || group >= DBW_KT_COUNT) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  ProfileGroup& pg = c->prof[group];
  for (int i = 0; i < pg.used; ++i) {
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, pg.start[i], pg.stop[i]));
    pg.done_ms += ms;
  }
  pg.done_launches += pg.used;
  pg.used = 0;
  *total_ms = pg.done_ms;
  *launches = pg.done_launches;
  return DBW_OK;
}

DBW_API dbw_status dbw_profile_reset(dbw_ctx* c) {
  if (!c) return DBW_EINVAL;
  if (dbw_status s = join_estimate(c); s != DBW_OK) return s;
  DeviceGuard dg(c->device);
  if (dbw_status s = sync_all(c); s != DBW_OK) return s;
  for (auto& pg : c->prof) {
    pg.used = 0;
    pg.done_ms = 0.0;
    pg.done_launches = 0;
  }
  return DBW_OK;
}
