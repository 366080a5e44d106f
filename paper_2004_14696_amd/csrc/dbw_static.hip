// dbw_grad_stats_static: the statistics of dbw_grad_stats without a context
// and without allocating, for callers that cannot allocate device memory.
//
// The kernels are those of dbw_grad_stats (mask to list, one pass over the
// selected rows against the given mean, fixed-order finish).  Their scratch
// -- the selection list, the per-row and per-tile partial sums -- lives in
// one file-scope device array per GPU, whose address is looked up once per
// device with hipGetSymbolAddress and used from then on (the array's name is
// a host-side stand-in in host code, not a device address).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <mutex>

#include "dbw.h"
#include "dbw_internal.h"

#define DBW_API extern "C" __attribute__((visibility("default")))

namespace {

static __device__ __align__(256) unsigned char scratch[DBW_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};     // per device: the address of its copy of `scratch`

// The current device's copy of the scratch array (looked up on first use).
hipError_t scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

constexpr size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Scratch bytes of one call: the per-row partial squared norms [n][tiles]
// and the per-tile partial sums [tiles][2].
size_t scratch_bytes(int32_t n, int64_t P) {
  const size_t tiles = static_cast<size_t>(dbw::agg_blocks(P));
  return align256(sizeof(float) * n * tiles) + align256(2 * sizeof(double) * tiles);
}

}  // namespace

DBW_API dbw_status dbw_grad_stats_static(int32_t n, int64_t P, const float* G, const uint8_t* mask, int32_t k,
                                         const float* g, const float* loss, double V_window, float* sqnorm,
                                         dbw_iter_stats* stats, void* stream) {
  using dbw::set_free_error;
  if (n < 1 || n > DBW_MAX_N || P < 1)
    return set_free_error(DBW_EINVAL, "dbw_grad_stats_static: n=%d outside [1, %d] or P=%lld < 1", n, DBW_MAX_N,
                          (long long)P);
  if (!G || !mask || !g || !loss || !sqnorm || !stats)
    return set_free_error(DBW_EINVAL, "dbw_grad_stats_static: a device pointer is NULL");
  if (k < 1 || k > n) return set_free_error(DBW_ERANGE, "dbw_grad_stats_static: k=%d outside [1, %d]", k, n);
  if (!std::isfinite(V_window)) return set_free_error(DBW_EINVAL, "dbw_grad_stats_static: V_window is not finite");
  if (P > (int64_t{1} << 29))
    return set_free_error(DBW_EUNSUPPORTED, "dbw_grad_stats_static: P=%lld: a row must stay below 2 GiB",
                          (long long)P);
  const size_t need = scratch_bytes(n, P);
  if (need > DBW_STATIC_SCRATCH_BYTES)
    return set_free_error(DBW_EUNSUPPORTED,
                          "dbw_grad_stats_static: n=%d, P=%lld need %zu bytes of scratch, above the %u-byte maximum",
                          n, (long long)P, need, static_cast<unsigned>(DBW_STATIC_SCRATCH_BYTES));
  void* base = nullptr;
  if (hipError_t e = scratch_on_current_device(&base); e != hipSuccess)
    return set_free_error(DBW_EHIP, "dbw_grad_stats_static: address of the scratch array: %s", hipGetErrorString(e));
  const int64_t tiles = dbw::agg_blocks(P);
  unsigned char* p = static_cast<unsigned char*>(base);
  float* sqpart = reinterpret_cast<float*>(p);
  double* part = reinterpret_cast<double*>(p + align256(sizeof(float) * n * tiles));
  hipStream_t s = static_cast<hipStream_t>(stream);
  // every scratch value a kernel reads was written earlier in this call:
  // nothing needs clearing
  dbw::AggArgs aa{};
  aa.G = G; aa.P = P; aa.n = n; aa.sel_mask = mask; aa.k_imm = k; aa.g_in = g;
  aa.sqpart = sqpart; aa.part = part; aa.mode = dbw::AGG_STATS_GIVEN_MEAN;
  if (dbw::launch_aggregate(aa, s) != hipSuccess)
    return set_free_error(DBW_EHIP, "dbw_grad_stats_static: launch failed");
  dbw::FinalizeArgs fa{};
  fa.sqpart = sqpart; fa.part = part; fa.nblocks = tiles; fa.mask = mask; fa.k_imm = k;
  fa.loss = loss; fa.n = n; fa.sqnorm = sqnorm; fa.stats = stats; fa.st = nullptr;
  fa.bookkeeping = 0; fa.v_window_given = 1; fa.v_window = V_window; fa.err = nullptr;
  if (dbw::launch_finalize(fa, s) != hipSuccess)
    return set_free_error(DBW_EHIP, "dbw_grad_stats_static: launch failed");
  return DBW_OK;
}
