// Parameter-server kernels of the DBW iteration (gfx950).
//
//  k_choose_select  one block: the DBW choice of k (Sect. 3.3, Eqs. gain,
//                   greedy, greedy2) from the device estimator state, then the
//                   fastest-k selection (Sect. 2, Eq. grad_bw) by rank of
//                   (tick, worker index).
//  k_aggregate      streams the k selected gradient rows once: mean g_t
//                   (Eq. grad_bw), per-column sums of squared deviations for
//                   the variance estimate (Eq. sumvariancekt), per-row squared
//                   norms, and optionally the SGD update (Eq. update).
//  k_finalize       reduces the per-block partials in a fixed order: the
//                   iteration statistics (Eqs. sumvariancekt, normsquarekt,
//                   loss estimate), per-worker squared norms, and the
//                   estimator-state push of Eq. estimateL and the D windows.
//
// All reductions run in a fixed order, so results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dbw_buffer.h"
#include "dbw_internal.h"

namespace dbw {
namespace {

constexpr int WAVE = 64;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

// Fixed-order block sum of doubles (blockDim.x == 256); result in all threads.
__device__ double block_sum_256(double v, double* sh /*[4]*/) {
  v = wave_sum_d(v);
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  double r = ((sh[0] + sh[1]) + sh[2]) + sh[3];
  __syncthreads();
  return r;
}

// Cooperative copy of the estimator state into LDS (whole 4-byte words).
__device__ __forceinline__ void load_state(const dbw_estimator_state* g, dbw_estimator_state* sh) {
  const uint32_t* src = reinterpret_cast<const uint32_t*>(g);
  uint32_t* dst = reinterpret_cast<uint32_t*>(sh);
  constexpr int W = sizeof(dbw_estimator_state) / 4;
  for (int i = threadIdx.x; i < W; i += blockDim.x) dst[i] = src[i];
}

__device__ __forceinline__ void store_state(const dbw_estimator_state* sh, dbw_estimator_state* g) {
  const uint32_t* src = reinterpret_cast<const uint32_t*>(sh);
  uint32_t* dst = reinterpret_cast<uint32_t*>(g);
  constexpr int W = sizeof(dbw_estimator_state) / 4;
  for (int i = threadIdx.x; i < W; i += blockDim.x) dst[i] = src[i];
}

// (objective, k) of the better choice: larger objective, then larger k.
__device__ __forceinline__ void better(double& r, int& k, double r2, int k2) {
  if (k2 != 0 && (k == 0 || r2 > r || (r2 == r && k2 > k))) {
    r = r2;
    k = k2;
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_choose_select(ChooseArgs a) {
#pragma clang fp contract(off)
  __shared__ dbw_estimator_state st;
  __shared__ double sh_T[DBW_MAX_N];
  __shared__ long long sh_t[DBW_MAX_N];
  __shared__ double sh_r[4], sh_g[4], sh_win[3];
  __shared__ int sh_k[4], sh_cnt[4];
  __shared__ int sh_kfinal;
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int n = a.n;

  // stage the inputs (T_hat and ticks may live in pinned host memory)
  if (a.do_choose) {
    load_state(a.st, &st);
    for (int k = tid; k < n; k += blockDim.x) {
      const double T = a.T_src[k];
      sh_T[k] = T;
      if (a.T_hat) a.T_hat[k] = T;
    }
  }
  if (a.do_select) {
    for (int i = tid; i < n; i += blockDim.x) {
      const long long t = a.ticks_src[i];
      sh_t[i] = t;
      if (a.ticks) a.ticks[i] = t;
    }
  }
  __syncthreads();

  if (a.do_choose) {
    // D-window means (oldest first, summed in order as the definition reads)
    if (tid == 0) {
      double V = 0.0, N = 0.0, L = 0.0;
      for (int i = 0; i < st.nV; ++i) V += st.hV[i];
      for (int i = 0; i < st.nV; ++i) N += st.hN[i];
      for (int i = 0; i < st.nL; ++i) L += st.hL[i];
      sh_win[0] = st.nV > 0 ? V / st.nV : 0.0;
      sh_win[1] = st.nV > 0 ? N / st.nV : 0.0;
      sh_win[2] = st.nL > 0 ? L / st.nL : 0.0;
    }
    __syncthreads();
    const bool hasL = st.nL > 0;
    const double V = sh_win[0], N = sh_win[1], L = sh_win[2];
    const double ga = a.eta - L * a.eta * a.eta / 2.0;
    const double gb = L * a.eta * a.eta / 2.0;
    double best_r = -INFINITY;
    int best_k = 0;
    double maxG = -INFINITY;
    for (int k = tid + 1; k <= n; k += blockDim.x) {
      const double Gk = ga * N - gb * V / k;
      const double T = sh_T[k - 1];
      const bool eligible = isfinite(T) && T > 0.0;
      const double r = eligible ? Gk / T : NAN;
      if (a.objective) a.objective[k - 1] = hasL ? r : NAN;
      maxG = fmax(maxG, Gk);
      if (eligible) better(best_r, best_k, r, k);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      better(best_r, best_k, __shfl_xor(best_r, o, WAVE), __shfl_xor(best_k, o, WAVE));
      maxG = fmax(maxG, __shfl_xor(maxG, o, WAVE));
    }
    if (lane == 0) {
      sh_r[wv] = best_r;
      sh_k[wv] = best_k;
      sh_g[wv] = maxG;
    }
    __syncthreads();
    if (tid == 0) {
      double r = sh_r[0], g = sh_g[0];
      int kb = sh_k[0];
      for (int w = 1; w < 4; ++w) {
        better(r, kb, sh_r[w], sh_k[w]);
        g = fmax(g, sh_g[w]);
      }
      int k = (!hasL || kb == 0 || g < 0.0) ? n : kb;
      // loss guard: never decrease k while the loss estimate rises
      if (st.nF >= 2 && st.F_prev > a.beta * st.F_prev2 && st.k_prev < n) k = max(k, st.k_prev + 1);
      a.k_out[0] = k;
      a.b_out[0] = n - k;
      if (a.k_host) *a.k_host = k;
      sh_kfinal = k;
    }
  } else if (tid == 0) {
    sh_kfinal = a.k_imm;
  }
  __syncthreads();

  if (a.do_select) {
    const int k = sh_kfinal;
    int finite = 0;
    for (int i = tid; i < n; i += blockDim.x) {
      const long long ti = sh_t[i];
      int rank = 0;
      for (int j = 0; j < n; ++j) {
        const long long tj = sh_t[j];
        rank += (tj < ti) || (tj == ti && j < i);
      }
      const bool on = rank < k;
      a.mask[i] = on ? 1 : 0;
      if (on) a.sel[rank] = i;
      finite += ti < INT64_MAX;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) finite += __shfl_xor(finite, o, WAVE);
    if (lane == 0) sh_cnt[wv] = finite;
    __syncthreads();
    if (tid == 0 && k > sh_cnt[0] + sh_cnt[1] + sh_cnt[2] + sh_cnt[3]) atomicOr(a.err, ERR_K_RANGE);
  }
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_mask_to_sel(const uint8_t* mask, int n, int k, int32_t* sel,
                                                     int32_t* err) {
  if (threadIdx.x != 0) return;
  int c = 0;
  for (int j = 0; j < n; ++j)
    if (mask[j]) {
      if (c < n) sel[c] = j;
      ++c;
    }
  if (c != k) atomicOr(err, ERR_MASK_COUNT);
}

// ---------------------------------------------------------------------------
// Column tile: 256 columns.  VEC4: lane owns 4 consecutive columns (16-byte
// loads; needs P % 4 == 0).  Otherwise lane owns columns lane + 64 q.
template <bool VEC4>
__device__ __forceinline__ void load_tile(const float* __restrict__ row, int64_t base, int lane,
                                          int64_t P, float v[4], bool valid = true) {
  // columns >= P (and every column of an invalid row) read as 0
  const __amdgpu_buffer_rsrc_t r = make_rsrc(row, valid ? static_cast<uint32_t>(P * 4) : 0u);
  if (VEC4) {
    const float4 q = buf_f32x4(r, static_cast<uint32_t>((base + lane * 4) * 4));
    v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = buf_f32(r, static_cast<uint32_t>((base + lane + WAVE * q) * 4));
  }
}

template <bool VEC4>
__device__ __forceinline__ int col_index(int lane, int q) {
  return VEC4 ? lane * 4 + q : lane + WAVE * q;
}

template <bool VEC4, int MODE>
__global__ __launch_bounds__(AGG_WAVES * WAVE) void k_aggregate(AggArgs a) {
  __shared__ float sh_s1[AGG_WAVES][AGG_TILE];
  __shared__ float sh_s2[AGG_WAVES][AGG_TILE];
  __shared__ float sh_c[AGG_TILE];
  __shared__ double sh_red[4];
  const int tid = threadIdx.x;
  const int lane = tid % WAVE, wv = tid / WAVE;
  const int64_t P = a.P;
  const int64_t blk = blockIdx.x;
  const int64_t nblocks = gridDim.x;
  const int64_t base = blk * AGG_TILE;
  const int k = a.k_dev ? a.k_dev[0] : a.k_imm;

  // shift: the mean itself (given) or the fastest worker's row
  float c[4];
  if (MODE == AGG_STATS_GIVEN_MEAN) load_tile<VEC4>(a.g_in, base, lane, P, c);
  else load_tile<VEC4>(a.G + (int64_t)__builtin_amdgcn_readfirstlane(a.sel[0]) * P, base, lane, P, c);

  float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f};
  constexpr int U = 4;   // rows in flight per wave
  for (int r0 = wv; r0 < k; r0 += AGG_WAVES * U) {
    float x[U][4];
    int jj[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = r0 + u * AGG_WAVES;
      jj[u] = r < k ? __builtin_amdgcn_readfirstlane(a.sel[r]) : -1;   // uniform per wave
      load_tile<VEC4>(a.G + (int64_t)(jj[u] < 0 ? 0 : jj[u]) * P, base, lane, P, x[u], jj[u] >= 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (jj[u] < 0) break;
      float sq = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float dv = x[u][q] - c[q];
        s1[q] += dv;
        s2[q] = fmaf(dv, dv, s2[q]);
        sq = fmaf(x[u][q], x[u][q], sq);
      }
      if (MODE != AGG_MEAN) {
        sq = wave_sum(sq);
        if (lane == 0) a.sqpart[(int64_t)jj[u] * nblocks + blk] = sq;
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    sh_s1[wv][col_index<VEC4>(lane, q)] = s1[q];
    sh_s2[wv][col_index<VEC4>(lane, q)] = s2[q];
    if (wv == 0) sh_c[col_index<VEC4>(lane, q)] = c[q];
  }
  __syncthreads();

  const int64_t col = base + tid;
  const float kf = static_cast<float>(k);
  float S1 = 0.f, S2 = 0.f;
#pragma unroll
  for (int w = 0; w < AGG_WAVES; ++w) {
    S1 += sh_s1[w][tid];
    S2 += sh_s2[w][tid];
  }
  double m2 = 0.0, g2 = 0.0;
  if (col < P) {
    const float cs = sh_c[tid];
    float g;
    if (MODE == AGG_STATS_GIVEN_MEAN) {
      g = cs;
      m2 = S2;
    } else {
      g = cs + S1 / kf;
      a.g_out[col] = g;
      if (MODE == AGG_FUSED) {
        m2 = S2 - S1 * S1 / kf;
        if (a.w) a.w[col] = a.w[col] - a.eta * g;
      }
    }
    g2 = static_cast<double>(g) * g;
  }
  if (MODE != AGG_MEAN) {
    m2 = block_sum_256(m2, sh_red);
    g2 = block_sum_256(g2, sh_red);
    if (tid == 0) {
      a.part[blk * 2 + 0] = m2;
      a.part[blk * 2 + 1] = g2;
    }
  }
}

// ---------------------------------------------------------------------------
__device__ void push_window(double* h, int32_t* cnt, int D, double v) {
  if (*cnt < D) {
    h[*cnt] = v;
    *cnt += 1;
  } else {
    for (int i = 0; i + 1 < D; ++i) h[i] = h[i + 1];
    h[D - 1] = v;
  }
}

__global__ __launch_bounds__(256) void k_finalize(FinalizeArgs a) {
#pragma clang fp contract(off)
  __shared__ double sh_red[4];
  const int tid = threadIdx.x;
  const int k = a.k_dev ? a.k_dev[0] : a.k_imm;
  if (blockIdx.x > 0) {
    // per-worker squared norms: one wave per worker
    const int lane = tid % WAVE;
    const int j = (blockIdx.x - 1) * 4 + tid / WAVE;
    if (j >= a.n) return;
    if (!a.mask[j]) {
      if (lane == 0) a.sqnorm[j] = 0.f;
      return;
    }
    double s = 0.0;
    const float* p = a.sqpart + (int64_t)j * a.nblocks;
    for (int64_t b = lane; b < a.nblocks; b += WAVE) s += p[b];
    s = wave_sum_d(s);
    if (lane == 0) a.sqnorm[j] = static_cast<float>(s);
    return;
  }
  // block 0: statistics and estimator bookkeeping
  __shared__ dbw_estimator_state st;
  load_state(a.st, &st);
  double m2 = 0.0, g2 = 0.0, ls = 0.0, cnt = 0.0;
  for (int64_t b = tid; b < a.nblocks; b += blockDim.x) {
    m2 += a.part[b * 2 + 0];
    g2 += a.part[b * 2 + 1];
  }
  for (int j = tid; j < a.n; j += blockDim.x)
    if (a.mask[j]) {
      ls += static_cast<double>(a.loss[j]);
      cnt += 1.0;
    }
  m2 = block_sum_256(m2, sh_red);
  g2 = block_sum_256(g2, sh_red);
  ls = block_sum_256(ls, sh_red);
  cnt = block_sum_256(cnt, sh_red);
  if (tid == 0) {
    if (static_cast<int>(cnt) != k) atomicOr(a.err, ERR_MASK_COUNT);
    double V_plus;
    if (k >= 2) {
      V_plus = m2 / (k - 1);
    } else {
      double s = 0.0;
      for (int i = 0; i < st.nV; ++i) s += st.hV[i];
      V_plus = st.nV > 0 ? s / st.nV : 0.0;
    }
    const double N_plus = fmax(g2 - V_plus / k, 0.0);
    const double F_hat = ls / k;
    a.stats->gnorm2 = g2;
    a.stats->V_plus = V_plus;
    a.stats->N_plus = N_plus;
    a.stats->F_hat = F_hat;
    if (a.bookkeeping) {
      const double eta = a.eta;
      if (st.t >= 1 && st.nV >= 1) {
        const double Nl = st.hN[st.nV - 1], Vl = st.hV[st.nV - 1];
        const double den = eta * eta * (Nl + Vl / st.k_prev);
        if (den > 0.0) {
          const double Lp = 2.0 * (eta * Nl - (st.F_prev - F_hat)) / den;
          push_window(st.hL, &st.nL, a.D, Lp);
        }
      }
      int32_t nv = st.nV;
      push_window(st.hV, &nv, a.D, V_plus);
      nv = st.nV;
      push_window(st.hN, &nv, a.D, N_plus);
      st.nV = nv;
      st.F_prev2 = st.F_prev;
      st.F_prev = F_hat;
      st.nF = st.nF < 2 ? st.nF + 1 : 2;
      st.k_prev = k;
      st.t += 1;
    }
  }
  if (a.bookkeeping) {
    __syncthreads();
    store_state(&st, a.st);
  }
}

}  // namespace

hipError_t launch_choose_select(const ChooseArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_choose_select, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_mask_to_sel(const uint8_t* mask, int n, int k, int32_t* sel, int32_t* err,
                              hipStream_t s) {
  hipLaunchKernelGGL(k_mask_to_sel, dim3(1), dim3(64), 0, s, mask, n, k, sel, err);
  return hipGetLastError();
}

hipError_t launch_aggregate(const AggArgs& a, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>(agg_blocks(a.P)));
  const dim3 block(AGG_WAVES * WAVE);
  const bool vec4 = (a.P % 4) == 0;
#define DBW_AGG_LAUNCH(V, M) hipLaunchKernelGGL((k_aggregate<V, M>), grid, block, 0, s, a)
  if (vec4) {
    if (a.mode == AGG_MEAN) DBW_AGG_LAUNCH(true, AGG_MEAN);
    else if (a.mode == AGG_STATS_GIVEN_MEAN) DBW_AGG_LAUNCH(true, AGG_STATS_GIVEN_MEAN);
    else DBW_AGG_LAUNCH(true, AGG_FUSED);
  } else {
    if (a.mode == AGG_MEAN) DBW_AGG_LAUNCH(false, AGG_MEAN);
    else if (a.mode == AGG_STATS_GIVEN_MEAN) DBW_AGG_LAUNCH(false, AGG_STATS_GIVEN_MEAN);
    else DBW_AGG_LAUNCH(false, AGG_FUSED);
  }
#undef DBW_AGG_LAUNCH
  return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s) {
  const dim3 grid(1 + (a.n + 3) / 4);
  hipLaunchKernelGGL(k_finalize, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dbw
