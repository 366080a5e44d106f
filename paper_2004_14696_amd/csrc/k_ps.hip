// Parameter-server kernels of the DBW iteration (gfx950).
//
//  k_choose_select  one block: the DBW choice of k (Sect. 3.3, Eqs. gain,
//                   greedy, greedy2) from the device estimator state, then the
//                   fastest-k selection (Sect. 2, Eq. grad_bw) by rank of
//                   (tick, worker index).
//  k_aggregate      streams the k selected gradient rows once: mean g_t
//                   (Eq. grad_bw), per-column sums of squared deviations for
//                   the variance estimate (Eq. sumvariancekt), per-row squared
//                   norms, and optionally the SGD update (Eq. update).  For
//                   the standalone mean every block ranks the ticks itself;
//                   for the statistics every block lists the mask's rows.
//  k_step_ps        the two above fused for dbw_step: every block repeats the
//                   choice, the selection comes from the arrival order the
//                   host sorted, and each block aggregates its column tile.
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
// waves of a k_step_ps block: with few column tiles, each wave then has at
// most one round of row loads for k <= 64
constexpr int STEP_PS_WAVES = 16;

// Lane exchange within rows of 16 lanes (xor 1, xor 2, half-row mirror, row
// mirror): a butterfly whose four steps leave a row's combination in every
// lane of the row.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const int lo = dpp_i<CTRL>(static_cast<int>(static_cast<uint32_t>(b)));
  const int hi = dpp_i<CTRL>(static_cast<int>(static_cast<uint32_t>(b >> 32)));
  return __builtin_bit_cast(double, (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) |
                                        static_cast<uint32_t>(lo));
}
__device__ __forceinline__ double readlane_d(double v, int l) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(b)), l);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(b >> 32)), l);
  return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

// Sum over each row of 16 lanes by a DPP butterfly, in every lane of the row
// (a fixed order, so the result is reproducible).
__device__ __forceinline__ double row_sum_d(double v) {
  v += dpp_d<0xB1>(v);
  v += dpp_d<0x4E>(v);
  v += dpp_d<0x141>(v);
  v += dpp_d<0x140>(v);
  return v;
}

// Sums over the wave: a DPP butterfly in each 16-lane row, then the four
// row sums read from lanes 0, 16, 32, 48 (fixed order; the same value in
// every lane, on the vector ALUs with no LDS round trip).  Called with the
// whole wave active.
__device__ __forceinline__ float wave_sum(float v) {
  v += __builtin_bit_cast(float, dpp_i<0xB1>(__builtin_bit_cast(int, v)));
  v += __builtin_bit_cast(float, dpp_i<0x4E>(__builtin_bit_cast(int, v)));
  v += __builtin_bit_cast(float, dpp_i<0x141>(__builtin_bit_cast(int, v)));
  v += __builtin_bit_cast(float, dpp_i<0x140>(__builtin_bit_cast(int, v)));
  const int b = __builtin_bit_cast(int, v);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 16));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 48));
  return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ double wave_sum_d(double v) {
  v = row_sum_d(v);
  return (readlane_d(v, 0) + readlane_d(v, 16)) + (readlane_d(v, 32) + readlane_d(v, 48));
}

// Fixed-order sums of doubles over the block (blockDim.x a multiple of 64,
// at most 1024), M at a time; the results in all threads.
template <int M>
__device__ void block_sums_d(double (&v)[M], double* sh /*[16 M]*/) {
#pragma unroll
  for (int m = 0; m < M; ++m) v[m] = wave_sum_d(v[m]);
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, nw = blockDim.x / WAVE;
  __syncthreads();
  if (l == 0)
#pragma unroll
    for (int m = 0; m < M; ++m) sh[m * 16 + w] = v[m];
  __syncthreads();
#pragma unroll
  for (int m = 0; m < M; ++m) {
    double r = sh[m * 16];
    for (int i = 1; i < nw; ++i) r += sh[m * 16 + i];
    v[m] = r;
  }
  __syncthreads();
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

// LDS of the choice of k.
struct ChooseShared {
  dbw_estimator_state st;
  double T[DBW_MAX_N];
  int kfinal;
};

// The DBW choice of k_t from the staged state and T_hat (called by every
// thread; wave 0 computes, k in sh.kfinal afterwards).  B-DBW replaces the
// gain by k; a static policy keeps the objective and overrides k.  write:
// this block stores k, b, the objective and the pinned copy of k.
__device__ void choose_k(const ChooseArgs& a, ChooseShared& sh, bool write) {
#pragma clang fp contract(off)
  const int tid = threadIdx.x, lane = tid % WAVE;
  const int n = a.n;
  const dbw_estimator_state& st = sh.st;
  if (tid < WAVE) {
    // D-window means (oldest first, summed in order as the definition
    // reads), the same sequence in every lane: lane i holds entry i (one
    // LDS read per window, D <= 64), the additions run in order on lane
    // reads instead of a chain of dependent LDS reads
    const int nV = __builtin_amdgcn_readfirstlane(st.nV), nL = __builtin_amdgcn_readfirstlane(st.nL);
    const double hv = lane < nV ? st.hV[lane] : 0.0;
    const double hn = lane < nV ? st.hN[lane] : 0.0;
    const double hl = lane < nL ? st.hL[lane] : 0.0;
    double V = 0.0, N = 0.0, L = 0.0;
    for (int i = 0; i < nV; ++i) {
      V += readlane_d(hv, i);
      N += readlane_d(hn, i);
    }
    for (int i = 0; i < nL; ++i) L += readlane_d(hl, i);
    V = nV > 0 ? V / nV : 0.0;
    N = nV > 0 ? N / nV : 0.0;
    L = nL > 0 ? L / nL : 0.0;
    const bool hasL = st.nL > 0;
    const double ga = a.eta - L * a.eta * a.eta / 2.0;
    const double gb = L * a.eta * a.eta / 2.0;
    // each lane's best (objective, k) over k = lane + 1 + 64 m: ties go to
    // the later, larger k
    double best_r = -INFINITY;
    int best_k = 0;
    bool nonneg = false;   // some gain >= 0
    const bool blind = a.policy == DBW_POLICY_BLIND;
    for (int k = lane + 1; k <= n; k += WAVE) {
      // B-DBW takes the number of aggregated gradients as the gain
      const double Gk = blind ? static_cast<double>(k) : ga * N - gb * V / k;
      const double T = sh.T[k - 1];
      const bool eligible = isfinite(T) && T > 0.0;
      const double r = eligible ? Gk / T : NAN;
      if (write && a.objective) a.objective[k - 1] = hasL ? r : NAN;
      nonneg = nonneg || Gk >= 0.0;
      const bool take = eligible && !isnan(r) && (best_k == 0 || r >= best_r);
      best_r = take ? r : best_r;
      best_k = take ? k : best_k;
    }
    // the largest objective over the wave (rows of 16 lanes by DPP, then the
    // four rows), then the largest k that reaches it; both exact
    double rm = best_r;
#define DBW_MAX_STEP(CTRL) rm = fmax(rm, dpp_d<CTRL>(rm));
    DBW_MAX_STEP(0xB1)
    DBW_MAX_STEP(0x4E)
    DBW_MAX_STEP(0x141)
    DBW_MAX_STEP(0x140)
#undef DBW_MAX_STEP
    const double rmax = fmax(fmax(readlane_d(rm, 0), readlane_d(rm, 16)), fmax(readlane_d(rm, 32), readlane_d(rm, 48)));
    int kc = best_k != 0 && best_r == rmax ? best_k : 0;
#define DBW_KMAX_STEP(CTRL) kc = max(kc, dpp_i<CTRL>(kc));
    DBW_KMAX_STEP(0xB1)
    DBW_KMAX_STEP(0x4E)
    DBW_KMAX_STEP(0x141)
    DBW_KMAX_STEP(0x140)
#undef DBW_KMAX_STEP
    const int kb = max(max(__builtin_amdgcn_readlane(kc, 0), __builtin_amdgcn_readlane(kc, 16)),
                       max(__builtin_amdgcn_readlane(kc, 32), __builtin_amdgcn_readlane(kc, 48)));
    const bool all_negative = __builtin_amdgcn_ballot_w64(nonneg) == 0;
    if (lane == 0) {
      int k = (!hasL || kb == 0 || all_negative) ? n : kb;
      // loss guard: never decrease k while the loss estimate rises
      if (st.nF >= 2 && st.F_prev > a.beta * st.F_prev2 && st.k_prev < n) k = max(k, st.k_prev + 1);
      if (a.policy == DBW_POLICY_STATIC) k = a.k_static;
      if (write) {
        a.k_out[0] = k;
        a.b_out[0] = n - k;
        if (a.k_host) *a.k_host = k;
      }
      sh.kfinal = k;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_choose_select(ChooseArgs a) {
  __shared__ ChooseShared sh;
  __shared__ long long sh_t[DBW_MAX_N];
  __shared__ int32_t sh_o[DBW_MAX_N];
  __shared__ int sh_cnt[16];
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int n = a.n;

  // stage the inputs (T_hat, ticks and the arrival order may live in pinned
  // host memory); all loads are issued before their values are used
  if (a.do_choose) load_state(a.st, &sh.st);
  const bool ordered = a.do_select && a.order_src;
  for (int i = tid; i < n; i += blockDim.x) {
    const double T = a.do_choose ? a.T_src[i] : 0.0;
    const long long t = a.do_select ? a.ticks_src[i] : 0;
    const int32_t o = ordered ? a.order_src[i] : 0;
    if (a.do_choose) {
      sh.T[i] = T;
      if (a.T_hat) a.T_hat[i] = T;
    }
    if (a.do_select) {
      sh_t[i] = t;
      if (a.ticks) a.ticks[i] = t;
    }
    sh_o[i] = o;
  }
  __syncthreads();

  if (a.do_choose) {
    choose_k(a, sh, true);
  } else {
    if (tid == 0) sh.kfinal = a.k_imm;
    __syncthreads();
  }

  if (a.do_select) {
    const int k = sh.kfinal;
    int finite = 0;
    if (ordered) {
      // the host sorted the workers by (tick, index): position r holds the
      // worker of rank r
      for (int r = tid; r < n; r += blockDim.x) {
        const int wr = sh_o[r];
        a.mask[wr] = r < k ? 1 : 0;
        if (r < k) a.sel[r] = wr;
        finite += sh_t[r] < INT64_MAX;
      }
    } else {
      // rank of worker i by (tick, index): G consecutive lanes split the
      // comparisons (G = 4 up to a quarter of the block's threads, then 2,
      // then 1) and add their counts by quad DPP exchanges
      const int nt = static_cast<int>(blockDim.x);
      const int G = 4 * n <= nt ? 4 : 2 * n <= nt ? 2 : 1;
      for (int t = tid; t < G * n; t += nt) {
        const int i = t / G, q = t % G;
        const long long ti = sh_t[i];
        const int j1 = (q + 1) * n / G;
        int rank = 0;
        for (int j = q * n / G; j < j1; ++j) {
          const long long tj = sh_t[j];
          rank += (tj < ti) || (tj == ti && j < i);
        }
        if (G >= 2) rank += dpp_i<0xB1>(rank);
        if (G == 4) rank += dpp_i<0x4E>(rank);
        if (q == 0) {
          const bool on = rank < k;
          a.mask[i] = on ? 1 : 0;
          if (on) a.sel[rank] = i;
          finite += ti < INT64_MAX;
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) finite += __shfl_xor(finite, o, WAVE);
    if (lane == 0) sh_cnt[wv] = finite;
    __syncthreads();
    if (tid == 0) {
      int total = 0;
      for (int w = 0; w < static_cast<int>(blockDim.x / WAVE); ++w) total += sh_cnt[w];
      if (k > total) atomicOr(a.err, ERR_K_RANGE);
    }
  }
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

// Column of w (layout [d][C]) of element e of a slab partial; -1 for the
// padding features of the tile order.  Tile order: 64-feature groups of 64C
// floats; in a group, float4 piece (4 jq + g) C + m holds class m of features
// 16 g + 4 t + jq, t = 0..3.
// (Elements and columns fit 32 bits: a worker's partials are addressed by
// one buffer descriptor, below 2^32 bytes.)
template <int SRC>
__device__ __forceinline__ int slab_column(const AggArgs& a, int e) {
  if (e >= a.slab_len) return -1;
  if (SRC == SRC_SLABS) return e < a.P ? e : -1;
  const int C = a.C;
  const int grp = e / (64 * C);
  const int r = e - grp * 64 * C;
  const int piece = r >> 2, t = r & 3;
  const int m = piece % C, jg = piece / C;
  const int f = 64 * grp + 16 * (jg & 3) + 4 * t + (jg >> 2);
  return f < a.d ? f * C + m : -1;
}

// Columns of w of the lane's four elements e0 .. e0 + 3 (-1: padding or
// past the partial) and the mask of those that are columns.  The same for
// every row, so taken once.
template <int SRC>
__device__ __forceinline__ int slab_lane_cols(const AggArgs& a, int e0, int (&col)[4]) {
  int m = 0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    col[t] = slab_column<SRC>(a, e0 + t);
    if (col[t] >= 0) m |= 1 << t;
  }
  return m;
}

// Worker j's gradient at elements base + 4 lane .. + 3 of the slab layout:
// the sum of its slab partials in slab order (the same additions as the slab
// reduction); 0 for an invalid row and where vmask (slab_lane_mask) is clear.
// S > 0: a.slabs == S, so every load is issued before the first addition.
template <int SRC, int S>
__device__ __forceinline__ void load_slab_row(const AggArgs& a, int j, int64_t base, int lane, float v[4],
                                              bool valid, int vmask) {
  // the descriptor depends on the row only (uniform per wave: no per-lane
  // loop over descriptors); lanes outside vmask read in-range or zero
  // values that are dropped below
  const int64_t e0 = base + lane * 4;
  const __amdgpu_buffer_rsrc_t r = make_rsrc(a.Gp + (int64_t)(valid ? j : 0) * a.slabs * a.slab_len,
                                             valid ? static_cast<uint32_t>(a.slabs * a.slab_len * 4) : 0u);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if constexpr (S > 0) {
    float4 xs[S];
#pragma unroll
    for (int q = 0; q < S; ++q) xs[q] = buf_f32x4(r, static_cast<uint32_t>((q * a.slab_len + e0) * 4));
#pragma unroll
    for (int q = 0; q < S; ++q) {
      acc.x += xs[q].x; acc.y += xs[q].y; acc.z += xs[q].z; acc.w += xs[q].w;
    }
  } else {
    for (int q = 0; q < a.slabs; ++q) {
      const float4 x = buf_f32x4(r, static_cast<uint32_t>((q * a.slab_len + e0) * 4));
      acc.x += x.x; acc.y += x.y; acc.z += x.z; acc.w += x.w;
    }
  }
  v[0] = vmask & 1 ? acc.x : 0.f;
  v[1] = vmask & 2 ? acc.y : 0.f;
  v[2] = vmask & 4 ? acc.z : 0.f;
  v[3] = vmask & 8 ? acc.w : 0.f;
}

// LDS of one aggregation tile worked by NW waves.
template <int NW>
struct AggShared {
  float s1[NW][AGG_TILE];
  float s2[NW][AGG_TILE];
  float c[AGG_TILE];
  double red[32];
};

// Pieces of one block's column tile of the aggregation over the rows listed
// in sel (generic pointer: global or LDS).  The block's NW waves split the
// rows, AGG_U rows in flight per wave; the first AGG_TILE threads finish the
// columns.
constexpr int AGG_U = 4;

// Loads of rows r0 + u NW (u < U) below rmax; jj = -1 past rmax.
template <bool VEC4, int NW, int SRC = SRC_ROWS, int S = 0, int U = AGG_U>
__device__ __forceinline__ void agg_load_round(const AggArgs& a, const int32_t* sel, int r0, int rmax,
                                               float (&x)[U][4], int (&jj)[U], int vmask = 0) {
  const int lane = threadIdx.x % WAVE;
  const int64_t base = (int64_t)blockIdx.x * AGG_TILE;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int r = r0 + u * NW;
    // r is the same in every lane; taking the first lane's value makes the
    // row, and so the buffer descriptor, provably uniform (no per-lane
    // descriptor loop)
    const int jv = r < rmax ? sel[r] : -1;
    jj[u] = __builtin_amdgcn_readfirstlane(jv);
    if (SRC == SRC_ROWS)
      load_tile<VEC4>(a.G + (int64_t)(jj[u] < 0 ? 0 : jj[u]) * a.P, base, lane, a.P, x[u], jj[u] >= 0);
    else
      load_slab_row<SRC, S>(a, jj[u], base, lane, x[u], jj[u] >= 0, vmask);
  }
}

// Shifted sums of the loaded rows, and their squared norms; from slab
// partials, the rows are also stored in [d][C] order when G_rows is set.
template <int MODE, int SRC = SRC_ROWS, int U = AGG_U>
__device__ __forceinline__ void agg_accumulate(const AggArgs& a, const float (&x)[U][4], const int (&jj)[U],
                                               const float (&c)[4], float (&s1)[4], float (&s2)[4],
                                               int vmask = 0, const int* ocol = nullptr) {
  const int lane = threadIdx.x % WAVE;
#pragma unroll
  for (int u = 0; u < U; ++u) {
    if (jj[u] < 0) break;
    if (SRC != SRC_ROWS && a.G_rows) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (vmask >> q & 1) a.G_rows[(int64_t)jj[u] * a.P + ocol[q]] = x[u][q];
    }
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
      if (lane == 0) a.sqpart[(int64_t)jj[u] * gridDim.x + blockIdx.x] = sq;
    }
  }
}

// Column results from the waves' partial sums: g, the update, and the block
// partials of the statistics.
template <bool VEC4, int MODE, int NW, int SRC = SRC_ROWS>
__device__ void agg_finish(const AggArgs& a, int k, const float (&c)[4], const float (&s1)[4], const float (&s2)[4],
                           AggShared<NW>& sh, const float* w_old = nullptr) {
  const int tid = threadIdx.x;
  const int lane = tid % WAVE, wv = tid / WAVE;
  const int64_t P = a.P;
  const int64_t blk = blockIdx.x;
  const int64_t base = blk * AGG_TILE;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    sh.s1[wv][col_index<VEC4>(lane, q)] = s1[q];
    sh.s2[wv][col_index<VEC4>(lane, q)] = s2[q];
    if (wv == 0) sh.c[col_index<VEC4>(lane, q)] = c[q];
  }
  __syncthreads();

  const int64_t col = base + tid;
  // slab layouts: the element's column of w (-1 at padding, whose sums are 0)
  const int64_t out = SRC == SRC_ROWS ? col : slab_column<SRC>(a, static_cast<int>(col));
  const int64_t ncol = SRC == SRC_ROWS ? P : a.slab_len;
  const float kf = static_cast<float>(k);
  double m2 = 0.0, g2 = 0.0;
  if (tid < AGG_TILE && col < ncol) {
    float S1 = 0.f, S2 = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      S1 += sh.s1[w][tid];
      S2 += sh.s2[w][tid];
    }
    const float cs = sh.c[tid];
    float g;
    if (MODE == AGG_STATS_GIVEN_MEAN) {
      g = cs;
      m2 = S2;
    } else {
      g = cs + S1 / kf;
      if (out >= 0) a.g_out[out] = g;
      if (MODE == AGG_FUSED) {
        m2 = S2 - S1 * S1 / kf;
        if (a.w && out >= 0) a.w[out] = (w_old ? *w_old : a.w[out]) - a.eta * g;
      }
    }
    g2 = static_cast<double>(g) * g;
  }
  if (MODE != AGG_MEAN) {
    // the tile's sums: the AGG_TILE column threads fill the first waves;
    // a DPP tree in each, then those waves' sums in order
    constexpr int TW = AGG_TILE / WAVE;
    if (wv < TW) {
      m2 = row_sum_d(m2);
      g2 = row_sum_d(g2);
      // the four row sums are read with the whole wave active (a read
      // inside the lane-0 branch would let the compiler compute the other
      // rows' sums there, for lane 0 only)
      const double wm2 = readlane_d(m2, 0) + readlane_d(m2, 16) + readlane_d(m2, 32) + readlane_d(m2, 48);
      const double wg2 = readlane_d(g2, 0) + readlane_d(g2, 16) + readlane_d(g2, 32) + readlane_d(g2, 48);
      if (lane == 0) {
        sh.red[wv] = wm2;
        sh.red[TW + wv] = wg2;
      }
    }
    __syncthreads();
    if (tid == 0) {
      double s0 = sh.red[0], s1v = sh.red[TW];
#pragma unroll
      for (int w = 1; w < TW; ++w) {
        s0 += sh.red[w];
        s1v += sh.red[TW + w];
      }
      a.part[blk * 2 + 0] = s0;
      a.part[blk * 2 + 1] = s1v;
    }
  }
}

// The shift row's tile: the mean itself (given) or the fastest worker's row.
template <bool VEC4, int MODE, int SRC = SRC_ROWS, int S = 0>
__device__ __forceinline__ void agg_shift(const AggArgs& a, const int32_t* sel, float (&c)[4], int vmask = 0) {
  const int lane = threadIdx.x % WAVE;
  const int64_t base = (int64_t)blockIdx.x * AGG_TILE;
  if (MODE == AGG_STATS_GIVEN_MEAN) load_tile<VEC4>(a.g_in, base, lane, a.P, c);
  else if (SRC == SRC_ROWS)
    load_tile<VEC4>(a.G + (int64_t)__builtin_amdgcn_readfirstlane(sel[0]) * a.P, base, lane, a.P, c);
  else load_slab_row<SRC, S>(a, __builtin_amdgcn_readfirstlane(sel[0]), base, lane, c, true, vmask);
}

template <bool VEC4, int MODE, int NW>
__device__ void aggregate_tile(const AggArgs& a, const int32_t* sel, int k, AggShared<NW>& sh) {
  const int wv = threadIdx.x / WAVE;
  float c[4];
  agg_shift<VEC4, MODE>(a, sel, c);
  float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f};
  for (int r0 = wv; r0 < k; r0 += NW * AGG_U) {
    float x[AGG_U][4];
    int jj[AGG_U];
    agg_load_round<VEC4, NW>(a, sel, r0, k, x, jj);
    agg_accumulate<MODE>(a, x, jj, c, s1, s2);
  }
  agg_finish<VEC4, MODE, NW>(a, k, c, s1, s2, sh);
}

// The set entries of mask [n] in worker order into sel[0, k) (LDS), the
// entries past their count -1 (no row; a count other than k is reported by
// the statistics).  Ballots and prefix popcounts per wave, wave counts
// through LDS; every thread of the block calls it.
__device__ void mask_to_sel_block(const uint8_t* mask, int n, int k, int32_t* sel, int* sh_wc) {
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int nw = static_cast<int>(blockDim.x) / WAVE;
  const uint64_t below = (uint64_t{1} << lane) - 1;
  int c = 0;
  for (int base = 0; base < n; base += blockDim.x) {
    const int j = base + tid;
    const bool on = j < n && mask[j] != 0;
    const uint64_t b = __builtin_amdgcn_ballot_w64(on);
    if (lane == 0) sh_wc[wv] = __popcll(b);
    __syncthreads();
    int before = c, total = c;
    for (int w = 0; w < nw; ++w) {
      before += w < wv ? sh_wc[w] : 0;
      total += sh_wc[w];
    }
    const int r = before + __popcll(b & below);
    if (on && r < k) sel[r] = j;
    c = total;
    __syncthreads();
  }
  for (int r = c + tid; r < k; r += blockDim.x) sel[r] = -1;
  __syncthreads();
}

// The k fastest of n workers by (tick, index), listed in arrival order into
// sel (LDS) by every block of an aggregation; block 0 also writes the mask
// and reports k beyond the finite ticks.  Ranks are counts of the workers
// ahead (the same comparisons as the selection kernel).
__device__ void select_fastest_block(const int64_t* ticks, int n, int k, int32_t* sel, long long* sh_t,
                                     uint8_t* mask, int32_t* err, int* sh_cnt) {
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int nt = static_cast<int>(blockDim.x);
  for (int i = tid; i < n; i += nt) sh_t[i] = ticks[i];
  __syncthreads();
  const bool lead = blockIdx.x == 0;
  int finite = 0;
  for (int i = tid; i < n; i += nt) {
    const long long ti = sh_t[i];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const long long tj = sh_t[j];
      rank += (tj < ti) || (tj == ti && j < i);
    }
    if (rank < k) sel[rank] = i;
    if (lead) {
      mask[i] = rank < k ? 1 : 0;
      finite += ti < INT64_MAX;
    }
  }
  if (lead) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) finite += __shfl_xor(finite, o, WAVE);
    if (lane == 0) sh_cnt[wv] = finite;
  }
  __syncthreads();
  if (lead && tid == 0) {
    int total = 0;
    for (int w = 0; w < nt / WAVE; ++w) total += sh_cnt[w];
    if (k > total) atomicOr(err, ERR_K_RANGE);
  }
}

template <bool VEC4, int MODE, bool SELECT = false>
__global__ __launch_bounds__(AGG_WAVES * WAVE) void k_aggregate(AggArgs a) {
  __shared__ AggShared<AGG_WAVES> sh;
  const int k = a.k_dev ? a.k_dev[0] : a.k_imm;
  if constexpr (SELECT) {
    // the selection in every block: no launch of its own before this one
    __shared__ int32_t sh_sel[DBW_MAX_N];
    __shared__ long long sh_t[DBW_MAX_N];
    __shared__ int sh_cnt[AGG_WAVES];
    select_fastest_block(a.ticks_sel, a.n, k, sh_sel, sh_t, a.mask_out, a.err, sh_cnt);
    aggregate_tile<VEC4, MODE, AGG_WAVES>(a, sh_sel, k, sh);
  } else if constexpr (MODE == AGG_STATS_GIVEN_MEAN) {
    // the rows come as a mask: each block lists them itself (no separate
    // launch; the list is n bytes of L2-resident reads per block)
    __shared__ int32_t sh_sel[DBW_MAX_N];
    __shared__ int sh_wc[AGG_WAVES];
    mask_to_sel_block(a.sel_mask, a.n, k, sh_sel, sh_wc);
    aggregate_tile<VEC4, MODE, AGG_WAVES>(a, sh_sel, k, sh);
  } else {
    aggregate_tile<VEC4, MODE, AGG_WAVES>(a, a.sel, k, sh);
  }
}

// The PS side of one DBW iteration in one launch: every block makes the
// choice of k_t itself (the same fp64 arithmetic on the same staged inputs,
// so every block reaches the same k), takes the first k_t workers of the
// arrival order the host sorted (ties to the lower index), and aggregates its
// column tile with the SGD update; block 0 also stores the choice, the
// selection and the device copies of T_hat and the ticks.  With a slab
// source the rows are the selected workers' slab partials summed in place
// (tiles follow the partial's layout, results land at their [d][C] column),
// and block 0 also turns every worker's slab loss sums into its loss.
template <bool VEC4, int SRC = SRC_ROWS, int S = 0>
__global__ __launch_bounds__(STEP_PS_WAVES * WAVE) void k_step_ps(ChooseArgs ca, AggArgs a, StepInline inl) {
  constexpr int NW = STEP_PS_WAVES;
  // rows per wave and round: about 8 float4 loads in flight per lane within
  // the 128 registers a 16-wave block leaves each wave
  constexpr int RU = SRC == SRC_ROWS ? AGG_U : S > 0 ? (8 / S > 1 ? 8 / S : 1) : 2;
  __shared__ ChooseShared cs;
  __shared__ AggShared<NW> sh;
  __shared__ int32_t sh_order[DBW_MAX_N];
  __shared__ long long sh_t[DBW_MAX_N];
  __shared__ int sh_cnt[16];
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int n = ca.n;
  const bool lead = blockIdx.x == 0;
  // every host and device read of the prologue is issued before any use
  load_state(ca.st, &cs.st);
  const int64_t col = (int64_t)blockIdx.x * AGG_TILE + tid;
  int64_t wcol = col < a.P ? col : -1;
  if (SRC != SRC_ROWS) wcol = slab_column<SRC>(a, static_cast<int>(col));
  const float w_old = tid < AGG_TILE && wcol >= 0 && a.w ? a.w[wcol] : 0.f;
  const bool given = inl.n_inline == n;
  for (int i = tid; i < n; i += blockDim.x) {
    const double T = given ? inl.T[i] : ca.T_src[i];
    const int32_t o = given ? inl.order[i] : ca.order_src[i];
    const long long t = lead ? (given ? inl.ticks[i] : ca.ticks_src[i]) : 0;
    cs.T[i] = T;
    sh_order[i] = o;
    if (lead) {
      sh_t[i] = t;
      if (ca.T_hat) ca.T_hat[i] = T;
      if (ca.ticks) ca.ticks[i] = t;
    }
  }
  __syncthreads();
  // the first rows of the arrival order are loaded while the choice runs
  // (k_t >= 1 rows are needed; rows past k_t are dropped)
  int ocol[4];
  const int vmask = SRC == SRC_ROWS ? 0 : slab_lane_cols<SRC>(a, static_cast<int>(blockIdx.x) * AGG_TILE + lane * 4, ocol);
  float c[4];
  agg_shift<VEC4, AGG_FUSED, SRC, S>(a, sh_order, c, vmask);
  float x[RU][4];
  int jj[RU];
  agg_load_round<VEC4, NW, SRC, S, RU>(a, sh_order, wv, n, x, jj, vmask);
  choose_k(ca, cs, lead);
  const int k = cs.kfinal;
  if (SRC != SRC_ROWS && lead) {
    for (int i = tid; i < n; i += blockDim.x) {
      float l = 0.f;
      for (int q = 0; q < a.slabs; ++q) l += a.lossp[(int64_t)i * a.slabs + q];
      a.loss[i] = l / static_cast<float>(a.B);
    }
  }
  if (lead) {
    int finite = 0;
    for (int r = tid; r < n; r += blockDim.x) {
      const int i = sh_order[r];
      const long long t = sh_t[i];
      ca.mask[i] = r < k ? 1 : 0;
      if (r < k) ca.sel[r] = i;
      finite += t < INT64_MAX;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) finite += __shfl_xor(finite, o, WAVE);
    if (lane == 0) sh_cnt[wv] = finite;
    __syncthreads();
    if (tid == 0) {
      int total = 0;
      for (int w = 0; w < NW; ++w) total += sh_cnt[w];
      if (k > total) atomicOr(ca.err, ERR_K_RANGE);
    }
  }
#pragma unroll
  for (int u = 0; u < RU; ++u)
    if (wv + u * NW >= k) jj[u] = -1;
  float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f};
  agg_accumulate<AGG_FUSED, SRC, RU>(a, x, jj, c, s1, s2, vmask, ocol);
  for (int r0 = wv + NW * RU; r0 < k; r0 += NW * RU) {
    agg_load_round<VEC4, NW, SRC, S, RU>(a, sh_order, r0, k, x, jj, vmask);
    agg_accumulate<AGG_FUSED, SRC, RU>(a, x, jj, c, s1, s2, vmask, ocol);
  }
  agg_finish<VEC4, AGG_FUSED, NW, SRC>(a, k, c, s1, s2, sh, &w_old);
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_finalize(FinalizeArgs a) {
#pragma clang fp contract(off)
  __shared__ double sh_red[64];
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
    // the lane's entries in increasing order, eight loads in flight at a
    // time (a plain loop waits for each load before its addition); entries
    // past the row read as 0, and adding +0 to these sums of squares (>= 0)
    // changes no bit
    double s = 0.0;
    const __amdgpu_buffer_rsrc_t p = make_rsrc(a.sqpart + (int64_t)j * a.nblocks,
                                               static_cast<uint32_t>(a.nblocks * 4));
    for (int64_t b = lane; b < a.nblocks; b += 8 * WAVE) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = buf_f32(p, static_cast<uint32_t>((b + u * WAVE) * 4));
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    s = wave_sum_d(s);
    if (lane == 0) a.sqnorm[j] = static_cast<float>(s);
    return;
  }
  // block 0: statistics and estimator bookkeeping
  __shared__ dbw_estimator_state st;
  if (a.st) load_state(a.st, &st);
  double m2 = 0.0, g2 = 0.0, ls = 0.0, cnt = 0.0;
  {
    // in increasing tile order, four tiles' loads in flight at a time
    const int64_t nt = blockDim.x;
    int64_t b = tid;
    for (; b + 3 * nt < a.nblocks; b += 4 * nt) {
      double v[4][2];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v[u][0] = a.part[(b + u * nt) * 2 + 0];
        v[u][1] = a.part[(b + u * nt) * 2 + 1];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        m2 += v[u][0];
        g2 += v[u][1];
      }
    }
    for (; b < a.nblocks; b += nt) {
      m2 += a.part[b * 2 + 0];
      g2 += a.part[b * 2 + 1];
    }
  }
  for (int j = tid; j < a.n; j += blockDim.x)
    if (a.mask[j]) {
      ls += static_cast<double>(a.loss[j]);
      cnt += 1.0;
    }
  {
    double v[4] = {m2, g2, ls, cnt};
    block_sums_d<4>(v, sh_red);
    m2 = v[0];
    g2 = v[1];
    ls = v[2];
    cnt = v[3];
  }
  if (tid < WAVE) {
    // wave 0: every lane computes the same scalars (the same inputs and
    // operations); lane i holds entry i of each D-window (D <= 64), so the
    // window mean is one LDS read and in-order additions of lane reads, and
    // a full window shifts by one in a single read and write
    const int lane = tid;
    const int nV = __builtin_amdgcn_readfirstlane(st.nV), nL = __builtin_amdgcn_readfirstlane(st.nL);
    const double hv = lane < nV ? st.hV[lane] : 0.0;
    const double hn = lane < nV ? st.hN[lane] : 0.0;
    const double hl = lane < nL ? st.hL[lane] : 0.0;
    const bool count_ok = static_cast<int>(cnt) == k;
    if (lane == 0 && !count_ok && a.err) atomicOr(a.err, ERR_MASK_COUNT);
    double V_plus;
    if (k >= 2) {
      V_plus = m2 / (k - 1);
    } else if (a.v_window_given) {
      V_plus = a.v_window;
    } else {
      double s = 0.0;
      for (int i = 0; i < nV; ++i) s += readlane_d(hv, i);
      V_plus = nV > 0 ? s / nV : 0.0;
    }
    const double N_plus = fmax(g2 - V_plus / k, 0.0);
    const double F_hat = ls / k;
    // without an error flag, a mask that does not hold k ones is reported
    // through the statistics themselves
    const double bad = !count_ok && !a.err ? NAN : 0.0;
    if (lane == 0) {
      a.stats->gnorm2 = g2 + bad;
      a.stats->V_plus = V_plus + bad;
      a.stats->N_plus = N_plus + bad;
      a.stats->F_hat = F_hat + bad;
    }
    if (a.bookkeeping) {
      const double eta = a.eta;
      const int D = a.D;
      // append while the window is not full, else drop the oldest entry
      // (lane i takes lane i + 1's) and put v last; returns the new count
      auto push = [&](double* h, int cw, double held, double v) {
        const double next = __shfl_down(held, 1, WAVE);
        if (cw < D) {
          if (lane == cw) h[lane] = v;
          return cw + 1;
        }
        if (lane + 1 < D) h[lane] = next;
        else if (lane + 1 == D) h[lane] = v;
        return D;
      };
      int nL_new = nL;
      if (st.t >= 1 && nV >= 1) {
        const double Nl = readlane_d(hn, nV - 1), Vl = readlane_d(hv, nV - 1);
        const double den = eta * eta * (Nl + Vl / st.k_prev);
        if (den > 0.0) {
          const double Lp = 2.0 * (eta * Nl - (st.F_prev - F_hat)) / den;
          nL_new = push(st.hL, nL, hl, Lp);
        }
      }
      const int nV_new = push(st.hV, nV, hv, V_plus);
      (void)push(st.hN, nV, hn, N_plus);
      if (lane == 0) {
        st.nL = nL_new;
        st.nV = nV_new;
        st.F_prev2 = st.F_prev;
        st.F_prev = F_hat;
        st.nF = st.nF < 2 ? st.nF + 1 : 2;
        st.k_prev = k;
        st.t += 1;
      }
    }
  }
  if (a.bookkeeping) {
    __syncthreads();
    store_state(&st, a.st);
  }
}

}  // namespace

hipError_t launch_choose_select(const ChooseArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_choose_select, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_aggregate(const AggArgs& a, hipStream_t s) {
  const bool select = a.mode == AGG_MEAN && a.ticks_sel;
  if (select ? !a.mask_out || !a.err : a.mode == AGG_STATS_GIVEN_MEAN ? !a.sel_mask : !a.sel)
    return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(agg_blocks(a.P)));
  const dim3 block(AGG_WAVES * WAVE);
  const bool vec4 = (a.P % 4) == 0;
  if (select) {
    if (vec4) hipLaunchKernelGGL((k_aggregate<true, AGG_MEAN, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_aggregate<false, AGG_MEAN, true>), grid, block, 0, s, a);
    return hipGetLastError();
  }
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

template <int SRC>
void launch_step_ps_slabs(const ChooseArgs& ca, const AggArgs& a, const StepInline& inl, dim3 grid, dim3 block,
                          hipStream_t s) {
  switch (a.slabs) {
#define DBW_SLABS_CASE(S) \
    case S: hipLaunchKernelGGL((k_step_ps<true, SRC, S>), grid, block, 0, s, ca, a, inl); return;
    DBW_SLABS_CASE(2)
    DBW_SLABS_CASE(3)
    DBW_SLABS_CASE(4)
    DBW_SLABS_CASE(5)
    DBW_SLABS_CASE(6)
    DBW_SLABS_CASE(7)
    DBW_SLABS_CASE(8)
#undef DBW_SLABS_CASE
    default: hipLaunchKernelGGL((k_step_ps<true, SRC, 0>), grid, block, 0, s, ca, a, inl);
  }
}

hipError_t launch_step_ps(const ChooseArgs& ca, const AggArgs& a, const StepInline& inl, hipStream_t s) {
  if (inl.n_inline != 0 && (inl.n_inline != ca.n || ca.n > kInlineN)) return hipErrorInvalidValue;
  const dim3 block(STEP_PS_WAVES * WAVE);
  if (a.src != SRC_ROWS) {
    // slab partials: float4 pieces of 4 consecutive elements
    if (a.slab_len % 4 != 0 || !a.Gp || !a.lossp || !a.loss || a.slabs < 1) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(agg_blocks(a.slab_len)));
    if (a.src == SRC_SLAB_TILES) launch_step_ps_slabs<SRC_SLAB_TILES>(ca, a, inl, grid, block, s);
    else launch_step_ps_slabs<SRC_SLABS>(ca, a, inl, grid, block, s);
    return hipGetLastError();
  }
  const dim3 grid(static_cast<unsigned>(agg_blocks(a.P)));
  if ((a.P % 4) == 0) hipLaunchKernelGGL(k_step_ps<true>, grid, block, 0, s, ca, a, inl);
  else hipLaunchKernelGGL(k_step_ps<false>, grid, block, 0, s, ca, a, inl);
  return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s) {
  const dim3 grid(1 + (a.n + 3) / 4);
  hipLaunchKernelGGL(k_finalize, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dbw
