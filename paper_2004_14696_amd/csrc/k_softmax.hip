// Worker minibatch gradients of softmax regression (Sect. 2, Eq. gradient), gfx950.
//
// For worker i with minibatch rows x_{i,b} (b < B) and labels y_{i,b}:
//   z_b = x_b W,  p_b = softmax(z_b),  r_b = (p_b - onehot(y_b)) / B
//   G_i = sum_b x_b^T r_b  (d x C, laid out like W)
//   loss_i = (1/B) sum_b (logsumexp(z_b) - z_{b,y_b})
//
// Two implementations:
//  * k_softmax_fused -- small C (<= 16): one pass over X.  Each thread owns a
//    strided slice of the feature dimension and keeps both its slice of W
//    and of the gradient accumulator in registers.  Rows stream through in
//    chunks of R: per-thread partial logits are reduced across the block
//    through LDS, R threads run the softmax, and every thread folds the
//    residuals into its accumulator.  A worker's rows are split over
//    `slabs` blocks (to fill the 256 CUs); a second kernel sums the slab
//    partials in a fixed order.
//  * GEMM path -- any C: logits Z = X W (tiled fp32 GEMM), row softmax in
//    place (residuals), then a per-worker GEMM G_i = X_i^T R_i.
//
// Minibatch rows are read either from a materialised X [n][B][d] or by row
// index from a resident dataset; both read each sample once per pass.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dbw_buffer.h"
#include "dbw_internal.h"

namespace dbw {
namespace {

constexpr int WAVE = 64;
constexpr int NXCD = 8;

// Row pointer and label of sample b of worker i; invalid indices are
// reported and replaced by 0 so that no access leaves the buffers.
__device__ __forceinline__ int64_t sample_row(const SoftmaxArgs& a, int i, int b, bool report) {
  const int64_t m = (int64_t)i * a.B + b;
  if (!a.rows) return m;
  const int64_t r = a.rows[m];
  if (r < 0 || r >= a.S) {
    if (report) atomicOr(a.err, ERR_ROW_RANGE);
    return 0;
  }
  return r;
}

__device__ __forceinline__ int sample_label(const SoftmaxArgs& a, int64_t row, bool report) {
  const int lab = a.y[row];
  if (lab < 0 || lab >= a.C) {
    if (report) atomicOr(a.err, ERR_LABEL_RANGE);
    return 0;
  }
  return lab;
}

// Block index -> logical (worker, slab) so that a worker's slabs run on the
// same XCD (dispatch places block b on XCD b % 8): their partials then meet
// in one L2.
__device__ __forceinline__ int64_t xcd_logical(int64_t b, int64_t per_xcd) {
  return (b % NXCD) * per_xcd + b / NXCD;
}

constexpr int FUSED_MAX_ROWS = 1024;   // rows of one slab staged in LDS

template <int CP, int M, int T, int R>
__global__ __launch_bounds__(T) void k_softmax_fused(SoftmaxArgs a, int slabs, int rps, int64_t per_xcd) {
  constexpr int V = R * CP;            // partial logits per thread
  constexpr int G = T / V;             // reduction groups (>= 1)
  static_assert(G >= 1, "block too small for the chunk");
  static_assert(R == 4 && CP <= 16, "softmax wave layout: 4 rows x 16 lanes");
  __shared__ float red[T][V + 1];
  __shared__ float red2[G][V];
  __shared__ float rr[V];
  __shared__ float sh_loss[R];
  __shared__ int sh_row[FUSED_MAX_ROWS];
  __shared__ int sh_lab[FUSED_MAX_ROWS];

  const int64_t logical = xcd_logical(blockIdx.x, per_xcd);
  if (logical >= (int64_t)a.n * slabs) return;
  const int i = static_cast<int>(logical / slabs);
  const int q = static_cast<int>(logical % slabs);
  const int tid = threadIdx.x;
  const int d = a.d, C = a.C;
  const int64_t P = (int64_t)d * C;
  const int b0 = q * rps;
  const int b1 = min(a.B, b0 + rps);
  const int nrows = b1 - b0;

  // the slab's row indices and labels, validated once
  for (int r = tid; r < nrows; r += T) {
    const int64_t row = sample_row(a, i, b0 + r, true);
    sh_row[r] = static_cast<int>(row);
    sh_lab[r] = sample_label(a, row, true);
  }

  // this thread's slice of W; features j >= d and classes c >= C read as 0
  const __amdgpu_buffer_rsrc_t wrs = make_rsrc(a.W, static_cast<uint32_t>(P * 4));
  float wr[M][CP];
  float acc[M][CP];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int j = tid + m * T;
#pragma unroll
    for (int c = 0; c < CP; ++c) {
      const uint32_t off = c < C ? static_cast<uint32_t>((j * C + c) * 4) : kOutOfRange;
      wr[m][c] = buf_f32(wrs, off);
      acc[m][c] = 0.f;
    }
  }
  float loss_acc = 0.f;
  const float invB = 1.0f / static_cast<float>(a.B);
  __syncthreads();

  // rows of chunk `cb` (relative to b0) into x; rows past the slab read as 0
  auto load_chunk = [&](int cb, float (&x)[R][M]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int rr_ = cb + r;
      const bool row_ok = rr_ < nrows;
      const int row = __builtin_amdgcn_readfirstlane(sh_row[row_ok ? rr_ : 0]);
      // a resource over the row (empty past the slab): j >= d reads 0
      const __amdgpu_buffer_rsrc_t xr =
          make_rsrc(a.X + static_cast<int64_t>(row) * d, row_ok ? static_cast<uint32_t>(d * 4) : 0u);
#pragma unroll
      for (int m = 0; m < M; ++m) x[r][m] = buf_f32(xr, static_cast<uint32_t>((tid + m * T) * 4));
    }
  };

  float xa[R][M], xb[R][M];
  load_chunk(0, xa);
  for (int cb = 0; cb < nrows; cb += R) {
    // partial logits over this thread's slice of the features
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
      for (int c = 0; c < CP; ++c) {
        float z = 0.f;
#pragma unroll
        for (int m = 0; m < M; ++m) z = fmaf(xa[r][m], wr[m][c], z);
        red[tid][r * CP + c] = z;
      }
    }
    // next chunk's loads fly during the reduction and the softmax
    load_chunk(cb + R, xb);
    __syncthreads();
    if (tid < V * G) {
      const int v = tid % V, g = tid / V;
      float s = 0.f;
#pragma unroll 4
      for (int t = g; t < T; t += G) s += red[t][v];
      red2[g][v] = s;
    }
    __syncthreads();
    // wave 0: 16 lanes per row (R == 4) finish the reduction and run the
    // softmax; lane (r, c) holds logit c of row r.
    if (tid < WAVE) {
      const int r = tid / 16, c = tid % 16;
      const int rb = cb + r;
      float z = 0.f;
      if (c < CP) {
#pragma unroll
        for (int g = 0; g < G; ++g) z += red2[g][r * CP + c];
      }
      const bool valid = c < C;
      float zmax = valid ? z : -INFINITY;
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) zmax = fmaxf(zmax, __shfl_xor(zmax, o, 16));
      const float sh = z - zmax;
      const float e = valid ? expf(sh) : 0.f;
      float se = e;
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) se += __shfl_xor(se, o, 16);
      const bool row_ok = rb < nrows;
      const int lab = row_ok ? sh_lab[rb] : 0;
      const float zy = __shfl(sh, r * 16 + lab, WAVE);
      if (c < CP) rr[r * CP + c] = row_ok ? (e / se - (c == lab ? 1.f : 0.f)) * invB : 0.f;
      // CE = log(sum_c e^{z_c - zmax}) - (z_y - zmax)
      if (c == 0 && row_ok) loss_acc += logf(se) - zy;
    }
    __syncthreads();
    // fold the residuals into the gradient slice, row by row
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float rv[CP];
#pragma unroll
      for (int c = 0; c < CP; ++c) rv[c] = rr[r * CP + c];
#pragma unroll
      for (int m = 0; m < M; ++m)
#pragma unroll
        for (int c = 0; c < CP; ++c) acc[m][c] = fmaf(xa[r][m], rv[c], acc[m][c]);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) xa[r][m] = xb[r][m];
  }
  if (tid < WAVE && tid % 16 == 0) sh_loss[tid / 16] = loss_acc;
  __syncthreads();
  float block_loss = 0.f;
#pragma unroll
  for (int r = 0; r < R; ++r) block_loss += sh_loss[r];

  if (slabs == 1) {
#pragma unroll
    for (int m = 0; m < M; ++m) {
      const int j = tid + m * T;
      if (j < d)
#pragma unroll
        for (int c = 0; c < CP; ++c)
          if (c < C) a.G[(int64_t)i * P + (int64_t)j * C + c] = acc[m][c];
    }
    if (tid == 0) a.loss[i] = block_loss * invB;
    return;
  }
  float* gp = a.Gp + ((int64_t)i * slabs + q) * P;
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int j = tid + m * T;
    if (j < d)
#pragma unroll
      for (int c = 0; c < CP; ++c)
        if (c < C) gp[(int64_t)j * C + c] = acc[m][c];
  }
  if (tid == 0) a.lossp[(int64_t)i * slabs + q] = block_loss;
}

// Sum of the slab partials of every worker in slab order (a kernel of its
// own: the launch boundary orders the partial writes before these reads).
// blockIdx.y = worker; each thread adds 4 consecutive elements.
__global__ __launch_bounds__(256) void k_slab_reduce(SoftmaxArgs a, int slabs) {
  const int i = blockIdx.y;
  const int64_t P = (int64_t)a.d * a.C;
  const int64_t e0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  const float* src = a.Gp + (int64_t)i * slabs * P;
  float* dst = a.G + (int64_t)i * P;
  if (e0 < P) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(src, static_cast<uint32_t>(slabs * P * 4));
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    if ((P & 3) == 0) {
      for (int q = 0; q < slabs; ++q) {
        const float4 v = buf_f32x4(rs, static_cast<uint32_t>((q * P + e0) * 4));
        s0 += v.x; s1 += v.y; s2 += v.z; s3 += v.w;
      }
      *reinterpret_cast<float4*>(dst + e0) = make_float4(s0, s1, s2, s3);
    } else {
      float acc4[4] = {0.f, 0.f, 0.f, 0.f};
      for (int q = 0; q < slabs; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t idx = e0 + e;
          acc4[e] += buf_f32(rs, idx < P ? static_cast<uint32_t>((q * P + idx) * 4) : kOutOfRange);
        }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e0 + e < P) dst[e0 + e] = acc4[e];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    float s = 0.f;
    for (int q = 0; q < slabs; ++q) s += a.lossp[(int64_t)i * slabs + q];
    a.loss[i] = s / static_cast<float>(a.B);
  }
}

// ---------------------------------------------------------------------------
// GEMM path.  64 x 64 output tile, 16-deep K slices staged in LDS, 256
// threads each computing a 4 x 4 sub-tile.
constexpr int GBM = 64, GBN = 64, GBK = 16;

// Z[m][c] = sum_j X[row(m)][j] W[j][c] for m < n*B, c < C.
__global__ __launch_bounds__(256) void k_logits_gemm(SoftmaxArgs a) {
  __shared__ float As[GBK][GBM + 4];
  __shared__ float Bs[GBK][GBN + 4];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int64_t Mrows = (int64_t)a.n * a.B;
  const int64_t m0 = (int64_t)blockIdx.y * GBM;
  const int n0 = blockIdx.x * GBN;
  const int d = a.d, C = a.C;
  // A loader: row m0 + tid/4, k offset (tid%4)*4; out-of-range reads are 0
  const int la_m = tid / 4, la_k = (tid % 4) * 4;
  const int64_t am = m0 + la_m;
  const int64_t xrows = a.rows ? a.S : Mrows;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t ws = make_rsrc(a.W, static_cast<uint32_t>((int64_t)d * C * 4));
  int64_t arow = -1;
  if (am < Mrows) {
    const int wi = static_cast<int>(am / a.B), wb = static_cast<int>(am % a.B);
    arow = sample_row(a, wi, wb, la_k == 0);
  }
  const int lb_k = tid / 16, lb_n = (tid % 16) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < d; k0 += GBK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int kk = k0 + la_k + e;
      const uint32_t off = (arow >= 0 && kk < d) ? static_cast<uint32_t>((arow * d + kk) * 4) : kOutOfRange;
      As[la_k + e][la_m] = buf_f32(xs, off);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int kk = k0 + lb_k, nn = n0 + lb_n + e;
      const uint32_t off = (kk < d && nn < C) ? static_cast<uint32_t>(((int64_t)kk * C + nn) * 4) : kOutOfRange;
      Bs[lb_k][lb_n + e] = buf_f32(ws, off);
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        av[e] = As[kk][ty * 4 + e];
        bv[e] = Bs[kk][tx * 4 + e];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(av[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t m = m0 + ty * 4 + r;
    if (m >= Mrows) continue;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int nn = n0 + tx * 4 + c;
      if (nn < C) a.Z[m * C + nn] = acc[r][c];
    }
  }
}

// Row softmax in place: Z[m] <- (softmax(Z[m]) - onehot(y)) / B; ce[m] = CE.
__global__ __launch_bounds__(256) void k_rows_softmax(SoftmaxArgs a) {
  const int lane = threadIdx.x % WAVE;
  const int64_t m = (int64_t)blockIdx.x * 4 + threadIdx.x / WAVE;
  if (m >= (int64_t)a.n * a.B) return;
  const int C = a.C;
  float* z = a.Z + m * C;
  const int wi = static_cast<int>(m / a.B), wb = static_cast<int>(m % a.B);
  const int lab = sample_label(a, sample_row(a, wi, wb, false), lane == 0);
  float mx = -INFINITY;
  for (int c = lane; c < C; c += WAVE) mx = fmaxf(mx, z[c]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, WAVE));
  float se = 0.f;
  for (int c = lane; c < C; c += WAVE) se += expf(z[c] - mx);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) se += __shfl_xor(se, o, WAVE);
  const float zy = z[lab];
  const float inv = 1.0f / se, invB = 1.0f / static_cast<float>(a.B);
  __syncthreads();  // every lane has read z[lab] before it is overwritten
  for (int c = lane; c < C; c += WAVE) z[c] = (expf(z[c] - mx) * inv - (c == lab ? 1.f : 0.f)) * invB;
  if (lane == 0) a.ce[m] = (logf(se) + mx) - zy;
}

// G_i[j][c] = sum_b X_i[b][j] R_i[b][c]; blockIdx.z = worker.
__global__ __launch_bounds__(256) void k_grads_gemm(SoftmaxArgs a) {
  __shared__ float As[GBK][GBM + 4];
  __shared__ float Bs[GBK][GBN + 4];
  __shared__ float sh[256];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int i = blockIdx.z;
  const int j0 = blockIdx.y * GBM;
  const int n0 = blockIdx.x * GBN;
  const int d = a.d, C = a.C, B = a.B;
  const int64_t P = (int64_t)d * C;
  const int64_t xrows = a.rows ? a.S : (int64_t)a.n * B;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.Z + (int64_t)i * B * C, static_cast<uint32_t>((int64_t)B * C * 4));
  const int l_k = tid / 16, l_x = (tid % 16) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < B; k0 += GBK) {
    const int b = k0 + l_k;
    const int64_t xrow = b < B ? sample_row(a, i, b, false) : -1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = j0 + l_x + e;
      const uint32_t xo = (xrow >= 0 && j < d) ? static_cast<uint32_t>((xrow * d + j) * 4) : kOutOfRange;
      As[l_k][l_x + e] = buf_f32(xs, xo);
      const int nn = n0 + l_x + e;
      const uint32_t ro = (b < B && nn < C) ? static_cast<uint32_t>(((int64_t)b * C + nn) * 4) : kOutOfRange;
      Bs[l_k][l_x + e] = buf_f32(rs, ro);
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GBK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        av[e] = As[kk][ty * 4 + e];
        bv[e] = Bs[kk][tx * 4 + e];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(av[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int j = j0 + ty * 4 + r;
    if (j >= d) continue;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int nn = n0 + tx * 4 + c;
      if (nn < C) a.G[(int64_t)i * P + (int64_t)j * C + nn] = acc[r][c];
    }
  }
  if (blockIdx.x == 0 && blockIdx.y == 0) {
    // loss_i = mean CE over the worker's rows (fixed order)
    float s = 0.f;
    for (int b = tid; b < B; b += 256) s += a.ce[(int64_t)i * B + b];
    sh[tid] = s;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
      if (tid < st) sh[tid] += sh[tid + st];
      __syncthreads();
    }
    if (tid == 0) a.loss[i] = sh[0] / static_cast<float>(B);
  }
}

template <int CP, int M, int T>
hipError_t launch_fused_t(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  constexpr int R = 4;
  const int64_t nb = (int64_t)a.n * p.slabs;
  const int64_t per_xcd = (nb + NXCD - 1) / NXCD;
  hipLaunchKernelGGL((k_softmax_fused<CP, M, T, R>), dim3(static_cast<unsigned>(per_xcd * NXCD)), dim3(T), 0, s,
                     a, p.slabs, p.rows_per_slab, per_xcd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.slabs == 1) return e;
  const int64_t P = (int64_t)a.d * a.C;
  const dim3 g2(static_cast<unsigned>((P + 1023) / 1024), static_cast<unsigned>(a.n));
  hipLaunchKernelGGL(k_slab_reduce, g2, dim3(256), 0, s, a, p.slabs);
  return hipGetLastError();
}

template <int CP>
hipError_t launch_fused_c(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  if (p.threads == 256) {
    switch (p.per_thread) {
      case 1: return launch_fused_t<CP, 1, 256>(p, a, s);
      case 2: return launch_fused_t<CP, 2, 256>(p, a, s);
      case 4: return launch_fused_t<CP, 4, 256>(p, a, s);
    }
  } else {
    switch (p.per_thread) {
      case 2: return launch_fused_t<CP, 2, 512>(p, a, s);
      case 4: return launch_fused_t<CP, 4, 512>(p, a, s);
      case 6: return launch_fused_t<CP, 6, 512>(p, a, s);
      case 8: return launch_fused_t<CP, 8, 512>(p, a, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace

SoftmaxPlan softmax_plan(int n, int B, int d, int C) {
  SoftmaxPlan p;
  int cp = C <= 4 ? 4 : C <= 10 ? 10 : C <= 16 ? 16 : 0;
  int T = d <= 1024 ? 256 : 512;
  int M = (d + T - 1) / T;
  if (T == 256) M = M <= 1 ? 1 : M <= 2 ? 2 : M <= 4 ? 4 : 0;
  else M = M <= 2 ? 2 : M <= 4 ? 4 : M <= 6 ? 6 : M <= 8 ? 8 : 0;
  // register budget: no spills for M <= 6 (C <= 10) and M <= 4 (C <= 16)
  if ((cp == 16 && M > 4) || (cp == 10 && M > 6)) M = 0;
  if (cp == 0 || M == 0) {
    p.fused = 0;
    return p;
  }
  p.fused = 1;
  p.threads = T;
  p.per_thread = M;
  p.cpad = cp;
  // fill the chip: about 256 blocks, at least two 4-row chunks per slab
  int slabs = 256 / n;
  int max_slabs = B / 8;
  slabs = slabs < 1 ? 1 : slabs;
  max_slabs = max_slabs < 1 ? 1 : max_slabs;
  slabs = slabs > max_slabs ? max_slabs : slabs;
  p.slabs = slabs;
  p.rows_per_slab = (B + slabs - 1) / slabs;
  // round rows per slab up to the 4-row chunk
  p.rows_per_slab = (p.rows_per_slab + 3) / 4 * 4;
  if (p.rows_per_slab > 1024) p.rows_per_slab = 1024;   // rows staged in LDS
  p.slabs = (B + p.rows_per_slab - 1) / p.rows_per_slab;
  // one worker's partials are read through one buffer resource
  if ((int64_t)p.slabs * d * C * 4 > kMaxBufferBytes) p.fused = 0;
  return p;
}

hipError_t launch_softmax_grads(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  if (p.fused) {
    switch (p.cpad) {
      case 4: return launch_fused_c<4>(p, a, s);
      case 10: return launch_fused_c<10>(p, a, s);
      case 16: return launch_fused_c<16>(p, a, s);
    }
    return hipErrorInvalidValue;
  }
  const int64_t Mrows = (int64_t)a.n * a.B;
  dim3 g1((a.C + GBN - 1) / GBN, static_cast<unsigned>((Mrows + GBM - 1) / GBM));
  hipLaunchKernelGGL(k_logits_gemm, g1, dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rows_softmax, dim3(static_cast<unsigned>((Mrows + 3) / 4)), dim3(256), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g3((a.C + GBN - 1) / GBN, (a.d + GBM - 1) / GBM, a.n);
  hipLaunchKernelGGL(k_grads_gemm, g3, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dbw
