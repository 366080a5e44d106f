// Worker minibatch gradients of the two-layer ReLU MLP (Sect. 2, Eq. gradient), gfx950.
//
// For worker i with rows x_b (b < B), parameters [W1 (d x H) | b1 | W2 (H x C) | b2]:
//   A = X W1 + b1,  Hh = relu(A),  Z = Hh W2 + b2,  R = (softmax(Z) - Y) / B
//   dW2 = Hh^T R,  db2 = sum_b R,  dA = (R W2^T) * [A > 0],
//   dW1 = X^T dA,  db1 = sum_b dA,  loss = mean_b CE.
// ReLU'(0) = 0; [A > 0] is read from Hh > 0, which is the same predicate.
//
// Kernels (one stream, in order):
//  k_mlp_hidden  Hh for all n*B rows: an fp32 MFMA GEMM (v_mfma_f32_16x16x4f32)
//                over 64 x 64 output tiles, bias + ReLU in the epilogue.
//  k_mlp_head    per (worker, slab of rows): logits from Hh and W2 held in
//                registers (thread = hidden unit), LDS reduction, softmax in
//                wave 0, then dA rows and the slab partials of db1 | dW2 | db2.
//  k_mlp_dw1     per worker: dW1 = X_i^T dA_i, fp32 MFMA GEMM, K = B; an
//                extra grid row sums the head's slab partials into
//                G[i][d*H ...] (fixed order) and the loss.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "dbw_buffer.h"
#include "dbw_internal.h"
#include "mfma_gemm.h"

namespace dbw {
namespace {

constexpr int WAVE = 64;
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int64_t mlp_row(const MlpArgs& a, int i, int b, bool report) {
  const int64_t m = (int64_t)i * a.B + b;
  if (!a.rows) return m;
  const int64_t r = a.rows[m];
  if (r < 0 || r >= a.S) {
    if (report) atomicOr(a.err, ERR_ROW_RANGE);
    return 0;
  }
  return r;
}

// A label loaded by the caller, range-checked (bad labels are reported and
// read as class 0).
__device__ __forceinline__ int checked_label(const MlpArgs& a, int lab) {
  if (lab < 0 || lab >= a.C) {
    atomicOr(a.err, ERR_LABEL_RANGE);
    return 0;
  }
  return lab;
}

// ---------------------------------------------------------------------------
// MFMA tile: block 256 threads = 4 waves in 2 x 2, each wave 32 x 32 output
// (2 x 2 MFMA 16 x 16 tiles); K staged through LDS 16 at a time.
// Lane layout of v_mfma_f32_16x16x4f32 (wave64): A operand lane l holds
// A[l % 16][l / 16]; B operand lane l holds B[l / 16][l % 16]; accumulator
// element e of lane l is D[4 (l / 16) + e][l % 16].
constexpr int TM = 64, TN = 64, TK = 16;

__device__ __forceinline__ void mfma_tile_step(const float (&As)[TK][TM + 4], const float (&Bs)[TK][TN + 4],
                                               int wm, int wn, int lane, floatx4 (&acc)[2][2]) {
#pragma unroll
  for (int kk = 0; kk < TK; kk += 4) {
    float av[2], bv[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      av[t] = As[kk + lane / 16][wm * 32 + t * 16 + lane % 16];
      bv[t] = Bs[kk + lane / 16][wn * 32 + t * 16 + lane % 16];
    }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mi], bv[ni], acc[mi][ni], 0, 0, 0);
  }
}

// Hh[m][h] = relu(sum_j X[row(m)][j] W1[j][h] + b1[h]), m < n*B.
__global__ __launch_bounds__(256) void k_mlp_hidden(MlpArgs a) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int wm = wv / 2, wn = wv % 2;
  const int64_t Mrows = (int64_t)a.n * a.B;
  const int64_t m0 = (int64_t)blockIdx.y * TM;
  const int n0 = blockIdx.x * TN;
  const int d = a.d, H = a.H;
  const int64_t xrows = a.rows ? a.S : Mrows;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t ws = make_rsrc(a.w, static_cast<uint32_t>((int64_t)d * H * 4));
  // loaders: A tile 64 rows x 16 k (row tid/4, k (tid%4)*4..+3); B tile 16 k x 64 (k tid/16, n (tid%16)*4..)
  const int la_m = tid / 4, la_k = (tid % 4) * 4;
  const int64_t am = m0 + la_m;
  int64_t arow = -1;
  if (am < Mrows) arow = mlp_row(a, static_cast<int>(am / a.B), static_cast<int>(am % a.B), la_k == 0);
  const int lb_k = tid / 16, lb_n = (tid % 16) * 4;
  floatx4 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < d; k0 += TK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int kk = k0 + la_k + e;
      As[la_k + e][la_m] = buf_f32(xs, (arow >= 0 && kk < d) ? static_cast<uint32_t>((arow * d + kk) * 4) : kOutOfRange);
      const int kb = k0 + lb_k, nn = n0 + lb_n + e;
      Bs[lb_k][lb_n + e] = buf_f32(ws, (kb < d && nn < H) ? static_cast<uint32_t>(((int64_t)kb * H + nn) * 4) : kOutOfRange);
    }
    __syncthreads();
    mfma_tile_step(As, Bs, wm, wn, lane, acc);
    __syncthreads();
  }
  const float* b1 = a.w + (int64_t)d * H;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int nn = n0 + wn * 32 + ni * 16 + lane % 16;
      if (nn >= H) continue;
      const float bias = b1[nn];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t m = m0 + wm * 32 + mi * 16 + 4 * (lane / 16) + e;
        if (m < Mrows) a.Hh[m * H + nn] = fmaxf(acc[mi][ni][e] + bias, 0.f);
      }
    }
}

// Matrix-core versions on (32 WT)^2 tiles (mfma_gemm.h), used when d and H
// are multiples of 4 and a worker's rows fit the LDS stage.
template <int WT>
__global__ __launch_bounds__(256) void k_mlp_hidden_mfma(MlpArgs a) {
  constexpr int BM = 32 * WT, NP = mfma_pieces<WT>();
  __shared__ MfmaLds<WT> L;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  const int64_t Mrows = (int64_t)a.n * a.B;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const int n0 = blockIdx.x * BM;
  const int d = a.d, H = a.H;
  const int64_t xrows = a.rows ? a.S : Mrows;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t ws = make_rsrc(a.w, static_cast<uint32_t>((int64_t)d * H * 4));
  int64_t xrow[NP];
#pragma unroll
  for (int s2 = 0; s2 < NP; ++s2) {
    const int q = tid + s2 * 256;
    const int64_t m = m0 + q / 4;
    xrow[s2] = -1;
    if (m < Mrows) xrow[s2] = mlp_row(a, static_cast<int>(m / a.B), static_cast<int>(m % a.B), (q % 4) == 0);
  }
  mfma_f32x4 acc[WT][WT];
  mfma_zero<WT>(acc);
  // with ksplit 2, block z takes one half of K (a multiple of 16) and leaves
  // its raw sums in Hh (z = 0) or dA (z = 1); the head adds them, b1 and the
  // ReLU (two addends: the same sum in either order)
  const int kh = a.ksplit == 2 ? (d / 2 + MBK - 1) / MBK * MBK : d;
  const int kbeg = static_cast<int>(blockIdx.z) * kh;
  // two slices in flight: hidden layer 23.2 -> 22.0 us at 2048 x 784 x 512,
  // 69.8 -> 61.9 us at 8000 x 800 x 500 (the X^T dA product, K = B, is
  // slower that way and keeps one)
  mfma_gemm_rows_w<WT, 2>(L, xs, xrow, d, ws, H, n0, acc, kbeg, min(d, kbeg + kh));
  const float* b1 = a.w + (int64_t)d * H;
  float* out = blockIdx.z == 0 ? a.Hh : a.dA;
#pragma unroll
  for (int nt = 0; nt < WT; ++nt) {
    const int h = n0 + wn * 16 * WT + nt * 16 + (lane & 15);
    if (h >= H) continue;
    const float bias = b1[h];
#pragma unroll
    for (int mt = 0; mt < WT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm * 16 * WT + mt * 16 + 4 * (lane >> 4) + r;
        if (m < Mrows) out[m * H + h] = a.ksplit == 2 ? acc[mt][nt][r] : fmaxf(acc[mt][nt][r] + bias, 0.f);
      }
  }
}

// G[i][d*H + e] = sum_q Gp[i][q][e] for e < len (fixed slab order) and the
// loss of worker i: the head's slab partials, summed by the extra grid row of
// the dW1 kernels (part `part` of `nparts` blocks of 256 threads), which run
// beside the X^T dA tiles and write a disjoint part of G.
__device__ __forceinline__ void mlp_tail_sum(const MlpArgs& a, int slabs, int64_t len, int i, int part, int nparts) {
  const int64_t P = a.ldG ? a.ldG : (int64_t)a.d * a.H + len;   // row stride of G
  const bool keep = !a.row_mask || a.row_mask[i];
  for (int64_t e = (int64_t)part * 256 + threadIdx.x; e < len; e += (int64_t)nparts * 256) {
    const float* src = a.Gp + (int64_t)i * slabs * len + e;
    float s = 0.f;
    for (int q0 = 0; q0 < slabs; q0 += 8) {
      // eight slabs' loads in flight, then added in slab order
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = q0 + u < slabs ? src[(int64_t)(q0 + u) * len] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (q0 + u < slabs) s += v[u];
    }
    if (keep) a.G[(int64_t)i * P + (int64_t)a.d * a.H + e] = s;
  }
  if (part == 0 && threadIdx.x == 0) {
    float s = 0.f;
    for (int q = 0; q < slabs; ++q) s += a.lossp[(int64_t)i * slabs + q];
    a.loss[i] = s / static_cast<float>(a.B);
  }
}

template <int WT>
__global__ __launch_bounds__(256) void k_mlp_dw1_mfma(MlpArgs a, int slabs, int64_t tail) {
  if (blockIdx.y == gridDim.y - 1) {
    mlp_tail_sum(a, slabs, tail, static_cast<int>(blockIdx.z), static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x));
    return;
  }
  constexpr int BM = 32 * WT;
  __shared__ MfmaLds<WT> L;
  __shared__ int sh_row[1024];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  const int i = blockIdx.z;
  const int j0 = blockIdx.y * BM, n0 = blockIdx.x * BM;
  const int d = a.d, H = a.H, B = a.B;
  const int64_t P = a.ldG ? a.ldG : (int64_t)d * H + H + (int64_t)H * a.C + a.C;   // row stride of G
  const int64_t xrows = a.rows ? a.S : (int64_t)a.n * B;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t das = make_rsrc(a.dA + (int64_t)i * B * H, static_cast<uint32_t>((int64_t)B * H * 4));
  for (int b = tid; b < B; b += 256) sh_row[b] = static_cast<int>(mlp_row(a, i, b, false));
  __syncthreads();
  mfma_f32x4 acc[WT][WT];
  mfma_zero<WT>(acc);
  mfma_gemm_xt_r<WT>(L, xs, sh_row, d, j0, das, B, H, n0, acc);
  float* Gi = a.G + (int64_t)i * P;
#pragma unroll
  for (int mt = 0; mt < WT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = j0 + wm * 16 * WT + mt * 16 + 4 * (lane >> 4) + r;
      if (j >= d) continue;
#pragma unroll
      for (int nt = 0; nt < WT; ++nt) {
        const int h = n0 + wn * 16 * WT + nt * 16 + (lane & 15);
        if (h < H && (!a.row_mask || a.row_mask[i])) Gi[(int64_t)j * H + h] = acc[mt][nt][r];
      }
    }
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Max / sum over the 16 lanes of a DPP row: butterflies (xor 1, xor 2, half
// mirror, mirror) that leave the identical value in every lane of the row.
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  return fmaxf(v, dpp<0x140>(v));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  return v + dpp<0x140>(v);
}

// ---------------------------------------------------------------------------
// Head: thread j < H owns hidden unit j (T == H rounded up to a wave multiple
// is handled by the plan: T threads cover H with M units each).
template <int CP, int M, int T>
__global__ __launch_bounds__(T) void k_mlp_head(MlpArgs a, int slabs, int rps, int64_t L) {
  constexpr int R = 4;
  constexpr int V = R * CP;
  constexpr int G = T / V;
  static_assert(G >= 1 && CP <= 16, "head layout");
  __shared__ float red[T][V + 1];
  __shared__ float red2[G][V];
  __shared__ float rr[V];
  __shared__ float sh_loss[R];
  __shared__ float sh_db2[R][CP];
  __shared__ int sh_lab[1024];
  const int i = blockIdx.x / slabs, q = blockIdx.x % slabs;
  const int tid = threadIdx.x;
  const int H = a.H, C = a.C, d = a.d;
  const int b0 = q * rps, b1 = min(a.B, b0 + rps), nrows = b1 - b0;
  // Nothing waits on the row indices but the labels, and nothing on the
  // labels until the first softmax: the indices are loaded first, then the
  // first rows and W2, then the labels, which are checked and staged in LDS
  // before the first step's first barrier.
  constexpr int LPT = (1024 + T - 1) / T;   // slab rows per thread
  int64_t rowv[LPT];
#pragma unroll
  for (int k = 0; k < LPT; ++k) {
    const int r = tid + k * T;
    rowv[k] = r < nrows ? mlp_row(a, i, b0 + r, false) : 0;
  }
  const int64_t hrow0 = (int64_t)i * a.B;
  // rows cb .. cb + R - 1 as loaded: the activations, or with ksplit 2 the
  // two K halves' sums (the second half sits in dA; this thread writes a
  // row's dA entries only after it has read them).  The next rows are
  // loaded one step ahead, so their latency overlaps a step's reductions.
  auto load_rows = [&](int cb, float (&h1)[R][M], float (&h2)[R][M]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const bool ok = cb + r < nrows;
      const int64_t hoff = (hrow0 + b0 + (ok ? cb + r : 0)) * H;
      const __amdgpu_buffer_rsrc_t hs = make_rsrc(a.Hh + hoff, ok ? static_cast<uint32_t>(H * 4) : 0u);
      const __amdgpu_buffer_rsrc_t hd = make_rsrc(a.dA + hoff, ok && a.ksplit == 2 ? static_cast<uint32_t>(H * 4) : 0u);
#pragma unroll
      for (int m = 0; m < M; ++m) {
        h1[r][m] = buf_f32(hs, static_cast<uint32_t>((tid + m * T) * 4));
        h2[r][m] = buf_f32(hd, static_cast<uint32_t>((tid + m * T) * 4));
      }
    }
  };
  float h1[R][M], h2[R][M];
  load_rows(0, h1, h2);
  const float* W2 = a.w + (int64_t)d * H + H;
  const float* bias2 = W2 + (int64_t)H * C;
  const __amdgpu_buffer_rsrc_t w2s = make_rsrc(W2, static_cast<uint32_t>((int64_t)H * C * 4));
  float wr[M][CP], gw2[M][CP], gb1[M], b1v[M];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int j = tid + m * T;
    gb1[m] = 0.f;
    b1v[m] = j < H ? a.w[(int64_t)d * H + j] : 0.f;
#pragma unroll
    for (int c = 0; c < CP; ++c) {
      wr[m][c] = buf_f32(w2s, c < C ? static_cast<uint32_t>((j * C + c) * 4) : kOutOfRange);
      gw2[m][c] = 0.f;
    }
  }
  float loss_acc = 0.f, db2_acc = 0.f;
  const float invB = 1.0f / static_cast<float>(a.B);
  int labv[LPT];
#pragma unroll
  for (int k = 0; k < LPT; ++k) labv[k] = tid + k * T < nrows ? a.y[rowv[k]] : 0;
  for (int cb = 0; cb < nrows; cb += R) {
    float x[R][M];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < M; ++m) x[r][m] = a.ksplit == 2 ? fmaxf(h1[r][m] + h2[r][m] + b1v[m], 0.f) : h1[r][m];
    if (cb + R < nrows) load_rows(cb + R, h1, h2);
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int c = 0; c < CP; ++c) {
        float z = 0.f;
#pragma unroll
        for (int m = 0; m < M; ++m) z = fmaf(x[r][m], wr[m][c], z);
        red[tid][r * CP + c] = z;
      }
    if (cb == 0) {
#pragma unroll
      for (int k = 0; k < LPT; ++k)
        if (tid + k * T < nrows) sh_lab[tid + k * T] = checked_label(a, labv[k]);
    }
    __syncthreads();
    if (tid < V * G) {
      // four interleaved partial sums keep four LDS reads in flight
      const int v = tid % V, g = tid / V;
      float s4[4] = {0.f, 0.f, 0.f, 0.f};
      int t = g;
      for (; t + 3 * G < T; t += 4 * G) {
#pragma unroll
        for (int u = 0; u < 4; ++u) s4[u] += red[t + u * G][v];
      }
#pragma unroll
      for (int u = 0; u < 3; ++u)
        if (t + u * G < T) s4[u] += red[t + u * G][v];
      red2[g][v] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
    }
    __syncthreads();
    if (tid < WAVE) {
      const int r = tid / 16, c = tid % 16;
      const int rb = cb + r;
      float z = 0.f;
      if (c < CP) {
#pragma unroll
        for (int g = 0; g < G; ++g) z += red2[g][r * CP + c];
      }
      const bool valid = c < C;
      if (valid) z += bias2[c];
      const float zmax = row16_max(valid ? z : -INFINITY);
      const float sh = z - zmax;
      const float e = valid ? expf(sh) : 0.f;
      const float se = row16_sum(e);
      const bool row_ok = rb < nrows;
      const int lab = row_ok ? sh_lab[rb] : 0;
      const float zy = __shfl(sh, r * 16 + lab, WAVE);
      const float res = row_ok ? (e / se - (c == lab ? 1.f : 0.f)) * invB : 0.f;
      if (c < CP) rr[r * CP + c] = res;
      db2_acc += (c < C) ? res : 0.f;
      if (c == 0 && row_ok) loss_acc += logf(se) - zy;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float rv[CP];
#pragma unroll
      for (int c = 0; c < CP; ++c) rv[c] = rr[r * CP + c];
      const bool ok = cb + r < nrows;
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const int j = tid + m * T;
        float dh = 0.f;
#pragma unroll
        for (int c = 0; c < CP; ++c) {
          dh = fmaf(rv[c], wr[m][c], dh);
          gw2[m][c] = fmaf(x[r][m], rv[c], gw2[m][c]);
        }
        const float da = x[r][m] > 0.f ? dh : 0.f;
        gb1[m] += da;
        if (ok && j < H) a.dA[(hrow0 + b0 + cb + r) * H + j] = da;
      }
    }
  }
  if (tid < WAVE) {
    const int r = tid / 16, c = tid % 16;
    if (c == 0) sh_loss[r] = loss_acc;
    if (c < CP) sh_db2[r][c] = db2_acc;
  }
  __syncthreads();
  // slab partial, laid out like G's tail: [db1 (H) | dW2 (H x C) | db2 (C)],
  // assembled in the LDS of the reduction and written in 8-byte pieces (a
  // thread's C classes are C floats apart from the next thread's)
  static_assert(M * T + M * T * CP + CP <= T * (V + 1), "slab partial fits the reduction LDS");
  float* stage = &red[0][0];
#pragma unroll
  for (int m = 0; m < M; ++m) {
    const int j = tid + m * T;
    if (j < H) {
      stage[j] = gb1[m];
#pragma unroll
      for (int c = 0; c < CP; ++c)
        if (c < C) stage[H + j * C + c] = gw2[m][c];
    }
  }
  if (tid < C) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r) s += sh_db2[r][tid];
    stage[H + H * C + tid] = s;
  }
  if (tid == 0) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < R; ++r) s += sh_loss[r];
    a.lossp[(int64_t)i * slabs + q] = s;
  }
  __syncthreads();
  float* gp = a.Gp + ((int64_t)i * slabs + q) * L;
  const int len = static_cast<int>(L);
  if ((len & 1) == 0) {
    // L even: every slab's partial starts 8-byte aligned
    for (int k = tid; k < len / 2; k += T)
      reinterpret_cast<float2*>(gp)[k] = make_float2(stage[2 * k], stage[2 * k + 1]);
  } else {
    for (int k = tid; k < len; k += T) gp[k] = stage[k];
  }
}

// dW1[j][h] = sum_b X[row(i,b)][j] dA[i*B + b][h]; blockIdx.z = worker; the
// last grid row sums the head's slab partials.
__global__ __launch_bounds__(256) void k_mlp_dw1(MlpArgs a, int slabs, int64_t tail) {
  if (blockIdx.y == gridDim.y - 1) {
    mlp_tail_sum(a, slabs, tail, static_cast<int>(blockIdx.z), static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x));
    return;
  }
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tid = threadIdx.x, lane = tid % WAVE, wv = tid / WAVE;
  const int wm = wv / 2, wn = wv % 2;
  const int i = blockIdx.z;
  const int j0 = blockIdx.y * TM;
  const int n0 = blockIdx.x * TN;
  const int d = a.d, H = a.H, B = a.B;
  const int64_t P = a.ldG ? a.ldG : (int64_t)d * H + H + (int64_t)H * a.C + a.C;   // row stride of G
  const int64_t xrows = a.rows ? a.S : (int64_t)a.n * B;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t das = make_rsrc(a.dA + (int64_t)i * B * H, static_cast<uint32_t>((int64_t)B * H * 4));
  const int l_k = tid / 16, l_x = (tid % 16) * 4;
  floatx4 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < B; k0 += TK) {
    const int b = k0 + l_k;
    const int64_t xrow = b < B ? mlp_row(a, i, b, false) : -1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = j0 + l_x + e;
      As[l_k][l_x + e] = buf_f32(xs, (xrow >= 0 && j < d) ? static_cast<uint32_t>((xrow * d + j) * 4) : kOutOfRange);
      const int nn = n0 + l_x + e;
      Bs[l_k][l_x + e] = buf_f32(das, (b < B && nn < H) ? static_cast<uint32_t>(((int64_t)b * H + nn) * 4) : kOutOfRange);
    }
    __syncthreads();
    mfma_tile_step(As, Bs, wm, wn, lane, acc);
    __syncthreads();
  }
  float* Gi = a.G + (int64_t)i * P;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const int nn = n0 + wn * 32 + ni * 16 + lane % 16;
      if (nn >= H) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = j0 + wm * 32 + mi * 16 + 4 * (lane / 16) + e;
        if (j < d && (!a.row_mask || a.row_mask[i])) Gi[(int64_t)j * H + nn] = acc[mi][ni][e];
      }
    }
}

template <int CP, int M, int T>
hipError_t launch_head(const MlpPlan& p, const MlpArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_mlp_head<CP, M, T>), dim3(static_cast<unsigned>(a.n * p.slabs)), dim3(T), 0, s, a,
                     p.slabs, p.rows_per_slab, p.tail);
  return hipGetLastError();
}

}  // namespace

MlpPlan mlp_plan(int n, int B, int d, int H, int C) {
  MlpPlan p;
  p.tail = (int64_t)H + (int64_t)H * C + C;
  p.cpad = C <= 4 ? 4 : C <= 10 ? 10 : C <= 16 ? 16 : 0;
  p.threads = H <= 256 ? 256 : 512;
  p.per_thread = (H + p.threads - 1) / p.threads;
  if (p.cpad == 0 || p.per_thread > 2 || (p.cpad == 16 && p.per_thread > 1)) return p;   // ok = 0
  int slabs = 256 / n;
  int max_slabs = B / 8;
  slabs = slabs < 1 ? 1 : slabs;
  max_slabs = max_slabs < 1 ? 1 : max_slabs;
  slabs = slabs > max_slabs ? max_slabs : slabs;
  p.rows_per_slab = (B + slabs - 1) / slabs;
  p.rows_per_slab = (p.rows_per_slab + 3) / 4 * 4;
  if (p.rows_per_slab > 1024) p.rows_per_slab = 1024;
  p.slabs = (B + p.rows_per_slab - 1) / p.rows_per_slab;
  p.ok = 1;
  return p;
}

hipError_t launch_mlp_grads(const MlpPlan& p, const MlpArgs& args, hipStream_t s) {
  if (!p.ok) return hipErrorNotSupported;
  MlpArgs a = args;
  a.ksplit = 1;
  const int64_t Mrows = (int64_t)a.n * a.B;
  const bool big = a.d % 4 == 0 && a.H % 4 == 0 && a.B <= 1024;
  const int64_t small_tiles = (int64_t)((a.H + 63) / 64) * ((Mrows + 63) / 64);
  if (big && (int64_t)((a.H + 127) / 128) * ((Mrows + 127) / 128) >= kMfmaBigTiles) {
    hipLaunchKernelGGL(k_mlp_hidden_mfma<4>, dim3((a.H + 127) / 128, static_cast<unsigned>((Mrows + 127) / 128)),
                       dim3(256), 0, s, a);
  } else if (big) {
    // too few 64 x 64 tiles for two blocks per CU: split K in two halves
    if (small_tiles < kMfmaBigTiles && a.d >= 2 * MBK) a.ksplit = 2;
    hipLaunchKernelGGL(k_mlp_hidden_mfma<2>,
                       dim3((a.H + 63) / 64, static_cast<unsigned>((Mrows + 63) / 64), a.ksplit), dim3(256), 0, s, a);
  }
  else
    hipLaunchKernelGGL(k_mlp_hidden, dim3((a.H + TN - 1) / TN, static_cast<unsigned>((Mrows + TM - 1) / TM)),
                       dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (p.cpad * 100 + p.per_thread * 10 + (p.threads == 512)) {
    case 410: e = launch_head<4, 1, 256>(p, a, s); break;
    case 420: e = launch_head<4, 2, 256>(p, a, s); break;
    case 411: e = launch_head<4, 1, 512>(p, a, s); break;
    case 421: e = launch_head<4, 2, 512>(p, a, s); break;
    case 1010: e = launch_head<10, 1, 256>(p, a, s); break;
    case 1020: e = launch_head<10, 2, 256>(p, a, s); break;
    case 1011: e = launch_head<10, 1, 512>(p, a, s); break;
    case 1021: e = launch_head<10, 2, 512>(p, a, s); break;
    case 1610: e = launch_head<16, 1, 256>(p, a, s); break;
    case 1611: e = launch_head<16, 1, 512>(p, a, s); break;
    default: return hipErrorNotSupported;
  }
  if (e != hipSuccess) return e;
  // X_i^T dA_i contracts over the worker's B rows only: with few rows the
  // large tile's operand reuse buys little, and the short blocks of 64 x 64
  // tiles overlap one another's stores with their matrix work (MLP 32 x 64:
  // 75.7 -> 73.0 us per launch)
  // (one extra grid row sums the head's slab partials into the tail of G)
  if (big && a.B >= 256 && (int64_t)((a.H + 127) / 128) * ((a.d + 127) / 128) * a.n >= kMfmaBigTiles)
    hipLaunchKernelGGL(k_mlp_dw1_mfma<4>, dim3((a.H + 127) / 128, (a.d + 127) / 128 + 1, a.n), dim3(256), 0, s, a,
                       p.slabs, p.tail);
  else if (big)
    hipLaunchKernelGGL(k_mlp_dw1_mfma<2>, dim3((a.H + 63) / 64, (a.d + 63) / 64 + 1, a.n), dim3(256), 0, s, a,
                       p.slabs, p.tail);
  else
    hipLaunchKernelGGL(k_mlp_dw1, dim3((a.H + TN - 1) / TN, (a.d + TM - 1) / TM + 1, a.n), dim3(256), 0, s, a,
                       p.slabs, p.tail);
  return hipGetLastError();
}

}  // namespace dbw
