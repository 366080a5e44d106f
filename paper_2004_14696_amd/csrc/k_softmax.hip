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
#include <type_traits>

#include "dbw_buffer.h"
#include "dbw_internal.h"
#include "mfma_gemm.h"

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

// A label loaded by the caller, range-checked as in sample_label.
__device__ __forceinline__ int checked_label(const SoftmaxArgs& a, int lab) {
  if (lab < 0 || lab >= a.C) {
    atomicOr(a.err, ERR_LABEL_RANGE);
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
      if (j < d && (!a.row_mask || a.row_mask[i]))
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

// ---------------------------------------------------------------------------
// Matrix-core variant of the single pass (C <= 16, d % 4 == 0, d <= 3072).
//
// Eight waves split the feature dimension; wave w owns features
// w*64U + 64u + 4m + j (u < U, m < 16, j < 4).  Rows stream through in
// chunks of 8; lane (m, g) = (lane % 16, lane / 16) holds the float4
// X[row g + 4e][w*64U + 64u + 4m .. +3] for e = 0, 1 -- exactly the A
// operand of a 16x16x4 MFMA whose k index runs over rows and whose m index
// runs over 16 features.  So the gradient G_i += X^T R (contraction over
// rows) is a chain of MFMAs on the loaded registers, accumulated in 16U
// tiles of 16 features x 16 classes.  The logits (contraction over
// features, which sit on lane % 16) are computed on the vector ALUs: each
// lane dots its 4U features of a row with W (staged once per block in LDS,
// in lane order), a 16-lane DPP reduction sums the row group, and the eight
// waves' partials meet in LDS.  After one block barrier every wave sums the
// partials of the rows its lanes hold and runs their softmax (16-lane DPP
// max and sum), so lane (m, g) forms r[row g + 4e][class m] itself -- the
// B operand of the same MFMAs.  One block barrier per chunk.
constexpr int MF_WAVES = 8;
constexpr int MF_T = MF_WAVES * WAVE;
constexpr int MF_ROWS = 8;
static_assert(MF_ROWS == 8, "lane (m, g) holds rows g and g + 4 of a chunk");

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Sum / max over the 16 lanes of a DPP row; butterfly pairs (xor 1, xor 2,
// half-mirror, mirror) leave the identical value in all 16 lanes.
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  return v;
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return v;
}

__device__ __forceinline__ float f4_at(const float4& v, int j) {
  return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int U, int CW>
__global__ __launch_bounds__(MF_T) void k_softmax_mfma(SoftmaxArgs a, int slabs, int rps, int64_t per_xcd) {
  static_assert(CW % 2 == 0 && CW <= 16, "class padding");
  // W in lane order: lane (w, m) reads its 4U features x CW classes from one
  // contiguous run (features w 64U + 64u + 4m + j at (4u + j) CW); with the
  // run length SL = 4 U CW + 2 floats, SL / 2 is odd, so the 16 distinct
  // 8-byte reads of a row group fall on distinct bank pairs of the 32 banks
  // (runs start 8-byte aligned, so W is staged with 8-byte stores).  The same
  // LDS later assembles the block's slice of G ([d][C]).
  constexpr int SL = 4 * U * CW + 2;
  constexpr int WS = MF_WAVES * 16 * SL;
  __shared__ __attribute__((aligned(16))) float Ws[WS];
  __shared__ __attribute__((aligned(16))) float zb[2][MF_WAVES][MF_ROWS][16];  // per-wave partial logits
  __shared__ int sh_row[FUSED_MAX_ROWS];
  __shared__ int sh_lab[FUSED_MAX_ROWS];

  const int64_t logical = xcd_logical(blockIdx.x, per_xcd);
  if (logical >= (int64_t)a.n * slabs) return;
  const int i = static_cast<int>(logical / slabs);
  const int q = static_cast<int>(logical % slabs);
  const int tid = threadIdx.x;
  const int lane = tid & (WAVE - 1), w = tid >> 6;
  const int m = lane & 15, g = lane >> 4;
  const int d = a.d, C = a.C;
  const int64_t P = (int64_t)d * C;
  const int b0 = q * rps;
  const int nrows = min(a.B, b0 + rps) - b0;

  // The chain to the first products is the row indices, then the rows: the
  // indices are loaded first, then W (coalesced float4 pieces, P % 4 == 0
  // since d % 4 == 0), then the labels, which are checked and staged only
  // after the first rows are on their way (the wait for a load also waits
  // for every load issued before it, so the labels go out before the rows).
  constexpr int RPT = FUSED_MAX_ROWS / MF_T;   // slab rows per thread
  int64_t rowv[RPT];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int r = tid + k * MF_T;
    rowv[k] = r < nrows ? sample_row(a, i, b0 + r, true) : 0;
  }
  const int n4 = static_cast<int>(P / 4);
  constexpr int KMAX = (MF_T * U * CW / 4 + MF_T - 1) / MF_T;   // P <= 512 U CW
  float4 wl[KMAX];
  {
    const __amdgpu_buffer_rsrc_t wrs = make_rsrc(a.W, static_cast<uint32_t>(P * 4));
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const int e4 = tid + k * MF_T;
      wl[k] = buf_f32x4(wrs, e4 < n4 ? static_cast<uint32_t>(e4 * 16) : kOutOfRange);
    }
  }
  float4* w4 = reinterpret_cast<float4*>(Ws);
  if (d < MF_T * U) {
    // slots of features past d must read as 0 (their rows carry finite values
    // of the same row)
    for (int k = tid; k < WS / 4; k += MF_T) w4[k] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  int labv[RPT];
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int r = tid + k * MF_T;
    labv[k] = 0;
    if (r < nrows) {
      sh_row[r] = static_cast<int>(rowv[k]);
      labv[k] = a.y[rowv[k]];
    }
  }
  __syncthreads();

  const int64_t xrows = a.rows ? a.S : (int64_t)a.n * a.B;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const int fbase = w * 64 * U + 4 * m;
  // byte offset of row cb + g + 4e of the slab, or kOutOfRange past the slab
  auto row_off = [&](int cb, int e) -> uint32_t {
    const int r = cb + g + 4 * e;
    const int rc = r < nrows ? r : 0;
    const int64_t row = a.rows ? (int64_t)sh_row[rc] : (int64_t)i * a.B + b0 + rc;
    return r < nrows ? static_cast<uint32_t>(row * d * 4) : kOutOfRange;
  };
  // this lane's float4 of group u of a row.  A group past d reads features
  // 0..3 of the same row instead: its W entries are 0 and its gradient rows
  // are never stored, so only the row's own values enter (no bounds select
  // per load; kOutOfRange + 12 KiB stays out of range).
  auto load_u = [&](uint32_t roff, int u) -> float4 {
    const int f = fbase + 64 * u;
    return buf_f32x4(xr, roff + (f < d ? static_cast<uint32_t>(f * 4) : 0u));
  };
  float4 xa[2][U], xb[2][U];   // two chunks in flight, roles alternate
  {
    const uint32_t r0 = row_off(0, 0), r1 = row_off(0, 1);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      xa[0][u] = load_u(r0, u);
      xa[1][u] = load_u(r1, u);
    }
  }
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int r = tid + k * MF_T;
    if (r < nrows) sh_lab[r] = checked_label(a, labv[k]);
  }

  // Stage W.  Features 4h .. 4h+3 (group h = w' 16U + 16u + m') are 4C
  // contiguous elements of W and 4CW contiguous floats of run (w', m') at
  // 4u CW, so with C == CW a float4 of W lands as two float2 stores.
  {
    // float index in Ws of element r of group h's 4CW floats
    auto slot = [](int h, int r) { return ((h / (16 * U)) * 16 + h % 16) * SL + ((h % (16 * U)) / 16) * 4 * CW + r; };
    if (C == CW) {
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        const int e = 4 * (tid + k * MF_T);
        if (e < 4 * n4) {
          float2* w2 = reinterpret_cast<float2*>(Ws) + slot(e / (4 * CW), e % (4 * CW)) / 2;
          w2[0] = make_float2(wl[k].x, wl[k].y);
          w2[1] = make_float2(wl[k].z, wl[k].w);
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        const int e4 = tid + k * MF_T;
        if (e4 < n4) {
          int f = (4 * e4) / C, c = 4 * e4 - f * C;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            Ws[slot(f / 4, (f % 4) * CW + c)] = f4_at(wl[k], q);
            if (++c == C) {
              c = 0;
              ++f;
            }
          }
        }
      }
    }
  }
  __syncthreads();

  f32x4 acc[U][4];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[u][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float loss_acc = 0.f;
  const float invB = 1.0f / static_cast<float>(a.B);
  const bool cls_ok = m < C;
  const int nch = (nrows + MF_ROWS - 1) / MF_ROWS;
  float rv[2];   // residuals of the chunk whose MFMAs run next

  // Partial logits of rows g, g + 4 over this lane's 4U features.  wl0 is
  // this lane's W run.  The W reads run one feature ahead of the FMAs, and
  // the empty asm statements pin every step in place: left alone, the
  // compiler would hoist all 4U x CW reads to the front and hold them in
  // registers that the row buffers need.
  auto logits = [&](const float4 (&x)[2][U], float (&z)[2][CW], const float* wl0) {
    float wc[CW], wn[CW];
    auto read_w = [&](int t, float (&wv)[CW]) {
      const float2* wp = reinterpret_cast<const float2*>(wl0 + t * CW);
#pragma unroll
      for (int c2 = 0; c2 < CW / 2; ++c2) {
        const float2 v = wp[c2];
        wv[2 * c2] = v.x;
        wv[2 * c2 + 1] = v.y;
      }
    };
    read_w(0, wc);
#pragma unroll
    for (int t = 0; t < 4 * U; ++t) {
      if (t + 1 < 4 * U) read_w(t + 1, wn);
      const float x0 = f4_at(x[0][t / 4], t % 4), x1 = f4_at(x[1][t / 4], t % 4);
#pragma unroll
      for (int c = 0; c < CW; ++c) {
        z[0][c] = fmaf(x0, wc[c], z[0][c]);
        z[1][c] = fmaf(x1, wc[c], z[1][c]);
      }
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int c = 0; c < CW; ++c) asm volatile("" : "+v"(z[e][c]));
      asm volatile("" ::: "memory");
#pragma unroll
      for (int c = 0; c < CW; ++c) wc[c] = wn[c];
    }
  };
  // Sum the partial logits over the 16-lane row group; lane m == 0 stores
  // the wave's partials for the block (zb[buf]).
  auto reduce_logits = [&](float (&z)[2][CW], int buf) {
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int c = 0; c < CW; ++c) z[e][c] += dpp<0xB1>(z[e][c]);
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int c = 0; c < CW; ++c) z[e][c] += dpp<0x4E>(z[e][c]);
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int c = 0; c < CW; ++c) z[e][c] += dpp<0x141>(z[e][c]);
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int c = 0; c < CW; ++c) z[e][c] += dpp<0x140>(z[e][c]);
    if (m == 0) {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        float2* zp = reinterpret_cast<float2*>(&zb[buf][w][g + 4 * e][0]);
#pragma unroll
        for (int c2 = 0; c2 < CW / 2; ++c2) zp[c2] = make_float2(z[e][2 * c2], z[e][2 * c2 + 1]);
      }
    }
  };
  // After the barrier: the softmax of the chunk's rows from the eight waves'
  // partials, residuals into rv, cross entropy into the label's lane.
  auto softmax = [&](int cb, int buf) {
    // lane (m, g): rows g and g + 4 of the chunk, class m.  Every wave forms
    // the residuals it needs from the eight waves' partials (the same
    // arithmetic in every wave), so no second barrier; wave 0 keeps the
    // cross entropy.
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int r = cb + g + 4 * e;
      const bool row_ok = r < nrows;
      float zt = 0.f;
#pragma unroll
      for (int v = 0; v < MF_WAVES; ++v) zt += zb[buf][v][g + 4 * e][m];
      const float mx = row16_max(cls_ok ? zt : -INFINITY);
      const float ex = cls_ok ? __expf(zt - mx) : 0.f;
      const float se = row16_sum(ex);
      const int lab = sh_lab[row_ok ? r : 0];
      const bool hit = row_ok && m == lab;
      const float p = ex * __builtin_amdgcn_rcpf(se);
      rv[e] = row_ok && cls_ok ? (p - (hit ? 1.f : 0.f)) * invB : 0.f;
      if (w == 0) loss_acc += hit ? __logf(se) - (zt - mx) : 0.f;
    }
  };
  // One chunk: logits of chunk cb (rows in A) while chunk cb + 8 streams
  // into B, the block-wide softmax, then G += X^T R on the matrix cores.
  auto step = [&](float4 (&A)[2][U], float4 (&B)[2][U], int cb) {
    float z[2][CW];
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int c = 0; c < CW; ++c) z[e][c] = 0.f;
    {
      const uint32_t rn = row_off(cb + MF_ROWS, 0);
#pragma unroll
      for (int u = 0; u < U; ++u) B[0][u] = load_u(rn, u);
    }
    logits(A, z, &Ws[(w * 16 + m) * SL]);
    const int buf = (cb / MF_ROWS) & 1;
    reduce_logits(z, buf);
    {
      // rows g + 4 of the next chunk once the logit registers are released
      const uint32_t rn = row_off(cb + MF_ROWS, 1);
#pragma unroll
      for (int u = 0; u < U; ++u) B[1][u] = load_u(rn, u);
    }
    __syncthreads();
    softmax(cb, buf);
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[u][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(f4_at(A[e][u], j), rv[e], acc[u][j], 0, 0, 0);
  };
  int c = 0;
  for (; c + 1 < nch; c += 2) {
    step(xa, xb, c * MF_ROWS);
    step(xb, xa, (c + 1) * MF_ROWS);
  }
  if (c < nch) step(xa, xb, c * MF_ROWS);

  // lane (m, g) holds tile rows 4g + t (features w 64U + 64u + 16g + 4t + j)
  // of class m.
  if (slabs > 1) {
    // slab partial in tile order: float4 (t = 0..3) of (w, u, j, g, m) at
    // ((((w U + u) 4 + j) 4 + g) C + m) 4; k_slab_reduce_tiles sums the slabs
    // and restores the [d][C] order
    if (cls_ok) {
      float4* part = reinterpret_cast<float4*>(a.Gp + ((int64_t)i * slabs + q) * (int64_t)(MF_T * U * C));
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          part[(((w * U + u) * 4 + j) * 4 + g) * C + m] = make_float4(acc[u][j][0], acc[u][j][1], acc[u][j][2], acc[u][j][3]);
    }
  } else {
    // the worker's G ([d][C], P contiguous floats) is assembled in the LDS
    // that held W and written out in float4 pieces
    __syncthreads();
    if (cls_ok) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int f = w * 64 * U + 64 * u + 16 * g + 4 * t + j;
            if (f < d) Ws[f * C + m] = acc[u][j][t];
          }
    }
    __syncthreads();
    const float4* s4 = reinterpret_cast<const float4*>(Ws);
    float4* o4 = reinterpret_cast<float4*>(a.G + (int64_t)i * P);
    if (!a.row_mask || a.row_mask[i])
      for (int k = tid; k < static_cast<int>(P / 4); k += MF_T) o4[k] = s4[k];
  }
  if (w == 0) {
    // the loss of every row sits in its label's lane of wave 0
    float l = loss_acc;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o);
    if (lane == 0) {
      if (slabs == 1) a.loss[i] = l * invB;
      else a.lossp[(int64_t)i * slabs + q] = l;
    }
  }
}

// Sum of the tile-order slab partials of the matrix-core kernel, in slab
// order.  Block (x, i): features 64x .. 64x + 63 of worker i, whose 64C
// partial floats of one slab are contiguous (wave w' = x / U, group
// u = x % U).  Summed float4 pieces are put back in [d][C] order through LDS.
__global__ __launch_bounds__(256) void k_slab_reduce_tiles(SoftmaxArgs a, int slabs, int U) {
  __shared__ __attribute__((aligned(16))) float tile[64 * 16];
  const int i = blockIdx.y, x = blockIdx.x;
  const int C = a.C, d = a.d;
  const int64_t P = (int64_t)d * C;
  const int64_t part = (int64_t)MF_T * U * C;
  const int n4 = 16 * C;   // float4 pieces of the 64 features
  for (int k = threadIdx.x; k < n4; k += 256) {
    // piece k = ((j 4 + g) C + m): features 16g + 4t + j (t = 0..3), class m
    const int m = k % C, jg = k / C, g = jg % 4, j = jg / 4;
    const float* src = a.Gp + (int64_t)i * slabs * part + (int64_t)x * 64 * C + 4 * k;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int q0 = 0; q0 < slabs; q0 += 8) {
      // up to eight slabs' pieces in flight, then added in slab order (a
      // plain loop over a run-time slab count waits for each load in turn)
      float4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[u] = q0 + u < slabs ? *reinterpret_cast<const float4*>(src + (q0 + u) * part) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (q0 + u < slabs) {
          s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w;
        }
    }
    tile[(16 * g + 0 + j) * C + m] = s.x;
    tile[(16 * g + 4 + j) * C + m] = s.y;
    tile[(16 * g + 8 + j) * C + m] = s.z;
    tile[(16 * g + 12 + j) * C + m] = s.w;
  }
  __syncthreads();
  const int f0 = x * 64;
  const int nf = min(64, d - f0);   // features past d are not stored
  float* dst = a.G + (int64_t)i * P + (int64_t)f0 * C;
  if (!a.row_mask || a.row_mask[i])
    for (int k = threadIdx.x; k < nf * C / 4; k += 256)
      reinterpret_cast<float4*>(dst)[k] = reinterpret_cast<const float4*>(tile)[k];
  if (x == 0 && threadIdx.x == 0) {
    float l = 0.f;
    for (int q = 0; q < slabs; ++q) l += a.lossp[(int64_t)i * slabs + q];
    a.loss[i] = l / static_cast<float>(a.B);
  }
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
  if (e0 < P && (!a.row_mask || a.row_mask[i])) {
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
      if (nn < C && (!a.row_mask || a.row_mask[i])) a.G[(int64_t)i * P + (int64_t)j * C + nn] = acc[r][c];
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

// ---------------------------------------------------------------------------
// Matrix-core fp32 GEMMs for the large-C path (C % 4 == 0, d % 4 == 0):
// 128 x 128 tiles, or 64 x 64 when the large tiles cannot fill the chip;
// main loops in mfma_gemm.h.

// Z[m][c] = sum_j X[row(m)][j] W[j][c]; blockIdx.x = class tile, y = row tile.
template <int WT>
__global__ __launch_bounds__(256) void k_logits_mfma(SoftmaxArgs a) {
  constexpr int BM = 32 * WT, NP = mfma_pieces<WT>();
  __shared__ MfmaLds<WT> L;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  const int64_t Mrows = (int64_t)a.n * a.B;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const int n0 = blockIdx.x * BM;
  const int d = a.d, C = a.C;
  const int64_t xrows = a.rows ? a.S : Mrows;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t ws = make_rsrc(a.W, static_cast<uint32_t>((int64_t)d * C * 4));
  int64_t xrow[NP];
#pragma unroll
  for (int s2 = 0; s2 < NP; ++s2) {
    const int q = tid + s2 * 256;
    const int64_t m = m0 + q / 4;
    xrow[s2] = -1;
    if (m < Mrows) xrow[s2] = sample_row(a, static_cast<int>(m / a.B), static_cast<int>(m % a.B), (q % 4) == 0);
  }
  mfma_f32x4 acc[WT][WT];
  mfma_zero<WT>(acc);
  mfma_gemm_rows_w<WT>(L, xs, xrow, d, ws, C, n0, acc);
#pragma unroll
  for (int mt = 0; mt < WT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t m = m0 + wm * 16 * WT + mt * 16 + 4 * (lane >> 4) + r;
      if (m >= Mrows) continue;
#pragma unroll
      for (int nt = 0; nt < WT; ++nt) {
        const int c = n0 + wn * 16 * WT + nt * 16 + (lane & 15);
        if (c < C) a.Z[m * C + c] = acc[mt][nt][r];
      }
    }
}

// G_i[j][c] = sum_b X[row(i,b)][j] R_i[b][c]; blockIdx.x = class tile,
// y = feature tile, z = worker.  Block (0, 0, i) also writes loss_i.
template <int WT>
__global__ __launch_bounds__(256) void k_grads_mfma(SoftmaxArgs a) {
  constexpr int BM = 32 * WT;
  __shared__ MfmaLds<WT> L;
  __shared__ int sh_row[FUSED_MAX_ROWS];
  __shared__ float sh[256];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  const int i = blockIdx.z;
  const int j0 = blockIdx.y * BM, n0 = blockIdx.x * BM;
  const int d = a.d, C = a.C, B = a.B;
  const int64_t P = (int64_t)d * C;
  const int64_t xrows = a.rows ? a.S : (int64_t)a.n * B;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.Z + (int64_t)i * B * C, static_cast<uint32_t>((int64_t)B * C * 4));
  for (int b = tid; b < B; b += 256) sh_row[b] = static_cast<int>(sample_row(a, i, b, false));
  __syncthreads();
  mfma_f32x4 acc[WT][WT];
  mfma_zero<WT>(acc);
  mfma_gemm_xt_r<WT>(L, xs, sh_row, d, j0, rs, B, C, n0, acc);
  // the G rows of workers outside the row mask are computed but not stored
  const bool write_g = !a.row_mask || a.row_mask[i];
#pragma unroll
  for (int mt = 0; mt < WT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = j0 + wm * 16 * WT + mt * 16 + 4 * (lane >> 4) + r;
      if (j >= d) continue;
#pragma unroll
      for (int nt = 0; nt < WT; ++nt) {
        const int c = n0 + wn * 16 * WT + nt * 16 + (lane & 15);
        if (c < C && write_g) a.G[(int64_t)i * P + (int64_t)j * C + c] = acc[mt][nt][r];
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

// ---------------------------------------------------------------------------
// Matrix-core path for 16 < C <= 16 NT (C % 4 == 0): the narrow-N loops of
// mfma_gemm.h put all classes of a row in one wave, so the row softmax runs
// in the logits kernel's registers (a 16-lane DPP row holds the row's
// classes) and the residuals are written once; then G_i = X_i^T R_i with
// blocks of 64 MT features x all classes.
constexpr int NARROW_MT = 2;

// Z[m][c] = (softmax(x_m W)_c - [c = y_m]) / B, ce[m] = CE of row m;
// blockIdx.x = tile of 64 MT rows.  RS > 0: C = 16 (NT - 1) + 4 RS, the last
// tile in 4-wide stripes.
template <int MT, int NT, int RS>
__global__ __launch_bounds__(256, 4) void k_logits_softmax_mfma(SoftmaxArgs a) {
  using Lds = MfmaLdsN<MT, NT, 64 * MT + 4>;
  constexpr int BM = Lds::BM, BN = Lds::BN;
  constexpr int NPA = BM / 64;                          // A: BM rows x 4 float4
  constexpr int NPB = (4 * BN + 255) / 256;             // B: 16 k rows x BN / 4 float4
  __shared__ Lds L;
  __shared__ int sh_lab[BM];
  const int tid = threadIdx.x, lane = tid & 63, wm = tid >> 6;
  const int64_t Mrows = (int64_t)a.n * a.B;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int d = a.d, C = a.C;
  const int64_t xrows = a.rows ? a.S : Mrows;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t ws = make_rsrc(a.W, static_cast<uint32_t>((int64_t)d * C * 4));
  if (tid < BM) {
    const int64_t m = m0 + tid;
    int lab = 0;
    if (m < Mrows) {
      const int64_t row = sample_row(a, static_cast<int>(m / a.B), static_cast<int>(m % a.B), true);
      lab = sample_label(a, row, true);
    }
    sh_lab[tid] = lab;
  }
  int64_t xrow[NPA];
#pragma unroll
  for (int s2 = 0; s2 < NPA; ++s2) {
    const int64_t m = m0 + (tid + s2 * 256) / 4;
    xrow[s2] = m < Mrows ? sample_row(a, static_cast<int>(m / a.B), static_cast<int>(m % a.B), false) : -1;
  }
  // byte offsets of this thread's pieces at k0 = 0 (out of range where the
  // piece has no row or class); whole slices add k0 in the scalar offset
  uint32_t aoff[NPA], boff[NPB];
#pragma unroll
  for (int s2 = 0; s2 < NPA; ++s2) {
    const int kq = 4 * ((tid + s2 * 256) % 4);
    aoff[s2] = xrow[s2] >= 0 ? static_cast<uint32_t>((xrow[s2] * d + kq) * 4) : kOutOfRange;
  }
#pragma unroll
  for (int s2 = 0; s2 < NPB; ++s2) {
    const int q = tid + s2 * 256;
    const int kb = q / (BN / 4), nb = 4 * (q % (BN / 4));
    boff[s2] = q < 4 * BN && nb < C ? static_cast<uint32_t>((kb * C + nb) * 4) : kOutOfRange;
  }
  auto load = [&](int k0, float4 (&ra)[NPA], float4 (&rb)[NPB]) {
    if (k0 + MBK <= d) {
#pragma unroll
      for (int s2 = 0; s2 < NPA; ++s2) ra[s2] = buf_f32x4_s(xs, aoff[s2], static_cast<uint32_t>(k0 * 4));
#pragma unroll
      for (int s2 = 0; s2 < NPB; ++s2) rb[s2] = buf_f32x4_s(ws, boff[s2], static_cast<uint32_t>(k0 * C * 4));
      return;
    }
    // the last, partial slice: features past d read as 0
#pragma unroll
    for (int s2 = 0; s2 < NPA; ++s2) {
      const int k = k0 + 4 * ((tid + s2 * 256) % 4);
      ra[s2] = buf_f32x4(xs, xrow[s2] >= 0 && k < d ? static_cast<uint32_t>((xrow[s2] * d + k) * 4) : kOutOfRange);
    }
#pragma unroll
    for (int s2 = 0; s2 < NPB; ++s2) {
      const int q = tid + s2 * 256;
      const int kb = k0 + q / (BN / 4), nb = 4 * (q % (BN / 4));
      rb[s2] = buf_f32x4(ws, q < 4 * BN && kb < d && nb < C ? static_cast<uint32_t>(((int64_t)kb * C + nb) * 4)
                                                             : kOutOfRange);
    }
  };
  auto store = [&](int buf, const float4 (&ra)[NPA], const float4 (&rb)[NPB]) {
#pragma unroll
    for (int s2 = 0; s2 < NPA; ++s2) {
      const int q = tid + s2 * 256;
      const int r = q / 4, k = 4 * (q % 4);
      L.A[buf][k + 0][r] = ra[s2].x;
      L.A[buf][k + 1][r] = ra[s2].y;
      L.A[buf][k + 2][r] = ra[s2].z;
      L.A[buf][k + 3][r] = ra[s2].w;
    }
#pragma unroll
    for (int s2 = 0; s2 < NPB; ++s2) {
      const int q = tid + s2 * 256;
      if (q < 4 * BN) *reinterpret_cast<float4*>(&L.B[buf][q / (BN / 4)][4 * (q % (BN / 4))]) = rb[s2];
    }
  };
  mfma_f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
  mfma_pipeline_n<MT, NT, RS, 64 * MT + 4, NPA, NPB>(L, (d + MBK - 1) / MBK, load, store, acc);

  // row softmax: lane l holds rows 4 (l / 16) + r of each 16-row tile, class
  // 16 nt + l % 16; a row's classes are the 16 lanes of one DPP row
  const float invB = 1.0f / static_cast<float>(a.B);
  const int cl = lane & 15;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rl = wm * 16 * MT + mt * 16 + 4 * (lane >> 4) + r;
      float mx = -INFINITY;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        if (nt * 16 + cl < C) mx = fmaxf(mx, acc[mt][nt][r]);
      mx = row16_max(mx);
      float ex[NT];
      float se = 0.f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        ex[nt] = nt * 16 + cl < C ? expf(acc[mt][nt][r] - mx) : 0.f;
        se += ex[nt];
      }
      se = row16_sum(se);
      const int64_t m = m0 + rl;
      if (m < Mrows) {
        const int lab = sh_lab[rl];
        const float inv = 1.0f / se;
        float* z = a.Z + m * C;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int c = nt * 16 + cl;
          if (c < C) z[c] = (ex[nt] * inv - (c == lab ? 1.f : 0.f)) * invB;
          if (c == lab) a.ce[m] = (logf(se) + mx) - acc[mt][nt][r];
        }
      }
    }
}

// G_i[j][c] = sum_b X[row(i,b)][j] R_i[b][c] for a block of 64 MT features
// and all classes; blockIdx.x = feature tile, y = worker.  Block (0, i) also
// writes loss_i.  RS as for the logits.
template <int MT, int NT, int RS>
__global__ __launch_bounds__(256, 4) void k_grads_mfma_n(SoftmaxArgs a) {
  // A rows 16 mod 64 floats apart: the four k rows of an operand read fall on
  // disjoint bank quarters (the slice is stored as whole float4 rows)
  using Lds = MfmaLdsN<MT, NT, 64 * MT + 16>;
  constexpr int BM = Lds::BM, BN = Lds::BN;
  constexpr int NPA = BM / 64;                          // A: 16 rows x BM / 4 float4
  constexpr int NPB = (4 * BN + 255) / 256;             // B: 16 rows x BN / 4 float4
  __shared__ Lds L;
  __shared__ int sh_row[FUSED_MAX_ROWS];
  const int tid = threadIdx.x, lane = tid & 63, wm = tid >> 6;
  const int i = blockIdx.y;
  const int j0 = blockIdx.x * BM;
  const int d = a.d, C = a.C, B = a.B;
  const int64_t P = (int64_t)d * C;
  const int64_t xrows = a.rows ? a.S : (int64_t)a.n * B;
  const __amdgpu_buffer_rsrc_t xs = make_rsrc(a.X, static_cast<uint32_t>(xrows * d * 4));
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.Z + (int64_t)i * B * C, static_cast<uint32_t>((int64_t)B * C * 4));
  // byte offsets of the worker's rows (the dataset is addressed by one buffer
  // descriptor, below 2^31 bytes): no multiply per load
  for (int b = tid; b < B; b += 256) sh_row[b] = static_cast<int>(sample_row(a, i, b, false) * d * 4);
  __syncthreads();
  // residual pieces: byte offsets at k0 = 0 (out of range past the classes);
  // whole slices add k0 rows in the scalar offset
  uint32_t boff[NPB];
#pragma unroll
  for (int s2 = 0; s2 < NPB; ++s2) {
    const int q = tid + s2 * 256;
    const int b = q / (BN / 4), c = 4 * (q % (BN / 4));
    boff[s2] = q < 4 * BN && c < C ? static_cast<uint32_t>((b * C + c) * 4) : kOutOfRange;
  }
  auto load = [&](int k0, float4 (&ra)[NPA], float4 (&rb)[NPB]) {
    const bool whole = k0 + MBK <= B;
#pragma unroll
    for (int s2 = 0; s2 < NPA; ++s2) {
      const int q = tid + s2 * 256;
      const int b = k0 + q / (BM / 4), j = j0 + 4 * (q % (BM / 4));
      ra[s2] = buf_f32x4(xs, (whole || b < B) && j < d ? static_cast<uint32_t>(sh_row[b]) + static_cast<uint32_t>(j * 4)
                                                        : kOutOfRange);
    }
    if (whole) {
#pragma unroll
      for (int s2 = 0; s2 < NPB; ++s2) rb[s2] = buf_f32x4_s(rs, boff[s2], static_cast<uint32_t>(k0 * C * 4));
      return;
    }
#pragma unroll
    for (int s2 = 0; s2 < NPB; ++s2) {
      const int q = tid + s2 * 256;
      const int b = k0 + q / (BN / 4), c = 4 * (q % (BN / 4));
      rb[s2] = buf_f32x4(rs, q < 4 * BN && b < B && c < C ? static_cast<uint32_t>(((int64_t)b * C + c) * 4)
                                                         : kOutOfRange);
    }
  };
  auto store = [&](int buf, const float4 (&ra)[NPA], const float4 (&rb)[NPB]) {
#pragma unroll
    for (int s2 = 0; s2 < NPA; ++s2) {
      const int q = tid + s2 * 256;
      *reinterpret_cast<float4*>(&L.A[buf][q / (BM / 4)][4 * (q % (BM / 4))]) = ra[s2];
    }
#pragma unroll
    for (int s2 = 0; s2 < NPB; ++s2) {
      const int q = tid + s2 * 256;
      if (q < 4 * BN) *reinterpret_cast<float4*>(&L.B[buf][q / (BN / 4)][4 * (q % (BN / 4))]) = rb[s2];
    }
  };
  mfma_f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
  mfma_pipeline_n<MT, NT, RS, 64 * MT + 16, NPA, NPB>(L, (B + MBK - 1) / MBK, load, store, acc);
  // the G rows of workers outside the row mask are computed but not stored
  const bool write_g = !a.row_mask || a.row_mask[i];
  float* Gi = a.G + (int64_t)i * P;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int j = j0 + wm * 16 * MT + mt * 16 + 4 * (lane >> 4) + r;
      if (j >= d) continue;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int c = nt * 16 + (lane & 15);
        if (c < C && write_g) Gi[(int64_t)j * C + c] = acc[mt][nt][r];
      }
    }
  if (blockIdx.x == 0) {
    // loss_i = mean CE over the worker's rows (fixed order), reduced in the
    // LDS of the A tiles (free after the pipeline's last barrier)
    float* sh = &L.A[0][0][0];
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

template <int NT, int RS>
hipError_t launch_narrow_t(const SoftmaxArgs& a, hipStream_t s) {
  const int64_t Mrows = (int64_t)a.n * a.B;
  constexpr int BM = 64 * NARROW_MT;
  hipLaunchKernelGGL((k_logits_softmax_mfma<NARROW_MT, NT, RS>), dim3(static_cast<unsigned>((Mrows + BM - 1) / BM)),
                     dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_grads_mfma_n<NARROW_MT, NT, RS>), dim3(static_cast<unsigned>((a.d + BM - 1) / BM), a.n),
                     dim3(256), 0, s, a);
  return hipGetLastError();
}

// Classes per 16-wide MFMA tile for the narrow path (0: not taken).
int narrow_tiles(int C, int d, int B) {
  if (C <= 16 || C > 112 || C % 4 != 0 || d % 4 != 0 || B > FUSED_MAX_ROWS) return 0;
  return (C + 15) / 16;
}

template <int NT>
hipError_t launch_narrow_nt(const SoftmaxArgs& a, hipStream_t s) {
  // 4 or 8 classes in the last tile: 4-wide stripes (C = 16 (NT - 1) + 4 RS);
  // with 12 the saving is small and the third stripe's registers are not
  // free at 7 tiles, so a full tile is used
  switch ((a.C % 16) / 4) {
    case 1: return launch_narrow_t<NT, 1>(a, s);
    case 2: return launch_narrow_t<NT, 2>(a, s);
    default: return launch_narrow_t<NT, 0>(a, s);
  }
}

hipError_t launch_narrow(const SoftmaxArgs& a, hipStream_t s) {
  switch (narrow_tiles(a.C, a.d, a.B)) {
    case 2: return launch_narrow_nt<2>(a, s);
    case 3: return launch_narrow_nt<3>(a, s);
    case 4: return launch_narrow_nt<4>(a, s);
    case 5: return launch_narrow_nt<5>(a, s);
    case 6: return launch_narrow_nt<6>(a, s);
    case 7: return launch_narrow_nt<7>(a, s);
  }
  return hipErrorInvalidValue;
}

template <int CP, int M, int T>
hipError_t launch_fused_t(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  constexpr int R = 4;
  const int64_t nb = (int64_t)a.n * p.slabs;
  const int64_t per_xcd = (nb + NXCD - 1) / NXCD;
  hipLaunchKernelGGL((k_softmax_fused<CP, M, T, R>), dim3(static_cast<unsigned>(per_xcd * NXCD)), dim3(T), 0, s,
                     a, p.slabs, p.rows_per_slab, per_xcd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.slabs == 1 || a.keep_slabs) return e;
  const int64_t P = (int64_t)a.d * a.C;
  const dim3 g2(static_cast<unsigned>((P + 1023) / 1024), static_cast<unsigned>(a.n));
  hipLaunchKernelGGL(k_slab_reduce, g2, dim3(256), 0, s, a, p.slabs);
  return hipGetLastError();
}

template <int U, int CW>
hipError_t launch_mfma_t(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  const int64_t nb = (int64_t)a.n * p.slabs;
  const int64_t per_xcd = (nb + NXCD - 1) / NXCD;
  hipLaunchKernelGGL((k_softmax_mfma<U, CW>), dim3(static_cast<unsigned>(per_xcd * NXCD)), dim3(MF_T), 0, s, a,
                     p.slabs, p.rows_per_slab, per_xcd);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.slabs == 1 || a.keep_slabs) return e;
  const dim3 g2(static_cast<unsigned>((a.d + 63) / 64), static_cast<unsigned>(a.n));
  hipLaunchKernelGGL(k_slab_reduce_tiles, g2, dim3(256), 0, s, a, p.slabs, U);
  return hipGetLastError();
}

template <int CW>
hipError_t launch_mfma_c(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  switch (p.per_thread) {
    case 1: return launch_mfma_t<1, CW>(p, a, s);
    case 2: return launch_mfma_t<2, CW>(p, a, s);
    case 3: return launch_mfma_t<3, CW>(p, a, s);
    case 4: return launch_mfma_t<4, CW>(p, a, s);
    case 5: if constexpr (CW <= 10) return launch_mfma_t<5, CW>(p, a, s); break;
    case 6: if constexpr (CW <= 10) return launch_mfma_t<6, CW>(p, a, s); break;
  }
  return hipErrorInvalidValue;
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
  {
    // matrix-core single pass: 8 waves x 64U features, W staged in LDS
    const int cw = C <= 4 ? 4 : C <= 10 ? 10 : C <= 16 ? 16 : 0;
    const int U = (d + MF_T - 1) / MF_T;
    const bool fits = cw == 16 ? U <= 4 : U <= 6;
    if (cw && d % 4 == 0 && fits) {
      p.fused = 2;
      p.threads = MF_T;
      p.per_thread = U;
      p.cpad = cw;
      // about 256 blocks, at least four 8-row chunks per slab
      int slabs = 256 / n, max_slabs = B / (4 * MF_ROWS);
      slabs = slabs < 1 ? 1 : slabs;
      max_slabs = max_slabs < 1 ? 1 : max_slabs;
      slabs = slabs > max_slabs ? max_slabs : slabs;
      int rps = (B + slabs - 1) / slabs;
      rps = (rps + MF_ROWS - 1) / MF_ROWS * MF_ROWS;
      if (rps > FUSED_MAX_ROWS) rps = FUSED_MAX_ROWS;
      p.rows_per_slab = rps;
      p.slabs = (B + rps - 1) / rps;
      p.part = (int64_t)MF_T * U * C;   // tile-order partial
      if ((int64_t)p.slabs * p.part * 4 <= kMaxBufferBytes) return p;
      p = SoftmaxPlan{};
    }
  }
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
  p.part = (int64_t)d * C;
  // one worker's partials are read through one buffer resource
  if ((int64_t)p.slabs * d * C * 4 > kMaxBufferBytes) p.fused = 0;
  return p;
}

hipError_t launch_softmax_grads(const SoftmaxPlan& p, const SoftmaxArgs& a, hipStream_t s) {
  if (p.fused == 2) {
    switch (p.cpad) {
      case 4: return launch_mfma_c<4>(p, a, s);
      case 10: return launch_mfma_c<10>(p, a, s);
      case 16: return launch_mfma_c<16>(p, a, s);
    }
    return hipErrorInvalidValue;
  }
  if (p.fused) {
    switch (p.cpad) {
      case 4: return launch_fused_c<4>(p, a, s);
      case 10: return launch_fused_c<10>(p, a, s);
      case 16: return launch_fused_c<16>(p, a, s);
    }
    return hipErrorInvalidValue;
  }
  if (narrow_tiles(a.C, a.d, a.B)) return launch_narrow(a, s);
  const int64_t Mrows = (int64_t)a.n * a.B;
  // matrix cores when float4 pieces tile the rows of X, W and R exactly
  // (and a worker's row indices fit the LDS stage)
  const bool mfma = a.C % 4 == 0 && a.d % 4 == 0 && a.B <= FUSED_MAX_ROWS;
  if (mfma) {
    const int64_t tiles = (int64_t)((a.C + 127) / 128) * ((Mrows + 127) / 128);
    if (tiles >= kMfmaBigTiles) {
      dim3 g1((a.C + 127) / 128, static_cast<unsigned>((Mrows + 127) / 128));
      hipLaunchKernelGGL(k_logits_mfma<4>, g1, dim3(256), 0, s, a);
    } else {
      dim3 g1((a.C + 63) / 64, static_cast<unsigned>((Mrows + 63) / 64));
      hipLaunchKernelGGL(k_logits_mfma<2>, g1, dim3(256), 0, s, a);
    }
  } else {
    dim3 g1((a.C + GBN - 1) / GBN, static_cast<unsigned>((Mrows + GBM - 1) / GBM));
    hipLaunchKernelGGL(k_logits_gemm, g1, dim3(256), 0, s, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rows_softmax, dim3(static_cast<unsigned>((Mrows + 3) / 4)), dim3(256), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (mfma) {
    const int64_t tiles = (int64_t)((a.C + 127) / 128) * ((a.d + 127) / 128) * a.n;
    if (tiles >= kMfmaBigTiles) {
      dim3 g3((a.C + 127) / 128, (a.d + 127) / 128, a.n);
      hipLaunchKernelGGL(k_grads_mfma<4>, g3, dim3(256), 0, s, a);
    } else {
      dim3 g3((a.C + 63) / 64, (a.d + 63) / 64, a.n);
      hipLaunchKernelGGL(k_grads_mfma<2>, g3, dim3(256), 0, s, a);
    }
  } else {
    dim3 g3((a.C + GBN - 1) / GBN, (a.d + GBM - 1) / GBM, a.n);
    hipLaunchKernelGGL(k_grads_gemm, g3, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace dbw
