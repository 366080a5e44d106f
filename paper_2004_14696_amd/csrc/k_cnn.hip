// Worker minibatch gradients of the MNIST-shaped CNN (Sect. 4: two 5x5
// convolutions and two fully connected layers; Sect. 2, Eq. gradient), gfx950.
//
// Per image (28 x 28, one channel): conv 1 -> 20 channels (24 x 24), 2 x 2 max
// pooling and ReLU (20 x 12 x 12 = H1), conv 20 -> 50 (8 x 8), pooling and ReLU
// (50 x 4 x 4 = the 800 features F), then the fully connected part, which is
// the MLP 800-H-C (k_mlp.hip).  A pooling window passes its first largest
// value in row-major order; only that entry receives the gradient, and none
// when the pooled value is not positive (ReLU).  The window code 0..3 names
// the passing entry; code 4 marks a window whose ReLU is off, so unpooling
// by code applies the ReLU mask as well.
//
//  k_cnn_conv1_pool   one thread per pooled position of an image: the four
//                     conv outputs of its window for all 20 filters (vector
//                     ALU, filters in LDS), the pooled value, its ReLU and the
//                     window code; also gathers the image's label.
//  k_cnn_conv2_pool   the conv as a 64 x 64 x 500 GEMM per image on the fp32
//                     matrix cores (positions x filters x (channel, row,
//                     column) of the 5 x 5 patches), filter fragments held in
//                     registers by a persistent grid, the image's H1 in LDS;
//                     pooling and ReLU in the epilogue.
//  k_cnn_dfeat        dF = dA Wf1^T on the matrix cores (the ReLU mask of F is
//                     in the window codes).
//  k_cnn_conv2_dgrad  gradient at H1: per image and input channel the GEMM
//                     dcols = dZ2 W2 (positions x taps, K = filters) on the
//                     matrix cores, with the filters' fragments held in
//                     registers by a persistent grid; the fold of dcols back
//                     onto the 12 x 12 map reads zero-framed tap maps in LDS at
//                     fixed offsets.
//  k_cnn_conv2_wgrad  dW2 and db2 partials over chunks of a worker's images:
//                     dW2 += dZ2^T im2col(H1) per image (filters x taps, K =
//                     positions) on the matrix cores, accumulators kept over the
//                     chunk, the next image staged in LDS meanwhile.
//  k_cnn_conv1_wgrad  dW1 and db1 partials: dW1 += dZ1 im2col(X) per image
//                     (filters x taps, K = the 576 conv1 positions) on the
//                     matrix cores, dZ1 formed from the pooled gradient and
//                     window codes as the operand is read.
//  k_cnn_wreduce      sums the chunk partials in chunk order into G.
//
// Everything runs in a fixed order: results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dbw_buffer.h"
#include "dbw_internal.h"
#include "mfma_gemm.h"

namespace dbw {
namespace {

constexpr int IMG = CNN_IMG, KS = 5, NC1 = CNN_C1, NC2 = CNN_C2;
constexpr int Q1 = 12, NPOS1 = Q1 * Q1, H1LEN = NC1 * NPOS1;   // 2880 per image
constexpr int O2 = 8, NPOS2 = O2 * O2;                          // conv2 output positions
constexpr int Q2 = 4, NQ2 = Q2 * Q2, FEAT = CNN_FEAT;           // 800
constexpr int K2 = NC1 * KS * KS;                               // 500: conv2 patch length
constexpr int W1LEN = NC1 * KS * KS;                            // 500 conv1 weights

__device__ __forceinline__ int64_t cnn_row(const CnnArgs& a, int64_t m, bool report) {
  if (!a.rows) return m;
  const int64_t r = a.rows[m];
  if (r < 0 || r >= a.S) {
    if (report) atomicOr(a.err, ERR_ROW_RANGE);
    return -1;
  }
  return r;
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_cnn_conv1_pool(CnnArgs a) {
  __shared__ float sw[W1LEN + NC1];
  const int tid = threadIdx.x;
  for (int i = tid; i < W1LEN + NC1; i += 256) sw[i] = a.w[a.off_c1 + i];   // W1 then b1
  __syncthreads();
  const int64_t nB = (int64_t)a.n * a.B;
  const int64_t gidx = (int64_t)blockIdx.x * 256 + tid;
  if (gidx >= nB * NPOS1) return;
  const int64_t b = gidx / NPOS1;
  const int pos = static_cast<int>(gidx - b * NPOS1), py = pos / Q1, px = pos % Q1;
  const int64_t row = cnn_row(a, b, pos == 0);
  if (pos == 0) {
    int lab = row >= 0 ? a.y[row] : 0;
    if (lab < 0 || lab >= a.C) {
      atomicOr(a.err, ERR_LABEL_RANGE);
      lab = 0;
    }
    a.ylab[b] = lab;
  }
  // the 6 x 6 input patch under the window's four 5 x 5 filters
  float in[6][6];
  const float* img = a.X + (row >= 0 ? row : 0) * (int64_t)(IMG * IMG);
#pragma unroll
  for (int r = 0; r < 6; ++r)
#pragma unroll
    for (int c = 0; c < 6; ++c) in[r][c] = row >= 0 ? img[(2 * py + r) * IMG + 2 * px + c] : 0.f;
  float* h1 = a.H1 + b * H1LEN + pos;
  uint8_t* cd = a.code1 + b * H1LEN + pos;
#pragma unroll 1
  for (int o = 0; o < NC1; ++o) {
    float z[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int dy = q >> 1, dx = q & 1;
      float s = sw[W1LEN + o];
#pragma unroll
      for (int u = 0; u < KS; ++u)
#pragma unroll
        for (int v = 0; v < KS; ++v) s = fmaf(in[dy + u][dx + v], sw[o * 25 + u * KS + v], s);
      z[q] = s;
    }
    int code = 0;
    float best = z[0];
#pragma unroll
    for (int q = 1; q < 4; ++q)
      if (z[q] > best) {
        best = z[q];
        code = q;
      }
    h1[o * NPOS1] = best > 0.f ? best : 0.f;
    cd[o * NPOS1] = static_cast<uint8_t>(best > 0.f ? code : 4);
  }
}

// ---------------------------------------------------------------------------
// Conv2 as a GEMM per image: Z[m][o] = sum_k A[m][k] W2[o][k], m = output
// position (y, x) of the 8 x 8, k = (c, u, v), A[m][k] = H1[c][y+u][x+v].
// The K steps of 4 run over (tap t, channel quad): step 5 t + cq takes
// channels 4 cq .. 4 cq + 3 at tap t, so that every A read is the lane's own
// LDS offset plus a constant.  Wave w owns filters 16 w .. 16 w + 15 and holds
// their 125 W2 fragments in registers for the whole (persistent) launch; the
// next image's H1 is loaded while the current one is multiplied.  Bias, 2 x 2
// pooling and ReLU run from an LDS copy of Z.
constexpr int FW_KS = K2 / 4;            // 125 K steps
constexpr int kConvBlocks = 512;         // two blocks per CU
struct Conv2Lds {
  float h1[2][H1LEN];
  float z[2][NPOS2][NC2 + 1];
};

__global__ __launch_bounds__(256, 2) void k_cnn_conv2_pool(CnnArgs a) {
  __shared__ __align__(16) Conv2Lds L;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, g = lane >> 4, j = lane & 15;
  const float* W2 = a.w + a.off_c2;
  const float* b2 = W2 + NC2 * K2;
  const int o_mine = 16 * wv + j;
  float wb[FW_KS];
#pragma unroll
  for (int t = 0; t < 25; ++t)
#pragma unroll
    for (int cq = 0; cq < 5; ++cq)
      wb[5 * t + cq] = o_mine < NC2 ? W2[o_mine * K2 + (4 * cq + g) * 25 + t] : 0.f;
  const float bias = o_mine < NC2 ? b2[o_mine] : 0.f;
  // A operand of lane (g, j): channel 4 cq + g, position m = 16 mt + j
  const int abase = g * NPOS1 + (j >> 3) * Q1 + (j & 7);
  const int64_t nB = (int64_t)a.n * a.B;
  float4 rh[3];
  auto fetch = [&](int64_t b) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int e = tid + 256 * s;
      rh[s] = e < H1LEN / 4 ? reinterpret_cast<const float4*>(a.H1 + b * H1LEN)[e] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto stage = [&](float* h) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int e = tid + 256 * s;
      if (e < H1LEN / 4) reinterpret_cast<float4*>(h)[e] = rh[s];
    }
  };
  int64_t b = blockIdx.x;
  if (b < nB) {
    fetch(b);
    stage(L.h1[0]);
  }
  __syncthreads();
  for (int it = 0; b < nB; b += gridDim.x, ++it) {
    const int cur = it & 1;
    if (b + gridDim.x < nB) fetch(b + gridDim.x);
    mfma_f32x4 acc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) acc[mt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
    const float* h = L.h1[cur] + abase;
#pragma unroll
    for (int t = 0; t < 25; ++t)
#pragma unroll
      for (int cq = 0; cq < 5; ++cq) {
        const int off = 4 * cq * NPOS1 + (t / 5) * Q1 + t % 5;
        float av[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) av[mt] = h[off + 2 * mt * Q1];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
          acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt], wb[5 * t + cq], acc[mt], 0, 0, 0);
        if (cq == 4) __builtin_amdgcn_sched_barrier(0);   // bounds how far LDS reads run ahead
      }
    // acc[mt][r] = Z[m = 16 mt + 4 g + r][o = 16 wv + j]
    if (o_mine < NC2)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) L.z[cur][16 * mt + 4 * g + r][o_mine] = acc[mt][r] + bias;
    if (b + gridDim.x < nB) stage(L.h1[cur ^ 1]);
    __syncthreads();
    for (int f = tid; f < FEAT; f += 256) {
      const int o = f / NQ2, q = f % NQ2, y = 2 * (q / Q2), x = 2 * (q % Q2);
      float best = L.z[cur][y * O2 + x][o];
      int code = 0;
      const float z1 = L.z[cur][y * O2 + x + 1][o], z2 = L.z[cur][(y + 1) * O2 + x][o],
                  z3 = L.z[cur][(y + 1) * O2 + x + 1][o];
      if (z1 > best) { best = z1; code = 1; }
      if (z2 > best) { best = z2; code = 2; }
      if (z3 > best) { best = z3; code = 3; }
      a.F[b * FEAT + f] = best > 0.f ? best : 0.f;
      a.code2[b * FEAT + f] = static_cast<uint8_t>(best > 0.f ? code : 4);
    }
  }
}

// ---------------------------------------------------------------------------
// dP2[m][f] = sum_h dA[m][h] Wf1[f][h]; 64 x 64 tiles.
__global__ __launch_bounds__(256) void k_cnn_dfeat(CnnArgs a) {
  __shared__ MfmaLds<2> L;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  const int64_t nB = (int64_t)a.n * a.B;
  const int H = a.H;
  const int n0 = blockIdx.x * 64;
  const int64_t m0 = (int64_t)blockIdx.y * 64;
  const float* Wf1 = a.w;     // [800][H]
  auto load = [&](int k0, float (&ra)[4], float (&rb)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int e = tid + 256 * s;
      const int k = k0 + e % 16, i = e / 16;
      const int64_t m = m0 + i;
      ra[s] = k < H && m < nB ? a.dA[m * H + k] : 0.f;
      const int f = n0 + i;
      rb[s] = k < H && f < FEAT ? Wf1[(int64_t)f * H + k] : 0.f;
    }
  };
  auto store = [&](int buf, const float (&ra)[4], const float (&rb)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int e = tid + 256 * s;
      L.A[buf][e % 16][e / 16] = ra[s];
      L.B[buf][e % 16][e / 16] = rb[s];
    }
  };
  mfma_f32x4 acc[2][2];
  mfma_zero<2>(acc);
  float ra[4], rb[4];
  load(0, ra, rb);
  store(0, ra, rb);
  __syncthreads();
  const int nk = (H + MBK - 1) / MBK;
  for (int kt = 0; kt < nk; ++kt) {
    const int cbuf = kt & 1;
    if (kt + 1 < nk) load((kt + 1) * MBK, ra, rb);
    mfma_slice<2>(L, cbuf, wm, wn, lane, acc);
    if (kt + 1 < nk) store(cbuf ^ 1, ra, rb);
    __syncthreads();
  }
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm * 32 + mt * 16 + 4 * (lane >> 4) + r;
        const int f = n0 + wn * 32 + nt * 16 + (lane & 15);
        if (m < nB && f < FEAT) a.dP2[m * FEAT + f] = acc[mt][nt][r];
      }
}

// ---------------------------------------------------------------------------
// Gradient at H1.  Per image the pooled gradient is unpooled into dZ2[m][o]
// (its value at the window's passing entry, 0 at the other three), and
// dcols[m][(c, t)] = sum_o dZ2[m][o] W2[o][c][t] is a 64 x 25 x 50 GEMM per
// input channel c on the matrix cores (4 x 2 tiles of 16 x 16, K = 50 padded
// to 52).  Each wave owns five channels and holds their W2 fragments in
// registers for the whole (persistent) launch.  The fold back onto H1,
// dH1[c][p] = sum_{t = (u, v)} dcols[p - (u, v)][(c, t)], goes through a
// wave-private LDS copy of the channel's 25 tap maps, each stored in a
// zero-framed 12 x 12 tile (data in rows and columns 4..11) so that a target's
// 25 reads sit at fixed offsets from it and out-of-range taps read zeros.
constexpr int DG_CPW = NC1 / 4;          // channels per wave (4 waves)
constexpr int DG_KS = (NC2 + 3) / 4;     // 13 K steps of 4 filters
constexpr int SA_LD = 80;                // unpooled-gradient row stride (bank spread)
constexpr int DT = 12 * 12;              // one framed tap map
constexpr int DLEN = 25 * DT + 64;       // 25 maps and a zero tail
constexpr int kDgradBlocks = 512;        // two blocks per CU

__global__ __launch_bounds__(256, 2) void k_cnn_conv2_dgrad(CnnArgs a) {
  __shared__ float sA[52 * SA_LD];                     // [o][m]
  __shared__ __align__(16) float sD[4][DLEN];           // per wave
  // the next image's pooled gradient and codes, loaded straight into LDS
  // while the current image is multiplied
  __shared__ float rawg[FEAT];
  __shared__ uint32_t rawc[FEAT / 4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, g = lane >> 4, j = lane & 15;
  for (int i = tid; i < 4 * DLEN; i += 256) (&sD[0][0])[i] = 0.f;
  for (int i = tid; i < 2 * SA_LD; i += 256) sA[NC2 * SA_LD + i] = 0.f;   // rows o = 50, 51
  // B fragments: W2[o = 4 ks + g][c][t = 16 nt + j] of the wave's channels
  const float* W2 = a.w + a.off_c2;
  float wb[DG_CPW][2][DG_KS];
#pragma unroll
  for (int ci = 0; ci < DG_CPW; ++ci)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int ks = 0; ks < DG_KS; ++ks) {
        const int o = 4 * ks + g, t = 16 * nt + j, c = DG_CPW * wv + ci;
        wb[ci][nt][ks] = o < NC2 && t < 25 ? W2[o * K2 + c * 25 + t] : 0.f;
      }
  float* D = sD[wv];
  const int64_t nB = (int64_t)a.n * a.B;
  auto fetch = [&](int64_t bn) {
    // wave wv copies pieces wv, wv + 4, .. of 64 dwords; lanes past the end
    // stay idle
    for (int k = wv; k * 64 < FEAT + FEAT / 4; k += 4) {
      const int e = 64 * k + lane;
      if (e < FEAT)
        __builtin_amdgcn_global_load_lds(a.dP2 + bn * FEAT + e, rawg + 64 * k, 4, 0, 0);
      else if (e < FEAT + FEAT / 4)
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint32_t*>(a.code2 + bn * FEAT) + (e - FEAT),
                                         rawc + (64 * k - FEAT), 4, 0, 0);
    }
  };
  if (blockIdx.x < nB) fetch(blockIdx.x);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int64_t b = blockIdx.x; b < nB; b += gridDim.x) {
    // unpool: task (o, q) writes the four entries of its window in row o
    const uint8_t* rc = reinterpret_cast<const uint8_t*>(rawc);
    for (int e = tid; e < FEAT; e += 256) {
      const int o = e / NQ2, q = e % NQ2;
      const int m0 = 2 * (q / Q2) * O2 + 2 * (q % Q2);
      const float gv = rawg[e];
      const int cd = rc[e];
      float* row = sA + o * SA_LD + m0;
      row[0] = cd == 0 ? gv : 0.f;
      row[1] = cd == 1 ? gv : 0.f;
      row[O2] = cd == 2 ? gv : 0.f;
      row[O2 + 1] = cd == 3 ? gv : 0.f;
    }
    __syncthreads();
    if (b + gridDim.x < nB) fetch(b + gridDim.x);
    // dcols of channel ci on the matrix cores
    auto products = [&](int ci, mfma_f32x4 (&acc)[4][2]) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < DG_KS; ++ks) {
        float av[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) av[mt] = sA[(4 * ks + g) * SA_LD + 16 * mt + j];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int nt = 0; nt < 2; ++nt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt], wb[ci][nt][ks], acc[mt][nt], 0, 0, 0);
      }
    };
    // acc[mt][nt][r]: m = 16 mt + 4 g + r (y = 2 mt + g / 2, x = 4 (g % 2) + r),
    // tap t = 16 nt + j, into the framed tap maps
    auto store = [&](const mfma_f32x4 (&acc)[4][2]) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int t = 16 * nt + j;
          if (t < 25) {
            float* cell = D + t * DT + (2 * mt + (g >> 1) + 4) * 12 + 4 * (g & 1) + 4;
            *reinterpret_cast<float4*>(cell) =
                make_float4(acc[mt][nt][0], acc[mt][nt][1], acc[mt][nt][2], acc[mt][nt][3]);
          }
        }
    };
    auto fold = [&](int c) {
      float* dp1 = a.dP1 + b * H1LEN + c * NPOS1;
#pragma unroll
      for (int pp = 0; pp < 3; ++pp) {
        const int p = lane + 64 * pp;
        if (p < NPOS1) {
          // framed cell of (t, y = py - u, x = px - v) = p + 52 + 708 u + 143 v
          const float* src = D + p + 52;
          float su[KS];                  // one short add chain per tap row
#pragma unroll
          for (int u = 0; u < KS; ++u) {
            su[u] = src[708 * u];
#pragma unroll
            for (int v = 1; v < KS; ++v) su[u] += src[708 * u + 143 * v];
          }
          dp1[p] = ((su[0] + su[1]) + (su[2] + su[3])) + su[4];
        }
        // one target's reads in flight at a time; matrix-core work may cross
        __builtin_amdgcn_sched_barrier(0x8);
      }
    };
    // channel ci + 1's products run while channel ci is folded: they need
    // neither its maps nor its results
    mfma_f32x4 acc[4][2];
    products(0, acc);
#pragma unroll   // register index ci
    for (int ci = 0; ci < DG_CPW; ++ci) {
      store(acc);
      asm volatile("" ::: "memory");   // the wave's LDS ops stay in program order
      if (ci + 1 < DG_CPW) products(ci + 1, acc);
      fold(DG_CPW * wv + ci);
      asm volatile("" ::: "memory");
    }
    __builtin_amdgcn_s_waitcnt(0);   // the next image's copy has landed
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// dW2, db2 partial of chunk j of worker i (images i B + j chunk .., in order):
// dW2[o][n] += sum_m dZ2[m][o] H1[c][m + t] with n = (c, t) = 25 c + t, a
// 64 x 512 x 64 GEMM per image on the matrix cores (o padded to 64, n to 512;
// the padded columns read a zero region, except column 500, which reads ones
// and so collects db2).  Each of the four waves owns 8
// column tiles and keeps its 4 x 8 accumulator tiles over the chunk; the
// image's H1 and unpooled gradient are staged in LDS, the next image's loads
// in flight meanwhile.
constexpr int WG_NT = 8;                 // column tiles per wave
constexpr int WG_ZERO = H1LEN;           // zero region after the image's H1
constexpr int WG_ONES = H1LEN + 96;      // then a region of ones
constexpr int WG_H1 = H1LEN + 192;
struct WgradBuf {
  float h1[WG_H1];
  float A[NPOS2 * SA_LD];                // [m][o]
};

__global__ __launch_bounds__(256) void k_cnn_conv2_wgrad(CnnArgs a) {
  __shared__ __align__(16) WgradBuf L[2];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, g = lane >> 4, j = lane & 15;
  const int i = blockIdx.y, jc = blockIdx.x;
  const int b0 = jc * a.chunk, b1 = min(a.B, b0 + a.chunk);
  for (int e = tid; e < 2 * 192; e += 256) L[e / 192].h1[WG_ZERO + e % 192] = e % 192 < 96 ? 0.f : 1.f;
  for (int e = tid; e < 2 * NPOS2 * (SA_LD - NC2); e += 256) {
    const int bi = e / (NPOS2 * (SA_LD - NC2)), r = e % (NPOS2 * (SA_LD - NC2));
    L[bi].A[(r / (SA_LD - NC2)) * SA_LD + NC2 + r % (SA_LD - NC2)] = 0.f;
  }
  // per column tile: the lane's H1 offset of tap (c, u, v), or the zero region
  int colbase[WG_NT];
#pragma unroll
  for (int nt = 0; nt < WG_NT; ++nt) {
    const int n = 16 * (WG_NT * wv + nt) + j;
    const int c = n / 25, t = n % 25;
    colbase[nt] = (n < K2 ? c * NPOS1 + (t / 5) * Q1 + t % 5 : n == K2 ? WG_ONES : WG_ZERO) + g;
  }
  float4 rh[3];
  float rg[4];
  uint8_t rc[4];
  auto fetch = [&](int64_t b) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int e = tid + 256 * s;
      rh[s] = e < H1LEN / 4 ? reinterpret_cast<const float4*>(a.H1 + b * H1LEN)[e] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int e = tid + 256 * s;
      rg[s] = e < FEAT ? a.dP2[b * FEAT + e] : 0.f;
      rc[s] = e < FEAT ? a.code2[b * FEAT + e] : 0;
    }
  };
  auto stage = [&](WgradBuf& B) {
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const int e = tid + 256 * s;
      if (e < H1LEN / 4) reinterpret_cast<float4*>(B.h1)[e] = rh[s];
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int e = tid + 256 * s;
      if (e < FEAT) {
        const int o = e / NQ2, q = e % NQ2, m0 = 2 * (q / Q2) * O2 + 2 * (q % Q2);
        float* col = B.A + m0 * SA_LD + o;
        col[0] = rc[s] == 0 ? rg[s] : 0.f;
        col[SA_LD] = rc[s] == 1 ? rg[s] : 0.f;
        col[O2 * SA_LD] = rc[s] == 2 ? rg[s] : 0.f;
        col[(O2 + 1) * SA_LD] = rc[s] == 3 ? rg[s] : 0.f;
      }
    }
  };
  mfma_f32x4 acc[4][WG_NT];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < WG_NT; ++nt) acc[mt][nt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
  if (b0 < b1) {
    fetch((int64_t)i * a.B + b0);
    stage(L[0]);
  }
  __syncthreads();
  for (int bb = b0; bb < b1; ++bb) {
    const int cur = (bb - b0) & 1;
    const int64_t b = (int64_t)i * a.B + bb;
    if (bb + 1 < b1) fetch(b + 1);
    const float* A = L[cur].A + g * SA_LD + j;
    const float* H = L[cur].h1;
#pragma unroll
    for (int ks = 0; ks < NPOS2 / 4; ++ks) {
      // K index m = 4 ks + g: y = ks / 2, x = 4 (ks % 2) + g
      const int moff = (ks >> 1) * Q1 + 4 * (ks & 1);
      float av[4], bv[WG_NT];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) av[mt] = A[4 * ks * SA_LD + 16 * mt];
#pragma unroll
      for (int nt = 0; nt < WG_NT; ++nt) bv[nt] = H[colbase[nt] + moff];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < WG_NT; ++nt)
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt], bv[nt], acc[mt][nt], 0, 0, 0);
    }
    if (bb + 1 < b1) stage(L[cur ^ 1]);
    __syncthreads();
  }
  // partial [i][jc][W2 (50 x 500) | b2 (50)]; acc[mt][nt][r] is (o = 16 mt + 4 g + r, n)
  float* p = a.part2 + ((int64_t)i * gridDim.x + jc) * (NC2 * K2 + NC2);
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int nt = 0; nt < WG_NT; ++nt) {
      const int n = 16 * (WG_NT * wv + nt) + j;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = 16 * mt + 4 * g + r;
        if (o < NC2 && n <= K2) p[n < K2 ? o * K2 + n : NC2 * K2 + o] = acc[mt][nt][r];
      }
    }
}

// ---------------------------------------------------------------------------
// dW1, db1 partial of chunk j of worker i: dW1[o][t] += sum_m dZ1[o][m]
// X[m + t] over the 24 x 24 conv1 outputs m of each image, a GEMM (filters x
// taps, K = positions) on the matrix cores.  K runs over (pooled position p,
// window offset d): the lanes of group d = lane / 16 take the pooled gradient
// of p where the window's code is d and 0 elsewhere, which is the unpooled
// dZ1.  Tap column 25 is all ones, so it collects db1.  Each wave takes whole
// images of the chunk (every fourth), staged in its own LDS region while the
// next one is loaded into registers; the four waves' partial tiles are
// summed in wave order at the end.
constexpr int C1_LD = NPOS1 + 1;         // bank spread of the [o][p] rows
struct Wg1Buf {
  float x[IMG * IMG];
  float g[NC1 * C1_LD];
  uint8_t cd[NC1 * C1_LD + 12];
};
constexpr int C1_X4 = (IMG * IMG / 4 + 63) / 64;     // float4 pieces per lane
constexpr int C1_G4 = (H1LEN / 4 + 63) / 64;

__global__ __launch_bounds__(256, 2) void k_cnn_conv1_wgrad(CnnArgs a) {
  __shared__ __align__(16) Wg1Buf L[4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, g = lane >> 4, j = lane & 15;
  const int i = blockIdx.y, jc = blockIdx.x;
  const int b0 = jc * a.chunk, b1 = min(a.B, b0 + a.chunk);
  Wg1Buf& B = L[wv];
  // B operand of lane (d = g, tap t = 16 nt + j): X[(2 py + d / 2 + u) 28 + 2 px + d % 2 + v]
  int xb[2];
  float bconst[2];
  bool bx[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int t = 16 * nt + j;
    bx[nt] = t < 25;
    xb[nt] = t < 25 ? ((g >> 1) + t / 5) * IMG + (g & 1) + t % 5 : 0;
    bconst[nt] = t == 25 ? 1.f : 0.f;
  }
  // A operand row o = 16 mt + j (filters 20 .. 31 read row 0 and contribute 0)
  int arow[2];
  bool aval[2];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
    aval[mt] = 16 * mt + j < NC1;
    arow[mt] = aval[mt] ? (16 * mt + j) * C1_LD : 0;
  }
  float4 rx[C1_X4], rg[C1_G4];
  uint32_t rc[C1_G4];
  auto fetch = [&](int64_t b) {
    const int64_t row = cnn_row(a, b, false);
#pragma unroll
    for (int s = 0; s < C1_X4; ++s) {
      const int e = lane + 64 * s;
      rx[s] = e < IMG * IMG / 4 && row >= 0 ? reinterpret_cast<const float4*>(a.X + row * (IMG * IMG))[e]
                                            : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int s = 0; s < C1_G4; ++s) {
      const int e = lane + 64 * s;
      rg[s] = e < H1LEN / 4 ? reinterpret_cast<const float4*>(a.dP1 + b * H1LEN)[e] : make_float4(0.f, 0.f, 0.f, 0.f);
      rc[s] = e < H1LEN / 4 ? reinterpret_cast<const uint32_t*>(a.code1 + b * H1LEN)[e] : 0u;
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int s = 0; s < C1_X4; ++s) {
      const int e = lane + 64 * s;
      if (e < IMG * IMG / 4) reinterpret_cast<float4*>(B.x)[e] = rx[s];
    }
#pragma unroll
    for (int s = 0; s < C1_G4; ++s) {
      const int e = lane + 64 * s;
      if (e < H1LEN / 4) {
        const int o = (4 * e) / NPOS1, p = (4 * e) % NPOS1;   // 144 % 4 == 0: one row
        float* gd = B.g + o * C1_LD + p;
        uint8_t* cd = B.cd + o * C1_LD + p;
        gd[0] = rg[s].x; gd[1] = rg[s].y; gd[2] = rg[s].z; gd[3] = rg[s].w;
        cd[0] = rc[s] & 0xff; cd[1] = (rc[s] >> 8) & 0xff; cd[2] = (rc[s] >> 16) & 0xff; cd[3] = rc[s] >> 24;
      }
    }
  };
  mfma_f32x4 acc[2][2];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
  int bb = b0 + wv;
  if (bb < b1) fetch((int64_t)i * a.B + bb);
  for (; bb < b1; bb += 4) {
    stage();
    asm volatile("" ::: "memory");       // the wave's LDS writes precede its reads
    if (bb + 4 < b1) fetch((int64_t)i * a.B + bb + 4);
    // pooled row py, column px: every read is unconditional (padding lanes
    // read valid cells and select), offsets are immediates within a row
#pragma unroll 1
    for (int py = 0; py < Q1; ++py) {
      const float* gr0 = B.g + arow[0] + py * Q1;
      const float* gr1 = B.g + arow[1] + py * Q1;
      const uint8_t* cr0 = B.cd + arow[0] + py * Q1;
      const uint8_t* cr1 = B.cd + arow[1] + py * Q1;
      const float* xr0 = B.x + xb[0] + 2 * py * IMG;
      const float* xr1 = B.x + xb[1] + 2 * py * IMG;
#pragma unroll
      for (int px = 0; px < Q1; ++px) {
        const float g0 = gr0[px], g1 = gr1[px];
        const int c0 = cr0[px], c1 = cr1[px];
        const float x0 = xr0[2 * px], x1 = xr1[2 * px];
        const float av0 = ((c0 == g) & aval[0]) ? g0 : 0.f;
        const float av1 = ((c1 == g) & aval[1]) ? g1 : 0.f;
        const float bv0 = bx[0] ? x0 : bconst[0];
        const float bv1 = bx[1] ? x1 : bconst[1];
        acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av0, bv0, acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av0, bv1, acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av1, bv0, acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av1, bv1, acc[1][1], 0, 0, 0);
      }
    }
    asm volatile("" ::: "memory");       // reads done before the next image's writes
  }
  // acc[mt][nt][r] = (o = 16 mt + 4 g + r, t = 16 nt + j); the four waves'
  // tiles meet in the staging LDS, now free
  __syncthreads();
  float (*red)[32][33] = reinterpret_cast<float (*)[32][33]>(&L[0]);
  static_assert(sizeof(float) * 4 * 32 * 33 <= sizeof(L), "reduction tiles fit in the staging LDS");
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wv][16 * mt + 4 * g + r][16 * nt + j] = acc[mt][nt][r];
  __syncthreads();
  // partial [i][jc][W1 (20 x 25) | b1 (20)]
  float* part = a.part1 + ((int64_t)i * gridDim.x + jc) * (W1LEN + NC1);
  for (int e = tid; e < NC1 * 26; e += 256) {
    const int o = e / 26, t = e % 26;
    const float s = ((red[0][o][t] + red[1][o][t]) + red[2][o][t]) + red[3][o][t];
    part[t < 25 ? o * 25 + t : W1LEN + o] = s;
  }
}

// ---------------------------------------------------------------------------
// G[i][off_c1 + e] = sum over chunks in order of the partials (conv1 block
// then conv2 block, which are contiguous in w).
__global__ __launch_bounds__(256) void k_cnn_wreduce(CnnArgs a, int chunks) {
  const int i = blockIdx.y;
  const int e = blockIdx.x * 256 + threadIdx.x;
  constexpr int L1 = W1LEN + NC1, L2 = NC2 * K2 + NC2;
  if (e >= L1 + L2) return;
  const float* src = e < L1 ? a.part1 + (int64_t)i * chunks * L1 + e : a.part2 + (int64_t)i * chunks * L2 + (e - L1);
  const int64_t stride = e < L1 ? L1 : L2;
  float s = 0.f;
  for (int j0 = 0; j0 < chunks; j0 += 8) {
    // eight chunks' partials in flight, then added in chunk order (a plain
    // loop over the run-time chunk count waits for each load in turn)
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = j0 + u < chunks ? src[(j0 + u) * stride] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (j0 + u < chunks) s += v[u];
  }
  if (!a.row_mask || a.row_mask[i]) a.G[(int64_t)i * a.P + a.off_c1 + e] = s;
}

}  // namespace

int cnn_chunks(int B) { return (B + kCnnChunk - 1) / kCnnChunk; }

hipError_t launch_cnn_grads(const MlpPlan& mplan, const CnnArgs& a, hipStream_t s) {
  const int64_t nB = (int64_t)a.n * a.B;
  hipLaunchKernelGGL(k_cnn_conv1_pool, dim3(static_cast<unsigned>((nB * NPOS1 + 255) / 256)), dim3(256), 0, s, a);
  const int64_t cv_blocks = nB < kConvBlocks ? nB : kConvBlocks;
  hipLaunchKernelGGL(k_cnn_conv2_pool, dim3(static_cast<unsigned>(cv_blocks)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the fully connected part: the MLP 800-H-C on the features, its G block
  // at the start of each row of G
  MlpArgs m{};
  m.w = a.w; m.X = a.F; m.y = a.ylab; m.rows = nullptr; m.S = 0;
  m.n = a.n; m.B = a.B; m.d = FEAT; m.H = a.H; m.C = a.C;
  m.G = a.G; m.ldG = a.P; m.loss = a.loss;
  m.Hh = a.Hh; m.dA = a.dA; m.Gp = a.Gp; m.lossp = a.lossp; m.err = a.err; m.row_mask = a.row_mask;
  e = launch_mlp_grads(mplan, m, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_cnn_dfeat, dim3((FEAT + 63) / 64, static_cast<unsigned>((nB + 63) / 64)), dim3(256), 0, s, a);
  const int64_t dg_blocks = nB < kDgradBlocks ? nB : kDgradBlocks;
  hipLaunchKernelGGL(k_cnn_conv2_dgrad, dim3(static_cast<unsigned>(dg_blocks)), dim3(256), 0, s, a);
  const int chunks = cnn_chunks(a.B);
  hipLaunchKernelGGL(k_cnn_conv2_wgrad, dim3(chunks, a.n), dim3(256), 0, s, a);
  hipLaunchKernelGGL(k_cnn_conv1_wgrad, dim3(chunks, a.n), dim3(256), 0, s, a);
  constexpr int LW = W1LEN + NC1 + NC2 * K2 + NC2;
  hipLaunchKernelGGL(k_cnn_wreduce, dim3((LW + 255) / 256, a.n), dim3(256), 0, s, a, chunks);
  return hipGetLastError();
}

}  // namespace dbw
