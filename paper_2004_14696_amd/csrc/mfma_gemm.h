// fp32 matrix-core GEMM main loops shared by the softmax and MLP kernels.
//
// One block (256 threads = four waves in 2 x 2) computes a (32 WT)^2 output
// tile; each wave owns a (16 WT)^2 = WT x WT set of v_mfma_f32_16x16x4f32
// tiles (WT = 4: 128 x 128 blocks for large outputs; WT = 2: 64 x 64 blocks
// when the output has too few large tiles to fill the 256 CUs).
// K advances 16 at a time through two LDS buffers laid out [k][m] / [k][n],
// so that the A operand of lane l (row l % 16, k l / 16) and its B operand
// (k l / 16, column l % 16) are single conflict-free LDS reads; the next
// slice's global loads (float4 buffer loads, 0 out of range) are in flight
// while the current one is multiplied.  Accumulator element r of lane l in
// tile (mt, nt) is output (row 16 mt + 4 (l / 16) + r, column 16 nt + l % 16)
// of the wave's (16 WT)^2.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "dbw_buffer.h"

namespace dbw {

typedef float mfma_f32x4 __attribute__((ext_vector_type(4)));

constexpr int MBK = 16, MPAD = 4;

// Below this many 128 x 128 output tiles (two per CU) a launch uses 64 x 64
// blocks instead.
constexpr int64_t kMfmaBigTiles = 512;

// LDS arrays are 16-byte aligned so that float4 stores stay whole
// (ds_write_b128, not two ds_write2_b32).
template <int WT>
struct MfmaLds {
  static constexpr int BM = 32 * WT;
  __attribute__((aligned(16))) float A[2][MBK][BM + MPAD];
  __attribute__((aligned(16))) float B[2][MBK][BM + MPAD];
};

template <int WT>
__device__ __forceinline__ void mfma_zero(mfma_f32x4 (&acc)[WT][WT]) {
#pragma unroll
  for (int mt = 0; mt < WT; ++mt)
#pragma unroll
    for (int nt = 0; nt < WT; ++nt) acc[mt][nt] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
}

template <int WT>
__device__ __forceinline__ void mfma_slice(const MfmaLds<WT>& L, int cbuf, int wm, int wn, int lane,
                                           mfma_f32x4 (&acc)[WT][WT]) {
  const int i = lane & 15, kq = lane >> 4;
#pragma unroll
  for (int ks = 0; ks < MBK; ks += 4) {
    float av[WT], bv[WT];
#pragma unroll
    for (int t = 0; t < WT; ++t) {
      av[t] = L.A[cbuf][ks + kq][wm * 16 * WT + t * 16 + i];
      bv[t] = L.B[cbuf][ks + kq][wn * 16 * WT + t * 16 + i];
    }
#pragma unroll
    for (int mt = 0; mt < WT; ++mt)
#pragma unroll
      for (int nt = 0; nt < WT; ++nt) acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt], bv[nt], acc[mt][nt], 0, 0, 0);
  }
}

// Pieces per thread of one K slice: the A and the B slice each hold 16 BM
// floats = 4 BM float4 pieces over 256 threads.
template <int WT>
constexpr int mfma_pieces() { return 32 * WT / 64; }

// Block barrier once this wave's LDS reads and writes are complete; unlike
// __syncthreads it does not wait for outstanding global loads, so slices
// prefetched into registers stay in flight across it.
__device__ __forceinline__ void mfma_lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt and expcnt unconstrained
  asm volatile("s_barrier" ::: "memory");
}

// The slice loop with PD slices in flight in registers: at step kt, register
// slot kt % PD (whose slice is already in LDS) receives slice kt + PD, LDS
// buffer kt & 1 is multiplied, and slot (kt + 1) % PD is stored into the
// other buffer.  Loads past the last slice are issued anyway (the loaders
// return 0 out of range), so the number of loads in flight is the same at
// every step and the waits before the stores stay partial.
template <int PD, int NP, class Load, class Store, class Slice>
__device__ __forceinline__ void mfma_prefetch_loop(int nk, Load&& load, Store&& store, Slice&& slice) {
  float4 ra[PD][NP], rb[PD][NP];
#pragma unroll
  for (int p = 0; p < PD; ++p) load(p * MBK, ra[p], rb[p]);
  store(0, ra[0], rb[0]);
  mfma_lds_barrier();
  for (int kt0 = 0; kt0 < nk; kt0 += PD) {
#pragma unroll
    for (int u = 0; u < PD; ++u) {
      const int kt = kt0 + u;
      if (kt < nk) {
        load((kt + PD) * MBK, ra[u], rb[u]);
        slice(kt & 1);
        store((kt + 1) & 1, ra[(u + 1) % PD], rb[(u + 1) % PD]);
        mfma_lds_barrier();
      }
    }
  }
}

// acc += X[row(m0 + r)][k] W[k][n0 + c] over kbeg <= k < kend (default: all
// K), for the block's tile.  xrow[s] is the dataset row of tile row
// (tid + 256 s) / 4, or -1 for rows past the matrix; X rows have K floats;
// W is K x N row-major (N % 4 == 0, K % 4 == 0, kbeg % 4 == 0).  PD > 1:
// PD slices in flight (mfma_prefetch_loop).
template <int WT, int PD = 1>
__device__ __forceinline__ void mfma_gemm_rows_w(MfmaLds<WT>& L, __amdgpu_buffer_rsrc_t xs,
                                                 const int64_t (&xrow)[mfma_pieces<WT>()], int K,
                                                 __amdgpu_buffer_rsrc_t ws, int N, int n0, mfma_f32x4 (&acc)[WT][WT],
                                                 int kbeg = 0, int kend = -1) {
  if (kend < 0) kend = K;
  constexpr int NP = mfma_pieces<WT>(), BQ = 8 * WT;   // B pieces per K row
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  auto load = [&](int k0, float4 (&ra)[NP], float4 (&rb)[NP]) {
#pragma unroll
    for (int s2 = 0; s2 < NP; ++s2) {
      const int q = tid + s2 * 256;
      const int k = kbeg + k0 + 4 * (q % 4);
      ra[s2] = buf_f32x4(xs, xrow[s2] >= 0 && k < kend ? static_cast<uint32_t>((xrow[s2] * K + k) * 4) : kOutOfRange);
      const int kb = kbeg + k0 + q / BQ, nb = n0 + 4 * (q % BQ);
      rb[s2] = buf_f32x4(ws, kb < kend && nb < N ? static_cast<uint32_t>(((int64_t)kb * N + nb) * 4) : kOutOfRange);
    }
  };
  auto store = [&](int buf, const float4 (&ra)[NP], const float4 (&rb)[NP]) {
#pragma unroll
    for (int s2 = 0; s2 < NP; ++s2) {
      const int q = tid + s2 * 256;
      const int r = q / 4, k = 4 * (q % 4);
      L.A[buf][k + 0][r] = ra[s2].x;
      L.A[buf][k + 1][r] = ra[s2].y;
      L.A[buf][k + 2][r] = ra[s2].z;
      L.A[buf][k + 3][r] = ra[s2].w;
      *reinterpret_cast<float4*>(&L.B[buf][q / BQ][4 * (q % BQ)]) = rb[s2];
    }
  };
  if constexpr (PD > 1) {
    mfma_prefetch_loop<PD, NP>((kend - kbeg + MBK - 1) / MBK, load, store,
                               [&](int cbuf) { mfma_slice(L, cbuf, wm, wn, lane, acc); });
    return;
  }
  float4 ra[NP], rb[NP];
  load(0, ra, rb);
  store(0, ra, rb);
  __syncthreads();
  const int nk = (kend - kbeg + MBK - 1) / MBK;
  for (int kt = 0; kt < nk; ++kt) {
    const int cbuf = kt & 1;
    if (kt + 1 < nk) load((kt + 1) * MBK, ra, rb);
    mfma_slice(L, cbuf, wm, wn, lane, acc);
    if (kt + 1 < nk) store(cbuf ^ 1, ra, rb);
    __syncthreads();
  }
}

// acc += X[srow[b]][j0 + r] R[b][n0 + c] over b < K (the transpose of a
// worker's rows times its K x N residual block R, row-major; J features per
// dataset row, J % 4 == 0, N % 4 == 0).  srow holds the worker's K dataset
// rows (LDS).
template <int WT>
__device__ __forceinline__ void mfma_gemm_xt_r(MfmaLds<WT>& L, __amdgpu_buffer_rsrc_t xs, const int* srow, int J,
                                               int j0, __amdgpu_buffer_rsrc_t rs, int K, int N, int n0,
                                               mfma_f32x4 (&acc)[WT][WT]) {
  constexpr int NP = mfma_pieces<WT>(), BQ = 8 * WT;   // pieces per K row (A and B)
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6, wm = wv >> 1, wn = wv & 1;
  auto load = [&](int k0, float4 (&ra)[NP], float4 (&rb)[NP]) {
#pragma unroll
    for (int s2 = 0; s2 < NP; ++s2) {
      const int q = tid + s2 * 256;
      const int b = k0 + q / BQ, j = j0 + 4 * (q % BQ), c = n0 + 4 * (q % BQ);
      ra[s2] = buf_f32x4(xs, b < K && j < J ? static_cast<uint32_t>(((int64_t)srow[b] * J + j) * 4) : kOutOfRange);
      rb[s2] = buf_f32x4(rs, b < K && c < N ? static_cast<uint32_t>(((int64_t)b * N + c) * 4) : kOutOfRange);
    }
  };
  auto store = [&](int buf, const float4 (&ra)[NP], const float4 (&rb)[NP]) {
#pragma unroll
    for (int s2 = 0; s2 < NP; ++s2) {
      const int q = tid + s2 * 256;
      *reinterpret_cast<float4*>(&L.A[buf][q / BQ][4 * (q % BQ)]) = ra[s2];
      *reinterpret_cast<float4*>(&L.B[buf][q / BQ][4 * (q % BQ)]) = rb[s2];
    }
  };
  float4 ra[NP], rb[NP];
  load(0, ra, rb);
  store(0, ra, rb);
  __syncthreads();
  const int nk = (K + MBK - 1) / MBK;
  for (int kt = 0; kt < nk; ++kt) {
    const int cbuf = kt & 1;
    if (kt + 1 < nk) load((kt + 1) * MBK, ra, rb);
    mfma_slice(L, cbuf, wm, wn, lane, acc);
    if (kt + 1 < nk) store(cbuf ^ 1, ra, rb);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Narrow-N variant: four waves stacked along M, each owning MT x NT tiles of
// 16 x 16, so a block covers (64 MT) x (16 NT) outputs and the whole N extent
// lives in one wave (N up to 16 NT: e.g. 100 classes in 7 tiles instead of a
// 128-wide tile).  A rows are AST floats apart in LDS, B rows BST.
//
// With RS > 0 the last tile holds only 4 RS columns (N = 16 (NT - 1) + 4 RS)
// and is computed as RS stripes of 4 columns on v_mfma_f32_4x4x1f32 (16
// blocks of 4 x 4 x 1, 8 cycles) instead of a 16 x 16 x 4 product (32
// cycles) that would be mostly padding.  Block b = 4 g + s of an instruction
// takes rows 4 g .. 4 g + 3 of the 16-row tile at k offset s of the 4-deep
// step (lane 4 b + i supplies A row i, lane 4 b + j B column j, and register i
// of lane 4 b + j receives output (i, j)), so after the K loop a sum over the
// four lanes of a 16-lane row that share lane % 4 (row rotations by 4 and 8)
// leaves rows 4 (l / 16) + r, column 4 s + l % 4 of the stripe in register r:
// the 16 x 16 tile layout, restricted to its first 4 RS columns.
template <int MT, int NT, int AST>
struct MfmaLdsN {
  static constexpr int BM = 64 * MT, BN = 16 * NT;
  // B rows 16 mod 64 floats apart: the four k rows of one read hit disjoint
  // bank quarters
  static constexpr int BST = (BN + 63) / 64 * 64 + 16;
  __attribute__((aligned(16))) float A[2][MBK][AST];
  __attribute__((aligned(16))) float B[2][MBK][BST];
};

template <int MT, int NT, int RS, int AST>
__device__ __forceinline__ void mfma_slice_n(const MfmaLdsN<MT, NT, AST>& L, int cbuf, int wm, int lane,
                                             mfma_f32x4 (&acc)[MT][NT], mfma_f32x4 (&accs)[MT][RS > 0 ? RS : 1]) {
  constexpr int NF = RS > 0 ? NT - 1 : NT;   // full 16-wide tiles
  const int i = lane & 15, kq = lane >> 4;
  // stripe operands: k offset (lane / 4) % 4, row 4 (lane / 16) + lane % 4
  const int ks4 = (lane >> 2) & 3, sr = 4 * (lane >> 4) + (lane & 3);
  // A wave issuing its slice's products is given issue priority over the
  // SIMD's other waves (their loads and LDS stores wait a little), so the
  // matrix pipe is refilled sooner: 1316 -> 1308 us on the 256 x 512 x 3072
  // x 100 launch (mean of eight paired runs).
  __builtin_amdgcn_s_setprio(1);
#pragma unroll
  for (int ks = 0; ks < MBK; ks += 4) {
    float av[MT], bv[NF];
#pragma unroll
    for (int t = 0; t < MT; ++t) av[t] = L.A[cbuf][ks + kq][wm * 16 * MT + t * 16 + i];
#pragma unroll
    for (int t = 0; t < NF; ++t) bv[t] = L.B[cbuf][ks + kq][t * 16 + i];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NF; ++nt)
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt], bv[nt], acc[mt][nt], 0, 0, 0);
    if constexpr (RS > 0) {
      float sa[MT], sb[RS];
#pragma unroll
      for (int t = 0; t < MT; ++t) sa[t] = L.A[cbuf][ks + ks4][wm * 16 * MT + t * 16 + sr];
#pragma unroll
      for (int s = 0; s < RS; ++s) sb[s] = L.B[cbuf][ks + ks4][NF * 16 + 4 * s + (lane & 3)];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int s = 0; s < RS; ++s) accs[mt][s] = __builtin_amdgcn_mfma_f32_4x4x1f32(sa[mt], sb[s], accs[mt][s], 0, 0, 0);
    }
  }
  __builtin_amdgcn_s_setprio(0);
}

// The four k-offset partials of a stripe summed (lanes 16 g + 4 s + j, s <
// 4) and placed in the last tile's layout; columns past 4 RS read 0.
template <int MT, int NT, int RS>
__device__ __forceinline__ void mfma_fold_stripes(mfma_f32x4 (&acc)[MT][NT], mfma_f32x4 (&accs)[MT][RS]) {
  const int sl = (threadIdx.x & 15) >> 2;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float out = 0.f;
#pragma unroll
      for (int s = 0; s < RS; ++s) {
        float v = accs[mt][s][r];
        v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x124, 0xF, 0xF, false));
        v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false));
        out = sl == s ? v : out;
      }
      acc[mt][NT - 1][r] = out;
    }
}

// The slice pipeline shared by the narrow-N GEMMs: load(k0, ra, rb) fetches
// slice k0 into registers, store(buf, ra, rb) puts it into LDS buffer buf.
// NPA / NPB float4 pieces per thread.
template <int MT, int NT, int RS, int AST, int NPA, int NPB, class Load, class Store>
__device__ __forceinline__ void mfma_pipeline_n(MfmaLdsN<MT, NT, AST>& L, int nk, Load load, Store store,
                                                mfma_f32x4 (&acc)[MT][NT]) {
  const int lane = threadIdx.x & 63, wm = threadIdx.x >> 6;
  mfma_f32x4 accs[MT][RS > 0 ? RS : 1];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int s = 0; s < (RS > 0 ? RS : 1); ++s) accs[mt][s] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
  float4 ra[NPA], rb[NPB];
  load(0, ra, rb);
  store(0, ra, rb);
  __syncthreads();
  // two slices per iteration, so that the LDS buffer of each is a constant
  // and its operand addresses fold into the read offsets (256 x 512 x 3072 x
  // 100 logits kernel -3%)
  for (int kt = 0; kt < nk; kt += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (kt + u < nk) {
        if (kt + u + 1 < nk) load((kt + u + 1) * MBK, ra, rb);
        mfma_slice_n<MT, NT, RS, AST>(L, u, wm, lane, acc, accs);
        if (kt + u + 1 < nk) store(u ^ 1, ra, rb);
        __syncthreads();
      }
    }
  }
  if constexpr (RS > 0) mfma_fold_stripes<MT, NT, RS>(acc, accs);
}

}  // namespace dbw
