// Internal declarations of the DBW library: device workspace layout, kernel
// launchers and the host time estimator.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "dbw.h"

namespace dbw {

// Device error flags (OR-ed by kernels, read and cleared by dbw_sync).
enum : int32_t {
  ERR_ROW_RANGE = 1,    // minibatch row index outside [0, S)
  ERR_K_RANGE = 2,      // k larger than the number of workers that arrive
  ERR_LABEL_RANGE = 4,  // label outside [0, C)
  ERR_MASK_COUNT = 8,   // mask does not hold exactly k ones
};

// Column tile of the aggregation kernel: 64 lanes x 4 columns.
constexpr int AGG_TILE = 256;
constexpr int AGG_WAVES = 4;

inline int64_t agg_blocks(int64_t P) { return (P + AGG_TILE - 1) / AGG_TILE; }

// ---------------------------------------------------------------------------
// Worker-gradient plans.
struct SoftmaxPlan {
  int fused = 0;          // 2: matrix-core single pass; 1: VALU single pass; 0: GEMM path
  int threads = 0;        // fused: threads per block
  int per_thread = 0;     // fused 1: d-elements per thread (M); fused 2: float4 groups per lane (U)
  int cpad = 0;           // fused: class template (>= C)
  int slabs = 1;          // fused: row slabs per worker
  int rows_per_slab = 0;
  int64_t part = 0;       // floats of one slab partial (fused, slabs > 1)
};

struct MlpPlan {
  int ok = 0;
  int cpad = 0;           // class template (>= C)
  int threads = 0;        // head kernel threads per block
  int per_thread = 0;     // hidden units per head thread
  int slabs = 1;          // row slabs per worker in the head kernel
  int rows_per_slab = 0;
  int64_t tail = 0;       // H + H*C + C: the [b1 | W2 | b2] segment of G
};

// Softmax regression: G = per-worker gradient of the mean CE of softmax(X W).
struct SoftmaxArgs {
  const float* W;        // [d][C]
  const float* X;        // [n*B][d] or dataset [S][d]
  const int32_t* y;      // [n*B] or [S]
  const int32_t* rows;   // nullable [n*B]
  int64_t S;
  int n, B, d, C;
  float* G;              // [n][d*C]
  float* loss;           // [n]
  // workspace
  float* Gp;             // [n*slabs][d*C] slab partials (fused, slabs > 1)
  float* lossp;          // [n*slabs]
  float* Z;              // [n*B][C] logits / residuals (GEMM path)
  float* ce;             // [n*B] per-row CE (GEMM path)
  int32_t* err;
  int keep_slabs;        // 1: leave the slab partials for the PS kernel (no slab reduction)
  const uint8_t* row_mask;  // nullable [n]: G rows only of workers with a nonzero entry
};

SoftmaxPlan softmax_plan(int n, int B, int d, int C);
hipError_t launch_softmax_grads(const SoftmaxPlan& plan, const SoftmaxArgs& a, hipStream_t s);

struct MlpArgs {
  const float* w;        // [P] flat parameters
  const float* X;
  const int32_t* y;
  const int32_t* rows;
  int64_t S;
  int n, B, d, H, C;
  float* G;              // [n][ldG]: the MLP's P floats at the start of each row
  int64_t ldG;           // row stride of G (0: P)
  float* loss;           // [n]
  // workspace
  float* Hh;             // [n*B][H] hidden activations (with ksplit 2: the first
                         // K half's pre-activation sums, dA the second's)
  float* dA;             // [n*B][H] gradient w.r.t. pre-activations
  int ksplit;            // set by launch_mlp_grads
  float* Gp;             // [n*slabs][H + H*C + C] head slab partials
  float* lossp;          // [n*slabs]
  int32_t* err;
  const uint8_t* row_mask;  // nullable [n]: G rows only of workers with a nonzero entry
};
MlpPlan mlp_plan(int n, int B, int d, int H, int C);
hipError_t launch_mlp_grads(const MlpPlan& plan, const MlpArgs& a, hipStream_t s);

// The MNIST-shaped CNN: 28 x 28 images, conv 5 x 5 to 20 channels, 2 x 2 max
// pooling, ReLU, conv 5 x 5 to 50 channels, pooling, ReLU, then the MLP
// 800-H-C.  Parameters [MLP (800-H-C) | Wc1 (20x1x5x5) | bc1 | Wc2 (50x20x5x5) | bc2].
constexpr int CNN_IMG = 28, CNN_C1 = 20, CNN_C2 = 50, CNN_FEAT = 800;
constexpr int64_t CNN_CONV_PARAMS = CNN_C1 * 25 + CNN_C1 + CNN_C2 * CNN_C1 * 25 + CNN_C2;
constexpr int kCnnChunk = 16;   // images per weight-gradient partial
struct CnnArgs {
  const float* w;        // [P]
  const float* X;        // [n*B][784] or dataset [S][784]
  const int32_t* y;
  const int32_t* rows;   // nullable [n*B]
  int64_t S;
  int n, B, H, C;
  int64_t P, off_c1, off_c2;   // parameter count, offsets of Wc1 and Wc2
  float* G;              // [n][P]
  float* loss;           // [n]
  // workspace
  float* H1;             // [n*B][20][12][12] pooled, ReLU'd conv1 output
  uint8_t* code1;        // [n*B][20][12][12] window code of each pooled value (4: ReLU off)
  float* F;              // [n*B][800] pooled, ReLU'd conv2 output (the features)
  uint8_t* code2;        // [n*B][800] window codes of the features (4: ReLU off)
  int32_t* ylab;         // [n*B] gathered labels
  float* dP2;            // [n*B][800] gradient at the features (before their ReLU)
  float* dP1;            // [n*B][2880] gradient at H1 (before its ReLU)
  float* part1;          // [n][chunks][520] conv1 weight-gradient partials
  float* part2;          // [n][chunks][25050] conv2 weight-gradient partials
  int chunk;             // images per partial
  float* Hh;             // MLP workspace
  float* dA;
  float* Gp;
  float* lossp;
  int32_t* err;
  const uint8_t* row_mask;  // nullable [n]: G rows only of workers with a nonzero entry
};
int cnn_chunks(int B);
hipError_t launch_cnn_grads(const MlpPlan& mplan, const CnnArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// PS side.
struct ChooseArgs {
  const dbw_estimator_state* st;  // device
  const double* T_src;            // [n] time estimates (device or pinned host)
  const int64_t* ticks_src;       // [n] ticks (device or pinned host)
  const int32_t* order_src;       // [n] workers by (tick, index) (pinned host; k_step_ps only)
  double* T_hat;                  // nullable device copy of T_src
  int64_t* ticks;                 // nullable device copy of ticks_src
  int32_t* k_host;                // nullable pinned host copy of k
  int n;
  double eta, beta;
  int policy;                     // dbw_policy
  int k_static;                   // k under DBW_POLICY_STATIC
  int do_choose, do_select;
  int k_imm;                      // k when not choosing
  int32_t* k_out;                 // device (choose) -- also read by select
  int32_t* b_out;
  double* objective;              // nullable
  int32_t* sel;                   // device [n] arrival-ordered selection
  uint8_t* mask;                  // device [n]
  int32_t* err;
};
hipError_t launch_choose_select(const ChooseArgs& a, hipStream_t s);

enum AggMode { AGG_MEAN = 0, AGG_STATS_GIVEN_MEAN = 1, AGG_FUSED = 2 };
struct AggArgs {
  const float* G;       // [n][P]
  int64_t P;
  int n;
  const int32_t* sel;   // arrival order (AGG_MEAN, AGG_FUSED)
  // AGG_MEAN with ticks_sel set: every block takes the k fastest workers by
  // (tick, index) itself (sel unused); block 0 writes mask_out [n] and
  // reports k beyond the finite ticks in err
  const int64_t* ticks_sel;
  uint8_t* mask_out;
  int32_t* err;
  const uint8_t* sel_mask;  // AGG_STATS_GIVEN_MEAN: the selected rows, as a mask [n]
  const int32_t* k_dev; // nullable -> k_imm
  int k_imm;
  const float* g_in;    // AGG_STATS_GIVEN_MEAN
  float* g_out;         // AGG_MEAN, AGG_FUSED
  float* w;             // AGG_FUSED: updated in place (nullable: no update)
  float eta;
  float* sqpart;        // [n][nblocks]
  double* part;         // [nblocks][2]
  int mode;
  // k_step_ps only: where worker j's gradient row comes from
  int src;              // AggSrc
  const float* Gp;      // SRC_SLABS*: slab partials, worker j's slab q at (j slabs + q) slab_len
  int slabs;
  int64_t slab_len;     // floats of one slab partial (a multiple of 4)
  int d, C, B;
  const float* lossp;   // [n][slabs] slab loss sums -> loss[n] (the mean over B)
  float* loss;
  float* G_rows;        // nullable: the selected rows are written here in [d][C] order
};
// Gradient rows of k_step_ps: the G rows themselves, or the sum of a worker's
// slab partials in slab order, laid out as [d][C] or in the matrix-core
// kernel's tile order (64-feature groups; see k_softmax.hip).
enum AggSrc { SRC_ROWS = 0, SRC_SLABS = 1, SRC_SLAB_TILES = 2 };
hipError_t launch_aggregate(const AggArgs& a, hipStream_t s);
// Choice, selection by the host-sorted arrival order, and fused aggregation
// in one launch (dbw_step); ca.order_src must be set.  Used up to this many
// column tiles (about two blocks per CU).
constexpr int64_t kStepPsMaxBlocks = 512;
// T_hat, the arrival order and the ticks passed in k_step_ps's kernel
// arguments when n <= kInlineN (n_inline = n; 0: they are read from
// ca.T_src, ca.order_src and ca.ticks_src).  Every block reads them, so this
// replaces reads of uncached pinned host memory by reads of the argument
// segment.
constexpr int kInlineN = 64;
struct StepInline {
  double T[kInlineN];
  int64_t ticks[kInlineN];
  int32_t order[kInlineN];
  int n_inline;
};
hipError_t launch_step_ps(const ChooseArgs& ca, const AggArgs& a, const StepInline& inl, hipStream_t s);

struct FinalizeArgs {
  const float* sqpart;  // [n][nblocks]
  const double* part;   // [nblocks][2]
  int64_t nblocks;
  const uint8_t* mask;  // [n]
  const int32_t* k_dev; // nullable -> k_imm
  int k_imm;
  const float* loss;    // [n]
  int n;
  float* sqnorm;        // [n]
  dbw_iter_stats* stats;
  dbw_estimator_state* st;  // device; read (window mean), written if bookkeeping;
                            // nullable when bookkeeping is 0 and v_window_given is set
  double eta;
  int D;
  int bookkeeping;
  int v_window_given;       // V_plus for k = 1 is v_window, not the state's window mean
  double v_window;
  int32_t* err;             // nullable: a mask count other than k then gives NaN statistics
};
hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s);

// Error text of the context-free calls (per calling thread; dbw_last_error
// with a NULL context returns it).  Returns s.
dbw_status set_free_error(dbw_status s, const char* fmt, ...);


// ---------------------------------------------------------------------------
// Host time estimator (exact constrained least squares).  An IsoSolver keeps
// the previous solution and re-certifies it against new samples (exact warm
// start); time_estimate() is the stateless full solve.
class IsoSolver {
 public:
  IsoSolver();
  ~IsoSolver();
  IsoSolver(const IsoSolver&) = delete;
  IsoSolver& operator=(const IsoSolver&) = delete;
  // Returns 0 on success, -1 on invalid input (reason in *why).  With
  // changed_rows, the caller guarantees that only those rows (1-based) of the
  // grid differ from the previous call on this solver, which then validates
  // and diffs only them.
  int solve(int n, const int64_t* cnt, const int64_t* tsum, double* T_hat, std::string* why,
            const std::vector<int>* changed_rows = nullptr);
  void reset();
  int64_t full_solves() const;
  int64_t warm_solves() const;
  int64_t fast_solves() const;

 private:
  struct Impl;
  Impl* p_;
};
int time_estimate(int n, const int64_t* cnt, const int64_t* tsum, double* T_hat, std::string* why);

}  // namespace dbw
