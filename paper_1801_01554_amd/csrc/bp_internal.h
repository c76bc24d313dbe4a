// bp_internal.h -- launch interface between the C-ABI host code (bp_net.cpp)
// and the gfx950 kernels (bp_kernels.hip).  Not part of the public ABI.
//
// Matrices are fp32 row-major with an explicit leading dimension (in floats).
// Weight layer l is stored as (n_l + 1) rows x ldw columns, ldw = n_{l+1}
// rounded up to a multiple of 4; row n_l is the bias ("true unit") row.
//
// Options of the method, passed to the kernels they affect:
//   tab            the 256-entry sigmoid table (section 4.3) in device memory,
//                  or nullptr for the exact logistic;
//   limit, faults  the range check of summed changes (section 8): with
//                  limit > 0 every summed change outside [-limit, limit] (or
//                  NaN) is replaced by 0 and counted in *faults (device).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bpk {

// Measurement: when `start` is set, the next kernel launch of this thread
// records its execution start and end on these events (taken from the
// dispatch itself, hipExtLaunchKernel), then clears them and sets `used`.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  bool used = false;
};
LaunchEvents& launch_events();

template <class K, class... Args>
hipError_t launch_kernel(K kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t s, Args... args) {
  LaunchEvents& ev = launch_events();
  if (ev.start) {
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)shmem, s, ev.start, ev.stop, 0u, args...);
    ev.start = ev.stop = nullptr;
    ev.used = true;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  }
  return hipGetLastError();
}

// Rows of the per-tile column sums a delta-producing launch over M rows writes.
int colsum_rows(int M);

// out[m][n] = sigma(sum_k A[m][k] W[k][n] + bias[n]),  m < M, n < N, k < K.
hipError_t forward_layer(hipStream_t s, const float* A, int lda, const float* W, int ldw, int M, int N,
                         int K, const float* bias, float* out, int ldo, const float* tab);

// The first layer of an Elman step with its input built in the product
// (section 10.5): A[m][k] = X[m][k] (X rows n_ext wide) for k < n_ext and
// cont[m] H[m][k - n_ext] for k in [n_ext, K), H the previous step's first
// hidden layer, whose first K - n_ext units the context copies in order;
// out = sigma(A W + bias) as forward_layer.  rows_out (or nullptr) receives
// A, with zeros in [K, ld_rows).  Only for forward_ctx_fits(M, N, K);
// otherwise, or for a missing pointer, hipErrorInvalidValue.
bool forward_ctx_fits(int M, int N, int K);
hipError_t forward_ctx_layer(hipStream_t s, const float* X, int n_ext, const float* H, int ldh, const float* cont,
                             const float* W, int ldw, int M, int N, int K, const float* bias, float* out, int ldo,
                             float* rows_out, int ld_rows, const float* tab);

// An Elman net with one hidden layer: step t + 1's hidden layer (as
// forward_ctx_layer, from Hprev = step t's hidden rows into Hnext, rows built
// into rows_out or nowhere) and step t's output layer with its deltas (as
// forward_output_delta with A = Hprev) in one launch.  All hidden rows have
// stride ldh.  Only for elman_pair_fits(S, n0, n1, n2) (then
// output_delta_blocks(S, n2, n1) error partials); otherwise, or for a
// missing pointer, hipErrorInvalidValue.
bool elman_pair_fits(int S, int n0, int n1, int n2);
hipError_t elman_pair(hipStream_t s, const float* X, int n_ext, const float* Hprev, const float* cont,
                      const float* W0, int ldw0, const float* bias0, int n0, int n1, float* Hnext, float* rows_out,
                      int ld_rows, const float* W1, int ldw1, const float* bias1, int n2, int ldh, int S,
                      const float* T, int ldt, float* delta, int ldd, double* sse_part, float* colsum, int ldcs,
                      const float* tab, const float* mask);

// Output layer during training: y = sigma(A W + bias); e = (T - y) * mask[m]
// (mask == nullptr: no mask);
// delta[m][n] = e y (1 - y); sse_part[b] = sum of e^2 over the elements of
// block b (b < output_delta_blocks(M, N, K)); colsum[t][n] = sum of delta
// over rows [64 t, 64 t + 64) (t < colsum_rows(M)).  With
// output_delta_splits(M, N, K) > 1 the product writes split partials to `ws`
// (output_delta_workspace floats) and output_finish applies the epilogue.
int output_delta_blocks(int M, int N, int K);
int output_delta_splits(int M, int N, int K);
size_t output_delta_workspace(int M, int N, int K);
hipError_t forward_output_delta(hipStream_t s, const float* A, int lda, const float* W, int ldw, int M,
                                int N, int K, const float* bias, const float* T, int ldt, float* delta,
                                int ldd, double* sse_part, float* colsum, int ldcs, float* ws, const float* tab,
                                const float* mask);
hipError_t output_finish(hipStream_t s, int M, int N, int K, const float* bias, const float* T, int ldt, float* delta,
                         int ldd, double* sse_part, float* colsum, int ldcs, const float* ws, const float* tab,
                         const float* mask);

// Hidden deltas: out[m][n] = (sum_k D[m][k] W[n][k]) * act[m][n] (1 - act[m][n]),
// with W rows n < N the non-bias rows of the layer above (ldw floats apart);
// colsum as for the output layer.
hipError_t backward_layer(hipStream_t s, const float* D, int ldd, const float* W, int ldw, int M, int N,
                          int K, const float* act, int lda, float* out, int ldo, float* colsum, int ldcs);

// Number of K-splits change_update uses for an M x N change summed over K
// rows (1 = one block per output tile applies the update from its
// accumulators).
int change_splits(int M, int N, int K);

// Floats of split workspace change_update needs for an M x N change summed over K rows.
size_t change_update_workspace(int M, int N, int K);

// Arrival counters (one per output tile) a split change_update of an M x N
// change summed over K rows uses; 0 when it is not split.  Never more than
// kMaxArrivals: a product is split only when it has fewer output tiles than
// that.
constexpr int kMaxArrivals = 512;
int change_arrivals(int M, int N, int K);

// Weight change and update for the non-bias rows:
//   G[m][n] = sum_k A[k][m] D[k][n];  V = lr G + mom V;  W += V   (m < M, n < N).
// With change_splits(M, N, K) > 1 the blocks of each output tile write their
// partial sums to `ws` (change_update_workspace floats) and the last one to
// arrive adds them in split order and applies the update, counting arrivals
// in `arrivals` (kMaxArrivals ints, all zero before the launch and left zero
// after it; launches that use them must not overlap).
hipError_t change_update(hipStream_t s, const float* A, int lda, const float* D, int ldd, int M, int N,
                         int K, float* W, float* V, int ldw, float lr, float mom, float* ws, int* arrivals,
                         float limit, unsigned long long* faults);

// Bias-row change and update of one layer: G[n] = sum_{k < rows} D[k][n];
// V = lr G + mom V;  W += V.  D is the per-tile column-sum buffer of the
// deltas (rows = colsum_rows(batch)); Wb, Vb the bias rows of W and V.
struct BiasJob {
  const float* D;
  float* Wb;
  float* Vb;
  int ldd, rows, N;
  int block0;   // set by bias_update
};
constexpr int kMaxBiasJobs = 8;
struct BiasJobs {
  BiasJob j[kMaxBiasJobs];
  int n;
};
// The bias updates of n layers (independent: distinct D, Wb, Vb), up to
// kMaxBiasJobs per launch.
hipError_t bias_update(hipStream_t s, const BiasJob* jobs, int n, float lr, float mom, float limit,
                       unsigned long long* faults);

// One-hot first layer: net[p][j] = W0[n0][j] + sum_{k < n_active} W0[act[p][k]][j].
// mode 0: out[p][j] = sigma(net).  mode 1 (single-layer nets, training):
// y = sigma(net), out[p][j] = (T - y) y (1 - y) and sse_part[b] receives the
// block sums of (T - y)^2 (b < onehot_forward_blocks(rows, H)).
int onehot_forward_blocks(int rows, int H);
hipError_t onehot_forward(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw,
                          int n0, int H, int mode, float* out, int ldo, const float* T, int ldt,
                          double* sse_part, const float* tab);

// One-hot first-layer change and update for all n0 + 1 rows:
//   G[r][j] = sum over patterns p containing index r of D[p][j]  (r < n0),
//   G[n0][j] = sum_p D[p][j];  V = lr G + mom V;  W += V.
hipError_t onehot_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* D, int ldd,
                         int n0, int H, float* W, float* V, int ldw, float lr, float mom, float limit,
                         unsigned long long* faults);

// ---- fused path for small two-layer nets with one-hot inputs (bp_small.hip)
constexpr int kSmallMaxHidden = 256;
constexpr int kSmallMaxOut = 64;
constexpr int kSmallMaxActive = 32;   // active inputs per pattern

// True if a one-hot net n0 - H - O fits the fused path.
bool small_path_fits(int n0, int H, int O, int n_active);

// Number of blocks (and error partials) of small_fwdbwd for `rows` patterns.
int small_fwdbwd_blocks(int rows);

// Floats of scratch the fused path needs for a batch of `rows` patterns
// (the hidden activations in groups of four units).
size_t small_scratch_floats(int rows, int H);

// Per pattern: A1 = sigma(W0 gather + bias), Y = sigma(A1 W1 + bias1),
// D2 = (T - Y) Y (1 - Y), D1 = (D2 W1^T) A1 (1 - A1); error partials per
// block.  A1 is written in groups of four units: A1q[((j / 4) rows + p) 4 + j % 4].
hipError_t small_fwdbwd(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw0, int n0,
                        int H, const float* W1, int ldw1, int O, const float* T, float* A1q, float* D1, int ldd1,
                        float* D2, int ldd2, double* sse_part, const float* tab);

// Summed changes of both layers over the batch and the momentum update of all
// weights.  With sse_out != nullptr (the last update of a call) one more
// block writes the sum of sse_part[0, n_sse) to sse_out, as sse_reduce.
hipError_t small_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* A1q, const float* D1,
                        int ldd1, const float* D2, int ldd2, float* W0, float* V0, int ldw0, int n0, int H, float* W1,
                        float* V1, int ldw1, int O, float lr, float mom, float limit, unsigned long long* faults,
                        const double* sse_part = nullptr, int n_sse = 0, double* sse_out = nullptr);

// ---- Elman nets (bp_seq.hip, section 10.5)
// Hidden layers a context unit may copy from: 1 .. kCtxMaxLayer.
constexpr int kCtxMaxLayer = 8;

// Rows of the previous step's activations, per hidden layer (base[l] ==
// nullptr: no previous step, the context is 0 times the flag).
struct CtxSource {
  const float* base[kCtxMaxLayer + 1];
  int ld[kCtxMaxLayer + 1];
};

// Input rows of one step for S streams: A0[s][0 .. n_ext) = X[s][..];
// A0[s][n_ext + c] = cont[s] * src.base[layer[c]][s * ld + unit[c]];
// A0[s][n0 .. lda0) = 0.
hipError_t seq_assemble(hipStream_t s, const float* X, int n_ext, const float* cont, int S, int n_ctx,
                        const int32_t* ctx_layer, const int32_t* ctx_unit, const CtxSource& src, float* A0,
                        int lda0);

// The forward pass of one window of an Elman net with one hidden layer whose
// context copies the hidden units in order (section 10.5), all steps in one
// launch.  Streams are independent, so each block keeps the recurrence of
// its own streams: step k's input rows (X, then cont x the hidden units of
// step k - 1 of the same stream; step 0 takes them from Hprev, or zero),
// hidden units, output units and output deltas, with no exchange between
// blocks.  Step k of the window is rows k * S .. k * S + S - 1 of H, rows, D
// (and of X, cont, mask, T, each given at the window's first step).  Block b
// writes the error sum of its rows of step k to sse[k * blocks + b] and the
// column sums of its deltas over the whole window to colsum row b, blocks =
// elman_window_blocks(S).  Only for elman_window_fits(...); otherwise, or
// for a missing pointer, hipErrorInvalidValue.
struct ElmanWindow {
  const float* X;          // [steps * S][n_ext]
  int n_ext;
  const float* cont;       // [steps * S]
  const float* mask;       // [steps * S] or nullptr (no mask)
  const float* T;          // [steps * S][ldt]
  int ldt;
  const float* Hprev;      // context source of step 0: [S][ldhp], or nullptr
  int ldhp;
  const float* W0;         // [n0][ldw0], bias row b0
  int ldw0;
  const float* b0;
  const float* W1;         // [n1][ldw1], bias row b1
  int ldw1;
  const float* b1;
  int n0, n1, n2;
  float* H;                // hidden units [steps * S][ldh]
  int ldh;
  float* rows;             // input rows [steps * S][ldr]
  int ldr;
  float* D;                // output deltas [steps * S][ldd]
  int ldd;
  float* colsum;           // [blocks][ldcs]
  int ldcs;
  double* sse;             // [steps * blocks]
  const float* tab;
  int S, steps;
};
bool elman_window_fits(int S, int n_ext, int n0, int n1, int n2);
int elman_window_blocks(int S);
hipError_t elman_window(hipStream_t s, const ElmanWindow& w);

// out[0] = sum of part[0 .. n-1] in a fixed order (double).
hipError_t sse_reduce(hipStream_t s, const double* part, int n, double* out);

// Sets p[0, n) to zero with a kernel (no memset node when captured).
hipError_t zero_ints(hipStream_t s, int* p, int n);

}  // namespace bpk
