// bp_internal.h -- launch interface between the C-ABI host code (bp_net.cpp)
// and the gfx950 kernels (bp_kernels.hip).  Not part of the public ABI.
//
// Matrices are fp32 row-major with an explicit leading dimension (in floats).
// Weight layer l is stored as (n_l + 1) rows x ldw columns, ldw = n_{l+1}
// rounded up to a multiple of 4; row n_l is the bias ("true unit") row.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bpk {

// Number of blocks (and SSE partials) the output-layer forward launch uses.
int output_delta_blocks(int M, int N);

// out[m][n] = sigma(sum_k A[m][k] W[k][n] + bias[n]),  m < M, n < N, k < K.
hipError_t forward_layer(hipStream_t s, const float* A, int lda, const float* W, int ldw, int M, int N,
                         int K, const float* bias, float* out, int ldo);

// Output layer during training: y = sigma(A W + bias); e = T - y;
// delta[m][n] = e y (1 - y); sse_part[b] = sum of e^2 over the elements of
// block b (b < output_delta_blocks(M, N)).
hipError_t forward_output_delta(hipStream_t s, const float* A, int lda, const float* W, int ldw, int M,
                                int N, int K, const float* bias, const float* T, int ldt, float* delta,
                                int ldd, double* sse_part);

// Hidden deltas: out[m][n] = (sum_k D[m][k] W[n][k]) * act[m][n] (1 - act[m][n]),
// with W rows n < N the non-bias rows of the layer above (ldw floats apart).
hipError_t backward_layer(hipStream_t s, const float* D, int ldd, const float* W, int ldw, int M, int N,
                          int K, const float* act, int lda, float* out, int ldo);

// Number of K-splits change_update uses for an M x N change summed over K
// rows (1 = the product applies the update itself).
int change_splits(int M, int N, int K);

// Floats of split workspace change_update needs for an M x N change summed over K rows.
size_t change_update_workspace(int M, int N, int K);

// Weight change and update for the non-bias rows:
//   G[m][n] = sum_k A[k][m] D[k][n];  V = lr G + mom V;  W += V   (m < M, n < N).
// With change_splits(M, N, K) > 1 this launch only writes the partial sums
// to `ws` (change_update_workspace floats) and splitk_finish must follow.
hipError_t change_update(hipStream_t s, const float* A, int lda, const float* D, int ldd, int M, int N,
                         int K, float* W, float* V, int ldw, float lr, float mom, float* ws);

// Sums the split partials of change_update in split order, then updates V and W.
hipError_t splitk_finish(hipStream_t s, int M, int N, int K, float* W, float* V, int ldw, float lr, float mom,
                         const float* ws);

// Bias-row change and update: G[n] = sum_{k < rows} D[k][n];  V = lr G + mom V;  W += V.
hipError_t bias_update(hipStream_t s, const float* D, int ldd, int rows, int N, float* Wb, float* Vb,
                       float lr, float mom);

// One-hot first layer: net[p][j] = W0[n0][j] + sum_{k < n_active} W0[act[p][k]][j].
// mode 0: out[p][j] = sigma(net).  mode 1 (single-layer nets, training):
// y = sigma(net), out[p][j] = (T - y) y (1 - y) and sse_part[b] receives the
// block sums of (T - y)^2 (b < onehot_forward_blocks(rows, H)).
int onehot_forward_blocks(int rows, int H);
hipError_t onehot_forward(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw,
                          int n0, int H, int mode, float* out, int ldo, const float* T, int ldt,
                          double* sse_part);

// One-hot first-layer change and update for all n0 + 1 rows:
//   G[r][j] = sum over patterns p containing index r of D[p][j]  (r < n0),
//   G[n0][j] = sum_p D[p][j];  V = lr G + mom V;  W += V.
hipError_t onehot_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* D, int ldd,
                         int n0, int H, float* W, float* V, int ldw, float lr, float mom);

// out[0] = sum of part[0 .. n-1] in a fixed order (double).
hipError_t sse_reduce(hipStream_t s, const double* part, int n, double* out);

}  // namespace bpk
