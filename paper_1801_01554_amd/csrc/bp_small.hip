// bp_small.hip -- fused pooled update for small two-layer nets with one-hot
// inputs (the NETtalk shape: a 7 x 29 one-hot window, a hidden layer of a
// few hundred units at most, a few dozen outputs; section 6.3).
//
// The generic path runs six dependent launches per update, each far too
// small to fill the chip, so an update is bound by launch and pipeline
// latency.  Here one update is two launches:
//
//   small_fwdbwd   per pattern, entirely on chip: gather the active rows of
//                  W0 (+ bias) -> sigma -> hidden activations; output layer
//                  with W1 held in LDS -> sigma -> output deltas and squared
//                  error; hidden deltas from the same W1 (before its update).
//                  Each block handles P patterns.
//   small_update   the summed changes of both layers and the momentum update
//                  of every weight.  Each output element is summed over the
//                  batch in pattern order by a fixed set of lanes, partial
//                  sums combined in a fixed order: no atomics, run-to-run
//                  identical.
//
// Arithmetic per element is the method's (sections 3 and 6.2.1); only the
// grouping of the work differs from the generic path.
#include <hip/hip_runtime.h>

#include "bp_internal.h"

namespace bpk {
namespace {

constexpr int kT = 256;        // threads per forward/backward block
constexpr int kTU = 1024;      // threads per update block (16 waves)
constexpr int kWU = kTU / 64;
constexpr int kMaxP = 8;       // patterns per forward/backward block
constexpr int kU = 32;         // loads kept in flight per lane in the batch sums

__device__ __forceinline__ float logistic(float z) { return 1.0f / (1.0f + expf(-z)); }

// sum_{p in [r0, r1)} x[p * ldx] * y[p * ldy], added in pattern order; the
// loads of kU consecutive patterns are issued before their products are added.
__device__ __forceinline__ float dot_rows(const float* __restrict__ x, int ldx, const float* __restrict__ y, int ldy,
                                          int r0, int r1) {
  float g = 0.f;
  for (int p = r0; p < r1; p += kU) {
    float a[kU], d[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      a[u] = p + u < r1 ? x[(size_t)(p + u) * ldx] : 0.f;
      d[u] = p + u < r1 ? y[(size_t)(p + u) * ldy] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (p + u < r1) g += a[u] * d[u];
  }
  return g;
}

// sum_{p in [r0, r1)} y[p * ldy], added in pattern order, kU loads in flight.
__device__ __forceinline__ float sum_rows(const float* __restrict__ y, int ldy, int r0, int r1) {
  float g = 0.f;
  for (int p = r0; p < r1; p += kU) {
    float d[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) d[u] = p + u < r1 ? y[(size_t)(p + u) * ldy] : 0.f;
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (p + u < r1) g += d[u];
  }
  return g;
}

// Dynamic LDS of small_fwdbwd: W1 as (H + 1) x (O + 1) (odd row stride so
// that column walks by consecutive hidden units hit distinct banks), the
// hidden activations [P][H], the output deltas [P][O], the targets [P][O]
// and the active indices [P][n_active] of the block's patterns.
//
// The kernel has two rounds of global loads: (1) indices, targets and W1,
// all independent; (2) the gathered W0 rows of all the block's patterns.
__global__ __launch_bounds__(kT) void small_fwdbwd_kernel(const int32_t* __restrict__ act, int n_active, int rows,
                                                          int P, const float* __restrict__ W0, int ldw0, int n0,
                                                          int H, const float* __restrict__ W1, int ldw1, int O,
                                                          const float* __restrict__ T, float* A1, int lda1,
                                                          float* D1, float* D2, int ldd2, double* sse_part) {
  extern __shared__ float smem[];
  const int S1 = O + 1;
  float* w1s = smem;                                         // (H + 1) x S1
  float* hs = w1s + (H + 1) * S1;                            // P x H
  float* d2s = hs + P * H;                                   // P x O
  float* ts = d2s + P * O;                                   // P x O
  int* idx = reinterpret_cast<int*>(ts + P * O);             // P x n_active
  __shared__ float red[kT / 64];

  const int tid = threadIdx.x;
  const int p0 = blockIdx.x * P;
  const int np = min(P, rows - p0);

  // round 1 (np * n_active <= kT and np * O <= 2 kT by the path's limits)
  {
    const int ni = np * n_active, nt = np * O, nw1 = (H + 1) * O;
    const int iv = tid < ni ? act[(size_t)p0 * n_active + tid] : 0;       // rows of act are contiguous
    const float t0 = tid < nt ? T[(size_t)p0 * O + tid] : 0.f;            // rows of T are contiguous
    const float t1 = tid + kT < nt ? T[(size_t)p0 * O + tid + kT] : 0.f;
    for (int q0 = 0; q0 < nw1; q0 += 16 * kT) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int q = q0 + u * kT + tid;
        v[u] = q < nw1 ? W1[(size_t)(q / O) * ldw1 + q % O] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int q = q0 + u * kT + tid;
        if (q < nw1) w1s[(q / O) * S1 + q % O] = v[u];
      }
    }
    if (tid < ni) idx[tid] = iv;
    if (tid < nt) ts[tid] = t0;
    if (tid + kT < nt) ts[tid + kT] = t1;
  }
  __syncthreads();
  // round 2: hidden layer, net = bias + sum of the active rows of W0 (in index order)
  for (int j = tid; j < H; j += kT) {
    const float b = W0[(size_t)n0 * ldw0 + j];
    float v[kMaxP][8];
#pragma unroll
    for (int p = 0; p < kMaxP; ++p)
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[p][u] = (p < np && u < n_active) ? W0[(size_t)idx[p * n_active + u] * ldw0 + j] : 0.f;
#pragma unroll
    for (int p = 0; p < kMaxP; ++p) {
      if (p >= np) break;
      float net = b;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (u < n_active) net += v[p][u];
      for (int k = 8; k < n_active; ++k) net += W0[(size_t)idx[p * n_active + k] * ldw0 + j];
      const float h = logistic(net);
      hs[p * H + j] = h;
      A1[(size_t)(p0 + p) * lda1 + j] = h;
    }
  }
  __syncthreads();
  // Output layer, output deltas and squared error.  Each output (p, c) is
  // computed by `lpo` adjacent lanes, lane k summing a contiguous share of
  // the hidden units; the shares are combined by a butterfly, which gives
  // every lane of the group the same (commutative) sum.
  float sse = 0.f;
  {
    const int nout = np * O;
    int lpo = 8;
    while (lpo > 1 && nout * lpo > kT) lpo >>= 1;
    for (int t0 = 0; t0 < nout * lpo; t0 += kT) {
      const int t = t0 + tid;
      const int q = t / lpo, part = t % lpo;
      float z = 0.f;
      if (q < nout) {
        const int p = q / O, c = q % O;
        const float* h = hs + p * H;
        const int j0 = H * part / lpo, j1 = H * (part + 1) / lpo;
        for (int j = j0; j < j1; j += 8) {
          float hv[8], wv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            hv[u] = j + u < j1 ? h[j + u] : 0.f;
            wv[u] = j + u < j1 ? w1s[(j + u) * S1 + c] : 0.f;
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) z += hv[u] * wv[u];
        }
      }
      for (int m = 1; m < lpo; m <<= 1) z += __shfl_xor(z, m, 64);
      if (q < nout && part == 0) {
        const int p = q / O, c = q % O;
        const float y = logistic(w1s[H * S1 + c] + z);
        const float e = ts[q] - y;
        sse += e * e;
        const float d = e * y * (1.0f - y);
        d2s[q] = d;
        D2[(size_t)(p0 + p) * ldd2 + c] = d;
      }
    }
  }
  __syncthreads();
  // hidden deltas (W1 before its update, bias row excluded): one thread per (p, j)
  for (int t = tid; t < np * H; t += kT) {
    const int p = t / H, j = t % H;
    const float* wr = w1s + j * S1;
    const float* d = d2s + p * O;
    float s = 0.f;
    for (int c = 0; c < O; c += 8) {
      float wv[8], dv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        wv[u] = c + u < O ? wr[c + u] : 0.f;
        dv[u] = c + u < O ? d[c + u] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) s += wv[u] * dv[u];
    }
    const float h = hs[p * H + j];
    D1[(size_t)(p0 + p) * lda1 + j] = s * (h * (1.0f - h));
  }
  // block error partial, fixed order
  const int lane = tid & 63, wave = tid >> 6;
  for (int off = 32; off > 0; off >>= 1) sse += __shfl_xor(sse, off, 64);
  if (lane == 0) red[wave] = sse;
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < kT / 64; ++w) s += (double)red[w];
    sse_part[blockIdx.x] = s;
  }
}

// Sum of the kWU wave partials of one lane, in wave order.
__device__ __forceinline__ float combine(const float (*part)[64], int lane) {
  float s = part[0][lane];
  for (int w = 1; w < kWU; ++w) s += part[w][lane];
  return s;
}

// 1024 threads = 16 waves per block.  The weight and momentum a lane updates
// are loaded at the start, overlapping the batch sums.
// Blocks [0, nA): W1 changes, 64 consecutive elements (j, c) per block, the
//   16 waves summing consecutive sixteenths of the batch.
// Blocks [nA, nA + n0): row r of W0: the delta rows of the patterns whose
//   active list contains r, in pattern order (ballot compaction of 1024
//   patterns at a time); wave w owns the column strip (w % 4) and quarter
//   (w / 4) of each compacted list.
// Blocks [nA + n0, nA + n0 + nS): the bias row of W0, 64 columns per block,
//   the 16 waves summing consecutive sixteenths of the batch.
__global__ __launch_bounds__(kTU) void small_update_kernel(const int32_t* __restrict__ act, int n_active, int rows,
                                                           const float* __restrict__ A1, const float* __restrict__ D1,
                                                           int lda1, const float* __restrict__ D2, int ldd2,
                                                           float* W0, float* V0, int ldw0, int n0, int H, float* W1,
                                                           float* V1, int ldw1, int O, int nA, float lr, float mom) {
  __shared__ float part[kWU][64];
  __shared__ int list[kTU];
  __shared__ int wave_cnt[kWU];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const int r0 = (int)((int64_t)rows * wave / kWU), r1 = (int)((int64_t)rows * (wave + 1) / kWU);

  float* Wt;        // weight row this block updates
  float* Vt;
  int col, ncol;    // lane's column in that row, row length
  if (b < nA) {
    const int o = b * 64 + lane;
    const int j = o / O, c = o % O;
    Wt = W1 + (size_t)j * ldw1;
    Vt = V1 + (size_t)j * ldw1;
    col = c;
    ncol = o < (H + 1) * O ? O : 0;
  } else if (b < nA + n0) {
    Wt = W0 + (size_t)(b - nA) * ldw0;
    Vt = V0 + (size_t)(b - nA) * ldw0;
    col = (wave & 3) * 64 + lane;
    ncol = H;
  } else {
    Wt = W0 + (size_t)n0 * ldw0;
    Vt = V0 + (size_t)n0 * ldw0;
    col = (b - nA - n0) * 64 + lane;
    ncol = H;
  }
  const bool owner = (b < nA || b >= nA + n0) ? (wave == 0) : (wave < 4);
  const bool live = col < ncol;
  float w_old = 0.f, v_old = 0.f;
  if (owner && live) {
    w_old = Wt[col];
    v_old = Vt[col];
  }

  float g = 0.f;
  if (b < nA) {
    const int o = b * 64 + lane;
    const int j = o / O, c = o % O;
    if (live) g = (j < H) ? dot_rows(A1 + j, lda1, D2 + c, ldd2, r0, r1) : sum_rows(D2 + c, ldd2, r0, r1);
    part[wave][lane] = g;
    __syncthreads();
    if (owner) g = combine(part, lane);
  } else if (b < nA + n0) {
    const int r = b - nA;
    const int quarter = wave >> 2;
    for (int pc = 0; pc < rows; pc += kTU) {
      const int p = pc + tid;
      bool hit = false;
      if (p < rows) {
        const int32_t* a = act + (size_t)p * n_active;
        for (int k0 = 0; k0 < n_active; k0 += 8) {
          int iv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) iv[u] = k0 + u < n_active ? a[k0 + u] : -1;
#pragma unroll
          for (int u = 0; u < 8; ++u) hit |= (iv[u] == r);
        }
      }
      const unsigned long long bal = __ballot(hit);
      if (lane == 0) wave_cnt[wave] = __popcll(bal);
      __syncthreads();
      int base = 0, total = 0;
      for (int w = 0; w < kWU; ++w) {
        base += (w < wave) ? wave_cnt[w] : 0;
        total += wave_cnt[w];
      }
      if (hit) list[base + __popcll(bal & ((1ull << lane) - 1ull))] = p;
      __syncthreads();
      const int q0 = (int)((int64_t)total * quarter / 4), q1 = (int)((int64_t)total * (quarter + 1) / 4);
      float s = 0.f;
      if (live) {
        for (int q = q0; q < q1; q += 16) {
          float v[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) v[u] = q + u < q1 ? D1[(size_t)list[q + u] * lda1 + col] : 0.f;
#pragma unroll
          for (int u = 0; u < 16; ++u)
            if (q + u < q1) s += v[u];
        }
      }
      // quarters of this chunk are added to the running sum in list order
      part[wave][lane] = s;
      __syncthreads();
      if (owner) g = (((g + part[wave][lane]) + part[wave + 4][lane]) + part[wave + 8][lane]) + part[wave + 12][lane];
      __syncthreads();
    }
  } else {
    if (live) g = sum_rows(D1 + col, lda1, r0, r1);
    part[wave][lane] = g;
    __syncthreads();
    if (owner) g = combine(part, lane);
  }
  if (owner && live) {
    const float v = lr * g + mom * v_old;
    Vt[col] = v;
    Wt[col] = w_old + v;
  }
}

int patterns_per_block(int rows) {
  int p = rows / 256;
  return p < 1 ? 1 : (p > kMaxP ? kMaxP : p);
}

}  // namespace

bool small_path_fits(int n0, int H, int O, int n_active) {
  return H >= 1 && H <= kSmallMaxHidden && O >= 1 && O <= kSmallMaxOut && n0 >= 1 && n_active >= 1 &&
         n_active <= kSmallMaxActive;
}

int small_fwdbwd_blocks(int rows) {
  const int P = patterns_per_block(rows);
  return (rows + P - 1) / P;
}

hipError_t small_fwdbwd(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw0, int n0,
                        int H, const float* W1, int ldw1, int O, const float* T, float* A1, int lda1, float* D1,
                        float* D2, int ldd2, double* sse_part) {
  if (rows <= 0) return hipSuccess;
  const int P = patterns_per_block(rows);
  const size_t lds = sizeof(float) * ((size_t)(H + 1) * (O + 1) + (size_t)P * H + 2 * (size_t)P * O) +
                     sizeof(int) * (size_t)P * n_active;
  return launch_kernel(small_fwdbwd_kernel, small_fwdbwd_blocks(rows), kT, lds, s, act, n_active, rows, P, W0, ldw0, n0, H, W1, ldw1, O,
                                                                 T, A1, lda1, D1, D2, ldd2, sse_part);
}

hipError_t small_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* A1, const float* D1,
                        int lda1, const float* D2, int ldd2, float* W0, float* V0, int ldw0, int n0, int H, float* W1,
                        float* V1, int ldw1, int O, float lr, float mom) {
  if (rows <= 0) return hipSuccess;
  const int nA = ((H + 1) * O + 63) / 64;
  const int nS = (H + 63) / 64;
  return launch_kernel(small_update_kernel, nA + n0 + nS, kTU, 0, s, act, n_active, rows, A1, D1, lda1, D2, ldd2, W0, V0, ldw0, n0, H, W1,
                                                  V1, ldw1, O, nA, lr, mom);
}

}  // namespace bpk
