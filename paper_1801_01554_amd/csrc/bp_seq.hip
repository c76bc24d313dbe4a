// bp_seq.hip -- Elman nets (section 10.5): the context copy between the
// steps of a sequence.
//
// Sequences run in parallel across streams, as the paper parallelises them
// across processors; step t of every stream is one row block of S patterns.
// Before the forward pass of a step, each context unit c (the last n_ctx
// input units) takes the value its source hidden unit had after the
// previous step of the same stream, multiplied by the pattern's continuation
// flag (0 at the start of a sequence).  Everything else of the step reuses
// the feed-forward kernels.
#include <hip/hip_runtime.h>

#include "bp_device.h"
#include "bp_internal.h"

namespace bpk {
namespace {

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kAsmThreads = 256;

// One thread per element of the lda0-wide input rows; threads of a row are
// adjacent, so the stores and the reads of X are coalesced.
__global__ __launch_bounds__(kAsmThreads) void seq_assemble_kernel(const float* __restrict__ X, int n_ext,
                                                                   const float* __restrict__ cont, int S, int n_ctx,
                                                                   const int32_t* __restrict__ ctx_layer,
                                                                   const int32_t* __restrict__ ctx_unit,
                                                                   CtxSource src, float* A0, int lda0) {
  const int64_t i = (int64_t)blockIdx.x * kAsmThreads + threadIdx.x;
  if (i >= (int64_t)S * lda0) return;
  const int s = (int)(i / lda0), j = (int)(i % lda0);
  float v = 0.f;
  if (j < n_ext) {
    v = X[(size_t)s * n_ext + j];
  } else if (j < n_ext + n_ctx) {
    const int c = j - n_ext;
    const int l = ctx_layer[c];
    const float* b = src.base[l];
    const float prev = b ? b[(size_t)s * src.ld[l] + ctx_unit[c]] : 0.f;
    v = cont[s] * prev;
  }
  A0[(size_t)s * lda0 + j] = v;
}

// ---- one window of an Elman net in one launch
//
// A block owns R = 4 RG streams and all their units, so a step needs nothing
// from other blocks.  Products use v_mfma_f32_4x4x1_16b_f32 (16 blocks of a
// 4 x 4 outer product): lane l supplies row l % 4 of the block's A column and
// column l % 4 of block l / 4 of B, and register r of lane l returns row r,
// column l % 4 of block l / 4.  Here every block takes the same 4 rows (the
// streams) and lane l its own weight column, so one instruction adds the
// rank-1 term of one k to a 4 x 64 tile of the product; with C columns per
// lane (C l .. C l + C - 1, one 4-, 8- or 16-byte load per k) a wave covers
// 64 C columns.  The four waves split K into contiguous quarters and add
// their sums in wave order through LDS.
constexpr int kWinThreads = 320;      // 4 compute waves and one memory wave
constexpr int kWinMaxIn = 512;       // n0
constexpr int kWinMaxUnits = 256;    // n1, n2
constexpr int kWinRG = 1;            // row groups of 4 streams per block

template <int C>
__device__ __forceinline__ void load_cols(float* d, const float* p) {
  if constexpr (C == 4) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p);
    d[0] = v[0], d[1] = v[1], d[2] = v[2], d[3] = v[3];
  } else if constexpr (C == 2) {
    const f32x2 v = *reinterpret_cast<const f32x2*>(p);
    d[0] = v[0], d[1] = v[1];
  } else {
    d[0] = *p;
  }
}

// Partial products of the block's rows As (LDS, row stride as, zero from K
// to the end of the last wave's range) with B (K x N, row stride ldb >= N,
// a multiple of C, 4 C-aligned): wave w takes k in [w kc, w kc + kc), and
// its sums go to P[w][row][col] (row stride 64 C).  B rows stream through a
// ring of D groups of 4 k: D - 1 groups are in flight while one is
// multiplied, and the first D - 1 are loaded by prefetch(), which a caller
// issues ahead of the product.  Rows past K and columns past ldb - C are
// clamped to valid addresses (their A is zero or their columns unused).
template <int RG, int C, int D>
struct WinProduct {
  float ring[D][4][C];
  const float* bl;
  int k0, nit, K, ldb;

  __device__ __forceinline__ void init(const float* __restrict__ B, int ldb_, int K_, int wave, int lane) {
    K = K_;
    ldb = ldb_;
    const int kc = ((K + 15) >> 4) << 2;
    // the wave's range is uniform across its lanes: row addresses stay scalar
    k0 = __builtin_amdgcn_readfirstlane(wave * kc);
    nit = K > k0 ? (min(kc, K - k0) + 3) >> 2 : 0;
    bl = B + min(C * lane, ldb - C);
  }
  __device__ __forceinline__ void load(int slot, int it) {
    const int kb = k0 + 4 * it;
#pragma unroll
    for (int j = 0; j < 4; ++j) load_cols<C>(ring[slot][j], bl + (size_t)min(kb + j, K - 1) * ldb);
  }
  __device__ __forceinline__ void prefetch() {
#pragma unroll
    for (int d = 0; d < D - 1; ++d) load(d, d);
  }
  // NA = 4 / C accumulator sets (k mod NA) give 4 RG independent chains.
  static constexpr int NA = 4 / C;
  __device__ __forceinline__ void mul(f32x4 (&acc)[NA][RG][C], const float* As, int as, int slot, int it,
                                      int lane) {
    const int kb = k0 + 4 * it;
    f32x4 a[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) a[g] = *reinterpret_cast<const f32x4*>(As + (4 * g + (lane & 3)) * as + kb);
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int g = 0; g < RG; ++g)
          acc[j % NA][g][c] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[g][j], ring[slot][j][c], acc[j % NA][g][c], 0, 0, 0);
  }
  // After prefetch(): the product, and the partial sums to P.  Whole trips of
  // D groups run without branches (a branch between a load and its use
  // makes the compiler wait for every load in flight); the last nit % D
  // groups were already loaded and run after.
  __device__ __forceinline__ void run(const float* As, int as, float* P, int wave, int lane) {
    constexpr int R = 4 * RG;
    f32x4 acc[NA][RG][C];
#pragma unroll
    for (int h = 0; h < NA; ++h)
#pragma unroll
      for (int g = 0; g < RG; ++g)
#pragma unroll
        for (int c = 0; c < C; ++c) acc[h][g][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int full = nit / D;
    for (int t = 0; t < full; ++t) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        load((u + D - 1) % D, t * D + u + D - 1);
        mul(acc, As, as, u, t * D + u, lane);
      }
    }
#pragma unroll
    for (int u = 0; u < D - 1; ++u)
      if (full * D + u < nit) mul(acc, As, as, u, full * D + u, lane);
#pragma unroll
    for (int g = 0; g < RG; ++g)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float* q = P + (wave * R + 4 * g + r) * (64 * C) + C * lane;
#pragma unroll
        for (int c = 0; c < C; ++c) {
          float v = acc[0][g][c][r];
#pragma unroll
          for (int h = 1; h < NA; ++h) v += acc[h][g][c][r];
          q[c] = v;
        }
      }
  }
};

// The same product with B held in LDS (K x 64 columns, row stride 64, zero
// rows from K to the end of the last wave's range): one column per lane.
template <int RG>
struct WinProductLds {
  int k0, nit;
  __device__ __forceinline__ void init(int K, int wave) {
    const int kc = ((K + 15) >> 4) << 2;
    k0 = __builtin_amdgcn_readfirstlane(wave * kc);
    nit = K > k0 ? (min(kc, K - k0) + 3) >> 2 : 0;
  }
  __device__ __forceinline__ void run(const float* As, int as, const float* Bs, float* P, int wave, int lane) {
    constexpr int R = 4 * RG;
    f32x4 acc[4][RG];   // four chains: k mod 4
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int g = 0; g < RG; ++g) acc[h][g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int it = 0; it < nit; ++it) {
      const int kb = k0 + 4 * it;
      f32x4 a[RG];
      float b[4];
#pragma unroll
      for (int g = 0; g < RG; ++g) a[g] = *reinterpret_cast<const f32x4*>(As + (4 * g + (lane & 3)) * as + kb);
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[(kb + j) * 64 + lane];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int g = 0; g < RG; ++g) acc[j][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[g][j], b[j], acc[j][g], 0, 0, 0);
    }
#pragma unroll
    for (int g = 0; g < RG; ++g)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        P[(wave * R + 4 * g + r) * 64 + lane] = ((acc[0][g][r] + acc[1][g][r]) + acc[2][g][r]) + acc[3][g][r];
  }
};

template <int C>
constexpr int win_depth() { return C == 1 ? 8 : (C == 2 ? 6 : 4); }

// Waves 0-3 compute; wave 4 moves data between LDS and global memory (the
// input, target and flag rows in; the input rows, hidden units, deltas,
// column sums and error partials out).  A wave waits for its memory
// operations in issue order, so a compute wave that stored results would
// stall on those stores at its next weight load; the weight loads are the
// only global accesses of waves 0-3.  Elementwise work maps compute thread t
// to column t of all R rows: no division by a row length, and a thread's
// deltas give their column sum without exchange.
//
// Per step k, between the block's four barriers:
//   1. compute: hidden product.   wave 4: load X and flags of step k + 1,
//      targets and mask of step k.
//   2. compute: hidden units.     wave 4: store input rows k.
//   3. compute: output product, then input rows k + 1 (X, flag x hidden k).
//      wave 4: store hidden units k, deltas etc. of step k - 1.
//   4. compute: output units, deltas, column sums, error partials.
constexpr int kWinComputeThreads = 256;

template <int RG, int C1, int C2>
__global__ __launch_bounds__(kWinThreads) void elman_window_kernel(ElmanWindow p) {
  constexpr int R = 4 * RG;
  constexpr int AS = kWinMaxIn + 4, HS = kWinMaxUnits + 4;   // row strides: 4 rows 4 banks apart
  constexpr int US = kWinMaxUnits;
  __shared__ __attribute__((aligned(16))) float Arow[R * AS];   // input rows of the step
  __shared__ __attribute__((aligned(16))) float Hrow[R * HS];   // hidden units of the step
  __shared__ __attribute__((aligned(16))) float P[4 * R * US];  // per-wave partial products
  __shared__ __attribute__((aligned(16))) float Xl[R * US];     // external inputs of the next step
  __shared__ __attribute__((aligned(16))) float Tl[R * US];     // targets of the step
  __shared__ __attribute__((aligned(16))) float Dl[R * US];     // deltas of the step
  __shared__ float csl[US], ssl[US];                             // their column sums, error sums
  __shared__ float contN[R], maskC[R];                           // flags (next step, this step)
  // output weights, when one column per lane covers them (n2 <= 64)
  __shared__ __attribute__((aligned(16))) float W1s[C2 == 1 ? (kWinMaxUnits + 4) * 64 : 4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const bool io = tid >= kWinComputeThreads;
  const int S = p.S, n_ext = p.n_ext, n0 = p.n0, n1 = p.n1, n2 = p.n2, n_ctx = n0 - n_ext;
  const int m0 = blockIdx.x * R;
  const int rows_in = min(R, S - m0);   // rows of real streams in this block
  const int steps = p.steps;

  // wave 4: external inputs and continuation flags of step k into Xl, contN
  // (all loads issued before the first LDS write)
  auto io_load_x = [&](int k) {
    float xr[R][kWinMaxUnits / 64], cr[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const size_t row = (size_t)k * S + m0 + i;
#pragma unroll
      for (int q = 0; q < kWinMaxUnits / 64; ++q) {
        const int c = lane + 64 * q;
        xr[i][q] = (c < n_ext && i < rows_in) ? p.X[row * n_ext + c] : 0.f;
      }
      cr[i] = i < rows_in ? p.cont[row] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
#pragma unroll
      for (int q = 0; q < kWinMaxUnits / 64; ++q)
        if (lane + 64 * q < n_ext) Xl[i * US + lane + 64 * q] = xr[i][q];
      if (lane == 0) contN[i] = cr[i];
    }
  };
  // wave 4: targets and mask of step k into Tl, maskC
  auto io_load_t = [&](int k) {
    const size_t row0 = (size_t)k * S + m0;
    float tr[R][kWinMaxUnits / 64], mr[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
#pragma unroll
      for (int q = 0; q < kWinMaxUnits / 64; ++q) {
        const int c = lane + 64 * q;
        tr[i][q] = (c < n2 && i < rows_in) ? p.T[(row0 + i) * p.ldt + c] : 0.f;
      }
      mr[i] = (p.mask && i < rows_in) ? p.mask[row0 + i] : 1.f;
    }
#pragma unroll
    for (int i = 0; i < R; ++i) {
#pragma unroll
      for (int q = 0; q < kWinMaxUnits / 64; ++q)
        if (lane + 64 * q < n2) Tl[i * US + lane + 64 * q] = tr[i][q];
      if (lane == 0) maskC[i] = mr[i];
    }
  };
  // wave 4: deltas and error partial of step k from LDS; the column sums
  // added over the window's steps in step order
  float cacc[kWinMaxUnits / 64] = {};
  auto io_store_d = [&](int k) {
    const size_t row0 = (size_t)k * S + m0;
    for (int i = 0; i < rows_in; ++i)
      for (int c = 4 * lane; c < n2; c += 256)
        *reinterpret_cast<f32x4*>(p.D + (row0 + i) * p.ldd + c) = *reinterpret_cast<const f32x4*>(Dl + i * US + c);
    const size_t crow = (size_t)k * gridDim.x + blockIdx.x;
#pragma unroll
    for (int q = 0; q < kWinMaxUnits / 64; ++q)
      if (lane + 64 * q < n2) cacc[q] += csl[lane + 64 * q];
    // error partial: the compute threads' sums added in thread order
    double e = 0.0;
    for (int c = lane; c < n2; c += 64) e += (double)ssl[c];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) e += __shfl_down(e, o);
    if (lane == 0) p.sse[crow] = e;
  };

  // Zero rows past the units (read by the products' last k groups); the
  // context source of step 0; the first step's inputs.
  for (int e = tid; e < R * AS; e += kWinThreads) Arow[e] = 0.f;
  for (int e = tid; e < R * US; e += kWinThreads) Dl[e] = 0.f;
  // (loads of a thread issued together, then written)
  if constexpr (C2 == 1) {
    constexpr int Q = ((kWinMaxUnits + 4) * 16 + kWinThreads - 1) / kWinThreads;
    f32x4 v[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int e4 = tid + q * kWinThreads, kk = e4 >> 4, c = (e4 & 15) * 4;
      v[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (kk < n1 && c < n2) v[q] = *reinterpret_cast<const f32x4*>(p.W1 + (size_t)kk * p.ldw1 + c);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int e4 = tid + q * kWinThreads, c = (e4 & 15) * 4;
      if (e4 < (n1 + 4) * 16) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (c + j >= n2) v[q][j] = 0.f;
        *reinterpret_cast<f32x4*>(W1s + 4 * e4) = v[q];
      }
    }
  }
  {
    constexpr int Q = (R * HS + kWinThreads - 1) / kWinThreads;
    float v[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int e = tid + q * kWinThreads, i = e / HS, c = e - i * HS;
      v[q] = (e < R * HS && p.Hprev && c < n_ctx && i < rows_in) ? p.Hprev[(size_t)(m0 + i) * p.ldhp + c] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < Q; ++q)
      if (tid + q * kWinThreads < R * HS) Hrow[tid + q * kWinThreads] = v[q];
  }
  if (io) io_load_x(0);
  __syncthreads();

  WinProduct<RG, C1, win_depth<C1>()> ph;
  WinProduct<RG, C2, win_depth<C2>()> po;
  WinProductLds<RG> pol;
  ph.init(p.W0, p.ldw0, n0, wave, lane);
  if constexpr (C2 == 1) pol.init(n1, wave);
  else po.init(p.W1, p.ldw1, n1, wave, lane);
  const float bh = tid < n1 ? p.b0[tid] : 0.f;   // biases of this thread's columns
  const float bo = tid < n2 ? p.b1[tid] : 0.f;
  // input rows of the step: external inputs, then flag x context (zero past the streams)
  auto build_rows = [&]() {
    if (tid < n_ext) {
#pragma unroll
      for (int i = 0; i < R; ++i) Arow[i * AS + tid] = Xl[i * US + tid];
    }
    if (tid < n_ctx) {
#pragma unroll
      for (int i = 0; i < R; ++i) Arow[i * AS + n_ext + tid] = i < rows_in ? contN[i] * Hrow[i * HS + tid] : 0.f;
    }
  };
  if (!io) {
    build_rows();
    ph.prefetch();
  }
  __syncthreads();

  for (int k = 0; k < steps; ++k) {
    const size_t row0 = (size_t)k * S + m0;   // first row of the block at this step
    // 1. hidden product | loads for steps k + 1 and k (loads only: their wait
    //    does not include stores issued after them)
    if (!io) {
      ph.run(Arow, AS, P, wave, lane);
      if constexpr (C2 != 1) po.prefetch();
    } else {
      if (k + 1 < steps) io_load_x(k + 1);
      io_load_t(k);
    }
    __syncthreads();
    // 2. hidden units | store of input rows k
    if (io) {
      for (int i = 0; i < rows_in; ++i)
        for (int c = 4 * lane; c < n0; c += 256)
          *reinterpret_cast<f32x4*>(p.rows + (row0 + i) * p.ldr + c) = *reinterpret_cast<const f32x4*>(Arow + i * AS + c);
    }
    if (tid < n1) {
#pragma unroll
      for (int i = 0; i < R; ++i) {
        float z = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) z += P[(w * R + i) * (64 * C1) + tid];
        Hrow[i * HS + tid] = unit_sigma(z + bh, p.tab);
      }
    }
    __syncthreads();
    // 3. output product, next input rows | stores of hidden units k and of
    //    the deltas etc. of step k - 1
    if (!io) {
      if constexpr (C2 == 1) pol.run(Hrow, HS, W1s, P, wave, lane);
      else po.run(Hrow, HS, P, wave, lane);
      if (k + 1 < steps) {
        build_rows();
        ph.prefetch();
      }
    } else {
      for (int i = 0; i < rows_in; ++i)
        for (int c = 4 * lane; c < n1; c += 256)
          *reinterpret_cast<f32x4*>(p.H + (row0 + i) * p.ldh + c) = *reinterpret_cast<const f32x4*>(Hrow + i * HS + c);
      if (k > 0) io_store_d(k - 1);
    }
    __syncthreads();
    // 4. output units, deltas (zero past the streams), column sums in row order, error
    float sse = 0.f;
    if (tid < n2) {
      float cs = 0.f;
#pragma unroll
      for (int i = 0; i < R; ++i) {
        float d = 0.f;
        if (i < rows_in) {
          float z = 0.f;
#pragma unroll
          for (int w = 0; w < 4; ++w) z += P[(w * R + i) * (64 * C2) + tid];
          const float y = unit_sigma(z + bo, p.tab);
          const float err = (Tl[i * US + tid] - y) * maskC[i];
          sse += err * err;
          d = err * y * (1.0f - y);
        }
        Dl[i * US + tid] = d;
        cs += d;
      }
      csl[tid] = cs;
      ssl[tid] = sse;
    }
    __syncthreads();
  }
  if (io) {
    io_store_d(steps - 1);
#pragma unroll
    for (int q = 0; q < kWinMaxUnits / 64; ++q)
      if (lane + 64 * q < n2) p.colsum[(size_t)blockIdx.x * p.ldcs + lane + 64 * q] = cacc[q];
  }
}

template <int RG, int C1>
hipError_t launch_window_c2(hipStream_t s, const ElmanWindow& w, int C2) {
  const unsigned blocks = (unsigned)elman_window_blocks(w.S);
  if (C2 == 1) return launch_kernel(elman_window_kernel<RG, C1, 1>, blocks, kWinThreads, 0, s, w);
  if (C2 == 2) return launch_kernel(elman_window_kernel<RG, C1, 2>, blocks, kWinThreads, 0, s, w);
  return launch_kernel(elman_window_kernel<RG, C1, 4>, blocks, kWinThreads, 0, s, w);
}

int cols_per_lane(int n) { return n <= 64 ? 1 : (n <= 128 ? 2 : 4); }

}  // namespace

bool elman_window_fits(int S, int n_ext, int n0, int n1, int n2) {
  return S > 0 && n_ext >= 0 && n_ext <= 256 && n_ext <= n0 && n0 - n_ext <= n1 && n0 >= 1 &&
         n0 <= kWinMaxIn && n1 >= 1 && n1 <= kWinMaxUnits && n2 >= 1 && n2 <= kWinMaxUnits;
}

int elman_window_blocks(int S) { return (S + 4 * kWinRG - 1) / (4 * kWinRG); }

hipError_t elman_window(hipStream_t s, const ElmanWindow& w) {
  if (!elman_window_fits(w.S, w.n_ext, w.n0, w.n1, w.n2) || w.steps < 1 || (w.n_ext > 0 && !w.X) || !w.cont ||
      !w.T || !w.W0 || !w.b0 || !w.W1 || !w.b1 || !w.H || !w.rows || !w.D || !w.colsum || !w.sse)
    return hipErrorInvalidValue;
  const int C1 = cols_per_lane(w.n1), C2 = cols_per_lane(w.n2);
  // 16-byte aligned rows: weights wide enough for the column loads, outputs
  // for 16-byte stores up to the next multiple of 4 columns
  auto rows16 = [](const void* q, int ld, int n) {
    return (reinterpret_cast<uintptr_t>(q) & 15) == 0 && (ld & 3) == 0 && ld >= ((n + 3) & ~3);
  };
  if (!rows16(w.W0, w.ldw0, w.n1) || !rows16(w.W1, w.ldw1, w.n2) || !rows16(w.rows, w.ldr, w.n0) ||
      !rows16(w.H, w.ldh, w.n1) || !rows16(w.D, w.ldd, w.n2) || w.ldt < w.n2 || w.ldcs < w.n2 ||
      (w.Hprev && w.ldhp < w.n0 - w.n_ext))
    return hipErrorInvalidValue;
  if (C1 == 1) return launch_window_c2<kWinRG, 1>(s, w, C2);
  if (C1 == 2) return launch_window_c2<kWinRG, 2>(s, w, C2);
  return launch_window_c2<kWinRG, 4>(s, w, C2);
}

hipError_t seq_assemble(hipStream_t s, const float* X, int n_ext, const float* cont, int S, int n_ctx,
                        const int32_t* ctx_layer, const int32_t* ctx_unit, const CtxSource& src, float* A0,
                        int lda0) {
  const int64_t total = (int64_t)S * lda0;
  if (total <= 0) return hipSuccess;
  return launch_kernel(seq_assemble_kernel, (unsigned)((total + kAsmThreads - 1) / kAsmThreads), kAsmThreads, 0, s,
                       X, n_ext, cont, S, n_ctx, ctx_layer, ctx_unit, src, A0, lda0);
}

}  // namespace bpk
