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

#include "bp_device.h"
#include "bp_internal.h"

namespace bpk {
namespace {

constexpr int kT = 1024;       // threads per forward/backward block (16 waves)
constexpr int kTU = 1024;      // threads per update block (16 waves)
constexpr int kWU = kTU / 64;
constexpr int kMaxP = 8;       // patterns per forward/backward block
constexpr int kStageFloats = 32768;   // LDS floats the update blocks stage batch chunks in

typedef float f32x4 __attribute__((ext_vector_type(4)));

// q / d and q % d for 0 <= q < 2^16 and 1 <= d <= 2^10, through a float
// reciprocal: the float quotient is within 2^-8 / d of the true one, far from
// the next integer, so the truncation is exact.
__device__ __forceinline__ void divmod(int q, int d, float inv_d, int& quo, int& rem) {
  quo = (int)(((float)q + 0.5f) * inv_d);
  rem = q - quo * d;
}

// Dynamic LDS of small_fwdbwd: W1 as (H + 1) x (O + 1) (odd row stride so
// that column walks by consecutive hidden units hit distinct banks), the
// hidden activations [P][H], the output deltas [P][O], the targets [P][O]
// and the active indices [P][n_active] of the block's patterns.
//
// 1024 threads (16 waves, four per SIMD) per block of P patterns: every
// phase is spread over all of them, so each lane's chain of dependent LDS
// reads is short and the waves of a SIMD hide each other's latencies.
//   round 1   indices, targets and W1: independent loads, all in flight;
//   gather    one (pattern, hidden unit) pair per thread: bias + the active
//             rows of W0, in index order -> sigma;
//   output    each output (p, c) summed by 2^lg adjacent lanes, lane k over
//             the hidden units k, k + 2^lg, ..., combined by a butterfly;
//   deltas    each hidden delta (p, j) summed by 2^lq adjacent lanes, lane k
//             over the outputs k, k + 2^lq, ..., combined by a butterfly.
// The strided shares walk LDS by pointer increments, with no clamped or
// guarded reads in the inner loops.
// P (patterns per block) and TAB (table sigmoid) are template parameters so
// that each instantiation holds only the code it runs: these kernels are
// short enough that instruction-cache misses at launch are a visible part of
// their time.
template <int P, bool TAB>
__global__ __launch_bounds__(kT) void small_fwdbwd_kernel(const int32_t* __restrict__ act, int n_active, int rows,
                                                          const float* __restrict__ W0, int ldw0, int n0,
                                                          int H, const float* __restrict__ W1, int ldw1, int O,
                                                          const float* __restrict__ T, float* A1, int lda1,
                                                          float* D1, float* D2, int ldd2, double* sse_part,
                                                          const float* __restrict__ tab) {
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
  const float inv_O = 1.0f / (float)O, inv_H = 1.0f / (float)H;

  // round 1 (np * n_active <= 256 and np * O <= 512 <= kT by the path's
  // limits).  Every load reads a clamped, valid address and the predicate
  // only selects the value: no load sits behind a branch, so all are in
  // flight together.  (Rows of act and of T are contiguous.)
  {
    const int ni = np * n_active, nt = np * O;
    const int iv = act[(size_t)p0 * n_active + min(tid, ni - 1)];
    const float t0 = T[(size_t)p0 * O + min(tid, nt - 1)];
    // W1: lane column c = tid % cw, rows tid / cw + k (kT / cw)
    const int cw = O <= 32 ? 32 : 64, rpp = kT / cw;
    const int c = tid & (cw - 1), jt = tid / cw;
    for (int k0 = 0; k0 * rpp <= H; k0 += 4) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = jt + (k0 + u) * rpp;
        v[u] = W1[(size_t)min(j, H) * ldw1 + min(c, O - 1)];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = jt + (k0 + u) * rpp;
        if (c < O && j <= H) w1s[j * S1 + c] = v[u];
      }
    }
    if (tid < ni) idx[tid] = iv;
    if (tid < nt) ts[tid] = t0;
  }
  __syncthreads();
  // gather: net = bias + the active rows of W0 (in index order)
  for (int t = tid; t < np * H; t += kT) {
    int p = 0, j = 0;
    divmod(t, H, inv_H, p, j);
    const int* ip = idx + p * n_active;
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = W0[(size_t)ip[min(u, n_active - 1)] * ldw0 + j];
    float net = W0[(size_t)n0 * ldw0 + j];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (u < n_active) net += v[u];
    for (int k = 8; k < n_active; ++k) net += W0[(size_t)ip[k] * ldw0 + j];
    const float h = TAB ? logistic_table(net, tab) : logistic(net);
    hs[t] = h;
    A1[(size_t)(p0 + p) * lda1 + j] = h;
  }
  __syncthreads();
  // Output layer, output deltas and squared error.  Each output (p, c) is
  // computed by `lpo` adjacent lanes; the lanes' partial sums are combined by
  // a butterfly, which gives every lane of the group the same (commutative)
  // sum.
  float sse = 0.f;
  {
    const int nout = np * O;
    int lg = 4;
    while (lg > 0 && (nout << lg) > kT) --lg;
    const int lpo = 1 << lg;
    for (int t0 = 0; t0 < (nout << lg); t0 += kT) {
      const int t = t0 + tid;
      const int q = t >> lg, part = t & (lpo - 1);
      int p = 0, c = 0;
      divmod(q, O, inv_O, p, c);
      float z = 0.f;
      if (q < nout) {
        const float* hp = hs + p * H + part;           // units part, part + lpo, ...
        const float* wp = w1s + part * S1 + c;
        const int n = (H - part + lpo - 1) >> lg;       // units of this lane
        const int ws = lpo * S1;
        float z1 = 0.f;
        int k = 0;
        for (; k + 4 <= n; k += 4) {
          const float h0 = hp[0], h1 = hp[lpo], h2 = hp[2 * lpo], h3 = hp[3 * lpo];
          const float w0 = wp[0], w1 = wp[ws], w2 = wp[2 * ws], w3 = wp[3 * ws];
          z += h0 * w0;
          z1 += h1 * w1;
          z += h2 * w2;
          z1 += h3 * w3;
          hp += 4 * lpo;
          wp += 4 * ws;
        }
        for (; k < n; ++k) {
          z += hp[0] * wp[0];
          hp += lpo;
          wp += ws;
        }
        z += z1;
      }
      for (int m = 1; m < lpo; m <<= 1) z += __shfl_xor(z, m, 64);
      if (q < nout && part == 0) {
        const float zo = w1s[H * S1 + c] + z;
        const float y = TAB ? logistic_table(zo, tab) : logistic(zo);
        const float e = ts[q] - y;
        sse += e * e;
        const float d = e * y * (1.0f - y);
        d2s[q] = d;
        D2[(size_t)(p0 + p) * ldd2 + c] = d;
      }
    }
  }
  __syncthreads();
  // hidden deltas (W1 before its update, bias row excluded): each (p, j) by
  // `lpd` adjacent lanes, each summing a contiguous share of the outputs
  {
    const int nh = np * H;
    int lq = 3;
    while (lq > 0 && (nh << lq) > kT) --lq;
    const int lpd = 1 << lq;
    for (int t0 = 0; t0 < (nh << lq); t0 += kT) {
      const int t = t0 + tid;
      const int q = t >> lq, part = t & (lpd - 1);
      int p = 0, j = 0;
      divmod(q, H, inv_H, p, j);
      float sd = 0.f;
      if (q < nh) {
        const float* wp = w1s + j * S1 + part;         // outputs part, part + lpd, ...
        const float* dp = d2s + p * O + part;
        const int n = (O - part + lpd - 1) >> lq;
        float s1 = 0.f;
        int k = 0;
        for (; k + 4 <= n; k += 4) {
          const float w0 = wp[0], w1 = wp[lpd], w2 = wp[2 * lpd], w3 = wp[3 * lpd];
          const float d0 = dp[0], d1 = dp[lpd], d2 = dp[2 * lpd], d3 = dp[3 * lpd];
          sd += w0 * d0;
          s1 += w1 * d1;
          sd += w2 * d2;
          s1 += w3 * d3;
          wp += 4 * lpd;
          dp += 4 * lpd;
        }
        for (; k < n; ++k) {
          sd += wp[0] * dp[0];
          wp += lpd;
          dp += lpd;
        }
        sd += s1;
      }
      for (int m = 1; m < lpd; m <<= 1) sd += __shfl_xor(sd, m, 64);
      if (q < nh && part == 0) {
        const float h = hs[q];
        D1[(size_t)(p0 + p) * lda1 + j] = sd * (h * (1.0f - h));
      }
    }
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

// 1024 threads = 16 waves per block.  The weight and momentum a lane updates
// are loaded at the start, overlapping the sums.  Batch sums over patterns
// run in chunks of `ch` patterns staged in LDS with wide coalesced loads; wave
// w adds its sixteenth of each chunk in pattern order, and the 16 wave
// partials are combined in wave order.
// Blocks [0, nA): W1 elements o = 64 b + lane (row o / O, column o % O):
//   sum_p A1[p][j] D2[p][c] (the bias row H takes 1 for A1).
// Blocks [nA, nA + n0): row r of W0: the delta rows of the patterns whose
//   active list holds r, in pattern order (ballot compaction of 1024
//   patterns at a time); wave w owns the column strip (w % 4) and quarter
//   (w / 4) of each compacted list.
// Blocks [nA + n0, nA + n0 + nS): the bias row of W0, 64 columns per block:
//   sum_p D1[p][j].
// CHECK: the range check of the summed changes (limit > 0).
template <bool CHECK>
__global__ __launch_bounds__(kTU) void small_update_kernel(const int32_t* __restrict__ act, int n_active, int rows,
                                                           const float* __restrict__ A1, const float* __restrict__ D1,
                                                           int lda1, const float* __restrict__ D2, int ldd2,
                                                           float* W0, float* V0, int ldw0, int n0, int H, float* W1,
                                                           float* V1, int ldw1, int O, int nA, int ch, float lr,
                                                           float mom, float limit, unsigned long long* faults) {
  extern __shared__ float stage[];
  __shared__ float part[kWU][64];
  __shared__ int list[kTU];
  __shared__ int wave_cnt[kWU];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;

  float* Wt;        // weight row this block updates
  float* Vt;
  int col, ncol;    // lane's column in that row, row length
  int jrow = 0;     // W1 blocks: the lane's row
  if (b < nA) {
    const int o = b * 64 + lane;
    divmod(o, O, 1.0f / (float)O, jrow, col);
    Wt = W1 + (size_t)jrow * ldw1;
    Vt = V1 + (size_t)jrow * ldw1;
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
    // rows jlo .. jhi of W1 are touched by this block
    const int jlo = (b * 64) / O, jhi = min(H, (b * 64 + 63) / O), nj = jhi - jlo + 1;
    const float inv_nj = 1.0f / (float)nj;
    const int q4 = ldd2 >> 2;                       // float4 per D2 row (ldd2 % 4 == 0)
    float* d2s = stage;                             // [ch][ldd2]
    float* a1s = stage + ch * ldd2;                 // [ch][nj]
    for (int pc = 0; pc < rows; pc += ch) {
      const int cn = min(ch, rows - pc);
      const f32x4* src = reinterpret_cast<const f32x4*>(D2 + (size_t)pc * ldd2);
      // the chunk's delta rows and activation columns are loaded in one round
      const int nd = cn * q4, na = cn * nj;
      for (int i0 = tid; i0 < max(nd, na); i0 += 4 * kTU) {
        f32x4 v[4];
        float av[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = src[min(i0 + u * kTU, nd - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = min(i0 + u * kTU, na - 1);
          int p = 0, jj = 0;
          divmod(i, nj, inv_nj, p, jj);
          const float a = A1[(size_t)(pc + p) * lda1 + min(jlo + jj, H - 1)];
          av[u] = jlo + jj < H ? a : 1.f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (i0 + u * kTU < nd) reinterpret_cast<f32x4*>(d2s)[i0 + u * kTU] = v[u];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (i0 + u * kTU < na) a1s[i0 + u * kTU] = av[u];
      }
      __syncthreads();
      const int s0 = cn * wave / kWU, s1 = cn * (wave + 1) / kWU;
      if (live) {
        const int jj = jrow - jlo;
        for (int p = s0; p < s1; p += 8) {
          float av[8], dv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int pp = min(p + u, s1 - 1);
            av[u] = a1s[pp * nj + jj];
            dv[u] = d2s[pp * ldd2 + col];
          }
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (p + u < s1) g += av[u] * dv[u];
        }
      }
      __syncthreads();
    }
    part[wave][lane] = g;
    __syncthreads();
    if (owner) {
      g = part[0][lane];
      for (int w = 1; w < kWU; ++w) g += part[w][lane];
    }
  } else if (b < nA + n0) {
    const int r = b - nA;
    const int quarter = wave >> 2;
    for (int pc = 0; pc < rows; pc += kTU) {
      const int p = pc + tid;
      bool hit = false;
      if (p < rows) {
        const int32_t* a = act + (size_t)p * n_active;
        for (int q0 = 0; q0 < n_active; q0 += 8) {
          int iv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) iv[u] = a[min(q0 + u, n_active - 1)];
#pragma unroll
          for (int u = 0; u < 8; ++u) iv[u] = q0 + u < n_active ? iv[u] : -1;
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
          for (int u = 0; u < 16; ++u) v[u] = D1[(size_t)list[min(q + u, q1 - 1)] * lda1 + col];
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
    // bias row of W0: columns c0 .. c0 + 63 of D1, staged as float4 (a D1
    // row is lda1 floats, lda1 % 4 == 0; lanes past H are never summed)
    const int c0 = (b - nA - n0) * 64;
    float* d1s = stage;                             // [ch][64]
    for (int pc = 0; pc < rows; pc += ch) {
      const int cn = min(ch, rows - pc);
      for (int i0 = tid; i0 < cn * 16; i0 += 8 * kTU) {
        f32x4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = min(i0 + u * kTU, cn * 16 - 1);
          const int cc = min(c0 + (i & 15) * 4, lda1 - 4);
          v[u] = *reinterpret_cast<const f32x4*>(D1 + (size_t)(pc + (i >> 4)) * lda1 + cc);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (i0 + u * kTU < cn * 16) reinterpret_cast<f32x4*>(d1s)[i0 + u * kTU] = v[u];
      }
      __syncthreads();
      const int s0 = cn * wave / kWU, s1 = cn * (wave + 1) / kWU;
      if (live) {
        for (int p = s0; p < s1; p += 8) {
          float dv[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) dv[u] = d1s[min(p + u, s1 - 1) * 64 + lane];
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (p + u < s1) g += dv[u];
        }
      }
      __syncthreads();
    }
    part[wave][lane] = g;
    __syncthreads();
    if (owner) {
      g = part[0][lane];
      for (int w = 1; w < kWU; ++w) g += part[w][lane];
    }
  }
  if (owner) {   // whole waves
    int nf = 0;
    if (live) {
      if (CHECK) g = checked_change(g, limit, nf);
      const float v = lr * g + mom * v_old;
      Vt[col] = v;
      Wt[col] = w_old + v;
    }
    if (CHECK) add_faults(nf, faults);
  }
}

// Patterns per forward/backward block: a power of two, about rows / 256.
int patterns_per_block(int rows) {
  int p = 1;
  while (p < kMaxP && 2 * p * 256 <= rows) p *= 2;
  return p;
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

template <bool TAB>
hipError_t launch_fwdbwd(hipStream_t s, int P, int nb, size_t lds, const int32_t* act, int n_active, int rows,
                         const float* W0, int ldw0, int n0, int H, const float* W1, int ldw1, int O, const float* T,
                         float* A1, int lda1, float* D1, float* D2, int ldd2, double* sse_part, const float* tab) {
  switch (P) {
    case 1: return launch_kernel(small_fwdbwd_kernel<1, TAB>, nb, kT, lds, s, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1, lda1, D1, D2, ldd2, sse_part, tab);
    case 2: return launch_kernel(small_fwdbwd_kernel<2, TAB>, nb, kT, lds, s, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1, lda1, D1, D2, ldd2, sse_part, tab);
    case 4: return launch_kernel(small_fwdbwd_kernel<4, TAB>, nb, kT, lds, s, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1, lda1, D1, D2, ldd2, sse_part, tab);
    default: return launch_kernel(small_fwdbwd_kernel<8, TAB>, nb, kT, lds, s, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1, lda1, D1, D2, ldd2, sse_part, tab);
  }
}

hipError_t small_fwdbwd(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw0, int n0,
                        int H, const float* W1, int ldw1, int O, const float* T, float* A1, int lda1, float* D1,
                        float* D2, int ldd2, double* sse_part, const float* tab) {
  if (rows <= 0) return hipSuccess;
  const int P = patterns_per_block(rows);
  const size_t lds = sizeof(float) * ((size_t)(H + 1) * (O + 1) + (size_t)P * H + 2 * (size_t)P * O) +
                     sizeof(int) * (size_t)P * n_active;
  const int nb = small_fwdbwd_blocks(rows);
  if (tab)
    return launch_fwdbwd<true>(s, P, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1, lda1, D1, D2,
                               ldd2, sse_part, tab);
  return launch_fwdbwd<false>(s, P, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1, lda1, D1, D2,
                              ldd2, sse_part, tab);
}

hipError_t small_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* A1, const float* D1,
                        int lda1, const float* D2, int ldd2, float* W0, float* V0, int ldw0, int n0, int H, float* W1,
                        float* V1, int ldw1, int O, float lr, float mom, float limit, unsigned long long* faults) {
  if (rows <= 0) return hipSuccess;
  const int nA = ((H + 1) * O + 63) / 64;
  const int nS = (H + 63) / 64;
  // patterns staged per round: the largest power of two that fits
  // kStageFloats for both block types (>= 128 since ldd2 + njmax <= 134)
  const int njmax = 64 / O + 2;
  const int per = (ldd2 + njmax) > 64 ? (ldd2 + njmax) : 64;
  int ch = 1;
  while (ch * 2 * per <= kStageFloats) ch *= 2;
  const size_t lds = sizeof(float) * (size_t)ch * per;
  if (limit > 0.f)
    return launch_kernel(small_update_kernel<true>, nA + n0 + nS, kTU, lds, s, act, n_active, rows, A1, D1, lda1, D2,
                         ldd2, W0, V0, ldw0, n0, H, W1, V1, ldw1, O, nA, ch, lr, mom, limit, faults);
  return launch_kernel(small_update_kernel<false>, nA + n0 + nS, kTU, lds, s, act, n_active, rows, A1, D1, lda1, D2,
                       ldd2, W0, V0, ldw0, n0, H, W1, V1, ldw1, O, nA, ch, lr, mom, limit, faults);
}

}  // namespace bpk
