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
//                  of every weight.  Each element is summed over the batch
//                  in pattern order by a fixed set of lanes, partial sums
//                  combined in a fixed order: no atomics, run-to-run
//                  identical.
//
// Arithmetic per element is the method's (sections 3 and 6.2.1); only the
// grouping of the work differs from the generic path.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "bp_device.h"
#include "bp_internal.h"

namespace bpk {
namespace {

constexpr int kT = 1024;       // threads per forward/backward block (16 waves)
constexpr int kTU = 1024;      // threads per update block (16 waves)
constexpr int kWU = kTU / 64;
constexpr int kMaxP = 8;       // patterns per forward/backward block

typedef float f32x4 __attribute__((ext_vector_type(4)));

// q / d and q % d for 0 <= q < 2^16 and 1 <= d <= 2^10, through a float
// reciprocal: the float quotient is within 2^-8 / d of the true one, far from
// the next integer, so the truncation is exact.
__device__ __forceinline__ void divmod(int q, int d, float inv_d, int& quo, int& rem) {
  quo = (int)(((float)q + 0.5f) * inv_d);
  rem = q - quo * d;
}

// Sum over aligned groups of 2^lg adjacent lanes (lg <= 4) by DPP lane moves
// inside each row of 16 lanes: lanes i ^ 1, lanes i ^ 2, then the mirror
// images within 8 and within 16 lanes.  Every lane of a group ends with the
// same value (each step adds two equal-shaped partial sums, and float
// addition is commutative).  All lanes of the wave must make the call.
template <int kCtrl>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), kCtrl, 0xF, 0xF, false));
}

__device__ __forceinline__ float group_sum(float v, int lg) {
  if (lg >= 1) v += dpp_move<0xB1>(v);    // quad_perm [1, 0, 3, 2]
  if (lg >= 2) v += dpp_move<0x4E>(v);    // quad_perm [2, 3, 0, 1]
  if (lg >= 3) v += dpp_move<0x141>(v);   // row_half_mirror
  if (lg >= 4) v += dpp_move<0x140>(v);   // row_mirror
  return v;
}

// Padded extents of the LDS copies: hidden units to a multiple of 128 and
// outputs to a multiple of 32, so that every lane of the output and delta
// sums reads a fixed multiple of 8 (resp. 4) entries, the padding being zero.
// W1's row stride S1 = Op + 4 is 4 modulo 64: the lanes of an output sum
// (consecutive hidden units, a few adjacent outputs) and of a delta sum
// (consecutive hidden units, adjacent outputs) fall on distinct banks.
__host__ __device__ __forceinline__ int small_hp(int H) { return (H + 127) / 128 * 128; }
__host__ __device__ __forceinline__ int small_op(int O) { return (O + 31) / 32 * 32; }

// Dynamic LDS of small_fwdbwd (floats unless noted):
//   w1s  HP x S1      W1 rows 0 .. H-1 (rows H .. HP-1, columns O .. OP-1 zero)
//   b1s  OP + 64      the bias row of W1
//   hs   P x HP       hidden activations (units H .. HP-1 zero)
//   d2s  P x OP       output deltas (outputs O .. OP-1 zero)
//   ts   P x O + 64   targets
// (the 64 extra entries of b1s and ts take the round-1 stores of the lanes
// past the end, one entry per lane)
__host__ __device__ __forceinline__ size_t small_fwdbwd_lds_floats(int P, int H, int O) {
  const int Hp = small_hp(H), Op = small_op(O);
  return (size_t)Hp * (Op + 4) + Op + 64 + (size_t)P * (Hp + Op) + (size_t)P * O + 64;
}

// 1024 threads (16 waves, four per SIMD) per block of P patterns.  With so
// little work per phase, the kernel is bound by instruction issue (a wave64
// instruction takes four cycles of its SIMD) and by dependent latencies, so
// the padded extents HP = small_hp(H) and OP = small_op(O) are template
// parameters: every LDS read of the sums below uses a constant offset from
// one base address, and the staging loop has a fixed trip count.
//   loads     one issue of global loads: each gather item's active
//             indices, then targets, the bias row and W1 (HP OP / 1024
//             elements per thread), then the gather's W0 rows as soon as
//             their indices arrive;
//   gather    one (pattern, hidden unit) pair per thread: bias + the active
//             rows of W0, in index order -> sigma;
//   output    each output (p, c) summed by 16 adjacent lanes, lane k over
//             the hidden units k, k + 16, ..., combined by group_sum;
//   deltas    each hidden delta (p, j) summed by 4 adjacent lanes, lane k
//             over the outputs k, k + 4, ..., combined by group_sum.
// For the update, hidden activations go out in groups of four units,
// A1q[j / 4][p][j % 4] (one float4 per pattern for the four W1 rows a block
// of the update handles), output deltas as rows of D2 and hidden deltas as
// rows of D1.  The activations and output deltas are written after the last
// phase: a phase that follows global stores can wait on them (a register the
// store read is written again), so they leave the chip when nothing else
// waits.
template <int P, bool TAB, int HP, int OP>
__global__ __launch_bounds__(kT) void small_fwdbwd_kernel(const int32_t* __restrict__ act, int n_active, int rows,
                                                          const float* __restrict__ W0, int ldw0, int n0,
                                                          int H, const float* __restrict__ W1, int ldw1, int O,
                                                          const float* __restrict__ T, float* A1q, int ldq,
                                                          float* D1, int ldd1, float* D2, int ldd2,
                                                          double* sse_part, const float* __restrict__ tab) {
  constexpr int S1 = OP + 4;                                 // W1 row stride, 4 modulo 64
  constexpr int LHP = HP == 128 ? 7 : 8;
  constexpr int NW = HP * OP / kT;                           // W1 elements staged per thread
  constexpr int RPP = kT / OP;                               // W1 rows per staging pass
  extern __shared__ float smem[];
  float* w1s = smem;                                         // HP x S1
  float* b1s = w1s + HP * S1;                                // OP + 64
  float* hs = b1s + OP + 64;                                 // P x HP
  float* d2s = hs + P * HP;                                  // P x OP
  float* ts = d2s + P * OP;                                  // P x O + 64
  __shared__ float red[kT / 64];

  const int tid = threadIdx.x;
  // blocks of one XCD (hardware block b runs on XCD b % 8) take a contiguous
  // range of patterns
  const int nbk = gridDim.x, xcd = blockIdx.x & 7, qb = nbk >> 3, rb = nbk & 7;
  const int lb = xcd * qb + min(xcd, rb) + (blockIdx.x >> 3);
  const int p0 = lb * P;
  const int np = min(P, rows - p0);
  const float inv_O = 1.0f / (float)O, inv_H = 1.0f / (float)H;

  // Loads in three groups, all in flight before the first is waited on:
  // each gather item's active indices, then the staging round, then the
  // gather's W0 rows, issued as soon as their indices arrive.  The thread of
  // gather item t = (pattern p, hidden unit j) reads its pattern's indices
  // straight from global memory (they depend on nothing staged here), so the
  // gather's loads overlap the staging round instead of following it.  Items
  // past the block's patterns read clamped, valid addresses and store nothing.
  constexpr int NG = (P * HP + kT - 1) / kT;                 // gather items per thread
  int iv[NG][8];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int p = min((tid + g * kT) >> LHP, np - 1);
    const int32_t* ip = act + (size_t)(p0 + p) * n_active;
#pragma unroll
    for (int u = 0; u < 8; ++u) iv[g][u] = ip[min(u, n_active - 1)];
  }
  // an index outside [0, n0) selects no row: it reads the bias row (always
  // valid) and adds nothing
  const unsigned n0u = (unsigned)n0;
  // Staging round (np * O <= 512 and P * OP <= 512 <= kT by the path's
  // limits).  Every load reads a clamped, valid address and is stored to LDS
  // unconditionally (the value selected; lanes past the end store to a spare
  // entry of their own), so that no load is sunk behind a branch.  (Rows of T
  // are contiguous.)
  const int nt = np * O;
  const float t0 = T[(size_t)p0 * O + min(tid, nt - 1)];
  const float bv = W1[(size_t)H * ldw1 + min(tid, O - 1)];
  const int c1 = tid & (OP - 1), jt = tid / OP;
  float v1[NW];
  {
    const float* wsrc = W1 + min(c1, O - 1);
#pragma unroll
    for (int u = 0; u < NW; ++u) v1[u] = wsrc[(size_t)min(jt + u * RPP, H - 1) * ldw1];
  }
  // keep the W0 loads behind the staging loads: waiting for an index must not
  // hold back the staging round
  __builtin_amdgcn_sched_barrier(0);
  float gv[NG][8], gb[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int jc = min((tid + g * kT) & (HP - 1), H - 1);
#pragma unroll
    for (int u = 0; u < 8; ++u) gv[g][u] = W0[(size_t)((unsigned)iv[g][u] < n0u ? iv[g][u] : n0) * ldw0 + jc];
    gb[g] = W0[(size_t)n0 * ldw0 + jc];
  }
  {
#pragma unroll
    for (int u = 0; u < NW; ++u) {
      const int j = jt + u * RPP;
      w1s[j * S1 + c1] = (j < H && c1 < O) ? v1[u] : 0.f;
    }
    const int spare = tid & 63;
    b1s[tid < OP ? tid : OP + spare] = tid < O ? bv : 0.f;
    ts[tid < nt ? tid : P * O + spare] = t0;
    if (tid < P * OP && (tid & (OP - 1)) >= O) d2s[tid] = 0.f;
  }
  // gather: net = bias + the active rows of W0 (in index order); units
  // H .. HP-1 get 0
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int t = tid + g * kT;
    if (t < np * HP) {
      const int p = t >> LHP, j = t & (HP - 1), jc = min(j, H - 1);
      float net = gb[g];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (u < n_active && (unsigned)iv[g][u] < n0u) net += gv[g][u];
      const int32_t* ip = act + (size_t)(p0 + p) * n_active;
      for (int k = 8; k < n_active; ++k) {
        const int ix = ip[k];
        if ((unsigned)ix < n0u) net += W0[(size_t)ix * ldw0 + jc];
      }
      const float h = TAB ? logistic_table(net, tab) : logistic(net);
      hs[t] = j < H ? h : 0.f;
    }
  }
  __syncthreads();
  // Output layer, output deltas and squared error.
  float sse = 0.f;
  {
    const int nout = np * O, part = tid & 15;
    for (int q0 = 0; q0 < nout; q0 += kT / 16) {
      const int q = q0 + (tid >> 4);
      int p = 0, c = 0;
      divmod(min(q, nout - 1), O, inv_O, p, c);
      const float* hp = hs + p * HP + part;             // units part, part + 16, ...
      const float* wp = w1s + part * S1 + c;
      float z0 = 0.f, z1 = 0.f;
#pragma unroll
      for (int u = 0; u < HP / 16; u += 2) {
        z0 += hp[16 * u] * wp[16 * u * S1];
        z1 += hp[16 * (u + 1)] * wp[16 * (u + 1) * S1];
      }
      const float z = group_sum(z0 + z1, 4);
      if (q < nout && part == 0) {
        const float zo = b1s[c] + z;
        const float y = TAB ? logistic_table(zo, tab) : logistic(zo);
        const float e = ts[q] - y;
        sse += e * e;
        d2s[p * OP + c] = e * y * (1.0f - y);
      }
    }
  }
  __syncthreads();
  // hidden deltas (W1 before its update, bias row excluded)
  {
    const int nh = np * H, part = tid & 3;
    for (int q0 = 0; q0 < nh; q0 += kT / 4) {
      const int q = q0 + (tid >> 2);
      int p = 0, j = 0;
      divmod(min(q, nh - 1), H, inv_H, p, j);
      const float* wp = w1s + j * S1 + part;            // outputs part, part + 4, ...
      const float* dp = d2s + p * OP + part;
      float s0 = 0.f, s1 = 0.f;
#pragma unroll
      for (int u = 0; u < OP / 4; u += 2) {
        s0 += wp[4 * u] * dp[4 * u];
        s1 += wp[4 * (u + 1)] * dp[4 * (u + 1)];
      }
      const float sd = group_sum(s0 + s1, 2);
      if (q < nh && part == 0) {
        const float h = hs[p * HP + j];
        D1[(size_t)(p0 + p) * ldd1 + j] = sd * (h * (1.0f - h));
      }
    }
  }
  // activations, quad-major so that a wave writes runs of P float4
  for (int t = tid; t < ((H + 3) >> 2) * 4 * P; t += kT) {
    const int r = t & 3, p = (t >> 2) & (P - 1), jq = t / (4 * P), j = 4 * jq + r;
    if (p < np && j < H) A1q[((size_t)jq * ldq + p0 + p) * 4 + r] = hs[p * HP + j];
  }
  for (int t = tid; t < np * O; t += kT) {
    int p = 0, c = 0;
    divmod(t, O, inv_O, p, c);
    D2[(size_t)(p0 + p) * ldd2 + c] = d2s[p * OP + c];
  }
  // block error partial, fixed order: rows of 16 lanes, then the four rows
  const int lane = tid & 63, wave = tid >> 6;
  sse = group_sum(sse, 4);
  sse = (__shfl(sse, 0, 64) + __shfl(sse, 16, 64)) + (__shfl(sse, 32, 64) + __shfl(sse, 48, 64));
  if (lane == 0) red[wave] = sse;
  __syncthreads();
  if (tid == 0) {
    double s = 0.0;
    for (int w = 0; w < kT / 64; ++w) s += (double)red[w];
    sse_part[lb] = s;
  }
}

// Patterns staged per chunk by the update's W1-tile blocks (D2 rows of
// Op / 4 float4 plus one float4 of activations each): 4096 float4 of D2.
__host__ __device__ __forceinline__ int small_update_chunk(int O) { return 4096 / (small_op(O) / 4); }

// 1024 threads = 16 waves per block.  The weight and momentum a thread
// updates are loaded in the block's first round of loads (loads that are
// still in flight at a loop head are waited for there, so they cannot be
// issued ahead of it).  Batch sums run over chunks of `ch` patterns staged in
// LDS by one round of coalesced loads, every load stored unconditionally so
// that none is sunk behind a branch.
// Blocks [0, nT): rows j0 .. j0+3 of W1 (j0 = 4 b; row H is the bias row,
//   activation 1), all O columns: G[j][c] = sum_p A1[p][j] D2[p][c].  The
//   first NCW threads compute: lane (sub, g) holds the 4 x 4 tile of rows
//   j0 .. j0+3 and columns 4 sub .. 4 sub + 3 over the patterns g, g + ng,
//   g + 2 ng, ... in order (ng = NCW / (Op / 4) lane groups); the group sums
//   are then added through LDS in a fixed tree.  NCW (128, 256 or 512) grows
//   with the batch: a small batch leaves most lanes without patterns, and
//   fewer group sums are cheaper to combine.
// Blocks [nT, nT + n0): row r of W0: the delta rows of the patterns whose
//   active list holds r, in pattern order (ballot compaction of 1024
//   patterns at a time); with ns = 1, 2 or 4 strips of 64 columns covering
//   H, wave w owns the column strip w % ns and the slice w / ns (of 16 / ns
//   equal slices) of each compacted list.
// Blocks [nT + n0, nT + n0 + nS): the bias row of W0, 32 columns per block:
//   sum_p D1[p][j], the half-wave h of wave w adding the (2 w + h)-th of 32
//   slices of each chunk in pattern order, the 32 slice sums combined in
//   slice order.
// CHECK: the range check of the summed changes (limit > 0).
// Sum of N values in a fixed pairwise tree.
template <int N>
__device__ __forceinline__ float tree_sum(const float* v) {
  if constexpr (N == 1)
    return v[0];
  else
    return tree_sum<N / 2>(v) + tree_sum<N / 2>(v + N / 2);
}

template <bool CHECK, int NCW>
__global__ __launch_bounds__(kTU) void small_update_kernel(const int32_t* __restrict__ act, int n_active, int rows,
                                                           const float* __restrict__ A1q, int ldq,
                                                           const float* __restrict__ D1, int ldd1,
                                                           const float* __restrict__ D2, int ldd2, float* W0,
                                                           float* V0, int ldw0, int n0, int H, float* W1, float* V1,
                                                           int ldw1, int O, int nT, int ch, float lr, float mom,
                                                           float limit, unsigned long long* faults,
                                                           const double* __restrict__ sse_part, int n_sse,
                                                           double* sse_out) {
  extern __shared__ f32x4 stage[];
  // The last update of a call has one more block, which sums the call's error
  // partials (all written by the forward/backward kernels before this launch).
  if (sse_out && (int)blockIdx.x == (int)gridDim.x - 1) {
    block_sum_partials<kTU>(sse_part, n_sse, sse_out, reinterpret_cast<double*>(stage));
    return;
  }
  __shared__ float part[kWU][64];
  __shared__ float tile_sum[256];
  __shared__ int list[kTU];
  __shared__ int wave_cnt[kWU];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const int Op = small_op(O), o4 = Op >> 2;

  float* Wt;        // weight row this block updates
  float* Vt;
  int col, ncol;    // thread's column in that row, row length
  bool owner;
  if (b < nT) {
    const int jj = tid / Op, j = b * 4 + jj;
    col = tid & (Op - 1);
    Wt = W1 + (size_t)min(j, H) * ldw1;
    Vt = V1 + (size_t)min(j, H) * ldw1;
    ncol = j <= H ? O : 0;
    owner = tid < 4 * Op;                            // whole waves
  } else if (b < nT + n0) {
    const int ns = H <= 64 ? 1 : (H <= 128 ? 2 : 4);
    Wt = W0 + (size_t)(b - nT) * ldw0;
    Vt = V0 + (size_t)(b - nT) * ldw0;
    col = (wave & (ns - 1)) * 64 + lane;
    ncol = H;
    owner = wave < ns;
  } else {
    Wt = W0 + (size_t)n0 * ldw0;
    Vt = V0 + (size_t)n0 * ldw0;
    col = lane < 32 ? (b - nT - n0) * 32 + lane : H;
    ncol = H;
    owner = wave == 0;
  }
  const bool live = col < ncol;
  const bool upd = owner && live;
  float w_old = 0.f, v_old = 0.f;

  float g = 0.f;
  if (b < nT) {
    const int j0 = b * 4;
    const int q4 = ldd2 >> 2;                        // float4 per D2 row (ldd2 % 4 == 0)
    const int lo4 = o4 == 8 ? 3 : 4;                 // log2(o4)
    f32x4* d2s = stage;                              // [ch][o4], columns past ldd2 zero
    f32x4* a1s = stage + ch * o4;                    // [ch + 64]: activations of rows j0 .. j0+3
    const f32x4* a1g = reinterpret_cast<const f32x4*>(A1q) + (size_t)min(b, (H - 1) >> 2) * ldq;
    const f32x4* d2g = reinterpret_cast<const f32x4*>(D2);
    const int sub = tid & (o4 - 1), grp = tid >> lo4, ng = NCW >> lo4;
    float acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.f;
    for (int pc = 0; pc < rows; pc += ch) {
      const int cn = min(ch, rows - pc);
      // one round: ch * o4 = 4096 float4 of D2 (4 per thread) and cn <= 1024
      // float4 of activations (1 per thread), clamped addresses, values
      // selected (row H is the bias row: activation 1; rows past it 0)
      {
        const int nd = cn * o4;
        if (pc == 0 && upd) {
          w_old = Wt[col];
          v_old = Vt[col];
        }
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = min(tid + u * kTU, nd - 1);
          const int p = i >> lo4, k = i & (o4 - 1);
          v[u] = d2g[(size_t)(pc + p) * q4 + min(k, q4 - 1)];
        }
        f32x4 av = a1g[pc + min(tid, cn - 1)];
#pragma unroll
        for (int r = 0; r < 4; ++r) av[r] = j0 + r < H ? av[r] : (j0 + r == H ? 1.0f : 0.f);
#pragma unroll
        for (int u = 0; u < 4; ++u) {             // ch * o4 = 4 kTU slots
          const int i = tid + u * kTU;
          d2s[i] = (i < nd && (i & (o4 - 1)) < q4) ? v[u] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
        a1s[tid < ch ? tid : ch + lane] = av;
      }
      __syncthreads();
      if (tid < NCW) {
        for (int p = grp; p < cn; p += 4 * ng) {
          f32x4 a[4], d[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int pp = min(p + u * ng, cn - 1);
            a[u] = a1s[pp];
            d[u] = d2s[pp * o4 + sub];
          }
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (p + u * ng < cn) {
#pragma unroll
              for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int q = 0; q < 4; ++q) acc[r * 4 + q] += a[u][r] * d[u][q];
            }
        }
      }
      __syncthreads();
    }
    // the lane groups' tiles through LDS: group grp's 16 o4 sums at
    // accs[grp * S + i * Op + 4 sub + q] (acc[4 i + q]; row stride S = 16 o4
    // + 8 floats keeps both the writes and the strided reads below free of
    // bank conflicts).  Element el = i * Op + 4 sub + q is summed by
    // tpe = 1024 / (16 o4) adjacent threads, thread s over the NCW / 64
    // groups s, s + tpe, ..., the partial sums combined by group_sum.
    const int S4 = 4 * o4 + 2;                           // row stride in float4
    if (tid < NCW) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        stage[grp * S4 + i * o4 + sub] = f32x4{acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]};
    }
    __syncthreads();
    {
      const int lt = 6 - lo4, tpe = 1 << lt;             // 8 (o4 = 8) or 4 (o4 = 16)
      const int el = tid >> lt, sl = tid & (tpe - 1);
      const float* src = reinterpret_cast<const float*>(stage) + el;
      constexpr int GPT = NCW / 64;                      // ng = GPT tpe groups
      float v[GPT];
#pragma unroll
      for (int u = 0; u < GPT; ++u) v[u] = src[(sl + tpe * u) * (4 * S4)];
      float x = tree_sum<GPT>(v);
      x = group_sum(x, lt);
      if (sl == 0) tile_sum[el] = x;
    }
    __syncthreads();
    if (owner) g = tile_sum[tid];                       // tid = jj Op + col
  } else if (b < nT + n0) {
    const int r = b - nT;
    const int ns = H <= 64 ? 1 : (H <= 128 ? 2 : 4), nsl = kWU / ns, slice = wave / ns;
    for (int pc = 0; pc < rows; pc += kTU) {
      const int p = pc + tid;
      if (pc == 0 && upd) {
        w_old = Wt[col];
        v_old = Vt[col];
      }
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
      const int q0 = (int)((int64_t)total * slice / nsl), q1 = (int)((int64_t)total * (slice + 1) / nsl);
      float s = 0.f;
      if (live) {
        for (int q = q0; q < q1; q += 4) {
          float v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = D1[(size_t)list[min(q + u, q1 - 1)] * ldd1 + col];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (q + u < q1) s += v[u];
        }
      }
      // the slices of this chunk are added to the running sum in list order
      part[wave][lane] = s;
      __syncthreads();
      if (owner)
        for (int k = 0; k < nsl; ++k) g += part[k * ns + wave][lane];
      __syncthreads();
    }
  } else {
    // bias row of W0: columns c0 .. c0 + 31 of D1, staged as float4 (a D1
    // row is ldd1 floats, ldd1 % 4 == 0; columns past H are never summed),
    // 512 patterns per chunk
    const int c0 = (b - nT - n0) * 32, c = lane & 31, h = lane >> 5;
    f32x4* d1s = stage;                              // [512][8]
    for (int pc = 0; pc < rows; pc += 512) {
      const int cn = min(512, rows - pc), nd = cn * 8;
      if (pc == 0 && upd) {
        w_old = Wt[col];
        v_old = Vt[col];
      }
      f32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = min(tid + u * kTU, nd - 1);
        const int cc = min(c0 + (i & 7) * 4, ldd1 - 4);
        v[u] = *reinterpret_cast<const f32x4*>(D1 + (size_t)(pc + (i >> 3)) * ldd1 + cc);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) d1s[tid + u * kTU] = v[u];   // 512 x 8 slots; past nd unread
      __syncthreads();
      const int sl = 2 * wave + h, s0 = cn * sl / 32, s1 = cn * (sl + 1) / 32;
      const float* col_s = reinterpret_cast<const float*>(d1s) + c;
      float sum = 0.f;
      for (int p = s0; p < s1; p += 8) {
        float dv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) dv[u] = col_s[min(p + u, s1 - 1) * 32];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (p + u < s1) sum += dv[u];
      }
      part[wave][lane] = sum;
      __syncthreads();
      if (owner && lane < 32)
        for (int w = 0; w < kWU; ++w) g = (g + part[w][lane]) + part[w][lane + 32];
      __syncthreads();
    }
  }
  if (owner) {   // whole waves
    int nf = 0;
    if (upd) {
      if (CHECK) g = checked_change(g, limit, nf);
      const float v = momentum_step(g, v_old, lr, mom);
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

size_t small_scratch_floats(int rows, int H) { return rows > 0 ? (size_t)((H + 3) / 4) * 4 * rows : 0; }

template <int P, bool TAB>
hipError_t launch_fwdbwd_p(hipStream_t s, int nb, size_t lds, const int32_t* act, int n_active, int rows,
                           const float* W0, int ldw0, int n0, int H, const float* W1, int ldw1, int O, const float* T,
                           float* A1q, float* D1, int ldd1, float* D2, int ldd2, double* sse_part, const float* tab) {
  const int hp = small_hp(H), op = small_op(O);
#define BP_FB(HPV, OPV)                                                                                      \
  if (hp == HPV && op == OPV)                                                                                \
    return launch_kernel(small_fwdbwd_kernel<P, TAB, HPV, OPV>, nb, kT, lds, s, act, n_active, rows, W0, ldw0, \
                         n0, H, W1, ldw1, O, T, A1q, rows, D1, ldd1, D2, ldd2, sse_part, tab);
  BP_FB(128, 32)
  BP_FB(128, 64)
  BP_FB(256, 32)
  BP_FB(256, 64)
#undef BP_FB
  return hipErrorInvalidValue;
}

template <bool TAB>
hipError_t launch_fwdbwd(hipStream_t s, int P, int nb, size_t lds, const int32_t* act, int n_active, int rows,
                         const float* W0, int ldw0, int n0, int H, const float* W1, int ldw1, int O, const float* T,
                         float* A1q, float* D1, int ldd1, float* D2, int ldd2, double* sse_part, const float* tab) {
  switch (P) {
    case 1: return launch_fwdbwd_p<1, TAB>(s, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1q, D1, ldd1, D2, ldd2, sse_part, tab);
    case 2: return launch_fwdbwd_p<2, TAB>(s, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1q, D1, ldd1, D2, ldd2, sse_part, tab);
    case 4: return launch_fwdbwd_p<4, TAB>(s, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1q, D1, ldd1, D2, ldd2, sse_part, tab);
    default: return launch_fwdbwd_p<8, TAB>(s, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1q, D1, ldd1, D2, ldd2, sse_part, tab);
  }
}

hipError_t small_fwdbwd(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw0, int n0,
                        int H, const float* W1, int ldw1, int O, const float* T, float* A1q, float* D1, int ldd1,
                        float* D2, int ldd2, double* sse_part, const float* tab) {
  if (rows <= 0) return hipSuccess;
  const int P = patterns_per_block(rows);
  const size_t lds = sizeof(float) * small_fwdbwd_lds_floats(P, H, O);
  const int nb = small_fwdbwd_blocks(rows);
  if (tab)
    return launch_fwdbwd<true>(s, P, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1q, D1, ldd1,
                               D2, ldd2, sse_part, tab);
  return launch_fwdbwd<false>(s, P, nb, lds, act, n_active, rows, W0, ldw0, n0, H, W1, ldw1, O, T, A1q, D1, ldd1, D2,
                              ldd2, sse_part, tab);
}

hipError_t small_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* A1q, const float* D1,
                        int ldd1, const float* D2, int ldd2, float* W0, float* V0, int ldw0, int n0, int H, float* W1,
                        float* V1, int ldw1, int O, float lr, float mom, float limit, unsigned long long* faults,
                        const double* sse_part, int n_sse, double* sse_out) {
  if (rows <= 0) return hipSuccess;
  const int nT = (H + 1 + 3) / 4;
  const int nS = (H + 31) / 32;
  const int ch = small_update_chunk(O), o4 = small_op(O) / 4;
  // tile chunks: ch (o4 + 1) + 64 float4; bias-row chunks: 512 rows of 8 float4
  // (at least kTU doubles for the error sum)
  const size_t lds = 16 * std::max((size_t)ch * (size_t)(o4 + 1) + 64, (size_t)512 * 8);
  const int blocks = nT + n0 + nS + (sse_out ? 1 : 0);
  // W1-tile compute width by batch (measured at 16 rows: 512 lanes 7.62, 256
  // lanes 7.41, 128 lanes 7.39 us per update; at 512 rows 512 lanes are best)
  const int ncw = rows <= 64 ? 128 : (rows <= 256 ? 256 : 512);
#define BP_UPD(CHK, NCWV)                                                                                          \
  if (ncw == NCWV)                                                                                                 \
    return launch_kernel(small_update_kernel<CHK, NCWV>, blocks, kTU, lds, s, act, n_active, rows, A1q, rows, D1, \
                         ldd1, D2, ldd2, W0, V0, ldw0, n0, H, W1, V1, ldw1, O, nT, ch, lr, mom, limit, faults,      \
                         sse_part, n_sse, sse_out);
  if (limit > 0.f) {
    BP_UPD(true, 128)
    BP_UPD(true, 256)
    BP_UPD(true, 512)
  } else {
    BP_UPD(false, 128)
    BP_UPD(false, 256)
    BP_UPD(false, 512)
  }
#undef BP_UPD
  return hipErrorInvalidValue;
}

}  // namespace bpk
