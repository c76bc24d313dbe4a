// bp_kernels.hip -- gfx950 (CDNA4) kernels of pooled back-propagation, fp32.
//
// The three weight contractions of one pooled update (forward, hidden deltas,
// summed change) are dense fp32 products and run on the matrix cores
// (v_mfma_f32_32x32x2_f32) with LDS-staged tiles; each one fuses the
// elementwise step that follows it in the method:
//   forward     A_{l+1} = sigma(A_l W_l + bias)             (section 3)
//   output      delta_L = (T - Y) Y (1 - Y), error partials  (section 3, fn 5)
//   backward    delta_l = (delta_{l+1} W_l^T) * A_l (1 - A_l) (section 3)
//   change      V = lr (A_l^T delta_{l+1}) + mom V; W += V    (sections 3, 6.2.1)
// The one-hot first layer of the NETtalk-style input window (section 6.3)
// gathers and scatters weight rows instead of multiplying by a 0/1 matrix.
//
// Every reduction runs in a fixed order: results are run-to-run identical.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "bp_device.h"
#include "bp_internal.h"

namespace bpk {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;

// --------------------------------------------------------------------------
// Epilogues.  apply() gets one element of the product (row m, column n) plus
// the per-column value column() returned, and returns the value that enters
// the per-tile column sums; its last argument is a per-lane statistic: the
// squared error for kSSE epilogues (added into a per-block partial), the
// number of range-check faults for kFaults epilogues (added to the fault
// counter).  kColSum marks epilogues that write per-tile column sums of the
// deltas they produce (colsum[tile row][n]; the bias-row change of the layer
// below is the sum of these over the tile rows).  `tab` is the sigmoid table
// (nullptr: exact logistic).
//
// load() returns the per-element operands an epilogue reads from memory
// (Pre).  The kernel loads them for a whole 32 x 32 block before the
// block's first store, so the loads are in flight together instead of each
// waiting behind the stores of the elements before it (which the compiler
// must assume may alias them).

typedef float f32x2 __attribute__((ext_vector_type(2)));
struct NoPre {};

struct EpiSigmoid {
  const float* bias;
  float* out;
  int ldo;
  const float* tab;
  static constexpr bool kSSE = false;
  static constexpr bool kColSum = false;
  static constexpr bool kFaults = false;
  using Pre = NoPre;
  __device__ Pre load(int, int) const { return {}; }
  __device__ float column(int n) const { return bias[n]; }
  __device__ float apply(int m, int n, float acc, float b, Pre, float&) const {
    out[(size_t)m * ldo + n] = unit_sigma(acc + b, tab);
    return 0.f;
  }
};

struct EpiOutputDelta {
  const float* bias;
  const float* T;
  int ldt;
  float* delta;
  int ldd;
  double* sse_part;
  float* colsum;
  int ldcs;
  const float* tab;
  const float* mask;     // per-row error multiplier (section 10.5), or nullptr
  static constexpr bool kSSE = true;
  static constexpr bool kColSum = true;
  static constexpr bool kFaults = false;
  using Pre = f32x2;     // target, mask
  __device__ Pre load(int m, int n) const { return {T[(size_t)m * ldt + n], mask ? mask[m] : 1.0f}; }
  __device__ float column(int n) const { return bias[n]; }
  __device__ float apply(int m, int n, float acc, float b, Pre tm, float& sse) const {
    const float y = unit_sigma(acc + b, tab);
    float e = tm.x - y;
    if (mask) e *= tm.y;
    sse += e * e;
    const float d = e * y * (1.0f - y);
    delta[(size_t)m * ldd + n] = d;
    return d;
  }
};

struct EpiHiddenDelta {
  const float* act;
  int lda;
  float* out;
  int ldo;
  float* colsum;
  int ldcs;
  static constexpr bool kSSE = false;
  static constexpr bool kColSum = true;
  static constexpr bool kFaults = false;
  using Pre = float;     // activation
  __device__ Pre load(int m, int n) const { return act[(size_t)m * lda + n]; }
  __device__ float column(int) const { return 0.f; }
  __device__ float apply(int m, int n, float acc, float, Pre a, float&) const {
    const float d = acc * (a * (1.0f - a));
    out[(size_t)m * ldo + n] = d;
    return d;
  }
};

struct EpiUpdate {
  float* W;
  float* V;
  int ldw;
  float lr, mom;
  float limit;                      // range check of the summed change (> 0: on)
  unsigned long long* faults;
  static constexpr bool kSSE = false;
  static constexpr bool kColSum = false;
  static constexpr bool kFaults = true;
  using Pre = f32x2;     // momentum, weight
  __device__ Pre load(int m, int n) const {
    const size_t i = (size_t)m * ldw + n;
    return {V[i], W[i]};
  }
  __device__ float column(int) const { return 0.f; }
  __device__ float apply(int m, int n, float acc, float, Pre vw, float& nf) const {
    const size_t i = (size_t)m * ldw + n;
    int f = 0;
    const float g = checked_change(acc, limit, f);
    nf += (float)f;
    const float v = momentum_step(g, vw.x, lr, mom);
    V[i] = v;
    W[i] = vw.y + v;
    return 0.f;
  }
};

// Split-K partial: P[z][m][n] for z = blockIdx.z.
struct EpiPartial {
  float* P;
  int ldp;
  size_t split_stride;
  static constexpr bool kSSE = false;
  static constexpr bool kColSum = false;
  static constexpr bool kFaults = false;
  using Pre = NoPre;
  __device__ Pre load(int, int) const { return {}; }
  __device__ float column(int) const { return 0.f; }
  __device__ float apply(int m, int n, float acc, float, Pre, float&) const {
    P[blockIdx.z * split_stride + (size_t)m * ldp + n] = acc;
    return 0.f;
  }
};

// Split-K change product fused with the update (the update routine of
// section 6.2.1 applied to the batch-summed change).  The blocks of one
// output tile each sum one K range of the batch.  Every block stores its
// partial sums and counts its arrival (one counter per output tile); the
// block that arrives last adds the tile's partials in split order, taking
// its own from registers, and applies the range check and the momentum
// update to them, as the epilogue of an unsplit product does.  The sum does
// not depend on which block arrives last (results are run-to-run identical)
// and the summed change itself never reaches memory.
//
// Partials are stored in the accumulator layout, lane fastest: 4-float slot
// u of lane l in wave w of block (tile t, split z) is at float offset
//   (((z * tiles + t) * waves + w) * slots + u) * 256 + 4 l,
// so every store or load instruction of a wave covers 1 KB of contiguous
// memory.  They are written and read with the device-coherent cache policy
// (written through the L2 of the XCD, read from the coherent level), so
// blocks on different XCDs see each other's partials without a fence (a
// device-scope fence would write back, or drop, the whole L2 of the XCD).
struct EpiSplitUpdate {
  float* P;                         // partials (split_workspace floats)
  float* W;
  float* V;
  int ldw;
  float lr, mom;
  float limit;                      // range check of the summed change (> 0: on)
  unsigned long long* faults;
  int* arrivals;                    // per output tile; zero before and after every launch
  int splits;
  static constexpr bool kColSum = false;
  static constexpr bool kFaults = true;
};

constexpr int kCoherent = 16;       // buffer cache policy bit sc1: device-coherent access

__device__ __forceinline__ __amdgpu_buffer_rsrc_t partial_rsrc(float* base) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, 0x7fffffff, 0x00020000);
}

// Every thread of the block calls this after storing its partial slots.
// Each wave waits until its stores are complete (performed at the coherent
// level) before the block's arrival is counted.  Returns true, in every
// thread, in the block that arrives last at `tile`; that block also resets
// the tile's counter for the next launch.
__device__ __forceinline__ bool split_arrive(const EpiSplitUpdate& e, int tile) {
  __shared__ int last;
  __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): this wave's partial stores are complete
  __syncthreads();
  if (threadIdx.x == 0) {
    const bool l =
        __hip_atomic_fetch_add(e.arrivals + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == e.splits - 1;
    if (l) __hip_atomic_store(e.arrivals + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = l;
  }
  __syncthreads();
  return last;
}

// g[u] = the sum over splits 0 .. S-1, in split order, of this lane's slot
// `slot0 + u` (split z's own value from `own`).  `r` addresses split 0 of
// the block's partials; splits are `zstride` bytes apart, slots 1 KB.  The
// other splits' slots are loaded in groups of ZB splits, all in flight
// together: by default one split at a time for 4 slots (a 32 x 32 block of
// 128-row tiles of gemm_kernel: more would cost it its second wave per
// SIMD), 16 splits for one slot.  The 64 x 64 tiles, launched about one
// block per CU, load 8 splits at a time (Elman epoch 1.3% faster).
template <int NS, int ZB = (NS >= 4 ? 1 : 16 / NS)>   // ZB: splits per load group
__device__ __forceinline__ void ordered_split_sum(f32x4 (&g)[NS], const f32x4 (&own)[NS], __amdgpu_buffer_rsrc_t r,
                                                  int zstride, int slot0, int lane, int z, int S) {
#pragma unroll
  for (int u = 0; u < NS; ++u) g[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int z0 = 0; z0 < S; z0 += ZB) {
    f32x4 t[ZB][NS];
#pragma unroll
    for (int d = 0; d < ZB; ++d) {
      const int zz = z0 + d;
      if (zz < S && zz != z) {
#pragma unroll
        for (int u = 0; u < NS; ++u)
          t[d][u] = __builtin_amdgcn_raw_buffer_load_b128(r, zz * zstride + ((slot0 + u) * 64 + lane) * 16, 0,
                                                          kCoherent);
      }
    }
#pragma unroll
    for (int d = 0; d < ZB; ++d) {
      const int zz = z0 + d;
      if (zz < S) {
#pragma unroll
        for (int u = 0; u < NS; ++u) g[u] += zz == z ? own[u] : t[d][u];
      }
    }
  }
}

// --------------------------------------------------------------------------
// Tiled fp32 MFMA product C[M][N] = sum_k A(m, k) B(k, n).
//
// Operand storage (global and LDS alike, so tiles are copied without a
// transpose):  A_KM false: A[m * lda + k]   true: A[k * lda + m]
//              B_NK false: B[k * ldb + n]   true: B[n * ldb + k]
// 256 threads = 4 waves in a 2 x 2 grid; each wave owns a (BM/2) x (BN/2)
// sub-tile made of 32 x 32 MFMA blocks.  Within a group of 8 k values, MFMA
// t (t = 0..3) pairs k = 8g + t (lanes 0-31) with k = 8g + 4 + t (lanes
// 32-63); A and B use the same assignment, so each lane can fetch its four k
// values of a k-contiguous tile with one 16-byte LDS read.
template <int BM, int BN, int BK, bool A_KM, bool B_NK, int NTH = kThreads>
struct Tile {
  // wave grid: 2 x 2 waves for 256 threads, 2 x 4 for 512 (wave tile 128 x 64)
  static constexpr int WGM = 2, WGN = NTH / 128;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int SA = A_KM ? (BM + 8) : (BK + 4);   // LDS row strides (floats)
  static constexpr int SB = B_NK ? (BK + 4) : (BN + 8);
  static constexpr int A_ELEMS = A_KM ? BK * SA : BM * SA;
  static constexpr int B_ELEMS = B_NK ? BN * SB : BK * SB;
  static constexpr int LA = BM * BK / 4 / NTH;             // float4 loads per thread per stage
  static constexpr int LB = BN * BK / 4 / NTH;
  static_assert(BM % 64 == 0 && BN % 64 == 0 && BK % 8 == 0, "tile shape");
  static_assert(LA * 4 * NTH == BM * BK && LB * 4 * NTH == BN * BK, "tile split");
};

// Loads a TO x TD tile (TD contiguous) whose origin is (o0, d0) into
// registers; elements outside [0, O_lim) x [0, D_lim) read as zero.
template <int TO, int TD, bool VEC, int NTH = kThreads>
__device__ __forceinline__ void load_tile(const float* __restrict__ base, int ld, int o0, int d0, int O_lim,
                                          int D_lim, f32x4* r, int tid) {
  constexpr int PER = TO * TD / 4 / NTH;
  constexpr int D4 = TD / 4;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int f = tid + q * NTH;
    const int go = o0 + f / D4, gd = d0 + (f % D4) * 4;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (go < O_lim) {
      const float* p = base + (size_t)go * ld + gd;
      if (VEC && gd + 4 <= D_lim) {
        v = *reinterpret_cast<const f32x4*>(p);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (gd + e < D_lim) v[e] = p[e];
      }
    }
    r[q] = v;
  }
}

// Loads a TO x TD tile that lies entirely inside the matrix, 16 bytes per
// load, with no bounds checks (interior tiles of 16-byte aligned operands).
template <int TO, int TD, int NTH = kThreads>
__device__ __forceinline__ void load_tile_full(const float* __restrict__ base, int ld, int o0, int d0, f32x4* r,
                                               int tid) {
  constexpr int PER = TO * TD / 4 / NTH;
  constexpr int D4 = TD / 4;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int f = tid + q * NTH;
    r[q] = *reinterpret_cast<const f32x4*>(base + (size_t)(o0 + f / D4) * ld + d0 + (f % D4) * 4);
  }
}

template <int TO, int TD, int S, int NTH = kThreads>
__device__ __forceinline__ void store_tile(float* lds, const f32x4* r, int tid) {
  constexpr int PER = TO * TD / 4 / NTH;
  constexpr int D4 = TD / 4;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int f = tid + q * NTH;
    *reinterpret_cast<f32x4*>(lds + (f / D4) * S + (f % D4) * 4) = r[q];
  }
}

// A TO x TD tile (TD contiguous, inside the matrix) copied from global memory
// straight into its LDS image [TO][S] by the LDS-DMA load: one wave
// instruction writes 64 consecutive 16-byte chunks of the image (lane l the
// l-th), each lane loading its chunk's global address.  The image is taken in
// blocks of 64 chunks, block b by wave b % NW; a chunk of row padding
// (S - TD floats per row) loads a copy of the row's last data chunk.  Its
// global offsets relative to the tile origin are fixed across K stages, so
// they are computed once (off) and a stage passes the origin.
template <int TO, int TD, int S, int NTH>
struct DmaTile {
  static constexpr int CPR = S / 4;                   // chunks per image row
  static constexpr int Q = TO * CPR;                  // chunks
  static constexpr int NB = (Q + 63) / 64;            // 64-chunk blocks
  static constexpr int NW = NTH / 64;
  static constexpr int PER = (NB + NW - 1) / NW;      // blocks per wave (at most)
  static_assert(S % 4 == 0 && TD % 4 == 0 && S >= TD, "DMA tile shape");
  int off[PER];                                       // element offsets from the origin
  __device__ __forceinline__ void init(int ld, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = min((wave + i * NW) * 64 + lane, Q - 1);
      const int row = q / CPR, c = min(q % CPR, TD / 4 - 1);
      off[i] = row * ld + 4 * c;
    }
  }
  // the tile with origin `org` (global) into the image `lds`
  __device__ __forceinline__ void copy(const float* org, float* lds, int wave, int lane) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = wave + i * NW;
#if defined(__HIP_DEVICE_COMPILE__)   // (a device instruction: the host pass only sees the kernel's signature)
      if (b < NB && (b < NB - 1 || lane < Q - 64 * (NB - 1)))
        __builtin_amdgcn_global_load_lds(org + off[i],
                                         (__attribute__((address_space(3))) void*)(lds + 256 * b), 16, 0, 0);
#endif
    }
  }
};

// Maps the hardware block index to a tile.  Blocks reach the eight XCDs
// round-robin (hardware index mod 8); each XCD is given a contiguous range
// of the tile order, and the tile order walks groups of 8 tile rows column by
// column, so the blocks an XCD runs at once cover about 8 x 8 tiles and
// share both their A and their B tiles in that XCD's L2.
constexpr int kGroupM = 8;
__device__ __forceinline__ void xcd_tile(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int per = nblocks >> 3;
  const int t = bid >= (per << 3) ? bid : (bid & 7) * per + (bid >> 3);
  const int band = t / (kGroupM * tiles_n);
  const int first = band * kGroupM;
  const int rows = min(tiles_m - first, kGroupM);
  const int in_band = t - band * kGroupM * tiles_n;
  tm = first + in_band % rows;
  tn = in_band / rows;
}

template <int BM, int BN, int BK, bool A_KM, bool B_NK, bool AVEC, bool BVEC, class Epi, int NTH = kThreads>
__global__ __launch_bounds__(NTH) void gemm_kernel(const float* __restrict__ A, int lda,
                                                   const float* __restrict__ B, int ldb, int M, int N,
                                                   int K, int k_chunk, Epi epi) {
  using T = Tile<BM, BN, BK, A_KM, B_NK, NTH>;
  // 512-thread blocks (256 x 256 tiles) only for full tiles of the sigmoid and
  // hidden-delta products, which end through the row epilogue
  static_assert(NTH == kThreads || ((std::is_same_v<Epi, EpiSigmoid> || std::is_same_v<Epi, EpiHiddenDelta>) &&
                                    BM == 256 && BN == 256),
                "512-thread tiles: full-tile sigmoid and hidden-delta products");
  __shared__ __attribute__((aligned(16))) float As[2][T::A_ELEMS];
  __shared__ __attribute__((aligned(16))) float Bs[2][T::B_ELEMS];

  const int tiles_n = (N + BN - 1) / BN, tiles_m = (M + BM - 1) / BM;
  int tm, tn;
  xcd_tile(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x;
  const int kb = blockIdx.z * k_chunk;
  const int ke = min(K, kb + k_chunk);

  const int wave = tid >> 6, lane = tid & 63;
  const int wm0 = (wave / T::WGN) * T::WM, wn0 = (wave % T::WGN) * T::WN;
  const int r = lane & 31, h = lane >> 5;

  f32x16 acc[T::TM][T::TN];
#pragma unroll
  for (int i = 0; i < T::TM; ++i)
#pragma unroll
    for (int j = 0; j < T::TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // Two register sets: the tile of stage s + 2 is loaded while stage s is
  // multiplied, so a global load has two stages of MFMA work to land before
  // its registers are written to LDS.
  f32x4 ra0[T::LA], rb0[T::LB], ra1[T::LA], rb1[T::LB];
  // Interior tiles (the block-uniform common case) take the unchecked path.
  const bool a_rows_in = m0 + BM <= M, b_rows_in = n0 + BN <= N;
  auto load_stage = [&](int k, f32x4* ra, f32x4* rb) {
    if constexpr (NTH != kThreads) {   // launched only on whole tiles: M, N, K multiples of the tile
      if (A_KM) load_tile_full<BK, BM, NTH>(A, lda, k, m0, ra, tid);
      else load_tile_full<BM, BK, NTH>(A, lda, m0, k, ra, tid);
      if (B_NK) load_tile_full<BN, BK, NTH>(B, ldb, n0, k, rb, tid);
      else load_tile_full<BK, BN, NTH>(B, ldb, k, n0, rb, tid);
      return;
    }
    const bool k_in = k + BK <= ke;
    if (AVEC && a_rows_in && k_in) {
      if (A_KM) load_tile_full<BK, BM, NTH>(A, lda, k, m0, ra, tid);
      else load_tile_full<BM, BK, NTH>(A, lda, m0, k, ra, tid);
    } else {
      if (A_KM) load_tile<BK, BM, AVEC, NTH>(A, lda, k, m0, ke, M, ra, tid);
      else load_tile<BM, BK, AVEC, NTH>(A, lda, m0, k, M, ke, ra, tid);
    }
    if (BVEC && b_rows_in && k_in) {
      if (B_NK) load_tile_full<BN, BK, NTH>(B, ldb, n0, k, rb, tid);
      else load_tile_full<BK, BN, NTH>(B, ldb, k, n0, rb, tid);
    } else {
      if (B_NK) load_tile<BN, BK, BVEC, NTH>(B, ldb, n0, k, N, ke, rb, tid);
      else load_tile<BK, BN, BVEC, NTH>(B, ldb, k, n0, ke, N, rb, tid);
    }
  };
  auto store_stage = [&](int buf, const f32x4* ra, const f32x4* rb) {
    if (A_KM) store_tile<BK, BM, T::SA, NTH>(As[buf], ra, tid);
    else store_tile<BM, BK, T::SA, NTH>(As[buf], ra, tid);
    if (B_NK) store_tile<BN, BK, T::SB, NTH>(Bs[buf], rb, tid);
    else store_tile<BK, BN, T::SB, NTH>(Bs[buf], rb, tid);
  };
  auto compute = [&](int buf) {
    const float* as = As[buf];
    const float* bs = Bs[buf];
#pragma unroll
    for (int g = 0; g < BK / 8; ++g) {
      f32x4 af[T::TM], bf[T::TN];
#pragma unroll
      for (int i = 0; i < T::TM; ++i) {
        const int m = wm0 + i * 32 + r;
        if (A_KM) {
#pragma unroll
          for (int t = 0; t < 4; ++t) af[i][t] = as[(g * 8 + 4 * h + t) * T::SA + m];
        } else {
          af[i] = *reinterpret_cast<const f32x4*>(as + m * T::SA + g * 8 + 4 * h);
        }
      }
#pragma unroll
      for (int j = 0; j < T::TN; ++j) {
        const int n = wn0 + j * 32 + r;
        if (B_NK) {
          bf[j] = *reinterpret_cast<const f32x4*>(bs + n * T::SB + g * 8 + 4 * h);
        } else {
#pragma unroll
          for (int t = 0; t < 4; ++t) bf[j][t] = bs[(g * 8 + 4 * h + t) * T::SB + n];
        }
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < T::TM; ++i)
#pragma unroll
          for (int j = 0; j < T::TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][t], bf[j][t], acc[i][j], 0, 0, 0);
    }
  };
  // One pipeline step at stage s: registers `rl` (which held stage s, already
  // in LDS) receive stage s + 2; LDS buffer s % 2 is multiplied; registers
  // `rs` (stage s + 1) are written to the other LDS buffer.
  const int nst = ke > kb ? (ke - kb + BK - 1) / BK : 0;
  auto step = [&](int s, f32x4* rla, f32x4* rlb, const f32x4* rsa, const f32x4* rsb) {
    if (s + 2 < nst) load_stage(kb + (s + 2) * BK, rla, rlb);
    compute(s & 1);
    if (s + 1 < nst) store_stage((s + 1) & 1, rsa, rsb);
    __syncthreads();
  };
  if constexpr (NTH != kThreads && B_NK) {
    // 512-thread blocks hold twice the accumulators per wave; one register
    // set suffices there, as a stage is twice the MFMA work per SIMD (two
    // waves of 128 x 64 each): the load of stage s + 1 lands while stage s
    // is multiplied.
    if (nst > 0) {
      load_stage(kb, ra0, rb0);
      store_stage(0, ra0, rb0);
      __syncthreads();
    }
    for (int s = 0; s < nst; ++s) {
      if (s + 1 < nst) load_stage(kb + (s + 1) * BK, ra0, rb0);
      compute(s & 1);
      if (s + 1 < nst) store_stage((s + 1) & 1, ra0, rb0);
      __syncthreads();
    }
  } else if constexpr (NTH != kThreads) {
    // The sigmoid products' 512-thread blocks (whole tiles only) copy each
    // stage straight into LDS with the LDS-DMA load: stage s + 1 is copied
    // into the other buffer while stage s is multiplied, and the barrier that
    // ends stage s waits for the copy; no staging registers, no LDS stores.
    // (Measured: forward products 1.3% faster; the hidden-delta products, whose
    // B tile is also sliced into 128-byte rows, 3% slower, so they stage
    // through registers.)
    DmaTile<A_KM ? BK : BM, A_KM ? BM : BK, T::SA, NTH> da;
    DmaTile<B_NK ? BN : BK, B_NK ? BK : BN, T::SB, NTH> db;
    da.init(lda, wave, lane);
    db.init(ldb, wave, lane);
    // stage origins: the tile's first row and column at depth k
    auto a_org = [&](int k) { return A_KM ? A + (size_t)k * lda + m0 : A + (size_t)m0 * lda + k; };
    auto b_org = [&](int k) { return B_NK ? B + (size_t)n0 * ldb + k : B + (size_t)k * ldb + n0; };
    if (nst > 0) {
      da.copy(a_org(kb), As[0], wave, lane);
      db.copy(b_org(kb), Bs[0], wave, lane);
      __syncthreads();
    }
    for (int s = 0; s < nst; ++s) {
      if (s + 1 < nst) {
        da.copy(a_org(kb + (s + 1) * BK), As[(s + 1) & 1], wave, lane);
        db.copy(b_org(kb + (s + 1) * BK), Bs[(s + 1) & 1], wave, lane);
      }
      compute(s & 1);
      __syncthreads();
    }
  } else {
    if (nst > 0) {
      load_stage(kb, ra0, rb0);
      if (nst > 1) load_stage(kb + BK, ra1, rb1);
      store_stage(0, ra0, rb0);
      __syncthreads();
    }
    int s = 0;
    for (; s + 1 < nst; s += 2) {
      step(s, ra0, rb0, ra1, rb1);       // even stage: loads s + 2 into set 0, stores set 1 (stage s + 1)
      step(s + 1, ra1, rb1, ra0, rb0);   // odd stage: loads s + 3 into set 1, stores set 0 (stage s + 2)
    }
    if (s < nst) step(s, ra0, rb0, ra1, rb1);
  }

  // Accumulator layout of a 32 x 32 block: register e of lane (h, r) holds
  // row 8 (e / 4) + 4 h + (e % 4), column r.
  if constexpr (std::is_same_v<Epi, EpiSplitUpdate>) {
    // The block's partial (slot (i TN + j) 4 + q of a wave = registers 4 q
    // .. 4 q + 3 of block (i, j)), its arrival, and in the last block of the
    // tile the ordered sum of the splits and the update.
    constexpr int kSlots = T::TM * T::TN * 4;
    const int tile = tm * tiles_n + tn;
    const int zstride = tiles_m * tiles_n * BM * BN * 4;
    const __amdgpu_buffer_rsrc_t pr = partial_rsrc(epi.P + (size_t)tile * BM * BN + wave * kSlots * 256);
    const int z = blockIdx.z;
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
      for (int j = 0; j < T::TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          __builtin_amdgcn_raw_buffer_store_b128(v, pr, z * zstride + (((i * T::TN + j) * 4 + q) * 64 + lane) * 16, 0,
                                                 kCoherent);
        }
    if (!split_arrive(epi, tile)) return;
    int nf = 0;
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
      for (int j = 0; j < T::TN; ++j) {
        const int n = n0 + wn0 + j * 32 + r, nc = min(n, N - 1);
        float vo[16], wo[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const size_t idx = (size_t)min(m0 + wm0 + i * 32 + 8 * (e >> 2) + 4 * h + (e & 3), M - 1) * epi.ldw + nc;
          vo[e] = epi.V[idx];
          wo[e] = epi.W[idx];
        }
        f32x4 own[4], g[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          own[q] = f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        ordered_split_sum<4, (BM == 64 && BN == 64) ? 8 : 1>(g, own, pr, zstride, (i * T::TN + j) * 4, lane, z,
                                                              epi.splits);
        if (n < N) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int m = m0 + wm0 + i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
            if (m < M) {
              const size_t idx = (size_t)m * epi.ldw + n;
              const float v = momentum_step(checked_change(g[e >> 2][e & 3], epi.limit, nf), vo[e], epi.lr, epi.mom);
              epi.V[idx] = v;
              epi.W[idx] = wo[e] + v;
            }
          }
        }
      }
    if (epi.limit > 0.f) add_faults(nf, epi.faults);
  } else {
    // Row epilogue of full 128 x 128 and 256 x 256 tiles for the sigmoid and
    // hidden-delta products, 128 rows at a time: the accumulators of those
    // rows go to LDS (the idle stage buffers, rows 0-63 in As and 64-127 in
    // Bs, row stride BN + 8 floats: the two lane halves of a register write
    // land 32 banks apart), then each thread takes 4 adjacent columns of 16
    // rows (rows t / (BN / 4) + 8 i) as float4: one 16-byte load of the
    // operand and one 16-byte store per row instead of four 4-byte ones, every
    // wave instruction covering whole cache lines.
    constexpr bool kRowEpi = (std::is_same_v<Epi, EpiSigmoid> || std::is_same_v<Epi, EpiHiddenDelta>) &&
                             ((BM == 128 && BN == 128) || (BM == 256 && BN == 256));
    if constexpr (kRowEpi) {
      constexpr int RS = BN + 8, C4N = BN / 4, SL = NTH / C4N;   // row stride; float4 per row; row slices
      static_assert(SL == 8 && 64 * RS <= 2 * T::A_ELEMS && 64 * RS <= 2 * T::B_ELEMS,
                    "row epilogue fits the stage buffers");
      bool vec = m0 + BM <= M && n0 + BN <= N && (epi.ldo & 3) == 0 && (reinterpret_cast<uintptr_t>(epi.out) & 15) == 0;
      if constexpr (std::is_same_v<Epi, EpiHiddenDelta>)
        vec = vec && (epi.lda & 3) == 0 && (reinterpret_cast<uintptr_t>(epi.act) & 15) == 0;
      if (NTH != kThreads || vec) {
        float* lo = &As[0][0];
        float* hi = &Bs[0][0];
        const int c4 = tid % C4N, r0 = tid / C4N;
        const int n = n0 + 4 * c4;
        f32x4 b4 = {0.f, 0.f, 0.f, 0.f};
        if constexpr (std::is_same_v<Epi, EpiSigmoid>)
          b4 = f32x4{epi.bias[n], epi.bias[n + 1], epi.bias[n + 2], epi.bias[n + 3]};
#pragma unroll
        for (int hf = 0; hf < BM / 128; ++hf) {
          if (hf > 0) __syncthreads();                     // the previous half is read
          // a wave's rows lie in one half (WM <= 128); rb is their first row
          // within it, a multiple of 64, so the buffer of each 32-row block
          // is wave-uniform
          const int rb = wm0 - 128 * hf;
          if (rb >= 0 && rb < 128) {
#pragma unroll
            for (int i = 0; i < T::TM; ++i) {
              float* dst = (rb + i * 32 < 64 ? lo : hi) + ((rb + i * 32) & 63) * RS + wn0 + r;
#pragma unroll
              for (int j = 0; j < T::TN; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) dst[(8 * (e >> 2) + 4 * h + (e & 3)) * RS + j * 32] = acc[i][j][e];
            }
          }
          __syncthreads();
          f32x4 cs[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
          for (int g = 0; g < 2; ++g) {
            const int mg = m0 + 128 * hf + 64 * g;
            f32x4 pre[8];
            if constexpr (std::is_same_v<Epi, EpiHiddenDelta>) {
#pragma unroll
              for (int i = 0; i < 8; ++i)
                pre[i] = *reinterpret_cast<const f32x4*>(epi.act + (size_t)(mg + r0 + 8 * i) * epi.lda + n);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              const int row = r0 + 8 * i;
              const f32x4 a = *reinterpret_cast<const f32x4*>((g ? hi : lo) + row * RS + 4 * c4);
              f32x4 v;
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                if constexpr (std::is_same_v<Epi, EpiSigmoid>)
                  v[q] = unit_sigma(a[q] + b4[q], epi.tab);
                else
                  v[q] = a[q] * (pre[i][q] * (1.0f - pre[i][q]));
              }
              *reinterpret_cast<f32x4*>(epi.out + (size_t)(mg + row) * epi.ldo + n) = v;
              if constexpr (Epi::kColSum) cs[g] += v;
            }
          }
          if constexpr (Epi::kColSum) {
            // per 64-row group: the 8 row slices (r0) of each column added in
            // slice order
            __syncthreads();
            f32x4* red = reinterpret_cast<f32x4*>(lo);        // [2][8][C4N] float4
#pragma unroll
            for (int g = 0; g < 2; ++g) red[(g * 8 + r0) * C4N + c4] = cs[g];
            __syncthreads();
            if (tid < 2 * C4N) {
              const int g = tid / C4N, cc = tid % C4N;
              f32x4 t = red[(g * 8) * C4N + cc];
              for (int k = 1; k < 8; ++k) t += red[(g * 8 + k) * C4N + cc];
              *reinterpret_cast<f32x4*>(epi.colsum + (size_t)(tm * (BM / 64) + 2 * hf + g) * epi.ldcs + n0 + 4 * cc) =
                  t;
            }
          }
        }
        return;
      }
    }
    if constexpr (NTH == kThreads) {
    float sse = 0.f;   // the epilogue's per-lane statistic (error, or fault count: exact below 2^24)
    // The per-element operands of each 32 x 32 block are loaded together
    // (clamped, always valid addresses; values outside the matrix are never
    // used) before the block's stores: one memory round trip per block, with
    // few extra registers.
    float csum[T::TN];
#pragma unroll
    for (int j = 0; j < T::TN; ++j) {
      csum[j] = 0.f;
      const int n = n0 + wn0 + j * 32 + r;
      if (n < N) {
        const float cv = epi.column(n);
#pragma unroll
        for (int i = 0; i < T::TM; ++i) {
          typename Epi::Pre pre[16];
#pragma unroll
          for (int e = 0; e < 16; ++e)
            pre[e] = epi.load(min(m0 + wm0 + i * 32 + 8 * (e >> 2) + 4 * h + (e & 3), M - 1), n);
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int m = m0 + wm0 + i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
            if (m < M) csum[j] += epi.apply(m, n, acc[i][j][e], cv, pre[e], sse);
          }
        }
      }
    }
    if constexpr (Epi::kColSum) {
      // Column sums per 64-row group of the tile (a 128-row tile has two, one
      // per wave row; a 64-row tile one, over both wave rows).  Lanes h = 0, 1
      // hold the same column (different rows); the wave rows of a group are
      // then added in a fixed order.
      static_assert(BM == 64 || BM == 128, "column-sum groups assume 64- or 128-row tiles");
      constexpr int kGroups = BM / 64, kWaveRowsPerGroup = 2 / kGroups;
      __shared__ float cs[2][BN];
#pragma unroll
      for (int j = 0; j < T::TN; ++j) {
        const float v = csum[j] + __shfl_xor(csum[j], 32, 64);
        if (h == 0) cs[wave >> 1][wn0 + j * 32 + r] = v;
      }
      __syncthreads();
#pragma unroll
      for (int g = 0; g < kGroups; ++g) {
        const int crow = tm * kGroups + g;
        if (crow * 64 >= M) break;
        for (int c = threadIdx.x; c < BN; c += kThreads) {
          if (n0 + c >= N) continue;
          float v = cs[g * kWaveRowsPerGroup][c];
          for (int w = 1; w < kWaveRowsPerGroup; ++w) v += cs[g * kWaveRowsPerGroup + w][c];
          epi.colsum[(size_t)crow * epi.ldcs + n0 + c] = v;
        }
      }
    }
    if constexpr (Epi::kFaults) {
      if (epi.limit > 0.f) add_faults((int)sse, epi.faults);
    }
    if constexpr (Epi::kSSE) {
      __shared__ float red[kThreads / 64];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) sse += __shfl_xor(sse, off, 64);
      if (lane == 0) red[wave] = sse;
      __syncthreads();
      if (threadIdx.x == 0) {
        double s = 0.0;
        for (int w = 0; w < kThreads / 64; ++w) s += (double)red[w];
        epi.sse_part[blockIdx.x] = s;
      }
    }
    }
  }
}

// Tile configurations: 128 x 128 x 32 (wave tile 64 x 64, two blocks per
// CU, 72 KB of LDS with both buffers) for products with at least one tile
// per CU or deep enough in K for split-K to fill the chip, 128 x 64 among
// those when N <= 64 (half of a 128-wide tile would be empty columns);
// 64 x 64 x 32 (wave tile 32 x 32) for the other, small products, which
// gives them four times the blocks (and wastes less of an edge tile).  (A
// 256 x 128 x 16 tile, one block per CU round for more products, measured
// slower on the wide and deep nets.)
constexpr int kTileK = 32;
constexpr int kChunkAlign = kTileK;   // split-K chunks are multiples of BK
constexpr int kCUs = 256;

inline int tiles_of(int M, int N, int t) { return ((M + t - 1) / t) * ((N + t - 1) / t); }
// Edge of the square tile an M x N product summed over K uses.
inline int tile_edge(int M, int N, int K) { return (tiles_of(M, N, 128) >= kCUs || K >= 1024) ? 128 : 64; }
// Column edge of that tile.
inline int tile_cols(int M, int N, int K) {
  const int t = tile_edge(M, N, K);
  return t == 128 && N <= 64 ? 64 : t;
}
inline int tile_count(int M, int N, int K) {
  const int bm = tile_edge(M, N, K), bn = tile_cols(M, N, K);
  return ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
}

template <int BM, int BN, int BK, bool A_KM, bool B_NK, class Epi>
hipError_t launch_gemm(hipStream_t s, const float* A, int lda, const float* B, int ldb, int M, int N, int K,
                       int splits, int k_chunk, const Epi& epi) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const bool avec = (lda % 4 == 0) && ((reinterpret_cast<uintptr_t>(A) & 15) == 0);
  const bool bvec = (ldb % 4 == 0) && ((reinterpret_cast<uintptr_t>(B) & 15) == 0);
  dim3 grid(tiles, 1, splits), block(kThreads);
  if (avec && bvec)
    return launch_kernel(gemm_kernel<BM, BN, BK, A_KM, B_NK, true, true, Epi>, grid, block, 0, s, A, lda, B, ldb, M,
                         N, K, k_chunk, epi);
  if (avec)
    return launch_kernel(gemm_kernel<BM, BN, BK, A_KM, B_NK, true, false, Epi>, grid, block, 0, s, A, lda, B, ldb, M,
                         N, K, k_chunk, epi);
  if (bvec)
    return launch_kernel(gemm_kernel<BM, BN, BK, A_KM, B_NK, false, true, Epi>, grid, block, 0, s, A, lda, B, ldb, M,
                         N, K, k_chunk, epi);
  return launch_kernel(gemm_kernel<BM, BN, BK, A_KM, B_NK, false, false, Epi>, grid, block, 0, s, A, lda, B, ldb, M, N,
                       K, k_chunk, epi);
}

template <bool A_KM, bool B_NK, class Epi>
hipError_t launch_cfg(hipStream_t s, const float* A, int lda, const float* B, int ldb, int M, int N, int K, int splits,
                      int k_chunk, const Epi& epi) {
  if (tile_edge(M, N, K) == 128) {
    if (tile_cols(M, N, K) == 64)
      return launch_gemm<128, 64, kTileK, A_KM, B_NK>(s, A, lda, B, ldb, M, N, K, splits, k_chunk, epi);
    return launch_gemm<128, 128, kTileK, A_KM, B_NK>(s, A, lda, B, ldb, M, N, K, splits, k_chunk, epi);
  }
  return launch_gemm<64, 64, kTileK, A_KM, B_NK>(s, A, lda, B, ldb, M, N, K, splits, k_chunk, epi);
}

// --------------------------------------------------------------------------
// Products with few output tiles (an Elman net's per-step layers: M = the
// sequence streams, N = the layer, K = the layer below).  A 64 x 64 tile grid
// would keep a fraction of the CUs busy, each wave with a long chain of
// dependent loads and MFMAs.  Here a block owns RB 32 x 32 MFMA blocks of
// one 32-column strip (a 32 RB-row tile) and splits K over four wave groups:
// wave w works on row block w % RB and K group w / RB.  K is cut into four
// ranges of KC = 2 KH values, KH a multiple of 16; within a range, MFMA step
// i pairs k = k0 + i (lanes 0-31) with k = k0 + KH + i (lanes 32-63), so that
// each lane reads its A row (and its B row when B is stored [n][k])
// contiguously.  Each lane loads its operands straight from global memory,
// 16 steps at a time with the next 32 in flight.  The four K partials of a
// row block are added through LDS in K order, and the four waves of the row
// block share its epilogue (RB = 2 for epilogues with 64-row column sums).
//
// With EpiSplitUpdate the kernel is a split-K change product (section
// 6.2.1, the batch-summed change of one layer's weights when the batch is
// long and the layer small): A is stored k-major (A[k][m], the activations),
// the block covers K range [z k_chunk, (z + 1) k_chunk) of split z and
// stores its partial sums; the last block of each tile adds them in split
// order and applies the update (EpiSplitUpdate).  Blocks are ordered split-major and handed to
// the XCDs in contiguous ranges, so each XCD reads one K range of both
// operands.
//
// With CTX, A is the input of an Elman step built on the fly (section 10.5):
// A[m][k] = X[m][k] for k < n_ext, cont[m] H[m][k - n_ext] for the context
// units, H being the previous step's first hidden layer (the context copies
// its units in order).  The blocks of the first column strip also write the
// rows they built to `out` (zeros in [K, ldo)), which the window's change
// product reads.
constexpr int kSkinnyChunk = 16;   // MFMA steps per load round

// 256 x 256 tiles of 512 threads (one block per CU) for products made of at
// least one full such tile per CU: one round of blocks instead of two rounds
// of 128 x 128 tiles, so one prologue and one epilogue per CU and no second
// round starting behind the first round's slowest blocks.
inline bool big_tiles(int M, int N, int K) {
  return M % 256 == 0 && N % 256 == 0 && K % kTileK == 0 && K > 0 && tiles_of(M, N, 256) >= kCUs;
}
inline bool vec16(const void* p, int ld) { return (ld & 3) == 0 && (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

inline bool use_skinny(int M, int N, int K) { return K <= 2048 && tiles_of(M, N, 64) < 128; }

struct CtxInput {
  const float* H = nullptr;   // previous step's hidden rows [M][ldh]
  int ldh = 0;
  const float* cont = nullptr;
  int n_ext = 0;              // X = A, rows [M][lda]
  float* out = nullptr;       // built rows [M][ldo], or nullptr
  int ldo = 0;
};

// The work of block `bid` of `nblocks` (a kernel may give a range of its
// blocks to each of several products); `part` is the block's LDS for the K
// partials.
template <int RB, bool A_KM, bool B_NK, bool AVEC, bool BVEC, bool CTX, class Epi>
__device__ __forceinline__ void skinny_body(int bid, int nblocks, float (&part)[4][RB][16][64],
                                            const float* __restrict__ A, int lda, const float* __restrict__ B,
                                            int ldb, int M, int N, int K, int k_chunk, const Epi& epi,
                                            const CtxInput& ctx) {
  constexpr bool SPLIT = std::is_same_v<Epi, EpiSplitUpdate>;
  static_assert(!Epi::kFaults || SPLIT, "unsplit update epilogues take gemm_kernel");
  static_assert(!Epi::kColSum || RB == 2, "64-row column sums need RB = 2");
  static_assert(!A_KM || (SPLIT && !AVEC && !CTX), "k-major A is the change product's");
  constexpr int C = kSkinnyChunk;
  const int tiles_m = (M + 32 * RB - 1) / (32 * RB), tiles_n = (N + 31) / 32;
  int tm, tn, z = 0;
  if constexpr (SPLIT) {
    const int per = nblocks >> 3;
    const int t = bid >= (per << 3) ? bid : (bid & 7) * per + (bid >> 3);
    const int tiles = tiles_m * tiles_n;
    z = t / tiles;
    tm = (t - z * tiles) / tiles_n;
    tn = t - z * tiles - tm * tiles_n;
  } else {
    xcd_tile(bid, nblocks, tiles_m, tiles_n, tm, tn);
  }
  const int kstart = z * k_chunk, kend = min(K, kstart + k_chunk);
  const int m0 = tm * 32 * RB, n0 = tn * 32;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rb = wave % RB, kg = wave / RB;
  const int r = lane & 31, h = lane >> 5;
  const int kh = ((kend - kstart + 7) / 8 + C - 1) / C * C;   // KH
  const int kbase = kstart + kg * 2 * kh + h * kh;            // this lane's first k
  const int m = m0 + rb * 32 + r, n = n0 + r;        // A row and B column of this lane
  const int mc = min(m, M - 1), nc = min(n, N - 1);
  const float* arow = A + (size_t)mc * lda;
  const float* hrow = CTX ? ctx.H + (size_t)mc * ctx.ldh : nullptr;
  const float cm = CTX ? ctx.cont[mc] : 1.f;
  const bool store_rows = CTX && ctx.out && tn == 0 && m < M;

  // operands of MFMA steps c C .. c C + C - 1 (zero past K, M or N).  Every
  // load reads a clamped, valid address and is issued before any mask is
  // applied; masks are bitwise ANDs, so the compiler has no branch to sink a
  // load into (a load sunk behind a predicate waits for itself) and masked
  // elements are exact zeros.
  const int mrow = m < M ? -1 : 0, ncol = n < N ? -1 : 0;
  auto masked = [](float v, int keep) { return __builtin_bit_cast(float, __builtin_bit_cast(int, v) & keep); };
  auto load = [&](int c, float* a, float* b) {
    const int k0 = kbase + c * C;
    if (CTX && AVEC) {
      // n_ext % 4 == 0: each 4-vector lies in X or in H
      f32x4 v[C / 4];
#pragma unroll
      for (int q = 0; q < C / 4; ++q) {
        const int k = k0 + 4 * q;
        const float* p = k < ctx.n_ext ? arow + k : hrow + min(k - ctx.n_ext, ctx.ldh - 4);
        v[q] = *reinterpret_cast<const f32x4*>(p);
      }
#pragma unroll
      for (int q = 0; q < C / 4; ++q) {
        const float sc = k0 + 4 * q < ctx.n_ext ? 1.f : cm;
#pragma unroll
        for (int e = 0; e < 4; ++e) a[4 * q + e] = masked(v[q][e] * sc, k0 + 4 * q + e < kend ? mrow : 0);
      }
    } else if (CTX) {
#pragma unroll
      for (int i = 0; i < C; ++i) {
        const int k = k0 + i;
        const float* p = k < ctx.n_ext ? arow + k : hrow + min(k - ctx.n_ext, ctx.ldh - 1);
        a[i] = *p;
      }
#pragma unroll
      for (int i = 0; i < C; ++i) a[i] = masked(a[i] * (k0 + i < ctx.n_ext ? 1.f : cm), k0 + i < kend ? mrow : 0);
    } else if (A_KM) {
#pragma unroll
      for (int i = 0; i < C; ++i) a[i] = A[(size_t)min(k0 + i, K - 1) * lda + mc];
#pragma unroll
      for (int i = 0; i < C; ++i) a[i] = masked(a[i], k0 + i < kend ? mrow : 0);
    } else if (AVEC) {
      f32x4 v[C / 4];
#pragma unroll
      for (int q = 0; q < C / 4; ++q) v[q] = *reinterpret_cast<const f32x4*>(arow + min(k0 + 4 * q, lda - 4));
#pragma unroll
      for (int q = 0; q < C / 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) a[4 * q + e] = masked(v[q][e], k0 + 4 * q + e < kend ? mrow : 0);
    } else {
#pragma unroll
      for (int i = 0; i < C; ++i) a[i] = arow[min(k0 + i, K - 1)];
#pragma unroll
      for (int i = 0; i < C; ++i) a[i] = masked(a[i], k0 + i < kend ? mrow : 0);
    }
    if (B_NK && BVEC) {
      const float* brow = B + (size_t)nc * ldb;
      f32x4 v[C / 4];
#pragma unroll
      for (int q = 0; q < C / 4; ++q) v[q] = *reinterpret_cast<const f32x4*>(brow + min(k0 + 4 * q, ldb - 4));
#pragma unroll
      for (int q = 0; q < C / 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) b[4 * q + e] = masked(v[q][e], k0 + 4 * q + e < kend ? ncol : 0);
    } else {
#pragma unroll
      for (int i = 0; i < C; ++i)
        b[i] = B_NK ? B[(size_t)nc * ldb + min(k0 + i, K - 1)] : B[(size_t)min(k0 + i, K - 1) * ldb + nc];
#pragma unroll
      for (int i = 0; i < C; ++i) b[i] = masked(b[i], k0 + i < kend ? ncol : 0);
    }
  };

  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
  // three register sets: chunks c + 1 and c + 2 are in flight while chunk c
  // is multiplied (up to three chunks, K <= 384, all loads precede the first
  // MFMA)
  const int nchunk = kh / C;
  float a0[C], b0[C], a1[C], b1[C], a2[C], b2[C];
  auto mfma = [&](int c, const float* a, const float* b) {
    if (store_rows) {
      // the built row segment, once the chunk's operands are in registers
      const int k0 = kbase + c * C;
      float* o = ctx.out + (size_t)m * ctx.ldo + k0;
      if (AVEC) {
#pragma unroll
        for (int q = 0; q < C / 4; ++q)
          if (k0 + 4 * q < ctx.ldo)
            *reinterpret_cast<f32x4*>(o + 4 * q) = f32x4{a[4 * q], a[4 * q + 1], a[4 * q + 2], a[4 * q + 3]};
      } else {
#pragma unroll
        for (int i = 0; i < C; ++i)
          if (k0 + i < ctx.ldo) o[i] = a[i];
      }
    }
#pragma unroll
    for (int i = 0; i < C; ++i) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[i], acc, 0, 0, 0);
  };
  if (nchunk > 0) load(0, a0, b0);
  if (nchunk > 1) load(1, a1, b1);
  for (int c = 0; c < nchunk; c += 3) {
    if (c + 2 < nchunk) load(c + 2, a2, b2);
    mfma(c, a0, b0);
    if (c + 1 >= nchunk) break;
    if (c + 3 < nchunk) load(c + 3, a0, b0);
    mfma(c + 1, a1, b1);
    if (c + 2 >= nchunk) break;
    if (c + 4 < nchunk) load(c + 4, a1, b1);
    mfma(c + 2, a2, b2);
  }

  // The K partials go through LDS; wave (rb, kg) then adds, in K-group
  // order, registers 4 kg .. 4 kg + 3 of its row block (rows 8 kg + 4 h + q
  // of the 32 x 32 block: register e of lane (h, r) holds row 8 (e / 4) +
  // 4 h + (e % 4), column r) and applies the epilogue to them, so that all
  // waves share the epilogue.
#pragma unroll
  for (int e = 0; e < 16; ++e) part[kg][rb][e][lane] = acc[e];
  __syncthreads();
  if constexpr (SPLIT) {
    // One 4-float slot per thread (slot = wave): rows 8 kg + 4 h + q of row
    // block rb, column n.  Then the arrival, and in the last block of the
    // tile the ordered sum of the splits and the update.
    f32x4 own[1], g[1];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * kg + q;
      own[0][q] = ((part[0][rb][e][lane] + part[1][rb][e][lane]) + part[2][rb][e][lane]) + part[3][rb][e][lane];
    }
    const int tile = tm * tiles_n + tn;
    const int zstride = tiles_m * tiles_n * 32 * RB * 32 * 4;
    const __amdgpu_buffer_rsrc_t pr = partial_rsrc(epi.P + (size_t)tile * 32 * RB * 32);
    __builtin_amdgcn_raw_buffer_store_b128(own[0], pr, z * zstride + (wave * 64 + lane) * 16, 0, kCoherent);
    if (!split_arrive(epi, tile)) return;
    const int nc = min(n, N - 1);
    float vo[4], wo[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const size_t idx = (size_t)min(m0 + rb * 32 + 8 * kg + 4 * h + q, M - 1) * epi.ldw + nc;
      vo[q] = epi.V[idx];
      wo[q] = epi.W[idx];
    }
    ordered_split_sum<1>(g, own, pr, zstride, wave, lane, z, epi.splits);
    int nf = 0;
    if (n < N) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int mm = m0 + rb * 32 + 8 * kg + 4 * h + q;
        if (mm < M) {
          const size_t idx = (size_t)mm * epi.ldw + n;
          const float v = momentum_step(checked_change(g[0][q], epi.limit, nf), vo[q], epi.lr, epi.mom);
          epi.V[idx] = v;
          epi.W[idx] = wo[q] + v;
        }
      }
    }
    if (epi.limit > 0.f) add_faults(nf, epi.faults);
  } else {
    float sse = 0.f, csum = 0.f;
    if (n < N) {
      const float cv = epi.column(n);
      float v[4];
      typename Epi::Pre pre[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = 4 * kg + q;
        v[q] = ((part[0][rb][e][lane] + part[1][rb][e][lane]) + part[2][rb][e][lane]) + part[3][rb][e][lane];
        pre[q] = epi.load(min(m0 + rb * 32 + 8 * kg + 4 * h + q, M - 1), n);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int mm = m0 + rb * 32 + 8 * kg + 4 * h + q;
        if (mm < M) csum += epi.apply(mm, n, v[q], cv, pre[q], sse);
      }
    }
    if constexpr (Epi::kColSum) {
      // the 64-row tile's column sums: per wave over its 8 rows (lanes h = 0,
      // 1 hold the same column), then the waves in (row block, K group) order
      __shared__ float cs[2][4][32];
      const float v = csum + __shfl_xor(csum, 32, 64);
      if (h == 0) cs[rb][kg][r] = v;
      __syncthreads();
      if (threadIdx.x < 32 && n0 + (int)threadIdx.x < N) {
        float t = 0.f;
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
          for (int g = 0; g < 4; ++g) t += cs[b2][g][threadIdx.x];
        epi.colsum[(size_t)tm * epi.ldcs + n0 + threadIdx.x] = t;
      }
    }
    if constexpr (Epi::kSSE) {
      __shared__ float red[4 * RB];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) sse += __shfl_xor(sse, off, 64);
      if (lane == 0) red[wave] = sse;
      __syncthreads();
      if (threadIdx.x == 0) {
        double s = 0.0;
        for (int w = 0; w < 4 * RB; ++w) s += (double)red[w];
        epi.sse_part[bid] = s;
      }
    }
  }
}

template <int RB, bool A_KM, bool B_NK, bool AVEC, bool BVEC, bool CTX, class Epi>
__global__ __launch_bounds__(256 * RB) void skinny_kernel(const float* __restrict__ A, int lda,
                                                          const float* __restrict__ B, int ldb, int M, int N,
                                                          int K, int k_chunk, Epi epi, CtxInput ctx) {
  __shared__ float part[4][RB][16][64];
  skinny_body<RB, A_KM, B_NK, AVEC, BVEC, CTX>(blockIdx.x, gridDim.x, part, A, lda, B, ldb, M, N, K, k_chunk, epi,
                                               ctx);
}

// Two independent products of an Elman net with one hidden layer in one
// launch (section 10.5): the hidden layer of step t + 1 (input built in the
// product) and the output layer of step t with its deltas, which both read
// step t's hidden rows and nothing the other writes.  Blocks [0, nh) take
// the first, the rest the second; 64 x 32 tiles for both.
template <bool AVEC_H, bool AVEC_O>
__global__ __launch_bounds__(512) void elman_pair_kernel(const float* __restrict__ X, int n_ext,
                                                         const float* __restrict__ W0, int ldw0, int n0, int n1,
                                                         EpiSigmoid eh, CtxInput ctx,
                                                         const float* __restrict__ H, int ldh,
                                                         const float* __restrict__ W1, int ldw1, int n2,
                                                         EpiOutputDelta eo, int S, int nh) {
  __shared__ float part[4][2][16][64];
  if ((int)blockIdx.x < nh)
    skinny_body<2, false, false, AVEC_H, false, true>(blockIdx.x, nh, part, X, n_ext, W0, ldw0, S, n1, n0, n0, eh,
                                                      ctx);
  else
    skinny_body<2, false, false, AVEC_O, false, false>(blockIdx.x - nh, gridDim.x - nh, part, H, ldh, W1, ldw1, S, n2,
                                                       n1, n1, eo, CtxInput{});
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <int RB, bool B_NK, class Epi>
hipError_t launch_skinny(hipStream_t s, const float* A, int lda, const float* B, int ldb, int M, int N, int K,
                         const Epi& epi) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const int tiles = ((M + 32 * RB - 1) / (32 * RB)) * ((N + 31) / 32);
  const bool avec = (lda % 4 == 0) && aligned16(A);
  const bool bvec = B_NK && (ldb % 4 == 0) && aligned16(B);
  const CtxInput none{};
  if (avec && bvec)
    return launch_kernel(skinny_kernel<RB, false, B_NK, true, true, false, Epi>, tiles, 256 * RB, 0, s, A, lda, B, ldb,
                         M, N, K, K, epi, none);
  if (avec)
    return launch_kernel(skinny_kernel<RB, false, B_NK, true, false, false, Epi>, tiles, 256 * RB, 0, s, A, lda, B,
                         ldb, M, N, K, K, epi, none);
  if (bvec)
    return launch_kernel(skinny_kernel<RB, false, B_NK, false, true, false, Epi>, tiles, 256 * RB, 0, s, A, lda, B,
                         ldb, M, N, K, K, epi, none);
  return launch_kernel(skinny_kernel<RB, false, B_NK, false, false, false, Epi>, tiles, 256 * RB, 0, s, A, lda, B, ldb,
                       M, N, K, K, epi, none);
}

// Split-K output layer: sums the split partials in split order, then applies
// the output-delta epilogue (bias, sigma, e = T - y, delta = e y (1 - y)).
// Block (x, y) covers rows [128 x, 128 x + 128) and columns [64 y, 64 y + 64)
// with 16 waves; lane = column, wave w = rows 8 w .. 8 w + 7 (their loads
// issued together).  Writes the block's error partial and the 64-row column
// sums of the deltas (waves 0-7 and 8-15; the grouping of the fused
// epilogue), both in wave order.
constexpr int kFin = 1024;
__global__ __launch_bounds__(kFin) void output_finish_kernel(const float* __restrict__ P, int splits, size_t stride,
                                                             int ldp, int M, int N, const float* __restrict__ bias,
                                                             const float* __restrict__ T, int ldt, float* delta,
                                                             int ldd, double* sse_part, float* colsum, int ldcs,
                                                             const float* __restrict__ tab,
                                                             const float* __restrict__ mask) {
  constexpr int W = kFin / 64, R = 128 / W;
  __shared__ float cs[W][64];
  __shared__ float red[W];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = blockIdx.y * 64 + lane;
  const int m0 = blockIdx.x * 128 + wave * R;
  float sse = 0.f, csum = 0.f;
  if (n < N) {
    // rows are clamped to M - 1 so that every load is unconditional (all in
    // flight together); rows past M are never used
    const float b = bias[n];
    float z[R], t[R], mk[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int m = min(m0 + r, M - 1);
      z[r] = 0.f;
      t[r] = T[(size_t)m * ldt + n];
      mk[r] = mask ? mask[m] : 1.0f;
    }
    for (int sp = 0; sp < splits; ++sp) {
      float v[R];
#pragma unroll
      for (int r = 0; r < R; ++r) v[r] = P[sp * stride + (size_t)min(m0 + r, M - 1) * ldp + n];
#pragma unroll
      for (int r = 0; r < R; ++r) z[r] += v[r];
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (m0 + r >= M) break;
      const float y = unit_sigma(z[r] + b, tab);
      float e = t[r] - y;
      if (mask) e *= mk[r];
      sse += e * e;
      const float d = e * y * (1.0f - y);
      delta[(size_t)(m0 + r) * ldd + n] = d;
      csum += d;
    }
  }
  cs[wave][lane] = csum;
  for (int off = 32; off > 0; off >>= 1) sse += __shfl_xor(sse, off, 64);
  if (lane == 0) red[wave] = sse;
  __syncthreads();
  if (wave < 2 && n < N && blockIdx.x * 128 + wave * 64 < M) {
    constexpr int kHalf = W / 2;
    float c = cs[wave * kHalf][lane];
    for (int w = 1; w < kHalf; ++w) c += cs[wave * kHalf + w][lane];
    colsum[(size_t)(2 * blockIdx.x + wave) * ldcs + n] = c;
  }
  if (threadIdx.x == 0) {
    double tt = 0.0;
    for (int w = 0; w < W; ++w) tt += (double)red[w];
    sse_part[blockIdx.y * gridDim.x + blockIdx.x] = tt;
  }
}

// Bias-row changes of several layers in one launch: column sums of each
// layer's D over its `rows` rows, then the update.  Blocks [block0, next
// job's block0) take the job's 64-column strips.  Block = 1024 threads = 16
// waves; lane = column within a strip; wave w sums its contiguous share of
// the rows in order, then the 16 partial sums are added in wave order.
constexpr int kBiasWaves = 16;
__global__ __launch_bounds__(64 * kBiasWaves) void bias_update_kernel(BiasJobs jobs, float lr, float mom,
                                                                       float limit, unsigned long long* faults) {
  __shared__ float part[kBiasWaves][64];
  int q = 0;
  while (q + 1 < jobs.n && (int)blockIdx.x >= jobs.j[q + 1].block0) ++q;
  const float* __restrict__ D = jobs.j[q].D;
  float* Wb = jobs.j[q].Wb;
  float* Vb = jobs.j[q].Vb;
  const int ldd = jobs.j[q].ldd, rows = jobs.j[q].rows, N = jobs.j[q].N;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n = ((int)blockIdx.x - jobs.j[q].block0) * 64 + lane;
  const int r0 = (int)((int64_t)rows * wave / kBiasWaves), r1 = (int)((int64_t)rows * (wave + 1) / kBiasWaves);
  float s = 0.f;
  if (n < N) {
    int k = r0;
    for (; k + 4 <= r1; k += 4) {
      const float a0 = D[(size_t)k * ldd + n], a1 = D[(size_t)(k + 1) * ldd + n];
      const float a2 = D[(size_t)(k + 2) * ldd + n], a3 = D[(size_t)(k + 3) * ldd + n];
      s += a0;
      s += a1;
      s += a2;
      s += a3;
    }
    for (; k < r1; ++k) s += D[(size_t)k * ldd + n];
  }
  part[wave][lane] = s;
  __syncthreads();
  if (wave == 0) {
    int nf = 0;
    if (n < N) {
      float g = 0.f;
      for (int w = 0; w < kBiasWaves; ++w) g += part[w][lane];
      g = checked_change(g, limit, nf);
      const float v = momentum_step(g, Vb[n], lr, mom);
      Vb[n] = v;
      Wb[n] = Wb[n] + v;
    }
    if (limit > 0.f) add_faults(nf, faults);
  }
}

// One-hot first layer forward.  One wave per (pattern, 64-column strip).
__global__ __launch_bounds__(kThreads) void onehot_forward_kernel(const int32_t* __restrict__ act, int n_active,
                                                                  int rows, const float* __restrict__ W0, int ldw,
                                                                  int n0, int H, int strips, int mode, float* out,
                                                                  int ldo, const float* __restrict__ T, int ldt,
                                                                  double* sse_part, const float* __restrict__ tab) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int item = blockIdx.x * (kThreads / 64) + wave;
  const int p = item / strips, col = (item % strips) * 64 + lane;
  float sse = 0.f;
  if (p < rows && col < H) {
    float net = W0[(size_t)n0 * ldw + col];
    const int32_t* a = act + (size_t)p * n_active;
    for (int k = 0; k < n_active; ++k) {
      const int ix = a[k];   // an index outside [0, n0) selects no row
      if ((unsigned)ix < (unsigned)n0) net += W0[(size_t)ix * ldw + col];
    }
    const float y = unit_sigma(net, tab);
    if (mode == 0) {
      out[(size_t)p * ldo + col] = y;
    } else {
      const float e = T[(size_t)p * ldt + col] - y;
      sse = e * e;
      out[(size_t)p * ldo + col] = e * y * (1.0f - y);
    }
  }
  if (mode == 1) {
    __shared__ float red[kThreads / 64];
    for (int off = 32; off > 0; off >>= 1) sse += __shfl_xor(sse, off, 64);
    if (lane == 0) red[wave] = sse;
    __syncthreads();
    if (threadIdx.x == 0) {
      double s = 0.0;
      for (int w = 0; w < kThreads / 64; ++w) s += (double)red[w];
      sse_part[blockIdx.x] = s;
    }
  }
}

// One-hot first-layer change + update.  Block (r, c): weight row r (r == n0 is
// the bias row) and columns [256 c, 256 c + 256).  The patterns containing
// index r are listed in pattern order (ballot compaction, 256 patterns at a
// time) and their delta rows summed in that order.
__global__ __launch_bounds__(kThreads) void onehot_update_kernel(const int32_t* __restrict__ act, int n_active,
                                                                 int rows, const float* __restrict__ D, int ldd,
                                                                 int n0, int H, float* W, float* V, int ldw,
                                                                 float lr, float mom, float limit,
                                                                 unsigned long long* faults) {
  __shared__ int list[kThreads];
  __shared__ int wave_cnt[kThreads / 64];
  const int r = blockIdx.x;
  const int col = blockIdx.y * kThreads + threadIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float g = 0.f;
  for (int p0 = 0; p0 < rows; p0 += kThreads) {
    const int p = p0 + threadIdx.x;
    bool hit = false;
    if (p < rows) {
      if (r == n0) {
        hit = true;
      } else {
        const int32_t* a = act + (size_t)p * n_active;
        for (int k = 0; k < n_active; ++k) hit |= (a[k] == r);
      }
    }
    const unsigned long long bal = __ballot(hit);
    if (lane == 0) wave_cnt[wave] = __popcll(bal);
    __syncthreads();
    int base = 0, total = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      if (w < wave) base += wave_cnt[w];
      total += wave_cnt[w];
    }
    if (hit) {
      const unsigned long long below = lane ? (bal & ((1ull << lane) - 1ull)) : 0ull;
      list[base + __popcll(below)] = p;
    }
    __syncthreads();
    if (col < H)
      for (int q = 0; q < total; ++q) g += D[(size_t)list[q] * ldd + col];
    __syncthreads();
  }
  int nf = 0;
  if (col < H) {
    g = checked_change(g, limit, nf);
    const size_t i = (size_t)r * ldw + col;
    const float v = momentum_step(g, V[i], lr, mom);
    V[i] = v;
    W[i] = W[i] + v;
  }
  if (limit > 0.f) add_faults(nf, faults);
}

// Zero fill of n ints (counters that must start at zero, in work a caller
// may capture into a graph, where a memset node is avoided).
__global__ __launch_bounds__(kThreads) void zero_ints_kernel(int* p, int n) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Fixed-order sum of n doubles by one block of 1024 threads: thread t adds
// elements t, t + 1024, ... (loads issued eight at a time), then a tree.
constexpr int kRed = 1024;
__global__ __launch_bounds__(kRed) void sse_reduce_kernel(const double* __restrict__ part, int n, double* out) {
  __shared__ double red[kRed];
  block_sum_partials<kRed>(part, n, out, red);
}

// K-splits for a product with few output tiles: enough blocks for two per
// CU (512), each split at least 256 deep in K.
int choose_splits(int M, int N, int K) {
  const int tiles = tile_count(M, N, K);
  if (K < 1024 || tiles >= 512) return 1;
  int s = (512 + tiles - 1) / tiles;
  const int max_s = K / 256;
  if (s > max_s) s = max_s;
  return s < 1 ? 1 : s;
}

int choose_output_splits(int M, int N, int K) { return use_skinny(M, N, K) ? 1 : choose_splits(M, N, K); }

int chunk_for(int K, int splits) {
  int c = (K + splits - 1) / splits;
  return (c + kChunkAlign - 1) / kChunkAlign * kChunkAlign;
}

}  // namespace

// --------------------------------------------------------------------------
// Launch wrappers (declared in bp_internal.h).

LaunchEvents& launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}

int colsum_rows(int M) { return (M + 63) / 64; }

int output_delta_blocks(int M, int N, int K) {
  if (use_skinny(M, N, K)) return ((M + 63) / 64) * ((N + 31) / 32);
  if (choose_output_splits(M, N, K) > 1) return ((M + 127) / 128) * ((N + 63) / 64);
  return tile_count(M, N, K);
}

size_t output_delta_workspace(int M, int N, int K) {
  const int sp = choose_output_splits(M, N, K);
  if (sp <= 1) return 0;
  return (size_t)sp * M * ((N + 3) / 4 * 4);
}

int output_delta_splits(int M, int N, int K) { return choose_output_splits(M, N, K); }

hipError_t forward_layer(hipStream_t s, const float* A, int lda, const float* W, int ldw, int M, int N, int K,
                         const float* bias, float* out, int ldo, const float* tab) {
  EpiSigmoid e{bias, out, ldo, tab};
  if (use_skinny(M, N, K)) return launch_skinny<1, false>(s, A, lda, W, ldw, M, N, K, e);
  if (big_tiles(M, N, K) && vec16(A, lda) && vec16(W, ldw) && vec16(out, ldo))
    return launch_kernel(gemm_kernel<256, 256, kTileK, false, false, true, true, EpiSigmoid, 2 * kThreads>,
                         tiles_of(M, N, 256), 2 * kThreads, 0, s, A, lda, W, ldw, M, N, K, K, e);
  return launch_cfg<false, false>(s, A, lda, W, ldw, M, N, K, 1, K, e);
}

bool forward_ctx_fits(int M, int N, int K) { return use_skinny(M, N, K); }

hipError_t forward_ctx_layer(hipStream_t s, const float* X, int n_ext, const float* H, int ldh, const float* cont,
                             const float* W, int ldw, int M, int N, int K, const float* bias, float* out, int ldo,
                             float* rows_out, int ld_rows, const float* tab) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (!use_skinny(M, N, K) || !H || !cont || n_ext < 0 || n_ext > K || (n_ext > 0 && !X) ||
      ldh < K - n_ext || (rows_out && ld_rows < K))
    return hipErrorInvalidValue;
  EpiSigmoid e{bias, out, ldo, tab};
  const CtxInput ctx{H, ldh, cont, n_ext, rows_out, ld_rows};
  const float* A = n_ext > 0 ? X : H;   // X is not read when n_ext == 0
  const int tiles = ((M + 31) / 32) * ((N + 31) / 32);
  const bool avec = n_ext % 4 == 0 && aligned16(A) && ldh % 4 == 0 && aligned16(H) &&
                    (!rows_out || (ld_rows % 4 == 0 && aligned16(rows_out)));
  if (avec)
    return launch_kernel(skinny_kernel<1, false, false, true, false, true, EpiSigmoid>, tiles, 256, 0, s, A, n_ext, W,
                         ldw, M, N, K, K, e, ctx);
  return launch_kernel(skinny_kernel<1, false, false, false, false, true, EpiSigmoid>, tiles, 256, 0, s, A, n_ext, W,
                       ldw, M, N, K, K, e, ctx);
}

bool elman_pair_fits(int S, int n0, int n1, int n2) { return use_skinny(S, n1, n0) && use_skinny(S, n2, n1); }

hipError_t elman_pair(hipStream_t s, const float* X, int n_ext, const float* Hprev, const float* cont,
                      const float* W0, int ldw0, const float* bias0, int n0, int n1, float* Hnext, float* rows_out,
                      int ld_rows, const float* W1, int ldw1, const float* bias1, int n2, int ldh, int S,
                      const float* T, int ldt, float* delta, int ldd, double* sse_part, float* colsum, int ldcs,
                      const float* tab, const float* mask) {
  if (S <= 0 || n1 <= 0 || n2 <= 0) return hipSuccess;
  if (!elman_pair_fits(S, n0, n1, n2) || !Hprev || !cont || !Hnext || n_ext < 0 || n_ext > n0 ||
      (n_ext > 0 && !X) || ldh < n1 || (rows_out && ld_rows < n0))
    return hipErrorInvalidValue;
  const float* A = n_ext > 0 ? X : Hprev;   // X is not read when n_ext == 0
  EpiSigmoid eh{bias0, Hnext, ldh, tab};
  const CtxInput ctx{Hprev, ldh, cont, n_ext, rows_out, ld_rows};
  EpiOutputDelta eo{bias1, T, ldt, delta, ldd, sse_part, colsum, ldcs, tab, mask};
  const int nh = ((S + 63) / 64) * ((n1 + 31) / 32), no = ((S + 63) / 64) * ((n2 + 31) / 32);
  const bool avh = n_ext % 4 == 0 && aligned16(A) && ldh % 4 == 0 && aligned16(Hprev) &&
                   (!rows_out || (ld_rows % 4 == 0 && aligned16(rows_out)));
  const bool avo = ldh % 4 == 0 && aligned16(Hprev);
  if (avh && avo)
    return launch_kernel(elman_pair_kernel<true, true>, nh + no, 512, 0, s, A, n_ext, W0, ldw0, n0, n1, eh, ctx, Hprev,
                         ldh, W1, ldw1, n2, eo, S, nh);
  if (avh)
    return launch_kernel(elman_pair_kernel<true, false>, nh + no, 512, 0, s, A, n_ext, W0, ldw0, n0, n1, eh, ctx,
                         Hprev, ldh, W1, ldw1, n2, eo, S, nh);
  if (avo)
    return launch_kernel(elman_pair_kernel<false, true>, nh + no, 512, 0, s, A, n_ext, W0, ldw0, n0, n1, eh, ctx,
                         Hprev, ldh, W1, ldw1, n2, eo, S, nh);
  return launch_kernel(elman_pair_kernel<false, false>, nh + no, 512, 0, s, A, n_ext, W0, ldw0, n0, n1, eh, ctx, Hprev,
                       ldh, W1, ldw1, n2, eo, S, nh);
}

hipError_t forward_output_delta(hipStream_t s, const float* A, int lda, const float* W, int ldw, int M, int N, int K,
                                const float* bias, const float* T, int ldt, float* delta, int ldd, double* sse_part,
                                float* colsum, int ldcs, float* ws, const float* tab, const float* mask) {
  const int sp = choose_output_splits(M, N, K);
  if (sp <= 1) {
    EpiOutputDelta e{bias, T, ldt, delta, ldd, sse_part, colsum, ldcs, tab, mask};
    if (use_skinny(M, N, K)) return launch_skinny<2, false>(s, A, lda, W, ldw, M, N, K, e);
    return launch_cfg<false, false>(s, A, lda, W, ldw, M, N, K, 1, K, e);
  }
  const int ldp = (N + 3) / 4 * 4;
  EpiPartial e{ws, ldp, (size_t)M * ldp};
  return launch_cfg<false, false>(s, A, lda, W, ldw, M, N, K, sp, chunk_for(K, sp), e);
}

hipError_t output_finish(hipStream_t s, int M, int N, int K, const float* bias, const float* T, int ldt, float* delta,
                         int ldd, double* sse_part, float* colsum, int ldcs, const float* ws, const float* tab,
                         const float* mask) {
  const int sp = choose_output_splits(M, N, K);
  if (M <= 0 || N <= 0 || sp <= 1) return hipSuccess;
  const int ldp = (N + 3) / 4 * 4;
  dim3 grid((M + 127) / 128, (N + 63) / 64);
  return launch_kernel(output_finish_kernel, grid, kFin, 0, s, ws, sp, (size_t)M * ldp, ldp, M, N, bias, T, ldt,
                       delta, ldd, sse_part, colsum, ldcs, tab, mask);
}

hipError_t backward_layer(hipStream_t s, const float* D, int ldd, const float* W, int ldw, int M, int N, int K,
                          const float* act, int lda, float* out, int ldo, float* colsum, int ldcs) {
  EpiHiddenDelta e{act, lda, out, ldo, colsum, ldcs};
  if (use_skinny(M, N, K)) return launch_skinny<2, true>(s, D, ldd, W, ldw, M, N, K, e);
  if (big_tiles(M, N, K) && vec16(D, ldd) && vec16(W, ldw) && vec16(out, ldo) && vec16(act, lda))
    return launch_kernel(gemm_kernel<256, 256, kTileK, false, true, true, true, EpiHiddenDelta, 2 * kThreads>,
                         tiles_of(M, N, 256), 2 * kThreads, 0, s, D, ldd, W, ldw, M, N, K, K, e);
  return launch_cfg<false, true>(s, D, ldd, W, ldw, M, N, K, 1, K, e);
}

// The change product of a layer: few output tiles and a long batch take the
// split-K skinny kernel (64 x 32 tiles), with the largest K chunk of 1024,
// 512, 256 or 128 that still gives kSkinnyChangeBlocks blocks (one per CU:
// every block pays the arrival's round trips once); the others
// take gemm_kernel, split over K when the batch is long (choose_splits).
// Split products apply the update in the last block of each tile
// (EpiSplitUpdate); the others in every block's epilogue (EpiUpdate).
constexpr int kSkinnyChangeBlocks = 256;
struct ChangePlan {
  bool skinny;
  int splits;
  int chunk;
  int tiles;        // output tiles
  int tile_elems;   // floats per output tile
  bool tiles64 = false;  // 64 x 64 tiles on gemm_kernel
};

ChangePlan change_plan(int M, int N, int K) {
  // long K over 16-127 output tiles of 64 x 64: those tiles split over K on
  // about one block per CU
  if (K >= 4096 && tiles_of(M, N, 64) >= 16 && tiles_of(M, N, 64) < 128) {
    const int tiles = tiles_of(M, N, 64);
    const int sp = std::min((kCUs + tiles - 1) / tiles, K / 256);
    return {false, sp, chunk_for(K, sp), tiles, 64 * 64, true};
  }
  if (K >= 1024 && tiles_of(M, N, 64) < 128) {
    const int tiles = ((M + 63) / 64) * ((N + 31) / 32);
    int chunk = 1024;
    while (chunk > 128 && (long)tiles * ((K + chunk - 1) / chunk) < kSkinnyChangeBlocks) chunk /= 2;
    const int sp = (K + chunk - 1) / chunk;
    if (sp >= 2) return {true, sp, chunk, tiles, 64 * 32};
  }
  const int sp = choose_splits(M, N, K);
  return {false, sp, sp > 1 ? chunk_for(K, sp) : K, tile_count(M, N, K), tile_edge(M, N, K) * tile_cols(M, N, K)};
}

int change_splits(int M, int N, int K) { return change_plan(M, N, K).splits; }

size_t change_update_workspace(int M, int N, int K) {
  const ChangePlan pl = change_plan(M, N, K);
  return pl.splits > 1 ? (size_t)pl.splits * pl.tiles * pl.tile_elems : 0;
}

int change_arrivals(int M, int N, int K) {
  const ChangePlan pl = change_plan(M, N, K);
  return pl.splits > 1 ? pl.tiles : 0;
}

hipError_t change_update(hipStream_t s, const float* A, int lda, const float* D, int ldd, int M, int N, int K,
                         float* W, float* V, int ldw, float lr, float mom, float* ws, int* arrivals, float limit,
                         unsigned long long* faults) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const ChangePlan pl = change_plan(M, N, K);
  if (pl.splits <= 1) {
    EpiUpdate e{W, V, ldw, lr, mom, limit, faults};
    return launch_cfg<true, false>(s, A, lda, D, ldd, M, N, K, 1, K, e);
  }
  if (!arrivals || !ws || pl.tiles > kMaxArrivals) return hipErrorInvalidValue;
  EpiSplitUpdate e{ws, W, V, ldw, lr, mom, limit, faults, arrivals, pl.splits};
  if (pl.tiles64) return launch_gemm<64, 64, kTileK, true, false>(s, A, lda, D, ldd, M, N, K, pl.splits, pl.chunk, e);
  if (pl.skinny)
    return launch_kernel(skinny_kernel<2, true, false, false, false, false, EpiSplitUpdate>, pl.tiles * pl.splits, 512,
                         0, s, A, lda, D, ldd, M, N, K, pl.chunk, e, CtxInput{});
  return launch_cfg<true, false>(s, A, lda, D, ldd, M, N, K, pl.splits, pl.chunk, e);
}

hipError_t bias_update(hipStream_t s, const BiasJob* jobs, int n, float lr, float mom, float limit,
                       unsigned long long* faults) {
  for (int j0 = 0; j0 < n; j0 += kMaxBiasJobs) {
    BiasJobs b{};
    int blocks = 0;
    for (int j = j0; j < n && j < j0 + kMaxBiasJobs; ++j) {
      if (jobs[j].N <= 0) continue;
      b.j[b.n] = jobs[j];
      b.j[b.n].block0 = blocks;
      blocks += (jobs[j].N + 63) / 64;
      ++b.n;
    }
    if (blocks == 0) continue;
    const hipError_t e = launch_kernel(bias_update_kernel, blocks, 64 * kBiasWaves, 0, s, b, lr, mom, limit, faults);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

int onehot_forward_blocks(int rows, int H) {
  const int strips = (H + 63) / 64;
  const long items = (long)rows * strips;
  return (int)((items + 3) / 4);
}

hipError_t onehot_forward(hipStream_t s, const int32_t* act, int n_active, int rows, const float* W0, int ldw,
                          int n0, int H, int mode, float* out, int ldo, const float* T, int ldt, double* sse_part,
                          const float* tab) {
  if (rows <= 0 || H <= 0) return hipSuccess;
  const int strips = (H + 63) / 64;
  return launch_kernel(onehot_forward_kernel, onehot_forward_blocks(rows, H), kThreads, 0, s, act, n_active, rows, W0, ldw, n0, H,
                                                                            strips, mode, out, ldo, T, ldt, sse_part, tab);
}

hipError_t onehot_update(hipStream_t s, const int32_t* act, int n_active, int rows, const float* D, int ldd, int n0,
                         int H, float* W, float* V, int ldw, float lr, float mom, float limit,
                         unsigned long long* faults) {
  if (H <= 0) return hipSuccess;
  dim3 grid(n0 + 1, (H + kThreads - 1) / kThreads);
  return launch_kernel(onehot_update_kernel, grid, kThreads, 0, s, act, n_active, rows, D, ldd, n0, H, W, V, ldw, lr,
                       mom, limit, faults);
}

hipError_t sse_reduce(hipStream_t s, const double* part, int n, double* out) {
  return launch_kernel(sse_reduce_kernel, 1, kRed, 0, s, part, n, out);
}

hipError_t zero_ints(hipStream_t s, int* p, int n) {
  if (n <= 0) return hipSuccess;
  return launch_kernel(zero_ints_kernel, (n + kThreads - 1) / kThreads, kThreads, 0, s, p, n);
}

}  // namespace bpk
