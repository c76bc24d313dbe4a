// bp_device.h -- device helpers shared by the gfx950 kernels: the unit
// nonlinearity (exact or table, section 4.3) and the range check of summed
// weight changes (section 8).
#pragma once

#include <hip/hip_runtime.h>

namespace bpk {

// Table sigmoid geometry (section 4.3, figure 3): 256 entries, the logistic
// at equally spaced points of [-15, 15]; [-15, 15] maps onto [0, 255] by
// (z + 15) * 255 / 30, and 255 / 30 = 8.5 is exact in float.
constexpr int kSigTableSize = 256;
constexpr float kSigTableEnd = 15.0f;
constexpr float kSigTableScale = 8.5f;

// The logistic 1 / (1 + e^-z) from the hardware's base-2 exponential and
// reciprocal: t = -z log2(e) is carried as t_hi + t_lo (the rounding error
// of the product and of the constant), e^-z = 2^t_hi (1 + t_lo ln 2).
// Measured against a double reference over [-40, 40]: at most 3.8 ulp (2.4e-7
// relative), against 2.4 ulp for expf and an IEEE divide, at a fraction of
// their instructions.  NaN stays NaN; z < -88 gives 0 (a denormal at most).
__device__ __forceinline__ float logistic(float z) {
  const float kLog2e = 1.44269502f, kLog2eLo = 1.925963e-8f, kLn2 = 0.693147181f;
  const float th = -z * kLog2e;
  const float tl = fmaf(-z, kLog2e, -th) + (-z) * kLog2eLo;
  float e = __builtin_amdgcn_exp2f(th);
  e = fabsf(th) < 126.f ? e * fmaf(tl, kLn2, 1.0f) : e;
  return __builtin_amdgcn_rcpf(1.0f + e);
}

// Inputs outside [-15, 15] take the end entries; inside, the integer part of
// the mapped value picks an entry and the fractional part interpolates
// linearly towards the next one.  NaN stays NaN.
__device__ __forceinline__ float logistic_table(float z, const float* __restrict__ tab) {
  if (z != z) return z;
  const float zc = fminf(fmaxf(z, -kSigTableEnd), kSigTableEnd);
  const float x1 = (zc + kSigTableEnd) * kSigTableScale;        // [0, 255]
  const int i = min((int)x1, kSigTableSize - 2);                // x1 >= 0: truncation is the floor
  const float f = x1 - (float)i;                                // 1 at x1 = 255: the last entry
  const float a = tab[i], b = tab[i + 1];
  return a + f * (b - a);
}

// The unit nonlinearity: the table when one is given, else the exact logistic.
__device__ __forceinline__ float unit_sigma(float z, const float* __restrict__ tab) {
  return tab ? logistic_table(z, tab) : logistic(z);
}

// Range check of one summed change: with limit > 0, a change outside
// [-limit, limit] (or NaN) becomes 0 and is counted in `faults`.
__device__ __forceinline__ float checked_change(float g, float limit, int& faults) {
  if (limit > 0.f && !(fabsf(g) <= limit)) {
    ++faults;
    return 0.f;
  }
  return g;
}

// The momentum step V = lr G + mom V (section 6.2.1) with its rounding
// fixed: mom V is rounded, lr G is fused into the add.  Written out so that
// no kernel or template instance is left to the compiler's choice of which
// product to fuse, which would change the last bit between otherwise equal
// code paths.
__device__ __forceinline__ float momentum_step(float g, float v_old, float lr, float mom) {
  return fmaf(lr, g, mom * v_old);
}

// The error of a training call (section 10.1 reports the total squared
// error): out[0] = the sum of part[0, n) in double, in a fixed order (each of
// the NT threads adds a strided subset, eight loads in flight, then a tree
// over the threads).  Every thread of the NT-thread block must call it;
// `red` is NT doubles of LDS.
template <int NT>
__device__ __forceinline__ void block_sum_partials(const double* __restrict__ part, int n, double* out,
                                                   double* red) {
  double s = 0.0;
  for (int i0 = threadIdx.x; i0 < n; i0 += 8 * NT) {
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = i0 + u * NT < n ? part[i0 + u * NT] : 0.0;
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = NT / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

// Adds the fault counts of a wave to the device counter: a wave sum, then one
// atomic from lane 0 when the sum is nonzero.  Every lane of the wave must
// reach this call.
__device__ __forceinline__ void add_faults(int faults, unsigned long long* counter) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) faults += __shfl_xor(faults, off, 64);
  if ((threadIdx.x & 63) == 0 && faults > 0) atomicAdd(counter, (unsigned long long)faults);
}

}  // namespace bpk
