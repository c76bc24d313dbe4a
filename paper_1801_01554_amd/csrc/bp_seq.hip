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

#include "bp_internal.h"

namespace bpk {
namespace {

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

}  // namespace

hipError_t seq_assemble(hipStream_t s, const float* X, int n_ext, const float* cont, int S, int n_ctx,
                        const int32_t* ctx_layer, const int32_t* ctx_unit, const CtxSource& src, float* A0,
                        int lda0) {
  const int64_t total = (int64_t)S * lda0;
  if (total <= 0) return hipSuccess;
  return launch_kernel(seq_assemble_kernel, (unsigned)((total + kAsmThreads - 1) / kAsmThreads), kAsmThreads, 0, s,
                       X, n_ext, cont, S, n_ctx, ctx_layer, ctx_unit, src, A0, lda0);
}

}  // namespace bpk
