// bp_net.cpp -- host side of the C-ABI in include/bp.h.
//
// Owns the device state of a net (weights W, momentum V, workspace), checks
// every argument before any device work, and enqueues the launch sequence of
// one pooled update per batch (sections 3 and 4.1 of the paper):
//   forward l = 0 .. L-1  ->  output deltas + error partials
//   for l = L-1 .. 1:  hidden deltas of layer l (with the pre-update W_l),
//                      then the change and update of W_l
//   change and update of W_0 (dense product, or the one-hot row scatter).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "bp.h"
#include "bp_internal.h"

struct bp_net {
  int L = 0;                          // weight layers
  std::vector<int> n;                 // n[0..L]
  std::vector<int> ldw;               // padded row length of W_l (floats)
  std::vector<int> lda;               // padded row length of activations/deltas of layer l
  std::vector<int64_t> woff;          // device offset of W_l (floats)
  std::vector<int64_t> foff;          // offset of W_l in the flat ABI layout
  int64_t wtotal = 0;                 // device floats of W (padding included)
  int64_t nweights = 0;               // connection count
  float* W = nullptr;
  float* V = nullptr;
  hipStream_t stream = nullptr;
  int device = 0;
  // workspace
  int64_t ws_rows = 0;
  int64_t ws_csum_top = 0;            // rows of csum[L] (per-step tiling of sequence windows)
  std::vector<float*> act;            // act[l], l = 1 .. L-1 : [ws_rows][lda[l]]
  std::vector<float*> del;            // del[l], l = 1 .. L   : [ws_rows][lda[l]]
  std::vector<float*> csum;           // csum[l], l = 1 .. L  : [colsum_rows(ws_rows)][lda[l]]
  float* fwd_tmp[2] = {nullptr, nullptr};  // forward-only ping-pong buffers
  int64_t fwd_rows = 0;
  size_t fwd_cap = 0;
  float* splitk = nullptr;
  size_t splitk_cap = 0;
  int* arrivals = nullptr;            // split-K arrival counters (bpk::kMaxArrivals), zero between launches
  double* sse_part = nullptr;
  size_t sse_cap = 0;
  double* sse_dev = nullptr;
  double* host_sse = nullptr;         // pinned host word: the error sum's read-back
  // options (section 4.3 table sigmoid; section 8 range check)
  float* sig_tab = nullptr;           // device table, set while the table sigmoid is selected
  float* sig_tab_mem = nullptr;       // its allocation (kept once made)
  float fault_limit = 0.f;            // > 0: range check on
  unsigned long long* faults = nullptr;
  // checkpoint of W and V (section 10.4) and the guard that uses it
  float* ckW = nullptr;
  float* ckV = nullptr;
  // Elman context (section 10.5): context unit c (input n0 - n_ctx + c)
  // copies unit ctx_unit[c] of hidden layer ctx_layer[c]
  int n_ctx = 0;
  bool ctx_in_order = false;          // ctx_layer[c] == 1 and ctx_unit[c] == c for every c
  int32_t* ctx_layer_dev = nullptr;
  int32_t* ctx_unit_dev = nullptr;
  float* seq_in = nullptr;            // assembled input rows of a window [rows][lda[0]]
  size_t seq_in_cap = 0;
  struct Guard {
    bool on = false;
    int every = 1;
    double jump = 0.0;
    int since = 0;                    // epochs accepted since the checkpoint
    int retry_at = -1;                // epoch (from the checkpoint) already rolled back once
    bool have_last = false;
    double last_sse = 0.0;            // error of the last accepted epoch
    bool ck_have = false;
    double ck_sse = 0.0;              // error of the epoch the checkpoint was taken at
  } guard;
  // measurement: launches bracketed by events while `prof` is set
  bool prof = false;
  struct Rec {
    int kind;
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> ev_pool;
  int64_t prof_n[BP_K_COUNT] = {};
  double prof_ms[BP_K_COUNT] = {};
  // graph replay of a repeated training call: the second of two calls with
  // the same arguments captures its launches into a HIP graph, and later
  // calls with those arguments replay it.  `gen` changes whenever something
  // a captured call depends on changes (workspace, sigmoid, range check).
  struct TrainKey {
    const void* x = nullptr;
    const void* act = nullptr;
    const void* t = nullptr;
    int64_t n = 0;
    int32_t batch = 0, n_active = 0, ldx = 0;
    uint32_t lr = 0, mom = 0;
    uint64_t gen = 0;
    bool operator==(const TrainKey& o) const {
      return x == o.x && act == o.act && t == o.t && n == o.n && batch == o.batch && n_active == o.n_active &&
             ldx == o.ldx && lr == o.lr && mom == o.mom && gen == o.gen;
    }
  };
  bool graph_on = true;
  uint64_t gen = 0;
  bool have_last = false;
  TrainKey last_key, graph_key;
  hipStream_t cap_stream = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t graph_exec = nullptr;
  mutable std::string err;            // message of the last failure (read-only calls set it too)
};

// Workspace of bp_train_batches_noalloc, for callers that cannot allocate:
// one array per GPU, held until the process ends.  Host code never uses the
// array's name as an address (on the host it is a stand-in, not device
// memory): bp_create looks up each device's copy once, with that device
// current, and the entry point takes that address.  Every call on a GPU
// shares the GPU's copy, so calls that overlap on one GPU race.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device` (which must be current on the
// first call for it); nullptr on failure.
float* scratch_on(int device, hipError_t* err) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  *err = hipSuccess;
  if (device < 0 || device >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*err != hipSuccess) return nullptr;
    if (!p) {
      *err = hipErrorInvalidSymbol;
      return nullptr;
    }
    g_scratch_ptr[device] = static_cast<float*>(p);
  }
  return g_scratch_ptr[device];
}

thread_local std::string g_create_err;

int fail(const bp_net* net, int code, const std::string& msg) {
  if (net) net->err = msg;
  else g_create_err = msg;
  return code;
}

int hip_fail(const bp_net* net, hipError_t e, const char* what) {
  char buf[256];
  std::snprintf(buf, sizeof(buf), "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
  return fail(net, e == hipErrorOutOfMemory ? BP_ENOMEM : BP_EDEVICE, buf);
}

#define BP_HIP(net, expr)                                   \
  do {                                                      \
    hipError_t e_ = (expr);                                 \
    if (e_ != hipSuccess) return hip_fail((net), e_, #expr); \
  } while (0)

// The call's error sum: copied from the device into the net's pinned host
// word (a copy into pageable memory goes through a staging path and costs
// more than the whole update of a small net), then the stream is waited for.
int read_sse(bp_net* net, const double* src, hipStream_t s, double* sse_out) {
  BP_HIP(net, hipMemcpyAsync(net->host_sse, src, sizeof(double), hipMemcpyDeviceToHost, s));
  BP_HIP(net, hipStreamSynchronize(s));
  *sse_out = *net->host_sse;
  return BP_OK;
}

// Weight, activation and delta rows are padded to 32 floats, one 128-byte
// cache line: a row that one block writes then shares no line with a row
// that a block on another XCD writes (each XCD has its own L2).
int row_pad(int v) { return (v + 31) / 32 * 32; }

hipEvent_t take_event(bp_net* net) {
  if (!net->ev_pool.empty()) {
    hipEvent_t e = net->ev_pool.back();
    net->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Runs one launch; while profiling, the kernel records its execution start
// and end (from its own dispatch) on a pair of events.
template <class F>
hipError_t launch(bp_net* net, int kind, F&& f) {
  if (!net->prof) return f();
  hipEvent_t a = take_event(net), b = take_event(net);
  if (!a || !b) return hipErrorOutOfMemory;
  bpk::LaunchEvents& ev = bpk::launch_events();
  ev.start = a;
  ev.stop = b;
  ev.used = false;
  const hipError_t e = f();
  const bool used = ev.used;
  ev = bpk::LaunchEvents();
  if (used) {
    net->recs.push_back({kind, a, b});
  } else {
    net->ev_pool.push_back(a);
    net->ev_pool.push_back(b);
  }
  return e;
}

#define BP_LAUNCH(net, kind, expr) BP_HIP(net, launch(net, kind, [&]() { return (expr); }))

void free_ptr(void* p) {
  if (p) (void)hipFree(p);
}

void free_workspace(bp_net* net) {
  for (float* p : net->act) free_ptr(p);
  for (float* p : net->del) free_ptr(p);
  for (float* p : net->csum) free_ptr(p);
  net->act.assign(net->L + 1, nullptr);
  net->del.assign(net->L + 1, nullptr);
  net->csum.assign(net->L + 1, nullptr);
  net->ws_rows = 0;
  net->ws_csum_top = 0;
  free_ptr(net->splitk);
  net->splitk = nullptr;
  net->splitk_cap = 0;
  ++net->gen;
}

// Floats of split-K workspace one forward pass over `fwd_rows` patterns and
// the change products over `chg_rows` patterns need (used one at a time).
// The output layer's need is not monotonic in its row count (fewer rows,
// more splits), so callers ask for every row count they will use.
size_t splitk_floats(const bp_net* net, int64_t fwd_rows, int64_t chg_rows) {
  size_t sk = fwd_rows > 0 ? bpk::output_delta_workspace((int)fwd_rows, net->n[net->L], net->n[net->L - 1]) : 0;
  for (int l = 0; l < net->L && chg_rows > 0; ++l)
    sk = std::max(sk, bpk::change_update_workspace(net->n[l], net->n[l + 1], (int)chg_rows));
  return sk;
}

// Workspace for batches of up to `rows` patterns, `top_csum` column-sum rows
// of the output deltas (sequence windows tile them per step) and `splitk`
// floats of split-K partials.  Grows only.
int ensure_workspace(bp_net* net, int64_t rows, int64_t top_csum, size_t splitk) {
  top_csum = std::max<int64_t>(top_csum, bpk::colsum_rows((int)rows));
  if (rows <= net->ws_rows && top_csum <= net->ws_csum_top && splitk <= net->splitk_cap) return BP_OK;
  rows = std::max(rows, net->ws_rows);
  top_csum = std::max(top_csum, net->ws_csum_top);
  splitk = std::max(splitk, net->splitk_cap);
  BP_HIP(net, hipStreamSynchronize(net->stream));
  free_workspace(net);
  for (int l = 1; l <= net->L; ++l) {
    const size_t bytes = sizeof(float) * (size_t)rows * net->lda[l];
    if (l < net->L) BP_HIP(net, hipMalloc(&net->act[l], bytes));
    BP_HIP(net, hipMalloc(&net->del[l], bytes));
    const int64_t cr = l == net->L ? top_csum : bpk::colsum_rows((int)rows);
    BP_HIP(net, hipMalloc(&net->csum[l], sizeof(float) * (size_t)cr * net->lda[l]));
  }
  if (splitk) BP_HIP(net, hipMalloc(&net->splitk, sizeof(float) * splitk));
  net->splitk_cap = splitk;
  net->ws_rows = rows;
  net->ws_csum_top = top_csum;
  return BP_OK;
}

int ensure_sse(bp_net* net, size_t count) {
  if (!net->sse_dev) BP_HIP(net, hipMalloc(&net->sse_dev, sizeof(double)));
  if (count <= net->sse_cap) return BP_OK;
  BP_HIP(net, hipStreamSynchronize(net->stream));
  free_ptr(net->sse_part);
  net->sse_part = nullptr;
  net->sse_cap = 0;
  BP_HIP(net, hipMalloc(&net->sse_part, sizeof(double) * count));
  net->sse_cap = count;
  ++net->gen;
  return BP_OK;
}

bool aligned_ptr(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

float* wl(bp_net* net, int l) { return net->W + net->woff[l]; }
float* vl(bp_net* net, int l) { return net->V + net->woff[l]; }
float* wbias(bp_net* net, int l) { return wl(net, l) + (size_t)net->n[l] * net->ldw[l]; }
float* vbias(bp_net* net, int l) { return vl(net, l) + (size_t)net->n[l] * net->ldw[l]; }

// Copies between the flat ABI layout (host) and the padded device layout.
int copy_layers(const bp_net* net, float* dev, const float* host_src, float* host_dst) {
  for (int l = 0; l < net->L; ++l) {
    const size_t rows = (size_t)net->n[l] + 1, cols = (size_t)net->n[l + 1];
    float* d = dev + net->woff[l];
    if (host_src)
      BP_HIP(net, hipMemcpy2DAsync(d, sizeof(float) * net->ldw[l], host_src + net->foff[l], sizeof(float) * cols,
                                   sizeof(float) * cols, rows, hipMemcpyHostToDevice, net->stream));
    else
      BP_HIP(net, hipMemcpy2DAsync(host_dst + net->foff[l], sizeof(float) * cols, d, sizeof(float) * net->ldw[l],
                                   sizeof(float) * cols, rows, hipMemcpyDeviceToHost, net->stream));
  }
  BP_HIP(net, hipStreamSynchronize(net->stream));
  return BP_OK;
}

// Inputs of one batch: dense rows or one-hot index rows.
struct BatchInput {
  const float* x = nullptr;       // dense [rows][ldx]
  int ldx = 0;                    // row stride of x (0: n0)
  const int32_t* act = nullptr;   // one-hot [rows][n_active]
  int n_active = 0;
  // An Elman step whose input rows the first product builds: x holds the
  // external inputs (ldx = n_ext), ctx_h the previous step's first hidden
  // layer, cont the flags; the built rows go to rows_out (or nowhere).
  const float* ctx_h = nullptr;
  const float* cont = nullptr;
  float* rows_out = nullptr;
};

int ldx_of(const bp_net* net, const BatchInput& in) { return in.ldx > 0 ? in.ldx : net->n[0]; }

// Where a training forward pass writes its output layer: deltas, their
// per-tile column sums, and the optional per-pattern error mask.
struct OutputView {
  float* delta = nullptr;
  float* csum = nullptr;
  const float* mask = nullptr;
};

// Forward pass of `rows` patterns; the last layer either applies the output
// delta epilogue (training, T != nullptr) or writes sigma to `out`.
int run_forward(bp_net* net, const BatchInput& in, int rows, const float* T, double* sse_part,
                float* out, int ldo, float* const* acts, OutputView ov = OutputView(), int l_begin = 0,
                int l_end = -1) {
  if (!ov.delta) ov.delta = net->del[net->L];
  if (!ov.csum) ov.csum = net->csum[net->L];
  const int L = net->L;
  hipStream_t s = net->stream;
  for (int l = l_begin; l < (l_end < 0 ? L : l_end); ++l) {
    const bool last = (l == L - 1);
    float* dst = last ? (T ? ov.delta : out) : acts[l + 1];
    const int ldd = last ? (T ? net->lda[L] : ldo) : net->lda[l + 1];
    if (l == 0 && in.act) {
      BP_LAUNCH(net, BP_K_GATHER,
                bpk::onehot_forward(s, in.act, in.n_active, rows, wl(net, 0), net->ldw[0], net->n[0], net->n[1],
                                    (last && T) ? 1 : 0, dst, ldd, T, net->n[L], sse_part, net->sig_tab));
      continue;
    }
    if (l == 0 && in.ctx_h) {
      BP_LAUNCH(net, BP_K_FORWARD,
                bpk::forward_ctx_layer(s, in.x, in.ldx, in.ctx_h, net->lda[1], in.cont, wl(net, 0), net->ldw[0], rows,
                                       net->n[1], net->n[0], wbias(net, 0), dst, ldd, in.rows_out, net->lda[0],
                                       net->sig_tab));
      continue;
    }
    const float* A = (l == 0) ? in.x : acts[l];
    const int ldA = (l == 0) ? ldx_of(net, in) : net->lda[l];
    if (last && T) {
      BP_LAUNCH(net, BP_K_OUTPUT,
                bpk::forward_output_delta(s, A, ldA, wl(net, l), net->ldw[l], rows, net->n[l + 1], net->n[l],
                                          wbias(net, l), T, net->n[L], dst, ldd, sse_part, ov.csum,
                                          net->lda[L], net->splitk, net->sig_tab, ov.mask));
      if (bpk::output_delta_splits(rows, net->n[l + 1], net->n[l]) > 1)
        BP_LAUNCH(net, BP_K_OUTFIN,
                  bpk::output_finish(s, rows, net->n[l + 1], net->n[l], wbias(net, l), T, net->n[L], dst, ldd,
                                     sse_part, ov.csum, net->lda[L], net->splitk, net->sig_tab, ov.mask));
    } else
      BP_LAUNCH(net, BP_K_FORWARD,
                bpk::forward_layer(s, A, ldA, wl(net, l), net->ldw[l], rows, net->n[l + 1], net->n[l],
                                   wbias(net, l), dst, ldd, net->sig_tab));
  }
  return BP_OK;
}

// One-hot two-layer nets small enough for the fused two-launch update.
bool use_small(const bp_net* net, const BatchInput& in) {
  return in.act && net->L == 2 && bpk::small_path_fits(net->n[0], net->n[1], net->n[2], in.n_active);
}

int sse_blocks(const bp_net* net, const BatchInput& in, int rows) {
  if (use_small(net, in)) return bpk::small_fwdbwd_blocks(rows);
  if (net->L == 1 && in.act) return bpk::onehot_forward_blocks(rows, net->n[1]);
  return bpk::output_delta_blocks(rows, net->n[net->L], net->n[net->L - 1]);
}

// One pooled update of a small one-hot two-layer net: two launches.
// The fused two-launch update of one batch; with n_sse >= 0 (the call's last
// batch) the update launch also sums the call's n_sse error partials.
int run_small(bp_net* net, const BatchInput& in, int rows, const float* T, double* sse_part, float lr, float mom,
              int n_sse = -1) {
  hipStream_t s = net->stream;
  const int n0 = net->n[0], H = net->n[1], O = net->n[2];
  BP_LAUNCH(net, BP_K_FUSED_FB,
            bpk::small_fwdbwd(s, in.act, in.n_active, rows, wl(net, 0), net->ldw[0], n0, H, wl(net, 1), net->ldw[1], O,
                              T, net->splitk, net->del[1], net->lda[1], net->del[2], net->lda[2], sse_part,
                              net->sig_tab));
  BP_LAUNCH(net, BP_K_FUSED_UPD,
            bpk::small_update(s, in.act, in.n_active, rows, net->splitk, net->del[1], net->lda[1], net->del[2],
                              net->lda[2], wl(net, 0), vl(net, 0), net->ldw[0], n0, H, wl(net, 1), vl(net, 1),
                              net->ldw[1], O, lr, mom, net->fault_limit, net->faults, net->sse_part, n_sse,
                              n_sse >= 0 ? net->sse_dev : nullptr));
  return BP_OK;
}

// Backward pass and update of one batch whose deltas of the output layer are
// in del[L].  The bias rows, which no delta or change product reads, are
// updated together in one launch after the last change product.
int run_backward_update(bp_net* net, const BatchInput& in, int rows, float lr, float mom, int top_csum = 0) {
  hipStream_t s = net->stream;
  bpk::BiasJob bias[bpk::kMaxBiasJobs];
  int nb = 0;
  for (int l = net->L - 1; l >= 0; --l) {
    // Hidden deltas of layer l use W_l before its update.
    if (l >= 1)
      BP_LAUNCH(net, BP_K_BACKWARD,
                bpk::backward_layer(s, net->del[l + 1], net->lda[l + 1], wl(net, l), net->ldw[l], rows, net->n[l],
                                    net->n[l + 1], net->act[l], net->lda[l], net->del[l], net->lda[l], net->csum[l],
                                    net->lda[l]));
    if (l == 0 && in.act) {
      BP_LAUNCH(net, BP_K_SCATTER,
                bpk::onehot_update(s, in.act, in.n_active, rows, net->del[1], net->lda[1], net->n[0], net->n[1],
                                   wl(net, 0), vl(net, 0), net->ldw[0], lr, mom, net->fault_limit, net->faults));
      continue;
    }
    const float* A = (l == 0) ? in.x : net->act[l];
    const int ldA = (l == 0) ? ldx_of(net, in) : net->lda[l];
    const bool split = bpk::change_splits(net->n[l], net->n[l + 1], rows) > 1;
    BP_LAUNCH(net, split ? BP_K_SPLITK : BP_K_CHANGE,
              bpk::change_update(s, A, ldA, net->del[l + 1], net->lda[l + 1], net->n[l], net->n[l + 1], rows,
                                 wl(net, l), vl(net, l), net->ldw[l], lr, mom, net->splitk, net->arrivals,
                                 net->fault_limit, net->faults));
    bias[nb++] = {net->csum[l + 1], wbias(net, l), vbias(net, l), net->lda[l + 1],
                  (l + 1 == net->L && top_csum > 0) ? top_csum : bpk::colsum_rows(rows), net->n[l + 1], 0};
    if (nb == bpk::kMaxBiasJobs) {
      BP_LAUNCH(net, BP_K_BIAS, bpk::bias_update(s, bias, nb, lr, mom, net->fault_limit, net->faults));
      nb = 0;
    }
  }
  if (nb > 0) BP_LAUNCH(net, BP_K_BIAS, bpk::bias_update(s, bias, nb, lr, mom, net->fault_limit, net->faults));
  return BP_OK;
}

// The launches of one training call: every batch, then the error reduction
// (kernels only, on net->stream; no allocation, copy or synchronisation, so
// that the sequence can be captured into a graph).
int train_launches(bp_net* net, const BatchInput& in, const float* targets, int64_t n, int32_t batch, float lr,
                   float mom) {
  int rc = BP_OK;
  size_t used = 0;
  for (int64_t p0 = 0; p0 < n; p0 += batch) {
    const int rows = (int)std::min<int64_t>(batch, n - p0);
    BatchInput b = in;
    if (b.x) b.x += (size_t)p0 * net->n[0];
    if (b.act) b.act += (size_t)p0 * b.n_active;
    const float* Tb = targets + (size_t)p0 * net->n[net->L];
    if (use_small(net, b)) {
      const bool last = p0 + batch >= n;
      const size_t total = used + (size_t)sse_blocks(net, b, rows);
      rc = run_small(net, b, rows, Tb, net->sse_part + used, lr, mom, last ? (int)total : -1);
      if (rc) return rc;
      used = total;
      if (last) return BP_OK;   // the error sum went with the last update
      continue;
    }
    rc = run_forward(net, b, rows, Tb, net->sse_part + used, nullptr, 0, net->act.data());
    if (rc) return rc;
    used += (size_t)sse_blocks(net, b, rows);
    rc = run_backward_update(net, b, rows, lr, mom);
    if (rc) return rc;
  }
  BP_LAUNCH(net, BP_K_REDUCE, bpk::sse_reduce(net->stream, net->sse_part, (int)used, net->sse_dev));
  return BP_OK;
}

void drop_graph(bp_net* net) {
  if (net->graph_exec) (void)hipGraphExecDestroy(net->graph_exec);
  if (net->graph) (void)hipGraphDestroy(net->graph);
  net->graph_exec = nullptr;
  net->graph = nullptr;
}

// Captures train_launches on the net's private capture stream and
// instantiates the graph (replacing the previous one).
int capture_train(bp_net* net, const BatchInput& in, const float* targets, int64_t n, int32_t batch, float lr,
                  float mom) {
  if (!net->cap_stream) BP_HIP(net, hipStreamCreateWithFlags(&net->cap_stream, hipStreamNonBlocking));
  drop_graph(net);
  BP_HIP(net, hipStreamBeginCapture(net->cap_stream, hipStreamCaptureModeThreadLocal));
  hipStream_t user = net->stream;
  net->stream = net->cap_stream;
  const int rc = train_launches(net, in, targets, n, batch, lr, mom);
  net->stream = user;
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(net->cap_stream, &g);
  if (rc) {
    if (g) (void)hipGraphDestroy(g);
    return rc;
  }
  if (e != hipSuccess) return hip_fail(net, e, "hipStreamEndCapture");
  hipGraphExec_t ex = nullptr;
  const hipError_t ei = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
  if (ei != hipSuccess) {
    (void)hipGraphDestroy(g);
    return hip_fail(net, ei, "hipGraphInstantiate");
  }
  net->graph = g;
  net->graph_exec = ex;
  return BP_OK;
}

int train(bp_net* net, const BatchInput& in, const float* targets, int64_t n, int32_t batch, float lr, float mom,
          double* sse_out) {
  if (n == 0) {
    if (sse_out) *sse_out = 0.0;
    return BP_OK;
  }
  const int64_t rows_max = std::min<int64_t>(batch, n);
  // every batch but the last has rows_max rows
  const int64_t nb = (n + batch - 1) / batch;
  const int last_rows = (int)(n - (nb - 1) * (int64_t)batch);
  size_t sk = std::max(splitk_floats(net, rows_max, rows_max), splitk_floats(net, last_rows, last_rows));
  if (use_small(net, in))   // the fused path's grouped activations take the split-K workspace
    sk = std::max(sk, bpk::small_scratch_floats((int)rows_max, net->n[1]));
  int rc = ensure_workspace(net, rows_max, 0, sk);
  if (rc) return rc;
  // exact number of error partials
  const size_t need = (size_t)sse_blocks(net, in, (int)rows_max) * (size_t)(nb - 1) +
                      (size_t)sse_blocks(net, in, last_rows);
  rc = ensure_sse(net, need);
  if (rc) return rc;
  // A call of one batch launches directly: its three or so launches cost
  // less host time than a graph launch.
  if (net->graph_on && !net->prof && nb >= 2) {
    bp_net::TrainKey key;
    key.x = in.x;
    key.act = in.act;
    key.t = targets;
    key.n = n;
    key.batch = batch;
    key.n_active = in.n_active;
    key.ldx = in.ldx;
    std::memcpy(&key.lr, &lr, sizeof(float));
    std::memcpy(&key.mom, &mom, sizeof(float));
    key.gen = net->gen;
    if (!(net->graph_exec && key == net->graph_key)) {
      if (net->have_last && key == net->last_key) {
        rc = capture_train(net, in, targets, n, batch, lr, mom);
        if (rc) return rc;
        net->graph_key = key;
      } else {
        rc = train_launches(net, in, targets, n, batch, lr, mom);
        if (rc) return rc;
        net->last_key = key;
        net->have_last = true;
        key.n = -1;   // no replay this time
      }
    }
    if (key.n >= 0) BP_HIP(net, hipGraphLaunch(net->graph_exec, net->stream));
  } else {
    rc = train_launches(net, in, targets, n, batch, lr, mom);
    if (rc) return rc;
  }
  if (sse_out) return read_sse(net, net->sse_dev, net->stream, sse_out);
  return BP_OK;
}

// A training call whose workspace is carved out of the device's `scratch`
// instead of the net's allocations: the same launches as train(), issued
// directly (no graph, no profiling events), with the net's workspace views
// pointed into the scratch for the call and restored afterwards.
int train_noalloc(bp_net* net, const BatchInput& in, const float* targets, int64_t n, int32_t batch, float lr,
                  float mom, double* sse_out) {
  if (n == 0) {
    if (sse_out) *sse_out = 0.0;
    return BP_OK;
  }
  hipError_t e = hipSuccess;
  float* base = scratch_on(net->device, &e);
  if (!base) return hip_fail(net, e, "bp_train_batches_noalloc: scratch address");
  const int64_t rows_max = std::min<int64_t>(batch, n);
  const int64_t nb = (n + batch - 1) / batch;
  const int last_rows = (int)(n - (nb - 1) * (int64_t)batch);
  const size_t sk = std::max(splitk_floats(net, rows_max, rows_max), splitk_floats(net, last_rows, last_rows));
  const size_t n_sse = (size_t)sse_blocks(net, in, (int)rows_max) * (size_t)(nb - 1) +
                       (size_t)sse_blocks(net, in, last_rows);
  // layout, each piece on a 256-byte boundary: act[1..L-1], del[1..L],
  // csum[1..L], split partials, arrival counters, error partials, error sum
  size_t off = 0;
  auto take = [&](size_t floats) {
    const size_t o = off;
    off += (floats + 63) / 64 * 64;
    return o;
  };
  std::vector<size_t> oa(net->L + 1, 0), od(net->L + 1, 0), oc(net->L + 1, 0);
  for (int l = 1; l <= net->L; ++l) {
    if (l < net->L) oa[l] = take((size_t)rows_max * net->lda[l]);
    od[l] = take((size_t)rows_max * net->lda[l]);
    oc[l] = take((size_t)bpk::colsum_rows((int)rows_max) * net->lda[l]);
  }
  const size_t osk = take(sk);
  const size_t oarr = take(bpk::kMaxArrivals);
  const size_t osp = take(2 * n_sse);
  const size_t osd = take(2);
  if (off * sizeof(float) > kScratchBytes) {
    char buf[256];
    std::snprintf(buf, sizeof(buf),
                  "bp_train_batches_noalloc: the call needs %zu bytes of workspace, more than the %zu-byte "
                  "scratch (use a smaller batch, or bp_train_batches)",
                  off * sizeof(float), kScratchBytes);
    return fail(net, BP_EINVAL, buf);
  }
  // swap the views in, run, swap back
  std::vector<float*> act = net->act, del = net->del, csum = net->csum;
  float* splitk = net->splitk;
  int* arrivals = net->arrivals;
  double* sse_part = net->sse_part;
  double* sse_dev = net->sse_dev;
  const bool prof = net->prof;
  for (int l = 1; l <= net->L; ++l) {
    net->act[l] = l < net->L ? base + oa[l] : nullptr;
    net->del[l] = base + od[l];
    net->csum[l] = base + oc[l];
  }
  net->splitk = base + osk;
  net->arrivals = reinterpret_cast<int*>(base + oarr);
  net->sse_part = reinterpret_cast<double*>(base + osp);
  net->sse_dev = reinterpret_cast<double*>(base + osd);
  net->prof = false;
  // the counters start at zero (every finished launch leaves them so; an
  // earlier call that failed part way might not have)
  const hipError_t ez = bpk::zero_ints(net->stream, net->arrivals, bpk::kMaxArrivals);
  int rc = ez == hipSuccess ? BP_OK : hip_fail(net, ez, "bp_train_batches_noalloc: counter reset");
  if (rc == BP_OK) rc = train_launches(net, in, targets, n, batch, lr, mom);
  double* sum = net->sse_dev;
  net->act = act;
  net->del = del;
  net->csum = csum;
  net->splitk = splitk;
  net->arrivals = arrivals;
  net->sse_part = sse_part;
  net->sse_dev = sse_dev;
  net->prof = prof;
  if (rc) return rc;
  if (sse_out) return read_sse(net, sum, net->stream, sse_out);
  return BP_OK;
}

// ---- Elman nets (section 10.5)

// Activation rows of `step` (S rows each) in the window buffers, per hidden
// layer, as the context source of the next step.
bpk::CtxSource ctx_source(bp_net* net, int64_t step, int S) {
  bpk::CtxSource src{};
  for (int l = 1; l < net->L && l <= bpk::kCtxMaxLayer; ++l) {
    src.base[l] = step < 0 ? nullptr : net->act[l] + (size_t)step * S * net->lda[l];
    src.ld[l] = net->lda[l];
  }
  return src;
}

// The first product builds a step's input rows itself when the context
// copies hidden layer 1 in order and the product takes the skinny kernel.
bool fuse_ctx_input(const bp_net* net, int S) {
  return net->ctx_in_order && bpk::forward_ctx_fits(S, net->n[1], net->n[0]);
}

// Input of a step whose first product builds the rows: external inputs of
// the step, the context source `step` (S rows of hidden layer 1), the flags,
// and where the built rows go.
BatchInput ctx_input(bp_net* net, const float* X, int n_ext, const float* cont, int64_t step, int S, float* rows_out) {
  BatchInput in;
  in.x = n_ext > 0 ? X : nullptr;
  in.ldx = n_ext;
  in.ctx_h = net->act[1] + (size_t)step * S * net->lda[1];
  in.cont = cont;
  in.rows_out = rows_out;
  return in;
}

int ensure_seq_in(bp_net* net, int64_t rows) {
  const size_t need = (size_t)rows * net->lda[0];
  if (need <= net->seq_in_cap) return BP_OK;
  BP_HIP(net, hipStreamSynchronize(net->stream));
  free_ptr(net->seq_in);
  net->seq_in = nullptr;
  net->seq_in_cap = 0;
  BP_HIP(net, hipMalloc(&net->seq_in, sizeof(float) * need));
  net->seq_in_cap = need;
  return BP_OK;
}

// The forward pass of the window of `steps` steps starting at step w0 (of B
// steps per window) in one launch (one hidden layer, context in order).
int run_window(bp_net* net, const float* X, const float* targets, const float* cont, const float* mask, int64_t w0,
               int steps, int B, int S, int per_step) {
  const int n_ext = net->n[0] - net->n_ctx, nL = net->n[2], lda1 = net->lda[1];
  bpk::ElmanWindow ew;
  ew.X = n_ext > 0 ? X + (size_t)w0 * S * n_ext : nullptr;
  ew.n_ext = n_ext;
  ew.cont = cont + (size_t)w0 * S;
  ew.mask = mask + (size_t)w0 * S;
  ew.T = targets + (size_t)w0 * S * nL;
  ew.ldt = nL;
  // context source of the window's first step: the last step of the
  // previous (full) window; none in the first window of the call
  ew.Hprev = w0 > 0 ? net->act[1] + (size_t)(B - 1) * S * lda1 : nullptr;
  ew.ldhp = lda1;
  ew.W0 = wl(net, 0);
  ew.ldw0 = net->ldw[0];
  ew.b0 = wbias(net, 0);
  ew.W1 = wl(net, 1);
  ew.ldw1 = net->ldw[1];
  ew.b1 = wbias(net, 1);
  ew.n0 = net->n[0];
  ew.n1 = net->n[1];
  ew.n2 = nL;
  ew.H = net->act[1];
  ew.ldh = lda1;
  ew.rows = net->seq_in;
  ew.ldr = net->lda[0];
  ew.D = net->del[2];
  ew.ldd = net->lda[2];
  ew.colsum = net->csum[2];
  ew.ldcs = net->lda[2];
  ew.sse = net->sse_part + (size_t)w0 * per_step;
  ew.tab = net->sig_tab;
  ew.S = S;
  ew.steps = steps;
  BP_LAUNCH(net, BP_K_SEQ_WIN, bpk::elman_window(net->stream, ew));
  return BP_OK;
}

// Training over n_steps x S patterns: windows of B steps; within a window,
// step by step: assemble the input rows (external inputs, flag x context),
// forward pass with masked output deltas; then one backward pass and pooled
// update over all rows of the window.  Rows of a window are step-major.
int train_sequences(bp_net* net, const float* X, const float* targets, const float* cont, const float* mask,
                    int64_t T, int S, int B, float lr, float mom, double* sse_out) {
  if (T == 0) {
    if (sse_out) *sse_out = 0.0;
    return BP_OK;
  }
  const int L = net->L, n_ext = net->n[0] - net->n_ctx, nL = net->n[L];
  const int steps_max = (int)std::min<int64_t>(B, T);
  const int last_steps = (int)(T - (T - 1) / B * B);
  const int64_t rows_max = (int64_t)steps_max * S;
  const bool fuse_ctx = fuse_ctx_input(net, S);
  // one hidden layer: the window's forward pass in one launch, each block
  // carrying the recurrence of its own streams
  const bool window = net->ctx_in_order && L == 2 && bpk::elman_window_fits(S, n_ext, net->n[0], net->n[1], nL);
  // otherwise, with one hidden layer, step k's hidden layer and step k - 1's
  // output layer share a launch; a window's first hidden layer and last
  // output layer run alone
  const bool pair =
      !window && fuse_ctx && L == 2 && B > 1 && bpk::elman_pair_fits(S, net->n[0], net->n[1], net->n[2]);
  // output-layer column-sum rows of a step (of a window for the one-launch
  // window), and error partials of a step
  const int csS = window ? bpk::elman_window_blocks(S) : bpk::colsum_rows(S);
  const int per_step = window ? bpk::elman_window_blocks(S) : bpk::output_delta_blocks(S, nL, net->n[L - 1]);
  int rc = ensure_workspace(net, rows_max, (int64_t)steps_max * csS,
                            std::max({splitk_floats(net, S, rows_max), splitk_floats(net, 0, (int64_t)last_steps * S)}));
  if (rc) return rc;
  rc = ensure_seq_in(net, rows_max);
  if (rc) return rc;
  rc = ensure_sse(net, (size_t)T * per_step);
  if (rc) return rc;
  hipStream_t s = net->stream;
  const int lda1 = net->lda[1], ldL = net->lda[L];
  std::vector<float*> acts(L + 1, nullptr);
  // the output layer's view of step k of the window (step g of the call)
  auto view = [&](int k, int64_t g) {
    OutputView ov;
    ov.delta = net->del[L] + (size_t)k * S * ldL;
    ov.csum = net->csum[L] + (size_t)k * csS * ldL;
    ov.mask = mask + (size_t)g * S;
    return ov;
  };
  for (int64_t w0 = 0; w0 < T; w0 += B) {
    const int steps = (int)std::min<int64_t>(B, T - w0);
    if (window) {
      rc = run_window(net, X, targets, cont, mask, w0, steps, B, S, per_step);
      if (rc) return rc;
    }
    for (int k = 0; k < steps && !window; ++k) {
      const int64_t g = w0 + k;
      if (pair && k > 0) {
        const OutputView ov = view(k - 1, g - 1);
        const float* hp = net->act[1] + (size_t)(k - 1) * S * lda1;
        BP_LAUNCH(net, BP_K_SEQ_PAIR,
                  bpk::elman_pair(s, n_ext > 0 ? X + (size_t)g * S * n_ext : nullptr, n_ext, hp, cont + (size_t)g * S,
                                  wl(net, 0), net->ldw[0], wbias(net, 0), net->n[0], net->n[1],
                                  net->act[1] + (size_t)k * S * lda1, net->seq_in + (size_t)k * S * net->lda[0],
                                  net->lda[0], wl(net, 1), net->ldw[1], wbias(net, 1), nL, lda1, S,
                                  targets + (size_t)(g - 1) * S * nL, nL, ov.delta, ldL,
                                  net->sse_part + (size_t)(g - 1) * per_step, ov.csum, ldL, net->sig_tab, ov.mask));
        continue;
      }
      // context source: the previous step of this window, or the last step of
      // the previous (full) window, or none at the first step of the call
      const int64_t prev = k > 0 ? k - 1 : (w0 > 0 ? B - 1 : -1);
      float* A0 = net->seq_in + (size_t)k * S * net->lda[0];
      BatchInput in;
      // (with one step per window the source rows are the ones this step
      // writes: those steps build the rows first)
      if (fuse_ctx && prev >= 0 && prev != k) {
        in = ctx_input(net, X + (size_t)g * S * n_ext, n_ext, cont + (size_t)g * S, prev, S, A0);
      } else {
        BP_LAUNCH(net, BP_K_SEQ_IN,
                  bpk::seq_assemble(s, X + (size_t)g * S * n_ext, n_ext, cont + (size_t)g * S, S, net->n_ctx,
                                    net->ctx_layer_dev, net->ctx_unit_dev, ctx_source(net, prev, S), A0,
                                    net->lda[0]));
        in.x = A0;
        in.ldx = net->lda[0];
      }
      for (int l = 1; l < L; ++l) acts[l] = net->act[l] + (size_t)k * S * net->lda[l];
      rc = run_forward(net, in, S, targets + (size_t)g * S * nL, net->sse_part + (size_t)g * per_step, nullptr, 0,
                       acts.data(), view(k, g), 0, pair ? L - 1 : L);
      if (rc) return rc;
    }
    if (pair) {
      const int k = steps - 1;
      const int64_t g = w0 + k;
      acts[1] = net->act[1] + (size_t)k * S * lda1;
      rc = run_forward(net, BatchInput(), S, targets + (size_t)g * S * nL, net->sse_part + (size_t)g * per_step,
                       nullptr, 0, acts.data(), view(k, g), L - 1, L);
      if (rc) return rc;
    }
    BatchInput win;
    win.x = net->seq_in;
    win.ldx = net->lda[0];
    rc = run_backward_update(net, win, steps * S, lr, mom, window ? csS : steps * csS);
    if (rc) return rc;
  }
  BP_LAUNCH(net, BP_K_REDUCE, bpk::sse_reduce(s, net->sse_part, (int)(T * per_step), net->sse_dev));
  if (sse_out) return read_sse(net, net->sse_dev, s, sse_out);
  return BP_OK;
}

// Forward passes of the sequences (no update): hidden activations ping-pong
// between two S-row halves of the workspace, the previous step's half being
// the context source.
int forward_sequences(bp_net* net, const float* X, const float* cont, int64_t T, int S, float* out) {
  if (T == 0) return BP_OK;
  const int L = net->L, n_ext = net->n[0] - net->n_ctx, nL = net->n[L];
  int rc = ensure_workspace(net, 2 * (int64_t)S, 0, 0);
  if (rc) return rc;
  rc = ensure_seq_in(net, S);
  if (rc) return rc;
  const bool fuse_ctx = fuse_ctx_input(net, S);
  std::vector<float*> acts(L + 1, nullptr);
  for (int64_t g = 0; g < T; ++g) {
    const int64_t half = g & 1;
    BatchInput in;
    if (fuse_ctx && g > 0) {
      in = ctx_input(net, X + (size_t)g * S * n_ext, n_ext, cont + (size_t)g * S, 1 - half, S, nullptr);
    } else {
      BP_LAUNCH(net, BP_K_SEQ_IN,
                bpk::seq_assemble(net->stream, X + (size_t)g * S * n_ext, n_ext, cont + (size_t)g * S, S, net->n_ctx,
                                  net->ctx_layer_dev, net->ctx_unit_dev, ctx_source(net, g > 0 ? 1 - half : -1, S),
                                  net->seq_in, net->lda[0]));
      in.x = net->seq_in;
      in.ldx = net->lda[0];
    }
    for (int l = 1; l < L; ++l) acts[l] = net->act[l] + (size_t)half * S * net->lda[l];
    rc = run_forward(net, in, S, nullptr, nullptr, out + (size_t)g * S * nL, nL, acts.data());
    if (rc) return rc;
  }
  return BP_OK;
}

int forward_only(bp_net* net, const BatchInput& in, int64_t n, float* out) {
  if (n == 0) return BP_OK;
  const int64_t chunk = std::min<int64_t>(n, 8192);
  // ping-pong activation buffers sized for the widest hidden layer
  int widest = 4;
  for (int l = 1; l < net->L; ++l) widest = std::max(widest, net->lda[l]);
  const size_t need = (size_t)chunk * widest;
  if (net->L > 1 && need > net->fwd_cap) {
    BP_HIP(net, hipStreamSynchronize(net->stream));
    free_ptr(net->fwd_tmp[0]);
    free_ptr(net->fwd_tmp[1]);
    net->fwd_tmp[0] = net->fwd_tmp[1] = nullptr;
    net->fwd_cap = 0;
    BP_HIP(net, hipMalloc(&net->fwd_tmp[0], sizeof(float) * need));
    BP_HIP(net, hipMalloc(&net->fwd_tmp[1], sizeof(float) * need));
    net->fwd_cap = need;
  }
  std::vector<float*> acts(net->L + 1, nullptr);
  for (int l = 1; l < net->L; ++l) acts[l] = net->fwd_tmp[l & 1];
  for (int64_t p0 = 0; p0 < n; p0 += chunk) {
    const int rows = (int)std::min<int64_t>(chunk, n - p0);
    BatchInput b = in;
    if (b.x) b.x += (size_t)p0 * net->n[0];
    if (b.act) b.act += (size_t)p0 * b.n_active;
    int rc = run_forward(net, b, rows, nullptr, nullptr, out + (size_t)p0 * net->n[net->L], net->n[net->L],
                         acts.data());
    if (rc) return rc;
  }
  return BP_OK;
}

int checkpoint_save(bp_net* net) {
  const size_t bytes = sizeof(float) * net->wtotal;
  if (!net->ckW) {
    BP_HIP(net, hipStreamSynchronize(net->stream));
    BP_HIP(net, hipMalloc(&net->ckW, bytes));
    const hipError_t e = hipMalloc(&net->ckV, bytes);
    if (e != hipSuccess) {
      free_ptr(net->ckW);
      net->ckW = nullptr;
      return hip_fail(net, e, "hipMalloc(checkpoint)");
    }
  }
  BP_HIP(net, hipMemcpyAsync(net->ckW, net->W, bytes, hipMemcpyDeviceToDevice, net->stream));
  BP_HIP(net, hipMemcpyAsync(net->ckV, net->V, bytes, hipMemcpyDeviceToDevice, net->stream));
  return BP_OK;
}

int checkpoint_restore(bp_net* net) {
  const size_t bytes = sizeof(float) * net->wtotal;
  BP_HIP(net, hipMemcpyAsync(net->W, net->ckW, bytes, hipMemcpyDeviceToDevice, net->stream));
  BP_HIP(net, hipMemcpyAsync(net->V, net->ckV, bytes, hipMemcpyDeviceToDevice, net->stream));
  return BP_OK;
}

int check_net(const bp_net* net) { return net ? BP_OK : BP_EINVAL; }

}  // namespace

extern "C" {

int bp_create(const int32_t* layer_sizes, int32_t n_layers, bp_net** out) {
  if (!out) return fail(nullptr, BP_EINVAL, "bp_create: out is NULL");
  *out = nullptr;
  if (!layer_sizes) return fail(nullptr, BP_EINVAL, "bp_create: layer_sizes is NULL");
  if (n_layers < 2) return fail(nullptr, BP_EINVAL, "bp_create: need at least 2 layer sizes");
  for (int i = 0; i < n_layers; ++i)
    if (layer_sizes[i] < 1 || layer_sizes[i] > (1 << 24))
      return fail(nullptr, BP_EINVAL, "bp_create: layer sizes must be in [1, 2^24]");
  bp_net* net = new bp_net();
  net->L = n_layers - 1;
  net->n.assign(layer_sizes, layer_sizes + n_layers);
  net->ldw.resize(net->L);
  net->woff.resize(net->L);
  net->foff.resize(net->L);
  net->lda.resize(net->L + 1);
  for (int l = 0; l <= net->L; ++l) net->lda[l] = row_pad(net->n[l]);
  for (int l = 0; l < net->L; ++l) {
    net->ldw[l] = row_pad(net->n[l + 1]);
    net->woff[l] = net->wtotal;
    net->foff[l] = net->nweights;
    net->wtotal += (int64_t)(net->n[l] + 1) * net->ldw[l];
    net->nweights += (int64_t)(net->n[l] + 1) * net->n[l + 1];
  }
  net->act.assign(net->L + 1, nullptr);
  net->del.assign(net->L + 1, nullptr);
  net->csum.assign(net->L + 1, nullptr);
  hipError_t e = hipGetDevice(&net->device);
  if (e == hipSuccess) e = hipMalloc(&net->W, sizeof(float) * net->wtotal);
  if (e == hipSuccess) e = hipMalloc(&net->V, sizeof(float) * net->wtotal);
  if (e == hipSuccess) e = hipMemset(net->W, 0, sizeof(float) * net->wtotal);
  if (e == hipSuccess) e = hipMemset(net->V, 0, sizeof(float) * net->wtotal);
  if (e == hipSuccess) e = hipMalloc(&net->arrivals, sizeof(int) * bpk::kMaxArrivals);
  if (e == hipSuccess) e = hipMemset(net->arrivals, 0, sizeof(int) * bpk::kMaxArrivals);
  if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&net->host_sse), sizeof(double), hipHostMallocDefault);
  if (e == hipSuccess) (void)scratch_on(net->device, &e);   // this device's scratch address, once
  if (e != hipSuccess) {
    hip_fail(nullptr, e, "bp_create");
    const int code = e == hipErrorOutOfMemory ? BP_ENOMEM : BP_EDEVICE;
    free_ptr(net->W);
    free_ptr(net->V);
    free_ptr(net->arrivals);
    if (net->host_sse) (void)hipHostFree(net->host_sse);
    delete net;
    return code;
  }
  *out = net;
  return BP_OK;
}

void bp_destroy(bp_net* net) {
  if (!net) return;
  (void)hipStreamSynchronize(net->stream);
  free_workspace(net);
  free_ptr(net->fwd_tmp[0]);
  free_ptr(net->fwd_tmp[1]);
  free_ptr(net->sse_part);
  free_ptr(net->sse_dev);
  free_ptr(net->sig_tab_mem);
  free_ptr(net->faults);
  free_ptr(net->ckW);
  free_ptr(net->ckV);
  free_ptr(net->ctx_layer_dev);
  free_ptr(net->ctx_unit_dev);
  free_ptr(net->seq_in);
  free_ptr(net->W);
  free_ptr(net->V);
  free_ptr(net->arrivals);
  if (net->host_sse) (void)hipHostFree(net->host_sse);
  for (auto& r : net->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (hipEvent_t e : net->ev_pool) (void)hipEventDestroy(e);
  drop_graph(net);
  if (net->cap_stream) (void)hipStreamDestroy(net->cap_stream);
  delete net;
}

int bp_set_stream(bp_net* net, void* hip_stream) {
  if (check_net(net)) return BP_EINVAL;
  if (net->stream != (hipStream_t)hip_stream) BP_HIP(net, hipStreamSynchronize(net->stream));
  net->stream = (hipStream_t)hip_stream;
  return BP_OK;
}

int64_t bp_num_weights(const bp_net* net) { return net ? net->nweights : -1; }

int bp_set_weights(bp_net* net, const float* w_host, int64_t n) {
  if (check_net(net)) return BP_EINVAL;
  if (!w_host) return fail(net, BP_EINVAL, "bp_set_weights: w_host is NULL");
  if (n != net->nweights) return fail(net, BP_EINVAL, "bp_set_weights: n != bp_num_weights");
  BP_HIP(net, hipStreamSynchronize(net->stream));
  BP_HIP(net, hipMemsetAsync(net->W, 0, sizeof(float) * net->wtotal, net->stream));
  BP_HIP(net, hipMemsetAsync(net->V, 0, sizeof(float) * net->wtotal, net->stream));
  // the split-K arrival counters are zero between launches; clear them here too,
  // in case a failed launch left some set
  BP_HIP(net, hipMemsetAsync(net->arrivals, 0, sizeof(int) * bpk::kMaxArrivals, net->stream));
  return copy_layers(net, net->W, w_host, nullptr);
}

int bp_get_weights(const bp_net* net, float* w_host, int64_t n) {
  if (check_net(net)) return BP_EINVAL;
  if (!w_host) return fail(net, BP_EINVAL, "bp_get_weights: w_host is NULL");
  if (n != net->nweights) return fail(net, BP_EINVAL, "bp_get_weights: n != bp_num_weights");
  return copy_layers(net, net->W, nullptr, w_host);
}

int bp_set_momentum(bp_net* net, const float* v_host, int64_t n) {
  if (check_net(net)) return BP_EINVAL;
  if (!v_host) return fail(net, BP_EINVAL, "bp_set_momentum: v_host is NULL");
  if (n != net->nweights) return fail(net, BP_EINVAL, "bp_set_momentum: n != bp_num_weights");
  BP_HIP(net, hipStreamSynchronize(net->stream));
  return copy_layers(net, net->V, v_host, nullptr);
}

int bp_get_momentum(const bp_net* net, float* v_host, int64_t n) {
  if (check_net(net)) return BP_EINVAL;
  if (!v_host) return fail(net, BP_EINVAL, "bp_get_momentum: v_host is NULL");
  if (n != net->nweights) return fail(net, BP_EINVAL, "bp_get_momentum: n != bp_num_weights");
  return copy_layers(net, net->V, nullptr, v_host);
}

static int check_train(bp_net* net, const void* in, const float* targets, int64_t n, int32_t batch,
                       const char* who) {
  if (check_net(net)) return BP_EINVAL;
  std::string w(who);
  if (n < 0) return fail(net, BP_EINVAL, w + ": n_patterns < 0");
  if (n > ((int64_t)1 << 31) - 1) return fail(net, BP_EINVAL, w + ": n_patterns too large");
  if (batch < 1) return fail(net, BP_EINVAL, w + ": batch < 1");
  if (n > 0 && (!in || !targets)) return fail(net, BP_EINVAL, w + ": NULL input or target pointer");
  if (n > 0 && (!aligned_ptr(in, 4) || !aligned_ptr(targets, 4)))
    return fail(net, BP_EINVAL, w + ": pointers must be 4-byte aligned");
  return BP_OK;
}

int bp_train_batches(bp_net* net, const float* inputs_dev, const float* targets_dev, int64_t n_patterns,
                     int32_t batch, float lr, float momentum, double* sse_out) {
  int rc = check_train(net, inputs_dev, targets_dev, n_patterns, batch, "bp_train_batches");
  if (rc) return rc;
  BatchInput in;
  in.x = inputs_dev;
  return train(net, in, targets_dev, n_patterns, batch, lr, momentum, sse_out);
}

int bp_train_batches_noalloc(bp_net* net, const float* inputs_dev, const float* targets_dev, int64_t n_patterns,
                             int32_t batch, float lr, float momentum, double* sse_out) {
  int rc = check_train(net, inputs_dev, targets_dev, n_patterns, batch, "bp_train_batches_noalloc");
  if (rc) return rc;
  BatchInput in;
  in.x = inputs_dev;
  return train_noalloc(net, in, targets_dev, n_patterns, batch, lr, momentum, sse_out);
}

int bp_train_batches_onehot(bp_net* net, const int32_t* active_dev, int32_t n_active, const float* targets_dev,
                            int64_t n_patterns, int32_t batch, float lr, float momentum, double* sse_out) {
  int rc = check_train(net, active_dev, targets_dev, n_patterns, batch, "bp_train_batches_onehot");
  if (rc) return rc;
  if (n_active < 1 || n_active > net->n[0])
    return fail(net, BP_EINVAL, "bp_train_batches_onehot: n_active must be in [1, n_0]");
  BatchInput in;
  in.act = active_dev;
  in.n_active = n_active;
  return train(net, in, targets_dev, n_patterns, batch, lr, momentum, sse_out);
}

int bp_forward(bp_net* net, const float* inputs_dev, int64_t n_patterns, float* outputs_dev) {
  if (check_net(net)) return BP_EINVAL;
  if (n_patterns < 0 || n_patterns > ((int64_t)1 << 31) - 1)
    return fail(net, BP_EINVAL, "bp_forward: bad n_patterns");
  if (n_patterns > 0 && (!inputs_dev || !outputs_dev)) return fail(net, BP_EINVAL, "bp_forward: NULL pointer");
  BatchInput in;
  in.x = inputs_dev;
  return forward_only(net, in, n_patterns, outputs_dev);
}

int bp_forward_onehot(bp_net* net, const int32_t* active_dev, int32_t n_active, int64_t n_patterns,
                      float* outputs_dev) {
  if (check_net(net)) return BP_EINVAL;
  if (n_patterns < 0 || n_patterns > ((int64_t)1 << 31) - 1)
    return fail(net, BP_EINVAL, "bp_forward_onehot: bad n_patterns");
  if (n_patterns > 0 && (!active_dev || !outputs_dev))
    return fail(net, BP_EINVAL, "bp_forward_onehot: NULL pointer");
  if (n_active < 1 || n_active > net->n[0])
    return fail(net, BP_EINVAL, "bp_forward_onehot: n_active must be in [1, n_0]");
  BatchInput in;
  in.act = active_dev;
  in.n_active = n_active;
  return forward_only(net, in, n_patterns, outputs_dev);
}

int bp_set_graph_replay(bp_net* net, int on) {
  if (check_net(net)) return BP_EINVAL;
  BP_HIP(net, hipStreamSynchronize(net->stream));
  net->graph_on = on != 0;
  net->have_last = false;
  drop_graph(net);
  return BP_OK;
}

int bp_profile(bp_net* net, int on) {
  if (check_net(net)) return BP_EINVAL;
  if (on) {
    BP_HIP(net, hipStreamSynchronize(net->stream));
    for (auto& r : net->recs) {
      net->ev_pool.push_back(r.a);
      net->ev_pool.push_back(r.b);
    }
    net->recs.clear();
    for (int k = 0; k < BP_K_COUNT; ++k) {
      net->prof_n[k] = 0;
      net->prof_ms[k] = 0.0;
    }
  }
  net->prof = on != 0;
  return BP_OK;
}

int bp_profile_report(bp_net* net, int64_t* launches, double* ms, int32_t n_kinds) {
  if (check_net(net)) return BP_EINVAL;
  if (!launches || !ms || n_kinds < 0 || n_kinds > BP_K_COUNT)
    return fail(net, BP_EINVAL, "bp_profile_report: bad output arrays");
  BP_HIP(net, hipStreamSynchronize(net->stream));
  for (auto& r : net->recs) {
    float t = 0.f;
    BP_HIP(net, hipEventElapsedTime(&t, r.a, r.b));
    net->prof_n[r.kind] += 1;
    net->prof_ms[r.kind] += (double)t;
    net->ev_pool.push_back(r.a);
    net->ev_pool.push_back(r.b);
  }
  net->recs.clear();
  for (int k = 0; k < n_kinds; ++k) {
    launches[k] = net->prof_n[k];
    ms[k] = net->prof_ms[k];
  }
  return BP_OK;
}

int bp_set_context(bp_net* net, int32_t n_ctx, const int32_t* from_layer, const int32_t* from_unit) {
  if (check_net(net)) return BP_EINVAL;
  if (n_ctx < 0 || n_ctx > net->n[0]) return fail(net, BP_EINVAL, "bp_set_context: n_ctx must be in [0, n_0]");
  if (n_ctx > 0 && (!from_layer || !from_unit)) return fail(net, BP_EINVAL, "bp_set_context: NULL source arrays");
  if (n_ctx > 0 && net->L < 2) return fail(net, BP_EINVAL, "bp_set_context: the net has no hidden layer");
  for (int c = 0; c < n_ctx; ++c) {
    const int l = from_layer[c];
    if (l < 1 || l > net->L - 1 || l > bpk::kCtxMaxLayer || from_unit[c] < 0 || from_unit[c] >= net->n[l])
      return fail(net, BP_EINVAL, "bp_set_context: a source is not a hidden unit (layers 1 .. min(L-1, 8))");
  }
  BP_HIP(net, hipStreamSynchronize(net->stream));
  free_ptr(net->ctx_layer_dev);
  free_ptr(net->ctx_unit_dev);
  net->ctx_layer_dev = net->ctx_unit_dev = nullptr;
  net->n_ctx = 0;
  net->ctx_in_order = false;
  if (n_ctx > 0) {
    BP_HIP(net, hipMalloc(&net->ctx_layer_dev, sizeof(int32_t) * n_ctx));
    BP_HIP(net, hipMalloc(&net->ctx_unit_dev, sizeof(int32_t) * n_ctx));
    BP_HIP(net, hipMemcpy(net->ctx_layer_dev, from_layer, sizeof(int32_t) * n_ctx, hipMemcpyHostToDevice));
    BP_HIP(net, hipMemcpy(net->ctx_unit_dev, from_unit, sizeof(int32_t) * n_ctx, hipMemcpyHostToDevice));
  }
  net->n_ctx = n_ctx;
  net->ctx_in_order = n_ctx > 0;
  for (int c = 0; c < n_ctx; ++c)
    if (from_layer[c] != 1 || from_unit[c] != c) net->ctx_in_order = false;
  return BP_OK;
}

static int check_seq(bp_net* net, const void* X, const void* cont, int64_t T, int32_t S, const char* who) {
  std::string w(who);
  if (T < 0 || S < 1) return fail(net, BP_EINVAL, w + ": need n_steps >= 0 and n_streams >= 1");
  if (T * (int64_t)S > ((int64_t)1 << 31) - 1) return fail(net, BP_EINVAL, w + ": too many patterns");
  if (T > 0 && (!cont || (!X && net->n[0] > net->n_ctx))) return fail(net, BP_EINVAL, w + ": NULL pointer");
  if (T > 0 && (!aligned_ptr(X, 4) || !aligned_ptr(cont, 4)))
    return fail(net, BP_EINVAL, w + ": pointers must be 4-byte aligned");
  return BP_OK;
}

int bp_train_sequences(bp_net* net, const float* inputs_dev, const float* targets_dev, const float* cont_dev,
                       const float* mask_dev, int64_t n_steps, int32_t n_streams, int32_t steps_per_update, float lr,
                       float momentum, double* sse_out) {
  if (check_net(net)) return BP_EINVAL;
  int rc = check_seq(net, inputs_dev, cont_dev, n_steps, n_streams, "bp_train_sequences");
  if (rc) return rc;
  if (steps_per_update < 1) return fail(net, BP_EINVAL, "bp_train_sequences: steps_per_update < 1");
  if ((int64_t)steps_per_update * n_streams > ((int64_t)1 << 30))
    return fail(net, BP_EINVAL, "bp_train_sequences: steps_per_update x n_streams too large");
  if (n_steps > 0 && (!targets_dev || !mask_dev || !aligned_ptr(targets_dev, 4) || !aligned_ptr(mask_dev, 4)))
    return fail(net, BP_EINVAL, "bp_train_sequences: NULL or misaligned targets or mask");
  return train_sequences(net, inputs_dev, targets_dev, cont_dev, mask_dev, n_steps, n_streams, steps_per_update, lr,
                         momentum, sse_out);
}

int bp_forward_sequences(bp_net* net, const float* inputs_dev, const float* cont_dev, int64_t n_steps,
                         int32_t n_streams, float* outputs_dev) {
  if (check_net(net)) return BP_EINVAL;
  int rc = check_seq(net, inputs_dev, cont_dev, n_steps, n_streams, "bp_forward_sequences");
  if (rc) return rc;
  if (n_steps > 0 && !outputs_dev) return fail(net, BP_EINVAL, "bp_forward_sequences: outputs_dev is NULL");
  return forward_sequences(net, inputs_dev, cont_dev, n_steps, n_streams, outputs_dev);
}

int bp_set_sigmoid(bp_net* net, int32_t mode) {
  if (check_net(net)) return BP_EINVAL;
  if (mode != BP_SIGMOID_EXACT && mode != BP_SIGMOID_TABLE)
    return fail(net, BP_EINVAL, "bp_set_sigmoid: mode must be BP_SIGMOID_EXACT or BP_SIGMOID_TABLE");
  BP_HIP(net, hipStreamSynchronize(net->stream));
  if (mode == BP_SIGMOID_EXACT) {
    net->sig_tab = nullptr;
    ++net->gen;
    return BP_OK;
  }
  if (!net->sig_tab_mem) {
    // entry i: the logistic at -15 + 30 i / 255, evaluated in double (section 4.3)
    float host[256];
    for (int i = 0; i < 256; ++i) {
      const double x = -15.0 + 30.0 * (double)i / 255.0;
      host[i] = (float)(1.0 / (1.0 + std::exp(-x)));
    }
    BP_HIP(net, hipMalloc(&net->sig_tab_mem, sizeof(host)));
    BP_HIP(net, hipMemcpy(net->sig_tab_mem, host, sizeof(host), hipMemcpyHostToDevice));
  }
  net->sig_tab = net->sig_tab_mem;
  ++net->gen;
  return BP_OK;
}

int bp_set_fault_limit(bp_net* net, float limit) {
  if (check_net(net)) return BP_EINVAL;
  if (!(limit >= 0.f)) return fail(net, BP_EINVAL, "bp_set_fault_limit: limit must be >= 0");
  BP_HIP(net, hipStreamSynchronize(net->stream));
  if (!net->faults) BP_HIP(net, hipMalloc(&net->faults, sizeof(unsigned long long)));
  const unsigned long long zero = 0;
  BP_HIP(net, hipMemcpy(net->faults, &zero, sizeof(zero), hipMemcpyHostToDevice));
  net->fault_limit = limit;
  ++net->gen;
  return BP_OK;
}

int bp_get_fault_count(bp_net* net, int64_t* count) {
  if (check_net(net)) return BP_EINVAL;
  if (!count) return fail(net, BP_EINVAL, "bp_get_fault_count: count is NULL");
  unsigned long long c = 0;
  if (net->faults) {
    BP_HIP(net, hipMemcpyAsync(&c, net->faults, sizeof(c), hipMemcpyDeviceToHost, net->stream));
    BP_HIP(net, hipStreamSynchronize(net->stream));
  }
  *count = (int64_t)c;
  return BP_OK;
}

int bp_checkpoint_save(bp_net* net) {
  if (check_net(net)) return BP_EINVAL;
  return checkpoint_save(net);
}

int bp_checkpoint_restore(bp_net* net) {
  if (check_net(net)) return BP_EINVAL;
  if (!net->ckW) return fail(net, BP_EINVAL, "bp_checkpoint_restore: no checkpoint saved");
  return checkpoint_restore(net);
}

int bp_guard_config(bp_net* net, int32_t every, double jump) {
  if (check_net(net)) return BP_EINVAL;
  if (every < 1 || !(jump > 0.0)) return fail(net, BP_EINVAL, "bp_guard_config: need every >= 1 and jump > 0");
  const int rc = checkpoint_save(net);
  if (rc) return rc;
  net->guard = bp_net::Guard();
  net->guard.on = true;
  net->guard.every = every;
  net->guard.jump = jump;
  return BP_OK;
}

int bp_guard_epoch(bp_net* net, double sse, int32_t* rolled_back) {
  if (check_net(net)) return BP_EINVAL;
  if (!rolled_back) return fail(net, BP_EINVAL, "bp_guard_epoch: rolled_back is NULL");
  if (!net->guard.on) return fail(net, BP_EINVAL, "bp_guard_epoch: call bp_guard_config first");
  bp_net::Guard& g = net->guard;
  const int pos = g.since + 1;
  // a NaN error compares false: it counts as a jump
  const bool jumped = g.have_last && !(sse <= g.jump * g.last_sse);
  if (jumped && g.retry_at != pos) {
    const int rc = checkpoint_restore(net);
    if (rc) return rc;
    g.retry_at = pos;
    g.since = 0;
    g.have_last = g.ck_have;
    g.last_sse = g.ck_sse;
    *rolled_back = 1;
    return BP_OK;
  }
  // accepted (a jump that recurs at the epoch already rolled back is the
  // learning itself: the replay is deterministic)
  g.have_last = true;
  g.last_sse = sse;
  g.since = pos;
  if (g.since == g.every) {
    const int rc = checkpoint_save(net);
    if (rc) return rc;
    g.ck_have = true;
    g.ck_sse = sse;
    g.since = 0;
    g.retry_at = -1;
  }
  *rolled_back = 0;
  return BP_OK;
}

const char* bp_last_error(const bp_net* net) { return net ? net->err.c_str() : g_create_err.c_str(); }

}  // extern "C"
