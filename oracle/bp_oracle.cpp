/*
 * bp_oracle.cpp -- CPU oracle for pooled back-propagation.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load or run this file.  It shares no code,
 * header, table or helper with the HIP library, and the library never calls
 * it.
 *
 * It is a plain, slow, obviously correct implementation of what the paper's
 * simulator computes (Witbrock & Zagha, "An Implementation of
 * Back-Propagation Learning on GF11", CMU-CS-89-208):
 *
 *   forward   a_{l+1}[j] = sigma( W_l[n_l][j] + sum_i a_l[i] * W_l[i][j] )
 *             -- a unit's net input is the weighted sum of the activations
 *             feeding it (section 3); the always-on "true unit" feeds every
 *             non-input layer (section 6.3), stored as the last row of W_l;
 *             sigma(x) = 1 / (1 + e^-x) (section 3, footnote 4).
 *   error     e = t - y, reported error = sum over patterns and outputs of e^2
 *             ("summed squared difference", section 3 footnote 5; "total
 *             squared error", section 8).
 *   deltas    delta_L = e * y * (1 - y); for l = L-1 .. 1:
 *             delta_l[i] = a_l[i] (1 - a_l[i]) * sum_j W_l[i][j] delta_{l+1}[j]
 *             -- partial derivatives taken from the output weights backwards
 *             (section 3); input units get no back-propagated error (the
 *             backward cycle count of section 6.1 charges input connections
 *             one add and one multiply only); the bias row is not used.
 *   pooled    G_l[i][j] = sum over the patterns of a batch of
 *             a_l[i] * delta_{l+1}[j]  (bias row: sum of delta_{l+1}[j]),
 *             i.e. the weight changes of all patterns summed and applied once
 *             (sections 3 and 4.1).
 *   update    V_l = lr * G_l + momentum * V_l ;  W_l += V_l
 *             -- learning rate and momentum applied to the summed change,
 *             with the previous change kept (sections 6.2.1 and 9).
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes): the batch change is the SUM (not the mean) over patterns;
 * delta carries no factor 2 (the gradient is that of half the squared error,
 * while the reported error has no half); momentum in the classical form above;
 * V starts at zero and persists across batches and epochs; a short last batch
 * is applied like any other; patterns are taken in order; the exact logistic.
 *
 * Precision: the net is templated on the STORAGE type Real (float or double).
 * Weights, momentum, activations and deltas are stored as Real; every sum
 * (net input, delta dot product, batch sum, error) uses a double accumulator,
 * sigma is evaluated in double and then rounded to Real.  The double instance
 * is the plain definition; the float instance rounds at the storage points a
 * float32 implementation has, which measures the float32 noise floor.
 *
 * Options (off by default):
 *   table sigmoid   the second of the two sigmoid evaluations of section 4.3:
 *             inputs outside [-15, 15] are taken to the ends of that range, the
 *             range is mapped onto [0, 255] by an add and a multiply, the
 *             integer part of the result indexes a 256-entry table of the
 *             logistic at equally spaced points of [-15, 15], and the
 *             fractional part interpolates linearly to the next entry.  The
 *             index (an integer that floating point decides) is computed in
 *             single precision, the interpolation in double.  Table entries
 *             are Real.
 *   range check     each summed change G (the "total weight change" of section
 *             8) outside [-limit, limit], or not a number, is set to zero
 *             before the update and counted as a fault (section 8).
 *   recurrence      Elman nets (section 10.5): the last n_ctx input units are
 *             context units; before each pattern of a sequence, context unit
 *             c receives a copy of unit ctx_unit[c] of hidden layer
 *             ctx_layer[c] as it was after the previous pattern of the same
 *             sequence, multiplied by the pattern's continuation flag (1 to
 *             continue a sequence, 0 at a sequence start).  Sequences are
 *             handled in parallel across streams: pattern (t, s) is step t
 *             of stream s, and the error of every pattern is multiplied by
 *             its mask flag (0 for the padding after a stream's last
 *             sequence), so a masked pattern back-propagates nothing.  A
 *             pooled update follows every `steps_per_update` steps (all
 *             streams); context values are inputs to the change like any
 *             other input (no propagation through time).  Context starts at
 *             zero in every call.
 *   checkpoint      one stored copy of W and V (section 10.4), and a guard that
 *             saves it every `every` accepted epochs and restores it when an
 *             epoch's error exceeds `jump` times the last accepted epoch's
 *             error.  A jump that recurs at the same epoch after a rollback is
 *             accepted: the training is deterministic, so a recurring jump is
 *             the learning itself, not a transient fault.
 *
 * Parallelism (OpenMP) only splits independent work: patterns in the forward
 * and backward passes, and output rows in the batch sum, where every element
 * is still accumulated over the patterns in pattern order.  Results do not
 * depend on the thread count.
 */
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <type_traits>
#include <vector>

#include <omp.h>

namespace {

double sigmoid(double z) { return 1.0 / (1.0 + std::exp(-z)); }

constexpr int kTableSize = 256;     // entries of the sigmoid table (section 4.3, figure 3)
constexpr double kTableEnd = 15.0;  // the table covers [-15, 15]

// Checkpoint guard state (see the header comment).
struct Guard {
  bool on = false;
  int every = 1;
  double jump = 0.0;
  int since = 0;            // epochs accepted since the checkpoint
  int retry_at = -1;        // epoch (counted from the checkpoint) that was already rolled back
  bool have_last = false;
  double last_sse = 0.0;    // error of the last accepted epoch
  bool ck_have = false;
  double ck_sse = 0.0;      // error of the epoch at which the checkpoint was taken
};

template <typename Real>
struct Net {
  int L = 0;                    // number of weight layers
  std::vector<int> n;           // n[0..L]
  std::vector<int64_t> off;     // offset of W_l in the flat arrays
  int64_t total = 0;            // sum (n_l + 1) * n_{l+1}
  std::vector<Real> W, V;       // flat, layer l row-major (n_l + 1) x n_{l+1}
  int sig_mode = 0;             // 0: exact logistic, 1: table
  std::vector<Real> table;      // sigmoid table, kTableSize entries
  double fault_limit = 0.0;     // > 0: range check of the summed changes
  int64_t faults = 0;
  std::vector<Real> ckW, ckV;   // checkpoint
  Guard guard;
  std::vector<int> ctx_layer, ctx_unit;   // Elman context: source of context unit c

  const Real* w(int l) const { return W.data() + off[l]; }
  Real* w(int l) { return W.data() + off[l]; }
  Real* v(int l) { return V.data() + off[l]; }

  // The unit nonlinearity in use, evaluated on a net input z.
  double act(double z) const {
    if (sig_mode == 0) return sigmoid(z);
    if (std::isnan(z)) return z;
    float zf = (float)z;
    if (zf < (float)-kTableEnd) zf = (float)-kTableEnd;
    if (zf > (float)kTableEnd) zf = (float)kTableEnd;
    // [-15, 15] -> [0, 255]: add 15, multiply by 255 / 30 = 8.5 (exact in float)
    const float x1 = (zf + (float)kTableEnd) * (float)((kTableSize - 1) / (2.0 * kTableEnd));
    const int i = (int)std::floor(x1);
    if (i >= kTableSize - 1) return (double)table[kTableSize - 1];
    const double f = (double)x1 - (double)i;
    return (double)table[i] + f * ((double)table[i + 1] - (double)table[i]);
  }
};

// Entry i of the sigmoid table: the logistic at -15 + 30 i / 255.
template <typename Real>
void build_table(Net<Real>& net) {
  net.table.assign(kTableSize, (Real)0);
  for (int i = 0; i < kTableSize; ++i)
    net.table[i] = (Real)sigmoid(-kTableEnd + 2.0 * kTableEnd * (double)i / (double)(kTableSize - 1));
}

// Per-batch state: activations a_0..a_L and deltas delta_1..delta_L of every
// pattern, stored row by row ([pattern][unit]).
template <typename Real>
struct BatchState {
  std::vector<std::vector<Real>> a;    // a[l] : rows x n_l
  std::vector<std::vector<Real>> d;    // d[l] : rows x n_l (l >= 1)
  std::vector<double> sse_p;           // squared error of each pattern
  // One-hot inputs (section 6.3): only the active input units take part in the
  // first layer, in the forward sum and in the summed change (inactive units
  // are 0 and contribute nothing; this differs from a dense 0/1 product only
  // when a weight or a delta is not finite, where 0 * NaN would be NaN).
  bool sparse0 = false;
};

// Forward pass of one pattern: a[0] already holds the inputs.
template <typename Real>
void forward_pattern(const Net<Real>& net, std::vector<Real*>& a, bool sparse0) {
  for (int l = 0; l < net.L; ++l) {
    const int n_in = net.n[l], n_out = net.n[l + 1];
    const Real* W = net.w(l);
    std::vector<double> acc(n_out);
    for (int j = 0; j < n_out; ++j) acc[j] = (double)W[(int64_t)n_in * n_out + j];  // true unit
    for (int i = 0; i < n_in; ++i) {
      const double ai = (double)a[l][i];
      if (l == 0 && sparse0 && ai == 0.0) continue;
      const Real* row = W + (int64_t)i * n_out;
      for (int j = 0; j < n_out; ++j) acc[j] += ai * (double)row[j];
    }
    for (int j = 0; j < n_out; ++j) a[l + 1][j] = (Real)net.act(acc[j]);
  }
}

// Deltas of one pattern from its activations and target; returns sum e^2.
template <typename Real>
double backward_pattern(const Net<Real>& net, Real* const* a, Real* const* d, const float* t, double mask = 1.0) {
  const int L = net.L, nL = net.n[L];
  double sse = 0.0;
  for (int k = 0; k < nL; ++k) {
    const double y = (double)a[L][k];
    const double e = mask * ((double)t[k] - y);     // the error times the pattern's mask flag
    sse += e * e;
    d[L][k] = (Real)(e * y * (1.0 - y));
  }
  for (int l = L - 1; l >= 1; --l) {
    const int n_in = net.n[l], n_out = net.n[l + 1];
    const Real* W = net.w(l);
    for (int i = 0; i < n_in; ++i) {
      const Real* row = W + (int64_t)i * n_out;
      double s = 0.0;
      for (int j = 0; j < n_out; ++j) s += (double)row[j] * (double)d[l + 1][j];
      const double ai = (double)a[l][i];
      d[l][i] = (Real)(ai * (1.0 - ai) * s);
    }
  }
  return sse;
}

// Forward and backward passes for `rows` patterns whose inputs are already in
// st.a[0].  With t == nullptr only the forward pass runs.
template <typename Real>
void run_batch(const Net<Real>& net, BatchState<Real>& st, int64_t rows, const float* t) {
  const int L = net.L;
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < rows; ++p) {
    std::vector<Real*> a(L + 1), d(L + 1, nullptr);
    for (int l = 0; l <= L; ++l) a[l] = st.a[l].data() + p * net.n[l];
    forward_pattern(net, a, st.sparse0);
    if (t) {
      for (int l = 1; l <= L; ++l) d[l] = st.d[l].data() + p * net.n[l];
      st.sse_p[p] = backward_pattern(net, a.data(), d.data(), t + p * net.n[L]);
    }
  }
}

// G_l[i][j] = sum_p a_l[p][i] * delta_{l+1}[p][j]; row n_l (true unit) = sum_p delta.
// Rows are split among threads; each element sums the patterns in order.
template <typename Real>
void batch_sum(const Net<Real>& net, const BatchState<Real>& st, int64_t rows, double* G) {
  for (int l = 0; l < net.L; ++l) {
    const int n_in = net.n[l], n_out = net.n[l + 1];
    double* Gl = G + net.off[l];
    const Real* A = st.a[l].data();
    const Real* D = st.d[l + 1].data();
#pragma omp parallel
    {
      const int nt = omp_get_num_threads(), tid = omp_get_thread_num();
      const int r0 = (int)((int64_t)(n_in + 1) * tid / nt);
      const int r1 = (int)((int64_t)(n_in + 1) * (tid + 1) / nt);
      for (int i = r0; i < r1; ++i)
        for (int j = 0; j < n_out; ++j) Gl[(int64_t)i * n_out + j] = 0.0;
      for (int64_t p = 0; p < rows; ++p) {
        const Real* dp = D + p * n_out;
        for (int i = r0; i < r1; ++i) {
          const double ai = (i < n_in) ? (double)A[p * n_in + i] : 1.0;
          if (l == 0 && st.sparse0 && ai == 0.0) continue;
          double* g = Gl + (int64_t)i * n_out;
          for (int j = 0; j < n_out; ++j) g[j] += ai * (double)dp[j];
        }
      }
    }
  }
}

template <typename Real>
void apply_update(Net<Real>& net, const double* G, double lr, double mom) {
  const int64_t total = net.total;
  Real* W = net.W.data();
  Real* V = net.V.data();
  const double limit = net.fault_limit;
  int64_t faults = 0;
#pragma omp parallel for schedule(static) reduction(+ : faults)
  for (int64_t k = 0; k < total; ++k) {
    double g = G[k];
    if (limit > 0.0 && !(std::fabs(g) <= limit)) {   // section 8: out of range -> zero, count
      g = 0.0;
      ++faults;
    }
    const Real v = (Real)(lr * g + mom * (double)V[k]);
    V[k] = v;
    W[k] = (Real)((double)W[k] + (double)v);
  }
  net.faults += faults;
}

template <typename Real>
void save_checkpoint(Net<Real>& net) {
  net.ckW = net.W;
  net.ckV = net.V;
}

template <typename Real>
int restore_checkpoint(Net<Real>& net) {
  if (net.ckW.size() != net.W.size()) return -1;
  net.W = net.ckW;
  net.V = net.ckV;
  return 0;
}

template <typename Real>
void guard_config(Net<Real>& net, int every, double jump) {
  net.guard = Guard();
  net.guard.on = true;
  net.guard.every = every;
  net.guard.jump = jump;
  save_checkpoint(net);
}

// 0: epoch accepted; 1: rolled back to the checkpoint.
template <typename Real>
int guard_epoch(Net<Real>& net, double sse) {
  Guard& g = net.guard;
  const int pos = g.since + 1;
  const bool jumped = g.have_last && !(sse <= g.jump * g.last_sse);
  if (jumped && g.retry_at != pos) {
    restore_checkpoint(net);
    g.retry_at = pos;
    g.since = 0;
    g.have_last = g.ck_have;
    g.last_sse = g.ck_sse;
    return 1;
  }
  g.have_last = true;
  g.last_sse = sse;
  g.since = pos;
  if (g.since == g.every) {
    save_checkpoint(net);
    g.ck_have = true;
    g.ck_sse = sse;
    g.since = 0;
    g.retry_at = -1;
  }
  return 0;
}

template <typename Real>
void alloc_state(const Net<Real>& net, BatchState<Real>& st, int64_t rows) {
  st.a.assign(net.L + 1, {});
  st.d.assign(net.L + 1, {});
  for (int l = 0; l <= net.L; ++l) {
    st.a[l].assign((size_t)(rows * net.n[l]), (Real)0);
    if (l >= 1) st.d[l].assign((size_t)(rows * net.n[l]), (Real)0);
  }
  st.sse_p.assign((size_t)rows, 0.0);
}

// Input rows of patterns [p0, p0 + rows): dense copy or one-hot expansion.
template <typename Real>
void load_inputs(const Net<Real>& net, BatchState<Real>& st, int64_t p0, int64_t rows,
                 const float* x, const int32_t* act, int n_active) {
  const int n0 = net.n[0];
  Real* a0 = st.a[0].data();
  st.sparse0 = (x == nullptr);
  if (x) {
    for (int64_t p = 0; p < rows; ++p)
      for (int i = 0; i < n0; ++i) a0[p * n0 + i] = (Real)x[(p0 + p) * n0 + i];
  } else {
    std::memset(a0, 0, sizeof(Real) * (size_t)(rows * n0));
    for (int64_t p = 0; p < rows; ++p)
      for (int k = 0; k < n_active; ++k) a0[p * n0 + act[(p0 + p) * n_active + k]] = (Real)1;
  }
}

// Checks one-hot indices: in range and distinct within each pattern.
int check_active(const int32_t* act, int n_active, int64_t n, int n0) {
  if (n > 0 && (!act || n_active < 1 || n_active > n0)) return -1;
  for (int64_t p = 0; p < n; ++p) {
    const int32_t* r = act + p * n_active;
    for (int k = 0; k < n_active; ++k) {
      if (r[k] < 0 || r[k] >= n0) return -1;
      for (int q = 0; q < k; ++q)
        if (r[q] == r[k]) return -1;
    }
  }
  return 0;
}

template <typename Real>
int train_epoch(Net<Real>& net, const float* x, const int32_t* act, int n_active, const float* t,
                int64_t n, int32_t batch, double lr, double mom, double* sse, double* batch_sse) {
  if (batch < 1 || n < 0 || (n > 0 && !t) || (n > 0 && !x && !act)) return -1;
  if (!x && check_active(act, n_active, n, net.n[0])) return -1;
  BatchState<Real> st;
  alloc_state(net, st, std::min<int64_t>(batch, std::max<int64_t>(n, 1)));
  std::vector<double> G((size_t)net.total);
  double total = 0.0;
  int64_t b = 0;
  for (int64_t p0 = 0; p0 < n; p0 += batch, ++b) {
    const int64_t rows = std::min<int64_t>(batch, n - p0);
    load_inputs(net, st, p0, rows, x, act, n_active);
    run_batch(net, st, rows, t + p0 * net.n[net.L]);
    double bs = 0.0;
    for (int64_t p = 0; p < rows; ++p) bs += st.sse_p[p];
    batch_sum(net, st, rows, G.data());
    apply_update(net, G.data(), lr, mom);
    if (batch_sse) batch_sse[b] = bs;
    total += bs;
  }
  if (sse) *sse = total;
  return 0;
}

// Elman training over n_steps x n_streams patterns (see the header comment).
// x: [n_steps][n_streams][n_ext], t: [n_steps][n_streams][n_L],
// cont, mask: [n_steps][n_streams]; window_sse receives each update's error.
// With train == false only the forward passes run and y (if given) receives
// the outputs [n_steps][n_streams][n_L].
template <typename Real>
int train_sequences(Net<Real>& net, const float* x, const float* t, const float* cont, const float* mask,
                    int64_t n_steps, int n_streams, int steps_per_update, double lr, double mom, double* sse,
                    double* window_sse, double* y, bool train) {
  const int L = net.L, n0 = net.n[0], nL = net.n[L];
  const int n_ctx = (int)net.ctx_layer.size(), n_ext = n0 - n_ctx;
  if (n_steps < 0 || n_streams < 1 || steps_per_update < 1 || (n_steps > 0 && (!x || !cont))) return -1;
  if (train && n_steps > 0 && (!t || !mask)) return -1;
  if (n_ctx > 0 && L < 2) return -1;
  const int S = n_streams;
  std::vector<double> prev((size_t)S * n_ctx, 0.0);   // context sources after the previous step
  const int64_t rows_max = (int64_t)std::min<int64_t>(steps_per_update, std::max<int64_t>(n_steps, 1)) * S;
  BatchState<Real> st;
  alloc_state(net, st, rows_max);
  std::vector<double> G(train ? (size_t)net.total : 0);
  double total = 0.0;
  int64_t wi = 0;
  for (int64_t w0 = 0; w0 < n_steps; w0 += steps_per_update, ++wi) {
    const int steps = (int)std::min<int64_t>(steps_per_update, n_steps - w0);
    for (int k = 0; k < steps; ++k) {
      const int64_t g = w0 + k;
#pragma omp parallel for schedule(static)
      for (int s = 0; s < S; ++s) {
        const int64_t p = (int64_t)k * S + s;            // row within the window
        const int64_t q = g * S + s;                     // pattern (step g, stream s)
        std::vector<Real*> a(L + 1), d(L + 1, nullptr);
        for (int l = 0; l <= L; ++l) a[l] = st.a[l].data() + p * net.n[l];
        for (int i = 0; i < n_ext; ++i) a[0][i] = (Real)x[q * n_ext + i];
        for (int c = 0; c < n_ctx; ++c) a[0][n_ext + c] = (Real)((double)cont[q] * prev[(size_t)s * n_ctx + c]);
        forward_pattern(net, a, false);
        if (train) {
          for (int l = 1; l <= L; ++l) d[l] = st.d[l].data() + p * net.n[l];
          st.sse_p[p] = backward_pattern(net, a.data(), d.data(), t + q * nL, (double)mask[q]);
        } else if (y) {
          for (int j = 0; j < nL; ++j) y[q * nL + j] = (double)a[L][j];
        }
        for (int c = 0; c < n_ctx; ++c) prev[(size_t)s * n_ctx + c] = (double)a[net.ctx_layer[c]][net.ctx_unit[c]];
      }
    }
    if (!train) continue;
    const int64_t rows = (int64_t)steps * S;
    double bs = 0.0;
    for (int64_t p = 0; p < rows; ++p) bs += st.sse_p[p];
    batch_sum(net, st, rows, G.data());
    apply_update(net, G.data(), lr, mom);
    if (window_sse) window_sse[wi] = bs;
    total += bs;
  }
  if (sse) *sse = total;
  return 0;
}

template <typename Real>
int gradient(Net<Real>& net, const float* x, const int32_t* act, int n_active, const float* t,
             int64_t n, double* G, double* sse) {
  if (n < 1 || !t || !G || (!x && !act)) return -1;
  if (!x && check_active(act, n_active, n, net.n[0])) return -1;
  BatchState<Real> st;
  alloc_state(net, st, n);
  load_inputs(net, st, 0, n, x, act, n_active);
  run_batch(net, st, n, t);
  batch_sum(net, st, n, G);
  if (sse) {
    double s = 0.0;
    for (int64_t p = 0; p < n; ++p) s += st.sse_p[p];
    *sse = s;
  }
  return 0;
}

template <typename Real>
int forward(Net<Real>& net, const float* x, const int32_t* act, int n_active, int64_t n, double* y) {
  if (n < 0 || (n > 0 && (!y || (!x && !act)))) return -1;
  if (!x && check_active(act, n_active, n, net.n[0])) return -1;
  if (n == 0) return 0;
  BatchState<Real> st;
  alloc_state(net, st, n);
  load_inputs(net, st, 0, n, x, act, n_active);
  run_batch(net, st, n, nullptr);
  const int nL = net.n[net.L];
  for (int64_t k = 0; k < n * nL; ++k) y[k] = (double)st.a[net.L][k];
  return 0;
}

// Activations a_1..a_L and deltas delta_1..delta_L of a batch at the current
// weights, each layer as [n][n_l] (concatenated over l = 1..L).
template <typename Real>
int batch_state(Net<Real>& net, const float* x, const int32_t* act, int n_active, const float* t,
                int64_t n, double* acts, double* deltas) {
  if (n < 1 || !t || (!x && !act)) return -1;
  if (!x && check_active(act, n_active, n, net.n[0])) return -1;
  BatchState<Real> st;
  alloc_state(net, st, n);
  load_inputs(net, st, 0, n, x, act, n_active);
  run_batch(net, st, n, t);
  int64_t o = 0;
  for (int l = 1; l <= net.L; ++l) {
    for (int64_t k = 0; k < n * net.n[l]; ++k, ++o) {
      if (acts) acts[o] = (double)st.a[l][k];
      if (deltas) deltas[o] = (double)st.d[l][k];
    }
  }
  return 0;
}

}  // namespace

extern "C" {

struct orc_net {
  int bits;             // 32 or 64: storage precision
  Net<float> f;
  Net<double> d;
};

static bool init_shape(std::vector<int>& n, std::vector<int64_t>& off, int64_t& total, int& L,
                       const int32_t* sizes, int32_t n_sizes) {
  if (!sizes || n_sizes < 2) return false;
  L = n_sizes - 1;
  n.assign(sizes, sizes + n_sizes);
  for (int v : n)
    if (v < 1) return false;
  off.assign(L, 0);
  total = 0;
  for (int l = 0; l < L; ++l) {
    off[l] = total;
    total += (int64_t)(n[l] + 1) * n[l + 1];
  }
  return true;
}

orc_net* orc_create(const int32_t* sizes, int32_t n_sizes, int32_t storage_bits) {
  if (storage_bits != 32 && storage_bits != 64) return nullptr;
  orc_net* h = new orc_net();
  h->bits = storage_bits;
  bool ok = storage_bits == 32 ? init_shape(h->f.n, h->f.off, h->f.total, h->f.L, sizes, n_sizes)
                               : init_shape(h->d.n, h->d.off, h->d.total, h->d.L, sizes, n_sizes);
  if (!ok) {
    delete h;
    return nullptr;
  }
  if (storage_bits == 32) {
    h->f.W.assign((size_t)h->f.total, 0.f);
    h->f.V.assign((size_t)h->f.total, 0.f);
  } else {
    h->d.W.assign((size_t)h->d.total, 0.0);
    h->d.V.assign((size_t)h->d.total, 0.0);
  }
  return h;
}

void orc_destroy(orc_net* h) { delete h; }

int64_t orc_num_weights(const orc_net* h) { return h->bits == 32 ? h->f.total : h->d.total; }

void orc_set_threads(int32_t n) {
  if (n > 0) omp_set_num_threads(n);
}

int32_t orc_get_threads(void) { return omp_get_max_threads(); }

#define ORC_DISPATCH(h, call) ((h)->bits == 32 ? call((h)->f) : call((h)->d))

int orc_set_weights(orc_net* h, const double* w, int64_t n) {
  if (!h || !w || n != orc_num_weights(h)) return -1;
  auto set = [&](auto& net) {
    using R = typename std::decay<decltype(net.W[0])>::type;
    for (int64_t k = 0; k < n; ++k) {
      net.W[k] = (R)w[k];
      net.V[k] = (R)0;
    }
    return 0;
  };
  return ORC_DISPATCH(h, set);
}

int orc_get_weights(const orc_net* h, double* w, int64_t n) {
  if (!h || !w || n != orc_num_weights(h)) return -1;
  for (int64_t k = 0; k < n; ++k) w[k] = h->bits == 32 ? (double)h->f.W[k] : h->d.W[k];
  return 0;
}

int orc_set_momentum(orc_net* h, const double* v, int64_t n) {
  if (!h || !v || n != orc_num_weights(h)) return -1;
  for (int64_t k = 0; k < n; ++k) {
    if (h->bits == 32) h->f.V[k] = (float)v[k];
    else h->d.V[k] = v[k];
  }
  return 0;
}

int orc_get_momentum(const orc_net* h, double* v, int64_t n) {
  if (!h || !v || n != orc_num_weights(h)) return -1;
  for (int64_t k = 0; k < n; ++k) v[k] = h->bits == 32 ? (double)h->f.V[k] : h->d.V[k];
  return 0;
}

// Sigmoid evaluation: 0 exact logistic, 1 the 256-entry table (section 4.3).
int orc_set_sigmoid(orc_net* h, int32_t mode) {
  if (!h || (mode != 0 && mode != 1)) return -1;
  auto f = [&](auto& net) {
    net.sig_mode = mode;
    if (mode == 1) build_table(net);
    return 0;
  };
  return ORC_DISPATCH(h, f);
}

// The net's unit nonlinearity at each z[k] (for checking it on its own).
int orc_eval_sigmoid(const orc_net* h, const double* z, int64_t n, double* y) {
  if (!h || n < 0 || (n > 0 && (!z || !y))) return -1;
  for (int64_t k = 0; k < n; ++k) y[k] = h->bits == 32 ? (double)(float)h->f.act(z[k]) : h->d.act(z[k]);
  return 0;
}

// Range check of the summed changes (section 8): limit > 0 enables, 0 disables; resets the count.
int orc_set_fault_limit(orc_net* h, double limit) {
  if (!h || !(limit >= 0.0)) return -1;
  auto f = [&](auto& net) {
    net.fault_limit = limit;
    net.faults = 0;
    return 0;
  };
  return ORC_DISPATCH(h, f);
}

int64_t orc_fault_count(const orc_net* h) { return !h ? -1 : (h->bits == 32 ? h->f.faults : h->d.faults); }

int orc_checkpoint_save(orc_net* h) {
  if (!h) return -1;
  auto f = [&](auto& net) {
    save_checkpoint(net);
    return 0;
  };
  return ORC_DISPATCH(h, f);
}

int orc_checkpoint_restore(orc_net* h) {
  if (!h) return -1;
  auto f = [&](auto& net) { return restore_checkpoint(net); };
  return ORC_DISPATCH(h, f);
}

int orc_guard_config(orc_net* h, int32_t every, double jump) {
  if (!h || every < 1 || !(jump > 0.0)) return -1;
  auto f = [&](auto& net) {
    guard_config(net, every, jump);
    return 0;
  };
  return ORC_DISPATCH(h, f);
}

int orc_guard_epoch(orc_net* h, double sse) {
  if (!h) return -1;
  auto f = [&](auto& net) { return net.guard.on ? guard_epoch(net, sse) : -1; };
  return ORC_DISPATCH(h, f);
}

// Elman context (section 10.5): context unit c (input unit n_0 - n_ctx + c)
// copies unit from_unit[c] of hidden layer from_layer[c] (1 <= layer <= L-1).
// n_ctx == 0 removes the context.
int orc_set_context(orc_net* h, int32_t n_ctx, const int32_t* from_layer, const int32_t* from_unit) {
  if (!h || n_ctx < 0 || (n_ctx > 0 && (!from_layer || !from_unit))) return -1;
  auto f = [&](auto& net) {
    if (n_ctx > net.n[0] || (n_ctx > 0 && net.L < 2)) return -1;
    for (int c = 0; c < n_ctx; ++c)
      if (from_layer[c] < 1 || from_layer[c] > net.L - 1 || from_unit[c] < 0 || from_unit[c] >= net.n[from_layer[c]])
        return -1;
    net.ctx_layer.assign(from_layer, from_layer + n_ctx);
    net.ctx_unit.assign(from_unit, from_unit + n_ctx);
    return 0;
  };
  return ORC_DISPATCH(h, f);
}

int orc_train_sequences(orc_net* h, const float* x, const float* t, const float* cont, const float* mask,
                        int64_t n_steps, int32_t n_streams, int32_t steps_per_update, double lr, double mom,
                        double* sse, double* window_sse) {
  if (!h) return -1;
  auto f = [&](auto& net) {
    return train_sequences(net, x, t, cont, mask, n_steps, n_streams, steps_per_update, lr, mom, sse, window_sse,
                           nullptr, true);
  };
  return ORC_DISPATCH(h, f);
}

// Outputs y [n_steps][n_streams][n_L] of the sequences at the current weights (no update).
int orc_forward_sequences(orc_net* h, const float* x, const float* cont, int64_t n_steps, int32_t n_streams,
                          double* y) {
  if (!h || (n_steps > 0 && !y)) return -1;
  auto f = [&](auto& net) {
    return train_sequences(net, x, nullptr, cont, nullptr, n_steps, n_streams, 1, 0.0, 0.0, nullptr, nullptr, y,
                           false);
  };
  return ORC_DISPATCH(h, f);
}

int orc_forward(orc_net* h, const float* x, int64_t n, double* y) {
  if (!h || (n > 0 && !x)) return -1;
  auto f = [&](auto& net) { return forward(net, x, nullptr, 0, n, y); };
  return ORC_DISPATCH(h, f);
}

int orc_forward_onehot(orc_net* h, const int32_t* act, int32_t n_active, int64_t n, double* y) {
  if (!h || (n > 0 && !act)) return -1;
  auto f = [&](auto& net) { return forward(net, (const float*)nullptr, act, n_active, n, y); };
  return ORC_DISPATCH(h, f);
}

int orc_gradient(orc_net* h, const float* x, const float* t, int64_t n, double* G, double* sse) {
  if (!h || !x) return -1;
  auto f = [&](auto& net) { return gradient(net, x, nullptr, 0, t, n, G, sse); };
  return ORC_DISPATCH(h, f);
}

int orc_gradient_onehot(orc_net* h, const int32_t* act, int32_t n_active, const float* t, int64_t n,
                        double* G, double* sse) {
  if (!h || !act) return -1;
  auto f = [&](auto& net) { return gradient(net, (const float*)nullptr, act, n_active, t, n, G, sse); };
  return ORC_DISPATCH(h, f);
}

int orc_batch_state(orc_net* h, const float* x, const float* t, int64_t n, double* acts, double* deltas) {
  if (!h || !x) return -1;
  auto f = [&](auto& net) { return batch_state(net, x, nullptr, 0, t, n, acts, deltas); };
  return ORC_DISPATCH(h, f);
}

int orc_train_epoch(orc_net* h, const float* x, const float* t, int64_t n, int32_t batch, double lr,
                    double mom, double* sse, double* batch_sse) {
  if (!h || (n > 0 && !x)) return -1;
  auto f = [&](auto& net) { return train_epoch(net, x, nullptr, 0, t, n, batch, lr, mom, sse, batch_sse); };
  return ORC_DISPATCH(h, f);
}

int orc_train_epoch_onehot(orc_net* h, const int32_t* act, int32_t n_active, const float* t, int64_t n,
                           int32_t batch, double lr, double mom, double* sse, double* batch_sse) {
  if (!h || (n > 0 && !act)) return -1;
  auto f = [&](auto& net) {
    return train_epoch(net, (const float*)nullptr, act, n_active, t, n, batch, lr, mom, sse, batch_sse);
  };
  return ORC_DISPATCH(h, f);
}

}  // extern "C"
