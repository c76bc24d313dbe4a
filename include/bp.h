/*
 * bp.h -- C-ABI of libbp.so: pooled back-propagation for fully connected
 * sigmoid nets, fp32, on one MI355X (gfx950).
 *
 * The method (Witbrock & Zagha, "An Implementation of Back-Propagation
 * Learning on GF11", CMU-CS-89-208):
 *   - forward: each unit takes the weighted sum of the units feeding it plus
 *     the weight from the always-on "true unit", then the logistic
 *     1/(1+e^-x) (section 3 and footnote 4; true unit: section 6.3);
 *   - error: summed squared difference of targets and outputs (section 3
 *     footnote 5, section 8);
 *   - backward: deltas from the output layer back to the first hidden layer;
 *     the input layer gets none (section 3; the cycle counts of section 6.1);
 *   - pooled update: the weight changes of all patterns of a batch are summed
 *     and applied once, with learning rate and momentum (sections 3, 4.1,
 *     6.2.1 and 9):  V = lr * G + momentum * V;  W += V,
 *     G[i][j] = sum over the batch of a_l[i] * delta_{l+1}[j].
 *
 * Layer sizes n_0 .. n_L (n_layers = L + 1 >= 2 entries).  Weight layout for
 * bp_set_weights / bp_get_weights / bp_*_momentum: the concatenation over
 * l = 0 .. L-1 of W_l, each (n_l + 1) x n_{l+1} row-major, row i = input unit
 * i, last row = the true unit (bias).  Its length is the paper's connection
 * count, sum (n_l + 1) * n_{l+1} (13,826 for the 203-60-26 NETtalk net).
 *
 * Ownership: the net owns its weights, momentum and workspace (device
 * memory).  Callers own every buffer they pass; "_dev" pointers are device
 * memory, contiguous row-major; "_host" pointers are host memory.
 *
 * Errors: every entry point returns BP_OK or a negative code; nothing throws
 * across this boundary.  Arguments are checked on the host before any device
 * work, so a BP_EINVAL return leaves the net unchanged.  BP_EDEVICE reports a
 * HIP runtime error; weights and momentum are then undefined until the next
 * bp_set_weights.  bp_last_error gives the message of the last failure.
 *
 * Streams: work is enqueued on the net's stream (bp_set_stream; default: the
 * null stream).  Train and forward calls return once the work is enqueued,
 * except that a non-NULL sse_out waits for the result.  A net is not
 * thread-safe; distinct nets are independent.
 */
#ifndef BP_H
#define BP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct bp_net bp_net;

enum {
  BP_OK = 0,
  BP_EINVAL = -1,   /* bad argument; nothing was done */
  BP_ENOMEM = -2,   /* device allocation failed */
  BP_EDEVICE = -3   /* HIP runtime error */
};

/* Creates a net with layer sizes layer_sizes[0 .. n_layers-1] (each >= 1 and
 * <= 2^24, n_layers >= 2; host array, read during the call) on the current
 * HIP device: a fully connected feed-forward net given by its topology, as
 * the paper's simulator builds its code from a topology file (section 2),
 * each non-input layer also fed by the true unit (section 6.3).  Weights and
 * momentum start at zero.  *out receives the handle (NULL on failure); the
 * caller releases it with bp_destroy.  BP_EINVAL for a NULL out or
 * layer_sizes, or sizes out of range; BP_ENOMEM / BP_EDEVICE if the device
 * allocation fails (nothing is left allocated). */
int bp_create(const int32_t* layer_sizes, int32_t n_layers, bp_net** out);

/* Frees the net and its device memory after its stream has drained.  NULL is a no-op. */
void bp_destroy(bp_net* net);

/* Sets the HIP stream (a hipStream_t, e.g. torch.cuda.current_stream().cuda_stream)
 * all later work of this net is enqueued on.  NULL selects the null stream. */
int bp_set_stream(bp_net* net, void* hip_stream);

/* Number of weights = connections, bias rows included: the paper's
 * connection count (section 6.3) that its throughput unit counts (section
 * 7.1).  Returns -1 for a NULL net. */
int64_t bp_num_weights(const bp_net* net);

/* The state a net keeps between updates is its weights and the weight
 * changes of the previous update (section 9; the update routine of section
 * 6.2.1 reads both).  These four calls copy it between host memory (the
 * caller's array of n == bp_num_weights floats, layout above) and the net.
 * All are synchronous: they wait for the net's stream, then copy.
 * BP_EINVAL for a NULL net or array, or n != bp_num_weights.
 *
 * bp_set_weights loads the weights and zeroes the momentum (a fresh start).
 * bp_get_weights reads the current weights (it does not change the net). */
int bp_set_weights(bp_net* net, const float* w_host, int64_t n);
int bp_get_weights(const bp_net* net, float* w_host, int64_t n);

/* Momentum state V (the previous change), same layout as the weights.
 * Needed for an exact resume. */
int bp_set_momentum(bp_net* net, const float* v_host, int64_t n);
int bp_get_momentum(const bp_net* net, float* v_host, int64_t n);

/* One pass (epoch) over n_patterns dense patterns, in order, with one pooled
 * update per `batch` patterns (ceil(n_patterns / batch) updates; a short last
 * batch is applied like the others).  Each update is the paper's: forward
 * pass, output and hidden deltas (section 3), the changes summed over the
 * batch (section 4.1; section 3 allows pooling over fewer than all
 * patterns), then learning rate and momentum applied to the sum (the update
 * routine of section 6.2.1).  Momentum persists across batches and calls.
 *   inputs_dev  : float [n_patterns][n_0]
 *   targets_dev : float [n_patterns][n_L]
 *   batch >= 1; lr and momentum are used exactly as given (the change is the
 *   SUM over the batch; pass lr / batch for a mean).
 *   sse_out     : if non-NULL, receives the summed squared error of the epoch,
 *                 each pattern measured with the weights of its own batch's
 *                 forward pass; the call then waits for the stream.
 * Returns BP_EINVAL for NULL pointers (n_patterns > 0), n_patterns < 0 or
 * batch < 1. */
int bp_train_batches(bp_net* net, const float* inputs_dev, const float* targets_dev, int64_t n_patterns,
                     int32_t batch, float lr, float momentum, double* sse_out);

/* bp_train_batches for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): same arguments, same launches and the same results, bit for
 * bit.  The call's workspace (activations, deltas, column sums, split-K
 * partials and counters, error partials) lives in a fixed 64 MiB array per
 * GPU, held by the library until the process ends, instead of in the net's
 * own allocations; nothing is allocated or freed, and no graph is captured
 * (every launch is issued directly).  The array is shared by every net and
 * every call on that GPU and keeps the last call's contents: calls that
 * overlap on one GPU (different streams, or host threads) race.  Returns
 * BP_EINVAL, with a message giving the bytes needed, when the call's
 * workspace exceeds 64 MiB (it grows with batch x the layer widths: batch
 * 512 on a 512-2048-2048-2048-64 net needs about 26 MB, batch 1024 about
 * 84 MB); otherwise as bp_train_batches. */
int bp_train_batches_noalloc(bp_net* net, const float* inputs_dev, const float* targets_dev, int64_t n_patterns,
                             int32_t batch, float lr, float momentum, double* sse_out);

/* As bp_train_batches, for inputs that are 0/1 with exactly n_active ones per
 * pattern (the NETtalk window coding: 7 positions x 29 symbols, section 6.3),
 * given as the indices of the ones:
 *   active_dev : int32 [n_patterns][n_active], each in [0, n_0) and distinct
 *                within a pattern.  An index outside [0, n_0) selects no
 *                weight row (the pattern is treated as lacking that one);
 *                duplicates are not detected.
 * The first layer gathers the n_active weight rows instead of multiplying;
 * its change touches only those rows, while the momentum term still moves
 * every row.  1 <= n_active <= n_0. */
int bp_train_batches_onehot(bp_net* net, const int32_t* active_dev, int32_t n_active,
                            const float* targets_dev, int64_t n_patterns, int32_t batch, float lr,
                            float momentum, double* sse_out);

/* Forward pass only (no update; section 3: each unit applies the logistic to
 * the weighted sum of the units feeding it and the true unit): outputs_dev
 * float [n_patterns][n_L] receives the output activations for inputs_dev
 * float [n_patterns][n_0] (both device memory, caller-owned).  Enqueued on
 * the net's stream; returns without waiting.  BP_EINVAL for a NULL pointer
 * (n_patterns > 0) or n_patterns outside [0, 2^31). */
int bp_forward(bp_net* net, const float* inputs_dev, int64_t n_patterns, float* outputs_dev);

/* Forward pass only for one-hot inputs given as active indices (see
 * bp_train_batches_onehot). */
int bp_forward_onehot(bp_net* net, const int32_t* active_dev, int32_t n_active, int64_t n_patterns,
                      float* outputs_dev);

/* ---- Elman nets (section 10.5: recurrent nets trained in parallel across
 * sequences).
 *
 * Context units are the last n_ctx units of the input layer: context unit c
 * (input unit n_0 - n_ctx + c) receives, before each pattern of a sequence,
 * a copy of unit from_unit[c] of hidden layer from_layer[c] (1 <= layer <=
 * min(L - 1, 8)) as it was after the previous pattern of the same sequence
 * (the paper's list of (from unit, to unit) pairs).  The other n_0 - n_ctx
 * inputs are the pattern's external inputs.  from_layer and from_unit are
 * host arrays of n_ctx entries; n_ctx = 0 removes the context.  Waits for the
 * net's stream. */
int bp_set_context(bp_net* net, int32_t n_ctx, const int32_t* from_layer, const int32_t* from_unit);

/* Trains on n_streams sequence streams of n_steps patterns each, pattern
 * (t, s) being step t of stream s (the paper gives each processor its own
 * sequences; here each stream is one).  Row-major device arrays:
 *   inputs_dev  float [n_steps][n_streams][n_0 - n_ctx]  external inputs
 *   targets_dev float [n_steps][n_streams][n_L]
 *   cont_dev    float [n_steps][n_streams]  continuation flag: the copied
 *               context is multiplied by it (1 continues the stream's
 *               sequence, 0 starts a new one)
 *   mask_dev    float [n_steps][n_streams]  the pattern's error is multiplied
 *               by it (0 for the padding after a stream's last sequence, so
 *               that it back-propagates nothing and adds no error)
 * One pooled update (summed change, lr and momentum, as bp_train_batches)
 * follows every steps_per_update steps of all streams, and one after the last
 * step.  The context takes part in the change as an ordinary input (no
 * propagation through time) and starts at zero in every call.  sse_out: the
 * summed squared masked error, as bp_train_batches.  Returns BP_EINVAL for
 * NULL pointers (n_steps > 0; inputs_dev may be NULL when n_0 == n_ctx),
 * n_steps < 0, n_streams < 1 or steps_per_update < 1. */
int bp_train_sequences(bp_net* net, const float* inputs_dev, const float* targets_dev, const float* cont_dev,
                       const float* mask_dev, int64_t n_steps, int32_t n_streams, int32_t steps_per_update,
                       float lr, float momentum, double* sse_out);

/* Forward passes of sequences (no update): outputs_dev float
 * [n_steps][n_streams][n_L]; inputs and flags as bp_train_sequences. */
int bp_forward_sequences(bp_net* net, const float* inputs_dev, const float* cont_dev, int64_t n_steps,
                         int32_t n_streams, float* outputs_dev);

/* ---- Options of the method (all off after bp_create). */

/* Unit nonlinearity (section 4.3).  BP_SIGMOID_EXACT: 1 / (1 + e^-x) in fp32
 * (the default).  BP_SIGMOID_TABLE: the paper's second evaluation: x is taken
 * to the nearest end of [-15, 15] when outside it, mapped onto [0, 255] as
 * x1 = (x + 15) * 255 / 30, and the logistic is read from a 256-entry table
 * of its values at -15 + 30 i / 255 (entry floor(x1)) with linear
 * interpolation to the next entry by x1 - floor(x1); NaN stays NaN.  Maximum
 * error 1.67e-4 (the linear-interpolation bound h^2 / 8 max|sigma''|).  The
 * derivative used in the deltas stays y (1 - y).  Applies to every later
 * train and forward call; waits for the net's stream. */
enum { BP_SIGMOID_EXACT = 0, BP_SIGMOID_TABLE = 1 };
int bp_set_sigmoid(bp_net* net, int32_t mode);

/* Range check of the summed weight changes (section 8: each total weight
 * change is tested for a reasonable range; one out of range is set to zero
 * and counted as a fault).  limit > 0: every summed change G (the batch sum,
 * before the learning rate) with |G| > limit or NaN is replaced by 0, so that
 * weight moves by its momentum term only, and the fault counter is
 * incremented.  limit == 0 disables the check.  Also resets the counter to 0.
 * Returns BP_EINVAL for a negative or NaN limit.  Waits for the net's stream. */
int bp_set_fault_limit(bp_net* net, float limit);

/* Faults counted since the last bp_set_fault_limit (0 if never set).  Waits
 * for the net's stream; *count is a host int64. */
int bp_get_fault_count(bp_net* net, int64_t* count);

/* In-HBM checkpoint of the weights and momentum (section 10.4): one slot
 * owned by the net (allocated by the first save).  Save and restore are
 * device-to-device copies enqueued on the net's stream.  Restore without a
 * saved checkpoint returns BP_EINVAL. */
int bp_checkpoint_save(bp_net* net);
int bp_checkpoint_restore(bp_net* net);

/* Rollback guard (section 10.4: copy weights to a checkpoint every few epochs
 * and copy them back when the error jumps between epochs).  bp_guard_config
 * saves a checkpoint now and arms the guard: every >= 1 accepted epochs
 * between checkpoints, jump > 0 the error ratio that counts as a jump.  After
 * each epoch the caller reports its summed squared error to bp_guard_epoch:
 *   - if the error exceeds jump x the last accepted epoch's error (or is NaN),
 *     W and V are restored from the checkpoint, *rolled_back = 1, and the
 *     caller resumes from the checkpoint's epoch;
 *   - otherwise the epoch is accepted (*rolled_back = 0), and every `every`
 *     accepted epochs the checkpoint is renewed.
 * A jump that recurs at the same epoch after a rollback is accepted: training
 * is deterministic, so a jump that replays is the learning itself rather than
 * a transient fault.  bp_guard_epoch without bp_guard_config returns
 * BP_EINVAL. */
int bp_guard_config(bp_net* net, int32_t every, double jump);
int bp_guard_epoch(bp_net* net, double sse, int32_t* rolled_back);

/* Measurement support (not part of the method).  Kernel kinds a net launches: */
enum {
  BP_K_FORWARD = 0,   /* hidden-layer forward product + sigmoid            */
  BP_K_OUTPUT = 1,    /* output-layer forward product + deltas + error      */
  BP_K_BACKWARD = 2,  /* hidden-delta product + derivative                  */
  BP_K_CHANGE = 3,    /* summed-change product + momentum update           */
  BP_K_SPLITK = 4,    /* summed-change product split over the batch; the  */
                      /* last block of each tile adds the partials in     */
                      /* split order and applies the momentum update      */
  BP_K_BIAS = 5,      /* bias-row column sums + momentum update             */
  BP_K_GATHER = 6,    /* one-hot first-layer forward                        */
  BP_K_SCATTER = 7,   /* one-hot first-layer change + momentum update       */
  BP_K_REDUCE = 8,    /* epoch error reduction                              */
  BP_K_FUSED_FB = 9,  /* small one-hot nets: whole forward + backward pass  */
  BP_K_FUSED_UPD = 10,/* small one-hot nets: both layers' change + update   */
  BP_K_OUTFIN = 11,   /* split-K output layer: partial sums + deltas + error */
  BP_K_SEQ_IN = 12,   /* Elman nets: input rows of a step with the context copy */
  BP_K_SEQ_PAIR = 13, /* Elman nets: hidden layer of a step + output layer of the step before */
  BP_K_SEQ_WIN = 14,  /* Elman nets, one hidden layer: forward pass + output deltas of a window */
  BP_K_COUNT = 15
};

/* Graph replay of repeated training calls (on by default).  With on != 0,
 * a call of bp_train_batches / bp_train_batches_onehot whose arguments (data
 * pointers, sizes, lr, momentum) equal those of the previous call captures
 * its kernel launches into a HIP graph, and later calls with the same
 * arguments replay that graph instead of launching each kernel: same
 * kernels, same results bit for bit, less launch overhead per update.  A
 * change of workspace size, sigmoid mode or range check, or profiling,
 * drops back to direct launches.  Calls of a single batch always launch
 * directly (a graph launch costs more host time than their few kernels).  The graph reads the argument buffers at
 * replay time, so their contents may change between calls.  on == 0: every
 * call launches directly.  Waits for the net's stream; drops any graph. */
int bp_set_graph_replay(bp_net* net, int on);

/* on != 0: from now on every kernel launch of this net is bracketed by HIP
 * events on the net's stream (adds launch overhead; for measurement runs
 * only); clears the counters.  on == 0: stops recording. */
int bp_profile(bp_net* net, int on);

/* Waits for the stream and writes, for each kind k < n_kinds (<= BP_K_COUNT),
 * the number of launches recorded and their summed device time in
 * milliseconds (launches[k], ms[k]; host arrays). */
int bp_profile_report(bp_net* net, int64_t* launches, double* ms, int32_t n_kinds);

/* Message describing the last non-OK return on this net (or of bp_create
 * when net is NULL).  Valid until the next call on the net. */
const char* bp_last_error(const bp_net* net);

#ifdef __cplusplus
}
#endif

#endif /* BP_H */
