/*
 * rnnbkt.h -- C ABI of librnnbkt.so: the single-GPU hot path of
 * sequence-bucketed recurrent-network training on AMD Instinct MI355X (gfx950).
 *
 * Method: Khomenko et al., "Accelerating Recurrent Neural Network Training
 * using Sequence Bucketing and Multi-GPU Data Parallelization" (arXiv
 * 1708.05604).  The planner implements the dynamic-programming bucketing of
 * Sec. III.A (eqs. 1-2 and the DYNAMICBUCKETING procedure); the batch
 * schedule follows Sec. III (reshuffle every epoch) and Sec. IV.A (shortest
 * bucket first); the model calls run one mini-batch of a stacked LSTM (the
 * paper's model, its ref. [1]) or GRU (its ref. [2], Sec. I) forward and
 * backward through time, with a per-frame softmax cross-entropy loss in place
 * of the paper's CTC cost, and a plain SGD step in place of ADADELTA.
 *
 * Conventions for every call
 *   - Return value: RNNBKT_OK (0) or a negative error code.  On error,
 *     rnnbkt_last_error() returns a message (thread-local, valid until the
 *     next call on the same thread).  No C++ exception crosses the ABI.
 *   - Argument validation happens before any GPU work is enqueued: a call
 *     that returns RNNBKT_EINVAL or RNNBKT_EUNSUPPORTED has launched nothing.
 *   - "device" pointers are HIP device memory owned by the caller; "host"
 *     pointers are read (or written) synchronously during the call.  The
 *     library never allocates or frees device memory.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     GPU work is enqueued on it asynchronously; the library never
 *     synchronises the device.  An asynchronous kernel fault surfaces as
 *     RNNBKT_EHIP from a later call or from rnnbkt_sync_check().
 */
#ifndef RNNBKT_H
#define RNNBKT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RNNBKT_OK 0
#define RNNBKT_EINVAL (-1)       /* bad argument (null pointer, bad size, unsorted lengths...) */
#define RNNBKT_EUNSUPPORTED (-2) /* valid but not supported shape/option (e.g. hidden % 32 != 0) */
#define RNNBKT_EHIP (-3)         /* a HIP runtime call or kernel launch failed */

#define RNNBKT_CELL_LSTM 0 /* gates i, f, g, o */
#define RNNBKT_CELL_GRU 1  /* gates r, z, n */
#define RNNBKT_CELL_LSTM_PEEPHOLE 2 /* LSTM with diagonal peepholes (Sec. IV.A: the
                                       paper's Lasagne LSTM has them by default) */

#define RNNBKT_GEMM_FP32 0 /* GEMM operands and accumulation in fp32 */
#define RNNBKT_GEMM_BF16 1 /* GEMM operands rounded to bf16 (nearest-even), fp32 accumulate */

/* Library version string, e.g. "rnnbkt 0.1.0 gfx950". */
const char* rnnbkt_version(void);

/* Message of the last error on this thread ("" if none). */
const char* rnnbkt_last_error(void);

/* Waits for `stream` and reports any asynchronous HIP error as RNNBKT_EHIP.
 * Also RNNBKT_EHIP when a wait of a resident recurrence launch (see
 * rnnbkt_lstm_fwd) gave up since the last report: the results of the launch
 * it belonged to are invalid.  Such a launch still runs to its end (its
 * later waits return at once) and other launches are not affected; the
 * report clears the count, so a later call returns RNNBKT_OK unless new
 * waits gave up.  The count is per device and process: call this while no
 * other stream runs the library's launches, or the report may name them. */
int32_t rnnbkt_sync_check(void* stream);

/*
 * rnnbkt_bucket_plan -- optimal length bucketing (Sec. III.A, the
 * DYNAMICBUCKETING dynamic program over the length histogram).
 *
 * Splits the sequences, ordered by length, into K_eff = min(K, D) buckets of
 * contiguous length ranges (D = number of distinct lengths) so that
 * sum_b upper_b * count_b -- every sequence padded to its bucket's upper
 * length -- is minimal.  Among equal-cost splits the one the paper's loop
 * order selects is returned: at every level the largest split point
 * (the DP scans split points downwards and replaces only on a strictly
 * smaller score).
 *
 *   lengths       host int32[n], every value >= 1 (any order)
 *   n             number of sequences, >= 1
 *   K             requested number of buckets, >= 1
 *   bucket_upper  host int32[K] out: first *K_eff entries = upper length of
 *                 each bucket, strictly increasing, last = max(lengths)
 *   bucket_of     host int32[n] out: bucket of each sequence (0-based), the
 *                 smallest b with lengths[s] <= bucket_upper[b]
 *   K_eff         host out: number of buckets actually used
 *   padded_steps  host out: the optimum, sum_b upper_b * count_b
 * Host-only (no GPU needed).  Errors: EINVAL for null pointers, n < 1,
 * K < 1 or a length < 1.
 */
int32_t rnnbkt_bucket_plan(const int32_t* lengths, int64_t n, int32_t K,
                           int32_t* bucket_upper, int32_t* bucket_of,
                           int32_t* K_eff, int64_t* padded_steps);

/*
 * rnnbkt_epoch_schedule -- the mini-batches of one epoch (Sec. III: data
 * reshuffled every epoch; Sec. IV.A: the shortest bucket is fed first, then
 * the bucket index increases; K_eff = 1 is the paper's unbucketed baseline,
 * a purely random split into mini-batches).
 *
 * For b = 0..K_eff-1: the sequences of bucket b are ordered by
 * (keys[s], s) ascending -- the keys are the epoch's random shuffle -- and
 * cut into consecutive batches of B (the last one may be smaller); each
 * batch is then ordered by (length descending, index ascending), so the
 * sequences still running at step t are a prefix of the batch.
 *
 *   lengths      host int32[n] (>= 1)
 *   bucket_of    host int32[n] from rnnbkt_bucket_plan (values in [0, K_eff))
 *   keys         host uint64[n] shuffle keys of this epoch
 *   B            batch size >= 1
 *   order        host int64[n] out: sequence indices, batch after batch
 *   batch_start  host int64[n+1] out: batch i is order[batch_start[i] ..
 *                batch_start[i+1]); only the first *num_batches+1 are set
 *   num_batches  host out
 * Host-only.  Errors: EINVAL.
 */
int32_t rnnbkt_epoch_schedule(const int32_t* lengths, const int32_t* bucket_of,
                              int64_t n, int32_t K_eff, const uint64_t* keys,
                              int32_t B, int64_t* order, int64_t* batch_start,
                              int64_t* num_batches);

/* Feeding orders of rnnbkt_epoch_schedule_ordered.  The paper feeds the
 * buckets shortest first (Sec. IV.A) and leaves other orders to future work
 * (Sec. V); every ordering feeds the same batches. */
#define RNNBKT_ORDER_ASCENDING 0        /* bucket 0, 1, ..., K_eff-1 (the paper's order) */
#define RNNBKT_ORDER_DESCENDING 1       /* bucket K_eff-1, ..., 0 */
#define RNNBKT_ORDER_RANDOM_BUCKETS 2   /* whole buckets by (order_keys[b], b) ascending */
#define RNNBKT_ORDER_SHUFFLED_BATCHES 3 /* batches of all buckets interleaved: the
                                           ascending list of batches sorted by
                                           (order_keys[i], i), i = ascending position */

/*
 * rnnbkt_epoch_schedule_ordered -- rnnbkt_epoch_schedule with a choice of
 * feeding order.  The batches are built exactly as rnnbkt_epoch_schedule
 * builds them; only their sequence in `order` / `batch_start` differs.
 *
 *   ordering     RNNBKT_ORDER_*
 *   order_keys   host uint64[n] random keys, read for RANDOM_BUCKETS (entries
 *                0..K_eff-1; then K_eff <= n) and SHUFFLED_BATCHES (entries
 *                0..num_batches-1); may be null for the other two
 *   other arguments as for rnnbkt_epoch_schedule, which equals this call
 *   with RNNBKT_ORDER_ASCENDING.
 * Host-only.  Errors: EINVAL (as rnnbkt_epoch_schedule; unknown ordering;
 * null order_keys where it is read).
 */
int32_t rnnbkt_epoch_schedule_ordered(const int32_t* lengths, const int32_t* bucket_of,
                                      int64_t n, int32_t K_eff, const uint64_t* keys,
                                      int32_t B, int32_t ordering,
                                      const uint64_t* order_keys, int64_t* order,
                                      int64_t* batch_start, int64_t* num_batches);

/* Model description.  Shapes: G = 4 (LSTM, either kind) or 3 (GRU) gates, H = hidden,
 * dirs = 2 if bidirectional else 1, D_in(layer 0) = input_dim,
 * D_in(layer > 0) = dirs * H, H_top = dirs * H. */
typedef struct {
  int32_t cell;          /* RNNBKT_CELL_LSTM, RNNBKT_CELL_GRU or RNNBKT_CELL_LSTM_PEEPHOLE */
  int32_t num_layers;    /* >= 1 */
  int32_t input_dim;     /* multiple of 4 */
  int32_t hidden;        /* multiple of 32 */
  int32_t num_classes;   /* multiple of 4, at most 1024 */
  int32_t bidirectional; /* 0 or 1 */
  int32_t gemm_dtype;    /* RNNBKT_GEMM_FP32 or RNNBKT_GEMM_BF16 */
} rnnbkt_model_desc;

/*
 * Flat fp32 parameter layout (row-major), the order of rnnbkt_param_count:
 *   for layer = 0..num_layers-1, for direction = forward, reverse:
 *     W_ih [G*H, D_in]  gate blocks in the order above
 *     W_hh [G*H, H]
 *     LSTM: b [G*H]          GRU: b_ih [3H], then b_hh [3H]
 *     LSTM with peepholes: b [G*H], then p [3H] = (p_i, p_f, p_o)
 *   W_out [C, H_top], b_out [C]
 * LSTM:  a = W_ih x + W_hh h + b; i,f,o = sigmoid, g = tanh;
 *        c' = f*c + i*g; h' = o*tanh(c').
 * Peephole LSTM: as LSTM but i = sigmoid(a_i + p_i*c), f = sigmoid(a_f +
 *        p_f*c), and after the cell update o = sigmoid(a_o + p_o*c').
 * GRU:   r,z = sigmoid(W_i x + b_i + W_h h + b_h) of their blocks;
 *        n = tanh(W_in x + b_in + r*(W_hn h + b_hn)); h' = (1-z)*n + z*h.
 * Initial states are zero; the reverse direction runs over each sequence's
 * own length; a bidirectional layer outputs [h_fwd ; h_bwd] per frame.
 * Returns the number of floats, or a negative error code.
 */
int64_t rnnbkt_param_count(const rnnbkt_model_desc* desc);

/*
 * Bytes of the two caller-owned device buffers a batch needs:
 *   reserve   -- written by rnnbkt_lstm_fwd, used by rnnbkt_lstm_bwd of the
 *                same batch: activations kept for backpropagation, and the
 *                backward's gate gradients (the forward prepares them for
 *                the backward's workgroups to exchange); must not be
 *                modified in between
 *   workspace -- scratch of either call (no content carried between calls)
 * Depends on (desc, T_max, B, n_valid) only and is non-decreasing in each,
 * so sizing with an epoch's maxima covers every batch of the epoch.
 *   T_max    longest sequence of the batch;  B  batch size;
 *   n_valid  sum of the batch's lengths.
 */
int32_t rnnbkt_buffer_sizes(const rnnbkt_model_desc* desc, int32_t T_max, int32_t B,
                            int64_t n_valid, size_t* reserve_bytes,
                            size_t* workspace_bytes);

/*
 * rnnbkt_lstm_fwd -- forward pass and loss of one mini-batch (LSTM or GRU
 * per desc->cell).
 *
 *   params     device fp32[param_count], layout above
 *   x          device fp32[T_max][B][input_dim], time-major padded batch;
 *              frames t >= lengths[b] are never read (may hold anything)
 *   labels     device int32[T_max][B], class of every valid frame in
 *              [0, num_classes); pad entries are never read
 *   lengths    host int32[B], non-increasing, lengths[0] == T_max, all >= 1
 *   reserve / workspace  device buffers of at least the sizes returned by
 *              rnnbkt_buffer_sizes(desc, T_max, B, sum(lengths))
 *   loss       device fp32[1] out: mean over the batch's valid frames of
 *              -log softmax(W_out h_top + b_out)[label]
 * The loss gradient w.r.t. the logits, and its product with W_out (the
 * gradient w.r.t. the top layer's output), are computed here and kept in
 * reserve.  When the top layer runs in a resident launch (fp32, one stream
 * declared), the output layer and loss are computed by extra workgroups of
 * that launch, on rows of the top layer as they are published;
 * RNNBKT_OUTPUT=after runs them as separate kernels after the recurrence.
 * Recurrence kernels (this call and rnnbkt_lstm_bwd): all steps of a layer
 * (or of a unidirectional stack) in one launch whose workgroups stay
 * resident, when the grid fits (see rnnbkt_set_concurrency), else one
 * launch per step.  Environment: RNNBKT_RECURRENCE=steps forces the
 * per-step kernels; RNNBKT_MAX_POLLS=n sets the poll budget of one wait of
 * a resident launch (default 2^20; a test hook: 0 makes every wait give up
 * at its first miss, which rnnbkt_sync_check then reports).
 * Errors: EINVAL (null pointer, bad lengths, buffers too small),
 * EUNSUPPORTED (hidden % 32 != 0, input_dim % 4 != 0, num_classes % 4 != 0
 * or > 1024), EHIP.
 */
int32_t rnnbkt_lstm_fwd(const rnnbkt_model_desc* desc, const float* params,
                        const float* x, const int32_t* labels,
                        const int32_t* lengths, int32_t T_max, int32_t B,
                        void* reserve, size_t reserve_bytes, void* workspace,
                        size_t workspace_bytes, float* loss, void* stream);

/*
 * rnnbkt_ctc_workspace_bytes -- bytes of the extra caller-owned device
 * workspace rnnbkt_lstm_fwd_ctc needs for batches of up to T_max frames,
 * B sequences and U_max labels per target (scratch; nothing carried between
 * calls).  Errors: EINVAL (non-positive sizes), EUNSUPPORTED (U_max > 1023).
 */
int32_t rnnbkt_ctc_workspace_bytes(int32_t T_max, int32_t B, int32_t U_max, size_t* bytes);

/*
 * rnnbkt_lstm_fwd_ctc -- rnnbkt_lstm_fwd with the connectionist temporal
 * classification loss, the cost the paper trains with (Sec. IV.A), in place
 * of the per-frame loss.  Class 0 of the output layer is the blank; each
 * sequence has an unaligned target string over classes 1..num_classes-1.
 *
 *   targets         device int32[B][U_max]: row b holds sequence b's labels
 *                   in its first target_lengths[b] entries (the rest are
 *                   never read); a label outside 1..num_classes-1 is clamped
 *                   into that range (device data is not checked)
 *   target_lengths  host int32[B], 1 <= target_lengths[b] <= min(U_max,
 *                   lengths[b])
 *   ctc_ws          device buffer of at least
 *                   rnnbkt_ctc_workspace_bytes(T_max, B, U_max) bytes,
 *                   16-byte aligned
 *   loss            device fp32[1] out: mean over the B sequences of
 *                   -ln p(target | x), p summing over every frame path that
 *                   collapses to the target (repeats merged, blanks dropped)
 * Other arguments as in rnnbkt_lstm_fwd (no per-frame labels).  The loss
 * gradient w.r.t. the logits is kept in reserve, so rnnbkt_lstm_bwd follows
 * unchanged (the output layer runs after the recurrence).  A target no path of its sequence's length can produce (equal
 * neighbours need a blank between them) gives an infinite loss and zero
 * gradient rows for that sequence.  Probabilities are renormalised every
 * frame in fp32; the per-sequence log-likelihood is summed in fp64.
 * Errors: as rnnbkt_lstm_fwd, plus EINVAL (bad target lengths, ctc_ws too
 * small) and EUNSUPPORTED (U_max > 1023).
 */
int32_t rnnbkt_lstm_fwd_ctc(const rnnbkt_model_desc* desc, const float* params, const float* x,
                            const int32_t* targets, const int32_t* target_lengths,
                            int32_t U_max, const int32_t* lengths, int32_t T_max, int32_t B,
                            void* reserve, size_t reserve_bytes, void* workspace,
                            size_t workspace_bytes, void* ctc_ws, size_t ctc_ws_bytes,
                            float* loss, void* stream);

/*
 * rnnbkt_lstm_bwd -- backpropagation through time of the batch last run
 * through rnnbkt_lstm_fwd with the same (desc, params, x, lengths, reserve).
 *   grads   device fp32[param_count] out: d loss / d params (overwritten
 *           entirely, same layout as params)
 * Other arguments as in rnnbkt_lstm_fwd (labels are not needed again).
 * For an fp32 unidirectional LSTM stack in one resident launch (one stream
 * declared), the layer weight gradients are computed by extra workgroups of
 * that launch as the gate gradients are published (RNNBKT_WGRAD=after:
 * GEMMs after it).  The
 * output layer's weight gradients run on an internal stream beside the
 * recurrence when one stream is declared; the call returns with all of its
 * work ordered on `stream`.
 * Reductions run in a fixed order: results are bitwise reproducible.
 */
int32_t rnnbkt_lstm_bwd(const rnnbkt_model_desc* desc, const float* params,
                        const int32_t* lengths, int32_t T_max, int32_t B,
                        void* reserve, size_t reserve_bytes, void* workspace,
                        size_t workspace_bytes, float* grads, void* stream);

/*
 * rnnbkt_lstm_bwd_noalloc -- rnnbkt_lstm_bwd for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): no workspace argument, no allocation,
 * no stream or event creation.  Its scratch is a 128 MiB array the library
 * holds on each device it runs on (from its first use there until the
 * process ends).  A batch whose backward needs more is refused with
 * RNNBKT_EUNSUPPORTED before anything is enqueued: a unidirectional stack
 * on the resident kernels needs only its split-K, weight-gradient and bias
 * partials (every batch of a 2-layer H=512 LSTM with B=128 and 4000 steps
 * fits), other plans the full backward workspace of rnnbkt_buffer_sizes.
 * Everything runs on `stream` (no internal side stream); results equal
 * rnnbkt_lstm_bwd's bit for bit.  All calls on one device share its scratch:
 * calls that overlap on one device (different streams or threads) race, so
 * serialise them.  Nothing in the scratch needs clearing between calls.
 * Arguments and errors otherwise as rnnbkt_lstm_bwd.
 */
int32_t rnnbkt_lstm_bwd_noalloc(const rnnbkt_model_desc* desc, const float* params,
                                const int32_t* lengths, int32_t T_max, int32_t B,
                                void* reserve, size_t reserve_bytes, float* grads,
                                void* stream);

/* rnnbkt_sgd_apply -- params[i] -= lr * grads[i] for i < n (device fp32). */
int32_t rnnbkt_sgd_apply(float* params, const float* grads, int64_t n, float lr,
                         void* stream);

/* rnnbkt_adadelta_apply -- one ADADELTA step, the update rule of the paper's
 * training processes (Sec. III.B, step 4; Zeiler's method, its ref. [21]),
 * elementwise over n device fp32 values, in this order:
 *   acc_g2[i]  <- rho * acc_g2[i] + (1 - rho) * g^2            (g = grads[i])
 *   dx          = -sqrt(acc_dx2[i] + eps) / sqrt(acc_g2[i] + eps) * g
 *                 (acc_g2 already updated, acc_dx2 not yet)
 *   acc_dx2[i] <- rho * acc_dx2[i] + (1 - rho) * dx^2
 *   params[i]  <- params[i] + lr * dx
 *   acc_g2, acc_dx2  caller-owned optimiser state of n floats each, zero
 *                    before the first step, kept between steps
 *   rho in [0, 1) (0.95 in the published method), eps > 0 (1e-6), lr > 0
 *   (1 = the method as published; it has no learning rate of its own).
 * All four arrays 16-byte aligned; params, acc_g2, acc_dx2 updated in place.
 * Errors: RNNBKT_EINVAL (null pointer, n < 0, misalignment, constants out of
 * range), before any launch. */
int32_t rnnbkt_adadelta_apply(float* params, const float* grads, float* acc_g2, float* acc_dx2,
                              int64_t n, float rho, float eps, float lr, void* stream);

/* rnnbkt_epoch_aggregate -- the epoch-end step of the paper's parallel
 * training (Sec. III.B, step 5, eq. 3 with alpha = 1): R replicas trained on
 * separate portions of the epoch are merged into
 *   V(t) = (1/R) sum_r V_r(t) - beta * V(t-1)
 * and every replica starts the next epoch from V(t).  In place, for i < n:
 *   replicas   device fp32; replica r's parameters at replicas + r*stride
 *              (r = 0..R-1); in: V_r(t), out: V(t) in every replica
 *   R          1..1024
 *   stride     floats between replicas, >= n and a multiple of 4
 *   prev       device fp32[n]; in: V(t-1) (the initial parameters for the
 *              first epoch), out: V(t); must not overlap any replica's n values
 *   beta       finite (1e-6 in the paper)
 * The sum and the scaling run in double; each result is rounded to float
 * once.  replicas and prev 16-byte aligned.  On one GPU the replicas are R
 * concurrent training streams (rnnbkt_set_concurrency); across GPUs an
 * all-reduce of the replicas would come first.
 * Errors: RNNBKT_EINVAL (null pointer, R, n or stride out of range,
 * misalignment, overlap, non-finite beta), before any launch. */
int32_t rnnbkt_epoch_aggregate(float* replicas, int32_t R, int64_t stride, int64_t n,
                               float* prev, float beta, void* stream);

/* rnnbkt_set_concurrency -- declares how many streams may run this
 * library's training calls at the same time in this process (default 1).
 * The recurrence kernels keep all their workgroups resident for a whole
 * batch (each waits for values other workgroups publish); with `streams`
 * declared, each such launch claims at most 1/streams of the GPU's capacity
 * for it, so the launches of all streams can be resident together.  A
 * batch whose grid does not fit its share runs on the per-step kernels
 * instead.  Running more streams than declared can make the waits of a
 * launch time out: the results are then invalid and rnnbkt_sync_check
 * reports it (no hang: every wait is bounded).  Set it while no call is in
 * flight.  Errors: RNNBKT_EINVAL if streams is outside [1, 64]. */
int32_t rnnbkt_set_concurrency(int32_t streams);

/*
 * rnnbkt_top_hidden -- copies the top layer's per-frame output of the batch
 * held in `reserve` (after rnnbkt_lstm_fwd) into the padded layout
 * out[T_max][B][H_top] (device fp32); pad frames are set to 0.
 * Arguments as in rnnbkt_lstm_fwd.
 */
int32_t rnnbkt_top_hidden(const rnnbkt_model_desc* desc, const int32_t* lengths,
                          int32_t T_max, int32_t B, const void* reserve,
                          size_t reserve_bytes, float* out, void* stream);

/*
 * Kernel timer -- measurement support for the benchmark (not part of the
 * method).  While enabled, the model calls and rnnbkt_sgd_apply bracket every
 * kernel launch with a pair of HIP events recorded on the call's stream and
 * note the launch's algorithmic work: recurrent launches count the flops of
 * their products (forward x.W_ih and h.W_hh, backward dA.W_hh and, where a
 * launch takes a stack of layers, the upper layer's dA.W_ih), GEMMs 2*M*N*K,
 * the loss kernel 8*C+4 bytes per frame, SGD 12 and ADADELTA 28 bytes per
 * parameter, the batch preparation the bytes it moves.
 * Kinds: see RNNBKT_KERNEL_*.  The events add a small gap between launches,
 * so time a run with the timer off and use the timer in a separate pass.
 *   rnnbkt_kernel_timer(1) clears the records and starts recording,
 *   rnnbkt_kernel_timer(0) stops.  Host-side state, one per process.
 *   rnnbkt_kernel_timer_read waits for the recorded events and returns, for
 *   one kind, the summed event-to-event time (ms), the number of launches
 *   and the summed algorithmic flops and bytes.
 */
#define RNNBKT_KERNEL_STEP_FWD 0 /* recurrent step, forward */
#define RNNBKT_KERNEL_STEP_BWD 1 /* recurrent step, backward through time */
#define RNNBKT_KERNEL_GEMM 2     /* dense contractions incl. split-K folds */
#define RNNBKT_KERNEL_XENT 3     /* output loss and its gradient (cross-entropy or CTC) */
#define RNNBKT_KERNEL_SGD 4      /* parameter update (SGD, ADADELTA, eq. 3 aggregation) */
#define RNNBKT_KERNEL_OTHER 5    /* batch tables, packing, column sums, loss sum */
#define RNNBKT_KERNEL_SIDE 6     /* any work on the library's internal side stream, which
                                    runs beside other work of the backward (output-layer
                                    weight gradients; recurrent weight gradients when the
                                    launch does not compute them): overlapped time */
#define RNNBKT_KERNEL_PREPARE 7  /* start of a forward: batch tables, packing of the padded
                                    batch into valid frames and the sentinel fills of the
                                    resident launches (bytes: everything the launch moves) */
#define RNNBKT_KERNEL_KINDS 8

int32_t rnnbkt_kernel_timer(int32_t enable);
int32_t rnnbkt_kernel_timer_read(int32_t kind, double* total_ms, int64_t* launches,
                                 double* alg_flops, double* alg_bytes);

#ifdef __cplusplus
}
#endif

#endif /* RNNBKT_H */
