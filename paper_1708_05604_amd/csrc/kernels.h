// Internal launch interface between the C-ABI layer (api.hip) and the HIP
// kernels.  Every launcher enqueues on `stream` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "rnnbkt.h"

namespace rnnbkt {

// A buffer of n 32-bit words to set to one value (16-byte aligned).
constexpr int kFillJobs = 8;
struct FillJob {
  unsigned* p;
  int64_t n;
};


// Cell nonlinearities of both recurrence implementations (device code):
// the logistic function from the hardware exp and reciprocal (relative
// error a few ulp), and tanh x = 2 sigma(2x) - 1 (absolute error a few
// 1e-8 near 0).  Saturating inputs give exactly 0 / 1 (-1 / 1 for tanh).
__device__ inline float act_sigmoid(float x) {
  return __builtin_amdgcn_rcpf(1.f + __expf(-x));
}
__device__ inline float act_tanh(float x) { return 2.f * act_sigmoid(2.f * x) - 1.f; }

// ---------------------------------------------------------------- GEMM
// C[M x N] = op(A) . op(B) (+ bias[n]) (+ C if accumulate), fp32 in memory;
// operands rounded to bf16 on the way to the matrix cores when bf16 != 0.
//   a_kcontig: A element (m, k) at A[m*lda + k], else at A[k*lda + m]
//   b_kcontig: B element (k, n) at B[n*ldb + k], else at B[row(k)*ldb + n]
//              where row(k) = gather_b ? gather_b[k] : k (a negative
//              gather entry reads as a zero row)
// With splits > 1 the K range is cut into `splits` slices of k_per_split
// (a multiple of 32); each slice writes partial[s][M][N] and
// splitk_reduce() folds them in slice order (deterministic).
// A second term (K2 > 0): C = op(A) op(B) + op(A2) op(B2), A2 and B2 in the
// layouts of A and B with strides lda2, ldb2 and reduction length K2 (no
// gather, no split-K; K % 32 == 0).
struct GemmArgs {
  const float* A;
  const float* B;
  float* C;
  const float* bias;
  const int32_t* gather_b;
  float* partial;
  int64_t lda, ldb, ldc;
  int32_t M, N, K;
  int32_t k_per_split;
  int32_t splits;
  int32_t accumulate;
  const float* A2;
  const float* B2;
  int64_t lda2, ldb2;
  int32_t K2;
  int32_t beside;  // 1: runs beside a resident recurrence (bf16: the gentler tiling)
  int32_t a_bf16;  // 1: A (and A2) hold bf16 values, 2 bytes each (bf16 path only)
};

// Output tile of the GEMM kernels, rows x columns: 64 x 64 (fp32), 128 x 128
// (bf16).  Split-K counts are chosen per tile size.
inline int32_t gemm_tile(bool bf16) { return bf16 ? 128 : 64; }

hipError_t launch_gemm(const GemmArgs& g, bool a_kcontig, bool b_kcontig, bool bf16,
                       hipStream_t stream);

// out[m*ldc + n] = (accumulate ? out : 0) + sum_s partial[s][m][n] (+ bias[n])
hipError_t launch_splitk_reduce(const float* partial, int32_t S, int32_t M, int32_t N,
                                float* out, int64_t ldc, const float* bias, int32_t accumulate,
                                hipStream_t stream);

// Several folds of the form above (no bias, no accumulation) in one launch:
// out[m*ldc + n] = sum_s partial[s][m][n], each job its own sizes.
constexpr int kFoldJobs = 16;
struct FoldJob {
  const float* partial;
  int32_t S, M, N;
  float* out;
  int64_t ldc;
};
hipError_t launch_splitk_reduce_multi(const FoldJob* jobs, int32_t njobs, hipStream_t stream);

// Column sums of A[rows x cols] (row stride lda), deterministic:
// partial[s][c] over row slices of `rows_per_split`, then folded into out[c].
hipError_t launch_colsum(const float* A, int64_t rows, int32_t cols, int64_t lda,
                         int64_t rows_per_split, float* partial, float* out,
                         hipStream_t stream);

// ---------------------------------------------------------------- batch tables
// batch_sizes[t] = #{b : lengths[b] > t} for t < T_max (lengths copied into
// kernel arguments in chunks), offsets[t] = sum_{t' < t} batch_sizes[t'],
// offsets[T_max] = n_valid.
hipError_t launch_batch_tables(const int32_t* lengths_host, int32_t B, int32_t T_max,
                               int32_t* batch_sizes, int32_t* offsets, hipStream_t stream);

// One launch for the start of a batch: what launch_batch_tables and
// launch_pack do (when B > 0; B <= kPrepMaxB, lengths non-increasing), plus
// filling fills[0..nfill) with `value` (16-byte aligned buffers).  With B = 0
// it only fills.
constexpr int kPrepMaxB = 256;
// zero_word (if not null) is set to 0.
hipError_t launch_prepare(const int32_t* lengths_host, int32_t B, int32_t T_max, const float* x,
                          const int32_t* labels, int32_t D, int32_t* batch_sizes,
                          int32_t* offsets, float* Xp, int32_t* Yp, int32_t* prev_fwd,
                          int32_t* prev_rev, const FillJob* fills, int32_t nfill, unsigned value,
                          unsigned* zero_word, hipStream_t stream);

// Padded time-major batch -> packed valid frames (frame of (t, b) = offsets[t] + b):
// Xp[f][:] = x[t][b][:], Yp[f] = labels[t][b] (labels may be null),
// prev_fwd[f] = frame of (t-1, b) or -1, prev_rev[f] = frame of (t+1, b) or -1.
hipError_t launch_pack(const float* x, const int32_t* labels, const int32_t* batch_sizes,
                       const int32_t* offsets, int32_t T_max, int32_t B, int32_t D, float* Xp,
                       int32_t* Yp, int32_t* prev_fwd, int32_t* prev_rev, hipStream_t stream);

// out[t][b][:] = H[offsets[t] + b][:] for b < batch_sizes[t], else 0.
hipError_t launch_unpack(const float* H, int32_t width, const int32_t* batch_sizes,
                         const int32_t* offsets, int32_t T_max, int32_t B, float* out,
                         hipStream_t stream);

// ---------------------------------------------------------------- loss, SGD
// In place over logits[N x C]: dlogits = (softmax - onehot(y)) / N;
// loss_partial[block] = sum over the block's frames of -log softmax[y].
// Returns the number of partials through *num_partials.
hipError_t launch_softmax_xent(float* logits, const int32_t* labels, int64_t N, int32_t C,
                               float* loss_partial, int32_t* num_partials, hipStream_t stream);

// out[0] = scale * sum_i partial[i] (fixed order).
hipError_t launch_sum(const float* partial, int32_t n, float scale, float* out,
                      hipStream_t stream);

hipError_t launch_sgd(float* params, const float* grads, int64_t n, float lr,
                      hipStream_t stream);
// ---------------------------------------------------------------- CTC
// Loss and logit gradient of a batch (packed frames, class 0 = blank).
//   z        [N x C] logits in, gradient d loss / d logits out (x scale)
//   targets  device int32 [B][U_max] label strings
//   tab      device int32 [2B]: target lengths, then sequence lengths
//   e, alpha, beta  device [B][T][S_stride] scratch (S_stride = 64 * states
//            per lane, see ctc_states_per_lane): log emissions and the two
//            shifted log recursions; chain [B][2*U_max] scratch (label
//            chains); lse [N]; loss_part [B] out (per-sequence -ln p, +inf
//            when no path exists)
struct CtcArgs {
  float* z;
  int C;
  const int32_t* bs;
  const int32_t* off;
  int T, B;
  const int32_t* targets;
  int U_max;
  const int32_t* tab;
  int S_stride;
  float* e;
  float* alpha;
  float* beta;
  int32_t* chain;
  float* lse;
  float* loss_part;
  float scale;
};
// States per lane of the sequential kernel for targets of up to U_max
// labels (a power of two, 0 if above 32).
int ctc_states_per_lane(int U_max);
hipError_t launch_ctc(const CtcArgs& a, hipStream_t st);
// dst[i] = values[i] for i < n, from host memory through kernel arguments.
hipError_t launch_store_ints(const int32_t* values, int n, int32_t* dst, hipStream_t st);

// One ADADELTA step over n elements (p, eg2, edx2 updated in place).
hipError_t launch_adadelta(float* p, const float* g, float* eg2, float* edx2, int64_t n,
                           float rho, float eps, float lr, hipStream_t st);
// Eq. 3 in place: replicas r = 0..R-1 at reps + r*stride (16-byte aligned,
// stride % 4 == 0) and prev all receive mean_r(reps) - beta * prev.
hipError_t launch_aggregate(float* reps, int R, int64_t stride, int64_t n, float* prev,
                            float beta, hipStream_t st);

// ---------------------------------------------------------------- recurrent steps
// One time step of one layer/direction over the active rows [0, rows) of the
// batch.  State of row b at the previous step (in recurrence order) lives in
// frame prev0 + b when b < prev_rows, else the state is zero.
struct StepFwdArgs {
  const float* gx;   // [N x G*H] input projection incl. input bias
  const float* whh;  // [G*H x H]
  const float* bhh;  // GRU: [3H] recurrent bias; LSTM: unused
  float* hout;       // layer output, already offset to this direction's columns
  float* stash;      // [N x 4H] gate activations (LSTM i,f,g,o; GRU r,z,n,W_hn h + b_hn)
  float* cst;        // LSTM: [N x H] cell state; GRU: unused
  const float* peep; // LSTM peepholes [3H] (p_i, p_f, p_o), or nullptr
  int32_t H, ldh;
  int32_t row0, rows;
  int32_t prev0, prev_rows;
};

// One step of backpropagation through time.  "next" is the following step
// of the forward recurrence (processed just before this one here).
struct StepBwdArgs {
  const float* da_next;  // LSTM: dA, GRU: dAh rows of the next step
  const float* whh;      // [G*H x H]
  const float* dh_in;    // gradient from above, offset to this direction's columns
  const float* stash;
  const float* cst;      // LSTM cell state
  const float* hout;     // GRU: layer output (previous state), offset to direction
  float* da;             // [N x G*H] LSTM dA / GRU dAx
  float* dah;            // GRU: [N x 3H] dAh
  float* carry;          // [B x H] LSTM: gradient reaching c_t from the next step
                         // (dc*f + peephole terms); GRU: dh*z of the next step
  const float* peep;     // LSTM peepholes [3H], or nullptr
  float* peep_acc;       // with peep: [B x 3H] per-row sums over the steps of
                         // da_i*c_{t-1}, da_f*c_{t-1}, da_o*c_t (zeroed before the first step)
  int32_t H, ldd, ldh;
  int32_t row0, rows;
  int32_t next0, next_rows;
  int32_t prev0, prev_rows;
};

hipError_t launch_step_fwd(const StepFwdArgs& a, int cell, bool bf16, hipStream_t stream);
hipError_t launch_step_bwd(const StepBwdArgs& a, int cell, bool bf16, hipStream_t stream);

// ---------------------------------------------------------------- persistent recurrence
// All T steps of a set of recurrences (the layers of a unidirectional stack,
// or the two directions of one layer) in one resident launch.  Tables
// bs/off are the device batch tables.  Every array published during the
// launch (hout of each unit forward; LSTM dA, GRU dAh and, when read by a
// unit below, GRU dAx backward) must hold the sentinel 0xFFFFFFFF in every
// element when the launch starts.  *fits reports whether the grid can be
// resident at once and the shape is supported; if not, nothing is launched.
constexpr int kMaxUnits = 4;

// Bounded waits of one resident launch.  `gen` identifies the launch: a wait
// that gives up marks its own launch, whose later waits then return at once
// (so it still ends), while other launches keep waiting normally.
// `max_polls` is the poll budget of one wait.  Both are set by the launcher.
struct WaitCtl {
  uint32_t gen;
  uint32_t max_polls;
};

// One (layer, direction) recurrence inside a forward launch.  The input
// projection is done per step inside the kernel: the reduction operand of
// a step is [input row (kin floats, zero-padded to a chunk multiple) ;
// previous state h (H floats)] against [W_ih ; W_hh].
struct FwdUnit {
  const float* in;     // input rows: frame f at in + f*ld_in (packed X or a layer output)
  const float* wih;    // [G*H x kin]
  const float* whh;    // [G*H x H]
  const float* b;      // LSTM b / GRU b_ih [G*H]
  const float* bhh;    // GRU b_hh [3H]; LSTM unused
  float* hout;         // layer output base [N x ldh]; this unit writes columns hcol..hcol+H-1
  float* stash;        // [N x 4H] (LSTM i,f,g,o; GRU r,z,n,W_hn h + b_hn)
  float* cst;          // LSTM [N x H]; GRU unused
  const float* peep;   // LSTM peepholes [3H] (p_i, p_f, p_o), or nullptr
  uint32_t in_bytes;   // bytes of the array `in` addresses (< 2^31 - 16)
  uint32_t out_bytes;  // bytes of hout (< 2^31 - 16)
  unsigned* hx;        // bf16: the output again, rounded to bf16, two units per 32-bit word
                       // ([N x ldh/2] words, same element order as hout): the recurrent
                       // poll reads it instead of hout
  uint32_t hx_bytes;   // bytes of hx's array (< 2^31 - 16)
  const unsigned* inx;  // bf16, above the first layer: the input as bf16 pairs (the packed
                        // copy of the layer below), read instead of `in`; else nullptr
  uint32_t inx_bytes;   // bytes of inx's array (< 2^31 - 16)
  int32_t ld_in, kin;  // input row stride and length
  int32_t in_published;  // 1: `in` is published by another unit of the same launch
  int32_t out_polled;    // bf16: 1 if another unit of the same launch polls hout (its
                         // input, when inx is not given); else hout gets plain stores
  int32_t dir, hcol;     // direction (0 forward in time, 1 reverse) and output column
  int32_t wg_begin;      // first workgroup of this unit
};

// Output layer run by extra workgroups of the forward launch that holds the
// top layer (fp32, per-frame loss): blocks of kOutRows frames in time order,
// each waiting (device-scope polls of the sentinel) for its rows of the top
// layer's published output, then logits = h W_out^T + b_out, softmax
// cross-entropy against the frame's label (loss terms summed per block into
// partial[block]), dlogits = (softmax - onehot) * inv_n into dz, and dh =
// dlogits W_out.  W_out is staged in LDS once per workgroup; usable when
// output_stream_lds(C, Htop) is nonzero.
constexpr int kOutRows = 32;
struct OutStreamArgs {
  const float* h;    // top layer output [N x Htop], published by the launch
  uint32_t h_bytes;  // bytes of h's array (< 2^31 - 16)
  int32_t Htop, C;
  const float* W;    // W_out [C x Htop]
  const float* bias; // b_out [C]
  const int32_t* y;  // packed labels [N]
  int64_t N;
  float inv_n;
  float* dz;         // [N x C]
  float* dh;         // [N x Htop]
  float* partial;    // [nblocks]
  int32_t nblocks;
  // Before the output layer, these workgroups set fill[0..nfill) to the
  // publication sentinel (buffers of a later launch).  After it, the last
  // of them to finish (counted in *done, zero before the launch) writes
  // loss[0] = inv_n * sum of partial, summed in a fixed order.
  FillJob fill[kFillJobs];
  int32_t nfill;
  unsigned* done;
  float* loss;
};
// Output-layer workgroups of a launch at most.
constexpr int kOutStreamGrid = 32;
// Dynamic LDS of an output-layer workgroup (0: shape not supported).
size_t output_stream_lds(int32_t C, int32_t Htop);

struct FwdLaunch {
  FwdUnit u[kMaxUnits];
  int32_t nunits;
  const int32_t* bs;
  const int32_t* off;
  int32_t H, ldh, T;
  int32_t slices, rgroups;  // set by the launcher
  // fp32 only: out_blocks > 0 adds that many output-layer workgroups after
  // the recurrence ones, reading the last unit's published output.
  OutStreamArgs out;
  int32_t out_blocks;
  WaitCtl wait;  // set by the launcher
};

// One (layer, direction) recurrence inside a backward launch.  The
// reduction operand of a step is [gate gradient of the layer above at the
// same frame (k_up floats; absent for the top layer) ; this layer's
// recurrent gate gradient of the next step (G*H floats)] against
// [W_ih of the layer above ; W_hh], restricted to this workgroup's units.
struct BwdUnit {
  const float* up;       // layer above: LSTM dA / GRU dAx rows [N x k_up]; nullptr = none
                         // (bf16 LSTM: bf16 pairs, k_up / 2 words per row, as da below)
  const float* wih_up;   // W_ih of the layer above [k_up x din_up]
  const float* whh;      // [G*H x H]
  const float* dh_in;    // plain gradient w.r.t. this unit's output (column hcol), or nullptr
  const float* stash;    // [N x 4H]
  const float* cst;      // LSTM [N x H]
  const float* hout;     // layer output [N x ldh] (GRU previous state), column hcol
  float* da;             // LSTM dA / GRU dAx [N x G*H]; a bf16 LSTM publishes dA
                         // rounded to bf16, two per 32-bit word ([N x G*H/2] words)
  float* dah;            // GRU dAh [N x 3H]
  float* bias_part;      // [rgroups x G*H]: per row group, sum over frames of dA / dAx
  float* bias_part_h;    // GRU: [rgroups x 3H] sums of dAh
  const float* peep;     // LSTM peepholes [3H], or nullptr
  float* peep_part;      // with peep: [rgroups x 3H] sums of da_i*c_{t-1}, da_f*c_{t-1}, da_o*c_t
  uint32_t up_bytes;     // bytes of `up`'s array (< 2^31 - 16)
  uint32_t rec_bytes;    // bytes of the recurrent array (LSTM da, GRU dah; < 2^31 - 16)
  int32_t k_up, din_up;  // columns of `up` and of W_ih above
  int32_t up_published;  // 1: `up` is published by another unit of this launch
  int32_t publish_dax;   // GRU: 1 if a unit below reads dAx during this launch
  int32_t ld_dh, dir, hcol;
  int32_t wg_begin;
};

// Weight gradients computed by extra workgroups of the backward launch of
// an fp32 LSTM stack: C = A^T B summed over the valid frames, for every
// (A, B) job, while the recurrence is still publishing A.  The frames are
// taken in chunks of `spc` time steps from the last step down (the order the
// recurrence finishes them).  A workgroup of 64*NW threads holds NW/4
// sub-tiles of 256 threads, each owning one 64 x 64 output tile; all of them
// accumulate every `reps`-th chunk (the same chunks, so they keep step at
// the workgroup's barriers) in registers, waiting (device-scope polls of the
// sentinel) for the A rows they read.  Each writes one partial tile;
// partial[r] of job j (r < reps) are then summed in order.
constexpr int kWgJobs = 8;      // two per layer, up to kMaxUnits layers
constexpr int kWgRepsMax = 8;   // workgroups per output tile, at most
struct WgJob {
  const float* A;          // published gate gradients [frames x lda] (LSTM dA)
  uint32_t a_bytes;        // bytes of A's array (< 2^31 - 16)
  int32_t lda;
  const float* B;          // B rows: frame f reads row gather ? gather[f] : f (-1 = zeros)
  int64_t ldb;
  const int32_t* gather;
  int32_t M, N;            // output M x N (M = columns of A used, N = columns of B)
  int32_t tile_begin;      // first tile index of this job
  float* partial;          // [reps][M][N]
};
struct WgStreamArgs {
  WgJob job[kWgJobs];
  int32_t njobs, tiles, reps;
  const int32_t* off;      // device frame offsets per step [T+1]
  int32_t T, spc, nchunks;
};
// One step per chunk: the last chunk, all that is left once the recurrence
// ends, is then a single step's frames (measured against 2, 4 and longer
// chunks, and 4-step chunks ending in single steps).
constexpr int kWgStepsPerChunk = 1;
// Output tiles of one job (64 x 64).
inline int32_t wg_tiles(int32_t M, int32_t N) { return ((M + 63) / 64) * ((N + 63) / 64); }

struct BwdLaunch {
  BwdUnit u[kMaxUnits];
  int32_t nunits;
  const int32_t* bs;
  const int32_t* off;
  int32_t H, ldh, T;
  int32_t slices, rgroups;  // set by the launcher
  // fp32 LSTM only: wg_on adds the weight-gradient workgroups, ceil(tiles /
  // (NW/4)) * reps of them after the recurrence ones (wg_blocks: set by the
  // launcher).
  WgStreamArgs wg;
  int32_t wg_on, wg_blocks;
  WaitCtl wait;  // set by the launcher
};

// Workgroups a forward launch of these units would need (0 = shape not
// supported by the persistent kernel).
int fwd_persistent_blocks(const FwdLaunch& a, int cell, bool bf16, int B);
hipError_t launch_fwd_persistent(FwdLaunch a, int cell, bool bf16, int B, hipStream_t stream,
                                 bool* fits);
int bwd_persistent_blocks(const BwdLaunch& a, int cell, bool bf16, int B);
hipError_t launch_bwd_persistent(BwdLaunch a, int cell, bool bf16, int B, hipStream_t stream,
                                 bool* fits);
// Compute units of the current device (0 on error).
int cu_count();

// Streams that may run persistent launches at once (each launch then claims
// at most 1/streams of the GPU's co-resident capacity).
void set_concurrency(int streams);
int concurrency();
// Number of waits for published values that gave up since the last reset
// (0 unless something went wrong), and its reset to 0 (device synchronous).
hipError_t read_wait_timeouts(unsigned* count);
hipError_t reset_wait_timeouts();
constexpr unsigned kPublishSentinel = 0xFFFFFFFFu;

// out[c * ld_out + r] = in[r * ld_in + c] for r < rows, c < cols.
hipError_t launch_transpose(const float* in, int32_t rows, int32_t cols, int64_t ld_in, float* out,
                            int64_t ld_out, hipStream_t stream);

// Fills n 32-bit words with `value` (a kernel, so it may sit in a captured graph).
hipError_t launch_fill_u32(unsigned* p, int64_t n, unsigned value, hipStream_t stream);

}  // namespace rnnbkt
