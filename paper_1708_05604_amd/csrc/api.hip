// C-ABI entry points of the model calls: argument validation, buffer
// carving, and the enqueue order of the kernels for one mini-batch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "common.h"
#include "kernels.h"

namespace rnnbkt {

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Shape {
  int G, H, D, C, L, dirs, Htop;
  bool bf16;
  int cell;   // RNNBKT_CELL_LSTM (either kind) or RNNBKT_CELL_GRU
  bool peep;  // LSTM with peepholes
  int din(int l) const { return l == 0 ? D : dirs * H; }
};

int32_t check_desc(const rnnbkt_model_desc* d, Shape* s) {
  RNNBKT_REQUIRE(d != nullptr, RNNBKT_EINVAL, "model desc is null");
  RNNBKT_REQUIRE(d->cell == RNNBKT_CELL_LSTM || d->cell == RNNBKT_CELL_GRU ||
                     d->cell == RNNBKT_CELL_LSTM_PEEPHOLE,
                 RNNBKT_EINVAL, "desc.cell must be 0 (LSTM), 1 (GRU) or 2 (peephole LSTM), got %d",
                 d->cell);
  RNNBKT_REQUIRE(d->num_layers >= 1 && d->input_dim >= 1 && d->hidden >= 1 &&
                     d->num_classes >= 1,
                 RNNBKT_EINVAL, "desc sizes must be >= 1");
  RNNBKT_REQUIRE(d->bidirectional == 0 || d->bidirectional == 1, RNNBKT_EINVAL,
                 "desc.bidirectional must be 0 or 1");
  RNNBKT_REQUIRE(d->gemm_dtype == RNNBKT_GEMM_FP32 || d->gemm_dtype == RNNBKT_GEMM_BF16,
                 RNNBKT_EINVAL, "desc.gemm_dtype must be 0 (fp32) or 1 (bf16)");
  RNNBKT_REQUIRE(d->hidden % 32 == 0, RNNBKT_EUNSUPPORTED,
                 "hidden must be a multiple of 32 (got %d)", d->hidden);
  RNNBKT_REQUIRE(d->input_dim % 4 == 0, RNNBKT_EUNSUPPORTED,
                 "input_dim must be a multiple of 4 (got %d)", d->input_dim);
  RNNBKT_REQUIRE(d->num_classes % 4 == 0 && d->num_classes <= 1024, RNNBKT_EUNSUPPORTED,
                 "num_classes must be a multiple of 4 and <= 1024 (got %d)", d->num_classes);
  s->cell = d->cell == RNNBKT_CELL_GRU ? RNNBKT_CELL_GRU : RNNBKT_CELL_LSTM;
  s->peep = d->cell == RNNBKT_CELL_LSTM_PEEPHOLE;
  s->G = s->cell == RNNBKT_CELL_LSTM ? 4 : 3;
  s->H = d->hidden;
  s->D = d->input_dim;
  s->C = d->num_classes;
  s->L = d->num_layers;
  s->dirs = d->bidirectional ? 2 : 1;
  s->Htop = s->dirs * s->H;
  s->bf16 = d->gemm_dtype == RNNBKT_GEMM_BF16;
  return RNNBKT_OK;
}

// Offsets (in floats) of each block of the flat parameter vector.
struct ParamOffsets {
  std::vector<int64_t> wih, whh, b, bhh, peep;  // indexed by layer*dirs + dir
  int64_t wout = 0, bout = 0, total = 0;
};

ParamOffsets param_offsets(const Shape& s) {
  ParamOffsets p;
  int64_t pos = 0;
  const int64_t GH = (int64_t)s.G * s.H;
  for (int l = 0; l < s.L; ++l)
    for (int d = 0; d < s.dirs; ++d) {
      p.wih.push_back(pos);
      pos += GH * s.din(l);
      p.whh.push_back(pos);
      pos += GH * s.H;
      p.b.push_back(pos);
      pos += GH;
      if (s.cell == RNNBKT_CELL_GRU) {
        p.bhh.push_back(pos);
        pos += GH;
      } else {
        p.bhh.push_back(-1);
      }
      if (s.peep) {
        p.peep.push_back(pos);
        pos += 3 * (int64_t)s.H;
      } else {
        p.peep.push_back(-1);
      }
    }
  p.wout = pos;
  pos += (int64_t)s.C * s.Htop;
  p.bout = pos;
  pos += s.C;
  p.total = pos;
  return p;
}

// Split-K choice for the weight-gradient reductions over the frames.
struct SplitK {
  int S;
  int kps;
};

// Slices of the reduction so that a GEMM launches about one round of
// workgroups, each slice at least 256 deep, for output tiles of `tile` x
// `tile`: 768 for the bf16 kernel (three per CU; alone at bilstm3's shapes
// dW_hh 113 -> 88 us against 512, and 120 us with 1024, a second round),
// 256 beside a resident recurrence, which takes half the CUs (bilstm3 +2%
// useful timesteps/s against 512), 1024 for the fp32 kernel's 64 x 64
// tiles (gru2's weight gradients: +3% against 512).  The buffers are sized
// with the largest.
constexpr int64_t kBesideSplitTarget = 256;
SplitK choose_splitk(int64_t M, int64_t N, int64_t K, int tile, bool beside = false) {
  const int64_t tiles = ((M + tile - 1) / tile) * ((N + tile - 1) / tile);
  const int64_t target = tile < 128 ? 1024 : beside ? kBesideSplitTarget : 768;
  int64_t S = std::max<int64_t>(1, (target + tiles - 1) / tiles);
  S = std::min<int64_t>(S, std::max<int64_t>(1, K / 256));
  int64_t kps = (K + S - 1) / S;
  kps = (kps + 31) / 32 * 32;
  S = std::max<int64_t>(1, (K + kps - 1) / kps);
  return SplitK{(int)S, (int)kps};
}

// Column sums: rows are cut into at most kColsumSplits slices.
constexpr int64_t kColsumSplits = 64;
int64_t colsum_rows(int64_t N) { return std::max<int64_t>(1, (N + kColsumSplits - 1) / kColsumSplits); }

// Byte offsets of every buffer a batch uses.
struct Carve {
  // reserve
  size_t bs, off, xp, yp, prev_f, prev_r, dz;
  size_t dhtop;                    // dH of the top layer's output, dZ W_out [N x Htop]
  std::vector<size_t> da, dah;     // backward gate gradients per layer*dirs [N x G*H]
  std::vector<size_t> hout;        // per layer [N x dirs*H]
  std::vector<size_t> stash, cst;  // per layer*dirs
  size_t reserve;
  // workspace (forward)
  size_t gx[2], loss_part;
  size_t out_done;  // counter of the output-layer workgroups that finished
  std::vector<size_t> hx;  // bf16: each layer's output as bf16 pairs, for the recurrent polls
  size_t ws_fwd;
  // workspace (backward)
  size_t dha, dhb, carry, peep_acc, splitk, colsum;
  size_t wt;  // W_ih of a layer above the first, transposed (both directions), for its dX GEMM
  size_t splitk_out, colsum_out;  // output-layer gradients (run beside the recurrence)
  size_t splitk_rec;              // weight gradients on the side stream
  size_t wgpart;                  // streamed weight gradients: partial tiles of every layer
  std::vector<size_t> bpart, bpart_h;  // bias-gradient partials per layer*dirs
  std::vector<size_t> ppart;           // peephole-gradient partials per layer*dirs

  size_t ws_bwd_resident_uni;  // the first bytes, all a resident unidirectional plan uses
  size_t ws_bwd;
  size_t workspace;
};

Carve carve(const Shape& s, int T, int B, int64_t N) {
  Carve c{};
  const int64_t GH = (int64_t)s.G * s.H;
  size_t pos = 0;
  auto take = [&](size_t bytes) {
    const size_t at = pos;
    pos = align_up(pos + bytes);
    return at;
  };
  c.bs = take(sizeof(int32_t) * T);
  c.off = take(sizeof(int32_t) * (T + 1));
  c.xp = take(sizeof(float) * N * s.D);
  c.yp = take(sizeof(int32_t) * N);
  c.prev_f = take(sizeof(int32_t) * N);
  c.prev_r = take(sizeof(int32_t) * N);
  c.dz = take(sizeof(float) * N * s.C);
  c.dhtop = take(sizeof(float) * N * s.Htop);
  // The backward's gate gradients, exchanged between its workgroups: kept
  // here so that the forward can set their sentinel beside its recurrence.
  // (A bf16 LSTM's resident backward fills the first half, as bf16 pairs.)
  for (int q = 0; q < s.L * s.dirs; ++q) {
    c.da.push_back(take(sizeof(float) * N * GH));
    c.dah.push_back(s.cell == RNNBKT_CELL_GRU ? take(sizeof(float) * N * GH) : 0);
  }
  for (int l = 0; l < s.L; ++l) c.hout.push_back(take(sizeof(float) * N * s.dirs * s.H));
  for (int l = 0; l < s.L; ++l)
    for (int d = 0; d < s.dirs; ++d) {
      c.stash.push_back(take(sizeof(float) * N * 4 * s.H));
      c.cst.push_back(s.cell == RNNBKT_CELL_LSTM ? take(sizeof(float) * N * s.H) : 0);
    }
  c.reserve = pos;

  pos = 0;
  const size_t common = pos;
  for (int d = 0; d < 2; ++d) c.gx[d] = d < s.dirs ? take(sizeof(float) * N * GH) : c.gx[0];
  c.loss_part = take(sizeof(float) * ((N + 15) / 16 + 1));
  c.out_done = take(sizeof(unsigned));
  for (int l = 0; l < s.L; ++l) c.hx.push_back(s.bf16 ? take(2 * (size_t)N * s.dirs * s.H) : 0);
  c.ws_fwd = pos;

  pos = common;
  // Backward, first what every resident (persistent) launch plan of a
  // unidirectional stack uses: the output layer's split-K partials and
  // column sums, the weight-gradient partials, the bias partials.
  const int tile = gemm_tile(s.bf16);
  size_t sk = 0;
  auto need = [&](int64_t M, int64_t Nn, int64_t K) {
    const SplitK p = choose_splitk(M, Nn, K, tile);
    if (p.S > 1) sk = std::max(sk, (size_t)p.S * M * Nn);
  };
  {
    const SplitK p = choose_splitk(s.C, s.Htop, N, tile);
    c.splitk_out = take(sizeof(float) * (p.S > 1 ? (size_t)p.S * s.C * s.Htop : 1));
  }
  c.colsum_out = take(sizeof(float) * kColsumSplits * s.C);
  {
    // Products on the side stream: dW_hh, and dW_ih of layers whose weight
    // gradients run beside the recurrence of the layers below.
    size_t rec = 1;
    for (int l = 0; l < s.L; ++l)
      for (const int64_t cols : {(int64_t)s.H, (int64_t)s.din(l)}) {
        const SplitK p = choose_splitk(GH, cols, N, tile);
        if (p.S > 1) rec = std::max(rec, (size_t)p.S * GH * cols);
      }
    c.splitk_rec = take(sizeof(float) * rec);
  }
  {
    size_t wg = 0;  // kWgRepsMax partial copies of dW_ih and dW_hh of every layer
    if (s.dirs == 1 && s.cell == RNNBKT_CELL_LSTM && !s.bf16)
      for (int l = 0; l < s.L; ++l) wg += (size_t)kWgRepsMax * GH * (s.din(l) + s.H);
    c.wgpart = take(sizeof(float) * std::max<size_t>(wg, 1));
  }
  for (int l = 0; l < s.L; ++l) {
    need(GH, s.din(l), N);
    need(GH, s.H, N);
  }
  c.splitk = take(sizeof(float) * std::max<size_t>(sk, 1));
  const int rgroups = (B + 15) / 16;
  for (int q = 0; q < s.L * s.dirs; ++q) {
    c.bpart.push_back(take(sizeof(float) * rgroups * GH));
    c.bpart_h.push_back(s.cell == RNNBKT_CELL_GRU ? take(sizeof(float) * rgroups * GH) : 0);
    c.ppart.push_back(s.peep ? take(sizeof(float) * rgroups * 3 * s.H) : 0);
  }
  c.ws_bwd_resident_uni = pos;
  // Then what only the per-step kernels or bidirectional layers use: the
  // gradient w.r.t. a layer's input between layer launches (ping-pong), the
  // per-step carries and running sums, column-sum partials.
  c.wt = take(sizeof(float) * 2 * (size_t)s.Htop * GH);
  c.dha = take(sizeof(float) * N * s.Htop);
  c.dhb = take(sizeof(float) * N * s.Htop);
  c.carry = take(sizeof(float) * (size_t)B * s.H);
  c.peep_acc = s.peep ? take(sizeof(float) * (size_t)B * 3 * s.H) : 0;
  // Column sums run over N frames (bias gradients) or B rows (peephole
  // running sums): at most kColsumSplits partial rows either way.
  c.colsum = take(sizeof(float) * kColsumSplits * std::max<int64_t>(GH, s.C));
  c.ws_bwd = pos;
  c.workspace = std::max(c.ws_fwd, c.ws_bwd);
  return c;
}

int32_t check_lengths(const int32_t* lengths, int T, int B, int64_t* n_valid) {
  RNNBKT_REQUIRE(lengths != nullptr, RNNBKT_EINVAL, "lengths is null");
  RNNBKT_REQUIRE(B >= 1, RNNBKT_EINVAL, "batch size must be >= 1 (got %d)", B);
  RNNBKT_REQUIRE(T >= 1, RNNBKT_EINVAL, "T_max must be >= 1 (got %d)", T);
  RNNBKT_REQUIRE(lengths[0] == T, RNNBKT_EINVAL, "lengths[0] (%d) must equal T_max (%d)",
                 lengths[0], T);
  int64_t n = 0;
  for (int b = 0; b < B; ++b) {
    RNNBKT_REQUIRE(lengths[b] >= 1, RNNBKT_EINVAL, "lengths[%d] = %d < 1", b, lengths[b]);
    RNNBKT_REQUIRE(b == 0 || lengths[b] <= lengths[b - 1], RNNBKT_EINVAL,
                   "lengths must be non-increasing (lengths[%d] = %d > lengths[%d] = %d)", b,
                   lengths[b], b - 1, lengths[b - 1]);
    n += lengths[b];
  }
  RNNBKT_REQUIRE(n <= (int64_t)INT32_MAX / 4, RNNBKT_EUNSUPPORTED,
                 "too many valid frames in one batch (%lld)", (long long)n);
  *n_valid = n;
  return RNNBKT_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

#define RNNBKT_HIP(expr)                                                              \
  do {                                                                                \
    hipError_t _e = (expr);                                                           \
    if (_e != hipSuccess) {                                                           \
      ::rnnbkt::set_error("%s failed: %s", #expr, hipGetErrorString(_e));             \
      return RNNBKT_EHIP;                                                             \
    }                                                                                 \
  } while (0)

// ---------------------------------------------------------------- kernel timer
struct TimerRec {
  int kind;
  hipEvent_t a, b;
  double flops, bytes;
};
std::mutex g_tmu;
bool g_timer_on = false;
std::vector<TimerRec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t pooled_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Brackets one launch with events when the timer is on.
bool is_side_stream(hipStream_t st);

// Work recorded on an internal side stream counts as RNNBKT_KERNEL_SIDE
// whatever kind it is.
class Timed {
 public:
  Timed(int kind, double flops, double bytes, hipStream_t st) : st_(st) {
    if (!g_timer_on) return;
    if (is_side_stream(st)) kind = RNNBKT_KERNEL_SIDE;
    std::lock_guard<std::mutex> lk(g_tmu);
    rec_.kind = kind;
    rec_.flops = flops;
    rec_.bytes = bytes;
    rec_.a = pooled_event();
    rec_.b = pooled_event();
    if (rec_.a && rec_.b && hipEventRecord(rec_.a, st_) == hipSuccess) active_ = true;
  }
  ~Timed() {
    if (!active_) return;
    std::lock_guard<std::mutex> lk(g_tmu);
    if (hipEventRecord(rec_.b, st_) == hipSuccess) g_recs.push_back(rec_);
  }

 private:
  hipStream_t st_;
  TimerRec rec_{};
  bool active_ = false;
};

// A side stream per caller stream, with the two events that fork work onto
// it and join it back.  Created on first use and kept for the process.
struct Side {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;
std::vector<std::pair<hipStream_t, Side>> g_sides;

bool is_side_stream(hipStream_t st) {
  std::lock_guard<std::mutex> lk(g_side_mu);
  for (auto& e : g_sides)
    if (e.second.s == st) return true;
  return false;
}

hipError_t side_for(hipStream_t st, Side* out) {
  std::lock_guard<std::mutex> lk(g_side_mu);
  for (auto& e : g_sides)
    if (e.first == st) {
      *out = e.second;
      return hipSuccess;
    }
  Side sd;
  hipError_t e = hipStreamCreateWithFlags(&sd.s, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&sd.fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&sd.join, hipEventDisableTiming);
  if (e != hipSuccess) return e;
  g_sides.emplace_back(st, sd);
  *out = sd;
  return hipSuccess;
}

// Reserve buffers whose backward exchange buffers (dA, GRU dAh) the last
// forward on them left holding the sentinel; the backward takes the mark, or
// sets the sentinel itself.
std::mutex g_pre_mu;
std::vector<const void*> g_prefilled;

void note_prefilled(const void* reserve, bool yes) {
  std::lock_guard<std::mutex> lk(g_pre_mu);
  auto it = std::find(g_prefilled.begin(), g_prefilled.end(), reserve);
  if (yes && it == g_prefilled.end()) g_prefilled.push_back(reserve);
  if (!yes && it != g_prefilled.end()) g_prefilled.erase(it);
}

bool take_prefilled(const void* reserve) {
  std::lock_guard<std::mutex> lk(g_pre_mu);
  auto it = std::find(g_prefilled.begin(), g_prefilled.end(), reserve);
  if (it == g_prefilled.end()) return false;
  g_prefilled.erase(it);
  return true;
}

// Host copy of the batch tables (active rows per step and frame offsets).
void host_tables(const int32_t* len, int T, int B, std::vector<int>& bs, std::vector<int>& off) {
  bs.assign(T, 0);
  off.assign(T + 1, 0);
  for (int b = 0; b < B; ++b)
    for (int t = 0; t < len[b]; ++t) bs[t]++;
  for (int t = 0; t < T; ++t) off[t + 1] = off[t] + bs[t];
}

// Recurrence kernels: "persistent" (default; all steps of a layer in one
// launch) or "steps" (one launch per time step).  RNNBKT_RECURRENCE selects.
bool use_persistent() {
  const char* e = getenv("RNNBKT_RECURRENCE");
  return !(e && strcmp(e, "steps") == 0);
}

template <typename P>
P* at(void* base, size_t off) {
  return reinterpret_cast<P*>(static_cast<char*>(base) + off);
}
template <typename P>
const P* at(const void* base, size_t off) {
  return reinterpret_cast<const P*>(static_cast<const char*>(base) + off);
}

// Second reduction term of a GEMM: C += op(A2) op(B2) over K2 (see GemmArgs).
struct Term2 {
  const float* A2;
  int64_t lda2;
  const float* B2;
  int64_t ldb2;
  int K2;
};

hipError_t gemm(const float* A, int64_t lda, bool a_kc, const float* Bm, int64_t ldb, bool b_kc,
                float* C, int64_t ldc, int M, int N, int K, const float* bias, int accumulate,
                bool bf16, hipStream_t st, const int32_t* gather = nullptr,
                float* splitk_buf = nullptr, const Term2* t2 = nullptr, bool beside = false,
                bool a_bf16 = false) {
  GemmArgs g{};
  g.beside = beside ? 1 : 0;
  g.a_bf16 = a_bf16 ? 1 : 0;
  if (t2) {
    g.A2 = t2->A2;
    g.lda2 = t2->lda2;
    g.B2 = t2->B2;
    g.ldb2 = t2->ldb2;
    g.K2 = t2->K2;
  }
  g.A = A;
  g.B = Bm;
  g.C = C;
  g.bias = bias;
  g.gather_b = gather;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.M = M;
  g.N = N;
  g.K = K;
  g.accumulate = accumulate;
  g.splits = 1;
  g.k_per_split = (K + 31) / 32 * 32;
  if (splitk_buf && !t2) {
    const SplitK p = choose_splitk(M, N, K, gemm_tile(bf16), beside);
    g.splits = p.S;
    g.k_per_split = p.kps;
    g.partial = splitk_buf;
  }
  if (M == 0 || N == 0) return hipSuccess;
  Timed tm(RNNBKT_KERNEL_GEMM, 2.0 * M * N * (K + (t2 ? t2->K2 : 0)), 0.0, st);
  hipError_t e = launch_gemm(g, a_kc, b_kc, bf16, st);
  if (e != hipSuccess || g.splits == 1) return e;
  return launch_splitk_reduce(splitk_buf, g.splits, M, N, C, ldc, bias, accumulate, st);
}

}  // namespace

}  // namespace rnnbkt

using namespace rnnbkt;

extern "C" const char* rnnbkt_version(void) { return "rnnbkt 0.1.0 gfx950"; }

extern "C" int32_t rnnbkt_sync_check(void* stream) {
  clear_error();
  RNNBKT_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
  RNNBKT_HIP(hipGetLastError());
  unsigned timeouts = 0;
  RNNBKT_HIP(read_wait_timeouts(&timeouts));
  if (timeouts != 0) {
    // Reported once: the count restarts, and later launches were never
    // affected (each launch only abandons its own waits).
    RNNBKT_HIP(reset_wait_timeouts());
    RNNBKT_REQUIRE(false, RNNBKT_EHIP,
                   "%u waits for values published by other workgroups timed out: results of the "
                   "affected launches are invalid",
                   timeouts);
  }
  return RNNBKT_OK;
}

extern "C" int64_t rnnbkt_param_count(const rnnbkt_model_desc* desc) {
  clear_error();
  Shape s;
  const int32_t rc = check_desc(desc, &s);
  if (rc != RNNBKT_OK) return rc;
  return param_offsets(s).total;
}

extern "C" int32_t rnnbkt_buffer_sizes(const rnnbkt_model_desc* desc, int32_t T_max, int32_t B,
                                       int64_t n_valid, size_t* reserve_bytes,
                                       size_t* workspace_bytes) {
  clear_error();
  Shape s;
  int32_t rc = check_desc(desc, &s);
  if (rc != RNNBKT_OK) return rc;
  RNNBKT_REQUIRE(reserve_bytes && workspace_bytes, RNNBKT_EINVAL, "null output pointer");
  RNNBKT_REQUIRE(T_max >= 1 && B >= 1 && n_valid >= 1 && n_valid <= (int64_t)T_max * B,
                 RNNBKT_EINVAL, "need T_max >= 1, B >= 1, 1 <= n_valid <= T_max*B");
  const Carve c = carve(s, T_max, B, n_valid);
  *reserve_bytes = c.reserve;
  *workspace_bytes = c.workspace;
  return RNNBKT_OK;
}

namespace {

// CTC scratch of a batch: per-sequence table (target and sequence lengths),
// log emissions and the two log recursions [B][T][S_stride], label chains,
// per-frame log-sum-exp, per-sequence losses.
struct CtcCarve {
  size_t tab, e, alpha, beta, chain, lse, loss_part, total;
  int S_stride;
};

CtcCarve ctc_carve(int T, int B, int U_max) {
  CtcCarve c{};
  c.S_stride = 64 * ctc_states_per_lane(U_max);
  size_t pos = 0;
  auto take = [&](size_t bytes) {
    const size_t at = pos;
    pos = align_up(pos + bytes);
    return at;
  };
  const size_t rows = (size_t)B * T * c.S_stride;
  c.tab = take(sizeof(int32_t) * 2 * B);
  c.e = take(sizeof(float) * rows);
  c.alpha = take(sizeof(float) * rows);
  c.beta = take(sizeof(float) * rows);
  c.chain = take(sizeof(int32_t) * 2 * (size_t)B * U_max);
  c.lse = take(sizeof(float) * (size_t)B * T);
  c.loss_part = take(sizeof(float) * B);
  c.total = pos;
  return c;
}

struct CtcInputs {
  const int32_t* targets;
  const int32_t* target_lengths;
  int32_t U_max;
  void* ws;
  size_t ws_bytes;
};

int32_t forward(const rnnbkt_model_desc* desc, const float* params, const float* x,
                const int32_t* labels, const CtcInputs* ctc, const int32_t* lengths, int32_t T,
                int32_t B, void* reserve, size_t reserve_bytes, void* workspace,
                size_t workspace_bytes, float* loss, void* stream) {
  clear_error();
  Shape s;
  int32_t rc = check_desc(desc, &s);
  if (rc != RNNBKT_OK) return rc;
  int64_t N = 0;
  rc = check_lengths(lengths, T, B, &N);
  if (rc != RNNBKT_OK) return rc;
  RNNBKT_REQUIRE(params && x && (labels || ctc) && reserve && workspace && loss, RNNBKT_EINVAL,
                 "lstm_fwd: null pointer");
  CtcCarve cc{};
  if (ctc) {
    RNNBKT_REQUIRE(ctc->targets && ctc->target_lengths && ctc->ws, RNNBKT_EINVAL,
                   "lstm_fwd_ctc: null pointer");
    RNNBKT_REQUIRE(ctc->U_max >= 1, RNNBKT_EINVAL, "lstm_fwd_ctc: U_max must be >= 1");
    RNNBKT_REQUIRE(ctc_states_per_lane(ctc->U_max) > 0, RNNBKT_EUNSUPPORTED,
                   "lstm_fwd_ctc: targets longer than 1023 labels are not supported");
    RNNBKT_REQUIRE(aligned16(ctc->ws), RNNBKT_EINVAL, "lstm_fwd_ctc: ctc_ws must be 16-byte aligned");
    for (int b = 0; b < B; ++b)
      RNNBKT_REQUIRE(ctc->target_lengths[b] >= 1 && ctc->target_lengths[b] <= ctc->U_max &&
                         ctc->target_lengths[b] <= lengths[b],
                     RNNBKT_EINVAL,
                     "lstm_fwd_ctc: target_lengths[%d] = %d outside [1, min(U_max %d, length %d)]",
                     b, ctc->target_lengths[b], ctc->U_max, lengths[b]);
    cc = ctc_carve(T, B, ctc->U_max);
    RNNBKT_REQUIRE(ctc->ws_bytes >= cc.total, RNNBKT_EINVAL,
                   "lstm_fwd_ctc: ctc_ws too small (%zu < %zu)", ctc->ws_bytes, cc.total);
  }
  RNNBKT_REQUIRE(aligned16(params) && aligned16(x) && aligned16(reserve) && aligned16(workspace),
                 RNNBKT_EINVAL, "lstm_fwd: params, x, reserve and workspace must be 16-byte aligned");
  const Carve c = carve(s, T, B, N);
  RNNBKT_REQUIRE(reserve_bytes >= c.reserve && workspace_bytes >= c.workspace, RNNBKT_EINVAL,
                 "lstm_fwd: buffers too small (reserve %zu < %zu or workspace %zu < %zu)",
                 reserve_bytes, c.reserve, workspace_bytes, c.workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  RNNBKT_HIP(hipGetLastError());
  const ParamOffsets po = param_offsets(s);
  std::vector<int> bs, off;
  host_tables(lengths, T, B, bs, off);

  int32_t* d_bs = at<int32_t>(reserve, c.bs);
  int32_t* d_off = at<int32_t>(reserve, c.off);
  float* Xp = at<float>(reserve, c.xp);
  int32_t* Yp = at<int32_t>(reserve, c.yp);
  int32_t* pf = at<int32_t>(reserve, c.prev_f);
  int32_t* pr = at<int32_t>(reserve, c.prev_r);
  float* dz = at<float>(reserve, c.dz);
  float* lp = at<float>(workspace, c.loss_part);

  const int GH = s.G * s.H;
  const int ldh = s.dirs * s.H;
  const bool persist = use_persistent();
  // Batch tables, packing and, for the resident kernels, the sentinel in
  // every layer's output: one launch when the batch fits its arguments.
  // The CTC loss has no per-frame labels: nothing to pack (labels are read
  // only when given somewhere to put them).
  // The backward's exchange buffers, which the forward sets to the
  // sentinel when the resident kernels run: beside the recurrence (by the
  // output-layer workgroups) when the output layer runs there, else here.
  FillJob bwd_fill[kFillJobs];
  int nbwd = 0;
  if (persist && s.L * s.dirs * (s.cell == RNNBKT_CELL_GRU ? 2 : 1) <= kFillJobs) {
    for (int q = 0; q < s.L * s.dirs; ++q) {
      // (a bf16 LSTM's resident backward publishes packed bf16: half the words)
      bwd_fill[nbwd++] = {reinterpret_cast<unsigned*>(at<float>(reserve, c.da[q])),
                          s.bf16 && s.cell != RNNBKT_CELL_GRU ? N * GH / 2 : N * GH};
      if (s.cell == RNNBKT_CELL_GRU)
        bwd_fill[nbwd++] = {reinterpret_cast<unsigned*>(at<float>(reserve, c.dah[q])), N * GH};
    }
  }
  unsigned* out_done = at<unsigned>(workspace, c.out_done);
  // Set again below once this call has enqueued the fills: a call that
  // fails part-way leaves no mark behind.
  note_prefilled(reserve, false);
  bool prefilled = false;
  {
    // Sentinels: every layer output (bf16: its packed copy, which the
    // recurrence and the layer above poll instead), then the output-layer
    // workgroups' loss partials.
    std::vector<FillJob> jobs;
    if (persist) {
      for (int l = 0; l < s.L; ++l) {
        if (!s.bf16)
          jobs.push_back({reinterpret_cast<unsigned*>(at<float>(reserve, c.hout[l])), N * ldh});
        if (s.bf16) jobs.push_back({at<unsigned>(workspace, c.hx[l]), N * ldh / 2});
      }
      jobs.push_back({reinterpret_cast<unsigned*>(lp), (N + kOutRows - 1) / kOutRows});
    }
    FillJob pre[kFillJobs];
    const int npre = (int)jobs.size();
    for (int q = 0; q < npre && q < kFillJobs; ++q) pre[q] = jobs[q];
    // Bytes moved: each valid frame's features and label read and written
    // packed, its two neighbour indices written, the tables, the fills.
    double moved = (double)N * (8.0 * s.D + (ctc ? 0.0 : 8.0) + 8.0) + 8.0 * (T + 1);
    for (const FillJob& j : jobs) moved += 4.0 * (double)j.n;
    Timed tm(RNNBKT_KERNEL_PREPARE, 0.0, moved, st);
    if (B <= kPrepMaxB && npre <= kFillJobs) {
      RNNBKT_HIP(launch_prepare(lengths, B, T, x, ctc ? nullptr : labels, s.D, d_bs, d_off, Xp,
                                ctc ? nullptr : Yp, pf, pr, pre, npre, kPublishSentinel, out_done,
                                st));
      prefilled = true;
    } else {
      RNNBKT_HIP(launch_batch_tables(lengths, B, T, d_bs, d_off, st));
      RNNBKT_HIP(launch_pack(x, ctc ? nullptr : labels, d_bs, d_off, T, B, s.D, Xp,
                             ctc ? nullptr : Yp, pf, pr, st));
      RNNBKT_HIP(launch_fill_u32(out_done, 1, 0u, st));
      RNNBKT_HIP(launch_fill_u32(reinterpret_cast<unsigned*>(lp), (N + kOutRows - 1) / kOutRows,
                                 kPublishSentinel, st));
    }
  }

  const uint64_t hout_bytes = sizeof(float) * (uint64_t)N * ldh;
  // One recurrence unit (layer l, direction d) of a persistent launch.
  auto make_unit = [&](int l, int d, bool in_published) {
    FwdUnit u{};
    const int ld = l * s.dirs + d;
    u.in = l == 0 ? Xp : at<float>(reserve, c.hout[l - 1]);
    u.ld_in = s.din(l);
    u.kin = s.din(l);
    const uint64_t ib = sizeof(float) * (uint64_t)N * u.ld_in;
    u.in_bytes = ib < 0x7FFFFFF0u ? (uint32_t)ib : 0x7FFFFFF0u;
    u.in_published = in_published ? 1 : 0;
    u.wih = params + po.wih[ld];
    u.whh = params + po.whh[ld];
    u.b = params + po.b[ld];
    u.bhh = s.cell == RNNBKT_CELL_GRU ? params + po.bhh[ld] : nullptr;
    u.hout = at<float>(reserve, c.hout[l]);
    u.out_bytes = hout_bytes < 0x7FFFFFF0u ? (uint32_t)hout_bytes : 0x7FFFFFF0u;
    if (s.bf16) {
      u.hx = at<unsigned>(workspace, c.hx[l]);
      u.hx_bytes = hout_bytes / 2 < 0x7FFFFFF0u ? (uint32_t)(hout_bytes / 2) : 0x7FFFFFF0u;
      if (l > 0) {
        // the layer below's packed copy (rows of din = dirs*H elements): the
        // layers that run resident are a prefix of the stack (the first that
        // does not fit sends itself and those above to the per-step kernels),
        // so that copy is complete, or published within the same launch
        u.inx = at<unsigned>(workspace, c.hx[l - 1]);
        u.inx_bytes = u.hx_bytes;
      }
    }
    u.stash = at<float>(reserve, c.stash[ld]);
    u.cst = s.cell == RNNBKT_CELL_LSTM ? at<float>(reserve, c.cst[ld]) : nullptr;
    u.peep = s.peep ? params + po.peep[ld] : nullptr;
    u.dir = d;
    u.hcol = d * s.H;
    return u;
  };
  auto base_launch = [&]() {
    FwdLaunch L{};
    L.bs = d_bs;
    L.off = d_off;
    L.H = s.H;
    L.ldh = ldh;
    L.T = T;
    return L;
  };
  // Algorithmic flops of the step products of one unit.
  auto unit_flops = [&](int l) {
    double fl = 0;
    for (int t = 0; t < T; ++t) fl += 2.0 * bs[t] * GH * (s.din(l) + s.H);
    return fl;
  };
  // Layers [l, l+n) of a unidirectional stack in one launch, each layer
  // reading the one below as it is published.  Returns the largest n that
  // the persistent kernel can keep resident (0 if none).
  auto stack_fits = [&](int l0) {
    int best = 0;
    for (int n = 1; n <= kMaxUnits && l0 + n <= s.L; ++n) {
      FwdLaunch L = base_launch();
      for (int q = 0; q < n; ++q) L.u[q] = make_unit(l0 + q, 0, q > 0);
      L.nunits = n;
      if (fwd_persistent_blocks(L, s.cell, s.bf16, B) > 0) best = n;
    }
    return best;
  };
  // Output layer and loss run by extra workgroups of the launch that holds
  // the top layer, on its rows as they are published: fp32 with per-frame
  // labels, W_out plus a block of rows within a workgroup's LDS, and the
  // grid still resident with them; one stream declared (several streams
  // already fill the GPU between them).  RNNBKT_OUTPUT=after runs them after
  // the recurrence as separate kernels.
  const char* out_env = getenv("RNNBKT_OUTPUT");
  const bool stream_out_ok = concurrency() == 1 && !ctc && !s.bf16 &&
                             output_stream_lds(s.C, s.Htop) > 0 &&
                             hout_bytes < 0x7FFFFFF0u &&
                             !(out_env && strcmp(out_env, "after") == 0);
  const int nblk = (int)((N + kOutRows - 1) / kOutRows);
  bool streamed_out = false;
  std::vector<char> layer_done(s.L, 0);
  if (persist) {
    int l = 0;
    while (l < s.L) {
      FwdLaunch L = base_launch();
      int n = 0;
      if (s.dirs == 1) {
        n = stack_fits(l);
        for (int q = 0; q < n; ++q) {
          L.u[q] = make_unit(l + q, 0, q > 0);
          // (bf16: the layer above reads the packed copy instead)
          L.u[q].out_polled = q + 1 < n && !s.bf16 ? 1 : 0;
        }
      } else {
        n = 1;
        for (int d = 0; d < 2; ++d) L.u[d] = make_unit(l, d, false);
      }
      L.nunits = s.dirs == 1 ? n : 2;
      bool fits = false;
      if (n > 0) {
        double fl = 0;
        for (int q = 0; q < n; ++q) fl += s.dirs * unit_flops(l + q);
        if (!prefilled) {
          Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
          for (int q = 0; q < n; ++q) {
            RNNBKT_HIP(launch_fill_u32(reinterpret_cast<unsigned*>(at<float>(reserve, c.hout[l + q])),
                                       N * ldh, kPublishSentinel, st));
            if (s.bf16)
              RNNBKT_HIP(launch_fill_u32(at<unsigned>(workspace, c.hx[l + q]), N * ldh / 2,
                                         kPublishSentinel, st));
          }
        }
        if (l + n == s.L && stream_out_ok) {
          OutStreamArgs& oa = L.out;
          oa.h = at<float>(reserve, c.hout[s.L - 1]);
          oa.h_bytes = (uint32_t)hout_bytes;
          oa.Htop = s.Htop;
          oa.C = s.C;
          oa.W = params + po.wout;
          oa.bias = params + po.bout;
          oa.y = Yp;
          oa.N = N;
          oa.inv_n = 1.0f / (float)N;
          oa.dz = dz;
          oa.dh = at<float>(reserve, c.dhtop);
          oa.partial = lp;
          oa.nblocks = nblk;
          for (int q = 0; q < nbwd; ++q) oa.fill[q] = bwd_fill[q];
          oa.nfill = nbwd;
          oa.done = out_done;
          oa.loss = loss;
          L.out_blocks = std::min(kOutStreamGrid, nblk);
          if (fwd_persistent_blocks(L, s.cell, s.bf16, B) == 0) L.out_blocks = 0;
        }
        Timed tm(RNNBKT_KERNEL_STEP_FWD, fl, 0.0, st);
        RNNBKT_HIP(launch_fwd_persistent(L, s.cell, s.bf16, B, st, &fits));
        streamed_out = fits && L.out_blocks > 0;
      }
      if (!fits) break;  // this layer and the ones above take the per-step kernels
      for (int q = 0; q < n; ++q) layer_done[l + q] = 1;
      l += n;
    }
  }
  // Per-step kernels for layers the persistent kernel does not take: input
  // projection of all frames as one GEMM, then one launch per time step.
  for (int l = 0; l < s.L; ++l) {
    if (layer_done[l]) continue;
    const float* xin = l == 0 ? Xp : at<float>(reserve, c.hout[l - 1]);
    const int din = s.din(l);
    float* hout = at<float>(reserve, c.hout[l]);
    for (int d = 0; d < s.dirs; ++d) {
      const int ld = l * s.dirs + d;
      RNNBKT_HIP(gemm(xin, din, true, params + po.wih[ld], din, true, at<float>(workspace, c.gx[d]),
                      GH, (int)N, GH, din, params + po.b[ld], 0, s.bf16, st));
    }
    for (int d = 0; d < s.dirs; ++d) {
      const int ld = l * s.dirs + d;
      StepFwdArgs a{};
      a.gx = at<float>(workspace, c.gx[d]);
      a.whh = params + po.whh[ld];
      a.bhh = s.cell == RNNBKT_CELL_GRU ? params + po.bhh[ld] : nullptr;
      a.hout = hout + d * s.H;
      a.stash = at<float>(reserve, c.stash[ld]);
      a.cst = s.cell == RNNBKT_CELL_LSTM ? at<float>(reserve, c.cst[ld]) : nullptr;
      a.peep = s.peep ? params + po.peep[ld] : nullptr;
      a.H = s.H;
      a.ldh = ldh;
      for (int k = 0; k < T; ++k) {
        const int t = d == 0 ? k : T - 1 - k;
        a.row0 = off[t];
        a.rows = bs[t];
        if (d == 0) {
          a.prev0 = t > 0 ? off[t - 1] : 0;
          a.prev_rows = t > 0 ? bs[t] : 0;
        } else {
          a.prev0 = t + 1 < T ? off[t + 1] : 0;
          a.prev_rows = t + 1 < T ? bs[t + 1] : 0;
        }
        Timed tm(RNNBKT_KERNEL_STEP_FWD, 2.0 * a.prev_rows * GH * s.H, 0.0, st);
        RNNBKT_HIP(launch_step_fwd(a, s.cell, s.bf16, st));
      }
    }
  }
  // The loss was summed by the output-layer workgroups, which also set the
  // backward's sentinels; otherwise they are set here (the separate output
  // kernels below run after this launch).
  if (!streamed_out && nbwd > 0) {
    Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
    RNNBKT_HIP(launch_prepare(nullptr, 0, 0, nullptr, nullptr, 0, nullptr, nullptr, nullptr,
                              nullptr, nullptr, nullptr, bwd_fill, nbwd, kPublishSentinel, nullptr,
                              st));
  }
  note_prefilled(reserve, nbwd > 0);
  if (streamed_out) return RNNBKT_OK;
  // Output layer and loss, then dH of the top layer for the backward.
  const float* top = at<float>(reserve, c.hout[s.L - 1]);
  float* dhtop = at<float>(reserve, c.dhtop);
  RNNBKT_HIP(gemm(top, s.Htop, true, params + po.wout, s.Htop, true, dz, s.C, (int)N, s.C,
                  s.Htop, params + po.bout, 0, s.bf16, st));
  if (ctc) {
    CtcArgs a{};
    a.z = dz;
    a.C = s.C;
    a.bs = d_bs;
    a.off = d_off;
    a.T = T;
    a.B = B;
    a.targets = ctc->targets;
    a.U_max = ctc->U_max;
    int32_t* tab = at<int32_t>(ctc->ws, cc.tab);
    a.tab = tab;
    a.S_stride = cc.S_stride;
    a.e = at<float>(ctc->ws, cc.e);
    a.alpha = at<float>(ctc->ws, cc.alpha);
    a.beta = at<float>(ctc->ws, cc.beta);
    a.chain = at<int32_t>(ctc->ws, cc.chain);
    a.lse = at<float>(ctc->ws, cc.lse);
    a.loss_part = at<float>(ctc->ws, cc.loss_part);
    a.scale = 1.0f / (float)B;
    {
      Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
      RNNBKT_HIP(launch_store_ints(ctc->target_lengths, B, tab, st));
      RNNBKT_HIP(launch_store_ints(lengths, B, tab + B, st));
    }
    {
      Timed tm(RNNBKT_KERNEL_XENT, 0.0, (8.0 * s.C + 4.0) * N, st);
      RNNBKT_HIP(launch_ctc(a, st));
    }
    {
      Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
      RNNBKT_HIP(launch_sum(a.loss_part, B, 1.0f / (float)B, loss, st));
    }
    RNNBKT_HIP(gemm(dz, s.C, true, params + po.wout, s.Htop, false, dhtop, s.Htop, (int)N,
                    s.Htop, s.C, nullptr, 0, s.bf16, st));
    return RNNBKT_OK;
  }
  int32_t nparts = 0;
  {
    Timed tm(RNNBKT_KERNEL_XENT, 0.0, (8.0 * s.C + 4.0) * N, st);
    RNNBKT_HIP(launch_softmax_xent(dz, Yp, N, s.C, lp, &nparts, st));
  }
  {
    Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
    RNNBKT_HIP(launch_sum(lp, nparts, 1.0f / (float)N, loss, st));
  }
  RNNBKT_HIP(gemm(dz, s.C, true, params + po.wout, s.Htop, false, dhtop, s.Htop, (int)N, s.Htop,
                  s.C, nullptr, 0, s.bf16, st));
  return RNNBKT_OK;
}

}  // namespace

extern "C" int32_t rnnbkt_lstm_fwd(const rnnbkt_model_desc* desc, const float* params,
                                   const float* x, const int32_t* labels,
                                   const int32_t* lengths, int32_t T, int32_t B, void* reserve,
                                   size_t reserve_bytes, void* workspace,
                                   size_t workspace_bytes, float* loss, void* stream) {
  return forward(desc, params, x, labels, nullptr, lengths, T, B, reserve, reserve_bytes,
                 workspace, workspace_bytes, loss, stream);
}

extern "C" int32_t rnnbkt_ctc_workspace_bytes(int32_t T_max, int32_t B, int32_t U_max,
                                              size_t* bytes) {
  clear_error();
  RNNBKT_REQUIRE(bytes, RNNBKT_EINVAL, "ctc_workspace_bytes: null pointer");
  RNNBKT_REQUIRE(T_max >= 1 && B >= 1 && U_max >= 1, RNNBKT_EINVAL,
                 "ctc_workspace_bytes: T_max, B and U_max must be >= 1");
  RNNBKT_REQUIRE(ctc_states_per_lane(U_max) > 0, RNNBKT_EUNSUPPORTED,
                 "ctc_workspace_bytes: targets longer than 1023 labels are not supported");
  *bytes = ctc_carve(T_max, B, U_max).total;
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_lstm_fwd_ctc(const rnnbkt_model_desc* desc, const float* params,
                                       const float* x, const int32_t* targets,
                                       const int32_t* target_lengths, int32_t U_max,
                                       const int32_t* lengths, int32_t T, int32_t B,
                                       void* reserve, size_t reserve_bytes, void* workspace,
                                       size_t workspace_bytes, void* ctc_ws, size_t ctc_ws_bytes,
                                       float* loss, void* stream) {
  clear_error();
  RNNBKT_REQUIRE(target_lengths, RNNBKT_EINVAL, "lstm_fwd_ctc: null pointer");
  const CtcInputs ctc{targets, target_lengths, U_max, ctc_ws, ctc_ws_bytes};
  return forward(desc, params, x, nullptr, &ctc, lengths, T, B, reserve, reserve_bytes, workspace,
                 workspace_bytes, loss, stream);
}

namespace {

// The backward of rnnbkt_lstm_bwd.  noalloc: the workspace is the library's
// per-device scratch array (workspace_bytes = its size), only the part the
// launch plan uses must fit, and all work stays on the caller's stream.
int32_t backward(const rnnbkt_model_desc* desc, const float* params, const int32_t* lengths,
                 int32_t T, int32_t B, void* reserve, size_t reserve_bytes, void* workspace,
                 size_t workspace_bytes, float* grads, void* stream, bool noalloc) {
  Shape s;
  int32_t rc = check_desc(desc, &s);
  if (rc != RNNBKT_OK) return rc;
  int64_t N = 0;
  rc = check_lengths(lengths, T, B, &N);
  if (rc != RNNBKT_OK) return rc;
  RNNBKT_REQUIRE(params && reserve && workspace && grads, RNNBKT_EINVAL,
                 "lstm_bwd: null pointer");
  RNNBKT_REQUIRE(aligned16(params) && aligned16(reserve) && aligned16(workspace) &&
                     aligned16(grads),
                 RNNBKT_EINVAL, "lstm_bwd: params, reserve, workspace and grads must be 16-byte aligned");
  const Carve c = carve(s, T, B, N);
  RNNBKT_REQUIRE(reserve_bytes >= c.reserve && (noalloc || workspace_bytes >= c.workspace),
                 RNNBKT_EINVAL,
                 "lstm_bwd: buffers too small (reserve %zu < %zu or workspace %zu < %zu)",
                 reserve_bytes, c.reserve, workspace_bytes, c.workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  RNNBKT_HIP(hipGetLastError());
  const ParamOffsets po = param_offsets(s);
  std::vector<int> bs, off;
  host_tables(lengths, T, B, bs, off);

  const int32_t* d_bs = at<int32_t>(reserve, c.bs);
  const int32_t* d_off = at<int32_t>(reserve, c.off);
  const float* Xp = at<float>(reserve, c.xp);
  const int32_t* pf = at<int32_t>(reserve, c.prev_f);
  const int32_t* pr = at<int32_t>(reserve, c.prev_r);
  const float* dz = at<float>(reserve, c.dz);
  float* dha = at<float>(workspace, c.dha);
  float* dhb = at<float>(workspace, c.dhb);
  float* carry = at<float>(workspace, c.carry);
  float* sk = at<float>(workspace, c.splitk);
  float* cs = at<float>(workspace, c.colsum);
  const int GH = s.G * s.H;
  const int n = (int)N;
  const bool gru = s.cell == RNNBKT_CELL_GRU;

  const float* dhtop = at<float>(reserve, c.dhtop);

  auto da_of = [&](int l, int d) { return at<float>(reserve, c.da[l * s.dirs + d]); };
  auto dah_of = [&](int l, int d) {
    return gru ? at<float>(reserve, c.dah[l * s.dirs + d]) : nullptr;
  };
  // A bf16 LSTM's resident backward publishes its gate gradients as packed
  // bf16 (two per 32-bit word, rounded as every consumer rounds them).
  const bool pk = s.bf16 && !gru;
  const uint64_t rec_b = (pk ? 2ull : 4ull) * (uint64_t)N * GH;
  const uint32_t rec_bytes = rec_b < 0x7FFFFFF0u ? (uint32_t)rec_b : 0x7FFFFFF0u;
  // Unit (layer l, direction d) of a persistent backward launch.  up: the
  // layer above runs in the same launch (unidirectional stacks), and this
  // layer multiplies its gate gradients by W_ih of that layer as they are
  // published.
  auto make_unit = [&](int l, int d, const float* dh, bool up, bool publish_dax) {
    BwdUnit u{};
    const int ld = l * s.dirs + d;
    if (up) {
      u.up = da_of(l + 1, 0);
      u.wih_up = params + po.wih[l + 1];
      u.k_up = GH;
      u.din_up = s.din(l + 1);
      u.up_bytes = rec_bytes;
      u.up_published = 1;
    }
    u.whh = params + po.whh[ld];
    u.dh_in = dh;
    u.ld_dh = s.Htop;
    u.stash = at<float>(reserve, c.stash[ld]);
    u.cst = gru ? nullptr : at<float>(reserve, c.cst[ld]);
    u.hout = at<float>(reserve, c.hout[l]);
    u.da = da_of(l, d);
    u.dah = dah_of(l, d);
    u.bias_part = at<float>(workspace, c.bpart[ld]);
    u.bias_part_h = gru ? at<float>(workspace, c.bpart_h[ld]) : nullptr;
    u.peep = s.peep ? params + po.peep[ld] : nullptr;
    u.peep_part = s.peep ? at<float>(workspace, c.ppart[ld]) : nullptr;
    u.rec_bytes = rec_bytes;
    u.publish_dax = publish_dax ? 1 : 0;
    u.dir = d;
    u.hcol = d * s.H;
    return u;
  };
  auto base_launch = [&]() {
    BwdLaunch Lc{};
    Lc.bs = d_bs;
    Lc.off = d_off;
    Lc.H = s.H;
    Lc.ldh = s.dirs * s.H;
    Lc.T = T;
    return Lc;
  };
  // Launch plan: unidirectional stacks run top-down, as many layers per
  // launch as stay resident (each layer reads the one above as it is
  // published); bidirectional layers run one layer (both directions) per
  // launch.  Between launches the gradient w.r.t. the lower layer's output
  // is a GEMM (dX = dA W_ih of the launch's lowest layer), which the next
  // launch's top layer reads like dH of the output layer: an input segment
  // multiplied inside the recurrence would double the weight fragments a
  // wave holds and spill them for wide layers.
  struct Group {
    int hi, n;
    bool frees_cus;  // its resident grid leaves CUs free for work beside it
  };
  std::vector<Group> groups;
  bool persistent = use_persistent();
  if (persistent) {
    int hi = s.L - 1;
    while (hi >= 0 && persistent) {
      int best = 0;
      bool frees = false;
      const int maxn = s.dirs == 1 ? std::min(kMaxUnits, hi + 1) : 1;
      for (int n = 1; n <= maxn; ++n) {
        BwdLaunch Lc = base_launch();
        for (int q = 0; q < n; ++q)
          for (int d = 0; d < s.dirs; ++d)
            Lc.u[q * s.dirs + d] = make_unit(hi - q, d, q == 0 ? dha : nullptr,
                                             s.dirs == 1 && q > 0, gru && q + 1 < n);
        Lc.nunits = n * s.dirs;
        const int blocks = bwd_persistent_blocks(Lc, s.cell, s.bf16, B);
        if (blocks > 0) {
          best = n;
          frees = blocks < cu_count();
        }
      }
      if (best == 0) persistent = false;
      groups.push_back({hi, best, frees});
      hi -= best;
    }
  }
  if (noalloc) {
    // A resident plan of a unidirectional stack in one launch uses only the
    // first bytes.
    const size_t need =
        (persistent && s.dirs == 1 && groups.size() == 1) ? c.ws_bwd_resident_uni : c.ws_bwd;
    RNNBKT_REQUIRE(need <= workspace_bytes, RNNBKT_EUNSUPPORTED,
                   "lstm_bwd_noalloc: this batch needs %zu bytes of scratch, above the %zu "
                   "the library holds",
                   need, workspace_bytes);
  }
  // Whether the forward left the exchange buffers holding the sentinel.
  const bool prefilled = take_prefilled(reserve);

  // Output layer: dW_out = dZ^T H_top, db_out = colsum dZ (dH_top = dZ W_out
  // was left in the reserve by the forward).
  // dW_out and db_out need nothing the recurrence produces: they run on a
  // side stream beside it (the resident recurrence grids leave most CUs
  // idle), into buffers of their own, and are joined before the layer weight
  // gradients.  With several streams declared (rnnbkt_set_concurrency) the
  // caller's streams already share the GPU and more queues would only
  // contend: the side work then stays on the caller's stream.
  const float* top = at<float>(reserve, c.hout[s.L - 1]);
  Side side;
  const bool one_stream = concurrency() == 1;
  const bool split = one_stream && !noalloc;
  if (split)
    RNNBKT_HIP(side_for(st, &side));
  else
    side.s = st;
  auto fork = [&]() -> hipError_t {
    if (!split) return hipSuccess;
    const hipError_t e = hipEventRecord(side.fork, st);
    return e != hipSuccess ? e : hipStreamWaitEvent(side.s, side.fork, 0);
  };
  auto mark_join = [&]() { return split ? hipEventRecord(side.join, side.s) : hipSuccess; };
  auto wait_join = [&]() { return split ? hipStreamWaitEvent(st, side.join, 0) : hipSuccess; };
  RNNBKT_HIP(fork());
  RNNBKT_HIP(gemm(dz, s.C, false, top, s.Htop, false, grads + po.wout, s.Htop, s.C, s.Htop, n,
                  nullptr, 0, s.bf16, side.s, nullptr, at<float>(workspace, c.splitk_out),
                  nullptr, split && persistent && groups.front().frees_cus));
  {
    Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, side.s);
    RNNBKT_HIP(launch_colsum(dz, N, s.C, s.C, colsum_rows(N), at<float>(workspace, c.colsum_out),
                             grads + po.bout, side.s));
  }
  // Weight gradients computed beside the recurrence by extra workgroups of
  // its launch: fp32 unidirectional LSTM stacks whose layers all run in one
  // resident launch, one stream declared (with several, the other streams'
  // launches already fill the GPU).  RNNBKT_WGRAD=after computes them after.
  const char* wg_env = getenv("RNNBKT_WGRAD");
  bool streamw = persistent && one_stream && !gru && s.dirs == 1 && !s.bf16 && groups.size() == 1 &&
                 !(wg_env && strcmp(wg_env, "after") == 0);
  FoldJob wg_folds[kWgJobs];
  int nwg_folds = 0;
  double wg_flops = 0;

  // Weight gradients dW_ih and dW_hh of layer l (both directions), reduced
  // over every valid frame: dW_ih on s_ih with split-K buffer buf_ih, dW_hh
  // on s_hh with the buffer of its own stream's products.
  float* sk_rec = at<float>(workspace, c.splitk_rec);
  // Layers whose gate gradients the resident backward left packed as bf16.
  std::vector<char> da_pk(s.L, 0);
  // beside: the products run beside the recurrence of the layers below.
  auto layer_wgrad = [&](int l, hipStream_t s_ih, float* buf_ih, hipStream_t s_hh,
                         bool beside) -> hipError_t {
    const float* xin = l == 0 ? Xp : at<float>(reserve, c.hout[l - 1]);
    const int din = s.din(l);
    const float* hout = at<float>(reserve, c.hout[l]);
    for (int d = 0; d < s.dirs; ++d) {
      const int ld = l * s.dirs + d;
      const float* dax = da_of(l, d);
      const float* dahh = gru ? dah_of(l, d) : dax;
      // The second direction swaps the streams (each keeps its split-K
      // buffer), so that two streams carry one dW_ih and one dW_hh each.
      const bool sw = d == 1;
      hipError_t e = gemm(dax, GH, false, xin, din, false, grads + po.wih[ld], din, GH, din, n,
                          nullptr, 0, s.bf16, sw ? s_hh : s_ih, nullptr, sw ? sk_rec : buf_ih,
                          nullptr, beside, da_pk[l] != 0);
      if (e != hipSuccess) return e;
      e = gemm(dahh, GH, false, hout + d * s.H, s.dirs * s.H, false, grads + po.whh[ld], s.H, GH,
               s.H, n, nullptr, 0, s.bf16, sw ? s_ih : s_hh, d == 0 ? pf : pr,
               sw ? buf_ih : sk_rec, nullptr, beside, da_pk[l] != 0);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  };
  // Layers whose weight gradients are already enqueued (on the side stream,
  // beside the recurrence of the layers below).
  std::vector<char> wg_done(s.L, 0);

  if (persistent) {
    // Gradient w.r.t. the output of the top layer of the next group; the
    // dX GEMMs of bidirectional layers alternate between dha and dhb.
    const float* dh_in = dhtop;
    float* dx = dha;
    float* spare = dhb;
    for (const Group& g : groups) {
      BwdLaunch Lc = base_launch();
      for (int q = 0; q < g.n; ++q) {
        const int l = g.hi - q;
        // Only the group's top layer reads a plain gradient from above: dH of
        // the output layer, or the dX GEMM after the launch above.
        const float* dh = q == 0 ? dh_in : nullptr;
        for (int d = 0; d < s.dirs; ++d)
          Lc.u[q * s.dirs + d] = make_unit(l, d, dh, s.dirs == 1 && q > 0, gru && q + 1 < g.n);
      }
      Lc.nunits = g.n * s.dirs;
      double fl = 0;
      for (int q = 0; q < g.n; ++q) {
        const double kup = (s.dirs == 1 && q > 0) ? GH : 0;
        for (int t = 0; t < T; ++t) fl += 2.0 * s.dirs * bs[t] * (kup + GH) * s.H;
      }
      if (!prefilled) {
        // The sentinel in every buffer the launch publishes, in one launch.
        Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
        FillJob fills[2 * kMaxUnits];
        int nf = 0;
        for (int q = 0; q < Lc.nunits; ++q) {
          const BwdUnit& u = Lc.u[q];
          fills[nf++] = {reinterpret_cast<unsigned*>(gru ? u.dah : u.da), pk ? N * GH / 2 : N * GH};
          if (gru && u.publish_dax) fills[nf++] = {reinterpret_cast<unsigned*>(u.da), N * GH};
        }
        for (int q0 = 0; q0 < nf; q0 += kFillJobs)
          RNNBKT_HIP(launch_prepare(nullptr, 0, 0, nullptr, nullptr, 0, nullptr, nullptr, nullptr,
                                    nullptr, nullptr, nullptr, fills + q0,
                                    std::min(kFillJobs, nf - q0), kPublishSentinel, nullptr, st));
      }
      if (streamw) {
        // As many workgroups per output tile as stay resident with the
        // recurrence (at least one, else the products run after it).
        WgStreamArgs& wa = Lc.wg;
        wa = WgStreamArgs{};
        for (int l = 0; l < s.L; ++l) {
          const float* xin = l == 0 ? Xp : at<float>(reserve, c.hout[l - 1]);
          WgJob ji{}, jh{};
          ji.A = jh.A = da_of(l, 0);
          ji.a_bytes = jh.a_bytes = rec_bytes;
          ji.lda = jh.lda = GH;
          ji.M = jh.M = GH;
          ji.B = xin;
          ji.ldb = s.din(l);
          ji.N = s.din(l);
          jh.B = at<float>(reserve, c.hout[l]);
          jh.ldb = s.H;
          jh.gather = pf;
          jh.N = s.H;
          for (WgJob* j : {&ji, &jh}) {
            j->tile_begin = wa.tiles;
            wa.tiles += wg_tiles(j->M, j->N);
            wa.job[wa.njobs++] = *j;
          }
        }
        wa.off = d_off;
        wa.T = T;
        wa.spc = kWgStepsPerChunk;
        wa.nchunks = (T + kWgStepsPerChunk - 1) / kWgStepsPerChunk;
        Lc.wg_on = 1;
        wa.reps = kWgRepsMax;
        while (wa.reps >= 1 && bwd_persistent_blocks(Lc, s.cell, s.bf16, B) == 0) --wa.reps;
        if (wa.reps < 1) {
          Lc.wg_on = 0;
          streamw = false;
        } else {
          float* part = at<float>(workspace, c.wgpart);
          for (int q = 0; q < wa.njobs; ++q) {
            wa.job[q].partial = part;
            part += (size_t)wa.reps * wa.job[q].M * wa.job[q].N;
            const int l = q / 2;
            wg_folds[nwg_folds++] = {wa.job[q].partial, wa.reps, wa.job[q].M, wa.job[q].N,
                                     grads + (q % 2 == 0 ? po.wih[l] : po.whh[l]), wa.job[q].N};
          }
          for (int l = 0; l < s.L; ++l) wg_flops += 2.0 * N * GH * (s.din(l) + s.H);
        }
      }
      bool fits = false;
      {
        Timed tm(RNNBKT_KERNEL_STEP_BWD, fl + wg_flops, 0.0, st);
        RNNBKT_HIP(launch_bwd_persistent(Lc, s.cell, s.bf16, B, st, &fits));
      }
      RNNBKT_REQUIRE(fits, RNNBKT_EHIP, "lstm_bwd: persistent launch no longer fits");
      for (int q = 0; q < g.n; ++q) da_pk[g.hi - q] = pk ? 1 : 0;
      // Gradient w.r.t. the output of the layer below the launch's lowest
      // layer: dX = dA W_ih (bidirectional: dA_fwd W_ih,fwd + dA_bwd W_ih,bwd,
      // one GEMM with two terms).
      const int lo = g.hi - g.n + 1;
      if (lo > 0) {
        // W_ih [G*H x din] of each direction transposed to [din x G*H], so that
        // the GEMM reads both operands with k contiguous (no transposing LDS
        // stores in its tile loop).
        float* wt = at<float>(workspace, c.wt);
        const int din = s.din(lo);
        {
          Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 8.0 * s.dirs * din * GH, st);
          for (int d = 0; d < s.dirs; ++d)
            RNNBKT_HIP(launch_transpose(params + po.wih[lo * s.dirs + d], GH, din, din,
                                        wt + (size_t)d * din * GH, GH, st));
        }
        Term2 t2{};
        if (s.dirs == 2) t2 = Term2{da_of(lo, 1), GH, wt + (size_t)din * GH, GH, GH};
        RNNBKT_HIP(gemm(da_of(lo, 0), GH, true, wt, GH, true, dx, din, n, din, GH, nullptr, 0,
                        s.bf16, st, nullptr, nullptr, s.dirs == 2 ? &t2 : nullptr, false,
                        da_pk[lo] != 0));
        dh_in = dx;
        std::swap(dx, spare);
      }
      // The group's gate gradients are complete: its weight gradients run on
      // the side stream beside the recurrence of the groups below (which
      // leave most CUs idle).  The last group's run after it, split over
      // both streams.
      if (split && !streamw && &g != &groups.back()) {
        RNNBKT_HIP(fork());
        for (int q = 0; q < g.n; ++q) {
          RNNBKT_HIP(layer_wgrad(g.hi - q, side.s, sk_rec, side.s, (&g + 1)->frees_cus));
          wg_done[g.hi - q] = 1;
        }
      }
    }
  } else {
    // One launch per time step: each layer needs the full gradient from above.
    const float* dh_in = dhtop;
    float* dx = dha;
    float* spare = dhb;
    for (int l = s.L - 1; l >= 0; --l) {
      const float* hout = at<float>(reserve, c.hout[l]);
      for (int d = 0; d < s.dirs; ++d) {
        const int ld = l * s.dirs + d;
        StepBwdArgs a{};
        a.da_next = gru ? dah_of(l, d) : da_of(l, d);
        a.whh = params + po.whh[ld];
        a.dh_in = dh_in + d * s.H;
        a.stash = at<float>(reserve, c.stash[ld]);
        a.cst = gru ? nullptr : at<float>(reserve, c.cst[ld]);
        a.hout = hout + d * s.H;
        a.da = da_of(l, d);
        a.dah = dah_of(l, d);
        a.carry = carry;
        a.peep = s.peep ? params + po.peep[ld] : nullptr;
        a.peep_acc = s.peep ? at<float>(workspace, c.peep_acc) : nullptr;
        if (a.peep_acc) {
          Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
          RNNBKT_HIP(launch_fill_u32(reinterpret_cast<unsigned*>(a.peep_acc),
                                     (int64_t)B * 3 * s.H, 0u, st));
        }
        a.H = s.H;
        a.ldd = s.Htop;
        a.ldh = s.dirs * s.H;
        for (int k = 0; k < T; ++k) {
          const int t = d == 0 ? T - 1 - k : k;
          a.row0 = off[t];
          a.rows = bs[t];
          if (d == 0) {
            a.next0 = t + 1 < T ? off[t + 1] : 0;
            a.next_rows = t + 1 < T ? bs[t + 1] : 0;
            a.prev0 = t > 0 ? off[t - 1] : 0;
            a.prev_rows = t > 0 ? bs[t] : 0;
          } else {
            a.next0 = t > 0 ? off[t - 1] : 0;
            a.next_rows = t > 0 ? bs[t] : 0;
            a.prev0 = t + 1 < T ? off[t + 1] : 0;
            a.prev_rows = t + 1 < T ? bs[t + 1] : 0;
          }
          Timed tm(RNNBKT_KERNEL_STEP_BWD, 2.0 * a.next_rows * GH * s.H, 0.0, st);
          RNNBKT_HIP(launch_step_bwd(a, s.cell, s.bf16, st));
        }
        if (a.peep_acc) {
          // Peephole gradients: the per-row running sums, summed over rows.
          Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
          RNNBKT_HIP(launch_colsum(a.peep_acc, B, 3 * s.H, 3 * s.H, colsum_rows(B), cs,
                                   grads + po.peep[ld], st));
        }
      }
      if (l > 0) {
        for (int d = 0; d < s.dirs; ++d) {
          const int ld = l * s.dirs + d;
          RNNBKT_HIP(gemm(da_of(l, d), GH, true, params + po.wih[ld], s.din(l), false, dx,
                          s.din(l), n, s.din(l), GH, nullptr, d > 0 ? 1 : 0, s.bf16, st));
        }
        dh_in = dx;
        std::swap(dx, spare);
      }
    }
  }

  if (persistent) {
    // Bias (GRU: both biases; peephole weights) gradients: the recurrence
    // kernels left one partial per row group; folded in one launch with the
    // partial tiles of the weight gradients computed in the launch, which
    // only needs this stream's kernels (it runs before the join).
    const int rgroups = (B + 15) / 16;
    std::vector<FoldJob> folds(wg_folds, wg_folds + nwg_folds);
    for (int ld = 0; ld < s.L * s.dirs; ++ld) {
      folds.push_back({at<float>(workspace, c.bpart[ld]), rgroups, 1, GH, grads + po.b[ld], GH});
      if (gru)
        folds.push_back(
            {at<float>(workspace, c.bpart_h[ld]), rgroups, 1, GH, grads + po.bhh[ld], GH});
      if (s.peep)
        folds.push_back(
            {at<float>(workspace, c.ppart[ld]), rgroups, 1, 3 * s.H, grads + po.peep[ld], 3 * s.H});
    }
    Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
    for (size_t q0 = 0; q0 < folds.size(); q0 += kFoldJobs)
      RNNBKT_HIP(launch_splitk_reduce_multi(folds.data() + q0,
                                            (int32_t)std::min<size_t>(kFoldJobs, folds.size() - q0),
                                            st));
  }
  // Weight gradients of the layers not enqueued yet (unless the recurrence
  // launch computed them).  The input and recurrent products of a layer read
  // the same dA and are independent: the recurrent ones run on the side
  // stream (own split-K buffer), overlapping the other stream's products.
  if (!streamw) RNNBKT_HIP(fork());
  for (int l = 0; l < s.L; ++l) {
    if (!streamw && !wg_done[l]) RNNBKT_HIP(layer_wgrad(l, st, sk, side.s, false));
    for (int d = 0; d < s.dirs; ++d) {
      const int ld = l * s.dirs + d;
      const float* dax = da_of(l, d);
      const float* dahh = gru ? dah_of(l, d) : dax;
      if (!persistent) {
        Timed tm(RNNBKT_KERNEL_OTHER, 0.0, 0.0, st);
        RNNBKT_HIP(launch_colsum(dax, N, GH, GH, colsum_rows(N), cs, grads + po.b[ld], st));
        if (gru)
          RNNBKT_HIP(launch_colsum(dahh, N, GH, GH, colsum_rows(N), cs, grads + po.bhh[ld], st));
      }
    }
  }
  // Everything on the side stream (output-layer gradients, weight
  // gradients) is ordered before the caller's later work.
  RNNBKT_HIP(mark_join());
  RNNBKT_HIP(wait_join());
  return RNNBKT_OK;
}

// Scratch of rnnbkt_lstm_bwd_noalloc: one array per device, held from the
// library's first use on that device until the process ends.  Host code must
// not use the array's name as an address: it stands for the array on the
// host side only.  Its device address comes from hipGetSymbolAddress, once
// per device, and is kept in g_scratch_ptr.
constexpr size_t kScratchBytes = size_t(128) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int32_t scratch_of_current_device(void** out) {
  int dev = 0;
  RNNBKT_HIP(hipGetDevice(&dev));
  RNNBKT_REQUIRE(dev >= 0 && dev < kMaxDevices, RNNBKT_EUNSUPPORTED,
                 "lstm_bwd_noalloc: device index %d above %d", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    RNNBKT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    RNNBKT_REQUIRE(p != nullptr, RNNBKT_EHIP, "lstm_bwd_noalloc: no address for the scratch array");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return RNNBKT_OK;
}

}  // namespace

extern "C" int32_t rnnbkt_lstm_bwd(const rnnbkt_model_desc* desc, const float* params,
                                   const int32_t* lengths, int32_t T, int32_t B,
                                   void* reserve, size_t reserve_bytes, void* workspace,
                                   size_t workspace_bytes, float* grads, void* stream) {
  clear_error();
  return backward(desc, params, lengths, T, B, reserve, reserve_bytes, workspace,
                  workspace_bytes, grads, stream, false);
}

extern "C" int32_t rnnbkt_lstm_bwd_noalloc(const rnnbkt_model_desc* desc, const float* params,
                                           const int32_t* lengths, int32_t T, int32_t B,
                                           void* reserve, size_t reserve_bytes, float* grads,
                                           void* stream) {
  clear_error();
  void* ws = nullptr;
  const int32_t rc = scratch_of_current_device(&ws);
  if (rc != RNNBKT_OK) return rc;
  return backward(desc, params, lengths, T, B, reserve, reserve_bytes, ws, kScratchBytes, grads,
                  stream, true);
}

extern "C" int32_t rnnbkt_sgd_apply(float* params, const float* grads, int64_t n, float lr,
                                    void* stream) {
  clear_error();
  RNNBKT_REQUIRE(params && grads, RNNBKT_EINVAL, "sgd_apply: null pointer");
  RNNBKT_REQUIRE(n >= 0, RNNBKT_EINVAL, "sgd_apply: n < 0");
  RNNBKT_REQUIRE(aligned16(params) && aligned16(grads), RNNBKT_EINVAL,
                 "sgd_apply: params and grads must be 16-byte aligned");
  if (n == 0) return RNNBKT_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Timed tm(RNNBKT_KERNEL_SGD, 0.0, 12.0 * n, st);
  RNNBKT_HIP(launch_sgd(params, grads, n, lr, st));
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_adadelta_apply(float* params, const float* grads, float* acc_g2,
                                         float* acc_dx2, int64_t n, float rho, float eps,
                                         float lr, void* stream) {
  clear_error();
  RNNBKT_REQUIRE(params && grads && acc_g2 && acc_dx2, RNNBKT_EINVAL,
                 "adadelta_apply: null pointer");
  RNNBKT_REQUIRE(n >= 0, RNNBKT_EINVAL, "adadelta_apply: n < 0");
  RNNBKT_REQUIRE(aligned16(params) && aligned16(grads) && aligned16(acc_g2) && aligned16(acc_dx2),
                 RNNBKT_EINVAL, "adadelta_apply: all four arrays must be 16-byte aligned");
  RNNBKT_REQUIRE(rho >= 0.f && rho < 1.f, RNNBKT_EINVAL, "adadelta_apply: rho must be in [0, 1)");
  RNNBKT_REQUIRE(eps > 0.f, RNNBKT_EINVAL, "adadelta_apply: eps must be > 0");
  RNNBKT_REQUIRE(lr > 0.f, RNNBKT_EINVAL, "adadelta_apply: lr must be > 0");
  if (n == 0) return RNNBKT_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Timed tm(RNNBKT_KERNEL_SGD, 0.0, 28.0 * n, st);
  RNNBKT_HIP(launch_adadelta(params, grads, acc_g2, acc_dx2, n, rho, eps, lr, st));
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_epoch_aggregate(float* replicas, int32_t R, int64_t stride, int64_t n,
                                          float* prev, float beta, void* stream) {
  clear_error();
  RNNBKT_REQUIRE(replicas && prev, RNNBKT_EINVAL, "epoch_aggregate: null pointer");
  RNNBKT_REQUIRE(R >= 1 && R <= 1024, RNNBKT_EINVAL, "epoch_aggregate: R = %d outside [1, 1024]",
                 R);
  RNNBKT_REQUIRE(n >= 0 && stride >= n && stride % 4 == 0, RNNBKT_EINVAL,
                 "epoch_aggregate: need n >= 0 and stride >= n, a multiple of 4");
  RNNBKT_REQUIRE(aligned16(replicas) && aligned16(prev), RNNBKT_EINVAL,
                 "epoch_aggregate: replicas and prev must be 16-byte aligned");
  RNNBKT_REQUIRE(std::isfinite(beta), RNNBKT_EINVAL, "epoch_aggregate: beta must be finite");
  if (n == 0) return RNNBKT_OK;
  // prev must not overlap any replica's n values.
  const uintptr_t p0 = reinterpret_cast<uintptr_t>(prev), p1 = p0 + sizeof(float) * n;
  for (int32_t r = 0; r < R; ++r) {
    const uintptr_t r0 = reinterpret_cast<uintptr_t>(replicas + (int64_t)r * stride);
    const uintptr_t r1 = r0 + sizeof(float) * n;
    RNNBKT_REQUIRE(p1 <= r0 || r1 <= p0, RNNBKT_EINVAL,
                   "epoch_aggregate: prev overlaps replica %d", r);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  Timed tm(RNNBKT_KERNEL_SGD, 0.0, 8.0 * (R + 1) * n, st);
  RNNBKT_HIP(launch_aggregate(replicas, R, stride, n, prev, beta, st));
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_set_concurrency(int32_t streams) {
  clear_error();
  RNNBKT_REQUIRE(streams >= 1 && streams <= 64, RNNBKT_EINVAL,
                 "set_concurrency: streams = %d outside [1, 64]", streams);
  set_concurrency(streams);
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_kernel_timer(int32_t enable) {
  clear_error();
  std::lock_guard<std::mutex> lk(g_tmu);
  if (enable) {
    for (auto& r : g_recs) {
      g_pool.push_back(r.a);
      g_pool.push_back(r.b);
    }
    g_recs.clear();
  }
  g_timer_on = enable != 0;
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_kernel_timer_read(int32_t kind, double* total_ms, int64_t* launches,
                                            double* alg_flops, double* alg_bytes) {
  clear_error();
  RNNBKT_REQUIRE(kind >= 0 && kind < RNNBKT_KERNEL_KINDS, RNNBKT_EINVAL,
                 "kernel_timer_read: kind %d out of range", kind);
  RNNBKT_REQUIRE(total_ms && launches && alg_flops && alg_bytes, RNNBKT_EINVAL,
                 "kernel_timer_read: null pointer");
  std::lock_guard<std::mutex> lk(g_tmu);
  double ms = 0.0, fl = 0.0, by = 0.0;
  int64_t cnt = 0;
  for (auto& r : g_recs) {
    if (r.kind != kind) continue;
    RNNBKT_HIP(hipEventSynchronize(r.b));
    float e = 0.f;
    RNNBKT_HIP(hipEventElapsedTime(&e, r.a, r.b));
    ms += e;
    fl += r.flops;
    by += r.bytes;
    ++cnt;
  }
  *total_ms = ms;
  *launches = cnt;
  *alg_flops = fl;
  *alg_bytes = by;
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_top_hidden(const rnnbkt_model_desc* desc, const int32_t* lengths,
                                     int32_t T, int32_t B, const void* reserve,
                                     size_t reserve_bytes, float* out, void* stream) {
  clear_error();
  Shape s;
  int32_t rc = check_desc(desc, &s);
  if (rc != RNNBKT_OK) return rc;
  int64_t N = 0;
  rc = check_lengths(lengths, T, B, &N);
  if (rc != RNNBKT_OK) return rc;
  RNNBKT_REQUIRE(reserve && out, RNNBKT_EINVAL, "top_hidden: null pointer");
  const Carve c = carve(s, T, B, N);
  RNNBKT_REQUIRE(reserve_bytes >= c.reserve, RNNBKT_EINVAL, "top_hidden: reserve too small");
  RNNBKT_HIP(launch_unpack(at<float>(reserve, c.hout[s.L - 1]), s.Htop,
                           at<int32_t>(reserve, c.bs), at<int32_t>(reserve, c.off), T, B, out,
                           static_cast<hipStream_t>(stream)));
  return RNNBKT_OK;
}
