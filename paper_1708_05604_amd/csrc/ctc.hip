// Connectionist temporal classification (CTC) loss and its gradient with
// respect to the output logits: the training cost of the paper's experiments
// (Sec. IV.A).  Class 0 is the blank; a target is a label string l_1..l_U
// over classes 1..C-1, extended to l' = (blank, l_1, blank, ..., l_U, blank)
// of S = 2U + 1 states.
//
// Three kernels per batch:
//   k_ctc_emit  one wave per valid frame (all frames in parallel): the
//               frame's log-sum-exp and, for every state s of its sequence,
//               the log emission probability ln y_t(l'_s);
//   k_ctc_seq   one wave per sequence, the only sequential part: the forward
//               variables over t in log space, shifted every step so that
//               their maximum is 0 (the shifts summed in double precision give
//               the loss), then the backward variables over t in reverse, the
//               same way, forming the state occupancies alpha beta / y
//               (normalised by their maximum, then their sum) and their
//               per-class sums over the target's classes (one lane per class,
//               in state order: deterministic);
//   k_ctc_grad  one wave per valid frame: y_t(k) minus the class sums,
//               scaled by the batch normalisation, written over the logits.
// Log space keeps every path's weight representable: in linear space with
// per-step scaling the forward and backward variables of a long sequence
// underflow exactly where the posterior lives (the unconstrained forward
// progress runs ahead of it).  Emissions and forward variables are read a
// few steps ahead, so the sequential kernel's steps wait only on their own
// arithmetic.
#include <hip/hip_runtime.h>

#include <cmath>

#include "kernels.h"

namespace rnnbkt {

namespace {

__device__ inline float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Cross-lane steps of the sequential kernel as DPP moves (no LDS round trip).
// dpp<CTRL, ROWS>(fill, v): v from the lane CTRL names; lanes in rows not in
// ROWS, or with no source lane, get fill.
template <int CTRL, int ROWS = 0xf>
__device__ inline float dpp(float fill, float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(fill), __float_as_int(v), CTRL,
                                                    ROWS, 0xf, false));
}
constexpr int kQuadSwap1 = 0xB1;     // quad_perm (1, 0, 3, 2)
constexpr int kQuadSwap2 = 0x4E;     // quad_perm (2, 3, 0, 1)
constexpr int kRowHalfMirror = 0x141;
constexpr int kRowMirror = 0x140;
constexpr int kRowBcast15 = 0x142;
constexpr int kRowBcast31 = 0x143;
constexpr int kWaveShl1 = 0x130;     // lane i <- lane i+1
constexpr int kWaveShr1 = 0x138;     // lane i <- lane i-1

// Sum / maximum over the wave, returned in every lane (the total forms in
// lane 63 and is read back as a scalar).
__device__ inline float dpp_wave_sum(float v) {
  v += dpp<kQuadSwap1>(0.f, v);
  v += dpp<kQuadSwap2>(0.f, v);
  v += dpp<kRowHalfMirror>(0.f, v);
  v += dpp<kRowMirror>(0.f, v);
  v += dpp<kRowBcast15, 0xa>(0.f, v);
  v += dpp<kRowBcast31, 0xc>(0.f, v);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ inline float dpp_wave_max(float v) {
  v = fmaxf(v, dpp<kQuadSwap1>(-INFINITY, v));
  v = fmaxf(v, dpp<kQuadSwap2>(-INFINITY, v));
  v = fmaxf(v, dpp<kRowHalfMirror>(-INFINITY, v));
  v = fmaxf(v, dpp<kRowMirror>(-INFINITY, v));
  v = fmaxf(v, dpp<kRowBcast15, 0xa>(-INFINITY, v));
  v = fmaxf(v, dpp<kRowBcast31, 0xc>(-INFINITY, v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Target classes are read from device memory the host cannot check: a value
// outside 1..C-1 is clamped into that range (wrong numbers, never an access
// outside the logits).
__device__ inline int label_at(const CtcArgs& a, const int32_t* tg, int u) {
  return min(max(tg[u], 1), a.C - 1);
}

// Frame (t, b) of the packed batch, or -1 past the sequence's end.
__device__ inline int64_t frame_of(const CtcArgs& a, int t, int b) {
  return b < a.bs[t] ? (int64_t)a.off[t] + b : -1;
}

constexpr int kEmitWaves = 4;

__global__ __launch_bounds__(64 * kEmitWaves) void k_ctc_emit(CtcArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t id = (int64_t)blockIdx.x * kEmitWaves + (threadIdx.x >> 6);
  if (id >= (int64_t)a.T * a.B) return;
  const int t = (int)(id / a.B), b = (int)(id % a.B);
  const int64_t f = frame_of(a, t, b);
  if (f < 0) return;
  const float* row = a.z + f * a.C;
  float m = -INFINITY;
  for (int k = lane; k < a.C; k += 64) m = fmaxf(m, row[k]);
  m = wave_max(m);
  float sum = 0.f;
  for (int k = lane; k < a.C; k += 64) sum += __expf(row[k] - m);
  const float lse = m + __logf(wave_sum(sum));
  if (lane == 0) a.lse[f] = lse;
  const int U = a.tab[b];
  const int S = 2 * U + 1;
  const int32_t* tg = a.targets + (int64_t)b * a.U_max;
  float* e = a.e + ((int64_t)b * a.T + t) * a.S_stride;
  for (int s = lane; s < a.S_stride; s += 64) {
    float v = -INFINITY;
    if (s < S) v = row[(s & 1) ? label_at(a, tg, s >> 1) : 0] - lse;
    e[s] = v;
  }
}

// Reads the lane's NS consecutive floats of a [T][S_stride] array at row t.
template <int NS>
__device__ inline void load_row(const float* base, int64_t stride, int t, int s0, float (&v)[NS]) {
  const float* p = base + (int64_t)t * stride + s0;
  if constexpr (NS % 4 == 0) {
#pragma unroll
    for (int i = 0; i < NS; i += 4) {
      const float4 x = *reinterpret_cast<const float4*>(p + i);
      v[i] = x.x;
      v[i + 1] = x.y;
      v[i + 2] = x.z;
      v[i + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < NS; ++i) v[i] = p[i];
  }
}

template <int NS>
__device__ inline void store_row(float* base, int64_t stride, int t, int s0, const float (&v)[NS]) {
  float* p = base + (int64_t)t * stride + s0;
  if constexpr (NS % 4 == 0) {
#pragma unroll
    for (int i = 0; i < NS; i += 4)
      *reinterpret_cast<float4*>(p + i) = make_float4(v[i], v[i + 1], v[i + 2], v[i + 3]);
  } else {
#pragma unroll
    for (int i = 0; i < NS; ++i) p[i] = v[i];
  }
}

// Steps between a row's load and its use: deep enough to cover a load from
// HBM at a fraction of a microsecond per step, within the register budget
// (two queues of D rows of NS floats in the backward pass).
template <int NS>
constexpr int ahead() {
  return NS <= 4 ? 16 : 64 / NS;
}

// ln(e^x + e^y + e^z) with -inf terms allowed (all -inf gives -inf).
__device__ inline float log_add3(float x, float y, float z) {
  const float m = fmaxf(fmaxf(x, y), z);
  if (m == -INFINITY) return -INFINITY;
  return m + __logf(__expf(x - m) + __expf(y - m) + __expf(z - m));
}


// Label chains of a target, one entry per label position u: nxt[u] = the
// next position with the same class (-1: none), head[u] = 1 at the first
// position of each class.  Written by the forward block of each sequence.
__device__ inline void build_chains(const CtcArgs& a, int b, const int32_t* tg, int U) {
  int32_t* nxt = a.chain + (int64_t)b * 2 * a.U_max;
  int32_t* head = nxt + a.U_max;
  for (int u = threadIdx.x; u < U; u += 64) {
    const int k = label_at(a, tg, u);
    int h = 1;
    for (int v = 0; v < u; ++v)
      if (label_at(a, tg, v) == k) {
        h = 0;
        break;
      }
    int n = -1;
    for (int v = u + 1; v < U; ++v)
      if (label_at(a, tg, v) == k) {
        n = v;
        break;
      }
    nxt[u] = n;
    head[u] = h;
  }
}

// The two recursions of one sequence, one wave each: block b < B runs the
// forward variables of sequence b over t = 0..L-1, block B + b the backward
// variables over t = L-1..0.  Both are kept in log space and shifted every
// step so that their maximum is 0; each stores its rows for the gradient
// kernel.  Lane owns states s0 = lane*NS .. s0+NS-1.
template <int NS>
__global__ __launch_bounds__(64) void k_ctc_seq(CtcArgs a) {
  const bool backward = (int)blockIdx.x >= a.B;
  const int b = backward ? blockIdx.x - a.B : blockIdx.x;
  const int lane = threadIdx.x;
  const int U = a.tab[b], L = a.tab[a.B + b];
  const int S = 2 * U + 1;
  const int s0 = lane * NS;
  const int32_t* tg = a.targets + (int64_t)b * a.U_max;
  const int64_t stride = a.S_stride;
  const float* eb = a.e + (int64_t)b * a.T * stride;
  float* out = (backward ? a.beta : a.alpha) + (int64_t)b * a.T * stride;
  if (!backward) build_chains(a, b, tg, U);

  // skip[i]: the transition between s and s-2 (forward) / s+2 (backward)
  // exists: the farther state is a label different from the nearer one.
  // (labels are read only at positions inside the target)
  bool skip[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const int s = s0 + i;
    const int far = backward ? s + 2 : s - 2;
    const bool lbl = s < S && (s & 1);
    skip[i] = lbl && far >= 1 && far < S && label_at(a, tg, far >> 1) != label_at(a, tg, s >> 1);
  }

  constexpr int D = ahead<NS>();
  float q[D][NS];
  // row of step k (t = k forward, L-1-k backward), clamped inside the sequence
  auto fetch = [&](int k, float (&v)[NS]) {
    const int kk = k < L ? k : L - 1;
    load_row<NS>(eb, stride, backward ? L - 1 - kk : kk, s0, v);
  };
#pragma unroll
  for (int j = 0; j < D; ++j) fetch(j, q[j]);
  float cur[NS];
  double logc = 0.0;
  bool dead = false;
  auto step = [&](int k, const float (&ev)[NS]) {
    float nx[NS];
    if (k == 0) {
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        const int s = s0 + i;
        const bool start = backward ? (s == S - 1 || s == S - 2) : s < 2;
        nx[i] = start ? ev[i] : -INFINITY;
      }
    } else if (!backward) {
      // states s0-1 and s0-2 live in the lanes below (-inf below lane 0)
      const float m1 = dpp<kWaveShr1>(-INFINITY, cur[NS - 1]);
      const float m2 = NS >= 2 ? dpp<kWaveShr1>(-INFINITY, cur[NS >= 2 ? NS - 2 : 0])
                               : dpp<kWaveShr1>(-INFINITY, m1);
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        const float n1 = i >= 1 ? cur[i - 1] : m1;
        const float n2 = i >= 2 ? cur[i - 2] : (i == 1 ? m1 : m2);
        nx[i] = log_add3(cur[i], n1, skip[i] ? n2 : -INFINITY) + ev[i];
      }
    } else {
      // states s0+NS and s0+NS+1 live in the lanes above (-inf past lane 63)
      const float p1 = dpp<kWaveShl1>(-INFINITY, cur[0]);
      const float p2 = NS >= 2 ? dpp<kWaveShl1>(-INFINITY, cur[NS >= 2 ? 1 : 0])
                               : dpp<kWaveShl1>(-INFINITY, p1);
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        const float n1 = i + 1 < NS ? cur[i + 1] : p1;
        const float n2 = i + 2 < NS ? cur[i + 2] : (i + 1 == NS ? p2 : p1);
        nx[i] = log_add3(cur[i], n1, skip[i] ? n2 : -INFINITY) + ev[i];
      }
    }
    float part = -INFINITY;
#pragma unroll
    for (int i = 0; i < NS; ++i) part = fmaxf(part, nx[i]);
    const float mx = dpp_wave_max(part);
    if (mx == -INFINITY) dead = true;
    const float sh = mx == -INFINITY ? 0.f : mx;
    logc += (double)sh;
#pragma unroll
    for (int i = 0; i < NS; ++i) cur[i] = nx[i] - sh;
    store_row<NS>(out, stride, backward ? L - 1 - k : k, s0, cur);
  };
  for (int k0 = 0; k0 < L; k0 += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      if (k0 + j < L) {
        step(k0 + j, q[j]);
        fetch(k0 + j + D, q[j]);
      }
    }
  }
  if (backward) return;
  // ln p = sum of the shifts + ln(alpha(S-1) + alpha(S-2)) at the last frame
  float endp = 0.f;
#pragma unroll
  for (int i = 0; i < NS; ++i)
    if (s0 + i == S - 1 || s0 + i == S - 2) endp += __expf(cur[i]);
  endp = dpp_wave_sum(endp);
  dead = dead || !(endp > 0.f);
  if (lane == 0) a.loss_part[b] = dead ? INFINITY : (float)(-(logc + (double)__logf(endp)));
}

// Gradient rows, one wave per valid frame: the state occupancies
// alpha beta / y of the frame (from the two stored recursions, normalised
// by their maximum, then their sum), their per-class sums (blank: all even
// states; a label class: its positions along the chain, in order), and
// y_t(k) minus those sums, times the loss scale, over the logits.
constexpr int kMaxStates = 2048;
__global__ __launch_bounds__(64 * kEmitWaves) void k_ctc_grad(CtcArgs a) {
  __shared__ float row_s[kEmitWaves][1024];
  __shared__ float occ_s[kEmitWaves][kMaxStates / 2];  // odd states: label positions
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t id = (int64_t)blockIdx.x * kEmitWaves + w;
  if (id >= (int64_t)a.T * a.B) return;
  const int t = (int)(id / a.B), b = (int)(id % a.B);
  const int64_t f = frame_of(a, t, b);
  if (f < 0) return;
  float* row = a.z + f * a.C;
  float* rs = row_s[w];
  float* oc = occ_s[w];
  const int U = a.tab[b];
  const int S = 2 * U + 1;
  const bool dead = !(a.loss_part[b] < INFINITY);
  const int64_t ro = ((int64_t)b * a.T + t) * a.S_stride;
  const float* al = a.alpha + ro;
  const float* be = a.beta + ro;
  const float* ee = a.e + ro;
  // ln(alpha beta / y) per state; its maximum; occupancies; their sum
  float mx = -INFINITY;
  for (int s = lane; s < S; s += 64) {
    const float x = al[s], y = be[s];
    const float lg = (x == -INFINITY || y == -INFINITY) ? -INFINITY : x + y - ee[s];
    mx = fmaxf(mx, lg);
  }
  mx = wave_max(mx);
  float z = 0.f, blank = 0.f;
  for (int s = lane; s < S; s += 64) {
    const float x = al[s], y = be[s];
    const float o = (x == -INFINITY || y == -INFINITY || mx == -INFINITY)
                        ? 0.f : __expf(x + y - ee[s] - mx);
    z += o;
    if (s & 1)
      oc[s >> 1] = o;
    else
      blank += o;
  }
  z = wave_sum(z);
  blank = wave_sum(blank);
  const float zinv = (z > 0.f && !dead) ? 1.f / z : 0.f;
  const float lse = a.lse[f];
  for (int k = lane; k < a.C; k += 64) rs[k] = __expf(row[k] - lse);
  __builtin_amdgcn_wave_barrier();
  if (lane == 0) rs[0] -= blank * zinv;
  // one lane per class (the first position of each class), in position order
  const int32_t* tg = a.targets + (int64_t)b * a.U_max;
  const int32_t* nxt = a.chain + (int64_t)b * 2 * a.U_max;
  const int32_t* head = nxt + a.U_max;
  for (int u = lane; u < U; u += 64) {
    if (!head[u]) continue;
    float v = 0.f;
    for (int q = u; q >= 0; q = nxt[q]) v += oc[q];
    rs[label_at(a, tg, u)] -= v * zinv;
  }
  __builtin_amdgcn_wave_barrier();
  for (int k = lane; k < a.C; k += 64) row[k] = dead ? 0.f : rs[k] * a.scale;
}

}  // namespace

int ctc_states_per_lane(int U_max) {
  const int S = 2 * U_max + 1;
  int ns = 1;
  while (64 * ns < S) ns *= 2;
  return ns <= 32 ? ns : 0;
}

hipError_t launch_ctc(const CtcArgs& a, hipStream_t st) {
  const int64_t waves = (int64_t)a.T * a.B;
  const unsigned blocks = (unsigned)((waves + kEmitWaves - 1) / kEmitWaves);
  hipLaunchKernelGGL(k_ctc_emit, dim3(blocks), dim3(64 * kEmitWaves), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  switch (a.S_stride / 64) {
    case 1: hipLaunchKernelGGL(k_ctc_seq<1>, dim3(2 * a.B), dim3(64), 0, st, a); break;
    case 2: hipLaunchKernelGGL(k_ctc_seq<2>, dim3(2 * a.B), dim3(64), 0, st, a); break;
    case 4: hipLaunchKernelGGL(k_ctc_seq<4>, dim3(2 * a.B), dim3(64), 0, st, a); break;
    case 8: hipLaunchKernelGGL(k_ctc_seq<8>, dim3(2 * a.B), dim3(64), 0, st, a); break;
    case 16: hipLaunchKernelGGL(k_ctc_seq<16>, dim3(2 * a.B), dim3(64), 0, st, a); break;
    case 32: hipLaunchKernelGGL(k_ctc_seq<32>, dim3(2 * a.B), dim3(64), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_ctc_grad, dim3(blocks), dim3(64 * kEmitWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace rnnbkt
