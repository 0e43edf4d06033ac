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

constexpr int kAhead = 4;  // steps between a row's load and its use

// ln(e^x + e^y + e^z) with -inf terms allowed (all -inf gives -inf).
__device__ inline float log_add3(float x, float y, float z) {
  const float m = fmaxf(fmaxf(x, y), z);
  if (m == -INFINITY) return -INFINITY;
  return m + __logf(__expf(x - m) + __expf(y - m) + __expf(z - m));
}


// One wave per sequence; lane owns states s0 = lane*NS .. s0+NS-1.
template <int NS>
__global__ __launch_bounds__(64) void k_ctc_seq(CtcArgs a) {
  constexpr int SP = 64 * NS;
  __shared__ int lab[SP];     // l'_s (0 past S)
  __shared__ int nx[SP];      // next state with the same label (-1: none)
  __shared__ float occ[SP];   // normalised occupancies of the current frame
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int U = a.tab[b], L = a.tab[a.B + b];
  const int S = 2 * U + 1;
  const int s0 = lane * NS;
  const int32_t* tg = a.targets + (int64_t)b * a.U_max;
  const int64_t stride = a.S_stride;
  float* eb = a.e + (int64_t)b * a.T * stride;
  float* ab = a.alpha + (int64_t)b * a.T * stride;

  int ext[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const int s = s0 + i;
    ext[i] = (s < S && (s & 1)) ? label_at(a, tg, s >> 1) : 0;
    lab[s] = ext[i];
  }
  __syncthreads();
  // into[i]: the transition s-2 -> s exists; from[i]: s -> s+2 exists;
  // head[i]: s is the first state carrying its label (its lane sums the
  // class's occupancies along the nx chain, in state order).
  bool into[NS], from[NS], head[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    const int s = s0 + i;
    const bool lbl = s < S && (s & 1);
    into[i] = lbl && s >= 3 && ext[i] != lab[s - 2];
    from[i] = s + 2 < S && ((s + 2) & 1) && lab[s + 2] != ext[i];
    head[i] = lbl;
    int next = -1;
    if (lbl) {
      for (int q = s - 2; q >= 1; q -= 2)
        if (lab[q] == ext[i]) {
          head[i] = false;
          break;
        }
      for (int q = s + 2; q < S; q += 2)
        if (lab[q] == ext[i]) {
          next = q;
          break;
        }
    }
    nx[s] = next;
  }

  // ---- forward variables
  float al[NS];
  double logc = 0.0;
  bool dead = false;
  float q0[NS], q1[NS], q2[NS], q3[NS];
  auto fetch_e = [&](int t, float (&q)[NS]) { load_row<NS>(eb, stride, t < L ? t : L - 1, s0, q); };
  fetch_e(0, q0);
  fetch_e(1, q1);
  fetch_e(2, q2);
  fetch_e(3, q3);
  auto fwd_step = [&](int t, const float (&ev)[NS]) {
    float an[NS];
    if (t == 0) {
#pragma unroll
      for (int i = 0; i < NS; ++i) an[i] = (s0 + i) < 2 ? ev[i] : -INFINITY;
    } else {
      // states s0-1 and s0-2 live in the lanes below
      float m1 = __shfl_up(al[NS - 1], 1, 64);
      float m2 = NS >= 2 ? __shfl_up(al[NS >= 2 ? NS - 2 : 0], 1, 64) : __shfl_up(al[0], 2, 64);
      if (lane < 1) m1 = -INFINITY;
      if (lane < (NS >= 2 ? 1 : 2)) m2 = -INFINITY;
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        const float a1 = i >= 1 ? al[i - 1] : m1;
        const float a2 = i >= 2 ? al[i - 2] : (i == 1 ? m1 : m2);
        an[i] = log_add3(al[i], a1, into[i] ? a2 : -INFINITY) + ev[i];
      }
    }
    float part = -INFINITY;
#pragma unroll
    for (int i = 0; i < NS; ++i) part = fmaxf(part, an[i]);
    const float mx = wave_max(part);
    if (mx == -INFINITY) dead = true;
    const float sh = mx == -INFINITY ? 0.f : mx;
    logc += (double)sh;
#pragma unroll
    for (int i = 0; i < NS; ++i) al[i] = an[i] - sh;
    store_row<NS>(ab, stride, t, s0, al);
  };
  for (int t = 0; t < L; t += kAhead) {
    fwd_step(t, q0);
    fetch_e(t + 4, q0);
    if (t + 1 < L) {
      fwd_step(t + 1, q1);
      fetch_e(t + 5, q1);
    }
    if (t + 2 < L) {
      fwd_step(t + 2, q2);
      fetch_e(t + 6, q2);
    }
    if (t + 3 < L) {
      fwd_step(t + 3, q3);
      fetch_e(t + 7, q3);
    }
  }
  // ln p = sum of the shifts + ln(alpha(S-1) + alpha(S-2)) at the last frame
  float endp = 0.f;
#pragma unroll
  for (int i = 0; i < NS; ++i)
    if (s0 + i == S - 1 || s0 + i == S - 2) endp += __expf(al[i]);
  endp = wave_sum(endp);
  dead = dead || !(endp > 0.f);
  if (lane == 0) a.loss_part[b] = dead ? INFINITY : (float)(-(logc + (double)__logf(endp)));

  // ---- backward variables and occupancies
  float be[NS];
  float r0[NS], r1[NS], r2[NS], r3[NS];  // alpha rows, read ahead like the e rows
  auto fetch_a = [&](int t, float (&q)[NS]) { load_row<NS>(ab, stride, t >= 0 ? t : 0, s0, q); };
  auto fetch_eb = [&](int t, float (&q)[NS]) { load_row<NS>(eb, stride, t >= 0 ? t : 0, s0, q); };
  // The backward pass reads back the forward pass's alpha rows: wait for
  // every store of this wave first.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  fetch_eb(L - 1, q0);
  fetch_eb(L - 2, q1);
  fetch_eb(L - 3, q2);
  fetch_eb(L - 4, q3);
  fetch_a(L - 1, r0);
  fetch_a(L - 2, r1);
  fetch_a(L - 3, r2);
  fetch_a(L - 4, r3);
  float* csum = eb;  // occupancy sums overwrite e row t once it has been used
  auto bwd_step = [&](int t, const float (&ev)[NS], const float (&av)[NS]) {
    float bn[NS];
    if (t == L - 1) {
#pragma unroll
      for (int i = 0; i < NS; ++i)
        bn[i] = (s0 + i == S - 1 || s0 + i == S - 2) ? ev[i] : -INFINITY;
    } else {
      float p1 = __shfl_down(be[0], 1, 64);
      float p2 = NS >= 2 ? __shfl_down(be[NS >= 2 ? 1 : 0], 1, 64) : __shfl_down(be[0], 2, 64);
      if (lane >= 63) p1 = -INFINITY;
      if (lane >= (NS >= 2 ? 63 : 62)) p2 = -INFINITY;
#pragma unroll
      for (int i = 0; i < NS; ++i) {
        const float b1 = i + 1 < NS ? be[i + 1] : p1;
        const float b2 = i + 2 < NS ? be[i + 2] : (i + 1 == NS ? p2 : p1);
        bn[i] = log_add3(be[i], b1, from[i] ? b2 : -INFINITY) + ev[i];
      }
    }
    float part = -INFINITY;
#pragma unroll
    for (int i = 0; i < NS; ++i) part = fmaxf(part, bn[i]);
    const float mb = wave_max(part);
    const float shb = mb == -INFINITY ? 0.f : mb;
    // ln of alpha beta / y per state, then occupancies relative to their
    // maximum (which is therefore 1: the normaliser cannot underflow)
    float lg[NS];
    float lpart = -INFINITY;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      be[i] = bn[i] - shb;
      lg[i] = (av[i] == -INFINITY || be[i] == -INFINITY) ? -INFINITY : av[i] + be[i] - ev[i];
      lpart = fmaxf(lpart, lg[i]);
    }
    const float mg = wave_max(lpart);
    float g[NS];
    float gpart = 0.f;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      g[i] = mg == -INFINITY ? 0.f : __expf(lg[i] - mg);
      gpart += g[i];
    }
    const float z = wave_sum(gpart);
    const float zinv = (z > 0.f && !dead) ? 1.f / z : 0.f;
    float blank = 0.f;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      g[i] *= zinv;
      occ[s0 + i] = g[i];
      if (!((s0 + i) & 1)) blank += g[i];
    }
    blank = wave_sum(blank);
    __syncthreads();
    // Entry 1+u of the row: the class sum at the first position u of each
    // label, -1 at later positions of a repeated label; entry 0: blank.
    float* cs = csum + (int64_t)t * stride;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const int s = s0 + i;
      if (!(s < S && (s & 1))) continue;
      float v = -1.f;
      if (head[i]) {
        v = g[i];
        for (int q = nx[s]; q >= 0; q = nx[q]) v += occ[q];
      }
      cs[1 + (s >> 1)] = v;
    }
    if (lane == 0) cs[0] = blank;
    __syncthreads();
  };
  for (int t = L - 1; t >= 0; t -= kAhead) {
    bwd_step(t, q0, r0);
    fetch_eb(t - 4, q0);
    fetch_a(t - 4, r0);
    if (t - 1 >= 0) {
      bwd_step(t - 1, q1, r1);
      fetch_eb(t - 5, q1);
      fetch_a(t - 5, r1);
    }
    if (t - 2 >= 0) {
      bwd_step(t - 2, q2, r2);
      fetch_eb(t - 6, q2);
      fetch_a(t - 6, r2);
    }
    if (t - 3 >= 0) {
      bwd_step(t - 3, q3, r3);
      fetch_eb(t - 7, q3);
      fetch_a(t - 7, r3);
    }
  }
}

// Gradient rows: y_t(k) - (class k's occupancy), times the loss scale.
__global__ __launch_bounds__(64 * kEmitWaves) void k_ctc_grad(CtcArgs a) {
  __shared__ float row_s[kEmitWaves][1024];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t id = (int64_t)blockIdx.x * kEmitWaves + w;
  const bool live = id < (int64_t)a.T * a.B;
  const int t = live ? (int)(id / a.B) : 0, b = live ? (int)(id % a.B) : 0;
  const int64_t f = live ? frame_of(a, t, b) : -1;
  float* row = f >= 0 ? a.z + f * a.C : nullptr;
  float* rs = row_s[w];
  if (f >= 0) {
    const float lse = a.lse[f];
    for (int k = lane; k < a.C; k += 64) rs[k] = __expf(row[k] - lse);
  }
  __syncthreads();
  if (f >= 0) {
    const int U = a.tab[b];
    const int32_t* tg = a.targets + (int64_t)b * a.U_max;
    const float* cs = a.e + ((int64_t)b * a.T + t) * a.S_stride;
    // Class sums sit at the first position of each label (distinct classes,
    // so lanes never meet on a class); later positions hold -1.
    if (lane == 0) rs[0] -= cs[0];
    for (int u = lane; u < U; u += 64) {
      const float v = cs[1 + u];
      if (v >= 0.f) rs[label_at(a, tg, u)] -= v;
    }
  }
  __syncthreads();
  if (f >= 0) {
    const bool dead = !(a.loss_part[b] < INFINITY);
    for (int k = lane; k < a.C; k += 64) row[k] = dead ? 0.f : rs[k] * a.scale;
  }
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
    case 1: hipLaunchKernelGGL(k_ctc_seq<1>, dim3(a.B), dim3(64), 0, st, a); break;
    case 2: hipLaunchKernelGGL(k_ctc_seq<2>, dim3(a.B), dim3(64), 0, st, a); break;
    case 4: hipLaunchKernelGGL(k_ctc_seq<4>, dim3(a.B), dim3(64), 0, st, a); break;
    case 8: hipLaunchKernelGGL(k_ctc_seq<8>, dim3(a.B), dim3(64), 0, st, a); break;
    case 16: hipLaunchKernelGGL(k_ctc_seq<16>, dim3(a.B), dim3(64), 0, st, a); break;
    case 32: hipLaunchKernelGGL(k_ctc_seq<32>, dim3(a.B), dim3(64), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_ctc_grad, dim3(blocks), dim3(64 * kEmitWaves), 0, st, a);
  return hipGetLastError();
}

}  // namespace rnnbkt
