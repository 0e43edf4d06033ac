// Whole-sequence recurrence of one LSTM/GRU layer (both directions) in one
// launch, forward and backward through time.
//
// A launch keeps every workgroup resident (cooperative launch) and walks
// the T steps of the batch itself.  Each workgroup owns a fixed block of 16
// batch rows and a fixed slice of hidden units, so
//   - its slice of W_hh stays in registers for the whole launch (each lane
//     holds the MFMA operand fragments it feeds; read from HBM once),
//   - the recurrent state of its (row, unit) pairs (c for the LSTM, h for
//     the GRU update, the dc / dh carries backward) stays in registers,
//   - per-step operands that do not depend on other workgroups (the input
//     projection row, the saved gate activations) are fetched early.
//
// Exchange between workgroups without a grid barrier: the buffer a step
// publishes (h forward, the recurrent gate gradient backward) is filled
// with a sentinel bit pattern before the launch; every element of it is
// written exactly once during the launch with a relaxed device-scope atomic
// store (a value equal to the sentinel is replaced by the canonical NaN), and
// a reader polls its elements with relaxed device-scope atomic loads until
// none holds the sentinel.  Single-location coherence of atomics is all this
// needs: no fence, no cache write-back or invalidation, and a workgroup
// waits only for the rows it reads (sequences are independent).  Polls are
// bounded; after a timeout the wait gives up, counts it (reported by
// rnnbkt_sync_check) and later waits return at once, so a launch always ends.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "kernels.h"

namespace rnnbkt {

__device__ unsigned g_wait_timeouts = 0;

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

__device__ inline float sigm(float x) { return 1.f / (1.f + __expf(-x)); }


constexpr unsigned kSentinel = 0xFFFFFFFFu;
constexpr unsigned kCanonicalNan = 0x7FC00000u;

__device__ inline void publish(float* p, float v) {
  unsigned u = __float_as_uint(v);
  if (u == kSentinel) u = kCanonicalNan;
  __hip_atomic_store(reinterpret_cast<unsigned*>(p), u, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}


typedef unsigned u4 __attribute__((ext_vector_type(4)));

// Buffer resource over a published array of `bytes` bytes.  Loads through it
// use the device-scope cache policy (sc1), the policy of a relaxed
// device-scope atomic load; every 32-bit element of a 128-bit load is read
// atomically, which is all the sentinel protocol needs.  Offsets at or past
// `bytes` read as zero.
__device__ inline __amdgpu_buffer_rsrc_t published_rsrc(const float* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, (int)bytes, 0x00020000);
}
constexpr unsigned kNoRow = 0x7FFFFFF0u;  // an offset past every published array
constexpr int kDeviceScope = 16;           // sc1
constexpr int kMaxSteps = 6144;  // batch tables kept in LDS: T_max above this is not handled here
constexpr int kBwdUnits = 16;    // hidden units per backward workgroup

// Reduction-dimension chunking of one MFMA group: fp32 16x16x4 takes 4
// k per lane group (4 groups), bf16 16x16x32 takes 8.
template <bool BF16>
struct Chunk;
template <>
struct Chunk<false> {
  static constexpr int CH = 16;
  static constexpr int CPL = 4;
};
template <>
struct Chunk<true> {
  static constexpr int CH = 32;
  static constexpr int CPL = 8;
};

// A lane's weight fragments for its chunks, kept in registers for the whole
// launch: element (k, column) of the 16-column weight block for
// k = c*CH + koff + e.  fp32: 4 floats per chunk; bf16: 8 values per chunk.
template <bool BF16>
struct WFrag;
template <>
struct WFrag<false> {
  using T = f4;
};
template <>
struct WFrag<true> {
  using T = bf8;
};

// acc += A(16 x K) . W(K x 16) over the chunks held in u (see fetch_published)
// with the lane's weight fragments w (one per chunk slot).
template <bool BF16, int MAXC>
__device__ inline f4 mma_chunks(const unsigned (&u)[Chunk<BF16>::CPL * MAXC],
                                const typename WFrag<BF16>::T (&w)[MAXC], int first, int stride,
                                int nchunks) {
  constexpr int CPL = Chunk<BF16>::CPL;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = first + i * stride;
    if (c >= nchunks) break;
    if constexpr (BF16) {
      bf8 av;
#pragma unroll
      for (int e = 0; e < CPL; ++e) av[e] = (__bf16)__uint_as_float(u[i * CPL + e]);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, w[i], acc, 0, 0, 0);
    } else {
#pragma unroll
      for (int e = 0; e < CPL; ++e)
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(u[i * CPL + e]), w[i][e], acc,
                                                   0, 0, 0);
    }
  }
  return acc;
}

// Loads the lane's weight fragments: wk(k) returns the weight for reduction
// index k of this lane's column (0 for padding columns).
template <bool BF16, int MAXC, typename F>
__device__ inline void load_wfrags(typename WFrag<BF16>::T (&w)[MAXC], int first, int stride,
                                   int nchunks, int koff, F wk) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int CPL = Chunk<BF16>::CPL;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = first + i * stride;
#pragma unroll
    for (int e = 0; e < CPL; ++e) {
      const float v = c < nchunks ? wk(c * CH + koff + e) : 0.f;
      if constexpr (BF16)
        w[i][e] = (__bf16)v;
      else
        w[i][e] = v;
    }
  }
}

// Step indices of launch-relative step k for direction d.
struct StepIdx {
  int t, rows, row0, prev0, prev_rows;
};

__device__ inline StepIdx fwd_step(const int32_t* bs, const int32_t* off, int T, int d, int k) {
  StepIdx s;
  s.t = d == 0 ? k : T - 1 - k;
  s.rows = bs[s.t];
  s.row0 = off[s.t];
  if (d == 0) {
    s.prev0 = s.t > 0 ? off[s.t - 1] : 0;
    s.prev_rows = s.t > 0 ? s.rows : 0;
  } else {
    s.prev0 = s.t + 1 < T ? off[s.t + 1] : 0;
    s.prev_rows = s.t + 1 < T ? bs[s.t + 1] : 0;
  }
  return s;
}

// Reads the lane's operand slots of one step: slot i (chunk c = first +
// i*stride) holds NV 128-bit pieces at byte offsets offs[i][v] in the input
// array (from_in[i]) or in the output array; slots with chk[i] are published
// values and are re-read until none holds the sentinel.  from_in / chk are
// uniform across the wave.
template <int NV, int MAXC>
__device__ inline void fetch_slots(__amdgpu_buffer_rsrc_t rin, __amdgpu_buffer_rsrc_t rout,
                                   const unsigned (&offs)[MAXC][NV], const bool (&from_in)[MAXC],
                                   const bool (&chk)[MAXC], unsigned (&u)[MAXC * NV * 4]) {
  unsigned spins = 0;
  for (;;) {
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const u4 x = from_in[i]
                         ? __builtin_amdgcn_raw_buffer_load_b128(rin, offs[i][v], 0, kDeviceScope)
                         : __builtin_amdgcn_raw_buffer_load_b128(rout, offs[i][v], 0, kDeviceScope);
#pragma unroll
        for (int e = 0; e < 4; ++e) u[(i * NV + v) * 4 + e] = x[e];
      }
    bool ready = true;
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
      if (chk[i])
#pragma unroll
        for (int e = 0; e < NV * 4; ++e) ready &= u[i * NV * 4 + e] != kSentinel;
    if (__all(ready)) return;
    if (spins == 0 && __hip_atomic_load(&g_wait_timeouts, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT) != 0u)
      return;
    if (++spins == (1u << 20)) {
      if ((threadIdx.x & 63) == 0)
        __hip_atomic_fetch_add(&g_wait_timeouts, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Copies unit `ui` out of the kernel arguments without dynamic indexing.
__device__ inline FwdUnit pick_unit(const FwdLaunch& a, int ui) {
  FwdUnit u = a.u[0];
  if (ui == 1) u = a.u[1];
  if (ui == 2) u = a.u[2];
  if (ui == 3) u = a.u[3];
  return u;
}

// Forward recurrence of the launch's units.  Workgroup = 16 rows x 4*NT
// hidden units of one unit; column block nt holds, for its 4 units, the
// LSTM gates (i, f, g, o) or the GRU groups (r, z, n from the input, n from
// the state), so one MFMA tile per block yields every pre-activation a
// unit's update needs.  NW waves split the reduction dimension; waves
// 0..NT-1 then run the state update of one column block each.
template <int G, bool BF16, int NW, int MAXC, int NT>
__global__ __launch_bounds__(64 * NW) void k_fwd_persistent(FwdLaunch a) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int CPL = Chunk<BF16>::CPL;
  constexpr int NV = CPL / 4;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* red = reinterpret_cast<float*>(smem);                     // [NW][NT][256]
  int32_t* tbs = reinterpret_cast<int32_t*>(red + NW * NT * 256);  // batch sizes [T]
  int32_t* toff = tbs + a.T;                                       // offsets [T+1]
  for (int i = threadIdx.x; i <= a.T; i += blockDim.x) {
    if (i < a.T) tbs[i] = a.bs[i];
    toff[i] = a.off[i];
  }
  int ui = 0;
  for (int q = 1; q < a.nunits; ++q)
    if ((int)blockIdx.x >= a.u[q].wg_begin) ui = q;
  const FwdUnit U = pick_unit(a, ui);
  const int rem = blockIdx.x - U.wg_begin;
  const int slice = rem % a.slices;
  const int rg = rem / a.slices;
  const int H = a.H;
  const int j0 = slice * 4 * NT;
  const int r0 = rg * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  const int kin_pad = (U.kin + CH - 1) / CH * CH;
  const int nin = kin_pad / CH;
  const int nch = nin + H / CH;

  // Weight fragments: this lane feeds column lr of every column block.
  typename WFrag<BF16>::T w[NT][MAXC];
  {
    const int grp = lr >> 2, uu = lr & 3;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = j0 + 4 * nt + uu;
      // gate row of W_ih / W_hh feeding this column for the input part and
      // the state part (-1 = none)
      int gi, gh;
      if (G == 4) {
        gi = grp;
        gh = grp;
      } else {
        gi = grp == 3 ? -1 : grp;
        gh = grp == 2 ? -1 : (grp == 3 ? 2 : grp);
      }
      const float* wi = gi >= 0 ? U.wih + (int64_t)(gi * H + j) * U.kin : nullptr;
      const float* wh = gh >= 0 ? U.whh + (int64_t)(gh * H + j) * H : nullptr;
      load_wfrags<BF16, MAXC>(w[nt], wave, NW, nch, lq * CPL, [&](int k) {
        if (k < kin_pad) return (wi && k < U.kin) ? wi[k] : 0.f;
        return wh ? wh[k - kin_pad] : 0.f;
      });
    }
  }
  // State-update lanes: wave nt < NT owns row r0 + (lane >> 2), unit
  // j0 + 4*nt + (lane & 3) for the whole launch.
  const bool epi = wave < NT;
  const int erow = r0 + (lane >> 2);
  const int ej = j0 + 4 * (epi ? wave : 0) + (lane & 3);
  float bi[4] = {0.f, 0.f, 0.f, 0.f}, bh[3] = {0.f, 0.f, 0.f};
  if (epi) {
#pragma unroll
    for (int g = 0; g < G; ++g) bi[g] = U.b[g * H + ej];
    if constexpr (G == 3) {
#pragma unroll
      for (int g = 0; g < 3; ++g) bh[g] = U.bhh[g * H + ej];
    }
  }
  float c_state = 0.f, h_state = 0.f;
  const __amdgpu_buffer_rsrc_t rin = published_rsrc(U.in, U.in_bytes);
  const __amdgpu_buffer_rsrc_t rout = published_rsrc(U.hout, U.out_bytes);
  __syncthreads();

  StepIdx s = fwd_step(tbs, toff, a.T, U.dir, 0);
  for (int k = 0; k < a.T; ++k) {
    StepIdx nx = s;
    if (k + 1 < a.T) nx = fwd_step(tbs, toff, a.T, U.dir, k + 1);
    const bool active = r0 < s.rows;
    if (active) {
      const int r = r0 + lr;
      unsigned offs[MAXC][NV];
      bool from_in[MAXC], chk[MAXC];
#pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        const int c = wave + i * NW;
        from_in[i] = c < nin;
        chk[i] = c < nin ? U.in_published != 0 : c < nch;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int kk = c * CH + lq * CPL + 4 * v;
          unsigned o = kNoRow;
          if (c < nin) {
            if (r < s.rows && kk < U.kin)
              o = 4u * (unsigned)((int64_t)(s.row0 + r) * U.ld_in + kk);
          } else if (c < nch) {
            if (r < s.prev_rows)
              o = 4u * (unsigned)((int64_t)(s.prev0 + r) * a.ldh + U.hcol + (kk - kin_pad));
          }
          offs[i][v] = o;
        }
      }
      unsigned uu[MAXC * NV * 4];
      fetch_slots<NV, MAXC>(rin, rout, offs, from_in, chk, uu);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const f4 acc = mma_chunks<BF16, MAXC>(uu, w[nt], wave, NW, nch);
#pragma unroll
        for (int q = 0; q < 4; ++q) red[(wave * NT + nt) * 256 + (lq * 4 + q) * 16 + lr] = acc[q];
      }
    }
    __syncthreads();
    if (epi && active && erow < s.rows) {
      const int rr = lane >> 2, u4_ = lane & 3;
      float sg[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float v = 0.f;
#pragma unroll
        for (int w_ = 0; w_ < NW; ++w_) v += red[(w_ * NT + wave) * 256 + rr * 16 + g * 4 + u4_];
        sg[g] = v;
      }
      const bool has_prev = erow < s.prev_rows;
      const int64_t f = s.row0 + erow;
      float* st = U.stash + f * 4 * H;
      if constexpr (G == 4) {
        const float ig = sigm(sg[0] + bi[0]);
        const float fg = sigm(sg[1] + bi[1]);
        const float gg = tanhf(sg[2] + bi[2]);
        const float og = sigm(sg[3] + bi[3]);
        const float cp = has_prev ? c_state : 0.f;
        c_state = fg * cp + ig * gg;
        h_state = og * tanhf(c_state);
        st[ej] = ig;
        st[H + ej] = fg;
        st[2 * H + ej] = gg;
        st[3 * H + ej] = og;
        U.cst[f * H + ej] = c_state;
      } else {
        const float rg_ = sigm(sg[0] + bi[0] + bh[0]);
        const float z = sigm(sg[1] + bi[1] + bh[1]);
        const float ahn = sg[3] + bh[2];
        const float n = tanhf(sg[2] + bi[2] + rg_ * ahn);
        const float hp = has_prev ? h_state : 0.f;
        h_state = (1.f - z) * n + z * hp;
        st[ej] = rg_;
        st[H + ej] = z;
        st[2 * H + ej] = n;
        st[3 * H + ej] = ahn;
      }
      publish(U.hout + f * a.ldh + U.hcol + ej, h_state);
    }
    s = nx;
    __syncthreads();  // red is rewritten by the next step
  }
}

// Backward.  "next" = the following step of the forward recurrence.
struct BwdIdx {
  int t, rows, row0, next0, next_rows, prev0, prev_rows;
};

__device__ inline BwdIdx bwd_step(const int32_t* bs, const int32_t* off, int T, int d, int k) {
  BwdIdx s;
  s.t = d == 0 ? T - 1 - k : k;
  s.rows = bs[s.t];
  s.row0 = off[s.t];
  if (d == 0) {
    s.next0 = s.t + 1 < T ? off[s.t + 1] : 0;
    s.next_rows = s.t + 1 < T ? bs[s.t + 1] : 0;
    s.prev0 = s.t > 0 ? off[s.t - 1] : 0;
    s.prev_rows = s.t > 0 ? s.rows : 0;
  } else {
    s.next0 = s.t > 0 ? off[s.t - 1] : 0;
    s.next_rows = s.t > 0 ? s.rows : 0;
    s.prev0 = s.t + 1 < T ? off[s.t + 1] : 0;
    s.prev_rows = s.t + 1 < T ? bs[s.t + 1] : 0;
  }
  return s;
}

__device__ inline BwdUnit pick_unit(const BwdLaunch& a, int ui) {
  BwdUnit u = a.u[0];
  if (ui == 1) u = a.u[1];
  if (ui == 2) u = a.u[2];
  if (ui == 3) u = a.u[3];
  return u;
}

__device__ inline void store_or_publish(float* p, float v, bool pub) {
  if (pub)
    publish(p, v);
  else
    *p = v;
}

// Backpropagation through time of the launch's units.  Workgroup = 16 rows
// x 16 hidden units of one unit; NW waves split the reduction dimension;
// threads 0..255 then run the gate-gradient algebra of one (row, unit) each,
// carrying dc*f (LSTM) or dh*z (GRU) of their row and unit in a register.
template <int G, bool BF16, int NW, int MAXC>
__global__ __launch_bounds__(64 * NW) void k_bwd_persistent(BwdLaunch a) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int CPL = Chunk<BF16>::CPL;
  constexpr int NV = CPL / 4;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* red = reinterpret_cast<float*>(smem);
  int32_t* tbs = reinterpret_cast<int32_t*>(red + NW * 256);  // batch sizes [T]
  int32_t* toff = tbs + a.T;                                  // offsets [T+1]
  for (int i = threadIdx.x; i <= a.T; i += blockDim.x) {
    if (i < a.T) tbs[i] = a.bs[i];
    toff[i] = a.off[i];
  }
  int ui = 0;
  for (int q = 1; q < a.nunits; ++q)
    if ((int)blockIdx.x >= a.u[q].wg_begin) ui = q;
  const BwdUnit U = pick_unit(a, ui);
  const int rem = blockIdx.x - U.wg_begin;
  const int slice = rem % a.slices;
  const int rg = rem / a.slices;
  const int H = a.H;
  const int GH = G * H;
  const int j0 = slice * kBwdUnits;
  const int r0 = rg * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  const bool has_up = U.up != nullptr;
  const int kup = has_up ? U.k_up : 0;
  const int nup = kup / CH;
  const int nch = nup + GH / CH;

  // Weight fragments: column lr is hidden unit j0 + lr.
  typename WFrag<BF16>::T w[MAXC];
  {
    const int j = j0 + lr;
    const float* wu = has_up ? U.wih_up + U.hcol + j : nullptr;
    const float* wh = U.whh + j;
    load_wfrags<BF16, MAXC>(w, wave, NW, nch, lq * CPL, [&](int k) {
      return k < kup ? wu[(int64_t)k * U.din_up] : wh[(int64_t)(k - kup) * H];
    });
  }
  // Gate-gradient threads: 0..255 -> row r0 + (tid >> 4), unit j0 + (tid & 15).
  const bool epi = threadIdx.x < 256;
  const int erow = r0 + ((threadIdx.x & 255) >> 4);
  const int ej = j0 + (threadIdx.x & 15);
  float carry = 0.f;
  const float* rec = G == 3 ? U.dah : U.da;
  const __amdgpu_buffer_rsrc_t rup = published_rsrc(has_up ? U.up : U.da, U.up_bytes);
  const __amdgpu_buffer_rsrc_t rrec = published_rsrc(rec, U.rec_bytes);
  const bool pub_dax = G == 4 || U.publish_dax != 0;
  __syncthreads();

  BwdIdx s = bwd_step(tbs, toff, a.T, U.dir, 0);
  for (int k = 0; k < a.T; ++k) {
    BwdIdx nx = s;
    if (k + 1 < a.T) nx = bwd_step(tbs, toff, a.T, U.dir, k + 1);
    const bool active = r0 < s.rows;
    // Operands that do not depend on other workgroups, loaded without
    // branches inside the gate-gradient threads (inactive rows read frame
    // 0 and are ignored).
    float dhv = 0.f, st0, st1, st2, st3, cc, cprev;
    const int64_t f = erow < s.rows ? s.row0 + erow : 0;
    const bool has_prev = erow < s.prev_rows;
    if (epi) {
      const int64_t fp = has_prev ? s.prev0 + erow : 0;
      if (U.dh_in) dhv = U.dh_in[f * U.ld_dh + U.hcol + ej];
      const float* st = U.stash + f * 4 * H;
      st0 = st[ej];
      st1 = st[H + ej];
      st2 = st[2 * H + ej];
      st3 = st[3 * H + ej];
      if constexpr (G == 4) {
        cc = U.cst[f * H + ej];
        cprev = U.cst[fp * H + ej];
      } else {
        cc = 0.f;
        cprev = U.hout[fp * a.ldh + U.hcol + ej];
      }
    }
    if (active) {
      const int r = r0 + lr;
      unsigned offs[MAXC][NV];
      bool from_up[MAXC], chk[MAXC];
#pragma unroll
      for (int i = 0; i < MAXC; ++i) {
        const int c = wave + i * NW;
        from_up[i] = c < nup;
        chk[i] = c < nup ? U.up_published != 0 : c < nch;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int kk = c * CH + lq * CPL + 4 * v;
          unsigned o = kNoRow;
          if (c < nup) {
            if (r < s.rows) o = 4u * (unsigned)((int64_t)(s.row0 + r) * kup + kk);
          } else if (c < nch) {
            if (r < s.next_rows) o = 4u * (unsigned)((int64_t)(s.next0 + r) * GH + (kk - kup));
          }
          offs[i][v] = o;
        }
      }
      unsigned uu[MAXC * NV * 4];
      fetch_slots<NV, MAXC>(rup, rrec, offs, from_up, chk, uu);
      const f4 acc = mma_chunks<BF16, MAXC>(uu, w, wave, NW, nch);
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave * 256 + (lq * 4 + q) * 16 + lr] = acc[q];
    }
    __syncthreads();
    if (epi && active && erow < s.rows) {
      const bool has_next = erow < s.next_rows;
      float dh_red = 0.f;
#pragma unroll
      for (int w_ = 0; w_ < NW; ++w_) dh_red += red[w_ * 256 + threadIdx.x];
      if constexpr (G == 4) {
        const float dh = dhv + dh_red;
        const float tc = tanhf(cc);
        const float dc = dh * st3 * (1.f - tc * tc) + (has_next ? carry : 0.f);
        const float cp = has_prev ? cprev : 0.f;
        float* dar = U.da + f * GH;
        publish(dar + ej, dc * st2 * st0 * (1.f - st0));
        publish(dar + H + ej, dc * cp * st1 * (1.f - st1));
        publish(dar + 2 * H + ej, dc * st0 * (1.f - st2 * st2));
        publish(dar + 3 * H + ej, dh * tc * st3 * (1.f - st3));
        carry = dc * st1;
      } else {
        const float dh = dhv + dh_red + (has_next ? carry : 0.f);
        const float r = st0, z = st1, n = st2, ahn = st3;
        const float hp = has_prev ? cprev : 0.f;
        const float dn = dh * (1.f - z);
        const float dz = dh * (hp - n);
        const float dan = dn * (1.f - n * n);
        const float dar_ = dan * ahn * r * (1.f - r);
        const float daz = dz * z * (1.f - z);
        float* dx = U.da + f * GH;
        float* dhh = U.dah + f * GH;
        store_or_publish(dx + ej, dar_, pub_dax);
        store_or_publish(dx + H + ej, daz, pub_dax);
        store_or_publish(dx + 2 * H + ej, dan, pub_dax);
        publish(dhh + ej, dar_);
        publish(dhh + H + ej, daz);
        publish(dhh + 2 * H + ej, dan * r);
        carry = dh * z;
      }
    }
    s = nx;
    __syncthreads();  // red is rewritten by the next step
  }
}

// Dynamic LDS above 64 KiB has to be allowed per kernel once.
hipError_t allow_lds(const void* kernel, size_t shmem) {
  static std::mutex mu;
  static std::vector<std::pair<const void*, size_t>> done;
  std::lock_guard<std::mutex> lk(mu);
  for (auto& p : done)
    if (p.first == kernel && p.second >= shmem) return hipSuccess;
  hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)shmem);
  if (e == hipSuccess) done.emplace_back(kernel, shmem);
  return e;
}

// Co-resident workgroups a launch of `kernel` can have (0 on error).
int max_coresident(const void* kernel, int threads, size_t shmem) {
  int dev = 0, cus = 0, per_cu = 0;
  if (allow_lds(kernel, shmem) != hipSuccess) return 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, shmem) != hipSuccess)
    return 0;
  return cus * per_cu;
}

// Launches a grid that must be resident all at once.  By default the
// runtime's cooperative launch guarantees it; RNNBKT_LAUNCH=plain uses an
// ordinary launch instead (for tools that cannot follow cooperative
// launches), relying on the occupancy check alone -- if another stream
// occupied the GPU, waits would time out and rnnbkt_sync_check reports it.
hipError_t coop_launch(const void* kernel, int blocks, int threads, size_t shmem, void* args,
                       hipStream_t st, bool* fits) {
  if (blocks > max_coresident(kernel, threads, shmem)) {
    *fits = false;
    return hipSuccess;
  }
  *fits = true;
  void* argv[] = {args};
  const char* mode = getenv("RNNBKT_LAUNCH");
  if (mode && strcmp(mode, "plain") == 0)
    return hipLaunchKernel(kernel, dim3(blocks), dim3(threads), argv, shmem, st);
  return hipLaunchCooperativeKernel(kernel, dim3(blocks), dim3(threads), argv, shmem, st);
}

}  // namespace

namespace {

// Chunks per wave (a power of two) for a reduction of nch chunks over 4
// waves; 0 if above the per-lane budget.
int fwd_maxc(int nch, bool bf16) {
  const int per = (nch + 3) / 4;
  int m = 1;
  while (m < per) m *= 2;
  return m <= (bf16 ? 8 : 16) ? m : 0;
}

template <int G, bool BF16, int NT>
const void* fwd_kernel_nt(int maxc) {
  switch (maxc) {
    case 1: return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, 1, NT>);
    case 2: return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, 2, NT>);
    case 4: return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, 4, NT>);
    case 8: return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, 8, NT>);
  }
  if constexpr (!BF16)
    if (maxc == 16) return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, 16, NT>);
  return nullptr;
}

const void* fwd_kernel(int cell, bool bf16, int nt, int maxc) {
  if (cell == RNNBKT_CELL_LSTM) {
    if (bf16) return nt == 1 ? fwd_kernel_nt<4, true, 1>(maxc) : fwd_kernel_nt<4, true, 2>(maxc);
    return nt == 1 ? fwd_kernel_nt<4, false, 1>(maxc) : fwd_kernel_nt<4, false, 2>(maxc);
  }
  if (bf16) return nt == 1 ? fwd_kernel_nt<3, true, 1>(maxc) : fwd_kernel_nt<3, true, 2>(maxc);
  return nt == 1 ? fwd_kernel_nt<3, false, 1>(maxc) : fwd_kernel_nt<3, false, 2>(maxc);
}

struct FwdPlan {
  const void* kernel;
  int nt, maxc, blocks;
  size_t shmem;
};

// Column blocks per workgroup: 2 (8 units) for wide layers, else 1 (4 units).
FwdPlan plan_fwd(const FwdLaunch& a, int cell, bool bf16, int B) {
  FwdPlan p{nullptr, 0, 0, 0, 0};
  const int ch = bf16 ? 32 : 16;
  if (a.T > kMaxSteps || a.nunits < 1 || a.nunits > kMaxUnits || a.H % ch != 0) return p;
  int nch = 0;
  for (int q = 0; q < a.nunits; ++q) {
    const FwdUnit& u = a.u[q];
    if (u.kin < 1 || u.kin % 4 != 0 || u.in_bytes >= kNoRow || u.out_bytes >= kNoRow) return p;
    nch = std::max(nch, (u.kin + ch - 1) / ch + a.H / ch);
  }
  p.nt = a.H >= 256 && a.H % 8 == 0 ? 2 : 1;
  p.maxc = fwd_maxc(nch, bf16);
  if (p.maxc == 0) return p;
  p.blocks = a.nunits * (a.H / (4 * p.nt)) * ((B + 15) / 16);
  p.shmem = sizeof(float) * 4 * p.nt * 256 + sizeof(int32_t) * (2 * a.T + 1);
  p.kernel = fwd_kernel(cell, bf16, p.nt, p.maxc);
  return p;
}

}  // namespace

int fwd_persistent_blocks(const FwdLaunch& a, int cell, bool bf16, int B) {
  const FwdPlan p = plan_fwd(a, cell, bf16, B);
  if (!p.kernel) return 0;
  if (p.blocks > max_coresident(p.kernel, 256, p.shmem)) return 0;
  return p.blocks;
}

hipError_t launch_fwd_persistent(FwdLaunch a, int cell, bool bf16, int B, hipStream_t st,
                                 bool* fits) {
  *fits = false;
  const FwdPlan p = plan_fwd(a, cell, bf16, B);
  if (!p.kernel) return hipSuccess;
  a.slices = a.H / (4 * p.nt);
  a.rgroups = (B + 15) / 16;
  const int per_unit = a.slices * a.rgroups;
  for (int q = 0; q < a.nunits; ++q) a.u[q].wg_begin = q * per_unit;
  return coop_launch(p.kernel, p.blocks, 256, p.shmem, &a, st, fits);
}

namespace {

template <int G, bool BF16, int NW>
const void* bwd_kernel_nw(int maxc) {
  switch (maxc) {
    case 1: return reinterpret_cast<const void*>(k_bwd_persistent<G, BF16, NW, 1>);
    case 2: return reinterpret_cast<const void*>(k_bwd_persistent<G, BF16, NW, 2>);
    case 4: return reinterpret_cast<const void*>(k_bwd_persistent<G, BF16, NW, 4>);
    case 8: return reinterpret_cast<const void*>(k_bwd_persistent<G, BF16, NW, 8>);
  }
  if constexpr (!BF16)
    if (maxc == 16) return reinterpret_cast<const void*>(k_bwd_persistent<G, BF16, NW, 16>);
  return nullptr;
}

const void* bwd_kernel(int cell, bool bf16, int nw, int maxc) {
  if (cell == RNNBKT_CELL_LSTM) {
    if (bf16) return nw == 4 ? bwd_kernel_nw<4, true, 4>(maxc) : bwd_kernel_nw<4, true, 16>(maxc);
    return nw == 4 ? bwd_kernel_nw<4, false, 4>(maxc) : bwd_kernel_nw<4, false, 16>(maxc);
  }
  if (bf16) return nw == 4 ? bwd_kernel_nw<3, true, 4>(maxc) : bwd_kernel_nw<3, true, 16>(maxc);
  return nw == 4 ? bwd_kernel_nw<3, false, 4>(maxc) : bwd_kernel_nw<3, false, 16>(maxc);
}

struct BwdPlan {
  const void* kernel;
  int nw, maxc, blocks;
  size_t shmem;
};

// Waves: 4, or 16 when a wave's share of the reduction would exceed the
// per-lane budget (16 chunks fp32, 8 chunks bf16).
BwdPlan plan_bwd(const BwdLaunch& a, int cell, bool bf16, int B) {
  BwdPlan p{nullptr, 0, 0, 0, 0};
  const int ch = bf16 ? 32 : 16;
  const int G = cell == RNNBKT_CELL_LSTM ? 4 : 3;
  if (a.T > kMaxSteps || a.nunits < 1 || a.nunits > kMaxUnits || a.H % kBwdUnits != 0) return p;
  if ((G * a.H) % ch != 0) return p;
  int nch = 0;
  for (int q = 0; q < a.nunits; ++q) {
    const BwdUnit& u = a.u[q];
    if (u.rec_bytes >= kNoRow || (u.up && (u.k_up % ch != 0 || u.up_bytes >= kNoRow))) return p;
    nch = std::max(nch, (u.up ? u.k_up / ch : 0) + G * a.H / ch);
  }
  const int cap = bf16 ? 8 : 16;
  for (int nw : {4, 16}) {
    const int per = (nch + nw - 1) / nw;
    int m = 1;
    while (m < per) m *= 2;
    if (m <= cap) {
      p.nw = nw;
      p.maxc = m;
      break;
    }
  }
  if (p.nw == 0) return p;
  p.blocks = a.nunits * (a.H / kBwdUnits) * ((B + 15) / 16);
  p.shmem = sizeof(float) * p.nw * 256 + sizeof(int32_t) * (2 * a.T + 1);
  p.kernel = bwd_kernel(cell, bf16, p.nw, p.maxc);
  return p;
}

}  // namespace

int bwd_persistent_blocks(const BwdLaunch& a, int cell, bool bf16, int B) {
  const BwdPlan p = plan_bwd(a, cell, bf16, B);
  if (!p.kernel) return 0;
  if (p.blocks > max_coresident(p.kernel, 64 * p.nw, p.shmem)) return 0;
  return p.blocks;
}

hipError_t launch_bwd_persistent(BwdLaunch a, int cell, bool bf16, int B, hipStream_t st,
                                 bool* fits) {
  *fits = false;
  const BwdPlan p = plan_bwd(a, cell, bf16, B);
  if (!p.kernel) return hipSuccess;
  a.slices = a.H / kBwdUnits;
  a.rgroups = (B + 15) / 16;
  const int per_unit = a.slices * a.rgroups;
  for (int q = 0; q < a.nunits; ++q) a.u[q].wg_begin = q * per_unit;
  return coop_launch(p.kernel, p.blocks, 64 * p.nw, p.shmem, &a, st, fits);
}

hipError_t read_wait_timeouts(unsigned* count) {
  return hipMemcpyFromSymbol(count, HIP_SYMBOL(g_wait_timeouts), sizeof(unsigned), 0,
                             hipMemcpyDeviceToHost);
}

}  // namespace rnnbkt
