// Whole-sequence recurrences of LSTM/GRU layers in one launch, forward and
// backward through time: all layers of a unidirectional stack (each layer
// consuming the one below as it is published), or both directions of one
// bidirectional layer.
//
// A launch keeps every workgroup resident (its grid fits the GPU at once) and walks
// the T steps of the batch itself.  Each workgroup owns a fixed block of 16
// batch rows and a fixed slice of hidden units, so
//   - its slice of W_hh stays in registers for the whole launch (each lane
//     holds the MFMA operand fragments it feeds; read from HBM once),
//   - the recurrent state of its (row, unit) pairs (c for the LSTM, h for
//     the GRU update, the dc / dh carries backward) stays in registers,
//   - per-step operands that do not depend on other workgroups (the input
//     projection row, the saved gate activations) are fetched early.
//
// Each step reduces over two segments: first the input part (the layer
// input row forward, the gate gradient of the layer above backward), which
// does not depend on this recurrence and is fetched one step ahead, then the
// recurrent part, which other workgroups publish during the previous step.
//
// Exchange between workgroups without a grid barrier: the buffer a step
// publishes (h forward, the recurrent gate gradient backward) is filled
// with a sentinel bit pattern before the launch; every element of it is
// written exactly once during the launch with a relaxed device-scope atomic
// store (a value equal to the sentinel is replaced by the canonical NaN; a
// bf16 LSTM's backward stores its gate gradients as bf16 pairs, one word
// each, a pair equal to the sentinel becoming two canonical NaNs), and
// a reader polls its elements with device-scope loads until none holds the
// sentinel.  Single-location coherence of atomics is all this
// needs: no fence, no cache write-back or invalidation, and a workgroup
// waits only for the rows it reads (sequences are independent).  Polls are
// bounded; after a timeout the wait gives up, counts it (reported, then
// cleared, by rnnbkt_sync_check) and the later waits of the same launch
// return at once, so a launch always ends; other launches are not affected.
#include <hip/hip_runtime.h>

#include <atomic>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "kernels.h"

namespace rnnbkt {

// Waits that gave up since the host last cleared the count, and the
// generation of the last launch that had one (launch generations start at 1).
__device__ unsigned g_wait_timeouts = 0;
__device__ unsigned g_abandoned_gen = 0;

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));



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
constexpr int kEpiWaves = 4;     // backward waves running the gate-gradient algebra (256 threads)

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

// The lane's slots of one segment: slot i is chunk c = first + i*stride of
// the segment (used while c < nchunks).
struct Slots {
  int first, stride, nchunks, koff;
};

// Loads the lane's weight fragments of one segment: wk(k) returns the
// weight for segment-local reduction index k of this lane's column.
template <bool BF16, int MAXC, typename F>
__device__ inline void load_wfrags(typename WFrag<BF16>::T (&w)[MAXC], const Slots& sl, F wk) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int CPL = Chunk<BF16>::CPL;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = sl.first + i * sl.stride;
#pragma unroll
    for (int e = 0; e < CPL; ++e) {
      const float v = c < sl.nchunks ? wk(c * CH + sl.koff + e) : 0.f;
      if constexpr (BF16)
        w[i][e] = (__bf16)v;
      else
        w[i][e] = v;
    }
  }
}

// Issues the lane's loads of one segment: piece v of slot i is read at byte
// offset row_off + 4*(c*CH + koff + 4v) of the array behind `r` when the row
// exists (row_off != kNoRow) and the piece starts below klim; other pieces
// read zero.  AUX: the loads' cache policy -- device scope for arrays that
// other workgroups of the launch publish, 0 (cached) for complete ones.
template <bool BF16, int MAXC, int AUX = kDeviceScope>
__device__ inline void issue_segment(__amdgpu_buffer_rsrc_t r, unsigned row_off, const Slots& sl,
                                     int klim, unsigned (&u)[Chunk<BF16>::CPL * MAXC]) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int NV = Chunk<BF16>::CPL / 4;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = sl.first + i * sl.stride;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int kk = c * CH + sl.koff + 4 * v;
      const unsigned o =
          (row_off != kNoRow && c < sl.nchunks && kk < klim) ? row_off + 4u * (unsigned)kk : kNoRow;
      const u4 x = __builtin_amdgcn_raw_buffer_load_b128(r, o, 0, AUX);
#pragma unroll
      for (int e = 0; e < 4; ++e) u[(i * NV + v) * 4 + e] = x[e];
    }
  }
}

template <int NE>
__device__ inline bool segment_clear(const unsigned (&u)[NE]) {
  bool ready = true;
#pragma unroll
  for (int j = 0; j < NE; ++j) ready &= u[j] != kSentinel;
  return __all(ready);
}

// True once some wait of this launch has given up: its later waits return
// at once, so the launch still ends.
__device__ inline bool waits_abandoned(const WaitCtl& w) {
  return __hip_atomic_load(&g_abandoned_gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == w.gen;
}

// Counts a wait that gave up and marks the launch (one thread per call).
__device__ inline void note_timeout(const WaitCtl& w) {
  __hip_atomic_fetch_add(&g_wait_timeouts, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(&g_abandoned_gen, w.gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline void report_timeout(const WaitCtl& w) {
  if ((threadIdx.x & 63) == 0) note_timeout(w);
}

// The buffer loads are pure reads to the compiler: between two polls of the
// same addresses it must be told that memory may have changed, or it merges
// the polls into one (no code is emitted for this).
__device__ inline void poll_fence() { __asm__ __volatile__("" ::: "memory"); }

// Poll budget of one wait unless RNNBKT_MAX_POLLS sets another.
constexpr unsigned kMaxPolls = 1u << 20;

// Re-reads the segment until no element holds the sentinel (wave-uniform).
// One poll at a time: keeping a second poll in flight detects arrivals
// sooner, but its load is still pending when the next step issues, which
// costs more than it saves.
template <bool BF16, int MAXC>
__device__ inline void settle_segment(__amdgpu_buffer_rsrc_t r, unsigned row_off, const Slots& sl,
                                      int klim, unsigned (&u)[Chunk<BF16>::CPL * MAXC],
                                      const WaitCtl& w) {
  if (segment_clear(u)) return;
  for (unsigned polls = 1;; ++polls) {
    __builtin_amdgcn_s_sleep(1);
    poll_fence();
    issue_segment<BF16, MAXC>(r, row_off, sl, klim, u);
    if (segment_clear(u)) return;
    // The abandoned flag is a device-scope load: checking it only every
    // 1024 polls keeps its round trip off the path of a wait that is about
    // to succeed (checked at every wait's first miss, it cost a round trip
    // per step).
    if ((polls & 1023u) == 0 && waits_abandoned(w)) return;
    if (polls >= w.max_polls) {
      report_timeout(w);
      return;
    }
  }
}

// acc += (16 rows x segment) . (segment x 16 columns) over the lane's slots.
template <bool BF16, int MAXC>
__device__ inline void mma_segment(f4& acc, const unsigned (&u)[Chunk<BF16>::CPL * MAXC],
                                   const typename WFrag<BF16>::T (&w)[MAXC], const Slots& sl) {
  constexpr int CPL = Chunk<BF16>::CPL;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = sl.first + i * sl.stride;
    if (c >= sl.nchunks) break;
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
}

// Packed bf16 segments (the gate gradients a bf16 LSTM backward publishes):
// element k of a row at byte row_off + 2k, two elements per 32-bit word (the
// sentinel test stays per word).  A slot is one 16-byte load of the 8
// consecutive k it feeds to one MFMA, which takes the words as they are:
// every consumer of these values rounds them to bf16 anyway, so storing
// them rounded changes no result and halves what each step exchanges.
template <int MAXC, int AUX = kDeviceScope>
__device__ inline void issue_segment_pk(__amdgpu_buffer_rsrc_t r, unsigned row_off, const Slots& sl,
                                        int klim, unsigned (&u)[4 * MAXC]) {
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = sl.first + i * sl.stride;
    const int kk = c * 32 + sl.koff;
    const unsigned o =
        (row_off != kNoRow && c < sl.nchunks && kk < klim) ? row_off + 2u * (unsigned)kk : kNoRow;
    const u4 x = __builtin_amdgcn_raw_buffer_load_b128(r, o, 0, AUX);
#pragma unroll
    for (int e = 0; e < 4; ++e) u[i * 4 + e] = x[e];
  }
}

template <int MAXC>
__device__ inline void settle_segment_pk(__amdgpu_buffer_rsrc_t r, unsigned row_off,
                                         const Slots& sl, int klim, unsigned (&u)[4 * MAXC],
                                         const WaitCtl& w) {
  if (segment_clear(u)) return;
  for (unsigned polls = 1;; ++polls) {
    __builtin_amdgcn_s_sleep(1);
    poll_fence();
    issue_segment_pk<MAXC>(r, row_off, sl, klim, u);
    if (segment_clear(u)) return;
    if ((polls & 1023u) == 0 && waits_abandoned(w)) return;
    if (polls >= w.max_polls) {
      report_timeout(w);
      return;
    }
  }
}

template <int MAXC>
__device__ inline void mma_segment_pk(f4& acc, const unsigned (&u)[4 * MAXC],
                                      const bf8 (&w)[MAXC], const Slots& sl) {
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = sl.first + i * sl.stride;
    if (c >= sl.nchunks) break;
    const u4 x = {u[i * 4], u[i * 4 + 1], u[i * 4 + 2], u[i * 4 + 3]};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, x), w[i], acc, 0, 0, 0);
  }
}

// The value of the neighbouring lane (lane ^ 1): a DPP quad permutation
// [1, 0, 3, 2] on the VALU, where a shuffle would go through the LDS and be
// waited for.
__device__ inline float lane_xor1(float v) {
  const int i = __float_as_int(v);
  return __int_as_float(__builtin_amdgcn_update_dpp(i, i, 0xB1, 0xF, 0xF, false));
}

// Publishes two bf16 values as one word (lo at the lower address); a word
// equal to the sentinel becomes a pair of canonical NaNs.
__device__ inline void publish_pk(unsigned* p, float lo, float hi) {
  unsigned u = (unsigned)__builtin_bit_cast(unsigned short, (__bf16)lo) |
               ((unsigned)__builtin_bit_cast(unsigned short, (__bf16)hi) << 16);
  if (u == kSentinel) u = 0x7FC07FC0u;
  __hip_atomic_store(p, u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

// Copies unit `ui` out of the kernel arguments without dynamic indexing.
__device__ inline FwdUnit pick_unit(const FwdLaunch& a, int ui) {
  FwdUnit u = a.u[0];
  if (ui == 1) u = a.u[1];
  if (ui == 2) u = a.u[2];
  if (ui == 3) u = a.u[3];
  return u;
}

// Workgroups are dispatched to the 8 XCDs in turn (block b on XCD b mod 8),
// each XCD with its own L2.  The S workgroups of one (unit, row group)
// cluster exchange values every step, so each cluster is kept on one XCD.
// With a cluster count nc that is a multiple of 8, consecutive logical ids
// share an XCD (nc / 8 whole clusters each: logical_block).  Otherwise the
// GRU backward pads its grid to ceil(nc / 8) cluster places per XCD
// (rec_grid, cluster_block): XCD x takes clusters x, x + 8, ..., and the
// workgroups of the empty places exit at once (-1), and so does the forward
// with 12 or 16 units per workgroup.  The 8-unit forward keeps the plain
// numbering: padded, gru2's 48-workgroup clusters put two workgroups on half
// the CUs of an XCD and its step got slower (14.1 -> 18.4 us).
constexpr int kXcds = 8;
__device__ inline int logical_block(int n) {
  const int b = blockIdx.x;
  if (n % kXcds != 0) return b;
  return (b % kXcds) * (n / kXcds) + b / kXcds;
}
__device__ inline int cluster_block(int rec_blocks, int nc, int S) {
  if (nc % kXcds == 0) return logical_block(rec_blocks);
  const int b = blockIdx.x;
  const int c = b % kXcds + kXcds * (b / kXcds / S);
  return c < nc ? c * S + b / kXcds % S : -1;
}

// ---------------------------------------------------------------- output layer
// See OutStreamArgs.  One 256-thread workgroup takes blocks first, first +
// stride, ...  LDS: W_out [C][Htop + 1] (the +1 keeps the 16 rows a fragment
// reads in different banks), the block's h rows [kOutRows][Htop + 1], its
// logits / dlogits [kOutRows][C + 1], 4 wave sums.  Products on
// v_mfma_f32_16x16x4_f32 as in the recurrence.
constexpr int kOutGroup = 256 / kOutRows;  // threads per row in the softmax
constexpr size_t kOutLdsMax = 96 * 1024;

__device__ inline float out_group_max(float v) {
#pragma unroll
  for (int o = kOutGroup / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kOutGroup));
  return v;
}
__device__ inline float out_group_sum(float v) {
#pragma unroll
  for (int o = kOutGroup / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kOutGroup);
  return v;
}

__device__ void output_consumer(const OutStreamArgs& a, int first, int stride, char* out_smem,
                                const WaitCtl& w) {
  const int Htop = a.Htop, C = a.C;
  const int WL = Htop + 1, ZL = C + 1;
  float* Ws = reinterpret_cast<float*>(out_smem);  // [C][WL]
  float* Hs = Ws + (size_t)C * WL;                 // [kOutRows][WL]
  float* Zs = Hs + (size_t)kOutRows * WL;          // [kOutRows][ZL]
  float* wsum = Zs + (size_t)kOutRows * ZL;        // [4]
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lq = lane >> 4;
  for (int i = tid; i < C * Htop; i += 256) Ws[(i / Htop) * WL + i % Htop] = a.W[i];
  // The sentinel fills are paced by the output blocks: block blk takes
  // quads [blk * per, (blk + 1) * per) of the fills laid end to end, so the
  // writes spread over the recurrence instead of contending with its first
  // steps (non-temporal stores: the lines are next read by another launch).
  int64_t fill_quads = 0;
  for (int j = 0; j < a.nfill; ++j) fill_quads += (a.fill[j].n + 3) / 4;
  const int64_t per = (fill_quads + a.nblocks - 1) / a.nblocks;
  auto fill_share = [&](int blk) {
    const u4 v4 = {kSentinel, kSentinel, kSentinel, kSentinel};
    const int64_t q1 = min(fill_quads, (int64_t)(blk + 1) * per);
    int64_t base = 0;
    for (int j = 0; j < a.nfill; ++j) {
      const int64_t n = a.fill[j].n, nq = (n + 3) / 4;
      const int64_t lo = max((int64_t)blk * per, base), hi = min(q1, base + nq);
      unsigned* p = a.fill[j].p;
      for (int64_t q = lo + tid; q < hi; q += 256) {
        const int64_t i4 = (q - base) * 4;
        if (i4 + 3 < n) {
          __builtin_nontemporal_store(v4, reinterpret_cast<u4*>(p + i4));
        } else {
          for (int64_t i = i4; i < n; ++i) p[i] = kSentinel;
        }
      }
      base += nq;
    }
  };
  const __amdgpu_buffer_rsrc_t rh = published_rsrc(a.h, a.h_bytes);
  constexpr int RT = kOutRows / 16;
  const int ctiles = (C + 15) / 16, htiles = Htop / 16;
  for (int blk = first; blk < a.nblocks; blk += stride) {
    if (a.nfill > 0) fill_share(blk);
    const int64_t f0 = (int64_t)blk * kOutRows;
    // this block's h rows, re-read until published
    for (int i = tid; i < kOutRows * Htop / 4; i += 256) {
      const int r = (4 * i) / Htop, k = (4 * i) % Htop;
      const unsigned o =
          f0 + r < a.N ? 4u * (unsigned)((f0 + r) * Htop + k) : kNoRow;
      u4 v = __builtin_amdgcn_raw_buffer_load_b128(rh, o, 0, kDeviceScope);
      for (unsigned polls = 1; v[0] == kSentinel || v[1] == kSentinel || v[2] == kSentinel ||
                               v[3] == kSentinel;
           ++polls) {
        __builtin_amdgcn_s_sleep(32);
        poll_fence();
        v = __builtin_amdgcn_raw_buffer_load_b128(rh, o, 0, kDeviceScope);
        if ((polls & 1023u) == 0 && waits_abandoned(w)) break;
        if (polls >= w.max_polls) {
          note_timeout(w);
          break;
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) Hs[r * WL + k + e] = __uint_as_float(v[e]);
    }
    __syncthreads();
    for (int t = wave; t < RT * ctiles; t += 4) {
      const int r0 = (t % RT) * 16, c0 = (t / RT) * 16;
      const int c = c0 + lr;
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < Htop; k += 4) {
        const float av = Hs[(r0 + lr) * WL + k + lq];
        const float bv = c < C ? Ws[c * WL + k + lq] : 0.f;
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
      }
      if (c < C) {
        const float b = a.bias[c];
#pragma unroll
        for (int q = 0; q < 4; ++q) Zs[(r0 + lq * 4 + q) * ZL + c] = acc[q] + b;
      }
    }
    __syncthreads();
    {
      const int r = tid / kOutGroup, g = tid % kOutGroup;
      const int64_t f = f0 + r;
      float* zr = Zs + r * ZL;
      float m = -INFINITY;
      for (int c = g; c < C; c += kOutGroup) m = fmaxf(m, zr[c]);
      m = out_group_max(m);
      float sacc = 0.f;
      for (int c = g; c < C; c += kOutGroup) sacc += expf(zr[c] - m);
      sacc = out_group_sum(sacc);
      const float lse = m + logf(sacc);
      const int label = f < a.N ? a.y[f] : -1;
      float zy = 0.f;
      for (int c = g; c < C; c += kOutGroup) {
        if (c == label) zy = zr[c];
        const float d = (expf(zr[c] - lse) - (c == label ? 1.f : 0.f)) * a.inv_n;
        zr[c] = f < a.N ? d : 0.f;
        if (f < a.N) a.dz[f * C + c] = d;
      }
      zy = out_group_sum(zy);
      float term = 0.f;
      if (g == 0 && f < a.N) term = (label >= 0 && label < C) ? lse - zy : NAN;
      // block sum of the row terms, fixed order: butterfly in a wave, then waves
      for (int o = 32; o > 0; o >>= 1) term += __shfl_xor(term, o, 64);
      if (lane == 0) wsum[wave] = term;
    }
    __syncthreads();
    if (tid == 0) publish(a.partial + blk, (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]));
    for (int t = wave; t < RT * htiles; t += 4) {
      const int r0 = (t % RT) * 16, h0 = (t / RT) * 16;
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < C; k += 4) {
        const float av = Zs[(r0 + lr) * ZL + k + lq];
        const float bv = Ws[(k + lq) * WL + h0 + lr];
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc, 0, 0, 0);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t f = f0 + r0 + lq * 4 + q;
        if (f < a.N) a.dh[f * Htop + h0 + lr] = acc[q];
      }
    }
    __syncthreads();  // Hs, Zs and wsum are rewritten for the next block
  }
  // The last workgroup to finish sums the partials.  The counter is a
  // relaxed atomic and orders nothing: the partials are published values
  // (sentinel until written), so the last workgroup polls each of them.
  if (tid == 0) {
    const unsigned prev = __hip_atomic_fetch_add(a.done, 1u, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_AGENT);
    wsum[0] = prev + 1 == (unsigned)stride ? 1.f : 0.f;
  }
  __syncthreads();
  if (wsum[0] != 0.f) {
    // The partials are published (sentinel until written): poll them.
    const __amdgpu_buffer_rsrc_t rp = published_rsrc(a.partial, 4u * (unsigned)a.nblocks);
    float v = 0.f;
    for (int i = tid; i < a.nblocks; i += 256) {
      unsigned x = __builtin_amdgcn_raw_buffer_load_b32(rp, 4u * (unsigned)i, 0, kDeviceScope);
      for (unsigned polls = 1; x == kSentinel; ++polls) {
        __builtin_amdgcn_s_sleep(1);
        poll_fence();
        x = __builtin_amdgcn_raw_buffer_load_b32(rp, 4u * (unsigned)i, 0, kDeviceScope);
        if ((polls & 1023u) == 0 && waits_abandoned(w)) break;
        if (polls >= w.max_polls) {
          note_timeout(w);
          break;
        }
      }
      v += __uint_as_float(x);
    }
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    __syncthreads();
    if (lane == 0) wsum[wave] = v;
    __syncthreads();
    if (tid == 0) a.loss[0] = ((wsum[0] + wsum[1]) + (wsum[2] + wsum[3])) * a.inv_n;
  }
}

// Copies the batch tables into LDS.
__device__ inline void load_tables(const int32_t* bs, const int32_t* off, int T, int32_t* tbs,
                                   int32_t* toff) {
  for (int i = threadIdx.x; i <= T; i += blockDim.x) {
    if (i < T) tbs[i] = bs[i];
    toff[i] = off[i];
  }
}

// Forward recurrence of the launch's units.  Workgroup = 16 rows x 4*NT
// hidden units of one unit; column block nt holds, for its 4 units, the
// LSTM gates (i, f, g, o) or the GRU groups (r, z, n from the input, n from
// the state), so one MFMA tile per block yields every pre-activation a
// unit's update needs.  NW waves split each segment's reduction; waves
// 0..NT-1 then run the state update of one column block each.
// MAXC: slots per wave of the widest segment; MR (<= MAXC): slots of the
// recurrent segment, whose poll is on the step's critical path and is
// compiled for its own width.  MR < MAXC only where no unit of the launch
// reads an input that the launch publishes: the input is then read through
// the caches (the workgroups of a row group share one XCD and read the
// same input rows).
template <int G, bool BF16, int NW, int MAXC, int NT, int MR>
__global__ __launch_bounds__(64 * NW) void k_fwd_persistent(FwdLaunch a) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int CPL = Chunk<BF16>::CPL;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* red = reinterpret_cast<float*>(smem);                     // [NW][NT][256]
  int32_t* tbs = reinterpret_cast<int32_t*>(red + NW * NT * 256);  // batch sizes [T]
  int32_t* toff = tbs + a.T;                                       // offsets [T+1]
  // Output-layer workgroups follow the recurrence ones (physical ids, so the
  // renumbering below is that of the recurrence grid alone).
  const int rec_blocks = gridDim.x - a.out_blocks;
  if constexpr (!BF16) {
    if ((int)blockIdx.x >= rec_blocks) {
      output_consumer(a.out, blockIdx.x - rec_blocks, a.out_blocks, smem, a.wait);
      return;
    }
  }
  load_tables(a.bs, a.off, a.T, tbs, toff);
  int bid;
  if constexpr (NT >= 3) {
    bid = cluster_block(rec_blocks, a.nunits * a.rgroups, a.slices);
    if (bid < 0) return;
  } else {
    bid = logical_block(rec_blocks);
  }
  int ui = 0;
  for (int q = 1; q < a.nunits; ++q)
    if (bid >= a.u[q].wg_begin) ui = q;
  const FwdUnit U = pick_unit(a, ui);
  const int rem = bid - U.wg_begin;
  const int slice = rem % a.slices;
  const int rg = rem / a.slices;
  const int H = a.H;
  const int j0 = slice * 4 * NT;
  const int r0 = rg * 16;
  const int lane = threadIdx.x & 63;
  // Wave-uniform: the per-slot tests below then become scalar branches.  An
  // MFMA placed in a lane-masked region still reads every lane, so a slot
  // must be skipped by the whole wave, never by masking.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const Slots sin{wave, NW, (U.kin + CH - 1) / CH, lq * CPL};
  const Slots srec{wave, NW, H / CH, lq * CPL};

  // Weight fragments: this lane feeds column lr of every column block.
  typename WFrag<BF16>::T win[NT][MAXC], wrec[NT][MR];
  {
    const int grp = lr >> 2, uu = lr & 3;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = j0 + 4 * nt + uu;
      // gate row of W_ih / W_hh feeding this column (-1 = none)
      const int gi = G == 4 ? grp : (grp == 3 ? -1 : grp);
      const int gh = G == 4 ? grp : (grp == 2 ? -1 : (grp == 3 ? 2 : grp));
      const float* wi = gi >= 0 ? U.wih + (int64_t)(gi * H + j) * U.kin : nullptr;
      const float* wh = gh >= 0 ? U.whh + (int64_t)(gh * H + j) * H : nullptr;
      load_wfrags<BF16, MAXC>(win[nt], sin, [&](int k) { return (wi && k < U.kin) ? wi[k] : 0.f; });
      load_wfrags<BF16, MR>(wrec[nt], srec, [&](int k) { return wh ? wh[k] : 0.f; });
    }
  }
  // State-update lanes: wave nt < NT owns row r0 + (lane >> 2), unit
  // j0 + 4*nt + (lane & 3) for the whole launch.
  const bool epi = wave < NT;
  const int erow = r0 + (lane >> 2);
  const int ej = j0 + 4 * (epi ? wave : 0) + (lane & 3);
  float bi[4] = {0.f, 0.f, 0.f, 0.f}, bh[3] = {0.f, 0.f, 0.f};
  // LSTM peepholes of this unit (the test is uniform over the workgroup).
  const bool peep = G == 4 && U.peep != nullptr;
  float pi = 0.f, pf = 0.f, po = 0.f;
  if (epi) {
    if (peep) {
      pi = U.peep[ej];
      pf = U.peep[H + ej];
      po = U.peep[2 * H + ej];
    }
#pragma unroll
    for (int g = 0; g < G; ++g) bi[g] = U.b[g * H + ej];
    if constexpr (G == 3) {
#pragma unroll
      for (int g = 0; g < 3; ++g) bh[g] = U.bhh[g * H + ej];
    }
  }
  float c_state = 0.f, h_state = 0.f;
  // bf16 above the first layer: the input rows come from the packed copy of
  // the layer below (half the bytes; rounded to bf16 by the products anyway).
  const bool in_pk = BF16 && U.inx != nullptr;
  const __amdgpu_buffer_rsrc_t rin =
      in_pk ? published_rsrc(reinterpret_cast<const float*>(U.inx), U.inx_bytes)
            : published_rsrc(U.in, U.in_bytes);
  const __amdgpu_buffer_rsrc_t rout = published_rsrc(U.hout, U.out_bytes);
  // bf16: the recurrent segment is polled from the packed copy of the
  // output (half the bytes; the products round it to bf16 anyway).
  const __amdgpu_buffer_rsrc_t rhx =
      published_rsrc(reinterpret_cast<const float*>(U.hx), U.hx_bytes);
  const int r = r0 + lr;
  __syncthreads();
  // Publishes element e of the output row layout as half of a bf16 pair:
  // units ej and ej + 1 sit in neighbouring lanes of one row, and the even
  // lane stores the word.
  auto publish_hx = [&](int64_t e, float v) {
    const float other = lane_xor1(v);
    if ((e & 1) == 0) publish_pk(U.hx + (e >> 1), v, other);
  };
  // The new state: bf16, first the packed copy the next step polls, then the
  // output itself (published only where a unit of this launch polls it).
  auto put_h = [&](int64_t e, float v) {
    if constexpr (BF16) {
      publish_hx(e, v);
      if (U.out_polled)
        publish(U.hout + e, v);
      else
        U.hout[e] = v;
    } else {
      publish(U.hout + e, v);
    }
  };

  auto in_off = [&](const StepIdx& q) {
    return r < q.rows ? (in_pk ? 2u : 4u) * (unsigned)((int64_t)(q.row0 + r) * U.ld_in) : kNoRow;
  };
  StepIdx s = fwd_step(tbs, toff, a.T, U.dir, 0);
  unsigned uin[CPL * MAXC];
  // The packed input uses the first 4 words of each slot.
  unsigned (&uin_pk)[4 * MAXC] = *reinterpret_cast<unsigned (*)[4 * MAXC]>(&uin[0]);
  auto issue_in = [&](const StepIdx& q) {
    if (in_pk)
      issue_segment_pk<MAXC, MR < MAXC ? 0 : kDeviceScope>(rin, in_off(q), sin, U.kin, uin_pk);
    else
      issue_segment<BF16, MAXC, MR < MAXC ? 0 : kDeviceScope>(rin, in_off(q), sin, U.kin, uin);
  };
  issue_in(s);
  for (int k = 0; k < a.T; ++k) {
    StepIdx nx = s;
    if (k + 1 < a.T) nx = fwd_step(tbs, toff, a.T, U.dir, k + 1);
    const bool active = r0 < s.rows;
    if (active) {
      f4 acc[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
      // Input part (fetched one step ahead; a published input may still be
      // arriving), then the recurrent poll.  (Polling first and multiplying
      // the input while the poll is in flight made bilstm3's upper-layer
      // launches slower: 1.92 against 1.37 ms.)
      if constexpr (BF16) {
        if (in_pk) {
          if (U.in_published) settle_segment_pk<MAXC>(rin, in_off(s), sin, U.kin, uin_pk, a.wait);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) mma_segment_pk<MAXC>(acc[nt], uin_pk, win[nt], sin);
        } else {
          if (U.in_published) settle_segment<BF16, MAXC>(rin, in_off(s), sin, U.kin, uin, a.wait);
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) mma_segment<BF16, MAXC>(acc[nt], uin, win[nt], sin);
        }
      } else {
        if (U.in_published) settle_segment<BF16, MAXC>(rin, in_off(s), sin, U.kin, uin, a.wait);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mma_segment<BF16, MAXC>(acc[nt], uin, win[nt], sin);
      }
      // Recurrent part.
      const int64_t rel = (int64_t)(s.prev0 + r) * a.ldh + U.hcol;
      if constexpr (BF16) {
        const unsigned roff = r < s.prev_rows ? 2u * (unsigned)rel : kNoRow;
        unsigned urec[4 * MR];
        issue_segment_pk<MR>(rhx, roff, srec, H, urec);
        settle_segment_pk<MR>(rhx, roff, srec, H, urec, a.wait);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mma_segment_pk<MR>(acc[nt], urec, wrec[nt], srec);
      } else {
        const unsigned roff = r < s.prev_rows ? 4u * (unsigned)rel : kNoRow;
        unsigned urec[CPL * MR];
        issue_segment<BF16, MR>(rout, roff, srec, H, urec);
        settle_segment<BF16, MR>(rout, roff, srec, H, urec, a.wait);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) mma_segment<BF16, MR>(acc[nt], urec, wrec[nt], srec);
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          red[(wave * NT + nt) * 256 + (lq * 4 + q) * 16 + lr] = acc[nt][q];
    }
    if (k + 1 < a.T) issue_in(nx);
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
        const float cp = has_prev ? c_state : 0.f;
        float ai = sg[0] + bi[0], af = sg[1] + bi[1], ao = sg[3] + bi[3];
        if (peep) {
          ai += pi * cp;
          af += pf * cp;
        }
        const float ig = act_sigmoid(ai);
        const float fg = act_sigmoid(af);
        const float gg = act_tanh(sg[2] + bi[2]);
        c_state = fg * cp + ig * gg;
        if (peep) ao += po * c_state;
        const float og = act_sigmoid(ao);
        h_state = og * act_tanh(c_state);
        put_h(f * a.ldh + U.hcol + ej, h_state);
        st[ej] = ig;
        st[H + ej] = fg;
        st[2 * H + ej] = gg;
        st[3 * H + ej] = og;
        U.cst[f * H + ej] = c_state;
      } else {
        const float rg_ = act_sigmoid(sg[0] + bi[0] + bh[0]);
        const float z = act_sigmoid(sg[1] + bi[1] + bh[1]);
        const float ahn = sg[3] + bh[2];
        const float n = act_tanh(sg[2] + bi[2] + rg_ * ahn);
        const float hp = has_prev ? h_state : 0.f;
        h_state = (1.f - z) * n + z * hp;
        put_h(f * a.ldh + U.hcol + ej, h_state);
        st[ej] = rg_;
        st[H + ej] = z;
        st[2 * H + ej] = n;
        st[3 * H + ej] = ahn;
      }
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

// ---------------------------------------------------------------- weight gradients
// C = A^T B over the frames of the batch, by workgroups of the backward
// launch beside the recurrence that publishes A (see WgStreamArgs).  The
// tile loop of a 256-thread sub-tile is the fp32 TN product of the GEMM
// kernels: 32-frame K-tiles staged untransposed in LDS ([k][m] and [k][n],
// rows padded by 16 floats), fed to v_mfma_f32_16x16x4_f32 with 4 waves of
// 32 x 32 each.  A's K-tile is read with device-scope loads and re-read until
// no element holds the sentinel.
constexpr int kWgBK = 32;
constexpr int kWgLD = 64 + 16;

constexpr size_t kWgSubLds = sizeof(float) * 2 * kWgBK * kWgLD;  // A and B K-tiles

__device__ inline void wg_load_a(u4 (&v)[2], __amdgpu_buffer_rsrc_t r, int lda, int c0, int clim,
                                 int k0, int klim, int tid) {
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int k = (tid >> 4) + rep * 16;
    const int c = (tid & 15) * 4;
    const unsigned o = (k0 + k < klim && c0 + c < clim)
                           ? 4u * (unsigned)((int64_t)(k0 + k) * lda + c0 + c)
                           : kNoRow;
    v[rep] = __builtin_amdgcn_raw_buffer_load_b128(r, o, 0, kDeviceScope);
  }
}

__device__ inline bool wg_clear(const u4 (&v)[2]) {
  bool ok = true;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep)
#pragma unroll
    for (int e = 0; e < 4; ++e) ok &= v[rep][e] != kSentinel;
  return ok;
}

// Waits until element (k, c0) of A is published: one word, the same for
// every thread (one load per wave), polled before whole K-tiles are read.
__device__ inline void wg_wait_word(__amdgpu_buffer_rsrc_t r, int lda, int c0, int k,
                                    const WaitCtl& w) {
  const unsigned o = 4u * (unsigned)((int64_t)k * lda + c0);
  unsigned x = __builtin_amdgcn_raw_buffer_load_b32(r, o, 0, kDeviceScope);
  for (unsigned polls = 1; x == kSentinel; ++polls) {
    __builtin_amdgcn_s_sleep(32);
    poll_fence();
    x = __builtin_amdgcn_raw_buffer_load_b32(r, o, 0, kDeviceScope);
    if ((polls & 1023u) == 0 && waits_abandoned(w)) return;
    if (polls >= w.max_polls) {
      note_timeout(w);
      return;
    }
  }
}

// Re-reads this thread's part of an A K-tile until it is all published.
__device__ inline void wg_settle_a(u4 (&v)[2], __amdgpu_buffer_rsrc_t r, int lda, int c0,
                                   int clim, int k0, int klim, int tid, const WaitCtl& w) {
  if (wg_clear(v)) return;
  for (unsigned polls = 1;; ++polls) {
    // (not on the recurrence's path: polling gently leaves it the memory
    // system; measured best of sleeps 2..64)
    __builtin_amdgcn_s_sleep(32);
    poll_fence();
    wg_load_a(v, r, lda, c0, clim, k0, klim, tid);
    if (wg_clear(v)) return;
    if ((polls & 1023u) == 0 && waits_abandoned(w)) return;
    if (polls >= w.max_polls) {
      note_timeout(w);
      return;
    }
  }
}

__device__ inline void wg_load_b(f4 (&v)[2], const float* P, int64_t ld, const int32_t* gather,
                                 int c0, int clim, int k0, int klim, int tid) {
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int k = (tid >> 4) + rep * 16;
    const int c = (tid & 15) * 4;
    f4 x = {0.f, 0.f, 0.f, 0.f};
    if (k0 + k < klim && c0 + c < clim) {
      int64_t row = k0 + k;
      if (gather) row = gather[row];
      if (row >= 0) x = *reinterpret_cast<const f4*>(P + row * ld + c0 + c);
    }
    v[rep] = x;
  }
}

__device__ inline void wg_store(float* S, const f4 (&v)[2], int tid) {
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int k = (tid >> 4) + rep * 16;
    const int c = (tid & 15) * 4;
    *reinterpret_cast<f4*>(S + k * kWgLD + c) = v[rep];
  }
}

__device__ inline void wg_store(float* S, const u4 (&v)[2], int tid) {
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int k = (tid >> 4) + rep * 16;
    const int c = (tid & 15) * 4;
    *reinterpret_cast<u4*>(S + k * kWgLD + c) = v[rep];
  }
}

__device__ inline WgJob pick_job(const WgStreamArgs& a, int j) {
  WgJob u = a.job[0];
#pragma unroll
  for (int q = 1; q < kWgJobs; ++q)
    if (j == q) u = a.job[q];
  return u;
}

// Role of workgroup wb (of the weight-gradient ones) in a backward launch of
// 64*NW threads: sub-tile threadIdx.x / 256 takes tile (wb % groups) * NW/4 +
// sub of repetition wb / groups; past the last tile it repeats the last one
// without storing, to keep step at the barriers.  LDS: NW/4 * kWgSubLds.
template <int NW>
__device__ void wgrad_role(const WgStreamArgs& a, int wb, float* lds, const WaitCtl& w) {
  constexpr int SUBS = NW / 4;
  const int sub = threadIdx.x >> 8, tid = threadIdx.x & 255;
  const int groups = (a.tiles + SUBS - 1) / SUBS;
  const int rep = wb / groups;
  const int t_raw = (wb % groups) * SUBS + sub;
  const bool owner = t_raw < a.tiles;
  const int tile = owner ? t_raw : a.tiles - 1;
  float* As = lds + (size_t)sub * 2 * kWgBK * kWgLD;
  float* Bs = As + kWgBK * kWgLD;
  int j = 0;
  for (int q = 1; q < a.njobs; ++q)
    if (tile >= a.job[q].tile_begin) j = q;
  const WgJob J = pick_job(a, j);
  const int lt = tile - J.tile_begin;
  const int mtiles = (J.M + 63) / 64;
  const int m0 = (lt % mtiles) * 64, n0 = (lt / mtiles) * 64;
  const __amdgpu_buffer_rsrc_t ra = published_rsrc(J.A, J.a_bytes);
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int lr = lane & 15, lq = lane >> 4;
  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) acc[i][jj] = f4{0.f, 0.f, 0.f, 0.f};

  for (int c = rep; c < a.nchunks; c += a.reps) {
    // chunk c: steps [t_lo, t_hi), the c-th group of spc steps from the end
    const int t_hi = a.T - c * a.spc;
    const int t_lo = t_hi - a.spc > 0 ? t_hi - a.spc : 0;
    const int kbeg = a.off[t_lo], kend = a.off[t_hi];
    u4 ua[2];
    f4 rb[2];
    // The chunk's last frame, first column of the tile: published at about
    // the time the rest of the chunk is, and one word to poll instead of
    // whole K-tiles while the recurrence has not reached the chunk yet (the
    // per-element check below stays the test of completeness).
    wg_wait_word(ra, J.lda, m0, kend - 1, w);
    wg_load_a(ua, ra, J.lda, m0, J.M, kbeg, kend, tid);
    wg_load_b(rb, J.B, J.ldb, J.gather, n0, J.N, kbeg, kend, tid);
    for (int k0 = kbeg; k0 < kend; k0 += kWgBK) {
      wg_settle_a(ua, ra, J.lda, m0, J.M, k0, kend, tid, w);
      wg_store(As, ua, tid);
      wg_store(Bs, rb, tid);
      __syncthreads();
      if (k0 + kWgBK < kend) {
        wg_load_a(ua, ra, J.lda, m0, J.M, k0 + kWgBK, kend, tid);
        wg_load_b(rb, J.B, J.ldb, J.gather, n0, J.N, k0 + kWgBK, kend, tid);
      }
#pragma unroll
      for (int kk = 0; kk < kWgBK; kk += 4) {
        const int kr = (kk + lq) * kWgLD;
        float av[2], bv[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) av[i] = As[kr + wm + i * 16 + lr];
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) bv[jj] = Bs[kr + wn + jj * 16 + lr];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
            acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[jj], acc[i][jj], 0, 0, 0);
      }
      __syncthreads();  // the K-tile in LDS is rewritten next
    }
  }
  if (!owner) return;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int n = n0 + wn + jj * 16 + lr;
      if (n >= J.N) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int m = m0 + wm + i * 16 + lq * 4 + q;
        if (m < J.M) J.partial[((int64_t)rep * J.M + m) * J.N + n] = acc[i][jj][q];
      }
    }
}

// Backpropagation through time of the launch's units.  Workgroup = 16 rows
// x 16 hidden units of one unit; NW waves split each segment's reduction;
// threads 0..255 then run the gate-gradient algebra of one (row, unit) each,
// carrying dc*f (LSTM) or dh*z (GRU) of their row and unit in a register and
// summing the unit's gate gradients over the steps for the bias gradients.
// UP = false: no unit of the launch reads a gradient from a layer above in
// the kernel (bidirectional layers, the top of a stack): the input segment's
// fragments and operands are not kept at all, which leaves their registers
// to the recurrent segment.
template <int G, bool BF16, int NW, int MAXC, bool SPLIT, bool UP>
__global__ __launch_bounds__(64 * NW) void k_bwd_persistent(BwdLaunch a) {
  constexpr int CH = Chunk<BF16>::CH;
  constexpr int CPL = Chunk<BF16>::CPL;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* red = reinterpret_cast<float*>(smem);                // [max(NW, 8)][256]
  int32_t* tbs = reinterpret_cast<int32_t*>(red + (NW < 8 ? 8 : NW) * 256);
  int32_t* toff = tbs + a.T;
  // Weight-gradient workgroups follow the recurrence ones.
  const int rec_blocks = gridDim.x - a.wg_blocks;
  if constexpr (G == 4 && !BF16) {
    if ((int)blockIdx.x >= rec_blocks) {
      wgrad_role<NW>(a.wg, blockIdx.x - rec_blocks, reinterpret_cast<float*>(smem), a.wait);
      return;
    }
  }
  load_tables(a.bs, a.off, a.T, tbs, toff);
  int bid;
  if constexpr (G == 3) {
    bid = cluster_block(rec_blocks, a.nunits * a.rgroups, a.slices);
    if (bid < 0) return;
  } else {
    bid = logical_block(rec_blocks);
  }
  int ui = 0;
  for (int q = 1; q < a.nunits; ++q)
    if (bid >= a.u[q].wg_begin) ui = q;
  const BwdUnit U = pick_unit(a, ui);
  const int rem = bid - U.wg_begin;
  const int slice = rem % a.slices;
  const int rg = rem / a.slices;
  const int H = a.H;
  const int GH = G * H;
  const int j0 = slice * kBwdUnits;
  const int r0 = rg * 16;
  const int lane = threadIdx.x & 63;
  // Wave-uniform: the per-slot tests below then become scalar branches.  An
  // MFMA placed in a lane-masked region still reads every lane, so a slot
  // must be skipped by the whole wave, never by masking.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 15, lq = lane >> 4;
  const bool has_up = U.up != nullptr;
  const int kup = has_up ? U.k_up : 0;
  // SPLIT (8 or 16 waves): the four gate-gradient waves neither poll nor
  // multiply.  Their per-step operand loads (saved gates, cell states, the
  // gradient from above) come from HBM, and loads complete in issue order,
  // so in a polling wave they would hold up every poll behind them.
  static_assert(!SPLIT || NW >= 8, "the split needs waves beyond the gate-gradient ones");
  constexpr int NMMA = SPLIT ? NW - kEpiWaves : NW;
  const bool mma_wave = !SPLIT || wave >= kEpiWaves;
  const int mw = SPLIT ? wave - kEpiWaves : wave;
  const int first = mma_wave ? mw : (1 << 20);  // no slots for the others
  const Slots sup{first, NMMA, kup / CH, lq * CPL};
  const Slots srec{first, NMMA, GH / CH, lq * CPL};
  // A bf16 LSTM publishes its gate gradients as packed bf16 (two per word).
  constexpr bool PK = BF16 && G == 4;
  constexpr int WPS = PK ? 4 : CPL;      // 32-bit words a slot loads
  constexpr unsigned kEB = PK ? 2u : 4u;  // bytes per published element
  auto seg_issue = [&](__amdgpu_buffer_rsrc_t rr, unsigned off, const Slots& sl, int klim,
                       auto& u) {
    if constexpr (PK)
      issue_segment_pk<MAXC>(rr, off, sl, klim, u);
    else
      issue_segment<BF16, MAXC>(rr, off, sl, klim, u);
  };
  auto seg_settle = [&](__amdgpu_buffer_rsrc_t rr, unsigned off, const Slots& sl, int klim,
                        auto& u) {
    if constexpr (PK)
      settle_segment_pk<MAXC>(rr, off, sl, klim, u, a.wait);
    else
      settle_segment<BF16, MAXC>(rr, off, sl, klim, u, a.wait);
  };
  auto seg_mma = [&](f4& acc, const auto& u, const auto& wf, const Slots& sl) {
    if constexpr (PK)
      mma_segment_pk<MAXC>(acc, u, wf, sl);
    else
      mma_segment<BF16, MAXC>(acc, u, wf, sl);
  };

  // Weight fragments: column lr is hidden unit j0 + lr.
  constexpr int MU = UP ? MAXC : 1;
  typename WFrag<BF16>::T wup[MU], wrec[MAXC];
  {
    const int j = j0 + lr;
    const float* wu = has_up ? U.wih_up + U.hcol + j : nullptr;
    const float* wh = U.whh + j;
    if constexpr (UP)
      load_wfrags<BF16, MAXC>(wup, sup, [&](int k) { return wu ? wu[(int64_t)k * U.din_up] : 0.f; });
    load_wfrags<BF16, MAXC>(wrec, srec, [&](int k) { return wh[(int64_t)k * H]; });
  }
  // Gate-gradient threads: 0..255 -> row r0 + (tid >> 4), unit j0 + (tid & 15).
  const bool epi = threadIdx.x < 256;
  const int erow = r0 + ((threadIdx.x & 255) >> 4);
  const int ej = j0 + (threadIdx.x & 15);
  float carry = 0.f;
  float bsum[4] = {0.f, 0.f, 0.f, 0.f};  // sum over steps of this (row, unit)'s dA (LSTM) / dAx (GRU)
  float bsumh[3] = {0.f, 0.f, 0.f};      // GRU: sum of dAh; peephole LSTM: peephole gradients
  // LSTM peepholes of this unit (the test is uniform over the workgroup).
  const bool peep = G == 4 && U.peep != nullptr;
  float pi = 0.f, pf = 0.f, po = 0.f;
  if (epi && peep) {
    pi = U.peep[ej];
    pf = U.peep[H + ej];
    po = U.peep[2 * H + ej];
  }
  const float* rec = G == 3 ? U.dah : U.da;
  const __amdgpu_buffer_rsrc_t rup = published_rsrc(has_up ? U.up : U.da, has_up ? U.up_bytes : 0u);
  const __amdgpu_buffer_rsrc_t rrec = published_rsrc(rec, U.rec_bytes);
  const bool pub_dax = G == 4 || U.publish_dax != 0;
  const int r = r0 + lr;
  __syncthreads();

  auto up_off = [&](const BwdIdx& q) {
    return (has_up && r < q.rows) ? kEB * (unsigned)((int64_t)(q.row0 + r) * kup) : kNoRow;
  };
  // Operands of the gate-gradient algebra that do not depend on other
  // workgroups (inactive rows read frame 0 and are ignored).
  auto fetch_ops = [&](const BwdIdx& q, float& dhv_, float& s0_, float& s1_, float& s2_,
                       float& s3_, float& cc_, float& cp_) {
    const int64_t fq = erow < q.rows ? q.row0 + erow : 0;
    const int64_t fp = erow < q.prev_rows ? q.prev0 + erow : 0;
    dhv_ = U.dh_in ? U.dh_in[fq * U.ld_dh + U.hcol + ej] : 0.f;
    const float* st = U.stash + fq * 4 * H;
    s0_ = st[ej];
    s1_ = st[H + ej];
    s2_ = st[2 * H + ej];
    s3_ = st[3 * H + ej];
    if constexpr (G == 4) {
      cc_ = U.cst[fq * H + ej];
      cp_ = U.cst[fp * H + ej];
    } else {
      cc_ = 0.f;
      cp_ = U.hout[fp * a.ldh + U.hcol + ej];
    }
  };
  // Operands of the gate-gradient algebra.  Fetched one step ahead
  // (kAheadOps), one set per step in flight: the loop then runs two steps
  // per iteration with the sets in turn, so a fetched set is never copied (a
  // copy would wait for its loads at the end of every step).
  struct Ops {
    float dhv = 0.f, st0 = 0.f, st1 = 0.f, st2 = 0.f, st3 = 0.f, cc = 0.f, cprev = 0.f;
  };
  Ops oa, ob;
  // Without the split the gate-gradient waves also poll, and loads complete
  // in issue order, so operands fetched at the top of a step hold up that
  // wave's poll: with few slots per wave they are fetched one step ahead,
  // after the step's poll has completed (bilstm3's backward, 2 slots: 1.94
  // -> 1.71 ms per launch; with 4 slots, longtail's, it was slower: 1.36 ->
  // 1.42).  With the split, fetching them ahead measured slower too.
  constexpr bool kAheadOps = !SPLIT && MAXC <= 2;
  BwdIdx s = bwd_step(tbs, toff, a.T, U.dir, 0);
  unsigned uup[WPS * MU];
  if constexpr (UP)
    if (mma_wave) seg_issue(rup, up_off(s), sup, kup, uup);
  // The first step's operands are fetched before the loop: fetched inside it
  // (under k == 0), their registers would count as possibly pending at every
  // step, and the compiler would wait for all loads in flight -- the next
  // step's operands included -- before the cell algebra.
  if constexpr (kAheadOps) {
    if (epi && a.T > 0) fetch_ops(s, oa.dhv, oa.st0, oa.st1, oa.st2, oa.st3, oa.cc, oa.cprev);
    // and waited for here (vmcnt 0), so that no step starts with them pending
    __builtin_amdgcn_s_waitcnt(0x0F70);
  }
  auto step = [&](int k, Ops& cur, Ops& nxt) {
    BwdIdx nx = s;
    if (k + 1 < a.T) nx = bwd_step(tbs, toff, a.T, U.dir, k + 1);
    const bool active = r0 < s.rows;
    const int64_t f = erow < s.rows ? s.row0 + erow : 0;
    const bool has_prev = erow < s.prev_rows;
    // Loaded at the top of the step, or (kAheadOps) one step ahead.
    if constexpr (!kAheadOps)
      if (epi) fetch_ops(s, cur.dhv, cur.st0, cur.st1, cur.st2, cur.st3, cur.cc, cur.cprev);
    if (active && mma_wave) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      // Gradient arriving from the layer above (fetched one step ahead).
      if constexpr (UP) {
        if (U.up_published) seg_settle(rup, up_off(s), sup, kup, uup);
        seg_mma(acc, uup, wup, sup);
      }
      // Recurrent part.
      const unsigned roff =
          r < s.next_rows ? kEB * (unsigned)((int64_t)(s.next0 + r) * GH) : kNoRow;
      unsigned urec[WPS * MAXC];
      seg_issue(rrec, roff, srec, GH, urec);
      seg_settle(rrec, roff, srec, GH, urec);
      seg_mma(acc, urec, wrec, srec);
#pragma unroll
      for (int q = 0; q < 4; ++q) red[mw * 256 + (lq * 4 + q) * 16 + lr] = acc[q];
    }
    // (kAheadOps) This step's operands, fetched a step ago, are waited for
    // before anything else is issued (they have long arrived): the compiler
    // then knows them complete, and the cell algebra waits for no load.
    if constexpr (kAheadOps) __builtin_amdgcn_s_waitcnt(0x0F70);
    if constexpr (UP)
      if (k + 1 < a.T && mma_wave) seg_issue(rup, up_off(nx), sup, kup, uup);
    if constexpr (kAheadOps)
      if (epi && k + 1 < a.T) fetch_ops(nx, nxt.dhv, nxt.st0, nxt.st1, nxt.st2, nxt.st3, nxt.cc, nxt.cprev);
    __syncthreads();
    if (epi && active && erow < s.rows) {
      const bool has_next = erow < s.next_rows;
      // All the partials are read before the first sum (the scheduling
      // barrier keeps the reads together), then summed in a fixed order
      // (bilstm3's backward 1.20 -> 1.11 ms per launch; the same in the
      // forward's state update made bf16 forwards slower).
      float part[NMMA];
#pragma unroll
      for (int w_ = 0; w_ < NMMA; ++w_) part[w_] = red[w_ * 256 + threadIdx.x];
      __builtin_amdgcn_sched_barrier(0);
      float dh_red = 0.f;
#pragma unroll
      for (int w_ = 0; w_ < NMMA; ++w_) dh_red += part[w_];
      if constexpr (G == 4) {
        const float dh = cur.dhv + dh_red;
        const float tc = act_tanh(cur.cc);
        const float dout = dh * tc * cur.st3 * (1.f - cur.st3);
        // c_t reaches the loss through h_t, the next step and the output peephole
        float dc = dh * cur.st3 * (1.f - tc * tc) + (has_next ? carry : 0.f);
        if (peep) dc += dout * po;
        const float cp = has_prev ? cur.cprev : 0.f;
        const float di = dc * cur.st2 * cur.st0 * (1.f - cur.st0);
        const float df = dc * cp * cur.st1 * (1.f - cur.st1);
        const float dg = dc * cur.st0 * (1.f - cur.st2 * cur.st2);
        if constexpr (PK) {
          // Units ej and ej + 1 sit in neighbouring lanes of the same row:
          // the even lane publishes the pair.
          // (Measured: one gate after another where the operands are fetched
          // ahead -- bilstm3's backward 1.26 against 1.20 ms per launch --
          // and the four gates' stores together otherwise -- longtail's
          // 0.86 against 0.83 ms.)
          const float gv[4] = {di, df, dg, dout};
          unsigned* dw = reinterpret_cast<unsigned*>(U.da) + ((f * GH + ej) >> 1);
          if constexpr (kAheadOps) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const float other = lane_xor1(gv[g]);
              if ((ej & 1) == 0) publish_pk(dw + ((g * H) >> 1), gv[g], other);
            }
          } else {
            float other[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) other[g] = lane_xor1(gv[g]);
            if ((ej & 1) == 0) {
#pragma unroll
              for (int g = 0; g < 4; ++g) publish_pk(dw + ((g * H) >> 1), gv[g], other[g]);
            }
          }
        } else {
          float* dar = U.da + f * GH;
          publish(dar + ej, di);
          publish(dar + H + ej, df);
          publish(dar + 2 * H + ej, dg);
          publish(dar + 3 * H + ej, dout);
        }
        // c_{t-1} reaches the loss through the forget path and two peepholes
        carry = dc * cur.st1;
        bsum[0] += di;
        bsum[1] += df;
        bsum[2] += dg;
        bsum[3] += dout;
        if (peep) {
          carry += di * pi + df * pf;
          bsumh[0] += di * cp;
          bsumh[1] += df * cp;
          bsumh[2] += dout * cur.cc;
        }
      } else {
        const float dh = cur.dhv + dh_red + (has_next ? carry : 0.f);
        const float rr = cur.st0, z = cur.st1, n = cur.st2, ahn = cur.st3;
        const float hp = has_prev ? cur.cprev : 0.f;
        const float dn = dh * (1.f - z);
        const float dz = dh * (hp - n);
        const float dan = dn * (1.f - n * n);
        const float dar_ = dan * ahn * rr * (1.f - rr);
        const float daz = dz * z * (1.f - z);
        const float dhn = dan * rr;
        float* dhh = U.dah + f * GH;
        publish(dhh + ej, dar_);
        publish(dhh + H + ej, daz);
        publish(dhh + 2 * H + ej, dhn);
        float* dx = U.da + f * GH;
        store_or_publish(dx + ej, dar_, pub_dax);
        store_or_publish(dx + H + ej, daz, pub_dax);
        store_or_publish(dx + 2 * H + ej, dan, pub_dax);
        carry = dh * z;
        bsum[0] += dar_;
        bsum[1] += daz;
        bsum[2] += dan;
        bsumh[0] += dar_;
        bsumh[1] += daz;
        bsumh[2] += dhn;
      }
    }
    s = nx;
    __syncthreads();  // red is rewritten by the next step
  };
  if constexpr (kAheadOps) {
    for (int k = 0; k < a.T; k += 2) {
      step(k, oa, ob);
      if (k + 1 < a.T) step(k + 1, ob, oa);
    }
  } else {
    for (int k = 0; k < a.T; ++k) step(k, oa, oa);  // fetched at the top of each step
  }
  // Bias gradients of this workgroup: sum its 16 rows in a fixed order and
  // write one partial per row group (folded over row groups afterwards).
  // Peephole gradients likewise (LSTM with peepholes): slots 4..6.
  const bool second = G == 3 || peep;
  if (epi) {
#pragma unroll
    for (int g = 0; g < G; ++g) red[g * 256 + threadIdx.x] = bsum[g];
    if (second) {
#pragma unroll
      for (int g = 0; g < 3; ++g) red[(4 + g) * 256 + threadIdx.x] = bsumh[g];
    }
  }
  __syncthreads();
  const int nsum = G + (second ? 3 : 0);
  if ((int)threadIdx.x < nsum * 16) {
    const int g = threadIdx.x >> 4, u = threadIdx.x & 15;
    const bool hi = g >= G;  // a sum of the second set
    const int slot = hi ? 4 + (g - G) : g;
    float v = 0.f;
    for (int row = 0; row < 16; ++row) v += red[slot * 256 + row * 16 + u];
    const int gate = hi ? g - G : g;
    if (hi)
      (G == 3 ? U.bias_part_h : U.peep_part)[(int64_t)rg * 3 * H + gate * H + j0 + u] = v;
    else
      U.bias_part[(int64_t)rg * GH + gate * H + j0 + u] = v;
  }
}

// Streams that may run persistent launches at the same time (>= 1).
std::atomic<int> g_concurrency{1};

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

// Co-resident workgroups a launch of `kernel` may claim (0 on error): the
// GPU's capacity for it divided among the streams that may run persistent
// launches at the same time.
int max_coresident(const void* kernel, int threads, size_t shmem) {
  int dev = 0, cus = 0, per_cu = 0;
  if (allow_lds(kernel, shmem) != hipSuccess) return 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, shmem) != hipSuccess)
    return 0;
  return cus * per_cu / g_concurrency.load();
}

// Launches a grid that must be resident all at once, as an ordinary launch:
// the grid fits in its share of the GPU (the check above), so every
// workgroup is dispatched once the work already running drains -- kernels
// of other streams that do not wait on this one.  Several streams may each
// run a persistent launch at once provided rnnbkt_set_concurrency declared
// them (each then claims at most its share).  Waits stay bounded: a launch
// whose grid could not all be resident ends with timeouts that
// rnnbkt_sync_check reports.
hipError_t resident_launch(const void* kernel, int blocks, int threads, size_t shmem, void* args,
                           hipStream_t st, bool* fits) {
  if (blocks > max_coresident(kernel, threads, shmem)) {
    *fits = false;
    return hipSuccess;
  }
  *fits = true;
  void* argv[] = {args};
  return hipLaunchKernel(kernel, dim3(blocks), dim3(threads), argv, shmem, st);
}

// Wait control of the next launch: a fresh generation (never 0, the value
// the device flag starts from) and the poll budget, RNNBKT_MAX_POLLS when set
// (0: a wait gives up at its first miss -- used to test the reporting path).
std::atomic<uint32_t> g_launch_gen{0};
WaitCtl next_wait_ctl() {
  WaitCtl w;
  do {
    w.gen = g_launch_gen.fetch_add(1) + 1;
  } while (w.gen == 0);
  w.max_polls = kMaxPolls;
  if (const char* e = getenv("RNNBKT_MAX_POLLS")) {
    char* end = nullptr;
    const unsigned long v = strtoul(e, &end, 10);
    if (end != e && v <= 0xFFFFFFFFul) w.max_polls = (uint32_t)v;
  }
  return w;
}

}  // namespace

namespace {

// Chunks per wave (a power of two) for the longer segment of nch chunks
// split over 4 waves; 0 if above the per-lane budget.
int fwd_maxc(int nch, bool bf16) {
  const int per = (nch + 3) / 4;
  int m = 1;
  while (m < per) m *= 2;
  // 24 fp32 chunks (H = 384) take six slots, none left empty: gru2's forward
  // launches 1.68 -> 1.58 ms.
  if (!bf16 && per == 6) m = 6;
  return m <= (bf16 ? 8 : 16) ? m : 0;
}

// mr: the recurrent segment's slots, maxc or (an input segment twice as
// wide, complete before the launch) maxc / 2.
template <int G, bool BF16, int NT, int M>
const void* fwd_kernel_m(int mr) {
  if (mr == M) return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, M, NT, M>);
  if constexpr (M == 4 || M == 8)
    if (mr == M / 2) return reinterpret_cast<const void*>(k_fwd_persistent<G, BF16, 4, M, NT, M / 2>);
  return nullptr;
}

template <int G, bool BF16, int NT>
const void* fwd_kernel_nt(int maxc, int mr) {
  switch (maxc) {
    case 1: return fwd_kernel_m<G, BF16, NT, 1>(mr);
    case 2: return fwd_kernel_m<G, BF16, NT, 2>(mr);
    case 4: return fwd_kernel_m<G, BF16, NT, 4>(mr);
    case 8: return fwd_kernel_m<G, BF16, NT, 8>(mr);
  }
  if constexpr (!BF16) {
    if (maxc == 6) return fwd_kernel_m<G, BF16, NT, 6>(mr);
    if (maxc == 16) return fwd_kernel_m<G, BF16, NT, 16>(mr);
  }
  return nullptr;
}

const void* fwd_kernel(int cell, bool bf16, int nt, int maxc, int mr) {
  if (cell == RNNBKT_CELL_LSTM) {
    if (nt == 3) return nullptr;
    if (nt == 4) return bf16 ? fwd_kernel_nt<4, true, 4>(maxc, mr) : nullptr;
    if (bf16)
      return nt == 1 ? fwd_kernel_nt<4, true, 1>(maxc, mr)
                     : fwd_kernel_nt<4, true, 2>(maxc, mr);
    return nt == 1 ? fwd_kernel_nt<4, false, 1>(maxc, mr)
                   : fwd_kernel_nt<4, false, 2>(maxc, mr);
  }
  if (nt >= 3) return bf16 || nt == 4 ? nullptr : fwd_kernel_nt<3, false, 3>(maxc, mr);
  if (bf16)
    return nt == 1 ? fwd_kernel_nt<3, true, 1>(maxc, mr)
                   : fwd_kernel_nt<3, true, 2>(maxc, mr);
  return nt == 1 ? fwd_kernel_nt<3, false, 1>(maxc, mr)
                 : fwd_kernel_nt<3, false, 2>(maxc, mr);
}

// Workgroups of a recurrence grid of nc clusters of S (see cluster_block).
int rec_grid(int nc, int S) {
  return nc % kXcds == 0 ? nc * S : kXcds * ((nc + kXcds - 1) / kXcds) * S;
}

struct FwdPlan {
  const void* kernel;
  int nt, maxc, mr, blocks;
  size_t shmem;
};

// Column blocks per workgroup: 2 (8 units) for wide layers, else 1 (4 units).
// An fp32 GRU whose 8-unit grid has more workgroups than the GPU has CUs
// takes 3 (12 units) when H allows, a bf16 LSTM 4 (16 units): each
// workgroup then has a CU of its own (gru2: 192 workgroups instead of 288,
// 32 of them sharing a CU), and the row-group clusters are kept whole on
// one XCD (rec_grid).
FwdPlan plan_fwd(const FwdLaunch& a, int cell, bool bf16, int B) {
  FwdPlan p{};
  const int ch = bf16 ? 32 : 16;
  if (a.T > kMaxSteps || a.nunits < 1 || a.nunits > kMaxUnits || a.H % ch != 0) return p;
  int nch = 0;
  bool published = false;
  for (int q = 0; q < a.nunits; ++q) {
    const FwdUnit& u = a.u[q];
    if (u.kin < 1 || u.kin % 4 != 0 || u.in_bytes >= kNoRow || u.out_bytes >= kNoRow) return p;
    if (bf16 && (!u.hx || u.hx_bytes >= kNoRow)) return p;
    if (u.inx && (!bf16 || u.inx_bytes >= kNoRow || u.kin % ch != 0)) return p;
    nch = std::max(nch, std::max((u.kin + ch - 1) / ch, a.H / ch));
    published = published || u.in_published;
  }
  p.nt = a.H >= 256 && a.H % 8 == 0 ? 2 : 1;
  p.maxc = fwd_maxc(nch, bf16);
  if (p.maxc == 0) return p;
  // An input segment twice as wide as the recurrent one, complete before
  // the launch: the recurrent poll and products compiled for their own
  // width, and the input read through the caches (bilstm3's upper layers,
  // input 2H: 1.50 -> 1.37 ms per launch with the narrower recurrent code,
  // -> 1.23 ms with cached input reads; cached reads of a launch-complete
  // input as wide as the layer, gru2's and longtail's second layers,
  // changed nothing).
  p.mr = !published && fwd_maxc(a.H / ch, bf16) * 2 == p.maxc ? p.maxc / 2 : p.maxc;
  p.blocks = a.nunits * (a.H / (4 * p.nt)) * ((B + 15) / 16);
  p.shmem = sizeof(float) * 4 * p.nt * 256 + sizeof(int32_t) * (2 * a.T + 1);
  size_t out_lds = 0;
  if (a.out_blocks > 0) {
    out_lds = output_stream_lds(a.out.C, a.out.Htop);
    if (bf16 || out_lds == 0) return p;
    p.blocks += a.out_blocks;
    p.shmem = std::max(p.shmem, out_lds);
  }
  p.kernel = fwd_kernel(cell, bf16, p.nt, p.maxc, p.mr);
  // Wider workgroups: 12 units for an fp32 GRU, 16 for a bf16 LSTM.
  const int wide = cell == RNNBKT_CELL_GRU ? (bf16 ? 0 : 3) : (bf16 ? 4 : 0);
  if (wide > 0 && p.nt == 2 && a.H % (4 * wide) == 0 && p.blocks > cu_count()) {
    const void* kw = fwd_kernel(cell, bf16, wide, p.maxc, p.mr);
    const int bw = rec_grid(a.nunits * ((B + 15) / 16), a.H / (4 * wide)) + a.out_blocks;
    const size_t shw =
        std::max(sizeof(float) * 4 * wide * 256 + sizeof(int32_t) * (2 * a.T + 1), out_lds);
    if (kw && bw <= max_coresident(kw, 256, shw)) {
      p.nt = wide;
      p.blocks = bw;
      p.shmem = shw;
      p.kernel = kw;
    }
  }
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
  a.wait = next_wait_ctl();
  return resident_launch(p.kernel, p.blocks, 256, p.shmem, &a, st, fits);
}

namespace {

// Chunks per wave a workgroup of nw waves holds in registers without
// spilling (512, 256 and 128 VGPRs per lane at 1, 2 and 4 waves per SIMD),
// and the largest instantiated (16 waves may spill for very wide layers).
constexpr int bwd_maxc_fit(int nw, bool bf16) {
  return (nw == 4 ? 16 : nw == 8 ? 8 : 4) / (bf16 ? 2 : 1);
}
constexpr int bwd_maxc_cap(int nw, bool bf16) {
  return nw == 16 ? (bf16 ? 8 : 16) : bwd_maxc_fit(nw, bf16);
}

template <int G, bool BF16, int NW, int M, bool SP, bool UP>
const void* bwd_kernel_m() {
  if constexpr (M <= bwd_maxc_cap(NW, BF16) && (!SP || NW >= 8) && (SP || NW != 8) &&
                (M != 5 || (NW == 16 && !SP)))
    return reinterpret_cast<const void*>(k_bwd_persistent<G, BF16, NW, M, SP, UP>);
  return nullptr;
}

template <int G, bool BF16, int NW, bool SP, bool UP>
const void* bwd_kernel_nw(int maxc) {
  switch (maxc) {
    case 1: return bwd_kernel_m<G, BF16, NW, 1, SP, UP>();
    case 2: return bwd_kernel_m<G, BF16, NW, 2, SP, UP>();
    case 3: return bwd_kernel_m<G, BF16, NW, 3, SP, UP>();
    case 4: return bwd_kernel_m<G, BF16, NW, 4, SP, UP>();
    case 5: return bwd_kernel_m<G, BF16, NW, 5, SP, UP>();
    case 8: return bwd_kernel_m<G, BF16, NW, 8, SP, UP>();
    case 16: return bwd_kernel_m<G, BF16, NW, 16, SP, UP>();
  }
  return nullptr;
}

template <int G, bool BF16, bool UP>
const void* bwd_kernel_g(int nw, int maxc, bool split) {
  switch (nw) {
    case 4: return split ? nullptr : bwd_kernel_nw<G, BF16, 4, false, UP>(maxc);
    case 8: return split ? bwd_kernel_nw<G, BF16, 8, true, UP>(maxc) : nullptr;
    case 16:
      return split ? bwd_kernel_nw<G, BF16, 16, true, UP>(maxc)
                   : bwd_kernel_nw<G, BF16, 16, false, UP>(maxc);
  }
  return nullptr;
}

const void* bwd_kernel(int cell, bool bf16, int nw, int maxc, bool split, bool up) {
  if (up) {
    if (cell == RNNBKT_CELL_LSTM)
      return bf16 ? bwd_kernel_g<4, true, true>(nw, maxc, split)
                  : bwd_kernel_g<4, false, true>(nw, maxc, split);
    return bf16 ? bwd_kernel_g<3, true, true>(nw, maxc, split)
                : bwd_kernel_g<3, false, true>(nw, maxc, split);
  }
  if (cell == RNNBKT_CELL_LSTM)
    return bf16 ? bwd_kernel_g<4, true, false>(nw, maxc, split)
                : bwd_kernel_g<4, false, false>(nw, maxc, split);
  return bf16 ? bwd_kernel_g<3, true, false>(nw, maxc, split)
              : bwd_kernel_g<3, false, false>(nw, maxc, split);
}

struct BwdPlan {
  const void* kernel;
  int nw, maxc, blocks, wg_blocks;
  bool split;
  size_t shmem;
};

// Waves per workgroup and slots per wave: each slot is a serial MFMA group
// on the step's critical path, and gate-gradient waves that also poll delay
// their polls behind their HBM operand loads (worth about 1.5 slots on
// lstm2); more waves cost a little in the barriers.  The cheapest candidate
// that fits in registers without spilling wins.
BwdPlan plan_bwd(const BwdLaunch& a, int cell, bool bf16, int B) {
  BwdPlan p{nullptr, 0, 0, 0, 0, false, 0};
  const int ch = bf16 ? 32 : 16;
  const int G = cell == RNNBKT_CELL_LSTM ? 4 : 3;
  if (a.T > kMaxSteps || a.nunits < 1 || a.nunits > kMaxUnits || a.H % kBwdUnits != 0) return p;
  if ((G * a.H) % ch != 0) return p;
  int nch = 0;
  bool up = false;
  for (int q = 0; q < a.nunits; ++q) {
    const BwdUnit& u = a.u[q];
    if (u.rec_bytes >= kNoRow || (u.up && (u.k_up % ch != 0 || u.up_bytes >= kNoRow))) return p;
    nch = std::max(nch, std::max(u.up ? u.k_up / ch : 0, G * a.H / ch));
    up = up || u.up != nullptr;
  }
  // A candidate fits when its compiled kernel needs no scratch (a bf16
  // LSTM's packed gate gradients take half the registers of fp32 ones, so
  // its launches with an input segment fit more slots than the others).
  auto fits_regs = [&](int nw, int m, bool split) {
    const void* k = bwd_kernel(cell, bf16, nw, m, split, up);
    hipFuncAttributes fa{};
    return k && hipFuncGetAttributes(&fa, k) == hipSuccess && fa.localSizeBytes == 0;
  };
  struct Cand {
    int nw;
    bool split;
  };
  float best = 1e30f;
  for (const Cand c : {Cand{4, false}, Cand{8, true}, Cand{16, true}, Cand{16, false}}) {
    const int nmma = c.split ? c.nw - kEpiWaves : c.nw;  // waves that poll and multiply
    const int per = (nch + nmma - 1) / nmma;
    // Slots per wave: 1, 2, 3 or a power of two.  (Six for gru2's 72 chunks
    // over 12 multiplying waves, instead of eight, made its backward slower:
    // 1.77 against 1.73 ms per launch.)
    int m = 1;
    while (m < per) m = m == 2 && per == 3 ? 3 : m * 2;
    if (!fits_regs(c.nw, m, c.split)) continue;
    // Without the split the gate-gradient loads delay the polls: worth 1.5
    // fp32 chunks (four MFMAs each) but only 0.4 bf16 chunks (one MFMA each;
    // bilstm3's backward: 1.95 against 1.99 ms per batch unsplit, 2 chunks).
    const float unsplit = bf16 ? 0.4f : 1.5f;
    const float cost =
        m + (c.split ? 0.f : unsplit) + (c.nw == 16 ? 0.5f : c.nw == 8 ? 0.25f : 0.f);
    if (cost < best) {
      best = cost;
      p.nw = c.nw;
      p.maxc = m;
      p.split = c.split;
    }
  }
  if (p.nw == 0 && !up) {
    // Very wide layers: 16 polling waves with spilled registers (5 slots
    // spill far less than 8, e.g. for 72 chunks).  Not for a launch with an
    // input segment: the caller then runs the layers in launches of their
    // own, with the gradient between them from a GEMM (gru2's small batches,
    // whose two layers would otherwise share a launch with 12 VGPRs spilled).
    const int per = (nch + 15) / 16;
    int m = per == 5 ? 5 : 1;
    while (m < per) m *= 2;
    if (m <= bwd_maxc_cap(16, bf16)) {
      p.nw = 16;
      p.maxc = m;
      p.split = false;
    }
  }
  if (p.nw == 0) return p;
  const int nc = a.nunits * ((B + 15) / 16);
  p.blocks = G == 3 ? rec_grid(nc, a.H / kBwdUnits) : nc * (a.H / kBwdUnits);
  p.shmem = sizeof(float) * std::max(p.nw, 8) * 256 + sizeof(int32_t) * (2 * a.T + 1);
  p.wg_blocks = 0;
  if (a.wg_on) {
    if (bf16 || G != 4 || a.wg.tiles < 1 || a.wg.reps < 1) return p;
    const int subs = p.nw / 4;
    p.wg_blocks = (a.wg.tiles + subs - 1) / subs * a.wg.reps;
    p.blocks += p.wg_blocks;
    p.shmem = std::max(p.shmem, subs * kWgSubLds);
  }
  p.kernel = bwd_kernel(cell, bf16, p.nw, p.maxc, p.split, up);
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
  a.wg_blocks = p.wg_blocks;
  const int per_unit = a.slices * a.rgroups;
  for (int q = 0; q < a.nunits; ++q) a.u[q].wg_begin = q * per_unit;
  a.wait = next_wait_ctl();
  return resident_launch(p.kernel, p.blocks, 64 * p.nw, p.shmem, &a, st, fits);
}

size_t output_stream_lds(int32_t C, int32_t Htop) {
  if (C % 4 != 0 || Htop % 16 != 0) return 0;
  const size_t b =
      sizeof(float) * ((size_t)(C + kOutRows) * (Htop + 1) + (size_t)kOutRows * (C + 1) + 4);
  return b <= kOutLdsMax ? b : 0;
}

int cu_count() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  return cus;
}


void set_concurrency(int streams) { g_concurrency.store(streams); }
int concurrency() { return g_concurrency.load(); }

hipError_t read_wait_timeouts(unsigned* count) {
  return hipMemcpyFromSymbol(count, HIP_SYMBOL(g_wait_timeouts), sizeof(unsigned), 0,
                             hipMemcpyDeviceToHost);
}

hipError_t reset_wait_timeouts() {
  const unsigned zero = 0;
  return hipMemcpyToSymbol(HIP_SYMBOL(g_wait_timeouts), &zero, sizeof(unsigned), 0,
                           hipMemcpyHostToDevice);
}

}  // namespace rnnbkt
