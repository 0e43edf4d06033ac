// Whole-sequence recurrence of one LSTM/GRU layer (both directions) in one
// launch, forward and backward through time.
//
// A launch keeps every workgroup resident (cooperative launch) and walks
// the T steps of the batch itself; between steps the workgroups meet at a
// grid barrier (a monotonic arrival counter per launch: release on arrival,
// acquire while waiting).  Each workgroup owns a fixed block of 16 batch
// rows and a fixed slice of hidden units, so
//   - its slice of W_hh stays in LDS for the whole launch (read from HBM
//     once instead of once per step),
//   - the recurrent state of its (row, unit) pairs (c for the LSTM, h for
//     the GRU update, the dc / dh carries backward) stays in registers,
//   - per-step operands that do not depend on the barrier (the input
//     projection row, the saved gate activations) are fetched before the
//     barrier wait, so only the exchange of h (forward) or dA (backward)
//     between workgroups sits on the critical path.
// Rows that have already ended at a step do no work but still meet the
// barrier, so every workgroup arrives exactly T times.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "kernels.h"

namespace rnnbkt {

__device__ unsigned g_barrier_timeouts = 0;

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

__device__ inline float sigm(float x) { return 1.f / (1.f + __expf(-x)); }

__device__ inline bf8 to_bf8(f4 lo, f4 hi) {
  bf8 r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    r[e] = (__bf16)lo[e];
    r[e + 4] = (__bf16)hi[e];
  }
  return r;
}

// Every workgroup of the grid arrives once per call; returns when all
// `target` arrivals (cumulative over the launch) have happened.  The wait
// is bounded: after ~2^20 polls (about a second) the workgroup gives up and
// counts a timeout; once any timeout has been counted, later waits return
// at once.  The launch therefore always ends, and rnnbkt_sync_check reports
// the timeout as an error.
__device__ inline void grid_barrier(unsigned* counter, unsigned target) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    if (__hip_atomic_load(&g_barrier_timeouts, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
      unsigned spins = 0;
      while (__hip_atomic_load(counter, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins == (1u << 20)) {
          __hip_atomic_fetch_add(&g_barrier_timeouts, 1u, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
      }
    }
  }
  __syncthreads();
}

constexpr int kWaves = 4;
constexpr int kFwdUnits = 4;   // hidden units per forward workgroup (x G gates <= 16 columns)
constexpr int kBwdUnits = 16;  // hidden units per backward workgroup

template <bool BF16>
struct LdsT;
template <>
struct LdsT<false> {
  using T = float;
  static constexpr int CH = 16;  // k per MFMA group: 4 lane groups x 4
  static constexpr int PAD = 4;
};
template <>
struct LdsT<true> {
  using T = __bf16;
  static constexpr int CH = 32;  // 4 lane groups x 8
  static constexpr int PAD = 8;
};

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

template <int G, bool BF16>
__global__ __launch_bounds__(256) void k_fwd_persistent(PersistFwdArgs a) {
  using T = typename LdsT<BF16>::T;
  constexpr int CH = LdsT<BF16>::CH;
  constexpr int NC = 16;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int H = a.H;
  const int LDW = H + LdsT<BF16>::PAD;
  T* Ws = reinterpret_cast<T*>(smem);
  float* red = reinterpret_cast<float*>(smem + ((NC * LDW * sizeof(T) + 15) / 16) * 16);

  const int per_dir = a.slices * a.rgroups;
  const int d = blockIdx.x / per_dir;
  const int rem = blockIdx.x % per_dir;
  const int slice = rem % a.slices;
  const int rg = rem / a.slices;
  const int j0 = slice * kFwdUnits;
  const int r0 = rg * 16;
  const int GH = G * H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;

  // W slice: column c = g*4 + u holds row g*H + j0 + u of W_hh (zero for g >= G).
  const float* whh = a.whh[d];
  for (int i = threadIdx.x; i < NC * H; i += blockDim.x) {
    const int c = i / H, k = i % H;
    const int g = c >> 2, u = c & 3;
    const float v = g < G ? whh[(int64_t)(g * H + j0 + u) * H + k] : 0.f;
    Ws[c * LDW + k] = (T)v;
  }
  // Epilogue lanes of wave 0: row r0 + (lane >> 2), unit j0 + (lane & 3).
  const int erow = r0 + (lane >> 2);
  const int ej = j0 + (lane & 3);
  float bhh[3] = {0.f, 0.f, 0.f};
  if constexpr (G == 3) {
    if (wave == 0)
      for (int g = 0; g < 3; ++g) bhh[g] = a.bhh[d][g * H + ej];
  }
  float c_state = 0.f, h_state = 0.f;
  const float* gxd = a.gx[d];
  float* stash = a.stash[d];
  float* cst = a.cst[d];
  float* hout = a.hout + d * H;
  const unsigned nwg = gridDim.x;
  __syncthreads();

  StepIdx s = fwd_step(a.bs, a.off, a.T, d, 0);
  for (int k = 0; k < a.T; ++k) {
    const bool active = r0 < s.rows;
    // Operands that do not depend on other workgroups: the input projection
    // of this step's rows (wave 0, epilogue lanes).
    float gxv[G];
    const bool erow_on = active && wave == 0 && erow < s.rows;
    if (erow_on) {
      const float* gr = gxd + (int64_t)(s.row0 + erow) * GH;
#pragma unroll
      for (int g = 0; g < G; ++g) gxv[g] = gr[g * H + ej];
    }
    if (active) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      const int r = r0 + lr;
      const float* arow =
          r < s.prev_rows ? hout + (int64_t)(s.prev0 + r) * a.ldh : nullptr;
      const T* wrow = Ws + lr * LDW;
      const int nchunks = H / CH;
      for (int c = wave; c < nchunks; c += kWaves) {
        if constexpr (BF16) {
          const int kk = c * CH + lq * 8;
          f4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0;
          if (arow) {
            a0 = *reinterpret_cast<const f4*>(arow + kk);
            a1 = *reinterpret_cast<const f4*>(arow + kk + 4);
          }
          const bf8 w = *reinterpret_cast<const bf8*>(wrow + kk);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(to_bf8(a0, a1), w, acc, 0, 0, 0);
        } else {
          const int kk = c * CH + lq * 4;
          f4 av = {0.f, 0.f, 0.f, 0.f};
          if (arow) av = *reinterpret_cast<const f4*>(arow + kk);
          const f4 w = *reinterpret_cast<const f4*>(wrow + kk);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], w[e], acc, 0, 0, 0);
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave * 256 + (lq * 4 + q) * 16 + lr] = acc[q];
    }
    __syncthreads();
    if (erow_on) {
      const int rr = lane >> 2, u = lane & 3;
      float sg[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) v += red[w * 256 + rr * 16 + g * 4 + u];
        sg[g] = v;
      }
      const bool has_prev = erow < s.prev_rows;
      const int64_t f = s.row0 + erow;
      float* st = stash + f * 4 * H;
      if constexpr (G == 4) {
        const float ig = sigm(gxv[0] + sg[0]);
        const float fg = sigm(gxv[1] + sg[1]);
        const float gg = tanhf(gxv[2] + sg[2]);
        const float og = sigm(gxv[3] + sg[3]);
        const float cp = has_prev ? c_state : 0.f;
        c_state = fg * cp + ig * gg;
        h_state = og * tanhf(c_state);
        st[ej] = ig;
        st[H + ej] = fg;
        st[2 * H + ej] = gg;
        st[3 * H + ej] = og;
        cst[f * H + ej] = c_state;
      } else {
        const float ahr = sg[0] + bhh[0];
        const float ahz = sg[1] + bhh[1];
        const float ahn = sg[2] + bhh[2];
        const float rg_ = sigm(gxv[0] + ahr);
        const float z = sigm(gxv[1] + ahz);
        const float n = tanhf(gxv[2] + rg_ * ahn);
        const float hp = has_prev ? h_state : 0.f;
        h_state = (1.f - z) * n + z * hp;
        st[ej] = rg_;
        st[H + ej] = z;
        st[2 * H + ej] = n;
        st[3 * H + ej] = ahn;
      }
      hout[f * a.ldh + ej] = h_state;
    }
    // Next step's indices (constant tables) before the barrier wait.
    StepIdx nxt = s;
    if (k + 1 < a.T) nxt = fwd_step(a.bs, a.off, a.T, d, k + 1);
    grid_barrier(a.barrier, nwg * (unsigned)(k + 1));
    s = nxt;
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

template <int G, bool BF16>
__global__ __launch_bounds__(256) void k_bwd_persistent(PersistBwdArgs a) {
  using T = typename LdsT<BF16>::T;
  constexpr int CH = LdsT<BF16>::CH;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int H = a.H;
  const int GH = G * H;
  const int LDW = GH + LdsT<BF16>::PAD;
  T* Ws = reinterpret_cast<T*>(smem);  // Ws[u][k] = W_hh[k][j0 + u]
  float* red = reinterpret_cast<float*>(smem + ((kBwdUnits * LDW * sizeof(T) + 15) / 16) * 16);

  const int per_dir = a.slices * a.rgroups;
  const int d = blockIdx.x / per_dir;
  const int rem = blockIdx.x % per_dir;
  const int slice = rem % a.slices;
  const int rg = rem / a.slices;
  const int j0 = slice * kBwdUnits;
  const int r0 = rg * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;

  const float* whh = a.whh[d];
  for (int i = threadIdx.x; i < kBwdUnits * GH; i += blockDim.x) {
    const int k = i / kBwdUnits, u = i % kBwdUnits;
    Ws[u * LDW + k] = (T)whh[(int64_t)k * H + j0 + u];
  }
  // Epilogue: thread -> row r0 + (tid >> 4), unit j0 + (tid & 15).
  const int erow = r0 + (threadIdx.x >> 4);
  const int ej = j0 + (threadIdx.x & 15);
  float carry = 0.f;
  const float* stash = a.stash[d];
  const float* cst = a.cst[d];
  const float* hout = a.hout + d * H;
  const float* dh_in = a.dh_in + d * H;
  float* da = a.da[d];
  float* dah = a.dah[d];
  const float* da_next = G == 3 ? dah : da;
  const unsigned nwg = gridDim.x;
  __syncthreads();

  BwdIdx s = bwd_step(a.bs, a.off, a.T, d, 0);
  for (int k = 0; k < a.T; ++k) {
    const bool active = r0 < s.rows;
    const bool erow_on = active && erow < s.rows;
    // Barrier-independent operands of this step.
    float dhv = 0.f, st0 = 0.f, st1 = 0.f, st2 = 0.f, st3 = 0.f, cc = 0.f, cp = 0.f, hp = 0.f;
    int64_t f = 0;
    if (erow_on) {
      f = s.row0 + erow;
      dhv = dh_in[f * a.ldd + ej];
      const float* st = stash + f * 4 * H;
      st0 = st[ej];
      st1 = st[H + ej];
      st2 = st[2 * H + ej];
      st3 = st[3 * H + ej];
      if constexpr (G == 4) {
        cc = cst[f * H + ej];
        if (erow < s.prev_rows) cp = cst[(int64_t)(s.prev0 + erow) * H + ej];
      } else {
        if (erow < s.prev_rows) hp = hout[(int64_t)(s.prev0 + erow) * a.ldh + ej];
      }
    }
    if (active && r0 < s.next_rows) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      const int r = r0 + lr;
      const float* arow = r < s.next_rows ? da_next + (int64_t)(s.next0 + r) * GH : nullptr;
      const T* wrow = Ws + lr * LDW;
      const int nchunks = GH / CH;
      for (int c = wave; c < nchunks; c += kWaves) {
        if constexpr (BF16) {
          const int kk = c * CH + lq * 8;
          f4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0;
          if (arow) {
            a0 = *reinterpret_cast<const f4*>(arow + kk);
            a1 = *reinterpret_cast<const f4*>(arow + kk + 4);
          }
          const bf8 w = *reinterpret_cast<const bf8*>(wrow + kk);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(to_bf8(a0, a1), w, acc, 0, 0, 0);
        } else {
          const int kk = c * CH + lq * 4;
          f4 av = {0.f, 0.f, 0.f, 0.f};
          if (arow) av = *reinterpret_cast<const f4*>(arow + kk);
          const f4 w = *reinterpret_cast<const f4*>(wrow + kk);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], w[e], acc, 0, 0, 0);
        }
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave * 256 + (lq * 4 + q) * 16 + lr] = acc[q];
    } else if (active) {
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave * 256 + (lq * 4 + q) * 16 + lr] = 0.f;
    }
    __syncthreads();
    if (erow_on) {
      const bool has_next = erow < s.next_rows;
      float dh_rec = 0.f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) dh_rec += red[w * 256 + threadIdx.x];
      if constexpr (G == 4) {
        const float dh = dhv + (has_next ? dh_rec : 0.f);
        const float tc = tanhf(cc);
        const float dc = dh * st3 * (1.f - tc * tc) + (has_next ? carry : 0.f);
        float* dar = da + f * GH;
        dar[ej] = dc * st2 * st0 * (1.f - st0);
        dar[H + ej] = dc * cp * st1 * (1.f - st1);
        dar[2 * H + ej] = dc * st0 * (1.f - st2 * st2);
        dar[3 * H + ej] = dh * tc * st3 * (1.f - st3);
        carry = dc * st1;
      } else {
        const float dh = dhv + (has_next ? dh_rec + carry : 0.f);
        const float r = st0, z = st1, n = st2, ahn = st3;
        const float dn = dh * (1.f - z);
        const float dz = dh * (hp - n);
        const float dan = dn * (1.f - n * n);
        const float dar_ = dan * ahn * r * (1.f - r);
        const float daz = dz * z * (1.f - z);
        float* dx = da + f * GH;
        float* dhh = dah + f * GH;
        dx[ej] = dar_;
        dx[H + ej] = daz;
        dx[2 * H + ej] = dan;
        dhh[ej] = dar_;
        dhh[H + ej] = daz;
        dhh[2 * H + ej] = dan * r;
        carry = dh * z;
      }
    }
    BwdIdx nxt = s;
    if (k + 1 < a.T) nxt = bwd_step(a.bs, a.off, a.T, d, k + 1);
    grid_barrier(a.barrier, nwg * (unsigned)(k + 1));
    s = nxt;
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

template <typename K>
hipError_t coop_launch(K kernel, int blocks, size_t shmem, void* args, hipStream_t st) {
  void* argv[] = {args};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(kernel), dim3(blocks),
                                    dim3(256), argv, shmem, st);
}

size_t fwd_shmem(int H, bool bf16) {
  const size_t w = 16 * (size_t)(H + (bf16 ? 8 : 4)) * (bf16 ? 2 : 4);
  return (w + 15) / 16 * 16 + sizeof(float) * kWaves * 256;
}

size_t bwd_shmem(int GH, bool bf16) {
  const size_t w = kBwdUnits * (size_t)(GH + (bf16 ? 8 : 4)) * (bf16 ? 2 : 4);
  return (w + 15) / 16 * 16 + sizeof(float) * kWaves * 256;
}

template <typename K>
int max_coresident(K kernel, size_t shmem) {
  int dev = 0, cus = 0, per_cu = 0;
  if (allow_lds(reinterpret_cast<const void*>(kernel), shmem) != hipSuccess) return 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kernel),
                                                   256, shmem) != hipSuccess)
    return 0;
  return cus * per_cu;
}

}  // namespace

int persistent_fwd_blocks(int H, int B, int dirs) { return dirs * (H / kFwdUnits) * ((B + 15) / 16); }
int persistent_bwd_blocks(int H, int B, int dirs) { return dirs * (H / kBwdUnits) * ((B + 15) / 16); }

hipError_t launch_fwd_persistent(PersistFwdArgs a, int cell, bool bf16, int B, int dirs,
                                 hipStream_t st, bool* fits) {
  a.slices = a.H / kFwdUnits;
  a.rgroups = (B + 15) / 16;
  const int blocks = dirs * a.slices * a.rgroups;
  const size_t sh = fwd_shmem(a.H, bf16);
#define RNNBKT_FWD(G_, BF_)                                                           \
  {                                                                                   \
    auto kern = k_fwd_persistent<G_, BF_>;                                            \
    if (blocks > max_coresident(kern, sh)) {                                          \
      *fits = false;                                                                  \
      return hipSuccess;                                                              \
    }                                                                                 \
    *fits = true;                                                                     \
    return coop_launch(kern, blocks, sh, &a, st);                                     \
  }
  if (cell == RNNBKT_CELL_LSTM) {
    if (bf16) RNNBKT_FWD(4, true) else RNNBKT_FWD(4, false)
  } else {
    if (bf16) RNNBKT_FWD(3, true) else RNNBKT_FWD(3, false)
  }
#undef RNNBKT_FWD
}

hipError_t launch_bwd_persistent(PersistBwdArgs a, int cell, bool bf16, int B, int dirs,
                                 hipStream_t st, bool* fits) {
  a.slices = a.H / kBwdUnits;
  a.rgroups = (B + 15) / 16;
  const int G = cell == RNNBKT_CELL_LSTM ? 4 : 3;
  const int blocks = dirs * a.slices * a.rgroups;
  const size_t sh = bwd_shmem(G * a.H, bf16);
#define RNNBKT_BWD(G_, BF_)                                                           \
  {                                                                                   \
    auto kern = k_bwd_persistent<G_, BF_>;                                            \
    if (blocks > max_coresident(kern, sh)) {                                          \
      *fits = false;                                                                  \
      return hipSuccess;                                                              \
    }                                                                                 \
    *fits = true;                                                                     \
    return coop_launch(kern, blocks, sh, &a, st);                                     \
  }
  if (cell == RNNBKT_CELL_LSTM) {
    if (bf16) RNNBKT_BWD(4, true) else RNNBKT_BWD(4, false)
  } else {
    if (bf16) RNNBKT_BWD(3, true) else RNNBKT_BWD(3, false)
  }
#undef RNNBKT_BWD
}

hipError_t read_barrier_timeouts(unsigned* count) {
  return hipMemcpyFromSymbol(count, HIP_SYMBOL(g_barrier_timeouts), sizeof(unsigned), 0,
                             hipMemcpyDeviceToHost);
}

}  // namespace rnnbkt
