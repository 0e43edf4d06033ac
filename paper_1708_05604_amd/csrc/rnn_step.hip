// One recurrent time step of an LSTM or GRU layer, forward and backward,
// over the rows of the batch that are still active at that step.
//
// Forward: a_t = gx_t + h_{t-1} W_hh^T on the matrix cores, fused with the
// gate nonlinearities and the state update.  Backward: the recurrent
// gradient dA_{next} W_hh on the matrix cores, fused with the gate-gradient
// algebra of the step.
//
// Work split: one 256-thread workgroup owns a tile of 16 batch rows x 16
// hidden units (all gates of those units, so the state update stays local);
// its 4 waves split the reduction dimension and combine their 16x16
// accumulators through LDS in a fixed order.  Rows at or beyond `rows` (the
// sequences that have already ended) are neither read nor written.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace rnnbkt {

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));


__device__ inline bf8 to_bf8(f4 lo, f4 hi) {
  bf8 r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    r[e] = (__bf16)lo[e];
    r[e + 4] = (__bf16)hi[e];
  }
  return r;
}

constexpr int kWaves = 4;

// acc[g] += A(16 rows x K) . W_g(K x 16 units)^T over this wave's K chunks,
// A rows from `arow` (nullptr = zero row), W_g rows from wrow[g].
// fp32: chunks of 16 (lane group q holds k = 4q..4q+3 of the chunk);
// bf16: chunks of 32 (lane group q holds k = 8q..8q+7).
template <int NG, bool BF16>
__device__ inline void mma_rows_kcontig(f4 (&acc)[NG], const float* arow,
                                        const float* const (&wrow)[NG], int K, int wave,
                                        int lq) {
  constexpr int CH = BF16 ? 32 : 16;
  const int nchunks = K / CH;
  for (int c = wave; c < nchunks; c += kWaves) {
    if constexpr (BF16) {
      const int k = c * CH + lq * 8;
      f4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0;
      if (arow) {
        a0 = *reinterpret_cast<const f4*>(arow + k);
        a1 = *reinterpret_cast<const f4*>(arow + k + 4);
      }
      const bf8 a = to_bf8(a0, a1);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const f4 w0 = *reinterpret_cast<const f4*>(wrow[g] + k);
        const f4 w1 = *reinterpret_cast<const f4*>(wrow[g] + k + 4);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, to_bf8(w0, w1), acc[g], 0, 0, 0);
      }
    } else {
      const int k = c * CH + lq * 4;
      f4 a = {0.f, 0.f, 0.f, 0.f};
      if (arow) a = *reinterpret_cast<const f4*>(arow + k);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const f4 w = *reinterpret_cast<const f4*>(wrow[g] + k);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], w[e], acc[g], 0, 0, 0);
      }
    }
  }
}

// Forward step.  G = 4 (LSTM) or 3 (GRU).
template <int G, bool BF16>
__global__ __launch_bounds__(256) void k_step_fwd(StepFwdArgs a) {
  __shared__ float red[kWaves][G][256];
  const int H = a.H;
  const int j0 = blockIdx.x * 16;
  const int r0 = blockIdx.y * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;

  f4 acc[G];
#pragma unroll
  for (int g = 0; g < G; ++g) acc[g] = f4{0.f, 0.f, 0.f, 0.f};
  {
    const int r = r0 + lr;
    const float* arow = r < a.prev_rows ? a.hout + (int64_t)(a.prev0 + r) * a.ldh : nullptr;
    const float* wrow[G];
#pragma unroll
    for (int g = 0; g < G; ++g) wrow[g] = a.whh + (int64_t)(g * H + j0 + lr) * H;
    mma_rows_kcontig<G, BF16>(acc, arow, wrow, H, wave, lq);
  }
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][g][(lq * 4 + r) * 16 + lr] = acc[g][r];
  __syncthreads();

  const int row = r0 + (threadIdx.x >> 4);
  const int j = j0 + (threadIdx.x & 15);
  if (row >= a.rows) return;
  float s[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += red[w][g][threadIdx.x];
    s[g] = v;
  }
  const int64_t f = a.row0 + row;
  const int GH = G * H;
  const float* gx = a.gx + f * GH;
  const bool has_prev = row < a.prev_rows;
  if constexpr (G == 4) {
    const float cp = has_prev ? a.cst[(int64_t)(a.prev0 + row) * H + j] : 0.f;
    float ai = gx[j] + s[0], af = gx[H + j] + s[1], ao = gx[3 * H + j] + s[3];
    if (a.peep) {
      ai += a.peep[j] * cp;
      af += a.peep[H + j] * cp;
    }
    const float ig = act_sigmoid(ai);
    const float fg = act_sigmoid(af);
    const float gg = act_tanh(gx[2 * H + j] + s[2]);
    const float c = fg * cp + ig * gg;
    if (a.peep) ao += a.peep[2 * H + j] * c;
    const float og = act_sigmoid(ao);
    const float h = og * act_tanh(c);
    float* st = a.stash + f * 4 * H;
    st[j] = ig;
    st[H + j] = fg;
    st[2 * H + j] = gg;
    st[3 * H + j] = og;
    a.cst[f * H + j] = c;
    a.hout[f * a.ldh + j] = h;
  } else {
    const float ahr = s[0] + a.bhh[j];
    const float ahz = s[1] + a.bhh[H + j];
    const float ahn = s[2] + a.bhh[2 * H + j];
    const float r = act_sigmoid(gx[j] + ahr);
    const float z = act_sigmoid(gx[H + j] + ahz);
    const float n = act_tanh(gx[2 * H + j] + r * ahn);
    const float hp = has_prev ? a.hout[(int64_t)(a.prev0 + row) * a.ldh + j] : 0.f;
    const float h = (1.f - z) * n + z * hp;
    float* st = a.stash + f * 4 * H;
    st[j] = r;
    st[H + j] = z;
    st[2 * H + j] = n;
    st[3 * H + j] = ahn;
    a.hout[f * a.ldh + j] = h;
  }
}

// Backward step.  dh_rec = dA_next . W_hh (K = G*H, N = H) on the matrix
// cores; W_hh is read column-wise (lanes of a group read 16 consecutive
// units of one row, so the loads stay coalesced).
template <int G, bool BF16>
__global__ __launch_bounds__(256) void k_step_bwd(StepBwdArgs a) {
  __shared__ float red[kWaves][256];
  const int H = a.H;
  const int GH = G * H;
  const int j0 = blockIdx.x * 16;
  const int r0 = blockIdx.y * 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lq = lane >> 4;

  f4 acc = {0.f, 0.f, 0.f, 0.f};
  if (a.next_rows > r0) {
    const int r = r0 + lr;
    const float* arow = r < a.next_rows ? a.da_next + (int64_t)(a.next0 + r) * GH : nullptr;
    const float* wcol = a.whh + j0 + lr;
    constexpr int CH = BF16 ? 32 : 16;
    const int nchunks = GH / CH;
    for (int c = wave; c < nchunks; c += kWaves) {
      if constexpr (BF16) {
        const int k = c * CH + lq * 8;
        f4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0;
        if (arow) {
          a0 = *reinterpret_cast<const f4*>(arow + k);
          a1 = *reinterpret_cast<const f4*>(arow + k + 4);
        }
        f4 w0, w1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          w0[e] = wcol[(int64_t)(k + e) * H];
          w1[e] = wcol[(int64_t)(k + 4 + e) * H];
        }
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(to_bf8(a0, a1), to_bf8(w0, w1), acc, 0, 0,
                                                      0);
      } else {
        const int k = c * CH + lq * 4;
        f4 av = {0.f, 0.f, 0.f, 0.f};
        if (arow) av = *reinterpret_cast<const f4*>(arow + k);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], wcol[(int64_t)(k + e) * H], acc, 0,
                                                     0, 0);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) red[wave][(lq * 4 + r) * 16 + lr] = acc[r];
  __syncthreads();

  const int row = r0 + (threadIdx.x >> 4);
  const int j = j0 + (threadIdx.x & 15);
  if (row >= a.rows) return;
  float dh_rec = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) dh_rec += red[w][threadIdx.x];
  const int64_t f = a.row0 + row;
  const bool has_next = row < a.next_rows;
  const bool has_prev = row < a.prev_rows;
  const float* st = a.stash + f * 4 * H;
  float* carry = a.carry + (int64_t)row * H + j;
  if constexpr (G == 4) {
    const float dh = a.dh_in[f * a.ldd + j] + (has_next ? dh_rec : 0.f);
    const float ig = st[j], fg = st[H + j], gg = st[2 * H + j], og = st[3 * H + j];
    const float c = a.cst[f * H + j];
    const float tc = act_tanh(c);
    const float dout = dh * tc * og * (1.f - og);
    float dc = dh * og * (1.f - tc * tc) + (has_next ? *carry : 0.f);
    if (a.peep) dc += dout * a.peep[2 * H + j];
    const float cp = has_prev ? a.cst[(int64_t)(a.prev0 + row) * H + j] : 0.f;
    const float di = dc * gg * ig * (1.f - ig);
    const float df = dc * cp * fg * (1.f - fg);
    float* da = a.da + f * GH;
    da[j] = di;
    da[H + j] = df;
    da[2 * H + j] = dc * ig * (1.f - gg * gg);
    da[3 * H + j] = dout;
    float cr = dc * fg;
    if (a.peep) {
      // c_{t-1} also feeds the input and forget gates; this thread owns
      // (row, j) at every step, so the running sums need no atomics.
      cr += di * a.peep[j] + df * a.peep[H + j];
      float* acc = a.peep_acc + (int64_t)row * 3 * H + j;
      acc[0] += di * cp;
      acc[H] += df * cp;
      acc[2 * H] += dout * c;
    }
    *carry = cr;
  } else {
    const float dh = a.dh_in[f * a.ldd + j] + (has_next ? dh_rec + *carry : 0.f);
    const float r = st[j], z = st[H + j], n = st[2 * H + j], ahn = st[3 * H + j];
    const float hp = has_prev ? a.hout[(int64_t)(a.prev0 + row) * a.ldh + j] : 0.f;
    const float dn = dh * (1.f - z);
    const float dz = dh * (hp - n);
    const float dan = dn * (1.f - n * n);
    const float dar = dan * ahn * r * (1.f - r);
    const float daz = dz * z * (1.f - z);
    float* dx = a.da + f * GH;
    float* dhh = a.dah + f * GH;
    dx[j] = dar;
    dx[H + j] = daz;
    dx[2 * H + j] = dan;
    dhh[j] = dar;
    dhh[H + j] = daz;
    dhh[2 * H + j] = dan * r;
    *carry = dh * z;
  }
}

}  // namespace

hipError_t launch_step_fwd(const StepFwdArgs& a, int cell, bool bf16, hipStream_t st) {
  dim3 grid(a.H / 16, (a.rows + 15) / 16);
  dim3 block(256);
  if (cell == RNNBKT_CELL_LSTM) {
    if (bf16)
      hipLaunchKernelGGL((k_step_fwd<4, true>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((k_step_fwd<4, false>), grid, block, 0, st, a);
  } else {
    if (bf16)
      hipLaunchKernelGGL((k_step_fwd<3, true>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((k_step_fwd<3, false>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_step_bwd(const StepBwdArgs& a, int cell, bool bf16, hipStream_t st) {
  dim3 grid(a.H / 16, (a.rows + 15) / 16);
  dim3 block(256);
  if (cell == RNNBKT_CELL_LSTM) {
    if (bf16)
      hipLaunchKernelGGL((k_step_bwd<4, true>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((k_step_bwd<4, false>), grid, block, 0, st, a);
  } else {
    if (bf16)
      hipLaunchKernelGGL((k_step_bwd<3, true>), grid, block, 0, st, a);
    else
      hipLaunchKernelGGL((k_step_bwd<3, false>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace rnnbkt
