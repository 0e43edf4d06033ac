// Dense contractions of the training step on the gfx950 matrix cores:
// input projection of all frames (X W_ih^T), output layer (H W_out^T), and
// the backward products (dZ W_out, dA W_ih, and the weight gradients
// dA^T X, dA^T H_prev, dZ^T H, reduced over all valid frames).
//
// Tile 64 x 64 x 32 per 256-thread workgroup (4 wave64s in a 2 x 2 grid,
// each wave owning a 32 x 32 block = 2 x 2 MFMA 16x16 tiles).  Operands are
// staged through LDS with K contiguous per row, so every lane feeds the
// matrix core from one 16-byte LDS read per MFMA group.  fp32 uses
// v_mfma_f32_16x16x4_f32; bf16 rounds to nearest-even when writing LDS and
// uses v_mfma_f32_16x16x32_bf16, always accumulating in fp32.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace rnnbkt {

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf4 __attribute__((ext_vector_type(4)));

constexpr int BM = 64, BN = 64, BK = 32;
constexpr int PAD32 = 4;   // fp32 LDS row padding (floats)
constexpr int PAD16 = 8;   // bf16 LDS row padding (elements)

template <bool BF16>
struct Lds;
template <>
struct Lds<false> {
  using T = float;
  static constexpr int LD = BK + PAD32;
};
template <>
struct Lds<true> {
  using T = __bf16;
  static constexpr int LD = BK + PAD16;
};

template <bool BF16>
__device__ inline void store4(typename Lds<BF16>::T* dst, f4 v) {
  if constexpr (BF16) {
    bf4 b = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
    *reinterpret_cast<bf4*>(dst) = b;
  } else {
    *reinterpret_cast<f4*>(dst) = v;
  }
}

template <bool BF16>
__device__ inline void store1(typename Lds<BF16>::T* dst, float v) {
  if constexpr (BF16) {
    *dst = (__bf16)v;
  } else {
    *dst = v;
  }
}

// Loads the BM x BK tile of an operand whose element (row r, k) lives at
// P[r*ld + k] (K contiguous) into S[r][k].
template <bool BF16>
__device__ inline void load_kcontig(typename Lds<BF16>::T* S, const float* P, int64_t ld,
                                    int r0, int rlim, int k0, int klim) {
  constexpr int LD = Lds<BF16>::LD;
  const int tid = threadIdx.x;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int idx = tid + rep * 256;
    const int r = idx >> 3;
    const int kq = (idx & 7) * 4;
    f4 v = {0.f, 0.f, 0.f, 0.f};
    if (r0 + r < rlim && k0 + kq < klim)
      v = *reinterpret_cast<const f4*>(P + (int64_t)(r0 + r) * ld + k0 + kq);
    store4<BF16>(S + r * LD + kq, v);
  }
}

// Loads the BK x BM tile of an operand whose element (row r, k) lives at
// P[row(k)*ld + r] (rows contiguous) into S[r][k] (transposed on the way).
template <bool BF16>
__device__ inline void load_rcontig(typename Lds<BF16>::T* S, const float* P, int64_t ld,
                                    const int32_t* gather, int r0, int rlim, int k0,
                                    int klim) {
  constexpr int LD = Lds<BF16>::LD;
  const int tid = threadIdx.x;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int idx = tid + rep * 256;
    const int k = idx >> 4;
    const int rq = (idx & 15) * 4;
    f4 v = {0.f, 0.f, 0.f, 0.f};
    if (r0 + rq < rlim && k0 + k < klim) {
      int64_t row = k0 + k;
      if (gather) row = gather[row];
      if (row >= 0) v = *reinterpret_cast<const f4*>(P + row * ld + r0 + rq);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) store1<BF16>(S + (rq + e) * LD + k, v[e]);
  }
}

template <bool A_KC, bool B_KC, bool BF16>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g) {
  using T = typename Lds<BF16>::T;
  constexpr int LD = Lds<BF16>::LD;
  __shared__ __attribute__((aligned(16))) T As[BM * LD];
  __shared__ __attribute__((aligned(16))) T Bs[BN * LD];

  const int m0 = blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int split = blockIdx.z;
  const int kbeg = split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * 32;
  const int wn = (wave & 1) * 32;
  const int lr = lane & 15;  // row of the A fragment / column of the B fragment
  const int lq = lane >> 4;  // k group of the fragment

  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    if constexpr (A_KC)
      load_kcontig<BF16>(As, g.A, g.lda, m0, g.M, k0, kend);
    else
      load_rcontig<BF16>(As, g.A, g.lda, nullptr, m0, g.M, k0, kend);
    if constexpr (B_KC)
      load_kcontig<BF16>(Bs, g.B, g.ldb, n0, g.N, k0, kend);
    else
      load_rcontig<BF16>(Bs, g.B, g.ldb, g.gather_b, n0, g.N, k0, kend);
    __syncthreads();
    if constexpr (BF16) {
      const int kk = lq * 8;
      bf8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const bf8*>(As + (wm + i * 16 + lr) * LD + kk);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const bf8*>(Bs + (wn + j * 16 + lr) * LD + kk);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    } else {
#pragma unroll
      for (int kc = 0; kc < BK; kc += 16) {
        const int kk = kc + lq * 4;
        f4 a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
          a[i] = *reinterpret_cast<const f4*>(As + (wm + i * 16 + lr) * LD + kk);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          b[j] = *reinterpret_cast<const f4*>(Bs + (wn + j * 16 + lr) * LD + kk);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
              acc[i][j] =
                  __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // Accumulator layout of a 16x16 MFMA tile: lane holds column (lane & 15),
  // rows 4*(lane >> 4) + r for r = 0..3.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn + j * 16 + lr;
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + i * 16 + lq * 4 + r;
        if (m >= g.M) continue;
        float v = acc[i][j][r];
        if (g.splits > 1) {
          g.partial[((int64_t)split * g.M + m) * g.N + n] = v;
        } else {
          if (g.bias) v += g.bias[n];
          float* c = g.C + (int64_t)m * g.ldc + n;
          if (g.accumulate) v += *c;
          *c = v;
        }
      }
    }
}

// fp32 C = A^T B with both operands K-outer (A element (m, k) at
// A[k*lda + m], B element (k, n) at B[row(k)*ldb + n]): the weight-gradient
// products, reduced over all valid frames.  Tiles are staged untransposed
// ([k][m] and [k][n], float4 stores, rows padded by 16 floats so the four
// k-rows a wave reads sit in different banks), which is the order
// v_mfma_f32_16x16x4_f32 wants: lane (row r, group q) feeds element
// (m0 + r, k0 + q) -- one float per lane per MFMA.  K-tiles are double
// buffered: the next tile's global loads are in flight during this tile's
// MFMAs.
constexpr int TN_LD = BM + 16;

__device__ inline void tn_load(f4 (&v)[2], const float* P, int64_t ld, const int32_t* gather,
                               int c0, int clim, int k0, int klim) {
  const int tid = threadIdx.x;
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

__device__ inline void tn_store(float* S, const f4 (&v)[2]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int k = (tid >> 4) + rep * 16;
    const int c = (tid & 15) * 4;
    *reinterpret_cast<f4*>(S + k * TN_LD + c) = v[rep];
  }
}

__global__ __launch_bounds__(256) void k_gemm_tn_f32(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) float As[2][BK * TN_LD];
  __shared__ __attribute__((aligned(16))) float Bs[2][BK * TN_LD];
  const int m0 = blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int split = blockIdx.z;
  const int kbeg = split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * 32;
  const int wn = (wave & 1) * 32;
  const int lr = lane & 15;
  const int lq = lane >> 4;

  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  f4 ra[2], rb[2];
  tn_load(ra, g.A, g.lda, nullptr, m0, g.M, kbeg, kend);
  tn_load(rb, g.B, g.ldb, g.gather_b, n0, g.N, kbeg, kend);
  int buf = 0;
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    tn_store(As[buf], ra);
    tn_store(Bs[buf], rb);
    __syncthreads();
    if (k0 + BK < kend) {
      tn_load(ra, g.A, g.lda, nullptr, m0, g.M, k0 + BK, kend);
      tn_load(rb, g.B, g.ldb, g.gather_b, n0, g.N, k0 + BK, kend);
    }
    const float* a_s = As[buf];
    const float* b_s = Bs[buf];
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      const int kr = (kk + lq) * TN_LD;
      float a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = a_s[kr + wm + i * 16 + lr];
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = b_s[kr + wn + j * 16 + lr];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    buf ^= 1;
  }

#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn + j * 16 + lr;
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + i * 16 + lq * 4 + r;
        if (m >= g.M) continue;
        float v = acc[i][j][r];
        if (g.splits > 1) {
          g.partial[((int64_t)split * g.M + m) * g.N + n] = v;
        } else {
          if (g.bias) v += g.bias[n];
          float* c = g.C + (int64_t)m * g.ldc + n;
          if (g.accumulate) v += *c;
          *c = v;
        }
      }
    }
}

__global__ void k_splitk_reduce(const float* __restrict__ partial, int S, int M, int N,
                                float* __restrict__ out, int64_t ldc,
                                const float* __restrict__ bias, int accumulate) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t MN = (int64_t)M * N;
  if (idx >= MN) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  // Four independent partial sums keep several loads in flight; the folding
  // order is fixed, so the result is deterministic.
  float v0 = 0.f, v1 = 0.f, v2 = 0.f, v3 = 0.f;
  int s = 0;
  for (; s + 4 <= S; s += 4) {
    v0 += partial[(int64_t)s * MN + idx];
    v1 += partial[(int64_t)(s + 1) * MN + idx];
    v2 += partial[(int64_t)(s + 2) * MN + idx];
    v3 += partial[(int64_t)(s + 3) * MN + idx];
  }
  for (; s < S; ++s) v0 += partial[(int64_t)s * MN + idx];
  float v = (v0 + v1) + (v2 + v3);
  if (bias) v += bias[n];
  float* c = out + (int64_t)m * ldc + n;
  if (accumulate) v += *c;
  *c = v;
}

struct FoldArgs {
  FoldJob job[kFoldJobs];
  int64_t first[kFoldJobs + 1];  // first element of each job, then the total
  int32_t njobs;
};

// One thread per output element of the job its index falls in; the partials
// are folded in the order of k_splitk_reduce.
__global__ void k_splitk_reduce_multi(FoldArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= a.first[a.njobs]) return;
  int q = 0;
  while (q + 1 < a.njobs && idx >= a.first[q + 1]) ++q;
  FoldJob j = a.job[0];
  for (int r = 1; r < kFoldJobs; ++r)
    if (r == q) j = a.job[r];
  const int64_t e = idx - a.first[q];
  const int64_t MN = (int64_t)j.M * j.N;
  const int m = (int)(e / j.N), n = (int)(e % j.N);
  float v0 = 0.f, v1 = 0.f, v2 = 0.f, v3 = 0.f;
  int s = 0;
  for (; s + 4 <= j.S; s += 4) {
    v0 += j.partial[(int64_t)s * MN + e];
    v1 += j.partial[(int64_t)(s + 1) * MN + e];
    v2 += j.partial[(int64_t)(s + 2) * MN + e];
    v3 += j.partial[(int64_t)(s + 3) * MN + e];
  }
  for (; s < j.S; ++s) v0 += j.partial[(int64_t)s * MN + e];
  j.out[(int64_t)m * j.ldc + n] = (v0 + v1) + (v2 + v3);
}

__global__ void k_colsum_partial(const float* __restrict__ A, int64_t rows, int cols,
                                 int64_t lda, int64_t rows_per_split,
                                 float* __restrict__ partial) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  const int s = blockIdx.y;
  if (c >= cols) return;
  const int64_t r0 = (int64_t)s * rows_per_split;
  const int64_t r1 = min(rows, r0 + rows_per_split);
  float v0 = 0.f, v1 = 0.f, v2 = 0.f, v3 = 0.f;
  int64_t r = r0;
  for (; r + 4 <= r1; r += 4) {
    v0 += A[r * lda + c];
    v1 += A[(r + 1) * lda + c];
    v2 += A[(r + 2) * lda + c];
    v3 += A[(r + 3) * lda + c];
  }
  for (; r < r1; ++r) v0 += A[r * lda + c];
  partial[(int64_t)s * cols + c] = (v0 + v1) + (v2 + v3);
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, bool a_kc, bool b_kc, bool bf16, hipStream_t st) {
  dim3 grid((g.M + BM - 1) / BM, (g.N + BN - 1) / BN, g.splits > 1 ? g.splits : 1);
  dim3 block(256);
#define RNNBKT_GEMM_CASE(AK, BKC, BF)                                      \
  if (a_kc == AK && b_kc == BKC && bf16 == BF) {                           \
    hipLaunchKernelGGL((k_gemm<AK, BKC, BF>), grid, block, 0, st, g);     \
    return hipGetLastError();                                              \
  }
  RNNBKT_GEMM_CASE(true, true, false)
  RNNBKT_GEMM_CASE(true, true, true)
  RNNBKT_GEMM_CASE(true, false, false)
  RNNBKT_GEMM_CASE(true, false, true)
  if (!a_kc && !b_kc && !bf16) {
    hipLaunchKernelGGL(k_gemm_tn_f32, grid, block, 0, st, g);
    return hipGetLastError();
  }
  RNNBKT_GEMM_CASE(false, false, true)
#undef RNNBKT_GEMM_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_splitk_reduce(const float* partial, int32_t S, int32_t M, int32_t N,
                                float* out, int64_t ldc, const float* bias, int32_t accumulate,
                                hipStream_t st) {
  const int64_t total = (int64_t)M * N;
  if (total == 0) return hipSuccess;
  const int threads = 256;
  hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)((total + threads - 1) / threads)),
                     dim3(threads), 0, st, partial, S, M, N, out, ldc, bias, accumulate);
  return hipGetLastError();
}

hipError_t launch_splitk_reduce_multi(const FoldJob* jobs, int32_t njobs, hipStream_t st) {
  if (njobs < 1 || njobs > kFoldJobs) return hipErrorInvalidValue;
  FoldArgs a{};
  a.njobs = njobs;
  int64_t total = 0;
  for (int q = 0; q < njobs; ++q) {
    a.job[q] = jobs[q];
    a.first[q] = total;
    total += (int64_t)jobs[q].M * jobs[q].N;
  }
  a.first[njobs] = total;
  if (total == 0) return hipSuccess;
  const int threads = 256;
  hipLaunchKernelGGL(k_splitk_reduce_multi, dim3((unsigned)((total + threads - 1) / threads)),
                     dim3(threads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_colsum(const float* A, int64_t rows, int32_t cols, int64_t lda,
                         int64_t rows_per_split, float* partial, float* out, hipStream_t st) {
  const int S = (int)((rows + rows_per_split - 1) / rows_per_split);
  const int threads = 256;
  hipLaunchKernelGGL(k_colsum_partial, dim3((cols + threads - 1) / threads, S), dim3(threads),
                     0, st, A, rows, cols, lda, rows_per_split, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_splitk_reduce(partial, S, 1, cols, out, cols, nullptr, 0, st);
}

}  // namespace rnnbkt
