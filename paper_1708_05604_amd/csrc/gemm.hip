// Dense contractions of the training step on the gfx950 matrix cores:
// input projection of all frames (X W_ih^T), output layer (H W_out^T), and
// the backward products (dZ W_out, dA W_ih, and the weight gradients
// dA^T X, dA^T H_prev, dZ^T H, reduced over all valid frames).
//
// fp32: tile 64 x 64 x 32 per 256-thread workgroup (4 wave64s in a 2 x 2
// grid, each wave owning a 32 x 32 block = 2 x 2 MFMA 16x16 tiles) on
// v_mfma_f32_16x16x4_f32.  Operands are staged through LDS with K contiguous
// per row, so every lane feeds the matrix core from one 16-byte LDS read per
// MFMA group.
//
// bf16 (k_gemm_bf16): tile 128 x 128 x 32 per 256-thread workgroup, each
// wave owning 64 x 64 = 4 x 4 tiles of v_mfma_f32_16x16x32_bf16 with fp32
// accumulators.  fp32 operands are rounded to bf16 (nearest-even) between
// their 16-byte global loads and LDS, where both operands sit as [row][k]
// bf16 (K-tiles double buffered, one barrier per K-tile); an operand stored
// K-outer in memory is transposed in registers on the way (each thread
// loads four k-rows of four columns and writes four 4-k pieces), with the
// 16-byte chunks of each LDS row permuted so that those stores spread over
// the banks.  Workgroups are renumbered so that the ones sharing an A row
// block run on one XCD.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace rnnbkt {

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int BM = 64, BN = 64, BK = 32;
constexpr int LD32 = BK + 4;  // fp32 LDS row (floats), padded

// Loads the BM x BK tile of an operand whose element (row r, k) lives at
// P[r*ld + k] (K contiguous) into S[r][k].
__device__ inline void load_kcontig(float* S, const float* P, int64_t ld, int r0, int rlim,
                                    int k0, int klim) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int rep = 0; rep < 2; ++rep) {
    const int idx = tid + rep * 256;
    const int r = idx >> 3;
    const int kq = (idx & 7) * 4;
    f4 v = {0.f, 0.f, 0.f, 0.f};
    if (r0 + r < rlim && k0 + kq < klim)
      v = *reinterpret_cast<const f4*>(P + (int64_t)(r0 + r) * ld + k0 + kq);
    *reinterpret_cast<f4*>(S + r * LD32 + kq) = v;
  }
}

// Loads the BK x BM tile of an operand whose element (row r, k) lives at
// P[row(k)*ld + r] (rows contiguous) into S[r][k] (transposed on the way).
__device__ inline void load_rcontig(float* S, const float* P, int64_t ld, const int32_t* gather,
                                    int r0, int rlim, int k0, int klim) {
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
    for (int e = 0; e < 4; ++e) S[(rq + e) * LD32 + k] = v[e];
  }
}

// fp32 C = op(A) op(B) with A K-contiguous (B either way).
template <bool A_KC, bool B_KC>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) float As[BM * LD32];
  __shared__ __attribute__((aligned(16))) float Bs[BN * LD32];

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
      load_kcontig(As, g.A, g.lda, m0, g.M, k0, kend);
    else
      load_rcontig(As, g.A, g.lda, nullptr, m0, g.M, k0, kend);
    if constexpr (B_KC)
      load_kcontig(Bs, g.B, g.ldb, n0, g.N, k0, kend);
    else
      load_rcontig(Bs, g.B, g.ldb, g.gather_b, n0, g.N, k0, kend);
    __syncthreads();
#pragma unroll
    for (int kc = 0; kc < BK; kc += 16) {
      const int kk = kc + lq * 4;
      f4 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const f4*>(As + (wm + i * 16 + lr) * LD32 + kk);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const f4*>(Bs + (wn + j * 16 + lr) * LD32 + kk);
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][e], b[j][e], acc[i][j], 0, 0, 0);
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

// ---------------------------------------------------------------- bf16
constexpr int TBM = 128, TBK = 32;
constexpr int TB_LD = TBK + 8;  // bf16 per LDS row: 80 bytes, so the 16-byte
                                // reads of 16 consecutive rows hit distinct banks
typedef __bf16 bf4v __attribute__((ext_vector_type(4)));

__device__ inline bf4v to_bf4(float a, float b, float c, float d) {
  return bf4v{(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
}

// LDS element offset of (row, k) in a K-tile: the four 16-byte chunks of a
// row are permuted by (row / 4) mod 4, so that the 8-byte stores of
// transposed operands (consecutive threads four rows apart) spread over the
// banks; the 16-byte fragment reads stay whole.
__device__ inline int tb_off(int row, int k) {
  return row * TB_LD + ((((k >> 3) ^ (row >> 2)) & 3) << 3) + (k & 7);
}

// One operand's K-tile of 128 rows x 32 k in registers, as loaded (fp32).
struct TileRegs {
  f4 v[4];
};

// Element (r, k) of an operand: KC at P[r*ld + k], else at P[row(k)*ld + r]
// with row(k) = gather ? gather[k] : k (negative = a zero row).
// KC: thread t loads rows (t >> 3) + 32 i, k = 4 (t & 7) .. + 3.
// RC: thread t loads k-rows 4 (t >> 5) + i, columns 4 (t & 31) .. + 3.
template <bool KC>
__device__ inline void tb_fetch(TileRegs& R, const float* P, int64_t ld, const int32_t* gather,
                                int r0, int rlim, int k0, int klim, int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f4 x = {0.f, 0.f, 0.f, 0.f};
    if constexpr (KC) {
      const int r = (tid >> 3) + 32 * i, k = k0 + (tid & 7) * 4;
      if (r0 + r < rlim) {
        const float* q = P + (int64_t)(r0 + r) * ld + k;
        if (k + 4 <= klim) {
          x = *reinterpret_cast<const f4*>(q);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (k + e < klim) x[e] = q[e];
        }
      }
    } else {
      const int k = k0 + 4 * (tid >> 5) + i, r = r0 + 4 * (tid & 31);
      if (k < klim && r < rlim) {
        int64_t row = k;
        if (gather) row = gather[k];
        if (row >= 0) {
          const float* q = P + row * ld + r;
          if (r + 4 <= rlim) {
            x = *reinterpret_cast<const f4*>(q);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (r + e < rlim) x[e] = q[e];
          }
        }
      }
    }
    R.v[i] = x;
  }
}

// An operand held as bf16 (the packed gate gradients of a bf16 LSTM): the
// same elements as tb_fetch, half the bytes, kept as loaded (two bf16 per
// word) until tb_store_bf16 writes them to LDS unchanged.  Widening them at
// fetch time made the loads complete before the stage's MFMAs (dX and
// weight-gradient products 1.4x slower).
struct TileRegsBf {
  uint2 v[4];
};

template <bool KC>
__device__ inline void tb_fetch_bf16(TileRegsBf& R, const float* Pf, int64_t ld, int r0, int rlim,
                                     int k0, int klim, int tid) {
  const unsigned short* P = reinterpret_cast<const unsigned short*>(Pf);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint2 x = {0u, 0u};
    if constexpr (KC) {
      const int r = (tid >> 3) + 32 * i, k = k0 + (tid & 7) * 4;
      if (r0 + r < rlim) {
        const unsigned short* q = P + (int64_t)(r0 + r) * ld + k;
        if (k + 4 <= klim) {
          x = *reinterpret_cast<const uint2*>(q);
        } else {
          unsigned h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (k + e < klim) h[e] = q[e];
          x = uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
        }
      }
    } else {
      const int k = k0 + 4 * (tid >> 5) + i, r = r0 + 4 * (tid & 31);
      if (k < klim && r < rlim) {
        const unsigned short* q = P + (int64_t)k * ld + r;
        if (r + 4 <= rlim) {
          x = *reinterpret_cast<const uint2*>(q);
        } else {
          unsigned h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (r + e < rlim) h[e] = q[e];
          x = uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
        }
      }
    }
    R.v[i] = x;
  }
}

// tb_store for TileRegsBf: KC rows go to LDS as loaded; otherwise element e
// of the four k-rows is gathered into row r + e (a transpose of bf16 halves).
template <bool KC>
__device__ inline void tb_store_bf16(__bf16* S, const TileRegsBf& R, int tid) {
  if constexpr (KC) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (tid >> 3) + 32 * i, k = (tid & 7) * 4;
      *reinterpret_cast<uint2*>(S + tb_off(r, k)) = R.v[i];
    }
  } else {
    const int k = 4 * (tid >> 5), r = 4 * (tid & 31);
    const unsigned w[2][4] = {{R.v[0].x, R.v[1].x, R.v[2].x, R.v[3].x},
                              {R.v[0].y, R.v[1].y, R.v[2].y, R.v[3].y}};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const unsigned* c = w[e >> 1];
      const uint2 o = (e & 1) == 0
                          ? uint2{(c[0] & 0xFFFFu) | (c[1] << 16), (c[2] & 0xFFFFu) | (c[3] << 16)}
                          : uint2{(c[0] >> 16) | (c[1] & 0xFFFF0000u),
                                  (c[2] >> 16) | (c[3] & 0xFFFF0000u)};
      *reinterpret_cast<uint2*>(S + tb_off(r + e, k)) = o;
    }
  }
}

// Writes the registers of tb_fetch into S[row][k] (bf16, row pitch TB_LD).
template <bool KC>
__device__ inline void tb_store(__bf16* S, const TileRegs& R, int tid) {
  if constexpr (KC) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (tid >> 3) + 32 * i, k = (tid & 7) * 4;
      *reinterpret_cast<bf4v*>(S + tb_off(r, k)) =
          to_bf4(R.v[i][0], R.v[i][1], R.v[i][2], R.v[i][3]);
    }
  } else {
    const int k = 4 * (tid >> 5), r = 4 * (tid & 31);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      *reinterpret_cast<bf4v*>(S + tb_off(r + e, k)) =
          to_bf4(R.v[0][e], R.v[1][e], R.v[2][e], R.v[3][e]);
  }
}

// Workgroup b of n -> logical index such that consecutive logical indices
// run on one XCD (workgroups are dispatched to the 8 XCDs in turn).
__device__ inline int xcd_logical(int b, int n) {
  const int per = n / 8, rem = n % 8, x = b % 8;
  return x * per + min(x, rem) + b / 8;
}

// SUB: K-tiles of 32 loaded per stage (the loads of a stage are waited for
// one stage after they are issued).  SUB = 2 doubles the LDS, so two
// workgroups fit a CU instead of three: slower alone, but the GEMMs that run
// beside a resident recurrence (on the CUs it leaves free) then slow its
// exchange less (bilstm3's backward launches 1.71 -> 1.60 ms).  The caller
// chooses it only for work beside a grid that leaves CUs free.
// ABF: the A operands are stored as bf16 (GemmArgs::a_bf16).
template <bool A_KC, bool B_KC, int SUB, bool ABF>
__global__ __launch_bounds__(256) void k_gemm_bf16(GemmArgs g) {
  constexpr int kTbSub = SUB;
  __shared__ __attribute__((aligned(16))) __bf16 As[2][kTbSub][TBM * TB_LD];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[2][kTbSub][TBM * TB_LD];
  const int mt = (g.M + TBM - 1) / TBM, nt = (g.N + TBM - 1) / TBM;
  const int l = xcd_logical(blockIdx.x, gridDim.x);
  const int n_i = l % nt, m_i = (l / nt) % mt, split = l / (nt * mt);
  const int m0 = m_i * TBM, n0 = n_i * TBM;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
  const int lr = lane & 15, lq = lane >> 4;

  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  int buf = 0;
  // One reduction term: A (lda) x B (ldb, gather) over k in [kbeg, kend).
  auto term = [&](const float* A, int64_t lda, const float* B, int64_t ldb,
                  const int32_t* gather, int kbeg, int kend) {
    if (kbeg >= kend) return;
    constexpr int KS = kTbSub * TBK;  // k per stage
    std::conditional_t<ABF, TileRegsBf, TileRegs> ra[kTbSub];
    TileRegs rb[kTbSub];
#pragma unroll
    for (int u = 0; u < kTbSub; ++u) {
      if constexpr (ABF)
        tb_fetch_bf16<A_KC>(ra[u], A, lda, m0, g.M, kbeg + u * TBK, kend, tid);
      else
        tb_fetch<A_KC>(ra[u], A, lda, nullptr, m0, g.M, kbeg + u * TBK, kend, tid);
      tb_fetch<B_KC>(rb[u], B, ldb, gather, n0, g.N, kbeg + u * TBK, kend, tid);
    }
    for (int k0 = kbeg; k0 < kend; k0 += KS) {
#pragma unroll
      for (int u = 0; u < kTbSub; ++u) {
        if constexpr (ABF)
          tb_store_bf16<A_KC>(As[buf][u], ra[u], tid);
        else
          tb_store<A_KC>(As[buf][u], ra[u], tid);
        tb_store<B_KC>(Bs[buf][u], rb[u], tid);
      }
      __syncthreads();
      if (k0 + KS < kend) {
#pragma unroll
        for (int u = 0; u < kTbSub; ++u) {
          if constexpr (ABF)
            tb_fetch_bf16<A_KC>(ra[u], A, lda, m0, g.M, k0 + KS + u * TBK, kend, tid);
          else
            tb_fetch<A_KC>(ra[u], A, lda, nullptr, m0, g.M, k0 + KS + u * TBK, kend, tid);
          tb_fetch<B_KC>(rb[u], B, ldb, gather, n0, g.N, k0 + KS + u * TBK, kend, tid);
        }
      }
#pragma unroll
      for (int u = 0; u < kTbSub; ++u) {
        if (k0 + u * TBK >= kend) break;  // uniform: a partial last stage
        const __bf16* a_s = As[buf][u];
        const __bf16* b_s = Bs[buf][u];
        bf8 a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          a[i] = *reinterpret_cast<const bf8*>(a_s + tb_off(wm + 16 * i + lr, 8 * lq));
#pragma unroll
        for (int j = 0; j < 4; ++j)
          b[j] = *reinterpret_cast<const bf8*>(b_s + tb_off(wn + 16 * j + lr, 8 * lq));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
      buf ^= 1;
    }
  };
  const int kbeg = split * g.k_per_split;
  term(g.A, g.lda, g.B, g.ldb, g.gather_b, kbeg, min(g.K, kbeg + g.k_per_split));
  if (g.K2 > 0) term(g.A2, g.lda2, g.B2, g.ldb2, nullptr, 0, g.K2);

  // Accumulator layout of a 16x16 MFMA tile: lane holds column (lane & 15),
  // rows 4*(lane >> 4) + r for r = 0..3.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + wn + 16 * j + lr;
      if (n >= g.N) continue;
      const float bv = (g.splits == 1 && g.bias) ? g.bias[n] : 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + 16 * i + 4 * lq + r;
        if (m >= g.M) continue;
        float v = acc[i][j][r];
        if (g.splits > 1) {
          g.partial[((int64_t)split * g.M + m) * g.N + n] = v;
        } else {
          float* c = g.C + (int64_t)m * g.ldc + n;
          v += bv;
          if (g.accumulate) v += *c;
          *c = v;
        }
      }
    }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& g, bool a_kc, bool b_kc, bool bf16, hipStream_t st) {
  if (g.K2 > 0 && (g.splits > 1 || g.K % 32 != 0 || g.gather_b)) return hipErrorInvalidValue;
  if (bf16) {
    const int64_t blocks = (int64_t)((g.M + TBM - 1) / TBM) * ((g.N + TBM - 1) / TBM) *
                           (g.splits > 1 ? g.splits : 1);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(256);
#define RNNBKT_BF16_CASE(AK, BKC)                                              \
  if (a_kc == AK && b_kc == BKC) {                                             \
    if (g.beside && g.a_bf16)                                                  \
      hipLaunchKernelGGL((k_gemm_bf16<AK, BKC, 2, true>), grid, block, 0, st, g); \
    else if (g.beside)                                                         \
      hipLaunchKernelGGL((k_gemm_bf16<AK, BKC, 2, false>), grid, block, 0, st, g); \
    else if (g.a_bf16)                                                         \
      hipLaunchKernelGGL((k_gemm_bf16<AK, BKC, 1, true>), grid, block, 0, st, g); \
    else                                                                       \
      hipLaunchKernelGGL((k_gemm_bf16<AK, BKC, 1, false>), grid, block, 0, st, g); \
    return hipGetLastError();                                                  \
  }
    RNNBKT_BF16_CASE(true, true)
    RNNBKT_BF16_CASE(true, false)
    RNNBKT_BF16_CASE(false, false)
    RNNBKT_BF16_CASE(false, true)
#undef RNNBKT_BF16_CASE
    return hipErrorInvalidValue;
  }
  if (g.a_bf16) return hipErrorInvalidValue;  // bf16-stored operands only on the bf16 path
  if (g.K2 > 0) {
    // fp32: the second term as a second launch accumulating into C.
    GemmArgs g1 = g, g2 = g;
    g1.K2 = 0;
    g2.A = g.A2;
    g2.B = g.B2;
    g2.lda = g.lda2;
    g2.ldb = g.ldb2;
    g2.K = g.K2;
    g2.k_per_split = (g.K2 + 31) / 32 * 32;
    g2.K2 = 0;
    g2.bias = nullptr;
    g2.accumulate = 1;
    hipError_t e = launch_gemm(g1, a_kc, b_kc, false, st);
    return e != hipSuccess ? e : launch_gemm(g2, a_kc, b_kc, false, st);
  }
  dim3 grid((g.M + BM - 1) / BM, (g.N + BN - 1) / BN, g.splits > 1 ? g.splits : 1);
  dim3 block(256);
#define RNNBKT_GEMM_CASE(AK, BKC)                                          \
  if (a_kc == AK && b_kc == BKC) {                                         \
    hipLaunchKernelGGL((k_gemm<AK, BKC>), grid, block, 0, st, g);         \
    return hipGetLastError();                                              \
  }
  RNNBKT_GEMM_CASE(true, true)
  RNNBKT_GEMM_CASE(true, false)
  if (!a_kc && !b_kc) {
    hipLaunchKernelGGL(k_gemm_tn_f32, grid, block, 0, st, g);
    return hipGetLastError();
  }
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
