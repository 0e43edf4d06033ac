// Memory-bound kernels of the training step: batch tables and packing of the
// padded batch into valid frames, the per-frame softmax cross-entropy with
// its gradient, deterministic reductions, and the parameter updates (SGD and
// ADADELTA).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.h"

namespace rnnbkt {

namespace {

constexpr int kLenChunk = 256;
struct LenChunk {
  int32_t len[kLenChunk];
};

__global__ void k_store_ints(LenChunk c, int count, int32_t* dst) {
  const int i = threadIdx.x;
  if (i < count) dst[i] = c.len[i];
}

// batch_sizes[t] (+)= #{b in chunk : len[b] > t}
__global__ void k_batch_sizes(LenChunk c, int count, int T, int32_t* bs, int first) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  int v = 0;
  for (int b = 0; b < count; ++b) v += c.len[b] > t ? 1 : 0;
  bs[t] = first ? v : bs[t] + v;
}

// offsets = exclusive prefix sum of batch_sizes; one 1024-thread block.
__global__ __launch_bounds__(1024) void k_offsets(const int32_t* __restrict__ bs, int T,
                                                  int32_t* __restrict__ off) {
  __shared__ int32_t part[1024];
  const int tid = threadIdx.x;
  const int per = (T + 1023) / 1024;
  const int t0 = tid * per;
  const int t1 = min(T, t0 + per);
  int32_t s = 0;
  for (int t = t0; t < t1; ++t) s += bs[t];
  part[tid] = s;
  __syncthreads();
  // Hillis-Steele inclusive scan of the 1024 partial sums.
  for (int d = 1; d < 1024; d <<= 1) {
    const int32_t add = tid >= d ? part[tid - d] : 0;
    __syncthreads();
    part[tid] += add;
    __syncthreads();
  }
  int32_t run = part[tid] - s;  // exclusive
  for (int t = t0; t < t1; ++t) {
    off[t] = run;
    run += bs[t];
  }
  if (tid == 1023) off[T] = part[1023];
}

__global__ void k_pack(const float* __restrict__ x, const int32_t* __restrict__ labels,
                       const int32_t* __restrict__ bs, const int32_t* __restrict__ off, int T,
                       int B, int D, float* __restrict__ Xp, int32_t* __restrict__ Yp,
                       int32_t* __restrict__ prev_fwd, int32_t* __restrict__ prev_rev) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)T * B) return;
  const int t = (int)(idx / B), b = (int)(idx % B);
  if (b >= bs[t]) return;
  const int64_t f = off[t] + b;
  const float* src = x + idx * D;
  float* dst = Xp + f * D;
  for (int k = 0; k < D; ++k) dst[k] = src[k];
  if (Yp) Yp[f] = labels[idx];
  prev_fwd[f] = t > 0 ? off[t - 1] + b : -1;
  prev_rev[f] = (t + 1 < T && b < bs[t + 1]) ? off[t + 1] + b : -1;
}

struct PrepArgs {
  int32_t len[kPrepMaxB];
  int32_t lsum[kPrepMaxB + 1];  // lsum[i] = sum of len[0..i)
  int32_t B, T, D;
  const float* x;
  const int32_t* labels;
  int32_t *bs, *off;
  float* Xp;
  int32_t *Yp, *pf, *pr;
  FillJob fill[kFillJobs];
  int32_t nfill;
  uint32_t value;
  unsigned* zero;
};

// #{b : len[b] > t} for non-increasing lengths (binary search).
__device__ inline int32_t rows_after(const PrepArgs& a, int t) {
  int lo = 0, hi = a.B;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a.len[mid] > t)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo;
}

// Packing with the tables written in passing: with lengths non-increasing,
// frame (t, b) is valid iff b < batch_sizes[t] = #{b : len[b] > t}, and
// offsets[t] = sum_b min(len[b], t) = t * batch_sizes[t] + sum of the lengths
// from batch_sizes[t] on, so each thread takes them from the lengths and
// their prefix sums (a few binary-search steps).  Then the fills,
// grid-stride, 16 bytes per store.
__global__ void k_prepare(PrepArgs a) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nth = (int64_t)gridDim.x * blockDim.x;
  const int64_t frames = (int64_t)a.T * a.B;
  if (gid == 0 && a.zero) *a.zero = 0u;
  const int32_t total = a.lsum[a.B];
  for (int64_t idx = gid; idx < frames; idx += nth) {
    const int t = (int)(idx / a.B), b = (int)(idx % a.B);
    const int32_t bs_t = rows_after(a, t);
    if (b >= bs_t) continue;
    const int32_t off_t = t * bs_t + total - a.lsum[bs_t];
    const int32_t bs_p = t > 0 ? rows_after(a, t - 1) : 0;
    const int32_t bs_n = t + 1 < a.T ? rows_after(a, t + 1) : 0;
    const int32_t off_p = off_t - bs_p;  // offsets[t - 1]
    if (b == 0) {
      a.bs[t] = bs_t;
      a.off[t] = off_t;
      if (t == a.T - 1) a.off[a.T] = off_t + bs_t;
    }
    const int64_t f = off_t + b;
    const float* src = a.x + idx * a.D;
    float* dst = a.Xp + f * a.D;
    for (int k = 0; k < a.D; ++k) dst[k] = src[k];
    if (a.Yp) a.Yp[f] = a.labels[idx];
    a.pf[f] = t > 0 ? off_p + b : -1;
    a.pr[f] = (t + 1 < a.T && b < bs_n) ? off_t + bs_t + b : -1;
  }
  const uint4 v4 = make_uint4(a.value, a.value, a.value, a.value);
  for (int j = 0; j < a.nfill; ++j) {
    unsigned* p = a.fill[j].p;
    const int64_t n = a.fill[j].n;
    for (int64_t i4 = gid * 4; i4 < n; i4 += nth * 4) {
      if (i4 + 3 < n) {
        *reinterpret_cast<uint4*>(p + i4) = v4;
      } else {
        for (int64_t i = i4; i < n; ++i) p[i] = a.value;
      }
    }
  }
}

__global__ void k_unpack(const float* __restrict__ H, int W, const int32_t* __restrict__ bs,
                         const int32_t* __restrict__ off, int T, int B,
                         float* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)T * B * W) return;
  const int64_t tb = idx / W;
  const int w = (int)(idx % W);
  const int t = (int)(tb / B), b = (int)(tb % B);
  out[idx] = b < bs[t] ? H[(int64_t)(off[t] + b) * W + w] : 0.f;
}

__device__ inline float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

constexpr int kXentRowsPerWave = 4;
constexpr int kXentWaves = 4;
constexpr int kXentMaxPerLane = 16;  // C <= 1024

// A wave per kXentRowsPerWave frames: max, log-sum-exp, loss term and
// gradient row of each.  MPL = ceil(C / 64) elements per lane and row; the
// loads of all the wave's rows are issued before any reduction, so a wave
// waits for memory once rather than once per row.
template <int MPL>
__global__ __launch_bounds__(256) void k_softmax_xent(float* __restrict__ z,
                                                      const int32_t* __restrict__ y, int64_t N,
                                                      int C, float inv_n,
                                                      float* __restrict__ partial) {
  __shared__ float wsum[kXentWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t base = ((int64_t)blockIdx.x * kXentWaves + wave) * kXentRowsPerWave;
  float v[kXentRowsPerWave][MPL];
  int label[kXentRowsPerWave];
#pragma unroll
  for (int rr = 0; rr < kXentRowsPerWave; ++rr) {
    const int64_t f = base + rr;
    const bool ok = f < N;
    label[rr] = ok ? y[f] : 0;
#pragma unroll
    for (int i = 0; i < MPL; ++i) {
      const int c = lane + 64 * i;
      v[rr][i] = ok && c < C ? z[f * C + c] : -INFINITY;
    }
  }
  float acc = 0.f;
#pragma unroll
  for (int rr = 0; rr < kXentRowsPerWave; ++rr) {
    const int64_t f = base + rr;
    if (f >= N) break;
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < MPL; ++i) m = fmaxf(m, v[rr][i]);
    m = wave_max(m);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < MPL; ++i) {
      const int c = lane + 64 * i;
      if (c < C) s += expf(v[rr][i] - m);
    }
    s = wave_sum(s);
    const float lse = m + logf(s);
    float zy = 0.f;
    float* row = z + f * C;
#pragma unroll
    for (int i = 0; i < MPL; ++i) {
      const int c = lane + 64 * i;
      if (c < C) {
        if (c == label[rr]) zy = v[rr][i];
        const float p = expf(v[rr][i] - lse);
        row[c] = (p - (c == label[rr] ? 1.f : 0.f)) * inv_n;
      }
    }
    zy = wave_sum(zy);
    acc += (label[rr] >= 0 && label[rr] < C) ? lse - zy : NAN;
  }
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
    for (int w = 0; w < kXentWaves; ++w) t += wsum[w];
    partial[blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(1024) void k_sum(const float* __restrict__ p, int n, float scale,
                                              float* __restrict__ out) {
  __shared__ float red[1024];
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += 1024) s += p[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int d = 512; d > 0; d >>= 1) {
    if ((int)threadIdx.x < d) red[threadIdx.x] += red[threadIdx.x + d];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0] * scale;
}

__global__ void k_sgd(float* __restrict__ p, const float* __restrict__ g, int64_t n, float lr) {
  const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 + 3 < n) {
    float4 pv = *reinterpret_cast<float4*>(p + i4);
    const float4 gv = *reinterpret_cast<const float4*>(g + i4);
    pv.x -= lr * gv.x;
    pv.y -= lr * gv.y;
    pv.z -= lr * gv.z;
    pv.w -= lr * gv.w;
    *reinterpret_cast<float4*>(p + i4) = pv;
  } else {
    for (int64_t i = i4; i < n; ++i) p[i] -= lr * g[i];
  }
}

// One ADADELTA step on element i (Zeiler's method, the update rule of the
// paper's training processes): the squared-gradient average first, the step
// from the previous squared-update average, then that average.
__device__ inline void adadelta1(float& p, float g, float& eg2, float& edx2, float rho, float eps,
                                 float lr) {
  const float e = rho * eg2 + (1.f - rho) * g * g;
  const float dx = -(sqrtf(edx2 + eps) / sqrtf(e + eps)) * g;
  edx2 = rho * edx2 + (1.f - rho) * dx * dx;
  eg2 = e;
  p += lr * dx;
}

__global__ void k_adadelta(float* __restrict__ p, const float* __restrict__ g,
                           float* __restrict__ eg2, float* __restrict__ edx2, int64_t n, float rho,
                           float eps, float lr) {
  const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 + 3 < n) {
    float4 pv = *reinterpret_cast<float4*>(p + i4);
    const float4 gv = *reinterpret_cast<const float4*>(g + i4);
    float4 a = *reinterpret_cast<float4*>(eg2 + i4);
    float4 b = *reinterpret_cast<float4*>(edx2 + i4);
    adadelta1(pv.x, gv.x, a.x, b.x, rho, eps, lr);
    adadelta1(pv.y, gv.y, a.y, b.y, rho, eps, lr);
    adadelta1(pv.z, gv.z, a.z, b.z, rho, eps, lr);
    adadelta1(pv.w, gv.w, a.w, b.w, rho, eps, lr);
    *reinterpret_cast<float4*>(p + i4) = pv;
    *reinterpret_cast<float4*>(eg2 + i4) = a;
    *reinterpret_cast<float4*>(edx2 + i4) = b;
  } else {
    for (int64_t i = i4; i < n; ++i) adadelta1(p[i], g[i], eg2[i], edx2[i], rho, eps, lr);
  }
}

// Eq. 3 over four consecutive parameters: the replica mean minus beta times
// the previous aggregate, accumulated in double (the result is the exact
// value rounded once to float), written back to every replica and to prev.
__device__ inline float4 aggregate4(const float* reps, int R, int64_t stride, int64_t i4,
                                    const float* prev, double beta) {
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  for (int r = 0; r < R; ++r) {
    const float4 v = *reinterpret_cast<const float4*>(reps + r * stride + i4);
    s0 += v.x;
    s1 += v.y;
    s2 += v.z;
    s3 += v.w;
  }
  const float4 pv = *reinterpret_cast<const float4*>(prev + i4);
  const double inv = 1.0 / R;
  return make_float4((float)(s0 * inv - beta * pv.x), (float)(s1 * inv - beta * pv.y),
                     (float)(s2 * inv - beta * pv.z), (float)(s3 * inv - beta * pv.w));
}

__global__ void k_aggregate(float* __restrict__ reps, int R, int64_t stride, int64_t n,
                            float* __restrict__ prev, double beta) {
  const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 + 3 < n) {
    const float4 v = aggregate4(reps, R, stride, i4, prev, beta);
    for (int r = 0; r < R; ++r) *reinterpret_cast<float4*>(reps + r * stride + i4) = v;
    *reinterpret_cast<float4*>(prev + i4) = v;
  } else {
    for (int64_t i = i4; i < n; ++i) {
      double s = 0.0;
      for (int r = 0; r < R; ++r) s += reps[r * stride + i];
      const float v = (float)(s * (1.0 / R) - beta * prev[i]);
      for (int r = 0; r < R; ++r) reps[r * stride + i] = v;
      prev[i] = v;
    }
  }
}

// out[c * ld_out + r] = in[r * ld_in + c] for r < rows, c < cols: 32 x 32
// tiles through LDS (rows of 33 floats: the column reads hit distinct banks).
__global__ __launch_bounds__(256) void k_transpose(const float* __restrict__ in, int rows, int cols,
                                                   int64_t ld_in, float* __restrict__ out,
                                                   int64_t ld_out) {
  __shared__ float t[32][33];
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int i = ty; i < 32; i += 8) {
    const int r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) t[i][tx] = in[(int64_t)r * ld_in + c];
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) out[(int64_t)c * ld_out + r] = t[tx][i];
  }
}

__global__ void k_fill_u32(unsigned* __restrict__ p, int64_t n, unsigned v) {
  const int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 + 3 < n) {
    *reinterpret_cast<uint4*>(p + i4) = make_uint4(v, v, v, v);
  } else {
    for (int64_t i = i4; i < n; ++i) p[i] = v;
  }
}

}  // namespace

hipError_t launch_transpose(const float* in, int32_t rows, int32_t cols, int64_t ld_in, float* out,
                            int64_t ld_out, hipStream_t st) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const dim3 grid((unsigned)((cols + 31) / 32), (unsigned)((rows + 31) / 32));
  hipLaunchKernelGGL(k_transpose, grid, dim3(256), 0, st, in, rows, cols, ld_in, out, ld_out);
  return hipGetLastError();
}

hipError_t launch_fill_u32(unsigned* p, int64_t n, unsigned v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int threads = 256;
  const int64_t quads = (n + 3) / 4;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)((quads + threads - 1) / threads)), dim3(threads),
                     0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_store_ints(const int32_t* values, int n, int32_t* dst, hipStream_t st) {
  for (int c0 = 0; c0 < n; c0 += kLenChunk) {
    LenChunk c{};
    const int cnt = std::min(kLenChunk, n - c0);
    for (int i = 0; i < cnt; ++i) c.len[i] = values[c0 + i];
    hipLaunchKernelGGL(k_store_ints, dim3(1), dim3(kLenChunk), 0, st, c, cnt, dst + c0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_batch_tables(const int32_t* lengths, int32_t B, int32_t T, int32_t* bs,
                               int32_t* off, hipStream_t st) {
  const int threads = 256;
  for (int c0 = 0; c0 < B; c0 += kLenChunk) {
    LenChunk c{};
    const int cnt = std::min(kLenChunk, B - c0);
    for (int i = 0; i < cnt; ++i) c.len[i] = lengths[c0 + i];
    hipLaunchKernelGGL(k_batch_sizes, dim3((T + threads - 1) / threads), dim3(threads), 0, st,
                       c, cnt, T, bs, c0 == 0 ? 1 : 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_offsets, dim3(1), dim3(1024), 0, st, bs, T, off);
  return hipGetLastError();
}

hipError_t launch_pack(const float* x, const int32_t* labels, const int32_t* bs,
                       const int32_t* off, int32_t T, int32_t B, int32_t D, float* Xp,
                       int32_t* Yp, int32_t* pf, int32_t* pr, hipStream_t st) {
  const int64_t total = (int64_t)T * B;
  const int threads = 256;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)((total + threads - 1) / threads)), dim3(threads),
                     0, st, x, labels, bs, off, T, B, D, Xp, Yp, pf, pr);
  return hipGetLastError();
}

hipError_t launch_prepare(const int32_t* lengths, int32_t B, int32_t T, const float* x,
                          const int32_t* labels, int32_t D, int32_t* bs, int32_t* off, float* Xp,
                          int32_t* Yp, int32_t* pf, int32_t* pr, const FillJob* fills,
                          int32_t nfill, unsigned value, unsigned* zero_word, hipStream_t st) {
  if (B < 0 || B > kPrepMaxB || nfill < 0 || nfill > kFillJobs) return hipErrorInvalidValue;
  PrepArgs a{};
  for (int i = 0; i < B; ++i) {
    a.len[i] = lengths[i];
    a.lsum[i + 1] = a.lsum[i] + lengths[i];
  }
  a.B = B;
  a.T = T;
  a.D = D;
  a.x = x;
  a.labels = labels;
  a.bs = bs;
  a.off = off;
  a.Xp = Xp;
  a.Yp = Yp;
  a.pf = pf;
  a.pr = pr;
  a.nfill = nfill;
  a.value = value;
  a.zero = zero_word;
  int64_t quads = 0;
  for (int j = 0; j < nfill; ++j) {
    a.fill[j] = fills[j];
    quads = std::max<int64_t>(quads, (fills[j].n + 3) / 4);
  }
  const int threads = 256;
  const int64_t want = std::max<int64_t>(std::max<int64_t>((int64_t)T * B, zero_word ? 1 : 0),
                                         std::min<int64_t>(quads, 4096 * threads));
  if (want == 0) return hipSuccess;
  hipLaunchKernelGGL(k_prepare, dim3((unsigned)((want + threads - 1) / threads)), dim3(threads), 0,
                     st, a);
  return hipGetLastError();
}

hipError_t launch_unpack(const float* H, int32_t W, const int32_t* bs, const int32_t* off,
                         int32_t T, int32_t B, float* out, hipStream_t st) {
  const int64_t total = (int64_t)T * B * W;
  const int threads = 256;
  hipLaunchKernelGGL(k_unpack, dim3((unsigned)((total + threads - 1) / threads)), dim3(threads),
                     0, st, H, W, bs, off, T, B, out);
  return hipGetLastError();
}

hipError_t launch_softmax_xent(float* z, const int32_t* y, int64_t N, int32_t C,
                               float* partial, int32_t* num_partials, hipStream_t st) {
  const int64_t rows_per_block = kXentRowsPerWave * kXentWaves;
  const int blocks = (int)((N + rows_per_block - 1) / rows_per_block);
  *num_partials = blocks;
  const int mpl = (C + 63) / 64;
  const dim3 g(blocks), t(256);
  const float inv_n = 1.0f / (float)N;
  if (mpl <= 1)
    hipLaunchKernelGGL(k_softmax_xent<1>, g, t, 0, st, z, y, N, C, inv_n, partial);
  else if (mpl <= 2)
    hipLaunchKernelGGL(k_softmax_xent<2>, g, t, 0, st, z, y, N, C, inv_n, partial);
  else if (mpl <= 4)
    hipLaunchKernelGGL(k_softmax_xent<4>, g, t, 0, st, z, y, N, C, inv_n, partial);
  else if (mpl <= 8)
    hipLaunchKernelGGL(k_softmax_xent<8>, g, t, 0, st, z, y, N, C, inv_n, partial);
  else if (mpl <= kXentMaxPerLane)
    hipLaunchKernelGGL(k_softmax_xent<kXentMaxPerLane>, g, t, 0, st, z, y, N, C, inv_n, partial);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_sum(const float* partial, int32_t n, float scale, float* out, hipStream_t st) {
  hipLaunchKernelGGL(k_sum, dim3(1), dim3(1024), 0, st, partial, n, scale, out);
  return hipGetLastError();
}

hipError_t launch_sgd(float* p, const float* g, int64_t n, float lr, hipStream_t st) {
  const int threads = 256;
  const int64_t quads = (n + 3) / 4;
  hipLaunchKernelGGL(k_sgd, dim3((unsigned)((quads + threads - 1) / threads)), dim3(threads), 0,
                     st, p, g, n, lr);
  return hipGetLastError();
}

hipError_t launch_adadelta(float* p, const float* g, float* eg2, float* edx2, int64_t n,
                           float rho, float eps, float lr, hipStream_t st) {
  const int threads = 256;
  const int64_t quads = (n + 3) / 4;
  hipLaunchKernelGGL(k_adadelta, dim3((unsigned)((quads + threads - 1) / threads)), dim3(threads),
                     0, st, p, g, eg2, edx2, n, rho, eps, lr);
  return hipGetLastError();
}

hipError_t launch_aggregate(float* reps, int R, int64_t stride, int64_t n, float* prev,
                            float beta, hipStream_t st) {
  const int threads = 256;
  const int64_t quads = (n + 3) / 4;
  hipLaunchKernelGGL(k_aggregate, dim3((unsigned)((quads + threads - 1) / threads)), dim3(threads),
                     0, st, reps, R, stride, n, prev, (double)beta);
  return hipGetLastError();
}

}  // namespace rnnbkt
