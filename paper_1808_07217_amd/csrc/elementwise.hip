// Bandwidth- and latency-bound kernels of the local-SGD step: index
// sampling, softmax cross-entropy, bias gradient + update, the fused
// momentum-SGD update, and the K-way replica average.
#include "kernels.h"
#include "device_common.h"

namespace lsgd {
namespace {

// One thread per (worker k, group of 4 slots): a Philox block gives the four
// uniform words of slots 4q .. 4q+3 of worker k at local step `step`.
__global__ void k_sample(uint32_t key0, uint32_t key1, uint32_t s_lo,
                         uint32_t s_hi, int K, long long N, int B,
                         int32_t* idx) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  const int k = blockIdx.y;
  if (4 * q >= B) return;
  const long long lo = (long long)k * N / K;
  const long long hi = (long long)(k + 1) * N / K;
  const uint64_t n = (uint64_t)(hi - lo);
  const uint4 r = philox4x32_10(make_uint4((uint32_t)q, s_lo, (uint32_t)k, s_hi),
                                key0, key1);
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int j = 4 * q + e;
    if (j < B) idx[(long long)k * B + j] = (int32_t)(lo + (long long)(((uint64_t)w[e] * n) >> 32));
  }
}

// One thread per (worker k = blockIdx.y, slot b): row pi_e(lo_k + jB + b).
__global__ void k_sample_epoch(uint32_t key0, uint32_t key1, uint32_t e, long long j,
                               int K, long long N, int B, int m, int32_t* idx) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  const int k = blockIdx.y;
  if (b >= B) return;
  const uint32_t q = (uint32_t)((long long)k * N / K + j * B + b);
  idx[(long long)k * B + b] = epoch_row(q, N, m, key0, key1, e);
}

// ------------------------------------------------------------------ loss
// Softmax cross-entropy over C classes for the B rows of replica k
// (blockIdx.x): dZ = (softmax(z) - onehot(y)) / B and the mean loss, summed
// in a fixed order (per-thread rows ascending, then a fixed LDS tree).
__global__ __launch_bounds__(256) void k_xent(const float* Z, const int32_t* y,
                                              const int32_t* idx, int B, int C,
                                              void* dZ, int dz_bf16,
                                              float* loss, int* nonfinite) {
  __shared__ float red[256];
  const int k = blockIdx.x;
  const float invB = 1.0f / (float)B;
  float part = 0.f;
  for (int b = threadIdx.x; b < B; b += blockDim.x) {
    const long long row = (long long)k * B + b;
    const float* z = Z + row * C;
    const int lab = y[idx[row]];
    float m = z[0];
    for (int j = 1; j < C; ++j) m = fmaxf(m, z[j]);
    float s = 0.f, rest = 0.f;
    for (int j = 0; j < C; ++j) {
      const float e = __expf(z[j] - m);
      s += e;
      if (j != lab) rest += e;
    }
    const float zy = z[lab];
    part += zy >= m ? log1pf(rest) : (m - zy) + logf(s);
    const float inv_s = 1.0f / s;
    for (int j = 0; j < C; ++j) {
      const float p = __expf(z[j] - m) * inv_s;
      const float d = (p - (j == lab ? 1.f : 0.f)) * invB;
      if (dz_bf16)
        ((bf16_t*)dZ)[row * C + j] = f32_to_bf16(d);
      else
        ((float*)dZ)[row * C + j] = d;
    }
  }
  red[threadIdx.x] = part;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float mean = red[0] * invB;
    if (loss) loss[k] = mean;
    if (nonfinite && !isfinite(mean)) *nonfinite = 1;
  }
}

// ------------------------------------------------------------------ update
__device__ __forceinline__ void sgd(float& w, float& u, float grad, float lr,
                                    float mom, float wd, int nesterov) {
  const float g = __builtin_fmaf(wd, w, grad);
  u = __builtin_fmaf(mom, u, g);
  const float d = step_dir(u, g, mom, nesterov);
  w = __builtin_fmaf(-lr, d, w);
}

__global__ void k_sgd_update4(float4* W, float4* U, const float4* G,
                              long long n4, float lr, float mom, float wd,
                              int nesterov) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
       i += (long long)gridDim.x * blockDim.x) {
    float4 w = W[i], u = U[i];
    const float4 g = G[i];
    sgd(w.x, u.x, g.x, lr, mom, wd, nesterov);
    sgd(w.y, u.y, g.y, lr, mom, wd, nesterov);
    sgd(w.z, u.z, g.z, lr, mom, wd, nesterov);
    sgd(w.w, u.w, g.w, lr, mom, wd, nesterov);
    W[i] = w;
    U[i] = u;
  }
}

__global__ void k_sgd_update1(float* W, float* U, const float* G, long long n,
                              float lr, float mom, float wd, int nesterov) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    float w = W[i], u = U[i];
    sgd(w, u, G[i], lr, mom, wd, nesterov);
    W[i] = w;
    U[i] = u;
  }
}

// ------------------------------------------------------------------ average
// Fixed summation tree over replicas lo .. lo+n-1: split at the largest power
// of two below n, left part first. For a power-of-two K this is the pairwise
// tree ((0+1)+(2+3))+..., under which identical replicas sum exactly.
__host__ __device__ constexpr int split_of(int n) {
  int h = 1;
  while (2 * h < n) h *= 2;
  return h;
}

template <int N, typename V>
struct Tree {
  __device__ __forceinline__ static V sum(const V* p, long long stride) {
    constexpr int H = split_of(N);
    return Tree<H, V>::sum(p, stride) + Tree<N - H, V>::sum(p + H * stride, stride);
  }
};
template <typename V>
struct Tree<1, V> {
  __device__ __forceinline__ static V sum(const V* p, long long) { return *p; }
};

__device__ __forceinline__ float4 operator+(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}
__device__ __forceinline__ float4 div4(float4 a, float k) {
  return make_float4(a.x / k, a.y / k, a.z / k, a.w / k);
}

// Same tree for a run-time K: a binary counter of power-of-two partial sums.
template <typename V>
__device__ V tree_sum_rt(const V* p, long long stride, int K) {
  V st[24];
  int sz[24];
  int top = 0;
  for (int k = 0; k < K; ++k) {
    V v = p[k * stride];
    int size = 1;
    while (top > 0 && sz[top - 1] == size) {
      v = st[top - 1] + v;
      size *= 2;
      --top;
    }
    st[top] = v;
    sz[top] = size;
    ++top;
  }
  V v = st[top - 1];
  for (int i = top - 2; i >= 0; --i) v = st[i] + v;
  return v;
}

__device__ __forceinline__ void store_bf16x4(bf16_t* p, float4 v) {
  const uint32_t a = f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
  const uint32_t b = f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
  *(uint2*)p = make_uint2(a, b);
}

// Vectorised average: thread i owns elements 4i .. 4i+3 of every replica.
// The grid's y index picks a block of K consecutive replicas (hierarchical
// averaging; a single block is the global average).
// mean_out != nullptr (one block): write the mean there (and its bf16 copy to
// Wb [n] when given) and leave W untouched.
template <int KT>
__global__ void k_average4(float* W, bf16_t* Wb, int K, long long n,
                           long long ld, float* mean_out) {
  W += blockIdx.y * (long long)K * ld;
  if (Wb) Wb += blockIdx.y * (long long)K * ld;
  const long long n4 = n / 4;
  const float4* W4 = (const float4*)W;
  const long long stride = ld / 4;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
       i += (long long)gridDim.x * blockDim.x) {
    float4 s;
    if constexpr (KT > 0)
      s = Tree<KT, float4>::sum(W4 + i, stride);
    else
      s = tree_sum_rt<float4>(W4 + i, stride, K);
    const float4 mean = div4(s, (float)K);
    if (mean_out) {
      ((float4*)mean_out)[i] = mean;
      if (Wb) store_bf16x4(Wb + 4 * i, mean);
      continue;
    }
    for (int k = 0; k < K; ++k) {
      ((float4*)W)[k * stride + i] = mean;
      if (Wb) store_bf16x4(Wb + k * ld + 4 * i, mean);
    }
  }
}

// Synchronisation with global momentum: the replica mean (the tree of
// k_average4), then u = mg u + (ws - mean) / lr and ws = ws - lr u, where ws
// holds the model of the previous synchronisation; every replica gets ws.
__device__ __forceinline__ float gm_step(float mean, float& ws, float& u,
                                         float mg, float lr) {
  u = mg * u + (ws - mean) / lr;
  ws = ws - lr * u;
  return ws;
}

template <int KT>
__global__ void k_average_gm4(float* W, bf16_t* Wb, int K, long long n,
                              long long ld, float* ws, float* ug, float mg,
                              float lr) {
  const long long n4 = n / 4;
  const float4* W4 = (const float4*)W;
  const long long stride = ld / 4;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n4;
       i += (long long)gridDim.x * blockDim.x) {
    float4 s;
    if constexpr (KT > 0)
      s = Tree<KT, float4>::sum(W4 + i, stride);
    else
      s = tree_sum_rt<float4>(W4 + i, stride, K);
    const float4 mean = div4(s, (float)K);
    float4 w = ((float4*)ws)[i], u = ((float4*)ug)[i];
    gm_step(mean.x, w.x, u.x, mg, lr);
    gm_step(mean.y, w.y, u.y, mg, lr);
    gm_step(mean.z, w.z, u.z, mg, lr);
    gm_step(mean.w, w.w, u.w, mg, lr);
    ((float4*)ws)[i] = w;
    ((float4*)ug)[i] = u;
    for (int k = 0; k < K; ++k) {
      ((float4*)W)[k * stride + i] = w;
      if (Wb) store_bf16x4(Wb + k * ld + 4 * i, w);
    }
  }
}

__global__ void k_average_gm1(float* W, bf16_t* Wb, int K, long long n,
                              long long ld, float* ws, float* ug, float mg,
                              float lr) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const float mean = tree_sum_rt<float>(W + i, ld, K) / (float)K;
    float w = ws[i], u = ug[i];
    gm_step(mean, w, u, mg, lr);
    ws[i] = w;
    ug[i] = u;
    for (int k = 0; k < K; ++k) {
      W[k * ld + i] = w;
      if (Wb) Wb[k * ld + i] = f32_to_bf16(w);
    }
  }
}

__global__ void k_average1(float* W, bf16_t* Wb, int K, long long n,
                           long long ld, float* mean_out) {
  W += blockIdx.y * (long long)K * ld;
  if (Wb) Wb += blockIdx.y * (long long)K * ld;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const float mean = tree_sum_rt<float>(W + i, ld, K) / (float)K;
    if (mean_out) {
      mean_out[i] = mean;
      if (Wb) Wb[i] = f32_to_bf16(mean);
      continue;
    }
    for (int k = 0; k < K; ++k) {
      W[k * ld + i] = mean;
      if (Wb) Wb[k * ld + i] = f32_to_bf16(mean);
    }
  }
}

__global__ void k_broadcast(const float* src, float* W, bf16_t* Wb, int K,
                            long long n, long long ld, int replica) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const float v = src[i];
    for (int k = 0; k < K; ++k) {
      if (replica >= 0 && k != replica) continue;
      W[k * ld + i] = v;
      if (Wb) Wb[k * ld + i] = f32_to_bf16(v);
    }
  }
}

__global__ void k_to_bf16(const float* x, bf16_t* y, long long n) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    y[i] = f32_to_bf16(x[i]);
}

// rows x n floats from src (row pitch spitch) to dst (row pitch dpitch):
// the sections of the state blob against the padded replica rows
__global__ void k_copy_rows(float* dst, long long dpitch, const float* src,
                            long long spitch, long long n, int rows) {
  const int r = blockIdx.y;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    dst[r * dpitch + i] = src[r * spitch + i];
}

__global__ void k_put_words(unsigned long long* dst, Words8 v) {
  if (threadIdx.x < 8) dst[threadIdx.x] = v.w[threadIdx.x];
}

__global__ void k_fill(float* x, float v, long long n) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    x[i] = v;
}

// One element (or float4) per thread over the whole range: measured on the
// fused update at 1 GB, a full grid streams 15% faster than a grid capped at
// 16384 workgroups with grid-stride loops. Ranges beyond 2^31 - 1 workgroups
// fall back to the grid-stride loop the kernels keep.
int grid_for(long long n, int threads) {
  long long b = (n + threads - 1) / threads;
  if (b > 0x7fffffffLL) b = 0x7fffffffLL;
  return b < 1 ? 1 : (int)b;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

hipError_t launch_sample(uint64_t seed, int64_t step, int K, int64_t N, int B,
                         int32_t* idx, hipStream_t s) {
  const int groups = (B + 3) / 4;
  dim3 grid((groups + 63) / 64, K);
  hipLaunchKernelGGL(k_sample, grid, dim3(64), 0, s, (uint32_t)seed,
                     (uint32_t)(seed >> 32), (uint32_t)step,
                     (uint32_t)((uint64_t)step >> 32), K, (long long)N, B, idx);
  return hipGetLastError();
}

hipError_t launch_sample_epoch(uint64_t seed, int64_t step, int K, int64_t N,
                               int B, int32_t* idx, hipStream_t s) {
  const long long S = (N / K) / B;  // batches per worker and epoch
  if (S < 1 || N > 0x7fffffffLL) return hipErrorInvalidValue;
  int m = 1;
  while ((1LL << (2 * m)) < N) ++m;
  const long long e = step / S, j = step % S;
  dim3 grid((B + 63) / 64, K);
  hipLaunchKernelGGL(k_sample_epoch, grid, dim3(64), 0, s, (uint32_t)seed,
                     (uint32_t)(seed >> 32), (uint32_t)e, j, K, (long long)N, B,
                     m, idx);
  return hipGetLastError();
}

hipError_t launch_xent(const float* Z, const int32_t* y, const int32_t* idx,
                       int K, int B, int C, void* dZ, int dz_bf16, float* loss,
                       int* nonfinite, hipStream_t s) {
  hipLaunchKernelGGL(k_xent, dim3(K), dim3(256), 0, s, Z, y, idx, B, C, dZ,
                     dz_bf16, loss, nonfinite);
  return hipGetLastError();
}

hipError_t launch_sgd_update(float* W, float* U, const float* G, long long n,
                             float lr, float mom, float wd, int nesterov,
                             hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 4 == 0 && aligned16(W) && aligned16(U) && aligned16(G))
    hipLaunchKernelGGL(k_sgd_update4, dim3(grid_for(n / 4, 256)), dim3(256), 0,
                       s, (float4*)W, (float4*)U, (const float4*)G, n / 4, lr,
                       mom, wd, nesterov);
  else
    hipLaunchKernelGGL(k_sgd_update1, dim3(grid_for(n, 256)), dim3(256), 0, s,
                       W, U, G, n, lr, mom, wd, nesterov);
  return hipGetLastError();
}

hipError_t launch_average_blocks(float* W, bf16_t* Wb, int Kb, int blocks,
                                 long long n, long long ld, float* mean_out,
                                 hipStream_t s) {
  if (n <= 0 || Kb <= 0 || blocks <= 0) return hipSuccess;
  if (blocks > 65535 || (mean_out && blocks != 1)) return hipErrorInvalidValue;
  const int K = Kb;
  const bool vec = n % 4 == 0 && ld % 4 == 0 && aligned16(W) &&
                   (mean_out == nullptr || aligned16(mean_out)) &&
                   (Wb == nullptr || ((uintptr_t)Wb & 7u) == 0);
  if (!vec) {
    hipLaunchKernelGGL(k_average1, dim3(grid_for(n, 256), blocks), dim3(256),
                       0, s, W, Wb, K, n, ld, mean_out);
    return hipGetLastError();
  }
  const dim3 grid(grid_for(n / 4, 256), blocks), block(256);
#define LSGD_AVG_CASE(KK)                                                    \
  case KK:                                                                   \
    hipLaunchKernelGGL(k_average4<KK>, grid, block, 0, s, W, Wb, K, n, ld,   \
                       mean_out);                                            \
    break;
  switch (K) {
    LSGD_AVG_CASE(1)
    LSGD_AVG_CASE(2)
    LSGD_AVG_CASE(3)
    LSGD_AVG_CASE(4)
    LSGD_AVG_CASE(8)
    LSGD_AVG_CASE(16)
    LSGD_AVG_CASE(32)
    LSGD_AVG_CASE(64)
    default:
      hipLaunchKernelGGL(k_average4<0>, grid, block, 0, s, W, Wb, K, n, ld,
                         mean_out);
  }
#undef LSGD_AVG_CASE
  return hipGetLastError();
}

hipError_t launch_average(float* W, bf16_t* Wb, int K, long long n,
                          long long ld, float* mean_out, hipStream_t s) {
  return launch_average_blocks(W, Wb, K, 1, n, ld, mean_out, s);
}

hipError_t launch_average_gm(float* W, bf16_t* Wb, int K, long long n,
                             long long ld, float* ws, float* ug, float mg,
                             float lr, hipStream_t s) {
  if (n <= 0 || K <= 0) return hipSuccess;
  const bool vec = n % 4 == 0 && ld % 4 == 0 && aligned16(W) && aligned16(ws) &&
                   aligned16(ug) && (Wb == nullptr || ((uintptr_t)Wb & 7u) == 0);
  if (!vec) {
    hipLaunchKernelGGL(k_average_gm1, dim3(grid_for(n, 256)), dim3(256), 0, s,
                       W, Wb, K, n, ld, ws, ug, mg, lr);
    return hipGetLastError();
  }
  const dim3 grid(grid_for(n / 4, 256)), block(256);
#define LSGD_AVG_GM_CASE(KK)                                                 \
  case KK:                                                                   \
    hipLaunchKernelGGL(k_average_gm4<KK>, grid, block, 0, s, W, Wb, K, n, ld, \
                       ws, ug, mg, lr);                                      \
    break;
  switch (K) {
    LSGD_AVG_GM_CASE(1)
    LSGD_AVG_GM_CASE(2)
    LSGD_AVG_GM_CASE(4)
    LSGD_AVG_GM_CASE(8)
    LSGD_AVG_GM_CASE(16)
    LSGD_AVG_GM_CASE(32)
    LSGD_AVG_GM_CASE(64)
    default:
      hipLaunchKernelGGL(k_average_gm4<0>, grid, block, 0, s, W, Wb, K, n, ld,
                         ws, ug, mg, lr);
  }
#undef LSGD_AVG_GM_CASE
  return hipGetLastError();
}

hipError_t launch_broadcast(const float* src, float* W, bf16_t* Wb, int K,
                            long long n, long long ld, int replica,
                            hipStream_t s) {
  hipLaunchKernelGGL(k_broadcast, dim3(grid_for(n, 256)), dim3(256), 0, s, src,
                     W, Wb, K, n, ld, replica);
  return hipGetLastError();
}

hipError_t launch_to_bf16(const float* x, bf16_t* y, long long n,
                          hipStream_t s) {
  hipLaunchKernelGGL(k_to_bf16, dim3(grid_for(n, 256)), dim3(256), 0, s, x, y,
                     n);
  return hipGetLastError();
}

hipError_t launch_copy_rows(float* dst, long long dpitch, const float* src,
                            long long spitch, long long n, int rows,
                            hipStream_t s) {
  if (rows <= 0 || n <= 0) return hipSuccess;
  long long b = (n + 255) / 256;
  if (b > 65535) b = 65535;
  hipLaunchKernelGGL(k_copy_rows, dim3((unsigned)b, rows), dim3(256), 0, s, dst,
                     dpitch, src, spitch, n, rows);
  return hipGetLastError();
}

hipError_t launch_put_words(void* dst, const Words8& v, hipStream_t s) {
  hipLaunchKernelGGL(k_put_words, dim3(1), dim3(64), 0, s,
                     (unsigned long long*)dst, v);
  return hipGetLastError();
}

hipError_t launch_fill(float* x, float v, long long n, hipStream_t s) {
  hipLaunchKernelGGL(k_fill, dim3(grid_for(n, 256)), dim3(256), 0, s, x, v, n);
  return hipGetLastError();
}

}  // namespace lsgd
