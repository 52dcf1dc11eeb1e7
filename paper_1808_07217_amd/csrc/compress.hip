// Sign-compressed synchronisation of (post-)local signSGD and EF-signSGD
// (Algorithms 3 and 4 of the appendix on compression): every worker sends
// its corrected model difference delta^k = w_s - w^k (+ e^k) as
// sign(delta^k) * ||delta^k||_1 / P, and every replica restarts from
// w_s - (1/K) sum_k sign(delta^k) ||delta^k||_1 / P.
//
// Three launches: per (replica, chunk) the l1 partial sums in fp64 (and,
// without error memories, the signs packed two bits per element); per
// replica the scale p^k from its partials in a fixed order; then the new
// model from the packed signs (or, with memories, from delta recomputed in
// the same arithmetic, which also updates e^k = delta^k - s^k p^k).
#include <mutex>

#include "kernels.h"

namespace lsgd {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kSgT = 256;                    // threads per workgroup
constexpr int kSgIters = 8;                  // float4 per thread and chunk
constexpr long long kSgChunk4 = kSgT * kSgIters;  // float4 per chunk

__device__ __forceinline__ float sgnf(float x) {
  return x > 0.f ? 1.f : (x < 0.f ? -1.f : 0.f);
}

// Phase 1, grid (chunks, K). Packed signs: for replica k and group q of 64
// float4 (256 elements, one wave), words 8q .. 8q+3 hold in bit l whether
// component j of float4 64q + l is > 0 (word 8q + j), words 8q+4 .. 8q+7
// whether it is < 0. Lanes past n4 count as zero.
template <bool EF>
__global__ __launch_bounds__(kSgT) void k_sign_l1(
    const float* W, const float* E, const float* ws, long long n4,
    long long sP4, long long ngroups, uint64_t* bits, double* part) {
  __shared__ double red[kSgT];
  const int k = blockIdx.y;
  const v4f* w4 = (const v4f*)W + k * sP4;
  const v4f* s4 = (const v4f*)ws;
  const int lane = threadIdx.x & 63;
  const long long base = (long long)blockIdx.x * kSgChunk4;
  double acc = 0.0;
  for (int it = 0; it < kSgIters; ++it) {
    const long long wave0 = base + it * kSgT + (threadIdx.x & ~63);
    const long long i = wave0 + lane;
    const bool ok = i < n4;
    const long long ic = ok ? i : n4 - 1;
    v4f d = s4[ic] - w4[ic];
    if constexpr (EF) d += ((const v4f*)E + k * sP4)[ic];
    if (!ok) d = (v4f){0.f, 0.f, 0.f, 0.f};
    acc += (double)fabsf(d.x) + (double)fabsf(d.y) + (double)fabsf(d.z) +
           (double)fabsf(d.w);
    if constexpr (!EF) {
      const uint64_t b[8] = {__ballot(d.x > 0.f), __ballot(d.y > 0.f),
                             __ballot(d.z > 0.f), __ballot(d.w > 0.f),
                             __ballot(d.x < 0.f), __ballot(d.y < 0.f),
                             __ballot(d.z < 0.f), __ballot(d.w < 0.f)};
      if (wave0 < n4 && lane < 8) {
        uint64_t v = b[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) v = lane == j ? b[j] : v;
        bits[(k * ngroups + wave0 / 64) * 8 + lane] = v;
      }
    }
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = kSgT / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) part[(long long)k * gridDim.x + blockIdx.x] = red[0];
}

// Phase 2, one workgroup per replica: p^k = (sum of its chunk partials) / P,
// thread t adding chunks t, t + 256, ... in order, then a fixed tree.
__global__ __launch_bounds__(kSgT) void k_sign_scale(const double* part,
                                                     int nchunks, long long P,
                                                     float* p) {
  __shared__ double red[kSgT];
  const int k = blockIdx.x;
  double acc = 0.0;
  for (int c = threadIdx.x; c < nchunks; c += kSgT)
    acc += part[(long long)k * nchunks + c];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = kSgT / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) p[k] = (float)(red[0] / (double)P);
}

__device__ __forceinline__ void store_bf16x4(bf16_t* q, v4f v) {
  const uint32_t a = f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
  const uint32_t b = f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
  *(uint2*)q = make_uint2(a, b);
}

// Phase 3, one thread per float4 of the model: the messages s^k p^k summed
// over k in ascending order, w_s -= sum / K, every replica := w_s.
template <bool EF>
__global__ __launch_bounds__(kSgT) void k_sign_apply(
    float* W, bf16_t* Wb, float* E, float* ws, int K, long long n4,
    long long sP4, long long ngroups, const uint64_t* bits, const float* p) {
  const long long i = blockIdx.x * (long long)kSgT + threadIdx.x;
  if (i >= n4) return;
  const v4f s0 = ((const v4f*)ws)[i];
  v4f acc = (v4f){0.f, 0.f, 0.f, 0.f};
  const int l = (int)(i & 63);
  for (int k = 0; k < K; ++k) {
    const float pk = p[k];
    v4f s;
    if constexpr (EF) {
      v4f* e4 = (v4f*)E + k * sP4;
      const v4f d = s0 - ((const v4f*)W + k * sP4)[i] + e4[i];
      s = (v4f){sgnf(d.x), sgnf(d.y), sgnf(d.z), sgnf(d.w)};
      e4[i] = d - s * pk;
    } else {
      const uint64_t* b = bits + (k * ngroups + i / 64) * 8;
      s.x = (float)((b[0] >> l) & 1) - (float)((b[4] >> l) & 1);
      s.y = (float)((b[1] >> l) & 1) - (float)((b[5] >> l) & 1);
      s.z = (float)((b[2] >> l) & 1) - (float)((b[6] >> l) & 1);
      s.w = (float)((b[3] >> l) & 1) - (float)((b[7] >> l) & 1);
    }
    acc += s * pk;
  }
  const v4f wn = s0 - acc / (float)K;
  ((v4f*)ws)[i] = wn;
  for (int k = 0; k < K; ++k) {
    ((v4f*)W)[k * sP4 + i] = wn;
    if (Wb) store_bf16x4(Wb + (k * sP4 + i) * 4, wn);
  }
}

size_t al256(size_t b) { return (b + 255) / 256 * 256; }

struct SignPlan {
  long long n4, ngroups;
  int nchunks;
  size_t bits_off, part_off, p_off, total;
};

SignPlan sign_plan(int K, long long Ps) {
  SignPlan q;
  q.n4 = Ps / 4;
  q.ngroups = (q.n4 + 63) / 64;
  q.nchunks = (int)((q.n4 + kSgChunk4 - 1) / kSgChunk4);
  q.bits_off = 0;
  q.part_off = al256((size_t)K * q.ngroups * 8 * sizeof(uint64_t));
  q.p_off = q.part_off + al256((size_t)K * q.nchunks * sizeof(double));
  q.total = q.p_off + al256((size_t)K * sizeof(float));
  return q;
}

}  // namespace

size_t sign_sync_scratch_bytes(int K, long long Ps) {
  return (K < 1 || Ps < 0) ? 0 : sign_plan(K, Ps).total;
}

// Scratch of the allocation-free sign synchronisation: one static array per
// device, alive until the process ends. Every call on a device shares it
// (calls that overlap on one device race); nothing in it needs clearing,
// since each launch writes all of the scratch it later reads.
__device__ __align__(256) unsigned char scratch[kSignSyncStaticBytes];

namespace {
// The array's device address, looked up once per device with that device
// current (the host-side name is only a stand-in for the symbol).
hipError_t static_scratch(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}
}  // namespace

hipError_t launch_sign_sync_static(float* W, float* E, float* ws, int K, long long P,
                                   hipStream_t s) {
  void* p = nullptr;
  hipError_t e = static_scratch(&p);
  if (e != hipSuccess) return e;
  return launch_sign_sync(W, nullptr, E, ws, K, P, P, p, kSignSyncStaticBytes, s);
}

hipError_t launch_sign_sync(float* W, bf16_t* Wb, float* E, float* ws, int K,
                            long long P, long long Ps, void* scratch,
                            size_t scratch_bytes, hipStream_t s) {
  if (K < 1 || P <= 0) return hipSuccess;
  if (Ps % 4 || Ps < P || ((uintptr_t)W | (uintptr_t)ws | (uintptr_t)E |
                           (uintptr_t)scratch) & 15u ||
      ((uintptr_t)Wb & 7u))
    return hipErrorInvalidValue;
  const SignPlan q = sign_plan(K, Ps);
  if (scratch_bytes < q.total || q.nchunks > 65535 * 256 || K > 65535)
    return hipErrorInvalidValue;
  char* base = (char*)scratch;
  uint64_t* bits = (uint64_t*)(base + q.bits_off);
  double* part = (double*)(base + q.part_off);
  float* p = (float*)(base + q.p_off);
  const long long sP4 = Ps / 4;
  if (E)
    hipLaunchKernelGGL(k_sign_l1<true>, dim3(q.nchunks, K), dim3(kSgT), 0, s, W, E,
                       ws, q.n4, sP4, q.ngroups, bits, part);
  else
    hipLaunchKernelGGL(k_sign_l1<false>, dim3(q.nchunks, K), dim3(kSgT), 0, s, W,
                       E, ws, q.n4, sP4, q.ngroups, bits, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sign_scale, dim3(K), dim3(kSgT), 0, s, part, q.nchunks, P, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)((q.n4 + kSgT - 1) / kSgT));
  if (E)
    hipLaunchKernelGGL(k_sign_apply<true>, grid, dim3(kSgT), 0, s, W, Wb, E, ws, K,
                       q.n4, sP4, q.ngroups, bits, p);
  else
    hipLaunchKernelGGL(k_sign_apply<false>, grid, dim3(kSgT), 0, s, W, Wb, E, ws, K,
                       q.n4, sP4, q.ngroups, bits, p);
  e = hipGetLastError();
  return e;
}

}  // namespace lsgd
