// Device functions shared by the sampling kernels and the single-launch
// round: the Philox4x32-10 generator, the per-epoch Feistel permutation, and
// the replica summation tree.
#pragma once
#include "kernels.h"

namespace lsgd {

// ------------------------------------------------------------------ Philox
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32->64-bit multiplies with a Weyl-sequence key schedule.
inline __device__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}

// Per-epoch reshuffled partition. Epoch e's permutation of [0, N) is a
// balanced Feistel network on 2m-bit words (4^m >= N) whose four round
// functions are word 0 of Philox4x32-10 at counter (right half, round, e,
// kShuffleStream), restricted to [0, N) by cycle walking: an image >= N is
// permuted again. The walk ends on the first in-range value of the cycle
// through the start, after about 4^m / N steps on average; a cap far above
// any plausible walk returns the position itself (still a valid row), so
// the kernel always finishes and a parity test would show the failure.
constexpr uint32_t kShuffleStream = 0x5348464Cu;
constexpr int kCycleWalkCap = 1 << 12;

inline __device__ uint32_t feistel4(uint32_t x, int m, uint32_t mask, uint32_t k0,
                                    uint32_t k1, uint32_t e) {
  uint32_t left = x >> m, right = x & mask;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint4 f = philox4x32_10(make_uint4(right, (uint32_t)r, e, kShuffleStream), k0, k1);
    const uint32_t t = left ^ (f.x & mask);
    left = right;
    right = t;
  }
  return (left << m) | right;
}

// Row pi_e(q) of the epoch permutation for position q < N.
inline __device__ int32_t epoch_row(uint32_t q, long long N, int m, uint32_t k0,
                                    uint32_t k1, uint32_t e) {
  const uint32_t mask = (1u << m) - 1u;
  uint32_t y = feistel4(q, m, mask, k0, k1, e);
  int walk = 0;
  while (y >= (uint64_t)N && walk < kCycleWalkCap) {
    y = feistel4(y, m, mask, k0, k1, e);
    ++walk;
  }
  return (int32_t)(y < (uint64_t)N ? y : q);
}

// Sum of p[0], p[stride], ..., p[(K-1) stride] in the replica-average order:
// split at the largest power of two below the count, left part first
// (a binary counter of power-of-two partial sums).
inline __device__ float tree_sum_f(const float* p, long long stride, int K) {
  float st[24];
  int sz[24];
  int top = 0;
  for (int k = 0; k < K; ++k) {
    float v = p[k * stride];
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
  float v = st[top - 1];
  for (int i = top - 2; i >= 0; --i) v = st[i] + v;
  return v;
}

}  // namespace lsgd
