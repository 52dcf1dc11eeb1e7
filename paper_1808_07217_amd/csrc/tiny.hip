// One launch per local-SGD round for softmax regression (one layer, fp32)
// when every replica and its momentum buffer fit in LDS: H local steps on all
// K replicas followed by the K-way average (eq. 2, Algorithm 1's round), in
// one workgroup. Small problems are bound by launch latency, not by work --
// the multi-kernel round of such a problem is 13 launches for H = 4 -- so the
// whole round runs from LDS with no launch between its steps.
//
// Two kernels: k_tiny_round_wide (further down) gives each of up to four
// replicas 256 threads and puts both products on the matrix cores;
// k_tiny_round, for more replicas or when the former's LDS does not fit:
//
// Workgroup layout: four waves; replica k belongs to wave k mod 4. Per local
// step and replica, its wave
//   samples B indices (the configured sampler),
//   forwards its rows (lane = row: C logits, the weight read from LDS by
//     broadcast), takes the stable softmax cross-entropy and
//     dZ = (softmax - onehot) / B into LDS, the mean loss by a fixed
//     butterfly,
//   forms dW[i][c] = sum_b x[b][i] dZ[b][c] in ascending b (lane = input
//     feature) and db[c], and applies the momentum-SGD step to the replica
//     in LDS.
// Then the replicas are averaged in the replica-average tree order and
// replicas and buffers are written back.
#include <atomic>

#include "kernels.h"
#include "device_common.h"

namespace lsgd {
namespace {

constexpr int kTinyThreads = 256;
typedef float v4f __attribute__((ext_vector_type(4)));

// Per-step scratch of one wave: dZ [B][C], the sampled row indices [B] and
// the rows themselves [B][D | 1].
__device__ __forceinline__ float wave_sum_fixed(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// CM >= C: classes padded to a compile-time count. Weights, buffers and dZ
// sit in LDS at a row pitch of CM (padded entries zero, so they stay zero
// through every update), the hot loops run over all CM columns with float4
// LDS reads, and the padded logits are masked to -inf: no loop branches on
// the class count.
template <int CM>
__global__ __launch_bounds__(kTinyThreads) void k_tiny_round(TinyArgs a) {
  extern __shared__ float lds[];
  const int K = a.K, B = a.B, D = a.D, C = a.C, P = D * C + C;
  const int PL = (D + 1) * CM;              // a replica in LDS: D rows + bias row
  float* Wl = lds;                          // [K][D + 1][CM]
  float* Ul = Wl + (long long)K * PL;       // [K][D + 1][CM]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int XP = D | 1;  // odd row pitch: lane-per-row reads miss no bank
  const int WS = (B * CM + B + B * XP + 3) & ~3;  // per-wave scratch, float4-aligned
  float* dz = Ul + (long long)K * PL + wave * WS;     // this wave's [B][CM]
  int32_t* rows = (int32_t*)(dz + B * CM);                            // [B]
  float* xs = dz + B * CM + B;                                        // [B][XP] its rows

#pragma unroll 8
  for (int e = threadIdx.x; e < K * PL; e += kTinyThreads) {
    const int k = e / PL, q = e - k * PL, i = q / CM, c = q - i * CM;
    const long long g = (long long)k * a.Ps + i * C + c;
    const bool ok = c < C;
    Wl[e] = ok ? a.W[g] : 0.f;
    Ul[e] = ok ? a.U[g] : 0.f;
  }
  __syncthreads();

  const float invB = 1.0f / (float)B;
  const int slots = (K + 3) / 4;
  for (int h = 0; h < a.H; ++h) {
    const long long step = a.step0 + h;
    const float lr = a.lr[h];
    for (int r = 0; r < slots; ++r) {
      // every wave passes the same barriers; waves without a replica in this
      // slot (k >= K) skip the work between them
      const int k = 4 * r + wave;
      const bool mine = k < K;
      float* W = Wl + (long long)(mine ? k : 0) * PL;
      float* U = Ul + (long long)(mine ? k : 0) * PL;
      const long long lo = (long long)k * a.N / K;
      if (mine) {
        // sampling
        if (a.S > 0) {  // per-epoch reshuffled partition
          const long long ep = step / a.S, j = step - ep * a.S;
          for (int b = lane; b < B; b += 64)
            rows[b] = epoch_row((uint32_t)(lo + j * B + b), a.N, a.m, a.key0, a.key1,
                                (uint32_t)ep);
        } else {        // i.i.d. from the worker's shard
          const uint64_t n = (uint64_t)((long long)(k + 1) * a.N / K - lo);
          for (int q = lane; 4 * q < B; q += 64) {
            const uint4 u = philox4x32_10(
                make_uint4((uint32_t)q, (uint32_t)step, (uint32_t)k,
                           (uint32_t)((uint64_t)step >> 32)), a.key0, a.key1);
            const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (4 * q + e < B)
                rows[4 * q + e] = (int32_t)(lo + (long long)(((uint64_t)w4[e] * n) >> 32));
          }
        }
      }
      __syncthreads();
      if (mine) {
        // the batch's rows into LDS, every load in flight before any store
        if ((D & 3) == 0) {
          const int D4 = D >> 2;
#pragma unroll 8
          for (int e = lane; e < B * D4; e += 64) {
            const int b = e / D4, i4 = e - b * D4;
            const v4f v = *(const v4f*)(a.X + (long long)rows[b] * D + 4 * i4);
            float* d = xs + b * XP + 4 * i4;
            d[0] = v[0];
            d[1] = v[1];
            d[2] = v[2];
            d[3] = v[3];
          }
        } else {
#pragma unroll 8
          for (int e = lane; e < B * D; e += 64) {
            const int b = e / D, i = e - b * D;
            xs[b * XP + i] = a.X[(long long)rows[b] * D + i];
          }
        }
      }
      __syncthreads();
      if (mine) {
        // forward, loss, dZ: lane = row
        float lsum = 0.f;
        for (int b0 = 0; b0 < B; b0 += 64) {
          const int b = b0 + lane;
          const bool live = b < B;
          const int row = live ? rows[b] : rows[0];
          const int lab = a.y[row];   // issued before the forward loop
          const float* x = xs + (live ? b : 0) * XP;
          float z[CM];
#pragma unroll
          for (int c = 0; c < CM; ++c) z[c] = 0.f;
#pragma unroll 4
          for (int i = 0; i < D; ++i) {
            const float xi = x[i];
#pragma unroll
            for (int c4 = 0; c4 < CM; c4 += 4) {
              const v4f wv = *(const v4f*)(W + i * CM + c4);
#pragma unroll
              for (int j = 0; j < 4; ++j) z[c4 + j] = __builtin_fmaf(xi, wv[j], z[c4 + j]);
            }
          }
          float m = -INFINITY;
#pragma unroll
          for (int c = 0; c < CM; ++c) {
            z[c] = c < C ? z[c] + W[D * CM + c] : -INFINITY;
            m = fmaxf(m, z[c]);
          }
          float s = 0.f, rest = 0.f, zy = 0.f;
#pragma unroll
          for (int c = 0; c < CM; ++c) {
            const float e = __expf(z[c] - m);   // 0 for the padded classes
            s += e;
            rest += c != lab ? e : 0.f;
            zy = c == lab ? z[c] : zy;
          }
          const float loss = zy >= m ? log1pf(rest) : (m - zy) + logf(s);
          const float inv_s = 1.0f / s;
          if (live) {
#pragma unroll
            for (int c4 = 0; c4 < CM; c4 += 4) {
              v4f v;
#pragma unroll
              for (int j = 0; j < 4; ++j)
                v[j] = (__expf(z[c4 + j] - m) * inv_s - (c4 + j == lab ? 1.f : 0.f)) * invB;
              *(v4f*)(dz + b * CM + c4) = v;
            }
            lsum += loss;
          }
        }
        lsum = wave_sum_fixed(lsum);
        if (lane == 0) {
          const float mean = lsum * invB;
          if (a.loss) a.loss[h * K + k] = mean;
          if (a.nonfinite && !isfinite(mean)) *a.nonfinite = 1;
        }
      }
      __syncthreads();
      if (mine) {
        // weight gradient and update: lane = input feature (and the bias row
        // as feature D, whose "input" is 1)
        for (int i0 = 0; i0 <= D; i0 += 64) {
          const int i = i0 + lane;
          if (i <= D) {
            float g[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c) g[c] = 0.f;
#pragma unroll 4
            for (int b = 0; b < B; ++b) {
              const float xi = i < D ? xs[b * XP + i] : 1.f;
#pragma unroll
              for (int c4 = 0; c4 < CM; c4 += 4) {
                const v4f dv = *(const v4f*)(dz + b * CM + c4);
#pragma unroll
                for (int j = 0; j < 4; ++j) g[c4 + j] = __builtin_fmaf(xi, dv[j], g[c4 + j]);
              }
            }
            const float wd = a.wd;   // coupled decay on weights and biases alike
#pragma unroll
            for (int c4 = 0; c4 < CM; c4 += 4) {
              v4f w = *(v4f*)(W + i * CM + c4), u = *(v4f*)(U + i * CM + c4);
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const float gg = __builtin_fmaf(wd, w[j], g[c4 + j]);
                u[j] = __builtin_fmaf(a.mom, u[j], gg);
                w[j] = __builtin_fmaf(-lr, step_dir(u[j], gg, a.mom, a.mode), w[j]);
              }
              *(v4f*)(W + i * CM + c4) = w;
              *(v4f*)(U + i * CM + c4) = u;
            }
          }
        }
      }
      __syncthreads();
    }
  }
  // the K-way average, every replica := mean; then write back
  for (int p = threadIdx.x; p < P; p += kTinyThreads) {
    const int i = p / C, c = p - i * C;
    const float mean = tree_sum_f(Wl + i * CM + c, PL, K) / (float)K;
    for (int k = 0; k < K; ++k) a.W[k * a.Ps + p] = mean;
  }
#pragma unroll 4
  for (int e = threadIdx.x; e < K * P; e += kTinyThreads) {
    const int k = e / P, p = e - k * P, i = p / C, c = p - i * C;
    a.U[k * a.Ps + p] = Ul[(long long)k * PL + i * CM + c];
  }
}

// The same round with a group of 256 threads (four waves) per replica, up
// to four replicas in 1024 threads. Both contractions of a step run on the
// matrix cores (v_mfma_f32_16x16x4f32) with their operands read from LDS:
//   logits Z^T = W^T X^T as blocks of 16 rows, over the input features;
//   gradient dW = X^T dZ (the bias as a feature whose input is 1) as blocks of
//     16 features x 16 classes, over the batch rows, each block followed by
//     the momentum step of its entries.
// Lane l then holds four classes of row l % 16, so a row's max, sums and
// label logit are one butterfly over four lanes; the logarithms of the row
// losses are taken by the wave with the fewest gradient blocks, which adds
// them lane-strided in ascending order, then by a fixed butterfly.
//
// LDS layout per replica (all pitches multiples of 4 floats, so that every
// MFMA operand of the forward and every update is one float4 access):
//   Wt, Ut [CM][DP]: class-major weights and buffers, entry (c, i) = weight
//     of input i (i = D: the bias) for class c; columns D + 1 .. DP - 1 and
//     classes C .. CM - 1 are zero and stay zero through every update.
//   xs [B16][XP] (two buffers, with labels [B]): the batch rows; columns D ..
//     XP - 1 and rows B .. B16 - 1 are zero, so the forward needs no masks.
//   dz [B16][CM]: dZ, rows B .. B16 - 1 zero; the rows' loss terms [B][2];
//     the sampled row indices of every step [H][B].
// The MFMA k index is remapped (lane quarter q takes k = 4 q .. 4 q + 3 of a
// 16-deep trip), so each lane's four k values are contiguous in LDS.
//
// The rows of all H steps are sampled up front; while a step computes, the
// next step's rows and labels are in flight into registers and are stored
// into the other buffer at the end of the step (two barriers per step). Wave
// ranks are rotated by replica, so a phase with fewer blocks than waves
// spreads over the four SIMDs. The average is the replica-average tree's.
constexpr int kWideThreads = 1024, kRepThreads = 256;

// Reductions over the four lanes l % 16 + 16 q of a wave (xor 16, then xor
// 32): each step adds two partials that both lanes of the pair form in the
// same order, so all four lanes end with bitwise the same value.
__device__ __forceinline__ float quad16_sum(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}
__device__ __forceinline__ float quad16_max(float v) {
  float o = __shfl_xor(v, 16, 64);
  v = o > v ? o : v;
  o = __shfl_xor(v, 32, 64);
  return o > v ? o : v;
}

// The replica average of k_tiny_round_wide (K <= 4) in the order of the
// replica-average tree: ((w0 + w1) + (w2 + w3)), ((w0 + w1) + w2), ...
__device__ __forceinline__ float tree_sum_le4(const float* p, int stride, int K) {
  if (K == 1) return p[0];
  const float a = p[0] + p[stride];
  if (K == 2) return a;
  if (K == 3) return a + p[2 * stride];
  return a + (p[2 * stride] + p[3 * stride]);
}

// Up to 4 * 256 float4 elements of a step's batch rows (the row-major
// [B][D] block, D % 4 == 0): element e at thread e % 256, slot e / 256.
constexpr int kPrefetch4 = 4 * kRepThreads;
__device__ __forceinline__ void rows_load(const float* X, const int32_t* r, int D4, int nel,
                                          int t, v4f (&v)[4]) {
  // unconditional loads (slots past the batch re-read element 0), so that
  // all four are in flight together
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = t + kRepThreads * j < nel ? t + kRepThreads * j : 0;
    const int b = e / D4, i4 = e - b * D4;
    v[j] = *(const v4f*)(X + (long long)r[b] * (4 * D4) + 4 * i4);
  }
}
__device__ __forceinline__ void rows_store(float* xs, int XP, int D4, int nel, int t,
                                           const v4f (&v)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = t + kRepThreads * j;
    if (e < nel) {
      const int b = e / D4, i4 = e - b * D4;
      *(v4f*)(xs + b * XP + 4 * i4) = v[j];
    }
  }
}

// Pitches of the wide kernel's LDS layout (see above).
__host__ __device__ inline int wide_dp(int D) {  // Wt row: >= D + 1 and >= ceil16(D)
  const int a = (D + 4) & ~3, b = (D + 15) & ~15;
  return a > b ? a : b;
}
__host__ __device__ inline int wide_xp(int D) { return ((D + 15) & ~15) + 4; }
__host__ __device__ inline int wide_rep_floats(int B, int D, int CM, int H) {
  const int B16 = (B + 15) & ~15;
  const int head = (B16 * CM + 2 * B + H * B + 3) & ~3;   // dz, loss terms, rows
  const int buf = (B16 * wide_xp(D) + B + 3) & ~3;         // xs + labels
  return head + 2 * buf;
}

template <int CM>
__global__ __launch_bounds__(kWideThreads) void k_tiny_round_wide(TinyArgs a) {
  constexpr int NCB = CM >= 16 ? CM / 16 : 1;  // blocks of 16 classes
  extern __shared__ float lds[];
  const int K = a.K, B = a.B, D = a.D, C = a.C, H = a.H;
  const int DP = wide_dp(D), XP = wide_xp(D), B16 = (B + 15) & ~15;
  const int PL = CM * DP;
  float* Wl = lds;                        // [K][CM][DP]
  float* Ul = Wl + (long long)K * PL;     // [K][CM][DP]
  const int k = threadIdx.x / kRepThreads, t = threadIdx.x % kRepThreads;
  // MFMA lane row and quarter; the wave's rank in its group, rotated by the
  // replica so that the first waves of the four groups (the only ones with
  // work when a phase has fewer blocks than waves) sit on different SIMDs
  const int l16 = t & 15, lq = (t & 63) >> 4, wr = ((t >> 6) - k) & 3;
  const bool mine = k < K;
  const int RS = wide_rep_floats(B, D, CM, H);
  float* dz = Ul + (long long)K * PL + (mine ? k : 0) * RS;   // [B16][CM]
  float* lrow = dz + B16 * CM;                                 // [B][2]
  int32_t* rows = (int32_t*)(lrow + 2 * B);                    // [H][B]
  const int BUF = (B16 * XP + B + 3) & ~3;
  float* const buf0 = dz + ((B16 * CM + 2 * B + H * B + 3) & ~3);
  float* xs = buf0;                                            // [B16][XP]
  int32_t* labs = (int32_t*)(buf0 + B16 * XP);                 // [B]

  const long long lo = (long long)k * a.N / K;
  if (mine) {
    // zero padding: both row buffers and dZ's rows past the batch
    for (int e = 4 * t; e < 2 * BUF; e += 4 * kRepThreads)
      *(v4f*)(buf0 + e) = (v4f){0.f, 0.f, 0.f, 0.f};
    for (int e = B * CM + t; e < B16 * CM; e += kRepThreads) dz[e] = 0.f;
    // every step's rows
    if (a.S > 0) {  // per-epoch reshuffled partition
      for (int e = t; e < H * B; e += kRepThreads) {
        const int h = e / B, b = e - h * B;
        const long long step = a.step0 + h, ep = step / a.S, j = step - ep * a.S;
        rows[e] = epoch_row((uint32_t)(lo + j * B + b), a.N, a.m, a.key0, a.key1,
                            (uint32_t)ep);
      }
    } else {        // i.i.d. from the worker's shard
      const uint64_t n = (uint64_t)((long long)(k + 1) * a.N / K - lo);
      const int nq = (B + 3) >> 2;
      for (int e = t; e < H * nq; e += kRepThreads) {
        const int h = e / nq, q = e - h * nq;
        const long long step = a.step0 + h;
        const uint4 u = philox4x32_10(
            make_uint4((uint32_t)q, (uint32_t)step, (uint32_t)k,
                       (uint32_t)((uint64_t)step >> 32)), a.key0, a.key1);
        const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (4 * q + j < B)
            rows[h * B + 4 * q + j] = (int32_t)(lo + (long long)(((uint64_t)w4[j] * n) >> 32));
      }
    }
  }
  __syncthreads();

  // the next step's batch fits four float4 per thread and its labels one
  // per thread: prefetched during the step; otherwise staged between steps
  const int D4 = D >> 2;
  const bool pf = (D & 3) == 0 && B * D4 <= kPrefetch4 && B <= kRepThreads;
  v4f pre[4];
  int lab_next = 0;
  auto stage_sync = [&](int h) {
    const int32_t* r = rows + h * B;
    if ((D & 3) == 0) {
#pragma unroll 4
      for (int e = t; e < B * D4; e += kRepThreads) {
        const int b = e / D4, i4 = e - b * D4;
        *(v4f*)(xs + b * XP + 4 * i4) = *(const v4f*)(a.X + (long long)r[b] * D + 4 * i4);
      }
    } else {
#pragma unroll 4
      for (int e = t; e < B * D; e += kRepThreads) {
        const int b = e / D, i = e - b * D;
        xs[b * XP + i] = a.X[(long long)r[b] * D + i];
      }
    }
    for (int b = t; b < B; b += kRepThreads) labs[b] = a.y[r[b]];
  };
  // step 0's rows and labels in flight together with the replicas' loads
  if (mine && pf) {
    rows_load(a.X, rows, D4, B * D4, t, pre);
    lab_next = a.y[rows[t < B ? t : 0]];
  }
  // the replicas, input-major over the padded layout (the row and class of
  // an entry are a shift and a mask), transposed into LDS: per chunk all
  // four replicas' loads (clamped, unconditional) before any store, so they
  // share one round trip
  for (int e0 = threadIdx.x; e0 < DP * CM; e0 += 2 * kWideThreads) {
    float wv[4][2], uv[4][2];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int e = min(e0 + r * kWideThreads, DP * CM - 1), i = e / CM, c = e % CM;
        const long long g =
            (long long)min(kk, K - 1) * a.Ps + (i <= D ? i : D) * C + (c < C ? c : 0);
        wv[kk][r] = a.W[g];
        uv[kk][r] = a.U[g];
      }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int e = e0 + r * kWideThreads, i = e / CM, c = e % CM;
        if (kk < K && e < DP * CM) {
          const bool ok = c < C && i <= D;
          Wl[kk * PL + c * DP + i] = ok ? wv[kk][r] : 0.f;
          Ul[kk * PL + c * DP + i] = ok ? uv[kk][r] : 0.f;
        }
      }
  }
  if (mine) {
    if (pf) {
      rows_store(xs, XP, D4, B * D4, t, pre);
      if (t < B) labs[t] = lab_next;
    } else {
      stage_sync(0);
    }
  }
  __syncthreads();

  const float invB = 1.0f / (float)B;
  float* W = Wl + (long long)(mine ? k : 0) * PL;
  float* U = Ul + (long long)(mine ? k : 0) * PL;
  for (int h = 0; h < H; ++h) {
    const float lr = a.lr[h];
    const bool next = h + 1 < H;
    xs = buf0 + (h & 1) * BUF;
    labs = (int32_t*)(xs + B16 * XP);
    if (mine && pf && next) {  // in flight while this step computes
      const int32_t* r = rows + (h + 1) * B;
      rows_load(a.X, r, D4, B * D4, t, pre);
      lab_next = a.y[r[t < B ? t : 0]];
    }
    if (mine) {
      // forward, loss terms, dZ: wave rank wr takes row blocks wr, wr + 4, ...
      const int nrb = B16 >> 4;
      for (int rb = wr; rb < nrb; rb += kRepThreads / 64) {
        const int br = rb * 16 + l16;
        const float* xb = xs + br * XP + 4 * lq;
        v4f acc[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = (v4f){0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < D; k0 += 16) {
          const v4f xv = *(const v4f*)(xb + k0);
          v4f wv[NCB];
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) {
            const int c = cb * 16 + l16;
            const v4f w = *(const v4f*)(W + (c < CM ? c : 0) * DP + k0 + 4 * lq);
            wv[cb] = c < CM ? w : (v4f){0.f, 0.f, 0.f, 0.f};
          }
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb)
              acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv[cb][u], xv[u], acc[cb], 0, 0, 0);
        }
        // lane holds the logits of row br, classes cb * 16 + 4 lq + j
        const bool rok = br < B;
        const int lab = labs[rok ? br : 0];
        float z[NCB][4], zl[NCB][4], m = -INFINITY;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int c = cb * 16 + 4 * lq + j;
            zl[cb][j] = acc[cb][j] + W[(c < C ? c : 0) * DP + D];
            z[cb][j] = c < C ? zl[cb][j] : -INFINITY;
            m = z[cb][j] > m ? z[cb][j] : m;
          }
        m = quad16_max(m);
        float s = 0.f, rest = 0.f, zy = -INFINITY;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int c = cb * 16 + 4 * lq + j;
            z[cb][j] = __expf(z[cb][j] - m);  // 0 for the padded classes
            s += z[cb][j];
            rest += c != lab ? z[cb][j] : 0.f;
            zy = c == lab ? zl[cb][j] : zy;
          }
        s = quad16_sum(s);
        rest = quad16_sum(rest);
        zy = quad16_max(zy);
        if (rok) {
          const float inv_s = 1.0f / s;
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) {
            const int c4 = cb * 16 + 4 * lq;
            if (c4 < CM) {
              v4f d;
#pragma unroll
              for (int j = 0; j < 4; ++j)
                d[j] = (z[cb][j] * inv_s - (c4 + j == lab ? 1.f : 0.f)) * invB;
              *(v4f*)(dz + br * CM + c4) = d;
            }
          }
          if (lq == 0) {  // the loss's terms; its logarithm on the loss wave
            lrow[2 * br] = m - zy;
            lrow[2 * br + 1] = zy >= m ? rest : s;
          }
        }
      }
    }
    __syncthreads();
    if (mine) {
      if (wr == 3) {  // mean loss (the wave with the fewest gradient blocks):
        // lane-strided rows in order, then a butterfly
        const int lane = t & 63;
        float lsum = 0.f;
        for (int b = lane; b < B; b += 64) {
          const float d = lrow[2 * b], v = lrow[2 * b + 1];
          lsum += d <= 0.f ? log1pf(v) : d + logf(v);  // d = 0: the label is the max
        }
        lsum = wave_sum_fixed(lsum);
        if (lane == 0) {
          const float mean = lsum * invB;
          if (a.loss) a.loss[h * K + k] = mean;
          if (a.nonfinite && !isfinite(mean)) *a.nonfinite = 1;
        }
      }
      // weight gradient and update: wave rank wr takes blocks wr, wr + 4, ...
      const int nib = (D + 16) >> 4;  // ceil((D + 1) / 16)
      for (int blk = wr; blk < nib * NCB; blk += kRepThreads / 64) {
        const int ib = blk / NCB, cb = blk - ib * NCB;
        const int ia = ib * 16 + l16, cn = cb * 16 + l16;
        const int iac = ia < XP ? ia : XP - 1;     // columns D + 1 .. XP - 1 are zero
        const int cnc = cn < CM ? cn : 0;
        v4f acc = (v4f){0.f, 0.f, 0.f, 0.f};
        for (int b0 = 0; b0 < B; b0 += 16) {  // rows past B are zero
          float av[4], bv[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int b = b0 + 4 * lq + u;
            const float x = xs[b * XP + iac], g = dz[b * CM + cnc];
            av[u] = ia == D ? 1.f : x;
            bv[u] = cn < CM ? g : 0.f;
          }
#pragma unroll
          for (int u = 0; u < 4; ++u)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[u], acc, 0, 0, 0);
        }
        // lane holds the gradient of inputs ib * 16 + 4 lq + j, class cn: one
        // float4 of Wt and Ut (padding entries get a zero gradient and stay 0)
        const int i0 = ib * 16 + 4 * lq;
        if (i0 < DP && cn < CM) {
          const float wd = a.wd;
          v4f w = *(v4f*)(W + cn * DP + i0), u = *(v4f*)(U + cn * DP + i0);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float gg = __builtin_fmaf(wd, w[j], acc[j]);
            u[j] = __builtin_fmaf(a.mom, u[j], gg);
            w[j] = __builtin_fmaf(-lr, step_dir(u[j], gg, a.mom, a.mode), w[j]);
          }
          *(v4f*)(W + cn * DP + i0) = w;
          *(v4f*)(U + cn * DP + i0) = u;
        }
      }
    }
    if (next && mine) {  // into the other buffer, last read two steps ago
      xs = buf0 + ((h + 1) & 1) * BUF;
      labs = (int32_t*)(xs + B16 * XP);
      if (pf) {
        rows_store(xs, XP, D4, B * D4, t, pre);
        if (t < B) labs[t] = lab_next;
      } else {
        stage_sync(h + 1);
      }
    }
    __syncthreads();
  }
  for (int e = threadIdx.x; e < (D + 1) * CM; e += kWideThreads) {
    const int i = e / CM, c = e % CM, p = i * C + c;
    if (c < C) {
      const float mean = tree_sum_le4(Wl + c * DP + i, PL, K) / (float)K;
      for (int kk = 0; kk < K; ++kk) {
        a.W[kk * a.Ps + p] = mean;
        a.U[kk * a.Ps + p] = Ul[kk * PL + c * DP + i];
      }
    }
  }
}

}  // namespace

int tiny_classes(int C) { return C <= 8 ? 8 : C <= 16 ? 16 : 32; }

size_t tiny_round_lds_bytes(int K, int B, int D, int C) {
  const int CM = tiny_classes(C);
  const long long wave = ((long long)B * CM + B + (long long)B * (D | 1) + 3) & ~3LL;
  return (size_t)(2LL * K * (D + 1) * CM + 4LL * wave) * sizeof(float);
}
size_t tiny_wide_lds_bytes(int K, int B, int D, int C, int H) {
  const int CM = tiny_classes(C);
  return (size_t)(2LL * K * CM * wide_dp(D) + (long long)K * wide_rep_floats(B, D, CM, H)) *
         sizeof(float);
}

// The kernel's dynamic LDS above the default 64 KB: requested once per
// device and instance (gfx950 compute units hold 160 KB). The per-device
// flags are atomics: contexts on different host threads may launch at once
// (the request itself is idempotent).
template <int CM, bool Wide>
hipError_t allow_lds(size_t bytes) {
  static std::atomic<bool> done[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= 64) return e != hipSuccess ? e : hipErrorInvalidDevice;
  if (bytes <= 64 * 1024 || done[dev].load(std::memory_order_acquire)) return hipSuccess;
  e = hipFuncSetAttribute(Wide ? (const void*)k_tiny_round_wide<CM> : (const void*)k_tiny_round<CM>,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)kTinyMaxLds);
  if (e == hipSuccess) done[dev].store(true, std::memory_order_release);
  return e;
}

// LDS one workgroup may opt in to on the current device (cached per device
// in an atomic; concurrent first queries store the same value).
size_t tiny_lds_limit() {
  static std::atomic<size_t> limit[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  size_t v = limit[dev].load(std::memory_order_acquire);
  if (!v) {
    int q = 0;
    if (hipDeviceGetAttribute(&q, hipDeviceAttributeSharedMemPerBlockOptin, dev) != hipSuccess ||
        q <= 0)
      q = 64 * 1024;
    v = (size_t)q;
    limit[dev].store(v, std::memory_order_release);
  }
  return v;
}

bool tiny_round_fits(int K, int B, int D, int C, int H) {
  if (K < 1 || B < 1 || D < 1 || C < 2 || C > kTinyMaxC || H < 1 || H > kTinyMaxH)
    return false;
  const size_t lds = tiny_round_lds_bytes(K, B, D, C);
  return lds <= kTinyMaxLds && lds <= tiny_lds_limit();
}

// Whether the 256-thread-per-replica kernel runs (up to four replicas, when
// its larger LDS request fits); otherwise the wave-per-replica kernel does.
bool tiny_round_wide(int K, int B, int D, int C, int H) {
  const size_t wide = tiny_wide_lds_bytes(K, B, D, C, H);
  return K * kRepThreads <= kWideThreads && wide <= kTinyMaxLds && wide <= tiny_lds_limit();
}

template <int CM>
hipError_t launch_round(const TinyArgs& a, hipStream_t s) {
  hipError_t e;
  if (tiny_round_wide(a.K, a.B, a.D, a.C, a.H)) {
    const size_t wide = tiny_wide_lds_bytes(a.K, a.B, a.D, a.C, a.H);
    if ((e = allow_lds<CM, true>(wide)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_tiny_round_wide<CM>, dim3(1), dim3(kWideThreads), wide, s, a);
  } else {
    const size_t lds = tiny_round_lds_bytes(a.K, a.B, a.D, a.C);
    if ((e = allow_lds<CM, false>(lds)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_tiny_round<CM>, dim3(1), dim3(kTinyThreads), lds, s, a);
  }
  return hipGetLastError();
}
// Up to four replicas take the 256-thread-per-replica kernel when its larger
// scratch fits; otherwise the wave-per-replica kernel runs.
hipError_t launch_tiny_round(const TinyArgs& a, hipStream_t s) {
  if (!tiny_round_fits(a.K, a.B, a.D, a.C, a.H)) return hipErrorInvalidValue;
  switch (tiny_classes(a.C)) {
    case 8: return launch_round<8>(a, s);
    case 16: return launch_round<16>(a, s);
    default: return launch_round<32>(a, s);
  }
}
}  // namespace lsgd
