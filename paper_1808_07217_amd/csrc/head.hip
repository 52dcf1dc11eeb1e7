// The output layer of the network with few classes (C <= 32), fused around
// the loss: the mean mini-batch cross-entropy whose gradient is the bracket of
// eq. 2 in the paper.
//
// k_head_fwd: one wavefront per sample row b of replica k. Lanes stride over
//   the D inputs to form the C logits, reduced across the wave by a fixed xor
//   butterfly; then softmax cross-entropy (stable form), dZ = (p - onehot)/B,
//   and, below the top layer, the input gradient dA[d] = sum_c dZ[c] W[d][c]
//   masked by the ReLU derivative (A > 0).
// k_head_wgrad: one workgroup per (replica, 64 inputs d): dW[d][c] =
//   sum_b A[b][d] dZ[b][c] in ascending b, fused with the momentum-SGD update;
//   workgroup 0 of each replica also updates the bias (sum_b dZ[b][c]) and
//   reduces the per-row losses in ascending b.
#include "kernels.h"

namespace lsgd {
namespace {

template <typename T>
__device__ __forceinline__ float ld(const T* p, long long i);
template <>
__device__ __forceinline__ float ld<float>(const float* p, long long i) {
  return p[i];
}
template <>
__device__ __forceinline__ float ld<bf16_t>(const bf16_t* p, long long i) {
  return bf16_to_f32(p[i]);
}
__device__ __forceinline__ void st(float* p, long long i, float v) { p[i] = v; }
__device__ __forceinline__ void st(bf16_t* p, long long i, float v) {
  p[i] = f32_to_bf16(v);
}
__device__ __forceinline__ float round_like(float v, const float*) { return v; }
__device__ __forceinline__ float round_like(float v, const bf16_t*) {
  return bf16_to_f32(f32_to_bf16(v));
}

// dst[i] = src[base + i] for i < n by the 256 threads of the workgroup, eight
// loads in flight per thread before the LDS stores.
template <typename T>
__device__ __forceinline__ void stage(float* dst, const T* src, long long base,
                                      int n) {
  for (int i0 = 0; i0 < n; i0 += 8 * 256) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * 256 + (int)threadIdx.x;
      v[u] = i < n ? ld(src, base + i) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * 256 + (int)threadIdx.x;
      if (i < n) dst[i] = v[u];
    }
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ void sgd_step(float& w, float& u, float grad,
                                         const HeadArgs& h) {
  const float g = __builtin_fmaf(h.wd, w, grad);
  u = __builtin_fmaf(h.mom, u, g);
  const float d = step_dir(u, g, h.mom, h.nesterov);
  w = __builtin_fmaf(-h.lr, d, w);
}

// Rows of W_L staged in LDS per pass: W chunk [DCH][C] plus nothing else.
template <int CMAX>
constexpr int head_chunk() { return CMAX <= 16 ? 1024 : 512; }

template <typename T, int CMAX, bool GATHER>
__global__ __launch_bounds__(256) void k_head_fwd(HeadArgs h) {
  constexpr int RPW = 2;             // sample rows per wavefront
  constexpr int DCH = head_chunk<CMAX>();
  __shared__ float Ws[DCH * CMAX];
  const int k = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int D = h.D, C = h.C;
  const T* Wg = (const T*)h.W + (long long)k * h.sW;
  const T* arow[RPW];
  long long rr[RPW];
  bool live[RPW];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int row = (blockIdx.x * 4 + wave) * RPW + q;
    live[q] = row < h.B;
    rr[q] = (long long)k * h.B + (live[q] ? row : 0);
    arow[q] = GATHER ? (const T*)h.A + (long long)h.rowmap[rr[q]] * D
                     : (const T*)h.A + (long long)k * h.sA +
                           (long long)(live[q] ? row : 0) * D;
  }

  float z[RPW][CMAX];
#pragma unroll
  for (int q = 0; q < RPW; ++q)
#pragma unroll
    for (int c = 0; c < CMAX; ++c) z[q][c] = 0.f;
  for (int d0 = 0; d0 < D; d0 += DCH) {
    const int nd = min(DCH, D - d0);
    __syncthreads();
    stage(Ws, Wg, (long long)d0 * C, nd * C);
    __syncthreads();
    // four strides of 64 per pass: all loads first, then the FMAs
    for (int db = 0; db < nd; db += 256) {
      float av[4][RPW];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db + u * 64 + lane;
#pragma unroll
        for (int q = 0; q < RPW; ++q) av[u][q] = d < nd ? ld(arow[q], d0 + d) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db + u * 64 + lane;
        if (d >= nd) continue;
#pragma unroll
        for (int c = 0; c < CMAX; ++c) {
          if (c >= C) continue;
          const float wdc = Ws[d * C + c];
#pragma unroll
          for (int q = 0; q < RPW; ++q) z[q][c] = __builtin_fmaf(av[u][q], wdc, z[q][c]);
        }
      }
    }
  }
  const float* bias = h.bias + (long long)k * h.sBias;
  const float invB = 1.0f / (float)h.B;
  float dz[RPW][CMAX];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
#pragma unroll
    for (int c = 0; c < CMAX; ++c)
      if (c < C) z[q][c] = wave_sum(z[q][c]) + bias[c];
    // softmax cross-entropy, identical in every lane
    const int lab = h.y[h.rowmap[rr[q]]];
    float m = z[q][0];
#pragma unroll
    for (int c = 1; c < CMAX; ++c)
      if (c < C) m = fmaxf(m, z[q][c]);
    float s = 0.f, rest = 0.f, zy = 0.f;
#pragma unroll
    for (int c = 0; c < CMAX; ++c)
      if (c < C) {
        const float e = __expf(z[q][c] - m);
        s += e;
        if (c != lab) rest += e;
        else zy = z[q][c];
      }
    const float loss = zy >= m ? log1pf(rest) : (m - zy) + logf(s);
    const float inv_s = 1.0f / s;
    float mine = 0.f;
#pragma unroll
    for (int c = 0; c < CMAX; ++c) {
      dz[q][c] = 0.f;
      if (c < C) {
        const float p = __expf(z[q][c] - m) * inv_s;
        dz[q][c] = round_like((p - (c == lab ? 1.f : 0.f)) * invB, (const T*)nullptr);
        if (c == lane) mine = dz[q][c];
      }
    }
    if (live[q]) {
      if (lane < C) st((T*)h.dZ, rr[q] * C + lane, mine);
      if (lane == 0) h.rowloss[rr[q]] = loss;
    }
  }

  if (!h.dZprev) return;  // uniform over the workgroup
  // input gradient of the top layer, ReLU-masked: needs W_L again
  for (int d0 = 0; d0 < D; d0 += DCH) {
    const int nd = min(DCH, D - d0);
    if (D > DCH) {  // the chunk in LDS is not the whole of W_L
      __syncthreads();
      stage(Ws, Wg, (long long)d0 * C, nd * C);
      __syncthreads();
    }
    for (int db = 0; db < nd; db += 256) {
      float mk[4][RPW];  // the ReLU mask operand, loaded up front
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db + u * 64 + lane;
#pragma unroll
        for (int q = 0; q < RPW; ++q)
          mk[u][q] = d < nd && live[q] ? ld(arow[q], d0 + d) : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = db + u * 64 + lane;
        if (d >= nd) continue;
        float v[RPW];
#pragma unroll
        for (int q = 0; q < RPW; ++q) v[q] = 0.f;
#pragma unroll
        for (int c = 0; c < CMAX; ++c) {
          if (c >= C) continue;
          const float wdc = Ws[d * C + c];
#pragma unroll
          for (int q = 0; q < RPW; ++q) v[q] = __builtin_fmaf(dz[q][c], wdc, v[q]);
        }
#pragma unroll
        for (int q = 0; q < RPW; ++q)
          if (live[q])
            st((T*)h.dZprev + rr[q] * D, d0 + d,
               (h.nomask || mk[u][q] > 0.f) ? v[q] : 0.f);
      }
    }
  }
}

template <typename T, int CMAX, bool GATHER>
__global__ __launch_bounds__(256) void k_head_wgrad(HeadArgs h) {
  constexpr int RB = 64;  // batch rows staged in LDS per pass
  constexpr int CJ = (CMAX + 3) / 4;
  __shared__ float dzs[RB * CMAX];
  __shared__ float As[RB][65];
  __shared__ float red[256];
  const int k = blockIdx.y;
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int D = h.D, C = h.C, B = h.B;
  const int dbase = blockIdx.x * 64, d = dbase + lane;
  const T* dZ = (const T*)h.dZ + (long long)k * B * C;
  const bool first = blockIdx.x == 0;

  float acc[CJ];
#pragma unroll
  for (int j = 0; j < CJ; ++j) acc[j] = 0.f;
  float bsum = 0.f;  // bias gradient of class threadIdx.x (first workgroup)
  for (int b0 = 0; b0 < B; b0 += RB) {
    const int nb = min(RB, B - b0);
    __syncthreads();
    stage(dzs, dZ, (long long)b0 * C, nb * C);
    // A[b0 + r][dbase .. dbase + 63]: each wave loads whole 64-wide rows,
    // eight rows per batch with every load issued before the LDS stores
    for (int r0 = grp; r0 < nb; r0 += 32) {
      long long base[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int r = r0 + 4 * u;
        const long long rr = (long long)k * B + b0 + (r < nb ? r : 0);
        base[u] = GATHER ? (long long)h.rowmap[rr] * D
                         : (long long)k * h.sA + (long long)(b0 + (r < nb ? r : 0)) * D;
      }
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[u] = (r0 + 4 * u < nb && d < D) ? ld((const T*)h.A, base[u] + d) : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (r0 + 4 * u < nb) As[r0 + 4 * u][lane] = v[u];
    }
    __syncthreads();
#pragma unroll 4
    for (int b = 0; b < nb; ++b) {
      const float av = As[b][lane];
#pragma unroll
      for (int j = 0; j < CJ; ++j) {
        const int c = grp + 4 * j;
        if (c < C) acc[j] = __builtin_fmaf(av, dzs[b * C + c], acc[j]);
      }
    }
    if (first && (int)threadIdx.x < C)
      for (int b = 0; b < nb; ++b) bsum += dzs[b * C + threadIdx.x];
  }
  if (d < D) {
#pragma unroll
    for (int j = 0; j < CJ; ++j) {
      const int c = grp + 4 * j;
      if (c >= C) continue;
      const long long o = (long long)k * h.sP + (long long)d * C + c;
      float w = h.Wsrc[(long long)k * h.sSrc + (long long)d * C + c], u = h.Um[o];
      sgd_step(w, u, acc[j], h);
      h.Wm[o] = w;
      h.Um[o] = u;
      if (h.Wb) h.Wb[o] = f32_to_bf16(w);
    }
  }
  if (!first) return;  // uniform over the workgroup
  if ((int)threadIdx.x < C) {
    const long long o = (long long)k * h.sP + threadIdx.x;
    float w = h.bsrc[(long long)k * h.sSrc + threadIdx.x], u = h.bias_u[o];
    sgd_step(w, u, bsum, h);
    h.bias_w[o] = w;
    h.bias_u[o] = u;
  }
  // mean loss of replica k: per-thread strided partial sums, then a fixed tree
  const float* rl = h.rowloss + (long long)k * B;
  float part = 0.f;
  for (int b = threadIdx.x; b < B; b += 256) part += rl[b];
  red[threadIdx.x] = part;
  __syncthreads();
  for (int w2 = 128; w2 > 0; w2 >>= 1) {
    if ((int)threadIdx.x < w2) red[threadIdx.x] += red[threadIdx.x + w2];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float mean = red[0] / (float)B;
    if (h.loss) h.loss[k] = mean;
    // a non-finite loss raises the context's flag (a plain store: every
    // writer stores the same value)
    if (h.nonfinite && !isfinite(mean)) *h.nonfinite = 1;
  }
}

// Weight gradient of the output layer in one memory round trip (fp32,
// C <= CM, D % 64 == 0, B <= 128): workgroup (x, k) owns inputs
// d = 64 x .. 64 x + 63 of replica k. Every load -- the activations A[b][d]
// of the lane's d for the group's rows b = grp + 4 r, dZ, this slice of W_L
// and U_L, the per-row losses -- is issued up front. Each of the 4 thread
// groups sums its quarter of the batch (rows grp, grp + 4, ... ascending);
// the four partials are then added in group order and the SGD step applied.
// Workgroup 0 of each replica also updates the bias and reduces the loss.
template <int CM, bool GATHER>
__global__ __launch_bounds__(256) void k_head_wgrad_vec(HeadArgs h) {
  constexpr int RPG = 32;                 // rows per group: B <= 128
  constexpr int WPT = (64 * CM + 255) / 256;  // weights per thread
  constexpr int ZPT = (128 * CM + 255) / 256; // dZ values per thread
  __shared__ float dzs[128 * CM];
  __shared__ float part[4][64][CM + 1];
  __shared__ float red[256];
  const int k = blockIdx.y;
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int D = h.D, C = h.C, B = h.B;
  const int dbase = blockIdx.x * 64, d = dbase + lane;
  const bool first = blockIdx.x == 0;
  const float* dZ = (const float*)h.dZ + (long long)k * B * C;

  // 1. all loads in flight together (clamped indices, values masked at use)
  float av[RPG];
#pragma unroll
  for (int r = 0; r < RPG; ++r) {
    const int b = min(grp + 4 * r, B - 1);
    const long long row = GATHER ? (long long)h.rowmap[(long long)k * B + b]
                                 : (long long)k * (h.sA / D) + b;
    av[r] = ((const float*)h.A)[row * D + d];
  }
  float zv[ZPT];
#pragma unroll
  for (int q = 0; q < ZPT; ++q) zv[q] = dZ[min((int)threadIdx.x + 256 * q, B * C - 1)];
  float wv[WPT], uv[WPT];
  const long long wbase = (long long)k * h.sP + (long long)dbase * C;
#pragma unroll
  for (int q = 0; q < WPT; ++q) {
    const int e = min((int)threadIdx.x + 256 * q, 64 * C - 1);
    wv[q] = h.Wsrc[(long long)k * h.sSrc + (long long)dbase * C + e];
    uv[q] = h.Um[wbase + e];
  }
  const float rl = first ? h.rowloss[(long long)k * B + min((int)threadIdx.x, B - 1)] : 0.f;

  // 2. dZ to LDS
#pragma unroll
  for (int q = 0; q < ZPT; ++q) {
    const int i = (int)threadIdx.x + 256 * q;
    if (i < B * C) dzs[i] = zv[q];
  }
  __syncthreads();

  // 3. this group's rows
  float acc[CM];
#pragma unroll
  for (int c = 0; c < CM; ++c) acc[c] = 0.f;
#pragma unroll
  for (int r = 0; r < RPG; ++r) {
    const int b = grp + 4 * r;
    if (b < B) {
#pragma unroll
      for (int c = 0; c < CM; ++c)
        if (c < C) acc[c] = __builtin_fmaf(av[r], dzs[b * C + c], acc[c]);
    }
  }
#pragma unroll
  for (int c = 0; c < CM; ++c) part[grp][lane][c] = acc[c];
  __syncthreads();

  // 4. partials in group order, SGD step on W_L[d][c]
#pragma unroll
  for (int q = 0; q < WPT; ++q) {
    const int e = (int)threadIdx.x + 256 * q;
    if (e < 64 * C) {
      const int dl = e / C, c = e - dl * C;
      const float g = ((part[0][dl][c] + part[1][dl][c]) + part[2][dl][c]) + part[3][dl][c];
      float w = wv[q], u = uv[q];
      sgd_step(w, u, g, h);
      h.Wm[wbase + e] = w;
      h.Um[wbase + e] = u;
    }
  }
  if (!first) return;  // uniform over the workgroup
  if ((int)threadIdx.x < C) {
    float bsum = 0.f;
    for (int b = 0; b < B; ++b) bsum += dzs[b * C + threadIdx.x];
    const long long o = (long long)k * h.sP + threadIdx.x;
    float w = h.bsrc[(long long)k * h.sSrc + threadIdx.x], u = h.bias_u[o];
    sgd_step(w, u, bsum, h);
    h.bias_w[o] = w;
    h.bias_u[o] = u;
  }
  red[threadIdx.x] = (int)threadIdx.x < B ? rl : 0.f;
  __syncthreads();
  for (int w2 = 128; w2 > 0; w2 >>= 1) {
    if ((int)threadIdx.x < w2) red[threadIdx.x] += red[threadIdx.x + w2];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float mean = red[0] / (float)B;
    if (h.loss) h.loss[k] = mean;
    // a non-finite loss raises the context's flag (a plain store: every
    // writer stores the same value)
    if (h.nonfinite && !isfinite(mean)) *h.nonfinite = 1;
  }
}

// Register-resident variant for fp32, a class count fixed at compile time,
// D % 256 == 0 and D <= 512: lane l
// owns inputs d = 256 j + 4 l .. +3 (j < D / 256) of two sample rows and the
// matching rows W_L[d][0..C-1]; all of them are loaded in one batch, so the
// logits, the loss, dZ and the masked input gradient cost one memory round
// trip. The loss and gradient formulas are those of k_head_fwd; only the
// split of the logit sums over lanes differs (each lane's inputs in ascending
// d, then the same xor butterfly).
template <int C, int NJ>
__global__ __launch_bounds__(256) void k_head_fwd_vec(HeadArgs h) {
  constexpr int RPW = 2;
  const int k = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int D = h.D;
  const float* Wg = (const float*)h.W + (long long)k * h.sW;
  long long rr[RPW];
  bool live[RPW];
  float4 a[RPW][NJ];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int row = (blockIdx.x * 4 + wave) * RPW + q;
    live[q] = row < h.B;
    rr[q] = (long long)k * h.B + (live[q] ? row : 0);
    const float* arow = (const float*)h.A + (long long)k * h.sA +
                        (long long)(live[q] ? row : 0) * D;
#pragma unroll
    for (int j = 0; j < NJ; ++j) a[q][j] = *(const float4*)(arow + 256 * j + 4 * lane);
  }
  // W rows d .. d+3 are 4*C consecutive floats (C float4 when C is even)
  static_assert(C % 2 == 0 && C <= 16, "class count");
  float wr[NJ][4 * C];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const float* wp = Wg + (long long)(256 * j + 4 * lane) * C;
#pragma unroll
    for (int v = 0; v < C; ++v) {
      const float4 t = *(const float4*)(wp + 4 * v);
      wr[j][4 * v] = t.x;
      wr[j][4 * v + 1] = t.y;
      wr[j][4 * v + 2] = t.z;
      wr[j][4 * v + 3] = t.w;
    }
  }
  float z[RPW][C];
#pragma unroll
  for (int q = 0; q < RPW; ++q)
#pragma unroll
    for (int c = 0; c < C; ++c) {
      float acc = 0.f;
      {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          acc = __builtin_fmaf(a[q][j].x, wr[j][0 * C + c], acc);
          acc = __builtin_fmaf(a[q][j].y, wr[j][1 * C + c], acc);
          acc = __builtin_fmaf(a[q][j].z, wr[j][2 * C + c], acc);
          acc = __builtin_fmaf(a[q][j].w, wr[j][3 * C + c], acc);
        }
      }
      z[q][c] = acc;
    }
  const float* bias = h.bias + (long long)k * h.sBias;
  const float invB = 1.0f / (float)h.B;
  float dz[RPW][C];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
#pragma unroll
    for (int c = 0; c < C; ++c)
      z[q][c] = wave_sum(z[q][c]) + bias[c];
    const int lab = h.y[h.rowmap[rr[q]]];
    float m = z[q][0];
#pragma unroll
    for (int c = 1; c < C; ++c)
      m = fmaxf(m, z[q][c]);
    float sum = 0.f, rest = 0.f, zy = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c)
      {
        const float e = __expf(z[q][c] - m);
        sum += e;
        if (c != lab) rest += e;
        else zy = z[q][c];
      }
    const float loss = zy >= m ? log1pf(rest) : (m - zy) + logf(sum);
    const float inv_s = 1.0f / sum;
    float mine = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      dz[q][c] = 0.f;
      {
        const float p = __expf(z[q][c] - m) * inv_s;
        dz[q][c] = (p - (c == lab ? 1.f : 0.f)) * invB;
        if (c == lane) mine = dz[q][c];
      }
    }
    if (live[q]) {
      if (lane < C) ((float*)h.dZ)[rr[q] * C + lane] = mine;
      if (lane == 0) h.rowloss[rr[q]] = loss;
    }
  }
  if (!h.dZprev) return;
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    if (!live[q]) continue;
    float* out = (float*)h.dZprev + rr[q] * D;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < C; ++c)
          acc = __builtin_fmaf(dz[q][c], wr[j][e * C + c], acc);
        v[e] = acc;
      }
      const float4 av = a[q][j];
      float4 o;
      o.x = (h.nomask || av.x > 0.f) ? v[0] : 0.f;
      o.y = (h.nomask || av.y > 0.f) ? v[1] : 0.f;
      o.z = (h.nomask || av.z > 0.f) ? v[2] : 0.f;
      o.w = (h.nomask || av.w > 0.f) ? v[3] : 0.f;
      *(float4*)(out + 256 * j + 4 * lane) = o;
    }
  }
}

// bf16 form: the bf16 copy of W_L and bf16 activations, a class count C
// fixed at compile time and D = 512 NJ. The replica's W_L ([D][C] bf16, D C / 8
// 16-byte words) is copied into LDS unchanged, every word loaded before the
// first is stored; lane l of a wave owns inputs d = 512 j + 8 l .. +7 of two
// sample rows, loaded in the same batch. The logits, the loss, dZ and the
// masked input gradient then need no further global read. Formulas and
// rounding points (dZ and the input gradient rounded to bf16) are those of
// k_head_fwd; each lane adds its inputs in ascending d before the xor
// butterfly.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) {
  return __uint_as_float(w & 0xFFFF0000u);
}
__device__ __forceinline__ float bf16_at(const uint4& v, int e) {
  const uint32_t w = e < 2 ? v.x : (e < 4 ? v.y : (e < 6 ? v.z : v.w));
  return (e & 1) ? bf16_hi(w) : bf16_lo(w);
}

template <int C, int NJ>
__global__ __launch_bounds__(256) void k_head_fwd_bf16(HeadArgs h) {
  constexpr int RPW = 2;
  constexpr int D = 512 * NJ;
  constexpr int WV = D * C / 8;            // 16-byte words of W_L
  constexpr int WPT = (WV + 255) / 256;    // per thread
  __shared__ uint4 Ws[WV];
  const int k = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint4* Wg = (const uint4*)((const bf16_t*)h.W + (long long)k * h.sW);
  uint4 wv[WPT];
#pragma unroll
  for (int u = 0; u < WPT; ++u) {
    const int i = u * 256 + (int)threadIdx.x;
    wv[u] = i < WV ? Wg[i] : make_uint4(0u, 0u, 0u, 0u);
  }
  long long rr[RPW];
  bool live[RPW];
  uint4 a[RPW][NJ];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
    const int row = (blockIdx.x * 4 + wave) * RPW + q;
    live[q] = row < h.B;
    rr[q] = (long long)k * h.B + (live[q] ? row : 0);
    const bf16_t* arow = (const bf16_t*)h.A + (long long)k * h.sA +
                         (long long)(live[q] ? row : 0) * D;
#pragma unroll
    for (int j = 0; j < NJ; ++j) a[q][j] = *(const uint4*)(arow + 512 * j + 8 * lane);
  }
#pragma unroll
  for (int u = 0; u < WPT; ++u) {
    const int i = u * 256 + (int)threadIdx.x;
    if (i < WV) Ws[i] = wv[u];
  }
  __syncthreads();
  // W_L[d][c] for the lane's d = 512 j + 8 l + t: element t C + c of the C
  // words starting at word (64 j + l) C
  float z[RPW][C];
#pragma unroll
  for (int q = 0; q < RPW; ++q)
#pragma unroll
    for (int c = 0; c < C; ++c) z[q][c] = 0.f;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    uint4 w[C];
#pragma unroll
    for (int v = 0; v < C; ++v) w[v] = Ws[(64 * j + lane) * C + v];
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
      for (int c = 0; c < C; ++c) {
        const int e = t * C + c;
        const float wdc = bf16_at(w[e / 8], e % 8);
#pragma unroll
        for (int q = 0; q < RPW; ++q)
          z[q][c] = __builtin_fmaf(bf16_at(a[q][j], t), wdc, z[q][c]);
      }
    __builtin_amdgcn_sched_barrier(0);  // one slice of W_L in registers at a time
  }
  const float* bias = h.bias + (long long)k * h.sBias;
  const float invB = 1.0f / (float)h.B;
  float dz[RPW][C];
#pragma unroll
  for (int q = 0; q < RPW; ++q) {
#pragma unroll
    for (int c = 0; c < C; ++c) z[q][c] = wave_sum(z[q][c]) + bias[c];
    const int lab = h.y[h.rowmap[rr[q]]];
    float m = z[q][0];
#pragma unroll
    for (int c = 1; c < C; ++c) m = fmaxf(m, z[q][c]);
    float sum = 0.f, rest = 0.f, zy = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const float e = __expf(z[q][c] - m);
      sum += e;
      if (c != lab) rest += e;
      else zy = z[q][c];
    }
    const float loss = zy >= m ? log1pf(rest) : (m - zy) + logf(sum);
    const float inv_s = 1.0f / sum;
    float mine = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const float p = __expf(z[q][c] - m) * inv_s;
      dz[q][c] = round_like((p - (c == lab ? 1.f : 0.f)) * invB, (const bf16_t*)nullptr);
      if (c == lane) mine = dz[q][c];
    }
    if (live[q]) {
      if (lane < C) ((bf16_t*)h.dZ)[rr[q] * C + lane] = f32_to_bf16(mine);
      if (lane == 0) h.rowloss[rr[q]] = loss;
    }
  }
  if (!h.dZprev) return;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    uint4 w[C];
#pragma unroll
    for (int v = 0; v < C; ++v) w[v] = Ws[(64 * j + lane) * C + v];
#pragma unroll
    for (int q = 0; q < RPW; ++q) {
      if (!live[q]) continue;
      uint32_t o[4];
#pragma unroll
      for (int t2 = 0; t2 < 4; ++t2) {
        uint32_t pair = 0u;
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
          const int t = 2 * t2 + hb;
          float acc = 0.f;
#pragma unroll
          for (int c = 0; c < C; ++c) {
            const int e = t * C + c;
            acc = __builtin_fmaf(dz[q][c], bf16_at(w[e / 8], e % 8), acc);
          }
          const float out = (h.nomask || bf16_at(a[q][j], t) > 0.f) ? acc : 0.f;
          pair |= (uint32_t)f32_to_bf16(out) << (16 * hb);
        }
        o[t2] = pair;
      }
      *(uint4*)((bf16_t*)h.dZprev + rr[q] * D + 512 * j + 8 * lane) =
          make_uint4(o[0], o[1], o[2], o[3]);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <typename T, int CMAX>
hipError_t launch_pair(const HeadArgs& h, hipStream_t s, int which) {
  const bool gather = h.gather != 0;  // the top layer is layer 1
  if (which == 0) {
    dim3 grid((h.B + 7) / 8, h.K);  // 4 waves x 2 rows per workgroup
    if (gather)
      hipLaunchKernelGGL((k_head_fwd<T, CMAX, true>), grid, dim3(256), 0, s, h);
    else
      hipLaunchKernelGGL((k_head_fwd<T, CMAX, false>), grid, dim3(256), 0, s, h);
  } else {
    dim3 grid((h.D + 63) / 64, h.K);
    if (gather)
      hipLaunchKernelGGL((k_head_wgrad<T, CMAX, true>), grid, dim3(256), 0, s, h);
    else
      hipLaunchKernelGGL((k_head_wgrad<T, CMAX, false>), grid, dim3(256), 0, s, h);
  }
  return hipGetLastError();
}

bool al16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

hipError_t launch_head(int dtype, const HeadArgs& h, hipStream_t s, int which) {
  if (h.C < 1 || h.C > kHeadMaxClasses) return hipErrorInvalidValue;
  if (h.K > 65535 || h.B < 1 || h.D < 1) return hipErrorInvalidValue;
  // register-resident forward when the shapes and alignment allow it
  if (which == 0 && dtype == 0 && !h.gather && h.C == 10 && h.D % 256 == 0 &&
      h.D <= 512 && h.sA % 4 == 0 && h.sW % 4 == 0 && al16(h.A) && al16(h.W) &&
      (h.dZprev == nullptr || al16(h.dZprev))) {
    dim3 grid((h.B + 7) / 8, h.K);
    if (h.D == 256)
      hipLaunchKernelGGL((k_head_fwd_vec<10, 1>), grid, dim3(256), 0, s, h);
    else
      hipLaunchKernelGGL((k_head_fwd_vec<10, 2>), grid, dim3(256), 0, s, h);
    return hipGetLastError();
  }
  // the same for bf16 operands, D a multiple of 512 up to 2048
  if (which == 0 && dtype == 1 && !h.gather && h.C == 10 && h.D % 512 == 0 &&
      h.D <= 2048 && h.sA % 8 == 0 && h.sW % 8 == 0 && al16(h.A) && al16(h.W) &&
      (h.dZprev == nullptr || al16(h.dZprev))) {
    dim3 grid((h.B + 7) / 8, h.K);
    switch (h.D / 512) {
      case 1: hipLaunchKernelGGL((k_head_fwd_bf16<10, 1>), grid, dim3(256), 0, s, h); break;
      case 2: hipLaunchKernelGGL((k_head_fwd_bf16<10, 2>), grid, dim3(256), 0, s, h); break;
      case 3: hipLaunchKernelGGL((k_head_fwd_bf16<10, 3>), grid, dim3(256), 0, s, h); break;
      default: hipLaunchKernelGGL((k_head_fwd_bf16<10, 4>), grid, dim3(256), 0, s, h); break;
    }
    return hipGetLastError();
  }
  // one-round-trip weight gradient: fp32, up to 16 classes, 64-input slices
  if (which == 1 && dtype == 0 && h.C <= 16 && h.D % 64 == 0 && h.B <= 128 &&
      h.Wb == nullptr && (h.gather || h.sA % h.D == 0)) {
    dim3 grid(h.D / 64, h.K);
    if (h.C == 10 && h.gather)
      hipLaunchKernelGGL((k_head_wgrad_vec<10, true>), grid, dim3(256), 0, s, h);
    else if (h.C == 10)
      hipLaunchKernelGGL((k_head_wgrad_vec<10, false>), grid, dim3(256), 0, s, h);
    else if (h.gather)
      hipLaunchKernelGGL((k_head_wgrad_vec<16, true>), grid, dim3(256), 0, s, h);
    else
      hipLaunchKernelGGL((k_head_wgrad_vec<16, false>), grid, dim3(256), 0, s, h);
    return hipGetLastError();
  }
  if (dtype == 1)
    return h.C <= 16 ? launch_pair<bf16_t, 16>(h, s, which)
                     : launch_pair<bf16_t, 32>(h, s, which);
  return h.C <= 16 ? launch_pair<float, 16>(h, s, which)
                   : launch_pair<float, 32>(h, s, which);
}

}  // namespace

hipError_t launch_head_fwd(int dtype, const HeadArgs& h, hipStream_t s) {
  return launch_head(dtype, h, s, 0);
}
hipError_t launch_head_wgrad(int dtype, const HeadArgs& h, hipStream_t s) {
  return launch_head(dtype, h, s, 1);
}

}  // namespace lsgd
