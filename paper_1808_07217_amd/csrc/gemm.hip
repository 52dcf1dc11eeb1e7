// Grouped (replica-batched) GEMM on the gfx950 matrix cores.
//
// Each of the G groups is one replica's layer contraction of the gradient in
// eq. 2 of the paper: forward Z = A W (+ bias, ReLU), the input gradient
// dA = dZ W^T (masked by the ReLU derivative), and the weight gradient
// G = A^T dZ, whose epilogue applies the local momentum-SGD update directly so
// the gradient never goes to memory.
//
// Block tile BM x BN x BK, 256 threads = 4 wavefronts in a 2 x 2 layout, each
// wave owning (BM/2) x (BN/2) as 32 x 32 MFMA blocks. Operands are staged
// global -> registers -> LDS with a double-buffered LDS ring: the next slab's
// global loads are in flight while the current slab feeds the MFMAs.
//
//  fp32: v_mfma_f32_32x32x2f32, BK = 16. LDS holds k-major tiles As[k][m],
//        Bs[k][n]; lane l feeds A[m = l%32][k = l/32], B[k = l/32][n = l%32].
//  bf16: v_mfma_f32_32x32x16_bf16, BK = 32. LDS holds k-contiguous rows
//        As[m][k], Bs[n][k]; lane l feeds 8 consecutive k starting at
//        8*(l/32) for row/column l%32.
//  Both: accumulator register v of lane l is C[8*(v/4) + 4*(l/32) + v%4][l%32].
#include "kernels.h"

namespace lsgd {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;

template <int EPI, bool OUTBF>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int g, int m, int n,
                                         float acc) {
  const long long o = (long long)g * a.sC + (long long)m * a.ldc + n;
  if constexpr (EPI == EPI_SGD) {
    float w = a.W[o];
    float u = a.U[o];
    float gr = __builtin_fmaf(a.wd, w, acc);
    u = __builtin_fmaf(a.mom, u, gr);
    float d = a.nesterov ? __builtin_fmaf(a.mom, u, gr) : u;
    w = __builtin_fmaf(-a.lr, d, w);
    a.W[o] = w;
    a.U[o] = u;
    if (a.Wb) a.Wb[o] = f32_to_bf16(w);
    return;
  } else {
    float v = acc;
    if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_RELU)
      v += a.bias[(long long)g * a.sBias + n];
    if constexpr (EPI == EPI_BIAS_RELU) v = v > 0.f ? v : 0.f;
    if constexpr (EPI == EPI_RELU_MASK) {
      float mk = OUTBF ? bf16_to_f32(((const bf16_t*)a.mask)[o])
                       : ((const float*)a.mask)[o];
      v = mk > 0.f ? v : 0.f;
    }
    if constexpr (OUTBF)
      ((bf16_t*)a.C)[o] = f32_to_bf16(v);
    else
      ((float*)a.C)[o] = v;
  }
}

// ------------------------------------------------------------------ fp32
template <bool AT, bool BT, int EPI, bool GATHER, int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_f32(GemmArgs a, int vecA,
                                                     int vecB) {
  constexpr int BK = 16, PAD = 4;
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 32, FN = WN / 32;
  constexpr int NA = BM * BK / 4 / kThreads;  // float4 loads per thread
  constexpr int NB = BN * BK / 4 / kThreads;
  static_assert(NA >= 1 && NB >= 1, "tile too small for 256 threads");
  __shared__ float As[2][BK][BM + PAD];
  __shared__ float Bs[2][BK][BN + PAD];

  const int g = blockIdx.z;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;
  const float* A = (const float*)a.A + (long long)g * a.sA;
  const float* B = (const float*)a.B + (long long)g * a.sB;
  // GATHER: rows of A come from a row map (the sampled mini-batch indices)
  const int32_t* rmap = GATHER ? a.rowmap + (long long)g * a.sRow : nullptr;
  const int M = a.M, N = a.N, Kd = a.Kd;

  float4 ra[NA], rb[NB];

  // Load 4 consecutive elements of storage row `row` starting at column
  // `col`; `avail` elements are valid, the rest read as zero.
  auto load4 = [](const float* p, int avail, int vec) -> float4 {
    if (vec && avail >= 4) return *(const float4*)p;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (avail > 0) v.x = p[0];
    if (avail > 1) v.y = p[1];
    if (avail > 2) v.z = p[2];
    if (avail > 3) v.w = p[3];
    return v;
  };

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (!AT) {  // storage [M][Kd]: rows m, 4 float4 per row
        const int r = q >> 2, c = k0 + (q & 3) * 4, row = m0 + r;
        ra[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row < M) {
          const long long sr = GATHER ? rmap[row] : row;
          ra[i] = load4(A + sr * a.lda + c, Kd - c, vecA);
        }
      } else {  // storage [Kd][M]: rows k, BM/4 float4 per row
        const int r = q / (BM / 4), c = m0 + (q % (BM / 4)) * 4, kr = k0 + r;
        ra[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (kr < Kd) {
          const long long sr = GATHER ? rmap[kr] : kr;
          ra[i] = load4(A + sr * a.lda + c, M - c, vecA);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT) {  // storage [N][Kd]
        const int r = q >> 2, c = k0 + (q & 3) * 4, row = n0 + r;
        rb[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row < N) rb[i] = load4(B + (long long)row * a.ldb + c, Kd - c, vecB);
      } else {  // storage [Kd][N]
        const int r = q / (BN / 4), c = n0 + (q % (BN / 4)) * 4, kr = k0 + r;
        rb[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (kr < Kd) rb[i] = load4(B + (long long)kr * a.ldb + c, N - c, vecB);
      }
    }
  };

  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (!AT) {
        const int r = q >> 2, kq = (q & 3) * 4;
        As[buf][kq + 0][r] = ra[i].x;
        As[buf][kq + 1][r] = ra[i].y;
        As[buf][kq + 2][r] = ra[i].z;
        As[buf][kq + 3][r] = ra[i].w;
      } else {
        const int r = q / (BM / 4), c = (q % (BM / 4)) * 4;
        *(float4*)&As[buf][r][c] = ra[i];
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT) {
        const int r = q >> 2, kq = (q & 3) * 4;
        Bs[buf][kq + 0][r] = rb[i].x;
        Bs[buf][kq + 1][r] = rb[i].y;
        Bs[buf][kq + 2][r] = rb[i].z;
        Bs[buf][kq + 3][r] = rb[i].w;
      } else {
        const int r = q / (BN / 4), c = (q % (BN / 4)) * 4;
        *(float4*)&Bs[buf][r][c] = rb[i];
      }
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = (Kd + BK - 1) / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  const int lk = lane >> 5, lr = lane & 31;
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) gload((t + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 2) {
      float av[FM], bv[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) av[i] = As[buf][kk + lk][wm0 + i * 32 + lr];
#pragma unroll
      for (int j = 0; j < FN; ++j) bv[j] = Bs[buf][kk + lk][wn0 + j * 32 + lr];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j],
                                                           acc[i][j], 0, 0, 0);
    }
    if (t + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm0 + i * 32 + (v >> 2) * 8 + lk * 4 + (v & 3);
        const int n = n0 + wn0 + j * 32 + lr;
        if (m < M && n < N) epilogue<EPI, false>(a, g, m, n, acc[i][j][v]);
      }
}

// ------------------------------------------------------------------ bf16
template <bool AT, bool BT, int EPI, bool GATHER, int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_bf16(GemmArgs a, int vecA,
                                                      int vecB) {
  constexpr int BK = 32, KP = BK + 8;  // row pitch 80 B keeps 16-B alignment
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 32, FN = WN / 32;
  constexpr int NA = BM * BK / 8 / kThreads;  // 8-element vectors per thread
  constexpr int NB = BN * BK / 8 / kThreads;
  static_assert(NA >= 1 && NB >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][KP];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][KP];

  const int g = blockIdx.z;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;
  const bf16_t* A = (const bf16_t*)a.A + (long long)g * a.sA;
  const bf16_t* B = (const bf16_t*)a.B + (long long)g * a.sB;
  // GATHER: rows of A come from a row map (the sampled mini-batch indices)
  const int32_t* rmap = GATHER ? a.rowmap + (long long)g * a.sRow : nullptr;
  const int M = a.M, N = a.N, Kd = a.Kd;

  uint4 ra[NA], rb[NB];

  auto load8 = [](const bf16_t* p, int avail, int vec) -> uint4 {
    if (vec && avail >= 8) return *(const uint4*)p;
    uint16_t t[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = e < avail ? p[e] : (uint16_t)0;
    return make_uint4(t[0] | ((uint32_t)t[1] << 16), t[2] | ((uint32_t)t[3] << 16),
                      t[4] | ((uint32_t)t[5] << 16), t[6] | ((uint32_t)t[7] << 16));
  };

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      ra[i] = make_uint4(0, 0, 0, 0);
      if constexpr (!AT) {  // [M][Kd]: 4 vectors per row
        const int r = q >> 2, c = k0 + (q & 3) * 8, row = m0 + r;
        if (row < M) {
          const long long sr = GATHER ? rmap[row] : row;
          ra[i] = load8(A + sr * a.lda + c, Kd - c, vecA);
        }
      } else {  // [Kd][M]: BM/8 vectors per row
        const int r = q / (BM / 8), c = m0 + (q % (BM / 8)) * 8, kr = k0 + r;
        if (kr < Kd) {
          const long long sr = GATHER ? rmap[kr] : kr;
          ra[i] = load8(A + sr * a.lda + c, M - c, vecA);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      rb[i] = make_uint4(0, 0, 0, 0);
      if constexpr (BT) {  // [N][Kd]
        const int r = q >> 2, c = k0 + (q & 3) * 8, row = n0 + r;
        if (row < N) rb[i] = load8(B + (long long)row * a.ldb + c, Kd - c, vecB);
      } else {  // [Kd][N]
        const int r = q / (BN / 8), c = n0 + (q % (BN / 8)) * 8, kr = k0 + r;
        if (kr < Kd) rb[i] = load8(B + (long long)kr * a.ldb + c, N - c, vecB);
      }
    }
  };

  auto scatter = [](bf16_t (*T)[KP], int r0, int k, uint4 v) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      T[r0 + 2 * e][k] = (bf16_t)(w[e] & 0xFFFFu);
      T[r0 + 2 * e + 1][k] = (bf16_t)(w[e] >> 16);
    }
  };

  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (!AT) {
        const int r = q >> 2, c = (q & 3) * 8;
        *(uint4*)&As[buf][r][c] = ra[i];
      } else {
        const int r = q / (BM / 8), c = (q % (BM / 8)) * 8;
        scatter(As[buf], c, r, ra[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT) {
        const int r = q >> 2, c = (q & 3) * 8;
        *(uint4*)&Bs[buf][r][c] = rb[i];
      } else {
        const int r = q / (BN / 8), c = (q % (BN / 8)) * 8;
        scatter(Bs[buf], c, r, rb[i]);
      }
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = (Kd + BK - 1) / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  const int lk = lane >> 5, lr = lane & 31;
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) gload((t + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 av[FM], bv[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        av[i] = *(const bf16x8*)&As[buf][wm0 + i * 32 + lr][kk + lk * 8];
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bv[j] = *(const bf16x8*)&Bs[buf][wn0 + j * 32 + lr][kk + lk * 8];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j],
                                                              acc[i][j], 0, 0, 0);
    }
    if (t + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm0 + i * 32 + (v >> 2) * 8 + lk * 4 + (v & 3);
        const int n = n0 + wn0 + j * 32 + lr;
        if (m < M && n < N) {
          if constexpr (EPI == EPI_BIAS_RELU || EPI == EPI_RELU_MASK)
            epilogue<EPI, true>(a, g, m, n, acc[i][j][v]);
          else
            epilogue<EPI, false>(a, g, m, n, acc[i][j][v]);
        }
      }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

template <bool AT, bool BT, int EPI, bool GATHER = false>
hipError_t dispatch(int dtype, const GemmArgs& a, hipStream_t s) {
  if (GATHER != (a.rowmap != nullptr)) {
    if (a.rowmap) return dispatch<AT, BT, EPI, true>(dtype, a, s);
    return hipErrorInvalidValue;
  }
  constexpr int BM = 64, BN = 64;
  dim3 grid((a.N + BN - 1) / BN, (a.M + BM - 1) / BM, a.G);
  const int esz = dtype == 1 ? 8 : 4;  // elements per vector load
  const int vecA = a.lda % esz == 0 && a.sA % esz == 0 && aligned16(a.A);
  const int vecB = a.ldb % esz == 0 && a.sB % esz == 0 && aligned16(a.B);
  if (dtype == 1)
    hipLaunchKernelGGL((gemm_bf16<AT, BT, EPI, GATHER, BM, BN>), grid, dim3(kThreads),
                       0, s, a, vecA, vecB);
  else
    hipLaunchKernelGGL((gemm_f32<AT, BT, EPI, GATHER, BM, BN>), grid, dim3(kThreads),
                       0, s, a, vecA, vecB);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int dtype, int trans_a, int trans_b, int epi,
                       int out_bf16, const GemmArgs& a, hipStream_t s) {
  if (a.G <= 0 || a.M <= 0 || a.N <= 0 || a.Kd <= 0) return hipSuccess;
  if (a.G > 65535) return hipErrorInvalidValue;
  // activations are bf16 exactly when the operands are
  if ((epi == EPI_BIAS_RELU || epi == EPI_RELU_MASK) && out_bf16 != (dtype == 1))
    return hipErrorInvalidValue;
  const int key = trans_a * 2 + trans_b;
  switch (epi) {
    case EPI_STORE:
      switch (key) {
        case 0: return dispatch<false, false, EPI_STORE>(dtype, a, s);
        case 1: return dispatch<false, true, EPI_STORE>(dtype, a, s);
        case 2: return dispatch<true, false, EPI_STORE>(dtype, a, s);
        default: return dispatch<true, true, EPI_STORE>(dtype, a, s);
      }
    case EPI_BIAS:
      if (key == 0) return dispatch<false, false, EPI_BIAS>(dtype, a, s);
      break;
    case EPI_BIAS_RELU:
      if (key == 0) return dispatch<false, false, EPI_BIAS_RELU>(dtype, a, s);
      break;
    case EPI_RELU_MASK:
      if (key == 1) return dispatch<false, true, EPI_RELU_MASK>(dtype, a, s);
      break;
    case EPI_SGD:
      if (key == 2) return dispatch<true, false, EPI_SGD>(dtype, a, s);
      break;
    default:
      break;
  }
  return hipErrorInvalidValue;
}

}  // namespace lsgd
