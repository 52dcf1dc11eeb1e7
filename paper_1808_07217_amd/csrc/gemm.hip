// Grouped (replica-batched) GEMM on the gfx950 matrix cores.
//
// Each of the G groups is one replica's layer contraction of the gradient in
// eq. 2 of the paper: forward Z = A W (+ bias, ReLU), the input gradient
// dA = dZ W^T (masked by the ReLU derivative), and the weight gradient
// G = A^T dZ, whose epilogue applies the local momentum-SGD update directly so
// the gradient never goes to memory; the same kernel sums dZ over the batch
// for the bias gradient and updates the bias.
//
// Block tile BM x BN, K slabs of BK, 256 threads = 4 wavefronts in a 2 x 2
// layout, each wave owning (BM/2) x (BN/2) as 32 x 32 MFMA blocks. Operands go
// global -> registers -> LDS through a double-buffered LDS ring: the next
// slab's global loads are in flight while the current slab feeds the MFMAs.
//
//  fp32: v_mfma_f32_32x32x2f32, BK = 32. LDS holds k-major tiles As[k][m],
//        Bs[k][n]; lane l feeds A[m = l%32][k = l/32], B[k = l/32][n = l%32].
//  bf16: v_mfma_f32_32x32x16_bf16, BK = 32. LDS holds k-contiguous rows
//        As[m][k], Bs[n][k]; lane l feeds 8 consecutive k starting at
//        8*(l/32) for row/column l%32.
//  Both: accumulator register v of lane l is C[8*(v/4) + 4*(l/32) + v%4][l%32].
//
// Work distribution: a 1-D grid of G * S * tilesM * tilesN workgroups. The
// hardware deals consecutive workgroup ids round-robin to the 8 XCDs (each
// with its own L2), so the id is remapped to give every XCD a contiguous range
// of tiles: the tiles of one replica then share that XCD's L2.
// Split-K (S > 1) gives skinny GEMMs enough workgroups: split s covers K range
// [s*kchunk, (s+1)*kchunk) and writes a raw fp32 partial; a second kernel sums
// the S partials in ascending s and applies the epilogue.
#include "kernels.h"

namespace lsgd {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;
constexpr int kXcds = 8;

// float4 moves through a native vector type: copying HIP's float4 struct
// straight from memory becomes a memcpy, which keeps register arrays of it
// in scratch memory
typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ldg4(const float* p) {
  const v4f v = *(const v4f*)p;
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void sts4(float* p, const float4& v) {
  *(v4f*)p = v4f{v.x, v.y, v.z, v.w};
}

struct Tile {
  int g, s, m0, n0;
};

__device__ __forceinline__ Tile decode_tile(const GemmArgs& a, int BM, int BN) {
  const int tn = (a.N + BN - 1) / BN, tm = (a.M + BM - 1) / BM;
  const int per_split = tn * tm, per_g = per_split * a.splits;
  const int total = per_g * a.G;
  const int p = blockIdx.x;
  int l = (total % kXcds == 0) ? (p % kXcds) * (total / kXcds) + p / kXcds : p;
  Tile t;
  t.g = l / per_g;
  l -= t.g * per_g;
  t.s = l / per_split;
  l -= t.s * per_split;
  t.m0 = (l / tn) * BM;
  t.n0 = (l % tn) * BN;
  return t;
}

__device__ __forceinline__ void sgd_step(float& w, float& u, float grad,
                                         const GemmArgs& a) {
  const float g = __builtin_fmaf(a.wd, w, grad);
  u = __builtin_fmaf(a.mom, u, g);
  const float d = step_dir(u, g, a.mom, a.nesterov);
  w = __builtin_fmaf(-a.lr, d, w);
}

// Epilogue applied to a finished value of C[g][m][n]. OUTBF: activations are
// bf16 (bf16 workloads) and so are the mask operand and the output.
template <int EPI, bool OUTBF>
__device__ __forceinline__ void finish(const GemmArgs& a, int g, int m, int n,
                                       float v) {
  const long long o = (long long)g * a.sC + (long long)m * a.ldc + n;
  if constexpr (EPI == EPI_SGD) {
    float w = a.Wsrc ? a.Wsrc[(long long)g * a.sWsrc + (long long)m * a.ldc + n] : a.W[o];
    float u = a.U[o];
    sgd_step(w, u, v, a);
    a.W[o] = w;
    a.U[o] = u;
    if (a.Wb) a.Wb[o] = f32_to_bf16(w);
  } else {
    if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_RELU)
      v += a.bias[(long long)g * a.sBias + n];
    if constexpr (EPI == EPI_BIAS_RELU) v = v > 0.f ? v : 0.f;
    if constexpr (EPI == EPI_RELU_MASK) {
      const float mk = OUTBF ? bf16_to_f32(((const bf16_t*)a.mask)[o])
                             : ((const float*)a.mask)[o];
      v = mk > 0.f ? v : 0.f;
    }
    if constexpr (OUTBF)
      ((bf16_t*)a.C)[o] = f32_to_bf16(v);
    else
      ((float*)a.C)[o] = v;
  }
}

template <int EPI, bool OUTBF>
__device__ __forceinline__ void emit(const GemmArgs& a, const Tile& t, int m,
                                     int n, float v) {
  if (a.splits > 1)
    a.part[(((long long)t.s * a.G + t.g) * a.M + m) * a.N + n] = v;
  else
    finish<EPI, OUTBF>(a, t.g, m, n, v);
}

// Bias of the weight-gradient workgroups with m0 == 0: db[n] = sum_b dZ[b][n]
// in ascending b, then the same update as the weights.
__device__ __forceinline__ void bias_update(const GemmArgs& a, const Tile& t,
                                            int n, float colsum) {
  const long long o = (long long)t.g * a.sBiasP + n;
  float w = a.bias_src ? a.bias_src[(long long)t.g * a.sBiasSrc + n] : a.bias_w[o];
  float u = a.bias_u[o];
  sgd_step(w, u, colsum, a);
  a.bias_w[o] = w;
  a.bias_u[o] = u;
}

// Epilogue over one wave's FM x FN fragment of 32 x 32 blocks, one block at
// a time. The operands the epilogue reads (W and U of the update, the ReLU
// mask) are loaded for the whole block before anything is stored, so those
// loads are in flight together instead of each waiting behind the previous
// element's stores (the compiler must assume the buffers may alias).
// Register v of a block sits at row 8*(v/4) + (v%4) below the lane's first
// row and in the lane's column: a 32-bit offset from one base per block.
template <int EPI, bool OUTBF, int FM, int FN>
__device__ __forceinline__ void epilogue_fragment(const GemmArgs& a, const Tile& t,
                                                  floatx16 (&acc)[FM][FN],
                                                  int mb, int nb, int lk, int lr) {
  const int M = a.M, N = a.N;
  if (EPI != EPI_SGD && a.splits > 1) {  // raw partial sums, [s][g][M][N]
    float* P = a.part + ((long long)t.s * a.G + t.g) * a.M * a.N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int m1 = mb + i * 32 + lk * 4, n = nb + j * 32 + lr;
        float* base = P + (long long)m1 * N + n;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int dr = (v >> 2) * 8 + (v & 3);
          if (m1 + dr < M && n < N) base[dr * N] = acc[i][j][v];
        }
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int m1 = mb + i * 32 + lk * 4, n = nb + j * 32 + lr;
      const long long o1 = (long long)t.g * a.sC + (long long)m1 * a.ldc + n;
      const int ldc = (int)a.ldc;
      bool ok[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) ok[v] = m1 + (v >> 2) * 8 + (v & 3) < M && n < N;
      if constexpr (EPI == EPI_SGD) {
        float* Wp = a.W + o1;
        float* Up = a.U + o1;
        const float* Wr = a.Wsrc ? a.Wsrc + (long long)t.g * a.sWsrc +
                                       (long long)m1 * a.ldc + n
                                 : Wp;
        float wv[16], uv[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int dr = ((v >> 2) * 8 + (v & 3)) * ldc;
          wv[v] = ok[v] ? Wr[dr] : 0.f;
          uv[v] = ok[v] ? Up[dr] : 0.f;
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if (!ok[v]) continue;
          const int dr = ((v >> 2) * 8 + (v & 3)) * ldc;
          sgd_step(wv[v], uv[v], acc[i][j][v], a);
          Wp[dr] = wv[v];
          Up[dr] = uv[v];
          if (a.Wb) a.Wb[o1 + dr] = f32_to_bf16(wv[v]);
        }
      } else if constexpr (EPI == EPI_RELU_MASK) {
        float mk[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int dr = ((v >> 2) * 8 + (v & 3)) * ldc;
          mk[v] = 0.f;
          if (ok[v])
            mk[v] = OUTBF ? bf16_to_f32(((const bf16_t*)a.mask)[o1 + dr])
                          : ((const float*)a.mask)[o1 + dr];
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if (!ok[v]) continue;
          const int dr = ((v >> 2) * 8 + (v & 3)) * ldc;
          const float r = mk[v] > 0.f ? acc[i][j][v] : 0.f;
          if constexpr (OUTBF)
            ((bf16_t*)a.C)[o1 + dr] = f32_to_bf16(r);
          else
            ((float*)a.C)[o1 + dr] = r;
        }
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (ok[v]) finish<EPI, OUTBF>(a, t.g, m1 + (v >> 2) * 8 + (v & 3), n, acc[i][j][v]);
      }
    }
}

// Vectorised update epilogue (EPI_SGD, ldc % 4 == 0): the accumulator tile
// goes through LDS, half of the rows at a time, so that every thread then
// updates whole float4 runs of W and U along n -- fully coalesced rows. The
// W/U reads of half 0 are issued at kernel entry (they overlap the MFMA
// loop) and those of half 1 before half 0's results go through LDS.
template <int BM, int BN>
struct SgdVec {
  static constexpr int CP = BN + 4;                      // LDS pitch
  static constexpr int PER = (BM / 2) * BN / 4 / kThreads;  // float4 per thread
  static_assert(PER >= 1 && (BM / 2) * BN / 4 % kThreads == 0, "tile too small");

  __device__ static void locate(const GemmArgs& a, const Tile& t, int half, int p,
                                int& r, int& c, long long& off, bool& ok) {
    const int idx = (int)threadIdx.x + p * kThreads;
    r = idx / (BN / 4);
    c = (idx % (BN / 4)) * 4;
    const int m = t.m0 + half * (BM / 2) + r, n = t.n0 + c;
    ok = m < a.M && n < a.N;
    off = (long long)t.g * a.sC + (long long)m * a.ldc + n;
  }
  __device__ static void fetch(const GemmArgs& a, const Tile& t, int half,
                               float4 (&wv)[PER], float4 (&uv)[PER]) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      int r, c;
      long long off;
      bool ok;
      locate(a, t, half, p, r, c, off, ok);
      if (ok) {
        const float* wr = a.Wsrc ? a.Wsrc + (off - (long long)t.g * a.sC) +
                                       (long long)t.g * a.sWsrc
                                 : a.W + off;
        wv[p] = *(const float4*)wr;
        uv[p] = *(const float4*)(a.U + off);
      }
    }
  }
  template <int FM, int FN>
  __device__ static void run(const GemmArgs& a, const Tile& t,
                             floatx16 (&acc)[FM][FN], float* smem, int wave,
                             int lk, int lr, float4 (&wv)[PER], float4 (&uv)[PER]) {
    const int wn0 = (wave & 1) * (BN / 2);
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      if (half == 1) fetch(a, t, 1, wv, uv);
      __syncthreads();
      if ((wave >> 1) == half) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int r = i * 32 + (v >> 2) * 8 + lk * 4 + (v & 3);
              smem[r * CP + wn0 + j * 32 + lr] = acc[i][j][v];
            }
      }
      __syncthreads();
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        int r, c;
        long long off;
        bool ok;
        locate(a, t, half, p, r, c, off, ok);
        if (!ok) continue;
        const float4 gr = *(const float4*)&smem[r * CP + c];
        float4 w = wv[p], u = uv[p];
        sgd_step(w.x, u.x, gr.x, a);
        sgd_step(w.y, u.y, gr.y, a);
        sgd_step(w.z, u.z, gr.z, a);
        sgd_step(w.w, u.w, gr.w, a);
        *(float4*)(a.W + off) = w;
        *(float4*)(a.U + off) = u;
        if (a.Wb) {
          const uint32_t lo = f32_to_bf16(w.x) | ((uint32_t)f32_to_bf16(w.y) << 16);
          const uint32_t hi = f32_to_bf16(w.z) | ((uint32_t)f32_to_bf16(w.w) << 16);
          *(uint2*)(a.Wb + off) = make_uint2(lo, hi);
        }
      }
    }
  }
};

// ------------------------------------------------------------------ fp32
// FULL: every tile is whole, every split covers whole BK slabs and the
// operands allow float4 loads (checked at launch). The loads then carry no
// bounds branches and the prefetch of slabs past the end is clamped to the
// last slab instead of skipped, so the compiler can count the loads in
// flight and wait only for the register set it is about to store.
template <bool AT, bool BT, int EPI, bool GATHER, int BM, int BN, int BK, bool FULL>
__global__ __launch_bounds__(kThreads) void gemm_f32(GemmArgs a, int vecA,
                                                     int vecB, int vecC) {
  // pitch: transposing stores (k-contiguous source) use pitch = 2 mod 8 to
  // spread banks; direct float4 stores need a 16-byte aligned pitch
  constexpr int PA = AT ? BM + 4 : BM + 2;
  constexpr int PB = BT ? BN + 2 : BN + 4;
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 32, FN = WN / 32;
  constexpr int KV = BK / 4;                  // float4 per k-contiguous row
  constexpr int NA = BM * BK / 4 / kThreads;  // float4 loads per thread
  constexpr int NB = BN * BK / 4 / kThreads;
  static_assert(NA >= 1 && NB >= 1, "tile too small for 256 threads");
  constexpr int OPER = 2 * BK * (PA + PB);
  constexpr int EPIF = EPI == EPI_SGD ? (BM / 2) * (BN + 4) : 0;
  __shared__ __attribute__((aligned(16))) float smem[OPER > EPIF ? OPER : EPIF];
  auto As = reinterpret_cast<float (*)[BK][PA]>(smem);
  auto Bs = reinterpret_cast<float (*)[BK][PB]>(smem + 2 * BK * PA);

  const Tile t = decode_tile(a, BM, BN);
  const int g = t.g, m0 = t.m0, n0 = t.n0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;
  const float* A = (const float*)a.A + (long long)g * a.sA;
  const float* B = (const float*)a.B + (long long)g * a.sB;
  // GATHER: rows of A come from a row map (the sampled mini-batch indices)
  const int32_t* rmap = GATHER ? a.rowmap + (long long)g * a.sRow : nullptr;
  const int M = a.M, N = a.N;
  const int kbeg = t.s * a.kchunk;
  const int kend = min(a.Kd, kbeg + a.kchunk);

  // two register sets: slab t+2 is loaded while slab t computes and slab t+1
  // waits in LDS, so each load has two compute phases to arrive (separate
  // arrays, not one indexed by the set: that index ends up in scratch)
  float4 ra0[NA], rb0[NB], ra1[NA], rb1[NB];
  // gathered rows: the forward operand's rows are fixed per thread, so their
  // dataset indices are read once; the weight gradient walks its rows per
  // slab, so the workgroup's indices are staged in LDS
  long long srow[AT ? 1 : NA];
  __shared__ int32_t srmap[AT && GATHER ? 512 : 1];  // beyond: read rmap
  if constexpr (!AT) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int row = m0 + (tid + i * kThreads) / KV;
      srow[i] = GATHER ? (row < M ? rmap[row] : 0) : row;
    }
  } else if constexpr (GATHER) {
    for (int i = tid; i < 512 && kbeg + i < kend; i += kThreads) srmap[i] = rmap[kbeg + i];
    __syncthreads();
  }

  auto load4 = [](const float* p, int avail, int vec) -> float4 {
    if (vec && avail >= 4) return *(const float4*)p;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (avail > 0) v.x = p[0];
    if (avail > 1) v.y = p[1];
    if (avail > 2) v.z = p[2];
    if (avail > 3) v.w = p[3];
    return v;
  };

  auto gload = [&](int k0, float4(&xa)[NA], float4(&xb)[NB]) __attribute__((always_inline)) {
    if constexpr (FULL) {
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const int q = tid + i * kThreads;
        if constexpr (!AT) {
          xa[i] = ldg4(A + srow[i] * a.lda + k0 + (q % KV) * 4);
        } else {
          const int r = q / (BM / 4), kr = k0 + r;
          const long long sr =
              GATHER ? (kr - kbeg < 512 ? srmap[kr - kbeg] : rmap[kr]) : kr;
          xa[i] = ldg4(A + sr * a.lda + m0 + (q % (BM / 4)) * 4);
        }
      }
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int q = tid + i * kThreads;
        if constexpr (BT)
          xb[i] = ldg4(B + (long long)(n0 + q / KV) * a.ldb + k0 + (q % KV) * 4);
        else
          xb[i] = ldg4(B + (long long)(k0 + q / (BN / 4)) * a.ldb + n0 + (q % (BN / 4)) * 4);
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      xa[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      if constexpr (!AT) {  // storage [M][Kd]: rows m, KV float4 per row
        const int r = q / KV, c = k0 + (q % KV) * 4, row = m0 + r;
        if (row < M && c < kend) xa[i] = load4(A + srow[i] * a.lda + c, kend - c, vecA);
      } else {  // storage [Kd][M]: rows k, BM/4 float4 per row
        const int r = q / (BM / 4), c = m0 + (q % (BM / 4)) * 4, kr = k0 + r;
        if (kr < kend) {
          const long long sr =
              GATHER ? (kr - kbeg < 512 ? srmap[kr - kbeg] : rmap[kr]) : kr;
          xa[i] = load4(A + sr * a.lda + c, M - c, vecA);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      xb[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      if constexpr (BT) {  // storage [N][Kd]
        const int r = q / KV, c = k0 + (q % KV) * 4, row = n0 + r;
        if (row < N && c < kend)
          xb[i] = load4(B + (long long)row * a.ldb + c, kend - c, vecB);
      } else {  // storage [Kd][N]
        const int r = q / (BN / 4), c = n0 + (q % (BN / 4)) * 4, kr = k0 + r;
        if (kr < kend) xb[i] = load4(B + (long long)kr * a.ldb + c, N - c, vecB);
      }
    }
  };

  auto lstore = [&](int buf, const float4(&xa)[NA], const float4(&xb)[NB]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (!AT) {
        const int r = q / KV, kq = (q % KV) * 4;
        As[buf][kq + 0][r] = xa[i].x;
        As[buf][kq + 1][r] = xa[i].y;
        As[buf][kq + 2][r] = xa[i].z;
        As[buf][kq + 3][r] = xa[i].w;
      } else {
        const int r = q / (BM / 4), c = (q % (BM / 4)) * 4;
        sts4(&As[buf][r][c], xa[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT) {
        const int r = q / KV, kq = (q % KV) * 4;
        Bs[buf][kq + 0][r] = xb[i].x;
        Bs[buf][kq + 1][r] = xb[i].y;
        Bs[buf][kq + 2][r] = xb[i].z;
        Bs[buf][kq + 3][r] = xb[i].w;
      } else {
        const int r = q / (BN / 4), c = (q % (BN / 4)) * 4;
        sts4(&Bs[buf][r][c], xb[i]);
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

  const bool do_bias = EPI == EPI_SGD && a.bias_w && m0 == 0;
  float colsum = 0.f;
  // EPI_SGD: W/U of the first half tile are read while the MFMAs run
  using SV = SgdVec<BM, BN>;
  float4 wpre[EPI == EPI_SGD ? SV::PER : 1], upre[EPI == EPI_SGD ? SV::PER : 1];
  if constexpr (EPI == EPI_SGD) {
    if (vecC) SV::fetch(a, t, 0, wpre, upre);
  }
  const int nk = (kend - kbeg + BK - 1) / BK;
  const int lk = lane >> 5, lr = lane & 31;
  auto compute = [&](int buf) __attribute__((always_inline)) {
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
    if (do_bias && tid < BN) {
#pragma unroll 8
      for (int k = 0; k < BK; ++k) colsum += Bs[buf][k][tid];
    }
  };
  // slab t lives in LDS buffer t % 2 and register set t % 2
  int it = 0;
  if constexpr (FULL) {
    // nk >= 1; prefetches past the last slab reload it (unused)
    auto slab = [&](int t) __attribute__((always_inline)) { return kbeg + min(t, nk - 1) * BK; };
    gload(slab(0), ra0, rb0);
    gload(slab(1), ra1, rb1);
    lstore(0, ra0, rb0);
    __syncthreads();
    for (; it + 1 < nk; it += 2) {
      gload(slab(it + 2), ra0, rb0);
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      lstore(1, ra1, rb1);
      __syncthreads();
      gload(slab(it + 3), ra1, rb1);
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      lstore(0, ra0, rb0);
      __syncthreads();
    }
  } else {
    if (nk > 0) gload(kbeg, ra0, rb0);
    if (nk > 1) gload(kbeg + BK, ra1, rb1);
    if (nk > 0) lstore(0, ra0, rb0);
    __syncthreads();
    for (; it + 1 < nk; it += 2) {
      if (it + 2 < nk) gload(kbeg + (it + 2) * BK, ra0, rb0);
      compute(0);
      lstore(1, ra1, rb1);
      __syncthreads();
      if (it + 3 < nk) gload(kbeg + (it + 3) * BK, ra1, rb1);
      compute(1);
      if (it + 2 < nk) lstore(0, ra0, rb0);
      __syncthreads();
    }
  }
  if (it < nk) compute(0);  // odd slab count: the last slab is in buffer 0

  if constexpr (EPI == EPI_SGD) {
    if (vecC)
      SV::template run<FM, FN>(a, t, acc, smem, wave, lk, lr, wpre, upre);
    else
      epilogue_fragment<EPI, false, FM, FN>(a, t, acc, m0 + wm0, n0 + wn0, lk, lr);
  } else {
    epilogue_fragment<EPI, false, FM, FN>(a, t, acc, m0 + wm0, n0 + wn0, lk, lr);
  }
  if (do_bias && tid < BN && n0 + tid < N) bias_update(a, t, n0 + tid, colsum);
}

// Two k halves per workgroup (fp32, A not transposed, whole tiles, no update
// epilogue): 512 threads, threads 256 h .. 256 h + 255 run gemm_f32's FULL
// pipeline over half h of the workgroup's k range (an even number of BK
// slabs) with an LDS ring of their own. Each SIMD then holds two MFMA
// wavefronts, one per half, and one's LDS and barrier waits are covered by
// the other's MFMAs. At the end half 1 hands its accumulators over through
// LDS and half 0 forms (first half) + (second half) and runs the epilogue.
template <bool BT, int EPI, bool GATHER, int BM, int BN, int BK>
__global__ __launch_bounds__(2 * kThreads) void gemm_f32_kh2(GemmArgs a) {
  constexpr int PA = BM + 2;  // As[k][m], transposing stores
  constexpr int PB = BT ? BN + 2 : BN + 4;
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 32, FN = WN / 32;
  constexpr int KV = BK / 4;
  constexpr int NA = BM * BK / 4 / kThreads, NB = BN * BK / 4 / kThreads;
  static_assert(NA >= 1 && NB >= 1, "tile too small for 256 threads per half");
  constexpr int HALF = 2 * BK * (PA + PB);  // floats of one half's ring
  constexpr int XCH = BM * BN;              // accumulator hand-over
  __shared__ __attribute__((aligned(16))) float smem[2 * HALF > XCH ? 2 * HALF : XCH];
  const int h = threadIdx.x >> 8, tid = threadIdx.x & (kThreads - 1);
  auto As = reinterpret_cast<float (*)[BK][PA]>(smem + h * HALF);
  auto Bs = reinterpret_cast<float (*)[BK][PB]>(smem + h * HALF + 2 * BK * PA);

  const Tile t = decode_tile(a, BM, BN);
  const int g = t.g, m0 = t.m0, n0 = t.n0;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;
  const float* A = (const float*)a.A + (long long)g * a.sA;
  const float* B = (const float*)a.B + (long long)g * a.sB;
  const int32_t* rmap = GATHER ? a.rowmap + (long long)g * a.sRow : nullptr;
  const int nk = a.kchunk / BK / 2;  // slabs per half
  const int kbeg = t.s * a.kchunk + h * nk * BK;

  long long srow[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = m0 + (tid + i * kThreads) / KV;
    srow[i] = GATHER ? rmap[row] : row;
  }
  auto gload = [&](int k0, float4(&xa)[NA], float4(&xb)[NB]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      xa[i] = ldg4(A + srow[i] * a.lda + k0 + (q % KV) * 4);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT)
        xb[i] = ldg4(B + (long long)(n0 + q / KV) * a.ldb + k0 + (q % KV) * 4);
      else
        xb[i] = ldg4(B + (long long)(k0 + q / (BN / 4)) * a.ldb + n0 + (q % (BN / 4)) * 4);
    }
  };
  auto lstore = [&](int buf, const float4(&xa)[NA], const float4(&xb)[NB]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      const int r = q / KV, kq = (q % KV) * 4;
      As[buf][kq + 0][r] = xa[i].x;
      As[buf][kq + 1][r] = xa[i].y;
      As[buf][kq + 2][r] = xa[i].z;
      As[buf][kq + 3][r] = xa[i].w;
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT) {
        const int r = q / KV, kq = (q % KV) * 4;
        Bs[buf][kq + 0][r] = xb[i].x;
        Bs[buf][kq + 1][r] = xb[i].y;
        Bs[buf][kq + 2][r] = xb[i].z;
        Bs[buf][kq + 3][r] = xb[i].w;
      } else {
        const int r = q / (BN / 4), c = (q % (BN / 4)) * 4;
        sts4(&Bs[buf][r][c], xb[i]);
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
  const int lk = lane >> 5, lr = lane & 31;
  auto compute = [&](int buf) __attribute__((always_inline)) {
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
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
  };
  // slab t of this half: LDS buffer t % 2, register set t % 2; prefetches
  // past the last slab reload it (unused)
  float4 ra0[NA], rb0[NB], ra1[NA], rb1[NB];
  auto slab = [&](int s) __attribute__((always_inline)) { return kbeg + min(s, nk - 1) * BK; };
  gload(slab(0), ra0, rb0);
  gload(slab(1), ra1, rb1);
  lstore(0, ra0, rb0);
  __syncthreads();
  int it = 0;
  for (; it + 1 < nk; it += 2) {
    gload(slab(it + 2), ra0, rb0);
    __builtin_amdgcn_sched_barrier(0);
    compute(0);
    lstore(1, ra1, rb1);
    __syncthreads();
    gload(slab(it + 3), ra1, rb1);
    __builtin_amdgcn_sched_barrier(0);
    compute(1);
    lstore(0, ra0, rb0);
    __syncthreads();
  }
  if (it < nk) compute(0);  // odd slab count per half: the last is in buffer 0

  // hand-over: register v of block (i, j) of wave w and lane l at
  // ((((w FM + i) FN + j) 16 + v) 64 + l)
  __syncthreads();  // both halves' operand reads are done
  if (h == 1) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          smem[(((wave * FM + i) * FN + j) * 16 + v) * 64 + lane] = acc[i][j][v];
  }
  __syncthreads();
  if (h == 1) return;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        acc[i][j][v] += smem[(((wave * FM + i) * FN + j) * 16 + v) * 64 + lane];
  epilogue_fragment<EPI, false, FM, FN>(a, t, acc, m0 + wm0, n0 + wn0, lk, lr);
}


// ------------------------------------------------- fp32 update, specialised
// Fused weight gradient + momentum-SGD update over the 128 x 128 tiles of one
// or several layers (a list of problems whose tiles are concatenated). A
// workgroup of 8 wavefronts stays resident and walks its share of the tile
// list; its waves have two roles that run concurrently:
//   MFMA waves 0-3 each compute a 64 x 64 quarter of tile j. A lane loads its
//     operands straight from global memory as float2 pairs along m (resp. n);
//     the two halves of a pair feed two different 32 x 32 MFMA blocks, so
//     block i's MFMA row r is m = 2 r + i (columns likewise) and no LDS
//     staging (and so no barrier among the MFMA waves) is needed. A ring of
//     D k-pairs of registers keeps D loads in flight.
//   Update waves 4-7 apply the SGD step to tile j-1 from the gradient tile
//     in LDS (float4 runs along n: coalesced W/U rows), then issue the W/U
//     reads of tile j, which arrive while tile j's MFMAs run.
// Two workgroup barriers per tile hand the LDS gradient buffer over. The
// HBM-bound update of one tile thus overlaps the MFMA phase of the next,
// where separate workgroups doing both phases in turn fall into step and
// alternate between compute-only and memory-only periods across the chip.
// Every problem needs M % 128 == 0, N % 128 == 0, 8-byte aligned operand
// rows, 16-byte aligned W/U rows and (gathered rows) Kd <= 512; all share
// lr, momentum, weight decay and Nesterov.
constexpr int kWsThreads = 512;
constexpr int kWsMaxRows = 512;
constexpr int kWsDepth = 8;        // k-pairs of operands in flight per lane
constexpr int kWsMinTiles = 1024;  // below: one tile per workgroup is as good

struct WsArgs {
  GemmArgs p[kWsMaxProblems];
  int start[kWsMaxProblems + 1];  // first tile of each problem; [np] = total
  int np;
};

struct WsTile {
  int pi, g, m0, n0;
};

__device__ __forceinline__ bool ws_tile(const WsArgs& w, int j, WsTile& t) {
  const int total = w.start[w.np];
  const int p = blockIdx.x, nwg = gridDim.x;
  int l;
  if (total % kXcds == 0 && nwg % kXcds == 0) {
    // XCD x = p % 8 owns tiles [x * total/8, (x+1) * total/8)
    const int chunk = total / kXcds, q = p / kXcds + j * (nwg / kXcds);
    if (q >= chunk) return false;
    l = (p % kXcds) * chunk + q;
  } else {
    const long long ll = p + (long long)j * nwg;
    if (ll >= total) return false;
    l = (int)ll;
  }
  int pi = 0;
  while (pi + 1 < w.np && l >= w.start[pi + 1]) ++pi;
  l -= w.start[pi];
  const int tn = w.p[pi].N / 128, per_g = tn * (w.p[pi].M / 128);
  t.pi = pi;
  t.g = l / per_g;
  l -= t.g * per_g;
  t.m0 = (l / tn) * 128;
  t.n0 = (l % tn) * 128;
  return true;
}

// Row list (sampled dataset indices) of a gathered tile: thread t < 256 of
// the MFMA role holds entries t and t + 256 (clamped to the last row).
struct WsRows {
  int32_t r0, r1;
};
__device__ __forceinline__ WsRows ws_rows_load(const WsArgs& w, const WsTile& t) {
  const GemmArgs& a = w.p[t.pi];
  const int32_t* rm = a.rowmap + (long long)t.g * a.sRow;
  const int last = a.Kd - 1, i = threadIdx.x;
  return WsRows{rm[min(i, last)], rm[min(i + 256, last)]};
}
__device__ __forceinline__ void ws_rows_store(int32_t* buf, const WsRows& r) {
  buf[threadIdx.x] = r.r0;
  buf[threadIdx.x + 256] = r.r1;
}

// Operand pairs of the MFMA role: two consecutive fp32 values (float2), or
// two consecutive bf16 values in one 32-bit word, widened to fp32 at use
// (bf16 x bf16 products are exact in fp32, so the fp32 MFMA computes what a
// bf16 MFMA with fp32 accumulation does, up to the order of the sums).
template <bool BF>
struct WsOp;
template <>
struct WsOp<false> {
  using E = float;
  using P = float2;
  __device__ static P ld(const E* p) { return *(const float2*)p; }
  __device__ static float lo(P v) { return v.x; }
  __device__ static float hi(P v) { return v.y; }
};
template <>
struct WsOp<true> {
  using E = bf16_t;
  using P = uint32_t;
  __device__ static P ld(const E* p) { return *(const uint32_t*)p; }
  __device__ static float lo(P v) { return __uint_as_float(v << 16); }
  __device__ static float hi(P v) { return __uint_as_float(v & 0xffff0000u); }
};

// k loop of one MFMA wave over a tile (its 64 x 64 quarter): rows
// k = 2 kp + lk, kp < nkp. A points at column m0 + wm0 + 2 lr of row 0
// (gathered: row srm[k]), B at column n0 + wn0 + 2 lr of row 0.
template <bool BF, int D>
struct WsK {
  using Op = WsOp<BF>;
  using E = typename Op::E;
  using P = typename Op::P;

  __device__ static void mfma(floatx16 (&acc)[2][2], P ra, P rb, float& cs0, float& cs1) {
    const float a0 = Op::lo(ra), a1 = Op::hi(ra), b0 = Op::lo(rb), b1 = Op::hi(rb);
    acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
    acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
    acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
    acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    cs0 += b0;
    cs1 += b1;
  }

  // Any batch size. Rows past the end are clamped to the last one and their
  // values replaced by zero at use, so the loads carry no branches and stay
  // countable in flight; a runtime loop's back edge still makes the compiler
  // wait for all of them at the top of each block.
  __device__ static void generic(floatx16 (&acc)[2][2], const E* A, const E* B,
                                 long long lda, long long ldb, int Kd, bool gather,
                                 const int32_t* srm, int lk, float& cs0, float& cs1) {
    P ra[D], rb[D];
    auto load = [&](int kp, P& x, P& y) __attribute__((always_inline)) {
      const int k = min(2 * kp + lk, Kd - 1);
      const int sr = srm[min(k, kWsMaxRows - 1)];
      const long long row = gather ? (long long)sr : (long long)k;
      x = Op::ld(A + row * lda);
      y = Op::ld(B + (long long)k * ldb);
    };
#pragma unroll
    for (int d = 0; d < D; ++d) load(d, ra[d], rb[d]);
    const int nblk = ((Kd + 1) / 2 + D - 1) / D;
    for (int blk = 0; blk < nblk; ++blk) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int kp = blk * D + d;
        const bool live = 2 * kp + lk < Kd;
        const P za = live ? ra[d] : P{}, zb = live ? rb[d] : P{};
        mfma(acc, za, zb, cs0, cs1);
        load(kp + D, ra[d], rb[d]);
        // keep each refill right behind its slot's MFMAs: left alone, the
        // scheduler sinks the refills to the end of the block, where they
        // have no time left to arrive
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  // ROWS (64 or 128) rows in straight-line code: the wait before each slot's
  // MFMAs counts exactly the D - 1 younger refills. The row indices sit in
  // ROWS / 64 registers per lane (rows lane, lane + 64) and a refill takes
  // its row by readlane at a compile-time lane instead of waiting on an LDS
  // read between MFMAs; B rows walk with one running pointer.
  template <int ROWS>
  __device__ static void unrolled(floatx16 (&acc)[2][2], const E* A, const E* B,
                                  long long lda, long long ldb, bool gather,
                                  const int32_t* srm, int lane, int lk, float& cs0,
                                  float& cs1) {
    static_assert(ROWS == 64 || ROWS == 128, "one or two index registers per lane");
    constexpr int NKP = ROWS / 2;
    P ra[D], rb[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int k = 2 * d + lk;
      const long long row = gather ? (long long)srm[k] : (long long)k;
      ra[d] = Op::ld(A + row * lda);
      rb[d] = Op::ld(B + (long long)k * ldb);
    }
    const int r_lo = srm[lane], r_hi = ROWS > 64 ? srm[lane + 64] : 0;
    const E* bq = B + (long long)(2 * D + lk) * ldb;
    const long long bstep = 2 * ldb;
#pragma unroll
    for (int kp = 0; kp < NKP; ++kp) {
      const int d = kp % D;
      const P ca = ra[d], cb = rb[d];
      const float a0 = Op::lo(ca), a1 = Op::hi(ca), b0 = Op::lo(cb), b1 = Op::hi(cb);
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      if (kp + D < NKP) {
        // refill of this slot with k-pair kp + D, between the MFMAs
        const int ke = 2 * (kp + D);
        const int src = ke < 64 ? r_lo : r_hi;
        const int se = __builtin_amdgcn_readlane(src, ke & 63);
        const int so = __builtin_amdgcn_readlane(src, (ke + 1) & 63);
        const long long row = gather ? (long long)(lk ? so : se) : (long long)(ke + lk);
        ra[d] = Op::ld(A + row * lda);
      }
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      if (kp + D < NKP) {
        rb[d] = Op::ld(bq);
        bq += bstep;
      }
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
      cs0 += b0;
      cs1 += b1;
      __builtin_amdgcn_sched_barrier(0);
    }
  }
};

// Both roles walk the same tile list and execute the same barriers: one
// before the first tile, then two per tile.
template <bool BF, int D>
__global__ __launch_bounds__(kWsThreads) void gemm_f32_sgd_ws(WsArgs w) {
  using K = WsK<BF, D>;
  using E = typename K::E;
  constexpr int T = 128, CP = T + 4;  // gradient tile pitch (16-byte rows)
  constexpr int PER = T * T / 4 / 256;  // float4 per update thread
  __shared__ __attribute__((aligned(16))) float Gs[T * CP];
  // row lists, double-buffered: tile j reads buffer j % 2 while the MFMA
  // role writes tile j+1's list into the other one after its k loop
  __shared__ int32_t srmap[2][kWsMaxRows];
  // wave index as a scalar: the role branch below is uniform per wave
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  WsTile cur, prev;
  bool prev_ok = false;

  if (wave < 4) {
    // ---- MFMA role: gradient tile j into LDS
    const int lk = lane >> 5, lr = lane & 31;
    const int wm0 = (wave >> 1) * 64, wn0 = (wave & 1) * 64;
    {
      WsTile t0;
      if (ws_tile(w, 0, t0) && w.p[t0.pi].rowmap) ws_rows_store(srmap[0], ws_rows_load(w, t0));
    }
    __syncthreads();  // row list of the first tile
    for (int j = 0;; ++j) {
      const bool ok = ws_tile(w, j, cur);  // uniform over the workgroup
      if (!ok && !prev_ok) break;
      floatx16 acc[2][2];
      if (ok) {
        // next tile's row list: issued now, stored after the k loop
        WsTile nxt;
        const bool nxt_rows = ws_tile(w, j + 1, nxt) && w.p[nxt.pi].rowmap;
        WsRows nr{0, 0};
        if (nxt_rows) nr = ws_rows_load(w, nxt);

        const GemmArgs& a = w.p[cur.pi];
        const int Kd = a.Kd;
        const bool gather = a.rowmap != nullptr;
        const int32_t* srm = srmap[j & 1];
        const E* A = (const E*)a.A + (long long)cur.g * a.sA + cur.m0 + wm0 + 2 * lr;
        const E* B = (const E*)a.B + (long long)cur.g * a.sB + cur.n0 + wn0 + 2 * lr;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][jj][v] = 0.f;
        float cs0 = 0.f, cs1 = 0.f;
        if (Kd == 128)
          K::template unrolled<128>(acc, A, B, a.lda, a.ldb, gather, srm, lane, lk, cs0, cs1);
        else if (Kd == 64)
          K::template unrolled<64>(acc, A, B, a.lda, a.ldb, gather, srm, lane, lk, cs0, cs1);
        else
          K::generic(acc, A, B, a.lda, a.ldb, Kd, gather, srm, lk, cs0, cs1);
        if (nxt_rows) ws_rows_store(srmap[(j + 1) & 1], nr);
        if (a.bias_w && cur.m0 == 0 && wm0 == 0) {
          // lanes < 32 summed the even batch rows, lanes >= 32 the odd ones
          cs0 += __shfl_xor(cs0, 32, 64);
          cs1 += __shfl_xor(cs1, 32, 64);
          if (lk == 0) {
            Tile bt;
            bt.g = cur.g;
            const int n = cur.n0 + wn0 + 2 * lr;
            bias_update(a, bt, n, cs0);
            bias_update(a, bt, n + 1, cs1);
          }
        }
      }
      __syncthreads();  // the update role has consumed gradient tile j-1
      if (ok) {
        // accumulator v of block (i, jj): row 8(v/4) + 4 lk + v%4, column lr
        // of the block, i.e. tile row wm0 + 2 R + i, column wn0 + 2 lr + jj
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int R = (v >> 2) * 8 + lk * 4 + (v & 3);
            *(float2*)&Gs[(wm0 + 2 * R + i) * CP + wn0 + 2 * lr] =
                make_float2(acc[i][0][v], acc[i][1][v]);
          }
      }
      __syncthreads();  // gradient tile j (and tile j+1's row list) in LDS
      prev_ok = ok;
    }
  } else {
    // ---- update role: SGD step of tile j-1, then tile j's W/U reads
    const int u = (int)threadIdx.x - 256;
    float4 wv[PER], uv[PER];
    __syncthreads();  // row list of the first tile
    for (int j = 0;; ++j) {
      const bool ok = ws_tile(w, j, cur);
      if (!ok && !prev_ok) break;
      if (prev_ok) {
        const GemmArgs& a = w.p[prev.pi];
#pragma unroll
        for (int p = 0; p < PER; ++p) {
          const int r = u / 32 + 8 * p, c = (u % 32) * 4;
          const long long off = (long long)prev.g * a.sC +
                                (long long)(prev.m0 + r) * a.ldc + prev.n0 + c;
          const float4 gr = *(const float4*)&Gs[r * CP + c];
          float4 wq = wv[p], uq = uv[p];
          sgd_step(wq.x, uq.x, gr.x, a);
          sgd_step(wq.y, uq.y, gr.y, a);
          sgd_step(wq.z, uq.z, gr.z, a);
          sgd_step(wq.w, uq.w, gr.w, a);
          *(float4*)(a.W + off) = wq;
          *(float4*)(a.U + off) = uq;
          if (a.Wb) {
            const uint32_t lo = f32_to_bf16(wq.x) | ((uint32_t)f32_to_bf16(wq.y) << 16);
            const uint32_t hi = f32_to_bf16(wq.z) | ((uint32_t)f32_to_bf16(wq.w) << 16);
            *(uint2*)(a.Wb + off) = make_uint2(lo, hi);
          }
        }
      }
      if (ok) {
        const GemmArgs& a = w.p[cur.pi];
#pragma unroll
        for (int p = 0; p < PER; ++p) {
          const int r = u / 32 + 8 * p, c = (u % 32) * 4;
          const long long in = (long long)(cur.m0 + r) * a.ldc + cur.n0 + c;
          const long long off = (long long)cur.g * a.sC + in;
          wv[p] = *(const float4*)(a.Wsrc ? a.Wsrc + (long long)cur.g * a.sWsrc + in
                                          : a.W + off);
          uv[p] = *(const float4*)(a.U + off);
        }
      }
      __syncthreads();  // gradient tile j-1 consumed
      __syncthreads();  // gradient tile j is in LDS
      prev = cur;
      prev_ok = ok;
    }
  }
}

// Shape and alignment rules of the specialised kernel for one problem.
// fp32 operands are read as float2, bf16 operands as pairs in one 32-bit word.
bool ws_eligible(int dtype, const GemmArgs& a) {
  auto al = [](const void* p, uintptr_t m) { return ((uintptr_t)p & m) == 0; };
  const uintptr_t pair = dtype == 0 ? 7 : 3;
  return (dtype == 0 || dtype == 1) && a.splits <= 1 && a.G > 0 && a.M > 0 &&
         a.N > 0 && a.Kd > 0 && a.M % 128 == 0 && a.N % 128 == 0 &&
         (a.rowmap == nullptr || a.Kd <= kWsMaxRows) &&
         a.lda % 2 == 0 && a.sA % 2 == 0 && al(a.A, pair) &&
         a.ldb % 2 == 0 && a.sB % 2 == 0 && al(a.B, pair) &&
         a.ldc % 4 == 0 && a.sC % 4 == 0 && al(a.W, 15) && al(a.U, 15) &&
         (a.Wb == nullptr || al(a.Wb, 7)) &&
         (a.Wsrc == nullptr || (al(a.Wsrc, 15) && a.sWsrc % 4 == 0));
}

// ------------------------------------------------------------------ bf16
template <bool AT, bool BT, int EPI, bool GATHER, int BM, int BN>
__global__ __launch_bounds__(kThreads) void gemm_bf16(GemmArgs a, int vecA,
                                                      int vecB, int vecC) {
  constexpr int BK = 32, KP = BK + 8;  // row pitch 80 B keeps 16-B alignment
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 32, FN = WN / 32;
  constexpr int NA = BM * BK / 8 / kThreads;  // 8-element vectors per thread
  constexpr int NB = BN * BK / 8 / kThreads;
  static_assert(NA >= 1 && NB >= 1, "tile too small for 256 threads");
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][KP];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][KP];

  const Tile t = decode_tile(a, BM, BN);
  const int g = t.g, m0 = t.m0, n0 = t.n0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;
  const bf16_t* A = (const bf16_t*)a.A + (long long)g * a.sA;
  const bf16_t* B = (const bf16_t*)a.B + (long long)g * a.sB;
  const int32_t* rmap = GATHER ? a.rowmap + (long long)g * a.sRow : nullptr;
  const int M = a.M, N = a.N;
  const int kbeg = t.s * a.kchunk;
  const int kend = min(a.Kd, kbeg + a.kchunk);

  uint4 ra[NA], rb[NB];

  auto load8 = [](const bf16_t* p, int avail, int vec) -> uint4 {
    if (vec && avail >= 8) return *(const uint4*)p;
    uint16_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = e < avail ? p[e] : (uint16_t)0;
    return make_uint4(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16),
                      h[4] | ((uint32_t)h[5] << 16), h[6] | ((uint32_t)h[7] << 16));
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
          ra[i] = load8(A + sr * a.lda + c, kend - c, vecA);
        }
      } else {  // [Kd][M]: BM/8 vectors per row
        const int r = q / (BM / 8), c = m0 + (q % (BM / 8)) * 8, kr = k0 + r;
        if (kr < kend) {
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
        if (row < N) rb[i] = load8(B + (long long)row * a.ldb + c, kend - c, vecB);
      } else {  // [Kd][N]
        const int r = q / (BN / 8), c = n0 + (q % (BN / 8)) * 8, kr = k0 + r;
        if (kr < kend) rb[i] = load8(B + (long long)kr * a.ldb + c, N - c, vecB);
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

  const bool do_bias = EPI == EPI_SGD && a.bias_w && m0 == 0;
  float colsum = 0.f;
  const int nk = (kend - kbeg + BK - 1) / BK;
  if (nk > 0) {
    gload(kbeg);
    lstore(0);
  }
  __syncthreads();
  const int lk = lane >> 5, lr = lane & 31;
  for (int it = 0; it < nk; ++it) {
    const int buf = it & 1;
    if (it + 1 < nk) gload(kbeg + (it + 1) * BK);
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
    if (do_bias && tid < BN) {
#pragma unroll 8
      for (int k = 0; k < BK; ++k) colsum += bf16_to_f32(Bs[buf][tid][k]);
    }
    if (it + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  constexpr bool OUTBF = EPI == EPI_BIAS_RELU || EPI == EPI_RELU_MASK;
  epilogue_fragment<EPI, OUTBF, FM, FN>(a, t, acc, m0 + wm0, n0 + wn0, lk, lr);
  if (do_bias && tid < BN && n0 + tid < N) bias_update(a, t, n0 + tid, colsum);
}

// bf16 operands, whole 64 x 64 tiles, A stored [M][Kd] (forward and input
// gradient): a HBM-bound contraction at small M, so the point is to keep
// many weight bytes in flight. Two register sets of branch-free 16-byte
// loads (slab t+2 is loaded while slab t computes and slab t+1 waits in
// LDS), BK = 64, prefetches past the end clamped to the last slab.
template <bool BT, int EPI, bool GATHER>
__global__ __launch_bounds__(kThreads) void gemm_bf16_full(GemmArgs a) {
  constexpr int BM = 64, BN = 64, BK = 64, KP = BK + 8;  // 144-B rows
  constexpr int FM = 1, FN = 1;
  constexpr int NA = BM * BK / 8 / kThreads, NB = BN * BK / 8 / kThreads;
  static_assert(NA == 2 && NB == 2, "tile shape");
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][KP];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][KP];

  const Tile t = decode_tile(a, BM, BN);
  const int g = t.g, m0 = t.m0, n0 = t.n0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 32, wn0 = (wave & 1) * 32;
  const bf16_t* A = (const bf16_t*)a.A + (long long)g * a.sA;
  const bf16_t* B = (const bf16_t*)a.B + (long long)g * a.sB;
  const int kbeg = t.s * a.kchunk;
  const int nk = a.kchunk / BK;
  // rows of A are fixed per thread: resolve the gathered indices once
  long long arow[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = m0 + (tid + i * kThreads) / (BK / 8);
    arow[i] = (GATHER ? (long long)a.rowmap[(long long)g * a.sRow + row] : (long long)row) * a.lda;
  }
  auto gload = [&](int k0, u32x4(&xa)[NA], u32x4(&xb)[NB]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      xa[i] = *(const u32x4*)(A + arow[i] + k0 + (q % (BK / 8)) * 8);
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT)  // [N][Kd]
        xb[i] = *(const u32x4*)(B + (long long)(n0 + q / (BK / 8)) * a.ldb + k0 + (q % (BK / 8)) * 8);
      else  // [Kd][N]
        xb[i] = *(const u32x4*)(B + (long long)(k0 + q / (BN / 8)) * a.ldb + n0 + (q % (BN / 8)) * 8);
    }
  };
  auto lstore = [&](int buf, const u32x4(&xa)[NA], const u32x4(&xb)[NB]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int q = tid + i * kThreads;
      *(u32x4*)&As[buf][q / (BK / 8)][(q % (BK / 8)) * 8] = xa[i];
    }
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int q = tid + i * kThreads;
      if constexpr (BT) {
        *(u32x4*)&Bs[buf][q / (BK / 8)][(q % (BK / 8)) * 8] = xb[i];
      } else {  // k row r, 8 consecutive n: transpose into Bs[n][k]
        const int r = q / (BN / 8), c = (q % (BN / 8)) * 8;
        const uint32_t wds[4] = {xb[i].x, xb[i].y, xb[i].z, xb[i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          Bs[buf][c + 2 * e][r] = (bf16_t)(wds[e] & 0xFFFFu);
          Bs[buf][c + 2 * e + 1][r] = (bf16_t)(wds[e] >> 16);
        }
      }
    }
  };
  floatx16 acc[FM][FN];
#pragma unroll
  for (int v = 0; v < 16; ++v) acc[0][0][v] = 0.f;
  const int lk = lane >> 5, lr = lane & 31;
  auto compute = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      const bf16x8 av = *(const bf16x8*)&As[buf][wm0 + lr][kk + lk * 8];
      const bf16x8 bv = *(const bf16x8*)&Bs[buf][wn0 + lr][kk + lk * 8];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[0][0], 0, 0, 0);
    }
  };
  u32x4 ra0[NA], rb0[NB], ra1[NA], rb1[NB];
  auto slab = [&](int s) __attribute__((always_inline)) { return kbeg + min(s, nk - 1) * BK; };
  gload(slab(0), ra0, rb0);
  gload(slab(1), ra1, rb1);
  lstore(0, ra0, rb0);
  __syncthreads();
  int it = 0;
  for (; it + 1 < nk; it += 2) {
    gload(slab(it + 2), ra0, rb0);
    __builtin_amdgcn_sched_barrier(0);
    compute(0);
    lstore(1, ra1, rb1);
    __syncthreads();
    gload(slab(it + 3), ra1, rb1);
    __builtin_amdgcn_sched_barrier(0);
    compute(1);
    lstore(0, ra0, rb0);
    __syncthreads();
  }
  if (it < nk) compute(0);  // odd slab count: the last slab is in buffer 0
  constexpr bool OUTBF = EPI == EPI_BIAS_RELU || EPI == EPI_RELU_MASK;
  epilogue_fragment<EPI, OUTBF, FM, FN>(a, t, acc, m0 + wm0, n0 + wn0, lk, lr);
}

// ------------------------------------------------------------------ split-K
// C[g][m][n] = epilogue(sum_{s=0}^{S-1} part[s][g][m][n]), s ascending. S is
// a template argument so all S loads are issued before the sum.
template <int EPI, bool OUTBF, int S>
__global__ void k_splitk_reduce(GemmArgs a) {
  const long long MN = (long long)a.M * a.N, total = MN * a.G;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    float p[S];
#pragma unroll
    for (int s = 0; s < S; ++s) p[s] = a.part[i + s * total];
    float v = p[0];
#pragma unroll
    for (int s = 1; s < S; ++s) v += p[s];
    const int g = (int)(i / MN);
    const long long r = i - g * MN;
    finish<EPI, OUTBF>(a, g, (int)(r / a.N), (int)(r % a.N), v);
  }
}

template <int EPI, bool OUTBF>
hipError_t launch_reduce(const GemmArgs& a, hipStream_t s) {
  const long long n = (long long)a.G * a.M * a.N;
  const int blocks = (int)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192);
  switch (a.splits) {
    case 2: hipLaunchKernelGGL((k_splitk_reduce<EPI, OUTBF, 2>), dim3(blocks), dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_splitk_reduce<EPI, OUTBF, 4>), dim3(blocks), dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_splitk_reduce<EPI, OUTBF, 8>), dim3(blocks), dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((k_splitk_reduce<EPI, OUTBF, 3>), dim3(blocks), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Tile shape for a problem: 128 x 128 (four MFMA chains per wave) when both
// output dimensions allow it on the fp32 path, else 64 x 64.
// 128 x 128 fp32 tiles when they fill the chip (256 or more) or the inner
// dimension is long enough for split-K to amortise them; otherwise 64 x 64
// tiles without split-K. Measured on the 512-wide MLP: its 512-deep layer
// GEMMs (64 big tiles) take 18 us as 64 x 64 tiles against 25 us as split-K
// 128 x 128 tiles plus the reduction; the 3072-deep first layer is fastest
// as 128 x 128 tiles split four ways.
bool big_tile(int dtype, int M, int N, int G, int Kd) {
  if (dtype != 0 || M < 128 || N < 128) return false;
  return (long long)(M / 128) * (N / 128) * G >= 256 || Kd >= 2048;
}

// Compute units and resident specialised-update workgroups per CU on the
// current device, queried once per device.
template <bool BF>
hipError_t ws_grid(long long tiles, int& grid) {
  struct Shape {
    int cus = 0, per_cu = 0;
  };
  static Shape cache[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  if (cache[dev].cus == 0) {
    Shape sh;
    e = hipDeviceGetAttribute(&sh.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &sh.per_cu, reinterpret_cast<const void*>(gemm_f32_sgd_ws<BF, kWsDepth>),
        kWsThreads, 0);
    if (e != hipSuccess) return e;
    if (sh.per_cu < 1) sh.per_cu = 1;
    cache[dev] = sh;
  }
  long long g = (long long)cache[dev].cus * cache[dev].per_cu;
  if (g > tiles) g = tiles;
  if (g >= kXcds) g -= g % kXcds;
  grid = (int)g;
  return hipSuccess;
}

}  // namespace

int gemm_sgd_multi_tiles(int dtype, const GemmArgs* list, int n) {
  if (n < 1 || n > kWsMaxProblems) return -1;
  long long total = 0;
  for (int i = 0; i < n; ++i) {
    if (!ws_eligible(dtype, list[i])) return -1;
    total += (long long)(list[i].M / 128) * (list[i].N / 128) * list[i].G;
  }
  return total < (1LL << 30) ? (int)total : -1;
}

hipError_t launch_gemm_sgd_multi(int dtype, const GemmArgs* list, int n,
                                 hipStream_t s) {
  const int total = gemm_sgd_multi_tiles(dtype, list, n);
  if (total < 0) return hipErrorInvalidValue;
  if (total == 0) return hipSuccess;
  WsArgs w{};
  w.np = n;
  w.start[0] = 0;
  for (int i = 0; i < n; ++i) {
    w.p[i] = list[i];
    w.p[i].splits = 1;
    w.start[i + 1] = w.start[i] + (list[i].M / 128) * (list[i].N / 128) * list[i].G;
    if (i > 0 && (list[i].lr != list[0].lr || list[i].mom != list[0].mom ||
                  list[i].wd != list[0].wd || list[i].nesterov != list[0].nesterov))
      return hipErrorInvalidValue;
  }
  int grid = 0;
  hipError_t e = dtype == 1 ? ws_grid<true>(total, grid) : ws_grid<false>(total, grid);
  if (e != hipSuccess) return e;
  if (dtype == 1)
    hipLaunchKernelGGL((gemm_f32_sgd_ws<true, kWsDepth>), dim3(grid), dim3(kWsThreads),
                       0, s, w);
  else
    hipLaunchKernelGGL((gemm_f32_sgd_ws<false, kWsDepth>), dim3(grid), dim3(kWsThreads),
                       0, s, w);
  return hipGetLastError();
}

namespace {

// k slab of the whole-tile 128 x 128 variant. 32 would halve the barriers
// per k but doubles the prefetch registers and LDS; measured on the 512-wide
// MLP it is slower, and costs the update epilogue an occupancy step.
template <int EPI>
constexpr int kBigFullBK = 16;

// Whole tiles, whole slabs per split, vector loads: the FULL kernel variant.
bool full(const GemmArgs& a, int T, int BK, int vecA, int vecB, int vecC) {
  return vecA && vecB && a.M % T == 0 && a.N % T == 0 && a.kchunk % BK == 0 &&
         (long long)a.kchunk * a.splits == a.Kd && (vecC || a.W == nullptr);
}

template <bool AT, bool BT, int EPI, bool GATHER>
hipError_t run(int dtype, GemmArgs a, hipStream_t s) {
  if constexpr (AT && !BT && EPI == EPI_SGD) {
    // one large layer: the specialised update kernel with a one-item list
    if (ws_eligible(dtype, a) &&
        (long long)(a.M / 128) * (a.N / 128) * a.G >= kWsMinTiles)
      return launch_gemm_sgd_multi(dtype, &a, 1, s);
  }
  const bool big = big_tile(dtype, a.M, a.N, a.G, a.Kd);
  const int BM = big ? 128 : 64, BN = BM;
  const long long tiles = (long long)((a.N + BN - 1) / BN) * ((a.M + BM - 1) / BM) * a.G;
  const long long total = tiles * a.splits;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  const int esz = dtype == 1 ? 8 : 4;  // elements per vector load
  const int vecA = a.lda % esz == 0 && a.sA % esz == 0 && aligned16(a.A);
  const int vecB = a.ldb % esz == 0 && a.sB % esz == 0 && aligned16(a.B);
  const int vecC = EPI == EPI_SGD && a.ldc % 4 == 0 && a.sC % 4 == 0 &&
                   aligned16(a.W) && aligned16(a.U) &&
                   (a.Wb == nullptr || ((uintptr_t)a.Wb & 7u) == 0) &&
                   (a.Wsrc == nullptr || (aligned16(a.Wsrc) && a.sWsrc % 4 == 0));
  if constexpr (!AT && EPI != EPI_SGD) {
    if (dtype == 1 && vecA && vecB && a.M % 64 == 0 && a.N % 64 == 0 &&
        a.kchunk % 64 == 0 && (long long)a.kchunk * a.splits == a.Kd) {
      hipLaunchKernelGGL((gemm_bf16_full<BT, EPI, GATHER>), dim3(total), dim3(kThreads),
                         0, s, a);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess || a.splits == 1) return e;
      constexpr bool OUTBF_ACT = EPI == EPI_BIAS_RELU || EPI == EPI_RELU_MASK;
      return launch_reduce<EPI, OUTBF_ACT>(a, s);
    }
  }
  // two k halves per workgroup (an even number of slabs per split)
  bool kh2 = false;
  if constexpr (!AT && EPI != EPI_SGD) {
    const int bk = big ? kBigFullBK<EPI> : 32;
    kh2 = dtype == 0 && full(a, BM, bk, vecA, vecB, vecC) && a.kchunk >= 2 * bk &&
          a.kchunk % (2 * bk) == 0;
    if (kh2 && big)
      hipLaunchKernelGGL((gemm_f32_kh2<BT, EPI, GATHER, 128, 128, kBigFullBK<EPI>>),
                         dim3(total), dim3(2 * kThreads), 0, s, a);
    else if (kh2)
      hipLaunchKernelGGL((gemm_f32_kh2<BT, EPI, GATHER, 64, 64, 32>), dim3(total),
                         dim3(2 * kThreads), 0, s, a);
  }
  if (kh2)
    ;
  else if (dtype == 1)
    hipLaunchKernelGGL((gemm_bf16<AT, BT, EPI, GATHER, 64, 64>), dim3(total),
                       dim3(kThreads), 0, s, a, vecA, vecB, vecC);
  else if (big && full(a, 128, kBigFullBK<EPI>, vecA, vecB, vecC))
    hipLaunchKernelGGL((gemm_f32<AT, BT, EPI, GATHER, 128, 128, kBigFullBK<EPI>, true>), dim3(total),
                       dim3(kThreads), 0, s, a, vecA, vecB, vecC);
  else if (big)
    hipLaunchKernelGGL((gemm_f32<AT, BT, EPI, GATHER, 128, 128, 16, false>), dim3(total),
                       dim3(kThreads), 0, s, a, vecA, vecB, vecC);
  else if (full(a, 64, 32, vecA, vecB, vecC))
    hipLaunchKernelGGL((gemm_f32<AT, BT, EPI, GATHER, 64, 64, 32, true>), dim3(total),
                       dim3(kThreads), 0, s, a, vecA, vecB, vecC);
  else
    hipLaunchKernelGGL((gemm_f32<AT, BT, EPI, GATHER, 64, 64, 32, false>), dim3(total),
                       dim3(kThreads), 0, s, a, vecA, vecB, vecC);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  constexpr bool OUTBF_ACT = EPI == EPI_BIAS_RELU || EPI == EPI_RELU_MASK;
  if (dtype == 1 && OUTBF_ACT) return launch_reduce<EPI, true>(a, s);
  return launch_reduce<EPI, false>(a, s);
}

template <bool AT, bool BT, int EPI>
hipError_t dispatch(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.rowmap) return run<AT, BT, EPI, true>(dtype, a, s);
  return run<AT, BT, EPI, false>(dtype, a, s);
}

}  // namespace

int gemm_splits(int dtype, int M, int N, int Kd, int G, int epi) {
  if (epi == EPI_SGD) return 1;
  const int T = big_tile(dtype, M, N, G, Kd) ? 128 : 64;
  const long long tiles = (long long)((N + T - 1) / T) * ((M + T - 1) / T) * G;
  int s = 1;
  // up to 8 splits while the grid has fewer workgroups than compute units
  // and every split keeps at least 128 of K
  while (s < 8 && tiles * s < 256 && Kd / (s * 2) >= 128) s *= 2;
  return s;
}

hipError_t launch_gemm(int dtype, int trans_a, int trans_b, int epi,
                       int out_bf16, const GemmArgs& args, hipStream_t s) {
  if (args.G <= 0 || args.M <= 0 || args.N <= 0 || args.Kd <= 0) return hipSuccess;
  GemmArgs a = args;
  if (a.splits < 1) a.splits = 1;
  if (a.splits > 1 && (a.part == nullptr || epi == EPI_SGD)) return hipErrorInvalidValue;
  a.kchunk = (a.Kd + a.splits - 1) / a.splits;
  a.kchunk = (a.kchunk + 31) / 32 * 32;
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
