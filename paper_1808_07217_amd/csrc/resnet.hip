// Kernels of the ResNet-20-shaped network (the CIFAR ResNet of the paper's
// model appendix and Table 5), per replica, NHWC activations:
//
//  * 3x3 convolutions (padding 1, stride 1 or 2) as implicit GEMMs on the
//    fp32 matrix cores. The operand loader maps GEMM coordinates to tensor
//    addresses on the fly -- no im2col buffer:
//      forward      y[m][co]  = sum_k x(m, k) W[k][co],       k = (kh, kw, ci)
//      input grad   dx[m][ci] = sum_k dy(m, k) W[(kh, kw, ci)][co], k = (kh, kw, co)
//      weight grad  dW[k][co] = sum_m x(m, k) dy[m][co]       (split over m)
//    where x(m, k) is the padded input at output position m and tap (kh, kw)
//    and dy(m, k) the output gradient that reaches input position m through
//    tap (kh, kw); the input gradient reads the weight in its forward layout
//    with the channel roles swapped as it stages it.
//  * batch normalisation with batch statistics per replica (the per-worker BN
//    of the CIFAR setup): fp64 partial sums per row chunk, reduced in a fixed
//    order, so the statistics are deterministic;
//  * ReLU, the option-A shortcut (every second pixel, channels zero-padded),
//    global average pooling.
#include <atomic>

#include "kernels.h"

namespace lsgd {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
constexpr int kT = 256;

// ------------------------------------------------------------ conv GEMM
enum ConvMode : int {
  CONV_FWD = CONV_FWD_MODE,
  CONV_DGRAD = CONV_DGRAD_MODE,
  CONV_WGRAD = CONV_WGRAD_MODE
};

// Geometry seen by one launch. For CONV_FWD / CONV_WGRAD the "input" is x
// (H x W x Cin) and the output y (Ho x Wo x Cout); for CONV_DGRAD the roles
// are as in the forward convolution (x is the input whose gradient is
// produced).
struct ConvArgs {
  int G, Bt;             // replicas, images per replica
  int H, W, Cin, Ho, Wo, Cout, stride;
  const float* x;        // input activations [G][Bt][H][W][Cin], or dataset
  long long sx;          //   group stride (0 with a row map)
  const int32_t* rowmap; // sampled image indices [G][Bt] (first convolution)
  const float* dy;       // output gradient [G][Bt][Ho][Wo][Cout]
  const float* Wk;       // weights [9*Cin][Cout] (every mode)
  long long sW;          //   group stride
  float* out;            // fwd: y; dgrad: dx; wgrad: partials [S][G][9Cin][Cout]
  int splits, mchunk;    // wgrad split over the m = (b, oh, ow) rows; stride-2 input
                         //   gradient: images per workgroup (mchunk)
  double* stats;         // fwd: per 256-row chunk q of replica g, (sum y, sum y^2)
                         //   per channel at [g][q][Cout][2], or nullptr
  const float* bn_mu;    // input BN-ReLU (see ConvGeom), or nullptr
  const float* bn_inv;
  const float* bn_g;
  const float* bn_b;
  long long bn_sP;
  // stage-1 input gradient epilogues (see ConvGeom): the shortcut share and
  // the backward BN sums of the layer whose activation gradient dx is
  const float* sc_dh;
  const unsigned* sc_hb;
  const float* bs_y;
  const unsigned* bs_hb;
  double* bs_part;
};

// The shifted, scaled BN output z = gamma * (y - mu) * inv + beta in one fixed
// rounding order, fma(y - mu, gamma * inv, beta): the forward pass takes
// relu(z) (+ the shortcut) with it, and
// the backward pass of a convolution followed by BN-ReLU alone recomputes the
// ReLU mask z > 0 with it instead of reading the activation back.
__device__ __forceinline__ float bn_z(float gm, float y, float m, float iv, float bt) {
  return __builtin_fmaf(y - m, gm * iv, bt);
}

typedef float v4f __attribute__((ext_vector_type(4)));

// ReLU masks as bits: a tensor's mask holds bit L % 32 of word L / 32 for its
// element at linear index L (whole tensor, [G][rows][C] order), set where the
// activation is positive. A block output's mask is written with it
// (k_bn_apply4); the backward passes that only need the activation's sign
// read 1/32 of its bytes.
__device__ __forceinline__ bool mask_bit(unsigned word, long long L) {
  return (word >> (unsigned)(L & 31)) & 1u;
}

// BN statistics and parameters of four consecutive input channels.
struct BnIn4 {
  v4f g, m, iv, b;
};
__device__ __forceinline__ BnIn4 bn_in_params(const ConvArgs& c, int g, int ch0) {
  BnIn4 p;
  p.m = *(const v4f*)(c.bn_mu + (long long)g * c.Cin + ch0);
  p.iv = *(const v4f*)(c.bn_inv + (long long)g * c.Cin + ch0);
  p.g = *(const v4f*)(c.bn_g + (long long)g * c.bn_sP + ch0);
  p.b = *(const v4f*)(c.bn_b + (long long)g * c.bn_sP + ch0);
  return p;
}
// relu(z) of four pre-BN values (the activation the BN pass would store)
__device__ __forceinline__ v4f bn_in(const BnIn4& p, v4f v) {
  v4f r;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float z = bn_z(p.g[e], v[e], p.m[e], p.iv[e], p.b[e]);
    r[e] = z > 0.f ? z : 0.f;
  }
  return r;
}

// BN statistics of a forward tile: lane partial sums (s0, s1) of one channel,
// added over the lanes xor-ed by `mask_bits` (a fixed butterfly), written by
// the lanes whose masked bits are zero.
__device__ __forceinline__ void stats_butterfly(double& s0, double& s1, int width_bits,
                                                int first_bit) {
  for (int b = 0; b < width_bits; ++b) {
    const int off = 1 << (first_bit + b);
    s0 += __shfl_xor(s0, off, 64);
    s1 += __shfl_xor(s1, off, 64);
  }
}

// Input-gradient epilogues (EPI bits; their operands are loaded while the
// last k work of a tile or band runs):
//   kEpiShortcut: dx += dh where h > 0 (c.sc_dh: the block output's
//     gradient, same shape; c.sc_hb: its activation's mask bits; the
//     identity shortcut);
//   kEpiBnSums: dx is the gradient of a BN-ReLU's output whose pre-BN values
//     c.bs_y and BN parameters come in c.bn_*: per 256 output rows, the
//     backward sums sum dz and sum dz x^ (dz = dx where the ReLU passed,
//     x^ = (y - mu) inv) go to c.bs_part as one chunk, in the forward
//     statistics' layout;
//   kEpiBnSumsAct: the same sums where the ReLU follows a shortcut add (a
//     block's second BN): dz = dx where the activation's mask bit (c.bs_hb)
//     is set.
// The shortcut combines with either sums (dx then includes the shortcut
// share); the sums' operands are then loaded after the k work, where the
// shortcut's are free.
constexpr int kEpiShortcut = 1, kEpiBnSums = 2, kEpiBnSumsAct = 4;

// Forward / input-gradient convolution for reduction channel counts that
// are multiples of 16 (every convolution after the first): the output tile
// is 256 spatial rows x all BN (= 16, 32 or 64) channels, so no MFMA lane is
// spent on channels that do not exist. Each wave owns 64 rows as 16 x 16
// blocks of v_mfma_f32_16x16x4f32 (lane l: A[m = l%16][k = l/16],
// B[k = l/16][n = l%16], accumulator v at C[4 (l/16) + v][l%16]). A k slab
// of 16 is one tap (kh, kw) and 16 consecutive channels, taken in the order
// 4 (l/16) + s at MFMA step s: a lane's four A values of a row are then one
// float4 of the activation, and the operands go from memory straight into
// the registers the MFMAs read -- no LDS staging and no barriers, every wave
// runs on its own. Operands are read through buffer resources: a lane
// decodes its four rows (image, position, which of the nine taps fall inside
// the image) once, a slab adds the tap's offset, and a tap outside the image
// reads at an offset past the resource's end, which the hardware returns as
// zero; the weights' slab offset is a scalar. Three register sets: slabs
// t + 1 and t + 2 are in flight while slab t computes. The input gradient
// here is that of a stride-1 convolution.
typedef float floatx4 __attribute__((ext_vector_type(4)));

// A raw buffer resource over `bytes` bytes at p (gfx9 word 3: 32-bit data
// format); loads at offsets at or past `bytes` return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* p, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes,
                                           0x00020000);
}
constexpr unsigned kOutside = 0x80000000u;  // an offset past every resource here

template <int BN>
struct RowsSlab {
  v4f a[4];          // A: rows 16 i + l%16, channels ch .. ch + 3
  v4f b[BN / 16];    // B: k = ch .. ch + 3, column 16 j + l%16
  unsigned okm;      // which of the four rows read inside the image (bit i)
  int ch;            // the lane's first reduction channel
};

template <int MODE, int BN, int EPI = 0>
__global__ __launch_bounds__(kT) void k_conv_rows(ConvArgs c) {
  static_assert(MODE == CONV_FWD || MODE == CONV_DGRAD, "row-tiled modes");
  static_assert(EPI == 0 || MODE == CONV_DGRAD, "epilogues of the input gradient");
  constexpr int BM = 256;
  constexpr int NBL = BN / 16;  // 16-wide column blocks

  const int Cr = MODE == CONV_FWD ? c.Cin : c.Cout;  // reduction channels
  const int HWo = MODE == CONV_FWD ? c.Ho * c.Wo : c.H * c.W;
  const int Mg = c.Bt * HWo;
  const int tiles = (Mg + BM - 1) / BM;
  const int g = blockIdx.x / tiles, m0 = (blockIdx.x - g * tiles) * BM;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lq = lane >> 4, lm = lane & 15;

  // the replica's operand tensor (the input, or the output gradient) and
  // weights W [9 Cin][Cout]
  const int Hs = MODE == CONV_FWD ? c.H : c.Ho, Ws = MODE == CONV_FWD ? c.W : c.Wo;
  const float* src = MODE == CONV_FWD ? c.x + (long long)g * c.sx
                                      : c.dy + (long long)g * c.Bt * c.Ho * c.Wo * c.Cout;
  const auto rsA = buffer_rsrc(src, (unsigned)c.Bt * Hs * Ws * Cr * 4u);
  const auto rsB = buffer_rsrc(c.Wk + (long long)g * c.sW, 9u * c.Cin * c.Cout * 4u);

  // rows of this lane: m0 + 64 wave + 16 i + l%16; off: byte offset of the
  // tap (1, 1) read plus the lane's channels; tapm: which taps are inside
  int off[4];
  unsigned tapm[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + wave * 64 + i * 16 + lm;
    const bool rok = m < Mg;
    const int mm = rok ? m : 0;
    const int b = mm / HWo, p = mm - b * HWo;
    int yc, xc;  // operand position of the centre tap
    if constexpr (MODE == CONV_FWD) {
      const int oh = p / c.Wo, ow = p - oh * c.Wo;
      yc = oh * c.stride;
      xc = ow * c.stride;
    } else {
      yc = p / c.W;
      xc = p - yc * c.W;
    }
    unsigned t = 0;
#pragma unroll
    for (int kh = 0; kh < 3; ++kh)
#pragma unroll
      for (int kw = 0; kw < 3; ++kw) {
        // forward: input (yc + kh - 1, xc + kw - 1); input gradient: output
        // gradient (yc + 1 - kh, xc + 1 - kw)
        const int yy = MODE == CONV_FWD ? yc + kh - 1 : yc + 1 - kh;
        const int xx = MODE == CONV_FWD ? xc + kw - 1 : xc + 1 - kw;
        const bool ok = rok && yy >= 0 && yy < Hs && xx >= 0 && xx < Ws;
        t |= (unsigned)ok << (kh * 3 + kw);
      }
    tapm[i] = t;
    off[i] = (((b * Hs + yc) * Ws + xc) * Cr + 4 * lq) * 4;
  }
  const int cpt = Cr / 16;     // slabs per tap
  const int nk = 9 * cpt;      // a multiple of 3
  // forward of a block's second convolution: the input BN-ReLU, statistics
  // and parameters of every input channel staged in LDS
  const bool bnin = MODE == CONV_FWD && c.bn_mu != nullptr;
  __shared__ __attribute__((aligned(16))) float bnp[4][64];
  constexpr bool kSc = (EPI & kEpiShortcut) != 0;
  constexpr bool kSums = (EPI & (kEpiBnSums | kEpiBnSumsAct)) != 0;
  constexpr bool kMaskAct = (EPI & kEpiBnSumsAct) != 0;
  if (bnin || kSums) {  // (the sums: the BN layer of dx, Cin channels)
    for (int t = tid; t < c.Cin; t += kT) {
      bnp[0][t] = c.bn_mu[(long long)g * c.Cin + t];
      bnp[1][t] = c.bn_inv[(long long)g * c.Cin + t];
      bnp[2][t] = c.bn_g[(long long)g * c.bn_sP + t];
      bnp[3][t] = c.bn_b[(long long)g * c.bn_sP + t];
    }
  }
  // Input gradient with up to 32 channels (and at most 32 reduction
  // channels): the replica's whole weight goes to LDS once, as B^T rows
  // [tap][n][k] with k contiguous (pitch BP), so a slab's B values are one
  // LDS float4 per column block; otherwise they are read from L1/L2 slab by
  // slab (measured: the forward's transposing staging costs it more than
  // the LDS reads save).
  constexpr bool kLdsB = MODE == CONV_DGRAD && BN <= 32;
  constexpr int BP = 32 + 4;
  __shared__ __attribute__((aligned(16))) float Bsm[kLdsB ? 9 * BN * BP : 4];
  if constexpr (kLdsB) {
    // W [9 Cin][Cout]: forward, B^T[tap][co][ci] = W[(tap, ci)][co]; input
    // gradient, B^T[tap][ci][co] = W[(tap, ci)][co]
    const float* Wg = c.Wk + (long long)g * c.sW;
    const int nq = 9 * c.Cin * c.Cout / 4;
    for (int q = tid; q < nq; q += kT) {
      const int e0 = 4 * q, row = e0 / c.Cout, co = e0 - row * c.Cout;
      const int tap = row / c.Cin, ci = row - tap * c.Cin;
      const v4f w = *(const v4f*)(Wg + e0);
      if constexpr (MODE == CONV_FWD) {
#pragma unroll
        for (int e = 0; e < 4; ++e) Bsm[(tap * BN + co + e) * BP + ci] = w[e];
      } else {
        *(v4f*)&Bsm[(tap * BN + ci) * BP + co] = w;
      }
    }
  }
  if (kLdsB || bnin || kSums) __syncthreads();
  // the lane's B offsets: forward, rows ch + e of W at column 16 j + l%16;
  // input gradient, row (tap, 16 j + l%16) of W at columns ch .. ch + 3
  int boff[NBL];
#pragma unroll
  for (int j = 0; j < NBL; ++j)
    boff[j] = MODE == CONV_FWD ? ((4 * lq) * BN + j * 16 + lm) * 4
                               : ((j * 16 + lm) * Cr + 4 * lq) * 4;
  auto gload = [&](int s, RowsSlab<BN>& t) __attribute__((always_inline)) {
    const int ti = s / cpt, cb = (s - ti * cpt) * 16;
    const int kh = ti / 3, kw = ti - kh * 3;
    // byte offset of tap (kh, kw), channel block cb, from the centre read
    const int dt = MODE == CONV_FWD ? (((kh - 1) * Ws + (kw - 1)) * Cr + cb) * 4
                                    : (((1 - kh) * Ws + (1 - kw)) * Cr + cb) * 4;
    unsigned okm = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool ok = tapm[i] >> ti & 1;
      const unsigned o = ok ? (unsigned)(off[i] + dt) : kOutside;
      t.a[i] = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(rsA, o, 0, 0));
      okm |= (unsigned)ok << i;
    }
    t.okm = okm;
    t.ch = cb + 4 * lq;
    if constexpr (kLdsB) {
      // B^T row (tap, 16 j + l%16), reduction channels ch .. ch + 3
      const float* bb = Bsm + (ti * BN + lm) * BP + cb + 4 * lq;
#pragma unroll
      for (int j = 0; j < NBL; ++j) t.b[j] = *(const v4f*)(bb + j * 16 * BP);
      return;
    }
    // scalar part of the weights' offset
    const int sb = MODE == CONV_FWD ? (ti * Cr + cb) * BN * 4 : (ti * BN * Cr + cb) * 4;
#pragma unroll
    for (int j = 0; j < NBL; ++j) {
      if constexpr (MODE == CONV_FWD) {
        // B[k = (tap, ci)][n = co] = W[(tap, ci)][co]: four rows of W
#pragma unroll
        for (int e = 0; e < 4; ++e)
          t.b[j][e] = __builtin_bit_cast(
              float, __builtin_amdgcn_raw_buffer_load_b32(rsB, boff[j] + e * BN * 4, sb, 0));
      } else {
        // B[k = (tap, co)][n = ci] = W[(tap, ci)][co]: four consecutive co
        t.b[j] = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(rsB, boff[j], sb, 0));
      }
    }
  };
  floatx4 acc[4][NBL];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NBL; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const RowsSlab<BN>& t) __attribute__((always_inline)) {
    v4f a[4];
    if (bnin) {
      BnIn4 p;
      p.m = *(const v4f*)&bnp[0][t.ch];
      p.iv = *(const v4f*)&bnp[1][t.ch];
      p.g = *(const v4f*)&bnp[2][t.ch];
      p.b = *(const v4f*)&bnp[3][t.ch];
#pragma unroll
      for (int i = 0; i < 4; ++i) {  // padding stays 0
        const v4f z = bn_in(p, t.a[i]);
        const bool ok = t.okm >> i & 1;
#pragma unroll
        for (int e = 0; e < 4; ++e) a[i][e] = ok ? z[e] : 0.f;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = t.a[i];  // zero outside the image
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NBL; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][s], t.b[j][s], acc[i][j], 0, 0, 0);
  };
  // epilogue operands of this lane's outputs (row block i, column block j,
  // register v): the shortcut's (eh, edh), or the sums' alone (ey and, with
  // the activation mask, ea), issued while the last slabs compute; the sums'
  // next to the shortcut's after the k work
  // (the masks as bit words: with BN a multiple of 32, a lane's column
  // blocks 2 jw and 2 jw + 1 of a row share word jw of that row, at bits
  // 16 (j % 2) + lm)
  static_assert(!(kSc || kMaskAct) || BN % 32 == 0, "mask words span 32 channels");
  constexpr int NW = (NBL + 1) / 2;
  unsigned eh[kSc ? 4 : 1][kSc ? NW : 1][4], ea[kMaskAct ? 4 : 1][kMaskAct ? NW : 1][4];
  float edh[kSc ? 4 : 1][kSc ? NBL : 1][4], ey[kSums ? 4 : 1][kSums ? NBL : 1][4];
  auto eoff = [&](int i, int j, int v) __attribute__((always_inline)) {
    const int m = min(m0 + wave * 64 + i * 16 + lq * 4 + v, Mg - 1);
    return ((long long)g * Mg + m) * BN + j * 16 + lm;
  };
  auto ebit = [&](unsigned w, int j) __attribute__((always_inline)) {
    return ((w >> (unsigned)(((j & 1) << 4) + lm)) & 1u) != 0u;
  };
  auto sc_load = [&]() __attribute__((always_inline)) {
    if constexpr (kSc) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
#pragma unroll
          for (int jw = 0; jw < NW; ++jw) eh[i][jw][v] = c.sc_hb[eoff(i, 2 * jw, v) >> 5];
#pragma unroll
          for (int j = 0; j < NBL; ++j) edh[i][j][v] = c.sc_dh[eoff(i, j, v)];
        }
    }
  };
  auto sums_load = [&]() __attribute__((always_inline)) {
    if constexpr (kSums) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
#pragma unroll
          for (int j = 0; j < NBL; ++j) ey[i][j][v] = c.bs_y[eoff(i, j, v)];
          if constexpr (kMaskAct) {
#pragma unroll
            for (int jw = 0; jw < NW; ++jw) ea[i][jw][v] = c.bs_hb[eoff(i, 2 * jw, v) >> 5];
          }
        }
    }
  };
  RowsSlab<BN> r0, r1, r2;
  gload(0, r0);
  gload(1, r1);
  int it = 0;
  // every prefetch a real slab while it + 4 < nk; then the last three slabs
  // with the epilogue loads in flight
  for (; it + 5 <= nk; it += 3) {
    gload(it + 2, r2);
    compute(r0);
    gload(it + 3, r0);
    compute(r1);
    gload(it + 4, r1);
    compute(r2);
  }
  gload(it + 2, r2);
  if constexpr (kSc)
    sc_load();
  else
    sums_load();
  compute(r0);
  compute(r1);
  compute(r2);
  if constexpr (kSc) sums_load();

  float* out = c.out + (long long)g * Mg * BN;
  if constexpr (MODE == CONV_FWD) {
    // BN statistics of the tile's 256 rows (one chunk; Mg is a multiple of
    // 256): each wave's 64 rows by a lane butterfly, the four waves in order
    if (c.stats) {
      __shared__ double red[4][BN][2];
#pragma unroll
      for (int j = 0; j < NBL; ++j) {
        double s0 = 0.0, s1 = 0.0;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const double y = (double)acc[i][j][v];
            s0 += y;
            s1 += y * y;
          }
        stats_butterfly(s0, s1, 2, 4);  // the four row groups lq
        if (lq == 0) {
          red[wave][j * 16 + lm][0] = s0;
          red[wave][j * 16 + lm][1] = s1;
        }
      }
      __syncthreads();
      if (tid < BN) {
        double* d = c.stats + (((long long)g * (Mg / 256) + m0 / 256) * BN + tid) * 2;
#pragma unroll
        for (int e = 0; e < 2; ++e)
          d[e] = ((red[0][tid][e] + red[1][tid][e]) + red[2][tid][e]) + red[3][tid][e];
      }
    }
  }
  if constexpr (EPI != 0) {
    // the shortcut share, or the BN backward sums of the tile's 256 rows
    // (Mg is then a multiple of 256: one chunk; lanes by a butterfly, then
    // the four waves in order)
    double bs0[NBL], bs1[NBL];
#pragma unroll
    for (int j = 0; j < NBL; ++j) {
      bs0[j] = 0.0;
      bs1[j] = 0.0;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NBL; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if constexpr (kSc) acc[i][j][v] += ebit(eh[i][j >> 1][v], j) ? edh[i][j][v] : 0.f;
          if constexpr (kSums) {
            const int ch = j * 16 + lm;
            const float y = ey[i][j][v], em = bnp[0][ch], ei = bnp[1][ch];
            bool pass;
            if constexpr (kMaskAct)
              pass = ebit(ea[i][j >> 1][v], j);
            else
              pass = bn_z(bnp[2][ch], y, em, ei, bnp[3][ch]) > 0.f;
            const float dz = pass ? acc[i][j][v] : 0.f;
            const float xh = (y - em) * ei;
            bs0[j] += (double)dz;
            bs1[j] += (double)dz * (double)xh;
          }
        }
    if constexpr (kSums) {
      __shared__ double bred[4][BN][2];
#pragma unroll
      for (int j = 0; j < NBL; ++j) {
        stats_butterfly(bs0[j], bs1[j], 2, 4);
        if (lq == 0) {
          bred[wave][j * 16 + lm][0] = bs0[j];
          bred[wave][j * 16 + lm][1] = bs1[j];
        }
      }
      __syncthreads();
      if (tid < BN) {
        double* d = c.bs_part + (((long long)g * (Mg / 256) + m0 / 256) * BN + tid) * 2;
#pragma unroll
        for (int e = 0; e < 2; ++e)
          d[e] = ((bred[0][tid][e] + bred[1][tid][e]) + bred[2][tid][e]) + bred[3][tid][e];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + wave * 64 + i * 16 + lq * 4 + v;
      if (m < Mg) {
#pragma unroll
        for (int j = 0; j < NBL; ++j) out[(long long)m * BN + j * 16 + lm] = acc[i][j][v];
      }
    }
}

// Input gradient of a stride-2 convolution whose output has twice its
// input's channels (the first convolution of the second and third stages):
// dx (W x W x CI) from dy (Wo x Wo x CO), Wo = W / 2, square images.
// Input position (2a + ph, 2j + pw) receives the taps kh = 1 when ph = 0 and
// kh in {0, 2} when ph = 1 (likewise kw by pw), from dy row
// a + (ph + 1 - kh) / 2 and column j + (pw + 1 - kw) / 2, so the four dy
// neighbours (a + dr, j + dc), dr, dc in {0, 1}, feed all nine taps of the
// four parity classes. A band of BH input rows (256 positions) splits into
// the four classes of BH/2 x Wo = 64 positions, four 16-row MFMA blocks
// each. The band's dy rows (one more below it, zero past the image) and
// columns 0 .. Wo (the last one zero) go to LDS, double buffered: the next
// band's loads are in flight while a band computes. Workgroup (g, i) takes
// the c.mchunk images i c.mchunk, ... of replica g, band by band, and each
// wave keeps the weights it needs in registers throughout:
//   CI = 16: wave w owns block w of every class over the whole reduction;
//   CI = 32: wave w owns every block of every class for input channels
//     16 (w / 2) .. + 15 over half of the output channels (w % 2); the two
//     halves are added through LDS, each wave storing two of the classes.
// The reduction over k = (tap, co) takes co as 16 chunk + 4 (l / 16) + s at
// MFMA step s of a chunk, so a lane reads its four k values of A and of B
// as one float4 each.
// SC: the option-A shortcut's share of the block-input gradient goes into dx
// as it is stored: input position (2 oh, 2 ow) -- the parity class (0, 0) --
// gains the block output's gradient c.sc_dh at (oh, ow) in its first CI
// channels where the output's mask bit (c.sc_hb) is set.
template <int CI, int CO, int W, bool SC>
__global__ __launch_bounds__(kT) __attribute__((amdgpu_waves_per_eu(CI == 16 ? 3 : 2))) void k_conv_dgrad_s2(
    ConvArgs c) {
  constexpr int Wo = W / 2, BH = 256 / W, BANDS = W / BH;
  constexpr int TR = BH / 2 + 1, TC = Wo + 1, PP = CO + 4;  // tile rows, cols, pitch
  constexpr int TQ = TR * TC * (CO / 4);                     // float4 of a tile
  constexpr int TPT = (TQ + kT - 1) / kT;
  constexpr bool kSplit = CI == 32;
  constexpr int NCH = CO / 16, NCW = kSplit ? NCH / 2 : NCH;  // chunks, per wave
  constexpr int NBW = kSplit ? 4 : 1;                         // blocks of a class per wave
  static_assert((CI == 16 || CI == 32) && CO == 2 * CI && (BH / 2) * Wo == 64 &&
                    BH * W == 256, "stage shapes");
  __shared__ __attribute__((aligned(16))) float T[2][TR * TC * PP];
  // halves handed over: [wave][2 classes][4 blocks][4][64 lanes]
  __shared__ __attribute__((aligned(16))) float X[kSplit ? 4 * 2 * 4 * 4 * 64 : 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lq = lane >> 4, lm = lane & 15;
  const int ipw = c.mchunk, groups = c.Bt / ipw, units = ipw * BANDS;
  const int g = blockIdx.x / groups, b0 = (blockIdx.x - g * groups) * ipw;
  const float* dyg = c.dy + ((long long)g * c.Bt + b0) * Wo * Wo * CO;
  const float* Wg = c.Wk + (long long)g * c.sW;  // W [9 CI][CO]
  const int nb = kSplit ? wave >> 1 : 0, half = kSplit ? wave & 1 : 0;
  const int blk0 = kSplit ? 0 : wave;            // first block of a class
  // unit u: image b0 + u / BANDS, band u % BANDS. The loads go out with
  // clamped addresses and are zeroed (bit i of ok clear) only as they are
  // stored to LDS, so that nothing waits for them before then.
  auto gload = [&](int u, v4f(&tv)[TPT], unsigned& ok) __attribute__((always_inline)) {
    const int bi = u / BANDS, oh0 = (u - bi * BANDS) * (BH / 2);
    const float* dy = dyg + (long long)bi * Wo * Wo * CO;
    ok = 0;
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int q = min(tid + kT * i, TQ - 1);
      const int pix = q / (CO / 4), c4 = (q - pix * (CO / 4)) * 4;
      const int tr = pix / TC, tc = pix - tr * TC, oh = oh0 + tr;
      const bool in = oh < Wo && tc < Wo;
      tv[i] = *(const v4f*)(dy + ((long long)(in ? oh : 0) * Wo + (in ? tc : 0)) * CO + c4);
      ok |= (unsigned)in << i;
    }
  };
  auto lstore = [&](float* Tb, const v4f(&tv)[TPT], unsigned ok) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int q = tid + kT * i;
      if (q < TQ) {
        const int pix = q / (CO / 4);
        *(v4f*)&Tb[pix * PP + (q - pix * (CO / 4)) * 4] =
            (ok >> i & 1) ? tv[i] : v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
  };
  // kDeep: two register sets, so unit u + 2's loads are issued before unit u
  // computes (the 32 -> 64 form has no registers to spare for them)
  constexpr bool kDeep = !kSplit;
  v4f tv[TPT], tw[kDeep ? TPT : 1];
  unsigned okv, okw = 0;
  gload(0, tv, okv);
  if constexpr (kDeep) {
    if (units > 1) gload(1, tw, okw);
  }
  // B[k][n] = W[(tap, ci)][co], n = ci - 16 nb = l % 16, co of this wave's chunks
  v4f Bf[9][NCW];
#pragma unroll
  for (int tap = 0; tap < 9; ++tap)
#pragma unroll
    for (int cw = 0; cw < NCW; ++cw)
      Bf[tap][cw] = *(const v4f*)(Wg + ((long long)tap * CI + nb * 16 + lm) * CO +
                                  (half * NCW + cw) * 16 + lq * 4);
  lstore(T[0], tv, okv);
  // every weight fragment in its registers before the loop (vmcnt(0)), so
  // that no wait for them is left inside it
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  // unit u with its tile in T[u & 1]; tn holds (or receives) unit u + 1's
  // loads, tf is free (kDeep)
  auto step = [&](int u, v4f(&tf)[TPT], unsigned& okf, v4f(&tn)[TPT], unsigned& okn)
      __attribute__((always_inline)) {
    const bool more = u + 1 < units;  // uniform over the workgroup
    if constexpr (kDeep) {
      if (u + 2 < units) gload(u + 2, tf, okf);
    } else if (more) {
      gload(u + 1, tn, okn);
    }
    const float* Tb = T[u & 1];
    const int bi = u / BANDS, band = u - bi * BANDS;
    floatx4 acc[4][NBW];
#pragma unroll
    for (int jb = 0; jb < NBW; ++jb) {
      // one block's operands in registers at a time
      if (jb > 0) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int cls = 0; cls < 4; ++cls) acc[cls][jb] = floatx4{0.f, 0.f, 0.f, 0.f};
      // block row m = l % 16 is class position 16 (blk0 + jb) + m: dy tile
      // row (16 / Wo) (blk0 + jb) + m / Wo, column m % Wo
      const float* ap = Tb + (((16 / Wo) * (blk0 + jb) + lm / Wo) * TC + lm % Wo) * PP +
                        half * NCW * 16 + lq * 4;
#pragma unroll
      for (int cw = 0; cw < NCW; ++cw) {
        v4f av[2][2];
#pragma unroll
        for (int dr = 0; dr < 2; ++dr)
#pragma unroll
          for (int dc = 0; dc < 2; ++dc)
            av[dr][dc] = *(const v4f*)(ap + (dr * TC + dc) * PP + cw * 16);
#pragma unroll
        for (int cls = 0; cls < 4; ++cls) {
          const int ph = cls >> 1, pw = cls & 1;
#pragma unroll
          for (int th = 0; th < 1 + ph; ++th) {
            const int kh = ph ? 2 * th : 1, dr = (ph + 1 - kh) / 2;
#pragma unroll
            for (int tw = 0; tw < 1 + pw; ++tw) {
              const int kw = pw ? 2 * tw : 1, dc = (pw + 1 - kw) / 2, tap = kh * 3 + kw;
#pragma unroll
              for (int s = 0; s < 4; ++s)
                acc[cls][jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                    av[dr][dc][s], Bf[tap][cw][s], acc[cls][jb], 0, 0, 0);
            }
          }
        }
      }
    }
    // the shortcut's operands of this lane's class-0 outputs (output
    // position (oh, ow) of block jb, register v), issued after the k work,
    // where its operand registers are free: the 16 -> 32 form once the next
    // tile is in LDS (its registers free too), and stores class 0 last
    float sdh[SC ? NBW : 1][4];
    unsigned swd[SC ? NBW : 1][4];
    auto sc_fetch = [&]() __attribute__((always_inline)) {
      if constexpr (SC) {
        if (!kSplit || half == 0) {
#pragma unroll
          for (int jb = 0; jb < NBW; ++jb) {
            // (v steps ow by one: CO floats, CO / 32 words)
            const int oh = band * (BH / 2) + (16 / Wo) * (blk0 + jb) + (4 * lq) / Wo;
            const long long e =
                ((((long long)g * c.Bt + b0 + bi) * Wo + oh) * Wo + (4 * lq) % Wo) * CO +
                nb * 16 + lm;
            const float* pd = c.sc_dh + e;
            const unsigned* pw = c.sc_hb + (e >> 5);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              sdh[jb][v] = pd[v * CO];
              swd[jb][v] = pw[v * (CO / 32)];
            }
          }
        }
      }
    };
    if constexpr (kSplit) sc_fetch();
    if (more) lstore(T[(u + 1) & 1], tn, okn);
    if constexpr (!kSplit) sc_fetch();
    // lane holds C[m = 4 (l/16) + v][n = l % 16] of each block: class
    // position 16 (blk0 + jb) + 4 (l/16) + v, i.e. a = (16 / Wo) (blk0 + jb) +
    // 4 (l/16) / Wo and j = 4 (l/16) % Wo + v, at input row band BH + 2 a + ph
    // and column 2 j + pw
    float* dx = c.out + ((long long)g * c.Bt + b0 + bi) * W * W * CI +
                (((long long)band * BH + 2 * ((16 / Wo) * blk0 + (4 * lq) / Wo)) * W +
                 2 * ((4 * lq) % Wo)) * CI + nb * 16 + lm;
    auto store = [&](int cls, int jb, floatx4 r) __attribute__((always_inline)) {
      if constexpr (SC) {
        // (channel nb 16 + lm < 32: its bit in the position's first word)
        if (cls == 0) {
#pragma unroll
          for (int v = 0; v < 4; ++v)
            r[v] += (swd[jb][v] >> (unsigned)(nb * 16 + lm)) & 1u ? sdh[jb][v] : 0.f;
        }
      }
#pragma unroll
      for (int v = 0; v < 4; ++v)
        dx[((2 * (16 / Wo) * jb + (cls >> 1)) * W + 2 * v + (cls & 1)) * CI] = r[v];
    };
    if constexpr (kSplit) {
      // half h stores classes 2h, 2h + 1 and hands the other two to its
      // partner wave (w ^ 1); the two partial sums are added once
      float* mine = X + wave * (2 * 4 * 4 * 64);
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
#pragma unroll
          for (int v = 0; v < 4; ++v)
            mine[((k * 4 + jb) * 4 + v) * 64 + lane] = half ? acc[k][jb][v] : acc[2 + k][jb][v];
        }
      __syncthreads();
      const float* other = X + (wave ^ 1) * (2 * 4 * 4 * 64);
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
          floatx4 r;
#pragma unroll
          for (int v = 0; v < 4; ++v)
            r[v] = (half ? acc[2 + k][jb][v] : acc[k][jb][v]) +
                   other[((k * 4 + jb) * 4 + v) * 64 + lane];
          store(2 * half + k, jb, r);
        }
    } else {
#pragma unroll
      for (int cls = 3; cls >= 0; --cls) store(cls, 0, acc[cls][0]);
    }
    __syncthreads();
  };
  if constexpr (kDeep) {
    for (int u = 0; u < units; u += 2) {
      step(u, tv, okv, tw, okw);
      if (u + 1 < units) step(u + 1, tw, okw, tv, okv);
    }
  } else {
    for (int u = 0; u < units; ++u) step(u, tv, okv, tv, okv);
  }
}

// The stem: a 3 x 3 stride-1 convolution of a 3-channel 32 x 32 image (read
// through the row map, or at group stride sx) to 16 channels. The image goes
// to LDS once as a zero-padded 34 x 34 x 3 tile; taps t = (kh, kw, ci) index
// the 27 rows of the [27][16] weight.
constexpr int kStemSide = 32, kStemTile = kStemSide + 2, kStemCin = 3, kStemCout = 16;
constexpr int kStemTaps = 9 * kStemCin;

__device__ __forceinline__ const float* stem_image(const ConvArgs& c, int g, int b) {
  const long long img = (long long)kStemSide * kStemSide * kStemCin;
  return c.rowmap ? c.x + (long long)c.rowmap[(long long)g * c.Bt + b] * img
                  : c.x + (long long)g * c.sx + (long long)b * img;
}

// Zero the tile, then scatter the image's 768 float4 into its interior.
__device__ __forceinline__ void stem_stage(float* T, const float* src) {
  constexpr int NT = kStemTile * kStemTile * kStemCin;
  constexpr int Q = kStemSide * kStemSide * kStemCin / 4;
  static_assert(Q % kT == 0, "whole float4 rounds");
  v4f v[Q / kT];
#pragma unroll
  for (int i = 0; i < Q / kT; ++i) v[i] = *(const v4f*)(src + 4 * (threadIdx.x + kT * i));
  for (int i = threadIdx.x; i < NT; i += kT) T[i] = 0.f;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < Q / kT; ++i) {
    const int e0 = 4 * (threadIdx.x + kT * i);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = e0 + j, pix = e / kStemCin, ci = e - pix * kStemCin;
      const int h = pix / kStemSide, w = pix - h * kStemSide;
      T[((h + 1) * kStemTile + w + 1) * kStemCin + ci] = v[i][j];
    }
  }
  __syncthreads();
}

// Tap t's input value for output position (h, w) from the tile; 0 for t >= 27.
__device__ __forceinline__ float stem_tap(const float* T, int t, int h, int w) {
  const int tt = t < kStemTaps ? t : 0;
  const int kh = tt / 9, kw = (tt / 3) % 3, ci = tt % 3;
  const float v = T[((h + kh) * kStemTile + w + kw) * kStemCin + ci];
  return t < kStemTaps ? v : 0.f;
}

// Forward, one workgroup per (replica, image): y^T = W^T X^T as
// v_mfma_f32_16x16x4f32 blocks of 16 output channels x 16 positions over
// 7 steps of 4 taps (the 28th tap is zero). Lane l holds channels
// 4 (l / 16) .. + 3 of position l % 16 of its block, one float4 store.
__global__ __launch_bounds__(kT) void k_conv_stem_fwd(ConvArgs c) {
  __shared__ float T[kStemTile * kStemTile * kStemCin];
  const int g = blockIdx.x / c.Bt, b = blockIdx.x - g * c.Bt;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lq = lane >> 4, lm = lane & 15;
  const float* Wg = c.Wk + (long long)g * c.sW;
  float wa[7];
#pragma unroll
  for (int ks = 0; ks < 7; ++ks) {
    const int t = 4 * ks + lq;
    wa[ks] = t < kStemTaps ? Wg[t * kStemCout + lm] : 0.f;
  }
  stem_stage(T, stem_image(c, g, b));
  float* out = c.out + ((long long)g * c.Bt + b) * kStemSide * kStemSide * kStemCout;
  // wave w: rows 8w .. 8w+7 (256 positions: one BN statistics chunk), two
  // blocks of 16 columns each
  double s0[4] = {0.0, 0.0, 0.0, 0.0}, s1[4] = {0.0, 0.0, 0.0, 0.0};
  for (int ch = 0; ch < 4; ++ch) {
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const int blk = 4 * ch + bb;
      const int h = 8 * wave + (blk >> 1), w = 16 * (blk & 1) + lm;
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 7; ++ks)
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[ks], stem_tap(T, 4 * ks + lq, h, w),
                                                   acc, 0, 0, 0);
      *(v4f*)(out + (h * kStemSide + 16 * (blk & 1) + lm) * kStemCout + 4 * lq) =
          v4f{acc[0], acc[1], acc[2], acc[3]};
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const double y = (double)acc[v];
        s0[v] += y;
        s1[v] += y * y;
      }
    }
  }
  if (c.stats) {
#pragma unroll
    for (int v = 0; v < 4; ++v) stats_butterfly(s0[v], s1[v], 4, 0);  // the 16 positions
    if (lm == 0) {
      const long long q = (long long)b * 4 + wave;
      double* d = c.stats + ((long long)g * c.Bt * 4 + q) * kStemCout * 2;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        d[(4 * lq + v) * 2] = s0[v];
        d[(4 * lq + v) * 2 + 1] = s1[v];
      }
    }
  }
}

// Weight gradient, workgroup (replica g, split s) over the s-th run of
// whole images (c.mchunk positions, a multiple of 1024):
//   dW[t][co] = sum_p x(p, tap t) dy[p][co]
// as two 16 x 16 blocks of taps (0-15, 16-31; taps 27-31 zero) x 16 output
// channels, 4 positions per v_mfma_f32_16x16x4f32 step. Wave w takes rows
// 8w .. 8w+7 of every image; the four waves' sums are added in wave order
// into the partial [S][G][27][16] for k_conv_wupdate.
__global__ __launch_bounds__(kT) void k_conv_wgrad_stem(ConvArgs c) {
  __shared__ float T[kStemTile * kStemTile * kStemCin];
  __shared__ float R[4][2 * 16 * 16];
  const int g = blockIdx.x / c.splits, s = blockIdx.x - g * c.splits;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lq = lane >> 4, lm = lane & 15;
  constexpr int HW = kStemSide * kStemSide;
  const int img0 = s * (c.mchunk / HW), nimg = c.mchunk / HW;
  floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < nimg && img0 + i < c.Bt; ++i) {
    const int b = img0 + i;
    if (i) __syncthreads();  // every wave is done with the previous tile
    stem_stage(T, stem_image(c, g, b));
    const float* dy = c.dy + ((long long)g * c.Bt + b) * HW * kStemCout;
#pragma unroll 4
    for (int q = 0; q < 64; ++q) {
      const int p = 256 * wave + 4 * q + lq;   // this lane's position
      const int h = p >> 5, w = p & 31;
      const float bv = dy[(long long)p * kStemCout + lm];
      acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(stem_tap(T, lm, h, w), bv, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(stem_tap(T, 16 + lm, h, w), bv, acc1,
                                                  0, 0, 0);
    }
  }
  // C[4 (l/16) + v][l % 16]: rows are taps, columns output channels
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    R[wave][(4 * lq + v) * 16 + lm] = acc0[v];
    R[wave][256 + (4 * lq + v) * 16 + lm] = acc1[v];
  }
  __syncthreads();
  float* part = c.out + ((long long)s * c.G + g) * kStemTaps * kStemCout;
  for (int e = threadIdx.x; e < kStemTaps * kStemCout; e += kT)
    part[e] = ((R[0][e] + R[1][e]) + R[2][e]) + R[3][e];
}

// Stride-1 convolution with 16 channels in and out on 32-wide images (the
// first stage): workgroup (g, b, band group) computes NBW bands of 8 output
// rows x 32 columns x 16 channels of image b, one after the other. The
// 144 x 16 weights go to LDS once per workgroup; per band the input rows
// h0-1 .. h0+8 (zero-padded) go to LDS and all 9 taps read shifted views of
// the tile, so each input value is fetched from memory about 1.25 times
// rather than once per tap, and the next band's rows are loaded into
// registers while a band computes. Input gradient: the same convolution
// applied to dy with the kernel flipped -- tap (kh, kw) uses weight row
// (2-kh, 2-kw) -- and the channels swapped, W[(2-kh, 2-kw, ci)][co] staged
// as [(kh, kw, co)][ci]. Wave w owns output rows h0 + 2w, h0 + 2w + 1 as
// four 16 x 16 blocks of v_mfma_f32_16x16x4f32.
// (EPI: the input-gradient epilogues, loaded at the start of each band)
template <int MODE, int NBW, int EPI = 0>
__global__ __launch_bounds__(kT) void k_conv_halo16(ConvArgs c) {
  constexpr int C = 16, CP = C + 4;          // 80-byte pixel pitch in LDS
  constexpr int W = 32, BH = 8;
  constexpr int TW = W + 2, TH = BH + 2;
  constexpr int TQ = TH * TW * (C / 4);      // float4 of the input tile
  constexpr int WQ = 9 * C * (C / 4);        // float4 of the weights
  constexpr int TPT = (TQ + kT - 1) / kT, WPT = (WQ + kT - 1) / kT;
  __shared__ __attribute__((aligned(16))) float T[TH * TW * CP];
  __shared__ __attribute__((aligned(16))) float Ws[9 * C * CP];
  const int H = c.H, bands = H / BH, groups = bands / NBW;
  int l = blockIdx.x;
  const int grp = l % groups;
  l /= groups;
  const int b = l % c.Bt, g = l / c.Bt;
  const float* src = MODE == CONV_FWD
                         ? c.x + (long long)g * c.sx + (long long)b * H * W * C
                         : c.dy + ((long long)g * c.Bt + b) * H * W * C;
  const float* Wg = c.Wk + (long long)g * c.sW;
  // forward of a block's second convolution: the input BN-ReLU of this
  // thread's four channels (c4 = 4 (tid % 4) for every float4 it stages)
  const bool bnin = MODE == CONV_FWD && c.bn_mu != nullptr;
  BnIn4 bp{};
  if (bnin) bp = bn_in_params(c, g, (threadIdx.x & 3) * 4);
  // a band's input rows into registers: clamped addresses, the padding
  // marked in okm and zeroed at the LDS store
  v4f tv[TPT];
  unsigned okm = 0;
  auto gload = [&](int h0) __attribute__((always_inline)) {
    okm = 0;
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int q = min((int)threadIdx.x + kT * i, TQ - 1);
      const int pix = q >> 2, c4 = (q & 3) * 4;
      const int tr = pix / TW, tc = pix - tr * TW;
      const int ih = h0 - 1 + tr, iw = tc - 1;
      const bool ok = ih >= 0 && ih < H && iw >= 0 && iw < W;
      tv[i] = *(const v4f*)(src + ((long long)(ok ? ih : 0) * W + (ok ? iw : 0)) * C + c4);
      okm |= (unsigned)ok << i;
    }
  };
  auto lstore = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int q = (int)threadIdx.x + kT * i;
      const bool in = okm >> i & 1;
      const v4f v = !in ? v4f{0.f, 0.f, 0.f, 0.f} : bnin ? bn_in(bp, tv[i]) : tv[i];
      if (q < TQ) *(v4f*)&T[(q >> 2) * CP + (q & 3) * 4] = v;
    }
  };
  gload(grp * NBW * BH);
  v4f wv[WPT];
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    // forward: Ws row (tap, ci) is W row (tap, ci); input gradient: Ws row
    // (tap, co) holds W[(8 - tap, ci)][co] over ci, so this thread reads W
    // row (8 - tap, ci) and scatters its four co below
    const int q = min((int)threadIdx.x + kT * i, WQ - 1);
    const int row = q >> 2, c4 = (q & 3) * 4;
    const int tap = row / C, r = row - tap * C;
    const int srow = MODE == CONV_FWD ? row : (8 - tap) * C + r;
    wv[i] = *(const v4f*)(Wg + (long long)srow * C + c4);
  }
  lstore();
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int q = (int)threadIdx.x + kT * i;
    if (q < WQ) {
      if (MODE == CONV_FWD) {
        *(v4f*)&Ws[(q >> 2) * CP + (q & 3) * 4] = wv[i];
      } else {
        const int row = q >> 2, tap = row / C, ci = row - tap * C, c4 = (q & 3) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) Ws[(tap * C + c4 + e) * CP + ci] = wv[i][e];
      }
    }
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lq = lane >> 4, lm = lane & 15;
  constexpr bool kSc = (EPI & kEpiShortcut) != 0;
  constexpr bool kSums = (EPI & (kEpiBnSums | kEpiBnSumsAct)) != 0;
  constexpr bool kMaskAct = (EPI & kEpiBnSumsAct) != 0;
  // BN parameters of this lane's channel (the sums)
  float em = 0.f, ei = 0.f, eg = 0.f, eb = 0.f;
  if constexpr (kSums) {
    em = c.bn_mu[(long long)g * C + lm];
    ei = c.bn_inv[(long long)g * C + lm];
    if constexpr (!kMaskAct) {
      eg = c.bn_g[(long long)g * c.bn_sP + lm];
      eb = c.bn_b[(long long)g * c.bn_sP + lm];
    }
  }
  const long long img = ((long long)g * c.Bt + b) * H * W * C;
  for (int u = 0; u < NBW; ++u) {
    const int band = grp * NBW + u, h0 = band * BH;
    if (u + 1 < NBW) gload(h0 + BH);  // the next band, in flight during this one
    // this lane's 16 outputs: element img + eoff(i, v)
    auto eoff = [&](int i, int v) __attribute__((always_inline)) {
      const int row = h0 + 2 * wave + (i >> 1), col = 16 * (i & 1) + 4 * lq + v;
      return ((long long)row * W + col) * C + lm;
    };
    // epilogue operands: the shortcut's (eh, edh), or the sums' alone (ey
    // and, with the activation mask, ea), issued at the band's start; the
    // sums' next to the shortcut's after the band's k work
    // (the masks as bit words: 16 channels, so the even column 2 vp and the
    // next one share a word, at bits 16 (v % 2) + lm; an image is a whole
    // number of words)
    unsigned eh[kSc ? 4 : 1][2], ea[kMaskAct ? 4 : 1][2];
    float edh[kSc ? 4 : 1][4], ey[kSums ? 4 : 1][4];
    auto ebit = [&](unsigned w, int v) __attribute__((always_inline)) {
      return ((w >> (unsigned)(((v & 1) << 4) + lm)) & 1u) != 0u;
    };
    auto sums_load = [&]() __attribute__((always_inline)) {
      if constexpr (kSums) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int v = 0; v < 4; ++v) ey[i][v] = c.bs_y[img + eoff(i, v)];
          if constexpr (kMaskAct) {
#pragma unroll
            for (int vp = 0; vp < 2; ++vp) ea[i][vp] = c.bs_hb[(img + eoff(i, 2 * vp)) >> 5];
          }
        }
      }
    };
    if constexpr (kSc) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int vp = 0; vp < 2; ++vp) eh[i][vp] = c.sc_hb[(img + eoff(i, 2 * vp)) >> 5];
#pragma unroll
        for (int v = 0; v < 4; ++v) edh[i][v] = c.sc_dh[img + eoff(i, v)];
      }
    } else {
      sums_load();
    }
    floatx4 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int kh = tap / 3, kw = tap - kh * 3;
#pragma unroll
      for (int cq = 0; cq < 4; ++cq) {
        const int ci = cq * 4 + lq;
        const float bv = Ws[(tap * C + ci) * CP + lm];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // output (row 2w + i/2, col 16 (i%2) + lm) reads tile (row + kh, col + kw)
          const int tr = 2 * wave + (i >> 1) + kh, tc = 16 * (i & 1) + lm + kw;
          const float av = T[(tr * TW + tc) * CP + ci];
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[i], 0, 0, 0);
        }
      }
    }
    if constexpr (kSc) sums_load();
    double bs0 = 0.0, bs1 = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float r = acc[i][v];
        if constexpr (kSc) r += ebit(eh[i][v >> 1], v) ? edh[i][v] : 0.f;
        if constexpr (kSums) {
          const float y = ey[i][v];
          bool pass;
          if constexpr (kMaskAct)
            pass = ebit(ea[i][v >> 1], v);
          else
            pass = bn_z(eg, y, em, ei, eb) > 0.f;
          const float dz = pass ? r : 0.f;
          const float xh = (y - em) * ei;
          bs0 += (double)dz;
          bs1 += (double)dz * (double)xh;
        }
        c.out[img + eoff(i, v)] = r;
      }
    if constexpr (kSums) {
      // the band's 256 positions: each wave's two rows by a lane butterfly,
      // the four waves in order
      __shared__ double bred[4][C][2];
      stats_butterfly(bs0, bs1, 2, 4);
      if (lq == 0) {
        bred[wave][lm][0] = bs0;
        bred[wave][lm][1] = bs1;
      }
      __syncthreads();
      if (threadIdx.x < C) {
        const int t = threadIdx.x;
        const long long q = (long long)b * bands + band;
        double* d = c.bs_part + (((long long)g * c.Bt * bands + q) * C + t) * 2;
#pragma unroll
        for (int e = 0; e < 2; ++e)
          d[e] = ((bred[0][t][e] + bred[1][t][e]) + bred[2][t][e]) + bred[3][t][e];
      }
    }
    if (MODE == CONV_FWD && c.stats) {
      // BN statistics of the band (8 x 32 = 256 positions: one chunk): each
      // wave's two rows by a lane butterfly, the four waves in order
      __shared__ double red[4][C][2];
      double s0 = 0.0, s1 = 0.0;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const double y = (double)acc[i][v];
          s0 += y;
          s1 += y * y;
        }
      stats_butterfly(s0, s1, 2, 4);
      if (lq == 0) {
        red[wave][lm][0] = s0;
        red[wave][lm][1] = s1;
      }
      __syncthreads();
      if (threadIdx.x < C) {
        const int t = threadIdx.x;
        const long long q = (long long)b * bands + band;
        double* d = c.stats + (((long long)g * c.Bt * bands + q) * C + t) * 2;
#pragma unroll
        for (int e = 0; e < 2; ++e)
          d[e] = ((red[0][t][e] + red[1][t][e]) + red[2][t][e]) + red[3][t][e];
      }
    }
    if (u + 1 < NBW) {
      __syncthreads();  // every wave is done with this band's tile (and red)
      lstore();
      __syncthreads();
    }
  }
}

// Weight gradient of the first-stage 16 -> 16 stride-1 convolution (32-wide
// images) from the same halo tiles: workgroup (g, split s) walks its bands
// of 8 x 32 output positions; per band the input rows h0-1 .. h0+8 and the
// band's output gradients go to LDS, and each wave takes 64 of the 256
// positions and accumulates all nine taps' 16 x 16 blocks
//   dW[tap][ci][co] += x(p shifted by tap)[ci] * dy[p][co].
// The next band's tiles are loaded into registers while a band computes.
// A lane reads channel l % 16 of position (l / 16), so unpadded 16-float
// pixel rows are read without bank conflicts, and the LDS (38 KB) leaves
// room for four workgroups per CU. The four waves' sums are added in wave
// order; the partial lands in [S][G][144][16] for k_conv_wupdate.
__global__ __launch_bounds__(kT) void k_conv_wgrad_halo16(ConvArgs c) {
  constexpr int C = 16, CP = C;
  constexpr int W = 32, BH = 8, TW = W + 2, TH = BH + 2;
  constexpr int TQ = TH * TW * (C / 4), DQ = BH * W * (C / 4);
  constexpr int TPT = (TQ + kT - 1) / kT, DPT = DQ / kT;
  static_assert(DQ % kT == 0, "band gradient tile");
  // one array: the input tile, the band's gradients, and at the end the
  // four waves' sums in the same space
  __shared__ __attribute__((aligned(16))) float lds[TH * TW * CP + BH * W * CP];
  float* T = lds;
  float* Dsh = lds + TH * TW * CP;
  const int H = c.H, bpi = H / BH;               // bands per image
  const int S = c.splits, sp = blockIdx.x % S, g = blockIdx.x / S;
  const int nb = c.Bt * bpi, per = (nb + S - 1) / S;
  const int bb = sp * per, be = min(nb, bb + per);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lq = lane >> 4, lm = lane & 15;
  floatx4 acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  // a block's second convolution: the input BN-ReLU of this thread's four
  // channels (c4 = 4 (tid % 4) for every float4 it stages)
  const bool bnin = c.bn_mu != nullptr;
  BnIn4 bp{};
  if (bnin) bp = bn_in_params(c, g, (threadIdx.x & 3) * 4);
  // band bd's tiles into registers: clamped addresses, padding marked in
  // okm and zeroed at the LDS store
  v4f tv[TPT], dv[DPT];
  unsigned okm = 0;
  auto gload = [&](int bd) __attribute__((always_inline)) {
    const int b = bd / bpi, h0 = (bd - b * bpi) * BH;
    const float* xs = c.x + (long long)g * c.sx + (long long)b * H * W * C;
    const float* ds = c.dy + (((long long)g * c.Bt + b) * H + h0) * W * C;
    okm = 0;
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int q = min((int)threadIdx.x + kT * i, TQ - 1);
      const int pix = q >> 2, c4 = (q & 3) * 4;
      const int tr = pix / TW, tc = pix - tr * TW;
      const int ih = h0 - 1 + tr, iw = tc - 1;
      const bool ok = ih >= 0 && ih < H && iw >= 0 && iw < W;
      tv[i] = *(const v4f*)(xs + ((long long)(ok ? ih : 0) * W + (ok ? iw : 0)) * C + c4);
      okm |= (unsigned)ok << i;
    }
#pragma unroll
    for (int i = 0; i < DPT; ++i) dv[i] = *(const v4f*)(ds + 4 * ((int)threadIdx.x + kT * i));
  };
  if (bb < be) gload(bb);
  for (int bd = bb; bd < be; ++bd) {
    __syncthreads();  // the previous band's tiles are no longer read
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      const int q = (int)threadIdx.x + kT * i;
      const bool in = okm >> i & 1;
      const v4f v = !in ? v4f{0.f, 0.f, 0.f, 0.f} : bnin ? bn_in(bp, tv[i]) : tv[i];
      if (q < TQ) *(v4f*)&T[(q >> 2) * CP + (q & 3) * 4] = v;
    }
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int q = (int)threadIdx.x + kT * i;
      *(v4f*)&Dsh[(q >> 2) * CP + (q & 3) * 4] = dv[i];
    }
    __syncthreads();
    if (bd + 1 < be) gload(bd + 1);  // uniform over the workgroup
#pragma unroll 2
    for (int ks = 0; ks < 16; ++ks) {
      // position of this lane's k: row 2w + ks/8, column 4 (ks%8) + lq
      const int pr = 2 * wave + (ks >> 3), pc = 4 * (ks & 7) + lq;
      const float bv = Dsh[(pr * W + pc) * CP + lm];
      // the nine taps at constant offsets from the lane's tile position
      const float* tb = T + (pr * TW + pc) * CP + lm;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int kh = t / 3, kw = t - kh * 3;
        const float av = tb[(kh * TW + kw) * CP];
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[t], 0, 0, 0);
      }
    }
  }
  // waves in order; block t register v of lane l: dW[t][4 (l/16) + v][l%16]
  __syncthreads();
  float* red = lds;  // 4 x 144 x 16 floats fit the tile space (5440 + 4096)
  static_assert(4 * 9 * C * C <= TH * TW * CP + BH * W * CP, "reduction space");
#pragma unroll
  for (int t = 0; t < 9; ++t)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      red[wave * 9 * C * C + (t * C + lq * 4 + v) * C + lm] = acc[t][v];
  __syncthreads();
  float* out = c.out + ((long long)sp * c.G + g) * 9 * C * C;
  for (int e = threadIdx.x; e < 9 * C * C; e += kT)
    out[e] = ((red[e] + red[9 * C * C + e]) + red[2 * 9 * C * C + e]) + red[3 * 9 * C * C + e];
}

// Weight gradient of the stage-2 and stage-3 convolutions (output rows of
// WO = 16 or 8 positions) from band tiles. A band is SP = 64 output positions,
// 64 / WO whole output rows of one image; per band the output gradients
// [64][CO] and the input rows its taps read, [(BH - 1) STRIDE + 3] x
// [(WO - 1) STRIDE + 3] x CI with the zero padding, go to LDS once for all
// nine taps (two buffers: the next band's loads are in flight while this band
// computes). The (tap, 16-column block) pairs of dW are dealt to the waves --
// pair p to wave p % 4 -- and each wave accumulates its pairs over all 64
// positions of every band (v_mfma_f32_16x16x4f32: lane l takes input channel
// 16 i + l % 16 and output channel 16 n + l % 16 at position 4 kk + l / 16),
// so no cross-wave sum is needed. Workgroup (g, split s) walks bands
// [s per, (s + 1) per) of replica g, per = ceil(bands / S), in ascending
// order; its partial sum lands in [S][G][9 CI][CO] for k_conv_wupdate.
// LDS bytes of a k_conv_wgrad_band instance (both buffers).
template <int CI, int CO, int STRIDE, int WO>
constexpr size_t wgrad_band_lds() {
  constexpr int BH = 64 / WO;
  constexpr int TH = (BH - 1) * STRIDE + 3, TW = (WO - 1) * STRIDE + 3;
  return ((size_t)2 * (TH * TW * (CI + 4) + 64 * (CO + 4)) + 4 * CI) * sizeof(float);
}
// Workgroups per CU a k_conv_wgrad_band instance is built for: one for the
// large accumulator sets (64 output channels), else as many as its LDS
// allows, at most three (the register budget follows).
template <int CI, int CO, int STRIDE, int WO>
constexpr int wgrad_band_min_wgs() {
  constexpr int lds_wgs = (int)(163840 / wgrad_band_lds<CI, CO, STRIDE, WO>());
  return (9 * (CO / 16) + 3) / 4 * (CI / 16) > 16 ? 1 : (lds_wgs < 3 ? lds_wgs : 3);
}

template <int CI, int CO, int STRIDE, int WO>
__global__ __launch_bounds__(kT, (wgrad_band_min_wgs<CI, CO, STRIDE, WO>())) void
k_conv_wgrad_band(ConvArgs c) {
  constexpr int SP = 64, BH = SP / WO;
  constexpr int TH = (BH - 1) * STRIDE + 3, TW = (WO - 1) * STRIDE + 3;
  constexpr int XP = CI + 4, DP = CO + 4;               // LDS pitches (16-byte rows)
  constexpr int XQ = TH * TW * (CI / 4), DQ = SP * (CO / 4);  // float4 per tile
  constexpr int XPT = (XQ + kT - 1) / kT, DPT = (DQ + kT - 1) / kT;
  constexpr int MB = CI / 16, NB = CO / 16, NP = 9 * NB, PPW = (NP + 3) / 4;
  constexpr int XF = TH * TW * XP, DF = SP * DP;        // floats per buffer
  static_assert(DQ % kT == 0, "whole float4 rounds of the gradient tile");
  // [2][XF], then [2][DF], then the input BN-ReLU's [4][CI]
  extern __shared__ __attribute__((aligned(16))) float lds[];
  float* Xs = lds;
  float* Ds = lds + 2 * XF;
  float* bnp = lds + 2 * (XF + DF);

  const int S = c.splits, sp = blockIdx.x % S, g = blockIdx.x / S;
  const int bpi = c.Ho / BH;                            // bands per image
  const int nbands = c.Bt * bpi, per = (nbands + S - 1) / S;
  const int b0 = sp * per, nbd = max(0, min(nbands, b0 + per) - b0);
  // Large accumulator sets (64 output channels: one wave per SIMD) read the
  // operands of step kk + 1 from LDS while step kk's MFMAs run; the smaller
  // ones keep several waves per SIMD and read each step's operands as they
  // go (measured: the read-ahead costs them occupancy and 50% more time).
  constexpr bool kBig = PPW * MB > 16;
  const int tid = threadIdx.x, lane = tid & 63;
  // (the small sets take the wave index as a scalar; measured: the large
  // ones schedule worse with it)
  const int wave = kBig ? tid >> 6 : __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lq = lane >> 4, lm = lane & 15;
  // a block's second convolution: the input BN-ReLU (statistics and
  // parameters per input channel in LDS; every float4 this thread stages
  // has channels c4 .. c4 + 3, c4 = 4 (tid % (CI / 4)))
  const bool bnin = c.bn_mu != nullptr;
  if (bnin) {
    for (int t = tid; t < CI; t += kT) {
      bnp[t] = c.bn_mu[(long long)g * CI + t];
      bnp[CI + t] = c.bn_inv[(long long)g * CI + t];
      bnp[2 * CI + t] = c.bn_g[(long long)g * c.bn_sP + t];
      bnp[3 * CI + t] = c.bn_b[(long long)g * c.bn_sP + t];
    }
    __syncthreads();
  }

  // every load of band bd in flight at once (clamped addresses, padding
  // zeroed at use)
  auto gload = [&](int bd, v4f(&xr)[XPT], v4f(&dr)[DPT], unsigned& okm)
      __attribute__((always_inline)) {
    okm = 0;
    const int b = bd / bpi, oh0 = (bd - b * bpi) * BH;
    const float* xs = c.x + (long long)g * c.sx + (long long)b * c.H * c.W * CI;
    const int ih0 = oh0 * STRIDE - 1;
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int q = min(tid + kT * i, XQ - 1);
      const int pix = q / (CI / 4), c4 = (q - pix * (CI / 4)) * 4;
      const int tr = pix / TW, tc = pix - tr * TW;
      const int ih = ih0 + tr, iw = tc - 1;
      const bool ok = ih >= 0 && ih < c.H && iw >= 0 && iw < c.W;
      xr[i] = *(const v4f*)(xs + ((long long)(ok ? ih : 0) * c.W + (ok ? iw : 0)) * CI + c4);
      if (!ok) xr[i] = v4f{0.f, 0.f, 0.f, 0.f};
      okm |= (unsigned)ok << i;
    }
    const float* ds = c.dy + (((long long)g * c.Bt + b) * c.Ho + oh0) * WO * CO;
#pragma unroll
    for (int i = 0; i < DPT; ++i) dr[i] = *(const v4f*)(ds + 4 * (tid + kT * i));
  };
  auto lstore = [&](int buf, const v4f(&xr)[XPT], const v4f(&dr)[DPT], unsigned okm)
      __attribute__((always_inline)) {
    BnIn4 p{};
    if (bnin) {
      const int c4 = (tid % (CI / 4)) * 4;
      p.m = *(const v4f*)&bnp[c4];
      p.iv = *(const v4f*)&bnp[CI + c4];
      p.g = *(const v4f*)&bnp[2 * CI + c4];
      p.b = *(const v4f*)&bnp[3 * CI + c4];
    }
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int q = tid + kT * i;
      if (q < XQ) {
        const int pix = q / (CI / 4), c4 = (q - pix * (CI / 4)) * 4;
        v4f v = xr[i];
        if (bnin) v = (okm >> i & 1) ? bn_in(p, v) : v4f{0.f, 0.f, 0.f, 0.f};  // padding stays 0
        *(v4f*)&Xs[buf * XF + pix * XP + c4] = v;
      }
    }
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int q = tid + kT * i;
      const int pos = q / (CO / 4), c4 = (q - pos * (CO / 4)) * 4;
      *(v4f*)&Ds[buf * DF + pos * DP + c4] = dr[i];
    }
  };
  floatx4 acc[PPW][MB];
#pragma unroll
  for (int pp = 0; pp < PPW; ++pp)
#pragma unroll
    for (int i = 0; i < MB; ++i) acc[pp][i] = floatx4{0.f, 0.f, 0.f, 0.f};
  // this wave's pairs: the offset of the pair's tap in the input tile and of
  // its column block in the gradient tile
  int xoff[PPW], doff[PPW];
#pragma unroll
  for (int pp = 0; pp < PPW; ++pp) {
    const int p = min(wave + 4 * pp, NP - 1);
    const int tap = p / NB, nbk = p - tap * NB, kh = tap / 3, kw = tap - kh * 3;
    xoff[pp] = (kh * TW + kw) * XP + lm;
    doff[pp] = nbk * 16 + lm;
  }
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const float* X = Xs + buf * XF;
    const float* D = Ds + buf * DF;
    if constexpr (!kBig) {
      // every pair slot computes (a slot past the last pair repeats the last
      // pair's operands into accumulators that are never stored), so the
      // reads of one step carry no branches and overlap the MFMAs
#pragma unroll 2
      for (int kk = 0; kk < SP / 4; ++kk) {
        const int pos = kk * 4 + lq, orow = pos / WO, ocol = pos - orow * WO;
        const int xb = (orow * STRIDE * TW + ocol * STRIDE) * XP, db = pos * DP;
        float av[PPW][MB], bv[PPW];
#pragma unroll
        for (int pp = 0; pp < PPW; ++pp) {
          bv[pp] = D[db + doff[pp]];
#pragma unroll
          for (int i = 0; i < MB; ++i) av[pp][i] = X[xb + xoff[pp] + i * 16];
        }
#pragma unroll
        for (int pp = 0; pp < PPW; ++pp)
#pragma unroll
          for (int i = 0; i < MB; ++i)
            acc[pp][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[pp][i], bv[pp], acc[pp][i], 0, 0, 0);
      }
      return;
    }
    float av[2][PPW][MB], bv[2][PPW];
    auto fetch = [&](int kk, int st) __attribute__((always_inline)) {
      const int pos = kk * 4 + lq, orow = pos / WO, ocol = pos - orow * WO;
      const int xb = (orow * STRIDE * TW + ocol * STRIDE) * XP, db = pos * DP;
#pragma unroll
      for (int pp = 0; pp < PPW; ++pp) {
        if (wave + 4 * pp < NP) {  // uniform over the wave
          bv[st][pp] = D[db + doff[pp]];
#pragma unroll
          for (int i = 0; i < MB; ++i) av[st][pp][i] = X[xb + xoff[pp] + i * 16];
        }
      }
    };
    fetch(0, 0);
#pragma unroll 2
    for (int kk = 0; kk < SP / 4; ++kk) {
      const int st = kk & 1;
      if (kk + 1 < SP / 4) fetch(kk + 1, st ^ 1);
#pragma unroll
      for (int pp = 0; pp < PPW; ++pp) {
        if (wave + 4 * pp < NP) {
#pragma unroll
          for (int i = 0; i < MB; ++i)
            acc[pp][i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[st][pp][i], bv[st][pp],
                                                              acc[pp][i], 0, 0, 0);
        }
      }
    }
  };
  // The large accumulator sets keep one register set of prefetched tiles:
  // band t + 1's loads are in flight while band t computes, then go to the
  // LDS buffer band t - 1 released at the last barrier.
  if constexpr (kBig) {
    if (nbd > 0) {
      v4f xr[XPT], dr[DPT];
      unsigned ok;
      gload(b0, xr, dr, ok);
      lstore(0, xr, dr, ok);
      __syncthreads();
      for (int t = 0; t < nbd; ++t) {
        const bool more = t + 1 < nbd;  // uniform over the workgroup
        if (more) gload(b0 + t + 1, xr, dr, ok);
        __builtin_amdgcn_sched_barrier(0);
        compute(t & 1);
        if (more) lstore((t + 1) & 1, xr, dr, ok);
        __syncthreads();
      }
    }
  } else if (nbd > 0) {
    v4f xr0[XPT], xr1[XPT], dr0[DPT], dr1[DPT];
    unsigned ok0, ok1;
    auto band = [&](int t) __attribute__((always_inline)) { return b0 + min(t, nbd - 1); };
    gload(band(0), xr0, dr0, ok0);
    gload(band(1), xr1, dr1, ok1);
    lstore(0, xr0, dr0, ok0);
    __syncthreads();
    int it = 0;
    for (; it + 1 < nbd; it += 2) {
      gload(band(it + 2), xr0, dr0, ok0);
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      lstore(1, xr1, dr1, ok1);
      __syncthreads();
      gload(band(it + 3), xr1, dr1, ok1);
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      lstore(0, xr0, dr0, ok0);
      __syncthreads();
    }
    if (it < nbd) compute(0);  // odd band count: the last band is in buffer 0
  }
  // block (pair, i) register v of lane l: dW[tap][16 i + 4 (l/16) + v][16 n + l%16]
  float* out = c.out + ((long long)sp * c.G + g) * 9 * CI * CO;
#pragma unroll
  for (int pp = 0; pp < PPW; ++pp) {
    const int p = wave + 4 * pp;
    if (p < NP) {
      const int tap = p / NB, nbk = p - tap * NB;
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          out[(long long)(tap * CI + i * 16 + 4 * lq + v) * CO + nbk * 16 + lm] = acc[pp][i][v];
    }
  }
}

// Weight gradient: sum the S partials (ascending s) and apply the update to
// the [9*Cin][Cout] weight of every replica.
template <int S>
__global__ void k_conv_wupdate(const float* part, int G, int n, float* W, float* U,
                               long long sP, float lr, float mom, float wd,
                               int nesterov) {
  const long long total = (long long)G * n;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    float p[S];
#pragma unroll
    for (int s = 0; s < S; ++s) p[s] = part[i + s * total];
    float grad = p[0];
#pragma unroll
    for (int s = 1; s < S; ++s) grad += p[s];
    const int g = (int)(i / n);
    const long long o = (long long)g * sP + (i - (long long)g * n);
    float w = W[o], u = U[o];
    const float gr = __builtin_fmaf(wd, w, grad);
    u = __builtin_fmaf(mom, u, gr);
    const float d = step_dir(u, gr, mom, nesterov);
    w = __builtin_fmaf(-lr, d, w);
    W[o] = w;
    U[o] = u;
  }
}

// ------------------------------------------------------------ batch norm
// Partial sums of one row chunk per workgroup, fp64: for the forward pass
// sum(y) and sum(y^2); for the backward pass sum(dz) and sum(dz * xhat),
// where dz = upstream gradient masked by the ReLU derivative -- the
// activation's mask bits when given, else bn_z(gamma, y, mu, inv, beta) > 0 -- and
// xhat = (y - mu) * inv. Channel count C divides 256. Rows per chunk: 1024
// for the largest layers, fewer for smaller ones so that every layer's
// launch has at least 32 chunks per replica to spread over the chip.
__host__ __device__ __forceinline__ int bn_chunk_rows(int R) {
  return R >= (1 << 17) ? 1024 : R >= (1 << 15) ? 512 : 256;
}

// Backward coefficients per (replica g, channel c), field f at
// coef[f * G * C + g * C + c]: gamma * inv, dbeta / R, dgamma / R, and gamma,
// beta as they were before this step's update.

// Running statistics of a BN layer after a training batch of R values per
// channel: exponential averages (factor kBnRunMomentum) of the batch mean and
// of the unbiased variance var R / (R - 1), in fp64 and stored as fp32.
constexpr double kBnRunMomentum = 0.1;
__device__ __forceinline__ void bn_running(float* rm, float* rv, long long o, double m,
                                           double var, int R) {
  const double a = kBnRunMomentum;
  rm[o] = (float)((1.0 - a) * (double)rm[o] + a * m);
  rv[o] = (float)((1.0 - a) * (double)rv[o] + a * (var * ((double)R / (double)(R - 1))));
}

// Finalisation of one BN layer, one workgroup per replica: lane q of channel
// c adds the chunk partials q, q + L, q + 2L, ... (L = 256 / C lanes,
// ascending), then the lanes are added in a fixed tree, and thread c < C
// finalises channel c.
// Forward: mu, inv = 1/sqrt(var + eps) (and the running statistics).
// Backward: the input-gradient coefficients and the update of gamma, beta:
//   dbeta = sum dz, dgamma = sum dz*xhat,
//   dy = gamma*inv*(dz - dbeta/R - xhat*dgamma/R)  -> coef = (gamma*inv,
//   dbeta/R, dgamma/R, gamma, beta); then gamma, beta take a momentum-SGD step
//   (no decay).
__global__ __launch_bounds__(kT) void k_bn_finalize_wg(
    const double* part, int nchunk, int C, int R, float* mu, float* inv, float* coef,
    float* gamma, float* beta, float* ug, float* ub, long long sP, float lr, float mom,
    int nesterov, float eps, float* rm, float* rv, long long sRS, float* gsnap,
    float* bsnap) {
  __shared__ double red[2][kT];
  const int g = blockIdx.x, t = threadIdx.x;
  const int L = kT / C, c = t % C, q = t / C;
  double s0 = 0.0, s1 = 0.0;
#pragma unroll 8
  for (int ch = q; ch < nchunk; ch += L) {
    const double* p = part + (((long long)g * nchunk + ch) * C + c) * 2;
    s0 += p[0];
    s1 += p[1];
  }
  red[0][t] = s0;
  red[1][t] = s1;
  __syncthreads();
  for (int w = kT / 2; w >= C; w >>= 1) {
    if (t < w) {
      red[0][t] += red[0][t + w];
      red[1][t] += red[1][t + w];
    }
    __syncthreads();
  }
  if (t >= C) return;
  s0 = red[0][t];
  s1 = red[1][t];
  const int i = g * C + c;
  if (coef == nullptr) {  // forward statistics
    const double m = s0 / R;
    double var = s1 / R - m * m;
    if (var < 0.0) var = 0.0;
    mu[i] = (float)m;
    inv[i] = (float)(1.0 / sqrt(var + (double)eps));
    if (rm) bn_running(rm, rv, (long long)g * sRS + c, m, var, R);
    if (gsnap) {  // the scale and shift this batch is normalised with
      gsnap[i] = gamma[(long long)g * sP + c];
      bsnap[i] = beta[(long long)g * sP + c];
    }
    return;
  }
  const long long o = (long long)g * sP + c;
  float gm = gamma[o], bt = beta[o];
  const int GC = (int)gridDim.x * C;
  coef[i] = gm * inv[i];
  coef[GC + i] = (float)(s0 / R);
  coef[2 * GC + i] = (float)(s1 / R);
  coef[3 * GC + i] = gm;
  coef[4 * GC + i] = bt;
  float u = ug[o];
  const float dgm = (float)s1;
  u = __builtin_fmaf(mom, u, dgm);
  float d = step_dir(u, dgm, mom, nesterov);
  gamma[o] = __builtin_fmaf(-lr, d, gm);
  ug[o] = u;
  u = ub[o];
  const float dbt = (float)s0;
  u = __builtin_fmaf(mom, u, dbt);
  d = step_dir(u, dbt, mom, nesterov);
  beta[o] = __builtin_fmaf(-lr, d, bt);
  ub[o] = u;
}

// ---- float4 forms of the BN passes (channel count C a power of two >= 16):
// the replica is the grid's y coordinate and a thread owns 4 consecutive
// channels of one row, so the channel is a mask of the index and no 64-bit
// division is left in the inner work.

// Partial sums of one row chunk per workgroup, 4 channels per thread: rows
// of a chunk interleaved over the 1024 / C row lanes of a workgroup, fp64
// sums per channel, then added in a fixed tree.
__global__ __launch_bounds__(kT) void k_bn_partial4(const float* y, int R, int C,
                                                    const float* gup, const unsigned* mbits,
                                                    const float* mu, const float* inv,
                                                    const float* gamma, const float* beta,
                                                    long long sP, double* part,
                                                    int nchunk) {
  __shared__ double red[2][4][kT];
  const int g = blockIdx.y, ch = blockIdx.x;
  const int cq = C / 4;  // threads per row
  const int c0 = (threadIdx.x % cq) * 4, lane_r = threadIdx.x / cq, rstep = kT / cq;
  const long long base = (long long)g * R * C;
  const int cr = bn_chunk_rows(R);
  const int r0 = ch * cr, r1 = min(R, r0 + cr);
  const bool bwd = gup != nullptr;
  const bool zmask = bwd && mbits == nullptr;
  float m_c[4], i_c[4], g_c[4], b_c[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    m_c[e] = bwd ? mu[g * C + c0 + e] : 0.f;
    i_c[e] = bwd ? inv[g * C + c0 + e] : 0.f;
    g_c[e] = zmask ? gamma[(long long)g * sP + c0 + e] : 0.f;
    b_c[e] = zmask ? beta[(long long)g * sP + c0 + e] : 0.f;
  }
  double s0[4] = {0.0, 0.0, 0.0, 0.0}, s1[4] = {0.0, 0.0, 0.0, 0.0};
  for (int rb = r0 + lane_r; rb < r1; rb += 4 * rstep) {
    v4f yv[4], gv[4];
    unsigned mw[4];  // the mask: bit e of (mw >> o % 32) is channel c0 + e's
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = min(rb + u * rstep, r1 - 1);
      const long long o = base + (long long)r * C + c0;
      yv[u] = *(const v4f*)(y + o);
      gv[u] = bwd ? *(const v4f*)(gup + o) : v4f{0.f, 0.f, 0.f, 0.f};
      mw[u] = mbits ? mbits[o >> 5] >> (unsigned)(o & 31) : 0u;
      if (zmask) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          mw[u] |= (bn_z(g_c[e], yv[u][e], m_c[e], i_c[e], b_c[e]) > 0.f ? 1u : 0u) << e;
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (rb + u * rstep >= r1) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (!bwd) {
          s0[e] += (double)yv[u][e];
          s1[e] += (double)yv[u][e] * (double)yv[u][e];
        } else {
          const float dz = (mw[u] >> e) & 1u ? gv[u][e] : 0.f;
          const float xh = (yv[u][e] - m_c[e]) * i_c[e];
          s0[e] += (double)dz;
          s1[e] += (double)dz * (double)xh;
        }
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    red[0][e][threadIdx.x] = s0[e];
    red[1][e][threadIdx.x] = s1[e];
  }
  __syncthreads();
  for (int w = kT / 2; w >= cq; w >>= 1) {
    if ((int)threadIdx.x < w) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        red[0][e][threadIdx.x] += red[0][e][threadIdx.x + w];
        red[1][e][threadIdx.x] += red[1][e][threadIdx.x + w];
      }
    }
    __syncthreads();
  }
  if ((int)threadIdx.x < cq) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double* p = part + (((long long)g * nchunk + ch) * C + c0 + e) * 2;
      p[0] = red[0][e][threadIdx.x];
      p[1] = red[1][e][threadIdx.x];
    }
  }
}

// BN output z = gamma*(y - mu)*inv + beta, 4 channels per thread (mu, inv,
// gamma, beta read as float4); then one of
//   mode 0: out = relu(z)
//   mode 1: out = relu(z + x_in)               (identity shortcut)
//   mode 2: out = relu(z + shortcutA(x_in))    (stride-2 option-A shortcut:
//           every second pixel, the first Cin channels)
__global__ __launch_bounds__(kT) void k_bn_apply4(const float* y, int R, int C, int cshift,
                                                  const float* mu, const float* inv,
                                                  const float* gamma, const float* beta,
                                                  long long sP, int mode, const float* xin,
                                                  int Ho, int Wo, int Cin, float* out,
                                                  unsigned* mbits) {
  const int g = blockIdx.y;
  const int j = blockIdx.x * kT + threadIdx.x;
  if (j >= R * C / 4) return;  // R C / 4 is a multiple of 8 with mbits
  const int e4 = 4 * j, c0 = e4 & (C - 1), r = e4 >> cshift;
  const long long o = (long long)g * R * C + e4;
  const v4f yv = *(const v4f*)(y + o);
  v4f xv = v4f{0.f, 0.f, 0.f, 0.f};
  if (mode == 1) {
    xv = *(const v4f*)(xin + o);
  } else if (mode == 2 && c0 < Cin) {
    const int HWo = Ho * Wo, b = r / HWo, p = r - b * HWo;
    const int oh = p / Wo, ow = p - oh * Wo;
    const int H = 2 * Ho, W = 2 * Wo, Bt = R / HWo;
    xv = *(const v4f*)(xin + (((long long)g * Bt + b) * H * W + (long long)(2 * oh) * W +
                              2 * ow) * Cin + c0);
  }
  const v4f m4 = *(const v4f*)(mu + g * C + c0), i4 = *(const v4f*)(inv + g * C + c0);
  const v4f g4 = *(const v4f*)(gamma + (long long)g * sP + c0);
  const v4f b4 = *(const v4f*)(beta + (long long)g * sP + c0);
  v4f res;
  unsigned nib = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float v = bn_z(g4[e], yv[e], m4[e], i4[e], b4[e]) + xv[e];
    res[e] = v > 0.f ? v : 0.f;
    nib |= (v > 0.f ? 1u : 0u) << e;
  }
  *(v4f*)(out + o) = res;
  if (mbits) {
    // the mask word of 32 consecutive elements: the nibbles of the eight
    // threads 8q .. 8q + 7 (all present: a group never straddles R C / 4)
    unsigned w = nib << (4 * (threadIdx.x & 7));
    w |= __shfl_xor(w, 1, 64);
    w |= __shfl_xor(w, 2, 64);
    w |= __shfl_xor(w, 4, 64);
    if ((threadIdx.x & 7) == 0) mbits[o >> 5] = w;
  }
}

// The BN input gradient, 4 channels per thread:
//   dy = gamma inv (dz - dbeta / R - x^ dgamma / R) with the coefficients of
// k_bn_finalize_wg, dz = gup where the ReLU passed (mask bits mbits, or, with
// mbits null, the recomputed sign of gamma (y - mu) inv + beta), x^ = (y - mu) inv.
__global__ __launch_bounds__(kT) void k_bn_bwd_apply4(const float* y, const float* gup,
                                                      const unsigned* mbits, int R, int C,
                                                      const float* mu, const float* inv,
                                                      const float* coef, float* dy) {
  const int g = blockIdx.y;
  const int j = blockIdx.x * kT + threadIdx.x;
  if (j >= R * C / 4) return;
  const int e4 = 4 * j, c0 = e4 & (C - 1);
  const long long o = (long long)g * R * C + e4;
  const int gc = g * C + c0, GC = (int)gridDim.y * C;
  const v4f yv = *(const v4f*)(y + o), gv = *(const v4f*)(gup + o);
  const v4f m4 = *(const v4f*)(mu + gc), i4 = *(const v4f*)(inv + gc);
  const v4f k0 = *(const v4f*)(coef + gc), k1 = *(const v4f*)(coef + GC + gc),
            k2 = *(const v4f*)(coef + 2 * GC + gc);
  unsigned mw = 0;  // bit e: channel c0 + e passes the ReLU
  if (mbits) {
    mw = mbits[o >> 5] >> (unsigned)(o & 31);
  } else {
    const v4f k3 = *(const v4f*)(coef + 3 * GC + gc), k4 = *(const v4f*)(coef + 4 * GC + gc);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      mw |= (bn_z(k3[e], yv[e], m4[e], i4[e], k4[e]) > 0.f ? 1u : 0u) << e;
  }
  v4f res;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float dz = (mw >> e) & 1u ? gv[e] : 0.f;
    const float xh = (yv[e] - m4[e]) * i4[e];
    res[e] = k0[e] * (dz - k1[e] - xh * k2[e]);
  }
  *(v4f*)(dy + o) = res;
}

// The shortcut's share of the block-input gradient, 4 channels per thread:
// dx += dh_out where the block output passed its ReLU (mask bits hb_out).
// Identity: every element of dx. Option A: one thread per (output position,
// 4 of the first Cin channels), adding to the even input pixel it was taken
// from.
__global__ __launch_bounds__(kT) void k_shortcut_grad4(float* dx, const float* dh_out,
                                                       const unsigned* hb_out, int Bt, int H,
                                                       int W, int Cin, int Cout, int mode) {
  const int g = blockIdx.y;
  const int j = blockIdx.x * kT + threadIdx.x;
  if (mode == 1) {
    if (j >= Bt * H * W * Cin / 4) return;
    const long long o = (long long)g * Bt * H * W * Cin + 4 * j;
    v4f d = *(const v4f*)(dx + o);
    const v4f gq = *(const v4f*)(dh_out + o);
    const unsigned mw = hb_out[o >> 5] >> (unsigned)(o & 31);
#pragma unroll
    for (int e = 0; e < 4; ++e) d[e] += (mw >> e) & 1u ? gq[e] : 0.f;
    *(v4f*)(dx + o) = d;
    return;
  }
  const int Ho = H / 2, Wo = W / 2, cq = Cin / 4;
  if (j >= Bt * Ho * Wo * cq) return;
  const int c0 = (j % cq) * 4, pos = j / cq;  // pos = (b, oh, ow)
  const int b = pos / (Ho * Wo), p = pos - b * Ho * Wo, oh = p / Wo, ow = p - oh * Wo;
  const long long oo = ((long long)g * Bt * Ho * Wo + pos) * Cout + c0;
  const long long oi = (((long long)g * Bt + b) * H * W + (long long)(2 * oh) * W + 2 * ow) * Cin + c0;
  v4f d = *(const v4f*)(dx + oi);
  const v4f gq = *(const v4f*)(dh_out + oo);
  const unsigned mw = hb_out[oo >> 5] >> (unsigned)(oo & 31);
#pragma unroll
  for (int e = 0; e < 4; ++e) d[e] += (mw >> e) & 1u ? gq[e] : 0.f;
  *(v4f*)(dx + oi) = d;
}

// Global average pool [G*Bt][S][C] -> [G*Bt][C] (sum in ascending position).
__global__ void k_gap(const float* h, int rows, int S, int C, float* feat) {
  const long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x;
  if (i >= (long long)rows * C) return;
  const long long r = i / C;
  const int c = (int)(i % C);
  float s = 0.f;
  for (int p = 0; p < S; ++p) s += h[(r * S + p) * C + c];
  feat[i] = s / (float)S;
}

// dh[r][p][c] = dfeat[r][c] / S (the pool's gradient).
__global__ void k_gap_bwd(const float* dfeat, int rows, int S, int C, float* dh) {
  const long long total = (long long)rows * S * C;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(i % C);
    const long long r = i / ((long long)S * C);
    dh[i] = dfeat[r * C + c] / (float)S;
  }
}

int blocks_for(long long n) {
  long long b = (n + kT - 1) / kT;
  return (int)(b < 1 ? 1 : (b > 16384 ? 16384 : b));
}

}  // namespace

// ------------------------------------------------------------ launchers
// The stem shape the dedicated kernels take: 3 -> 16 channels, stride 1,
// 32 x 32, 16-byte aligned image rows (3072 floats) and output.
static bool stem_shape(const ConvGeom& q) {
  return q.Cin == kStemCin && q.Cout == kStemCout && q.stride == 1 && q.H == kStemSide &&
         q.W == kStemSide && q.Ho == kStemSide && q.Wo == kStemSide &&
         ((uintptr_t)q.x & 15) == 0 && ((uintptr_t)q.dy & 15) == 0 &&
         ((uintptr_t)q.out & 15) == 0 && (q.rowmap || q.sx % 4 == 0);
}

// Row-tiled kernel: reduction channels a multiple of 16, output channels
// 16 / 32 / 64, 16-byte aligned tensors.
static bool rows_shape(const ConvGeom& q, int mode) {
  const int Cr = mode == CONV_FWD ? q.Cin : q.Cout;
  const int Ng = mode == CONV_DGRAD ? q.Cin : q.Cout;
  // one replica's operand tensor is read through a buffer resource with
  // 32-bit byte offsets
  const long long opb = 4LL * q.Bt *
                        (mode == CONV_FWD ? (long long)q.H * q.W * q.Cin
                                          : (long long)q.Ho * q.Wo * q.Cout);
  // (an input gradient with up to 32 channels stages the whole weight in
  // LDS: at most 32 reduction channels)
  return Cr % 16 == 0 && (Ng == 16 || Ng == 32 || Ng == 64) &&
         (mode == CONV_FWD || Ng == 64 || Cr <= 32) &&
         (q.stride == 1 || (q.stride == 2 && mode == CONV_FWD)) && ((uintptr_t)q.Wk & 15) == 0 &&
         (q.sW % 4 == 0) &&
         (mode == CONV_FWD ? ((uintptr_t)q.x & 15) == 0 : ((uintptr_t)q.dy & 15) == 0) &&
         (mode == CONV_DGRAD || (!q.rowmap && q.sx % 4 == 0)) && opb < (1LL << 31);
}

// Input gradients of the stride-2 convolutions: 16 -> 32 channels on 32-wide
// images and 32 -> 64 on 16-wide ones.
static bool dgrad_s2_shape(const ConvGeom& q) {
  return q.stride == 2 && q.H == q.W && q.H == 2 * q.Ho && q.W == 2 * q.Wo &&
         ((q.Cin == 16 && q.Cout == 32 && q.W == 32) ||
          (q.Cin == 32 && q.Cout == 64 && q.W == 16)) &&
         ((uintptr_t)q.Wk & 15) == 0 && q.sW % 4 == 0 && ((uintptr_t)q.dy & 15) == 0;
}

// Halo-tile kernel: the first stage's 16 -> 16 stride-1 convolutions.
// bands of 8 rows per workgroup of k_conv_halo16: the forward (with its
// statistics epilogue) one, the input gradient several
constexpr int kHaloBandsFwd = 1, kHaloBandsDgrad = 4;
static bool halo_shape(const ConvGeom& q, int mode) {
  return q.Cin == 16 && q.Cout == 16 && q.stride == 1 && q.W == 32 && q.Wo == 32 &&
         q.H == q.Ho && q.H % (8 * (mode == CONV_FWD ? kHaloBandsFwd : kHaloBandsDgrad)) == 0 &&
         !q.rowmap && ((uintptr_t)q.Wk & 15) == 0 &&
         q.sW % 4 == 0 && ((uintptr_t)(mode == CONV_FWD ? q.x : q.dy) & 15) == 0 &&
         (mode == CONV_DGRAD || q.sx % 4 == 0);
}

int conv_dgrad_epilogues(const ConvGeom& q) {
  if (halo_shape(q, CONV_DGRAD)) return kEpiShortcut | kEpiBnSums | kEpiBnSumsAct;
  if (dgrad_s2_shape(q)) return kEpiShortcut;  // option A
  if (q.stride != 1 || !rows_shape(q, CONV_DGRAD) || q.Cin != q.Cout) return 0;
  // the row kernel: 32 channels (at 64 the operands' registers cost more
  // occupancy than the separate passes); the sums need whole 256-row chunks
  const bool chunks = ((long long)q.Bt * q.H * q.W) % 256 == 0;
  return q.Cin == 32 ? kEpiShortcut | (chunks ? kEpiBnSums | kEpiBnSumsAct : 0) : 0;
}

namespace {
// The kernel instances' epilogue sets: none, one of the three, or the
// shortcut with either sums
bool epi_instance(int e) {
  return e == 0 || e == kEpiShortcut || e == kEpiBnSums || e == kEpiBnSumsAct ||
         e == (kEpiShortcut | kEpiBnSums) || e == (kEpiShortcut | kEpiBnSumsAct);
}
}  // namespace

bool conv_fwd_stats(const ConvGeom& q) {
  if (stem_shape(q) || halo_shape(q, CONV_FWD)) return true;
  return rows_shape(q, CONV_FWD) && ((long long)q.Bt * q.Ho * q.Wo) % 256 == 0;
}

// Splits of a weight gradient over the batch: a power of two that divides
// the batch (the stem's kernel takes whole images per split). The band
// kernel of the 16- and 8-wide stages takes 32 and 16 splits (about two and
// one workgroups per compute unit at 16 replicas, each with whole bands);
// the others at most 64 with at least 1024 positions per split.
int conv_wgrad_splits(int Bt, int Ho, int Wo) {
  const int rows = Bt * Ho * Wo;
  const int cap = Wo == 16 ? 32 : Wo == 8 ? 16 : 64;
  int s = 1;
  while (s < cap && rows / (2 * s) >= (Wo <= 16 ? 64 : 1024) && Bt % (2 * s) == 0) s *= 2;
  return s;
}

// One k_conv_wgrad_band launch; instances above 64 KB of LDS opt in to more
// once per device (the per-device flags are atomics, the request idempotent).
template <int CI, int CO, int STRIDE, int WO>
hipError_t launch_wgrad_band(const ConvArgs& c, hipStream_t st) {
  constexpr size_t lds = wgrad_band_lds<CI, CO, STRIDE, WO>();
  static_assert(lds <= 160 * 1024, "fits one compute unit's LDS");
  if (lds > 64 * 1024) {
    static std::atomic<bool> done[64] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    if (!done[dev].load(std::memory_order_acquire)) {
      e = hipFuncSetAttribute((const void*)k_conv_wgrad_band<CI, CO, STRIDE, WO>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
      done[dev].store(true, std::memory_order_release);
    }
  }
  hipLaunchKernelGGL((k_conv_wgrad_band<CI, CO, STRIDE, WO>), dim3((unsigned)(c.G * c.splits)),
                     dim3(kT), lds, st, c);
  return hipGetLastError();
}

hipError_t launch_conv(int mode, const ConvGeom& q, hipStream_t st) {
  ConvArgs c{};
  c.G = q.G;
  c.Bt = q.Bt;
  c.H = q.H;
  c.W = q.W;
  c.Cin = q.Cin;
  c.Ho = q.Ho;
  c.Wo = q.Wo;
  c.Cout = q.Cout;
  c.stride = q.stride;
  c.x = q.x;
  c.sx = q.sx;
  c.rowmap = q.rowmap;
  c.dy = q.dy;
  c.Wk = q.Wk;
  c.sW = q.sW;
  c.out = q.out;
  c.stats = mode == CONV_FWD ? q.stats : nullptr;
  c.bn_mu = mode == CONV_DGRAD && !q.bs_part ? nullptr : q.bn_mu;
  c.bn_inv = q.bn_inv;
  c.bn_g = q.bn_g;
  c.bn_b = q.bn_b;
  c.bn_sP = q.bn_sP;
  c.sc_dh = mode == CONV_DGRAD ? q.sc_dh : nullptr;
  c.sc_hb = q.sc_hb;
  c.bs_y = q.bs_y;
  c.bs_hb = q.bs_hb;
  c.bs_part = mode == CONV_DGRAD ? q.bs_part : nullptr;
  const int epi = (c.sc_dh ? kEpiShortcut : 0) |
                  (c.bs_part ? (c.bs_hb ? kEpiBnSumsAct : kEpiBnSums) : 0);
  if (epi && (!epi_instance(epi) || (conv_dgrad_epilogues(q) & epi) != epi ||
              (c.sc_dh && (!c.sc_hb || ((uintptr_t)c.sc_hb & 3))) ||
              (c.bs_hb && ((uintptr_t)c.bs_hb & 3)) ||
              (c.bs_part && (!c.bs_y || !c.bn_mu || !c.bn_inv ||
                             (!c.bs_hb && (!c.bn_g || !c.bn_b))))))
    return hipErrorInvalidValue;
  if (c.bn_mu && (q.Cin % 4 || q.bn_sP % 4 || ((uintptr_t)q.bn_mu | (uintptr_t)q.bn_inv |
                                              (uintptr_t)q.bn_g | (uintptr_t)q.bn_b) & 15))
    return hipErrorInvalidValue;
  const int Mg = mode == CONV_FWD ? q.Bt * q.Ho * q.Wo
               : mode == CONV_DGRAD ? q.Bt * q.H * q.W : 9 * q.Cin;
  const int Ng = mode == CONV_DGRAD ? q.Cin : q.Cout;
  if (mode == CONV_WGRAD) {
    c.splits = conv_wgrad_splits(q.Bt, q.Ho, q.Wo);
    const int rows = q.Bt * q.Ho * q.Wo;
    const bool halo = q.Cin == 16 && q.Cout == 16 && q.stride == 1 && q.W == 32 &&
                      q.Wo == 32 && q.H == q.Ho && q.H % 8 == 0 && !q.rowmap &&
                      ((uintptr_t)q.x & 15) == 0 && ((uintptr_t)q.dy & 15) == 0 &&
                      q.sx % 4 == 0;
    if (halo) {
      hipLaunchKernelGGL(k_conv_wgrad_halo16, dim3((unsigned)(q.G * c.splits)), dim3(kT), 0,
                         st, c);
      return hipGetLastError();
    }
    if (stem_shape(q)) {
      c.mchunk = rows / c.splits;  // whole images per split
      hipLaunchKernelGGL(k_conv_wgrad_stem, dim3((unsigned)(q.G * c.splits)), dim3(kT), 0,
                         st, c);
      return hipGetLastError();
    }
    // band tiles: 64 output positions (whole 16- or 8-wide rows) per band
    const bool bandk = !q.rowmap && (q.Wo == 16 || q.Wo == 8) && q.Ho % (64 / q.Wo) == 0 &&
                       ((q.stride == 1 && q.H == q.Ho && q.W == q.Wo) ||
                        (q.stride == 2 && q.H == 2 * q.Ho && q.W == 2 * q.Wo)) &&
                       ((uintptr_t)q.x & 15) == 0 && ((uintptr_t)q.dy & 15) == 0 &&
                       q.sx % 4 == 0;
    if (bandk) {
      if (q.Cin == 32 && q.Cout == 32 && q.stride == 1 && q.Wo == 16)
        return launch_wgrad_band<32, 32, 1, 16>(c, st);
      if (q.Cin == 16 && q.Cout == 32 && q.stride == 2 && q.Wo == 16)
        return launch_wgrad_band<16, 32, 2, 16>(c, st);
      if (q.Cin == 64 && q.Cout == 64 && q.stride == 1 && q.Wo == 8)
        return launch_wgrad_band<64, 64, 1, 8>(c, st);
      if (q.Cin == 32 && q.Cout == 64 && q.stride == 2 && q.Wo == 8)
        return launch_wgrad_band<32, 64, 2, 8>(c, st);
    }
    return hipErrorInvalidValue;  // no weight-gradient kernel for this shape
  } else {
    const bool rows = rows_shape(q, mode), halo = halo_shape(q, mode);
    if (mode == CONV_FWD && stem_shape(q)) {
      const long long nb = (long long)q.G * q.Bt;
      if (nb > 0x7fffffffLL) return hipErrorInvalidValue;
      hipLaunchKernelGGL(k_conv_stem_fwd, dim3((unsigned)nb), dim3(kT), 0, st, c);
      return hipGetLastError();
    }
    if (mode == CONV_DGRAD && q.stride == 2) {
      if (!dgrad_s2_shape(q)) return hipErrorInvalidValue;  // no kernel for this shape
      // images per workgroup: up to 4 (the weights are loaded once for all
      // of them) while at least 512 workgroups remain
      c.mchunk = 1;
      while (c.mchunk < 4 && q.Bt % (2 * c.mchunk) == 0 &&
             (long long)q.G * (q.Bt / (2 * c.mchunk)) >= 512)
        c.mchunk *= 2;
      const long long nb = (long long)q.G * (q.Bt / c.mchunk);
      if (nb > 0x7fffffffLL) return hipErrorInvalidValue;
      if (q.Cin == 16 && c.sc_dh)
        hipLaunchKernelGGL((k_conv_dgrad_s2<16, 32, 32, true>), dim3((unsigned)nb), dim3(kT), 0,
                           st, c);
      else if (q.Cin == 16)
        hipLaunchKernelGGL((k_conv_dgrad_s2<16, 32, 32, false>), dim3((unsigned)nb), dim3(kT),
                           0, st, c);
      else if (c.sc_dh)
        hipLaunchKernelGGL((k_conv_dgrad_s2<32, 64, 16, true>), dim3((unsigned)nb), dim3(kT), 0,
                           st, c);
      else
        hipLaunchKernelGGL((k_conv_dgrad_s2<32, 64, 16, false>), dim3((unsigned)nb), dim3(kT),
                           0, st, c);
      return hipGetLastError();
    }
    if (halo) {
      const long long nb = (long long)q.G * q.Bt *
                           (q.H / 8 / (mode == CONV_FWD ? kHaloBandsFwd : kHaloBandsDgrad));
      if (nb > 0x7fffffffLL) return hipErrorInvalidValue;
      if (mode == CONV_FWD)
        hipLaunchKernelGGL((k_conv_halo16<CONV_FWD, kHaloBandsFwd>), dim3((unsigned)nb),
                           dim3(kT), 0, st, c);
      else if (epi == kEpiShortcut)
        hipLaunchKernelGGL((k_conv_halo16<CONV_DGRAD, kHaloBandsDgrad, kEpiShortcut>),
                           dim3((unsigned)nb), dim3(kT), 0, st, c);
      else if (epi == kEpiBnSums)
        hipLaunchKernelGGL((k_conv_halo16<CONV_DGRAD, kHaloBandsDgrad, kEpiBnSums>),
                           dim3((unsigned)nb), dim3(kT), 0, st, c);
      else if (epi == (kEpiShortcut | kEpiBnSums))
        hipLaunchKernelGGL((k_conv_halo16<CONV_DGRAD, kHaloBandsDgrad, kEpiShortcut | kEpiBnSums>),
                           dim3((unsigned)nb), dim3(kT), 0, st, c);
      else if (epi == (kEpiShortcut | kEpiBnSumsAct))
        hipLaunchKernelGGL(
            (k_conv_halo16<CONV_DGRAD, kHaloBandsDgrad, kEpiShortcut | kEpiBnSumsAct>),
            dim3((unsigned)nb), dim3(kT), 0, st, c);
      else if (epi == kEpiBnSumsAct)
        hipLaunchKernelGGL((k_conv_halo16<CONV_DGRAD, kHaloBandsDgrad, kEpiBnSumsAct>),
                           dim3((unsigned)nb), dim3(kT), 0, st, c);
      else
        hipLaunchKernelGGL((k_conv_halo16<CONV_DGRAD, kHaloBandsDgrad>), dim3((unsigned)nb),
                           dim3(kT), 0, st, c);
    } else if (rows) {
      const long long rt = (long long)((Mg + 255) / 256) * q.G;
      if (rt > 0x7fffffffLL) return hipErrorInvalidValue;
#define LSGD_ROWS(MD, NB)                                                              \
  hipLaunchKernelGGL((k_conv_rows<MD, NB>), dim3((unsigned)rt), dim3(kT), 0, st, c)
      if (mode == CONV_FWD) {
        if (Ng == 16) LSGD_ROWS(CONV_FWD, 16);
        else if (Ng == 32) LSGD_ROWS(CONV_FWD, 32);
        else LSGD_ROWS(CONV_FWD, 64);
      } else {
#define LSGD_ROWS_E(NB, E)                                                                  \
  hipLaunchKernelGGL((k_conv_rows<CONV_DGRAD, NB, E>), dim3((unsigned)rt), dim3(kT), 0, st, c)
        if (Ng == 16) LSGD_ROWS(CONV_DGRAD, 16);
        else if (Ng == 32 && epi == kEpiShortcut) LSGD_ROWS_E(32, kEpiShortcut);
        else if (Ng == 32 && epi == kEpiBnSums) LSGD_ROWS_E(32, kEpiBnSums);
        else if (Ng == 32 && epi == kEpiBnSumsAct) LSGD_ROWS_E(32, kEpiBnSumsAct);
        else if (Ng == 32 && epi == (kEpiShortcut | kEpiBnSums))
          LSGD_ROWS_E(32, kEpiShortcut | kEpiBnSums);
        else if (Ng == 32 && epi == (kEpiShortcut | kEpiBnSumsAct))
          LSGD_ROWS_E(32, kEpiShortcut | kEpiBnSumsAct);
        else if (Ng == 32) LSGD_ROWS(CONV_DGRAD, 32);
        else LSGD_ROWS(CONV_DGRAD, 64);
#undef LSGD_ROWS_E
      }
#undef LSGD_ROWS
    } else {
      return hipErrorInvalidValue;  // no kernel for this shape
    }
  }
  return hipGetLastError();
}

hipError_t launch_conv_wupdate(const float* part, int splits, int G, int n, float* W,
                               float* U, long long sP, float lr, float mom, float wd,
                               int nesterov, hipStream_t st) {
  const int b = blocks_for((long long)G * n);
#define LSGD_WU(S)                                                                   \
  case S:                                                                            \
    hipLaunchKernelGGL(k_conv_wupdate<S>, dim3(b), dim3(kT), 0, st, part, G, n, W, U, \
                       sP, lr, mom, wd, nesterov);                                   \
    break;
  switch (splits) {
    LSGD_WU(1)
    LSGD_WU(2)
    LSGD_WU(4)
    LSGD_WU(8)
    LSGD_WU(16)
    LSGD_WU(32)
    LSGD_WU(64)
    default: return hipErrorInvalidValue;
  }
#undef LSGD_WU
  return hipGetLastError();
}

// Channel counts the float4 BN forms take: powers of two from 16, aligned.
int bn_vec_shift(int C) {
  if (C < 16 || (C & (C - 1))) return -1;
  int s = 0;
  while ((1 << s) < C) ++s;
  return s;
}
bool al16p(const void* p) { return p == nullptr || ((uintptr_t)p & 15u) == 0; }

int bn_chunks(int R) { return (R + bn_chunk_rows(R) - 1) / bn_chunk_rows(R); }

// The BN kernels take 4 channels per thread: C a power of two >= 16 (and
// <= 256), 16-byte aligned tensors, fewer than 2^31 values per replica and
// at most 65535 replicas (the ResNet-20 plan meets all of these; anything
// else is refused rather than run by a slower form).
static bool bn_shape_ok(int G, int R, int C) {
  return bn_vec_shift(C) >= 0 && C <= kT && (long long)R * C < (1LL << 31) && G <= 65535;
}

hipError_t launch_bn_stats(const float* y, int G, int R, int C, double* part,
                           float* mu, float* inv, float* rm, float* rv, long long sRS,
                           hipStream_t st, const float* gamma, const float* beta,
                           long long sP, float* gsnap, float* bsnap) {
  if (!bn_shape_ok(G, R, C) || !al16p(y) || (gsnap && (!gamma || !beta || !bsnap)))
    return hipErrorInvalidValue;
  const int nch = bn_chunks(R);
  hipLaunchKernelGGL(k_bn_partial4, dim3(nch, G), dim3(kT), 0, st, y, R, C, nullptr,
                     nullptr, nullptr, nullptr, nullptr, nullptr, 0LL, part, nch);
  hipLaunchKernelGGL(k_bn_finalize_wg, dim3(G), dim3(kT), 0, st, part, nch, C, R, mu,
                     inv, nullptr, (float*)gamma, (float*)beta, nullptr, nullptr, sP, 0.f,
                     0.f, 0, 1e-5f, rm, rv, sRS, gsnap, bsnap);
  return hipGetLastError();
}

hipError_t launch_bn_finalize_chunks(const double* part, int nchunk, int G, int R, int C,
                                     float* mu, float* inv, float* rm, float* rv,
                                     long long sRS, hipStream_t st, const float* gamma,
                                     const float* beta, long long sP, float* gsnap,
                                     float* bsnap) {
  if (!bn_shape_ok(G, R, C) || (gsnap && (!gamma || !beta || !bsnap)))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_bn_finalize_wg, dim3(G), dim3(kT), 0, st, part, nchunk, C, R, mu,
                     inv, nullptr, (float*)gamma, (float*)beta, nullptr, nullptr, sP, 0.f,
                     0.f, 0, 1e-5f, rm, rv, sRS, gsnap, bsnap);
  return hipGetLastError();
}

hipError_t launch_bn_apply(const float* y, int G, int R, int C, const float* mu,
                           const float* inv, const float* gamma, const float* beta,
                           long long sP, int mode, const float* xin, int Ho, int Wo,
                           int Cin, float* out, unsigned* mbits, hipStream_t st) {
  if (!bn_shape_ok(G, R, C) || !al16p(y) || !al16p(out) || !al16p(xin) || !al16p(mu) ||
      !al16p(inv) || !al16p(gamma) || !al16p(beta) || sP % 4 || Cin % 4 ||
      (mbits && ((R * C) % 32 || !al16p(mbits))))
    return hipErrorInvalidValue;
  const dim3 grid((R * C / 4 + kT - 1) / kT, G);
  hipLaunchKernelGGL(k_bn_apply4, grid, dim3(kT), 0, st, y, R, C, bn_vec_shift(C), mu, inv,
                     gamma, beta, sP, mode, xin, Ho, Wo, Cin, out, mbits);
  return hipGetLastError();
}

hipError_t launch_bn_backward(const float* y, const float* gup, const unsigned* mbits,
                              int G, int R, int C, double* part, const float* mu,
                              const float* inv, float* coef, float* gamma, float* beta,
                              float* ug, float* ub, long long sP, float lr, float mom,
                              int nesterov, float* dy, int fused_nchunk, hipStream_t st) {
  if (!bn_shape_ok(G, R, C) || !al16p(y) || !al16p(gup) || !al16p(mbits) || !al16p(dy) ||
      !al16p(mu) || !al16p(inv) || !al16p(coef) || fused_nchunk < 0 ||
      (mbits && (R * C) % 32))
    return hipErrorInvalidValue;
  const int nch = fused_nchunk > 0 ? fused_nchunk : bn_chunks(R);
  if (fused_nchunk == 0)
    hipLaunchKernelGGL(k_bn_partial4, dim3(nch, G), dim3(kT), 0, st, y, R, C, gup, mbits,
                       mu, inv, gamma, beta, sP, part, nch);
  hipLaunchKernelGGL(k_bn_finalize_wg, dim3(G), dim3(kT), 0, st, part, nch, C, R,
                     (float*)mu, (float*)inv, coef, gamma, beta, ug, ub, sP, lr, mom,
                     nesterov, 1e-5f, nullptr, nullptr, 0LL, nullptr, nullptr);
  hipLaunchKernelGGL(k_bn_bwd_apply4, dim3((R * C / 4 + kT - 1) / kT, G), dim3(kT), 0,
                     st, y, gup, mbits, R, C, mu, inv, coef, dy);
  return hipGetLastError();
}

hipError_t launch_shortcut_grad(float* dx, const float* dh_out, const unsigned* hb_out,
                                int G, int Bt, int H, int W, int Cin, int Cout,
                                int mode, hipStream_t st) {
  if (Cin % 4 || Cout % 4 || !al16p(dx) || !al16p(dh_out) || !hb_out || !al16p(hb_out) ||
      (long long)Bt * H * W * Cin >= (1LL << 31) || G > 65535 || H % 2 || W % 2 ||
      (mode == 1 ? (long long)Bt * H * W * Cin : (long long)Bt * (H / 2) * (W / 2) * Cout) %
          32)
    return hipErrorInvalidValue;
  const long long n4 = mode == 1 ? (long long)Bt * H * W * Cin / 4
                                 : (long long)Bt * (H / 2) * (W / 2) * (Cin / 4);
  hipLaunchKernelGGL(k_shortcut_grad4, dim3((unsigned)((n4 + kT - 1) / kT), G), dim3(kT),
                     0, st, dx, dh_out, hb_out, Bt, H, W, Cin, Cout, mode);
  return hipGetLastError();
}

hipError_t launch_gap(const float* h, int rows, int S, int C, float* feat, bool bwd,
                      const float* dfeat, float* dh, hipStream_t st) {
  if (!bwd)
    hipLaunchKernelGGL(k_gap, dim3((rows * C + 255) / 256), dim3(256), 0, st, h, rows, S,
                       C, feat);
  else
    hipLaunchKernelGGL(k_gap_bwd, dim3(blocks_for((long long)rows * S * C)), dim3(kT), 0,
                       st, dfeat, rows, S, C, dh);
  return hipGetLastError();
}

}  // namespace lsgd
