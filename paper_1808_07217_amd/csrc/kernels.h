// Internal declarations shared by the HIP translation units of liblsgd.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsgd {

// Local-step mode, carried in the `nesterov` field of the update arguments:
// bit 0 Nesterov (d = g + m u) instead of heavy ball (d = u); bit 1 moves
// by sign(d) (the signSGD local step), sign(0) = 0.
constexpr int kModeNesterov = 1, kModeSign = 2;

__device__ __forceinline__ float step_dir(float u, float g, float mom, int mode) {
  float d = (mode & kModeNesterov) ? __builtin_fmaf(mom, u, g) : u;
  if (mode & kModeSign) d = d > 0.f ? 1.f : (d < 0.f ? -1.f : 0.f);
  return d;
}


typedef uint16_t bf16_t;  // bfloat16 bit pattern

// fp32 -> bf16, round to nearest even (finite inputs; overflow gives inf).
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  uint32_t b = __float_as_uint(x);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (bf16_t)(b >> 16);
}
__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// ---------------------------------------------------------------- GEMM
enum Epilogue : int {
  EPI_STORE = 0,       // C = acc (fp32)
  EPI_BIAS = 1,        // C = acc + bias[n] (fp32 logits)
  EPI_BIAS_RELU = 2,   // C = relu(acc + bias[n]) (activation dtype)
  EPI_RELU_MASK = 3,   // C = acc * (mask[m][n] > 0) (activation dtype)
  EPI_SGD = 4          // fused parameter update of W[m][n] with acc as grad
};

struct GemmArgs {
  int G, M, N, Kd;
  // operand A: element (m, k) at A + g*sA + row(r)*lda + c, where the
  // storage (r, c) is (m, k) for trans_a == 0 and (k, m) otherwise; row(r)
  // is rowmap[g*sRow + r] when rowmap != nullptr, else r.
  const void* A;
  long long lda, sA;
  const int32_t* rowmap;
  long long sRow;
  // operand B: element (k, n); storage (k, n) for trans_b == 0, (n, k) else.
  const void* B;
  long long ldb, sB;
  // output / epilogue operands (leading dimension ldc, group stride sC)
  void* C;
  long long ldc, sC;
  const float* bias;
  long long sBias;
  const void* mask;  // same layout as C (activation dtype)
  // fused update (EPI_SGD): W, U fp32 and Wb bf16 copy share ldc / sC
  float* W;
  float* U;
  bf16_t* Wb;
  // when set, the update reads the weights (and the bias) it steps from here
  // instead of W (bias_w): the synchronised model of a pending lazy average,
  // same layout, replica stride sWsrc (sBiasSrc); it still writes W, U, Wb
  const float* Wsrc;
  long long sWsrc;
  const float* bias_src;
  long long sBiasSrc;
  float lr, mom, wd;
  int nesterov;
  // EPI_SGD: when bias_w != nullptr the kernel also forms the bias gradient
  // sum_k B[k][n] and updates bias_w / bias_u (group stride sBiasP)
  float* bias_w;
  float* bias_u;
  long long sBiasP;
  // split-K: `splits` partial sums of K range kchunk each, written to `part`
  // ([splits][G][M][N] fp32) and reduced by a second kernel
  int splits;
  int kchunk;  // set by launch_gemm
  float* part;
};

// Split count launch_gemm would like for a problem (1 = no split-K).
int gemm_splits(int dtype, int M, int N, int Kd, int G, int epi);

hipError_t launch_gemm(int dtype, int trans_a, int trans_b, int epi,
                       int out_bf16, const GemmArgs& a, hipStream_t s);

// Fused weight gradient + update (trans_a = 1, trans_b = 0, EPI_SGD) of up to
// kWsMaxProblems layers in one persistent launch, their tiles concatenated.
// gemm_sgd_multi_tiles: the list's total 128 x 128 tile count, or -1 when a
// problem does not fit the kernel (fp32, M and N multiples of 128, aligned
// rows, at most 512 gathered rows).
constexpr int kWsMaxProblems = 8;
int gemm_sgd_multi_tiles(int dtype, const GemmArgs* list, int n);
hipError_t launch_gemm_sgd_multi(int dtype, const GemmArgs* list, int n,
                                 hipStream_t s);

// ---------------------------------------------------------------- head
// Output layer with few classes, fused around the loss (head.hip).
constexpr int kHeadMaxClasses = 32;
struct HeadArgs {
  int K, B, D, C;            // replicas, batch, inputs, classes
  const void* A;             // layer input: activations [K][B][D] (group
  long long sA;              //   stride sA) or, if gather, dataset rows
  int gather;                //   selected by rowmap
  const int32_t* rowmap;     // sampled indices [K][B]
  const int32_t* y;          // labels [N]
  const void* W;             // W_L [D][C] operand (fp32 master or bf16 copy)
  long long sW;              //   group stride
  float* Wm;                 // W_L master, momentum, bf16 copy (update)
  float* Um;
  bf16_t* Wb;
  const float* bias;         // b_L (read by the forward pass)
  float* bias_w;             // b_L and its momentum (update)
  float* bias_u;
  long long sP;              // replica stride of the parameter buffers
  void* dZ;                  // [K][B][C] out (activation dtype)
  void* dZprev;              // [K][B][D] masked input gradient, or nullptr
  float* rowloss;            // [K][B]
  float* loss;               // [K] or nullptr
  // the forward reads b_L at bias + k sBias; the update reads the W_L and b_L
  // it steps at Wsrc / bsrc + k sSrc (the replica's own, or the shared model
  // of a pending lazy average) and writes Wm / bias_w
  long long sBias;
  const float* Wsrc;
  const float* bsrc;
  long long sSrc;
  int* nonfinite;            // set to 1 when a replica's mean loss is not
                             //   finite (never cleared here), or nullptr
  float lr, mom, wd;
  int nesterov;
  int nomask;                // dZprev without the ReLU mask (pooled inputs)
};
hipError_t launch_head_fwd(int dtype, const HeadArgs& h, hipStream_t s);
hipError_t launch_head_wgrad(int dtype, const HeadArgs& h, hipStream_t s);

// ---------------------------------------------------------------- ResNet
// 3x3 convolution geometry of one launch (resnet.hip). x: input activations
// [G][Bt][H][W][Cin] with group stride sx, or with a row map the dataset
// rows (images) selected per replica; dy: output gradient
// [G][Bt][Ho][Wo][Cout]; Wk: [9*Cin][Cout] (forward, weight gradient) or the
// swapped copy [9*Cout][Cin] (input gradient), group stride sW; out: forward
// y, input gradient dx, or the weight gradient's split partials.
struct ConvGeom {
  int G, Bt, H, W, Cin, Ho, Wo, Cout, stride;
  const float* x;
  long long sx;
  const int32_t* rowmap;
  const float* dy;
  const float* Wk;
  long long sW;
  float* out;
  double* stats;  // forward: BN statistics per 256-row chunk (see conv_fwd_stats)
  // forward / weight gradient of a block's second convolution: x is the
  // first convolution's pre-BN output and the input is relu(BN(x)) with the
  // replica's statistics (mu, inv at g * Cin + c) and parameters (gamma,
  // beta at g * bn_sP + c), formed as the tiles are loaded; nullptr: x as is
  const float* bn_mu;
  const float* bn_inv;
  const float* bn_g;
  const float* bn_b;
  long long bn_sP;
  // input gradient, where conv_dgrad_epilogues(q) (nullptr: none):
  //  * sc_dh, sc_hb: the block output's gradient and its activation's ReLU
  //    mask as bits (bit L % 32 of word L / 32 for linear element L, as
  //    launch_bn_apply writes it): dx gains sc_dh where the bit is set --
  //    element for element (identity shortcut, same shape as dx), or, for a
  //    stride-2 input gradient (option A, output [G][Bt][Ho][Wo][Cout]), at
  //    input position (2 oh, 2 ow) from output (oh, ow), first Cin channels;
  //  * bs_part: dx (with the shortcut's share, when both are set) is the
  //    gradient of a BN-ReLU's output whose pre-BN values are bs_y (same
  //    shape) and whose statistics and parameters come in bn_* (as above):
  //    the BN backward sums (sum dz, sum dz x^ with x^ = (y - mu) inv) are
  //    written per 256-row chunk, [G][R/256][Cin][2] doubles, for
  //    launch_bn_backward's fused_nchunk; dz = dx where
  //    gamma (y - mu) inv + beta > 0, or, with bs_hb set (a BN whose ReLU
  //    follows a shortcut add), where its activation's mask bit is set (bn_g, bn_b
  //    then unused)
  const float* sc_dh;
  const unsigned* sc_hb;
  const float* bs_y;
  const unsigned* bs_hb;
  double* bs_part;
};
enum { CONV_FWD_MODE = 0, CONV_DGRAD_MODE = 1, CONV_WGRAD_MODE = 2 };
// Which epilogues the input-gradient launch of q takes: bit 0 the shortcut
// share (sc_*; option A for the stride-2 ones), bit 1 the BN backward sums
// with the recomputed mask (bs_*),
// bit 2 the sums with the activation mask (bs_hb). A launch takes one of them,
// or the shortcut with one kind of sums.
int conv_dgrad_epilogues(const ConvGeom& q);
int conv_wgrad_splits(int Bt, int Ho, int Wo);
// Whether the forward convolution of q writes its output's BN statistics
// (per 256-row chunk, [G][R/256][Cout][2] doubles: sum, sum of squares) when
// q.stats is set; the caller then finalises with launch_bn_finalize_chunks.
bool conv_fwd_stats(const ConvGeom& q);
// Both finalisers also update the running statistics when rm is set: the
// running means rm[g * sRS + c] and variances rv[g * sRS + c] of replica g
// (factor 0.1 on the batch mean and the unbiased batch variance); and, when
// gsnap is set, copy the BN scale and shift the batch is normalised with
// (gamma, beta at g * sP + c) to gsnap, bsnap [G][C], so that readers of the
// forward's BN-ReLU see them after the backward pass has stepped gamma, beta.
hipError_t launch_bn_finalize_chunks(const double* part, int nchunk, int G, int R, int C,
                                     float* mu, float* inv, float* rm, float* rv,
                                     long long sRS, hipStream_t st,
                                     const float* gamma = nullptr,
                                     const float* beta = nullptr, long long sP = 0,
                                     float* gsnap = nullptr, float* bsnap = nullptr);
int bn_chunks(int R);
hipError_t launch_conv(int mode, const ConvGeom& q, hipStream_t st);
hipError_t launch_conv_wupdate(const float* part, int splits, int G, int n, float* W,
                               float* U, long long sP, float lr, float mom, float wd,
                               int nesterov, hipStream_t st);
hipError_t launch_bn_stats(const float* y, int G, int R, int C, double* part,
                           float* mu, float* inv, float* rm, float* rv, long long sRS,
                           hipStream_t st, const float* gamma = nullptr,
                           const float* beta = nullptr, long long sP = 0,
                           float* gsnap = nullptr, float* bsnap = nullptr);
// BN output with the shortcut add (mode 1 identity, 2 option A from xin) and
// ReLU into out; with mbits set, also the ReLU mask as bits (bit L % 32 of
// word L / 32 set where out at linear element L is positive; R C a multiple
// of 32), which the backward passes read instead of out.
hipError_t launch_bn_apply(const float* y, int G, int R, int C, const float* mu,
                           const float* inv, const float* gamma, const float* beta,
                           long long sP, int mode, const float* xin, int Ho, int Wo,
                           int Cin, float* out, unsigned* mbits, hipStream_t st);
// BN backward with the gamma/beta step: the upstream gradient gup is masked
// by the activation's mask bits mbits (launch_bn_apply's) or, with mbits null,
// by the sign of the recomputed pre-ReLU BN output (a BN-ReLU with no shortcut
// add). coef holds 5 floats per (replica, channel).
// fused_nchunk > 0: the sums are already in part (fused_nchunk chunks per
// replica, from an input-gradient epilogue) and are not formed again.
// dy may be gup (the input gradient in place over it).
hipError_t launch_bn_backward(const float* y, const float* gup, const unsigned* mbits,
                              int G, int R, int C, double* part, const float* mu,
                              const float* inv, float* coef, float* gamma, float* beta,
                              float* ug, float* ub, long long sP, float lr, float mom,
                              int nesterov, float* dy, int fused_nchunk, hipStream_t st);
// The shortcut's share dx += dh_out where the block output's mask bit
// (hb_out, launch_bn_apply's) is set: identity (mode 1) or option A (mode 2).
hipError_t launch_shortcut_grad(float* dx, const float* dh_out, const unsigned* hb_out,
                                int G, int Bt, int H, int W, int Cin, int Cout,
                                int mode, hipStream_t st);
hipError_t launch_gap(const float* h, int rows, int S, int C, float* feat, bool bwd,
                      const float* dfeat, float* dh, hipStream_t st);

// ---------------------------------------------------------------- others
// The per-epoch reshuffled partition sampler (epoch = step / S, batch
// step % S with S = floor(floor(N / K) / B) >= 1, else hipErrorInvalidValue).
hipError_t launch_sample_epoch(uint64_t seed, int64_t step, int K, int64_t N,
                               int B, int32_t* idx, hipStream_t s);
hipError_t launch_sample(uint64_t seed, int64_t step, int K, int64_t N,
                         int B, int32_t* idx, hipStream_t s);
hipError_t launch_xent(const float* Z, const int32_t* y, const int32_t* idx,
                       int K, int B, int C, void* dZ, int dz_bf16,
                       float* loss, int* nonfinite, hipStream_t s);
hipError_t launch_sgd_update(float* W, float* U, const float* G, long long n,
                             float lr, float mom, float wd, int nesterov,
                             hipStream_t s);
// K-way average of the first n elements of K rows spaced ld apart: every
// row (and its bf16 copy in Wb) := the mean; with mean_out, only the mean is
// written, to mean_out [n] (and its bf16 copy to Wb [n] when given).
hipError_t launch_average(float* W, bf16_t* Wb, int K, long long n,
                          long long ld, float* mean_out, hipStream_t s);
// The K-way average with global momentum: mean of the K rows, then
// ug = mg ug + (ws - mean) / lr, ws -= lr ug, and every row := ws (ws, ug:
// [n] fp32, updated in place).
hipError_t launch_average_gm(float* W, bf16_t* Wb, int K, long long n,
                             long long ld, float* ws, float* ug, float mg,
                             float lr, hipStream_t s);
// Single-launch round for softmax regression (tiny.hip): every replica and
// its buffer live in LDS for the H steps and the average.
constexpr int kTinyMaxC = 32, kTinyMaxH = 64;
constexpr size_t kTinyMaxLds = 160 * 1024;
struct TinyArgs {
  const float* X;      // [N][D]
  const int32_t* y;    // [N]
  float* W;            // [K][Ps] replicas (read, then the averaged model)
  float* U;            // [K][Ps] momentum buffers
  float* loss;         // [H][K] or nullptr
  int* nonfinite;      // set to 1 on a non-finite mean loss, or nullptr
  long long N, Ps, step0;
  long long S;         // batches per epoch of the reshuffle sampler; 0: i.i.d.
  int K, B, D, C, H, m;
  uint32_t key0, key1;
  float mom, wd;
  int mode;            // kModeNesterov | kModeSign
  float lr[kTinyMaxH];
};
size_t tiny_round_lds_bytes(int K, int B, int D, int C);
bool tiny_round_fits(int K, int B, int D, int C, int H);
// true when the round takes the 256-thread-per-replica kernel
bool tiny_round_wide(int K, int B, int D, int C, int H);
hipError_t launch_tiny_round(const TinyArgs& a, hipStream_t s);
// Sign-compressed synchronisation (compress.hip): W fp32 [K][Ps] replicas
// (the first P elements of each row are the model), ws fp32 [Ps] the model
// of the previous synchronisation (updated), E fp32 [K][Ps] error memories
// or nullptr (Algorithm 4 / 3), Wb the bf16 copy or nullptr. Ps % 4 == 0,
// 16-byte aligned buffers; scratch of sign_sync_scratch_bytes(K, Ps).
size_t sign_sync_scratch_bytes(int K, long long Ps);
hipError_t launch_sign_sync(float* W, bf16_t* Wb, float* E, float* ws, int K,
                            long long P, long long Ps, void* scratch,
                            size_t scratch_bytes, hipStream_t s);
// The same on plain [K][P] arrays with the scratch in a static device array
// of kSignSyncStaticBytes (no allocation; hipErrorInvalidValue when the
// problem needs more).
constexpr size_t kSignSyncStaticBytes = 16u << 20;
hipError_t launch_sign_sync_static(float* W, float* E, float* ws, int K, long long P,
                                   hipStream_t s);
// The same average within each of `blocks` groups of Kb consecutive rows
// (mean_out only with blocks == 1).
hipError_t launch_average_blocks(float* W, bf16_t* Wb, int Kb, int blocks,
                                 long long n, long long ld, float* mean_out,
                                 hipStream_t s);
hipError_t launch_broadcast(const float* src, float* W, bf16_t* Wb, int K,
                            long long n, long long ld, int replica,
                            hipStream_t s);
hipError_t launch_to_bf16(const float* x, bf16_t* y, long long n,
                          hipStream_t s);
hipError_t launch_fill(float* x, float v, long long n, hipStream_t s);
// rows x n floats between row-pitched buffers (pitches in floats)
hipError_t launch_copy_rows(float* dst, long long dpitch, const float* src,
                            long long spitch, long long n, int rows,
                            hipStream_t s);
// eight 64-bit words, passed by value, stored at dst (8-byte aligned)
struct Words8 { unsigned long long w[8]; };
hipError_t launch_put_words(void* dst, const Words8& v, hipStream_t s);

}  // namespace lsgd
