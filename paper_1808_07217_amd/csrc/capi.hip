// C ABI and host runtime of liblsgd: workspace layout, the launch sequence
// of one local step, the round driver and error latching.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/lsgd.h"
#include "kernels.h"

using lsgd::bf16_t;
using lsgd::GemmArgs;

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kReplicaPad = 64;  // replica stride in elements: 256 B

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ResNet-20 plan: the 19 convolutions (stem; 3 stages x 3 blocks x 2) with
// their geometry, parameter offsets and activation buffers.
struct ConvSpec {
  int Cin, Cout, stride, H, W, Ho, Wo;
  int64_t offW, offG, offB;  // weight [9*Cin][Cout], BN scale, BN shift
  size_t y, act;             // pre-BN output, post-BN activation (ReLU'd)
  size_t mbits;              // block outputs: the activation's ReLU mask as bits
};
constexpr int kResConvs = 19;
struct ResPlan {
  ConvSpec cv[kResConvs];
  int64_t offFcW = 0, offFcB = 0;
  int classes = 0, feat = 64, side_out = 8;
  // gradient buffers: gio the block-output and block-input gradients (the
  // two swap roles block by block), bgrad[b] block b's two BN input gradients
  size_t featb = 0, dfeat = 0, dzh = 0, gio[2] = {}, bgrad[9][2] = {}, mu = 0, inv = 0,
         coef = 0,
         bnpart = 0, bnpart2 = 0, wpart = 0, wpart0 = 0;
  // per BN layer, the scale and shift its forward batch was normalised with
  // ([kResConvs][K][64], layer i's [K][Cout] from i K 64)
  size_t gsnap = 0, bsnap = 0;
  // BN running statistics [K][Rs] fp32: per replica the running means of
  // every BN layer in convolution order (layer i from rsoff[i]), then the
  // running variances in the same order (from rs_half); R = 2 rs_half
  size_t rs = 0;
  int rsoff[kResConvs] = {};
  int rs_half = 0;
  int64_t Rs = 0;
};

struct Layout {
  int L = 0;
  bool resnet = false;
  ResPlan rp;
  int64_t P = 0, Ps = 0;
  int64_t offW[LSGD_MAX_LAYERS] = {}, offB[LSGD_MAX_LAYERS] = {};
  size_t esz = 4;  // activation / operand element size
  // byte offsets into the workspace
  size_t W = 0, U = 0, Wb = 0, Xb = 0, idx = 0, Z = 0, part = 0, rowloss = 0;
  size_t idx2 = 0;  // second index buffer: the next step's rows, sampled early
  size_t Wsync = 0, Ug = 0;  // model at the last sync; global momentum buffer
  size_t E = 0, sign = 0, sign_bytes = 0;  // error memories; sign-sync scratch
  size_t flag = 0;    // int32: set by the loss kernels on a non-finite loss
  size_t Wbar = 0, Wbarb = 0;  // lazy average: the mean [Ps] fp32 (+ bf16)
  bool head = false;  // top layer through the fused head kernels
  size_t act[LSGD_MAX_LAYERS] = {}, dZ[LSGD_MAX_LAYERS + 1] = {};
  size_t total = 0;
};

// The local step's mode bits: Nesterov, and the sign step of Algorithm 3.
int upd_mode(const lsgd_config& cf) {
  return (cf.nesterov ? lsgd::kModeNesterov : 0) |
         (cf.scheme == LSGD_SCHEME_SIGN ? lsgd::kModeSign : 0);
}

bool valid_config(const lsgd_config* c) {
  if (!c) return false;
  if (c->model == LSGD_MODEL_RESNET20) {
    // B_loc below 2^17 keeps each replica's largest activation under 2^31
    // values (the BN and shortcut kernels index it in 32 bits)
    if (c->n_layers != 1 || c->widths[0] != 3072 || c->widths[1] < 2 ||
        c->widths[1] > lsgd::kHeadMaxClasses || c->gemm_dtype != LSGD_FP32 ||
        c->B_loc >= (1 << 17))
      return false;
  } else if (c->model != LSGD_MODEL_MLP) {
    return false;
  }
  if (c->n_layers < 1 || c->n_layers > LSGD_MAX_LAYERS) return false;
  for (int i = 0; i <= c->n_layers; ++i)
    if (c->widths[i] < 1 || c->widths[i] > (1 << 20)) return false;
  if (c->widths[c->n_layers] < 2) return false;  // classes
  if (c->K < 1 || c->K > 65535) return false;
  if (c->B_loc < 1 || c->B_loc > (1 << 20)) return false;
  if (c->gemm_dtype != LSGD_FP32 && c->gemm_dtype != LSGD_BF16) return false;
  if (c->nesterov != 0 && c->nesterov != 1) return false;
  if (!std::isfinite(c->momentum) || c->momentum < 0.f || c->momentum >= 1.f)
    return false;
  if (!std::isfinite(c->weight_decay) || c->weight_decay < 0.f) return false;
  if (!std::isfinite(c->global_momentum) || c->global_momentum < 0.f ||
      c->global_momentum >= 1.f)
    return false;
  if (c->scheme < LSGD_SCHEME_LOCAL || c->scheme > LSGD_SCHEME_EF_SIGN) return false;
  if (c->sampler != LSGD_SAMPLER_IID && c->sampler != LSGD_SAMPLER_EPOCH) return false;
  if (c->sampler == LSGD_SAMPLER_EPOCH && (c->N / c->K) / c->B_loc < 1) return false;
  if (c->scheme != LSGD_SCHEME_LOCAL && c->global_momentum != 0.f) return false;
  if (c->N < c->K || c->N > (int64_t)INT32_MAX) return false;
  return true;
}

Layout make_resnet_layout(const lsgd_config* c) {
  Layout l;
  l.resnet = true;
  l.L = 1;
  ResPlan& r = l.rp;
  r.classes = c->widths[1];
  const int stages[3] = {16, 32, 64};
  int n = 0, ci = 3, side = 32;
  r.cv[n++] = {3, 16, 1, 32, 32, 32, 32, 0, 0, 0, 0, 0};
  ci = 16;
  for (int st = 0; st < 3; ++st) {
    for (int b = 0; b < 3; ++b) {
      const int co = stages[st], stride = (st > 0 && b == 0) ? 2 : 1;
      const int so = side / stride;
      r.cv[n++] = {ci, co, stride, side, side, so, so, 0, 0, 0, 0, 0};
      r.cv[n++] = {co, co, 1, so, so, so, so, 0, 0, 0, 0, 0};
      ci = co;
      side = so;
    }
  }
  int64_t o = 0;
  for (int i = 0; i < kResConvs; ++i) {
    r.cv[i].offW = o;
    o += 9LL * r.cv[i].Cin * r.cv[i].Cout;
    r.cv[i].offG = o;
    o += r.cv[i].Cout;
    r.cv[i].offB = o;
    o += r.cv[i].Cout;
  }
  r.offFcW = o;
  o += 64LL * r.classes;
  r.offFcB = o;
  o += r.classes;
  l.P = o;
  l.Ps = (o + kReplicaPad - 1) / kReplicaPad * kReplicaPad;
  const size_t K = c->K, B = c->B_loc;
  size_t t = 0;
  auto take = [&](size_t bytes) {
    size_t at = t;
    t = align_up(t + bytes, kAlign);
    return at;
  };
  l.W = take(K * l.Ps * 4);
  l.U = take(K * l.Ps * 4);
  for (int i = 0; i < kResConvs; ++i) {
    r.rsoff[i] = r.rs_half;
    r.rs_half += r.cv[i].Cout;
  }
  r.Rs = (2 * r.rs_half + kReplicaPad - 1) / kReplicaPad * kReplicaPad;
  r.rs = take(K * r.Rs * 4);
  l.flag = take(4);
  if (c->global_momentum != 0.f || c->scheme != LSGD_SCHEME_LOCAL)
    l.Wsync = take(l.Ps * 4);
  if (c->global_momentum != 0.f) l.Ug = take(l.Ps * 4);
  if (c->scheme == LSGD_SCHEME_EF_SIGN) l.E = take(K * l.Ps * 4);
  if (c->scheme != LSGD_SCHEME_LOCAL) {
    l.sign_bytes = lsgd::sign_sync_scratch_bytes((int)K, l.Ps);
    l.sign = take(l.sign_bytes);
  }
  l.idx = take(K * B * 4);
  l.rowloss = take(K * B * 4);
  size_t maxact = 0, maxpart = 0, maxbn = 0;
  for (int i = 0; i < kResConvs; ++i) {
    const ConvSpec& q = r.cv[i];
    const size_t sz = K * B * q.Ho * q.Wo * q.Cout * 4;
    r.cv[i].y = take(sz);
    // a block's first BN-ReLU output is never stored (its consumers form it);
    // a block output's mask bits serve the backward passes that need its sign
    if (i % 2 == 0) r.cv[i].act = take(sz);
    if (i % 2 == 0 && i > 0) r.cv[i].mbits = take(sz / 32);
    maxact = std::max(maxact, std::max(sz, K * B * q.H * q.W * q.Cin * 4));
    maxpart = std::max(maxpart, (size_t)lsgd::conv_wgrad_splits(c->B_loc, q.Ho, q.Wo) *
                                    K * 9 * q.Cin * q.Cout * 4);
    maxbn = std::max(maxbn, K * lsgd::bn_chunks(c->B_loc * q.Ho * q.Wo) * q.Cout * 2 * 8);
    // the forward convolutions' statistics: one partial per 256 output rows
    maxbn = std::max(maxbn, K * ((size_t)c->B_loc * q.Ho * q.Wo / 256 + 1) * q.Cout * 2 * 8);
  }
  r.featb = take(K * B * 64 * 4);
  r.dfeat = take(K * B * 64 * 4);
  r.dzh = take(K * B * r.classes * 4);
  for (int i = 0; i < 2; ++i) r.gio[i] = take(maxact);
  // each block's own BN input gradients (its second convolution's output size):
  // the main stream never rewrites one that the side stream may still read
  for (int b = 0; b < 9; ++b)
    for (int j = 0; j < 2; ++j)
      r.bgrad[b][j] = take(K * B * r.cv[2 * b + 2].Ho * r.cv[2 * b + 2].Wo *
                           r.cv[2 * b + 2].Cout * 4);
  r.mu = take(kResConvs * K * 64 * 4);
  r.inv = take(kResConvs * K * 64 * 4);
  r.gsnap = take(kResConvs * K * 64 * 4);
  r.bsnap = take(kResConvs * K * 64 * 4);
  r.coef = take(K * 64 * 5 * 4);
  r.bnpart = take(maxbn);
  r.bnpart2 = take(maxbn);  // the second half's forward statistics
  r.wpart = take(maxpart);
  // the stem's weight-gradient partials apart: the main stream forms them
  // while the side stream may still use wpart
  r.wpart0 = take((size_t)lsgd::conv_wgrad_splits(c->B_loc, r.cv[0].Ho, r.cv[0].Wo) * K * 9 *
                  r.cv[0].Cin * r.cv[0].Cout * 4);
  l.total = t;
  return l;
}

Layout make_layout(const lsgd_config* c) {
  if (c->model == LSGD_MODEL_RESNET20) return make_resnet_layout(c);
  Layout l;
  l.L = c->n_layers;
  int64_t o = 0;
  for (int i = 0; i < l.L; ++i) {
    l.offW[i] = o;
    o += (int64_t)c->widths[i] * c->widths[i + 1];
    l.offB[i] = o;
    o += c->widths[i + 1];
  }
  l.P = o;
  l.Ps = (o + kReplicaPad - 1) / kReplicaPad * kReplicaPad;
  const bool bf = c->gemm_dtype == LSGD_BF16;
  l.esz = bf ? 2 : 4;
  const size_t K = c->K, B = c->B_loc;
  size_t t = 0;
  auto take = [&](size_t bytes) {
    size_t at = t;
    t = align_up(t + bytes, kAlign);
    return at;
  };
  l.W = take(K * l.Ps * 4);
  l.U = take(K * l.Ps * 4);
  l.flag = take(4);
  // the synchronised model of a lazy average (and its bf16 copy)
  l.Wbar = take(l.Ps * 4);
  if (c->gemm_dtype == LSGD_BF16) l.Wbarb = take(l.Ps * 2);
  if (c->global_momentum != 0.f || c->scheme != LSGD_SCHEME_LOCAL)
    l.Wsync = take(l.Ps * 4);
  if (c->global_momentum != 0.f) l.Ug = take(l.Ps * 4);
  if (c->scheme == LSGD_SCHEME_EF_SIGN) l.E = take(K * l.Ps * 4);
  if (c->scheme != LSGD_SCHEME_LOCAL) {
    l.sign_bytes = lsgd::sign_sync_scratch_bytes((int)K, l.Ps);
    l.sign = take(l.sign_bytes);
  }
  if (bf) {
    l.Wb = take(K * l.Ps * 2);
    l.Xb = take((size_t)c->N * c->widths[0] * 2);
  }
  l.idx = take(K * B * 4);
  l.idx2 = take(K * B * 4);
  for (int i = 1; i < l.L; ++i) l.act[i] = take(K * B * c->widths[i] * l.esz);
  l.Z = take(K * B * c->widths[l.L] * 4);
  for (int i = 1; i <= l.L; ++i) l.dZ[i] = take(K * B * c->widths[i] * l.esz);
  // split-K partial sums of the forward and input-gradient GEMMs
  size_t part = 0;
  for (int i = 1; i <= l.L; ++i) {
    const int din = c->widths[i - 1], dout = c->widths[i];
    const int dt = c->gemm_dtype;
    const size_t f = lsgd::gemm_splits(dt, c->B_loc, dout, din, c->K, lsgd::EPI_BIAS);
    if (f > 1) part = std::max(part, f * K * B * dout);
    if (i > 1) {
      const size_t d = lsgd::gemm_splits(dt, c->B_loc, din, dout, c->K, lsgd::EPI_RELU_MASK);
      if (d > 1) part = std::max(part, d * K * B * din);
    }
  }
  l.part = take(part * 4);
  l.head = c->widths[l.L] <= lsgd::kHeadMaxClasses;
  l.rowloss = take(K * B * 4);
  l.total = t;
  return l;
}

}  // namespace

// Opt-in per-launch timing: a pair of HIP events on the context's stream
// around every kernel launch, tagged by launch site.
struct Profiler {
  bool on = false;
  std::string only;  // non-empty: bracket only launches with this tag,
  int every = 1;     // and of those only every `every`-th
  long long seen = 0;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  struct Rec { std::string tag; hipEvent_t a, b; };
  std::vector<Rec> recs;

  hipError_t event(hipEvent_t* e) {
    if (used == pool.size()) {
      hipEvent_t ev;
      // timing only: no system-scope fence (and its cache writeback) at
      // each record, so the bracketed kernels run as they would unobserved
      hipError_t r = hipEventCreateWithFlags(&ev, hipEventDisableSystemFence);
      if (r != hipSuccess) return r;
      pool.push_back(ev);
    }
    *e = pool[used++];
    return hipSuccess;
  }
  bool wants(const std::string& tag) {
    if (only.empty()) return true;
    return tag == only && seen++ % every == 0;
  }
  ~Profiler() {
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }
};

struct lsgd_ctx {
  lsgd_config cfg;
  Profiler prof;
  // side streams for weight updates that do not feed the rest of the step
  // (default priority), with fork/join events; created at init
  hipStream_t side[2] = {nullptr, nullptr};
  hipEvent_t fork[2] = {nullptr, nullptr}, join[2] = {nullptr, nullptr};
  // ResNet: completion of a step's side-stream work (its weight gradients)
  hipEvent_t done = nullptr;
  bool use_side = false;
  Layout lay;
  const float* X = nullptr;
  const int32_t* y = nullptr;
  char* ws = nullptr;
  hipStream_t stream = nullptr;
  int64_t step = 0;
  lsgd_status latched = LSGD_OK;
  std::string err;

  float* W() const { return (float*)(ws + lay.W); }
  float* U() const { return (float*)(ws + lay.U); }
  int* flag() const { return (int*)(ws + lay.flag); }
  // Lazy average (MLP, plain scheme): the synchronisation writes the mean
  // once to Wbar and sets `pending`; the next local step reads the weights
  // from Wbar (replica stride 0) and writes every replica. Anything else that
  // reads the replica array first materialises the mean into it.
  bool lazy = false, pending = false;
  float* Wbar() const { return (float*)(ws + lay.Wbar); }
  bf16_t* Wbarb() const { return lay.Wbarb ? (bf16_t*)(ws + lay.Wbarb) : nullptr; }
  // BN running statistics (ResNet), else nullptr
  float* RS() const { return lay.resnet ? (float*)(ws + lay.rp.rs) : nullptr; }
  bool gm() const { return cfg.global_momentum != 0.f; }
  bool signed_sync() const { return cfg.scheme != LSGD_SCHEME_LOCAL; }
  bool ef() const { return cfg.scheme == LSGD_SCHEME_EF_SIGN; }
  // w_s, the model of the previous synchronisation (global momentum and
  // the sign-compressed schemes keep it)
  float* Wsync() const {
    return gm() || signed_sync() ? (float*)(ws + lay.Wsync) : nullptr;
  }
  float* Ug() const { return gm() ? (float*)(ws + lay.Ug) : nullptr; }
  float* E() const { return ef() ? (float*)(ws + lay.E) : nullptr; }
  bf16_t* Wb() const { return bf16() ? (bf16_t*)(ws + lay.Wb) : nullptr; }
  bf16_t* Xb() const { return (bf16_t*)(ws + lay.Xb); }
  // Sampled rows of the current step. The MLP step samples the next step's
  // rows on side stream 0 into the other buffer (idx_next); `presampled` is
  // the step they belong to (-1: none), and the buffers swap when it starts.
  int idx_alt = 0;
  int64_t presampled = -1;
  int32_t* idx() const { return (int32_t*)(ws + (idx_alt ? lay.idx2 : lay.idx)); }
  int32_t* idx_next() const { return (int32_t*)(ws + (idx_alt ? lay.idx : lay.idx2)); }
  void* act(int l) const { return ws + lay.act[l]; }
  float* Z() const { return (float*)(ws + lay.Z); }
  float* part() const { return (float*)(ws + lay.part); }
  float* rowloss() const { return (float*)(ws + lay.rowloss); }
  void* dZ(int l) const { return ws + lay.dZ[l]; }
  bool bf16() const { return cfg.gemm_dtype == LSGD_BF16; }

  ~lsgd_ctx() {
    for (int i = 0; i < 2; ++i) {
      if (side[i]) {
        (void)hipStreamSynchronize(side[i]);
        (void)hipStreamDestroy(side[i]);
      }
      if (fork[i]) (void)hipEventDestroy(fork[i]);
      if (join[i]) (void)hipEventDestroy(join[i]);
    }
    if (done) (void)hipEventDestroy(done);
  }

  lsgd_status fail(hipError_t e, const char* what) {
    latched = LSGD_E_HIP;
    char buf[256];
    std::snprintf(buf, sizeof buf, "%s: %s", what, hipGetErrorString(e));
    err = buf;
    return LSGD_E_HIP;
  }
};

#define LSGD_CK(ctx, expr)                                  \
  do {                                                      \
    hipError_t e_ = (expr);                                 \
    if (e_ != hipSuccess) return (ctx)->fail(e_, #expr);    \
  } while (0)

// A kernel launch on stream `st`, bracketed by profiling events on that
// stream when profiling is on (and the tag is selected).
#define LSGD_LAUNCH_ON(ctx, st, tag, expr)                                 \
  do {                                                                     \
    hipEvent_t a_ = nullptr, b_ = nullptr;                                 \
    const bool p_ = (ctx)->prof.on && (ctx)->prof.wants(tag);              \
    if (p_) {                                                              \
      LSGD_CK(ctx, (ctx)->prof.event(&a_));                                \
      LSGD_CK(ctx, (ctx)->prof.event(&b_));                                \
      LSGD_CK(ctx, hipEventRecord(a_, (st)));                              \
    }                                                                      \
    LSGD_CK(ctx, expr);                                                    \
    if (p_) {                                                              \
      LSGD_CK(ctx, hipEventRecord(b_, (st)));                              \
      (ctx)->prof.recs.push_back({std::string(tag), a_, b_});              \
    }                                                                      \
  } while (0)
#define LSGD_LAUNCH(ctx, tag, expr) LSGD_LAUNCH_ON(ctx, (ctx)->stream, tag, expr)

namespace {

lsgd_status do_local_step_resnet(lsgd_ctx* c, float lr, float* d_loss);

// The index sets of local step `step` by the configured sampler.
hipError_t sample(const lsgd_ctx* c, int64_t step, int32_t* idx, hipStream_t s) {
  const lsgd_config& cf = c->cfg;
  if (cf.sampler == LSGD_SAMPLER_EPOCH)
    return lsgd::launch_sample_epoch(cf.seed, step, cf.K, cf.N, cf.B_loc, idx, s);
  return lsgd::launch_sample(cf.seed, step, cf.K, cf.N, cf.B_loc, idx, s);
}

// Tiles (128 x 128) from which one persistent launch over all hidden layers
// updates beats per-layer launches (about four per compute unit).
constexpr int kMergedMinTiles = 1024;

// Weight gradient of layer l fused with its momentum-SGD step and the bias
// step: G_l = A_{l-1}^T dZ_l over the batch, per replica.
GemmArgs wgrad_args(const lsgd_ctx* c, int l, float lr) {
  const lsgd_config& cf = c->cfg;
  const Layout& ly = c->lay;
  const int K = cf.K, B = cf.B_loc;
  const int din = cf.widths[l - 1], dout = cf.widths[l];
  const bool dt = c->bf16();
  GemmArgs a{};
  a.G = K;
  a.M = din;
  a.N = dout;
  a.Kd = B;
  if (l == 1) {
    a.A = dt ? (const void*)c->Xb() : (const void*)c->X;
    a.sA = 0;
    a.rowmap = c->idx();
    a.sRow = B;
  } else {
    a.A = c->act(l - 1);
    a.sA = (long long)B * din;
  }
  a.lda = din;
  a.B = c->dZ(l);
  a.ldb = dout;
  a.sB = (long long)B * dout;
  a.ldc = dout;
  a.sC = ly.Ps;
  a.W = c->W() + ly.offW[l - 1];
  a.U = c->U() + ly.offW[l - 1];
  a.Wb = dt ? c->Wb() + ly.offW[l - 1] : nullptr;
  a.lr = lr;
  a.mom = cf.momentum;
  a.wd = cf.weight_decay;
  a.nesterov = upd_mode(cf);
  a.bias_w = c->W() + ly.offB[l - 1];
  a.bias_u = c->U() + ly.offB[l - 1];
  a.sBiasP = ly.Ps;
  if (c->pending) {  // step the shared mean of a lazy average
    a.Wsrc = c->Wbar() + ly.offW[l - 1];
    a.sWsrc = 0;
    a.bias_src = c->Wbar() + ly.offB[l - 1];
    a.sBiasSrc = 0;
  }
  a.splits = 1;
  return a;
}

lsgd_status do_local_step(lsgd_ctx* c, float lr, float* d_loss) {
  if (c->lay.resnet) return do_local_step_resnet(c, lr, d_loss);
  const lsgd_config& cf = c->cfg;
  const Layout& ly = c->lay;
  const int K = cf.K, B = cf.B_loc, L = ly.L;
  const int* w = cf.widths;
  const int dt = c->bf16() ? 1 : 0;
  const hipStream_t s = c->stream;
  float* W = c->W();
  float* U = c->U();
  bf16_t* Wb = c->Wb();
  const void* X0 = dt ? (const void*)c->Xb() : (const void*)c->X;
  // where this step reads the weights: the replicas, or the shared mean of
  // a pending lazy average
  const float* Wr = c->pending ? c->Wbar() : W;
  const bf16_t* Wbr = c->pending ? c->Wbarb() : Wb;
  const long long sWr = c->pending ? 0 : ly.Ps;

  // this step's rows: sampled by the step before on the side stream, or now
  if (c->presampled == c->step && c->lay.idx2 != 0)
    c->idx_alt ^= 1;
  else
    LSGD_LAUNCH(c, "sample", sample(c, c->step, c->idx(), s));
  c->presampled = -1;
  bool presample = false;
  bool side0 = false, side1 = false;  // work forked onto the side streams

  // forward: Z_l = A_{l-1} W_l + b_l, A_l = relu(Z_l) below the top layer
  const int Lg = ly.head ? L - 1 : L;  // layers through the generic GEMMs
  for (int l = 1; l <= Lg; ++l) {
    const int din = w[l - 1], dout = w[l];
    GemmArgs a{};
    a.G = K;
    a.M = B;
    a.N = dout;
    a.Kd = din;
    if (l == 1) {
      a.A = X0;
      a.sA = 0;
      a.rowmap = c->idx();
      a.sRow = B;
    } else {
      a.A = c->act(l - 1);
      a.sA = (long long)B * din;
    }
    a.lda = din;
    a.B = dt ? (const void*)(Wbr + ly.offW[l - 1]) : (const void*)(Wr + ly.offW[l - 1]);
    a.ldb = dout;
    a.sB = sWr;
    a.bias = Wr + ly.offB[l - 1];
    a.sBias = sWr;
    a.ldc = dout;
    a.sC = (long long)B * dout;
    a.splits = lsgd::gemm_splits(dt, B, dout, din, K, lsgd::EPI_BIAS);
    a.part = c->part();
    if (l < L) {
      a.C = c->act(l);
      LSGD_LAUNCH(c, "fwd" + std::to_string(l),
                  lsgd::launch_gemm(dt, 0, 0, lsgd::EPI_BIAS_RELU, dt, a, s));
    } else {
      a.C = c->Z();
      LSGD_LAUNCH(c, "fwd" + std::to_string(l),
                  lsgd::launch_gemm(dt, 0, 0, lsgd::EPI_BIAS, 0, a, s));
    }
  }

  lsgd::HeadArgs h{};
  if (ly.head) {
    h.K = K;
    h.B = B;
    h.D = w[L - 1];
    h.C = w[L];
    h.gather = L == 1;
    h.A = L == 1 ? X0 : c->act(L - 1);
    h.sA = (long long)B * w[L - 1];
    h.rowmap = c->idx();
    h.y = c->y;
    h.W = dt ? (const void*)(Wbr + ly.offW[L - 1]) : (const void*)(Wr + ly.offW[L - 1]);
    h.sW = sWr;
    h.Wm = W + ly.offW[L - 1];
    h.Um = U + ly.offW[L - 1];
    h.Wb = dt ? Wb + ly.offW[L - 1] : nullptr;
    h.bias = Wr + ly.offB[L - 1];
    h.sBias = sWr;
    h.Wsrc = Wr + ly.offW[L - 1];
    h.bsrc = Wr + ly.offB[L - 1];
    h.sSrc = sWr;
    h.bias_w = W + ly.offB[L - 1];
    h.bias_u = U + ly.offB[L - 1];
    h.sP = ly.Ps;
    h.dZ = c->dZ(L);
    h.dZprev = L > 1 ? c->dZ(L - 1) : nullptr;
    h.rowloss = c->rowloss();
    h.loss = d_loss;
    h.nonfinite = c->flag();
    h.lr = lr;
    h.mom = cf.momentum;
    h.wd = cf.weight_decay;
    h.nesterov = upd_mode(cf);
    // logits, loss, dZ_L and the masked input gradient of the top layer
    LSGD_LAUNCH(c, "head_fwd", lsgd::launch_head_fwd(dt, h, s));
    // the top layer's weight gradient feeds nothing else in this step: it
    // runs on side stream 0 while the backward pass continues
    if (c->use_side) {
      LSGD_CK(c, hipEventRecord(c->fork[0], s));
      LSGD_CK(c, hipStreamWaitEvent(c->side[0], c->fork[0], 0));
      LSGD_LAUNCH_ON(c, c->side[0], "head_wgrad",
                     lsgd::launch_head_wgrad(dt, h, c->side[0]));
      // the next step's rows, off the critical path, into the buffer this
      // step does not read (its previous rows' readers, the step before,
      // precede head_fwd, after which this stream runs)
      if (c->lay.idx2 != 0) {
        LSGD_LAUNCH_ON(c, c->side[0], "sample",
                       sample(c, c->step + 1, c->idx_next(), c->side[0]));
        presample = true;
      }
      LSGD_CK(c, hipEventRecord(c->join[0], c->side[0]));
      side0 = true;
    } else {
      LSGD_LAUNCH(c, "head_wgrad", lsgd::launch_head_wgrad(dt, h, s));
    }
  } else {
    LSGD_LAUNCH(c, "xent", lsgd::launch_xent(c->Z(), c->y, c->idx(), K, B, w[L],
                                               c->dZ(L), dt, d_loss, c->flag(), s));
  }

  // backward, top layer first. The input gradient of layer l reads the
  // pre-update W_l, so it is enqueued before W_l's fused update. When every
  // hidden layer's update fits the persistent update kernel and together
  // they fill the chip, the input gradients go first and one launch then
  // updates all of those layers (their tiles in one list).
  GemmArgs upd[lsgd::kWsMaxProblems];
  int nupd = 0;
  bool merged = false;
  if (Lg >= 1 && Lg <= lsgd::kWsMaxProblems) {
    for (int l = 1; l <= Lg; ++l) upd[l - 1] = wgrad_args(c, l, lr);
    const int tiles = lsgd::gemm_sgd_multi_tiles(dt, upd, Lg);
    merged = tiles >= kMergedMinTiles;
    nupd = Lg;
  }
  for (int l = Lg; l >= 1; --l) {
    const int din = w[l - 1], dout = w[l];
    if (l > 1 && !(ly.head && l == L)) {
      GemmArgs a{};
      a.G = K;
      a.M = B;
      a.N = din;
      a.Kd = dout;
      a.A = c->dZ(l);
      a.lda = dout;
      a.sA = (long long)B * dout;
      a.B = dt ? (const void*)(Wbr + ly.offW[l - 1]) : (const void*)(Wr + ly.offW[l - 1]);
      a.ldb = dout;
      a.sB = sWr;
      a.C = c->dZ(l - 1);
      a.ldc = din;
      a.sC = (long long)B * din;
      a.mask = c->act(l - 1);
      a.splits = lsgd::gemm_splits(dt, B, din, dout, K, lsgd::EPI_RELU_MASK);
      a.part = c->part();
      LSGD_LAUNCH(c, "dgrad" + std::to_string(l),
                  lsgd::launch_gemm(dt, 0, 1, lsgd::EPI_RELU_MASK, dt, a, s));
    }
    if (merged) continue;
    const GemmArgs a = wgrad_args(c, l, lr);
    if (c->use_side && l > 1) {
      // after its input gradient, layer l's update only has to finish by the
      // end of the step: side stream 1, overlapping the layers below
      LSGD_CK(c, hipEventRecord(c->fork[1], s));
      LSGD_CK(c, hipStreamWaitEvent(c->side[1], c->fork[1], 0));
      LSGD_LAUNCH_ON(c, c->side[1], "wgrad_update" + std::to_string(l),
                     lsgd::launch_gemm(dt, 1, 0, lsgd::EPI_SGD, 0, a, c->side[1]));
      side1 = true;
    } else {
      LSGD_LAUNCH(c, "wgrad_update" + std::to_string(l),
                  lsgd::launch_gemm(dt, 1, 0, lsgd::EPI_SGD, 0, a, s));
    }
  }
  if (merged)
    LSGD_LAUNCH(c, "wgrad_update", lsgd::launch_gemm_sgd_multi(dt, upd, nupd, s));
  // join: the step ends when all of its updates have; a side stream with no
  // work this step is not waited for (each wait costs the stream some µs)
  if (side0) LSGD_CK(c, hipStreamWaitEvent(s, c->join[0], 0));
  if (side1) {
    LSGD_CK(c, hipEventRecord(c->join[1], c->side[1]));
    LSGD_CK(c, hipStreamWaitEvent(s, c->join[1], 0));
  }
  c->step += 1;
  c->pending = false;  // every replica now holds its own stepped model
  if (presample) c->presampled = c->step;
  return LSGD_OK;
}

lsgd_status do_local_step_resnet(lsgd_ctx* c, float lr, float* d_loss) {
  const lsgd_config& cf = c->cfg;
  const ResPlan& r = c->lay.rp;
  const int K = cf.K, B = cf.B_loc;
  const long long Ps = c->lay.Ps;
  const hipStream_t s = c->stream;
  float* W = c->W();
  float* U = c->U();
  auto F = [&](size_t off) { return (float*)(c->ws + off); };
  auto M = [&](size_t off) { return (unsigned*)(c->ws + off); };
  float* mu = F(r.mu);
  float* inv = F(r.inv);
  double* bnpart = (double*)(c->ws + r.bnpart);
  auto geom = [&](int i) {
    const ConvSpec& q = r.cv[i];
    lsgd::ConvGeom g{};
    g.G = K;
    g.Bt = B;
    g.H = q.H;
    g.W = q.W;
    g.Cin = q.Cin;
    g.Ho = q.Ho;
    g.Wo = q.Wo;
    g.Cout = q.Cout;
    g.stride = q.stride;
    g.sx = (long long)B * q.H * q.W * q.Cin;
    g.Wk = W + q.offW;
    g.sW = Ps;
    return g;
  };
  auto rows = [&](int i) { return B * r.cv[i].Ho * r.cv[i].Wo; };

  LSGD_LAUNCH(c, "sample", sample(c, c->step, c->idx(), s));

  // the input of a block's second convolution is the first convolution's
  // BN-ReLU output, which is never stored: the kernels form it from that
  // convolution's pre-BN output (BN layer j) as they load it
  // (the scale and shift as the forward batch used them: the backward pass
  // steps gamma and beta while weight gradients that read them may still run)
  float* gsnap = F(r.gsnap);
  float* bsnap = F(r.bsnap);
  auto bn_input = [&](lsgd::ConvGeom& g, int j) {
    g.bn_mu = mu + (size_t)j * K * 64;
    g.bn_inv = inv + (size_t)j * K * 64;
    g.bn_g = gsnap + (size_t)j * K * 64;
    g.bn_b = bsnap + (size_t)j * K * 64;
    g.bn_sP = r.cv[j].Cout;
  };

  // The forward pass of replicas g0 .. g0 + Kh - 1 on stream fs, its BN
  // statistics' partials in part: layer i of the stem and blocks (a:
  // conv-BN-ReLU, b: conv-BN + shortcut, ReLU), then the head (pool,
  // classifier, loss and the classifier's update). Every tensor is per
  // replica, so a subset of them is a pointer offset and a smaller grid.
  const ConvSpec& last = r.cv[kResConvs - 1];
  const int S = last.Ho * last.Wo;
  auto per = [&](int i) {  // values per replica of conv i's output
    return (long long)B * r.cv[i].Ho * r.cv[i].Wo * r.cv[i].Cout;
  };
  auto fwd_layer = [&](int i, int g0, int Kh, hipStream_t fs, double* part) -> lsgd_status {
    const ConvSpec& q = r.cv[i];
    const int C = q.Cout;
    lsgd::ConvGeom g = geom(i);
    g.G = Kh;
    g.Wk += (size_t)g0 * Ps;
    if (i == 0) {
      g.x = c->X;
      g.sx = 0;
      g.rowmap = c->idx() + (size_t)g0 * B;
    } else if (i % 2 == 0) {  // second convolution of a block
      g.x = F(r.cv[i - 1].y) + g0 * g.sx;
      bn_input(g, i - 1);
      const int Cj = r.cv[i - 1].Cout;
      g.bn_mu += (size_t)g0 * Cj;
      g.bn_inv += (size_t)g0 * Cj;
      g.bn_g += (size_t)g0 * Cj;
      g.bn_b += (size_t)g0 * Cj;
    } else {  // first convolution: the block input (stem or previous block output)
      g.x = F(r.cv[i - 1].act) + g0 * g.sx;
    }
    float* y = F(q.y) + g0 * per(i);
    g.out = y;
    // the convolution writes its BN statistics per 256-row chunk where its
    // kernel can; otherwise a separate pass reads the output
    const bool fused = lsgd::conv_fwd_stats(g) && rows(i) % 256 == 0;
    g.stats = fused ? part : nullptr;
    LSGD_LAUNCH_ON(c, fs, "conv_fwd", lsgd::launch_conv(lsgd::CONV_FWD_MODE, g, fs));
    float* mi = mu + (size_t)i * K * 64 + (size_t)g0 * C;
    float* ii = inv + (size_t)i * K * 64 + (size_t)g0 * C;
    // this replica's running statistics of BN layer i follow the batch
    float* rm = c->RS() + r.rsoff[i] + g0 * r.Rs;
    float* rv = c->RS() + r.rs_half + r.rsoff[i] + g0 * r.Rs;
    float* gs = gsnap + (size_t)i * K * 64 + (size_t)g0 * C;
    float* bs = bsnap + (size_t)i * K * 64 + (size_t)g0 * C;
    float* gm = W + q.offG + (size_t)g0 * Ps;
    float* bt = W + q.offB + (size_t)g0 * Ps;
    if (fused)
      LSGD_LAUNCH_ON(c, fs, "bn_stats",
                     lsgd::launch_bn_finalize_chunks(part, rows(i) / 256, Kh, rows(i), C, mi,
                                                     ii, rm, rv, r.Rs, fs, gm, bt, Ps, gs,
                                                     bs));
    else
      LSGD_LAUNCH_ON(c, fs, "bn_stats",
                     lsgd::launch_bn_stats(y, Kh, rows(i), C, part, mi, ii, rm, rv, r.Rs, fs,
                                           gm, bt, Ps, gs, bs));
    if (i % 2 == 1) return LSGD_OK;  // a block's first BN-ReLU: formed by its consumers
    int mode = 0;
    const float* blk_in = nullptr;
    int cin_blk = 0;
    if (i > 0) {  // second convolution of a block
      const ConvSpec& qa = r.cv[i - 1];
      blk_in = F(r.cv[i - 2].act) + g0 * per(i - 2);
      cin_blk = qa.Cin;
      mode = (qa.stride == 1 && qa.Cin == q.Cout) ? 1 : 2;
    }
    LSGD_LAUNCH_ON(c, fs, "bn_apply",
                   lsgd::launch_bn_apply(y, Kh, rows(i), C, mi, ii, gm, bt, Ps, mode, blk_in,
                                         q.Ho, q.Wo, cin_blk, F(q.act) + g0 * per(i),
                                         i > 0 ? M(q.mbits) + g0 * per(i) / 32 : nullptr,
                                         fs));
    return LSGD_OK;
  };
  auto fwd_head = [&](int g0, int Kh, hipStream_t fs) -> lsgd_status {
    // head: global average pool, classifier, loss
    LSGD_LAUNCH_ON(c, fs, "gap",
                   lsgd::launch_gap(F(last.act) + g0 * per(kResConvs - 1), Kh * B, S, 64,
                                    F(r.featb) + (size_t)g0 * B * 64, false, nullptr, nullptr,
                                    fs));
    const size_t pg = (size_t)g0 * Ps;
    lsgd::HeadArgs h{};
    h.K = Kh;
    h.B = B;
    h.D = 64;
    h.C = r.classes;
    h.gather = 0;
    h.A = F(r.featb) + (size_t)g0 * B * 64;
    h.sA = (long long)B * 64;
    h.rowmap = c->idx() + (size_t)g0 * B;
    h.y = c->y;
    h.W = W + r.offFcW + pg;
    h.sW = Ps;
    h.Wm = W + r.offFcW + pg;
    h.Um = U + r.offFcW + pg;
    h.bias = W + r.offFcB + pg;
    h.sBias = Ps;
    h.Wsrc = W + r.offFcW + pg;
    h.bsrc = W + r.offFcB + pg;
    h.sSrc = Ps;
    h.bias_w = W + r.offFcB + pg;
    h.bias_u = U + r.offFcB + pg;
    h.sP = Ps;
    h.dZ = F(r.dzh) + (size_t)g0 * B * r.classes;
    h.dZprev = F(r.dfeat) + (size_t)g0 * B * 64;
    h.nomask = 1;
    h.rowloss = c->rowloss() + (size_t)g0 * B;
    h.loss = d_loss ? d_loss + g0 : nullptr;
    h.nonfinite = c->flag();
    h.lr = lr;
    h.mom = cf.momentum;
    h.wd = cf.weight_decay;
    h.nesterov = upd_mode(cf);
    LSGD_LAUNCH_ON(c, fs, "head_fwd", lsgd::launch_head_fwd(0, h, fs));
    LSGD_LAUNCH_ON(c, fs, "head_wgrad", lsgd::launch_head_wgrad(0, h, fs));
    return LSGD_OK;
  };
  // With side streams, the two halves of the replicas run their forward
  // passes on the main and the side stream: nothing passes between replicas,
  // and each half's memory-bound BN passes overlap the other's convolutions.
  // The launches go out layer by layer, alternating, so that both streams
  // have work from the start (the second half started a layer behind the
  // first measured no different).
  if (c->use_side && K % 2 == 0) {
    const int Kh = K / 2;
    hipStream_t s2 = c->side[1];
    double* part2 = (double*)(c->ws + r.bnpart2);
    LSGD_CK(c, hipEventRecord(c->fork[1], s));
    LSGD_CK(c, hipStreamWaitEvent(s2, c->fork[1], 0));
    for (int i = 0; i < kResConvs; ++i) {
      if (lsgd_status st = fwd_layer(i, 0, Kh, s, bnpart)) return st;
      if (lsgd_status st = fwd_layer(i, Kh, Kh, s2, part2)) return st;
    }
    if (lsgd_status st = fwd_head(0, Kh, s)) return st;
    if (lsgd_status st = fwd_head(Kh, Kh, s2)) return st;
    LSGD_CK(c, hipEventRecord(c->join[1], s2));
    LSGD_CK(c, hipStreamWaitEvent(s, c->join[1], 0));
  } else {
    for (int i = 0; i < kResConvs; ++i)
      if (lsgd_status st = fwd_layer(i, 0, K, s, bnpart)) return st;
    if (lsgd_status st = fwd_head(0, K, s)) return st;
  }

  // backward
  float* gb[2] = {F(r.gio[0]), F(r.gio[1])};
  float* coef = F(r.coef);
  float* wpart = F(r.wpart);
  LSGD_LAUNCH(c, "gap_bwd", lsgd::launch_gap(nullptr, K * B, S, 64, nullptr, true,
                                             F(r.dfeat), gb[0], s));
  int cur = 0;  // gb[cur] holds the gradient of the current block output
  // BN backward (coefficients, gamma/beta update, input gradient into dy)
  // (fused_nchunk > 0: the sums are in bnpart already, from the input
  // gradient that produced gup)
  auto bn_bwd = [&](int i, const float* gup, const unsigned* mbits, float* dy,
                    int fused_nchunk) {
    const ConvSpec& q = r.cv[i];
    return lsgd::launch_bn_backward(F(q.y), gup, mbits, K, rows(i), q.Cout, bnpart,
                                    mu + (size_t)i * K * 64, inv + (size_t)i * K * 64,
                                    coef, W + q.offG, W + q.offB, U + q.offG,
                                    U + q.offB, Ps, lr, cf.momentum, upd_mode(cf), dy,
                                    fused_nchunk, s);
  };
  // weight gradient of conv i from its input x and output gradient dy into
  // per-split partials, then their fixed-order sum and the update (after
  // any input gradient that reads the old weight)
  // (bn_layer >= 0: x is that BN layer's pre-BN output, see bn_input)
  auto wgrad = [&](int i, const float* x, const float* dy, int bn_layer, hipStream_t ws,
                   float* part) -> lsgd_status {
    const ConvSpec& q = r.cv[i];
    lsgd::ConvGeom g = geom(i);
    if (i == 0) {
      g.x = c->X;
      g.sx = 0;
      g.rowmap = c->idx();
    } else {
      g.x = x;
      if (bn_layer >= 0) bn_input(g, bn_layer);
    }
    g.dy = dy;
    g.out = part;
    LSGD_LAUNCH_ON(c, ws, "conv_wgrad", lsgd::launch_conv(lsgd::CONV_WGRAD_MODE, g, ws));
    LSGD_LAUNCH_ON(c, ws, "conv_wupdate",
                   lsgd::launch_conv_wupdate(part, lsgd::conv_wgrad_splits(B, q.Ho, q.Wo),
                                             K, 9 * q.Cin * q.Cout, W + q.offW, U + q.offW,
                                             Ps, lr, cf.momentum, cf.weight_decay,
                                             upd_mode(cf), ws));
    return LSGD_OK;
  };
  // The weight gradients (and updates) of a block run on side stream 1: they
  // fork after the block's last input gradient (the last reader of its
  // weights) and overlap the next block's BN backward passes and input
  // gradients on the main stream (memory-bound passes beside the weight
  // gradients' matrix work; a fork after the next BN's sums and coefficients,
  // which then run alone, set the weight gradients against the input
  // gradients' matrix work instead and was slower). A block's two BN input
  // gradients (the second BN's, and the first BN's formed in place over the
  // gradient it came from) have buffers of their own, so the main stream
  // waits for the side stream only at the step's end (with buffers shared
  // by parity, a wait before each block cost the main stream some µs each);
  // one wpart serves all blocks, in the side stream's order (the
  // stem's weight gradient, on the main stream, has its own). Without side
  // streams everything runs in order on the main stream.
  const bool sidew = c->use_side;
  hipStream_t ws = sidew ? c->side[1] : s;
  bool pend = false;
  auto join_side = [&]() -> lsgd_status {  // the main stream waits for event done
    if (pend) LSGD_CK(c, hipStreamWaitEvent(s, c->done, 0));
    pend = false;
    return LSGD_OK;
  };
  // the weight gradients of block (ib, ia) with its BN input gradients g1, g2
  // and input h_in, forked to the side stream
  // (the last block's, block 0's, records done after all of the side
  // stream's work of the step)
  auto fork = [&](int ib, int ia, bool last, const float* g1, const float* g2,
                  const float* h_in) -> lsgd_status {
    if (sidew) {
      LSGD_CK(c, hipEventRecord(c->fork[1], s));
      LSGD_CK(c, hipStreamWaitEvent(ws, c->fork[1], 0));
    }
    if (lsgd_status st = wgrad(ib, F(r.cv[ia].y), g1, ia, ws, wpart)) return st;
    if (lsgd_status st = wgrad(ia, h_in, g2, -1, ws, wpart)) return st;
    if (sidew && last) {
      LSGD_CK(c, hipEventRecord(c->done, ws));
      pend = true;
    }
    return LSGD_OK;
  };
  // input gradient of conv i (reads the old weight, before its update).
  // Where the kernel takes the epilogues: with sc_dh, sc_hb the identity
  // shortcut's share of the block-output gradient goes into dx (*sc_fused);
  // with bs_layer >= 0 the backward sums of BN layer bs_layer, whose
  // activation's gradient dx is, go to bnpart (*sums_fused) -- its ReLU mask
  // recomputed from the pre-BN output, or, with bs_act, read from that
  // activation's mask bits (a BN whose ReLU follows a shortcut add).
  auto dgrad = [&](int i, const float* dy, float* dx, const float* sc_dh,
                   const unsigned* sc_hb, int bs_layer, const unsigned* bs_act,
                   bool* sc_fused, bool* sums_fused) -> lsgd_status {
    lsgd::ConvGeom g = geom(i);
    g.dy = dy;
    g.out = dx;
    const int cap = lsgd::conv_dgrad_epilogues(g);
    *sc_fused = sc_dh && (cap & 1);
    *sums_fused = bs_layer >= 0 && (cap & (bs_act ? 4 : 2)) &&
                  rows(bs_layer) == B * r.cv[i].H * r.cv[i].W && rows(bs_layer) % 256 == 0;
    if (*sc_fused) {
      g.sc_dh = sc_dh;
      g.sc_hb = sc_hb;
    }
    if (*sums_fused) {
      g.bs_y = F(r.cv[bs_layer].y);
      g.bs_hb = bs_act;
      g.bs_part = bnpart;
      bn_input(g, bs_layer);
    }
    LSGD_LAUNCH(c, "conv_dgrad", lsgd::launch_conv(lsgd::CONV_DGRAD_MODE, g, s));
    return LSGD_OK;
  };

  // (out_sums: the backward sums of the BN whose output's gradient the last
  // block-input gradient was are in bnpart already)
  bool out_sums = false;
  for (int blk = 8; blk >= 0; --blk) {
    const int ia = 2 * blk + 1, ib = 2 * blk + 2;
    const ConvSpec& qa = r.cv[ia];
    const int nxt = 1 - cur;
    float* g1 = F(r.bgrad[blk][0]);
    float* g2 = F(r.bgrad[blk][1]);
    // second convolution: its output went through the shortcut add and ReLU
    const unsigned* mb = M(r.cv[ib].mbits);
    LSGD_LAUNCH(c, "bn_bwd", bn_bwd(ib, gb[cur], mb, g1, out_sums ? rows(ib) / 256 : 0));
    bool sums_fused = false, sc_fused = false, unused = false;
    if (lsgd_status st = dgrad(ib, g1, g2, nullptr, nullptr, ia, nullptr, &unused, &sums_fused))
      return st;
    // first convolution: ReLU'd BN output, the mask recomputed from its input
    // (dy in place over its gradient)
    LSGD_LAUNCH(c, "bn_bwd", bn_bwd(ia, g2, nullptr, g2, sums_fused ? rows(ia) / 256 : 0));
    // the block-input gradient: the convolution path, and the shortcut's share
    // of the block-output gradient, and (identity blocks) the backward sums of
    // the BN before the block input -- the previous block's second BN, masked
    // by its activation, or the stem's -- in the input gradient's epilogue
    // where it can
    const int mode = (qa.stride == 1 && qa.Cin == qa.Cout) ? 1 : 2;
    const int prev_bn = ia - 1;
    if (lsgd_status st = dgrad(ia, g2, gb[nxt], gb[cur], mb, mode == 1 ? prev_bn : -1,
                               prev_bn > 0 ? M(r.cv[prev_bn].mbits) : nullptr, &sc_fused,
                               &out_sums))
      return st;
    if (lsgd_status st = fork(ib, ia, blk == 0, g1, g2, F(r.cv[ia - 1].act))) return st;
    if (!sc_fused)
      LSGD_LAUNCH(c, "shortcut_bwd",
                  lsgd::launch_shortcut_grad(gb[nxt], gb[cur], mb, K, B, qa.H, qa.W, qa.Cin,
                                             qa.Cout, mode, s));
    cur = nxt;
  }
  // the stem: its BN input gradient in place over the gradient it came from
  // (the side stream reads neither of gio), its weight gradient into
  // its own partials; then the join (the side stream's last work, block 0's,
  // was recorded last: all its updates are done)
  LSGD_LAUNCH(c, "bn_bwd", bn_bwd(0, gb[cur], nullptr, gb[cur], out_sums ? rows(0) / 256 : 0));
  if (lsgd_status st = wgrad(0, nullptr, gb[cur], -1, s, F(r.wpart0))) return st;
  if (lsgd_status st = join_side()) return st;
  c->step += 1;
  return LSGD_OK;
}

// The BN running statistics (ResNet) take the plain mean over the replicas
// (over each block of Kb for a block synchronisation) at every
// synchronisation, whatever the scheme: they are not trained parameters.
lsgd_status average_running_stats(lsgd_ctx* c, int Kb) {
  if (!c->RS()) return LSGD_OK;
  const int K = c->cfg.K;
  const long long Rs = c->lay.rp.Rs;
  if (Kb == K)
    LSGD_LAUNCH(c, "average_bn_running",
                lsgd::launch_average(c->RS(), nullptr, K, Rs, Rs, nullptr, c->stream));
  else if (Kb > 1)
    LSGD_LAUNCH(c, "average_bn_running",
                lsgd::launch_average_blocks(c->RS(), nullptr, Kb, K / Kb, Rs, Rs, nullptr,
                                            c->stream));
  return LSGD_OK;
}

// A pending lazy average written out: every replica (and its bf16 copy)
// := the mean. Bit for bit what the plain average would have left there.
lsgd_status materialise(lsgd_ctx* c) {
  if (!c->pending) return LSGD_OK;
  LSGD_LAUNCH(c, "average_materialise",
              lsgd::launch_broadcast(c->Wbar(), c->W(), c->Wb(), c->cfg.K, c->lay.Ps,
                                     c->lay.Ps, -1, c->stream));
  c->pending = false;
  return LSGD_OK;
}

lsgd_status do_average(lsgd_ctx* c) {
  if (lsgd_status st = materialise(c)) return st;  // average the replicas as stored
  if (c->lazy) {
    // the mean once (and its bf16 copy); the next step reads it for every
    // replica
    LSGD_LAUNCH(c, "average",
                lsgd::launch_average(c->W(), c->Wbarb(), c->cfg.K, c->lay.Ps, c->lay.Ps,
                                     c->Wbar(), c->stream));
    c->pending = true;
    return LSGD_OK;
  }
  LSGD_LAUNCH(c, "average",
              lsgd::launch_average(c->W(), c->Wb(), c->cfg.K, c->lay.Ps,
                                   c->lay.Ps, nullptr, c->stream));
  return average_running_stats(c, c->cfg.K);
}

// The end-of-round synchronisation: the plain average, or with a global
// momentum factor its momentum form at step size lr.
lsgd_status do_synchronise(lsgd_ctx* c, float lr) {
  if (c->signed_sync()) {
    LSGD_LAUNCH(c, "sign_sync",
                lsgd::launch_sign_sync(c->W(), c->Wb(), c->E(), c->Wsync(),
                                       c->cfg.K, c->lay.P, c->lay.Ps,
                                       c->ws + c->lay.sign, c->lay.sign_bytes,
                                       c->stream));
    return average_running_stats(c, c->cfg.K);
  }
  if (!c->gm()) return do_average(c);
  LSGD_LAUNCH(c, "average",
              lsgd::launch_average_gm(c->W(), c->Wb(), c->cfg.K, c->lay.Ps,
                                      c->lay.Ps, c->Wsync(), c->Ug(),
                                      c->cfg.global_momentum, lr, c->stream));
  return average_running_stats(c, c->cfg.K);
}

lsgd_status do_average_blocks(lsgd_ctx* c, int Kb) {
  if (Kb == c->cfg.K) return do_average(c);
  if (Kb == 1) return LSGD_OK;  // every block holds one replica
  if (lsgd_status st = materialise(c)) return st;
  LSGD_LAUNCH(c, "average_blocks",
              lsgd::launch_average_blocks(c->W(), c->Wb(), Kb, c->cfg.K / Kb,
                                          c->lay.Ps, c->lay.Ps, nullptr,
                                          c->stream));
  return average_running_stats(c, Kb);
}

// A whole round of softmax regression (one fp32 layer, plain local SGD and
// averaging) in one launch when the replicas fit in LDS.
bool tiny_round_ok(const lsgd_ctx* c, int H) {
  const lsgd_config& cf = c->cfg;
  return cf.model == LSGD_MODEL_MLP && cf.n_layers == 1 && cf.gemm_dtype == LSGD_FP32 &&
         cf.scheme == LSGD_SCHEME_LOCAL && cf.global_momentum == 0.f &&
         lsgd::tiny_round_fits(cf.K, cf.B_loc, cf.widths[0], cf.widths[1], H);
}

lsgd_status do_tiny_round(lsgd_ctx* c, int H, const float* h_lr, float* d_loss) {
  if (lsgd_status st = materialise(c)) return st;
  const lsgd_config& cf = c->cfg;
  lsgd::TinyArgs a{};
  a.X = c->X;
  a.y = c->y;
  a.W = c->W();
  a.U = c->U();
  a.loss = d_loss;
  a.nonfinite = c->flag();
  a.N = cf.N;
  a.Ps = c->lay.Ps;
  a.step0 = c->step;
  a.K = cf.K;
  a.B = cf.B_loc;
  a.D = cf.widths[0];
  a.C = cf.widths[1];
  a.H = H;
  a.key0 = (uint32_t)cf.seed;
  a.key1 = (uint32_t)(cf.seed >> 32);
  a.mom = cf.momentum;
  a.wd = cf.weight_decay;
  a.mode = upd_mode(cf);
  if (cf.sampler == LSGD_SAMPLER_EPOCH) {
    a.S = (cf.N / cf.K) / cf.B_loc;
    a.m = 1;
    while ((1LL << (2 * a.m)) < cf.N) ++a.m;
  }
  for (int h = 0; h < H; ++h) a.lr[h] = h_lr[h];
  // the two kernels launch under their own tags
  const char* tag = lsgd::tiny_round_wide(a.K, a.B, a.D, a.C, a.H) ? "tiny_round_wide"
                                                                  : "tiny_round";
  LSGD_LAUNCH(c, tag, lsgd::launch_tiny_round(a, c->stream));
  c->step += H;
  return LSGD_OK;
}

// The state blob of lsgd_read_state / lsgd_write_state: a header of eight
// 64-bit words, then the sections present for the configuration, each at a
// 256-byte aligned offset, rows of P (or R) contiguous fp32 values.
enum { kSecW = 0, kSecU, kSecRS, kSecWsync, kSecUg, kSecE, kSecCount };
constexpr uint64_t kStateMagic = 0x3154535F4447534CULL;  // "LSGD_ST1"
constexpr size_t kStateHeader = 256;

struct StatePlan {
  int64_t K = 0, P = 0, R = 0;
  uint64_t mask = 0;
  size_t off[kSecCount] = {};
  size_t total = 0;
  uint64_t digest = 0;
};

uint64_t fnv1a(uint64_t h, int64_t v) {
  for (int i = 0; i < 8; ++i) {
    h ^= (uint64_t)((v >> (8 * i)) & 0xff);
    h *= 0x100000001b3ULL;
  }
  return h;
}

StatePlan state_plan(const lsgd_config& cf, const Layout& ly) {
  StatePlan sp;
  sp.K = cf.K;
  sp.P = ly.P;
  sp.R = ly.resnet ? 2LL * ly.rp.rs_half : 0;
  const bool gm = cf.global_momentum != 0.f, sgn = cf.scheme != LSGD_SCHEME_LOCAL;
  const bool present[kSecCount] = {true, true, sp.R > 0, gm || sgn, gm,
                                   cf.scheme == LSGD_SCHEME_EF_SIGN};
  const int64_t floats[kSecCount] = {sp.K * sp.P, sp.K * sp.P, sp.K * sp.R, sp.P, sp.P,
                                     sp.K * sp.P};
  size_t t = kStateHeader;
  for (int i = 0; i < kSecCount; ++i) {
    if (!present[i]) continue;
    sp.mask |= 1ULL << i;
    sp.off[i] = t;
    t = align_up(t + (size_t)floats[i] * 4, kAlign);
  }
  sp.total = t;
  uint64_t h = 0xcbf29ce484222325ULL;
  h = fnv1a(h, cf.model);
  h = fnv1a(h, cf.n_layers);
  for (int i = 0; i <= cf.n_layers; ++i) h = fnv1a(h, cf.widths[i]);
  h = fnv1a(h, sp.K);
  h = fnv1a(h, sp.P);
  h = fnv1a(h, sp.R);
  h = fnv1a(h, (int64_t)sp.mask);
  sp.digest = h;
  return sp;
}

#define LSGD_USABLE(ctx)                                   \
  do {                                                     \
    if (!(ctx)) return LSGD_E_INVALID;                     \
    if ((ctx)->latched != LSGD_OK) return LSGD_E_STATE;    \
  } while (0)

}  // namespace

extern "C" {

lsgd_status lsgd_param_count(const lsgd_config* cfg, int64_t* P) {
  if (!valid_config(cfg) || !P) return LSGD_E_INVALID;
  *P = make_layout(cfg).P;
  return LSGD_OK;
}

lsgd_status lsgd_workspace_bytes(const lsgd_config* cfg, size_t* bytes) {
  if (!valid_config(cfg) || !bytes) return LSGD_E_INVALID;
  *bytes = make_layout(cfg).total;
  return LSGD_OK;
}

lsgd_status lsgd_init_replicas(const lsgd_config* cfg, const float* d_X,
                               const int32_t* d_y, const float* d_w0,
                               void* d_ws, size_t ws_bytes, void* stream,
                               lsgd_ctx** out) {
  if (!out) return LSGD_E_INVALID;
  *out = nullptr;
  if (!valid_config(cfg) || !d_X || !d_y || !d_w0 || !d_ws) return LSGD_E_INVALID;
  if (((uintptr_t)d_ws) % kAlign) return LSGD_E_INVALID;
  Layout ly = make_layout(cfg);
  if (ws_bytes < ly.total) return LSGD_E_WORKSPACE;
  lsgd_ctx* c = new (std::nothrow) lsgd_ctx();
  if (!c) return LSGD_E_INVALID;
  c->cfg = *cfg;
  c->lay = ly;
  c->X = d_X;
  c->y = d_y;
  c->ws = (char*)d_ws;
  c->stream = (hipStream_t)stream;
  const int K = cfg->K;
  lsgd_status st = LSGD_OK;
  auto check = [&](hipError_t e, const char* what) {
    if (st == LSGD_OK && e != hipSuccess) st = c->fail(e, what);
  };
  check(lsgd::launch_fill(c->W(), 0.f, (long long)K * ly.Ps, c->stream), "fill W");
  check(lsgd::launch_fill(c->U(), 0.f, (long long)K * ly.Ps, c->stream), "fill U");
  check(lsgd::launch_broadcast(d_w0, c->W(), c->Wb(), K, ly.P, ly.Ps, -1,
                               c->stream), "broadcast w0");
  if (c->Wsync()) {  // w_(0) is the first synchronised model
    check(lsgd::launch_fill(c->Wsync(), 0.f, ly.Ps, c->stream), "fill w_sync");
    check(lsgd::launch_broadcast(d_w0, c->Wsync(), nullptr, 1, ly.P, ly.Ps, -1,
                                 c->stream), "w_sync := w0");
  }
  if (c->gm())  // the global buffer starts at 0
    check(lsgd::launch_fill(c->Ug(), 0.f, ly.Ps, c->stream), "fill u_global");
  if (c->ef())  // and so do the error memories
    check(lsgd::launch_fill(c->E(), 0.f, (long long)K * ly.Ps, c->stream), "fill e");
  if (c->bf16())
    check(lsgd::launch_to_bf16(d_X, c->Xb(), (long long)cfg->N * cfg->widths[0],
                               c->stream), "dataset to bf16");
  check(lsgd::launch_fill((float*)c->flag(), 0.f, 1, c->stream), "clear the loss flag");
  if (c->RS()) {  // running means 0 and variances 1, in every replica
    const ResPlan& r = ly.rp;
    check(lsgd::launch_fill(c->RS(), 0.f, (long long)K * r.Rs, c->stream), "fill RS");
    check(lsgd::launch_fill(c->RS() + r.rs_half, 1.f, r.rs_half, c->stream),
          "running variances := 1");
    if (K > 1)  // rows 1..K-1 from row 0
      check(lsgd::launch_copy_rows(c->RS() + r.Rs, r.Rs, c->RS(), 0, r.Rs, K - 1,
                                   c->stream), "running statistics to every replica");
  }
  // side streams pay off once there is a hidden layer (an update that can
  // overlap the rest of the backward pass), and for ResNet-20 (its weight
  // gradients overlap the BN backward passes)
  const bool resnet = c->cfg.model == LSGD_MODEL_RESNET20;
  if (st == LSGD_OK && ((ly.head && ly.L >= 2) || resnet)) {
    for (int i = 0; i < 2; ++i) {
      check(hipStreamCreateWithFlags(&c->side[i], hipStreamNonBlocking), "side stream");
      check(hipEventCreateWithFlags(&c->fork[i], hipEventDisableTiming), "fork event");
      check(hipEventCreateWithFlags(&c->join[i], hipEventDisableTiming), "join event");
    }
    if (resnet) check(hipEventCreateWithFlags(&c->done, hipEventDisableTiming), "done event");
    c->use_side = st == LSGD_OK;
  }
  if (st != LSGD_OK) {
    delete c;
    return st;
  }
  *out = c;
  return LSGD_OK;
}

lsgd_status lsgd_local_step(lsgd_ctx* ctx, float lr, float* d_loss) {
  LSGD_USABLE(ctx);
  if (!std::isfinite(lr)) return LSGD_E_INVALID;
  return do_local_step(ctx, lr, d_loss);
}

lsgd_status lsgd_average(lsgd_ctx* ctx) {
  LSGD_USABLE(ctx);
  // global momentum needs the step size, the sign schemes compress: both
  // synchronise through lsgd_synchronise
  if (ctx->gm() || ctx->signed_sync()) return LSGD_E_INVALID;
  return do_average(ctx);
}

lsgd_status lsgd_synchronise(lsgd_ctx* ctx, float lr) {
  LSGD_USABLE(ctx);
  if (!std::isfinite(lr) || (ctx->gm() && lr == 0.f)) return LSGD_E_INVALID;
  return do_synchronise(ctx, lr);
}

lsgd_status lsgd_run_round(lsgd_ctx* ctx, int32_t H, const float* h_lr,
                           float* d_loss) {
  LSGD_USABLE(ctx);
  if (H < 0 || (H > 0 && !h_lr)) return LSGD_E_INVALID;
  for (int h = 0; h < H; ++h)
    if (!std::isfinite(h_lr[h])) return LSGD_E_INVALID;
  if (ctx->gm() && (H == 0 || h_lr[H - 1] == 0.f)) return LSGD_E_INVALID;
  if (tiny_round_ok(ctx, H)) return do_tiny_round(ctx, H, h_lr, d_loss);
  for (int h = 0; h < H; ++h) {
    lsgd_status st = do_local_step(ctx, h_lr[h],
                                   d_loss ? d_loss + (size_t)h * ctx->cfg.K : nullptr);
    if (st != LSGD_OK) return st;
  }
  return do_synchronise(ctx, H > 0 ? h_lr[H - 1] : 0.f);
}

lsgd_status lsgd_average_blocks(lsgd_ctx* ctx, int32_t Kb) {
  LSGD_USABLE(ctx);
  if (Kb < 1 || ctx->cfg.K % Kb) return LSGD_E_INVALID;
  return do_average_blocks(ctx, Kb);
}

lsgd_status lsgd_run_hierarchical_round(lsgd_ctx* ctx, int32_t H, int32_t Hb,
                                        int32_t Kb, const float* h_lr,
                                        float* d_loss) {
  LSGD_USABLE(ctx);
  if (H < 0 || Hb < 1 || Kb < 1 || ctx->cfg.K % Kb) return LSGD_E_INVALID;
  if (ctx->gm() && H == 0) return LSGD_E_INVALID;  // no step size to sync with
  const long long steps = (long long)H * Hb;
  if (steps > 0 && !h_lr) return LSGD_E_INVALID;
  for (long long h = 0; h < steps; ++h)
    if (!std::isfinite(h_lr[h])) return LSGD_E_INVALID;
  for (int b = 0; b < Hb; ++b) {
    for (int h = 0; h < H; ++h) {
      const long long t = (long long)b * H + h;
      lsgd_status st = do_local_step(
          ctx, h_lr[t], d_loss ? d_loss + (size_t)t * ctx->cfg.K : nullptr);
      if (st != LSGD_OK) return st;
    }
    // the last block synchronisation is absorbed by the global one: the
    // mean of equal-sized block means is the global mean
    lsgd_status st = b + 1 < Hb ? do_average_blocks(ctx, Kb)
                                : do_synchronise(ctx, h_lr[steps - 1]);
    if (st != LSGD_OK) return st;
  }
  return LSGD_OK;
}

lsgd_status lsgd_read_params(lsgd_ctx* ctx, int32_t replica, float* d_dst) {
  LSGD_USABLE(ctx);
  if (!d_dst || replica < -1 || replica >= ctx->cfg.K) return LSGD_E_INVALID;
  if (ctx->pending) {  // every replica is the pending mean
    LSGD_CK(ctx, hipMemcpyAsync(d_dst, ctx->Wbar(), ctx->lay.P * sizeof(float),
                                hipMemcpyDeviceToDevice, ctx->stream));
    return LSGD_OK;
  }
  if (replica >= 0) {
    LSGD_CK(ctx, hipMemcpyAsync(d_dst, ctx->W() + (size_t)replica * ctx->lay.Ps,
                                ctx->lay.P * sizeof(float),
                                hipMemcpyDeviceToDevice, ctx->stream));
  } else {
    LSGD_CK(ctx, lsgd::launch_average(ctx->W(), nullptr, ctx->cfg.K, ctx->lay.P,
                                      ctx->lay.Ps, d_dst, ctx->stream));
  }
  return LSGD_OK;
}

lsgd_status lsgd_read_momentum(lsgd_ctx* ctx, int32_t replica, float* d_dst) {
  LSGD_USABLE(ctx);
  if (!d_dst || replica < 0 || replica >= ctx->cfg.K) return LSGD_E_INVALID;
  LSGD_CK(ctx, hipMemcpyAsync(d_dst, ctx->U() + (size_t)replica * ctx->lay.Ps,
                              ctx->lay.P * sizeof(float),
                              hipMemcpyDeviceToDevice, ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_write_params(lsgd_ctx* ctx, int32_t replica,
                              const float* d_src) {
  LSGD_USABLE(ctx);
  if (!d_src || replica < -1 || replica >= ctx->cfg.K) return LSGD_E_INVALID;
  if (replica >= 0) {  // the other replicas keep the pending mean
    if (lsgd_status st = materialise(ctx)) return st;
  }
  ctx->pending = false;
  LSGD_CK(ctx, lsgd::launch_broadcast(d_src, ctx->W(), ctx->Wb(), ctx->cfg.K,
                                      ctx->lay.P, ctx->lay.Ps, replica,
                                      ctx->stream));
  if (replica == -1 && ctx->Wsync())  // the written model is the synchronised one
    LSGD_CK(ctx, lsgd::launch_broadcast(d_src, ctx->Wsync(), nullptr, 1,
                                        ctx->lay.P, ctx->lay.Ps, -1, ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_read_error_memory(lsgd_ctx* ctx, int32_t replica, float* d_dst) {
  LSGD_USABLE(ctx);
  if (!d_dst || !ctx->ef() || replica < 0 || replica >= ctx->cfg.K)
    return LSGD_E_INVALID;
  LSGD_CK(ctx, hipMemcpyAsync(d_dst, ctx->E() + (size_t)replica * ctx->lay.Ps,
                              ctx->lay.P * sizeof(float), hipMemcpyDeviceToDevice,
                              ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_write_error_memory(lsgd_ctx* ctx, int32_t replica,
                                    const float* d_src) {
  LSGD_USABLE(ctx);
  if (!d_src || !ctx->ef() || replica < 0 || replica >= ctx->cfg.K)
    return LSGD_E_INVALID;
  LSGD_CK(ctx, hipMemcpyAsync(ctx->E() + (size_t)replica * ctx->lay.Ps, d_src,
                              ctx->lay.P * sizeof(float), hipMemcpyDeviceToDevice,
                              ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_write_momentum(lsgd_ctx* ctx, int32_t replica,
                                const float* d_src) {
  LSGD_USABLE(ctx);
  if (!d_src || replica < 0 || replica >= ctx->cfg.K) return LSGD_E_INVALID;
  LSGD_CK(ctx, hipMemcpyAsync(ctx->U() + (size_t)replica * ctx->lay.Ps, d_src,
                              ctx->lay.P * sizeof(float), hipMemcpyDeviceToDevice,
                              ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_read_global_momentum(lsgd_ctx* ctx, float* d_dst) {
  LSGD_USABLE(ctx);
  if (!d_dst || !ctx->gm()) return LSGD_E_INVALID;
  LSGD_CK(ctx, hipMemcpyAsync(d_dst, ctx->Ug(), ctx->lay.P * sizeof(float),
                              hipMemcpyDeviceToDevice, ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_write_global_momentum(lsgd_ctx* ctx, const float* d_src) {
  LSGD_USABLE(ctx);
  if (!d_src || !ctx->gm()) return LSGD_E_INVALID;
  LSGD_CK(ctx, hipMemcpyAsync(ctx->Ug(), d_src, ctx->lay.P * sizeof(float),
                              hipMemcpyDeviceToDevice, ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_state_bytes(const lsgd_config* cfg, size_t* bytes) {
  if (!valid_config(cfg) || !bytes) return LSGD_E_INVALID;
  *bytes = state_plan(*cfg, make_layout(cfg)).total;
  return LSGD_OK;
}

lsgd_status lsgd_read_state(lsgd_ctx* ctx, void* d_dst) {
  LSGD_USABLE(ctx);
  if (!d_dst || ((uintptr_t)d_dst) % kAlign) return LSGD_E_INVALID;
  if (lsgd_status st = materialise(ctx)) return st;
  const StatePlan sp = state_plan(ctx->cfg, ctx->lay);
  char* dst = (char*)d_dst;
  lsgd::Words8 h{};
  h.w[0] = kStateMagic;
  h.w[1] = sp.digest;
  h.w[2] = (uint64_t)sp.K;
  h.w[3] = (uint64_t)sp.P;
  h.w[4] = (uint64_t)sp.R;
  h.w[5] = (uint64_t)ctx->step;
  h.w[6] = sp.mask;
  h.w[7] = (uint64_t)sp.total;
  const hipStream_t s = ctx->stream;
  const long long P = sp.P, Ps = ctx->lay.Ps;
  LSGD_CK(ctx, lsgd::launch_put_words(dst, h, s));
  // the rest of the header and the alignment gaps are zeros, so that equal
  // states give equal blobs
  LSGD_CK(ctx, lsgd::launch_fill((float*)(dst + 64), 0.f, (kStateHeader - 64) / 4, s));
  const int64_t nfl[kSecCount] = {sp.K * P, sp.K * P, sp.K * sp.R, P, P, sp.K * P};
  for (int i = 0; i < kSecCount; ++i) {
    if (!(sp.mask >> i & 1)) continue;
    size_t next = sp.total;
    for (int j = i + 1; j < kSecCount; ++j)
      if (sp.mask >> j & 1) {
        next = sp.off[j];
        break;
      }
    const size_t end = sp.off[i] + (size_t)nfl[i] * 4;
    if (next > end) LSGD_CK(ctx, lsgd::launch_fill((float*)(dst + end), 0.f, (next - end) / 4, s));
  }
  auto rows = [&](int sec, const float* src, long long n, long long pitch, int k) {
    return lsgd::launch_copy_rows((float*)(dst + sp.off[sec]), n, src, pitch, n, k, s);
  };
  LSGD_CK(ctx, rows(kSecW, ctx->W(), P, Ps, sp.K));
  LSGD_CK(ctx, rows(kSecU, ctx->U(), P, Ps, sp.K));
  if (sp.mask & (1u << kSecRS)) LSGD_CK(ctx, rows(kSecRS, ctx->RS(), sp.R, ctx->lay.rp.Rs, sp.K));
  if (sp.mask & (1u << kSecWsync)) LSGD_CK(ctx, rows(kSecWsync, ctx->Wsync(), P, Ps, 1));
  if (sp.mask & (1u << kSecUg)) LSGD_CK(ctx, rows(kSecUg, ctx->Ug(), P, Ps, 1));
  if (sp.mask & (1u << kSecE)) LSGD_CK(ctx, rows(kSecE, ctx->E(), P, Ps, sp.K));
  return LSGD_OK;
}

lsgd_status lsgd_write_state(lsgd_ctx* ctx, const void* d_src) {
  LSGD_USABLE(ctx);
  if (!d_src || ((uintptr_t)d_src) % kAlign) return LSGD_E_INVALID;
  const StatePlan sp = state_plan(ctx->cfg, ctx->lay);
  const hipStream_t s = ctx->stream;
  // the header decides whether the blob fits this context: read it first
  uint64_t h[8] = {};
  LSGD_CK(ctx, hipMemcpyAsync(h, d_src, sizeof h, hipMemcpyDeviceToHost, s));
  LSGD_CK(ctx, hipStreamSynchronize(s));
  if (h[0] != kStateMagic || h[1] != sp.digest || h[2] != (uint64_t)sp.K ||
      h[3] != (uint64_t)sp.P || h[4] != (uint64_t)sp.R || h[6] != sp.mask ||
      h[7] != (uint64_t)sp.total || (int64_t)h[5] < 0)
    return LSGD_E_INVALID;
  const char* src = (const char*)d_src;
  const long long P = sp.P, Ps = ctx->lay.Ps;
  auto sec = [&](int i) { return (const float*)(src + sp.off[i]); };
  // replicas through the broadcast kernel, which also refreshes the bf16 copy
  for (int k = 0; k < sp.K; ++k)
    LSGD_CK(ctx, lsgd::launch_broadcast(sec(kSecW) + (size_t)k * P, ctx->W(), ctx->Wb(),
                                        (int)sp.K, P, Ps, k, s));
  LSGD_CK(ctx, lsgd::launch_copy_rows(ctx->U(), Ps, sec(kSecU), P, P, (int)sp.K, s));
  if (sp.mask & (1u << kSecRS))
    LSGD_CK(ctx, lsgd::launch_copy_rows(ctx->RS(), ctx->lay.rp.Rs, sec(kSecRS), sp.R, sp.R,
                                        (int)sp.K, s));
  if (sp.mask & (1u << kSecWsync))
    LSGD_CK(ctx, lsgd::launch_copy_rows(ctx->Wsync(), Ps, sec(kSecWsync), P, P, 1, s));
  if (sp.mask & (1u << kSecUg))
    LSGD_CK(ctx, lsgd::launch_copy_rows(ctx->Ug(), Ps, sec(kSecUg), P, P, 1, s));
  if (sp.mask & (1u << kSecE))
    LSGD_CK(ctx, lsgd::launch_copy_rows(ctx->E(), Ps, sec(kSecE), P, P, (int)sp.K, s));
  // a restored state starts without a non-finite loss on record
  LSGD_CK(ctx, lsgd::launch_fill((float*)ctx->flag(), 0.f, 1, s));
  ctx->step = (int64_t)h[5];
  ctx->presampled = -1;
  ctx->pending = false;
  return LSGD_OK;
}

lsgd_status lsgd_set_lazy_average(lsgd_ctx* ctx, int32_t enable) {
  LSGD_USABLE(ctx);
  if (enable != 0 && enable != 1) return LSGD_E_INVALID;
  const lsgd_config& cf = ctx->cfg;
  if (enable && (ctx->lay.resnet || cf.scheme != LSGD_SCHEME_LOCAL ||
                 cf.global_momentum != 0.f))
    return LSGD_E_UNSUPPORTED;
  if (!enable)
    if (lsgd_status st = materialise(ctx)) return st;
  ctx->lazy = enable != 0;
  return LSGD_OK;
}

lsgd_status lsgd_get_step(lsgd_ctx* ctx, int64_t* step) {
  if (!ctx || !step) return LSGD_E_INVALID;
  *step = ctx->step;
  return LSGD_OK;
}

lsgd_status lsgd_set_step(lsgd_ctx* ctx, int64_t step) {
  LSGD_USABLE(ctx);
  if (step < 0) return LSGD_E_INVALID;
  ctx->step = step;
  ctx->presampled = -1;
  return LSGD_OK;
}

lsgd_status lsgd_sample_indices(lsgd_ctx* ctx, int64_t step, int32_t* d_idx) {
  LSGD_USABLE(ctx);
  if (!d_idx || step < 0) return LSGD_E_INVALID;
  LSGD_CK(ctx, sample(ctx, step, d_idx, ctx->stream));
  return LSGD_OK;
}

lsgd_status lsgd_sync(lsgd_ctx* ctx) {
  LSGD_USABLE(ctx);
  LSGD_CK(ctx, hipStreamSynchronize(ctx->stream));
  int flag = 0;
  LSGD_CK(ctx, hipMemcpy(&flag, ctx->flag(), sizeof flag, hipMemcpyDeviceToHost));
  return flag ? LSGD_E_NONFINITE : LSGD_OK;
}

lsgd_status lsgd_destroy(lsgd_ctx* ctx) {
  if (!ctx) return LSGD_E_INVALID;
  delete ctx;
  return LSGD_OK;
}

const char* lsgd_status_string(lsgd_status s) {
  switch (s) {
    case LSGD_OK: return "ok";
    case LSGD_E_INVALID: return "invalid argument";
    case LSGD_E_WORKSPACE: return "workspace too small";
    case LSGD_E_HIP: return "HIP runtime error";
    case LSGD_E_NONFINITE: return "non-finite loss";
    case LSGD_E_STATE: return "context unusable after an earlier HIP error";
    case LSGD_E_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

lsgd_status lsgd_profile_enable(lsgd_ctx* ctx, int32_t enable) {
  LSGD_USABLE(ctx);
  if (enable != 0 && enable != 1) return LSGD_E_INVALID;
  ctx->prof.on = enable != 0;
  return LSGD_OK;
}

lsgd_status lsgd_profile_select(lsgd_ctx* ctx, const char* tag, int32_t every) {
  LSGD_USABLE(ctx);
  if ((tag && std::strlen(tag) > 64) || every < 1) return LSGD_E_INVALID;
  ctx->prof.only = tag ? tag : "";
  ctx->prof.every = every;
  ctx->prof.seen = 0;
  return LSGD_OK;
}

lsgd_status lsgd_profile_report(lsgd_ctx* ctx, char* h_buf, size_t len) {
  LSGD_USABLE(ctx);
  if (!h_buf || len == 0) return LSGD_E_INVALID;
  LSGD_CK(ctx, hipStreamSynchronize(ctx->stream));
  std::vector<std::string> tags;
  std::vector<double> ms;
  std::vector<long long> n;
  for (const auto& r : ctx->prof.recs) {
    float t = 0.f;
    LSGD_CK(ctx, hipEventElapsedTime(&t, r.a, r.b));
    size_t i = 0;
    while (i < tags.size() && tags[i] != r.tag) ++i;
    if (i == tags.size()) {
      tags.push_back(r.tag);
      ms.push_back(0.0);
      n.push_back(0);
    }
    ms[i] += t;
    n[i] += 1;
  }
  std::string out;
  for (size_t i = 0; i < tags.size(); ++i) {
    char line[160];
    std::snprintf(line, sizeof line, "%s %lld %.6f\n", tags[i].c_str(), n[i], ms[i]);
    out += line;
  }
  ctx->prof.recs.clear();
  ctx->prof.used = 0;
  if (out.size() + 1 > len) return LSGD_E_INVALID;
  std::memcpy(h_buf, out.c_str(), out.size() + 1);
  return LSGD_OK;
}

const char* lsgd_last_error(const lsgd_ctx* ctx) {
  return ctx ? ctx->err.c_str() : "";
}

lsgd_status lsgd_grouped_gemm(int32_t dtype, int32_t trans_a, int32_t trans_b,
                              int32_t G, int32_t M, int32_t N, int32_t Kd,
                              const void* d_A, int64_t lda, int64_t sA,
                              const void* d_B, int64_t ldb, int64_t sB,
                              float* d_C, int32_t splits, float* d_part,
                              void* stream) {
  if (splits < 1 || splits > 8 || splits == 5 || splits == 6 || splits == 7 ||
      (splits > 1 && !d_part))
    return LSGD_E_INVALID;
  if ((dtype != LSGD_FP32 && dtype != LSGD_BF16) || (trans_a | trans_b) & ~1)
    return LSGD_E_INVALID;
  if (G < 1 || M < 1 || N < 1 || Kd < 1 || G > 65535) return LSGD_E_INVALID;
  if (!d_A || !d_B || !d_C || sA < 0 || sB < 0) return LSGD_E_INVALID;
  if (lda < (trans_a ? M : Kd) || ldb < (trans_b ? Kd : N)) return LSGD_E_INVALID;
  GemmArgs a{};
  a.G = G;
  a.M = M;
  a.N = N;
  a.Kd = Kd;
  a.A = d_A;
  a.lda = lda;
  a.sA = sA;
  a.B = d_B;
  a.ldb = ldb;
  a.sB = sB;
  a.C = d_C;
  a.ldc = N;
  a.sC = (long long)M * N;
  a.splits = splits;
  a.part = d_part;
  hipError_t e = lsgd::launch_gemm(dtype, trans_a, trans_b, lsgd::EPI_STORE, 0, a,
                                   (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : LSGD_E_HIP;
}

lsgd_status lsgd_replica_average(float* d_W, int32_t K, int64_t P, void* stream) {
  if (!d_W || K < 1 || P < 0) return LSGD_E_INVALID;
  hipError_t e = lsgd::launch_average(d_W, nullptr, K, P, P, nullptr,
                                      (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : LSGD_E_HIP;
}

lsgd_status lsgd_replica_average_blocks(float* d_W, int32_t K, int32_t Kb,
                                       int64_t P, void* stream) {
  if (!d_W || K < 1 || Kb < 1 || K % Kb || P < 0) return LSGD_E_INVALID;
  hipError_t e = lsgd::launch_average_blocks(d_W, nullptr, Kb, K / Kb, P, P,
                                             nullptr, (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : LSGD_E_HIP;
}

lsgd_status lsgd_replica_average_global_momentum(float* d_W, int32_t K,
                                                 int64_t P, float* d_wsync,
                                                 float* d_ug, float m_global,
                                                 float lr, void* stream) {
  if (!d_W || !d_wsync || !d_ug || K < 1 || P < 0 || !std::isfinite(m_global) ||
      m_global < 0.f || m_global >= 1.f || !std::isfinite(lr) || lr == 0.f)
    return LSGD_E_INVALID;
  hipError_t e = lsgd::launch_average_gm(d_W, nullptr, K, P, P, d_wsync, d_ug,
                                         m_global, lr, (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : LSGD_E_HIP;
}

lsgd_status lsgd_sign_sync_scratch_bytes(int32_t K, int64_t P, size_t* bytes) {
  if (!bytes || K < 1 || P < 0 || P % 4) return LSGD_E_INVALID;
  *bytes = lsgd::sign_sync_scratch_bytes(K, P);
  return LSGD_OK;
}

lsgd_status lsgd_replica_sign_sync(float* d_W, int32_t K, int64_t P,
                                   float* d_wsync, float* d_E, void* d_scratch,
                                   size_t scratch_bytes, void* stream) {
  if (!d_W || !d_wsync || !d_scratch || K < 1 || P < 0 || P % 4)
    return LSGD_E_INVALID;
  if (scratch_bytes < lsgd::sign_sync_scratch_bytes(K, P)) return LSGD_E_WORKSPACE;
  hipError_t e = lsgd::launch_sign_sync(d_W, nullptr, d_E, d_wsync, K, P, P,
                                        d_scratch, scratch_bytes,
                                        (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : (e == hipErrorInvalidValue ? LSGD_E_INVALID
                                                                : LSGD_E_HIP);
}

lsgd_status lsgd_replica_sign_sync_static(float* d_W, int32_t K, int64_t P,
                                          float* d_wsync, float* d_E, void* stream) {
  static_assert(LSGD_SIGN_SYNC_STATIC_BYTES == lsgd::kSignSyncStaticBytes,
                "the header states the static scratch size");
  if (!d_W || !d_wsync || K < 1 || P < 0 || P % 4) return LSGD_E_INVALID;
  if (lsgd::sign_sync_scratch_bytes(K, P) > lsgd::kSignSyncStaticBytes)
    return LSGD_E_WORKSPACE;
  hipError_t e = lsgd::launch_sign_sync_static(d_W, d_E, d_wsync, K, P, (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : (e == hipErrorInvalidValue ? LSGD_E_INVALID
                                                                : LSGD_E_HIP);
}

lsgd_status lsgd_sgd_update(float* d_W, float* d_U, const float* d_G, int64_t n,
                            float lr, float momentum, float weight_decay,
                            int32_t nesterov, void* stream) {
  if (!d_W || !d_U || !d_G || n < 0 || (nesterov & ~3)) return LSGD_E_INVALID;
  hipError_t e = lsgd::launch_sgd_update(d_W, d_U, d_G, n, lr, momentum,
                                         weight_decay, nesterov,
                                         (hipStream_t)stream);
  return e == hipSuccess ? LSGD_OK : LSGD_E_HIP;
}

}  // extern "C"
