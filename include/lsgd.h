/*
 * lsgd.h -- C ABI of the MI355X (gfx950) local-SGD hot path.
 *
 * Method: local SGD and post-local SGD of Lin, Stich, Patel, Jaggi, "Don't Use
 * Large Mini-Batches, Use Local SGD" (ICLR 2020). K workers each run H
 * sequential mini-batch SGD steps of batch B_loc on their own model copy, then
 * the K models are replaced by their mean (eq. 2; Algorithm 1). Post-local SGD
 * runs rounds with H = 1 first (eq. "post-local SGD", Algorithm 2); that
 * schedule is a sequence of run_round calls.
 *
 * On one GPU the K workers are K model replicas resident in device memory.
 *
 * Conventions for every call:
 *  - Pointers prefixed d_ are device pointers, h_ host pointers. The caller owns
 *    all memory; the library never allocates device memory. Device buffers
 *    handed to lsgd_init_replicas (dataset, labels, workspace) must stay alive
 *    and unmodified by the caller until lsgd_destroy.
 *  - Work is enqueued asynchronously on the stream given at init (a
 *    hipStream_t passed as void*, NULL = the null stream). Results are valid
 *    once that stream has been synchronised (lsgd_sync does it). Inside a
 *    local step, weight updates that feed nothing else in the step may run on
 *    two internal streams of default priority; they are joined back into the
 *    given stream before the step's last command, so stream order on the
 *    given stream still covers all of the step's work.
 *  - Every call returns a status. Argument errors return LSGD_E_INVALID and
 *    change nothing. A failed HIP call returns LSGD_E_HIP and latches: from
 *    then on every call on that context returns LSGD_E_STATE until destroy.
 *  - One context must not be used from two host threads at once. Distinct
 *    contexts are independent.
 *  - Failure detection: every local step checks on the device, with no host
 *    synchronisation, that each replica's mean mini-batch loss is finite; a
 *    non-finite one sets a flag in the workspace that lsgd_sync reports as
 *    LSGD_E_NONFINITE. The flag stays set (the context remains usable)
 *    until lsgd_write_state restores a state or the context is destroyed.
 *    A loss is taken at the pre-update weights, so a step whose update makes
 *    a parameter non-finite shows up at the next step's loss; a non-finite
 *    hidden pre-activation that a ReLU maps to 0 does not reach it.
 *
 * Flat parameter layout of one replica ([P] fp32): for each layer l = 1..L in
 * order, W_l row-major [d_{l-1}][d_l] (element (i, j) maps input i to output
 * j), then the bias b_l [d_l].
 */
#ifndef LSGD_H
#define LSGD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lsgd_ctx lsgd_ctx; /* opaque, host-side */

typedef enum lsgd_status {
  LSGD_OK = 0,
  LSGD_E_INVALID = 1,     /* bad argument; no state was changed */
  LSGD_E_WORKSPACE = 2,   /* workspace smaller than lsgd_workspace_bytes */
  LSGD_E_HIP = 3,         /* a HIP runtime call or launch failed (latched) */
  LSGD_E_STATE = 4,       /* context unusable after an earlier HIP error */
  LSGD_E_UNSUPPORTED = 5, /* valid request the library does not implement */
  LSGD_E_NONFINITE = 6    /* a local step's loss was not finite (sticky; see
                             lsgd_sync) */
} lsgd_status;

/* LSGD_MODEL_MLP: ReLU MLP with widths d_0 .. d_L (L = 1 is softmax
 * regression). LSGD_MODEL_RESNET20: the CIFAR ResNet-20 of the paper's Table 5
 * on 32x32x3 NHWC images (widths[0] = 3072, widths[1] = classes <= 32,
 * n_layers = 1, fp32, B_loc < 131072): a 3x3 stem convolution to 16 channels, three stages of
 * three basic blocks at 16/32/64 channels (stride 2 entering stages 2 and 3,
 * option-A shortcuts: subsample and zero-pad channels), batch normalisation
 * with per-replica batch statistics after every convolution (no weight decay
 * on its scale and shift), global average pooling and a 64 -> classes
 * classifier. Parameter layout: per convolution in order its weight
 * [3][3][c_in][c_out], BN scale [c_out], BN shift [c_out]; then the
 * classifier weight [64][classes] and bias [classes]. Each replica also keeps
 * BN running statistics (they do not enter the training loss): R = 1376
 * values, the running means of the 19 BN layers in convolution order, then
 * their running variances; they start at 0 and 1, follow every local step as
 * r = 0.9 r + 0.1 s (s the batch mean, or the unbiased batch variance
 * var * n / (n - 1) over the n values per channel), and take the plain mean
 * over the replicas at every synchronisation (over the block at a block
 * synchronisation), whatever the scheme. They are read and written through
 * the state blob. */
enum { LSGD_MODEL_MLP = 0, LSGD_MODEL_RESNET20 = 1 };
enum { LSGD_FP32 = 0, LSGD_BF16 = 1 };
/* Local-step / synchronisation scheme (the appendix on compression):
 * LSGD_SCHEME_LOCAL   plain local steps, plain mean (eq. 2);
 * LSGD_SCHEME_SIGN    Algorithm 3: local steps move by sign(d) (d the update
 *                     direction after weight decay and momentum, sign(0) =
 *                     0); the synchronisation sends each worker's model
 *                     difference Delta^k = w_s - w^k as sign(Delta^k) *
 *                     ||Delta^k||_1 / P and sets every replica to
 *                     w_s - (1/K) sum_k of those messages;
 * LSGD_SCHEME_EF_SIGN Algorithm 4: plain local steps; the synchronisation
 *                     compresses Delta^k + e^k the same way and keeps the
 *                     error memory e^k = Delta^k + e^k - message (e^k = 0 at
 *                     init, per worker, never averaged).
 * w_s is the model of the previous synchronisation (w0 at init). */
enum { LSGD_SCHEME_LOCAL = 0, LSGD_SCHEME_SIGN = 1, LSGD_SCHEME_EF_SIGN = 2 };
/* Index sampler. With n_k = floor((k+1)N/K) - floor(kN/K) rows in worker
 * k's slice [floor(kN/K), floor((k+1)N/K)):
 * LSGD_SAMPLER_IID    every local step draws B_loc rows i.i.d. with
 *                     replacement from the worker's fixed slice (eq. 1's
 *                     sampling from the local data): Philox4x32-10, key
 *                     (seed lo, seed hi), counter (j / 4, s lo, k, s hi),
 *                     slot j takes word j mod 4, u -> lo + floor(u n_k / 2^32);
 * LSGD_SAMPLER_EPOCH  the data is repartitioned by a fresh global permutation
 *                     every epoch (the CIFAR training procedure): with
 *                     S = floor(floor(N / K) / B_loc) batches per epoch
 *                     (must be >= 1), step s is batch j = s mod S of epoch
 *                     e = s / S and takes rows pi_e(lo_k + j B_loc + b),
 *                     b < B_loc. pi_e is a 4-round balanced Feistel network on
 *                     2m-bit words (m the smallest >= 1 with 4^m >= N; left
 *                     half the high m bits; round r maps (L, R) to
 *                     (R, L xor (F_r(R) & (2^m - 1)))), F_r(R) word 0 of
 *                     Philox4x32-10 at counter (R, r, e, 0x5348464C) with the
 *                     same key, restricted to [0, N) by cycle walking. */
enum { LSGD_SAMPLER_IID = 0, LSGD_SAMPLER_EPOCH = 1 };
#define LSGD_MAX_LAYERS 8

/*
 * Problem statement, after the REQUIRE list of Algorithms 1 and 2: model,
 * mini-batch size per worker, number of workers, momentum, plus the sampler
 * key. The step size and H are per call (run_round), so schedules such as
 * post-local SGD stay on the host.
 */
typedef struct lsgd_config {
  int32_t model;                          /* LSGD_MODEL_MLP / _RESNET20 */
  int32_t n_layers;                       /* L, 1..LSGD_MAX_LAYERS */
  int32_t widths[LSGD_MAX_LAYERS + 1];    /* d_0 (features) .. d_L (classes) */
  int32_t K;                              /* workers = replicas, >= 1 */
  int32_t B_loc;                          /* local mini-batch, >= 1 */
  int32_t gemm_dtype;                     /* LSGD_FP32 or LSGD_BF16 */
  int32_t nesterov;                       /* 0 heavy ball, 1 Nesterov */
  float momentum;                         /* m in [0, 1) */
  float weight_decay;                     /* coupled L2 on weights and biases */
  float global_momentum;                  /* m_g in [0, 1) at the global
                                             synchronisation; 0: plain mean */
  int32_t scheme;                         /* LSGD_SCHEME_*; a sign scheme
                                             needs global_momentum == 0 */
  int32_t sampler;                        /* LSGD_SAMPLER_* */
  uint64_t seed;                          /* Philox4x32-10 key for sampling */
  int64_t N;                              /* dataset rows, >= K */
} lsgd_config;

/* Number of parameters P of one replica. */
lsgd_status lsgd_param_count(const lsgd_config* cfg, int64_t* P);

/* Bytes of device workspace lsgd_init_replicas needs (replicas, momentum
 * buffers, activations, indices, and for bf16 the operand copies). */
lsgd_status lsgd_workspace_bytes(const lsgd_config* cfg, size_t* bytes);

/*
 * Create a context and synchronise all replicas to w0 (first line of
 * Algorithm 1: w^k_(0) := w_(0)); momentum buffers are zeroed and the local
 * step counter s is set to 0.
 *  d_X   fp32 [N][d_0] row-major dataset, d_y int32 [N] labels in [0, d_L).
 *  d_w0  fp32 [P], copied (stream-ordered); may be freed after the stream
 *        has passed this call.
 *  d_ws  workspace of ws_bytes >= lsgd_workspace_bytes, 256-byte aligned.
 * For LSGD_BF16 the dataset is converted once to a bf16 copy in the
 * workspace (round to nearest even).
 */
lsgd_status lsgd_init_replicas(const lsgd_config* cfg, const float* d_X,
                               const int32_t* d_y, const float* d_w0,
                               void* d_ws, size_t ws_bytes, void* stream,
                               lsgd_ctx** out);

/*
 * One local step on every replica (inner loop of Algorithm 1, local update
 * of eq. 2 with per-replica momentum): sample B_loc indices per worker from
 * its shard, forward, softmax cross-entropy, backward, and
 *   g = grad + wd * w;  u = m u + g;  d = nesterov ? g + m u : u;
 *   w = w - lr * d.
 * d_loss: fp32 [K] receives each replica's mean mini-batch loss at the
 * pre-update weights, or NULL. Increments s.
 */
lsgd_status lsgd_local_step(lsgd_ctx* ctx, float lr, float* d_loss);

/* Synchronisation of eq. 2: every replica becomes (1/K) sum_k w^k, summed in
 * a fixed pairwise tree over k. Momentum buffers are left as they are.
 * LSGD_E_INVALID when the configuration sets a global momentum factor or a
 * sign scheme (those synchronise through lsgd_synchronise). */
lsgd_status lsgd_average(lsgd_ctx* ctx);

/*
 * The form of the plain average (lsgd_average, and the synchronisation of
 * lsgd_run_round without global momentum or a sign scheme). enable = 0 (the
 * default): the mean is written back into all K replicas (K P floats read
 * and K P written). enable = 1, the lazy form that eq. 2 allows since every
 * replica holds the same w after it: the mean is written once (P floats,
 * plus its bf16 copy for LSGD_BF16); the next local step reads that copy as
 * every replica's weights and writes each replica's stepped model. Results
 * are bit for bit those of the default form: every call that reads the
 * replicas (read_params, read_state, block averages, the single-launch
 * softmax round, write_params of one replica) first writes the pending mean
 * into them. MLP models under LSGD_SCHEME_LOCAL without global momentum
 * only, else LSGD_E_UNSUPPORTED; enable outside {0, 1}: LSGD_E_INVALID.
 * Switching it off writes a pending mean out.
 */
lsgd_status lsgd_set_lazy_average(lsgd_ctx* ctx, int32_t enable);

/*
 * The end-of-round synchronisation. With a sign scheme it is the
 * sign-compressed synchronisation of Algorithm 3 or 4 (lr unused; see
 * LSGD_SCHEME_*). With global_momentum == 0 it is lsgd_average (lr unused). Otherwise it is local SGD with global momentum
 * (the momentum appendix's paragraph on global momentum; with local
 * momentum also on, its hybrid scheme): with w_s the model of the previous
 * synchronisation (w0 at init) and u the global buffer (0 at init),
 *   mean = (1/K) sum_k w^k  (the tree of lsgd_average),
 *   u = m_g u + (w_s - mean) / lr,   w_s = w_s - lr u,   every w^k := w_s.
 * The paper's (1/K) sum_k (w_s - w^k) is computed as w_s - mean. lr is the
 * step size of the round's local steps; lr must be finite, and non-zero
 * when m_g != 0, else LSGD_E_INVALID.
 */
lsgd_status lsgd_synchronise(lsgd_ctx* ctx, float lr);

/* H local steps with step sizes h_lr[0..H-1] (host array), then
 * lsgd_synchronise(ctx, h_lr[H-1]) (lsgd_average without global momentum).
 * d_loss: fp32 [H][K] or NULL. With global momentum, H == 0 or a zero last
 * step size is LSGD_E_INVALID.
 * A one-layer fp32 model (softmax regression) under the plain local scheme
 * without global momentum, with 1 <= H <= 64, at most 32 classes and all
 * replicas and buffers within one workgroup's LDS, runs the whole round as a
 * single launch. Its products sum in a different fixed order than the
 * step-by-step path, so the two agree to fp32 rounding, not bit for bit;
 * each is deterministic. */
lsgd_status lsgd_run_round(lsgd_ctx* ctx, int32_t H, const float* h_lr,
                           float* d_loss);

/*
 * Block synchronisation of hierarchical local SGD (Appendix D, the
 * hierarchical local SGD equation; the inner all-reduce of Algorithm 5):
 * replicas 0..K-1 form K/Kb blocks of Kb consecutive replicas and each
 * replica becomes the mean of its block, summed in the same fixed tree as
 * lsgd_average (within the block). Momentum buffers are left as they are.
 * Kb must divide K, else LSGD_E_INVALID; Kb == K is lsgd_average (bit for
 * bit), Kb == 1 changes nothing.
 */
lsgd_status lsgd_average_blocks(lsgd_ctx* ctx, int32_t Kb);

/*
 * One outer round of hierarchical local SGD (Algorithm 5): Hb times, run H
 * local steps then the block synchronisation over blocks of Kb replicas;
 * the last block synchronisation is replaced by the global synchronisation
 * (lsgd_synchronise with the last step size; lsgd_average without global
 * momentum), which the plain block mean would not change in exact
 * arithmetic. h_lr: host
 * array of H * Hb step sizes in step order. d_loss: fp32 [Hb * H][K] or
 * NULL. Kb must divide K; H >= 0, Hb >= 1, else LSGD_E_INVALID. Hb == 1 is
 * lsgd_run_round; Kb == K runs Hb plain rounds of period H.
 */
lsgd_status lsgd_run_hierarchical_round(lsgd_ctx* ctx, int32_t H, int32_t Hb,
                                        int32_t Kb, const float* h_lr,
                                        float* d_loss);

/* Copy replica `replica`'s parameters (or, for replica == -1, their mean by
 * the same tree as lsgd_average, without changing state) to d_dst fp32 [P]. */
lsgd_status lsgd_read_params(lsgd_ctx* ctx, int32_t replica, float* d_dst);

/* Copy replica `replica`'s momentum buffer to d_dst fp32 [P] / overwrite it
 * from d_src fp32 [P] (checkpoint and resume). replica outside [0, K):
 * LSGD_E_INVALID. */
lsgd_status lsgd_read_momentum(lsgd_ctx* ctx, int32_t replica, float* d_dst);
lsgd_status lsgd_write_momentum(lsgd_ctx* ctx, int32_t replica,
                                const float* d_src);

/* Copy the global momentum buffer u to d_dst fp32 [P] / overwrite it from
 * d_src fp32 [P] (checkpoint and resume; the synchronised model w_s is set
 * by lsgd_write_params with replica == -1). LSGD_E_INVALID without global
 * momentum. */
lsgd_status lsgd_read_global_momentum(lsgd_ctx* ctx, float* d_dst);
lsgd_status lsgd_write_global_momentum(lsgd_ctx* ctx, const float* d_src);

/* Copy replica `replica`'s error memory e^k (LSGD_SCHEME_EF_SIGN) to d_dst
 * fp32 [P] / overwrite it from d_src fp32 [P]. LSGD_E_INVALID for other
 * schemes or a replica outside [0, K). */
lsgd_status lsgd_read_error_memory(lsgd_ctx* ctx, int32_t replica, float* d_dst);
lsgd_status lsgd_write_error_memory(lsgd_ctx* ctx, int32_t replica,
                                    const float* d_src);

/* Overwrite replica `replica` (or all replicas for -1) with d_src fp32 [P]
 * (and the bf16 operand copy). For checkpoint restore and tests. With global
 * momentum, replica == -1 also sets the synchronised model w_s. */
lsgd_status lsgd_write_params(lsgd_ctx* ctx, int32_t replica,
                              const float* d_src);

/* Local step counter s (the sampler counter of the next local step). */
lsgd_status lsgd_get_step(lsgd_ctx* ctx, int64_t* step);
lsgd_status lsgd_set_step(lsgd_ctx* ctx, int64_t step);

/* The indices the configured sampler (LSGD_SAMPLER_*) draws at local step
 * `step`: int32 [K][B_loc] into d_idx. */
lsgd_status lsgd_sample_indices(lsgd_ctx* ctx, int64_t step, int32_t* d_idx);

/* Synchronise the context's stream; returns the latched status, else
 * LSGD_E_NONFINITE when a local step since init (or the last
 * lsgd_write_state) had a non-finite loss, else LSGD_OK. */
lsgd_status lsgd_sync(lsgd_ctx* ctx);

/*
 * Checkpoint and resume: the whole training state of a context as one
 * device blob -- what the paper's post-local runs restart from (they switch
 * to local SGD from a mini-batch SGD checkpoint). Layout (all little-endian):
 *   bytes 0..255: header, eight uint64 words: magic 0x3154535F4447534C
 *     ("LSGD_ST1"), a digest of the layout (model, widths, K, P, R and the
 *     section mask, FNV-1a), K, P, R (BN running statistics per replica; 0
 *     for the MLP), the local step counter s, the section mask, the blob's
 *     total bytes; the rest of the 256 bytes is unused;
 *   then, each at the next 256-byte aligned offset and present when its mask
 *   bit is set: bit 0 the replicas fp32 [K][P], bit 1 the momentum buffers
 *   [K][P] (always present), bit 2 the BN running statistics [K][R]
 *   (ResNet-20), bit 3 the synchronised model w_s [P] (global momentum and
 *   the sign schemes), bit 4 the global momentum buffer [P] (global
 *   momentum), bit 5 the error memories [K][P] (LSGD_SCHEME_EF_SIGN).
 * lsgd_state_bytes gives the size for a configuration (no device needed).
 * lsgd_read_state writes the blob to d_dst (stream-ordered, no host sync).
 * lsgd_write_state restores it from d_src: it synchronises the stream to
 * read the header, returns LSGD_E_INVALID without changing anything unless
 * the header matches this context's configuration (magic, digest, K, P, R,
 * mask, size), then overwrites every section (and the bf16 operand copy),
 * sets s and clears the non-finite flag. d_dst / d_src: caller-owned device
 * memory of lsgd_state_bytes bytes, 256-byte aligned, else LSGD_E_INVALID.
 * A context resumed from a blob continues bit for bit as the one that wrote
 * it (same configuration, dataset and step sizes).
 */
lsgd_status lsgd_state_bytes(const lsgd_config* cfg, size_t* bytes);
lsgd_status lsgd_read_state(lsgd_ctx* ctx, void* d_dst);
lsgd_status lsgd_write_state(lsgd_ctx* ctx, const void* d_src);

/* Release the host context (device memory stays with the caller). */
lsgd_status lsgd_destroy(lsgd_ctx* ctx);

/* Static description of a status; never NULL. */
const char* lsgd_status_string(lsgd_status s);

/* Text of the last error recorded on ctx ("" if none); never NULL. */
const char* lsgd_last_error(const lsgd_ctx* ctx);

/* Per-launch timing (a measurement aid, off by default): while enabled,
 * every kernel the context launches is bracketed by two HIP events on its
 * stream, tagged by launch site (sample, fwd<l>, xent, dgrad<l>,
 * wgrad_update<l>, average; a split-K GEMM's tag covers both of its
 * kernels). */
lsgd_status lsgd_profile_enable(lsgd_ctx* ctx, int32_t enable);

/* Restrict the bracketing to launches tagged `tag` (host string, at most 64
 * characters, copied; NULL or "" selects every launch again), and of those
 * to the 1st, (every+1)-th, (2 every+1)-th ... counted from this call, so
 * that one kernel can be timed inside a run at a sampling rate that leaves
 * the run's own speed nearly undisturbed (each bracket costs some
 * microseconds of stream time). LSGD_E_INVALID for a longer tag or
 * every < 1. */
lsgd_status lsgd_profile_select(lsgd_ctx* ctx, const char* tag, int32_t every);

/* Synchronise, then write one line "tag launches total_ms" per tag into the
 * host buffer h_buf (NUL-terminated; LSGD_E_INVALID if len is too small) and
 * clear the records. */
lsgd_status lsgd_profile_report(lsgd_ctx* ctx, char* h_buf, size_t len);

/*
 * Building blocks, exposed for kernel-level tests and bandwidth sweeps.
 */

/* Grouped GEMM over G independent problems (the per-replica layer
 * contractions of the gradient in eq. 2):
 *   C_g[M][N] = opA(A_g)[M][Kd] * opB(B_g)[Kd][N]   (fp32 accumulation)
 * trans_a = 0: A_g is [M][Kd] row-major with leading dimension lda;
 *         = 1: A_g is [Kd][M] row-major (lda >= M).
 * trans_b = 0: B_g is [Kd][N] (ldb >= N); = 1: B_g is [N][Kd] (ldb >= Kd).
 * dtype LSGD_FP32: A, B are float; LSGD_BF16: A, B are bfloat16 bit patterns
 * (uint16). C is fp32 [G][M][N] with leading dimension N, group stride M*N.
 * Group strides sA, sB are in elements. splits in {2, 3, 4, 8} splits K into
 * that many ranges whose fp32 partial sums go to d_part ([splits][G][M][N],
 * caller owned) and are then added in ascending order; splits == 1 needs no
 * d_part; other counts return LSGD_E_INVALID.
 */
lsgd_status lsgd_grouped_gemm(int32_t dtype, int32_t trans_a, int32_t trans_b,
                              int32_t G, int32_t M, int32_t N, int32_t Kd,
                              const void* d_A, int64_t lda, int64_t sA,
                              const void* d_B, int64_t ldb, int64_t sB,
                              float* d_C, int32_t splits, float* d_part,
                              void* stream);

/* In-place K-way replica average of d_W fp32 [K][P] (the kernel behind
 * lsgd_average). */
lsgd_status lsgd_replica_average(float* d_W, int32_t K, int64_t P,
                                 void* stream);

/* The global-momentum synchronisation of lsgd_synchronise on plain arrays:
 * d_W fp32 [K][P] replicas (all set to the new model), d_wsync fp32 [P] the
 * previous synchronised model and d_ug fp32 [P] the global buffer, both
 * updated in place. m_global in [0, 1), lr finite and non-zero, else
 * LSGD_E_INVALID. */
lsgd_status lsgd_replica_average_global_momentum(float* d_W, int32_t K,
                                                 int64_t P, float* d_wsync,
                                                 float* d_ug, float m_global,
                                                 float lr, void* stream);

/* Scratch bytes lsgd_replica_sign_sync needs for K rows of P elements
 * (P % 4 == 0, else LSGD_E_INVALID). */
lsgd_status lsgd_sign_sync_scratch_bytes(int32_t K, int64_t P, size_t* bytes);

/* The sign-compressed synchronisation of lsgd_synchronise on plain arrays:
 * d_W fp32 [K][P] replicas (all set to the new model), d_wsync fp32 [P] the
 * previous synchronised model (updated), d_E fp32 [K][P] the error memories
 * (updated; Algorithm 4) or NULL (Algorithm 3). d_scratch: caller-owned
 * device memory of lsgd_sign_sync_scratch_bytes (LSGD_E_WORKSPACE if
 * smaller). Pointers 16-byte aligned and P % 4 == 0, else LSGD_E_INVALID.
 * Summation orders: each |delta| partial in fp64 over fixed chunks of 8192
 * elements, chunks added in a fixed order; messages added over k in
 * ascending order in fp32. */
lsgd_status lsgd_replica_sign_sync(float* d_W, int32_t K, int64_t P,
                                   float* d_wsync, float* d_E, void* d_scratch,
                                   size_t scratch_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * lsgd_replica_sign_sync with its scratch taken from a static device array
 * of LSGD_SIGN_SYNC_STATIC_BYTES that the library holds on each GPU it runs
 * on until the process ends, so the call allocates nothing (the caller
 * still passes d_W, d_wsync and d_E). Same arguments, kernels and results as
 * lsgd_replica_sign_sync, bit for bit. Problems needing more scratch than
 * the array holds (lsgd_sign_sync_scratch_bytes(K, P) > 16 MiB, i.e.
 * about K * P > 6.7e7 elements) return LSGD_E_WORKSPACE and launch nothing.
 * Every call on one GPU shares the array: calls that overlap on one GPU
 * (different streams or host threads) race and must be ordered by the
 * caller. The array keeps the last call's contents; nothing in it needs to
 * start at zero.
 */
#define LSGD_SIGN_SYNC_STATIC_BYTES (16u << 20)
lsgd_status lsgd_replica_sign_sync_static(float* d_W, int32_t K, int64_t P,
                                          float* d_wsync, float* d_E,
                                          void* stream);

/* In-place block average of d_W fp32 [K][P]: each of the K/Kb groups of Kb
 * consecutive rows is replaced by its mean (the kernel behind
 * lsgd_average_blocks). Kb must divide K, else LSGD_E_INVALID. */
lsgd_status lsgd_replica_average_blocks(float* d_W, int32_t K, int32_t Kb,
                                        int64_t P, void* stream);

/* Fused update over n elements (the kernel behind the parameter update of
 * lsgd_local_step): g = d_G + wd * w; u = m u + g; d = (nesterov & 1) ?
 * g + m u : u; with nesterov & 2, d = sign(d) (the sign step); w -= lr * d.
 * d_W, d_U updated in place. nesterov outside [0, 3]: LSGD_E_INVALID. */
lsgd_status lsgd_sgd_update(float* d_W, float* d_U, const float* d_G,
                            int64_t n, float lr, float momentum,
                            float weight_decay, int32_t nesterov,
                            void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LSGD_H */
