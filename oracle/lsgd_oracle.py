"""CPU oracle for (post-)local SGD -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module. The product path never calls it.

Plain, slow and fp64. It follows "Don't Use Large Mini-Batches, Use Local SGD"
(Lin, Stich, Patel, Jaggi, ICLR 2020); every function names the passage it
implements. It shares no code with the HIP path: the only common module is
``workloads`` (seeded inputs, no arithmetic of the method).

Readings of the paper taken here (it is silent or garbled on these points):

* sampling -- each worker draws its B_loc indices i.i.d. with replacement
  from its own contiguous shard [floor(kN/K), floor((k+1)N/K)), using
  Philox4x32-10 (Salmon et al., SC'11) keyed by the seed, with counter
  (slot // 4, step low word, worker, step high word); slot j takes output word
  j mod 4 and maps u in [0, 2^32) to the shard by the multiply-shift
  lo + floor(u * n / 2^32);
* averaging -- the plain mean of eq. (2); the Delta form of Algorithms 1 and 2
  is the same thing once the stray step size is dropped (all replicas start a
  round equal);
* optimiser -- coupled L2 decay g = grad + wd * w, buffer u = m u + g, step
  d = u (heavy ball) or d = g + m u (Nesterov), w = w - lr * d; buffers start
  at zero, belong to one replica and are never averaged; decay applies to
  weights and biases;
* post-local switch -- rounds 1..t' use one local step, later rounds H, with
  the decayed step size from round t'+1 on; momentum buffers carry over;
* loss -- per-sample cross-entropy in the numerically stable form, mean over
  the local batch, taken in the forward pass before the update;
* bf16 workloads -- GEMM operands (gathered inputs, hidden activations after
  ReLU, weight copies, and the back-propagated dZ including the one used for
  the bias gradient) are rounded to bfloat16 with round-to-nearest-even;
  everything else stays at full precision.
"""
from __future__ import annotations

import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)

# Philox4x32 constants (Salmon, Moraes, Dror, Shaw, "Parallel random numbers:
# as easy as 1, 2, 3", SC'11): the two round multipliers and the Weyl key
# increments (golden ratio and sqrt(3) - 1 in 0.32 fixed point).
PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint64(0x9E3779B9)
PHILOX_W1 = np.uint64(0xBB67AE85)


# --------------------------------------------------------------------------
# Sampling (eq. 1: index sets drawn from the worker's local data; setup
# section: data partitioned among workers, local mini-batches sampled among
# the local data)
# --------------------------------------------------------------------------
def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds.

    ``ctr``: four arrays of 32-bit words (any integer dtype, same shape);
    ``key``: two 32-bit words. Returns four uint64 arrays holding 32-bit words.
    Each round multiplies words 0 and 2 by the two constants, and the new
    state is (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0));
    the key is bumped by the Weyl increments between rounds.
    """
    c0, c1, c2, c3 = (np.asarray(c).astype(np.uint64) & MASK32 for c in ctr)
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    for r in range(10):
        if r:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = PHILOX_M0 * c0          # < 2^64, exact in uint64
        p1 = PHILOX_M1 * c2
        c0, c1, c2, c3 = ((p1 >> np.uint64(32)) ^ c1 ^ k0, p1 & MASK32,
                          (p0 >> np.uint64(32)) ^ c3 ^ k1, p0 & MASK32)
    return c0, c1, c2, c3


def shard(k: int, K: int, N: int):
    """Worker k's disjoint slice [lo, hi) of the N training rows."""
    return (k * N) // K, ((k + 1) * N) // K


def sample_indices(seed: int, step: int, k: int, K: int, N: int, B: int):
    """I^k for local step ``step`` (counted from init over all rounds).

    Returns int64 [B], i.i.d. uniform (with replacement) over worker k's
    shard.
    """
    lo, hi = shard(k, K, N)
    n = hi - lo
    j = np.arange(B, dtype=np.uint64)
    ctr = (j >> np.uint64(2),
           np.full(B, step & 0xFFFFFFFF, np.uint64),
           np.full(B, k, np.uint64),
           np.full(B, (step >> 32) & 0xFFFFFFFF, np.uint64))
    words = np.stack(philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32)))
    u = words[(j & np.uint64(3)).astype(np.int64), np.arange(B)]
    return lo + ((u * np.uint64(n)) >> np.uint64(32)).astype(np.int64)


# Per-epoch global reshuffle (the CIFAR training procedure: the data is
# partitioned disjointly among the workers and reshuffled globally every
# epoch; each worker then takes its local mini-batches from its part).
# The permutation of epoch e is a counter-based pseudo-random permutation:
# a balanced Feistel network (Luby and Rackoff) on 2m-bit words, 4^m >= N,
# whose round function is word 0 of Philox4x32-10 at counter
# (right half, round, e, SHUFFLE_STREAM), restricted to [0, N) by cycle
# walking (Black and Rogaway): values >= N are permuted again until they
# fall in range.
SHUFFLE_STREAM = 0x5348464C
FEISTEL_ROUNDS = 4


def feistel_bits(N: int) -> int:
    """Half width m: the smallest m >= 1 with 4^m >= N."""
    m = 1
    while (1 << (2 * m)) < N:
        m += 1
    return m


def feistel(x, m: int, seed: int, epoch: int):
    """The Feistel permutation of [0, 4^m) applied to the array ``x``."""
    x = np.asarray(x, np.uint64)
    mask = np.uint64((1 << m) - 1)
    left, right = x >> np.uint64(m), x & mask
    for r in range(FEISTEL_ROUNDS):
        f = philox4x32_10((right, np.full_like(right, r),
                           np.full_like(right, epoch & 0xFFFFFFFF),
                           np.full_like(right, SHUFFLE_STREAM)),
                          (seed & 0xFFFFFFFF, seed >> 32))[0]
        left, right = right, left ^ (f & mask)
    return (left << np.uint64(m)) | right


def epoch_permutation(positions, N: int, seed: int, epoch: int):
    """pi_e(q) for the array of positions q in [0, N)."""
    m = feistel_bits(N)
    y = feistel(np.asarray(positions, np.uint64), m, seed, epoch)
    out = y.copy()
    todo = out >= np.uint64(N)
    while todo.any():
        out[todo] = feistel(out[todo], m, seed, epoch)
        todo = out >= np.uint64(N)
    return out.astype(np.int64)


def steps_per_epoch(K: int, N: int, B: int) -> int:
    """Whole local mini-batches per epoch: every worker's part holds at least
    floor(N / K) rows, of which floor(floor(N / K) / B) batches are taken
    (the rest of a part is left for that epoch; the next reshuffle moves
    every row to a random place)."""
    return (N // K) // B


def sample_indices_epoch(seed: int, step: int, k: int, K: int, N: int, B: int):
    """I^k for local step ``step`` under the per-epoch reshuffle: epoch
    e = step // S, batch j = step % S (S = steps_per_epoch); worker k's part
    of epoch e is pi_e restricted to its slice [lo_k, hi_k) of positions, and
    batch j is positions lo_k + jB .. lo_k + jB + B - 1 of it (without
    replacement within the epoch)."""
    S = steps_per_epoch(K, N, B)
    if S < 1:
        raise ValueError("a worker's part must hold at least one batch")
    e, j = divmod(step, S)
    lo, _ = shard(k, K, N)
    q = lo + j * B + np.arange(B, dtype=np.int64)
    return epoch_permutation(q, N, seed, e)


def worker_indices(wl, step: int, k: int):
    """The index set of worker k at a local step, by the workload's
    sampler ("iid": with replacement from a fixed shard; "epoch": the
    per-epoch reshuffled partition)."""
    if getattr(wl, "sampler", "iid") == "epoch":
        return sample_indices_epoch(wl.sample_seed, step, k, wl.K, wl.N, wl.B_loc)
    return sample_indices(wl.sample_seed, step, k, wl.K, wl.N, wl.B_loc)


# --------------------------------------------------------------------------
# bfloat16 rounding (operand precision of the bf16 workload)
# --------------------------------------------------------------------------
def rne_bf16(x):
    """Round to the nearest bfloat16 value, ties to even; returns float64.

    bfloat16 keeps 8 significant bits and fp32's exponent range: normal
    values below 2^-126 fall onto the fixed subnormal grid of 2^-133.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                       # x = m * 2^e, |m| in [0.5, 1)
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)   # spacing of bf16 near x
    r = np.round(x / q) * q                  # np.round is half-to-even
    big = np.abs(r) > 3.3895313892515355e38  # beyond the largest bf16
    if np.any(big):
        r = np.where(big, np.sign(r) * np.inf, r)
    return r


# --------------------------------------------------------------------------
# The model: fully-connected ReLU network with a softmax cross-entropy loss
# (f_i of the sum-structured objective in the introduction); with no hidden
# layer it is softmax regression.
# --------------------------------------------------------------------------
def unpack(w, widths):
    """Views (W_l [d_in][d_out], b_l [d_out]) into a flat parameter vector."""
    out, o = [], 0
    for din, dout in zip(widths[:-1], widths[1:]):
        W = w[o:o + din * dout].reshape(din, dout)
        o += din * dout
        b = w[o:o + dout]
        o += dout
        out.append((W, b))
    assert o == w.size, (o, w.size)
    return out


def cross_entropy(z, y):
    """Per-row loss -log softmax(z)_y and the softmax probabilities.

    Stable form: with m = max_j z_j, the loss is log1p(sum_{j != y} e^{z_j-m})
    when z_y is the maximum, else (m - z_y) + log(sum_j e^{z_j - m}).
    """
    z = np.asarray(z, np.float64)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1)
    rows = np.arange(z.shape[0])
    zy = z[rows, y]
    is_max = zy >= m[:, 0]
    others = e.copy()
    others[rows, y] = 0.0
    rest = others.sum(axis=1)         # summed directly: no cancellation
    loss = np.where(is_max, np.log1p(rest), (m[:, 0] - zy) + np.log(s))
    p = e / s[:, None]
    return loss, p


def loss_and_grad(w, widths, A0, y, bf16=False):
    """Mean mini-batch loss and its gradient (the bracket of eq. 2).

    ``A0`` [B][d_in] are the gathered rows, ``y`` their labels. Returns
    (loss_mean, flat gradient in the layout of ``w``).
    """
    rnd = rne_bf16 if bf16 else (lambda v: v)
    B = A0.shape[0]
    layers = unpack(np.asarray(w, np.float64), widths)
    L = len(layers)
    Wq = [rnd(W) for W, _ in layers]
    acts = [rnd(np.asarray(A0, np.float64))]
    pre = []
    for l, (W, b) in enumerate(layers):
        z = acts[-1] @ Wq[l] + b
        pre.append(z)
        if l < L - 1:
            acts.append(rnd(np.maximum(z, 0.0)))
    loss, p = cross_entropy(pre[-1], y)
    dz = p.copy()
    dz[np.arange(B), y] -= 1.0
    dz /= B
    grads = [None] * L
    for l in range(L - 1, -1, -1):
        dzq = rnd(dz)
        gW = acts[l].T @ dzq
        gb = dzq.sum(axis=0)
        grads[l] = (gW, gb)
        if l > 0:
            dz = (dzq @ Wq[l].T) * (pre[l - 1] > 0.0)
    flat = np.concatenate([np.concatenate([gW.ravel(), gb]) for gW, gb in grads])
    return float(loss.mean()), flat


def decay_mask(widths):
    """1 where weight decay applies: every weight and bias of the network."""
    return np.ones(sum(a * b + b for a, b in zip(widths[:-1], widths[1:])))


# --------------------------------------------------------------------------
# Optimiser step (local update of eq. 2 with the local momentum of the
# appendix on local SGD with momentum; Nesterov, no dampening, weight decay
# from the CIFAR hyper-parameter paragraph)
# --------------------------------------------------------------------------
def sgd_update(w, u, grad, lr, momentum, weight_decay, nesterov, wd_mask=1.0,
               sign_step=False):
    """One local step on one replica: returns (w_new, u_new). With
    ``sign_step`` the replica moves by the sign of its update direction (the
    local step of the signSGD variant, Algorithm 3: the direction may
    include weight decay and momentum); sign(0) = 0."""
    g = grad + (weight_decay * wd_mask) * w
    u = momentum * u + g
    d = g + momentum * u if nesterov else u
    if sign_step:
        d = np.sign(d)
    return w - lr * d, u


# --------------------------------------------------------------------------
# Synchronisation (eq. 2, right part; Algorithms 1 and 2)
# --------------------------------------------------------------------------
def average(W):
    """Replace every replica by the mean of the K replicas. W: [K][P]."""
    W = np.asarray(W, np.float64)
    wbar = W.sum(axis=0) / W.shape[0]
    return np.broadcast_to(wbar, W.shape).copy()


def average_delta_form(W_start, W_end):
    """Algorithm 1's form: w_(t) - (1/K) sum_k Delta^k with Delta^k =
    w^k_(t) - w^k_(t)+H, read without the stray step size; all rows of
    ``W_start`` are the synchronised w_(t)."""
    D = np.asarray(W_start, np.float64) - np.asarray(W_end, np.float64)
    wbar = np.asarray(W_start, np.float64)[0] - D.sum(axis=0) / D.shape[0]
    return np.broadcast_to(wbar, D.shape).copy()


def average_global_momentum(W, w_sync, u_global, m_global, lr):
    """Synchronisation of local SGD with global momentum (momentum appendix,
    the paragraph on local SGD with global momentum; with local momentum on
    as well it is the hybrid scheme of the next paragraph). The round's
    model differences Delta^k = w_(t) - w^k_(t)+H, averaged over the workers
    and divided by the step size, feed a momentum buffer u held with the
    synchronised model:
        u_(t)   = m_g u_(t-1) + (1/lr) (1/K) sum_k Delta^k,
        w_(t+1) = w_(t) - lr u_(t).
    W: [K][P] replicas at the end of the round; w_sync = w_(t). Returns
    (every replica set to w_(t+1), w_(t+1), u_(t)). With m_g = 0 this is the
    plain average up to rounding."""
    W = np.asarray(W, np.float64)
    w_sync = np.asarray(w_sync, np.float64)
    deltas = w_sync[None, :] - W
    u = m_global * np.asarray(u_global, np.float64) + deltas.sum(axis=0) / W.shape[0] / lr
    w = w_sync - lr * u
    return np.broadcast_to(w, W.shape).copy(), w.copy(), u


def compress_sign(delta):
    """The compressor of Algorithms 3 and 4: the sign vector s = sign(delta)
    (sign(0) = 0) and the scale p = ||delta||_1 / d, d the model size."""
    delta = np.asarray(delta, np.float64)
    return np.sign(delta), np.abs(delta).sum() / delta.size


def average_sign_compressed(W, w_sync, E=None):
    """Sign-compressed synchronisation (Algorithm 3's; Algorithm 4's when the
    error memories E are given). Each worker's model difference
    Delta^k = w_(t) - w^k_(t)+H, plus e^k for Algorithm 4, is sent as
    s^k p^k; the new synchronised model is w_(t) - (1/K) sum_k s^k p^k.
    Algorithm 4 keeps what the message missed, e^k = Delta^k - s^k p^k
    (error feedback: the memory holds the part of the corrected difference
    that was not transmitted). Returns (every replica set to w_(t+1),
    w_(t+1), new E or None)."""
    W = np.asarray(W, np.float64)
    w_sync = np.asarray(w_sync, np.float64)
    K = W.shape[0]
    sent = np.zeros_like(W)
    newE = None if E is None else np.zeros_like(W)
    for k in range(K):
        delta = w_sync - W[k]
        if E is not None:
            delta = delta + E[k]
        s, p = compress_sign(delta)
        sent[k] = s * p
        if E is not None:
            newE[k] = delta - sent[k]
    w = w_sync - sent.sum(axis=0) / K
    return np.broadcast_to(w, W.shape).copy(), w.copy(), newE


def synchronise(state, wl, lr):
    """The global synchronisation at the end of a round: the plain average of
    eq. (2); the global-momentum form when the workload sets a global
    momentum factor (read with the step size of the round's local steps);
    the sign-compressed forms of Algorithms 3 ("sign") and 4 ("ef_sign")."""
    m_g = getattr(wl, "global_momentum", 0.0)
    scheme = getattr(wl, "scheme", "local")
    if scheme in ("sign", "ef_sign"):
        state.W, state.w_sync, E = average_sign_compressed(
            state.W, state.w_sync, state.E if scheme == "ef_sign" else None)
        if E is not None:
            state.E = E
    elif m_g:
        state.W, state.w_sync, state.u_global = average_global_momentum(
            state.W, state.w_sync, state.u_global, m_g, lr)
    else:
        state.W = average(state.W)
        state.w_sync = state.W[0].copy()
    if getattr(state, "RS", None) is not None:
        # BN running statistics are not trained: every scheme takes their
        # plain mean over the workers
        state.RS = average(state.RS)


def average_blocks(W, Kb):
    """Hierarchical local SGD's block synchronisation (Appendix D, the
    hierarchical local SGD equation, middle line; Algorithm 5's inner
    all-reduce, read as a plain mean like the global one): replicas are
    grouped into blocks of Kb consecutive workers and every replica is
    replaced by the mean of its block. W: [K][P], K a multiple of Kb."""
    W = np.asarray(W, np.float64)
    K = W.shape[0]
    if Kb < 1 or K % Kb:
        raise ValueError("the block size must divide K")
    blocks = W.reshape(K // Kb, Kb, -1)
    means = blocks.sum(axis=1) / Kb
    return np.repeat(means, Kb, axis=0)


# --------------------------------------------------------------------------
# Drivers
# --------------------------------------------------------------------------
class State:
    """K replicas w^k, their momentum buffers u^k, and the step counter; for
    global momentum also the synchronised model w_(t) and its buffer u; for
    the ResNet its per-replica BN running statistics RS [K][R] (created at the
    first local step, see resnet_running_init)."""

    def __init__(self, w0, K):
        self.W = np.repeat(np.asarray(w0, np.float64)[None, :], K, axis=0)
        self.U = np.zeros_like(self.W)
        self.step = 0
        self.w_sync = np.asarray(w0, np.float64).copy()
        self.u_global = np.zeros_like(self.w_sync)
        self.E = np.zeros_like(self.W)     # error memories e^k (Algorithm 4)
        self.RS = None


def local_step(state, wl, X, y, lr, replicas=None):
    """One local step (inner loop body of Algorithm 1) on each replica.

    ``wl`` is a ``workloads.Workload``. Returns the per-replica mini-batch
    losses (NaN for replicas not in ``replicas``).
    """
    K = state.W.shape[0]
    ks = range(K) if replicas is None else replicas
    losses = np.full(K, np.nan)
    mask = model_decay_mask(wl)
    resnet = wl.model == "resnet20"
    if resnet and getattr(state, "RS", None) is None:
        state.RS = np.repeat(resnet_running_init(resnet_arch())[None, :], K, axis=0)
    for k in ks:
        idx = worker_indices(wl, state.step, k)
        A0 = np.asarray(X[idx], np.float64)
        if resnet:
            # per-worker BN: replica k's running statistics follow its batches
            stats = []
            loss, grad = resnet_loss_and_grad(state.W[k], resnet_arch(), A0, y[idx], stats)
            half = state.RS.shape[1] // 2
            for (_, o, c), (mu, var, n) in zip(resnet_running_layout(resnet_arch()), stats):
                state.RS[k, o:o + c], state.RS[k, half + o:half + o + c] = \
                    bn_running_update(state.RS[k, o:o + c],
                                      state.RS[k, half + o:half + o + c], mu, var, n)
        else:
            loss, grad = model_loss_and_grad(wl, state.W[k], A0, y[idx])
        state.W[k], state.U[k] = sgd_update(
            state.W[k], state.U[k], grad, lr, wl.momentum, wl.weight_decay,
            wl.nesterov, mask, sign_step=getattr(wl, "scheme", "local") == "sign")
        losses[k] = loss
    state.step += 1
    return losses


def model_loss_and_grad(wl, w, A0, y):
    """Loss and gradient of the workload's model on one mini-batch."""
    if wl.model == "resnet20":
        return resnet_loss_and_grad(w, resnet_arch(), A0, y)
    return loss_and_grad(w, wl.widths, A0, y, bf16=(wl.dtype == "bf16"))


def model_decay_mask(wl):
    if wl.model == "resnet20":
        return resnet_decay_mask(resnet_arch())
    return decay_mask(wl.widths)


def run_round(state, wl, X, y, H, lr):
    """H local steps on every replica, then the synchronisation (the average,
    or its global-momentum form); returns [H][K] losses. ``lr`` is one step
    size for the round or a list of H, one per local step (the
    synchronisation uses the last)."""
    lrs = list(lr) if np.ndim(lr) else [lr] * H
    if len(lrs) != H:
        raise ValueError("one step size per local step")
    losses = np.stack([local_step(state, wl, X, y, a) for a in lrs])
    synchronise(state, wl, lrs[-1] if lrs else lr)
    return losses


def run_hierarchical_round(state, wl, X, y, H, Hb, Kb, lr):
    """One outer round of hierarchical local SGD (Appendix D, Algorithm 5):
    Hb block rounds, each H local steps on every replica followed by the
    block average over Kb consecutive replicas, then the global average.
    Momentum buffers stay local. Returns the [Hb * H][K] losses."""
    losses = []
    for _ in range(Hb):
        for _ in range(H):
            losses.append(local_step(state, wl, X, y, lr))
        state.W = average_blocks(state.W, Kb)
        if getattr(state, "RS", None) is not None:
            state.RS = average_blocks(state.RS, Kb)
    synchronise(state, wl, lr)
    return np.stack(losses)


def schedule(wl):
    """(H_t, lr_t) per round: the post-local rule H_(t) = 1 for t <= t',
    else H (section 3), with the decayed step size after the switch."""
    out = []
    for t in range(1, wl.warm_rounds + wl.rounds + 1):
        if t <= wl.warm_rounds:
            out.append((1, wl.lr))
        else:
            out.append((wl.H, wl.lr_after_switch if wl.warm_rounds else wl.lr))
    return out


# --------------------------------------------------------------------------
# Schedules of the training procedure (host side): the large-batch learning
# rate schemes (linear scaling and gradual warm-up), the step decay at 50%
# and 75% of the sample budget, and the local-step warm-up strategies.
# --------------------------------------------------------------------------
def goyal_lr(step: int, lr: float, scale: float, warmup_steps: int) -> float:
    """Step size of local step ``step`` (0-based) under the large-batch
    schemes: the target lr * scale (the linear scaling rule), reached from lr
    by a constant increment per iteration, (target - lr) / warmup_steps. With
    warmup_steps = 5 N / (K B) (five epochs) this is the appendix's
    increment. warmup_steps = 0: the target from the start."""
    target = lr * scale
    if warmup_steps <= 0 or step >= warmup_steps:
        return target
    return lr + step * (target - lr) / warmup_steps


def decay_factor(step: int, samples_per_step: int, total_samples: int,
                 milestones=(0.5, 0.75), factor: float = 0.1) -> float:
    """The step decay of the CIFAR procedure: the step size is divided by 10
    once the run has accessed 50% of its sample budget and again at 75%;
    ``step`` local steps (of samples_per_step samples over all workers) have
    been taken before the step in question."""
    f = 1.0
    for m in milestones:
        if step * samples_per_step >= m * total_samples:
            f *= factor
    return f


def local_steps_of_epoch(epoch: int, H: int, kind, warmup_epochs: int) -> int:
    """Local-step warm-up (the appendix on it and the ImageNet runs): during
    the first ``warmup_epochs`` epochs H grows from 1 -- "linear": by equal
    increments, 1 + floor((H - 1) e / W); "exponential": doubling, min(H, 2^e)
    (H = 8 over three epochs gives 1, 2, 4, as in the ImageNet runs);
    "constant": 1 throughout -- and is H afterwards."""
    if kind is None or epoch >= warmup_epochs:
        return H
    if kind == "linear":
        return 1 + ((H - 1) * epoch) // warmup_epochs
    if kind == "exponential":
        return min(H, 2 ** epoch)
    if kind == "constant":
        return 1
    raise ValueError(kind)


def schedule_rounds(total_steps: int, steps_per_ep: int, H: int, lr_of_step,
                    h_kind=None, h_warmup_epochs: int = 0,
                    switch_step=None):
    """The rounds of a run as [(H_t, [step size of each of its steps])]: a
    round's H_t is that of the epoch in which it starts (local-step warm-up),
    or -- post-local SGD -- 1 before ``switch_step`` and H from it on; the
    last round is cut so that the run takes exactly ``total_steps`` local
    steps (every method accesses the same number of samples)."""
    rounds, s = [], 0
    while s < total_steps:
        if switch_step is not None:
            Ht = 1 if s < switch_step else H
        else:
            Ht = local_steps_of_epoch(s // steps_per_ep, H, h_kind, h_warmup_epochs)
        Ht = min(Ht, total_steps - s)
        rounds.append((Ht, [lr_of_step(s + h) for h in range(Ht)]))
        s += Ht
    return rounds


def run(wl, X, y, w0, rounds=None):
    """Whole (post-)local SGD run (Algorithm 2; Algorithm 1 when t' = 0).

    Returns (state, per-round list of [H_t][K] loss arrays).
    """
    st = State(w0, wl.K)
    sched = schedule(wl)
    if rounds is not None:
        sched = sched[:rounds]
    traj = [run_round(st, wl, X, y, H, lr) for H, lr in sched]
    return st, traj


def minibatch_sgd(wl, X, y, w0, steps, lr):
    """Plain mini-batch SGD of eq. (1) with one global momentum buffer (the
    distributed mini-batch momentum recursion of the momentum appendix): the
    gradient is taken over the union of the K workers' index sets at once.
    Used only as the comparator of the H = 1 special case."""
    w = np.asarray(w0, np.float64).copy()
    u = np.zeros_like(w)
    mask = model_decay_mask(wl)
    for s in range(steps):
        idx = np.concatenate([
            worker_indices(wl, s, k)
            for k in range(wl.K)])
        _, grad = model_loss_and_grad(wl, w, np.asarray(X[idx], np.float64), y[idx])
        g = grad + wl.weight_decay * mask * w
        u = wl.momentum * u + g
        d = g + wl.momentum * u if wl.nesterov else u
        w = w - lr * d
    return w


# --------------------------------------------------------------------------
# ResNet-20-shaped network (the CIFAR ResNet of the appendix on models and
# Table 5: 0.27M parameters, 0.041 G multiply-adds per image). NHWC images;
# 3x3 convolutions, padding 1; per-worker batch normalisation (training-mode
# batch statistics, the per-worker BN of the CIFAR setup paragraph); option-A
# shortcuts (subsample, zero-pad channels); global average pool; FC classifier.
# --------------------------------------------------------------------------
BN_EPS = 1e-5


def resnet_arch(side=32, cin=3, base=16, blocks=3, classes=10):
    return dict(side=side, cin=cin, base=base, blocks=blocks, classes=classes)


def resnet_convs(arch):
    """[(name, c_in, c_out, stride)] of every 3x3 convolution, in order."""
    out = [("conv1", arch["cin"], arch["base"], 1)]
    c = arch["base"]
    for s in range(3):
        co = arch["base"] * 2**s
        for b in range(arch["blocks"]):
            stride = 2 if (s > 0 and b == 0) else 1
            out.append((f"s{s}b{b}a", c, co, stride))
            out.append((f"s{s}b{b}b", co, co, 1))
            c = co
    return out


def resnet_layout(arch):
    """[(name, shape, decays)] of the flat parameter vector, in order: per
    convolution its weight [3][3][c_in][c_out] then BN gamma and beta; then
    the classifier weight [c][classes] and bias."""
    out = []
    for name, ci, co, _ in resnet_convs(arch):
        out += [(name + ".w", (3, 3, ci, co), True), (name + ".g", (co,), False),
                (name + ".be", (co,), False)]
    c = arch["base"] * 4
    out += [("fc.w", (c, arch["classes"]), True), ("fc.b", (arch["classes"],), True)]
    return out


def resnet_unpack(w, arch):
    out, o = {}, 0
    for name, shape, _ in resnet_layout(arch):
        n = int(np.prod(shape))
        out[name] = w[o:o + n].reshape(shape)
        o += n
    assert o == w.size
    return out


def resnet_decay_mask(arch):
    return np.concatenate([np.full(int(np.prod(s)), 1.0 if d else 0.0)
                           for _, s, d in resnet_layout(arch)])


def _im2col(x, stride):
    """x [B][H][W][C] -> patches [B][Ho][Wo][3][3][C] (zero padding 1)."""
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    win = np.lib.stride_tricks.sliding_window_view(xp, (3, 3), axis=(1, 2))
    win = win[:, ::stride, ::stride]               # [B][Ho][Wo][C][3][3]
    return np.ascontiguousarray(win.transpose(0, 1, 2, 4, 5, 3))


def conv3x3(x, W, stride):
    """Convolution with weight W [3][3][c_in][c_out]; returns (y, patches)."""
    cols = _im2col(x, stride)
    B, Ho, Wo = cols.shape[:3]
    y = cols.reshape(B * Ho * Wo, -1) @ W.reshape(-1, W.shape[3])
    return y.reshape(B, Ho, Wo, W.shape[3]), cols


def conv3x3_backward(dy, cols, W, x_shape, stride):
    """Gradients of conv3x3 w.r.t. its weight and its input."""
    B, Ho, Wo, co = dy.shape
    d2 = dy.reshape(-1, co)
    dW = (cols.reshape(d2.shape[0], -1).T @ d2).reshape(W.shape)
    dcols = (d2 @ W.reshape(-1, co).T).reshape(B, Ho, Wo, 3, 3, -1)
    H, Wd = x_shape[1], x_shape[2]
    dxp = np.zeros((B, H + 2, Wd + 2, x_shape[3]))
    for kh in range(3):
        for kw in range(3):
            dxp[:, kh:kh + stride * Ho:stride, kw:kw + stride * Wo:stride, :] += \
                dcols[:, :, :, kh, kw, :]
    return dW, dxp[:, 1:H + 1, 1:Wd + 1, :]


def batchnorm(x, g, be):
    """Training-mode BN over (batch, height, width), biased variance."""
    mu = x.mean(axis=(0, 1, 2))
    var = ((x - mu) ** 2).mean(axis=(0, 1, 2))
    inv = 1.0 / np.sqrt(var + BN_EPS)
    xh = (x - mu) * inv
    return g * xh + be, (xh, inv, g)


def batchnorm_backward(dy, cache):
    xh, inv, g = cache
    dbe = dy.sum(axis=(0, 1, 2))
    dg = (dy * xh).sum(axis=(0, 1, 2))
    dx = g * inv * (dy - dy.mean(axis=(0, 1, 2)) - xh * (dy * xh).mean(axis=(0, 1, 2)))
    return dx, dg, dbe


BN_MOMENTUM = 0.1


def bn_running_update(rm, rv, mean, var, n, momentum=BN_MOMENTUM):
    """Running statistics of one BN layer after a training-mode batch (the
    paper keeps BN per worker and is silent on its running statistics; read
    as the usual convention of its PyTorch implementation): an exponential
    average with factor ``momentum`` of the batch mean and of the unbiased
    batch variance var * n / (n - 1), ``var`` being the biased variance that
    normalised the batch over its ``n`` values per channel."""
    return ((1.0 - momentum) * rm + momentum * mean,
            (1.0 - momentum) * rv + momentum * var * (n / (n - 1.0)))


def resnet_running_layout(arch):
    """[(name, offset, channels)] of the running statistics of one replica:
    the running means of every BN layer in convolution order, then the
    running variances in the same order; the flat vector has 2 * sum(C)
    entries."""
    out, o = [], 0
    for name, _, co, _ in resnet_convs(arch):
        out.append((name, o, co))
        o += co
    return out


def resnet_running_init(arch):
    """Initial running statistics: means 0, variances 1."""
    n = sum(c for _, _, c in resnet_running_layout(arch))
    return np.concatenate([np.zeros(n), np.ones(n)])


def _shortcut(x, co):
    """Option A: every second pixel, channels zero-padded to co."""
    s = x[:, ::2, ::2, :]
    return np.concatenate([s, np.zeros(s.shape[:3] + (co - s.shape[3],))], axis=3)


def resnet_loss_and_grad(w, arch, A0, y, stats=None):
    """Mean mini-batch loss and flat gradient; A0 [B][side*side*cin] NHWC.
    With a list ``stats``, each BN layer appends (batch mean, biased batch
    variance, values per channel) in convolution order."""
    p = resnet_unpack(np.asarray(w, np.float64), arch)
    B = A0.shape[0]
    x = np.asarray(A0, np.float64).reshape(B, arch["side"], arch["side"], arch["cin"])
    convs = resnet_convs(arch)
    tape = []

    def cbr(x, name, stride, relu):
        y, cols = conv3x3(x, p[name + ".w"], stride)
        z, bc = batchnorm(y, p[name + ".g"], p[name + ".be"])
        if stats is not None:
            mu = y.mean(axis=(0, 1, 2))
            stats.append((mu, ((y - mu) ** 2).mean(axis=(0, 1, 2)),
                          y.shape[0] * y.shape[1] * y.shape[2]))
        tape.append((name, x.shape, stride, cols, bc))
        return np.maximum(z, 0.0) if relu else z, z

    h, _ = cbr(x, "conv1", 1, True)
    blocks = []  # (input, pre-activation of the output) per block
    for i in range(1, len(convs), 2):
        name_a, ci, co, stride = convs[i]
        name_b = convs[i + 1][0]
        a, za = cbr(h, name_a, stride, True)
        b, _ = cbr(a, name_b, 1, False)
        sc = h if (stride == 1 and ci == co) else _shortcut(h, co)
        out = b + sc
        blocks.append((h, za, out, stride, ci, co))
        h = np.maximum(out, 0.0)
    feat = h.mean(axis=(1, 2))                           # global average pool
    z = feat @ p["fc.w"] + p["fc.b"]
    loss, prob = cross_entropy(z, y)
    dz = prob.copy()
    dz[np.arange(B), y] -= 1.0
    dz /= B

    g = {"fc.w": feat.T @ dz, "fc.b": dz.sum(axis=0)}
    dh = np.broadcast_to((dz @ p["fc.w"].T)[:, None, None, :], h.shape) / (h.shape[1] * h.shape[2])
    t = len(tape) - 1
    for (hin, za, out, stride, ci, co) in reversed(blocks):
        dout = dh * (out > 0.0)
        # second convolution of the block (no ReLU after its BN)
        name_b, xs_b, st_b, cols_b, bc_b = tape[t]
        dyb, g[name_b + ".g"], g[name_b + ".be"] = batchnorm_backward(dout, bc_b)
        g[name_b + ".w"], da = conv3x3_backward(dyb, cols_b, p[name_b + ".w"], xs_b, st_b)
        t -= 1
        name_a, xs_a, st_a, cols_a, bc_a = tape[t]
        dza = da * (za > 0.0)
        dya, g[name_a + ".g"], g[name_a + ".be"] = batchnorm_backward(dza, bc_a)
        g[name_a + ".w"], dx = conv3x3_backward(dya, cols_a, p[name_a + ".w"], xs_a, st_a)
        t -= 1
        if stride == 1 and ci == co:
            dx = dx + dout
        else:
            dsc = np.zeros_like(hin)
            dsc[:, ::2, ::2, :] = dout[..., :ci]
            dx = dx + dsc
        dh = dx
    name, xs, st, cols, bc = tape[0]
    # conv1 output went through ReLU: its mask is the block-0 input > 0
    dz1 = dh * (blocks[0][0] > 0.0)
    dy1, g[name + ".g"], g[name + ".be"] = batchnorm_backward(dz1, bc)
    g[name + ".w"], _ = conv3x3_backward(dy1, cols, p[name + ".w"], xs, st)
    flat = np.concatenate([g[n].ravel() for n, _, _ in resnet_layout(arch)])
    return float(loss.mean()), flat


def resnet_param_count(arch):
    return sum(int(np.prod(s)) for _, s, _ in resnet_layout(arch))


def resnet_macs_per_image(arch):
    side, macs = arch["side"], 0
    for _, ci, co, stride in resnet_convs(arch):
        side //= stride
        macs += side * side * 9 * ci * co
    return macs + arch["base"] * 4 * arch["classes"]
