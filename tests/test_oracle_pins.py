"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each checks it against a
published vector, an independent library, a closed form, brute force in high
precision, or a special case of the method that reduces to a simpler,
separately written algorithm. No GPU is needed.
"""
import decimal
import math
import os
import shutil
import subprocess

import numpy as np
import pytest

import workloads as wk
from oracle import lsgd_oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


# ------------------------------------------------------------------ sampler
def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append([int(v, 16) for v in line.split()])
    return rows


def test_philox_known_answer_vectors():
    for r in _kat_rows():
        out = O.philox4x32_10([np.array([v]) for v in r[:4]], r[4:6])
        assert [int(o[0]) for o in out] == r[6:10]


def test_philox_matches_rocrand_engine(tmp_path):
    """rocRAND's Philox4x32-10 (host-callable ROCm header) on random blocks."""
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = tmp_path / "ref"
    subprocess.run([hipcc, "-x", "hip", "--offload-arch=gfx950", "-O1",
                    os.path.join(HERE, "rocrand_philox_ref.cpp"), "-o",
                    str(exe)], check=True, capture_output=True)
    rng = np.random.default_rng(7)
    blocks = rng.integers(0, 2**32, size=(500, 6), dtype=np.uint64)
    text = "\n".join(" ".join(f"{int(v):08x}" for v in b) for b in blocks)
    res = subprocess.run([str(exe)], input=text + "\n", check=True,
                         capture_output=True, text=True).stdout.split()
    got = np.array([int(v, 16) for v in res], dtype=np.uint64).reshape(-1, 4)
    mine = np.stack([
        np.stack(O.philox4x32_10([blocks[i:i + 1, c] for c in range(4)],
                                 (int(blocks[i, 4]), int(blocks[i, 5]))))[:, 0]
        for i in range(len(blocks))])
    np.testing.assert_array_equal(mine, got)


@pytest.mark.parametrize("K,N,sizes", [(4, 4096, {1024}), (16, 50000, {3125}),
                                       (64, 50000, {781, 782})])
def test_shards_partition_the_data(K, N, sizes):
    bounds = [O.shard(k, K, N) for k in range(K)]
    assert bounds[0][0] == 0 and bounds[-1][1] == N
    assert all(bounds[k][1] == bounds[k + 1][0] for k in range(K - 1))
    assert {hi - lo for lo, hi in bounds} == sizes


def test_sampler_stays_in_shard_and_is_deterministic():
    K, N, B = 64, 50000, 64
    for s in (0, 1, 17, 2**32 + 5):
        for k in (0, 1, 31, 63):
            lo, hi = O.shard(k, K, N)
            a = O.sample_indices(99, s, k, K, N, B)
            assert a.dtype == np.int64 and a.shape == (B,)
            assert a.min() >= lo and a.max() < hi
            np.testing.assert_array_equal(a, O.sample_indices(99, s, k, K, N, B))


def test_sampler_uniform_over_shard():
    """Chi-square test of the shard occupancy over many steps (n = 37)."""
    K, N, B = 4, 148, 32
    counts = np.zeros(N // K)
    for s in range(400):
        counts += np.bincount(O.sample_indices(5, s, 2, K, N, B) - 74,
                              minlength=N // K)
    exp = counts.sum() / counts.size
    chi2 = ((counts - exp) ** 2 / exp).sum()
    # 36 degrees of freedom: the 99.9% quantile is about 67.98
    assert chi2 < 68.0, chi2


def test_sampler_streams_differ_across_workers_and_steps():
    K, N, B = 2, 2**20, 256
    a = O.sample_indices(1, 3, 0, K, N, B).astype(float)
    b = O.sample_indices(1, 3, 1, K, N, B).astype(float) - N // 2
    c = O.sample_indices(1, 4, 0, K, N, B).astype(float)
    d = O.sample_indices(2, 3, 0, K, N, B).astype(float)
    for other in (b, c, d):
        assert abs(np.corrcoef(a, other)[0, 1]) < 0.25
        assert not np.array_equal(a, other)


# ------------------------------------------------------------------ bf16
@pytest.mark.parametrize("x,want", [
    (1.0, 1.0),
    (1.0 + 2.0**-8, 1.0),                         # tie -> even (mantissa 0)
    (1.0 + 3 * 2.0**-8, 1.0 + 2.0**-6),           # tie -> even (mantissa 2)
    (1.0 + 2.0**-8 + 2.0**-30, 1.0 + 2.0**-7),    # just above the tie
    (-(1.0 + 2.0**-8 + 2.0**-30), -(1.0 + 2.0**-7)),
    (3.0 * 2.0**-133 / 2, 2.0**-132),             # subnormal tie -> even
    (2.0**-134, 0.0),                             # half the smallest -> 0
    (0.0, 0.0),
    (255.5, 256.0),                               # 8 significant bits
])
def test_bf16_rounding_hand_values(x, want):
    assert O.rne_bf16(x) == want


def test_bf16_rounding_matches_torch_on_fp32_values():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(200000) *
         np.exp2(rng.integers(-140, 120, 200000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.rne_bf16(x.astype(np.float64)), ref)


def test_bf16_rounding_points_on_a_hand_computed_network():
    """The bf16 workload's rounding points, each made visible on a 1-1-2
    network with one sample of class 0 whose inputs sit at bf16 ties:
      x = 1 + 2^-8 (rounds to 1), W1 = 1 + 2^-8 (to 1), b1 = 2^-9 (fp32, not
      rounded), W2 = [1 + 2^-8, -(1/2 + 2^-9)] (to [1, -1/2]), b2 = 0.
    By hand: z1 = 1 + 2^-9, whose ReLU rounds to 1; z2 = [1, -1/2]; with
    s = 1 / (1 + e^1.5) = 0.18242552..., dZ2 = [-s, s], rounded to
    [-187, 187] 2^-10; dW2 = 1 * dZ2q; db2 = dZ2q; the input gradient
    dZ2q W2q^T = -187 * 1.5 * 2^-10 = -0.27392578125 (ReLU slope 1), rounded to
    -140 * 2^-9 = -0.2734375 = dW1 = db1; the loss is log(1 + e^-1.5).
    Each single change -- leaving x, W1, the hidden activation, W2 (forward
    or input gradient) or a dZ unrounded, or taking a bias gradient before
    its dZ's rounding -- moves at least one of these values by >= 2^-10
    relative (x or W1 unrounded gives a hidden activation that rounds to
    1 + 2^-7; an unrounded W2 in the input gradient gives 141 * 2^-9)."""
    q = 2.0 ** -8
    w = np.array([1 + q,                      # W1 [1][1]
                  2.0 ** -9,                  # b1
                  1 + q, -(0.5 + q / 2),      # W2 [1][2]
                  0.0, 0.0])                  # b2
    A0 = np.array([[1 + q]])
    loss, g = O.loss_and_grad(w, (1, 1, 2), A0, np.array([0]), bf16=True)
    s = 1.0 / (1.0 + math.exp(1.5))
    assert round(s * 1024) == 187 and abs(s * 1024 - 187) > 0.1   # not a tie
    dz2q = 187 * 2.0 ** -10
    dz1q = -140 * 2.0 ** -9
    want = np.array([dz1q, dz1q, -dz2q, dz2q, -dz2q, dz2q])
    np.testing.assert_array_equal(g, want)
    assert abs(loss - math.log1p(math.exp(-1.5))) <= 1e-15
    # the same network without any bf16 rounding gives other values
    _, g32 = O.loss_and_grad(w, (1, 1, 2), A0, np.array([0]), bf16=False)
    assert np.all(np.abs(g32 - want) >= 2.0 ** -10 * np.abs(want))


def test_bf16_rounding_points_with_a_batch_and_a_dead_unit():
    """Two samples and two hidden units, one of them below zero for the
    second sample (its mask and its rounded activation of 0): the bias
    gradients are the batch sums of the rounded dZ (each already divided by
    the batch size), the weight gradients the rounded activations times the
    rounded dZ. Checked against the per-sample scalar formulas written out
    here with the rounding applied at the same points."""
    r = O.rne_bf16
    q = 2.0 ** -8
    X = np.array([[1 + q, -(2 + 3 * q)], [0.75 + q / 4, 1 + 3 * q]])
    W1 = np.array([[1 + q, 0.5 + q / 2], [0.25 + q / 8, -(1 + 3 * q)]])
    b1 = np.array([2.0 ** -9, -0.1])
    W2 = np.array([[1.5 + q, -1.0], [-0.5 - q / 2, 0.75]])
    b2 = np.array([0.01, -0.02])
    y = np.array([1, 0])
    w = np.concatenate([W1.ravel(), b1, W2.ravel(), b2])
    loss, g = O.loss_and_grad(w, (2, 2, 2), X, y, bf16=True)
    gW1, gb1, gW2, gb2 = np.zeros((2, 2)), np.zeros(2), np.zeros((2, 2)), np.zeros(2)
    losses = []
    for b in range(2):
        xq = [r(v) for v in X[b]]
        z1 = [sum(xq[i] * r(W1[i, j]) for i in range(2)) + b1[j] for j in range(2)]
        hq = [r(max(v, 0.0)) for v in z1]
        z2 = [sum(hq[i] * r(W2[i, c]) for i in range(2)) + b2[c] for c in range(2)]
        m = max(z2)
        e = [math.exp(v - m) for v in z2]
        losses.append(math.log(sum(e)) + m - z2[y[b]])
        dz2q = [r((e[c] / sum(e) - (c == y[b])) / 2) for c in range(2)]
        for c in range(2):
            gb2[c] += dz2q[c]
            for i in range(2):
                gW2[i, c] += hq[i] * dz2q[c]
        dz1q = [r(sum(dz2q[c] * r(W2[j, c]) for c in range(2)) * (z1[j] > 0))
                for j in range(2)]
        for j in range(2):
            gb1[j] += dz1q[j]
            for i in range(2):
                gW1[i, j] += xq[i] * dz1q[j]
    assert z1[0] > 0 and z1[1] < 0            # the second sample's dead unit
    want = np.concatenate([gW1.ravel(), gb1, gW2.ravel(), gb2])
    np.testing.assert_allclose(g, want, rtol=1e-14, atol=1e-17)
    assert abs(loss - np.mean(losses)) <= 1e-14


# ------------------------------------------------------------------ loss
def _exact_ce(z, y):
    with decimal.localcontext() as ctx:
        ctx.prec = 60
        zs = [decimal.Decimal(float(v)) for v in z]
        m = max(zs)
        s = sum((v - m).exp() for v in zs)
        return float(m + s.ln() - zs[y])


def test_cross_entropy_against_high_precision():
    rng = np.random.default_rng(11)
    z = rng.standard_normal((40, 10)) * np.linspace(0.1, 40, 40)[:, None]
    y = rng.integers(0, 10, 40)
    # rows where the true class wins by a wide margin: loss near 1e-15
    z[:5, :] = 0.0
    z[np.arange(5), y[:5]] = np.linspace(20, 35, 5)
    loss, p = O.cross_entropy(z, y)
    for i in range(40):
        ref = _exact_ce(z[i], y[i])
        assert abs(loss[i] - ref) <= 1e-14 * max(ref, 1e-300) + 1e-300, (i, loss[i], ref)
    np.testing.assert_allclose(p.sum(1), 1.0, rtol=1e-15)


def test_initial_loss_is_log_of_classes():
    """Classifier weights ~ N(0, 0.01^2) give near-uniform softmax: loss ~ ln 10."""
    wl = wk.get("softmax_d64")
    X, y = wk.dataset(wl)
    loss, _ = O.loss_and_grad(wk.initial_weights(wl).astype(np.float64),
                              wl.widths, X[:512].astype(np.float64), y[:512])
    assert abs(loss - math.log(10.0)) < 0.1


# ------------------------------------------------------------------ gradient
@pytest.mark.parametrize("widths", [(5, 3), (6, 5, 4, 3), (7, 9, 3)])
def test_gradient_matches_central_differences(widths):
    rng = np.random.default_rng(sum(widths))
    P = wk.param_count(widths)
    w = rng.standard_normal(P) * 0.7
    A0 = rng.standard_normal((8, widths[0]))
    y = rng.integers(0, widths[-1], 8)
    _, g = O.loss_and_grad(w, widths, A0, y)
    eps = 1e-6
    fd = np.empty(P)
    for i in range(P):
        wp, wm = w.copy(), w.copy()
        wp[i] += eps
        wm[i] -= eps
        fd[i] = (O.loss_and_grad(wp, widths, A0, y)[0] -
                 O.loss_and_grad(wm, widths, A0, y)[0]) / (2 * eps)
    assert np.max(np.abs(fd - g)) <= 1e-7 * max(1.0, np.max(np.abs(g)))


def test_softmax_regression_gradient_closed_form():
    """For one layer the gradient is X^T (P - Y) / B and 1^T (P - Y) / B."""
    rng = np.random.default_rng(4)
    d, C, B = 6, 4, 10
    W = rng.standard_normal((d, C))
    b = rng.standard_normal(C)
    X = rng.standard_normal((B, d))
    y = rng.integers(0, C, B)
    Z = X @ W + b
    P = np.exp(Z - Z.max(1, keepdims=True))
    P /= P.sum(1, keepdims=True)
    Y = np.eye(C)[y]
    _, g = O.loss_and_grad(np.concatenate([W.ravel(), b]), (d, C), X, y)
    np.testing.assert_allclose(g[:d * C].reshape(d, C), X.T @ (P - Y) / B,
                               rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g[d * C:], (P - Y).sum(0) / B, rtol=1e-12,
                               atol=1e-15)


# ------------------------------------------------------------------ update
@pytest.mark.parametrize("nesterov", [False, True])
def test_local_momentum_closed_form_constant_gradient(nesterov):
    """H local momentum steps with a constant gradient g.

    Heavy ball follows the expansion of the local-momentum appendix:
    w_H = w_0 - lr (sum_{tau=1..H} m^tau u_0 + sum_{h=0..H-1} sum_{tau=0..H-1-h}
    m^tau g). Nesterov (d = g + m u) with u_0 = 0 sums to
    w_H = w_0 - lr g (H - m^2 (1 - m^H) / (1 - m)) / (1 - m).
    """
    rng = np.random.default_rng(5)
    w0 = rng.standard_normal(50)
    g = rng.standard_normal(50)
    u0 = rng.standard_normal(50) if not nesterov else np.zeros(50)
    lr, m, H = 0.07, 0.9, 13
    w, u = w0.copy(), u0.copy()
    for _ in range(H):
        w, u = O.sgd_update(w, u, g, lr, m, 0.0, nesterov)
    if nesterov:
        want = w0 - lr * g * (H - m * m * (1 - m**H) / (1 - m)) / (1 - m)
    else:
        acc = sum(m**tau for tau in range(1, H + 1)) * u0
        acc = acc + sum(sum(m**tau for tau in range(H - h)) for h in range(H)) * g
        want = w0 - lr * acc
    np.testing.assert_allclose(w, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("nesterov", [False, True])
def test_weight_decay_is_a_linear_recurrence(nesterov):
    """Zero loss gradient, decay lam: (w, u) evolves by a fixed 2x2 matrix."""
    lr, m, lam, H = 0.3, 0.8, 0.05, 25
    if nesterov:
        M = np.array([[1 - lr * lam * (1 + m), -lr * m * m], [lam, m]])
    else:
        M = np.array([[1 - lr * lam, -lr * m], [lam, m]])
    w, u = np.array([1.5, -2.0]), np.array([0.25, 0.5])
    want = np.linalg.matrix_power(M, H) @ np.stack([w, u])
    for _ in range(H):
        w, u = O.sgd_update(w, u, np.zeros(2), lr, m, lam, nesterov)
    np.testing.assert_allclose(np.stack([w, u]), want, rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------------ average
def test_average_identity_invariance_and_delta_form():
    rng = np.random.default_rng(6)
    w = rng.standard_normal(33)
    same = np.repeat(w[None], 8, axis=0)
    np.testing.assert_allclose(O.average(same), same, rtol=4e-16, atol=0)
    W = rng.standard_normal((8, 33))
    A = O.average(W)
    np.testing.assert_allclose(A.mean(0), W.mean(0), rtol=1e-14, atol=1e-15)
    assert np.all(A == A[0])
    np.testing.assert_allclose(O.average_delta_form(same, W), A,
                               rtol=1e-13, atol=1e-14)
    np.testing.assert_array_equal(O.average(W[:1]), W[:1])   # K = 1


# ------------------------------------------------------------------ method
def _small(nesterov, momentum=0.9, wd=1e-3, K=4, H=1, B=8, rounds=3):
    base = wk.get("softmax_d64")
    return base.scaled(widths=(64, 12, 10), K=K, B_loc=B, H=H, rounds=rounds,
                       lr=0.05, momentum=momentum, nesterov=nesterov,
                       weight_decay=wd)


@pytest.mark.parametrize("nesterov,momentum", [(False, 0.0), (False, 0.9),
                                               (True, 0.9)])
def test_h1_local_sgd_is_minibatch_sgd(nesterov, momentum):
    """H = 1 with averaging after each step equals mini-batch SGD with batch
    K*B_loc (introduction, below eq. 2), including coupled decay and, by
    linearity of the buffers, heavy-ball and Nesterov momentum."""
    wl = _small(nesterov, momentum, H=1, rounds=6)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(1).standard_normal(wk.param_count(wl.widths)) * 0.1
    st, _ = O.run(wl, X, y, w0)
    ref = O.minibatch_sgd(wl, X, y, w0, steps=6, lr=wl.lr)
    np.testing.assert_allclose(st.W[0], ref, rtol=1e-12, atol=1e-13)


def test_h1_local_sgd_is_minibatch_sgd_with_the_epoch_sampler():
    """The same identity with the per-epoch reshuffled partition, across an
    epoch boundary (the union batch is drawn without replacement)."""
    wl = _small(False, 0.9, K=4, H=1, B=8, rounds=40).scaled(sampler="epoch", N=400)
    X, y = wk.dataset(wl)
    assert O.steps_per_epoch(wl.K, wl.N, wl.B_loc) < 40
    w0 = np.random.default_rng(5).standard_normal(wk.param_count(wl.widths)) * 0.1
    st, _ = O.run(wl, X, y, w0)
    ref = O.minibatch_sgd(wl, X, y, w0, steps=40, lr=wl.lr)
    np.testing.assert_allclose(st.W[0], ref, rtol=1e-11, atol=1e-12)


def test_single_worker_is_sequential_sgd():
    wl = _small(False, 0.9, K=1, H=4, rounds=3)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(2).standard_normal(wk.param_count(wl.widths)) * 0.1
    st, _ = O.run(wl, X, y, w0)
    ref = O.minibatch_sgd(wl, X, y, w0, steps=12, lr=wl.lr)
    np.testing.assert_allclose(st.W[0], ref, rtol=1e-12, atol=1e-13)


def test_post_local_limits():
    """t' >= T is mini-batch SGD; t' = 0 is local SGD (section 3)."""
    X, y = wk.dataset(wk.get("softmax_d64"))
    w0 = np.random.default_rng(3).standard_normal(wk.param_count((64, 12, 10))) * 0.1
    warm_only = _small(True, 0.9, H=4, rounds=0).scaled(warm_rounds=5,
                                                        lr_after_switch=0.005)
    st, traj = O.run(warm_only, X, y, w0)
    assert [t.shape[0] for t in traj] == [1] * 5
    np.testing.assert_allclose(
        st.W[0], O.minibatch_sgd(warm_only, X, y, w0, 5, warm_only.lr),
        rtol=1e-12, atol=1e-13)
    # a switch after 2 warm rounds = 2 H=1 rounds, then H=4 rounds at lr/10
    post = _small(True, 0.9, H=4, rounds=2).scaled(warm_rounds=2,
                                                   lr_after_switch=0.005)
    assert O.schedule(post) == [(1, 0.05), (1, 0.05), (4, 0.005), (4, 0.005)]
    assert O.schedule(post.scaled(warm_rounds=0)) == [(4, 0.05), (4, 0.05)]


def test_momentum_buffers_stay_local():
    """Averaging touches the models only; each worker keeps its own u^k."""
    wl = _small(False, 0.9, H=3, rounds=1)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(4).standard_normal(wk.param_count(wl.widths)) * 0.1
    st, manual = O.State(w0, wl.K), O.State(w0, wl.K)
    O.run_round(st, wl, X, y, 3, wl.lr)
    for _ in range(3):
        O.local_step(manual, wl, X, y, wl.lr)
    np.testing.assert_array_equal(st.U, manual.U)
    assert not np.allclose(st.U[0], st.U[1])
    np.testing.assert_allclose(st.W[1], manual.W.mean(0), rtol=1e-15, atol=1e-16)


def test_round_matches_local_momentum_expansion():
    """After one round, each replica obeys the local-momentum expansion of
    the appendix: w^k_H = w^k_0 - lr (sum_tau m^tau u^k_0 + sum_h
    (sum_{tau<H-h} m^tau) grad^k_h); checked with decay off, using the
    replica's own per-step gradients."""
    wl = _small(False, 0.9, wd=0.0, H=5, rounds=1)
    X, y = wk.dataset(wl)
    rng = np.random.default_rng(8)
    w0 = rng.standard_normal(wk.param_count(wl.widths)) * 0.1
    st = O.State(w0, wl.K)
    st.U = rng.standard_normal(st.U.shape) * 0.01
    st.step = 40
    U0 = st.U.copy()
    W0 = st.W.copy()
    grads = [[None] * wl.K for _ in range(wl.H)]
    for h in range(wl.H):
        for k in range(wl.K):
            idx = O.sample_indices(wl.sample_seed, st.step, k, wl.K, wl.N, wl.B_loc)
            grads[h][k] = O.loss_and_grad(st.W[k], wl.widths, X[idx].astype(float),
                                          y[idx])[1]
        O.local_step(st, wl, X, y, wl.lr)
    m, H = wl.momentum, wl.H
    for k in range(wl.K):
        acc = sum(m**t for t in range(1, H + 1)) * U0[k]
        for h in range(H):
            acc = acc + sum(m**t for t in range(H - h)) * grads[h][k]
        np.testing.assert_allclose(st.W[k], W0[k] - wl.lr * acc, rtol=1e-11,
                                   atol=1e-13)


def test_replicas_are_independent_between_averages():
    wl = _small(True, 0.9, H=2, rounds=1)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(9).standard_normal(wk.param_count(wl.widths)) * 0.1
    a, b = O.State(w0, wl.K), O.State(w0, wl.K)
    for _ in range(2):
        O.local_step(a, wl, X, y, wl.lr)
        O.local_step(b, wl, X, y, wl.lr, replicas=[2])
    np.testing.assert_array_equal(a.W[2], b.W[2])
    np.testing.assert_array_equal(b.W[0], np.asarray(w0, float))


# ---------------------------------------------------- hierarchical local SGD
@pytest.mark.parametrize("K,Kb", [(8, 1), (8, 2), (8, 4), (8, 8), (6, 3)])
def test_block_average_structure(K, Kb):
    """Block synchronisation (Appendix D): members of a block of Kb
    consecutive workers become equal, the mean over all workers is kept,
    Kb = 1 is the identity, Kb = K is the global average, and a second block
    average changes nothing."""
    W = np.random.default_rng(K * 10 + Kb).standard_normal((K, 37))
    A = O.average_blocks(W, Kb)
    for b in range(K // Kb):
        blk = A[b * Kb:(b + 1) * Kb]
        np.testing.assert_array_equal(blk, np.broadcast_to(blk[0], blk.shape))
    np.testing.assert_allclose(A.mean(0), W.mean(0), rtol=1e-13, atol=1e-15)
    if Kb == 1:
        np.testing.assert_array_equal(A, W)
    if Kb == K:
        np.testing.assert_allclose(A, O.average(W), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(O.average_blocks(A, Kb), A, rtol=1e-14, atol=1e-15)
    if 1 < Kb < K:  # different blocks differ before the global average
        assert not np.allclose(A[0], A[Kb])
    with pytest.raises(ValueError):
        O.average_blocks(W, 5)


@pytest.mark.parametrize("nesterov", [False, True])
def test_hierarchical_limits_are_local_sgd(nesterov):
    """Appendix D's limits, against the separately pinned local SGD rounds:
    K' = K makes every block step a global average (H^b rounds of local SGD
    with period H); K' = 1 leaves only the global average (one round of
    H * H^b local steps); H^b = 1 is one round of period H for any K' --
    the mean of equal-sized block means is the global mean."""
    wl = _small(nesterov, 0.9, K=8, H=2, B=6, rounds=1)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(21).standard_normal(wk.param_count(wl.widths)) * 0.1
    H, Hb = 2, 3

    def pair():
        return O.State(w0, wl.K), O.State(w0, wl.K)

    a, b = pair()
    O.run_hierarchical_round(a, wl, X, y, H, Hb, wl.K, wl.lr)
    for _ in range(Hb):
        O.run_round(b, wl, X, y, H, wl.lr)
    np.testing.assert_allclose(a.W, b.W, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(a.U, b.U, rtol=1e-12, atol=1e-14)

    a, b = pair()
    O.run_hierarchical_round(a, wl, X, y, H, Hb, 1, wl.lr)
    O.run_round(b, wl, X, y, H * Hb, wl.lr)
    np.testing.assert_allclose(a.W, b.W, rtol=1e-12, atol=1e-14)

    for Kb in (2, 4):
        a, b = pair()
        O.run_hierarchical_round(a, wl, X, y, H, 1, Kb, wl.lr)
        O.run_round(b, wl, X, y, H, wl.lr)
        np.testing.assert_allclose(a.W, b.W, rtol=1e-12, atol=1e-14)


def test_hierarchical_round_blocks_between_global_averages():
    """Within an outer round, the blocks evolve separately: after the first
    block step, workers of one block agree and the blocks differ; after the
    round every worker holds the global mean, and buffers stay local."""
    wl = _small(False, 0.9, K=8, H=2, B=6, rounds=1)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(22).standard_normal(wk.param_count(wl.widths)) * 0.1
    st = O.State(w0, wl.K)
    for _ in range(2):
        O.local_step(st, wl, X, y, wl.lr)
    blk = O.average_blocks(st.W, 4)
    np.testing.assert_array_equal(blk[0], blk[3])
    assert not np.allclose(blk[0], blk[4])
    st2 = O.State(w0, wl.K)
    O.run_hierarchical_round(st2, wl, X, y, 2, 2, 4, wl.lr)
    np.testing.assert_array_equal(st2.W, np.broadcast_to(st2.W[0], st2.W.shape))
    assert not np.allclose(st2.U[0], st2.U[1])


# ------------------------------------------------- global / hybrid momentum
def test_global_momentum_average_closed_forms():
    """The global-momentum synchronisation against its rearranged closed
    forms: with all replicas starting the round at w_(t), the new model is
    the plain mean minus lr * m_g * u_(t-1), and the buffer gains the mean
    model change over lr. m_g = 0 is the plain average of eq. (2)."""
    rng = np.random.default_rng(41)
    K, P, lr, mg = 5, 33, 0.05, 0.7
    W = rng.standard_normal((K, P))
    w_sync = rng.standard_normal(P)
    u = rng.standard_normal(P)
    Wn, wn, un = O.average_global_momentum(W, w_sync, u, mg, lr)
    mean = W.mean(axis=0)
    np.testing.assert_allclose(wn, mean - lr * mg * u, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(un, mg * u + (w_sync - mean) / lr, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(Wn, np.broadcast_to(wn, (K, P)))
    W0, _, _ = O.average_global_momentum(W, w_sync, u, 0.0, lr)
    np.testing.assert_allclose(W0, O.average(W), rtol=1e-12, atol=1e-13)


def test_global_momentum_h1_is_minibatch_heavy_ball():
    """H = 1 without local momentum: the mean model change over lr is the
    mean gradient (coupled decay included), so local SGD with global
    momentum m_g is mini-batch SGD with heavy-ball momentum m_g on the
    union batch -- the block-momentum view of the global-momentum
    paragraph."""
    base = _small(False, 0.0, H=1, rounds=6)
    X, y = wk.dataset(base)
    w0 = np.random.default_rng(42).standard_normal(wk.param_count(base.widths)) * 0.1
    for mg in (0.5, 0.9):
        st, _ = O.run(base.scaled(global_momentum=mg), X, y, w0)
        ref = O.minibatch_sgd(base.scaled(momentum=mg), X, y, w0, steps=6, lr=base.lr)
        np.testing.assert_allclose(st.W[0], ref, rtol=1e-10, atol=1e-12)
        assert not np.allclose(st.W[0], O.minibatch_sgd(base, X, y, w0, 6, base.lr))


def test_hybrid_momentum_first_round_and_buffers():
    """Hybrid momentum (local buffers plus the global one): the global buffer
    starts at zero, so the first round ends at the plain average; from the
    second round on the models differ by -lr * m_g * u_(1), with u_(1) the
    first round's mean model change over lr. Local buffers stay local."""
    wl = _small(True, 0.9, H=3, rounds=2)
    hyb = wl.scaled(global_momentum=0.4)
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(43).standard_normal(wk.param_count(wl.widths)) * 0.1
    a, b = O.State(w0, wl.K), O.State(w0, wl.K)
    O.run_round(a, hyb, X, y, 3, wl.lr)
    O.run_round(b, wl, X, y, 3, wl.lr)
    np.testing.assert_allclose(a.W, b.W, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(a.u_global, (w0 - b.W[0]) / wl.lr, rtol=1e-10, atol=1e-10)
    np.testing.assert_array_equal(a.U, b.U)
    assert not np.allclose(a.U[0], a.U[1])
    # second round from the same start: the end models differ by the momentum term
    c = O.State(w0, wl.K)
    c.W, c.U, c.step = a.W.copy(), a.U.copy(), a.step
    c.w_sync = a.w_sync.copy()
    O.run_round(a, hyb, X, y, 3, wl.lr)
    O.run_round(c, wl, X, y, 3, wl.lr)
    np.testing.assert_allclose(a.W[0], c.W[0] - wl.lr * 0.4 * (w0 - b.W[0]) / wl.lr,
                               rtol=1e-9, atol=1e-12)


# ------------------------------------------- sign-compressed synchronisation
def test_sign_compressor_properties():
    """sign(0) = 0 and zeros count in the model size d; a difference whose
    entries share one magnitude passes unchanged; without zeros the message
    keeps the l1 norm and its residual is orthogonal to the sign vector
    (p = ||delta||_1 / d is then the l2-optimal scale of s)."""
    s_, p_ = O.compress_sign(np.array([2.0, 0.0, -2.0, 0.0]))
    np.testing.assert_array_equal(s_, [1.0, 0.0, -1.0, 0.0])
    assert p_ == 1.0
    rng = np.random.default_rng(61)
    flat = 0.25 * np.where(rng.random(1000) < 0.5, -1.0, 1.0)
    s_, p_ = O.compress_sign(flat)
    np.testing.assert_array_equal(s_ * p_, flat)
    delta = rng.standard_normal(997)
    s_, p_ = O.compress_sign(delta)
    np.testing.assert_allclose(np.abs(s_ * p_).sum(), np.abs(delta).sum(), rtol=1e-13)
    np.testing.assert_allclose(np.dot(s_, delta - s_ * p_), 0.0, atol=1e-10)
    c = np.dot(s_, delta) / np.dot(s_, s_)
    np.testing.assert_allclose(c, p_, rtol=1e-13)


def test_sign_sync_without_memory_and_constant_magnitudes_is_the_average():
    """If every worker's difference has one magnitude per worker and no
    zeros, Algorithm 3's synchronisation is exactly the plain average."""
    rng = np.random.default_rng(62)
    K, P = 4, 64
    w_sync = rng.standard_normal(P)
    mags = np.array([0.5, 0.25, 0.125, 0.0625])
    W = w_sync[None] - mags[:, None] * np.where(rng.random((K, P)) < 0.5, -1.0, 1.0)
    Wn, wn, E = O.average_sign_compressed(W, w_sync)
    assert E is None
    np.testing.assert_allclose(Wn, O.average(W), rtol=0, atol=1e-15)


def test_alg3_h1_is_signsgd_with_sign_averaging():
    """Algorithm 3 at H' = 1: each worker's round moves by lr * sign(d^k)
    exactly, so its message is that move and the synchronisation takes the
    average of the workers' signs -- signSGD with an average instead of a
    majority vote over signs, as the appendix on compression says. The
    reference below writes that update directly."""
    wl = _small(True, 0.9, K=4, H=1, B=8, rounds=5).scaled(scheme="sign")
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(63).standard_normal(wk.param_count(wl.widths)) * 0.1
    st, _ = O.run(wl, X, y, w0)
    w = w0.copy()
    u = np.zeros((wl.K, w.size))
    for s in range(5):
        signs = []
        for k in range(wl.K):
            idx = O.sample_indices(wl.sample_seed, s, k, wl.K, wl.N, wl.B_loc)
            _, grad = O.model_loss_and_grad(wl, w, np.asarray(X[idx], np.float64), y[idx])
            g = grad + wl.weight_decay * w
            u[k] = wl.momentum * u[k] + g
            signs.append(np.sign(g + wl.momentum * u[k]))
        w = w - wl.lr * np.mean(signs, axis=0)
    np.testing.assert_allclose(st.W[0], w, rtol=1e-12, atol=1e-13)


def test_alg4_local_steps_are_plain_and_memory_feeds_back():
    """Algorithm 4: the local steps are plain SGD steps (the replicas before
    the synchronisation equal those of local SGD), the memories start at 0,
    and error feedback telescopes: the model minus the mean memory moves by
    exactly the uncompressed mean model change of every round. Each memory
    is orthogonal to its sign vector and shorter than the corrected
    difference it came from."""
    wl = _small(False, 0.9, K=4, H=3, B=8, rounds=1).scaled(scheme="ef_sign")
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(64).standard_normal(wk.param_count(wl.widths)) * 0.1
    st, plain = O.State(w0, wl.K), O.State(w0, wl.K)
    tilde = st.w_sync - st.E.mean(axis=0)
    for t in range(4):
        for _ in range(3):
            O.local_step(st, wl, X, y, wl.lr)
            if t == 0:
                O.local_step(plain, wl.scaled(scheme="local"), X, y, wl.lr)
        if t == 0:
            np.testing.assert_array_equal(st.W, plain.W)
            assert not np.any(st.E)
        w_start, W_end, E_old = st.w_sync.copy(), st.W.copy(), st.E.copy()
        O.synchronise(st, wl, wl.lr)
        new_tilde = st.w_sync - st.E.mean(axis=0)
        np.testing.assert_allclose(new_tilde, tilde - (w_start - W_end.mean(axis=0)),
                                   rtol=1e-11, atol=1e-13)
        tilde = new_tilde
        for k in range(wl.K):
            delta = w_start - W_end[k] + E_old[k]
            s_ = np.sign(delta)
            np.testing.assert_allclose(np.dot(s_, st.E[k]), 0.0, atol=1e-12)
            assert np.linalg.norm(st.E[k]) < np.linalg.norm(delta)
        np.testing.assert_array_equal(st.W, np.broadcast_to(st.w_sync, st.W.shape))


def test_alg3_local_steps_move_by_signs():
    """Algorithm 3's local step moves every coordinate by exactly lr (the
    update direction has no zero entries here), unlike the plain step."""
    wl = _small(True, 0.9, K=2, H=1, B=8, rounds=1).scaled(scheme="sign")
    X, y = wk.dataset(wl)
    w0 = np.random.default_rng(65).standard_normal(wk.param_count(wl.widths)) * 0.1
    st = O.State(w0, wl.K)
    O.local_step(st, wl, X, y, wl.lr)
    np.testing.assert_allclose(np.abs(st.W - w0[None]), wl.lr, rtol=1e-9)


# ------------------------------------------- per-epoch reshuffle sampler
def _feistel_inverse(y, m, seed, epoch):
    """Undo the Feistel rounds (the network run backwards): a separate
    derivation, so the forward map is checked to be the permutation its
    definition says."""
    y = np.asarray(y, np.uint64)
    mask = np.uint64((1 << m) - 1)
    left, right = y >> np.uint64(m), y & mask
    for r in reversed(range(O.FEISTEL_ROUNDS)):
        f = O.philox4x32_10((left, np.full_like(left, r),
                             np.full_like(left, epoch & 0xFFFFFFFF),
                             np.full_like(left, O.SHUFFLE_STREAM)),
                            (seed & 0xFFFFFFFF, seed >> 32))[0]
        left, right = right ^ (f & mask), left
    return (left << np.uint64(m)) | right


@pytest.mark.parametrize("m", [1, 2, 3, 5, 8])
def test_feistel_is_a_permutation_with_its_inverse(m):
    for seed, epoch in ((0, 0), (2**64 - 1, 7), (12345, 2**31 + 5)):
        x = np.arange(1 << (2 * m), dtype=np.uint64)
        y = O.feistel(x, m, seed, epoch)
        assert np.array_equal(np.sort(y), x)
        assert np.array_equal(_feistel_inverse(y, m, seed, epoch), x)
        if m >= 3:
            assert not np.array_equal(y, x)


@pytest.mark.parametrize("N", [1, 2, 3, 5, 17, 1000, 4097, 50000])
def test_epoch_permutation_is_a_bijection_of_the_rows(N):
    for epoch in (0, 1, 99):
        pi = O.epoch_permutation(np.arange(N), N, 0x5EED, epoch)
        assert np.array_equal(np.sort(pi), np.arange(N))
    if N >= 17:
        a = O.epoch_permutation(np.arange(N), N, 0x5EED, 0)
        assert not np.array_equal(a, O.epoch_permutation(np.arange(N), N, 0x5EED, 1))
        assert not np.array_equal(a, O.epoch_permutation(np.arange(N), N, 0x5EEE, 0))


def test_epoch_sampler_partitions_each_epoch_disjointly():
    """Within an epoch no row is drawn twice across workers and steps, every
    worker's batches come from its part of that epoch's permutation, and the
    next epoch reshuffles (the parts change)."""
    K, N, B, seed = 4, 1000, 32, 99
    S = O.steps_per_epoch(K, N, B)
    assert S == 7
    for e in (0, 1):
        drawn = np.concatenate([O.sample_indices_epoch(seed, e * S + j, k, K, N, B)
                                for k in range(K) for j in range(S)])
        assert drawn.size == K * S * B == np.unique(drawn).size
        assert drawn.min() >= 0 and drawn.max() < N
        pi = O.epoch_permutation(np.arange(N), N, seed, e)
        for k in range(K):
            lo, hi = O.shard(k, K, N)
            mine = np.concatenate([O.sample_indices_epoch(seed, e * S + j, k, K, N, B)
                                   for j in range(S)])
            assert set(mine) <= set(pi[lo:hi])
    part0 = set(O.sample_indices_epoch(seed, 0, 0, K, N, B))
    part1 = set(O.sample_indices_epoch(seed, S, 0, K, N, B))
    assert part0 != part1
    with pytest.raises(ValueError):
        O.sample_indices_epoch(seed, 0, 0, 8, 100, 32)


def test_epoch_permutation_places_a_row_uniformly():
    """Over many epochs, row 0 lands in each of the N positions about
    equally often (chi-square)."""
    from scipy.stats import chisquare
    N, E = 10, 5000
    pos = np.array([int(np.argmax(O.epoch_permutation(np.arange(N), N, 7, e) == 0))
                    for e in range(E)])
    counts = np.bincount(pos, minlength=N)
    assert chisquare(counts).pvalue > 1e-4


# ------------------------------------------------------------- schedules
def test_goyal_warmup_matches_the_appendix_increment():
    """Five epochs of N / (K n) iterations from lr to k * lr with the
    appendix's per-iteration increment (k_hat lr - lr) / (5 N / (K n))."""
    K, n, S = 16, 128, 24
    N = S * K * n
    lr, scale = 0.1, K * n / 128
    warm = 5 * N // (K * n)
    inc = (scale * lr - lr) / (5 * N / (K * n))
    for s in (0, 1, 7, warm - 1):
        assert O.goyal_lr(s, lr, scale, warm) == pytest.approx(lr + s * inc, rel=1e-15)
    assert O.goyal_lr(warm, lr, scale, warm) == scale * lr
    assert O.goyal_lr(10 * warm, lr, scale, warm) == scale * lr
    assert O.goyal_lr(0, lr, scale, 0) == scale * lr


def test_step_decay_at_half_and_three_quarters_of_the_samples():
    spp, T = 2048, 2048 * 100
    f = [O.decay_factor(s, spp, T) for s in range(100)]
    assert f[:50] == [1.0] * 50
    assert all(v == pytest.approx(0.1) for v in f[50:75])
    assert all(v == pytest.approx(0.01) for v in f[75:])


def test_local_step_warmup_kinds():
    """The ImageNet example (fixture) for the exponential warm-up; linear
    and constant warm-up by their definitions' end points and monotonicity."""
    path = os.path.join(os.path.dirname(__file__), "golden", "local_step_warmup_imagenet.txt")
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        head, tail = line.split(":")
        kind, H, W = head.split()
        want = [int(v) for v in tail.split()]
        got = [O.local_steps_of_epoch(e, int(H), kind, int(W)) for e in range(len(want))]
        assert got == want
    lin = [O.local_steps_of_epoch(e, 16, "linear", 4) for e in range(6)]
    assert lin == [1, 4, 8, 12, 16, 16]
    assert [O.local_steps_of_epoch(e, 16, "constant", 3) for e in range(5)] == [1, 1, 1, 16, 16]
    assert [O.local_steps_of_epoch(e, 16, None, 3) for e in range(3)] == [16] * 3


@pytest.mark.parametrize("kind", [None, "linear", "exponential", "constant"])
def test_schedule_rounds_keep_the_sample_budget(kind):
    S, total, H = 24, 24 * 10 + 5, 16
    rounds = O.schedule_rounds(total, S, H, lambda s: 0.1 * (s + 1), h_kind=kind,
                               h_warmup_epochs=3)
    assert sum(h for h, _ in rounds) == total
    s = 0
    for h, lrs in rounds:
        want = O.local_steps_of_epoch(s // S, H, kind, 3)
        assert h == want or (h < want and s + h == total)
        assert lrs == [0.1 * (s + i + 1) for i in range(h)]
        s += h
    pl = O.schedule_rounds(total, S, H, lambda s: 1.0, switch_step=100)
    assert [h for h, _ in pl[:100]] == [1] * 100 and pl[100][0] == H
    assert sum(h for h, _ in pl) == total


def test_loss_decreases_on_every_workload_first_rounds():
    wl = wk.get("softmax_d64")
    X, y = wk.dataset(wl)
    _, traj = O.run(wl, X, y, wk.initial_weights(wl), rounds=10)
    means = [t.mean() for t in traj]
    assert means[-1] < 0.2 * means[0]


# ------------------------------------------------------------------ ResNet-20
def test_resnet20_shape_matches_table5():
    """Table 5: ResNet-20 (CIFAR-10) has 0.27 M parameters and 0.041 G
    multiply-adds per image; the network built here has 269,722 and
    40,551,040."""
    a = O.resnet_arch()
    assert O.resnet_param_count(a) == 269722
    assert O.resnet_macs_per_image(a) == 40551040
    assert round(O.resnet_param_count(a) / 1e6, 2) == 0.27
    assert round(O.resnet_macs_per_image(a) / 1e9, 3) == 0.041
    assert len(O.resnet_convs(a)) == 19          # 1 + 3 stages x 3 blocks x 2


def test_conv3x3_against_direct_loops():
    rng = np.random.default_rng(21)
    for stride in (1, 2):
        x = rng.standard_normal((2, 5, 6, 3))
        W = rng.standard_normal((3, 3, 3, 4))
        y, _ = O.conv3x3(x, W, stride)
        Ho, Wo = (5 + 2 - 3) // stride + 1, (6 + 2 - 3) // stride + 1
        assert y.shape == (2, Ho, Wo, 4)
        ref = np.zeros_like(y)
        for b in range(2):
            for i in range(Ho):
                for j in range(Wo):
                    for kh in range(3):
                        for kw in range(3):
                            r, c = i * stride + kh - 1, j * stride + kw - 1
                            if 0 <= r < 5 and 0 <= c < 6:
                                ref[b, i, j] += x[b, r, c] @ W[kh, kw]
        np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_batchnorm_normalises_per_channel():
    rng = np.random.default_rng(22)
    x = rng.standard_normal((4, 3, 3, 5)) * 3 + 2
    y, _ = O.batchnorm(x, np.ones(5), np.zeros(5))
    np.testing.assert_allclose(y.mean(axis=(0, 1, 2)), 0, atol=1e-12)
    var = x.var(axis=(0, 1, 2))
    np.testing.assert_allclose(y.var(axis=(0, 1, 2)), var / (var + O.BN_EPS), rtol=1e-10)


def test_resnet_gradient_matches_central_differences():
    """Tiny ResNet (4x4 images, channels 2/4/8, one block per stage): every
    parameter, including BN scales and shifts, stride-2 convolutions and the
    zero-padded shortcuts."""
    a = O.resnet_arch(side=4, cin=2, base=2, blocks=1, classes=3)
    P = O.resnet_param_count(a)
    rng = np.random.default_rng(23)
    w = rng.standard_normal(P) * 0.5
    A0 = rng.standard_normal((6, 4 * 4 * 2))
    y = rng.integers(0, 3, 6)
    _, g = O.resnet_loss_and_grad(w, a, A0, y)
    eps = 1e-6
    fd = np.empty(P)
    for i in range(P):
        wp, wm = w.copy(), w.copy()
        wp[i] += eps
        wm[i] -= eps
        fd[i] = (O.resnet_loss_and_grad(wp, a, A0, y)[0] -
                 O.resnet_loss_and_grad(wm, a, A0, y)[0]) / (2 * eps)
    assert np.max(np.abs(fd - g)) <= 1e-6 * max(1.0, np.max(np.abs(g)))


def test_resnet_decay_mask_exempts_batchnorm():
    a = O.resnet_arch()
    m = O.resnet_decay_mask(a)
    n_bn = sum(int(np.prod(s)) for nme, s, _ in O.resnet_layout(a)
               if nme.endswith(".g") or nme.endswith(".be"))
    assert m.size == 269722 and int((m == 0).sum()) == n_bn == 2 * (16 * 7 + 32 * 6 + 64 * 6)


# --------------------------------------- ResNet against torch's autograd / BN
def _torch_resnet(arch, w, bns=None):
    """The CIFAR ResNet of the oracle's architecture written with torch's
    functional ops (CPU, fp64) from the flat parameter vector, with its own
    unpacking: per 3x3 convolution (stem, then two per block) the weight
    [3][3][c_in][c_out], BN scale and shift; then the classifier [c][classes]
    and bias. BN is torch's training-mode batch_norm (momentum 0.1) on
    running-statistic buffers that persist across calls when ``bns`` (a list
    of (running mean, running variance) pairs) is passed back in. Returns
    (forward(x_nhwc, labels) -> mean loss, parameters as leaf tensors in
    vector order, the BN buffers)."""
    import torch
    import torch.nn.functional as F
    convs, c = [(arch["cin"], arch["base"], 1)], arch["base"]
    for s in range(3):
        co = arch["base"] * 2 ** s
        for b in range(arch["blocks"]):
            convs += [(c, co, 2 if (s > 0 and b == 0) else 1), (co, co, 1)]
            c = co
    params, o = [], 0
    w = np.asarray(w, np.float64)

    def take(shape):
        nonlocal o
        n = int(np.prod(shape))
        t = torch.tensor(w[o:o + n].reshape(shape), dtype=torch.float64, requires_grad=True)
        o += n
        params.append(t)
        return t
    layers = [(take((3, 3, ci, co)), take((co,)), take((co,)), st) for ci, co, st in convs]
    fcw, fcb = take((c, arch["classes"])), take((arch["classes"],))
    assert o == w.size
    if bns is None:
        bns = [(torch.zeros(co, dtype=torch.float64), torch.ones(co, dtype=torch.float64))
               for _, co, _ in convs]

    def cbr(x, i):
        Wt, g, be, st = layers[i]
        y = F.conv2d(x, Wt.permute(3, 2, 0, 1), stride=st, padding=1)
        return F.batch_norm(y, bns[i][0], bns[i][1], weight=g, bias=be, training=True,
                            momentum=0.1, eps=1e-5)

    def forward(x_nhwc, labels):
        x = torch.tensor(x_nhwc, dtype=torch.float64).permute(0, 3, 1, 2)
        h = torch.relu(cbr(x, 0))
        for i in range(1, len(convs), 2):
            ci, co, st = convs[i]
            a = torch.relu(cbr(h, i))
            b = cbr(a, i + 1)
            sc = h if (st == 1 and ci == co) else \
                F.pad(h[:, :, ::2, ::2], (0, 0, 0, 0, 0, co - ci))
            h = torch.relu(b + sc)
        z = h.mean(dim=(2, 3)) @ fcw + fcb
        return F.cross_entropy(z, torch.tensor(labels, dtype=torch.long))
    return forward, params, bns


def test_resnet_loss_gradient_and_batch_statistics_match_torch():
    """A small ResNet (8x8 images, channels 4/8/16, two blocks per stage) in
    torch's autograd with its BatchNorm2d (training mode): the same mean loss,
    the same gradient of every parameter, and the batch statistics the oracle
    reports per BN layer give torch's running statistics."""
    torch = pytest.importorskip("torch")
    a = O.resnet_arch(side=8, cin=3, base=4, blocks=2, classes=5)
    rng = np.random.default_rng(31)
    P = O.resnet_param_count(a)
    w = rng.standard_normal(P) * 0.4
    A0 = rng.standard_normal((6, 8 * 8 * 3))
    y = rng.integers(0, 5, 6)
    stats = []
    loss, g = O.resnet_loss_and_grad(w, a, A0, y, stats)
    fwd, params, bns = _torch_resnet(a, w)
    tl = fwd(A0.reshape(6, 8, 8, 3), y)
    tl.backward()
    tg = np.concatenate([p.grad.numpy().ravel() for p in params])
    assert abs(loss - tl.item()) <= 1e-12 * abs(loss)
    assert np.max(np.abs(g - tg)) <= 1e-10 * np.max(np.abs(tg))
    assert len(stats) == len(bns) == 1 + 3 * 2 * 2
    for (mu, var, n), (trm, trv) in zip(stats, bns):
        rm, rv = O.bn_running_update(np.zeros_like(mu), np.ones_like(var), mu, var, n)
        np.testing.assert_allclose(rm, trm.numpy(), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(rv, trv.numpy(), rtol=1e-12, atol=1e-14)


def test_bn_running_update_closed_form():
    """Repeating one batch T times: running mean (1 - 0.9^T) mu (from 0),
    running variance 0.9^T + (1 - 0.9^T) var n / (n - 1) (from 1)."""
    mu, var, n = np.array([0.3, -2.0]), np.array([1.5, 0.25]), 37
    rm, rv = np.zeros(2), np.ones(2)
    for _ in range(7):
        rm, rv = O.bn_running_update(rm, rv, mu, var, n)
    f = 0.9 ** 7
    np.testing.assert_allclose(rm, (1 - f) * mu, rtol=1e-14)
    np.testing.assert_allclose(rv, f + (1 - f) * var * n / (n - 1), rtol=1e-14)


def test_resnet20_running_statistics_per_worker_and_averaged():
    """The full ResNet-20 at 2 images per replica, K = 2, two local steps and
    the synchronisation: each replica's running statistics equal those of a
    torch ResNet-20 whose BatchNorm2d modules saw that replica's batches at
    that replica's weights, and the synchronisation leaves their mean in every
    replica."""
    torch = pytest.importorskip("torch")
    base = wk.get("resnet20")
    w = base.scaled(K=2, B_loc=2, N=64, H=2, momentum=0.9)
    X, y = wk.dataset(base)
    X, y = np.ascontiguousarray(X[:64]), np.ascontiguousarray(y[:64])
    st = O.State(wk.initial_weights(w), 2)
    arch = O.resnet_arch()
    bns = [None, None]
    for _ in range(2):
        W_before = st.W.copy()
        step = st.step
        O.local_step(st, w, X, y, w.lr)
        for k in range(2):
            fwd, _, bns[k] = _torch_resnet(arch, W_before[k], bns[k])
            idx = O.worker_indices(w, step, k)
            fwd(X[idx].reshape(2, 32, 32, 3).astype(np.float64), y[idx])
    half = st.RS.shape[1] // 2
    for k in range(2):
        for (_, o, c), (trm, trv) in zip(O.resnet_running_layout(arch), bns[k]):
            np.testing.assert_allclose(st.RS[k, o:o + c], trm.numpy(),
                                       rtol=1e-10, atol=1e-13)
            np.testing.assert_allclose(st.RS[k, half + o:half + o + c], trv.numpy(),
                                       rtol=1e-10)
    before = st.RS.copy()
    O.synchronise(st, w, w.lr)
    np.testing.assert_allclose(st.RS, np.repeat(before.mean(axis=0)[None], 2, axis=0),
                               rtol=1e-15, atol=0)
