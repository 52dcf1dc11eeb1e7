"""State blob (checkpoint / resume), failure detection and BN running
statistics of the HIP path, through the C ABI."""
import numpy as np
import pytest
import torch

import workloads as wk
from oracle import lsgd_oracle as O
from gpu_util import make_replicas, normwise, rel, device

pytestmark = pytest.mark.gpu


def _small(widths, K=3, B=20, N=999, H=3, momentum=0.9, nesterov=True, **kw):
    return wk.Workload(name="small", model="mlp", widths=widths, dtype="fp32", K=K,
                       B_loc=B, H=H, rounds=2, lr=0.02, momentum=momentum,
                       nesterov=nesterov, weight_decay=1e-3, data="custom", N=N,
                       sample_seed=0xC0FFEE + K, **kw)


def _small_data(w, seed=5):
    rng = np.random.default_rng(seed)
    C = w.widths[-1]
    mu = rng.standard_normal((C, w.widths[0]))
    y = rng.integers(0, C, w.N).astype(np.int32)
    X = (mu[y] + rng.standard_normal((w.N, w.widths[0]))).astype(np.float32)
    w0 = np.concatenate([
        np.concatenate([(rng.standard_normal(a * b) * np.sqrt(2.0 / a)),
                        rng.standard_normal(b) * 0.1])
        for a, b in wk.layer_shapes(w.widths)]).astype(np.float32)
    return X, y, w0


def _resnet_small(**kw):
    base = wk.get("resnet20")
    w = base.scaled(K=2, N=4096, H=2, **kw)
    X, y = wk.dataset(base)
    return w, np.ascontiguousarray(X[:4096]), np.ascontiguousarray(y[:4096])


CASES = {
    "mlp_ef_sign": lambda: _small((70, 48, 36, 10), K=4, B=12, scheme="ef_sign"),
    "mlp_global_momentum": lambda: _small((70, 48, 36, 10), K=4, B=12,
                                          global_momentum=0.3),
    "mlp_epoch_sampler": lambda: _small((70, 48, 10), K=3, B=8, N=400, sampler="epoch"),
}


def _setup(case):
    if case == "resnet20":
        w, X, y = _resnet_small()
        return w, X, y, wk.initial_weights(w)
    w = CASES[case]()
    X, y, w0 = _small_data(w, seed=len(case))
    return w, X, y, w0


@pytest.mark.parametrize("case", [*CASES, "resnet20"])
def test_state_blob_resumes_bit_exactly(case):
    """A context restored from lsgd_read_state's blob continues bit for bit:
    replicas, momentum buffers, losses, and the whole next blob (BN running
    statistics, synchronised model, global buffer, error memories and the
    step counter included)."""
    from paper_1808_07217_amd import lsgd as L
    w, X, y, w0 = _setup(case)
    print(f"state blob {case}", flush=True)
    H = w.H
    a = make_replicas(w, X, y, w0)
    for r in range(2):
        a.run_round([w.lr * (1 + 0.5 * r)] * H)
    blob = a.read_state().clone()
    la = torch.empty(H, w.K, device=device())
    a.run_round([w.lr] * H, la)
    c = make_replicas(w, X, y, w0)
    c.write_state(blob)
    assert c.step == 2 * H
    lc = torch.empty(H, w.K, device=device())
    c.run_round([w.lr] * H, lc)
    np.testing.assert_array_equal(la.cpu().numpy(), lc.cpu().numpy())
    ba, bc = a.read_state(), c.read_state()
    torch.cuda.synchronize()
    assert torch.equal(ba, bc)
    sa = L.parse_state(ba)
    for k in range(w.K):
        np.testing.assert_array_equal(sa["W"][k].cpu().numpy(), a.read_params(k).cpu().numpy())
        np.testing.assert_array_equal(sa["U"][k].cpu().numpy(), a.read_momentum(k).cpu().numpy())
    assert sa["step"] == 3 * H
    a.sync()
    c.sync()


def test_write_state_refuses_a_foreign_blob():
    """A blob of another configuration (different K, or damaged magic) is
    refused with LSGD_E_INVALID and changes nothing."""
    from paper_1808_07217_amd import lsgd as L
    w = _small((70, 48, 10), K=3, B=8)
    X, y, w0 = _small_data(w, seed=3)
    a = make_replicas(w, X, y, w0)
    a.run_round([w.lr] * 2)
    other = make_replicas(w.scaled(K=2), X, y, w0)
    before = a.read_params(0).cpu().numpy()
    with pytest.raises(L.LsgdError, match="invalid argument"):
        a.write_state(other.read_state())
    bad = a.read_state().clone()
    bad[0] ^= 1
    with pytest.raises(L.LsgdError, match="invalid argument"):
        a.write_state(bad)
    np.testing.assert_array_equal(a.read_params(0).cpu().numpy(), before)
    assert a.step == 2


@pytest.mark.parametrize("case", ["mlp_head", "mlp_xent", "softmax_single_launch",
                                  "resnet20"])
def test_nonfinite_loss_latches_and_clears_on_restore(case):
    """A NaN written into one replica's output-layer bias makes the next
    local step's loss non-finite: lsgd_sync then reports LSGD_E_NONFINITE
    (checked on the device inside the step, no host sync), keeps reporting it
    while the context goes on running, and a restored state clears it. Runs
    that stay finite never report it. (The output bias is chosen because a
    non-finite hidden weight need not reach the loss: the kernels' ReLU maps
    a NaN pre-activation to 0.)"""
    from paper_1808_07217_amd import lsgd as L
    if case == "resnet20":
        w, X, y = _resnet_small()
        w0 = wk.initial_weights(w)
    else:
        widths = {"mlp_head": (70, 48, 10), "mlp_xent": (70, 48, 45),
                  "softmax_single_launch": (64, 10)}[case]
        w = _small(widths, K=4, B=16, H=2)
        X, y, w0 = _small_data(w, seed=7)
    print(f"non-finite {case}", flush=True)
    reps = make_replicas(w, X, y, w0)
    if case == "softmax_single_launch":
        reps.profile(True)
    reps.run_round([w.lr] * w.H)
    reps.sync()                                   # finite so far
    good = reps.read_state().clone()
    p = reps.read_params(1)
    p[-1] = float("nan")                          # the last class's bias
    reps.write_params(p, replica=1)
    reps.run_round([w.lr] * w.H)
    with pytest.raises(L.NonFiniteLoss):
        reps.sync()
    reps.run_round([w.lr] * w.H)                  # the context stays usable
    with pytest.raises(L.NonFiniteLoss):
        reps.sync()
    if case == "softmax_single_launch":
        assert set(reps.profile_report()) == {"tiny_round_wide"}
    reps.write_state(good)
    reps.sync()
    reps.run_round([w.lr] * w.H)
    reps.sync()


def test_resnet20_bn_running_statistics_match_oracle():
    """Per-worker BN running statistics (K = 2 replicas at the workload's
    batch of 128 over a 4096-image subset): after every round of two local
    steps, each replica's running means and variances against the oracle's,
    which the synchronisation averages."""
    from paper_1808_07217_amd import lsgd as L
    w, X, y = _resnet_small()
    w0 = wk.initial_weights(w)
    reps = make_replicas(w, X, y, w0)
    st = O.State(w0, w.K)
    loss = torch.empty(2, w.K, device=device())
    for t in range(3):
        reps.run_round([w.lr] * 2, loss)
        want = O.run_round(st, w, X, y, 2, w.lr)
        assert np.all(rel(loss.cpu().numpy(), want) <= 1e-4), t
        s = L.parse_state(reps.read_state())
        got = s["RS"].cpu().numpy()
        assert got.shape == st.RS.shape == (2, 1376)
        err = normwise(got, st.RS)
        print(f"round {t}: running statistics {err:.3e}", flush=True)
        assert err <= 1e-5, t
        np.testing.assert_array_equal(got[0], got[1])   # averaged
