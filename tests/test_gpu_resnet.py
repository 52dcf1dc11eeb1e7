"""ResNet-20 workload: HIP path against the oracle through the C ABI."""
import numpy as np
import pytest
import torch

import workloads as wk
from oracle import lsgd_oracle as O
from gpu_util import make_replicas, normwise, rel, device

pytestmark = pytest.mark.gpu


def _compare(w, X, y, w0, steps, replicas, param_tol, loss_tol):
    reps = make_replicas(w, X, y, w0)
    st = O.State(w0, w.K)
    loss = torch.empty(w.K, device=device())
    worst = 0.0
    for s in range(steps):
        reps.local_step(w.lr, loss)
        ref = O.local_step(st, w, X, y, w.lr, replicas=replicas)
        got = loss.cpu().numpy()
        for k in replicas:
            assert rel(got[k], ref[k]) <= loss_tol, (s, k, got[k], ref[k])
            e = normwise(reps.read_params(k).cpu().numpy(), st.W[k])
            worst = max(worst, e)
            assert e <= param_tol, (s, k, e)
    return reps, st, worst


def test_resnet20_every_step():
    """ResNet-20 at the workload's batch (128 images per replica) on 2
    replicas over a 4096-image subset: every replica after every local step,
    then the average. (Smaller batches are not a fair check at a 1e-5 bar:
    with 8 or 32 images some channels' batch variance nearly vanishes and BN's
    1/sigma amplifies rounding -- perturbing the weights by 1e-7 moves the
    fp64 oracle's own gradients by 0.7-3% there, against 1.2e-6 at 128.)"""
    base = wk.get("resnet20")
    w = base.scaled(K=2, N=4096)
    X, y = wk.dataset(base)
    X, y = np.ascontiguousarray(X[:4096]), np.ascontiguousarray(y[:4096])
    w0 = wk.initial_weights(w)
    print("resnet20 K=2", flush=True)
    reps, st, worst = _compare(w, X, y, w0, 3, [0, 1], 1e-5, 1e-4)
    reps.average()
    st.W = O.average(st.W)
    e = normwise(reps.read_params(-1).cpu().numpy(), st.W[0])
    print(f"resnet20 K=2: worst step error {worst:.3e}, averaged {e:.3e}", flush=True)
    assert e <= 1e-5


def test_resnet20_odd_replica_count():
    """K = 3: the forward pass on one stream (an even replica count runs it
    as two halves on two streams), every replica after every local step,
    then the average."""
    base = wk.get("resnet20")
    w = base.scaled(K=3, N=4096)
    X, y = wk.dataset(base)
    X, y = np.ascontiguousarray(X[:4096]), np.ascontiguousarray(y[:4096])
    w0 = wk.initial_weights(w)
    print("resnet20 K=3", flush=True)
    reps, st, worst = _compare(w, X, y, w0, 2, [0, 1, 2], 1e-5, 1e-4)
    reps.average()
    st.W = O.average(st.W)
    e = normwise(reps.read_params(-1).cpu().numpy(), st.W[0])
    print(f"resnet20 K=3: worst step error {worst:.3e}, averaged {e:.3e}", flush=True)
    assert e <= 1e-5


def test_resnet20_batch_not_a_multiple_of_four():
    """B_loc = 10 (K = 2, 4096-image subset, three steps, then the average):
    the paths a batch of 128 never takes -- the stride-2 input gradients of
    stage 3 through the nine-tap row kernel (10 x 8 x 8 rows are not whole
    256-row parity-class tiles), BN statistics of stage 3 from a separate
    pass (its outputs are not whole 256-row chunks), and weight-gradient
    splits that divide 10. The sampler seed is one where perturbing the
    oracle's initial weights by 1e-7 moves its replicas by 3.4e-7 over these
    steps (small batches can put a channel's batch variance near zero)."""
    base = wk.get("resnet20")
    w = base.scaled(K=2, N=4096, B_loc=10, sample_seed=0x5EED0015)
    X, y = wk.dataset(base)
    X, y = np.ascontiguousarray(X[:4096]), np.ascontiguousarray(y[:4096])
    w0 = wk.initial_weights(w)
    print("resnet20 B=10", flush=True)
    reps, st, worst = _compare(w, X, y, w0, 3, [0, 1], 1e-5, 1e-4)
    reps.average()
    st.W = O.average(st.W)
    e = normwise(reps.read_params(-1).cpu().numpy(), st.W[0])
    print(f"resnet20 B=10: worst step error {worst:.3e}, averaged {e:.3e}", flush=True)
    assert e <= 1e-5


def test_resnet20_full_shape_first_steps():
    """Workload 5 at its real shape (K=16, B_loc=128): replicas 0 and 15 over
    the first two local steps."""
    w = wk.get("resnet20")
    X, y = wk.dataset(w)
    print("resnet20 full shape", flush=True)
    _, _, worst = _compare(w, X, y, wk.initial_weights(w), 2, [0, w.K - 1], 1e-5, 1e-3)
    print(f"resnet20 full shape: worst error {worst:.3e}", flush=True)


@pytest.mark.parametrize("variant", ["hybrid_epoch", "ef_sign"])
def test_resnet20_round_with_the_newer_schemes(variant):
    """ResNet-20 (K = 2, B = 128, a 4096-image subset) for one round of two
    local steps under hybrid momentum (local 0.9, global 0.3) with the
    per-epoch reshuffle sampler, and under EF-signSGD: the synchronised
    model against the oracle (for EF-signSGD, elements whose corrected
    difference is within the replicas' own fp32 error of zero may take
    either sign, as on the MLP)."""
    base = wk.get("resnet20")
    w = base.scaled(K=2, N=4096, H=2)
    w = (w.scaled(global_momentum=0.3, sampler="epoch") if variant == "hybrid_epoch"
         else w.scaled(scheme="ef_sign", nesterov=True))
    X, y = wk.dataset(base)
    X, y = np.ascontiguousarray(X[:4096]), np.ascontiguousarray(y[:4096])
    w0 = wk.initial_weights(w)
    print(f"resnet20 {variant}", flush=True)
    reps = make_replicas(w, X, y, w0)
    st = O.State(w0, w.K)
    loss = torch.empty(2, w.K, device=device())
    reps.run_round([w.lr] * 2, loss)
    want = [O.local_step(st, w, X, y, w.lr) for _ in range(2)]
    assert np.all(rel(loss.cpu().numpy(), np.stack(want)) <= 1e-4)
    scale = np.max(np.abs(st.W))
    if variant == "ef_sign":
        d = st.w_sync[None] - st.W
        p = np.abs(d).sum(axis=1) / d.shape[1]
        amb = np.abs(d) <= 1e-5 * scale
        allow = (2 * p[:, None] * amb).sum(axis=0) / w.K
    O.synchronise(st, w, w.lr)
    got = reps.read_params(0).cpu().numpy()
    err = np.abs(got - st.W[0])
    if variant == "ef_sign":
        assert np.all(err <= 1e-5 * scale + allow)
        assert np.max(err[allow == 0]) <= 1e-5 * scale
    else:
        assert normwise(got, st.W[0]) <= 1e-5
        u = reps.read_global_momentum().cpu().numpy()
        assert np.max(np.abs(u - st.u_global)) * w.lr <= 1e-5 * scale


def test_resnet20_full_shape_first_round_model():
    """Workload 5 at its real shape (K = 16, B_loc = 128, H = 16): the
    synchronised model after round 1 (eq. 2 / Algorithm 1 with per-worker BN)
    against the oracle's, which tests/golden/make_round_models.py wrote
    (oracle only), and the round's per-step mean losses. Bar: normwise 1e-5,
    or, where the oracle itself moves further when its initial weights are
    perturbed by 1e-7 (eight independent draws, same file), the largest of
    those distances times a factor calibrated on the draws alone, leave one
    out: the largest ratio of a draw to max(1e-5, the largest of the others)
    (at least 1) -- the largest of n draws understates where one more
    legitimate run may land."""
    import json
    import os
    here = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
    with open(os.path.join(here, "round1_resnet20.json")) as f:
        gold = json.load(f)
    model = np.load(os.path.join(here, "round1_resnet20_model.npy"))
    d = list(gold["perturbed_round1_normwise"])
    assert len(d) >= 3
    factor = max([1.0] + [d[i] / max(1e-5, max(d[:i] + d[i + 1:])) for i in range(len(d))])
    bar = max(1e-5, factor * max(d))
    w = wk.get("resnet20")
    X, y = wk.dataset(w)
    print("resnet20 full-shape round 1", flush=True)
    reps = make_replicas(w, X, y)
    loss = torch.empty(w.H, w.K, device=device())
    reps.run_round([w.lr] * w.H, loss)
    got = reps.read_params(0).cpu().numpy()
    np.testing.assert_array_equal(got, reps.read_params(w.K - 1).cpu().numpy())
    err = normwise(got, model)
    lerr = rel(loss.cpu().numpy().mean(axis=1), np.asarray(gold["round1_step_mean_loss"]))
    print(f"resnet20 round 1: model {err:.3e} (bar {bar:.3e}, leave-one-out factor "
          f"{factor:.3f}; oracle perturbed {d}), losses {lerr.max():.3e}", flush=True)
    assert err <= bar
    assert np.all(lerr <= 1e-3)
