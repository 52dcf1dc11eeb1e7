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


def test_resnet20_full_shape_first_steps():
    """Workload 5 at its real shape (K=16, B_loc=128): replicas 0 and 15 over
    the first two local steps."""
    w = wk.get("resnet20")
    X, y = wk.dataset(w)
    print("resnet20 full shape", flush=True)
    _, _, worst = _compare(w, X, y, wk.initial_weights(w), 2, [0, w.K - 1], 1e-5, 1e-3)
    print(f"resnet20 full shape: worst error {worst:.3e}", flush=True)
