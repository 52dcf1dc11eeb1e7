"""Helpers shared by the GPU tests: building replicas from a workload and the
parity metrics. No arithmetic of the method lives here."""
import numpy as np
import torch

import workloads as wk

U32 = 2.0**-24  # unit roundoff of fp32


def gamma(n, u=U32):
    """Higham's gamma_n = n u / (1 - n u): bound on n roundings in sequence."""
    return n * u / (1 - n * u)


def normwise(a, b):
    """max_i |a_i - b_i| / max_i |b_i| over the whole vector."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def rel(a, b, floor=1e-6):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b) / np.maximum(np.abs(b), floor)


def device():
    return torch.device("cuda", 0)


def to_dev(arr, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(arr))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device())


def make_replicas(w, X=None, y=None, w0=None):
    """A ``Replicas`` for workload ``w`` on cuda:0 with its seeded inputs."""
    from paper_1808_07217_amd import lsgd as L
    if X is None:
        X, y = wk.dataset(w)
    if w0 is None:
        w0 = wk.initial_weights(w)
    cfg = L.make_config(w.widths, w.K, w.B_loc, w.N, dtype=w.dtype,
                        momentum=w.momentum, weight_decay=w.weight_decay,
                        nesterov=w.nesterov, seed=w.sample_seed, model=w.model,
                        global_momentum=w.global_momentum, scheme=w.scheme,
                        sampler=w.sampler)
    Xd = to_dev(np.asarray(X, np.float32))
    yd = to_dev(np.asarray(y, np.int32))
    wd = to_dev(np.asarray(w0, np.float32))
    return L.Replicas(cfg, Xd, yd, wd)
