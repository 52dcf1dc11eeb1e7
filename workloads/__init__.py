"""Seeded synthetic inputs and the workload table for the local-SGD hot path.

This module holds inputs only: the hyper-parameters of each workload, the
synthetic datasets that stand in for the paper's CIFAR-10 / convex benchmarks,
and the initial weights. It contains none of the method's arithmetic (no
sampling, no forward/backward, no update, no averaging). Both the HIP path and
the CPU oracle take their inputs from here, as identical bytes.

Parameter layout of one replica (the flat `[P]` vector that crosses the C ABI):
for each fully-connected layer l = 1..L in order, the weight W_l stored
row-major as `[d_in][d_out]` (element (i, j) multiplies input feature i into
output j), followed by the bias b_l `[d_out]`.

Recipes (all numpy PCG64, drawn in fp64, cast to fp32 at the end):

* ``gauss64`` -- stands in for the paper's small convex problem (the w8a
  logistic-regression experiment of the appendix on local SGD's convergence):
  10 class means mu_c ~ N(0, I_64); labels y_i ~ U{0..9}; x_i = mu_{y_i} +
  0.5 * eps_i, eps_i ~ N(0, I_64); N = 4096 rows, raw features.
* ``img3072`` -- stands in for CIFAR-10 (50K colour images 32x32x3, 10
  classes; the dataset section of the appendix): per-class mean image
  m_c ~ N(0, I_3072) in CHW order; y ~ U{0..9}; x = m_y + 1.0 * eps; then the
  per-channel standardisation the paper applies to its inputs (channel mean
  and standard deviation over the whole set, computed in fp64).
"""
from __future__ import annotations

import dataclasses
import functools
from typing import Tuple

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "get", "dataset", "initial_weights",
    "layer_shapes", "param_count",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One (post-)local SGD workload.

    ``warm_rounds`` is the post-local switch point t': rounds 1..t' run with
    one local step each (mini-batch SGD), later rounds run ``H`` local steps.
    ``lr_after_switch`` is the step size used after the switch (equal to
    ``lr`` when there is no switch). ``Kb`` > 0 makes it hierarchical local
    SGD (Appendix D): blocks of ``Kb`` consecutive workers average every
    ``H`` steps, all workers every ``H * Hb`` steps (one outer round).
    """
    name: str
    model: str                 # "mlp" (softmax regression is the 1-layer MLP)
    widths: Tuple[int, ...]    # d_in, hidden..., classes
    dtype: str                 # "fp32" or "bf16" (GEMM operand type)
    K: int                     # workers == replicas
    B_loc: int                 # local mini-batch size
    H: int                     # local steps per round (local phase)
    rounds: int                # rounds of the local phase
    lr: float
    momentum: float
    nesterov: bool
    weight_decay: float
    warm_rounds: int = 0       # post-local switch point t'
    lr_after_switch: float = 0.0
    data: str = "img3072"
    N: int = 50000
    data_seed: int = 0
    init_seed: int = 0
    sample_seed: int = 0
    Kb: int = 0                # hierarchical block size K' (0: none)
    Hb: int = 1                # block rounds per global average, H^b
    global_momentum: float = 0.0   # m_g at the global average (0: plain mean)
    scheme: str = "local"      # "local"; "sign" (Algorithm 3); "ef_sign" (4)
    sampler: str = "iid"       # "iid" (fixed shards); "epoch" (reshuffled)

    @property
    def n_layers(self) -> int:
        return len(self.widths) - 1

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


_IMG = dict(data="img3072", N=50000)

WORKLOADS = {
    # softmax regression d=64 -> 10 classes, fp32, plain SGD
    "softmax_d64": Workload(
        name="softmax_d64", model="mlp", widths=(64, 10), dtype="fp32",
        K=4, B_loc=32, H=4, rounds=50, lr=0.1, momentum=0.0, nesterov=False,
        weight_decay=0.0, data="gauss64", N=4096,
        data_seed=101, init_seed=102, sample_seed=0x5EED0001),
    # MLP 3072-512-512-10, fp32, heavy-ball momentum, local buffers
    "mlp_512": Workload(
        name="mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=16, rounds=20, lr=0.001,
        momentum=0.9, nesterov=False, weight_decay=1e-4, **_IMG,
        data_seed=201, init_seed=202, sample_seed=0x5EED0002),
    # post-local SGD on the same MLP: 200 rounds of H=1, then 20 rounds of
    # H=16 with the step size decayed 10x at the switch; Nesterov momentum
    "postlocal_mlp_512": Workload(
        name="postlocal_mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=16, rounds=20, lr=0.001,
        momentum=0.9, nesterov=True, weight_decay=1e-4,
        warm_rounds=200, lr_after_switch=0.0001, **_IMG,
        data_seed=201, init_seed=302, sample_seed=0x5EED0003),
    # wide MLP 3072-2048-2048-10, bf16 GEMM operands, fp32 master weights
    "wide_mlp_2048_bf16": Workload(
        name="wide_mlp_2048_bf16", model="mlp", widths=(3072, 2048, 2048, 10),
        dtype="bf16", K=64, B_loc=64, H=8, rounds=10, lr=0.001,
        momentum=0.9, nesterov=False, weight_decay=1e-4, **_IMG,
        data_seed=201, init_seed=402, sample_seed=0x5EED0004),
    # hierarchical local SGD on the same MLP: 8 blocks of K'=2 workers (the
    # 8 x 2 topology of Appendix D's tables), block average every H=4 steps,
    # global average every H * H^b = 16 steps
    "hier_mlp_512": Workload(
        name="hier_mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=4, rounds=20, lr=0.001,
        momentum=0.9, nesterov=False, weight_decay=1e-4, Kb=2, Hb=4, **_IMG,
        data_seed=201, init_seed=202, sample_seed=0x5EED0006),
    # hybrid momentum on the same MLP: local heavy ball 0.9 plus a global
    # buffer with factor 0.3 at every synchronisation (the momentum
    # appendix's local/global grid, at one of its well-behaved settings)
    "hybrid_mlp_512": Workload(
        name="hybrid_mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=16, rounds=20, lr=0.001,
        momentum=0.9, nesterov=False, weight_decay=1e-4, global_momentum=0.3,
        **_IMG, data_seed=201, init_seed=202, sample_seed=0x5EED0007),
    # (post-)local SGD with sign compression on the same MLP, Nesterov and
    # weight decay on the local steps as the compression appendix used:
    # Algorithm 3 (sign local steps; a small step size since every
    # coordinate moves by it) and Algorithm 4 (EF-signSGD)
    "signsgd_mlp_512": Workload(
        name="signsgd_mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=16, rounds=20, lr=0.0001,
        momentum=0.9, nesterov=True, weight_decay=1e-4, scheme="sign",
        **_IMG, data_seed=201, init_seed=202, sample_seed=0x5EED0008),
    "efsign_mlp_512": Workload(
        name="efsign_mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=16, rounds=20, lr=0.001,
        momentum=0.9, nesterov=True, weight_decay=1e-4, scheme="ef_sign",
        **_IMG, data_seed=201, init_seed=202, sample_seed=0x5EED0009),
    # the same MLP round with the per-epoch reshuffled partition sampler
    # (the CIFAR procedure's data handling) instead of i.i.d. draws
    "epoch_mlp_512": Workload(
        name="epoch_mlp_512", model="mlp", widths=(3072, 512, 512, 10),
        dtype="fp32", K=16, B_loc=128, H=16, rounds=20, lr=0.001,
        momentum=0.9, nesterov=False, weight_decay=1e-4, sampler="epoch",
        **_IMG, data_seed=201, init_seed=202, sample_seed=0x5EED000A),
    # ResNet-20-shaped CNN, fp32, per-worker BN, heavy-ball momentum
    "resnet20": Workload(
        name="resnet20", model="resnet20", widths=(3072, 10), dtype="fp32",
        K=16, B_loc=128, H=16, rounds=5, lr=0.05, momentum=0.9,
        nesterov=False, weight_decay=1e-4, data="img3072_nhwc", N=50000,
        data_seed=201, init_seed=502, sample_seed=0x5EED0005),
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def layer_shapes(widths) -> list:
    """[(d_in, d_out), ...] of the fully-connected layers."""
    return [(widths[i], widths[i + 1]) for i in range(len(widths) - 1)]


def param_count(widths, model: str = "mlp") -> int:
    if model == "resnet20":
        return sum(int(np.prod(s)) for _, s in resnet_tensors(classes=widths[-1]))
    return sum(a * b + b for a, b in layer_shapes(widths))


@functools.lru_cache(maxsize=4)
def _dataset_cached(kind: str, N: int, seed: int):
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "gauss64":
        d, C = 64, 10
        mu = rng.standard_normal((C, d))
        y = rng.integers(0, C, size=N)
        X = mu[y] + 0.5 * rng.standard_normal((N, d))
    elif kind == "img3072":
        d, C, ch = 3072, 10, 3
        mu = rng.standard_normal((C, d))
        y = rng.integers(0, C, size=N)
        X = rng.standard_normal((N, d))
        X += mu[y]
        # per-channel standardisation, CHW order: channel c owns a contiguous
        # block of 1024 pixels
        Xc = X.reshape(N, ch, d // ch)
        mean = Xc.mean(axis=(0, 2), keepdims=True)
        std = Xc.std(axis=(0, 2), keepdims=True)
        Xc -= mean
        Xc /= std
    elif kind == "img3072_nhwc":
        # the same images, stored as [N][32][32][3] (channel innermost)
        Xc, y32 = _dataset_cached("img3072", N, seed)
        X = np.ascontiguousarray(
            Xc.reshape(N, 3, 32, 32).transpose(0, 2, 3, 1)).reshape(N, 3072)
        X.setflags(write=False)
        return X, y32
    else:
        raise ValueError(f"unknown dataset kind {kind!r}")
    X32 = np.ascontiguousarray(X, dtype=np.float32)
    y32 = y.astype(np.int32)
    X32.setflags(write=False)
    y32.setflags(write=False)
    return X32, y32


def dataset(w: Workload):
    """(X f32[N][d], y i32[N]) for a workload; read-only arrays, cached."""
    return _dataset_cached(w.data, w.N, w.data_seed)


RESNET_STAGES = (16, 32, 64)   # channels of the three stages


def resnet_tensors(blocks: int = 3, cin: int = 3, classes: int = 10):
    """[(kind, shape)] of the ResNet-20 parameter vector, in order: per 3x3
    convolution its weight [3][3][c_in][c_out] ("conv"), BN scale ("bn_g")
    and shift ("bn_b"); then the classifier weight [64][classes] ("fc_w")
    and bias ("fc_b"). Convolutions: the stem, then per stage and block two
    convolutions (the first of stages 2 and 3 has stride 2)."""
    out, c = [], RESNET_STAGES[0]
    convs = [(cin, c)]
    for co in RESNET_STAGES:
        for _ in range(blocks):
            convs += [(c, co), (co, co)]
            c = co
    for ci, co in convs:
        out += [("conv", (3, 3, ci, co)), ("bn_g", (co,)), ("bn_b", (co,))]
    out += [("fc_w", (RESNET_STAGES[-1], classes)), ("fc_b", (classes,))]
    return out


def initial_weights(w: Workload) -> np.ndarray:
    """The shared starting point w_(0), flat fp32 `[P]` in the layout above.

    Hidden layers: He normal, std sqrt(2 / fan_in); the classifier layer:
    N(0, 0.01^2); biases 0 (initialisation paragraph of the appendix on
    models). ResNet: convolutions He normal with fan_in = 9 c_in, BN scale 1
    and shift 0, classifier as above.
    """
    rng = np.random.Generator(np.random.PCG64(w.init_seed))
    if w.model == "resnet20":
        parts = []
        for kind, shape in resnet_tensors():
            n = int(np.prod(shape))
            if kind == "conv":
                parts.append(np.sqrt(2.0 / (9 * shape[2])) * rng.standard_normal(n))
            elif kind == "fc_w":
                parts.append(0.01 * rng.standard_normal(n))
            elif kind == "bn_g":
                parts.append(np.ones(n))
            else:
                parts.append(np.zeros(n))
        return np.concatenate(parts).astype(np.float32)
    parts = []
    shapes = layer_shapes(w.widths)
    for li, (din, dout) in enumerate(shapes):
        std = 0.01 if li == len(shapes) - 1 else np.sqrt(2.0 / din)
        parts.append((std * rng.standard_normal((din, dout))).ravel())
        parts.append(np.zeros(dout))
    return np.concatenate(parts).astype(np.float32)
