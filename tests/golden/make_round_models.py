"""Write the oracle's full-size round models and the sensitivity draws the
full-size parity tests are held to.

Usage (from the repository root):
    python tests/golden/make_round_models.py resnet20 [--jobs N]
    python tests/golden/make_round_models.py resnet20 --draws-only SEED ... [--jobs N]
    python tests/golden/make_round_models.py wide_mlp_2048_bf16 [--jobs N]

(--draws-only runs the perturbed draws of the given seeds and adds them to
the files already written, replacing a draw of the same seed.)

Only the oracle (``oracle.lsgd_oracle``) and the seeded input module
(``workloads``) are used. Replicas are independent between synchronisations
(eq. 2), so each round's local steps run one replica per task in a pool of
processes, each through the oracle's own ``local_step`` on a state holding
that replica; the parent applies the oracle's ``synchronise`` to the gathered
replicas. The arithmetic per replica is the oracle's, in its order.

resnet20 (K = 16, B_loc = 128, H = 16, five rounds):
  * the run from the workload's initial weights: the per-round step-mean
    losses (``trajectory_resnet20.json``) and the synchronised model after
    round 1 (``round1_resnet20_model.npy``, fp32 [P]);
  * eight runs from initial weights multiplied elementwise by (1 + 1e-7 z),
    z ~ N(0, 1), from eight independent seeds -- a change of the size of fp32
    rounding: their loss trajectories (``trajectory_resnet20_perturbed.json``)
    and how far each one's round-1 model lies from the unperturbed one
    (``round1_resnet20.json``). The spread measures how strongly the
    trajectory itself amplifies rounding.

wide_mlp_2048_bf16 (K = 64, B_loc = 64, H = 8, bf16 operands, round 1):
  * the synchronised model after round 1 at 65536 seeded sample positions
    plus its largest magnitude over the whole vector
    (``round1_wide_mlp_2048_bf16.npz``), the round's losses;
  * the same round with every bf16 rounding removed (fp32/fp64 operands):
    its normwise distance to the bf16 model and its loss distance, which
    bound from above how far a path that skipped the roundings would land;
  * three 1e-7-perturbed bf16 runs of the round: their distances.
"""
import os

# one BLAS thread per process; the pool provides the parallelism
for _v in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ[_v] = "1"

import argparse  # noqa: E402
import json  # noqa: E402
import multiprocessing as mp  # noqa: E402
import sys  # noqa: E402
import time  # noqa: E402

import numpy as np  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import workloads as wk  # noqa: E402
from oracle import lsgd_oracle as O  # noqa: E402

PERTURBATION = 1e-7
PERTURBATION_SEEDS = (12345, 23456, 34567, 45678, 56789, 67890, 78901, 89012)
WIDE_PERTURBATION_SEEDS = PERTURBATION_SEEDS[:3]
SAMPLE_SEED = 777
N_SAMPLES = 65536

_G = {}


def _pool_init(wl):
    _G["wl"] = wl
    _G["X"], _G["y"] = wk.dataset(wl)


def _replica_steps(task):
    """H local steps of replica k through the oracle's local_step."""
    k, step0, w_k, u_k, lrs = task
    wl, X, y = _G["wl"], _G["X"], _G["y"]
    st = O.State.__new__(O.State)
    # rows other than k stay untouched (and, being calloc'd, unallocated)
    st.W = np.zeros((wl.K, w_k.size))
    st.U = np.zeros((wl.K, w_k.size))
    st.W[k], st.U[k] = w_k, u_k
    st.step = step0
    losses = [O.local_step(st, wl, X, y, lr, replicas=[k])[k] for lr in lrs]
    return k, st.W[k].copy(), st.U[k].copy(), np.asarray(losses)


def initial(wl, seed=None):
    w0 = np.asarray(wk.initial_weights(wl), np.float64)
    if seed is not None:
        z = np.random.default_rng(seed).standard_normal(w0.size)
        w0 = w0 * (1.0 + PERTURBATION * z)
    return w0


def run(wl, w0, rounds, jobs, label):
    """Rounds of the oracle from w0. Returns (per-round [H][K] losses, the
    synchronised model after each round)."""
    K = wl.K
    st = O.State.__new__(O.State)
    st.W = np.repeat(w0[None, :], K, axis=0)
    st.w_sync = w0.copy()
    st.step = 0
    U = [np.zeros_like(w0) for _ in range(K)]
    losses, models = [], []
    t0 = time.time()
    ctx = mp.get_context("fork")
    with ctx.Pool(jobs, initializer=_pool_init, initargs=(wl,)) as pool:
        for t, (H, lr) in enumerate(O.schedule(wl)[:rounds]):
            lrs = [lr] * H
            tasks = [(k, st.step, st.W[k], U[k], lrs) for k in range(K)]
            L = np.zeros((H, K))
            for k, w_k, u_k, l_k in pool.imap_unordered(_replica_steps, tasks):
                st.W[k], U[k], L[:, k] = w_k, u_k, l_k
            st.step += H
            O.synchronise(st, wl, lrs[-1])
            losses.append(L)
            models.append(st.W[0].copy())
            print(f"{label}: round {t + 1} loss {L.mean():.6g} "
                  f"({time.time() - t0:.0f} s)", flush=True)
    return losses, models


def normwise(a, b):
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


def traj(losses):
    return [[float(v) for v in L.mean(axis=1)] for L in losses]


def make_resnet20(jobs, draws_only=None):
    wl = wk.get("resnet20")
    src = ("tests/golden/make_round_models.py: oracle.lsgd_oracle local_step per "
           "replica and synchronise, from workloads.initial_weights")
    if draws_only:
        # the unperturbed model and losses as written before
        base_m0 = np.load(os.path.join(HERE, "round1_resnet20_model.npy")).astype(np.float64)
        with open(os.path.join(HERE, "round1_resnet20.json")) as f:
            base_l0 = json.load(f)["round1_step_mean_loss"]
        with open(os.path.join(HERE, "trajectory_resnet20_perturbed.json")) as f:
            old = {d["seed"]: d for d in json.load(f)["draws"]}
        with open(os.path.join(HERE, "round1_resnet20.json")) as f:
            r1 = json.load(f)
        old_dist = dict(zip(r1["perturbation_seeds"], r1["perturbed_round1_normwise"]))
        seeds = list(draws_only)
    else:
        base_l, base_m = run(wl, initial(wl), wl.rounds, jobs, "resnet20")
        with open(os.path.join(HERE, "trajectory_resnet20.json"), "w") as f:
            json.dump({"workload": "resnet20", "source": src,
                       "per_round_step_mean_loss": traj(base_l)}, f)
        np.save(os.path.join(HERE, "round1_resnet20_model.npy"),
                base_m[0].astype(np.float32))
        # the float32 model as stored is what the draws are measured against
        base_m0 = base_m[0].astype(np.float32).astype(np.float64)
        base_l0 = traj(base_l)[0]
        old, old_dist, seeds = {}, {}, list(PERTURBATION_SEEDS)
    for seed in seeds:
        l, m = run(wl, initial(wl, seed), wl.rounds, jobs, f"resnet20 seed {seed}")
        old[seed] = {"seed": seed, "per_round_step_mean_loss": traj(l)}
        old_dist[seed] = normwise(m[0], base_m0)
        print(f"seed {seed}: round-1 model moved {old_dist[seed]:.3e}", flush=True)
    order = sorted(old)
    with open(os.path.join(HERE, "trajectory_resnet20_perturbed.json"), "w") as f:
        json.dump({"workload": "resnet20",
                   "source": src + f", initial weights x (1 + {PERTURBATION} z), "
                             "z ~ N(0,1) from each seed",
                   "draws": [old[k] for k in order]}, f)
    with open(os.path.join(HERE, "round1_resnet20.json"), "w") as f:
        json.dump({"workload": "resnet20", "source": src,
                   "model": "round1_resnet20_model.npy (fp32 [P], the "
                            "synchronised model after round 1)",
                   "round1_step_mean_loss": base_l0,
                   "perturbation": PERTURBATION,
                   "perturbation_seeds": order,
                   "perturbed_round1_normwise": [old_dist[k] for k in order]}, f,
                  indent=1)


def make_wide_bf16(jobs):
    wl = wk.get("wide_mlp_2048_bf16")
    base_l, base_m = run(wl, initial(wl), 1, jobs, "wide bf16")
    wbar = base_m[0]
    pos = np.sort(np.random.default_rng(SAMPLE_SEED).choice(
        wbar.size, N_SAMPLES, replace=False))
    nr = wl.scaled(dtype="fp32")            # every bf16 rounding removed
    nr_l, nr_m = run(nr, initial(wl), 1, jobs, "wide, no bf16 rounding")
    rel_loss = lambda a, b: float(np.max(np.abs(a - b) / np.abs(b)))
    base_steps = base_l[0].mean(axis=1)
    out = {"workload": "wide_mlp_2048_bf16",
           "source": "tests/golden/make_round_models.py: oracle.lsgd_oracle "
                     "local_step per replica and synchronise",
           "sample_seed": SAMPLE_SEED,
           "max_abs_model": float(np.max(np.abs(wbar))),
           "round1_step_mean_loss": [float(v) for v in base_steps],
           "no_rounding_normwise": normwise(nr_m[0], wbar),
           "no_rounding_sampled_normwise":
               float(np.max(np.abs(nr_m[0][pos] - wbar[pos])) / np.max(np.abs(wbar))),
           "no_rounding_step_loss_rel": rel_loss(nr_l[0].mean(axis=1), base_steps),
           "no_rounding_replica_loss_rel": rel_loss(nr_l[0], base_l[0]),
           "perturbation": PERTURBATION,
           "perturbation_seeds": list(WIDE_PERTURBATION_SEEDS),
           "perturbed_normwise": [], "perturbed_step_loss_rel": []}
    print(json.dumps({k: v for k, v in out.items() if "loss" not in k}), flush=True)
    for seed in WIDE_PERTURBATION_SEEDS:
        l, m = run(wl, initial(wl, seed), 1, jobs, f"wide bf16 seed {seed}")
        out["perturbed_normwise"].append(normwise(m[0], wbar))
        out["perturbed_step_loss_rel"].append(rel_loss(l[0].mean(axis=1), base_steps))
    np.savez(os.path.join(HERE, "round1_wide_mlp_2048_bf16.npz"),
             positions=pos.astype(np.int64), values=wbar[pos].astype(np.float32),
             losses=base_l[0].astype(np.float64))
    with open(os.path.join(HERE, "round1_wide_mlp_2048_bf16.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("workload", choices=["resnet20", "wide_mlp_2048_bf16"])
    ap.add_argument("--jobs", type=int, default=os.cpu_count())
    ap.add_argument("--draws-only", type=int, nargs="+", default=None)
    a = ap.parse_args()
    if a.workload == "resnet20":
        make_resnet20(a.jobs, a.draws_only)
    else:
        make_wide_bf16(a.jobs)


if __name__ == "__main__":
    main()
