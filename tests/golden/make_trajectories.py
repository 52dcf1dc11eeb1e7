"""Write the oracle's loss trajectories for the full workload runs.

Usage (from the repository root; takes tens of minutes on 8 cores):
    python tests/golden/make_trajectories.py [workload ...]

For each workload it runs the CPU oracle over the whole schedule from the
seeded inputs and stores, per round, the mean mini-batch loss of every local
step (averaged over the K replicas) in tests/golden/trajectory_<name>.json.
Only the oracle and the seeded input module are used.

ResNet-20's runs from perturbed initial weights (several independent draws,
trajectory_resnet20_perturbed.json) are written by make_round_models.py,
which also writes its unperturbed trajectory the same way.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import workloads as wk  # noqa: E402
from oracle import lsgd_oracle as O  # noqa: E402

FULL_RUNS = ["mlp_512", "postlocal_mlp_512", "wide_mlp_2048_bf16", "resnet20"]


def trajectory(name):
    w = wk.get(name)
    X, y = wk.dataset(w)
    w0 = np.asarray(wk.initial_weights(w), np.float64)
    st = O.State(w0, w.K)
    rounds = []
    t0 = time.time()
    for t, (H, lr) in enumerate(O.schedule(w)):
        losses = O.run_round(st, w, X, y, H, lr)       # [H][K]
        rounds.append([float(v) for v in losses.mean(axis=1)])
        if t % 10 == 0:
            print(f"{name}: round {t + 1} loss {np.mean(rounds[-1]):.6g} "
                  f"({time.time() - t0:.0f} s)", flush=True)
    return {
        "workload": name,
        "source": "oracle.lsgd_oracle.run_round over the post-local schedule "
                  "from workloads.initial_weights / workloads.dataset",
        "per_round_step_mean_loss": rounds,
    }


def main():
    names = sys.argv[1:] or FULL_RUNS
    for name in names:
        out = trajectory(name)
        path = os.path.join(HERE, f"trajectory_{name}.json")
        with open(path, "w") as f:
            json.dump(out, f)
        print(f"wrote {path}", flush=True)


if __name__ == "__main__":
    main()
