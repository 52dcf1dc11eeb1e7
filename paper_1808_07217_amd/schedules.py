"""Host-side schedules of the training procedure: which rounds to run, with
how many local steps, at which step sizes. Scalars only: every round they
describe runs on the GPU through ``Replicas.run_round``.

* Large-batch learning-rate schemes (appendix on large-batch training,
  after Goyal et al.): the linear scaling rule (step size times the factor
  by which the global mini-batch grew over a reference batch) and the
  gradual warm-up, a constant increment per iteration from the base step
  size to the scaled one over a number of iterations (five epochs there).
* Step decay of the CIFAR procedure: divide by 10 once 50% and again once
  75% of the run's sample budget has been accessed.
* Local-step warm-up (appendix on the warm-up of the number of local steps;
  the ImageNet runs): H grows from 1 to its final value over the first
  epochs -- linearly, by doubling, or held at 1 ("constant").
* Post-local SGD (section 3): one local step per round before the switch,
  H after it; the paper switches at the first step-size decay.

Rounds never change the sample budget: the last round is shortened so that
a run takes exactly the requested number of local steps.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from fractions import Fraction
from typing import Callable, List, Optional, Sequence, Tuple

Round = Tuple[int, List[float]]   # (local steps H_t, step size of each step)

WARMUP_KINDS = ("linear", "exponential", "constant")


def batches_per_epoch(K: int, N: int, B: int) -> int:
    """Local steps per epoch: whole batches of B rows in the smallest worker
    part (floor(N / K) rows); matches the per-epoch reshuffle sampler."""
    return (N // K) // B


@dataclass(frozen=True)
class StepSizes:
    """Step size of every local step of a run (0-based step index s).

    base: the single-worker step size; scale: linear-scaling factor (global
    batch / reference batch, 1 for none); warmup_steps: iterations of the
    gradual warm-up from base to base * scale (0: none); the decay divides
    by ``1 / factor`` at each milestone fraction of total_samples, counting
    the samples accessed before step s (s * samples_per_step)."""
    base: float
    scale: float = 1.0
    warmup_steps: int = 0
    samples_per_step: int = 1
    total_samples: int = 0
    milestones: Sequence[float] = (0.5, 0.75)
    factor: float = 0.1

    def __call__(self, s: int) -> float:
        peak = self.base * self.scale
        if 0 < self.warmup_steps and s < self.warmup_steps:
            value = self.base + (peak - self.base) * (s / self.warmup_steps)
        else:
            value = peak
        if self.total_samples > 0:
            seen = s * self.samples_per_step
            passed = sum(1 for m in self.milestones if seen >= m * self.total_samples)
            value *= self.factor ** passed
        return value

    def first_decay_step(self) -> Optional[int]:
        """The first local step taken at a decayed step size."""
        if self.total_samples <= 0 or not self.milestones:
            return None
        target = Fraction(min(self.milestones)) * self.total_samples
        return math.ceil(target / self.samples_per_step)


def warmup_local_steps(epoch: int, H: int, kind: Optional[str],
                       epochs: int) -> int:
    """H used by rounds that start in ``epoch`` under a local-step warm-up of
    ``epochs`` epochs: linear 1 + floor((H - 1) e / epochs), exponential
    min(H, 2^e), constant 1; H from then on (and with no warm-up)."""
    if kind is None or epoch >= epochs:
        return H
    if kind not in WARMUP_KINDS:
        raise ValueError(f"unknown local-step warm-up {kind!r}")
    if kind == "constant":
        return 1
    if kind == "exponential":
        h = 1
        for _ in range(epoch):
            h = min(H, 2 * h)
        return h
    return 1 + (H - 1) * epoch // epochs


def plan_rounds(total_steps: int, steps_per_epoch: int, H: int,
                step_size: Callable[[int], float], *,
                warmup: Optional[str] = None, warmup_epochs: int = 0,
                switch_step: Optional[int] = None) -> List[Round]:
    """Rounds covering exactly ``total_steps`` local steps. A round starting
    at local step s has H_t = warmup_local_steps(s // steps_per_epoch, ...)
    -- or, with ``switch_step`` (post-local SGD), 1 while s < switch_step and
    H from it on -- cut short if the budget ends inside it."""
    if total_steps < 0 or steps_per_epoch < 1 or H < 1:
        raise ValueError("need total_steps >= 0, steps_per_epoch >= 1, H >= 1")
    plan: List[Round] = []
    s = 0
    while s < total_steps:
        if switch_step is not None:
            h = H if s >= switch_step else 1
        else:
            h = warmup_local_steps(s // steps_per_epoch, H, warmup, warmup_epochs)
        h = min(h, total_steps - s)
        plan.append((h, [step_size(s + i) for i in range(h)]))
        s += h
    return plan


def cifar_plan(*, K: int, B: int, N: int, epochs: int, base_lr: float, H: int,
               ref_batch: Optional[int] = None, lr_warmup_epochs: int = 0,
               post_local: bool = False, warmup: Optional[str] = None,
               warmup_epochs: int = 0) -> List[Round]:
    """The CIFAR training procedure as rounds: ``epochs`` epochs of
    batches_per_epoch(K, N, B) local steps; step sizes scaled by K B /
    ref_batch (when given) with an optional gradual warm-up over
    lr_warmup_epochs epochs, decayed at 50% and 75% of the samples; rounds
    of H local steps, with post-local SGD switching at the first decay, or
    a local-step warm-up."""
    S = batches_per_epoch(K, N, B)
    if S < 1:
        raise ValueError("a worker's part must hold at least one batch")
    total = epochs * S
    sizes = StepSizes(base=base_lr,
                      scale=(K * B / ref_batch) if ref_batch else 1.0,
                      warmup_steps=lr_warmup_epochs * S,
                      samples_per_step=K * B, total_samples=total * K * B)
    switch = sizes.first_decay_step() if post_local else None
    return plan_rounds(total, S, H, sizes, warmup=warmup,
                       warmup_epochs=warmup_epochs, switch_step=switch)


def run_plan(reps, plan: Sequence[Round], loss=None) -> None:
    """Run the rounds of a plan on ``reps`` (a ``lsgd.Replicas``); ``loss``
    (fp32 [total steps][K] on the device) receives every step's losses."""
    row = 0
    for h, lrs in plan:
        reps.run_round(lrs, None if loss is None else loss[row:row + h])
        row += h
