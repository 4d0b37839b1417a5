"""Pose-estimation driver: the parallel Monte Carlo schedule of Sec. IV-B run
with the optimiser of Sec. IV-A and the setting of Sec. IV-D.

Phase 1 optimises P_N hypotheses independently for s1 steps.  Phase 2 is
repeated S times: rank the hypotheses by loss, keep the lowest-loss fraction r
and redraw the rest around them, then optimise all of them for s2 more steps;
r is halved after every round.  With the paper's constants (P_N = 64,
s1 = s2 = 512, S = 4, r = 0.25) a run takes 2560 steps and keeps 16, 8, 4
and 2 hypotheses at its four resampling rounds.

The loop is host code around the library's entry points: every step is one
pnerf_render_loss_grad and one pnerf_step_adam (or pnerf_step_momentum), and
each round one pnerf_resample_hypotheses, all on one stream.  Ranking uses the
losses of the last step (each hypothesis's loss on that step's pixel batch).
"""
from __future__ import annotations

import dataclasses
from typing import Callable

from . import pnerf


@dataclasses.dataclass(frozen=True)
class MCSchedule:
    """Constants of the Monte Carlo schedule (Sec. IV-B, values of Sec. IV-D)."""
    n_hypotheses: int = 64   # P_N
    s1: int = 512            # free-exploration steps
    s2: int = 512            # steps after each resampling round
    rounds: int = 4          # S
    keep_frac: float = 0.25  # r of the first round, halved every round

    def __post_init__(self):
        if self.n_hypotheses < 1 or self.s1 < 1 or self.s2 < 1 or self.rounds < 0:
            raise ValueError(f"invalid schedule {self}")
        if not 0.0 <= self.keep_frac <= 1.0:
            raise ValueError(f"keep_frac {self.keep_frac} outside [0, 1]")

    @property
    def total_steps(self) -> int:
        return self.s1 + self.rounds * self.s2

    def resample_round(self, steps_done: int) -> int:
        """The round (1..S) that resamples once `steps_done` steps have been
        taken, or 0 when none does."""
        if steps_done < self.s1 or (steps_done - self.s1) % self.s2:
            return 0
        j = (steps_done - self.s1) // self.s2 + 1
        return j if j <= self.rounds else 0

    def keep_fraction(self, round_idx: int) -> float:
        return self.keep_frac * 0.5 ** (round_idx - 1)

    def n_keep(self, round_idx: int) -> int:
        """Hypotheses kept by a round (the rule of pnerf_resample_hypotheses)."""
        k = int(self.n_hypotheses * self.keep_fraction(round_idx))
        return max(1, min(k, self.n_hypotheses))


PAPER_SCHEDULE = MCSchedule()


def invert(field: pnerf.Field, poses, observed, intr, pixels: Callable[[int], object],
           schedule: MCSchedule = PAPER_SCHEDULE, adam: pnerf.AdamParams | None = None,
           sigma_rot: float = 0.05, sigma_trans: float = 0.02, seed: int = 0,
           momentum: tuple[float, float] | None = None, stream=None,
           on_step: Callable[[int, object], None] | None = None):
    """Run the schedule on `poses` (device float32 [K][3][4], updated in place).

    pixels(it) returns the device int32 [K][P] pixel batch of step `it`.
    With `momentum` = (lr, beta) the heavy-ball step replaces Adam.  on_step,
    if given, is called after every step's update with (it, loss) -- loss being
    the device tensor of that step's per-hypothesis losses.  Returns the loss
    tensor of the last step; the state tensor is returned alongside it."""
    import torch
    K = poses.shape[0]
    if K != schedule.n_hypotheses:
        raise ValueError(f"{K} poses for a schedule of {schedule.n_hypotheses} hypotheses")
    dev = poses.device
    if momentum is None:
        adam = adam if adam is not None else pnerf.AdamParams()
        state = torch.zeros((K, pnerf.ADAM_STATE), dtype=torch.float32, device=dev)
    else:
        state = torch.zeros((K, 6), dtype=torch.float32, device=dev)
    loss = torch.empty(K, dtype=torch.float32, device=dev)
    dpose = torch.empty((K, 6), dtype=torch.float32, device=dev)
    for it in range(schedule.total_steps):
        field.render_loss_grad(poses, pixels(it), observed, intr, loss, dpose, stream=stream)
        if momentum is None:
            pnerf.step_adam(poses, state, dpose, it, adam, stream=stream)
        else:
            pnerf.step_momentum(poses, state, dpose, momentum[0], momentum[1], stream=stream)
        if on_step is not None:
            on_step(it, loss)
        j = schedule.resample_round(it + 1)
        if j:
            pnerf.resample_hypotheses(poses, state, loss, schedule.keep_fraction(j), sigma_rot,
                                      sigma_trans, seed, j, stream=stream)
    return loss, state
