"""Plain CPU oracle of hysteresis-guided reconfiguration (DynaResize Sec. 3.4, Exp#3).

TEST INFRASTRUCTURE ONLY (see oracle/__init__.py).  It shares no code with the
library's controller; both follow the rule written out below.

The paper treats resizing as a stabilized decision over a discrete, pre-specified
list of configurations: a measurement is not an immediate trigger; decisions pass
through hysteresis thresholds, dwell time, a cooldown after each resize and a
number of consecutive same-direction signals, so only sustained imbalance moves
the allocation (Sec. 3.4).  A resize pays off once the per-step saving has covered
its blocking cost (Exp#3: about 11 steps; the cooldown of more than 10 steps keeps
decisions beyond that point).

Written-out rule (the paper gives no formulas; this is the reading):

* configurations 0 .. K-1 are pre-specified GPU splits (training GPUs T_i,
  rollout GPUs R_i), ordered from the most training GPUs to the most rollout
  GPUs; a resize moves one position, +1 toward rollout, -1 toward training;
* per step, with rollout time tr and training time tt, the imbalance is
  r = (tr - tt) / max(tr, tt)  (0 when both are 0);
* hysteresis signal: off (0) becomes +1 when r > enter and -1 when r < -enter;
  +1 stays while r > exit, turns to -1 if r < -enter, else off; -1 symmetric;
* run: the number of consecutive steps with the same nonzero signal;
* at the start of every step the steps spent in the current configuration grow
  by one, and a pending cooldown counts down (a resize at step k blocks steps
  k+1 .. k+cooldown);
* a resize in direction s is issued when, in this order of checks,
  signal s != 0, run >= consecutive, no cooldown is pending, steps in the
  configuration >= dwell, configuration + s exists, and the resize pays off:
  over the last `consecutive` steps the stages' work is estimated as
  mean(tr) * R_cur and mean(tt) * T_cur GPU-seconds, the step time in the
  target is predicted as max(work_r / R_tgt, work_t / T_tgt), the gain per step
  is mean(max(tr, tt)) minus that prediction, and the resize needs gain > 0 and
  (switch_cost == 0 or gain * horizon >= switch_cost);
* after a resize the run, the signal and the steps in the configuration restart
  at 0 and the cooldown is set.

Parity pinned by the tests: closed-form traces (balanced, step change, oscillation,
in-band noise, hysteresis band, edges) and the paper's break-even arithmetic.  The
paper pins only the behaviour (sustained imbalance alone moves the allocation, a
cooldown beyond 10 steps, a resize amortizes in about 11 steps); the band, run,
dwell and predicted-gain formulas above are this reading, so beyond those
properties their parity is unpinned by the paper: the pins check the written rule
on hand-derived traces.
"""
from __future__ import annotations

from dataclasses import dataclass

BALANCED, PERSISTENCE, COOLDOWN, DWELL, EDGE, AMORTIZE, RESIZE = range(7)


@dataclass
class Params:
    train_gpus: list[int]
    rollout_gpus: list[int]
    initial: int
    enter: float
    exit: float
    consecutive: int
    dwell: int
    cooldown: int
    switch_cost: float = 0.0
    horizon: int = 0

    @property
    def num_configs(self) -> int:
        return len(self.train_gpus)


def break_even_steps(switch_cost: float, step_before: float, step_after: float) -> float:
    """Steps after which the saved time covers one resize (Exp#3)."""
    return switch_cost / (step_before - step_after)


def imbalance(tr: float, tt: float) -> float:
    m = max(tr, tt)
    return 0.0 if m == 0 else (tr - tt) / m


def predicted_gain(params: Params, cur: int, tgt: int, window: list[tuple[float, float]]) -> float:
    """Step time saved per step by moving from configuration cur to tgt, from the window's work."""
    n = len(window)
    mean_tr = sum(tr for tr, _ in window) / n
    mean_tt = sum(tt for _, tt in window) / n
    mean_step = sum(max(tr, tt) for tr, tt in window) / n
    work_r = mean_tr * params.rollout_gpus[cur]
    work_t = mean_tt * params.train_gpus[cur]
    return mean_step - max(work_r / params.rollout_gpus[tgt], work_t / params.train_gpus[tgt])


def _pays_off(params: Params, cur: int, tgt: int, window) -> bool:
    gain = predicted_gain(params, cur, tgt, window)
    return gain > 0 and (params.switch_cost == 0 or gain * params.horizon >= params.switch_cost)


def run(params: Params, trace: list[tuple[float, float]]) -> list[tuple[int, int, int]]:
    """Decisions for a trace of (rollout time, training time): (config after the step, action, reason)."""
    config = params.initial
    signal = 0
    run_len = 0
    in_config = 0
    cooldown_left = 0
    window: list[tuple[float, float]] = []
    out = []
    for tr, tt in trace:
        in_config += 1
        blocked = cooldown_left > 0
        if blocked:
            cooldown_left -= 1
        r = imbalance(tr, tt)
        if signal == 0:
            new = 1 if r > params.enter else (-1 if r < -params.enter else 0)
        elif signal == 1:
            new = 1 if r > params.exit else (-1 if r < -params.enter else 0)
        else:
            new = -1 if r < -params.exit else (1 if r > params.enter else 0)
        run_len = run_len + 1 if (new != 0 and new == signal) else (1 if new != 0 else 0)
        signal = new
        window = (window + [(tr, tt)])[-params.consecutive:]
        if signal == 0:
            reason = BALANCED
        elif run_len < params.consecutive:
            reason = PERSISTENCE
        elif blocked:
            reason = COOLDOWN
        elif in_config < params.dwell:
            reason = DWELL
        elif not 0 <= config + signal < params.num_configs:
            reason = EDGE
        elif not _pays_off(params, config, config + signal, window):
            reason = AMORTIZE
        else:
            reason = RESIZE
        action = 0
        if reason == RESIZE:
            action = signal
            config += signal
            signal = 0
            run_len = 0
            in_config = 0
            cooldown_left = params.cooldown
        out.append((config, action, reason))
    return out
