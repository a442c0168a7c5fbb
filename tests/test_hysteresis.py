"""Hysteresis-guided reconfiguration: oracle pins and parity of the native controller (C ABI).

Pins: hand-derived decisions on closed-form traces (balanced, a sustained step
change with consecutive/cooldown/dwell, oscillation, in-band noise, the
hysteresis band, the configuration edges, amortization) and the paper's
break-even arithmetic (Exp#3: 187 s over a 39.84 s -> 23.93 s step is about 11
steps).  Parity: the library and the oracle take identical decisions, step by
step, on random traces and parameters.
"""
import itertools

import numpy as np
import pytest

from oracle import controller as oc
from paper_2607_22614_amd import datagen, dr

R = oc.RESIZE


def splits(k):
    """k pre-specified splits of k+1 GPUs, most training first: (k:1), (k-1:2), ..., (1:k)."""
    return [k - i for i in range(k)], [i + 1 for i in range(k)]


def P(**kw):
    base = dict(train_gpus=[6, 5, 4, 3, 2], rollout_gpus=[2, 3, 4, 5, 6], initial=2, enter=0.2, exit=0.1,
                consecutive=3, dwell=0, cooldown=10)
    base.update(kw)
    return oc.Params(**base)


def resizes(decisions):
    return [(k, a) for k, (_, a, _) in enumerate(decisions) if a != 0]


def test_break_even_matches_the_paper():
    n = oc.break_even_steps(187.0, 39.84, 23.93)
    assert 11.0 < n < 12.0                       # Exp#3: a resize pays off after about 11 steps
    assert abs(n - 187.0 / 15.91) < 1e-12
    assert 10 < n                                # a >10-step cooldown sits at the amortization point
    assert dr.dr_break_even_steps(187.0, 39.84, 23.93) == n


def test_balanced_trace_never_resizes():
    d = oc.run(P(), [(10.0, 10.0)] * 50)
    assert resizes(d) == [] and all(r == oc.BALANCED for _, _, r in d)


def test_sustained_imbalance_resizes_after_consecutive_then_cooldown():
    # r = (30 - 10) / 30 = 0.667 > enter from step 5 on
    trace = [(10.0, 10.0)] * 5 + [(30.0, 10.0)] * 40
    d = oc.run(P(consecutive=3, cooldown=10), trace)
    # run reaches 3 at step 7 -> resize (config 3); steps 8..17 are cooled down while the restarted
    # run grows (8: 1, 9: 2, then cooldown), so the next resize is at 18 (config 4, the last one);
    # after it: 19 and 20 lack the run, 21..28 are cooled down, and from 29 on there is no config 5
    assert resizes(d) == [(7, 1), (18, 1)]
    assert [d[k][2] for k in (8, 9, 10, 17)] == [oc.PERSISTENCE, oc.PERSISTENCE, oc.COOLDOWN, oc.COOLDOWN]
    assert [d[k][2] for k in (19, 20, 21, 28, 29, 44)] == [oc.PERSISTENCE, oc.PERSISTENCE, oc.COOLDOWN,
                                                           oc.COOLDOWN, oc.EDGE, oc.EDGE]
    assert d[-1][0] == 4


def test_dwell_holds_a_fresh_configuration():
    trace = [(30.0, 10.0)] * 30
    d = oc.run(P(consecutive=2, cooldown=0, dwell=6), trace)
    # first resize needs 6 steps in the configuration (step 5); after it, 6 more (step 11)
    assert resizes(d) == [(5, 1), (11, 1)]
    assert d[4][2] == oc.DWELL


def test_oscillation_shorter_than_consecutive_never_resizes():
    trace = [(30.0, 10.0), (10.0, 30.0)] * 30
    assert resizes(oc.run(P(consecutive=2), trace)) == []


def test_noise_inside_the_band_never_resizes():
    trace = datagen.stage_time_trace(seed=1, steps=400, noise=0.03)
    assert max(abs(oc.imbalance(*t)) for t in trace) < 0.2
    assert resizes(oc.run(P(consecutive=1, cooldown=0), trace)) == []


def test_hysteresis_band_keeps_a_signal_alive():
    # r = 0.5 switches on, then r = 0.15 sits between exit 0.1 and enter 0.2: the signal holds
    tr_on, tr_mid = 20.0, 10.0 / 0.85
    trace = [(tr_on, 10.0)] + [(tr_mid, 10.0)] * 3
    d = oc.run(P(consecutive=4, cooldown=0), trace)
    assert resizes(d) == [(3, 1)]
    # without the hysteresis (exit == enter) the mid values turn the signal off
    assert resizes(oc.run(P(consecutive=4, cooldown=0, exit=0.2), trace)) == []


def test_edges_and_direction():
    down = oc.run(P(initial=0, consecutive=1, cooldown=0), [(10.0, 30.0)] * 3)
    assert resizes(down) == [] and down[0][2] == oc.EDGE
    up = oc.run(P(initial=0, consecutive=1, cooldown=0), [(30.0, 10.0)] * 6)
    assert [a for _, a in resizes(up)] == [1, 1, 1, 1] and up[-1][0] == 4


def test_amortization_blocks_a_switch_that_cannot_pay_off():
    # at 6:2 with rollout 30 s / training 10 s the work is 60 + 60 GPU-s; at 5:3 the step would take
    # max(60/3, 60/5) = 20 s, a gain of 10 s per step: 18 steps (180 s) do not cover 187 s, 19 do
    trace = [(30.0, 10.0)] * 20
    blocked = oc.run(P(initial=0, consecutive=3, switch_cost=187.0, horizon=18), trace)
    assert resizes(blocked) == [] and blocked[2][2] == oc.AMORTIZE
    assert resizes(oc.run(P(initial=0, consecutive=3, switch_cost=187.0, horizon=19), trace))[0] == (2, 1)
    assert oc.predicted_gain(P(initial=0), 0, 1, [(30.0, 10.0)]) == 10.0


def test_no_move_into_a_worse_split():
    # at 4:4, training 25.5 s vs rollout 20 s (r = -0.216) points toward training, but 5:3 would take
    # max(80/3, 102/5) = 26.7 s > 25.5 s: the controller holds instead of thrashing
    d = oc.run(P(initial=2, consecutive=2, cooldown=0), [(20.0, 25.5)] * 10)
    assert resizes(d) == [] and d[1][2] == oc.AMORTIZE and d[0][2] == oc.PERSISTENCE
    assert oc.predicted_gain(P(), 2, 1, [(20.0, 25.5)]) < 0


# ------------------------------------------------------------------ native controller == oracle
def _native(params, trace):
    h = dr.dr_hyst_create(params.train_gpus, params.rollout_gpus, params.initial, params.enter, params.exit,
                          params.consecutive, params.dwell, params.cooldown, params.switch_cost, params.horizon)
    out = []
    for tr, tt in trace:
        d = dr.dr_hyst_step(h, tr, tt)
        out.append((d["config"], d["action"], d["reason"]))
    h.close()
    return out


CASES = list(itertools.product([1, 3, 5], [0.1, 0.3], [0.0, 0.05, 0.1], [1, 2, 4], [0, 3], [0, 5, 11],
                               [(0.0, 0), (60.0, 20)]))


@pytest.mark.parametrize("part", range(4))
def test_native_controller_matches_oracle(part):
    rng = np.random.default_rng(part)
    for i, (k, enter, exit_, cons, dwell, cool, (cost, hor)) in enumerate(CASES[part::4]):
        if exit_ > enter:
            continue
        tg, rg = splits(k)
        params = P(train_gpus=tg, rollout_gpus=rg, initial=int(rng.integers(0, k)), enter=enter, exit=exit_,
                   consecutive=cons, dwell=dwell, cooldown=cool, switch_cost=cost, horizon=hor)
        trace = datagen.stage_time_trace(seed=100 * part + i, steps=120, noise=0.3,
                                         shift_at=int(rng.integers(0, 80)), shift_to=float(rng.uniform(-0.6, 0.6)))
        assert _native(params, trace) == oc.run(params, trace), (params, i)


def test_native_controller_rejects_bad_parameters():
    bad = [dict(train_gpus=[], rollout_gpus=[]), dict(initial=5), dict(enter=0.1, exit=0.2), dict(enter=1.0),
           dict(consecutive=0), dict(consecutive=(1 << 20) + 1), dict(dwell=-1), dict(cooldown=-1), dict(switch_cost=-1.0),
           dict(switch_cost=10.0, horizon=0), dict(train_gpus=[6, 5, 0, 3, 2]),
           dict(train_gpus=[5, 6, 4, 3, 2]), dict(rollout_gpus=[2, 3, 3, 5, 6]), dict(rollout_gpus=[2, 3, 4, 5])]
    for kw in bad:
        p = P(**kw)
        with pytest.raises(dr.DrError) as e:
            dr.dr_hyst_create(p.train_gpus, p.rollout_gpus, p.initial, p.enter, p.exit, p.consecutive, p.dwell,
                              p.cooldown, p.switch_cost, p.horizon)
        assert e.value.code == dr.DR_EINVAL, kw
    h = dr.dr_hyst_create([1, 1][:1], [1], 0, 0.2, 0.1, 1, 0, 0)
    for tr, tt in ((-1.0, 1.0), (float("nan"), 1.0), (1.0, float("inf"))):
        with pytest.raises(dr.DrError):
            dr.dr_hyst_step(h, tr, tt)
