"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of an oracle function (on the CPU, via
monkeypatch) and checks that at least one pin test fails with it.
"""
import numpy as np
import pytest

import oracle
import oracle.staging as st
from tests import test_oracle_cast as tc
from tests import test_oracle_checksum as tk
from tests import test_oracle_layout as tl

_ORIG_RNE = st.rne_bf16


def _fails(fn, *args):
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


def _patch(monkeypatch, name, fn):
    monkeypatch.setattr(st, name, fn)
    monkeypatch.setattr(oracle, name, fn)
    for mod in (tc, tk, tl):
        if hasattr(mod, name):
            monkeypatch.setattr(mod, name, fn)


# ------------------------------------------------------------------ cast mistakes
def _rne_half_up(bits):
    u = np.asarray(bits, dtype=np.uint32)
    out = (u + np.uint32(0x8000)) >> np.uint32(16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    return np.where(nan, (u >> np.uint32(16)) | np.uint32(0x40), out).astype(np.uint16)


def _rne_truncate(bits):
    return (np.asarray(bits, dtype=np.uint32) >> np.uint32(16)).astype(np.uint16)


def _rne_ftz(bits):
    u = np.asarray(bits, dtype=np.uint32)
    sub = (u & np.uint32(0x7F800000)) == 0
    return _ORIG_RNE(np.where(sub, u & np.uint32(0x80000000), u))


def _rne_nan_unquiet(bits):
    u = np.asarray(bits, dtype=np.uint32)
    out = _ORIG_RNE(u).astype(np.uint32)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    return np.where(nan, u >> np.uint32(16), out).astype(np.uint16)


@pytest.mark.parametrize("bad", [_rne_half_up, _rne_truncate, _rne_ftz, _rne_nan_unquiet])
def test_cast_mistakes_caught(bad, monkeypatch, golden_dir):
    _patch(monkeypatch, "rne_bf16", bad)
    caught = [
        _fails(tc.test_hand_derived_table, golden_dir),
        _fails(tc.test_exact_rational_rounding),
        _fails(tc.test_nan_stays_nan_with_sign_and_quiet_bit),
    ]
    assert any(caught)


# ------------------------------------------------------------------ layout mistakes
def _mutated_rollout_rank(kind):
    orig = st.rollout_rank

    def fn(src, m, t, r):
        out = orig(src, m, t, r)
        qh, kh, fr, vr = m.n_q_heads // t, m.n_kv_heads // t, m.ffn // t, m.vocab // t
        D = m.head_dim
        res = []
        for name, a in out:
            base = name.split(".")[-1]
            lay = name[: -len(base)]
            if kind == "qkv_order" and base == "qkv":
                a = np.concatenate([a[: qh * D], a[(qh + kh) * D:], a[qh * D:(qh + kh) * D]])
            elif kind == "o_wrong_rank" and base == "o":
                q = ((r + 1) % t) * qh * D
                a = _ORIG_RNE(src[lay + "o"][:, q:q + qh * D])
            elif kind == "down_wrong_rank" and base == "down":
                f = ((r + 1) % t) * fr
                a = _ORIG_RNE(src[lay + "down"][:, f:f + fr])
            elif kind == "embed_from_lm_head" and base == "embed":
                a = _ORIG_RNE(src["lm_head"][r * vr:(r + 1) * vr])
            elif kind == "norm_rank0_only" and base in ("ln1", "ln2") and r > 0:
                a = np.zeros_like(a)
            elif kind == "gate_up_swapped" and base == "gate_up":
                a = np.concatenate([a[fr:], a[:fr]])
            res.append((name, a))
        return res

    return fn


@pytest.mark.parametrize("kind", ["qkv_order", "o_wrong_rank", "down_wrong_rank", "embed_from_lm_head",
                                  "norm_rank0_only", "gate_up_swapped"])
def test_layout_mistakes_caught(kind, monkeypatch, golden_dir):
    _patch(monkeypatch, "rollout_rank", _mutated_rollout_rank(kind))
    caught = [_fails(tl.test_tiny_worked_example, golden_dir)] + [_fails(tl.test_tagged_brute_force, p) for p in range(2)]
    assert any(caught), kind


def test_training_order_mistake_caught(monkeypatch, golden_dir):
    orig = st.training_tensors

    def swapped(m):
        out = orig(m)
        i = next(k for k, (n, _) in enumerate(out) if n.endswith(".gate"))
        out[i], out[i + 1] = out[i + 1], out[i]
        return out

    _patch(monkeypatch, "training_tensors", swapped)
    assert _fails(tl.test_tiny_worked_example, golden_dir)


# ------------------------------------------------------------------ checksum / chunk mistakes
def _cks_j0(chunk):
    w = np.ascontiguousarray(chunk).view(np.uint8).ravel().view("<u4").astype(np.uint64)
    j = np.arange(w.size, dtype=np.uint64)
    return int(w.sum(dtype=np.uint64)), int((j * w).sum(dtype=np.uint64))


def _cks_big_endian(chunk):
    w = np.ascontiguousarray(chunk).view(np.uint8).ravel().view(">u4").astype(np.uint64)
    j = np.arange(1, w.size + 1, dtype=np.uint64)
    return int(w.sum(dtype=np.uint64)), int((j * w).sum(dtype=np.uint64))


@pytest.mark.parametrize("bad", [_cks_j0, _cks_big_endian])
def test_checksum_mistakes_caught(bad, monkeypatch):
    _patch(monkeypatch, "checksum", bad)
    caught = [_fails(tk.test_single_word_position), _fails(tk.test_little_endian_words_from_bf16_pairs),
              _fails(tk.test_big_int_reference_with_wraparound)]
    assert any(caught)


def test_chunk_span_mistake_caught(monkeypatch):
    def off_by_one(total, budget):
        return [(c, min(c + budget - 16, total)) for c in range(0, total, budget)]

    _patch(monkeypatch, "chunk_spans", off_by_one)
    assert _fails(tl.test_chunk_spans, 5264384, 262144)


# ------------------------------------------------------------------ reshard and moment-stream mistakes
def _reshard_pad_one(flat, n, w2):
    out = np.ones(st.padded_elems(n, w2), dtype=flat.dtype)
    out[:n] = flat[:n]
    return out


def _reshard_pad_half(flat, n, w2):
    size = -(-n // (w2 * 128)) * (w2 * 128)
    out = np.zeros(size, dtype=flat.dtype)
    out[:n] = flat[:n]
    return out


def _reshard_drop_last(flat, n, w2):
    out = np.zeros(st.padded_elems(n, w2), dtype=flat.dtype)
    out[:n - 1] = flat[:n - 1]
    return out


@pytest.mark.parametrize("bad", [_reshard_pad_one, _reshard_pad_half, _reshard_drop_last])
def test_reshard_mistakes_caught(bad, monkeypatch):
    _patch(monkeypatch, "reshard", bad)
    caught = [_fails(tl.test_reshard_keeps_every_element_and_repads, w, w2)
              for w, w2 in ((4, 3), (1, 8), (8, 1), (3, 64), (5, 5))]
    assert any(caught)


def _moments_interleaved(m_shards, v_shards):
    parts = []
    for m, v in zip(m_shards, v_shards):
        parts += [np.ascontiguousarray(m).view(np.uint8).ravel(), np.ascontiguousarray(v).view(np.uint8).ravel()]
    return np.concatenate(parts)


def _moments_v_first(m_shards, v_shards):
    return _ORIG_MOMENTS(v_shards, m_shards)


_ORIG_MOMENTS = st.moment_stream


@pytest.mark.parametrize("bad", [_moments_interleaved, _moments_v_first])
def test_moment_stream_mistakes_caught(bad, monkeypatch):
    _patch(monkeypatch, "moment_stream", bad)
    assert _fails(tk.test_moment_stream_order)


# ------------------------------------------------------------------ controller mistakes
from oracle import controller as oc  # noqa: E402
from tests import test_hysteresis as th  # noqa: E402


def _controller_variant(kind):
    orig = oc.run

    def fn(params, trace):
        p = oc.Params(**vars(params))
        if kind == "no_hysteresis":
            p.exit = p.enter
        elif kind == "short_cooldown":
            p.cooldown = max(0, p.cooldown - 1)
        elif kind == "no_dwell":
            p.dwell = 0
        elif kind == "no_amortize":
            p.switch_cost = 0.0
        elif kind == "one_less_signal":
            p.consecutive = max(1, p.consecutive - 1)
        return orig(p, trace)

    return fn


@pytest.mark.parametrize("kind", ["no_hysteresis", "short_cooldown", "no_dwell", "no_amortize", "one_less_signal"])
def test_controller_mistakes_caught(kind, monkeypatch):
    monkeypatch.setattr(oc, "run", _controller_variant(kind))
    caught = [_fails(f) for f in (th.test_sustained_imbalance_resizes_after_consecutive_then_cooldown,
                                  th.test_dwell_holds_a_fresh_configuration,
                                  th.test_hysteresis_band_keeps_a_signal_alive,
                                  th.test_amortization_blocks_a_switch_that_cannot_pay_off,
                                  th.test_oscillation_shorter_than_consecutive_never_resizes)]
    assert any(caught), kind


# ------------------------------------------------------------------ widening mistakes
def _widen_zero(bits16):
    return np.zeros(np.asarray(bits16).shape, dtype=np.uint32)


def _widen_shift15(bits16):
    return np.asarray(bits16, dtype=np.uint16).astype(np.uint32) << np.uint32(15)


def _widen_low_half(bits16):
    return np.asarray(bits16, dtype=np.uint16).astype(np.uint32)


@pytest.mark.parametrize("bad", [_widen_zero, _widen_shift15, _widen_low_half])
def test_widen_mistakes_caught(bad, monkeypatch):
    _patch(monkeypatch, "widen_bf16", bad)
    caught = [_fails(tc.test_widen_closed_forms), _fails(tc.test_widen_is_exact_on_every_pattern),
              _fails(tc.test_widen_against_torch), _fails(tc.test_cast_undoes_widen),
              _fails(tl.test_round_trip_inverse, 2)]
    assert all(caught[:4]) and caught[4], caught
