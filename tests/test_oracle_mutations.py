"""Plant plausible mistakes in the oracle (CPU only) and check that its pins catch each one.

A pin that cannot fail is no pin. Every mutation below is a mistake a reader of the
mixer's description could make; the brute-force loop, the hand-worked examples or the
closed forms must reject each.
"""
import math

import numpy as np
import pytest

from oracle import mixer as om
from oracle import naive
from paper_2602_21144_amd import synth

import test_oracle_pins as pins


def _pins_pass() -> bool:
    checks = [
        lambda: pins.test_oracle_matches_naive_loop_full_width(0),
        lambda: pins.test_tp_shards_match_naive_full_width(2),
        pins.test_scan_hand_worked_example,
        pins.test_conv_hand_worked_example,
        lambda: pins.test_lti_closed_form(0),
        pins.test_scan_special_cases,
        pins.test_conv_matches_torch_grouped_conv1d,
        lambda: pins.test_state_cache_invariant_prefill_then_decode("f64"),
        pins.test_bf16_rounding_points_worked_example,
        pins.test_bf16_storage_points_are_bf16_values,
    ]
    for c in checks:
        try:
            c()
        except AssertionError:
            return False
    return True


def test_unmutated_oracle_passes():
    assert _pins_pass()


_orig = {k: getattr(om, k) for k in ("in_proj", "conv1d_silu", "split_x_dbl", "discretize",
                                      "ssm_recurrence", "gate", "silu", "shard_weights", "x_proj",
                                      "dt_proj", "out_proj")}


def _swap_xz(w, x, act):
    xz = _orig["in_proj"](w, x, act)
    E = xz.shape[1] // 2
    return np.concatenate([xz[:, E:], xz[:, :E]], axis=1)


def _reversed_taps(w, xs, st0, act):
    w2 = dict(w)
    w2["conv_w"] = np.asarray(w["conv_w"])[:, ::-1]
    return _orig["conv1d_silu"](w2, xs, st0, act)


def _stale_history(w, xs, st0, act):
    u, st = _orig["conv1d_silu"](w, xs, st0, act)
    return u, np.roll(st, 1, axis=1)


def _swap_bc(x_dbl, R, N):
    d, B, C = _orig["split_x_dbl"](x_dbl, R, N)
    return d, C, B


def _no_softplus(dt, b_dt, A_log):
    _, A = _orig["discretize"](dt, b_dt, A_log)
    return dt + np.asarray(b_dt)[None, :], A


def _a_without_exp(dt, b_dt, A_log):
    d, _ = _orig["discretize"](dt, b_dt, A_log)
    return d, -np.asarray(A_log, np.float64)


def _zoh_b(u, delta, A, B, C, D, h0):
    # exact zero-order hold for B instead of the Delta*B reading
    u = np.asarray(u, np.float64)
    L, E = u.shape
    h = np.array(h0, dtype=np.float64, copy=True)
    y = np.empty((L, E))
    for t in range(L):
        dA = np.exp(delta[t][:, None] * A)
        h = dA * h + ((dA - 1.0) / A * u[t][:, None]) * B[t][None, :]
        y[t] = h @ C[t] + D * u[t]
    return y, h


def _no_d_skip(u, delta, A, B, C, D, h0):
    return _orig["ssm_recurrence"](u, delta, A, B, C, np.zeros_like(np.asarray(D)), h0)


def _state_before_update(u, delta, A, B, C, D, h0):
    # read out the state before it absorbs the current token
    u = np.asarray(u, np.float64)
    L, E = u.shape
    h = np.array(h0, dtype=np.float64, copy=True)
    y = np.empty((L, E))
    for t in range(L):
        y[t] = h @ C[t] + D * u[t]
        h = np.exp(delta[t][:, None] * A) * h + (delta[t] * u[t])[:, None] * B[t][None, :]
    return y, h


def _gate_without_silu(y, z, act):
    return om.rnd(np.asarray(y) * np.asarray(z), act)


def _silu_as_sigmoid(v):
    v = np.asarray(v, np.float64)
    return 1.0 / (1.0 + np.exp(-v))


def _shard_interleaved(full, r, P):
    s = _orig["shard_weights"](full, r, P)
    E_tot = full["conv_w"].shape[0]
    E = E_tot // P
    s["W_in"] = full["W_in"][np.r_[r * 2 * E: (r + 1) * 2 * E]] if 2 * E * (r + 1) <= 2 * E_tot else s["W_in"]
    return s


def _delta_unrounded(w, delta, act):
    # dt_proj fed the fp32 delta instead of its bf16 rounding
    return om.rnd(np.asarray(delta, np.float64) @ np.asarray(w["W_dt"], np.float64).T, act)


def _dt_unrounded(w, delta, act):
    return om.rnd(delta, act) @ np.asarray(w["W_dt"], np.float64).T


def _dt_rounded_after_bias(w, delta, act):
    # dt_proj's output kept exact; the rounding moved behind the bias add (below)
    return om.rnd(delta, act) @ np.asarray(w["W_dt"], np.float64).T


def _discretize_rounding_sum(dt, b_dt, A_log):
    v = om.round_bf16(np.asarray(dt, np.float64) + np.asarray(b_dt, np.float64)[None, :])
    return om.softplus(v), -np.exp(np.asarray(A_log, np.float64))


def _gate_unrounded(y, z, act):
    return np.asarray(y, np.float64) * om.silu(z)


def _out_proj_unrounded(w, g, act):
    return np.asarray(g, np.float64) @ np.asarray(w["W_out"], np.float64).T


def _u_unrounded(w, xs, st0, act):
    return _orig["conv1d_silu"](w, xs, st0, "f64")


def _xz_unrounded(w, x, act):
    return _orig["in_proj"](w, x, "f64")


MUTATIONS = {
    "x and z halves swapped": ("in_proj", _swap_xz),
    "convolution taps reversed": ("conv1d_silu", _reversed_taps),
    "conv history off by one": ("conv1d_silu", _stale_history),
    "B and C swapped": ("split_x_dbl", _swap_bc),
    "softplus dropped": ("discretize", _no_softplus),
    "A without exp": ("discretize", _a_without_exp),
    "zero-order-hold B": ("ssm_recurrence", _zoh_b),
    "D skip dropped": ("ssm_recurrence", _no_d_skip),
    "output read before update": ("ssm_recurrence", _state_before_update),
    "gate without SiLU": ("gate", _gate_without_silu),
    "SiLU as sigmoid": ("silu", _silu_as_sigmoid),
    "in_proj sliced as one block": ("shard_weights", _shard_interleaved),
    "delta not rounded before dt_proj": ("dt_proj", _delta_unrounded),
    "dt not rounded": ("dt_proj", _dt_unrounded),
    "xz not rounded": ("in_proj", _xz_unrounded),
    "u not rounded": ("conv1d_silu", _u_unrounded),
    "g not rounded": ("gate", _gate_unrounded),
    "y_partial not rounded": ("out_proj", _out_proj_unrounded),
}


def test_pins_catch_rounding_moved_behind_the_bias(monkeypatch):
    """dt kept exact by dt_proj and rounded only after the bias is added (two coordinated edits)."""
    monkeypatch.setattr(om, "dt_proj", _dt_rounded_after_bias)
    monkeypatch.setattr(om, "discretize", _discretize_rounding_sum)
    assert not _pins_pass()


@pytest.mark.parametrize("name", list(MUTATIONS))
def test_pins_catch_mutation(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(om, attr, fn)
    assert not _pins_pass(), f"pins did not catch: {name}"
