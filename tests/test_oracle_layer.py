"""Pins of the layer oracle (residual stream, pre-norm, Falcon-Mamba's delta/B/C norms,
stacks of layers, decoding without the cache) against things other than itself: torch's
RMS norm, an independent pure-Python stack loop, exact special cases and the cache and
shard invariants. Planted mistakes at the end must each fail a pin. No GPU needed.
"""
import numpy as np
import pytest
import torch

from oracle import layer as ol
from oracle import mixer as om
from oracle import naive
from paper_2602_21144_amd import synth


def _f64(w):
    return {k: np.asarray(v, np.float64) for k, v in w.items() if not k.startswith("_")}


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def _stack(n_layers, shard_count, seed, act="f64"):
    shape = synth.tiny_shape(shard_count=1, act="f32")
    st = synth.make_stack(shape, n_layers, seed, general=True)
    full = [_f64(w) for w in st["layers"]]
    layers = [[om.shard_weights(w, r, shard_count) for r in range(shard_count)] for w in full]
    return shape, st, full, layers


def _pools(shape, layers, S):
    E = shape.d_inner
    conv = [[np.zeros((S, len(w["conv_b"]), shape.d_conv - 1)) for w in sh] for sh in layers]
    ssm = [[np.zeros((S, len(w["conv_b"]), shape.d_state)) for w in sh] for sh in layers]
    assert sum(len(w["conv_b"]) for w in layers[0]) == E
    return conv, ssm


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(0)
    for d, eps in ((8, 1e-5), (37, 1e-6), (2560, 1e-5)):
        x = rng.normal(size=(5, d)) * rng.uniform(0.01, 100, size=(5, 1))
        w = rng.uniform(0.5, 1.5, size=d)
        ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (d,), torch.from_numpy(w), eps).numpy()
        assert _rel(ol.rms_norm(x, w, eps), ref) < 1e-14
        ref1 = torch.nn.functional.rms_norm(torch.from_numpy(x), (d,), None, eps).numpy()
        assert _rel(ol.rms_norm(x, None, eps), ref1) < 1e-14


def test_bcdt_rms_matches_torch_per_range():
    rng = np.random.default_rng(1)
    R, N = 5, 4
    x = rng.normal(size=(7, R + 2 * N)) * np.array([100.0] * R + [0.01] * N + [3.0] * N)
    got = ol.bcdt_rms(x, R, N, 1e-6)
    t = torch.from_numpy(x)
    for a, b in ((0, R), (R, R + N), (R + N, R + 2 * N)):
        ref = torch.nn.functional.rms_norm(t[:, a:b], (b - a,), None, 1e-6).numpy()
        assert _rel(got[:, a:b], ref) < 1e-14


@pytest.mark.parametrize("bcdt", [None, ol.BCDT_EPS])
def test_stack_matches_naive_loop(bcdt):
    shape, st, full, layers = _stack(2, 1, 3)
    rng = np.random.default_rng(2)
    L = 9
    x = rng.normal(size=(L, shape.d_model))
    conv, ssm = _pools(shape, layers, 1)
    got = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x, [0, L], [0], [0], conv, ssm, "f64",
                           bcdt_eps=bcdt)["out"]
    ref = naive.stack_sequence(full, st["norm_w"], st["final_w"], x.tolist(), ol.RMS_EPS, bcdt)
    assert _rel(got, ref) < 1e-12


def test_zero_mixer_output_leaves_the_residual():
    """Every out_proj zero: the stack's output is the final norm of its input, exactly."""
    shape, st, full, layers = _stack(3, 2, 4)
    for sh in layers:
        for w in sh:
            w["W_out"] = np.zeros_like(w["W_out"])
    rng = np.random.default_rng(3)
    x = rng.normal(size=(6, shape.d_model))
    conv, ssm = _pools(shape, layers, 1)
    r = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x, [0, 6], [0], [0], conv, ssm, "f64")
    assert np.array_equal(r["residual"], x)
    assert _rel(r["out"], ol.rms_norm(x, st["final_w"], ol.RMS_EPS)) < 1e-15


@pytest.mark.parametrize("bcdt", [None, ol.BCDT_EPS])
def test_stack_shard_invariant(bcdt):
    """Splitting every layer over 2 or 3 ranks leaves the stack's output unchanged."""
    rng = np.random.default_rng(5)
    x = rng.normal(size=(10, 8))
    outs = []
    for P in (1, 2, 3):
        shape, st, full, layers = _stack(2, P, 6)
        conv, ssm = _pools(shape, layers, 2)
        outs.append(ol.stack_prefill(layers, st["norm_w"], st["final_w"], x, [0, 4, 10], [1, 0], [0, 0], conv, ssm,
                                     "f64", bcdt_eps=bcdt)["out"])
    assert _rel(outs[1], outs[0]) < 1e-12 and _rel(outs[2], outs[0]) < 1e-12


@pytest.mark.parametrize("bcdt", [None, ol.BCDT_EPS])
def test_stack_cache_invariant_and_no_cache_decode(bcdt):
    """Prefill of L tokens then k decode steps = a prefill of L + k tokens, per sequence and
    layer; decoding without the cache (re-prefilling each prefix) gives the same outputs."""
    shape, st, full, layers = _stack(2, 2, 7)
    rng = np.random.default_rng(8)
    lens, k = [5, 3], 4
    seqs = [rng.normal(size=(n + k, shape.d_model)) for n in lens]
    args = (layers, st["norm_w"], st["final_w"])
    conv, ssm = _pools(shape, layers, 3)
    slots = np.array([2, 0])
    x = np.concatenate([s[:n] for s, n in zip(seqs, lens)])
    cu = [0, lens[0], sum(lens)]
    r = ol.stack_prefill(*args, x, cu, slots, [0, 0], conv, ssm, "f64", bcdt_eps=bcdt)
    cp, sp = r["conv_pools"], r["ssm_pools"]
    dec = []
    for j in range(k):
        xt = np.stack([s[n + j] for s, n in zip(seqs, lens)])
        d = ol.stack_decode_step(*args, xt, slots, cp, sp, "f64", bcdt_eps=bcdt)
        cp, sp = d["conv_pools"], d["ssm_pools"]
        dec.append(d["out"])
        e_conv, e_ssm = _pools(shape, layers, 2)
        nc = ol.stack_no_cache_step(*args, [s[:n + j + 1] for s, n in zip(seqs, lens)], e_conv, e_ssm, "f64",
                                    bcdt_eps=bcdt)
        assert _rel(nc, d["out"]) < 1e-12, f"no-cache step {j}"
    for i, (s, n) in enumerate(zip(seqs, lens)):
        conv1, ssm1 = _pools(shape, layers, 1)
        full_r = ol.stack_prefill(*args, s, [0, n + k], [0], [0], conv1, ssm1, "f64", bcdt_eps=bcdt)
        assert _rel(np.stack([dd[i] for dd in dec]), full_r["out"][n:]) < 1e-12
        for l in range(len(layers)):
            for rk in range(2):
                assert _rel(sp[l][rk][slots[i]], full_r["ssm_pools"][l][rk][0]) < 1e-12


def test_bcdt_norms_make_x_proj_scale_irrelevant():
    """With Falcon-Mamba's norms, scaling x_proj's weights by 3 changes nothing but the eps term."""
    shape, st, full, layers = _stack(1, 1, 9)
    rng = np.random.default_rng(10)
    x = rng.normal(size=(8, shape.d_model))
    conv, ssm = _pools(shape, layers, 1)
    a = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x, [0, 8], [0], [0], conv, ssm, "f64",
                         bcdt_eps=ol.BCDT_EPS)["out"]
    scaled = [[dict(w, W_x=3.0 * w["W_x"]) for w in sh] for sh in layers]
    b = ol.stack_prefill(scaled, st["norm_w"], st["final_w"], x, [0, 8], [0], [0], conv, ssm, "f64",
                         bcdt_eps=ol.BCDT_EPS)["out"]
    c = ol.stack_prefill(scaled, st["norm_w"], st["final_w"], x, [0, 8], [0], [0], conv, ssm, "f64")["out"]
    assert _rel(b, a) < 1e-4
    assert _rel(c, a) > 1e-3    # without the norms the scale does matter


# ------------------------------------------------------------------ planted mistakes
def _pins():
    return [lambda: test_stack_matches_naive_loop(None), lambda: test_stack_matches_naive_loop(ol.BCDT_EPS),
            test_zero_mixer_output_leaves_the_residual, lambda: test_stack_shard_invariant(ol.BCDT_EPS)]


def _caught():
    for p in _pins():
        try:
            p()
        except AssertionError:
            return True
    return False


_ORIG = {k: getattr(ol, k) for k in ("residual_norm", "bcdt_rms", "tp_layer_prefill", "rms_norm")}


def _residual_dropped(residual, y_parts, norm_w, eps, act):
    if len(y_parts):
        residual = np.sum([np.asarray(p, np.float64) for p in y_parts], axis=0)
    return _ORIG["residual_norm"](residual, [], norm_w, eps, act)


def _norm_weight_ignored(residual, y_parts, norm_w, eps, act):
    return _ORIG["residual_norm"](residual, y_parts, None, eps, act)


def _bcdt_over_whole_row(x_dbl, R, N, eps=ol.BCDT_EPS):
    return ol.rms_norm(x_dbl, None, eps)


def _bcdt_before_exchange(shards, h, cu, slots, has_init, conv_pools, ssm_pools, act, bcdt_eps=None):
    s1 = [om.prefill_stage1(w, h, cu, slots, has_init, cp, act) for w, cp in zip(shards, conv_pools)]
    E, N = shards[0]["A_log"].shape
    R = shards[0]["W_dt"].shape[1]
    parts = [s["x_dbl"] if bcdt_eps is None else _ORIG["bcdt_rms"](s["x_dbl"], R, N, bcdt_eps) for s in s1]
    red = np.sum(parts, axis=0)
    s2 = [om.prefill_stage2(w, a, red, cu, slots, has_init, sp, act) for w, a, sp in zip(shards, s1, ssm_pools)]
    return [s["y"] for s in s2], [s["conv_pool"] for s in s1], [s["ssm_pool"] for s in s2]


def _rms_without_mean(x, weight, eps):
    x = np.asarray(x, np.float64)
    r = x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)
    return r if weight is None else r * np.asarray(weight, np.float64)


@pytest.mark.parametrize("name,fn", [("residual_norm", _residual_dropped), ("residual_norm", _norm_weight_ignored),
                                     ("bcdt_rms", _bcdt_over_whole_row),
                                     ("tp_layer_prefill", _bcdt_before_exchange), ("rms_norm", _rms_without_mean)])
def test_planted_mistakes_are_caught(monkeypatch, name, fn):
    assert not _caught()
    monkeypatch.setattr(ol, name, fn)
    assert _caught(), f"planted mistake {fn.__name__} went unnoticed"
