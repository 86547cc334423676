"""Pins of the Mamba-2 (SSD) mixer oracle (CPU): the brute-force loop, the pinned Mamba-1
recurrence it reduces to, closed forms and special cases, the cache, chunking and shard
invariants, torch's RMS norm, and planted mistakes that each must fail a pin.
"""
import numpy as np
import pytest

from oracle import mamba2 as o2
from oracle import mixer as om
from oracle import naive
from paper_2602_21144_amd import synth

torch = pytest.importorskip("torch")


def _tiny(P=1, G=1, act="f64", stress=True, seed=0, H=4, Pd=3, N=5, dm=6):
    sh = synth.Mamba2Shape(dm, H, Pd, N, G, 4, P, act)
    full = synth.make_mamba2_layer(sh, seed, stress=stress)
    w = {k: np.asarray(v, np.float64) for k, v in full.items() if not k.startswith("_")}
    w["norm_w"] = np.random.default_rng(seed + 1).uniform(0.5, 1.5, size=w["norm_w"].shape)
    w["D"] = np.random.default_rng(seed + 2).normal(size=w["D"].shape)
    return sh, w


def _full_prefill(sh, w, x, act="f64"):
    """Unsplit layer on one sequence: y [L, d_model] and the final state."""
    r = 0
    H, Pd, N, K = sh.heads_shard, sh.headdim, sh.d_state, sh.d_conv
    C = sh.conv_dim_shard
    s1, ys = o2.tp_prefill(w, sh, x, [0, len(x)], [0], [0], [np.zeros((1, C, K - 1))], [np.zeros((1, H, Pd, N))], act)
    return ys[0], s1[0]["ssm_pool"][0]


@pytest.mark.parametrize("G", [1, 2])
def test_matches_naive_loop(G):
    sh, w = _tiny(G=G, H=4)
    x = np.random.default_rng(3).normal(size=(7, sh.d_model))
    y, h = _full_prefill(sh, w, x)
    yn, hn = naive.mamba2_sequence(w, sh.nheads, sh.headdim, sh.d_state, G, x)
    assert np.allclose(y, np.array(yn), rtol=1e-11, atol=1e-13)
    assert np.allclose(h, np.array(hn), rtol=1e-11, atol=1e-13)


def test_scan_reduces_to_mamba1_recurrence():
    """headdim 1, one head per channel, one B/C group: the Mamba-1 recurrence with A[c, n] = A[c]."""
    rng = np.random.default_rng(4)
    L, E, N = 9, 5, 6
    u, delta = rng.normal(size=(L, E)), rng.uniform(0.01, 0.5, size=(L, E))
    A = -rng.uniform(0.5, 3, size=E)
    B, C, D = rng.normal(size=(L, N)), rng.normal(size=(L, N)), rng.normal(size=E)
    h0 = rng.normal(size=(E, N))
    y2, h2 = o2.ssd_recurrence(u[:, :, None], delta, A, B[:, None, :], C[:, None, :], D, h0[:, None, :], np.zeros(E, int))
    y1, h1 = om.ssm_recurrence(u, delta, np.repeat(A[:, None], N, 1), B, C, D, h0)
    assert np.allclose(y2[:, :, 0], y1, rtol=1e-12) and np.allclose(h2[:, 0, :], h1, rtol=1e-12)


def test_lti_closed_form():
    """Constant Delta, B, C: y_t = sum_k (C.B) exp(Delta A (t-k)) Delta x_k + D x_t (+ decayed h0)."""
    rng = np.random.default_rng(5)
    L, H, Pd, N = 12, 3, 2, 4
    xs = rng.normal(size=(L, H, Pd))
    dl = np.full((L, H), 0.3)
    A = -np.array([0.5, 1.0, 2.0])
    b, c = rng.normal(size=N), rng.normal(size=N)
    D = rng.normal(size=H)
    h0 = rng.normal(size=(H, Pd, N))
    y, _ = o2.ssd_recurrence(xs, dl, A, np.tile(b, (L, 1, 1)), np.tile(c, (L, 1, 1)), D, h0, np.zeros(H, int))
    cb = float(c @ b)
    for t in range(L):
        for hh in range(H):
            ker = sum(cb * np.exp(0.3 * A[hh] * (t - k)) * 0.3 * xs[k, hh] for k in range(t + 1))
            ref = ker + D[hh] * xs[t, hh] + np.exp(0.3 * A[hh] * (t + 1)) * (h0[hh] @ c)
            assert np.allclose(y[t, hh], ref, rtol=1e-12)


def test_special_cases():
    rng = np.random.default_rng(6)
    L, H, Pd, N = 6, 2, 3, 4
    xs, dl = rng.normal(size=(L, H, Pd)), rng.uniform(0.1, 1, size=(L, H))
    B, C = rng.normal(size=(L, 1, N)), rng.normal(size=(L, 1, N))
    D = np.zeros(H)
    h0 = np.zeros((H, Pd, N))
    # no memory: y_t = Delta_t x_t (B_t . C_t)
    y, _ = o2.ssd_recurrence(xs, dl, np.full(H, -1e30), B, C, D, h0, np.zeros(H, int))
    assert np.allclose(y, dl[:, :, None] * xs * np.sum(B * C, axis=2)[:, :, None])
    # A = 0: the state is a running sum
    y, h = o2.ssd_recurrence(xs, dl, np.zeros(H), B, C, D, h0, np.zeros(H, int))
    href = np.einsum("th,thp,tn->hpn", dl, xs, B[:, 0])
    assert np.allclose(h, href)


def test_gated_norm_matches_torch_rms_norm():
    sh, w = _tiny(G=2, H=4)
    rng = np.random.default_rng(7)
    g = rng.normal(size=(5, sh.d_shard))
    y = o2.norm_out(w, sh, 0, g, o2.group_sumsq(sh, 0, g), "f64")
    gs = sh.d_inner // sh.ngroups
    tg = torch.from_numpy(g).reshape(5, sh.ngroups, gs)
    gn = torch.nn.functional.rms_norm(tg, (gs,), eps=o2.NORM_EPS).reshape(5, -1) * torch.from_numpy(w["norm_w"])
    ref = gn.numpy() @ w["W_out"].T
    assert np.allclose(y, ref, rtol=1e-12)


@pytest.mark.parametrize("act", ["f64", "f32"])
def test_state_cache_invariant(act):
    """Prefill of L tokens then k decode steps equals a prefill of L + k tokens."""
    sh, w = _tiny(G=1, H=4, act=act)
    rng = np.random.default_rng(8)
    L, k = 9, 4
    x = rng.normal(size=(L + k, sh.d_model))
    H, Pd, N, K, C = sh.heads_shard, sh.headdim, sh.d_state, sh.d_conv, sh.conv_dim_shard
    zc, zs = np.zeros((2, C, K - 1)), np.zeros((2, H, Pd, N))
    s_all, y_all = o2.tp_prefill(w, sh, x, [0, L + k], [1], [0], [zc], [zs], act)
    s_pre, y_pre = o2.tp_prefill(w, sh, x[:L], [0, L], [1], [0], [zc], [zs], act)
    cp, sp = [s_pre[0]["conv_pool"]], [s_pre[0]["ssm_pool"]]
    ys = [y_pre[0]]
    for i in range(k):
        d1, yd = o2.tp_decode_step(w, sh, x[L + i:L + i + 1], [1], cp, sp, act)
        cp, sp = [d1[0]["conv_pool"]], [d1[0]["ssm_pool"]]
        ys.append(yd[0])
    tol = 1e-12 if act == "f64" else 1e-5
    assert np.allclose(np.concatenate(ys), y_all[0], rtol=tol, atol=tol)
    assert np.allclose(sp[0][1], s_all[0]["ssm_pool"][1], rtol=tol, atol=tol)
    assert np.allclose(cp[0][1], s_all[0]["conv_pool"][1])


def test_chunked_prefill_and_packed_batch():
    """Two pieces through the cache equal one prefill; packing sequences changes nothing."""
    sh, w = _tiny(G=1, H=4)
    rng = np.random.default_rng(9)
    x = rng.normal(size=(13, sh.d_model))
    H, Pd, N, K, C = sh.heads_shard, sh.headdim, sh.d_state, sh.d_conv, sh.conv_dim_shard
    zc, zs = np.zeros((3, C, K - 1)), np.zeros((3, H, Pd, N))
    s_all, y_all = o2.tp_prefill(w, sh, x, [0, 13], [2], [0], [zc], [zs], "f64")
    s_a, y_a = o2.tp_prefill(w, sh, x[:2], [0, 2], [2], [0], [zc], [zs], "f64")     # piece shorter than K-1
    s_b, y_b = o2.tp_prefill(w, sh, x[2:], [0, 11], [2], [1], [s_a[0]["conv_pool"]], [s_a[0]["ssm_pool"]], "f64")
    assert np.allclose(np.concatenate([y_a[0], y_b[0]]), y_all[0], rtol=1e-12)
    assert np.allclose(s_b[0]["ssm_pool"][2], s_all[0]["ssm_pool"][2], rtol=1e-12)
    x2 = rng.normal(size=(5, sh.d_model))
    s_p, y_p = o2.tp_prefill(w, sh, np.concatenate([x, x2]), [0, 13, 18], [2, 0], [0, 0], [zc], [zs], "f64")
    s_2, y_2 = o2.tp_prefill(w, sh, x2, [0, 5], [0], [0], [zc], [zs], "f64")
    assert np.allclose(y_p[0][:13], y_all[0]) and np.allclose(y_p[0][13:], y_2[0])


@pytest.mark.parametrize("P,G", [(2, 1), (2, 2), (4, 2), (2, 4)])
def test_shards_sum_to_full_width(P, G):
    """Head split, group split or replication, and the sum-of-squares exchange: the shard
    partials add up to the unsplit layer and the shard states concatenate to its state."""
    sh1, w = _tiny(P=1, G=G, H=8, Pd=2, N=3)
    shP = synth.Mamba2Shape(sh1.d_model, sh1.nheads, sh1.headdim, sh1.d_state, G, 4, P, "f64")
    x = np.random.default_rng(10).normal(size=(6, sh1.d_model))
    y1, h1 = _full_prefill(sh1, w, x)
    H, Pd, N, K, C = shP.heads_shard, shP.headdim, shP.d_state, shP.d_conv, shP.conv_dim_shard
    s1, ys = o2.tp_prefill(w, shP, x, [0, 6], [0], [0], [np.zeros((1, C, K - 1))] * P, [np.zeros((1, H, Pd, N))] * P, "f64")
    assert np.allclose(sum(ys), y1, rtol=1e-11, atol=1e-13)
    assert np.allclose(np.concatenate([s["ssm_pool"][0] for s in s1]), h1, rtol=1e-11)


# ------------------------------------------------------------------ planted mistakes
def _pins():
    return [lambda: test_matches_naive_loop(2), test_scan_reduces_to_mamba1_recurrence, test_lti_closed_form,
            test_special_cases, test_gated_norm_matches_torch_rms_norm, lambda: test_state_cache_invariant("f64"),
            lambda: test_shards_sum_to_full_width(2, 1), lambda: test_shards_sum_to_full_width(4, 2)]


def _caught():
    for p in _pins():
        try:
            p()
        except AssertionError:
            return True
    return False


_ORIG = {k: getattr(o2, k) for k in ("ssd_recurrence", "head_groups", "norm_out", "split", "group_sumsq")}


def _decay_after_input(xs, delta, A, B, C, D, h0, groups):
    L, H, Pd = xs.shape
    h = np.array(h0, np.float64)
    y = np.zeros((L, H, Pd))
    for t in range(L):
        Bt, Ct = B[t][groups], C[t][groups]
        h = np.exp(delta[t] * A)[:, None, None] * (h + delta[t][:, None, None] * xs[t][:, :, None] * Bt[:, None, :])
        y[t] = np.einsum("hpn,hn->hp", h, Ct) + D[:, None] * xs[t]
    return y, h


def _groups_interleaved(shape, r):
    return _ORIG["head_groups"](shape, r)[::-1].copy()


def _norm_without_exchange(w, shape, r, g, sumsq, act):
    return _ORIG["norm_out"](w, shape, r, g, _ORIG["group_sumsq"](shape, r, g) * shape.shard_count, act)


def _swapped_zx(shape, zxbcdt):
    z, xbc, dt = _ORIG["split"](shape, zxbcdt)
    E = shape.d_shard
    xbc = xbc.copy()
    z2 = xbc[:, :E].copy()
    xbc[:, :E] = z
    return z2, xbc, dt


@pytest.mark.parametrize("name,fn", [("ssd_recurrence", _decay_after_input), ("head_groups", _groups_interleaved),
                                     ("norm_out", _norm_without_exchange), ("split", _swapped_zx)])
def test_planted_mistakes_are_caught(monkeypatch, name, fn):
    assert not _caught()
    monkeypatch.setattr(o2, name, fn)
    assert _caught(), f"planted mistake {fn.__name__} went unnoticed"
