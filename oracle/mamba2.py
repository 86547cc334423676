"""TEST INFRASTRUCTURE -- float64 oracle of one shard of a Mamba-2 (SSD) mixer layer. Only
tests/, smoke() and the CPU-baseline leg of bench.py use this module.

Section II-A and Section IV-E of the paper: Mamba-2 keeps the mixer pipeline (projection,
convolution, state update, gating, output projection) and reformulates the state update
so that it maps onto matrix products; tensor parallelism reuses the same sharding and
exchange principles, adapted to Mamba-2's packed parameter layout. The paper defers the
equations to the Mamba-2 paper; this module writes the published mixer out plainly, per
token and per head (the chunked matrix form is the GPU's business, not the oracle's):

  zxbcdt = W_in x                       packed rows [z | x | B | C | dt]
  u      = SiLU(causal depthwise conv over [x | B | C])      (cache: last K-1 inputs)
  Delta  = softplus(dt + dt_bias)       one per head;   A = -exp(A_log), one per head
  per head h (B, C of its group g):     h_t = exp(Delta_t A) h_{t-1} + Delta_t x_t B_t^T
                                        y_t = h_t C_t + D x_t          (h_t: headdim x N)
  g      = y * SiLU(z);  g_norm = g / sqrt(mean over the norm group of g^2 + eps) * norm_w
  y_partial = W_out g_norm              (this shard's out_proj partial sum)

Sharding (readings): heads are split; B/C groups are split when ngroups is a multiple of
the shard count and replicated otherwise; the gated norm's group is d_inner / ngroups
channels, so when it spans shards its sum of squares is exchanged (summed over shards)
before normalising. Stage 1 ends at that exchange, stage 2 normalises and projects.
Storage rounding (act dtype): the in_proj output, u, g and g_norm, y_partial; states fp32.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .mixer import rnd, silu, softplus

NORM_EPS = 1e-5


def _seq_ranges(cu) -> List[Tuple[int, int]]:
    cu = [int(v) for v in cu]
    return [(cu[i], cu[i + 1]) for i in range(len(cu) - 1)]


def _state_store(h, act):
    return h if act == "f64" else np.asarray(h, np.float64).astype(np.float32).astype(np.float64)


def shard_weights(full: Dict[str, np.ndarray], shape, r: int) -> Dict[str, np.ndarray]:
    """Shard r's slice of the full weights (Section IV-B, IV-E): its heads' rows of z, x and
    dt, its B/C groups (all of them when groups are replicated), its conv channels, its
    heads' dt_bias, A_log, D, its channels of norm_w and its columns of W_out."""
    H, P, N, G = shape.heads_shard, shape.headdim, shape.d_state, shape.ngroups
    E_tot, E = shape.d_inner, shape.d_shard
    Gs = shape.groups_shard
    g0 = r * Gs if shape.groups_split else 0
    c0 = r * E
    W_in = np.asarray(full["W_in"])
    zr = W_in[c0:c0 + E]
    xr = W_in[E_tot + c0:E_tot + c0 + E]
    Br = W_in[2 * E_tot + g0 * N:2 * E_tot + (g0 + Gs) * N]
    Cr = W_in[2 * E_tot + G * N + g0 * N:2 * E_tot + G * N + (g0 + Gs) * N]
    dtr = W_in[2 * E_tot + 2 * G * N + r * H:2 * E_tot + 2 * G * N + (r + 1) * H]
    cw, cb = np.asarray(full["conv_w"]), np.asarray(full["conv_b"])
    conv_idx = np.concatenate([np.arange(c0, c0 + E), E_tot + np.arange(g0 * N, (g0 + Gs) * N),
                               E_tot + G * N + np.arange(g0 * N, (g0 + Gs) * N)])
    hs = slice(r * H, (r + 1) * H)
    return {"W_in": np.concatenate([zr, xr, Br, Cr, dtr], axis=0), "conv_w": cw[conv_idx], "conv_b": cb[conv_idx],
            "dt_bias": np.asarray(full["dt_bias"])[hs], "A_log": np.asarray(full["A_log"])[hs],
            "D": np.asarray(full["D"])[hs], "norm_w": np.asarray(full["norm_w"])[c0:c0 + E],
            "W_out": np.asarray(full["W_out"])[:, c0:c0 + E]}


def head_groups(shape, r: int) -> np.ndarray:
    """Local B/C group index of each of the shard's heads."""
    hpg = shape.nheads // shape.ngroups
    g = (r * shape.heads_shard + np.arange(shape.heads_shard)) // hpg
    return g - r * shape.groups_shard if shape.groups_split else g


def norm_groups(shape, r: int) -> np.ndarray:
    """Global norm-group index of each of the shard's channels (group size d_inner / ngroups)."""
    return (r * shape.d_shard + np.arange(shape.d_shard)) // (shape.d_inner // shape.ngroups)


# ------------------------------------------------------------------ steps
def split(shape, zxbcdt):
    E, GN, H = shape.d_shard, shape.groups_shard * shape.d_state, shape.heads_shard
    return zxbcdt[:, :E], zxbcdt[:, E:2 * E + 2 * GN], zxbcdt[:, 2 * E + 2 * GN:2 * E + 2 * GN + H]


def conv1d_silu(w, xbc, conv_state0, act):
    """Causal depthwise conv + SiLU over [x | B | C] of one sequence; returns u and the new
    history (last K-1 inputs of history-then-inputs, oldest first)."""
    cw = np.asarray(w["conv_w"], np.float64)
    cb = np.asarray(w["conv_b"], np.float64)
    Cc, K = cw.shape
    L = xbc.shape[0]
    hist = np.zeros((K - 1, Cc)) if conv_state0 is None else np.asarray(conv_state0, np.float64).T
    xt = np.concatenate([hist, np.asarray(xbc, np.float64)], axis=0)
    acc = np.zeros((L, Cc)) + cb[None, :]
    for j in range(K):
        acc = acc + cw[None, :, j] * xt[j:j + L]
    return rnd(silu(acc), act), xt[L:L + K - 1].T.copy()


def ssd_recurrence(xs, delta, A, B, C, D, h0, groups):
    """Per-head scalar-decay recurrence, token by token.

    xs [L, H, P], delta [L, H], A [H] (negative), B and C [L, Gs, N], D [H], h0 [H, P, N],
    groups [H] (local group of each head). Returns y [L, H, P] and the final state."""
    L, H, Pd = xs.shape
    h = np.asarray(h0, np.float64).copy()
    y = np.zeros((L, H, Pd))
    for t in range(L):
        dA = np.exp(delta[t] * A)                                        # [H]
        Bt, Ct = B[t][groups], C[t][groups]                              # [H, N]
        h = dA[:, None, None] * h + delta[t][:, None, None] * xs[t][:, :, None] * Bt[:, None, :]
        y[t] = np.einsum("hpn,hn->hp", h, Ct) + D[:, None] * xs[t]
    return y, h


def mixer_core(w, shape, r, zxbcdt, conv_state0, h0, act):
    """One sequence from its in_proj output: conv, scan and gate. Returns g [L, E] (act-
    rounded), the new conv history and the final state."""
    H, Pd, N, Gs = shape.heads_shard, shape.headdim, shape.d_state, shape.groups_shard
    E = shape.d_shard
    z, xbc, dt = split(shape, zxbcdt)
    u, hist = conv1d_silu(w, xbc, conv_state0, act)
    L = u.shape[0]
    xs = u[:, :E].reshape(L, H, Pd)
    Bm = u[:, E:E + Gs * N].reshape(L, Gs, N)
    Cm = u[:, E + Gs * N:E + 2 * Gs * N].reshape(L, Gs, N)
    delta = softplus(dt + np.asarray(w["dt_bias"], np.float64)[None, :])
    A = -np.exp(np.asarray(w["A_log"], np.float64))
    y, h = ssd_recurrence(xs, delta, A, Bm, Cm, np.asarray(w["D"], np.float64), h0, head_groups(shape, r))
    g = rnd(y.reshape(L, E) * silu(z), act)
    return g, hist, h


def group_sumsq(shape, r, g) -> np.ndarray:
    """[T, ngroups]: sum of g^2 over the shard's channels of each norm group (a partial sum
    to be added over shards)."""
    ng = norm_groups(shape, r)
    out = np.zeros((g.shape[0], shape.ngroups))
    for k in range(shape.ngroups):
        m = ng == k
        if m.any():
            out[:, k] = np.sum(np.asarray(g, np.float64)[:, m] ** 2, axis=1)
    return out


def norm_out(w, shape, r, g, sumsq, act):
    """Gated RMSNorm's normalisation (with the summed sum of squares) and out_proj."""
    gsize = shape.d_inner // shape.ngroups
    ng = norm_groups(shape, r)
    inv = 1.0 / np.sqrt(np.asarray(sumsq, np.float64)[:, ng] / gsize + NORM_EPS)
    gn = rnd(np.asarray(g, np.float64) * inv * np.asarray(w["norm_w"], np.float64)[None, :], act)
    return rnd(gn @ np.asarray(w["W_out"], np.float64).T, act)


# ------------------------------------------------------------------ stages
def prefill_stage1(w, shape, r, x, cu, slots, has_init, conv_pool, ssm_pool, act) -> dict:
    """Packed prefill up to the norm exchange: g [T, E], the partial sums of squares
    [T, ngroups], and the updated pools (conv [S, C, K-1], ssm [S, H, P, N])."""
    zx = rnd(np.asarray(x, np.float64) @ np.asarray(w["W_in"], np.float64).T, act)
    conv_pool = np.array(conv_pool, np.float64, copy=True)
    ssm_pool = np.array(ssm_pool, np.float64, copy=True)
    T = zx.shape[0]
    g = np.zeros((T, shape.d_shard))
    H, Pd, N = shape.heads_shard, shape.headdim, shape.d_state
    for i, (a, b) in enumerate(_seq_ranges(cu)):
        s = int(slots[i])
        cont = bool(has_init[i])
        c0 = conv_pool[s] if cont else None
        h0 = ssm_pool[s] if cont else np.zeros((H, Pd, N))
        if b == a:
            if not cont:
                conv_pool[s] = 0.0
                ssm_pool[s] = 0.0
            continue
        gi, hist, h = mixer_core(w, shape, r, zx[a:b], c0, h0, act)
        g[a:b] = gi
        conv_pool[s] = rnd(hist, act)
        ssm_pool[s] = _state_store(h, act)
    return {"g": g, "sumsq": group_sumsq(shape, r, g), "conv_pool": conv_pool, "ssm_pool": ssm_pool}


def prefill_stage2(w, shape, r, st1, sumsq_reduced, act) -> np.ndarray:
    return norm_out(w, shape, r, st1["g"], sumsq_reduced, act)


def decode_stage1(w, shape, r, x_t, slots, conv_pool, ssm_pool, act) -> dict:
    """One token per active sequence (every one continues from its cached state)."""
    zx = rnd(np.asarray(x_t, np.float64) @ np.asarray(w["W_in"], np.float64).T, act)
    conv_pool = np.array(conv_pool, np.float64, copy=True)
    ssm_pool = np.array(ssm_pool, np.float64, copy=True)
    Bd = zx.shape[0]
    g = np.zeros((Bd, shape.d_shard))
    for i in range(Bd):
        s = int(slots[i])
        gi, hist, h = mixer_core(w, shape, r, zx[i:i + 1], conv_pool[s], ssm_pool[s], act)
        g[i] = gi[0]
        conv_pool[s] = rnd(hist, act)
        ssm_pool[s] = _state_store(h, act)
    return {"g": g, "sumsq": group_sumsq(shape, r, g), "conv_pool": conv_pool, "ssm_pool": ssm_pool}


def decode_stage2(w, shape, r, st1, sumsq_reduced, act) -> np.ndarray:
    return norm_out(w, shape, r, st1["g"], sumsq_reduced, act)


def tp_prefill(full, shape, x, cu, slots, has_init, conv_pools, ssm_pools, act):
    """All shards: stage 1 on each, the sums of squares added over shards, stage 2 on each.
    Returns (stage-1 results, y_partials)."""
    shards = [shard_weights(full, shape, r) for r in range(shape.shard_count)]
    s1 = [prefill_stage1(shards[r], shape, r, x, cu, slots, has_init, conv_pools[r], ssm_pools[r], act)
          for r in range(shape.shard_count)]
    red = np.sum([s["sumsq"] for s in s1], axis=0)
    return s1, [prefill_stage2(shards[r], shape, r, s1[r], red, act) for r in range(shape.shard_count)]


def tp_decode_step(full, shape, x_t, slots, conv_pools, ssm_pools, act):
    shards = [shard_weights(full, shape, r) for r in range(shape.shard_count)]
    s1 = [decode_stage1(shards[r], shape, r, x_t, slots, conv_pools[r], ssm_pools[r], act)
          for r in range(shape.shard_count)]
    red = np.sum([s["sumsq"] for s in s1], axis=0)
    return s1, [decode_stage2(shards[r], shape, r, s1[r], red, act) for r in range(shape.shard_count)]
