"""CPU oracle of one selective-SSM (Mamba-1) mixer layer on one channel shard.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's CPU
baseline may import this module; the product path never does. It shares no code with
the GPU library: it is a plain, slow, float64 restatement of what the mixer computes.

What it follows (paper: "Scaling State-Space Models on Multiple GPUs with Tensor
Parallelism"):
  * Section II-B and Fig. 1 give the mixer's op order: input projection, split into an
    SSM path and a gating path, a short channel-separable convolution, a projection to
    the packed token-dependent fields (Delta, B, C), discretisation of the per-channel
    dynamics A with Delta, the state update walked over the sequence with a per-channel
    D skip, elementwise gating and an output projection.
  * The paper states these steps in prose and takes their equations from the Mamba
    selective SSM (Gu & Dao). The readings used here, where the text is silent, are:
      - discretisation: Abar = exp(Delta * A) and Bbar = Delta * B;
      - Delta = softplus(dt_proj(delta) + b_dt), softplus(v) = v for v > 20 else log(1+e^v);
      - SiLU after the convolution and on the gate;
      - the convolution is a causal cross-correlation with a bias, left-padded with the
        cached history (or zeros), so tap K-1 multiplies the current token;
      - packed orders xz = [x | z] and x_dbl = [delta | B | C];
      - no bias on in_proj, x_proj and out_proj; A = -exp(A_log).
  * Section IV-A: the cache holds the final state and the last K-1 inputs of the
    convolution per sequence, both sharded by channel.
  * Section IV-B/IV-C: each rank owns a contiguous channel range; in_proj's x and z rows,
    the convolution, dt_proj, A, D are sliced by channel, x_proj and out_proj by column;
    the x_proj output is summed over ranks (the first of the two reductions) and the
    out_proj output is a partial sum (the second reduction, outside this layer).

Precision: all arithmetic is float64. ``act`` selects where values are stored in a
narrower type, exactly as the GPU path stores them: "bf16" rounds xz, u, dt (and delta
as dt_proj's input), g and y_partial to bf16 (ties to even); "f32" rounds the same
points to float32; "f64" rounds nothing and keeps the state in float64 (used by the
invariant checks). The SSM state is stored as float32 unless act == "f64".
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "round_bf16", "rnd", "softplus", "silu", "shard_weights", "in_proj", "conv1d_silu",
    "x_proj", "split_x_dbl", "dt_proj", "discretize", "ssm_recurrence", "gate", "out_proj",
    "selective_scan", "prefill_stage1", "prefill_stage2", "prefill", "decode_stage1",
    "decode_stage2", "decode_step", "tp_prefill", "tp_decode_step",
]


# ---------------------------------------------------------------------------- rounding
def round_bf16(a) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (8 significant bits, ties to even)."""
    a = np.asarray(a, dtype=np.float64)
    _, e = np.frexp(a)               # a = m * 2**e with 0.5 <= |m| < 1
    # spacing of bf16 values near a: 2**(e-8) for normal values, 2**-133 below 2**-126
    q = np.maximum(e, -125) - 8
    r = np.ldexp(np.rint(np.ldexp(a, -q)), q)
    return np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, a), r)


def rnd(a, act: str) -> np.ndarray:
    """Storage rounding to the activation dtype."""
    a = np.asarray(a, dtype=np.float64)
    if act == "bf16":
        return round_bf16(a)
    if act == "f32":
        return a.astype(np.float32).astype(np.float64)
    if act == "f64":
        return a
    raise ValueError(act)


def _state_store(h: np.ndarray, act: str) -> np.ndarray:
    return h if act == "f64" else h.astype(np.float32).astype(np.float64)


def softplus(v):
    """softplus(v) = log(1 + exp(v)), taken as v itself above 20."""
    v = np.asarray(v, dtype=np.float64)
    return np.where(v > 20.0, v, np.log1p(np.exp(np.minimum(v, 20.0))))


def silu(v):
    """SiLU(v) = v * sigmoid(v)."""
    v = np.asarray(v, dtype=np.float64)
    return v / (1.0 + np.exp(-v))


# ------------------------------------------------------------------ channel splitter
def shard_weights(full: Dict[str, np.ndarray], shard_index: int, shard_count: int) -> Dict[str, np.ndarray]:
    """Slice full-width layer weights to one rank's contiguous channel range (Section IV-B).

    in_proj's x rows and z rows are sliced separately so that the shard's packed output
    is [x_shard | z_shard]; x_proj and out_proj are sliced by input column; the
    convolution, dt_proj, b_dt, A_log and D by channel.
    """
    E_tot = full["conv_w"].shape[0]
    assert E_tot % shard_count == 0
    E = E_tot // shard_count
    c0, c1 = shard_index * E, (shard_index + 1) * E
    W_in = full["W_in"]
    return {
        "W_in": np.concatenate([W_in[c0:c1], W_in[E_tot + c0:E_tot + c1]], axis=0),
        "conv_w": full["conv_w"][c0:c1], "conv_b": full["conv_b"][c0:c1],
        "W_x": full["W_x"][:, c0:c1], "W_dt": full["W_dt"][c0:c1], "b_dt": full["b_dt"][c0:c1],
        "A_log": full["A_log"][c0:c1], "D": full["D"][c0:c1], "W_out": full["W_out"][:, c0:c1],
    }


# ------------------------------------------------------------------------- stages
def in_proj(w, x, act: str) -> np.ndarray:
    """Input projection to the packed [x | z] tensor (Section II-B, Fig. 1)."""
    return rnd(np.asarray(x, np.float64) @ np.asarray(w["W_in"], np.float64).T, act)


def conv1d_silu(w, xs: np.ndarray, conv_state0: Optional[np.ndarray], act: str) -> Tuple[np.ndarray, np.ndarray]:
    """Causal depthwise convolution over time for one sequence, then SiLU.

    xs: [L, E] SSM-path inputs. conv_state0: [E, K-1] cached history, oldest first, or
    None for a fresh sequence (zeros). Returns u [L, E] and the new history [E, K-1]:
    the last K-1 entries of history-then-inputs (Section IV-A, Section IV-B).
    """
    cw = np.asarray(w["conv_w"], np.float64)
    cb = np.asarray(w["conv_b"], np.float64)
    E, K = cw.shape
    L = xs.shape[0]
    hist = np.zeros((K - 1, E)) if conv_state0 is None else np.asarray(conv_state0, np.float64).T
    xt = np.concatenate([hist, np.asarray(xs, np.float64)], axis=0)       # [L+K-1, E]
    acc = np.zeros((L, E)) + cb[None, :]
    for j in range(K):
        acc = acc + cw[None, :, j] * xt[j:j + L]
    u = rnd(silu(acc), act)
    new_state = xt[L:L + K - 1].T.copy()                                  # [E, K-1]
    return u, new_state


def x_proj(w, u: np.ndarray) -> np.ndarray:
    """Projection to the packed token-dependent fields; a partial sum over the shard's channels."""
    return np.asarray(u, np.float64) @ np.asarray(w["W_x"], np.float64).T


def split_x_dbl(x_dbl: np.ndarray, R: int, N: int):
    """Unpack [delta | B | C] by column ranges (Section IV-C)."""
    return x_dbl[:, :R], x_dbl[:, R:R + N], x_dbl[:, R + N:R + 2 * N]


def dt_proj(w, delta: np.ndarray, act: str) -> np.ndarray:
    """Per-channel step-size projection of the low-rank delta (bias added at discretisation)."""
    return rnd(rnd(delta, act) @ np.asarray(w["W_dt"], np.float64).T, act)


def discretize(dt: np.ndarray, b_dt, A_log):
    """Delta = softplus(dt + b_dt) per token and channel; A = -exp(A_log) per channel and state."""
    return softplus(dt + np.asarray(b_dt, np.float64)[None, :]), -np.exp(np.asarray(A_log, np.float64))


def ssm_recurrence(u, delta, A, B, C, D, h0):
    """The state update walked over one sequence (Section II-B).

    h_t = exp(Delta_t * A) * h_{t-1} + Delta_t * B_t * u_t ;  y_t = C_t . h_t + D * u_t
    Shapes: u, delta [L, E]; A [E, N]; B, C [L, N]; D [E]; h0 [E, N]. Returns y [L, E], h [E, N].
    """
    u = np.asarray(u, np.float64)
    L, E = u.shape
    h = np.array(h0, dtype=np.float64, copy=True)
    y = np.empty((L, E))
    Dv = np.asarray(D, np.float64)
    for t in range(L):
        h = np.exp(delta[t][:, None] * A) * h + (delta[t] * u[t])[:, None] * B[t][None, :]
        y[t] = h @ C[t] + Dv * u[t]
    return y, h


def gate(y, z, act: str) -> np.ndarray:
    """Gating path: elementwise product with SiLU(z)."""
    return rnd(np.asarray(y, np.float64) * silu(z), act)


def out_proj(w, g, act: str) -> np.ndarray:
    """Output projection; on a shard this is a partial sum over its channels."""
    return rnd(np.asarray(g, np.float64) @ np.asarray(w["W_out"], np.float64).T, act)


def selective_scan(w, u, dt, z, B, C, h0, act: str):
    """Discretisation, recurrence, D skip and gate for one sequence. Returns g [L, E], h [E, N]."""
    delta, A = discretize(dt, w["b_dt"], w["A_log"])
    y, h = ssm_recurrence(u, delta, A, B, C, w["D"], h0)
    return gate(y, z, act), h


# ------------------------------------------------------------------- whole layer
def _seq_ranges(cu_seqlens) -> List[Tuple[int, int]]:
    cu = [int(v) for v in cu_seqlens]
    return [(cu[i], cu[i + 1]) for i in range(len(cu) - 1)]


def prefill_stage1(w, x, cu_seqlens, cache_slot, has_init, conv_pool, act: str) -> dict:
    """in_proj, convolution + SiLU and x_proj over packed sequences; writes conv history.

    Returns the stage's values and a new conv pool (the input pool is not modified).
    """
    E = w["conv_w"].shape[0]
    xz = in_proj(w, x, act)
    xs = xz[:, :E]
    u = np.empty_like(xs)
    pool = np.array(conv_pool, dtype=np.float64, copy=True)
    for i, (a, b) in enumerate(_seq_ranges(cu_seqlens)):
        s = int(cache_slot[i])
        st0 = pool[s] if has_init[i] else None
        u[a:b], pool[s] = conv1d_silu(w, xs[a:b], st0, act)
    return {"xz": xz, "u": u, "x_dbl": x_proj(w, u), "conv_pool": pool}


def prefill_stage2(w, st1: dict, x_dbl_reduced, cu_seqlens, cache_slot, has_init, ssm_pool, act: str) -> dict:
    """dt_proj, the selective scan per sequence and out_proj; writes the final states."""
    E, N = w["A_log"].shape
    R = w["W_dt"].shape[1]
    delta, B, C = split_x_dbl(np.asarray(x_dbl_reduced, np.float64), R, N)
    dt = dt_proj(w, delta, act)
    z = st1["xz"][:, E:2 * E]
    g = np.empty((z.shape[0], E))
    pool = np.array(ssm_pool, dtype=np.float64, copy=True)
    for i, (a, b) in enumerate(_seq_ranges(cu_seqlens)):
        s = int(cache_slot[i])
        h0 = pool[s] if has_init[i] else np.zeros((E, N))
        g[a:b], h = selective_scan(w, st1["u"][a:b], dt[a:b], z[a:b], B[a:b], C[a:b], h0, act)
        pool[s] = _state_store(h, act)
    return {"dt": dt, "g": g, "y": out_proj(w, g, act), "ssm_pool": pool}


def prefill(w, x, cu_seqlens, cache_slot, has_init, conv_pool, ssm_pool, act: str) -> dict:
    """One shard with the first reduction taken as the identity (exact when there is one shard)."""
    s1 = prefill_stage1(w, x, cu_seqlens, cache_slot, has_init, conv_pool, act)
    s2 = prefill_stage2(w, s1, s1["x_dbl"], cu_seqlens, cache_slot, has_init, ssm_pool, act)
    return {**s1, **s2}


def decode_stage1(w, x_t, cache_slot, conv_pool, act: str) -> dict:
    """One token per sequence: in_proj, then the cached window shifted by one and convolved."""
    cw = np.asarray(w["conv_w"], np.float64)
    cb = np.asarray(w["conv_b"], np.float64)
    E, K = cw.shape
    xz = in_proj(w, x_t, act)
    pool = np.array(conv_pool, dtype=np.float64, copy=True)
    u = np.empty((xz.shape[0], E))
    for i in range(xz.shape[0]):
        s = int(cache_slot[i])
        window = np.concatenate([pool[s], xz[i, :E][:, None]], axis=1)    # [E, K], oldest first
        u[i] = rnd(silu(cb + np.sum(cw * window, axis=1)), act)
        pool[s] = window[:, 1:]
    return {"xz": xz, "u": u, "x_dbl": x_proj(w, u), "conv_pool": pool}


def decode_stage2(w, st1: dict, x_dbl_reduced, cache_slot, ssm_pool, act: str) -> dict:
    """One recurrence step per sequence on its cached state, in place of a rescan (Section IV-A)."""
    E, N = w["A_log"].shape
    R = w["W_dt"].shape[1]
    delta, B, C = split_x_dbl(np.asarray(x_dbl_reduced, np.float64), R, N)
    dt = dt_proj(w, delta, act)
    Dlt, A = discretize(dt, w["b_dt"], w["A_log"])
    D = np.asarray(w["D"], np.float64)
    pool = np.array(ssm_pool, dtype=np.float64, copy=True)
    g = np.empty((dt.shape[0], E))
    for i in range(dt.shape[0]):
        s = int(cache_slot[i])
        u = st1["u"][i]
        h = np.exp(Dlt[i][:, None] * A) * pool[s] + (Dlt[i] * u)[:, None] * B[i][None, :]
        y = h @ C[i] + D * u
        g[i] = rnd(y * silu(st1["xz"][i, E:2 * E]), act)
        pool[s] = _state_store(h, act)
    return {"dt": dt, "g": g, "y": out_proj(w, g, act), "ssm_pool": pool}


def decode_step(w, x_t, cache_slot, conv_pool, ssm_pool, act: str) -> dict:
    s1 = decode_stage1(w, x_t, cache_slot, conv_pool, act)
    s2 = decode_stage2(w, s1, s1["x_dbl"], cache_slot, ssm_pool, act)
    return {**s1, **s2}


# -------------------------------------------------------------- tensor parallel
def tp_prefill(shards: Sequence[dict], x, cu_seqlens, cache_slot, has_init, conv_pools, ssm_pools, act: str):
    """All ranks of a channel split: x_proj partials are summed over ranks between the stages."""
    s1 = [prefill_stage1(w, x, cu_seqlens, cache_slot, has_init, cp, act) for w, cp in zip(shards, conv_pools)]
    red = np.sum([s["x_dbl"] for s in s1], axis=0)
    s2 = [prefill_stage2(w, a, red, cu_seqlens, cache_slot, has_init, sp, act)
          for w, a, sp in zip(shards, s1, ssm_pools)]
    return s1, s2, red


def tp_decode_step(shards: Sequence[dict], x_t, cache_slot, conv_pools, ssm_pools, act: str):
    s1 = [decode_stage1(w, x_t, cache_slot, cp, act) for w, cp in zip(shards, conv_pools)]
    red = np.sum([s["x_dbl"] for s in s1], axis=0)
    s2 = [decode_stage2(w, a, red, cache_slot, sp, act) for w, a, sp in zip(shards, s1, ssm_pools)]
    return s1, s2, red
