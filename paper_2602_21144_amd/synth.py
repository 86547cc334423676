"""Seeded synthetic inputs for one selective-SSM mixer layer.

This module only draws numbers. It holds none of the mixer's arithmetic, so both the
CPU oracle (through the tests) and the GPU path can take their inputs from it.

Shapes follow the Mamba-style mixer (Section II-B): full-width weights for an
``E_tot``-channel layer are drawn first, in a fixed order, from
``numpy.random.Generator(PCG64(seed))``; the token activations follow. Values meant
for bf16 storage are the fp32 draws rounded to bf16 with round-to-nearest-even, so
the same numbers reach the oracle (as float64) and the GPU (as bf16).

Init recipe (per layer):
  * ``W_in [2*E_tot, d_model]``, ``conv_w [E_tot, K]``, ``conv_b [E_tot]``,
    ``W_x [R+2N, E_tot]``, ``W_dt [E_tot, R]``, ``W_out [d_model, E_tot]`` ~ N(0, 0.02);
  * step-size bias: ``dt0 = exp(U[ln 1e-3, ln 0.1])`` per channel and ``b_dt`` its
    inverse softplus, so the initial step sizes are log-uniform in [1e-3, 0.1];
  * ``A_log[c, n] = log(n + 1)`` (n counted from 0) and ``D = 1``;
  * token activations ``x ~ N(0, 1)``.
The "stress" init instead scales the matrices so that the state path dominates the
output (``W_in ~ N(0, 1/sqrt(d_model))``, ``conv_w ~ N(0, 1/sqrt(K))``,
``W_x ~ N(0, 1/sqrt(E_tot))``, ``W_dt ~ N(0, 1/sqrt(R))``, ``D = 0``).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

__all__ = [
    "LayerShape", "CONFIGS", "round_bf16_f32", "make_layer", "make_general_layer", "make_tokens",
    "packed_schedule", "serving_schedule", "make_slots", "tiny_shape",
]


@dataclasses.dataclass(frozen=True)
class LayerShape:
    """Dimensions of one mixer layer and of the shard that is run on one GPU."""
    d_model: int
    d_inner: int          # E_tot, full width of the intermediate channels
    d_state: int          # N
    dt_rank: int          # R
    d_conv: int = 4       # K
    shard_count: int = 1  # P, channel-split degree
    act: str = "bf16"     # storage dtype of activations and weights: "bf16" | "f32"

    @property
    def d_shard(self) -> int:
        assert self.d_inner % self.shard_count == 0
        return self.d_inner // self.shard_count

    @property
    def w_dbl(self) -> int:
        return self.dt_rank + 2 * self.d_state


# Workloads: shapes of Mamba-130m, Mamba-2.8B, Falcon-Mamba-7B and a hybrid-stack mixer.
CONFIGS: Dict[str, dict] = {
    # Mamba-130m-shaped, full width, fp32; batch 1, prefill 256 then 16 decode steps.
    "mamba130m_f32": dict(shape=LayerShape(768, 1536, 16, 48, 4, 1, "f32"), seed=0,
                          batch=1, prefill_len=256, decode_steps=16),
    # Mamba-2.8B-shaped, shard of a 2-way split, bf16; batch 8, prefill 2048 then 128 decode.
    "mamba2.8b_tp2": dict(shape=LayerShape(2560, 5120, 16, 160, 4, 2, "bf16"), seed=1,
                          batch=8, prefill_len=2048, decode_steps=128),
    # Falcon-Mamba-7B-shaped long prefill, shard of a 4-way split; batch 4, L=16384.
    "falcon7b_tp4_long": dict(shape=LayerShape(4096, 8192, 16, 256, 4, 4, "bf16"), seed=2,
                              batch=4, prefill_len=16384, decode_steps=0),
    # Decode-heavy serving, Mamba-2.8B shape, shard of a 4-way split: 256 sequences,
    # 512-token prefill to fill the cache, then 512 decode steps.
    "mamba2.8b_tp4_decode": dict(shape=LayerShape(2560, 5120, 16, 160, 4, 4, "bf16"), seed=3,
                                 batch=256, prefill_len=512, decode_steps=512),
    # Hybrid-stack mixer, shard of a 2-way split: 64 prompts U[128, 8192], packed and
    # prefilled in 2048-token chunks interleaved with decode steps (64 per sequence).
    "hybrid3584_tp2_mixed": dict(shape=LayerShape(3584, 7168, 16, 224, 4, 2, "bf16"), seed=4,
                                 batch=64, len_range=(128, 8192), chunk=2048, decode_steps=64),
}


def tiny_shape(shard_count: int = 1, act: str = "f32", d_state: int = 4) -> LayerShape:
    """A layer small enough for pure-Python loops: d_model 8, E_tot 6, N 4, R 2, K 4."""
    return LayerShape(8, 6, d_state, 2, 4, shard_count, act)


def round_bf16_f32(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32 holding them."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # add 0x7FFF plus the lowest kept bit, then clear the 16 dropped bits; finite values
    # never carry out of 32 bits (the largest finite float rounds to infinity's pattern)
    r = (u >> 16) & 1
    r += 0x7FFF
    r += u
    r &= 0xFFFF0000
    out = r.view(np.float32)
    # NaN stays NaN (not produced by the draws; kept for completeness)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = a[nan]
    return out


def _store(a: np.ndarray, act: str) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    return round_bf16_f32(a) if act == "bf16" else a


def make_layer(shape: LayerShape, seed: int, stress: bool = False,
               rng: Optional[np.random.Generator] = None) -> Dict[str, np.ndarray]:
    """Full-width weights of one layer (float32 arrays; act-dtype ones already rounded).

    Returns the generator too (key ``"_rng"``) so that token draws continue the same stream.
    """
    g = rng if rng is not None else np.random.Generator(np.random.PCG64(seed))
    dm, E, N, R, K = shape.d_model, shape.d_inner, shape.d_state, shape.dt_rank, shape.d_conv
    W = R + 2 * N
    s = (lambda fan: 1.0 / math.sqrt(fan)) if stress else (lambda fan: 0.02)
    W_in = g.normal(0.0, s(dm), size=(2 * E, dm)).astype(np.float32)
    conv_w = g.normal(0.0, s(K), size=(E, K)).astype(np.float32)
    conv_b = g.normal(0.0, 0.02, size=(E,)).astype(np.float32)
    W_x = g.normal(0.0, s(E), size=(W, E)).astype(np.float32)
    W_dt = g.normal(0.0, s(R), size=(E, R)).astype(np.float32)
    log_dt0 = g.uniform(math.log(1e-3), math.log(0.1), size=(E,))
    W_out = g.normal(0.0, 0.02 if not stress else s(E), size=(dm, E)).astype(np.float32)
    dt0 = np.exp(log_dt0)
    # inverse of softplus at dt0: log(exp(dt0) - 1), written stably
    b_dt = (dt0 + np.log(-np.expm1(-dt0))).astype(np.float32)
    A_log = np.log(np.arange(1, N + 1, dtype=np.float64))[None, :].repeat(E, 0).astype(np.float32)
    D = np.zeros(E, np.float32) if stress else np.ones(E, np.float32)
    act = shape.act
    return {
        "W_in": _store(W_in, act), "conv_w": _store(conv_w, act), "conv_b": _store(conv_b, act),
        "W_x": _store(W_x, act), "W_dt": _store(W_dt, act), "W_out": _store(W_out, act),
        "b_dt": b_dt, "A_log": A_log, "D": D, "_rng": g,
    }


def make_general_layer(shape: LayerShape, seed: int) -> Dict[str, np.ndarray]:
    """Weights with no structure to lean on: every matrix ~ N(0, 1/sqrt(fan_in)), A_log ~
    U[-1, 1.5] independently per (channel, state), D ~ N(0, 1), b_dt ~ U[-4, 0].

    Used by the checks, so that a result cannot pass by accident of a symmetric A or D = 1.
    """
    g = np.random.Generator(np.random.PCG64(seed))
    dm, E, N, R, K = shape.d_model, shape.d_inner, shape.d_state, shape.dt_rank, shape.d_conv
    W = R + 2 * N
    nrm = lambda fan, size: g.normal(0.0, 1.0 / math.sqrt(fan), size=size).astype(np.float32)
    out = {
        "W_in": nrm(dm, (2 * E, dm)), "conv_w": nrm(K, (E, K)), "conv_b": nrm(4, (E,)),
        "W_x": nrm(E, (W, E)), "W_dt": nrm(R, (E, R)), "W_out": nrm(E, (dm, E)),
    }
    out = {k: _store(v, shape.act) for k, v in out.items()}
    out["b_dt"] = g.uniform(-4.0, 0.0, size=(E,)).astype(np.float32)
    out["A_log"] = g.uniform(-1.0, 1.5, size=(E, N)).astype(np.float32)
    out["D"] = g.normal(0.0, 1.0, size=(E,)).astype(np.float32)
    out["_rng"] = g
    return out


def make_stack(shape: LayerShape, n_layers: int, seed: int, general: bool = False, stress: bool = False) -> dict:
    """Weights of a stack of mixer layers with pre-norm residual blocks: full-width layer
    weights per layer (``make_layer`` or ``make_general_layer``, drawn one after another
    from one generator for make_layer), then per-channel norm weights 1 + U[-0.5, 0.5]
    (float32) for every layer and for the final norm."""
    g = np.random.Generator(np.random.PCG64(seed))
    if general:
        layers = [make_general_layer(shape, seed * 1000 + l) for l in range(n_layers)]
    else:
        layers = [make_layer(shape, seed, stress=stress, rng=g) for _ in range(n_layers)]
    for w in layers:
        w.pop("_rng", None)
    norm_w = [(1.0 + g.uniform(-0.5, 0.5, size=shape.d_model)).astype(np.float32) for _ in range(n_layers)]
    final_w = (1.0 + g.uniform(-0.5, 0.5, size=shape.d_model)).astype(np.float32)
    return {"layers": layers, "norm_w": norm_w, "final_w": final_w, "_rng": g}


def make_tokens(rng: np.random.Generator, n: int, d_model: int, act: str) -> np.ndarray:
    """``n`` token activations x ~ N(0, 1), drawn as float32 and stored in the act dtype."""
    return _store(rng.standard_normal(size=(n, d_model), dtype=np.float32), act)


def make_slots(rng: np.random.Generator, nseq: int, spare: int = 16) -> np.ndarray:
    """Distinct cache slots for ``nseq`` sequences inside a pool of ``nseq + spare`` slots."""
    return rng.permutation(nseq + spare)[:nseq].astype(np.int32)


def packed_schedule(lengths: List[int], chunk: int) -> List[dict]:
    """Split prompts, concatenated in index order, into windows of ``chunk`` packed tokens.

    Each window lists its pieces as (sequence index, offset in that sequence, length);
    a piece with offset > 0 continues a sequence begun in an earlier window.
    """
    starts = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    total = int(starts[-1])
    out = []
    for w0 in range(0, total, chunk):
        w1 = min(w0 + chunk, total)
        pieces = []
        i = int(np.searchsorted(starts, w0, side="right") - 1)
        while i < len(lengths) and starts[i] < w1:
            a = max(w0, int(starts[i]))
            b = min(w1, int(starts[i + 1]))
            if b > a:
                pieces.append((i, a - int(starts[i]), b - a))
            i += 1
        out.append({"start": w0, "stop": w1, "pieces": pieces})
    return out


# ------------------------------------------------------------------ Mamba-2 (SSD) mixer
@dataclasses.dataclass(frozen=True)
class Mamba2Shape:
    """Dimensions of one Mamba-2 mixer layer and of the shard run on one GPU. The split
    is by heads; B/C groups are split when ngroups is a multiple of the shard count and
    replicated on every shard otherwise."""
    d_model: int
    nheads: int           # total heads
    headdim: int          # P
    d_state: int          # N
    ngroups: int = 1      # G, B/C groups (heads nheads/G per group)
    d_conv: int = 4       # K
    shard_count: int = 1
    act: str = "bf16"

    @property
    def d_inner(self) -> int:
        return self.nheads * self.headdim

    @property
    def heads_shard(self) -> int:
        assert self.nheads % self.shard_count == 0
        return self.nheads // self.shard_count

    @property
    def d_shard(self) -> int:
        return self.heads_shard * self.headdim

    @property
    def groups_split(self) -> bool:
        return self.ngroups % self.shard_count == 0

    @property
    def groups_shard(self) -> int:
        return self.ngroups // self.shard_count if self.groups_split else self.ngroups

    @property
    def conv_dim_shard(self) -> int:
        return self.d_shard + 2 * self.groups_shard * self.d_state

    @property
    def in_rows_shard(self) -> int:
        return 2 * self.d_shard + 2 * self.groups_shard * self.d_state + self.heads_shard


MAMBA2_CONFIGS: Dict[str, dict] = {
    # Mamba-2 2.7B-shaped (80 heads of 64, N 128, one B/C group), shard 1 of a 2-way split;
    # batch 8 x prefill 2048, then 128 decode steps.
    "mamba2_2.7b_tp2": dict(shape=Mamba2Shape(2560, 80, 64, 128, 1, 4, 2, "bf16"), seed=11,
                            batch=8, prefill_len=2048, decode_steps=128),
}


def make_mamba2_layer(shape: Mamba2Shape, seed: int, stress: bool = False,
                      rng: Optional[np.random.Generator] = None) -> Dict[str, np.ndarray]:
    """Full-width Mamba-2 weights (float32 arrays; act-dtype ones rounded). Draw order:
    W_in ([z | x | B | C | dt] rows), conv_w, conv_b ([x | B | C] channels), dt0, A, W_out.
    dt_bias = softplus^-1(dt0) with dt0 log-uniform in [1e-3, 0.1] per head; A_log =
    log(U[1, 16]) per head; D = 1 (0 under stress); norm weight 1. Stress draws the
    matrices at 1/sqrt(fan_in) so that the state path carries y."""
    g = rng if rng is not None else np.random.Generator(np.random.PCG64(seed))
    dm, H, P, N, G, K = shape.d_model, shape.nheads, shape.headdim, shape.d_state, shape.ngroups, shape.d_conv
    E = H * P
    s = (lambda fan: 1.0 / math.sqrt(fan)) if stress else (lambda fan: 0.02)
    W_in = g.normal(0.0, s(dm), size=(2 * E + 2 * G * N + H, dm)).astype(np.float32)
    conv_w = g.normal(0.0, s(K), size=(E + 2 * G * N, K)).astype(np.float32)
    conv_b = g.normal(0.0, 0.02, size=(E + 2 * G * N,)).astype(np.float32)
    dt0 = np.exp(g.uniform(math.log(1e-3), math.log(0.1), size=(H,)))
    A = g.uniform(1.0, 16.0, size=(H,))
    W_out = g.normal(0.0, 0.02 if not stress else s(E), size=(dm, E)).astype(np.float32)
    act = shape.act
    return {
        "W_in": _store(W_in, act), "conv_w": _store(conv_w, act), "conv_b": _store(conv_b, act),
        "dt_bias": (dt0 + np.log(-np.expm1(-dt0))).astype(np.float32),
        "A_log": np.log(A).astype(np.float32),
        "D": np.zeros(H, np.float32) if stress else np.ones(H, np.float32),
        "norm_w": np.ones(E, np.float32), "W_out": _store(W_out, act), "_rng": g,
    }


def serving_schedule(lengths: List[int], chunk: int, decode_steps: int) -> List[tuple]:
    """The chunked serving schedule of a mixed batch: prompts concatenated in index order
    and prefilled in windows of ``chunk`` packed tokens (``packed_schedule``); after each
    window, one decode step for every sequence whose prompt is complete and that has fewer
    than ``decode_steps`` decode tokens; after the last window, decode steps until every
    sequence has ``decode_steps``.

    Returns a list of ("prefill", window) and ("decode", [(sequence, k), ...]) entries, k
    being that sequence's decode index (which decode input it consumes).
    """
    ndec = [0] * len(lengths)
    ready: List[int] = []
    out: List[tuple] = []

    def decode_round():
        batch = [(i, ndec[i]) for i in ready if ndec[i] < decode_steps]
        if batch:
            out.append(("decode", batch))
            for i, _ in batch:
                ndec[i] += 1

    for w in packed_schedule(lengths, chunk):
        out.append(("prefill", w))
        for p in w["pieces"]:
            if p[1] + p[2] == lengths[p[0]]:
                ready.append(p[0])
        decode_round()
    while any(n < decode_steps for n in ndec):
        decode_round()
    return out
