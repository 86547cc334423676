"""TEST INFRASTRUCTURE -- float64 oracle of the layer around the mixer shard: the residual
stream, the normalisations, stacks of layers and decoding without the SSM cache. Only
tests/, smoke() and the CPU-baseline leg of bench.py use this module; the product path
never does, and it shares no code with the GPU library.

What it follows:
  * Section II-B: after the output projection the block returns to the residual stream
    by adding the mixer output to the incoming hidden states. Under tensor parallelism
    that output is the sum over ranks of the out_proj partials (Section IV-B, the second
    reduction), so the residual add follows the exchange.
  * Section IV-E: Falcon-Mamba uses the same selective SSM mixer; its model definition
    normalises the token-dependent fields Delta (low rank), B and C each by their RMS,
    without a weight, before they are used.
  * Section V (ablation): without the SSM cache every generated token re-processes the
    whole prefix; with it, one decode step per token.

Readings (the paper is silent on these):
  * pre-norm: an RMSNorm with a per-channel weight (eps 1e-5) in front of every mixer, and
    a final RMSNorm after the last layer;
  * the residual stream is stored in float32 (nothing rounded for act "f64"); the mixer
    input (the normed residual) is stored in the act dtype;
  * the exchange sums the out_proj partials in float32, and the sum is added to the
    residual;
  * Falcon-Mamba's norms act on the reduced x_proj output (after the first exchange): the
    delta, B and C column ranges are each divided by sqrt(mean of squares + 1e-6); the
    normalised fields are kept in float32 like x_proj's output.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import numpy as np

from . import mixer as om

RMS_EPS = 1e-5
BCDT_EPS = 1e-6


def _f32(a, act: str) -> np.ndarray:
    a = np.asarray(a, np.float64)
    return a if act == "f64" else a.astype(np.float32).astype(np.float64)


def rms_norm(x, weight: Optional[np.ndarray], eps: float) -> np.ndarray:
    """x / sqrt(mean over the last axis of x^2 + eps), times weight when given."""
    x = np.asarray(x, np.float64)
    r = x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return r if weight is None else r * np.asarray(weight, np.float64)


def bcdt_rms(x_dbl, R: int, N: int, eps: float = BCDT_EPS) -> np.ndarray:
    """Falcon-Mamba's weightless RMS norms over the delta, B and C ranges of x_proj's output."""
    x_dbl = np.asarray(x_dbl, np.float64)
    d, B, C = om.split_x_dbl(x_dbl, R, N)
    return np.concatenate([rms_norm(d, None, eps), rms_norm(B, None, eps), rms_norm(C, None, eps)], axis=1)


def residual_norm(residual, y_parts: Sequence[np.ndarray], norm_w, eps: float, act: str):
    """residual <- residual + sum of the out_proj partials (float32); returns it and the
    normed residual in the act dtype (the next mixer's input, or the stack's output)."""
    r = np.asarray(residual, np.float64)
    if len(y_parts):
        y = _f32(np.sum([np.asarray(p, np.float64) for p in y_parts], axis=0), act)
        r = _f32(r + y, act)
    return r, om.rnd(rms_norm(r, norm_w, eps), act)


def _dims(w):
    E, N = np.asarray(w["A_log"]).shape
    return E, N, np.asarray(w["W_dt"]).shape[1]


def tp_layer_prefill(shards: Sequence[dict], h, cu, slots, has_init, conv_pools, ssm_pools, act: str,
                     bcdt_eps: Optional[float] = None):
    """One mixer layer on all ranks: stage 1, the x_proj exchange, Falcon-Mamba's norms
    when bcdt_eps is given, stage 2. Returns the ranks' out_proj partials and new pools."""
    s1 = [om.prefill_stage1(w, h, cu, slots, has_init, cp, act) for w, cp in zip(shards, conv_pools)]
    red = np.sum([s["x_dbl"] for s in s1], axis=0)
    if bcdt_eps is not None:
        _, N, R = _dims(shards[0])
        red = bcdt_rms(red, R, N, bcdt_eps)
    s2 = [om.prefill_stage2(w, a, red, cu, slots, has_init, sp, act) for w, a, sp in zip(shards, s1, ssm_pools)]
    return [s["y"] for s in s2], [s["conv_pool"] for s in s1], [s["ssm_pool"] for s in s2]


def tp_layer_decode(shards: Sequence[dict], h, slots, conv_pools, ssm_pools, act: str,
                    bcdt_eps: Optional[float] = None):
    s1 = [om.decode_stage1(w, h, slots, cp, act) for w, cp in zip(shards, conv_pools)]
    red = np.sum([s["x_dbl"] for s in s1], axis=0)
    if bcdt_eps is not None:
        _, N, R = _dims(shards[0])
        red = bcdt_rms(red, R, N, bcdt_eps)
    s2 = [om.decode_stage2(w, a, red, slots, sp, act) for w, a, sp in zip(shards, s1, ssm_pools)]
    return [s["y"] for s in s2], [s["conv_pool"] for s in s1], [s["ssm_pool"] for s in s2]


def stack_prefill(layers: Sequence[Sequence[dict]], norm_ws, final_w, x, cu, slots, has_init,
                  conv_pools, ssm_pools, act: str, eps: float = RMS_EPS, bcdt_eps: Optional[float] = None):
    """A stack of mixer layers, each split over len(layers[l]) ranks (one rank = full width).

    resid_0 = x; per layer l: h = RMSNorm_l(resid_l) in the act dtype, y = the sum over ranks
    of the mixer's out_proj partials, resid_{l+1} = resid_l + y; the output is
    RMSNorm_final(resid_L). conv_pools[l][r], ssm_pools[l][r] are the layer's rank caches;
    new ones are returned (the inputs are not modified).
    """
    resid = _f32(x, act)
    new_conv: List[list] = []
    new_ssm: List[list] = []
    y_parts: list = []
    for l, shards in enumerate(layers):
        resid, h = residual_norm(resid, y_parts, norm_ws[l], eps, act)
        y_parts, cp, sp = tp_layer_prefill(shards, h, cu, slots, has_init, conv_pools[l], ssm_pools[l], act, bcdt_eps)
        new_conv.append(cp)
        new_ssm.append(sp)
    resid, out = residual_norm(resid, y_parts, final_w, eps, act)
    return {"out": out, "residual": resid, "conv_pools": new_conv, "ssm_pools": new_ssm}


def stack_decode_step(layers, norm_ws, final_w, x_t, slots, conv_pools, ssm_pools, act: str,
                      eps: float = RMS_EPS, bcdt_eps: Optional[float] = None):
    """One token per sequence through the stack, every layer advancing its own caches."""
    resid = _f32(x_t, act)
    new_conv, new_ssm, y_parts = [], [], []
    for l, shards in enumerate(layers):
        resid, h = residual_norm(resid, y_parts, norm_ws[l], eps, act)
        y_parts, cp, sp = tp_layer_decode(shards, h, slots, conv_pools[l], ssm_pools[l], act, bcdt_eps)
        new_conv.append(cp)
        new_ssm.append(sp)
    resid, out = residual_norm(resid, y_parts, final_w, eps, act)
    return {"out": out, "residual": resid, "conv_pools": new_conv, "ssm_pools": new_ssm}


def stack_no_cache_step(layers, norm_ws, final_w, prefixes: Sequence[np.ndarray], empty_conv, empty_ssm,
                        act: str, eps: float = RMS_EPS, bcdt_eps: Optional[float] = None):
    """Decoding without the SSM cache (the ablation's baseline): every sequence's whole
    prefix, ending with the current token, is prefilled from empty caches and the last
    row of each is the step's output. prefixes[i]: [L_i, d_model]."""
    lens = [len(p) for p in prefixes]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n = len(prefixes)
    x = np.concatenate([np.asarray(p, np.float64) for p in prefixes], axis=0)
    r = stack_prefill(layers, norm_ws, final_w, x, cu, np.arange(n), np.zeros(n, np.int32),
                      empty_conv, empty_ssm, act, eps, bcdt_eps)
    return r["out"][cu[1:] - 1]
