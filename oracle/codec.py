"""TEST INFRASTRUCTURE -- the oracle of the quantized exchange. Only tests/, smoke() and
the CPU-baseline leg of bench.py use this module; the product path never does.

Section IV-D of the paper lowers the precision of the tensors that the two remaining
AllReduces carry (FP32 to FP16 in the paper) for transfer and reduction, and converts
the result back for the computation that follows. Here one exchange of P partial sums
is written out plainly:

    payload_r = encode(partial_r)          on every rank r
    result    = sum over r of decode(payload_r), in rank order

which is an all-gather of the payloads followed by a local reduction. Codecs:

  f16, bf16  element-wise rounding to IEEE half / bfloat16 (ties to even);
  fp8        OCP FP8 E4M3 (bias 7, 3 mantissa bits, largest finite 448) of the row
             scaled by 448 / max|row|, one fp32 scale per row;
  int8       round-half-even of the row scaled by 127 / max|row|, one fp32 scale per row.

Reading (the paper names FP16 only; fp8 and int8 follow the same boundary): scales are
computed per row (one token of the exchanged tensor) in fp32 arithmetic, s = amax / Q and
q = clamp(x * (Q / amax), -Q, Q) with Q = 448 or 127; a row of zeros has s = 0. The
decoded value is the code times s, rounded to fp32; the sum is exact here (float64).
Inputs are finite. Every function returns integer codes so that payloads can be
compared bit for bit.
"""
from __future__ import annotations

import numpy as np

from .mixer import round_bf16

CODECS = ("f16", "bf16", "fp8", "int8")
QMAX = {"fp8": 448.0, "int8": 127.0}


def _f32(a):
    return np.asarray(a, dtype=np.float64).astype(np.float32)


# ------------------------------------------------------------------ element formats

def f16_code(x) -> np.ndarray:
    """IEEE binary16 bit patterns of fp32 values (round to nearest, ties to even)."""
    with np.errstate(over="ignore"):                 # beyond 65504 rounds to infinity, as IEEE does
        return _f32(x).astype(np.float16).view(np.uint16)


def f16_value(code) -> np.ndarray:
    return np.asarray(code, np.uint16).view(np.float16).astype(np.float64)


def bf16_code(x) -> np.ndarray:
    """bfloat16 bit patterns: the upper half of the fp32 pattern after rounding to 8
    significant bits (ties to even)."""
    r = round_bf16(_f32(x).astype(np.float64)).astype(np.float32)
    return (r.view(np.uint32) >> 16).astype(np.uint16)


def bf16_value(code) -> np.ndarray:
    return (np.asarray(code, np.uint32) << 16).astype(np.uint32).view(np.float32).astype(np.float64)


def e4m3_code(v) -> np.ndarray:
    """OCP FP8 E4M3 codes of values with |v| <= 448, rounded to nearest, ties to even.

    Normal numbers: 2**(e-7) * (1 + m/8) for exponent field e in 1..15 (e = 15, m = 7 is
    NaN, so 448 is the largest); subnormals: m * 2**-9 for e = 0. The sign is bit 7 and
    is kept for values that round to zero."""
    v = np.asarray(v, np.float64)
    if np.any(np.abs(v) > 448.0) or not np.all(np.isfinite(v)):
        raise ValueError("e4m3_code takes finite values with |v| <= 448")
    a = np.abs(v)
    _, E = np.frexp(a)                          # a = f * 2**E, 0.5 <= f < 1 (E = 0 for a = 0)
    eu = np.maximum(E - 1, -6)                  # unbiased exponent; subnormals share 2**-6
    quantum = np.ldexp(1.0, eu - 3)             # spacing of representable values near a
    k = np.rint(a / quantum).astype(np.int64)   # exact division, ties to even
    up = k == 16                                # rounded up to the next binade
    eu = np.where(up, eu + 1, eu)
    k = np.where(up, 8, k)
    normal = k >= 8
    field_e = np.where(normal, eu + 7, 0)
    field_m = np.where(normal, k - 8, k)
    code = (field_e << 3) | field_m
    return (code | np.where(np.signbit(v), 0x80, 0)).astype(np.uint8)


def e4m3_value(code) -> np.ndarray:
    c = np.asarray(code, np.int64)
    e, m = (c >> 3) & 0xF, c & 0x7
    mag = np.where(e == 0, m * 2.0 ** -9, np.ldexp(1.0 + m / 8.0, e - 7))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(c & 0x80, -mag, mag)


# ------------------------------------------------------------------ codec

def row_scales(x, codec: str):
    """(s, inv) per row in fp32: s = amax / Q, inv = Q / amax (0 for an all-zero row)."""
    xf = _f32(x)
    amax = np.max(np.abs(xf), axis=-1).astype(np.float32)
    q = np.float32(QMAX[codec])
    with np.errstate(divide="ignore"):
        inv = np.where(amax > 0, (np.float64(q) / amax.astype(np.float64)).astype(np.float32), np.float32(0))
    s = (amax.astype(np.float64) / np.float64(q)).astype(np.float32)
    return s, inv.astype(np.float32)


def encode(x, codec: str) -> dict:
    """Payload of one rank's partial x [rows][cols] (values representable in fp32)."""
    x = np.asarray(x, np.float64)
    if codec == "f16":
        return {"codes": f16_code(x), "scales": None}
    if codec == "bf16":
        return {"codes": bf16_code(x), "scales": None}
    s, inv = row_scales(x, codec)
    Q = np.float32(QMAX[codec])
    qf = (_f32(x).astype(np.float64) * inv[..., None].astype(np.float64)).astype(np.float32)  # one fp32 rounding
    qf = np.clip(qf, -Q, Q).astype(np.float64)
    if codec == "fp8":
        return {"codes": e4m3_code(qf), "scales": s}
    if codec == "int8":
        return {"codes": np.rint(qf).astype(np.int64).astype(np.int8).view(np.uint8), "scales": s}
    raise ValueError(codec)


def decode(payload: dict, codec: str) -> np.ndarray:
    """The fp32 values a payload stands for (as float64)."""
    c = payload["codes"]
    if codec == "f16":
        return f16_value(c)
    if codec == "bf16":
        return bf16_value(c)
    if codec == "fp8":
        v = e4m3_value(c)
    elif codec == "int8":
        v = np.asarray(c, np.uint8).view(np.int8).astype(np.float64)
    else:
        raise ValueError(codec)
    s = payload["scales"].astype(np.float64)[..., None]
    return (v * s).astype(np.float32).astype(np.float64)   # code times scale, rounded to fp32


def exchange(partials, codec: str) -> np.ndarray:
    """Sum over ranks of the decoded payloads (exact, float64)."""
    out = None
    for p in partials:
        d = decode(encode(p, codec), codec)
        out = d if out is None else out + d
    return out


def exact_sum(partials) -> np.ndarray:
    """The unquantized exchange: sum of the partials in float64."""
    return np.sum([np.asarray(p, np.float64) for p in partials], axis=0)
