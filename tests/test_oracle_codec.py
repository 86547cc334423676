"""Pins of the exchange-codec oracle (CPU): bit patterns worked out from the IEEE binary16,
bfloat16 and OCP FP8 E4M3 definitions, the conversions of an independent library
(torch's CPU bfloat16 and float8_e4m3fn types), round-half-even cases, the per-row
scaling rules, error bounds of each format, and exchanges that must be exact.
Planted mistakes in the oracle at the end must each fail one of these pins.
"""
import numpy as np
import pytest

from oracle import codec as oc

torch = pytest.importorskip("torch")


# ------------------------------------------------------------------ binary16
def test_f16_bit_patterns_from_definition():
    # 1.0 = 0 01111 0000000000; -2 = 1 10000 0...; 65504 = 0 11110 1111111111; 2**-24 = smallest subnormal
    cases = {1.0: 0x3C00, -2.0: 0xC000, 65504.0: 0x7BFF, 2.0 ** -24: 0x0001, 2.0 ** -14: 0x0400,
             65520.0: 0x7C00,                       # halfway to 2**16 rounds up to infinity
             1.0 + 2.0 ** -11: 0x3C00,              # tie between 0x3C00 and 0x3C01: even
             1.0 + 3 * 2.0 ** -11: 0x3C02,          # tie between 0x3C01 and 0x3C02: even
             2.0 ** -25: 0x0000,                    # tie between 0 and the smallest subnormal: even
             3 * 2.0 ** -25: 0x0002}
    for v, c in cases.items():
        assert int(oc.f16_code([v])[0]) == c, (v, hex(c))
    third = np.float32(1.0) / np.float32(3.0)       # 0x3EAAAAAB -> 0 01101 0101010101 (+ rounding)
    assert int(oc.f16_code([third])[0]) == 0x3555


def test_f16_value_roundtrip_of_all_finite_codes():
    codes = np.arange(0x10000, dtype=np.uint16)
    v = oc.f16_value(codes)
    fin = np.isfinite(v)
    assert np.array_equal(oc.f16_code(v[fin]), codes[fin])


# ------------------------------------------------------------------ bfloat16
def test_bf16_codes_match_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-8, 8, 20000),
                        [1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -0.0, 3e38]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oc.bf16_code(x), ref)
    assert int(oc.bf16_code([1.0 + 2.0 ** -8])[0]) == 0x3F80   # tie: even
    assert int(oc.bf16_code([1.0 + 3 * 2.0 ** -8])[0]) == 0x3F82


# ------------------------------------------------------------------ FP8 E4M3
def test_e4m3_spec_values():
    cases = {448.0: 0x7E, -448.0: 0xFE, 2.0 ** -9: 0x01, 2.0 ** -6: 0x08, 0.875 * 2.0 ** -6: 0x07, 1.0: 0x38,
             -2.0: 0xC0, 240.0: 0x77, 1.0625: 0x38,        # tie between 1.0 and 1.125: even
             1.1875: 0x3A,                                 # tie between 1.125 and 1.25: even
             232.0: 0x76,                                  # tie between 224 and 240: even
             2.0 ** -10: 0x00, 3 * 2.0 ** -10: 0x02,       # subnormal ties
             -2.0 ** -11: 0x80}                            # sign kept on a value rounding to zero
    for v, c in cases.items():
        assert int(oc.e4m3_code([v])[0]) == c, (v, hex(c))


def test_e4m3_values_of_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    got = oc.e4m3_value(codes)
    both_nan = np.isnan(ref) & np.isnan(got)
    assert np.array_equal(np.where(both_nan, 0, got), np.where(both_nan, 0, ref))
    assert np.isnan(got).sum() == 2                       # S.1111.111 only


def test_e4m3_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([np.linspace(-448, 448, 100001), rng.standard_normal(50000) * 30,
                        rng.standard_normal(50000) * 2.0 ** -7]).astype(np.float32)
    x = np.clip(x, -448, 448)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oc.e4m3_code(x), ref)


def test_e4m3_rejects_out_of_range():
    with pytest.raises(ValueError):
        oc.e4m3_code([449.0])


# ------------------------------------------------------------------ scaled codecs
@pytest.mark.parametrize("codec", ["fp8", "int8"])
def test_row_scaling(codec):
    rng = np.random.default_rng(2)
    x = (rng.standard_normal((7, 33)) * np.array([1e-3, 1, 10, 100, 1e4, 0.5, 3])[:, None]).astype(np.float32)
    x[5] = 0.0                                             # a row of zeros
    p = oc.encode(x, codec)
    s = p["scales"]
    amax = np.abs(x).max(axis=1)
    Q = oc.QMAX[codec]
    assert s.dtype == np.float32 and s[5] == 0.0
    assert np.array_equal(s, (amax.astype(np.float64) / Q).astype(np.float32))
    d = oc.decode(p, codec)
    assert np.all(d[5] == 0.0)
    # the largest entry of each row takes the largest code
    i = np.abs(x).argmax(axis=1)
    top = oc.decode(p, codec)[np.arange(7), i]
    rows = [r for r in range(7) if r != 5]
    assert np.allclose(np.abs(top[rows]), amax[rows], rtol=2.0 ** -22)
    if codec == "int8":
        q = p["codes"].view(np.int8)
        assert np.all(np.abs(q[rows, i[rows]]) == 127)
        # |error| <= half a step (one step = s), plus fp32 rounding of x * (127 / amax) and of q * s
        assert np.all(np.abs(d - x) <= 0.5 * s[:, None] * (1 + 2.0 ** -20) + np.abs(x) * 2.0 ** -22)
    else:
        assert np.all(p["codes"][rows, i[rows]] & 0x7F == 0x7E)
        # 3 mantissa bits: relative error <= 2**-4 above 2**-6 * s, absolute <= 2**-10 * s below
        bound = np.maximum(np.abs(x) * 2.0 ** -4, 2.0 ** -10 * s[:, None]) * (1 + 2.0 ** -20)
        assert np.all(np.abs(d - x) <= bound + np.abs(x) * 2.0 ** -22)


def test_int8_ties_to_even():
    x = np.array([[127.0, 2.5, 3.5, -2.5, 0.5, -0.5, 1.5]], np.float32)   # amax = 127: scale exactly 1
    p = oc.encode(x, "int8")
    assert p["scales"][0] == 1.0
    assert list(p["codes"].view(np.int8)[0]) == [127, 2, 4, -2, 0, 0, 2]


# ------------------------------------------------------------------ exchanges
def test_exchange_exact_when_representable():
    rng = np.random.default_rng(3)
    parts = [rng.integers(-100, 100, size=(5, 40)).astype(np.float32) for _ in range(4)]
    exact = oc.exact_sum(parts)
    for codec in ("f16", "bf16"):
        assert np.array_equal(oc.exchange(parts, codec), exact)
    # integer rows whose largest magnitude is 127 are exact in int8
    for p in parts:
        p[:, 0] = 127.0
        np.clip(p, -127, 127, out=p)
    assert np.array_equal(oc.exchange(parts, "int8"), oc.exact_sum(parts))


@pytest.mark.parametrize("codec,rel", [("f16", 2.0 ** -11), ("bf16", 2.0 ** -8)])
def test_exchange_error_bound_elementwise(codec, rel):
    rng = np.random.default_rng(4)
    parts = [(rng.standard_normal((16, 64)) * 3).astype(np.float32) for _ in range(3)]
    err = np.abs(oc.exchange(parts, codec) - oc.exact_sum(parts))
    bound = sum(np.abs(p).astype(np.float64) for p in parts) * rel * (1 + 1e-6) + 2.0 ** -24 * len(parts)
    assert np.all(err <= bound)


# ------------------------------------------------------------------ planted mistakes
def _pins():
    return [test_f16_bit_patterns_from_definition, test_bf16_codes_match_torch, test_e4m3_spec_values,
            test_e4m3_rounding_matches_torch, lambda: test_row_scaling("fp8"), lambda: test_row_scaling("int8"),
            test_int8_ties_to_even, test_exchange_exact_when_representable]


def _some_pin_fails():
    for p in _pins():
        try:
            p()
        except AssertionError:
            return True
    return False


def _truncating_e4m3(v):
    v = np.asarray(v, np.float64)
    a = np.abs(v)
    _, E = np.frexp(a)
    eu = np.maximum(E - 1, -6)
    q = np.ldexp(1.0, eu - 3)
    k = np.floor(a / q).astype(np.int64)            # truncates instead of rounding
    up = k == 16
    eu, k = np.where(up, eu + 1, eu), np.where(up, 8, k)
    normal = k >= 8
    code = (np.where(normal, eu + 7, 0) << 3) | np.where(normal, k - 8, k)
    return (code | np.where(np.signbit(v), 0x80, 0)).astype(np.uint8)


def _bias8_e4m3(v):
    c = oc.e4m3_code.__wrapped__(v) if hasattr(oc.e4m3_code, "__wrapped__") else _ORIG["e4m3_code"](v)
    e = (c.astype(np.int64) >> 3) & 0xF
    return (((np.minimum(e + 1, 15)) << 3) | (c & 0x87)).astype(np.uint8)   # exponent off by one


def _scale_by_amax(x, codec):
    s, inv = _ORIG["row_scales"](x, codec)
    return s * np.float32(oc.QMAX[codec]), inv / np.float32(oc.QMAX[codec])   # amax instead of amax / Q


def _f16_truncate(x):
    a = np.asarray(x, np.float64).astype(np.float32)
    bits = a.view(np.uint32)
    # chop the mantissa (round toward zero) for normal numbers
    with np.errstate(over="ignore"):
        out = a.astype(np.float16).view(np.uint16).copy()
    down = np.abs(out.view(np.float16).astype(np.float64)) > np.abs(a.astype(np.float64))
    return np.where(down, out - 1, out).astype(np.uint16) if bits.size else out


_ORIG = {k: getattr(oc, k) for k in ("e4m3_code", "row_scales", "f16_code")}


@pytest.mark.parametrize("name,fn", [("e4m3_code", _truncating_e4m3), ("e4m3_code", _bias8_e4m3),
                                     ("row_scales", _scale_by_amax), ("f16_code", _f16_truncate)])
def test_planted_codec_mistakes_are_caught(monkeypatch, name, fn):
    assert not _some_pin_fails()
    monkeypatch.setattr(oc, name, fn)
    assert _some_pin_fails(), f"planted mistake in {name} ({fn.__name__}) went unnoticed"
