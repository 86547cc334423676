"""Quantized exchange on the GPU against the codec oracle: payload bytes (codes and fp32
scales) equal the oracle's bit for bit on the same inputs, the decoded sum over ranks
matches the oracle's sum of decoded payloads, and a two-shard prefill whose x_proj
exchange goes through each codec stays within the codec's error of the exact layer.
"""
import numpy as np
import pytest

from mixer_cases import TOL, GpuLayer, assert_close, f64, host
from oracle import codec as oc
from oracle import mixer as om
from paper_2602_21144_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _rows(rng, rows, cols, src):
    """Rows of very different magnitudes, one all-zero row, one with a single spike."""
    mag = 10.0 ** rng.uniform(-6, 3, size=(rows, 1))   # f16 stays finite
    x = (rng.standard_normal((rows, cols)) * mag).astype(np.float32)
    if rows > 2:
        x[1] = 0.0
        x[2] = 0.0
        x[2, cols // 3] = -3.5
    if src == "bf16":
        x = synth.round_bf16_f32(x)
    return x


def _payload_parts(buf, codec, rows, cols):
    b = buf.cpu().numpy()
    if codec in ("f16", "bf16"):
        return b[:rows * cols * 2].view(np.uint16).reshape(rows, cols), None
    off = (rows * 4 + 255) // 256 * 256
    return b[off:off + rows * cols].reshape(rows, cols), b[:rows * 4].view(np.float32)


@pytest.mark.parametrize("codec", oc.CODECS)
@pytest.mark.parametrize("src", ["f32", "bf16"])
@pytest.mark.parametrize("rows,cols,pad", [(1, 8, 0), (37, 192, 8), (300, 2560, 0), (5, 5000, 16), (64, 1032, 0)])
def test_payload_bits_and_sum_match_oracle(codec, src, rows, cols, pad):
    from paper_2602_21144_amd import binding as B
    rng = np.random.default_rng(rows * 7 + cols)
    tdt = torch.float32 if src == "f32" else torch.bfloat16
    parts = [_rows(rng, rows, cols, src) for _ in range(3)]
    acc = torch.full((rows, cols + pad), float("nan"), dtype=torch.float32, device="cuda")[:, :cols]
    for r, x in enumerate(parts):
        dev = torch.zeros(rows, cols + pad, dtype=tdt, device="cuda")
        dev[:, :cols] = torch.from_numpy(x).to(tdt)
        pay = B.exchange_payload(codec, rows, cols)
        B.ssm_exchange_encode(codec, dev[:, :cols], pay)
        codes, scales = _payload_parts(pay, codec, rows, cols)
        ref = oc.encode(x.astype(np.float64), codec)
        assert np.array_equal(codes, ref["codes"]), f"rank {r}: codes differ"
        if scales is not None:
            assert np.array_equal(scales.view(np.uint32), ref["scales"].view(np.uint32)), f"rank {r}: scales differ"
        B.ssm_exchange_decode_accumulate(codec, pay, acc, accumulate=r > 0)
    torch.cuda.synchronize()
    want = oc.exchange([p.astype(np.float64) for p in parts], codec)
    got = host(acc)
    # the GPU adds three fp32 values in rank order: within two fp32 roundings of the exact sum
    terms = sum(np.abs(oc.decode(oc.encode(p.astype(np.float64), codec), codec)) for p in parts)
    assert np.all(np.abs(got - want) <= 2.0 ** -23 * terms + 1e-45)


def test_accumulate_flag_overwrites_or_adds():
    from paper_2602_21144_amd import binding as B
    x = torch.arange(16 * 8, dtype=torch.float32, device="cuda").reshape(16, 8)
    pay = B.exchange_payload("f16", 16, 8)
    B.ssm_exchange_encode("f16", x, pay)
    acc = torch.full((16, 8), 7.0, device="cuda")
    B.ssm_exchange_decode_accumulate("f16", pay, acc, accumulate=True)
    assert torch.equal(acc, x + 7.0)
    B.ssm_exchange_decode_accumulate("f16", pay, acc, accumulate=False)
    assert torch.equal(acc, x)


@pytest.mark.parametrize("codec", oc.CODECS)
def test_quantized_x_proj_exchange_in_two_shard_prefill(codec):
    """Stage 1 on both shards, their x_proj partials exchanged through the codec, stage 2
    on shard 0: y_partial equals the oracle's with the same codec applied to the oracle's
    partials, and differs from the exact exchange by no more than the codec allows."""
    from paper_2602_21144_amd import binding as B
    shape = synth.LayerShape(64, 256, 16, 16, 4, 2, "bf16")
    full = synth.make_layer(shape, 21, stress=True)
    rng = np.random.default_rng(5)
    lens = [70, 33]
    cu = np.array([0, 70, 103], np.int32)
    slots = np.array([1, 0], np.int32)
    x = synth.make_tokens(rng, 103, shape.d_model, "bf16")
    g = GpuLayer(shape, full)
    meta = B.SeqMeta(cu, slots, [0, 0], 2)
    conv, ssm = g.new_pools(2)
    T, W = 103, shape.w_dbl
    xd = g.to_dev(x)
    parts = {}
    ws = {}
    for r in range(2):
        ws[r] = B.workspace(B.prefill_workspace_bytes(g.desc[r], T, 2))
        parts[r] = torch.empty(T, W, dtype=torch.float32, device="cuda")
        B.ssm_shard_prefill_stage1(g.desc[r], g.ws_struct[r], xd, meta, conv[r], parts[r], ws[r])
    red = torch.empty(T, W, dtype=torch.float32, device="cuda")
    for r in range(2):
        pay = B.exchange_payload(codec, T, W)
        B.ssm_exchange_encode(codec, parts[r], pay)
        B.ssm_exchange_decode_accumulate(codec, pay, red, accumulate=r > 0)
    y = torch.empty(T, shape.d_model, dtype=torch.bfloat16, device="cuda")
    B.ssm_shard_prefill_stage2(g.desc[0], g.ws_struct[0], red, meta, ssm[0], y, ws[0])
    assert B.take_status(ws[0]) == 0

    w64 = f64(full)
    shards = [om.shard_weights(w64, r, 2) for r in range(2)]
    zc, zs = np.zeros((2, 128, 3)), np.zeros((2, 128, 16))
    s1 = [om.prefill_stage1(w, x.astype(np.float64), cu, slots, [0, 0], zc, "bf16") for w in shards]
    q_sum = oc.exchange([s["x_dbl"] for s in s1], codec)
    ref = om.prefill_stage2(shards[0], s1[0], q_sum, cu, slots, [0, 0], zs, "bf16")
    assert_close(host(y), ref["y"], TOL["bf16"], f"y_partial with a {codec} exchange")
    # the exchange itself: GPU sum of decoded GPU partials vs the exact sum of the oracle partials
    # each rank's rounding error, per format: half an ulp of the element (f16, bf16), the
    # larger of 2**-4 of the element and half a subnormal step of the row scale (fp8), half
    # a step of the row scale (int8); plus the fp32-vs-fp64 difference of the partials
    exact = oc.exact_sum([s["x_dbl"] for s in s1])
    bound = np.zeros_like(exact)
    for s_ in s1:
        p = np.abs(s_["x_dbl"])
        amax = p.max(axis=1, keepdims=True)
        if codec == "f16":
            bound += p * 2.0 ** -11 + 2.0 ** -25
        elif codec == "bf16":
            bound += p * 2.0 ** -8
        elif codec == "fp8":
            bound += np.maximum(p * 2.0 ** -4, amax / 448 * 2.0 ** -10)
        else:
            bound += amax / 127 / 2
        bound += p * 1e-5
    err = np.abs(host(red) - exact)
    assert np.all(err <= bound * (1 + 1e-3) + 1e-7), f"{codec}: exchange error {float((err / bound).max()):.3e} of its bound"
