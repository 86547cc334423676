"""The decode step that allocates nothing (ssm_shard_decode_step_noalloc: its workspace is
a static device array of the library) against the decode step with a caller workspace
(ssm_shard_decode_step), through the C ABI: two calls in a row, the second with fewer
sequences, from identical caches; outputs and both caches must be bit-identical. Also the
host-side rejection of a batch whose workspace exceeds the static array."""
import numpy as np
import pytest

from mixer_cases import GpuLayer
from paper_2602_21144_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


CASES = {
    # Mamba-2.8B quarter shard (1280 channels): 200 sequences take the tiled projections
    # with split-K partials in the scratch, then 40 the fused kernels
    "bf16_quarter_shard": (synth.LayerShape(2560, 5120, 16, 160, 4, 4, "bf16"), [200, 40], True),
    # fp32: 9 rows on fp32 MFMA tiles, then 3 on the one-row-per-wave kernel
    "f32_small": (synth.LayerShape(96, 256, 16, 32, 4, 2, "f32"), [9, 3], False),
}


@pytest.mark.parametrize("case", list(CASES))
def test_noalloc_decode_matches_workspace_decode(case):
    from paper_2602_21144_amd import binding as B
    shape, batches, stress = CASES[case]
    full = synth.make_layer(shape, 31, stress=stress)
    g = GpuLayer(shape, full, shards=[0])
    d, w = g.desc[0], g.ws_struct[0]
    E, N, K = shape.d_shard, shape.d_state, shape.d_conv
    rng = np.random.default_rng(7)
    S = max(batches) + 8
    conv_a = g.to_dev(rng.normal(size=(S, E, K - 1)).astype(np.float32))
    ssm_a = torch.from_numpy((rng.normal(size=(S, E, N)) * 0.5).astype(np.float32)).cuda()
    conv_b, ssm_b = conv_a.clone(), ssm_a.clone()
    ws = B.workspace(B.decode_workspace_bytes(d, max(batches)))
    for step, bsz in enumerate(batches):
        slots = torch.from_numpy(rng.permutation(S)[:bsz].astype(np.int32)).cuda()
        x = g.to_dev(synth.make_tokens(rng, bsz, shape.d_model, shape.act))
        y_ref = torch.empty(bsz, shape.d_model, dtype=g.tdt, device="cuda")
        y_new = torch.full_like(y_ref, float("nan"))
        B.ssm_shard_decode_step(d, w, x, slots, conv_a, ssm_a, y_ref, ws)
        B.ssm_shard_decode_step_noalloc(d, w, x, slots, conv_b, ssm_b, y_new)
        torch.cuda.synchronize()
        assert torch.equal(y_new, y_ref), f"call {step} ({bsz} sequences): y_partial differs"
        assert torch.equal(ssm_b, ssm_a), f"call {step}: ssm pool differs"
        assert torch.equal(conv_b, conv_a), f"call {step}: conv pool differs"
    assert B.take_status(ws) == 0


def test_noalloc_decode_rejects_batches_beyond_the_scratch():
    """A batch whose workspace would not fit the static array is refused on the host with
    SSM_E_WORKSPACE before anything is enqueued (pools stay as they were)."""
    from paper_2602_21144_amd import binding as B
    shape = synth.LayerShape(4096, 8192, 16, 256, 4, 1, "bf16")
    d = B.make_desc(shape, 0)
    bsz = 2048
    assert B.decode_workspace_bytes(d, bsz) > B.SSM_NOALLOC_SCRATCH_BYTES
    dev = "cuda"
    w = B.empty_shard_weights(shape, dev)
    conv = torch.zeros(bsz, shape.d_shard, 3, dtype=torch.bfloat16, device=dev)
    ssm = torch.zeros(bsz, shape.d_shard, 16, dtype=torch.float32, device=dev)
    x = torch.zeros(bsz, shape.d_model, dtype=torch.bfloat16, device=dev)
    y = torch.zeros(bsz, shape.d_model, dtype=torch.bfloat16, device=dev)
    slots = torch.arange(bsz, dtype=torch.int32, device=dev)
    with pytest.raises(B.SsmError) as e:
        B.ssm_shard_decode_step_noalloc(d, w, x, slots, conv, ssm, y)
    assert e.value.code == B.SSM_E_WORKSPACE
    torch.cuda.synchronize()
    assert not torch.any(ssm != 0) and not torch.any(y != 0)
