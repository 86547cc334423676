"""Decode steps captured in a HIP graph (through torch's graph capture on a side stream) and
replayed several times, with eager work and synchronisations between the replays: every
replay must give exactly the outputs and caches of the same steps issued eagerly from the
same caches. Covers the fused kernels (up to 64 sequences), the tiled projections with
split-K partials (more than 64), float32, and the decode step without allocation."""
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
    "bf16_fused_40": (synth.LayerShape(320, 384, 16, 32, 4, 1, "bf16"), 40, "workspace"),
    "bf16_tiled_100": (synth.LayerShape(2560, 1280, 16, 160, 4, 1, "bf16"), 100, "workspace"),
    "f32_9": (synth.LayerShape(96, 256, 16, 32, 4, 1, "f32"), 9, "workspace"),
    "bf16_noalloc_40": (synth.LayerShape(320, 384, 16, 32, 4, 1, "bf16"), 40, "noalloc"),
    "bf16_noalloc_100": (synth.LayerShape(2560, 1280, 16, 160, 4, 1, "bf16"), 100, "noalloc"),
}


@pytest.mark.parametrize("case", list(CASES))
def test_captured_decode_steps_replay_like_eager(case):
    from paper_2602_21144_amd import binding as B
    shape, batch, entry = CASES[case]
    steps = 4
    full = synth.make_layer(shape, 41, stress=True)
    g = GpuLayer(shape, full)
    d, w = g.desc[0], g.ws_struct[0]
    E, N, K = shape.d_shard, shape.d_state, shape.d_conv
    rng = np.random.default_rng(5)
    S = batch + 6
    conv0 = g.to_dev(rng.normal(size=(S, E, K - 1)).astype(np.float32))
    ssm0 = torch.from_numpy((rng.normal(size=(S, E, N)) * 0.5).astype(np.float32)).cuda()
    slots = torch.from_numpy(rng.permutation(S)[:batch].astype(np.int32)).cuda()
    xs = [g.to_dev(synth.make_tokens(rng, batch, shape.d_model, shape.act)) for _ in range(steps)]
    conv, ssm = conv0.clone(), ssm0.clone()
    ys = [torch.empty(batch, shape.d_model, dtype=g.tdt, device="cuda") for _ in range(steps)]
    ws = B.workspace(B.decode_workspace_bytes(d, batch))
    s = torch.cuda.Stream()

    if entry == "workspace":
        calls = [B.bind("ssm_shard_decode_step", d, w, xs[k], slots, conv, ssm, ys[k], ws, stream=s)
                 for k in range(steps)]
    else:
        calls = [B.bind("ssm_shard_decode_step_noalloc", d, w, xs[k], slots, conv, ssm, ys[k], stream=s)
                 for k in range(steps)]

    def run():
        for c in calls:
            c()

    # eager reference from the initial caches
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        run()
    torch.cuda.synchronize()
    y_ref = [y.clone() for y in ys]
    conv_ref, ssm_ref = conv.clone(), ssm.clone()

    graph = torch.cuda.CUDAGraph()
    conv.copy_(conv0)
    ssm.copy_(ssm0)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=s):
        run()
    torch.cuda.synchronize()
    for rep in range(3):
        conv.copy_(conv0)
        ssm.copy_(ssm0)
        for y in ys:
            y.fill_(float("nan"))
        junk = torch.randn(1000, device="cuda") @ torch.randn(1000, device="cuda")   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in range(steps):
            assert torch.equal(ys[k], y_ref[k]), f"replay {rep}: y of step {k} differs from the eager run"
        assert torch.equal(conv, conv_ref) and torch.equal(ssm, ssm_ref), f"replay {rep}: caches differ"
        del junk
    assert B.take_status(ws) == 0
