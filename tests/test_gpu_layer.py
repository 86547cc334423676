"""The layer around the mixer on the GPU against the layer oracle (same seeded inputs):
the residual add + RMSNorm kernel, Falcon-Mamba's delta/B/C norms, stacks of layers split
over ranks (composed from the per-layer calls with the exchanges summed on the one GPU)
and at full width through the stack calls, decoding with and without the SSM cache, and a
Falcon-Mamba-7B-shaped layer with its norms.
"""
import numpy as np
import pytest

from mixer_cases import TOL, assert_close, f64, host
from oracle import layer as ol
from oracle import mixer as om
from paper_2602_21144_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _dev(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to("cuda", dt)


# ------------------------------------------------------------------ kernels
@pytest.mark.parametrize("d", [8, 768, 2568, 4096, 8192])
@pytest.mark.parametrize("nparts", [0, 1, 3])
@pytest.mark.parametrize("dts", [("bf16", "bf16", "bf16"), ("f32", "f32", "f32"), ("f32", "bf16", "bf16"),
                                 ("bf16", "f32", "f32")])
def test_residual_rmsnorm(d, nparts, dts):
    from paper_2602_21144_amd import binding as B
    bdt, pdt, odt = (torch.bfloat16 if t == "bf16" else torch.float32 for t in dts)
    rng = np.random.default_rng(d + 10 * nparts)
    T = 37
    scale = 10.0 ** rng.uniform(-3, 3, size=(T, 1))
    base = rng.normal(size=(T, d)) * scale
    parts = [rng.normal(size=(T, d)) * scale for _ in range(nparts)]
    if dts[0] == "bf16":
        base = synth.round_bf16_f32(base.astype(np.float32))
    if dts[1] == "bf16":
        parts = [synth.round_bf16_f32(p.astype(np.float32)) for p in parts]
    w = (1 + rng.uniform(-0.5, 0.5, size=d)).astype(np.float32)
    resid = torch.empty(T, d, dtype=torch.float32, device="cuda")
    normed = torch.empty(T, d, dtype=odt, device="cuda")
    B.ssm_residual_rmsnorm(_dev(base, bdt), [_dev(p, pdt) for p in parts], resid, _dev(w, torch.float32), 1e-5, normed)
    r_ref, n_ref = ol.residual_norm(np.asarray(base, np.float64), [np.asarray(p, np.float64) for p in parts], w,
                                    1e-5, "f64")
    got_r, got_n = host(resid), host(normed)
    # the residual: a float32 sum of the parts and the base, within a few float32 roundings
    terms = np.abs(base) + sum(np.abs(p) for p in parts)
    assert np.all(np.abs(got_r - r_ref) <= (nparts + 1) * 2.0 ** -23 * terms + 1e-30)
    # normed: float32 arithmetic, then at most one rounding to the output type on each side
    bound = (2.0 ** -7 if dts[2] == "bf16" else 1e-5) * np.abs(n_ref) + 1e-6 * np.max(np.abs(n_ref))
    assert np.all(np.abs(got_n - n_ref) <= bound)


def test_residual_rmsnorm_in_place():
    from paper_2602_21144_amd import binding as B
    rng = np.random.default_rng(3)
    T, d = 19, 2560
    r0 = rng.normal(size=(T, d)).astype(np.float32)
    y = synth.round_bf16_f32(rng.normal(size=(T, d)).astype(np.float32))
    w = np.ones(d, np.float32)
    resid = _dev(r0, torch.float32)
    normed = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    B.ssm_residual_rmsnorm(resid, [_dev(y, torch.bfloat16)], resid, _dev(w, torch.float32), 1e-5, normed)
    r_ref, n_ref = ol.residual_norm(r0.astype(np.float64), [y.astype(np.float64)], w, 1e-5, "bf16")
    assert_close(host(resid), r_ref, 1e-6, "residual in place")
    assert_close(host(normed), n_ref, 2.0 ** -7, "normed")


@pytest.mark.parametrize("R,N,pad", [(48, 16, 0), (160, 16, 5), (256, 16, 0), (3, 4, 1)])
def test_bcdt_rmsnorm(R, N, pad):
    from paper_2602_21144_amd import binding as B
    rng = np.random.default_rng(R)
    T, W = 301, R + 2 * N
    x = rng.normal(size=(T, W + pad)) * (10.0 ** rng.uniform(-4, 4, size=(T, 1)))
    x[5, :R] = 0.0       # an all-zero delta range: stays zero
    xd = _dev(x, torch.float32)
    B.ssm_bcdt_rmsnorm(xd, R, N, 1e-6)
    ref = ol.bcdt_rms(x[:, :W], R, N, 1e-6)
    got = host(xd)
    assert np.all(np.abs(got[:, :W] - ref) <= 2e-6 * np.abs(ref) + 1e-30)
    assert np.array_equal(got[:, W:], x[:, W:].astype(np.float32).astype(np.float64))


# ------------------------------------------------------------------ stacks
class GpuStackTP:
    """A stack whose layers are split over P ranks, composed from the per-layer calls on the
    one GPU: the exchanges are the library's reduce (x_proj) and the norm kernel's sum of
    the ranks' out_proj partials."""

    def __init__(self, shape, st, bcdt):
        from paper_2602_21144_amd import binding as B
        self.B, self.shape, self.bcdt = B, shape, bcdt
        self.P = shape.shard_count
        self.tdt = B.torch_act(shape.act)
        self.desc = [B.make_desc(shape, r) for r in range(self.P)]
        self.w = []
        for full in st["layers"]:
            fd = B.upload_weights(full, shape.act)
            per = []
            for r in range(self.P):
                o = B.empty_shard_weights(shape)
                B.ssm_shard_slice_weights(self.desc[r], fd, o)
                per.append((o, B.weights_struct(o)))
            self.w.append(per)
        self.norm_w = [_dev(w, torch.float32) for w in st["norm_w"]]
        self.final_w = _dev(st["final_w"], torch.float32)

    def pools(self, S):
        sh = self.shape
        conv = [[torch.zeros(S, sh.d_shard, sh.d_conv - 1, dtype=self.tdt, device="cuda") for _ in range(self.P)]
                for _ in self.w]
        ssm = [[torch.zeros(S, sh.d_shard, sh.d_state, dtype=torch.float32, device="cuda") for _ in range(self.P)]
               for _ in self.w]
        return conv, ssm

    def _run(self, x, rows, stage1, stage2):
        B, sh = self.B, self.shape
        resid = torch.empty(rows, sh.d_model, dtype=torch.float32, device="cuda")
        h = torch.empty(rows, sh.d_model, dtype=self.tdt, device="cuda")
        B.ssm_residual_rmsnorm(x, [], resid, self.norm_w[0], ol.RMS_EPS, h)
        for l in range(len(self.w)):
            parts = [torch.empty(rows, sh.w_dbl, dtype=torch.float32, device="cuda") for _ in range(self.P)]
            for r in range(self.P):
                stage1(l, r, h, parts[r])
            for r in range(1, self.P):
                B.ssm_reduce_add_f32(parts[0], parts[r])
            if self.bcdt:
                B.ssm_bcdt_rmsnorm(parts[0], sh.dt_rank, sh.d_state, ol.BCDT_EPS)
            ys = [torch.empty(rows, sh.d_model, dtype=self.tdt, device="cuda") for _ in range(self.P)]
            for r in range(self.P):
                stage2(l, r, parts[0], ys[r])
            last = l + 1 == len(self.w)
            out = torch.empty_like(h) if last else h
            B.ssm_residual_rmsnorm(resid, ys, resid, self.final_w if last else self.norm_w[l + 1], ol.RMS_EPS, out)
            h = out
        return h

    def prefill(self, x, meta, conv, ssm):
        B = self.B
        ws = [B.workspace(B.prefill_workspace_bytes(self.desc[r], meta.T, meta.nseq)) for r in range(self.P)]
        return self._run(
            x, meta.T,
            lambda l, r, h, part: B.ssm_shard_prefill_stage1(self.desc[r], self.w[l][r][1], h, meta, conv[l][r], part,
                                                             ws[r]),
            lambda l, r, red, y: B.ssm_shard_prefill_stage2(self.desc[r], self.w[l][r][1], red, meta, ssm[l][r], y,
                                                            ws[r]))

    def decode(self, x_t, slots, conv, ssm):
        B = self.B
        Bd = x_t.shape[0]
        ws = [B.workspace(B.decode_workspace_bytes(self.desc[r], Bd)) for r in range(self.P)]
        return self._run(
            x_t, Bd,
            lambda l, r, h, part: B.ssm_shard_decode_stage1(self.desc[r], self.w[l][r][1], h, slots, conv[l][r], part,
                                                            ws[r]),
            lambda l, r, red, y: B.ssm_shard_decode_stage2(self.desc[r], self.w[l][r][1], red, slots, ssm[l][r], y,
                                                           ws[r]))


def _oracle_stack(shape, st):
    full = [f64(w) for w in st["layers"]]
    return [[om.shard_weights(w, r, shape.shard_count) for r in range(shape.shard_count)] for w in full]


def _oracle_pools(shape, n_layers, S):
    P = shape.shard_count
    return ([[np.zeros((S, shape.d_shard, shape.d_conv - 1)) for _ in range(P)] for _ in range(n_layers)],
            [[np.zeros((S, shape.d_shard, shape.d_state)) for _ in range(P)] for _ in range(n_layers)])


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("P,bcdt", [(2, False), (2, True), (4, True)])
def test_split_stack_prefill_and_decode(act, P, bcdt):
    from paper_2602_21144_amd import binding as B
    shape = synth.LayerShape(64, 256, 16, 16, 4, P, act)
    st = synth.make_stack(shape, 3, 30 + P, stress=True)
    g = GpuStackTP(shape, st, bcdt)
    rng = np.random.default_rng(P)
    lens = [70, 1, 33]
    T = sum(lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    slots = np.array([2, 0, 3], np.int32)
    x = synth.make_tokens(rng, T, shape.d_model, act)
    S = 5
    meta = B.SeqMeta(cu, slots, [0, 0, 0], S)
    conv, ssm = g.pools(S)
    out = g.prefill(_dev(x, g.tdt), meta, conv, ssm)
    layers = _oracle_stack(shape, st)
    oc, osp = _oracle_pools(shape, 3, S)
    eps = ol.BCDT_EPS if bcdt else None
    ref = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x.astype(np.float64), cu, slots, [0, 0, 0], oc, osp,
                           act, bcdt_eps=eps)
    assert_close(host(out), ref["out"], TOL[act], "stack prefill output")
    cp, sp = ref["conv_pools"], ref["ssm_pools"]
    sl = torch.from_numpy(slots).cuda()
    for step in range(3):
        xt = synth.make_tokens(rng, 3, shape.d_model, act)
        o = g.decode(_dev(xt, g.tdt), sl, conv, ssm)
        d = ol.stack_decode_step(layers, st["norm_w"], st["final_w"], xt.astype(np.float64), slots, cp, sp, act,
                                 bcdt_eps=eps)
        cp, sp = d["conv_pools"], d["ssm_pools"]
        assert_close(host(o), d["out"], TOL[act], f"stack decode step {step}")
    # layer 0's input is the same on both sides, so its states are held to one bf16 step of
    # dt (2^-8); deeper layers take the previous layers' bf16 outputs, which differ at the
    # output tolerance, and so do their states
    for l in range(3):
        for r in range(P):
            tol = (2.0 ** -8 if l == 0 else TOL["bf16"]) if act == "bf16" else TOL["f32"]
            assert_close(host(ssm[l][r])[slots], sp[l][r][slots], tol, f"layer {l} rank {r} states")


class GpuStack:
    """A full-width stack through ssm_stack_prefill / ssm_stack_decode_step."""

    def __init__(self, shape, st, bcdt, S):
        from paper_2602_21144_amd import binding as B
        self.B, self.shape = B, shape
        self.tdt = B.torch_act(shape.act)
        self.sd = B.make_stack_desc(shape, len(st["layers"]), ol.RMS_EPS, ol.BCDT_EPS if bcdt else 0.0)
        self.dev_w = [B.upload_weights(w, shape.act) for w in st["layers"]]
        self.norm_w = [_dev(w, torch.float32) for w in st["norm_w"]]
        self.final_w = _dev(st["final_w"], torch.float32)
        self.sw = B.StackWeights(self.dev_w, self.norm_w, self.final_w)
        self.S = S
        self.new_pools()

    def new_pools(self):
        sh = self.shape
        self.conv = [torch.zeros(self.S, sh.d_inner, sh.d_conv - 1, dtype=self.tdt, device="cuda")
                     for _ in self.dev_w]
        self.ssm = [torch.zeros(self.S, sh.d_inner, sh.d_state, dtype=torch.float32, device="cuda") for _ in self.dev_w]
        self.pools = self.B.StackPools(self.conv, self.ssm)

    def prefill(self, x, meta):
        B = self.B
        ws = B.workspace(B.stack_prefill_workspace_bytes(self.sd, meta.T, meta.nseq))
        out = torch.empty(max(meta.T, 1), self.shape.d_model, dtype=self.tdt, device="cuda")
        B.ssm_stack_prefill(self.sd, self.sw, x, meta, self.pools, out, ws)
        assert B.take_status(ws) == 0
        return out[:meta.T]

    def decode(self, x_t, slots):
        B = self.B
        ws = B.workspace(B.stack_decode_workspace_bytes(self.sd, x_t.shape[0]))
        out = torch.empty(x_t.shape[0], self.shape.d_model, dtype=self.tdt, device="cuda")
        B.ssm_stack_decode_step(self.sd, self.sw, x_t, slots, self.pools, out, ws)
        assert B.take_status(ws) == 0
        return out


# K = 1: no conv history, the stack's conv pools are empty (null pointers)
@pytest.mark.parametrize("act,bcdt,K", [("f32", False, 4), ("bf16", False, 4), ("bf16", True, 4), ("bf16", False, 1)])
def test_full_width_stack_calls(act, bcdt, K):
    from paper_2602_21144_amd import binding as B
    shape = synth.LayerShape(128, 256, 16, 16, K, 1, act)
    st = synth.make_stack(shape, 4, 40, stress=True)
    S = 4
    g = GpuStack(shape, st, bcdt, S)
    rng = np.random.default_rng(41)
    lens = [90, 5]
    cu = np.array([0, 90, 95], np.int32)
    slots = np.array([3, 1], np.int32)
    x = synth.make_tokens(rng, 95, shape.d_model, act)
    out = g.prefill(_dev(x, g.tdt), B.SeqMeta(cu, slots, [0, 0], S))
    layers = _oracle_stack(shape, st)
    oc, osp = _oracle_pools(shape, 4, S)
    eps = ol.BCDT_EPS if bcdt else None
    ref = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x.astype(np.float64), cu, slots, [0, 0], oc, osp, act,
                           bcdt_eps=eps)
    assert_close(host(out), ref["out"], TOL[act], "stack prefill")
    cp, sp = ref["conv_pools"], ref["ssm_pools"]
    sl = torch.from_numpy(slots).cuda()
    for step in range(4):
        xt = synth.make_tokens(rng, 2, shape.d_model, act)
        o = g.decode(_dev(xt, g.tdt), sl)
        d = ol.stack_decode_step(layers, st["norm_w"], st["final_w"], xt.astype(np.float64), slots, cp, sp, act,
                                 bcdt_eps=eps)
        cp, sp = d["conv_pools"], d["ssm_pools"]
        assert_close(host(o), d["out"], TOL[act], f"stack decode {step}")
    # a second prefill that continues both sequences from their caches
    x2 = synth.make_tokens(rng, 7, shape.d_model, act)
    cu2 = np.array([0, 3, 7], np.int32)
    out2 = g.prefill(_dev(x2, g.tdt), B.SeqMeta(cu2, slots, [1, 1], S))
    ref2 = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x2.astype(np.float64), cu2, slots, [1, 1], cp, sp,
                            act, bcdt_eps=eps)
    assert_close(host(out2), ref2["out"], TOL[act], "continued prefill")


def test_decoding_with_and_without_the_cache():
    """The ablation's two ways of generating: prefill + decode steps from the cache, or a
    prefill of the whole prefix for every token. Both match the oracle and each other."""
    from paper_2602_21144_amd import binding as B
    shape = synth.LayerShape(128, 256, 16, 16, 4, 1, "bf16")
    st = synth.make_stack(shape, 3, 50, stress=True)
    g = GpuStack(shape, st, False, 2)
    rng = np.random.default_rng(51)
    L, k = 40, 6
    seq = synth.make_tokens(rng, L + k, shape.d_model, "bf16")
    g.prefill(_dev(seq[:L], g.tdt), B.SeqMeta([0, L], [0], [0], 2))
    sl = torch.zeros(1, dtype=torch.int32, device="cuda")
    cached = [host(g.decode(_dev(seq[L + j:L + j + 1], g.tdt), sl))[0] for j in range(k)]
    nocache = []
    for j in range(k):
        g.new_pools()
        n = L + j + 1
        nocache.append(host(g.prefill(_dev(seq[:n], g.tdt), B.SeqMeta([0, n], [0], [0], 2)))[-1])
    layers = _oracle_stack(shape, st)
    ref = []
    for j in range(k):
        oc, osp = _oracle_pools(shape, 3, 1)
        ref.append(ol.stack_no_cache_step(layers, st["norm_w"], st["final_w"], [seq[:L + j + 1].astype(np.float64)],
                                          oc, osp, "bf16")[0])
    assert_close(np.stack(cached), np.stack(ref), TOL["bf16"], "decode from the cache")
    assert_close(np.stack(nocache), np.stack(ref), TOL["bf16"], "re-prefill of the prefix")
    assert_close(np.stack(cached), np.stack(nocache), TOL["bf16"], "cache vs no cache")


def test_falcon_mamba_7b_shaped_layer_with_its_norms():
    """Falcon-Mamba-7B's mixer shape (d_model 4096, 8192 channels over 4 ranks, dt rank 256)
    with the delta/B/C norms: a packed prefill and two decode steps on all four ranks;
    rank 0's output and states against the oracle."""
    from paper_2602_21144_amd import binding as B
    shape = synth.LayerShape(4096, 8192, 16, 256, 4, 4, "bf16")
    st = synth.make_stack(shape, 1, 60, stress=True)
    g = GpuStackTP(shape, st, True)
    rng = np.random.default_rng(61)
    lens = [150, 70]
    cu = np.array([0, 150, 220], np.int32)
    slots = np.array([1, 0], np.int32)
    x = synth.make_tokens(rng, 220, shape.d_model, "bf16")
    meta = B.SeqMeta(cu, slots, [0, 0], 2)
    conv, ssm = g.pools(2)
    out = g.prefill(_dev(x, torch.bfloat16), meta, conv, ssm)
    layers = _oracle_stack(shape, st)
    oc, osp = _oracle_pools(shape, 1, 2)
    ref = ol.stack_prefill(layers, st["norm_w"], st["final_w"], x.astype(np.float64), cu, slots, [0, 0], oc, osp,
                           "bf16", bcdt_eps=ol.BCDT_EPS)
    assert_close(host(out), ref["out"], TOL["bf16"], "Falcon-shaped prefill")
    xt = synth.make_tokens(rng, 2, shape.d_model, "bf16")
    o = g.decode(_dev(xt, torch.bfloat16), torch.from_numpy(slots).cuda(), conv, ssm)
    d = ol.stack_decode_step(layers, st["norm_w"], st["final_w"], xt.astype(np.float64), slots, ref["conv_pools"],
                             ref["ssm_pools"], "bf16", bcdt_eps=ol.BCDT_EPS)
    assert_close(host(o), d["out"], TOL["bf16"], "Falcon-shaped decode")
    assert_close(host(ssm[0][0]), d["ssm_pools"][0][0], 2.0 ** -8, "rank 0 states")
