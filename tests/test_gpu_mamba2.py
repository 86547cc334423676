"""Mamba-2 (SSD) shard on the GPU against the float64 oracle on the same seeded inputs:
packed prefill with fresh and continuing sequences (including empty ones and ones shorter
than the convolution), the chunked state update across chunk and window boundaries, the
sum-of-squares exchange of the gated norm with split and with replicated B/C groups
(also through the decode out_proj that applies the norm to its operand as it loads it),
decode steps from the cache, and the Mamba-2 2.7B shard shape at full size (a sampled
sequence recomputed by the oracle).
"""
import numpy as np
import pytest

from mixer_cases import TOL, assert_close, host, poison_like
from oracle import mamba2 as o2
from paper_2602_21144_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# States are fp32 on both sides, but dt is rounded to bf16 by in_proj: a neighbouring
# rounding of one dt moves that token's Delta by up to one bf16 step (2^-8 relative).
STATE_TOL = 2.0 ** -8


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


class GpuLayer2:
    """All shards of a Mamba-2 layer on the GPU (weights sliced from full width on the GPU)."""

    def __init__(self, shape, full):
        from paper_2602_21144_amd import binding as B
        self.B, self.shape, self.P = B, shape, shape.shard_count
        full_dev = B.upload_weights2(full)
        dfull = B.make_desc2(shape, full=True)
        self.desc = [B.make_desc2(shape, r) for r in range(self.P)]
        self.w = []
        for r in range(self.P):
            out = B.empty_shard_weights2(shape)
            B.ssm2_shard_slice_weights(self.desc[r], full_dev, out)
            self.w.append(out)
        del full_dev, dfull
        self.ws_struct = [B.weights2_struct(w) for w in self.w]

    def new_pools(self, S, poison=True):
        sh = self.shape
        conv = [torch.zeros(S, sh.conv_dim_shard, sh.d_conv - 1, dtype=torch.bfloat16, device="cuda") for _ in range(self.P)]
        ssm = [torch.zeros(S, sh.heads_shard, sh.headdim, sh.d_state, dtype=torch.float32, device="cuda")
               for _ in range(self.P)]
        if poison:
            for t in conv + ssm:
                poison_like(t)
        return conv, ssm

    def prefill(self, x, meta, conv, ssm):
        B, sh = self.B, self.shape
        T = meta.T
        xd = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda().to(torch.bfloat16)
        self.ws = [B.workspace(B.m2_prefill_workspace_bytes(self.desc[r], T, meta.nseq)) for r in range(self.P)]
        parts = [torch.zeros(max(T, 1), sh.ngroups, dtype=torch.float32, device="cuda") for _ in range(self.P)]
        for r in range(self.P):
            B.ssm2_shard_prefill_stage1(self.desc[r], self.ws_struct[r], xd, meta, conv[r], ssm[r], parts[r], self.ws[r])
        for r in range(1, self.P):
            B.ssm_reduce_add_f32(parts[0], parts[r])
        ys = []
        for r in range(self.P):
            y = torch.empty(max(T, 1), sh.d_model, dtype=torch.bfloat16, device="cuda")
            B.ssm2_shard_prefill_stage2(self.desc[r], self.ws_struct[r], parts[0], T, y, self.ws[r])
            ys.append(y[:T])
        return ys

    def decode(self, x_t, slots_dev, conv, ssm):
        B, sh = self.B, self.shape
        Bd = x_t.shape[0]
        xd = torch.from_numpy(np.ascontiguousarray(x_t, np.float32)).cuda().to(torch.bfloat16)
        self.dws = [B.workspace(B.m2_decode_workspace_bytes(self.desc[r], Bd)) for r in range(self.P)]
        parts = [torch.zeros(Bd, sh.ngroups, dtype=torch.float32, device="cuda") for _ in range(self.P)]
        for r in range(self.P):
            B.ssm2_shard_decode_stage1(self.desc[r], self.ws_struct[r], xd, slots_dev, conv[r], ssm[r], parts[r],
                                       self.dws[r])
        for r in range(1, self.P):
            B.ssm_reduce_add_f32(parts[0], parts[r])
        ys = []
        for r in range(self.P):
            y = torch.empty(Bd, sh.d_model, dtype=torch.bfloat16, device="cuda")
            B.ssm2_shard_decode_stage2(self.desc[r], self.ws_struct[r], parts[0], Bd, y, self.dws[r])
            ys.append(y)
        return ys

    def status_ok(self, wss):
        return all(self.B.take_status(w) == 0 for w in wss)


def _f64(full):
    return {k: np.asarray(v, np.float64) for k, v in full.items() if not k.startswith("_")}


def _rand_pools(rng, sh, S):
    C, K = sh.conv_dim_shard, sh.d_conv
    cp = [synth.round_bf16_f32(rng.normal(size=(S, C, K - 1)).astype(np.float32)) for _ in range(sh.shard_count)]
    sp = [(rng.normal(size=(S, sh.heads_shard, sh.headdim, sh.d_state)) * 0.2).astype(np.float32)
          for _ in range(sh.shard_count)]
    return cp, sp


def _run_case(sh, full, lens, hi, seed, decode_steps=3):
    from paper_2602_21144_amd import binding as B
    rng = np.random.default_rng(seed)
    nseq = len(lens)
    S = nseq + 3
    slots = rng.permutation(S)[:nseq].astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    x = synth.make_tokens(rng, T, sh.d_model, "bf16")
    cp0, sp0 = _rand_pools(rng, sh, S)
    g = GpuLayer2(sh, full)
    conv, ssm = g.new_pools(S)
    for r in range(sh.shard_count):
        conv[r].copy_(torch.from_numpy(cp0[r]).cuda().to(torch.bfloat16))
        ssm[r].copy_(torch.from_numpy(sp0[r]).cuda())
    meta = B.SeqMeta(cu, slots, hi, S)
    ys = g.prefill(x, meta, conv, ssm)
    assert g.status_ok(g.ws)
    f64 = _f64(full)
    cps = [c.astype(np.float64) for c in cp0]
    sps = [s.astype(np.float64) for s in sp0]
    s1, yr = o2.tp_prefill(f64, sh, x.astype(np.float64), cu, slots, hi, cps, sps, "bf16")
    for r in range(sh.shard_count):
        assert_close(host(ys[r]), yr[r], TOL["bf16"], f"prefill y_partial shard {r}")
        assert_close(host(ssm[r]), s1[r]["ssm_pool"], STATE_TOL, f"prefill states shard {r}")
        assert_close(host(conv[r]), s1[r]["conv_pool"], TOL["bf16"], f"conv history shard {r}")
    dec = [i for i in range(nseq) if lens[i] > 0 or hi[i]]
    dslots = slots[dec]
    sl = torch.from_numpy(dslots).cuda()
    cps = [s["conv_pool"] for s in s1]
    sps = [s["ssm_pool"] for s in s1]
    for step in range(decode_steps):
        xt = synth.make_tokens(rng, len(dec), sh.d_model, "bf16")
        yd = g.decode(xt, sl, conv, ssm)
        assert g.status_ok(g.dws)
        d1, ydr = o2.tp_decode_step(f64, sh, xt.astype(np.float64), dslots, cps, sps, "bf16")
        cps = [d["conv_pool"] for d in d1]
        sps = [d["ssm_pool"] for d in d1]
        for r in range(sh.shard_count):
            assert_close(host(yd[r]), ydr[r], TOL["bf16"], f"decode step {step} shard {r}")
    for r in range(sh.shard_count):
        assert_close(host(ssm[r]), sps[r], STATE_TOL, f"states after decode, shard {r}")
    return g


@pytest.mark.parametrize("P,G", [(1, 1), (2, 1), (2, 2), (1, 4)])
@pytest.mark.parametrize("stress", [False, True])
def test_m2_prefill_then_decode(P, G, stress):
    sh = synth.Mamba2Shape(256, 16, 64, 128, G, 4, P, "bf16")
    full = synth.make_mamba2_layer(sh, 31 + G, stress=stress)
    lens = [70, 1, 0, 200, 65, 130, 3]
    hi = np.array([1, 0, 1, 0, 1, 1, 0], np.int32)
    _run_case(sh, full, lens, hi, seed=7 + P + G)


@pytest.mark.parametrize("K", [2, 3])
def test_m2_conv_widths(K):
    """Convolution widths 2 and 3 through prefill (continuing and fresh sequences) and the
    fused decode in_proj's conv window."""
    sh = synth.Mamba2Shape(128, 16, 64, 128, 2, K, 2, "bf16")
    full = synth.make_mamba2_layer(sh, 60 + K, stress=True)
    _run_case(sh, full, [40, 1, 0, 77], np.array([1, 0, 1, 1], np.int32), seed=60 + K)


# d_model 2048 gives out_proj 128 tiles of 16 columns, so decode batches of up to 16 take the
# streamed out_proj with the gated norm applied to its operand as loaded: 4-wave workgroups
# (K = 512 or 1024 per shard) and 8-wave ones (K = 2048), one norm group per row (G = 1) and
# several, split over the shards or replicated on each
@pytest.mark.parametrize("P,G,H", [(2, 1, 32), (2, 2, 16), (1, 4, 16), (1, 2, 32)])
def test_m2_fused_norm_out_proj(P, G, H):
    sh = synth.Mamba2Shape(2048, H, 64, 128, G, 4, P, "bf16")
    full = synth.make_mamba2_layer(sh, 80 + G + H)
    from paper_2602_21144_amd import binding as B
    B.ssm_timing_collect()
    B.ssm_timing_enable(True, "m2.decode.norm_out_proj")
    try:
        _run_case(sh, full, [20, 1, 0, 9, 33], np.array([1, 0, 1, 0, 1], np.int32), seed=80 + P + G, decode_steps=3)
        torch.cuda.synchronize()
    finally:
        B.ssm_timing_enable(False)
    # the decode steps took the fused launch (one per shard and step)
    assert B.ssm_timing_collect()["m2.decode.norm_out_proj"][0] == 3 * P


def test_m2_many_short_sequences():
    """60 sequences of 0..5 tokens, some continuing: chunks holding many sequence starts and
    ends, then decode steps."""
    sh = synth.Mamba2Shape(128, 16, 64, 128, 1, 4, 2, "bf16")
    full = synth.make_mamba2_layer(sh, 70, stress=True)
    rng = np.random.default_rng(70)
    lens = [int(v) for v in rng.integers(0, 6, 60)]
    hi = (rng.random(60) < 0.4).astype(np.int32)
    _run_case(sh, full, lens, hi, seed=71, decode_steps=2)


def test_m2_windows_of_several_chunks():
    """Long enough that each (window, head) workgroup walks several chunks, with a second
    sequence after it and a continuing start."""
    sh = synth.Mamba2Shape(128, 8, 64, 128, 1, 4, 1, "bf16")
    full = synth.make_mamba2_layer(sh, 5, stress=True)
    _run_case(sh, full, [9000, 333], np.array([1, 0], np.int32), seed=3, decode_steps=2)


# decode batches on each in_proj route: up to 16 sequences on the streamed kernel and up to
# 64 on the fragment kernel, both with the conv window in the in_proj epilogue; above 64
# in_proj, then the conv step as its own kernel
@pytest.mark.parametrize("Bd", [5, 16, 40, 64, 65, 129])
def test_m2_decode_batches(Bd):
    """Decode steps straight from random caches (no prefill) for a batch of sequences in
    scattered slots; outputs, states and the conv history against the oracle each step."""
    sh = synth.Mamba2Shape(256, 16, 64, 128, 2, 4, 2, "bf16")
    full = synth.make_mamba2_layer(sh, 40 + Bd)
    rng = np.random.default_rng(Bd)
    S = Bd + 7
    slots = rng.permutation(S)[:Bd].astype(np.int32)
    cp0, sp0 = _rand_pools(rng, sh, S)
    g = GpuLayer2(sh, full)
    conv, ssm = g.new_pools(S)
    for r in range(sh.shard_count):
        conv[r].copy_(torch.from_numpy(cp0[r]).cuda().to(torch.bfloat16))
        ssm[r].copy_(torch.from_numpy(sp0[r]).cuda())
    f64 = _f64(full)
    cps = [c.astype(np.float64) for c in cp0]
    sps = [s.astype(np.float64) for s in sp0]
    sl = torch.from_numpy(slots).cuda()
    for step in range(2):
        xt = synth.make_tokens(rng, Bd, sh.d_model, "bf16")
        yd = g.decode(xt, sl, conv, ssm)
        assert g.status_ok(g.dws)
        d1, ydr = o2.tp_decode_step(f64, sh, xt.astype(np.float64), slots, cps, sps, "bf16")
        cps = [d["conv_pool"] for d in d1]
        sps = [d["ssm_pool"] for d in d1]
        for r in range(sh.shard_count):
            assert_close(host(yd[r]), ydr[r], TOL["bf16"], f"decode step {step} shard {r}")
            assert_close(host(conv[r]), cps[r], TOL["bf16"], f"conv history step {step} shard {r}")
            assert_close(host(ssm[r]), sps[r], STATE_TOL, f"states step {step} shard {r}")


def test_m2_empty_batch_and_bad_slot():
    from paper_2602_21144_amd import binding as B
    sh = synth.Mamba2Shape(128, 8, 64, 128, 1, 4, 1, "bf16")
    full = synth.make_mamba2_layer(sh, 6)
    g = GpuLayer2(sh, full)
    conv, ssm = g.new_pools(4)
    # all sequences empty: fresh ones end with zero caches, continuing ones keep theirs
    meta = B.SeqMeta([0, 0, 0], [1, 2], [0, 1], 4)
    keep_c, keep_s = conv[0][2].clone(), ssm[0][2].clone()
    g.prefill(np.zeros((0, sh.d_model), np.float32), meta, conv, ssm)
    assert g.status_ok(g.ws)
    assert torch.all(conv[0][1] == 0) and torch.all(ssm[0][1] == 0)
    assert torch.equal(conv[0][2].view(torch.int16), keep_c.view(torch.int16))
    assert torch.equal(ssm[0][2].view(torch.int32), keep_s.view(torch.int32))
    # a slot outside the pool in decode is reported, not followed
    conv[0].zero_()
    ssm[0].zero_()
    xt = synth.make_tokens(np.random.default_rng(1), 2, sh.d_model, "bf16")
    g.decode(xt, torch.tensor([0, 9], dtype=torch.int32, device="cuda"), conv, ssm)
    assert B.take_status(g.dws[0]) & B.SSM_STATUS_BAD_SLOT


def test_m2_2p7b_shard_full_size():
    """Mamba-2 2.7B shard 1/2 (40 heads of 64, N 128, one replicated B/C group): 8 x 2048
    prefill and 16 decode steps; sequence 2 recomputed by the oracle through both shards."""
    from paper_2602_21144_amd import binding as B
    cfg = synth.MAMBA2_CONFIGS["mamba2_2.7b_tp2"]
    sh = cfg["shape"]
    full = synth.make_mamba2_layer(sh, cfg["seed"])
    rng = full["_rng"]
    Bsz, L, steps = cfg["batch"], cfg["prefill_len"], 16
    x = synth.make_tokens(rng, Bsz * L, sh.d_model, "bf16")
    xdec = [synth.make_tokens(rng, Bsz, sh.d_model, "bf16") for _ in range(steps)]
    slots = synth.make_slots(rng, Bsz)
    S = Bsz + 16
    g = GpuLayer2(sh, full)
    conv, ssm = g.new_pools(S)
    meta = B.SeqMeta(np.arange(0, Bsz * L + 1, L), slots, np.zeros(Bsz, np.int32), S)
    ys = g.prefill(x, meta, conv, ssm)
    assert g.status_ok(g.ws)
    i = 2
    y_pre = [host(ys[r][i * L:(i + 1) * L]) for r in range(2)]
    sl = torch.from_numpy(slots).cuda()
    y_dec = [[], []]
    for xt in xdec:
        yd = g.decode(xt, sl, conv, ssm)
        for r in range(2):
            y_dec[r].append(host(yd[r][i]))
    f64 = _f64(full)
    C, K, H = sh.conv_dim_shard, sh.d_conv, sh.heads_shard
    zc, zs = np.zeros((1, C, K - 1)), np.zeros((1, H, sh.headdim, sh.d_state))
    s1, yr = o2.tp_prefill(f64, sh, x[i * L:(i + 1) * L].astype(np.float64), [0, L], [0], [0], [zc, zc], [zs, zs], "bf16")
    cps = [s["conv_pool"] for s in s1]
    sps = [s["ssm_pool"] for s in s1]
    yd_ref = [[], []]
    for xt in xdec:
        d1, ydr = o2.tp_decode_step(f64, sh, xt[i:i + 1].astype(np.float64), [0], cps, sps, "bf16")
        cps = [d["conv_pool"] for d in d1]
        sps = [d["ssm_pool"] for d in d1]
        for r in range(2):
            yd_ref[r].append(ydr[r][0])
    for r in range(2):
        assert_close(y_pre[r], yr[r], TOL["bf16"], f"prefill y_partial of sequence {i}, shard {r}")
        assert_close(np.stack(y_dec[r]), np.stack(yd_ref[r]), TOL["bf16"], f"decode y_partial, shard {r}")
        assert_close(host(ssm[r][slots[i]]), sps[r][0], STATE_TOL, f"final state, shard {r}")
    spare = sorted(set(range(S)) - set(slots.tolist()))
    assert torch.all(ssm[0][spare].view(torch.int32) == 0x7FC0DEAD)
