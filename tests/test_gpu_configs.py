"""Parity at the five workload shapes, at full size, in the launch configuration the
benchmark uses: every shard of the channel split runs on the GPU (stage 1 on all, the
x_proj partials summed, stage 2 on shard 0). The oracle recomputes sampled whole
sequences (the 16k-token prefill in full). Each workload runs with the recipe's init and
with the stress init (matrices at 1/sqrt(fan-in), D = 0), under which the state path
carries y; the hybrid schedule also runs at float32, the precision of the headline
benchmark.

Inputs follow the seeded recipe: full-width weights, then the prompts, then the decode
inputs, from numpy PCG64(seed); bf16 values are RNE-rounded fp32 draws. The two inits
draw the same number of weight values, so the token streams that follow are the same.
"""
import dataclasses
import functools

import numpy as np
import pytest

from mixer_cases import TOL, GpuLayer, assert_close, f64, host, oracle_tp_sequence
from paper_2602_21144_amd import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

INITS = ["baseline", "stress"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _status_ok(g):
    for r in range(g.P):
        assert g.B.take_status(g.last_ws[r]) == 0


@functools.lru_cache(maxsize=1)
def _tokens_f32(cfg_name):
    """The workload's token draws at float32 (shared by both inits and both precisions)."""
    cfg = synth.CONFIGS[cfg_name]
    sh = dataclasses.replace(cfg["shape"], act="f32")
    rng = synth.make_layer(sh, cfg["seed"])["_rng"]
    if "len_range" in cfg:
        lo, hi = cfg["len_range"]
        lengths = [int(v) for v in rng.integers(lo, hi, endpoint=True, size=cfg["batch"])]
        x = synth.make_tokens(rng, int(sum(lengths)), sh.d_model, "f32")
        xdec = synth.make_tokens(rng, cfg["batch"] * cfg["decode_steps"], sh.d_model, "f32")
        xdec = xdec.reshape(cfg["batch"], cfg["decode_steps"], sh.d_model)
        slots = synth.make_slots(rng, cfg["batch"])
        return lengths, x, xdec, slots
    Bsz, L, steps = cfg["batch"], cfg["prefill_len"], cfg["decode_steps"]
    x = synth.make_tokens(rng, Bsz * L, sh.d_model, "f32")
    xdec = [synth.make_tokens(rng, Bsz, sh.d_model, "f32") for _ in range(steps)]
    slots = synth.make_slots(rng, Bsz)
    return None, x, xdec, slots


def _workload(cfg_name, init, act=None):
    cfg = synth.CONFIGS[cfg_name]
    sh = cfg["shape"] if act is None else dataclasses.replace(cfg["shape"], act=act)
    full = synth.make_layer(sh, cfg["seed"], stress=(init == "stress"))
    full.pop("_rng")
    lengths, x, xdec, slots = _tokens_f32(cfg_name)
    store = synth.round_bf16_f32 if sh.act == "bf16" else (lambda a: a)
    if lengths is None:
        return sh, full, store(x), [store(xt) for xt in xdec], slots
    return sh, full, lengths, store(x), store(xdec), slots


@pytest.mark.parametrize("init", INITS)
def test_mamba130m_f32_full_width(init):
    """Mamba-130m shape, fp32, full width: prefill 256 then 16 decode steps, all outputs."""
    sh, full, x, xdec, slots = _workload("mamba130m_f32", init)
    from paper_2602_21144_amd import binding as B
    g = GpuLayer(sh, full)
    S = len(slots) + 16
    conv, ssm = g.new_pools(S)
    meta = B.SeqMeta([0, 256], slots, [0], S)
    y = host(g.prefill(x, meta, conv, ssm)[0])
    _status_ok(g)
    sl = torch.from_numpy(slots).cuda()
    yd = np.stack([host(g.decode(xt, sl, conv, ssm)[0])[0] for xt in xdec])
    ref = oracle_tp_sequence(f64(full), sh, x, np.concatenate(xdec))[0]
    assert_close(y, ref["y"], TOL["f32"], "prefill y")
    assert_close(yd, ref["dec_y"], TOL["f32"], "decode y")
    assert_close(host(ssm[0][slots[0]]), ref["ssm"], TOL["f32"], "ssm state")
    assert_close(host(conv[0][slots[0]]), ref["conv"], TOL["f32"], "conv state")


@pytest.mark.parametrize("init", INITS)
def test_mamba28b_tp2_batch8(init):
    """Mamba-2.8B shard 1/2, bf16: 8 x 2048 prefill then 128 decode steps; sequence 5 sampled."""
    sh, full, x, xdec, slots = _workload("mamba2.8b_tp2", init)
    from paper_2602_21144_amd import binding as B
    Bsz, L = 8, 2048
    g = GpuLayer(sh, full, shards=[0])
    S = Bsz + 16
    conv, ssm = g.new_pools(S)
    meta = B.SeqMeta(np.arange(0, Bsz * L + 1, L), slots, np.zeros(Bsz, np.int32), S)
    y = g.prefill(x, meta, conv, ssm)[0]
    _status_ok(g)
    i = 5
    y_i = host(y[i * L:(i + 1) * L])
    h_pre = host(ssm[0][slots[i]])
    sl = torch.from_numpy(slots).cuda()
    yd = np.stack([host(g.decode(xt, sl, conv, ssm)[0][i]) for xt in xdec])
    ref_pre = oracle_tp_sequence(f64(full), sh, x[i * L:(i + 1) * L])[0]
    ref = oracle_tp_sequence(f64(full), sh, x[i * L:(i + 1) * L], np.stack([xt[i] for xt in xdec]))[0]
    assert_close(y_i, ref["y"], TOL["bf16"], "prefill y_partial of sequence 5")
    assert_close(h_pre, ref_pre["ssm"], TOL["bf16"], "ssm state after the prefill")
    assert_close(yd, ref["dec_y"], TOL["bf16"], "decode y_partial of sequence 5")
    assert_close(host(ssm[0][slots[i]]), ref["ssm"], TOL["bf16"], "ssm state")
    assert_close(host(conv[0][slots[i]]), ref["conv"], TOL["bf16"], "conv state")
    # spare slots untouched
    spare = sorted(set(range(S)) - set(slots.tolist()))
    assert torch.all(ssm[0][spare].view(torch.int32) == 0x7FC0DEAD)


@pytest.mark.parametrize("init", INITS)
def test_falcon7b_tp4_long_prefill(init):
    """Falcon-Mamba-7B shard 1/4, 4 x 16384 prefill. Sequence 1 is recomputed whole by the
    oracle: its y_partial over all 16384 tokens, the final SSM state and the conv history
    (the cache the prefill leaves, Section IV-A). The cache property is checked too:
    prefilling that sequence in two pieces, the second continuing from the cache, gives
    the same outputs and final state as the whole run."""
    sh, full, x, _, slots = _workload("falcon7b_tp4_long", init)
    from paper_2602_21144_amd import binding as B
    Bsz, L = 4, 16384
    g = GpuLayer(sh, full, shards=[0])
    S = Bsz + 16
    conv, ssm = g.new_pools(S)
    meta = B.SeqMeta(np.arange(0, Bsz * L + 1, L), slots, np.zeros(Bsz, np.int32), S)
    y = g.prefill(x, meta, conv, ssm)[0]
    _status_ok(g)
    i = 1
    y_full_i = host(y[i * L:(i + 1) * L])
    h_full = host(ssm[0][slots[i]])
    c_full = host(conv[0][slots[i]])
    del y
    ref = oracle_tp_sequence(f64(full), sh, x[i * L:(i + 1) * L])[0]
    assert_close(y_full_i, ref["y"], TOL["bf16"], "y_partial of sequence 1, all 16384 tokens")
    assert_close(h_full, ref["ssm"], TOL["bf16"], "final SSM state of sequence 1")
    assert_close(c_full, ref["conv"], TOL["bf16"], "conv history of sequence 1")
    # two pieces: 7001 tokens fresh, the rest continuing
    conv2, ssm2 = g.new_pools(2)
    cut = 7001
    xa = x[i * L:i * L + cut]
    xb = x[i * L + cut:(i + 1) * L]
    ya = host(g.prefill(xa, B.SeqMeta([0, cut], [1], [0], 2), conv2, ssm2)[0])
    yb = host(g.prefill(xb, B.SeqMeta([0, L - cut], [1], [1], 2), conv2, ssm2)[0])
    assert_close(np.concatenate([ya, yb]), y_full_i, TOL["bf16"], "two pieces vs whole (y)")
    assert_close(host(ssm2[0][1]), h_full, 1e-3, "two pieces vs whole (state)")
    assert np.array_equal(host(conv2[0][1]), c_full)


@pytest.mark.parametrize("init", INITS)
def test_mamba28b_tp4_decode_heavy(init):
    """Mamba-2.8B shard 1/4: 256 sequences prefilled with 512 tokens, then 512 decode steps;
    two sequences sampled at every decode step."""
    sh, full, x, xdec, slots = _workload("mamba2.8b_tp4_decode", init)
    from paper_2602_21144_amd import binding as B
    Bsz, L = 256, 512
    g = GpuLayer(sh, full, shards=[0])
    S = Bsz + 16
    conv, ssm = g.new_pools(S)
    meta = B.SeqMeta(np.arange(0, Bsz * L + 1, L), slots, np.zeros(Bsz, np.int32), S)
    y = g.prefill(x, meta, conv, ssm)[0]
    _status_ok(g)
    sample = [3, 200]
    y_pre = {i: host(y[i * L:(i + 1) * L]) for i in sample}
    del y
    sl = torch.from_numpy(slots).cuda()
    yd = {i: [] for i in sample}
    for xt in xdec:
        out = g.decode(xt, sl, conv, ssm)[0]
        for i in sample:
            yd[i].append(host(out[i]))
    for i in sample:
        ref = oracle_tp_sequence(f64(full), sh, x[i * L:(i + 1) * L], np.stack([xt[i] for xt in xdec]))[0]
        assert_close(y_pre[i], ref["y"], TOL["bf16"], f"prefill y of sequence {i}")
        assert_close(np.stack(yd[i]), ref["dec_y"], TOL["bf16"], f"decode y of sequence {i}")
        assert_close(host(ssm[0][slots[i]]), ref["ssm"], TOL["bf16"], f"state of sequence {i}")
        assert_close(host(conv[0][slots[i]]), ref["conv"], TOL["bf16"], f"conv of sequence {i}")
    spare = sorted(set(range(S)) - set(slots.tolist()))
    assert torch.all(ssm[0][spare].view(torch.int32) == 0x7FC0DEAD)


@pytest.mark.parametrize("act,init", [("bf16", "baseline"), ("bf16", "stress"), ("f32", "baseline"),
                                      ("f32", "stress")])
def test_hybrid3584_tp2_mixed_schedule(act, init):
    """Hybrid-stack mixer shard 1/2: 64 prompts U[128, 8192] packed into 2048-token chunks
    (per-sequence continuation through the cache), one decode step after each chunk for
    every sequence already prefilled, until each has 64 decode tokens (the serving schedule
    the benchmark times, at bf16 storage and at float32). Sampled sequences are recomputed
    whole by the oracle (prompt, then their 64 decode steps)."""
    cfg = synth.CONFIGS["hybrid3584_tp2_mixed"]
    sh, full, lengths, x_all, dec_x, slots = _workload("hybrid3584_tp2_mixed", init, act)
    nseq, steps = cfg["batch"], cfg["decode_steps"]
    starts = np.concatenate([[0], np.cumsum(lengths)])
    S = nseq + 16
    schedule = synth.serving_schedule(lengths, cfg["chunk"], steps)
    windows = [w for kind, w in schedule if kind == "prefill"]
    # sampled: the two shortest prompts that cross a chunk boundary, and the shortest one
    crossing = sorted({p[0] for w in windows for p in w["pieces"] if p[1] > 0}, key=lambda i: lengths[i])
    sample = sorted(set(crossing[:2] + [int(np.argmin(lengths))]))

    from paper_2602_21144_amd import binding as B
    g = GpuLayer(sh, full, shards=[0])
    conv, ssm = g.new_pools(S)
    got_pre = {i: [] for i in sample}
    got_dec = {i: [] for i in sample}
    for kind, what in schedule:
        if kind == "prefill":
            lens = [p[2] for p in what["pieces"]]
            cu = np.concatenate([[0], np.cumsum(lens)])
            seqs = [p[0] for p in what["pieces"]]
            meta = B.SeqMeta(cu, slots[seqs], [1 if p[1] > 0 else 0 for p in what["pieces"]], S)
            y = g.prefill(x_all[what["start"]:what["stop"]], meta, conv, ssm)[0]
            _status_ok(g)
            for k, p in enumerate(what["pieces"]):
                if p[0] in got_pre:
                    got_pre[p[0]].append(host(y[cu[k]:cu[k + 1]]))
        else:
            seqs = [i for i, _ in what]
            xt = np.stack([dec_x[i, k] for i, k in what])
            out = g.decode(xt, torch.from_numpy(slots[seqs]).cuda(), conv, ssm)[0]
            for r, i in enumerate(seqs):
                if i in got_dec:
                    got_dec[i].append(host(out[r]))
    for r in range(g.P):
        assert g.B.take_status(g._dws[r]) == 0

    tol = TOL[act]
    for i in sample:
        ref = oracle_tp_sequence(f64(full), sh, x_all[starts[i]:starts[i + 1]], dec_x[i])[0]
        assert_close(np.concatenate(got_pre[i]), ref["y"], tol, f"prefill y of sequence {i} (len {lengths[i]})")
        assert_close(np.stack(got_dec[i]), ref["dec_y"], tol, f"decode y of sequence {i}")
        assert_close(host(ssm[0][slots[i]]), ref["ssm"], tol, f"state of sequence {i}")
        assert_close(host(conv[0][slots[i]]), ref["conv"], tol, f"conv of sequence {i}")
