#!/usr/bin/env python3
"""Benchmark of the selective-SSM mixer shard on one MI355X.

Workload: a Mamba-2.8B-shaped layer (d_model 2560, d_inner 5120 split over 2 ranks, so
this GPU runs the 2560-channel shard 0; N 16, dt_rank 160, conv 4), bf16 activations
and weights with fp32 scan state; 8 prompts of 2048 tokens prefilled, then 128 decode
steps over the 8 sequences. One step = that prefill plus the 128 decode steps.

Per shard, the work of one step is: stage 1 (in_proj, conv1d+SiLU, x_proj), the sum of
the x_proj partials over ranks (here: shard 1's partial, computed outside the timed
region because it is the other GPU's work, added by the library's reduce kernel), and
stage 2 (dt_proj, selective scan, out_proj); the same for every decode step.

Prints one JSON line: prefill tokens/s (value), decode us/step, ms per step, a roofline
entry for the kernel that takes the most time in a step (its duration measured during the
timed region by HIP events bound to every 16th of its dispatches on the launch stream, its HBM
traffic from the committed rocprofv3 counter summary), a per-kernel breakdown from one
extra profiled step, and the CPU oracle timed on a bounded sample on the host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "selective-scan prefill tokens/s + decode µs/step per shard; % HBM/MFMA peak"
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
TIMING_EVERY = 16


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic(name, sh, T, Bd, nseq):
    """(roof, amount per launch, unit) of a kernel role: flops for the dense in/out
    projections in prefill, else bytes each operand must move once (s = act bytes)."""
    s = 2 if sh.act == "bf16" else 4
    E, dm, N, R, K, W = sh.d_shard, sh.d_model, sh.d_state, sh.dt_rank, sh.d_conv, sh.w_dbl
    M = T if name.startswith("prefill") else Bd
    table = {
        "prefill.in_proj": ("mfma", 2.0 * T * 2 * E * dm),
        "prefill.out_proj": ("mfma", 2.0 * T * dm * E),
        "prefill.x_proj": ("hbm", T * E * s + W * E * s + T * W * 4),
        "prefill.dt_round": ("hbm", T * R * 4 + T * R * 2),  # delta rounded to bf16 once
        "prefill.dt_proj": ("hbm", T * R * s + E * R * s + T * E * s),
        "prefill.conv1d": ("hbm", 2 * T * E * s + E * (K + 1) * s),
        "prefill.conv_history": ("hbm", 2 * nseq * E * (K - 1) * s),
        "prefill.scan_main": ("hbm", 4 * T * E * s + T * 2 * N * 4 + nseq * E * N * 4 + E * (N + 2) * 4),
        "decode.in_proj": ("hbm", 2 * E * dm * s + M * dm * s + M * 2 * E * s),
        # in_proj with the conv window fused: weights, x_t, u and z out, history read + write
        "decode.in_proj_conv": ("hbm", 2 * E * dm * s + M * dm * s + 2 * M * E * s + 2 * M * E * (K - 1) * s
                                + E * (K + 1) * s),
        # dt_proj with the state step fused: weights, delta, B and C, u and z, g, state read + write
        "decode.dt_proj_state": ("hbm", E * R * s + M * R * 4 + M * 2 * N * 4 + 3 * M * E * s + 2 * M * E * N * 4
                                 + E * (N + 2) * 4),
        "decode.conv": ("hbm", 2 * M * E * (K - 1) * s + 2 * M * E * s + E * (K + 1) * s),
        "decode.x_proj": ("hbm", W * E * s + M * E * s + M * W * 4),
        "decode.dt_proj": ("hbm", E * R * s + M * R * 4 + M * E * s),
        "decode.state_update": ("hbm", 2 * M * E * N * 4 + 4 * M * E * s + M * 2 * N * 4 + E * (N + 2) * 4),
        "decode.out_proj": ("hbm", dm * E * s + M * E * s + M * dm * s),
    }
    if name in table:
        roof, amt = table[name]
        return roof, float(amt), ("TFLOP/s" if roof == "mfma" else "GB/s")
    if name == "exchange.reduce_add":
        return "hbm", None, "GB/s"
    return "hbm", None, "GB/s"


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "mamba2.8b_shard0of2_b8x2048_dec128.traffic.txt")
ROLE_SOURCE = {"prefill.in_proj": "gemm.hip", "prefill.out_proj": "gemm.hip", "prefill.x_proj": "gemm.hip",
               "prefill.dt_proj": "gemm.hip", "prefill.dt_round": "gemm.hip", "prefill.conv1d": "conv.hip", "prefill.conv_history": "conv.hip",
               "prefill.scan_local": "scan.hip", "prefill.scan_link": "scan.hip", "prefill.scan_main": "scan.hip",
               "decode.in_proj_conv": "skinny.hip", "decode.x_proj": "skinny.hip", "decode.dt_proj_state": "skinny.hip",
               "decode.out_proj": "skinny.hip", "exchange.reduce_add": "misc.hip"}
ROLE_SOURCE.update({f"exchange.{op}_{c}": "codec.hip" for op in ("encode", "decode") for c in ("f16", "bf16", "fp8", "int8")})


def source_sha(src):
    import hashlib
    h = hashlib.sha256()
    for f in ("common.h", src):
        with open(os.path.join(ROOT, "paper_2602_21144_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(role):
    """HBM bytes per launch of a kernel role from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary (already scaled by the copy calibration), or None when there is
    no entry or the kernel's source has changed since the counters were taken."""
    src = ROLE_SOURCE.get(role)
    if src is None or not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        for line in f:
            parts = line.split()
            if line.startswith("#") or len(parts) < 5 or parts[0] != role:
                continue
            if parts[4] != source_sha(src):
                return None
            return {"fetch": float(parts[2]), "write": float(parts[3])}
    return None


def achieved(roof, amount, avg_ms):
    if amount is None or avg_ms <= 0:
        return None
    per_s = amount / (avg_ms * 1e-3)
    return per_s / 1e12 if roof == "mfma" else per_s / 1e9


def run(args):
    import numpy as np
    import torch

    from paper_2602_21144_amd import binding as B
    from paper_2602_21144_amd import synth

    cfg = synth.CONFIGS["mamba2.8b_tp2"]
    sh = cfg["shape"]
    Bsz, L, steps_dec = cfg["batch"], cfg["prefill_len"], cfg["decode_steps"]
    T = Bsz * L
    dev = "cuda"
    torch.cuda.set_device(0)
    B.lib()

    log("drawing seeded inputs")
    full = synth.make_layer(sh, cfg["seed"])
    rng = full["_rng"]
    x_host = synth.make_tokens(rng, T, sh.d_model, sh.act)
    xdec_host = np.stack([synth.make_tokens(rng, Bsz, sh.d_model, sh.act) for _ in range(steps_dec)])
    S = Bsz + 16
    slots = synth.make_slots(rng, Bsz)

    log("uploading and slicing weights")
    full_dev = B.upload_weights(full, sh.act, dev)
    desc = [B.make_desc(sh, r) for r in range(sh.shard_count)]
    wdev = []
    for r in range(sh.shard_count):
        out = B.empty_shard_weights(sh, dev)
        B.ssm_shard_slice_weights(desc[r], full_dev, out)
        wdev.append(out)
    del full_dev
    wst = [B.weights_struct(w) for w in wdev]
    act = B.torch_act(sh.act)
    x = torch.from_numpy(x_host).to(dev, act)
    xdec = torch.from_numpy(xdec_host).to(dev, act)
    cu = np.arange(0, T + 1, L, dtype=np.int32)
    meta = B.SeqMeta(cu, slots, np.zeros(Bsz, np.int32), S, dev)
    slots_dev = torch.from_numpy(slots).to(dev)
    E, N, K, W = sh.d_shard, sh.d_state, sh.d_conv, sh.w_dbl
    conv = [torch.zeros(S, E, K - 1, dtype=act, device=dev) for _ in range(sh.shard_count)]
    ssm = [torch.zeros(S, E, N, dtype=torch.float32, device=dev) for _ in range(sh.shard_count)]
    wsp = [B.workspace(B.prefill_workspace_bytes(desc[r], T, Bsz), dev) for r in range(sh.shard_count)]
    wsd = [B.workspace(B.decode_workspace_bytes(desc[r], Bsz), dev) for r in range(sh.shard_count)]
    p0 = torch.empty(T, W, dtype=torch.float32, device=dev)
    q0 = torch.empty(Bsz, W, dtype=torch.float32, device=dev)
    y = torch.empty(T, sh.d_model, dtype=act, device=dev)
    yd = torch.empty(Bsz, sh.d_model, dtype=act, device=dev)

    log("x_proj partials of the other shard (the other GPU's work, outside the timed region)")
    p1_pref = torch.zeros(T, W, dtype=torch.float32, device=dev)
    p1_dec = torch.zeros(steps_dec, Bsz, W, dtype=torch.float32, device=dev)
    pr = torch.empty(T, W, dtype=torch.float32, device=dev)
    qr = torch.empty(Bsz, W, dtype=torch.float32, device=dev)
    for r in range(1, sh.shard_count):
        B.ssm_shard_prefill_stage1(desc[r], wst[r], x, meta, conv[r], pr, wsp[r])
        B.ssm_reduce_add_f32(p1_pref, pr)
        for k in range(steps_dec):
            B.ssm_shard_decode_stage1(desc[r], wst[r], xdec[k], slots_dev, conv[r], qr, wsd[r])
            B.ssm_reduce_add_f32(p1_dec[k], qr)
    torch.cuda.synchronize()

    # the ABI calls of a step, marshalled once (a serving loop issues the same calls on the
    # same buffers every step)
    prefill_calls = (B.bind("ssm_shard_prefill_stage1", desc[0], wst[0], x, meta, conv[0], p0, wsp[0]),
                     B.bind("ssm_reduce_add_f32", p0, p1_pref),
                     B.bind("ssm_shard_prefill_stage2", desc[0], wst[0], p0, meta, ssm[0], y, wsp[0]))
    decode_calls = [(B.bind("ssm_shard_decode_stage1", desc[0], wst[0], xdec[k], slots_dev, conv[0], q0, wsd[0]),
                     B.bind("ssm_reduce_add_f32", q0, p1_dec[k]),
                     B.bind("ssm_shard_decode_stage2", desc[0], wst[0], q0, slots_dev, ssm[0], yd, wsd[0]))
                    for k in range(steps_dec)]

    def prefill():
        for c in prefill_calls:
            c()

    def decode(k):
        for c in decode_calls[k]:
            c()

    def step(evs=None):
        if evs:
            evs[0].record()
        prefill()
        if evs:
            evs[1].record()
        for k in range(steps_dec):
            decode(k)
        if evs:
            evs[2].record()

    log(f"warmup {args.warmup} step(s)")
    for _ in range(max(args.warmup, 1)):
        step()
    torch.cuda.synchronize()

    log("one profiled step (every kernel bracketed by events) for the breakdown")
    B.ssm_timing_collect()
    B.ssm_timing_enable(True)
    step()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    breakdown = B.ssm_timing_collect()
    dominant = max(breakdown, key=lambda n: breakdown[n][1])

    # every TIMING_EVERY-th launch of the dominant kernel is timed by its own dispatch events
    # (each timed dispatch costs about 5 us more; timing every launch would slow the step)
    log(f"timed region: {args.steps} step(s); events bracket every {TIMING_EVERY}th launch of {dominant}")
    B.ssm_timing_enable(True, dominant, every=TIMING_EVERY)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    B.ssm_timing_enable(False)
    dom_launches, dom_ms = B.ssm_timing_collect()[dominant]
    pre_ms = [e[0].elapsed_time(e[1]) for e in evs]
    dec_ms = [e[1].elapsed_time(e[2]) for e in evs]
    step_ms = evs[0][0].elapsed_time(evs[-1][2]) / args.steps
    assert B.take_status(wsp[0]) == 0 and B.take_status(wsd[0]) == 0
    log(f"prefill {np.mean(pre_ms):.3f} ms, decode {1e3 * np.mean(dec_ms) / steps_dec:.2f} us/step, "
        f"step {step_ms:.3f} ms (host wall {1e3 * wall / args.steps:.3f} ms)")

    kernels = {}
    for name, (n, ms) in sorted(breakdown.items(), key=lambda kv: -kv[1][1]):
        roof, amt, unit = algorithmic(name, sh, T, Bsz, Bsz)
        avg = ms / n
        a = achieved(roof, amt, avg)
        peak = PEAK_BF16_TFLOPS if roof == "mfma" else PEAK_HBM_GBS
        kernels[name] = {"launches": n, "avg_us": round(1e3 * avg, 3), "share_of_step": round(ms / sum(v[1] for v in breakdown.values()), 4),
                         "bound": roof, "achieved": None if a is None else round(a, 1), "unit": unit,
                         "frac": None if a is None else round(a / peak, 4)}
    roof, amt, unit = algorithmic(dominant, sh, T, Bsz, Bsz)
    dom_avg = dom_ms / dom_launches
    ach = achieved(roof, amt, dom_avg)
    peak = PEAK_BF16_TFLOPS if roof == "mfma" else PEAK_HBM_GBS
    tr = measured_traffic(dominant)
    roofline = {"kernel": dominant, "bound": roof, "achieved": None if ach is None else round(ach, 2), "peak": peak,
                "unit": unit, "frac": None if ach is None else round(ach / peak, 4),
                "traffic": None if tr is None else round(tr["fetch"] + tr["write"]),
                "traffic_fetch_write": None if tr is None else [round(tr["fetch"]), round(tr["write"])],
                "avg_us": round(1e3 * dom_avg, 3), "launches_timed": dom_launches, "timed_every": TIMING_EVERY,
                "algorithmic_per_launch": amt}

    scan_ms = sum(breakdown[k][1] for k in breakdown if k.startswith("prefill.scan"))
    result = {
        "metric": METRIC, "value": round(T / (np.mean(pre_ms) * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "Mamba-2.8B-shaped mixer layer, shard 0 of a 2-way channel split: d_model 2560, "
                               "d_inner 2560 of 5120, d_state 16, dt_rank 160, d_conv 4; batch 8 x prefill 2048, "
                               "then 128 decode steps; bf16 activations/weights, fp32 state; seed 1",
                   "d_model": sh.d_model, "d_inner_shard": sh.d_shard, "d_inner_total": sh.d_inner,
                   "d_state": sh.d_state, "dt_rank": sh.dt_rank, "d_conv": sh.d_conv, "batch": Bsz,
                   "prefill_len": L, "decode_steps": steps_dec, "shard": "0 of 2"},
        "prefill_ms": round(float(np.mean(pre_ms)), 4),
        "decode_us_per_step": round(float(1e3 * np.mean(dec_ms) / steps_dec), 3),
        # device time of the kernels alone (stage 1 + stage 2, exchange excluded), from the breakdown step
        "prefill_kernels_ms": round(sum(v[1] for k, v in breakdown.items() if k.startswith("prefill.")), 4),
        "decode_kernels_us_per_step": round(1e3 * sum(v[1] for k, v in breakdown.items() if k.startswith("decode."))
                                            / steps_dec, 3),
        "scan_tokens_per_s": round(T / (scan_ms * 1e-3), 1) if scan_ms > 0 else None,
        "roofline": roofline,
        "kernels": kernels,
    }
    if not args.no_codec:
        log("quantized exchange codecs on this workload's two exchange tensors (outside the timed region)")
        xa = torch.empty(T, W, dtype=torch.float32, device=dev)
        B.ssm_shard_prefill_stage1(desc[0], wst[0], x, meta, conv[0], xa, wsp[0])   # shard 0's x_proj partial
        y1 = torch.empty(T, sh.d_model, dtype=act, device=dev)
        ssm1 = torch.zeros(S, E, N, dtype=torch.float32, device=dev)
        B.ssm_shard_prefill_stage2(desc[1], wst[1], p0, meta, ssm1, y1, wsp[1])      # shard 1's out_proj partial
        result["codec"] = codec_figures(B, torch, {"x_dbl": [xa, p1_pref], "y_partial": [y, y1]})
    if not args.no_mamba2:
        log("Mamba-2 (SSD) shard on its workload (outside the timed region)")
        result["mamba2"] = mamba2_figures(B, torch, args.steps, args.warmup)
    if not args.no_ablation:
        log("cache vs no-cache generation through a 64-layer stack (outside the timed region)")
        result["ablation"] = ablation_figures(B, torch)
    if not args.no_decode_heavy:
        log("decode-heavy step: 256 cached sequences on the 2.8B quarter shard (outside the timed region)")
        result["decode_heavy"] = decode_heavy_figures(B, torch)
    return result, (sh, full, x_host, xdec_host, slots, S)


def mamba2_figures(B, torch, steps, warmup):
    """The Mamba-2 (SSD) shard on its 2.7B-shaped workload (shard 0 of 2: 40 heads of 64,
    N 128, one replicated B/C group): 8 x 2048 prefill and 128 decode steps, the other
    shard's sums of squares precomputed (the other GPU's work), per-dispatch kernel times."""
    import numpy as np
    from paper_2602_21144_amd import synth
    cfg = synth.MAMBA2_CONFIGS["mamba2_2.7b_tp2"]
    sh = cfg["shape"]
    Bsz, L, nd = cfg["batch"], cfg["prefill_len"], cfg["decode_steps"]
    T = Bsz * L
    dev = "cuda"
    full = synth.make_mamba2_layer(sh, cfg["seed"])
    rng = full["_rng"]
    x = torch.from_numpy(synth.make_tokens(rng, T, sh.d_model, "bf16")).to(dev, torch.bfloat16)
    xdec = torch.from_numpy(np.stack([synth.make_tokens(rng, Bsz, sh.d_model, "bf16") for _ in range(nd)])).to(
        dev, torch.bfloat16)
    slots = synth.make_slots(rng, Bsz)
    S = Bsz + 16
    fd = B.upload_weights2(full, dev)
    desc = [B.make_desc2(sh, r) for r in range(2)]
    w = []
    for r in range(2):
        o = B.empty_shard_weights2(sh, dev)
        B.ssm2_shard_slice_weights(desc[r], fd, o)
        w.append(B.weights2_struct(o))
        w[-1]._keep = o
    del fd
    meta = B.SeqMeta(np.arange(0, T + 1, L), slots, np.zeros(Bsz, np.int32), S, dev)
    sl = torch.from_numpy(slots).to(dev)
    conv = [torch.zeros(S, sh.conv_dim_shard, sh.d_conv - 1, dtype=torch.bfloat16, device=dev) for _ in range(2)]
    ssm = [torch.zeros(S, sh.heads_shard, 64, 128, dtype=torch.float32, device=dev) for _ in range(2)]
    wsp = [B.workspace(B.m2_prefill_workspace_bytes(desc[r], T, Bsz), dev) for r in range(2)]
    wsd = [B.workspace(B.m2_decode_workspace_bytes(desc[r], Bsz), dev) for r in range(2)]
    G = sh.ngroups
    ss0, ss1 = (torch.zeros(T, G, dtype=torch.float32, device=dev) for _ in range(2))
    q0 = torch.zeros(Bsz, G, dtype=torch.float32, device=dev)
    q1 = torch.zeros(nd, Bsz, G, dtype=torch.float32, device=dev)
    y = torch.empty(T, sh.d_model, dtype=torch.bfloat16, device=dev)
    yd = torch.empty(Bsz, sh.d_model, dtype=torch.bfloat16, device=dev)
    # the other shard's partial sums of squares (its GPU's work), outside the timed region
    B.ssm2_shard_prefill_stage1(desc[1], w[1], x, meta, conv[1], ssm[1], ss1, wsp[1])
    for k in range(nd):
        B.ssm2_shard_decode_stage1(desc[1], w[1], xdec[k], sl, conv[1], ssm[1], q1[k], wsd[1])
    pre = (B.bind("ssm2_shard_prefill_stage1", desc[0], w[0], x, meta, conv[0], ssm[0], ss0, wsp[0]),
           B.bind("ssm_reduce_add_f32", ss0, ss1),
           B.bind("ssm2_shard_prefill_stage2", desc[0], w[0], ss0, T, y, wsp[0]))
    dec = [(B.bind("ssm2_shard_decode_stage1", desc[0], w[0], xdec[k], sl, conv[0], ssm[0], q0, wsd[0]),
            B.bind("ssm_reduce_add_f32", q0, q1[k]),
            B.bind("ssm2_shard_decode_stage2", desc[0], w[0], q0, Bsz, yd, wsd[0])) for k in range(nd)]

    def step(evs=None):
        if evs:
            evs[0].record()
        for c in pre:
            c()
        if evs:
            evs[1].record()
        for k in range(nd):
            for c in dec[k]:
                c()
        if evs:
            evs[2].record()
    for _ in range(max(warmup, 1)):
        step()
    torch.cuda.synchronize()
    B.ssm_timing_collect()
    B.ssm_timing_enable(True)
    step()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    bd = B.ssm_timing_collect()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    assert B.take_status(wsp[0]) == 0 and B.take_status(wsd[0]) == 0
    pre_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    dec_us = float(np.mean([e[1].elapsed_time(e[2]) for e in evs])) * 1e3 / nd
    kernels = {k: {"launches": n, "avg_us": round(1e3 * ms / n, 3)} for k, (n, ms) in
               sorted(bd.items(), key=lambda kv: -kv[1][1])}
    # SSD main pass: per 64-token chunk and head, the four products (two of them on hi/lo
    # operand pairs) and the bytes the pass must move: x, z, B, C, dt in, g out
    E, H, N, P, Q = sh.d_shard, sh.heads_shard, 128, 64, 64
    flops = (T / Q) * H * (2 * Q * Q * N + 2 * Q * Q * P + 4 * Q * N * P + 4 * P * Q * N)
    nbytes = T * (3 * E * 2 + 2 * sh.groups_shard * N * 2 + H * 2)
    main = bd.get("prefill.ssd_main", (1, float("nan")))
    main_s = main[1] / main[0] * 1e-3
    return {"workload": "Mamba-2 2.7B-shaped mixer layer, shard 0 of a 2-way head split: d_model 2560, 40 of 80 "
                        "heads of 64, d_state 128, one B/C group (replicated), d_conv 4; batch 8 x prefill 2048, "
                        "then 128 decode steps; bf16 activations, fp32 state; seed 11",
            "prefill_ms": round(pre_ms, 4), "prefill_tokens_per_s": round(T / (pre_ms * 1e-3), 1),
            "decode_us_per_step": round(dec_us, 3),
            "ssd_main": {"avg_us": round(main_s * 1e6, 3), "TFLOP_per_s": round(flops / main_s / 1e12, 1),
                         "GB_per_s": round(nbytes / main_s / 1e9, 1), "flops": flops, "bytes": nbytes},
            "kernels": kernels}


def decode_heavy_figures(B, torch, steps=64):
    """Decode-heavy serving step on the Mamba-2.8B quarter shard (1280 of 5120 channels,
    d_model 2560): 256 sequences holding cached states, one single-token step each. Above
    64 sequences the step runs tiled projections, the conv-step kernel and the state-step
    kernel, whose traffic is the state cache (read and written once: 2 B E N 4 bytes).
    Weights are drawn on the GPU with the one-layer recipe; the cache pools hold seeded
    random values (the timing does not depend on them); the other shards' x_proj partial
    (their GPUs' work) is precomputed, as in the headline step.

    The 256 sequences' states (21 MB) stay in the 256 MB MALL from step to step, so the
    state kernel's rate is also measured with 16 groups of 256 sequences in a 4112-slot
    pool (337 MB of states), each step serving the next group: every step's states then
    come from HBM ("state_beyond_mall")."""
    import math
    import numpy as np
    from paper_2602_21144_amd import synth
    cfg = synth.CONFIGS["mamba2.8b_tp4_decode"]
    sh, Bd = cfg["shape"], cfg["batch"]
    E, dm, N, R, K, W = sh.d_shard, sh.d_model, sh.d_state, sh.dt_rank, sh.d_conv, sh.w_dbl
    dev = "cuda"
    g = torch.Generator(device=dev)
    g.manual_seed(cfg["seed"])

    def nrm(*size, std=0.02):
        return (torch.randn(*size, generator=g, device=dev) * std).to(torch.bfloat16)

    lo, hi = math.log(1e-3), math.log(0.1)
    dt0 = torch.exp(torch.rand(E, generator=g, device=dev) * (hi - lo) + lo)
    w = {"W_in": nrm(2 * E, dm), "conv_w": nrm(E, K), "conv_b": nrm(E), "W_x": nrm(W, E), "W_dt": nrm(E, R),
         "W_out": nrm(dm, E), "b_dt": (dt0 + torch.log(-torch.expm1(-dt0))).float(),
         "A_log": torch.log(torch.arange(1, N + 1, device=dev, dtype=torch.float32)).repeat(E, 1).contiguous(),
         "D": torch.ones(E, device=dev)}
    ws_ = B.weights_struct(w)
    d = B.make_desc(sh, 0)
    S = Bd + 16
    slots = torch.from_numpy(synth.make_slots(np.random.default_rng(cfg["seed"]), Bd)).to(dev)
    conv = nrm(S, E, K - 1, std=1.0)
    ssm = torch.randn(S, E, N, generator=g, device=dev) * 0.5
    wsd = B.workspace(B.decode_workspace_bytes(d, Bd), dev)
    xs = [nrm(Bd, dm, std=1.0) for _ in range(steps)]
    q0 = torch.empty(Bd, W, dtype=torch.float32, device=dev)
    other = torch.randn(Bd, W, generator=g, device=dev) * 0.1
    y = torch.empty(Bd, dm, dtype=torch.bfloat16, device=dev)
    calls = [(B.bind("ssm_shard_decode_stage1", d, ws_, xs[k], slots, conv, q0, wsd),
              B.bind("ssm_reduce_add_f32", q0, other),
              B.bind("ssm_shard_decode_stage2", d, ws_, q0, slots, ssm, y, wsd)) for k in range(steps)]

    def run():
        for cs in calls:
            for c in cs:
                c()
    run()
    torch.cuda.synchronize()
    B.ssm_timing_collect()
    B.ssm_timing_enable(True)
    run()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    bd = B.ssm_timing_collect()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    run()
    ev[1].record()
    torch.cuda.synchronize()
    assert B.take_status(wsd) == 0
    step_us = ev[0].elapsed_time(ev[1]) * 1e3 / steps

    # the same steps over 16 groups of sequences whose states together exceed the MALL
    groups = 16
    S2 = groups * Bd + 16
    perm = torch.from_numpy(np.random.default_rng(cfg["seed"] + 1).permutation(Bd).astype(np.int32)).to(dev)
    gslots = [perm + gi * Bd for gi in range(groups)]
    conv2 = nrm(S2, E, K - 1, std=1.0)
    ssm2 = torch.randn(S2, E, N, generator=g, device=dev) * 0.5
    calls2 = [(B.bind("ssm_shard_decode_stage1", d, ws_, xs[k], gslots[k % groups], conv2, q0, wsd),
               B.bind("ssm_reduce_add_f32", q0, other),
               B.bind("ssm_shard_decode_stage2", d, ws_, q0, gslots[k % groups], ssm2, y, wsd)) for k in range(steps)]

    def run2():
        for cs in calls2:
            for c in cs:
                c()
    run2()
    torch.cuda.synchronize()
    ev[0].record()
    run2()
    ev[1].record()
    torch.cuda.synchronize()
    step2_us = ev[0].elapsed_time(ev[1]) * 1e3 / steps
    B.ssm_timing_collect()
    B.ssm_timing_enable(True, "decode.state_update")
    run2()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    bd2 = B.ssm_timing_collect()
    assert B.take_status(wsd) == 0
    del conv2, ssm2
    state_bytes = 2 * Bd * E * N * 4 + 4 * Bd * E * 2 + Bd * 2 * N * 4 + E * (N + 2) * 4
    weight_bytes = (2 * E * dm + W * E + E * R + dm * E) * 2
    step_bytes = weight_bytes + state_bytes + 2 * Bd * E * (K - 1) * 2 + Bd * (dm + 2 * E + W * 4 + dm) * 2
    st = bd.get("decode.state_update", (1, float("nan")))
    st_us = 1e3 * st[1] / st[0]
    st2 = bd2.get("decode.state_update", (1, float("nan")))
    st2_us = 1e3 * st2[1] / st2[0]
    return {"workload": "Mamba-2.8B-shaped layer, shard 0 of a 4-way channel split (d_model 2560, 1280 of 5120 "
                        "channels, d_state 16, dt_rank 160, d_conv 4): 256 sequences with cached states, one "
                        "single-token decode step each; bf16, fp32 state; seed 3",
            "decode_us_per_step": round(step_us, 3),
            "step_bytes": step_bytes, "step_GBps": round(step_bytes / (step_us * 1e-6) / 1e9, 1),
            "step_frac_hbm": round(step_bytes / (step_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "state_kernel": {"avg_us": round(st_us, 3), "bytes": state_bytes,
                             "GBps": round(state_bytes / (st_us * 1e-6) / 1e9, 1),
                             "frac_hbm": round(state_bytes / (st_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)},
            "state_beyond_mall": {"pool_slots": S2, "state_pool_bytes": S2 * E * N * 4,
                                  "decode_us_per_step": round(step2_us, 3), "state_kernel_avg_us": round(st2_us, 3),
                                  "GBps": round(state_bytes / (st2_us * 1e-6) / 1e9, 1),
                                  "frac_hbm": round(state_bytes / (st2_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)},
            "kernels": {k: {"launches": n, "avg_us": round(1e3 * ms / n, 3)}
                        for k, (n, ms) in sorted(bd.items(), key=lambda kv: -kv[1][1])}}


def device_stack_weights(torch, sh, n_layers, seed, dev):
    """Seeded synthetic weights of a full-width stack drawn on the GPU (torch's Philox
    generator; drawing ~5 GB of normals on the host would dominate the run). The recipe is
    the one-layer recipe: matrices and conv ~N(0, 0.02) in bf16, dt0 log-uniform in
    [1e-3, 0.1] with b_dt = softplus^-1(dt0), A_log[c, n] = log(n + 1), D = 1; norm weights 1."""
    import math
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    E, dm, N, R, K = sh.d_inner, sh.d_model, sh.d_state, sh.dt_rank, sh.d_conv

    def nrm(*size):
        return (torch.randn(*size, generator=g, device=dev) * 0.02).to(torch.bfloat16)

    a_log = torch.log(torch.arange(1, N + 1, device=dev, dtype=torch.float32)).repeat(E, 1).contiguous()
    layers = []
    for _ in range(n_layers):
        lo, hi = math.log(1e-3), math.log(0.1)
        dt0 = torch.exp(torch.rand(E, generator=g, device=dev) * (hi - lo) + lo)
        layers.append({"W_in": nrm(2 * E, dm), "conv_w": nrm(E, K), "conv_b": nrm(E), "W_x": nrm(R + 2 * N, E),
                       "W_dt": nrm(E, R), "W_out": nrm(dm, E), "b_dt": (dt0 + torch.log(-torch.expm1(-dt0))).float(),
                       "A_log": a_log.clone(), "D": torch.ones(E, device=dev)})
    return layers, [torch.ones(dm, device=dev) for _ in range(n_layers)], torch.ones(dm, device=dev), g


def ablation_figures(B, torch, n_layers=64, prompt=256, generated=256):
    """Section V's ablation at kernel level on one GPU: per-token latency of generating
    `generated` tokens after a `prompt`-token prompt through a Mamba-2.8B-shaped stack at
    full width, batch 1, with the SSM cache (prefill of the prompt, then one decode step per
    token) and without it (the prompt, then a prefill of the whole prefix for every token).
    Inputs are seeded synthetic rows, not fed back (one stack, no LM head)."""
    import numpy as np
    from paper_2602_21144_amd import synth
    dev = "cuda"
    sh = synth.LayerShape(2560, 5120, 16, 160, 4, 1, "bf16")
    layers, norm_w, final_w, g = device_stack_weights(torch, sh, n_layers, 21, dev)
    sd = B.make_stack_desc(sh, n_layers)
    sw = B.StackWeights(layers, norm_w, final_w)
    conv = [torch.zeros(1, sh.d_inner, sh.d_conv - 1, dtype=torch.bfloat16, device=dev) for _ in range(n_layers)]
    ssm = [torch.zeros(1, sh.d_inner, sh.d_state, dtype=torch.float32, device=dev) for _ in range(n_layers)]
    pools = B.StackPools(conv, ssm)
    n = prompt + generated
    x = torch.randn(n, sh.d_model, generator=g, device=dev).to(torch.bfloat16)
    ws_p = B.workspace(B.stack_prefill_workspace_bytes(sd, n, 1), dev)
    ws_d = B.workspace(B.stack_decode_workspace_bytes(sd, 1), dev)
    out_p = torch.empty(n, sh.d_model, dtype=torch.bfloat16, device=dev)
    out_d = torch.empty(1, sh.d_model, dtype=torch.bfloat16, device=dev)
    slot = torch.zeros(1, dtype=torch.int32, device=dev)
    metas = {L: B.SeqMeta([0, L], [0], [0], 1, dev) for L in range(prompt, n + 1)}
    prefills = {L: B.bind("ssm_stack_prefill", sd, sw, x[:L], metas[L], pools, out_p[:L], ws_p) for L in metas}
    decodes = [B.bind("ssm_stack_decode_step", sd, sw, x[prompt + t:prompt + t + 1], slot, pools, out_d, ws_d)
               for t in range(generated)]

    def cached():
        prefills[prompt]()
        for c in decodes:
            c()

    def no_cache():
        prefills[prompt]()
        for L in range(prompt + 1, n + 1):
            prefills[L]()

    def timed(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    for L in (prompt, n):            # warm up both paths
        prefills[L]()
    decodes[0]()
    t_cache = timed(cached)
    last_cached = out_d.float().clone()
    t_pref = timed(lambda: prefills[prompt]())
    t_nocache = timed(no_cache)
    last_nocache = out_p[n - 1:n].float()
    assert B.take_status(ws_p) == 0 and B.take_status(ws_d) == 0
    diff = float((last_cached - last_nocache).abs().max() / last_nocache.abs().max())
    del layers, sw, conv, ssm, pools, ws_p, ws_d
    torch.cuda.empty_cache()
    return {"workload": f"Mamba-2.8B-shaped stack of {n_layers} layers at full width (d_model 2560, d_inner 5120, "
                        f"d_state 16, dt_rank 160, d_conv 4; pre-norm RMSNorm, fp32 residual), batch 1, "
                        f"{prompt}-token prompt then {generated} generated tokens; bf16; seeded synthetic weights "
                        f"and inputs",
            "cache_ms_per_token": round(t_cache / generated, 4),
            "no_cache_ms_per_token": round(t_nocache / generated, 4),
            "speedup": round(t_nocache / t_cache, 2),
            "prompt_prefill_ms": round(t_pref, 4),
            "decode_step_ms": round((t_cache - t_pref) / generated, 4),
            "last_token_rel_diff_cache_vs_no_cache": round(diff, 5)}


def codec_figures(B, torch, tensors):
    """Section IV-D exchange codecs on real partials of the two exchange points: encode and
    decode-accumulate device time (per-dispatch events), algorithmic GB/s, payload bytes,
    and the largest error of the decoded sum relative to the largest exact sum entry."""
    out = {}
    for tname, parts in tensors.items():
        rows, cols = parts[0].shape
        src_b = parts[0].element_size()
        exact = parts[0].float() + parts[1].float()
        amax = float(exact.abs().max())
        for codec in ("f16", "bf16", "fp8", "int8"):
            pays = [B.exchange_payload(codec, rows, cols) for _ in parts]
            acc = torch.empty(rows, cols, dtype=torch.float32, device=parts[0].device)

            def once():
                for r, t in enumerate(parts):
                    B.ssm_exchange_encode(codec, t, pays[r])
                for r in range(len(parts)):
                    B.ssm_exchange_decode_accumulate(codec, pays[r], acc, accumulate=r > 0)
            once()
            torch.cuda.synchronize()
            B.ssm_timing_collect()
            B.ssm_timing_enable(True)
            for _ in range(10):
                once()
            torch.cuda.synchronize()
            B.ssm_timing_enable(False)
            t = B.ssm_timing_collect()
            enc = t[f"exchange.encode_{codec}"]
            dec = t[f"exchange.decode_{codec}"]
            pb = B.exchange_payload_bytes(codec, rows, cols)
            enc_us, dec_us = 1e3 * enc[1] / enc[0], 1e3 * dec[1] / dec[0]
            # algorithmic bytes: encode reads the partial and writes the payload; decode reads the
            # payload and reads + writes the fp32 sum (the first rank's decode writes it only)
            enc_b = rows * cols * src_b + pb
            dec_b = pb + rows * cols * 4 * 1.5
            out[f"{tname}.{codec}"] = {
                "rows": rows, "cols": cols, "payload_bytes": pb, "raw_bytes": rows * cols * src_b,
                "encode_us": round(enc_us, 3), "encode_GBps": round(enc_b / enc_us / 1e3, 1),
                "decode_accumulate_us": round(dec_us, 3), "decode_accumulate_GBps": round(dec_b / dec_us / 1e3, 1),
                "max_err_rel_to_max": float(f"{float((acc - exact).abs().max()) / max(amax, 1e-30):.3e}")}
    return out


def cpu_baseline(ctx):
    """The oracle (float64 numpy, untuned) on a bounded sample of the same workload."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import mixer as om

    sh, full, x_host, xdec_host, slots, S = ctx
    w64 = {k: np.asarray(v, np.float64) for k, v in full.items() if not k.startswith("_")}
    shards = [om.shard_weights(w64, r, sh.shard_count) for r in range(sh.shard_count)]
    E, N, K = sh.d_shard, sh.d_state, sh.d_conv
    nb = len(slots)
    L = x_host.shape[0] // nb
    cu = np.arange(0, nb * L + 1, L)
    sl = np.arange(nb)
    zc = np.zeros((nb, E, K - 1))
    zs = np.zeros((nb, E, N))
    xs = x_host.astype(np.float64)
    # the other rank's x_proj partials are inputs here, as on the GPU (not timed)
    o1 = om.prefill_stage1(shards[1], xs, cu, sl, np.zeros(nb), zc, sh.act)
    t0 = time.perf_counter()
    s1 = om.prefill_stage1(shards[0], xs, cu, sl, np.zeros(nb), zc, sh.act)
    s2 = om.prefill_stage2(shards[0], s1, s1["x_dbl"] + o1["x_dbl"], cu, sl, np.zeros(nb), zs, sh.act)
    t_pre = time.perf_counter() - t0
    cp, sp, cp1 = s1["conv_pool"], s2["ssm_pool"], o1["conv_pool"]
    nsteps = xdec_host.shape[0]
    t_dec = 0.0
    for k in range(nsteps):
        xd = xdec_host[k].astype(np.float64)
        d1o = om.decode_stage1(shards[1], xd, sl, cp1, sh.act)
        cp1 = d1o["conv_pool"]
        t0 = time.perf_counter()
        d1 = om.decode_stage1(shards[0], xd, sl, cp, sh.act)
        d2 = om.decode_stage2(shards[0], d1, d1["x_dbl"] + d1o["x_dbl"], sl, sp, sh.act)
        t_dec += time.perf_counter() - t0
        cp, sp = d1["conv_pool"], d2["ssm_pool"]
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": round(nb * L / t_pre, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"the whole step on the host: shard 0 prefill of {nb} x {L} tokens (stage 1 + stage 2, "
                      f"float64 numpy, untuned) and {nsteps} decode steps of {nb} sequences; the other shard's "
                      f"x_proj partials are precomputed inputs, as on the GPU",
            "decode_us_per_step": round(1e6 * t_dec / nsteps, 1), "prefill_s": round(t_pre, 2),
            "host_cpus": len(os.sched_getaffinity(0))}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing (profiling runs)")
    ap.add_argument("--no-codec", action="store_true", help="skip the quantized-exchange codec figures")
    ap.add_argument("--no-mamba2", action="store_true", help="skip the Mamba-2 (SSD) shard figures")
    ap.add_argument("--no-ablation", action="store_true", help="skip the cache vs no-cache generation figures")
    ap.add_argument("--no-decode-heavy", action="store_true", help="skip the 256-sequence decode step figures")
    ap.add_argument("--mamba2-only", action="store_true",
                    help="print only the Mamba-2 (SSD) shard figures (its own kernel profile; the headline step "
                         "shares kernel names with it)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy 1 GiB device-to-device once (a kernel of known traffic, "
                         "to scale hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's shard; --gpus {args.gpus} is not supported (this build runs on one GPU)",
              file=sys.stderr)
        sys.exit(2)
    if args.mamba2_only:
        import torch
        from paper_2602_21144_amd import binding as B
        B.lib()
        torch.cuda.set_device(0)
        print(json.dumps({"mamba2": mamba2_figures(B, torch, args.steps, args.warmup)}), flush=True)
        return
    result, ctx = run(args)
    if args.copy_calibration:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copied 1 GiB for counter calibration")
    if not args.no_cpu_baseline:
        log("CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(ctx)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
