#!/usr/bin/env python3
"""Benchmark of the selective-SSM mixer shard on one MI355X.

Headline workload (the largest of the five): the hybrid-stack-shaped mixer, shard 0 of a
2-way channel split (d_model 3584, 3584 of 7168 channels, d_state 16, dt_rank 224,
d_conv 4), serving 64 prompts with lengths uniform in [128, 8192] packed and prefilled in
2048-token chunks, each chunk followed by one decode step for every sequence already
prefilled, until each has 64 decode tokens; seed 4. It runs at float32, the paper's
default precision (activations, weights, accumulation and state), and at bf16 storage
with fp32 state beside it. One step = the whole schedule.

Per shard, a prefill chunk or decode step is stage 1 (in_proj, conv1d + SiLU, x_proj),
the x_proj exchange (the sum of the shards' partials: a cross-GPU reduction, not this
shard's work) and stage 2 (dt_proj, selective scan, out_proj). The exchange is excluded:
an untimed pass runs every shard's stage 1 over the whole schedule and keeps the summed
x_proj output of each chunk and step on the device; the timed steps run shard 0's stage 1
and then stage 2 on that sum.

Prints one JSON line: prefill tokens per second of the whole schedule (value), ms per step,
prefill-only tokens/s, decode us/step, a roofline entry for the kernel that takes the most
time (its duration from HIP events bound to its own dispatches during the timed region, its
HBM traffic from the committed rocprofv3 counter summary), per-kernel figures from one
extra step with every kernel timed, the four other workloads and the bf16 run of the
headline schedule as extra objects, and the CPU oracle on a bounded sample.
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
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}     # dense MFMA
# VALU issue: 256 CUs x 4 SIMDs, one wave64 instruction per SIMD every 4 cycles, 2.4 GHz
PEAK_VALU_GINSTS = 256 * 4 * 2.4e9 / 4 / 1e9

CONFIG_KEYS = {"c0": "mamba130m_f32", "c1": "mamba2.8b_tp2", "c2": "falcon7b_tp4_long",
               "c3": "mamba2.8b_tp4_decode", "c4": "hybrid3584_tp2_mixed"}
WORKLOAD_TEXT = {
    "c0": "Mamba-130m-shaped mixer layer at full width (d_model 768, d_inner 1536, d_state 16, dt_rank 48, "
          "d_conv 4): batch 1, prefill 256 then 16 decode steps; seed 0",
    "c1": "Mamba-2.8B-shaped mixer layer, shard 0 of a 2-way channel split (d_model 2560, 2560 of 5120 channels, "
          "d_state 16, dt_rank 160, d_conv 4): batch 8, prefill 2048 then 128 decode steps; seed 1",
    "c2": "Falcon-Mamba-7B-shaped long-context prefill, shard 0 of a 4-way split (d_model 4096, 2048 of 8192 "
          "channels, d_state 16, dt_rank 256, d_conv 4): batch 4 x prefill 16384, final conv and SSM states "
          "written to the cache; seed 2",
    "c3": "Decode-heavy serving, Mamba-2.8B-shaped shard 0 of a 4-way split (d_model 2560, 1280 of 5120 "
          "channels, d_state 16, dt_rank 160, d_conv 4): 256 sequences prefilled with 512 tokens to fill the "
          "cache, then 512 single-token decode steps over all 256; seed 3",
    "c4": "Hybrid-stack-shaped mixer, shard 0 of a 2-way split (d_model 3584, 3584 of 7168 channels, d_state 16, "
          "dt_rank 224, d_conv 4): 64 prompts with lengths uniform in [128, 8192] packed in index order and "
          "prefilled in 2048-token chunks (per-sequence state continuation), one decode step after each chunk "
          "for every fully prefilled sequence, then decode steps until each sequence has 64; seed 4",
}
PROFILE_STEM = {"c0": "mamba130m_full_b1x256_dec16", "c1": "mamba2.8b_shard0of2_b8x2048_dec128",
                "c2": "falcon7b_shard0of4_b4x16384", "c3": "mamba2.8b_shard0of4_b256x512_dec512",
                "c4": "hybrid3584_shard0of2_64prompts_chunk2048"}


def profile_stem(key, act):
    """Stem of the committed rocprofv3 summaries of a workload (the headline workload runs
    at two precisions, so its stem names the precision)."""
    return PROFILE_STEM[key] + (f"_{act}" if key == "c4" else "")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------------ workloads (host)
def draw_workload(key, act=None, stress=False):
    """Seeded host arrays of one workload, in the recipe's draw order (full-width weights,
    then prompt lengths where they vary, prompts, decode inputs, cache slots), and its
    schedule: a list of phases, each a prefill call over packed pieces or a decode step over
    a batch of sequences. The same draws as the parity tests."""
    import dataclasses

    import numpy as np

    from paper_2602_21144_amd import synth
    cfg = synth.CONFIGS[CONFIG_KEYS[key]]
    sh = cfg["shape"] if act is None else dataclasses.replace(cfg["shape"], act=act)
    full = synth.make_layer(sh, cfg["seed"], stress=stress)
    rng = full.pop("_rng")
    phases = []
    if key == "c4":
        nseq, steps = cfg["batch"], cfg["decode_steps"]
        lo, hi = cfg["len_range"]
        lengths = [int(v) for v in rng.integers(lo, hi, endpoint=True, size=nseq)]
        x_all = synth.make_tokens(rng, int(sum(lengths)), sh.d_model, sh.act)
        dec_x = synth.make_tokens(rng, nseq * steps, sh.d_model, sh.act).reshape(nseq, steps, sh.d_model)
        slots = synth.make_slots(rng, nseq)
        for kind, what in synth.serving_schedule(lengths, cfg["chunk"], steps):
            if kind == "prefill":
                lens = [p[2] for p in what["pieces"]]
                seqs = [p[0] for p in what["pieces"]]
                phases.append({"kind": "prefill", "x": x_all[what["start"]:what["stop"]],
                               "cu": np.concatenate([[0], np.cumsum(lens)]).astype(np.int32),
                               "slots": slots[seqs].astype(np.int32),
                               "has_init": np.array([1 if p[1] > 0 else 0 for p in what["pieces"]], np.int32)})
            else:
                phases.append({"kind": "decode", "x": np.stack([dec_x[i, k] for i, k in what]),
                               "slots": slots[[i for i, _ in what]].astype(np.int32)})
        S = nseq + 16
        info = {"prompts": nseq, "prompt_tokens": int(sum(lengths)), "chunk": cfg["chunk"],
                "decode_tokens_per_sequence": steps}
    else:
        Bsz, L, nd = cfg["batch"], cfg["prefill_len"], cfg["decode_steps"]
        x = synth.make_tokens(rng, Bsz * L, sh.d_model, sh.act)
        xdec = [synth.make_tokens(rng, Bsz, sh.d_model, sh.act) for _ in range(nd)]
        slots = synth.make_slots(rng, Bsz)
        S = Bsz + 16
        phases.append({"kind": "prefill", "x": x, "cu": np.arange(0, Bsz * L + 1, L, dtype=np.int32),
                       "slots": slots, "has_init": np.zeros(Bsz, np.int32)})
        for xt in xdec:
            phases.append({"kind": "decode", "x": xt, "slots": slots})
        info = {"batch": Bsz, "prefill_len": L, "decode_steps": nd}
    return sh, full, phases, S, info


# ------------------------------------------------------------ algorithmic work per kernel
def kernel_work(sh, kind, n, nseq):
    """Kernel roles one prefill call of n tokens (nseq sequences) or one decode step of n
    sequences launches, as the library dispatches them, each with its roof and the work it
    must do: flops for the dense in/out projections in prefill, else the bytes each operand
    and result must move once (s = act bytes). The scan's three passes share one entry."""
    s = 2 if sh.act == "bf16" else 4
    E, dm, N, R, K, W = sh.d_shard, sh.d_model, sh.d_state, sh.dt_rank, sh.d_conv, sh.w_dbl
    bf = sh.act == "bf16"
    if kind == "prefill":
        T = n
        out = {"prefill.in_proj": ("mfma", 2.0 * T * 2 * E * dm),
               "prefill.conv1d": ("hbm", 2 * T * E * s + E * (K + 1) * s),
               "prefill.conv_history": ("hbm", 2 * nseq * E * (K - 1) * s),
               "prefill.x_proj": ("hbm", T * E * s + W * E * s + T * W * 4),
               "prefill.dt_proj": ("hbm", T * R * s + E * R * s + T * E * s),
               "prefill.scan": ("hbm", 4 * T * E * s + T * 2 * N * 4 + 2 * nseq * E * N * 4 + E * (N + 2) * 4),
               "prefill.out_proj": ("mfma", 2.0 * T * dm * E)}
        if bf and R % 32 == 0 and T > 64:
            out["prefill.dt_round"] = ("hbm", T * R * 4 + T * R * 2)
        return out
    M = n

    def proj(nbytes, flops):
        # a decode projection: both its bytes and its flops; its roof over a whole step is the
        # one that takes longer (work_by_role): float32 weights at 64 rows are MFMA-bound
        return ("proj", (nbytes, flops))

    # dt_proj with the state step fused (its epilogue up to 64 sequences, the state-step
    # kernel above): weights, delta, B and C, u and z, g, state read + write
    state = ("hbm", E * R * s + M * R * 4 + M * 2 * N * 4 + 3 * M * E * s + 2 * M * E * N * 4 + E * (N + 2) * 4)
    if bf and K >= 2 and M <= 512:
        return {
            # in_proj with the conv window fused: weights, x_t, u and z out, history read + write
            "decode.in_proj_conv": proj(2 * E * dm * s + M * dm * s + 2 * M * E * s + 2 * M * E * (K - 1) * s
                                        + E * (K + 1) * s, 2.0 * M * 2 * E * dm),
            "decode.x_proj": proj(W * E * s + M * E * s + M * W * 4, 2.0 * M * W * E),
            "decode.dt_proj_state": state,
            "decode.out_proj": proj(dm * E * s + M * E * s + M * dm * s, 2.0 * M * dm * E)}
    if not bf and K >= 2 and M <= 64 and dm % 32 == 0:
        # float32: in_proj with the conv window fused, up to 64 sequences
        return {
            "decode.in_proj_conv": proj(2 * E * dm * s + M * dm * s + 2 * M * E * s + 2 * M * E * (K - 1) * s
                                        + E * (K + 1) * s, 2.0 * M * 2 * E * dm),
            "decode.x_proj": proj(W * E * s + M * E * s + M * W * 4, 2.0 * M * W * E),
            "decode.dt_proj_state": state,
            "decode.out_proj": proj(dm * E * s + M * E * s + M * dm * s, 2.0 * M * dm * E)}
    return {"decode.in_proj": proj(2 * E * dm * s + M * dm * s + M * 2 * E * s, 2.0 * M * 2 * E * dm),
            "decode.conv": ("hbm", 2 * M * E * (K - 1) * s + 2 * M * E * s + E * (K + 1) * s),
            "decode.x_proj": proj(W * E * s + M * E * s + M * W * 4, 2.0 * M * W * E),
            "decode.dt_proj_state": state,
            "decode.out_proj": proj(dm * E * s + M * E * s + M * dm * s, 2.0 * M * dm * E)}


def keep_busy(torch, ms=1.0):
    """Queue a spin of about `ms` on the current stream right after a synchronisation, so that
    the GPU is at work while the host sets up and submits the launches that follow. The first
    kernels after an idle GPU read up to ~300 us each in their own dispatch events (a 5 us
    kernel), and a sampled dispatch that the GPU reaches before the host has submitted it
    reads that wait too; a spin longer than the host's submission of a whole step keeps
    every sampled dispatch behind queued work."""
    if hasattr(torch.cuda, "_sleep"):
        torch.cuda._sleep(int(ms * 2.0e6))


def role_of(name):
    return "prefill.scan" if name.startswith("prefill.scan_") else name


def source_sha(src):
    import hashlib
    h = hashlib.sha256()
    for f in ("common.h", src):
        with open(os.path.join(ROOT, "paper_2602_21144_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def profile_counters(stem, kind, role):
    """Per-launch counter values of a kernel role from a committed rocprofv3 summary
    (profiles/<stem>.<kind>.txt), or None when there is no entry or the kernel's source file
    (named on the line) has changed since the counters were taken. kind "traffic": HBM
    bytes already scaled by the copy calibration ({"fetch", "write"}); kind "util":
    {"valu", "trans"} wave instructions per dispatch."""
    path = os.path.join(ROOT, "profiles", f"{stem}.{kind}.txt")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            parts = line.split()
            if line.startswith("#") or not parts or parts[0] != role:
                continue
            try:
                if kind == "traffic":
                    if parts[4] != source_sha(parts[5]):
                        return None
                    return {"fetch": float(parts[2]), "write": float(parts[3])}
                if kind == "util":
                    if parts[8] != source_sha(parts[9]):
                        return None
                    return {"valu": float(parts[6]), "trans": float(parts[7])}
            except (IndexError, ValueError, OSError):
                return None
    return None


# ----------------------------------------------------------------- the GPU runner
class Workload:
    """One workload on the GPU: every shard's weights (sliced on the device from the
    full-width upload), cache pools, the summed x_proj output of every phase (from an
    untimed pass of all shards' stage 1), and shard 0's calls of a step, marshalled once."""

    def __init__(self, B, torch, key, sh, full, phases, S, info, keep_all=False):
        import numpy as np
        self.B, self.torch, self.key, self.sh, self.info = B, torch, key, sh, info
        dev = "cuda"
        act = B.torch_act(sh.act)
        P = sh.shard_count
        E, N, K, W = sh.d_shard, sh.d_state, sh.d_conv, sh.w_dbl
        full_dev = B.upload_weights(full, sh.act, dev)
        self.desc = [B.make_desc(sh, r) for r in range(P)]
        wdev = []
        for r in range(P):
            o = B.empty_shard_weights(sh, dev)
            B.ssm_shard_slice_weights(self.desc[r], full_dev, o)
            wdev.append(o)
        del full_dev
        self.wdev = wdev
        self.wst = [B.weights_struct(w) for w in wdev]
        self.conv = [torch.zeros(S, E, K - 1, dtype=act, device=dev) for _ in range(P)]
        self.ssm = [torch.zeros(S, E, N, dtype=torch.float32, device=dev) for _ in range(P)]
        maxT = max([len(p["x"]) for p in phases if p["kind"] == "prefill"] + [1])
        maxS = max([len(p["slots"]) for p in phases if p["kind"] == "prefill"] + [1])
        maxB = max([len(p["x"]) for p in phases if p["kind"] == "decode"] + [1])
        self.wsp = [B.workspace(B.prefill_workspace_bytes(self.desc[r], maxT, maxS), dev) for r in range(P)]
        self.wsd = [B.workspace(B.decode_workspace_bytes(self.desc[r], maxB), dev) for r in range(P)]
        self.phases = []
        for p in phases:
            q = {"kind": p["kind"], "n": len(p["x"]), "x": torch.from_numpy(np.ascontiguousarray(p["x"])).to(dev, act)}
            if p["kind"] == "prefill":
                q["meta"] = B.SeqMeta(p["cu"], p["slots"], p["has_init"], S, dev)
                q["nseq"] = len(p["slots"])
            else:
                q["slots"] = torch.from_numpy(np.ascontiguousarray(p["slots"], np.int32)).to(dev)
                q["nseq"] = len(p["slots"])
            self.phases.append(q)
        self.n_prefill_tokens = sum(q["n"] for q in self.phases if q["kind"] == "prefill")
        self.n_decode_steps = sum(1 for q in self.phases if q["kind"] == "decode")
        # the exchange, outside every timed step: all shards' stage 1 over the schedule, summed
        part = torch.empty(maxT, W, dtype=torch.float32, device=dev)
        for q in self.phases:
            n = q["n"]
            q["xdbl"] = torch.zeros(n, W, dtype=torch.float32, device=dev)
            for r in range(P):
                if q["kind"] == "prefill":
                    B.ssm_shard_prefill_stage1(self.desc[r], self.wst[r], q["x"], q["meta"], self.conv[r], part[:n],
                                               self.wsp[r])
                else:
                    B.ssm_shard_decode_stage1(self.desc[r], self.wst[r], q["x"], q["slots"], self.conv[r], part[:n],
                                              self.wsd[r])
                B.ssm_reduce_add_f32(q["xdbl"], part[:n])
        torch.cuda.synchronize()
        if not keep_all:               # the other shards' work is done
            self.wsp, self.wsd = self.wsp[:1], self.wsd[:1]
            self.conv, self.ssm, self.wst, self.desc = self.conv[:1], self.ssm[:1], self.wst[:1], self.desc[:1]
            self.wdev = self.wdev[:1]
            torch.cuda.empty_cache()
        self.y = torch.empty(max(maxT, maxB), sh.d_model, dtype=act, device=dev)
        self.p0 = torch.empty(max(maxT, maxB), W, dtype=torch.float32, device=dev)
        self.stream = torch.cuda.current_stream()
        self.calls = [self._bind(q) for q in self.phases]

    def _bind(self, q, stream=None):
        B = self.B
        d, w, n = self.desc[0], self.wst[0], q["n"]
        one_shard = self.sh.shard_count == 1   # the exchange is the identity: stage 2 reads stage 1's output
        xin = self.p0[:n] if one_shard else q["xdbl"]
        if q["kind"] == "prefill":
            return (B.bind("ssm_shard_prefill_stage1", d, w, q["x"], q["meta"], self.conv[0], self.p0[:n], self.wsp[0],
                           stream=stream),
                    B.bind("ssm_shard_prefill_stage2", d, w, xin, q["meta"], self.ssm[0], self.y[:n], self.wsp[0],
                           stream=stream))
        return (B.bind("ssm_shard_decode_stage1", d, w, q["x"], q["slots"], self.conv[0], self.p0[:n], self.wsd[0],
                       stream=stream),
                B.bind("ssm_shard_decode_stage2", d, w, xin, q["slots"], self.ssm[0], self.y[:n], self.wsd[0],
                       stream=stream))

    def step(self, evs=None):
        for i, cs in enumerate(self.calls):
            if evs is not None:
                evs[i].record()
            for c in cs:
                c()
        if evs is not None:
            evs[-1].record()

    def status_ok(self):
        return self.B.take_status(self.wsp[0]) == 0 and self.B.take_status(self.wsd[0]) == 0

    def work_by_role(self):
        """role -> (roof, [work of each launch in schedule order]) over one step. A decode
        projection takes the roof on which the step's launches take longer in all: their
        bytes at the HBM peak or their flops at the MFMA peak."""
        out, proj = {}, {}
        for q in self.phases:
            for role, (roof, amt) in kernel_work(self.sh, q["kind"], q["n"], q["nseq"]).items():
                if roof == "proj":
                    proj.setdefault(role, []).append(amt)
                else:
                    out.setdefault(role, (roof, []))[1].append(float(amt))
        for role, amts in proj.items():
            t_hbm = sum(b for b, _ in amts) / (PEAK_HBM_GBS * 1e9)
            t_mfma = sum(f for _, f in amts) / (PEAK_TFLOPS[self.sh.act] * 1e12)
            if t_mfma > t_hbm:
                out[role] = ("mfma", [float(f) for _, f in amts])
            else:
                out[role] = ("hbm", [float(b) for b, _ in amts])
        return out


def launches_per_step(wl):
    """Launches of each kernel name in one step: the roles of kernel_work, and the scan's
    three passes once per prefill call."""
    n = {role: len(amts) for role, (roof, amts) in wl.work_by_role().items()}
    if "prefill.scan" in n:
        for p in ("prefill.scan_local", "prefill.scan_link", "prefill.scan_main"):
            n[p] = n["prefill.scan"]
    return n


def measure(B, torch, wl, steps, warmup, dominant_every=None):
    """Warm-up steps; one breakdown step with every 16th launch of each kernel name timed (the
    first included) by events bound to its own dispatch; then the timed steps with events at
    every phase boundary and the dominant kernel's dispatches timed by their own events (every
    launch if it runs 200 us or more, else every 16th). A dispatch's events read its execution
    plus any time the GPU waits for it (for the host to submit it, or for work queued ahead of
    it); sampling few launches keeps the host ahead of the GPU, so that wait stays small."""
    import numpy as np
    for _ in range(max(warmup, 1)):
        wl.step()
    torch.cuda.synchronize()
    keep_busy(torch, 20.0)
    B.ssm_timing_collect()
    B.ssm_timing_enable(True, None, every=16)
    wl.step()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    sampled = B.ssm_timing_collect()
    per_step = launches_per_step(wl)
    # per kernel name: (launches per step, average ms of its sampled launches)
    breakdown = {k: (per_step.get(k, n), ms / n) for k, (n, ms) in sampled.items()}
    dominant = max(breakdown, key=lambda k: breakdown[k][0] * breakdown[k][1])
    dom_avg_ms = breakdown[dominant][1]
    every = dominant_every or (1 if dom_avg_ms >= 0.2 else 16)
    B.ssm_timing_enable(True, dominant, every=every)
    nph = len(wl.phases)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nph + 1)] for _ in range(steps)]
    torch.cuda.synchronize()
    keep_busy(torch)
    t0 = time.perf_counter()
    for i in range(steps):
        wl.step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    B.ssm_timing_enable(False)
    dom_launches, dom_ms = B.ssm_timing_collect()[dominant]
    assert wl.status_ok(), "a kernel flagged bad metadata"
    step_ms = [e[0].elapsed_time(e[-1]) for e in evs]
    pre_ms, dec_ms = [], []
    for e in evs:
        ph = [e[j].elapsed_time(e[j + 1]) for j in range(nph)]
        pre_ms.append(sum(t for t, q in zip(ph, wl.phases) if q["kind"] == "prefill"))
        dec_ms.append(sum(t for t, q in zip(ph, wl.phases) if q["kind"] == "decode"))
    # work of the sampled launches of the dominant kernel (its launches are numbered over
    # the timed steps; every `every`-th is timed, the first included)
    work = wl.work_by_role()
    dom_role = role_of(dominant)
    sampled_work = None
    if dom_role in work and not dom_role.startswith("prefill.scan"):
        amts = work[dom_role][1]
        n = len(amts)
        sampled_work = sum(amts[j % n] for j in range(0, steps * n, every))
    return {"breakdown": breakdown, "dominant": dominant, "every": every, "dom_launches": dom_launches,
            "dom_ms": dom_ms, "sampled_work": sampled_work, "step_ms": float(np.mean(step_ms)),
            "prefill_ms": float(np.mean(pre_ms)), "decode_ms": float(np.mean(dec_ms)), "wall_s": wall,
            "work": work}


def kernel_figures(wl, m):
    """Per-kernel (and per-role) figures from the breakdown step: launches per step, average
    time of the sampled launches, estimated share of the step, roof, achieved rate (work of
    the sampled launches over their time) and fraction of the roof's peak."""
    sh = wl.sh
    bd = m["breakdown"]
    total = sum(n * ms for n, ms in bd.values())
    mf_peak = PEAK_TFLOPS[sh.act]
    out = {}
    for name, (n, ms) in sorted(bd.items(), key=lambda kv: -kv[1][0] * kv[1][1]):
        e = {"launches": n, "avg_us": round(1e3 * ms, 3), "share_of_step": round(n * ms / total, 4)}
        role = role_of(name)
        if role in m["work"] and role == name:
            roof, amts = m["work"][role]
            sampled = amts[::16]
            rate = (sum(sampled) / len(sampled)) / (ms * 1e-3)
            if roof == "mfma":
                e.update(bound="mfma", achieved=round(rate / 1e12, 2), unit="TFLOP/s", peak=mf_peak,
                         frac=round(rate / 1e12 / mf_peak, 4))
            else:
                e.update(bound="hbm", achieved=round(rate / 1e9, 1), unit="GB/s", peak=PEAK_HBM_GBS,
                         frac=round(rate / 1e9 / PEAK_HBM_GBS, 4))
        out[name] = e
    # the scan's three passes together: the scan's bytes over their summed time, and the
    # VALU issue rate from the committed counter summary, when it matches the source
    scan = [k for k in bd if k.startswith("prefill.scan_")]
    if scan and "prefill.scan" in m["work"]:
        amts = m["work"]["prefill.scan"][1][::16]    # the sampled prefill calls
        ms = sum(bd[k][1] for k in scan) * len(amts)
        launches = len(amts)
        amt = sum(amts)
        gbs = amt / (ms * 1e-3) / 1e9
        e = {"passes": sorted(scan), "launches": launches, "avg_us": round(1e3 * ms / launches, 3), "bound": "alu",
             "hbm": {"achieved": round(gbs, 1), "unit": "GB/s", "peak": PEAK_HBM_GBS,
                     "frac": round(gbs / PEAK_HBM_GBS, 4), "bytes_per_launch": amt / launches}}
        insts = 0.0
        for k in scan:
            c = profile_counters(profile_stem(wl.key, wl.sh.act), "util", k)
            if c is None:
                insts = None
                break
            insts += c["valu"] + c["trans"]     # a transcendental takes two issue slots
        if insts is not None:
            rate = insts / (ms * 1e-3 / launches) / 1e9
            e["valu_issue"] = {"achieved": round(rate, 1), "unit": "G wave-instructions/s",
                               "peak": PEAK_VALU_GINSTS, "frac": round(rate / PEAK_VALU_GINSTS, 4),
                               "insts_per_launch": insts}
        out["prefill.scan (3 passes)"] = e
    return out


def roofline_entry(wl, m):
    sh = wl.sh
    dom = m["dominant"]
    role = role_of(dom)
    avg_ms = m["dom_ms"] / m["dom_launches"]
    roof = m["work"].get(role, ("hbm", None))[0]
    ach = peak = unit = per_launch = None
    if m["sampled_work"] is not None:
        rate = m["sampled_work"] / (m["dom_ms"] * 1e-3)
        per_launch = m["sampled_work"] / m["dom_launches"]
        if roof == "mfma":
            ach, peak, unit = rate / 1e12, PEAK_TFLOPS[sh.act], "TFLOP/s"
        else:
            ach, peak, unit = rate / 1e9, PEAK_HBM_GBS, "GB/s"
    tr = profile_counters(profile_stem(wl.key, sh.act), "traffic", dom)
    return {"kernel": dom, "bound": roof, "achieved": None if ach is None else round(ach, 2), "peak": peak,
            "unit": unit, "frac": None if ach is None else round(ach / peak, 4),
            "traffic": None if tr is None else round(tr["fetch"] + tr["write"]),
            "traffic_fetch_write": None if tr is None else [round(tr["fetch"]), round(tr["write"])],
            "avg_us": round(1e3 * avg_ms, 3), "launches_timed": m["dom_launches"], "timed_every": m["every"],
            "algorithmic_per_launch": per_launch,
            "dtype": sh.act}


def summarize(wl, m):
    steps_dec = wl.n_decode_steps
    return {"prefill_tokens": wl.n_prefill_tokens, "decode_steps": steps_dec,
            "ms_per_step": round(m["step_ms"], 4),
            "tokens_per_s_whole_step": round(wl.n_prefill_tokens / (m["step_ms"] * 1e-3), 1),
            "prefill_ms": round(m["prefill_ms"], 4),
            "prefill_tokens_per_s": round(wl.n_prefill_tokens / (m["prefill_ms"] * 1e-3), 1) if m["prefill_ms"] else None,
            "decode_us_per_step": round(1e3 * m["decode_ms"] / steps_dec, 3) if steps_dec else None}


def graph_decode_us(B, torch, wl, reps=3):
    """The decode steps of a workload captured once in a HIP graph and replayed: device time
    per step with launch overhead removed (exchange excluded as in the timed steps)."""
    s = torch.cuda.Stream()
    dec = [q for q in wl.phases if q["kind"] == "decode"]
    if not dec:
        return None
    calls = [wl._bind(q, stream=s) for q in dec]
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for cs in calls:            # warm on the capture stream
            for c in cs:
                c()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for cs in calls:
            for c in cs:
                c()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    keep_busy(torch)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    assert wl.status_ok()
    del g
    return e0.elapsed_time(e1) * 1e3 / (reps * len(dec))


def to_bf16(drawn):
    """The bf16 form of a workload drawn at float32: the same draws rounded to bf16 (ties
    to even), which is what the recipe stores for a bf16 workload."""
    import dataclasses

    from paper_2602_21144_amd import synth
    sh, full, phases, S, info = drawn
    act_keys = ("W_in", "conv_w", "conv_b", "W_x", "W_dt", "W_out")
    full16 = {k: (synth.round_bf16_f32(v) if k in act_keys else v) for k, v in full.items()}
    ph16 = [{**q, "x": synth.round_bf16_f32(q["x"])} for q in phases]
    return dataclasses.replace(sh, act="bf16"), full16, ph16, S, info


def run_workload(B, torch, key, act, steps, warmup, graph=False, drawn=None, keep_all=False):
    if drawn is None:
        log(f"{key} ({act}): drawing seeded host inputs")
        drawn = draw_workload(key, act)
    sh, full, phases, S, info = drawn
    log(f"{key} ({act}): uploading, slicing weights, precomputing the exchange")
    wl = Workload(B, torch, key, sh, full, phases, S, info, keep_all=keep_all)
    log(f"{key} ({act}): {warmup} warm-up and {steps} timed step(s) of {len(wl.phases)} phases")
    m = measure(B, torch, wl, steps, warmup)
    res = {"workload": WORKLOAD_TEXT[key], "dtype": act, **info, **summarize(wl, m),
           "roofline": roofline_entry(wl, m), "kernels": kernel_figures(wl, m)}
    if graph:
        res["decode_us_per_step_graph"] = round(graph_decode_us(B, torch, wl), 3)
    log(f"{key} ({act}): {res['ms_per_step']:.3f} ms/step, prefill {res['prefill_tokens_per_s']} tok/s, "
        f"decode {res['decode_us_per_step']} us/step")
    return res, wl, m


# ------------------------------------------------------------------- CPU baseline
def cpu_model():
    """The host CPU's model name as lscpu reports it (else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(drawn, n_chunks=20, n_decode=4):
    """The oracle (float64 numpy, untuned) on a bounded sample of the headline workload:
    shard 0's stage 1 + stage 2 over the first prefill chunks of the schedule (the other
    shard's x_proj partials precomputed, as on the GPU) and decode steps of 64 sequences;
    then the smallest workload on one core."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import mixer as om
    sh, full, phases, S, info = drawn
    act = sh.act
    w64 = {k: np.asarray(v, np.float64) for k, v in full.items()}
    shards = [om.shard_weights(w64, r, sh.shard_count) for r in range(sh.shard_count)]
    E, N, K = sh.d_shard, sh.d_state, sh.d_conv
    conv = [np.zeros((S, E, K - 1)) for _ in shards]
    ssm0 = np.zeros((S, E, N))
    pre = [q for q in phases if q["kind"] == "prefill"][:n_chunks]
    t_pre, tokens = 0.0, 0
    for q in pre:
        x = q["x"].astype(np.float64)
        others = []
        for r in range(1, len(shards)):
            o = om.prefill_stage1(shards[r], x, q["cu"], q["slots"], q["has_init"], conv[r], sh.act)
            conv[r] = o["conv_pool"]
            others.append(o["x_dbl"])
        t0 = time.perf_counter()
        s1 = om.prefill_stage1(shards[0], x, q["cu"], q["slots"], q["has_init"], conv[0], sh.act)
        red = s1["x_dbl"] + sum(others)
        s2 = om.prefill_stage2(shards[0], s1, red, q["cu"], q["slots"], q["has_init"], ssm0, sh.act)
        t_pre += time.perf_counter() - t0
        conv[0], ssm0 = s1["conv_pool"], s2["ssm_pool"]
        tokens += len(x)
    rng = np.random.default_rng(0)
    Bd = 64
    slots = np.arange(Bd)
    cp = [rng.normal(size=(Bd, E, K - 1)) for _ in shards]
    sp = rng.normal(size=(Bd, E, N)) * 0.5
    t_dec = 0.0
    for _ in range(n_decode):
        xt = rng.normal(size=(Bd, sh.d_model))
        others = []
        for r in range(1, len(shards)):
            o = om.decode_stage1(shards[r], xt, slots, cp[r], sh.act)
            cp[r] = o["conv_pool"]
            others.append(o["x_dbl"])
        t0 = time.perf_counter()
        d1 = om.decode_stage1(shards[0], xt, slots, cp[0], sh.act)
        d2 = om.decode_stage2(shards[0], d1, d1["x_dbl"] + sum(others), slots, sp, sh.act)
        t_dec += time.perf_counter() - t0
        cp[0], sp = d1["conv_pool"], d2["ssm_pool"]
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    # the smallest workload (Mamba-130m shape, full width, fp32) on one core
    sh0, full0, ph0, S0, _ = draw_workload("c0")
    w0 = {k: np.asarray(v, np.float64) for k, v in full0.items()}
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        q = ph0[0]
        E0, K0, N0 = sh0.d_shard, sh0.d_conv, sh0.d_state
        st = om.prefill(w0, q["x"].astype(np.float64), q["cu"], q["slots"], q["has_init"],
                        np.zeros((S0, E0, K0 - 1)), np.zeros((S0, E0, N0)), sh0.act)
        t_c0_pre = time.perf_counter() - t0
        cpool, spool = st["conv_pool"], st["ssm_pool"]
        t0 = time.perf_counter()
        for q in ph0[1:]:
            d = om.decode_step(w0, q["x"].astype(np.float64), q["slots"], cpool, spool, sh0.act)
            cpool, spool = d["conv_pool"], d["ssm_pool"]
        t_c0_dec = time.perf_counter() - t0
    return {"value": round(tokens / t_pre, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"the first {len(pre)} prefill chunks of the headline schedule ({tokens} tokens, "
                      f"{sum(len(q['slots']) for q in pre)} sequence pieces) through shard 0's stage 1 + stage 2 "
                      f"in {act}, and {n_decode} decode steps of {Bd} sequences; float64 numpy, untuned; the other "
                      f"shard's x_proj partials are precomputed inputs, as on the GPU",
            "decode_us_per_step": round(1e6 * t_dec / n_decode, 1), "prefill_s": round(t_pre, 2),
            "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
            "c0_one_core": {"workload": WORKLOAD_TEXT["c0"], "cores": 1,
                            "prefill_tokens_per_s": round(256 / t_c0_pre, 1),
                            "decode_us_per_step": round(1e6 * t_c0_dec / 16, 1)}}


# ------------------------------------------------------ the NEXT-row figures (extras)
def decode_beyond_mall(B, torch, groups=16):
    """The 2.8B quarter shard's decode step with states that cannot stay in the 256 MB MALL:
    16 groups of 256 sequences in a 4112-slot pool (337 MB of states), each step serving
    the next group, so every step's states come from HBM. Weights, states and inputs are
    seeded device draws (the timing does not depend on their values)."""
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
    S2 = groups * Bd + 16
    perm = torch.from_numpy(np.random.default_rng(cfg["seed"] + 1).permutation(Bd).astype(np.int32)).to(dev)
    gslots = [perm + gi * Bd for gi in range(groups)]
    conv2 = nrm(S2, E, K - 1, std=1.0)
    ssm2 = torch.randn(S2, E, N, generator=g, device=dev) * 0.5
    wsd = B.workspace(B.decode_workspace_bytes(d, Bd), dev)
    steps = 64
    xs = [nrm(Bd, dm, std=1.0) for _ in range(steps)]
    q0 = torch.empty(Bd, W, dtype=torch.float32, device=dev)
    xr = torch.randn(Bd, W, generator=g, device=dev) * 0.1
    y = torch.empty(Bd, dm, dtype=torch.bfloat16, device=dev)
    calls = [(B.bind("ssm_shard_decode_stage1", d, ws_, xs[k], gslots[k % groups], conv2, q0, wsd),
              B.bind("ssm_shard_decode_stage2", d, ws_, xr, gslots[k % groups], ssm2, y, wsd)) for k in range(steps)]

    def run():
        for cs in calls:
            for c in cs:
                c()
    run()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    run()
    ev[1].record()
    torch.cuda.synchronize()
    step_us = ev[0].elapsed_time(ev[1]) * 1e3 / steps
    keep_busy(torch, 20.0)
    B.ssm_timing_collect()
    # every 8th launch: timing every launch lets the host fall behind the GPU and the events
    # then include the wait for the host
    B.ssm_timing_enable(True, "decode.dt_proj_state", every=8)
    run()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    bd = B.ssm_timing_collect()
    assert B.take_status(wsd) == 0
    st = bd.get("decode.dt_proj_state", (1, float("nan")))
    st_us = 1e3 * st[1] / st[0]
    state_bytes = 2 * Bd * E * N * 4 + 3 * Bd * E * 2 + Bd * 2 * N * 4 + E * (N + 2) * 4 + E * R * 2 + Bd * R * 4
    return {"workload": "the decode-heavy step (2.8B quarter shard, 256 sequences) over 16 groups of 256 sequences "
                        "in a 4112-slot pool (337 MB of states), each step serving the next group",
            "state_pool_bytes": S2 * E * N * 4, "decode_us_per_step": round(step_us, 3),
            "state_kernel_avg_us": round(st_us, 3), "state_kernel_GBps": round(state_bytes / (st_us * 1e-6) / 1e9, 1),
            "state_kernel_frac_hbm": round(state_bytes / (st_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}


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
    # the exchange of the sums of squares, outside the timed region: both shards' stage 1
    # over the step, the partial sums added; the timed steps run shard 0's stage 1 and then
    # stage 2 on the summed values
    ssum = torch.zeros(T, G, dtype=torch.float32, device=dev)
    qsum = torch.zeros(nd, Bsz, G, dtype=torch.float32, device=dev)
    for r, part in ((0, ss0), (1, ss1)):
        B.ssm2_shard_prefill_stage1(desc[r], w[r], x, meta, conv[r], ssm[r], part, wsp[r])
        B.ssm_reduce_add_f32(ssum, part)
    for k in range(nd):
        for r, part in ((0, q0), (1, q1[k])):
            B.ssm2_shard_decode_stage1(desc[r], w[r], xdec[k], sl, conv[r], ssm[r], part, wsd[r])
            B.ssm_reduce_add_f32(qsum[k], part)
    pre = (B.bind("ssm2_shard_prefill_stage1", desc[0], w[0], x, meta, conv[0], ssm[0], ss0, wsp[0]),
           B.bind("ssm2_shard_prefill_stage2", desc[0], w[0], ssum, T, y, wsp[0]))
    dec = [(B.bind("ssm2_shard_decode_stage1", desc[0], w[0], xdec[k], sl, conv[0], ssm[0], q0, wsd[0]),
            B.bind("ssm2_shard_decode_stage2", desc[0], w[0], qsum[k], Bsz, yd, wsd[0])) for k in range(nd)]

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
    keep_busy(torch, 20.0)
    B.ssm_timing_collect()
    B.ssm_timing_enable(True, None, every=16)   # sampled, so the queue stays full
    step()
    torch.cuda.synchronize()
    B.ssm_timing_enable(False)
    bd = B.ssm_timing_collect()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    keep_busy(torch)
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    assert B.take_status(wsp[0]) == 0 and B.take_status(wsd[0]) == 0
    pre_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    dec_us = float(np.mean([e[1].elapsed_time(e[2]) for e in evs])) * 1e3 / nd
    kernels = {k: {"timed_launches": n, "avg_us": round(1e3 * ms / n, 3)} for k, (n, ms) in
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
                        "then 128 decode steps; bf16 activations, fp32 state; seed 11; the sum-of-squares exchange "
                        "excluded",
            "prefill_ms": round(pre_ms, 4), "prefill_tokens_per_s": round(T / (pre_ms * 1e-3), 1),
            "decode_us_per_step": round(dec_us, 3),
            "ssd_main": {"avg_us": round(main_s * 1e6, 3), "TFLOP_per_s": round(flops / main_s / 1e12, 1),
                         "GB_per_s": round(nbytes / main_s / 1e9, 1), "flops": flops, "bytes": nbytes},
            "kernels": kernels}


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


def codec_on_c1(B, torch, wl):
    """The codecs on the 2.8B half shard's two exchange tensors of its prefill: both shards'
    x_proj partials and both shards' out_proj partials."""
    q = wl.phases[0]
    n = q["n"]
    act = B.torch_act(wl.sh.act)
    p = [torch.empty(n, wl.sh.w_dbl, dtype=torch.float32, device="cuda") for _ in range(2)]
    y = [torch.empty(n, wl.sh.d_model, dtype=act, device="cuda") for _ in range(2)]
    for r in range(2):
        B.ssm_shard_prefill_stage1(wl.desc[r], wl.wst[r], q["x"], q["meta"], wl.conv[r], p[r], wl.wsp[r])
    for r in range(2):
        B.ssm_shard_prefill_stage2(wl.desc[r], wl.wst[r], q["xdbl"], q["meta"], wl.ssm[r], y[r], wl.wsp[r])
    return codec_figures(B, torch, {"x_dbl": p, "y_partial": y})


# ------------------------------------------------------------------------- main
def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", choices=sorted(CONFIG_KEYS), default="c4",
                    help="workload of the headline line (default c4, the largest)")
    ap.add_argument("--dtype", choices=["f32", "bf16"], default=None,
                    help="arithmetic of the headline run (default: f32 for c4, the paper's default precision; "
                         "the workload's own dtype otherwise)")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the headline workload (profiling runs): no other workloads, no NEXT-row figures")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing (profiling runs)")
    ap.add_argument("--no-next", action="store_true", help="skip the codec, Mamba-2 and ablation figures")
    ap.add_argument("--mamba2-only", action="store_true",
                    help="profiling runs of the Mamba-2 shard: only its figures, printed as one JSON line")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy 1 GiB device-to-device once (a kernel of known traffic, "
                         "to scale hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU's shard; --gpus {args.gpus} is not supported: this build runs on one GPU, "
              f"and the cross-GPU exchanges are outside it", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2602_21144_amd import binding as B
    from paper_2602_21144_amd import synth
    torch.cuda.set_device(0)
    B.lib()
    if args.mamba2_only:
        log("Mamba-2 (SSD) shard")
        print(json.dumps({"mamba2": mamba2_figures(B, torch, args.steps, args.warmup)}), flush=True)
        return
    key = args.config
    act = args.dtype or ("f32" if key == "c4" else synth.CONFIGS[CONFIG_KEYS[key]]["shape"].act)
    log(f"{key} ({act}): drawing seeded host inputs")
    drawn = draw_workload(key, "f32" if key == "c4" else act)
    if act == "bf16" and drawn[0].act == "f32":
        drawn = to_bf16(drawn)
    head, wl, m = run_workload(B, torch, key, act, args.steps, args.warmup, graph=(key in ("c1", "c3")),
                               drawn=drawn)
    if args.copy_calibration:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copied 1 GiB for counter calibration")
    sh = wl.sh
    result = {
        "metric": METRIC, "value": head["tokens_per_s_whole_step"], "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": act, "data": "synthetic",
        "config": {"workload": head["workload"] + f"; {act} activations, weights and state"
                   + ("" if act == "f32" else " (fp32 state)"), "key": key,
                   "d_model": sh.d_model, "d_inner_shard": sh.d_shard, "d_inner_total": sh.d_inner,
                   "d_state": sh.d_state, "dt_rank": sh.dt_rank, "d_conv": sh.d_conv,
                   "shard": f"0 of {sh.shard_count}", **wl.info},
        "value_is": "prefill tokens of the whole step (schedule) per second of the step, the interleaved decode "
                    "steps included; the x_proj exchange excluded",
        "prefill_tokens": head["prefill_tokens"], "decode_steps": head["decode_steps"],
        "prefill_ms": head["prefill_ms"], "prefill_tokens_per_s": head["prefill_tokens_per_s"],
        "decode_us_per_step": head["decode_us_per_step"],
        "roofline": head["roofline"], "kernels": head["kernels"],
    }
    if "decode_us_per_step_graph" in head:
        result["decode_us_per_step_graph"] = head["decode_us_per_step_graph"]
    del wl, m
    torch.cuda.empty_cache()
    sample = None
    if not args.no_cpu_baseline:
        # the oracle's sample: the first chunks of the headline schedule (kept before the
        # large arrays are dropped)
        sh_, full_, phases_, S_, info_ = drawn
        pre = [q for q in phases_ if q["kind"] == "prefill"][:20]
        sample = (sh_, full_, pre, S_, info_)
    if not args.no_extras:
        others = {}
        # the bf16 run of the hybrid schedule last (it keeps the headline's host arrays until then)
        head_bf16 = to_bf16(drawn) if key == "c4" and act == "f32" else None
        drawn = None
        for k in ("c0", "c1", "c2", "c3", "c4"):
            if k == key:
                continue
            a = synth.CONFIGS[CONFIG_KEYS[k]]["shape"].act
            r, w2, _ = run_workload(B, torch, k, a, max(1, min(args.steps, 3)), 2, graph=(k in ("c1", "c3")),
                                    keep_all=(k == "c1"))
            if k == "c1" and not args.no_next:
                log("quantized exchange codecs on the 2.8B half shard's exchange tensors")
                result["codec"] = codec_on_c1(B, torch, w2)
            others[k] = r
            del w2
            torch.cuda.empty_cache()
        if head_bf16 is not None:
            r, w2, _ = run_workload(B, torch, "c4", "bf16", max(1, min(args.steps, 3)), 2, drawn=head_bf16)
            others["c4_bf16"] = r
            del w2, head_bf16
            torch.cuda.empty_cache()
        result["workloads"] = others
        log("decode-heavy step with states beyond the MALL")
        result["decode_beyond_mall"] = decode_beyond_mall(B, torch)
        if not args.no_next:
            log("Mamba-2 (SSD) shard")
            result["mamba2"] = mamba2_figures(B, torch, max(1, min(args.steps, 3)), 1)
            log("cache vs no-cache generation through a 64-layer stack")
            result["ablation"] = ablation_figures(B, torch)
    drawn = None
    if sample is not None:
        log("CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(sample)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
