"""Helpers for the parity tests: seeded cases, the GPU path through the C ABI, and the
oracle on the same inputs.

The GPU side runs every shard of a channel split on the one GPU: stage 1 on each shard,
the x_proj partials summed with the library's reduce kernel (the first of the two
reductions), then stage 2 on the shards under test. The oracle side never sees a value
computed on the GPU.
"""
from __future__ import annotations

import numpy as np

from paper_2602_21144_amd import synth

# tolerances: relative error of a whole output tensor, in both the max norm and the 2-norm
TOL = {"f32": 1e-5, "bf16": 2e-2}


def rel_err(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    d = got - ref
    inf = float(np.max(np.abs(d)) / max(np.max(np.abs(ref)), 1e-300)) if ref.size else 0.0
    two = float(np.linalg.norm(d) / max(np.linalg.norm(ref), 1e-300)) if ref.size else 0.0
    return max(inf, two)


def assert_close(got, ref, tol, what=""):
    e = rel_err(got, ref)
    assert np.all(np.isfinite(np.asarray(got, np.float64))), f"{what}: non-finite values"
    assert e <= tol, f"{what}: relative error {e:.3e} > {tol:.1e}"
    return e


def f64(w):
    return {k: np.asarray(v, np.float64) for k, v in w.items() if not k.startswith("_")}


def poison_like(t):
    """Fill a pool with a recognisable NaN bit pattern (untouched slots must keep it)."""
    import torch
    if t.dtype == torch.float32:
        t.view(torch.int32).fill_(0x7FC0DEAD)
    else:
        t.view(torch.int16).fill_(0x7FC1)
    return t


class GpuLayer:
    """All shards of one layer on the GPU, fed from the same host arrays as the oracle."""

    def __init__(self, shape: synth.LayerShape, full_host: dict, shards=None, device="cuda"):
        import torch
        from paper_2602_21144_amd import binding as B
        self.B, self.torch = B, torch
        self.shape = shape
        self.P = shape.shard_count
        self.shards = list(range(self.P)) if shards is None else list(shards)
        self.act = shape.act
        self.tdt = B.torch_act(shape.act)
        full_dev = B.upload_weights(full_host, shape.act, device)
        self.desc = {r: B.make_desc(shape, r) for r in range(self.P)}
        self.w = {}
        for r in range(self.P):
            out = B.empty_shard_weights(shape, device)
            B.ssm_shard_slice_weights(self.desc[r], full_dev, out)
            self.w[r] = out
        self.ws_struct = {r: B.weights_struct(self.w[r]) for r in range(self.P)}
        del full_dev
        self.device = device

    # pools ---------------------------------------------------------------
    def new_pools(self, S, poison=True):
        torch = self.torch
        E, N, K = self.shape.d_shard, self.shape.d_state, self.shape.d_conv
        conv = {r: torch.zeros(S, E, K - 1, dtype=self.tdt, device=self.device) for r in range(self.P)}
        ssm = {r: torch.zeros(S, E, N, dtype=torch.float32, device=self.device) for r in range(self.P)}
        if poison:
            for r in range(self.P):
                poison_like(conv[r])
                poison_like(ssm[r])
        return conv, ssm

    def to_dev(self, a):
        return self.torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(self.device, self.tdt)

    # prefill / decode through the C ABI ---------------------------------------
    def prefill(self, x_host, meta, conv, ssm, ws_pref=None, run_shards=None):
        """Returns {rank: y_partial (device)} for the shards in run_shards (default: self.shards)."""
        B, torch = self.B, self.torch
        run = self.shards if run_shards is None else run_shards
        T = meta.T
        W = self.shape.w_dbl
        x = self.to_dev(x_host)
        ws = {}
        for r in range(self.P):
            n = B.prefill_workspace_bytes(self.desc[r], T, meta.nseq)
            ws[r] = ws_pref[r] if ws_pref is not None else B.workspace(n, self.device)
        parts = {r: torch.empty(max(T, 1), W, dtype=torch.float32, device=self.device) for r in range(self.P)}
        for r in range(self.P):
            B.ssm_shard_prefill_stage1(self.desc[r], self.ws_struct[r], x, meta, conv[r], parts[r], ws[r])
        red = parts[0]
        for r in range(1, self.P):
            B.ssm_reduce_add_f32(red, parts[r])
        ys = {}
        for r in run:
            y = torch.empty(max(T, 1), self.shape.d_model, dtype=self.tdt, device=self.device)
            B.ssm_shard_prefill_stage2(self.desc[r], self.ws_struct[r], red, meta, ssm[r], y, ws[r])
            ys[r] = y[:T]
        self.last_ws = ws
        return ys

    def decode(self, x_host, slots_dev, conv, ssm, run_shards=None):
        B, torch = self.B, self.torch
        run = self.shards if run_shards is None else run_shards
        Bd = x_host.shape[0]
        W = self.shape.w_dbl
        x = self.to_dev(x_host)
        if not hasattr(self, "_dws") or self._dws_b < Bd:
            self._dws = {r: B.workspace(B.decode_workspace_bytes(self.desc[r], Bd), self.device) for r in range(self.P)}
            self._dws_b = Bd
        parts = {r: torch.empty(Bd, W, dtype=torch.float32, device=self.device) for r in range(self.P)}
        for r in range(self.P):
            B.ssm_shard_decode_stage1(self.desc[r], self.ws_struct[r], x, slots_dev, conv[r], parts[r], self._dws[r])
        red = parts[0]
        for r in range(1, self.P):
            B.ssm_reduce_add_f32(red, parts[r])
        ys = {}
        for r in run:
            y = torch.empty(Bd, self.shape.d_model, dtype=self.tdt, device=self.device)
            B.ssm_shard_decode_stage2(self.desc[r], self.ws_struct[r], red, slots_dev, ssm[r], y, self._dws[r])
            ys[r] = y
        return ys


def host(t):
    import torch
    return t.detach().to("cpu", torch.float64).numpy() if t.dtype != torch.float64 else t.cpu().numpy()


def oracle_tp_sequence(full64: dict, shape: synth.LayerShape, x_seq, decode_x=None, ranks=(0,)):
    """Oracle of one sequence through all shards (fresh state): prefill, then decode steps.

    Stage 1 runs on every shard (their x_proj partials are summed, the first reduction);
    stage 2 only on the ranks asked for. Returns rank -> {"y": [L, dm], "conv": [E, K-1],
    "ssm": [E, N], "dec_y": [steps, dm]}.
    """
    from oracle import mixer as om
    P = shape.shard_count
    shards = [om.shard_weights(full64, r, P) for r in range(P)]
    E, N, K = shape.d_shard, shape.d_state, shape.d_conv
    L = x_seq.shape[0]
    x64 = np.asarray(x_seq, np.float64)
    cu, sl, hi = [0, L], [0], [0]
    s1 = [om.prefill_stage1(w, x64, cu, sl, hi, np.zeros((1, E, K - 1)), shape.act) for w in shards]
    red = np.sum([s["x_dbl"] for s in s1], axis=0)
    out, sps = {}, {}
    for r in ranks:
        s2 = om.prefill_stage2(shards[r], s1[r], red, cu, sl, hi, np.zeros((1, E, N)), shape.act)
        out[r] = {"y": s2["y"], "conv": s1[r]["conv_pool"][0], "ssm": s2["ssm_pool"][0], "dec_y": []}
        sps[r] = s2["ssm_pool"]
    cps = [s["conv_pool"] for s in s1]
    if decode_x is not None:
        for t in range(decode_x.shape[0]):
            xt = np.asarray(decode_x[t:t + 1], np.float64)
            d1 = [om.decode_stage1(w, xt, [0], cp, shape.act) for w, cp in zip(shards, cps)]
            dred = np.sum([d["x_dbl"] for d in d1], axis=0)
            cps = [d["conv_pool"] for d in d1]
            for r in ranks:
                d2 = om.decode_stage2(shards[r], d1[r], dred, [0], sps[r], shape.act)
                sps[r] = d2["ssm_pool"]
                out[r]["dec_y"].append(d2["y"][0])
        for r in ranks:
            out[r]["dec_y"] = np.array(out[r]["dec_y"])
            out[r]["conv"] = cps[r][0]
            out[r]["ssm"] = sps[r][0]
    return out
