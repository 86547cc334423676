"""Brute-force per-token mixer in pure Python, for tiny shapes only.

TEST INFRASTRUCTURE ONLY: it exists to pin the numpy oracle (``oracle.mixer``) by an
independent implementation. It is written with scalar loops and the ``math`` module,
shares no code with the oracle or with the GPU path, and rounds nothing (exact float64
arithmetic up to summation order).

It walks one sequence token by token through the full-width (unsharded) mixer in the
op order of Section II-B / Fig. 1, with the readings listed in ``oracle.mixer``: packed
[x | z] and [delta | B | C], a causal K-tap convolution with bias and SiLU,
Delta = softplus(dt_proj(delta) + b_dt), h <- exp(Delta*A) h + Delta*B*u,
y = C.h + D*u, gate y*SiLU(z), output projection.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence


def _silu(v: float) -> float:
    return v / (1.0 + math.exp(-v))


def _softplus(v: float) -> float:
    return v if v > 20.0 else math.log1p(math.exp(v))


def _row(m, i) -> List[float]:
    return [float(v) for v in m[i]]


def _rms_scaled(v: Sequence[float], eps: float, weight: Optional[Sequence[float]] = None) -> List[float]:
    ms = sum(a * a for a in v) / len(v)
    inv = 1.0 / math.sqrt(ms + eps)
    return [a * inv * (1.0 if weight is None else float(weight[i])) for i, a in enumerate(v)]


def mixer_sequence(w, x_rows: Sequence[Sequence[float]], conv_hist: Optional[Sequence[Sequence[float]]] = None,
                   h0: Optional[Sequence[Sequence[float]]] = None, bcdt_eps: Optional[float] = None):
    """Run one sequence through the full-width layer.

    w: dict of full-width weights (W_in [2E,dm], conv_w [E,K], conv_b [E], W_x [R+2N,E],
    W_dt [E,R], b_dt [E], A_log [E,N], D [E], W_out [dm,E]).
    x_rows: L rows of d_model values. conv_hist: [E][K-1] (oldest first) or None.
    h0: [E][N] or None. bcdt_eps: when given, delta, B and C are each divided by their
    RMS (Falcon-Mamba) before use. Returns (y rows [L][dm], new conv_hist [E][K-1], h [E][N]).
    """
    E = len(w["conv_b"])
    K = len(w["conv_w"][0])
    N = len(w["A_log"][0])
    R = len(w["W_dt"][0])
    dm = len(w["W_out"])
    hist = [[0.0] * (K - 1) for _ in range(E)] if conv_hist is None else [list(map(float, r)) for r in conv_hist]
    h = [[0.0] * N for _ in range(E)] if h0 is None else [list(map(float, r)) for r in h0]
    A = [[-math.exp(float(w["A_log"][c][n])) for n in range(N)] for c in range(E)]
    ys = []
    for x in x_rows:
        # input projection: channel c of the SSM path uses row c, gate row E + c
        xs = [sum(float(w["W_in"][c][k]) * float(x[k]) for k in range(dm)) for c in range(E)]
        zs = [sum(float(w["W_in"][E + c][k]) * float(x[k]) for k in range(dm)) for c in range(E)]
        # causal convolution over the window [hist..., current], tap K-1 on the current token
        u = []
        for c in range(E):
            window = hist[c] + [xs[c]]
            acc = float(w["conv_b"][c])
            for j in range(K):
                acc += float(w["conv_w"][c][j]) * window[j]
            u.append(_silu(acc))
            hist[c] = window[1:]
        # packed token fields
        W = R + 2 * N
        dbl = [sum(float(w["W_x"][r][c]) * u[c] for c in range(E)) for r in range(W)]
        delta_lr, Bt, Ct = dbl[:R], dbl[R:R + N], dbl[R + N:]
        if bcdt_eps is not None:
            delta_lr, Bt, Ct = (_rms_scaled(delta_lr, bcdt_eps), _rms_scaled(Bt, bcdt_eps), _rms_scaled(Ct, bcdt_eps))
        y_inner = []
        for c in range(E):
            dtc = sum(float(w["W_dt"][c][r]) * delta_lr[r] for r in range(R))
            D_step = _softplus(dtc + float(w["b_dt"][c]))
            acc = 0.0
            for n in range(N):
                h[c][n] = math.exp(D_step * A[c][n]) * h[c][n] + D_step * Bt[n] * u[c]
                acc += Ct[n] * h[c][n]
            acc += float(w["D"][c]) * u[c]
            y_inner.append(acc * _silu(zs[c]))
        ys.append([sum(float(w["W_out"][m][c]) * y_inner[c] for c in range(E)) for m in range(dm)])
    return ys, hist, h


def stack_sequence(layers, norm_ws, final_w, x_rows: Sequence[Sequence[float]], eps: float,
                   bcdt_eps: Optional[float] = None):
    """One fresh sequence through a stack of full-width layers with pre-norm residual
    blocks: h = RMSNorm_l(resid) * w_l, resid += mixer_l(h), output RMSNorm_final(resid)."""
    resid = [[float(v) for v in r] for r in x_rows]
    for w, nw in zip(layers, norm_ws):
        h = [_rms_scaled(r, eps, nw) for r in resid]
        ys, _, _ = mixer_sequence(w, h, bcdt_eps=bcdt_eps)
        resid = [[a + b for a, b in zip(r, y)] for r, y in zip(resid, ys)]
    return [_rms_scaled(r, eps, final_w) for r in resid]


def mamba2_sequence(w, nheads: int, headdim: int, d_state: int, ngroups: int, x_rows: Sequence[Sequence[float]],
                    eps: float = 1e-5):
    """One fresh sequence through a full-width Mamba-2 mixer, token by token, with scalar
    loops: packed [z | x | B | C | dt] projection, causal K-tap conv + SiLU over [x | B | C],
    Delta = softplus(dt + dt_bias) per head, per head h <- exp(Delta*A) h + Delta*x B^T,
    y = h C + D x, g = y*SiLU(z), RMS normalisation over groups of d_inner/ngroups
    channels times norm_w, output projection. Returns (outputs, final states [h][p][n])."""
    H, Pd, N, G = nheads, headdim, d_state, ngroups
    E = H * Pd
    Cc = E + 2 * G * N
    W_in = [_row(w["W_in"], i) for i in range(len(w["W_in"]))]
    K = len(w["conv_w"][0])
    conv_w = [_row(w["conv_w"], c) for c in range(Cc)]
    conv_b = [float(v) for v in w["conv_b"]]
    A = [-math.exp(float(v)) for v in w["A_log"]]
    D = [float(v) for v in w["D"]]
    dtb = [float(v) for v in w["dt_bias"]]
    nw = [float(v) for v in w["norm_w"]]
    W_out = [_row(w["W_out"], i) for i in range(len(w["W_out"]))]
    hist = [[0.0] * Cc for _ in range(K - 1)]
    h = [[[0.0] * N for _ in range(Pd)] for _ in range(H)]
    outs = []
    for xr in x_rows:
        xr = [float(v) for v in xr]
        proj = [sum(W_in[i][j] * xr[j] for j in range(len(xr))) for i in range(len(W_in))]
        z = proj[:E]
        xbc = proj[E:E + Cc]
        dt = proj[E + Cc:E + Cc + H]
        window = hist + [xbc]
        u = []
        for c in range(Cc):
            a = conv_b[c]
            for j in range(K):
                a += conv_w[c][j] * window[j][c]
            u.append(_silu(a))
        hist = window[1:]
        xs = u[:E]
        Bv = u[E:E + G * N]
        Cv = u[E + G * N:E + 2 * G * N]
        y = [0.0] * E
        for hh in range(H):
            grp = hh // (H // G)
            delta = _softplus(dt[hh] + dtb[hh])
            decay = math.exp(delta * A[hh])
            for p in range(Pd):
                xv = xs[hh * Pd + p]
                acc = 0.0
                for n in range(N):
                    h[hh][p][n] = decay * h[hh][p][n] + delta * xv * Bv[grp * N + n]
                    acc += h[hh][p][n] * Cv[grp * N + n]
                y[hh * Pd + p] = acc + D[hh] * xv
        g = [y[c] * _silu(z[c]) for c in range(E)]
        gs = E // G
        gn = [0.0] * E
        for k in range(G):
            ms = sum(g[c] * g[c] for c in range(k * gs, (k + 1) * gs)) / gs
            for c in range(k * gs, (k + 1) * gs):
                gn[c] = g[c] / math.sqrt(ms + eps) * nw[c]
        outs.append([sum(W_out[i][c] * gn[c] for c in range(E)) for i in range(len(W_out))])
    return outs, h
