"""Kernel-level parity on the GPU: each stage operator of the C ABI against the oracle's
stage function on the same seeded inputs (drawn on the host, never computed on the GPU).
"""
import numpy as np
import pytest

from mixer_cases import TOL, assert_close, f64, poison_like
from oracle import mixer as om
from paper_2602_21144_amd import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def B():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_21144_amd import binding
    binding.lib()
    return binding


def _rnd_host(rng, shape, act, scale=1.0):
    a = (rng.normal(size=shape) * scale).astype(np.float32)
    return synth.round_bf16_f32(a) if act == "bf16" else a


def _dev(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to("cuda", dt)


# ----------------------------------------------------------------------- GEMM
GEMM_SHAPES = [(1, 64, 16), (7, 130, 48), (300, 200, 32), (33, 200, 160), (64, 96, 224), (100, 300, 256), (257, 513, 64),
               (1000, 520, 768), (2048, 2048, 512), (300, 5120, 2560), (4089, 4091, 256), (200, 300, 96),
               # few rows with K a multiple of 64 (streamed-weight decode kernel: small grid of 16-wave
               # workgroups; large grids of 8 waves of up to 5 stages, 8 waves of up to 10 stages, and
               # 4 waves for K up to 1280, including waves left without a stage; 9..16 rows)
               (1, 200, 128), (5, 100, 640), (8, 5120, 2560), (16, 192, 2560), (13, 3000, 4096),
               (12, 2080, 1344), (9, 2100, 1280), (3, 4096, 64),
               # 17..64 rows over at least 192 tiles of 32 columns (32-column fragment kernel: 32- and
               # 64-row tiles, ragged N, a K tail of 8)
               (17, 6150, 512), (40, 6176, 808), (64, 7168, 1024),
               # decode batches of 17..512 rows, bf16 output, at least 128 tiles: the streamed tile
               # kernel (64x64 tiles above 128 rows, 64x32, 32x32; ragged last row and column tiles,
               # waves without a stage at K = 64); other outputs on the DMA tiles
               (256, 2560, 2560), (130, 8192, 1280), (500, 1100, 640), (17, 4104, 64), (33, 4096, 1344),
               (100, 4104, 2560), (129, 2560, 1280), (200, 4104, 3584), (511, 2568, 640), (40, 2560, 640),
               (60, 3584, 3584), (40, 4104, 640),
               # bf16 256x320 tiles (N a multiple of 320 whose 256-wide tiles would take an extra
               # round; ragged last row tile)
               (8000, 2560, 320),
               # bf16 256x256 tiles over two rounds (ragged last row and column tiles, three k-tiles)
               (8000, 4000, 192),
               # float32 at prefill sizes, by the tile model: 128x128 (2000 x 3588), 128x224 (1500 x 4100,
               # 1200 x 3500), 256x256 (2000 x 7900), 256x224 (2048 x 7168); ragged M and N, K of 96 to 3584
               (2000, 3588, 224), (1500, 4100, 96), (1200, 3500, 352), (2000, 7900, 256), (2048, 7168, 3584)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("kind", ["bf16_bf16", "bf16_f32", "f32a_bf16", "f32"])
def test_gemm_nt(B, M, N, K, kind):
    rng = np.random.default_rng(M * 7 + N * 3 + K)
    a_act = "f32" if kind in ("f32a_bf16", "f32") else "bf16"
    b_act = "f32" if kind == "f32" else "bf16"
    A = _rnd_host(rng, (M, K), a_act)
    Bm = _rnd_host(rng, (N, K), b_act, 1.0 / np.sqrt(K))
    c_dt = torch.float32 if kind in ("bf16_f32", "f32") else torch.bfloat16
    # ragged N: the output row stride is padded to a multiple of 4 and C is a view
    Cpad = torch.full((M, (N + 3) // 4 * 4), float("nan"), dtype=c_dt, device="cuda")
    C = Cpad[:, :N]
    B.ssm_gemm_nt(_dev(A, torch.float32 if a_act == "f32" else torch.bfloat16),
                  _dev(Bm, torch.float32 if b_act == "f32" else torch.bfloat16), C)
    torch.cuda.synchronize()
    A64 = A.astype(np.float64)
    if kind == "f32a_bf16":      # A is rounded to bf16 as it is loaded (dt_proj's input)
        A64 = om.round_bf16(A64)
    ref = A64 @ Bm.astype(np.float64).T
    if c_dt == torch.bfloat16:
        ref = om.round_bf16(ref)
    got = C.to(torch.float64).cpu().numpy()
    tol = 1e-5 if c_dt == torch.float32 else 8e-3
    assert_close(got, ref, tol, f"gemm {kind} {M}x{N}x{K}")


@pytest.mark.parametrize("M,N,K", [(16384, 2560, 128), (16140, 2560, 192)])
def test_gemm_wide_tiles(B, M, N, K):
    """Outputs whose 256-wide tiles would leave the last round of CUs part-empty take
    256x320 tiles when N is a multiple of 320 (the 2.8B half shard's out_proj is
    16384 x 2560); ragged M included. Rows sampled across every tile row."""
    rng = np.random.default_rng(M + K)
    A = _rnd_host(rng, (M, K), "bf16")
    Bm = _rnd_host(rng, (N, K), "bf16", 1.0 / np.sqrt(K))
    C = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    B.ssm_gemm_nt(_dev(A, torch.bfloat16), _dev(Bm, torch.bfloat16), C)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, M, 97), np.arange(M - 40, M)]))
    ref = om.round_bf16(A[rows].astype(np.float64) @ Bm.astype(np.float64).T)
    got = C[torch.from_numpy(rows).cuda()].to(torch.float64).cpu().numpy()
    assert_close(got, ref, 8e-3, f"gemm {M}x{N}x{K}")


SPLITK_SHAPES = [("out_proj", 600, 2560, 5120, False), ("in_proj", 600, 3000, 2560, False),
                 ("x_proj", 1000, 192, 5120, True), ("x_proj", 2048, 256, 3584, True), ("in_proj", 600, 2000, 2560, False),
                 ("out_proj", 700, 3584, 3584, False), ("generic", 129, 130, 1024, False), ("x_proj", 600, 80, 1536, True)]


@pytest.mark.parametrize("role,M,N,K,c_f32", SPLITK_SHAPES)
def test_gemm_split_k(B, role, M, N, K, c_f32):
    """Few output tiles and a long K: the product is cut into K-slices whose partials a
    second kernel adds; the result matches the float64 product and the unsplit run."""
    need = B.gemm_splitk_bytes(M, N, K, B.SSM_BF16, B.SSM_BF16, role)
    assert need > 0, "this shape is expected to run split-K"
    rng = np.random.default_rng(M + N + K)
    A = _rnd_host(rng, (M, K), "bf16")
    Bm = _rnd_host(rng, (N, K), "bf16", 1.0 / np.sqrt(K))
    c_dt = torch.float32 if c_f32 else torch.bfloat16
    Ad, Bd = _dev(A, torch.bfloat16), _dev(Bm, torch.bfloat16)
    scratch = torch.full((need // 4,), float("nan"), dtype=torch.float32, device="cuda")
    Np = (N + 3) // 4 * 4   # output rows padded to a multiple of 4 values; C is a view
    C = torch.full((M, Np), float("nan"), dtype=c_dt, device="cuda")[:, :N]
    B.ssm_gemm_nt_role(Ad, Bd, C, role, scratch)
    C1 = torch.full((M, Np), float("nan"), dtype=c_dt, device="cuda")[:, :N]
    B.ssm_gemm_nt_role(Ad, Bd, C1, role, None)          # no scratch: unsplit
    torch.cuda.synchronize()
    ref = A.astype(np.float64) @ Bm.astype(np.float64).T
    if not c_f32:
        ref = om.round_bf16(ref)
    tol = 1e-5 if c_f32 else 8e-3
    assert_close(C.to(torch.float64).cpu().numpy(), ref, tol, f"split-K {role} {M}x{N}x{K}")
    assert_close(C1.to(torch.float64).cpu().numpy(), ref, tol, f"unsplit {role} {M}x{N}x{K}")


@pytest.mark.parametrize("M,N,K", [(65, 192, 1280), (256, 192, 1280), (511, 256, 3584), (300, 80, 1536)])
def test_gemm_x_proj_decode_rows(B, M, N, K):
    """x_proj of a decode batch of 65..512 rows runs on 16-row tiles of the few-row kernel
    (no K-slices, no scratch needed); bf16 operands, float32 output."""
    assert B.gemm_splitk_bytes(M, N, K, B.SSM_BF16, B.SSM_BF16, "x_proj") == 0
    rng = np.random.default_rng(M + N + K)
    A = _rnd_host(rng, (M, K), "bf16")
    Bm = _rnd_host(rng, (N, K), "bf16", 1.0 / np.sqrt(K))
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    B.ssm_gemm_nt_role(_dev(A, torch.bfloat16), _dev(Bm, torch.bfloat16), C, "x_proj", None)
    torch.cuda.synchronize()
    ref = A.astype(np.float64) @ Bm.astype(np.float64).T
    assert_close(C.to(torch.float64).cpu().numpy(), ref, 1e-5, f"x_proj {M}x{N}x{K}")


F32_SPLITK_SHAPES = [("x_proj", 2048, 256, 3584), ("x_proj", 2000, 256, 3584), ("in_proj", 256, 3072, 768),
                     ("out_proj", 300, 770, 1536), ("generic", 129, 130, 1024)]


@pytest.mark.parametrize("role,M,N,K", F32_SPLITK_SHAPES)
def test_gemm_split_k_f32(B, role, M, N, K):
    """Float32 operands with few 128x128 tiles: K-slices on the tile kernel, their partials
    added by the reduce kernel (ragged M and N included); matches the float64 product and
    the unsplit run (64x64 tiles) to float32 accuracy."""
    need = B.gemm_splitk_bytes(M, N, K, B.SSM_F32, B.SSM_F32, role)
    assert need > 0, "this shape is expected to run split-K"
    rng = np.random.default_rng(M + 3 * N + K)
    A = _rnd_host(rng, (M, K), "f32")
    Bm = _rnd_host(rng, (N, K), "f32", 1.0 / np.sqrt(K))
    Ad, Bd = _dev(A, torch.float32), _dev(Bm, torch.float32)
    scratch = torch.full((need // 4,), float("nan"), dtype=torch.float32, device="cuda")
    Np = (N + 3) // 4 * 4
    C = torch.full((M, Np), float("nan"), dtype=torch.float32, device="cuda")[:, :N]
    B.ssm_gemm_nt_role(Ad, Bd, C, role, scratch)
    C1 = torch.full((M, Np), float("nan"), dtype=torch.float32, device="cuda")[:, :N]
    B.ssm_gemm_nt_role(Ad, Bd, C1, role, None)
    torch.cuda.synchronize()
    ref = A.astype(np.float64) @ Bm.astype(np.float64).T
    assert_close(C.to(torch.float64).cpu().numpy(), ref, 1e-5, f"split-K f32 {role} {M}x{N}x{K}")
    assert_close(C1.to(torch.float64).cpu().numpy(), ref, 1e-5, f"unsplit f32 {role} {M}x{N}x{K}")


def test_gemm_strided_operands(B):
    """dt_proj reads the first R columns of x_dbl (row stride R+2N) as its A operand."""
    rng = np.random.default_rng(5)
    T, R, N, E = 77, 48, 16, 192
    xdbl = rng.normal(size=(T, R + 2 * N)).astype(np.float32)
    W = synth.round_bf16_f32((rng.normal(size=(E, R)) / np.sqrt(R)).astype(np.float32))
    xd = _dev(xdbl, torch.float32)
    C = torch.empty(T, E, dtype=torch.bfloat16, device="cuda")
    B.ssm_gemm_nt(xd[:, :R], _dev(W, torch.bfloat16), C)
    torch.cuda.synchronize()
    ref = om.round_bf16(om.round_bf16(xdbl.astype(np.float64)[:, :R]) @ W.astype(np.float64).T)
    assert_close(C.to(torch.float64).cpu().numpy(), ref, 8e-3, "strided dt_proj")


# ------------------------------------------------------------------ conv1d
def _meta_case(rng, lens, S, init_frac=0.5):
    nseq = len(lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    slots = rng.permutation(S)[:nseq].astype(np.int32)
    hi = (rng.random(nseq) < init_frac).astype(np.int32)
    return cu, slots, hi


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("K", [4, 3, 2])
def test_conv1d_silu_prefill(B, act, K):
    rng = np.random.default_rng(11 + K)
    shape = synth.LayerShape(64, 128, 16, 16, K, 1, act)
    E = shape.d_shard
    lens = [5, 1, 0, 40, 2, 17, 1, 3]
    S = len(lens) + 4
    cu, slots, hi = _meta_case(rng, lens, S)
    hi[0], hi[1], hi[4] = 1, 1, 1      # short continuing pieces (fewer than K-1 tokens)
    T = int(cu[-1])
    xz = _rnd_host(rng, (T, 2 * E), act)
    w = f64(synth.make_general_layer(shape, 3))
    pool0 = _rnd_host(rng, (S, E, K - 1), act)
    dt_act = torch.float32 if act == "f32" else torch.bfloat16
    dw = B.upload_weights(synth.make_general_layer(shape, 3), act)
    d = B.make_desc(shape)
    meta = B.SeqMeta(cu, slots, hi, S)
    pool = _dev(pool0, dt_act)
    untouched = [s for s in range(S) if s not in set(slots.tolist())]
    for s in untouched:
        poison_like(pool[s])
    u = torch.full((T, E), float("nan"), dtype=dt_act, device="cuda")
    ws = B.workspace(4096)
    B.ssm_conv1d_silu(d, dw, _dev(xz, dt_act), meta, pool, u, ws)
    assert B.take_status(ws) == 0
    got_u = u.to(torch.float64).cpu().numpy()
    got_pool = pool.to(torch.float64).cpu().numpy()
    for i in range(len(lens)):
        a, b = cu[i], cu[i + 1]
        s = slots[i]
        ref_u, ref_st = om.conv1d_silu(w, xz[a:b, :E].astype(np.float64),
                                       pool0[s].astype(np.float64) if hi[i] else None, act)
        if b > a:
            assert_close(got_u[a:b], ref_u, TOL[act], f"u of sequence {i}")
        # the new history is a copy of inputs: bit-exact
        assert np.array_equal(got_pool[s], ref_st), f"history of sequence {i}"
    raw = pool.view(torch.int16 if act == "bf16" else torch.int32).cpu().numpy()
    for s in untouched:
        assert np.all(raw[s] == (0x7FC1 if act == "bf16" else 0x7FC0DEAD)), f"slot {s} was touched"


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_conv_decode(B, act):
    rng = np.random.default_rng(21)
    shape = synth.LayerShape(64, 192, 16, 16, 4, 1, act)
    E, K = shape.d_shard, 4
    S, Bd = 12, 5
    slots = np.array([3, 0, 11, 7, 5], np.int32)
    xz = _rnd_host(rng, (Bd, 2 * E), act)
    pool0 = _rnd_host(rng, (S, E, K - 1), act)
    hw = synth.make_general_layer(shape, 4)
    w = f64(hw)
    dt_act = torch.float32 if act == "f32" else torch.bfloat16
    d = B.make_desc(shape)
    pool = _dev(pool0, dt_act)
    u = torch.empty(Bd, E, dtype=dt_act, device="cuda")
    ws = B.workspace(4096)
    sl = torch.from_numpy(slots).cuda()
    B.ssm_decode_conv(d, B.upload_weights(hw, act), _dev(xz, dt_act), sl, pool, u, ws)
    assert B.take_status(ws) == 0
    gu = u.to(torch.float64).cpu().numpy()
    gp = pool.to(torch.float64).cpu().numpy()
    for i in range(Bd):
        s = slots[i]
        win = np.concatenate([pool0[s].astype(np.float64), xz[i, :E, None].astype(np.float64)], axis=1)
        ref = om.rnd(om.silu(w["conv_b"] + np.sum(w["conv_w"] * win, axis=1)), act)
        assert_close(gu[i], ref, TOL[act], f"decode u {i}")
        assert np.array_equal(gp[s], win[:, 1:]), "shifted window"
    for s in set(range(S)) - set(slots.tolist()):
        assert np.array_equal(gp[s], pool0[s].astype(np.float64))


# -------------------------------------------------------------------- scan
def _scan_inputs(rng, T, E, R, act, stress=False):
    N = 16
    u = _rnd_host(rng, (T, E), act)
    dt = _rnd_host(rng, (T, E), act, 0.7)
    xz = _rnd_host(rng, (T, 2 * E), act)
    xdbl = rng.normal(size=(T, R + 2 * N)).astype(np.float32)
    return u, dt, xz, xdbl


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("E", [128, 512])
# the last case: 200 sequences of 0..4 tokens, so that most 8-token blocks hold several
# sequence ends (the main pass's per-token path) and windows hold dozens of sequences
@pytest.mark.parametrize("lens", [[70, 1, 0, 33, 100, 31, 65], [300], [1, 2, 3, 31, 32, 33, 64, 65, 0, 5],
                                  [7, 0, 0, 9, 1], [int(v) for v in np.random.default_rng(9).integers(0, 5, 200)]])
def test_selective_scan(B, act, E, lens):
    rng = np.random.default_rng(sum(lens) + len(lens) + E)
    shape = synth.LayerShape(64, E, 16, 16, 4, 1, act)
    E, N, R = shape.d_shard, 16, 16
    S = len(lens) + 3
    cu, slots, hi = _meta_case(rng, lens, S)
    T = int(cu[-1])
    u, dt, xz, xdbl = _scan_inputs(rng, T, E, R, act)
    hw = synth.make_general_layer(shape, 8)
    w = f64(hw)
    pool0 = rng.normal(size=(S, E, N)).astype(np.float32)
    dt_act = torch.float32 if act == "f32" else torch.bfloat16
    d = B.make_desc(shape)
    meta = B.SeqMeta(cu, slots, hi, S)
    pool = torch.from_numpy(pool0).cuda()
    untouched = [s for s in range(S) if s not in set(slots.tolist())]
    for s in untouched:
        poison_like(pool[s])
    g = torch.full((max(T, 1), E), float("nan"), dtype=dt_act, device="cuda")
    ws = B.workspace(B.scan_scratch_workspace_bytes(d, T, len(lens)))
    B.ssm_selective_scan(d, B.upload_weights(hw, act), _dev(u, dt_act), _dev(dt, dt_act), _dev(xz, dt_act),
                         torch.from_numpy(xdbl).cuda(), meta, pool, g, ws)
    assert B.take_status(ws) == 0
    gg = g.to(torch.float64).cpu().numpy()
    gp = pool.to(torch.float64).cpu().numpy()
    Bm, Cm = xdbl[:, R:R + N].astype(np.float64), xdbl[:, R + N:].astype(np.float64)
    for i in range(len(lens)):
        a, b = cu[i], cu[i + 1]
        s = slots[i]
        h0 = pool0[s].astype(np.float64) if hi[i] else np.zeros((E, N))
        ref_g, ref_h = om.selective_scan(w, u[a:b].astype(np.float64), dt[a:b].astype(np.float64),
                                         xz[a:b, E:].astype(np.float64), Bm[a:b], Cm[a:b], h0, act)
        if b > a:
            assert_close(gg[a:b], ref_g, TOL[act], f"g of sequence {i} (len {b - a})")
        assert_close(gp[s], ref_h, 2e-5 if act == "f32" else 1e-4, f"state of sequence {i} (len {b - a})")
    raw = pool.view(torch.int32).cpu().numpy()
    for s in untouched:
        assert np.all(raw[s] == 0x7FC0DEAD), f"slot {s} was touched"


@pytest.mark.parametrize("act", ["f32", "bf16"])
@pytest.mark.parametrize("T", [3333, 9001])
def test_selective_scan_long_sequence_many_windows(B, act, T):
    """One long sequence crossing ~100 (~280) windows: exercises the window-to-window state
    links, with each of the link pass's ranges one (several, the last ragged) fetch batches long."""
    rng = np.random.default_rng(99 + T)
    shape = synth.LayerShape(64, 64, 16, 16, 4, 1, act)
    E, N, R = 64, 16, 16
    u, dt, xz, xdbl = _scan_inputs(rng, T, E, R, act)
    dt = (dt - 2.0).astype(np.float32)        # small steps: long memory across windows
    if act == "bf16":
        dt = synth.round_bf16_f32(dt)
    hw = synth.make_general_layer(shape, 9)
    w = f64(hw)
    dt_act = torch.float32 if act == "f32" else torch.bfloat16
    d = B.make_desc(shape)
    meta = B.SeqMeta([0, T], [1], [1], 2)
    pool0 = rng.normal(size=(2, E, N)).astype(np.float32)
    pool = torch.from_numpy(pool0).cuda()
    g = torch.empty(T, E, dtype=dt_act, device="cuda")
    ws = B.workspace(B.scan_scratch_workspace_bytes(d, T, 1))
    B.ssm_selective_scan(d, B.upload_weights(hw, act), _dev(u, dt_act), _dev(dt, dt_act), _dev(xz, dt_act),
                         torch.from_numpy(xdbl).cuda(), meta, pool, g, ws)
    assert B.take_status(ws) == 0
    ref_g, ref_h = om.selective_scan(w, u.astype(np.float64), dt.astype(np.float64), xz[:, E:].astype(np.float64),
                                     xdbl[:, R:R + N].astype(np.float64), xdbl[:, R + N:].astype(np.float64),
                                     pool0[1].astype(np.float64), act)
    assert_close(g.to(torch.float64).cpu().numpy(), ref_g, TOL[act], "g")
    assert_close(pool[1].to(torch.float64).cpu().numpy(), ref_h, 2e-5 if act == "f32" else 1e-4, "state")
    assert np.array_equal(pool[0].cpu().numpy(), pool0[0])


@pytest.mark.parametrize("act", ["f32", "bf16"])
def test_decode_ssm(B, act):
    rng = np.random.default_rng(31)
    shape = synth.LayerShape(64, 128, 16, 16, 4, 1, act)
    E, N, R = 128, 16, 16
    S, Bd = 9, 4
    slots = np.array([8, 2, 0, 5], np.int32)
    u, dt, xz, xdbl = _scan_inputs(rng, Bd, E, R, act)
    hw = synth.make_general_layer(shape, 12)
    w = f64(hw)
    pool0 = rng.normal(size=(S, E, N)).astype(np.float32)
    dt_act = torch.float32 if act == "f32" else torch.bfloat16
    d = B.make_desc(shape)
    pool = torch.from_numpy(pool0).cuda()
    g = torch.empty(Bd, E, dtype=dt_act, device="cuda")
    ws = B.workspace(4096)
    B.ssm_decode_ssm(d, B.upload_weights(hw, act), _dev(u, dt_act), _dev(dt, dt_act), _dev(xz, dt_act),
                     torch.from_numpy(xdbl).cuda(), torch.from_numpy(slots).cuda(), pool, g, ws)
    assert B.take_status(ws) == 0
    gg = g.to(torch.float64).cpu().numpy()
    gp = pool.cpu().numpy().astype(np.float64)
    for i in range(Bd):
        s = slots[i]
        ref_g, ref_h = om.selective_scan(w, u[i:i + 1].astype(np.float64), dt[i:i + 1].astype(np.float64),
                                         xz[i:i + 1, E:].astype(np.float64), xdbl[i:i + 1, R:R + N].astype(np.float64),
                                         xdbl[i:i + 1, R + N:].astype(np.float64), pool0[s].astype(np.float64), act)
        assert_close(gg[i], ref_g[0], TOL[act], f"g {i}")
        assert_close(gp[s], ref_h, 1e-5, f"state {i}")
    for s in set(range(S)) - set(slots.tolist()):
        assert np.array_equal(gp[s], pool0[s].astype(np.float64))


def test_bad_device_slot_is_reported_not_followed(B):
    """A slot outside the pool in device metadata: the kernels skip it and flag the status."""
    shape = synth.LayerShape(64, 64, 16, 16, 4, 1, "f32")
    d = B.make_desc(shape)
    hw = synth.make_general_layer(shape, 1)
    S = 3
    pool = torch.zeros(S, 64, 16, device="cuda")
    slots = torch.tensor([1, 7], dtype=torch.int32, device="cuda")
    u = torch.randn(2, 64, device="cuda")
    xz = torch.randn(2, 128, device="cuda")
    xdbl = torch.randn(2, 48, device="cuda")
    g = torch.empty(2, 64, device="cuda")
    ws = B.workspace(4096)
    B.ssm_decode_ssm(d, B.upload_weights(hw, "f32"), u, u, xz, xdbl, slots, pool, g, ws)
    st = B.take_status(ws)
    assert st & B.SSM_STATUS_BAD_SLOT
    assert torch.count_nonzero(pool[0]) == 0 and torch.count_nonzero(pool[2]) == 0
    assert torch.count_nonzero(pool[1]) > 0
    assert B.take_status(ws) == 0   # cleared by the read
