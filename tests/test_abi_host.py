"""Host-side checks of the C ABI (no GPU): the library loads, exports every function the
header declares, and rejects bad arguments before anything reaches a stream."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssm_shard.h")


@pytest.fixture(scope="module")
def B():
    from paper_2602_21144_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2602_21144_amd import build
        build.build()
    binding.lib()
    return binding


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(ssm2?_\w+)\(", src, flags=re.M)))


def test_exports_every_declared_function(B):
    names = _declared()
    assert len(names) >= 20
    L = ctypes.CDLL(B.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(B._SIGS), "binding signatures cover the header exactly"
    assert B.lib().ssm_shard_abi_version() == 1


def _desc(B, **kw):
    base = dict(d_model=2560, d_inner_total=5120, d_inner_shard=2560, d_state=16, dt_rank=160, d_conv=4,
                shard_index=0, shard_count=2, act_dtype=B.SSM_BF16)
    base.update(kw)
    return B.Desc(**base)


@pytest.mark.parametrize("bad", [
    dict(d_model=100), dict(d_inner_shard=2500, d_inner_total=5000), dict(shard_index=2), dict(d_state=8),
    dict(dt_rank=150), dict(d_conv=5), dict(d_conv=0), dict(act_dtype=7), dict(d_inner_total=5121)])
def test_descriptor_rejections(B, bad):
    rc = B.lib().ssm_shard_check_desc(ctypes.byref(_desc(B, **bad)))
    assert rc == -1
    assert B.lib().ssm_last_error()


def test_descriptor_ok(B):
    assert B.lib().ssm_shard_check_desc(ctypes.byref(_desc(B))) == 0


def _meta_rc(B, cu, sl, hi, T, S):
    cu = np.array(cu, np.int32)
    sl = np.array(sl, np.int32)
    hi = np.array(hi, np.int32)
    return B.lib().ssm_shard_check_meta_host(cu.ctypes.data, sl.ctypes.data, hi.ctypes.data, len(sl), T, S)


def test_meta_validation(B):
    assert _meta_rc(B, [0, 3, 3, 10], [0, 2, 1], [0, 1, 0], 10, 3) == 0
    assert _meta_rc(B, [1, 3, 10], [0, 1], [0, 0], 10, 3) == -5      # must start at 0
    assert _meta_rc(B, [0, 5, 3], [0, 1], [0, 0], 3, 3) == -5        # decreasing
    assert _meta_rc(B, [0, 3, 9], [0, 1], [0, 0], 10, 3) == -5       # does not end at T
    assert _meta_rc(B, [0, 3, 10], [0, 3], [0, 0], 10, 3) == -4      # slot out of range
    assert _meta_rc(B, [0, 3, 10], [1, 1], [0, 0], 10, 3) == -4      # slot used twice
    assert _meta_rc(B, [0, 3, 10], [0, 1], [0, 2], 10, 3) == -1      # flag not 0/1
    assert _meta_rc(B, [0], [], [], 0, 3) == 0                       # empty batch


def test_workspace_sizes_grow_with_tokens(B):
    d = _desc(B)
    sizes = [B.prefill_workspace_bytes(d, T, 8) for T in (0, 1, 31, 1000, 16384, 65536)]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))
    assert sizes[-2] > 16384 * 2560 * 2 * 5
    assert B.decode_workspace_bytes(d, 256) > B.decode_workspace_bytes(d, 1)


def test_entry_points_reject_before_enqueue(B):
    """Bad arguments return an error code; nothing is launched (there is no GPU here)."""
    L = B.lib()
    d = _desc(B)
    fake = 1 << 20                                    # never dereferenced: checks fail first
    w = B.Weights(*([fake] * 9))
    meta = B.SeqMetaC(fake, fake, fake, 1)
    need = B.prefill_workspace_bytes(d, 100, 1)
    args = lambda ws_bytes, x=fake: (ctypes.byref(d), ctypes.byref(w), ctypes.c_void_p(x), 100, ctypes.byref(meta),
                                     ctypes.c_void_p(fake), ctypes.c_void_p(fake), 4, ctypes.c_void_p(fake),
                                     ctypes.c_void_p(fake), ws_bytes, None)
    assert L.ssm_shard_prefill(*args(need - 1)) == -3                 # workspace too small
    assert L.ssm_shard_prefill(*args(need, x=fake + 2)) == -2         # misaligned input
    assert L.ssm_shard_prefill(*args(need, x=0)) == -1                # null input
    w_bad = B.Weights(*([fake] * 8 + [0]))
    assert L.ssm_shard_prefill(ctypes.byref(d), ctypes.byref(w_bad), *args(need)[2:]) == -1
    assert L.ssm_gemm_nt(4, 4, 12, fake, 16, 1, fake, 16, 1, fake, 4, 1, None) == -2   # K not a multiple of 8
    assert L.ssm_gemm_nt(4, 4, 16, fake, 16, 0, fake, 16, 0, fake, 4, 1, None) == -1   # f32 B needs f32 C
    assert L.ssm_reduce_add_f32(fake + 4, fake, 10, None) == -2
    assert L.ssm_shard_decode_step(ctypes.byref(d), ctypes.byref(w), ctypes.c_void_p(fake), 4, None,
                                   ctypes.c_void_p(fake), ctypes.c_void_p(fake), 4, ctypes.c_void_p(fake),
                                   ctypes.c_void_p(fake), 1 << 30, None) == -1        # null slot array


def test_channel_splitter_layout_matches_oracle_on_host():
    """The library's splitter copies the same row/column ranges the oracle slices; the
    ranges are stated once here as index arithmetic and checked against the oracle."""
    from oracle import mixer as om
    E_tot, P, dm, R, N, K = 12, 3, 4, 2, 2, 4
    full = {"W_in": np.arange(2 * E_tot * dm).reshape(2 * E_tot, dm), "conv_w": np.arange(E_tot * K).reshape(E_tot, K),
            "conv_b": np.arange(E_tot), "W_x": np.arange((R + 2 * N) * E_tot).reshape(R + 2 * N, E_tot),
            "W_dt": np.arange(E_tot * R).reshape(E_tot, R), "b_dt": np.arange(E_tot),
            "A_log": np.arange(E_tot * N).reshape(E_tot, N), "D": np.arange(E_tot),
            "W_out": np.arange(dm * E_tot).reshape(dm, E_tot)}
    E = E_tot // P
    for r in range(P):
        s = om.shard_weights(full, r, P)
        rows = list(range(r * E, (r + 1) * E)) + list(range(E_tot + r * E, E_tot + (r + 1) * E))
        assert np.array_equal(s["W_in"], full["W_in"][rows])
        assert np.array_equal(s["W_x"], full["W_x"][:, r * E:(r + 1) * E])
        assert np.array_equal(s["W_out"], full["W_out"][:, r * E:(r + 1) * E])


def test_exchange_codec_host_checks(B):
    """Payload sizes follow the documented layout; bad arguments fail before any launch."""
    L = B.lib()
    n = ctypes.c_size_t()
    assert L.ssm_exchange_payload_bytes(0, 16384, 192, ctypes.byref(n)) == 0 and n.value == 16384 * 192 * 2
    assert L.ssm_exchange_payload_bytes(1, 3, 8, ctypes.byref(n)) == 0 and n.value == 48
    # scaled codecs: fp32 scales padded to 256 bytes, then one byte per value
    assert L.ssm_exchange_payload_bytes(2, 100, 2560, ctypes.byref(n)) == 0 and n.value == 512 + 100 * 2560
    assert L.ssm_exchange_payload_bytes(3, 64, 16, ctypes.byref(n)) == 0 and n.value == 256 + 64 * 16
    assert L.ssm_exchange_payload_bytes(4, 1, 8, ctypes.byref(n)) == -1           # unknown codec
    assert L.ssm_exchange_payload_bytes(0, 1, 12, ctypes.byref(n)) == -2          # cols not a multiple of 8
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: every call below fails its host checks first
    assert L.ssm_exchange_encode(0, None, 0, 4, 8, 8, fake, 4096, None) == -1     # null source
    assert L.ssm_exchange_encode(0, fake, 2, 4, 8, 8, fake, 4096, None) == -1     # bad source dtype
    assert L.ssm_exchange_encode(2, fake, 0, 4, 8, 4, fake, 4096, None) == -1     # ld < cols
    assert L.ssm_exchange_encode(2, fake, 0, 4, 8, 12, fake, 4096, None) == -2    # ld not a multiple of 8
    assert L.ssm_exchange_encode(2, fake, 0, 4, 8, 8, fake, 100, None) == -3      # payload too small
    assert L.ssm_exchange_decode_accumulate(3, fake, 100, 4, 8, fake, 8, 0, None) == -3
    assert L.ssm_exchange_decode_accumulate(3, fake, 4096, 4, 8, None, 8, 0, None) == -1
    assert L.ssm_exchange_encode(1, fake, 0, 0, 8, 8, None, 0, None) == 0         # empty: nothing to do


def test_layer_and_stack_host_checks(B):
    """The residual norm, the Falcon-Mamba norms and the stack calls reject bad arguments
    before any launch; workspace sizes cover the layer's and the stack's buffers."""
    L = B.lib()
    fake = 1 << 20   # never dereferenced: every call below fails its host checks first
    f = ctypes.c_void_p(fake)
    parts = (ctypes.c_void_p * 2)(fake, fake + (1 << 24))
    norm = lambda base, bdt, n, pdt, res, d, T=4, eps=1e-5, odt=1: L.ssm_residual_rmsnorm(
        ctypes.c_void_p(base), bdt, parts, n, pdt, ctypes.c_void_p(res), f, ctypes.c_float(eps), f, odt, T, d, None)
    assert norm(fake, 0, 1, 1, fake, 12) == -1                 # d not a multiple of 8
    assert norm(fake, 0, 1, 1, fake, 8200) == -1               # d above 8192
    assert norm(fake, 0, 9, 1, fake, 16) == -1                 # more than 8 parts
    assert norm(fake, 3, 1, 1, fake, 16) == -1                 # bad base dtype
    assert norm(fake, 0, 1, 1, fake, 16, eps=0.0) == -1        # eps must be positive
    assert norm(fake, 0, 1, 1, fake + 64, 16) == -1            # base overlaps residual partially
    assert norm(fake + 4, 0, 1, 1, fake + 4096, 16) == -2      # misaligned base
    assert norm(fake, 0, 1, 1, fake, 16, T=0) == 0             # no rows: nothing to do
    assert L.ssm_bcdt_rmsnorm(f, 10, 8, 4, 15, ctypes.c_float(1e-6), None) == -1   # ld < R + 2N
    assert L.ssm_bcdt_rmsnorm(f, 10, 8, 4, 16, ctypes.c_float(0.0), None) == -1    # eps
    assert L.ssm_bcdt_rmsnorm(None, 10, 8, 4, 16, ctypes.c_float(1e-6), None) == -1
    d1 = _desc(B, d_inner_shard=5120, shard_count=1)
    sd = B.StackDesc(d1, 2, 1e-5, 0.0)
    n1, n2 = ctypes.c_size_t(), ctypes.c_size_t()
    assert L.ssm_stack_prefill_workspace_bytes(ctypes.byref(sd), 1000, 2, ctypes.byref(n1)) == 0
    assert n1.value >= B.prefill_workspace_bytes(d1, 1000, 2) + 1000 * 2560 * 8
    assert L.ssm_stack_decode_workspace_bytes(ctypes.byref(sd), 8, ctypes.byref(n2)) == 0
    w = (B.Weights * 2)(*[B.Weights(*([fake] * 9)) for _ in range(2)])
    nw = (ctypes.c_void_p * 2)(fake, fake)
    pools = (ctypes.c_void_p * 2)(fake, fake)
    meta = B.SeqMetaC(fake, fake, fake, 1)
    call = lambda sdesc, ws_bytes: L.ssm_stack_prefill(ctypes.byref(sdesc), w, nw, f, f, 100, ctypes.byref(meta),
                                                       pools, pools, 4, f, f, ws_bytes, None)
    assert call(B.StackDesc(_desc(B), 2, 1e-5, 0.0), 1 << 40) == -1         # split layers: not a stack
    assert call(B.StackDesc(d1, 0, 1e-5, 0.0), 1 << 40) == -1               # no layers
    assert call(B.StackDesc(d1, 2, 0.0, 0.0), 1 << 40) == -1                # norm eps
    assert call(B.StackDesc(d1, 2, 1e-5, -1.0), 1 << 40) == -1              # bcdt eps
    need = ctypes.c_size_t()
    L.ssm_stack_prefill_workspace_bytes(ctypes.byref(sd), 100, 1, ctypes.byref(need))
    assert call(sd, need.value - 1) == -3                                   # workspace too small


def test_timing_switch_arguments(B):
    """Kernel timing: 0 turns it off, k >= 1 samples every k-th launch, negative is rejected;
    collecting with nothing recorded returns no entries."""
    L = B.lib()
    assert L.ssm_timing_enable(-1, None) == -1
    assert L.ssm_timing_enable(4, b"decode.in_proj_conv") == 0
    assert L.ssm_timing_enable(0, None) == 0
    assert B.ssm_timing_collect() == {}
