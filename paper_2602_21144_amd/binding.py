"""ctypes binding of ``libssm_shard.so`` (declared in include/ssm_shard.h).

Argument marshalling only: torch tensors supply device memory and the current HIP
stream; every step of the mixer runs in the library's gfx950 kernels. There is no
fallback: if the library is missing, loading it raises.

Function names follow the C ABI; tensors replace pointer + size arguments.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np
import torch

from .synth import LayerShape

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libssm_shard.so")

SSM_F32, SSM_BF16 = 0, 1
SSM_OK = 0
ERRORS = {-1: "SSM_E_INVAL", -2: "SSM_E_ALIGN", -3: "SSM_E_WORKSPACE", -4: "SSM_E_SLOT",
          -5: "SSM_E_SEQLENS", -6: "SSM_E_HIP"}
SSM_STATUS_BAD_SLOT, SSM_STATUS_BAD_SEQLENS = 1, 2
SSM_E_INVAL, SSM_E_ALIGN, SSM_E_WORKSPACE = -1, -2, -3
SSM_NOALLOC_SCRATCH_BYTES = 32 << 20   # the static scratch of ssm_shard_decode_step_noalloc


class SsmError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class Desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "d_model", "d_inner_total", "d_inner_shard", "d_state", "dt_rank", "d_conv",
        "shard_index", "shard_count", "act_dtype")]


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "in_proj_w", "conv_w", "conv_b", "x_proj_w", "dt_proj_w", "out_proj_w",
        "dt_proj_b", "A_log", "D")]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


class SeqMetaC(ctypes.Structure):
    _fields_ = [("cu_seqlens", ctypes.c_void_p), ("cache_slot", ctypes.c_void_p),
                ("has_initial_state", ctypes.c_void_p), ("nseq", ctypes.c_int32)]


class Desc2(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "d_model", "nheads_total", "headdim", "d_state", "ngroups_total", "d_conv", "shard_index", "shard_count",
        "act_dtype")]


class Weights2(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "in_proj_w", "conv_w", "conv_b", "out_proj_w", "dt_bias", "A_log", "D", "norm_w")]


_lib: Optional[ctypes.CDLL] = None
_P, _I32, _I64, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t

_SIGS = {
    "ssm_shard_abi_version": ([], _I32),
    "ssm_last_error": ([], ctypes.c_char_p),
    "ssm_shard_check_desc": ([_P], _I32),
    "ssm_shard_check_meta_host": ([_P, _P, _P, _I32, _I64, _I32], _I32),
    "ssm_shard_prefill_workspace_bytes": ([_P, _I64, _I32, _P], _I32),
    "ssm_shard_decode_workspace_bytes": ([_P, _I32, _P], _I32),
    "ssm_shard_workspace_init": ([_P, _SZ, _P], _I32),
    "ssm_shard_take_status": ([_P, _SZ, _P, _P], _I32),
    "ssm_shard_prefill": ([_P, _P, _P, _I64, _P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_shard_prefill_stage1": ([_P, _P, _P, _I64, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_shard_prefill_stage2": ([_P, _P, _P, _I64, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_shard_decode_step": ([_P, _P, _P, _I32, _P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_shard_decode_step_noalloc": ([_P, _P, _P, _I32, _P, _P, _P, _I32, _P, _P], _I32),
    "ssm_shard_decode_stage1": ([_P, _P, _P, _I32, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_shard_decode_stage2": ([_P, _P, _P, _I32, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_shard_slice_weights": ([_P, _P, _P, _P], _I32),
    "ssm_reduce_add_f32": ([_P, _P, _I64, _P], _I32),
    "ssm_gemm_nt": ([_I64, _I64, _I64, _P, _I64, _I32, _P, _I64, _I32, _P, _I64, _I32, _P], _I32),
    "ssm_gemm_splitk_bytes": ([_I64, _I64, _I64, _I32, _I32, _I32, _P], _I32),
    "ssm_gemm_nt_role": ([_I64, _I64, _I64, _P, _I64, _I32, _P, _I64, _I32, _P, _I64, _I32, _I32, _P, _SZ, _P], _I32),
    "ssm_conv1d_silu": ([_P, _P, _P, _I64, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_selective_scan": ([_P, _P, _P, _P, _P, _P, _I64, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_decode_conv": ([_P, _P, _P, _I32, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_decode_ssm": ([_P, _P, _P, _P, _P, _P, _I32, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_exchange_payload_bytes": ([_I32, _I64, _I64, _P], _I32),
    "ssm_exchange_encode": ([_I32, _P, _I32, _I64, _I64, _I64, _P, _SZ, _P], _I32),
    "ssm_exchange_decode_accumulate": ([_I32, _P, _SZ, _I64, _I64, _P, _I64, _I32, _P], _I32),
    "ssm2_shard_check_desc": ([_P], _I32),
    "ssm2_shard_prefill_workspace_bytes": ([_P, _I64, _I32, _P], _I32),
    "ssm2_shard_decode_workspace_bytes": ([_P, _I32, _P], _I32),
    "ssm2_shard_slice_weights": ([_P, _P, _P, _P], _I32),
    "ssm2_shard_prefill_stage1": ([_P, _P, _P, _I64, _P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm2_shard_prefill_stage2": ([_P, _P, _P, _I64, _P, _P, _SZ, _P], _I32),
    "ssm2_shard_decode_stage1": ([_P, _P, _P, _I32, _P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm2_shard_decode_stage2": ([_P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_residual_rmsnorm": ([_P, _I32, _P, _I32, _I32, _P, _P, ctypes.c_float, _P, _I32, _I64, _I32, _P], _I32),
    "ssm_bcdt_rmsnorm": ([_P, _I64, _I32, _I32, _I64, ctypes.c_float, _P], _I32),
    "ssm_stack_prefill_workspace_bytes": ([_P, _I64, _I32, _P], _I32),
    "ssm_stack_decode_workspace_bytes": ([_P, _I32, _P], _I32),
    "ssm_stack_prefill": ([_P, _P, _P, _P, _P, _I64, _P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_stack_decode_step": ([_P, _P, _P, _P, _P, _I32, _P, _P, _P, _I32, _P, _P, _SZ, _P], _I32),
    "ssm_timing_enable": ([_I32, ctypes.c_char_p], _I32),
    "ssm_timing_collect": ([_P, _I32, _P], _I32),
}


def lib() -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2602_21144_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes, f.restype = args, res
        _lib = L
    return _lib


def _check(rc: int):
    if rc != SSM_OK:
        raise SsmError(rc, lib().ssm_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device tensor expected")
    if not t.is_contiguous():
        raise ValueError("contiguous tensor expected")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def torch_act(act: str):
    return torch.bfloat16 if act == "bf16" else torch.float32


def make_desc(shape: LayerShape, shard_index: int = 0) -> Desc:
    d = Desc(shape.d_model, shape.d_inner, shape.d_shard, shape.d_state, shape.dt_rank, shape.d_conv,
             shard_index, shape.shard_count, SSM_BF16 if shape.act == "bf16" else SSM_F32)
    _check(lib().ssm_shard_check_desc(ctypes.byref(d)))
    return d


_WKEYS = {"in_proj_w": "W_in", "conv_w": "conv_w", "conv_b": "conv_b", "x_proj_w": "W_x", "dt_proj_w": "W_dt",
          "out_proj_w": "W_out", "dt_proj_b": "b_dt", "A_log": "A_log", "D": "D"}
_F32_KEYS = ("b_dt", "A_log", "D")


def upload_weights(host: Dict[str, np.ndarray], act: str, device="cuda") -> Dict[str, torch.Tensor]:
    """Copy host weights (float32 arrays, act-typed ones already representable) to the device."""
    out = {}
    for k in _WKEYS.values():
        dt = torch.float32 if k in _F32_KEYS else torch_act(act)
        out[k] = torch.from_numpy(np.ascontiguousarray(host[k], np.float32)).to(device=device, dtype=dt)
    return out


def weights_struct(dev: Dict[str, torch.Tensor]) -> Weights:
    return Weights(*[_ptr(dev[_WKEYS[f]]) for f, _ in Weights._fields_])


def empty_shard_weights(shape: LayerShape, device="cuda") -> Dict[str, torch.Tensor]:
    E, dm, N, R, K = shape.d_shard, shape.d_model, shape.d_state, shape.dt_rank, shape.d_conv
    a = torch_act(shape.act)
    f = torch.float32
    shapes = {"W_in": ((2 * E, dm), a), "conv_w": ((E, K), a), "conv_b": ((E,), a), "W_x": ((R + 2 * N, E), a),
              "W_dt": ((E, R), a), "W_out": ((dm, E), a), "b_dt": ((E,), f), "A_log": ((E, N), f), "D": ((E,), f)}
    return {k: torch.empty(s, dtype=t, device=device) for k, (s, t) in shapes.items()}


def ssm_shard_slice_weights(desc: Desc, full: Dict[str, torch.Tensor], out: Dict[str, torch.Tensor], stream=None):
    fw, ow = weights_struct(full), weights_struct(out)
    _check(lib().ssm_shard_slice_weights(ctypes.byref(desc), ctypes.byref(fw), ctypes.byref(ow), _stream(stream)))


class SeqMeta:
    """Device-resident packed-batch metadata (int32), validated from its host copy."""

    def __init__(self, cu_seqlens, cache_slot, has_initial_state, num_slots: int, device="cuda"):
        cu = np.ascontiguousarray(cu_seqlens, np.int32)
        sl = np.ascontiguousarray(cache_slot, np.int32)
        hi = np.ascontiguousarray(has_initial_state, np.int32)
        self.nseq = int(sl.shape[0])
        self.T = int(cu[-1]) if cu.size else 0
        _check(lib().ssm_shard_check_meta_host(cu.ctypes.data, sl.ctypes.data, hi.ctypes.data, self.nseq,
                                               self.T, int(num_slots)))
        self.host = (cu, sl, hi)
        n = max(self.nseq, 1)
        self.cu = torch.zeros(n + 1, dtype=torch.int32, device=device)
        self.slot = torch.zeros(n, dtype=torch.int32, device=device)
        self.has_init = torch.zeros(n, dtype=torch.int32, device=device)
        if self.nseq:
            self.cu.copy_(torch.from_numpy(cu))
            self.slot.copy_(torch.from_numpy(sl))
            self.has_init.copy_(torch.from_numpy(hi))
        self.c = SeqMetaC(self.cu.data_ptr(), self.slot.data_ptr(), self.has_init.data_ptr(), self.nseq)


def prefill_workspace_bytes(desc: Desc, max_tokens: int, max_seqs: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm_shard_prefill_workspace_bytes(ctypes.byref(desc), max_tokens, max_seqs, ctypes.byref(n)))
    return n.value


def decode_workspace_bytes(desc: Desc, max_batch: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm_shard_decode_workspace_bytes(ctypes.byref(desc), max_batch, ctypes.byref(n)))
    return n.value


def workspace(nbytes: int, device="cuda", stream=None) -> torch.Tensor:
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    _check(lib().ssm_shard_workspace_init(_ptr(ws), ws.numel(), _stream(stream)))
    return ws


def take_status(ws: torch.Tensor, stream=None) -> int:
    v = ctypes.c_int32()
    _check(lib().ssm_shard_take_status(_ptr(ws), ws.numel(), ctypes.byref(v), _stream(stream)))
    return v.value


def _w(weights):
    return weights if isinstance(weights, Weights) else weights_struct(weights)


# Each ABI call is marshalled by a _m_<name> function returning (ctypes arguments, objects
# those arguments point into). The wrapper of the same name makes the call once; bind()
# keeps the marshalled arguments for repeated calls with the same tensors.

def _m_ssm_shard_prefill(desc, weights, x, meta: SeqMeta, conv_pool, ssm_pool, y_partial, ws, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x), meta.T, ctypes.byref(meta.c), _ptr(conv_pool),
            _ptr(ssm_pool), conv_pool.shape[0], _ptr(y_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w, meta)


def _m_ssm_shard_prefill_stage1(desc, weights, x, meta: SeqMeta, conv_pool, x_dbl_partial, ws, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x), meta.T, ctypes.byref(meta.c), _ptr(conv_pool),
            conv_pool.shape[0], _ptr(x_dbl_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w, meta)


def _m_ssm_shard_prefill_stage2(desc, weights, x_dbl, meta: SeqMeta, ssm_pool, y_partial, ws, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x_dbl), meta.T, ctypes.byref(meta.c), _ptr(ssm_pool),
            ssm_pool.shape[0], _ptr(y_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w, meta)


def _m_ssm_shard_decode_step(desc, weights, x_t, cache_slot, conv_pool, ssm_pool, y_partial, ws, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x_t), x_t.shape[0], _ptr(cache_slot), _ptr(conv_pool),
            _ptr(ssm_pool), conv_pool.shape[0], _ptr(y_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w)


def _m_ssm_shard_decode_step_noalloc(desc, weights, x_t, cache_slot, conv_pool, ssm_pool, y_partial, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x_t), x_t.shape[0], _ptr(cache_slot), _ptr(conv_pool),
            _ptr(ssm_pool), conv_pool.shape[0], _ptr(y_partial), _stream(stream)), (desc, w)


def _m_ssm_shard_decode_stage1(desc, weights, x_t, cache_slot, conv_pool, x_dbl_partial, ws, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x_t), x_t.shape[0], _ptr(cache_slot), _ptr(conv_pool),
            conv_pool.shape[0], _ptr(x_dbl_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w)


def _m_ssm_shard_decode_stage2(desc, weights, x_dbl, cache_slot, ssm_pool, y_partial, ws, stream=None):
    w = _w(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x_dbl), x_dbl.shape[0], _ptr(cache_slot), _ptr(ssm_pool),
            ssm_pool.shape[0], _ptr(y_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w)


def _m_ssm_reduce_add_f32(dst, src, stream=None):
    if dst.dtype != torch.float32 or src.dtype != torch.float32 or dst.numel() != src.numel():
        raise ValueError("ssm_reduce_add_f32: two float32 tensors of equal size expected")
    return (_ptr(dst), _ptr(src), dst.numel(), _stream(stream)), ()


_MARSHAL = {name[3:]: fn for name, fn in list(globals().items()) if name.startswith("_m_ssm_")}


def _call(name, *args, **kw):
    a, _keep = _MARSHAL[name](*args, **kw)
    _check(getattr(lib(), name)(*a))


def ssm_shard_prefill(desc, weights, x, meta: SeqMeta, conv_pool, ssm_pool, y_partial, ws, stream=None):
    _call("ssm_shard_prefill", desc, weights, x, meta, conv_pool, ssm_pool, y_partial, ws, stream)


def ssm_shard_prefill_stage1(desc, weights, x, meta: SeqMeta, conv_pool, x_dbl_partial, ws, stream=None):
    _call("ssm_shard_prefill_stage1", desc, weights, x, meta, conv_pool, x_dbl_partial, ws, stream)


def ssm_shard_prefill_stage2(desc, weights, x_dbl, meta: SeqMeta, ssm_pool, y_partial, ws, stream=None):
    _call("ssm_shard_prefill_stage2", desc, weights, x_dbl, meta, ssm_pool, y_partial, ws, stream)


def ssm_shard_decode_step(desc, weights, x_t, cache_slot, conv_pool, ssm_pool, y_partial, ws, stream=None):
    _call("ssm_shard_decode_step", desc, weights, x_t, cache_slot, conv_pool, ssm_pool, y_partial, ws, stream)


def ssm_shard_decode_step_noalloc(desc, weights, x_t, cache_slot, conv_pool, ssm_pool, y_partial, stream=None):
    _call("ssm_shard_decode_step_noalloc", desc, weights, x_t, cache_slot, conv_pool, ssm_pool, y_partial, stream)


def ssm_shard_decode_stage1(desc, weights, x_t, cache_slot, conv_pool, x_dbl_partial, ws, stream=None):
    _call("ssm_shard_decode_stage1", desc, weights, x_t, cache_slot, conv_pool, x_dbl_partial, ws, stream)


def ssm_shard_decode_stage2(desc, weights, x_dbl, cache_slot, ssm_pool, y_partial, ws, stream=None):
    _call("ssm_shard_decode_stage2", desc, weights, x_dbl, cache_slot, ssm_pool, y_partial, ws, stream)


def ssm_reduce_add_f32(dst, src, stream=None):
    _call("ssm_reduce_add_f32", dst, src, stream)


class BoundCall:
    """One ABI call with its arguments marshalled once. Calling it issues the call again
    with the same pointers, sizes and stream: the tensors must stay alive, unmoved and
    of the same shape (the object keeps references to them)."""

    __slots__ = ("_f", "_args", "_keep", "name")

    def __init__(self, name, args, keep):
        self.name = name
        self._f = getattr(lib(), name)
        self._args = args
        self._keep = keep

    def __call__(self):
        rc = self._f(*self._args)
        if rc != SSM_OK:
            _check(rc)


def bind(name: str, *args, **kw) -> BoundCall:
    """bind("ssm_shard_decode_stage1", desc, weights, x_t, ...) -> a callable issuing that call.
    Available for the prefill, decode and reduce entry points."""
    a, keep = _MARSHAL[name](*args, **kw)
    tensors = tuple(v for v in list(args) + list(kw.values()) if isinstance(v, torch.Tensor))
    return BoundCall(name, a, keep + tensors)


# ------------------------------------------------------------------ Mamba-2 (SSD) shard
_W2KEYS = {"in_proj_w": "W_in", "conv_w": "conv_w", "conv_b": "conv_b", "out_proj_w": "W_out",
           "dt_bias": "dt_bias", "A_log": "A_log", "D": "D", "norm_w": "norm_w"}
_W2_F32 = ("dt_bias", "A_log", "D", "norm_w")


def make_desc2(shape, shard_index: int = 0, full: bool = False) -> Desc2:
    """Descriptor of shard `shard_index` (or of the unsplit layer with full=True)."""
    d = Desc2(shape.d_model, shape.nheads, shape.headdim, shape.d_state, shape.ngroups, shape.d_conv,
              0 if full else shard_index, 1 if full else shape.shard_count, SSM_BF16)
    _check(lib().ssm2_shard_check_desc(ctypes.byref(d)))
    return d


def upload_weights2(host: Dict[str, np.ndarray], device="cuda") -> Dict[str, torch.Tensor]:
    return {k: torch.from_numpy(np.ascontiguousarray(host[k], np.float32)).to(
        device=device, dtype=torch.float32 if k in _W2_F32 else torch.bfloat16) for k in _W2KEYS.values()}


def weights2_struct(dev: Dict[str, torch.Tensor]) -> Weights2:
    return Weights2(*[_ptr(dev[_W2KEYS[f]]) for f, _ in Weights2._fields_])


def empty_shard_weights2(shape, device="cuda") -> Dict[str, torch.Tensor]:
    E, H, dm, K = shape.d_shard, shape.heads_shard, shape.d_model, shape.d_conv
    rows, Cc = shape.in_rows_shard, shape.conv_dim_shard
    b, f = torch.bfloat16, torch.float32
    shapes = {"W_in": ((rows, dm), b), "conv_w": ((Cc, K), b), "conv_b": ((Cc,), b), "W_out": ((dm, E), b),
              "dt_bias": ((H,), f), "A_log": ((H,), f), "D": ((H,), f), "norm_w": ((E,), f)}
    return {k: torch.empty(sz, dtype=t, device=device) for k, (sz, t) in shapes.items()}


def ssm2_shard_slice_weights(desc: Desc2, full: Dict[str, torch.Tensor], out: Dict[str, torch.Tensor], stream=None):
    fw, ow = weights2_struct(full), weights2_struct(out)
    _check(lib().ssm2_shard_slice_weights(ctypes.byref(desc), ctypes.byref(fw), ctypes.byref(ow), _stream(stream)))


def m2_prefill_workspace_bytes(desc: Desc2, max_tokens: int, max_seqs: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm2_shard_prefill_workspace_bytes(ctypes.byref(desc), max_tokens, max_seqs, ctypes.byref(n)))
    return n.value


def m2_decode_workspace_bytes(desc: Desc2, max_batch: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm2_shard_decode_workspace_bytes(ctypes.byref(desc), max_batch, ctypes.byref(n)))
    return n.value


def _w2(weights):
    return weights if isinstance(weights, Weights2) else weights2_struct(weights)


def _m_ssm2_shard_prefill_stage1(desc, weights, x, meta: SeqMeta, conv_pool, ssm_pool, sumsq_partial, ws, stream=None):
    w = _w2(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x), meta.T, ctypes.byref(meta.c), _ptr(conv_pool),
            _ptr(ssm_pool), conv_pool.shape[0], _ptr(sumsq_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w, meta)


def _m_ssm2_shard_prefill_stage2(desc, weights, sumsq, T, y_partial, ws, stream=None):
    w = _w2(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(sumsq), T, _ptr(y_partial), _ptr(ws), ws.numel(),
            _stream(stream)), (desc, w)


def _m_ssm2_shard_decode_stage1(desc, weights, x_t, cache_slot, conv_pool, ssm_pool, sumsq_partial, ws, stream=None):
    w = _w2(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(x_t), x_t.shape[0], _ptr(cache_slot), _ptr(conv_pool),
            _ptr(ssm_pool), conv_pool.shape[0], _ptr(sumsq_partial), _ptr(ws), ws.numel(), _stream(stream)), (desc, w)


def _m_ssm2_shard_decode_stage2(desc, weights, sumsq, batch, y_partial, ws, stream=None):
    w = _w2(weights)
    return (ctypes.byref(desc), ctypes.byref(w), _ptr(sumsq), batch, _ptr(y_partial), _ptr(ws), ws.numel(),
            _stream(stream)), (desc, w)


_MARSHAL.update({name[3:]: fn for name, fn in list(globals().items()) if name.startswith("_m_ssm2_")})


def ssm2_shard_prefill_stage1(desc, weights, x, meta, conv_pool, ssm_pool, sumsq_partial, ws, stream=None):
    _call("ssm2_shard_prefill_stage1", desc, weights, x, meta, conv_pool, ssm_pool, sumsq_partial, ws, stream)


def ssm2_shard_prefill_stage2(desc, weights, sumsq, T, y_partial, ws, stream=None):
    _call("ssm2_shard_prefill_stage2", desc, weights, sumsq, T, y_partial, ws, stream)


def ssm2_shard_decode_stage1(desc, weights, x_t, cache_slot, conv_pool, ssm_pool, sumsq_partial, ws, stream=None):
    _call("ssm2_shard_decode_stage1", desc, weights, x_t, cache_slot, conv_pool, ssm_pool, sumsq_partial, ws, stream)


def ssm2_shard_decode_stage2(desc, weights, sumsq, batch, y_partial, ws, stream=None):
    _call("ssm2_shard_decode_stage2", desc, weights, sumsq, batch, y_partial, ws, stream)


SSM_CODEC = {"f16": 0, "bf16": 1, "fp8": 2, "int8": 3}


def exchange_payload_bytes(codec: str, rows: int, cols: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm_exchange_payload_bytes(SSM_CODEC[codec], rows, cols, ctypes.byref(n)))
    return n.value


def exchange_payload(codec: str, rows: int, cols: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(exchange_payload_bytes(codec, rows, cols), 16), dtype=torch.uint8, device=device)


def ssm_exchange_encode(codec: str, src: torch.Tensor, payload: torch.Tensor, stream=None):
    """payload <- encode(src); src is [rows][cols] float32 or bfloat16 with unit column stride."""
    rows, cols = src.shape
    if src.stride(1) != 1:
        raise ValueError("unit column stride expected")
    _check(lib().ssm_exchange_encode(SSM_CODEC[codec], ctypes.c_void_p(src.data_ptr()), _dt(src), rows, cols,
                                     src.stride(0), _ptr(payload), payload.numel(), _stream(stream)))


def ssm_exchange_decode_accumulate(codec: str, payload: torch.Tensor, acc: torch.Tensor, accumulate: bool,
                                   stream=None):
    """acc [rows][cols] float32 = decode(payload) (+ acc when accumulate)."""
    rows, cols = acc.shape
    if acc.dtype != torch.float32 or acc.stride(1) != 1:
        raise ValueError("float32 accumulator with unit column stride expected")
    _check(lib().ssm_exchange_decode_accumulate(SSM_CODEC[codec], _ptr(payload), payload.numel(), rows, cols,
                                                ctypes.c_void_p(acc.data_ptr()), acc.stride(0),
                                                1 if accumulate else 0, _stream(stream)))


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SSM_F32
    if t.dtype == torch.bfloat16:
        return SSM_BF16
    raise ValueError(t.dtype)


def ssm_gemm_nt(A, B, C, stream=None):
    """C[M][N] = A[M][K] B[N][K]^T on the library's GEMM kernels (row strides from the tensors)."""
    M, K = A.shape
    N = B.shape[0]
    assert B.shape[1] == K and C.shape == (M, N)
    for t in (A, B, C):
        assert t.stride(1) == 1
    _check(lib().ssm_gemm_nt(M, N, K, ctypes.c_void_p(A.data_ptr()), A.stride(0), _dt(A),
                             ctypes.c_void_p(B.data_ptr()), B.stride(0), _dt(B), ctypes.c_void_p(C.data_ptr()),
                             C.stride(0), _dt(C), _stream(stream)))


GEMM_ROLE = {"generic": 0, "in_proj": 1, "x_proj": 2, "dt_proj": 3, "out_proj": 4}


def gemm_splitk_bytes(M, N, K, a_dtype, b_dtype, role: str) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm_gemm_splitk_bytes(M, N, K, a_dtype, b_dtype, GEMM_ROLE[role], ctypes.byref(n)))
    return n.value


def ssm_gemm_nt_role(A, B, C, role: str, scratch: Optional[torch.Tensor] = None, stream=None):
    """ssm_gemm_nt on one projection's kernel path, split-K into scratch when it fits."""
    M, K = A.shape
    N = B.shape[0]
    assert B.shape[1] == K and C.shape == (M, N)
    for t in (A, B, C):
        assert t.stride(1) == 1
    sp = ctypes.c_void_p(scratch.data_ptr()) if scratch is not None else None
    nb = scratch.numel() * scratch.element_size() if scratch is not None else 0
    _check(lib().ssm_gemm_nt_role(M, N, K, ctypes.c_void_p(A.data_ptr()), A.stride(0), _dt(A),
                                  ctypes.c_void_p(B.data_ptr()), B.stride(0), _dt(B), ctypes.c_void_p(C.data_ptr()),
                                  C.stride(0), _dt(C), GEMM_ROLE[role], sp, nb, _stream(stream)))


def ssm_conv1d_silu(desc, weights, xz, meta: SeqMeta, conv_pool, u, ws, stream=None):
    w = _w(weights)
    _check(lib().ssm_conv1d_silu(ctypes.byref(desc), ctypes.byref(w), _ptr(xz), meta.T, ctypes.byref(meta.c),
                                 _ptr(conv_pool), conv_pool.shape[0], _ptr(u), _ptr(ws), ws.numel(), _stream(stream)))


def ssm_selective_scan(desc, weights, u, dt, xz, x_dbl, meta: SeqMeta, ssm_pool, g, ws, stream=None):
    w = _w(weights)
    _check(lib().ssm_selective_scan(ctypes.byref(desc), ctypes.byref(w), _ptr(u), _ptr(dt), _ptr(xz), _ptr(x_dbl),
                                    meta.T, ctypes.byref(meta.c), _ptr(ssm_pool), ssm_pool.shape[0], _ptr(g),
                                    _ptr(ws), ws.numel(), _stream(stream)))


def ssm_decode_conv(desc, weights, xz, cache_slot, conv_pool, u, ws, stream=None):
    w = _w(weights)
    _check(lib().ssm_decode_conv(ctypes.byref(desc), ctypes.byref(w), _ptr(xz), xz.shape[0], _ptr(cache_slot),
                                 _ptr(conv_pool), conv_pool.shape[0], _ptr(u), _ptr(ws), ws.numel(), _stream(stream)))


def ssm_decode_ssm(desc, weights, u, dt, xz, x_dbl, cache_slot, ssm_pool, g, ws, stream=None):
    w = _w(weights)
    _check(lib().ssm_decode_ssm(ctypes.byref(desc), ctypes.byref(w), _ptr(u), _ptr(dt), _ptr(xz), _ptr(x_dbl),
                                u.shape[0], _ptr(cache_slot), _ptr(ssm_pool), ssm_pool.shape[0], _ptr(g), _ptr(ws),
                                ws.numel(), _stream(stream)))


def scan_scratch_workspace_bytes(desc: Desc, T: int, nseq: int) -> int:
    """Workspace large enough for ssm_selective_scan at (T, nseq) (header + scan scratch)."""
    return prefill_workspace_bytes(desc, T, nseq)


def ssm_timing_enable(on: bool = True, only: Optional[str] = None, every: int = 1):
    """Per-dispatch kernel timing on (every `every`-th launch of each kernel name) or off."""
    _check(lib().ssm_timing_enable((max(int(every), 1) if on else 0), only.encode() if only else None))


def ssm_timing_collect(max_kernels: int = 64) -> Dict[str, tuple]:
    """{kernel role: (launches, total ms)} since the last collection (waits for the events)."""
    buf = (KernelTime * max_kernels)()
    n = ctypes.c_int32()
    _check(lib().ssm_timing_collect(buf, max_kernels, ctypes.byref(n)))
    return {buf[i].name.decode(): (int(buf[i].launches), float(buf[i].total_ms)) for i in range(n.value)}


# ------------------------------------------------------------------ the layer around the mixer
class StackDesc(ctypes.Structure):
    _fields_ = [("layer", Desc), ("n_layers", ctypes.c_int32), ("norm_eps", ctypes.c_float),
                ("bcdt_eps", ctypes.c_float)]


def _dtype_of(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SSM_F32
    if t.dtype == torch.bfloat16:
        return SSM_BF16
    raise ValueError(f"float32 or bfloat16 tensor expected, got {t.dtype}")


def _m_ssm_residual_rmsnorm(base, parts, residual, norm_w, eps, normed, stream=None):
    """residual <- base + sum(parts); normed <- RMSNorm(residual) * norm_w. base, every part,
    residual and normed are [T][d]; parts is a list (possibly empty) of same-dtype tensors."""
    T, d = base.shape
    pdt = _dtype_of(parts[0]) if parts else SSM_F32
    arr = (ctypes.c_void_p * max(len(parts), 1))(*[p.data_ptr() for p in parts])
    for p in parts:
        _ptr(p)
        if p.shape != base.shape or _dtype_of(p) != pdt:
            raise ValueError("parts must match base's shape and share one dtype")
    return (_ptr(base), _dtype_of(base), arr, len(parts), pdt, _ptr(residual), _ptr(norm_w), float(eps),
            _ptr(normed), _dtype_of(normed), T, d, _stream(stream)), (arr,)


def _m_ssm_bcdt_rmsnorm(x_dbl, R, N, eps, stream=None):
    T, ld = x_dbl.shape
    if x_dbl.dtype != torch.float32:
        raise ValueError("x_dbl must be float32")
    return (_ptr(x_dbl), T, int(R), int(N), ld, float(eps), _stream(stream)), ()


def make_stack_desc(shape: LayerShape, n_layers: int, norm_eps: float = 1e-5, bcdt_eps: float = 0.0) -> StackDesc:
    return StackDesc(make_desc(shape), n_layers, norm_eps, bcdt_eps)


class StackWeights:
    """Host arrays (ctypes) of a stack's per-layer weight structs and device pointers."""

    def __init__(self, layers, norm_w, final_w):
        self.structs = [_w(w) for w in layers]
        self.layers = (Weights * len(layers))(*self.structs)
        self.norm_w = (ctypes.c_void_p * len(norm_w))(*[_ptr(t).value for t in norm_w])
        self.final_w = _ptr(final_w)
        self._keep = (layers, norm_w, final_w)


class StackPools:
    def __init__(self, conv, ssm):
        self.conv = (ctypes.c_void_p * len(conv))(*[_ptr(t).value for t in conv])
        self.ssm = (ctypes.c_void_p * len(ssm))(*[_ptr(t).value for t in ssm])
        self.S = conv[0].shape[0]
        self._keep = (conv, ssm)


def stack_prefill_workspace_bytes(sd: StackDesc, max_tokens: int, max_seqs: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm_stack_prefill_workspace_bytes(ctypes.byref(sd), max_tokens, max_seqs, ctypes.byref(n)))
    return n.value


def stack_decode_workspace_bytes(sd: StackDesc, max_batch: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().ssm_stack_decode_workspace_bytes(ctypes.byref(sd), max_batch, ctypes.byref(n)))
    return n.value


def _m_ssm_stack_prefill(sd, sw: StackWeights, x, meta: SeqMeta, pools: StackPools, out, ws, stream=None):
    return (ctypes.byref(sd), sw.layers, sw.norm_w, sw.final_w, _ptr(x), meta.T, ctypes.byref(meta.c), pools.conv,
            pools.ssm, pools.S, _ptr(out), _ptr(ws), ws.numel(), _stream(stream)), (sd, sw, meta, pools)


def _m_ssm_stack_decode_step(sd, sw: StackWeights, x_t, cache_slot, pools: StackPools, out, ws, stream=None):
    return (ctypes.byref(sd), sw.layers, sw.norm_w, sw.final_w, _ptr(x_t), x_t.shape[0], _ptr(cache_slot),
            pools.conv, pools.ssm, pools.S, _ptr(out), _ptr(ws), ws.numel(), _stream(stream)), (sd, sw, pools)


_MARSHAL.update({name[3:]: fn for name, fn in list(globals().items())
                 if name.startswith(("_m_ssm_residual", "_m_ssm_bcdt", "_m_ssm_stack"))})


def ssm_residual_rmsnorm(base, parts, residual, norm_w, eps, normed, stream=None):
    _call("ssm_residual_rmsnorm", base, parts, residual, norm_w, eps, normed, stream)


def ssm_bcdt_rmsnorm(x_dbl, R, N, eps, stream=None):
    _call("ssm_bcdt_rmsnorm", x_dbl, R, N, eps, stream)


def ssm_stack_prefill(sd, sw, x, meta, pools, out, ws, stream=None):
    _call("ssm_stack_prefill", sd, sw, x, meta, pools, out, ws, stream)


def ssm_stack_decode_step(sd, sw, x_t, cache_slot, pools, out, ws, stream=None):
    _call("ssm_stack_decode_step", sd, sw, x_t, cache_slot, pools, out, ws, stream)
