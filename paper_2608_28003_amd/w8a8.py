"""ctypes binding of ``libw8a8.so`` (C ABI in ``include/w8a8.h``).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  torch supplies device memory and the current stream.  The library
is loaded on first use; a missing or unloadable library raises, there is no
fallback.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libw8a8.so")

OK, EINVAL, EUNSUPPORTED, EHIP, EWORKSPACE, ETIMEOUT = 0, 1, 2, 3, 4, 5
F32, BF16 = 0, 1
MAX_K = 133144


class W8A8Error(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("w8a8 status %d: %s" % (status, msg))
        self.status = status


P = ctypes.c_void_p
I64 = ctypes.c_int64
SZ = ctypes.c_size_t
INT = ctypes.c_int


class LinearDesc(ctypes.Structure):
    _fields_ = [("n", I64), ("k", I64), ("wq", P), ("s_w", P), ("delta", P)]


class FfnDesc(ctypes.Structure):
    _fields_ = [("d", I64), ("f", I64), ("wq_gate", P), ("s_gate", P), ("wq_up", P),
                ("s_up", P), ("delta_gu", P), ("wq_down", P), ("s_down", P),
                ("delta_down", P)]


class Bf16FfnDesc(ctypes.Structure):
    _fields_ = [("d", I64), ("f", I64), ("wp_gate", P), ("wp_up", P), ("wp_down", P)]


class StackDesc(ctypes.Structure):
    _fields_ = [("n_layers", I64), ("d", I64), ("f", I64), ("vocab", I64),
                ("int8_ffn", ctypes.POINTER(FfnDesc)), ("bf16_ffn", ctypes.POINTER(Bf16FfnDesc)),
                ("lm_head_int8", LinearDesc), ("lm_head_bf16", P)]


_SIGS = {
    "w8a8_packed_bytes": (SZ, [I64, I64]),
    "w8a8_packed_bf16_bytes": (SZ, [I64, I64]),
    "w8a8_linear_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_ffn_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_bf16_ffn_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_lm_head_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_bf16_linear_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_stack_workspace_bytes": (SZ, [I64, I64, I64, I64]),
    "w8a8_col_absmax": (INT, [P, INT, I64, I64, P, P]),
    "w8a8_smooth_calibrate": (INT, [P, ctypes.POINTER(P), ctypes.POINTER(I64), INT, INT, I64,
                                    ctypes.c_float, P, P]),
    "w8a8_smooth_delta": (INT, [P, P, I64, ctypes.c_float, P, P]),
    "w8a8_geglu_requant": (INT, [P, P, I64, I64, P, P, P, P, P]),
    "w8a8_ffn_stack_status": (INT, [P, SZ, P]),
    "w8a8_set_plan_override": (INT, [ctypes.c_char_p, INT]),
    "w8a8_clear_plan_overrides": (None, []),
    "w8a8_quantize_weights": (INT, [P, INT, I64, I64, P, P, P, P]),
    "w8a8_unpack_weights": (INT, [P, I64, I64, P, P]),
    "w8a8_pack_bf16": (INT, [P, I64, I64, P, P]),
    "w8a8_quantize_act": (INT, [P, INT, I64, I64, P, P, P, P]),
    "w8a8_gemm_i8_i32": (INT, [P, I64, P, I64, I64, P, P, SZ, P]),
    "w8a8_linear": (INT, [ctypes.POINTER(LinearDesc), P, INT, I64, P, INT, P, SZ, P]),
    "w8a8_ffn_gate_up": (INT, [ctypes.POINTER(FfnDesc), P, P, I64, P, P]),
    "w8a8_ffn": (INT, [ctypes.POINTER(FfnDesc), P, I64, P, P, SZ, P]),
    "w8a8_ffn_noalloc": (INT, [ctypes.POINTER(FfnDesc), P, I64, P, P]),
    "w8a8_lm_head": (INT, [ctypes.POINTER(LinearDesc), P, I64, P, P, SZ, P]),
    "w8a8_fp8_linear_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_fp8_ffn_workspace_bytes": (SZ, [I64, I64, I64]),
    "w8a8_fp8_quantize_weights": (INT, [P, INT, I64, I64, P, P, P, P]),
    "w8a8_fp8_quantize_act": (INT, [P, INT, I64, I64, P, P, P, P]),
    "w8a8_fp8_gemm_f32": (INT, [P, I64, P, I64, I64, P, P, SZ, P]),
    "w8a8_fp8_linear": (INT, [ctypes.POINTER(LinearDesc), P, INT, I64, P, INT, P, SZ, P]),
    "w8a8_fp8_ffn_gate_up": (INT, [ctypes.POINTER(FfnDesc), P, P, I64, P, P]),
    "w8a8_fp8_ffn": (INT, [ctypes.POINTER(FfnDesc), P, I64, P, P, SZ, P]),
    "w8a8_fp8_lm_head": (INT, [ctypes.POINTER(LinearDesc), P, I64, P, P, SZ, P]),
    "w8a8_bf16_linear": (INT, [P, I64, P, I64, I64, P, P, SZ, P]),
    "w8a8_bf16_ffn": (INT, [ctypes.POINTER(Bf16FfnDesc), P, I64, P, P, SZ, P]),
    "w8a8_bf16_ffn_gate_up": (INT, [ctypes.POINTER(Bf16FfnDesc), P, I64, P, P]),
    "w8a8_rmsnorm": (INT, [P, I64, I64, P, P]),
    "w8a8_rmsnorm_residual": (INT, [P, P, I64, I64, P, P]),
    "w8a8_precision_map": (INT, [ctypes.c_char_p, P, INT]),
    "w8a8_ffn_stack": (INT, [ctypes.POINTER(StackDesc), P, INT, P, I64, P, P, SZ, P]),
    "w8a8_ffn_stack_trace": (INT, [ctypes.POINTER(StackDesc), P, INT, P, I64, P, P, P, SZ, P]),
    "w8a8_sqnr_workspace_bytes": (SZ, [I64]),
    "w8a8_sqnr": (INT, [P, P, INT, I64, P, P, SZ, P]),
    "w8a8_stack_sensitivity_workspace_bytes": (SZ, [I64, I64, I64, I64, I64]),
    "w8a8_stack_sensitivity": (INT, [ctypes.POINTER(StackDesc), P, P, I64, P, P, P, SZ, P]),
    "w8a8_rank_layers": (INT, [P, INT, P]),
    "w8a8_select_precision_map": (INT, [ctypes.POINTER(StackDesc), P, I64, ctypes.c_float, P, P,
                                        P, SZ, P]),
    "w8a8_kv_quantize": (INT, [P, I64, I64, P, P, P]),
    "w8a8_attn_decode_workspace_bytes": (SZ, [I64]),
    "w8a8_attn_decode": (INT, [P, INT, I64, I64, P, P, P, P, I64, P, P, SZ, P]),
    "w8a8_attn_decode_bf16": (INT, [P, INT, I64, I64, P, P, I64, P, P, SZ, P]),
    "w8a8_status_str": (ctypes.c_char_p, [INT]),
    "w8a8_last_error": (ctypes.c_char_p, []),
}

_lib = None


def lib():
    """Load ``libw8a8.so`` (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libw8a8.so is missing: build it with "
                               "`python -m paper_2608_28003_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def exported_names():
    return list(_SIGS)


def _check(status):
    if status != OK:
        raise W8A8Error(status, lib().w8a8_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t):
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t


def _dt(t):
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError("dtype %s not supported" % t.dtype)


def _empty(nbytes, device):
    # 256-byte aligned uint8 buffer
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ----------------------------------------------------------------- sizes

def packed_bytes(n, k):
    return lib().w8a8_packed_bytes(n, k)


def packed_bf16_bytes(n, k):
    return lib().w8a8_packed_bf16_bytes(n, k)


def linear_workspace_bytes(m, n, k):
    return lib().w8a8_linear_workspace_bytes(m, n, k)


def ffn_workspace_bytes(m, d, f):
    return lib().w8a8_ffn_workspace_bytes(m, d, f)


def bf16_ffn_workspace_bytes(m, d, f):
    return lib().w8a8_bf16_ffn_workspace_bytes(m, d, f)


def lm_head_workspace_bytes(m, n, k):
    return lib().w8a8_lm_head_workspace_bytes(m, n, k)


def bf16_linear_workspace_bytes(m, n, k):
    return lib().w8a8_bf16_linear_workspace_bytes(m, n, k)


def stack_workspace_bytes(m, d, f, vocab):
    return lib().w8a8_stack_workspace_bytes(m, d, f, vocab)


# ----------------------------------------------------------------- a1 / a2 / a3

def col_absmax(x, amax=None, stream=None):
    _dev(x)
    rows, k = x.shape
    if amax is None:
        amax = torch.zeros(k, dtype=torch.float32, device=x.device)
    _check(lib().w8a8_col_absmax(_ptr(x), _dt(x), rows, k, _ptr(amax), _stream(stream)))
    return amax


def smooth_calibrate(act_amax, weights, alpha=0.5, stream=None):
    """delta from the calibration statistic and every weight matrix (k columns,
    one dtype) that consumes the input; the weight maximum runs over all their
    rows stacked."""
    k = act_amax.numel()
    weights = [_dev(w) for w in weights]
    dt = _dt(weights[0])
    if any(_dt(w) != dt or w.shape[1] != k for w in weights):
        raise ValueError("weights must share dtype and have k columns")
    delta = torch.empty(k, dtype=torch.float32, device=act_amax.device)
    ptrs = (P * len(weights))(*[w.data_ptr() for w in weights])
    rows = (I64 * len(weights))(*[w.shape[0] for w in weights])
    _check(lib().w8a8_smooth_calibrate(_ptr(_dev(act_amax)), ptrs, rows, len(weights), dt, k,
                                       float(alpha), _ptr(delta), _stream(stream)))
    return delta


def smooth_delta(act_amax, w_amax, alpha=0.5, stream=None):
    """delta from both statistics already gathered (w8a8_col_absmax)."""
    k = act_amax.numel()
    delta = torch.empty(k, dtype=torch.float32, device=act_amax.device)
    _check(lib().w8a8_smooth_delta(_ptr(_dev(act_amax)), _ptr(_dev(w_amax)), k,
                                   float(alpha), _ptr(delta), _stream(stream)))
    return delta


def geglu_requant(g, u, delta=None, want_h=True, stream=None):
    """(packed codes of h / delta, per-row scales, h or None) with
    h = bf16(gelu_tanh(g) u) from binary32 g, u."""
    _dev(g)
    _dev(u)
    m, n = g.shape
    q = _empty(packed_bytes(m, n), g.device)
    s = torch.empty(m, dtype=torch.float32, device=g.device)
    h = torch.empty((m, n), dtype=torch.bfloat16, device=g.device) if want_h else None
    _check(lib().w8a8_geglu_requant(_ptr(g), _ptr(u), m, n, _ptr(delta), _ptr(q), _ptr(s),
                                    _ptr(h), _stream(stream)))
    return q, s, h


def set_plan_override(name, value):
    if lib().w8a8_set_plan_override(name.encode(), int(value)) != 0:
        raise ValueError("unknown planner override %r" % name)


def clear_plan_overrides():
    lib().w8a8_clear_plan_overrides()


def quantize_weights(w, delta=None, stream=None):
    """Returns (packed int8 codes as a uint8 tensor, s_w)."""
    _dev(w)
    n, k = w.shape
    wq = _empty(packed_bytes(n, k), w.device)
    s_w = torch.empty(n, dtype=torch.float32, device=w.device)
    _check(lib().w8a8_quantize_weights(_ptr(w), _dt(w), n, k, _ptr(delta), _ptr(wq), _ptr(s_w),
                                       _stream(stream)))
    return wq, s_w


def unpack_weights(wq, n, k, stream=None):
    q = torch.empty((n, k), dtype=torch.int8, device=wq.device)
    _check(lib().w8a8_unpack_weights(_ptr(wq), n, k, _ptr(q), _stream(stream)))
    return q


def pack_bf16(w, stream=None):
    _dev(w)
    n, k = w.shape
    wp = _empty(packed_bf16_bytes(n, k), w.device)
    _check(lib().w8a8_pack_bf16(_ptr(w), n, k, _ptr(wp), _stream(stream)))
    return wp


def quantize_act(x, delta=None, stream=None):
    """Returns (packed int8 codes, s_x)."""
    _dev(x)
    m, k = x.shape
    qx = _empty(packed_bytes(m, k), x.device)
    s_x = torch.empty(m, dtype=torch.float32, device=x.device)
    _check(lib().w8a8_quantize_act(_ptr(x), _dt(x), m, k, _ptr(delta), _ptr(qx), _ptr(s_x),
                                   _stream(stream)))
    return qx, s_x


# ----------------------------------------------------------------- layers

@dataclass
class LinearW8A8:
    n: int
    k: int
    wq: torch.Tensor
    s_w: torch.Tensor
    delta: torch.Tensor | None

    @classmethod
    def from_weight(cls, w, delta=None):
        wq, s_w = quantize_weights(w, delta)
        return cls(w.shape[0], w.shape[1], wq, s_w, delta)

    def desc(self):
        return LinearDesc(self.n, self.k, _ptr(self.wq), _ptr(self.s_w), _ptr(self.delta))


@dataclass
class FfnW8A8:
    d: int
    f: int
    gate: LinearW8A8
    up: LinearW8A8
    down: LinearW8A8

    @classmethod
    def from_weights(cls, w_gate, w_up, w_down, delta_gu, delta_down):
        return cls(w_gate.shape[1], w_gate.shape[0],
                   LinearW8A8.from_weight(w_gate, delta_gu),
                   LinearW8A8.from_weight(w_up, delta_gu),
                   LinearW8A8.from_weight(w_down, delta_down))

    def desc(self):
        return FfnDesc(self.d, self.f, _ptr(self.gate.wq), _ptr(self.gate.s_w), _ptr(self.up.wq),
                       _ptr(self.up.s_w), _ptr(self.gate.delta), _ptr(self.down.wq),
                       _ptr(self.down.s_w), _ptr(self.down.delta))


@dataclass
class FfnBF16:
    d: int
    f: int
    wp_gate: torch.Tensor
    wp_up: torch.Tensor
    wp_down: torch.Tensor

    @classmethod
    def from_weights(cls, w_gate, w_up, w_down):
        return cls(w_gate.shape[1], w_gate.shape[0], pack_bf16(w_gate), pack_bf16(w_up),
                   pack_bf16(w_down))

    def desc(self):
        return Bf16FfnDesc(self.d, self.f, _ptr(self.wp_gate), _ptr(self.wp_up),
                           _ptr(self.wp_down))


def gemm_i8_i32(qx, m, wq, n, k, ws=None, stream=None):
    acc = torch.empty((m, n), dtype=torch.int32, device=qx.device)
    need = linear_workspace_bytes(m, n, k)
    if ws is None:
        ws = _empty(need, qx.device)
    _check(lib().w8a8_gemm_i8_i32(_ptr(qx), m, _ptr(wq), n, k, _ptr(acc), _ptr(ws),
                                  ws.numel(), _stream(stream)))
    return acc


def linear(layer: LinearW8A8, x, out_dtype=torch.float32, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.n), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = _empty(linear_workspace_bytes(m, layer.n, layer.k), x.device)
    d = layer.desc()
    _check(lib().w8a8_linear(ctypes.byref(d), _ptr(x), _dt(x), m, _ptr(out), _dt(out), _ptr(ws),
                             ws.numel(), _stream(stream)))
    return out


def ffn_gate_up(ffn: FfnW8A8, qx, s_x, m, out=None, stream=None):
    if out is None:
        out = torch.empty((m, ffn.f), dtype=torch.bfloat16, device=qx.device)
    d = ffn.desc()
    _check(lib().w8a8_ffn_gate_up(ctypes.byref(d), _ptr(qx), _ptr(s_x), m, _ptr(out),
                                  _stream(stream)))
    return out


def ffn(layer: FfnW8A8, x, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.d), dtype=torch.bfloat16, device=x.device)
    if ws is None:
        ws = _empty(ffn_workspace_bytes(m, layer.d, layer.f), x.device)
    d = layer.desc()
    _check(lib().w8a8_ffn(ctypes.byref(d), _ptr(x), m, _ptr(out), _ptr(ws), ws.numel(),
                          _stream(stream)))
    return out


def ffn_noalloc(layer: FfnW8A8, x, out=None, stream=None):
    """w8a8_ffn with the library's per-GPU scratch array instead of a workspace."""
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.d), dtype=torch.bfloat16, device=x.device)
    d = layer.desc()
    _check(lib().w8a8_ffn_noalloc(ctypes.byref(d), _ptr(x), m, _ptr(out), _stream(stream)))
    return out


def lm_head(layer: LinearW8A8, x, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.n), dtype=torch.bfloat16, device=x.device)
    if ws is None:
        ws = _empty(lm_head_workspace_bytes(m, layer.n, layer.k), x.device)
    d = layer.desc()
    _check(lib().w8a8_lm_head(ctypes.byref(d), _ptr(x), m, _ptr(out), _ptr(ws), ws.numel(),
                              _stream(stream)))
    return out


# ----------------------------------------------------------------- FP8 variant
# E4M3 codes in the packed fragment layout; the layer containers above carry
# them unchanged (LinearW8A8 / FfnW8A8 built with the fp8_ constructors below).

def fp8_linear_workspace_bytes(m, n, k):
    return lib().w8a8_fp8_linear_workspace_bytes(m, n, k)


def fp8_ffn_workspace_bytes(m, d, f):
    return lib().w8a8_fp8_ffn_workspace_bytes(m, d, f)


def fp8_quantize_weights(w, delta=None, stream=None):
    """Returns (packed E4M3 codes as a uint8 tensor, s_w)."""
    _dev(w)
    n, k = w.shape
    wq = _empty(packed_bytes(n, k), w.device)
    s_w = torch.empty(n, dtype=torch.float32, device=w.device)
    _check(lib().w8a8_fp8_quantize_weights(_ptr(w), _dt(w), n, k, _ptr(delta), _ptr(wq),
                                           _ptr(s_w), _stream(stream)))
    return wq, s_w


def fp8_quantize_act(x, delta=None, stream=None):
    """Returns (packed E4M3 codes, s_x)."""
    _dev(x)
    m, k = x.shape
    qx = _empty(packed_bytes(m, k), x.device)
    s_x = torch.empty(m, dtype=torch.float32, device=x.device)
    _check(lib().w8a8_fp8_quantize_act(_ptr(x), _dt(x), m, k, _ptr(delta), _ptr(qx),
                                       _ptr(s_x), _stream(stream)))
    return qx, s_x


def fp8_linear_layer(w, delta=None) -> LinearW8A8:
    wq, s_w = fp8_quantize_weights(w, delta)
    return LinearW8A8(w.shape[0], w.shape[1], wq, s_w, delta)


def fp8_ffn_layer(w_gate, w_up, w_down, delta_gu, delta_down) -> FfnW8A8:
    return FfnW8A8(w_gate.shape[1], w_gate.shape[0], fp8_linear_layer(w_gate, delta_gu),
                   fp8_linear_layer(w_up, delta_gu), fp8_linear_layer(w_down, delta_down))


def fp8_gemm_f32(qx, m, wq, n, k, ws=None, stream=None):
    acc = torch.empty((m, n), dtype=torch.float32, device=qx.device)
    if ws is None:
        ws = _empty(fp8_linear_workspace_bytes(m, n, k), qx.device)
    _check(lib().w8a8_fp8_gemm_f32(_ptr(qx), m, _ptr(wq), n, k, _ptr(acc), _ptr(ws),
                                   ws.numel(), _stream(stream)))
    return acc


def fp8_linear(layer: LinearW8A8, x, out_dtype=torch.float32, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.n), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = _empty(fp8_linear_workspace_bytes(m, layer.n, layer.k), x.device)
    d = layer.desc()
    _check(lib().w8a8_fp8_linear(ctypes.byref(d), _ptr(x), _dt(x), m, _ptr(out), _dt(out),
                                 _ptr(ws), ws.numel(), _stream(stream)))
    return out


def fp8_ffn_gate_up(ffn: FfnW8A8, qx, s_x, m, out=None, stream=None):
    if out is None:
        out = torch.empty((m, ffn.f), dtype=torch.bfloat16, device=qx.device)
    d = ffn.desc()
    _check(lib().w8a8_fp8_ffn_gate_up(ctypes.byref(d), _ptr(qx), _ptr(s_x), m, _ptr(out),
                                      _stream(stream)))
    return out


def fp8_ffn(layer: FfnW8A8, x, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.d), dtype=torch.bfloat16, device=x.device)
    if ws is None:
        ws = _empty(fp8_ffn_workspace_bytes(m, layer.d, layer.f), x.device)
    d = layer.desc()
    _check(lib().w8a8_fp8_ffn(ctypes.byref(d), _ptr(x), m, _ptr(out), _ptr(ws), ws.numel(),
                              _stream(stream)))
    return out


def fp8_lm_head(layer: LinearW8A8, x, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.n), dtype=torch.bfloat16, device=x.device)
    if ws is None:
        ws = _empty(fp8_linear_workspace_bytes(m, layer.n, layer.k), x.device)
    d = layer.desc()
    _check(lib().w8a8_fp8_lm_head(ctypes.byref(d), _ptr(x), m, _ptr(out), _ptr(ws), ws.numel(),
                                  _stream(stream)))
    return out


def bf16_linear(x, wp, n, k, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, n), dtype=torch.bfloat16, device=x.device)
    need = bf16_linear_workspace_bytes(m, n, k)
    if ws is None and need:
        ws = _empty(need, x.device)
    _check(lib().w8a8_bf16_linear(_ptr(x), m, _ptr(wp), n, k, _ptr(out), _ptr(ws),
                                  0 if ws is None else ws.numel(), _stream(stream)))
    return out


def bf16_ffn(layer: FfnBF16, x, out=None, ws=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.d), dtype=torch.bfloat16, device=x.device)
    if ws is None:
        ws = _empty(bf16_ffn_workspace_bytes(m, layer.d, layer.f), x.device)
    d = layer.desc()
    _check(lib().w8a8_bf16_ffn(ctypes.byref(d), _ptr(x), m, _ptr(out), _ptr(ws), ws.numel(),
                               _stream(stream)))
    return out


def bf16_ffn_gate_up(layer: FfnBF16, x, out=None, stream=None):
    _dev(x)
    m = x.shape[0]
    if out is None:
        out = torch.empty((m, layer.f), dtype=torch.bfloat16, device=x.device)
    d = layer.desc()
    _check(lib().w8a8_bf16_ffn_gate_up(ctypes.byref(d), _ptr(x), m, _ptr(out), _stream(stream)))
    return out


def rmsnorm(x, out=None, stream=None):
    m, d = x.shape
    if out is None:
        out = torch.empty_like(x)
    _check(lib().w8a8_rmsnorm(_ptr(_dev(x)), m, d, _ptr(out), _stream(stream)))
    return out


def rmsnorm_residual(x, f, out=None, stream=None):
    m, d = x.shape
    if out is None:
        out = torch.empty_like(x)
    _check(lib().w8a8_rmsnorm_residual(_ptr(_dev(x)), _ptr(_dev(f)), m, d, _ptr(out),
                                       _stream(stream)))
    return out


def precision_map(name: str, n_layers: int = 26) -> np.ndarray:
    prec = np.zeros(n_layers, np.uint8)
    r = lib().w8a8_precision_map(name.encode(), prec.ctypes.data_as(P), n_layers)
    if r < 0:
        raise ValueError("unknown precision map %r" % name)
    return prec


class Stack:
    """Device weights of an FFN stack plus the host descriptor arrays."""

    def __init__(self, int8_layers, bf16_layers, lm_int8: LinearW8A8, lm_bf16_packed, vocab):
        self.int8_layers = int8_layers
        self.bf16_layers = bf16_layers
        self.lm_int8 = lm_int8
        self.lm_bf16 = lm_bf16_packed
        n = len(bf16_layers)
        L0 = bf16_layers[0]
        self.d, self.f, self.vocab, self.n_layers = L0.d, L0.f, vocab, n
        self._i8 = (FfnDesc * n)(*[l.desc() if l is not None else FfnDesc() for l in int8_layers])
        self._bf = (Bf16FfnDesc * n)(*[l.desc() for l in bf16_layers])
        self._desc = StackDesc(n, self.d, self.f, vocab, self._i8, self._bf,
                               lm_int8.desc() if lm_int8 is not None else LinearDesc(),
                               _ptr(lm_bf16_packed))

    def run(self, x, prec: np.ndarray, lm_head_int8: bool, out=None, ws=None, stream=None):
        m = x.shape[0]
        if out is None:
            out = torch.empty((m, self.vocab), dtype=torch.bfloat16, device=x.device)
        if ws is None:
            ws = _empty(stack_workspace_bytes(m, self.d, self.f, self.vocab), x.device)
        prec = np.ascontiguousarray(prec, dtype=np.uint8)
        _check(lib().w8a8_ffn_stack(ctypes.byref(self._desc), prec.ctypes.data_as(P),
                                    int(lm_head_int8), _ptr(_dev(x)), m, _ptr(out), _ptr(ws),
                                    ws.numel(), _stream(stream)))
        return out

    @staticmethod
    def status(ws, stream=None):
        """Synchronises the stream; raises W8A8Error (status ETIMEOUT) when the
        last run on workspace ws had a persistent decode launch give up."""
        _check(lib().w8a8_ffn_stack_status(_ptr(ws), ws.numel(), _stream(stream)))

    def trace(self, x, prec: np.ndarray, lm_head_int8: bool = False, logits: bool = False,
              ws=None, stream=None):
        """Token stream after every layer, (n_layers, m, d) bf16; with logits=True
        also the logits: returns (hidden, logits)."""
        m = x.shape[0]
        hidden = torch.empty((self.n_layers, m, self.d), dtype=torch.bfloat16, device=x.device)
        out = (torch.empty((m, self.vocab), dtype=torch.bfloat16, device=x.device)
               if logits else None)
        if ws is None:
            ws = _empty(stack_workspace_bytes(m, self.d, self.f, self.vocab), x.device)
        prec = np.ascontiguousarray(prec, dtype=np.uint8)
        _check(lib().w8a8_ffn_stack_trace(ctypes.byref(self._desc), prec.ctypes.data_as(P),
                                          int(lm_head_int8), _ptr(_dev(x)), m, _ptr(out),
                                          _ptr(hidden), _ptr(ws), ws.numel(), _stream(stream)))
        return (hidden, out) if logits else hidden

    def _sens_ws(self, m, device):
        return _empty(lib().w8a8_stack_sensitivity_workspace_bytes(m, self.d, self.f, self.vocab,
                                                                   self.n_layers), device)

    def sensitivity(self, x, prec=None, stream=None):
        """(isolated_db, propagated_db) per layer as float32 arrays; propagated
        is None without a precision map."""
        m = x.shape[0]
        iso = np.zeros(self.n_layers, np.float32)
        prop = None if prec is None else np.zeros(self.n_layers, np.float32)
        pr = None if prec is None else np.ascontiguousarray(prec, dtype=np.uint8)
        ws = self._sens_ws(m, x.device)
        _check(lib().w8a8_stack_sensitivity(
            ctypes.byref(self._desc), None if pr is None else pr.ctypes.data_as(P), _ptr(_dev(x)),
            m, iso.ctypes.data_as(P), None if prop is None else prop.ctypes.data_as(P), _ptr(ws),
            ws.numel(), _stream(stream)))
        return iso, prop

    def select_map(self, x, budget_db, stream=None):
        """Automatic precision map: (prec uint8[n_layers], SQNR of the chosen map)."""
        m = x.shape[0]
        prec = np.zeros(self.n_layers, np.uint8)
        fin = np.zeros(1, np.float32)
        ws = self._sens_ws(m, x.device)
        _check(lib().w8a8_select_precision_map(ctypes.byref(self._desc), _ptr(_dev(x)), m,
                                               float(budget_db), prec.ctypes.data_as(P),
                                               fin.ctypes.data_as(P), _ptr(ws), ws.numel(),
                                               _stream(stream)))
        return prec, float(fin[0])


def sqnr(ref, test, stream=None):
    """(sum ref^2, sum (ref - test)^2, SQNR dB), computed on the GPU in binary64."""
    _dev(ref)
    _dev(test)
    assert ref.dtype == test.dtype and ref.numel() == test.numel()
    n = ref.numel()
    out = torch.empty(3, dtype=torch.float64, device=ref.device)
    ws = _empty(lib().w8a8_sqnr_workspace_bytes(n), ref.device)
    _check(lib().w8a8_sqnr(_ptr(ref), _ptr(test), _dt(ref), n, _ptr(out), _ptr(ws), ws.numel(),
                           _stream(stream)))
    return tuple(float(v) for v in out.cpu())


def rank_layers(isolated_db) -> np.ndarray:
    iso = np.ascontiguousarray(isolated_db, dtype=np.float32)
    order = np.zeros(iso.size, np.int32)
    if lib().w8a8_rank_layers(iso.ctypes.data_as(P), iso.size, order.ctypes.data_as(P)) != 0:
        raise ValueError("rank_layers: bad arguments")
    return order


# ----------------------------------------------------------------- layout helpers

# ---------------------------------------------------------------- key/value cache, attention decode

HEAD_DIM = 256


class KVCache:
    """One layer's key/value cache of t_max rows of 256: INT8 codes with
    per-row scales, or bf16 rows."""

    def __init__(self, t_max, int8=True, device="cuda"):
        self.t_max, self.int8 = t_max, int8
        if int8:
            self.k = torch.zeros((t_max, HEAD_DIM), dtype=torch.int8, device=device)
            self.v = torch.zeros((t_max, HEAD_DIM), dtype=torch.int8, device=device)
            self.sk = torch.zeros(t_max, dtype=torch.float32, device=device)
            self.sv = torch.zeros(t_max, dtype=torch.float32, device=device)
        else:
            self.k = torch.zeros((t_max, HEAD_DIM), dtype=torch.bfloat16, device=device)
            self.v = torch.zeros((t_max, HEAD_DIM), dtype=torch.bfloat16, device=device)

    def fill(self, t0, k, v, stream=None):
        """Rows t0 .. t0 + n - 1 from bf16 keys and values (n x 256 views with
        unit column stride, e.g. column slices of a fused QKV output)."""
        n = k.shape[0]
        if self.int8:
            kv_quantize(k, self.k[t0:t0 + n], self.sk[t0:t0 + n], stream)
            kv_quantize(v, self.v[t0:t0 + n], self.sv[t0:t0 + n], stream)
        else:
            self.k[t0:t0 + n].copy_(k)
            self.v[t0:t0 + n].copy_(v)


def kv_quantize(kv, codes=None, scales=None, stream=None):
    """Rows of 256 bf16 values (row stride kv.stride(0)) -> (INT8 codes
    [rows, 256], scales [rows])."""
    if not kv.is_cuda or kv.dim() != 2 or kv.shape[1] != HEAD_DIM or kv.stride(1) != 1 \
            or kv.dtype != torch.bfloat16:
        raise ValueError("kv must be a bf16 GPU tensor of rows of 256 with unit column stride")
    rows = kv.shape[0]
    if codes is None:
        codes = torch.empty((rows, HEAD_DIM), dtype=torch.int8, device=kv.device)
    if scales is None:
        scales = torch.empty(rows, dtype=torch.float32, device=kv.device)
    _check(lib().w8a8_kv_quantize(_ptr(kv), rows, kv.stride(0), _ptr(codes), _ptr(scales),
                                  _stream(stream)))
    return codes, scales


def attn_decode_workspace_bytes(t_max):
    return lib().w8a8_attn_decode_workspace_bytes(t_max)


def attn_decode(qkv, cache: KVCache, pos, window, n_heads=4, out=None, ws=None, stream=None):
    """Append the token's key and value (from its fused QKV row, bf16) at row
    pos of the cache and attend rows max(0, pos + 1 - window) .. pos; returns
    the bf16 attention output (n_heads * 256)."""
    _dev(qkv)
    if out is None:
        out = torch.empty(n_heads * HEAD_DIM, dtype=torch.bfloat16, device=qkv.device)
    if ws is None:
        ws = _empty(max(1, attn_decode_workspace_bytes(cache.t_max)), qkv.device)
    if cache.int8:
        _check(lib().w8a8_attn_decode(_ptr(qkv), n_heads, pos, window, _ptr(cache.k), _ptr(cache.sk),
                                      _ptr(cache.v), _ptr(cache.sv), cache.t_max, _ptr(out),
                                      _ptr(ws), ws.numel(), _stream(stream)))
    else:
        _check(lib().w8a8_attn_decode_bf16(_ptr(qkv), n_heads, pos, window, _ptr(cache.k),
                                           _ptr(cache.v), cache.t_max, _ptr(out), _ptr(ws),
                                           ws.numel(), _stream(stream)))
    return out


def frag_to_rowmajor(packed: np.ndarray, rows: int, k: int) -> np.ndarray:
    """Packed int8 fragment layout (include/w8a8.h) -> row-major rows x k."""
    rp, kp = -(-rows // 16) * 16, -(-k // 64) * 64
    a = np.asarray(packed, dtype=np.uint8).view(np.int8)[: rp * kp]
    # [rb, kb, g, r16, e16] -> [rb, r16, kb, g, e16]
    a = a.reshape(rp // 16, kp // 64, 4, 16, 16).transpose(0, 3, 1, 2, 4)
    return np.ascontiguousarray(a.reshape(rp, kp)[:rows, :k])


def rowmajor_to_frag(q: np.ndarray) -> np.ndarray:
    """Row-major int8 rows x k -> packed fragment layout (zero padded), as uint8."""
    rows, k = q.shape
    rp, kp = -(-rows // 16) * 16, -(-k // 64) * 64
    a = np.zeros((rp, kp), np.int8)
    a[:rows, :k] = q
    a = a.reshape(rp // 16, 16, kp // 64, 4, 16).transpose(0, 2, 3, 1, 4)
    return np.ascontiguousarray(a).reshape(-1).view(np.uint8)
