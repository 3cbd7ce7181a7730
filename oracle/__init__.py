"""CPU oracle for the W8A8 SmoothQuant path of arxiv 2608.28003.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain reference the GPU
library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it; the product package
never does, and the two share no code.

The arithmetic lives in ``w8a8_oracle.c`` (plain C loops, one function per
definition of the paper); this module only marshals numpy arrays and composes
those functions in the order the paper states:

* calibration, eq. ``delta-attn`` / ``delta-lmhead`` (Sec. 4 and Sec. 6);
* smoothing, eq. ``xhat-lmhead`` / ``what-lmhead`` (Sec. 6);
* per-output-channel weight quantisation, eq. ``si`` / ``what-ffn`` (Sec. 3);
* dynamic per-token activation quantisation, eq. ``stx`` / ``xint8`` (Sec. 6);
* the INT8 product and its two-scale dequantisation, eq. ``gemm-final``;
* the gated FFN between the projections (Sec. 3, Tab. 1 ``fused_fc``/``proj``);
* the FFN layer subsets, eq. ``ffn55`` / ``ffn1010`` / ``ffnall26``;
* the attention-projection layer subsets and the INT8 key/value cache with the
  one-token attention that reads it (Sec. 4, further speed-ups; Sec. 5, eq.
  ``attnffn55`` / ``attnffn1010``).

bf16 tensors are passed as ``numpy.uint16`` bit patterns.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "w8a8_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liborc.so")
# a prebuilt oracle library to load instead (the sanitizer test's instrumented
# build); when set, build() compiles nothing
_LIB_OVERRIDE = os.environ.get("W8A8_ORACLE_LIB")

MODE_DIV = 0  # activations: x / delta
MODE_MUL = 1  # weights:     W * delta

# GELU's tanh form, RMSNorm epsilon and the calibration floor are readings of
# a paper that leaves them implicit; see the module docstring of the C file.
RMS_EPS = 1e-6
CAL_EPS = 1e-5
ALPHA = 0.5  # SmoothQuant migration strength used throughout the paper


def build(force: bool = False) -> str:
    """Compile ``w8a8_oracle.c`` into ``liborc.so`` with gcc."""
    if _LIB_OVERRIDE:
        return _LIB_OVERRIDE
    if force or not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _L():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        D = ctypes.c_double
        sigs = {
            "orc_bf16_to_f32": [P, I64, P],
            "orc_f32_to_bf16": [P, I64, P],
            "orc_f64_to_bf16": [P, I64, P],
            "orc_col_absmax": [P, I64, I64, P],
            "orc_smooth_delta": [P, P, I64, D, D, P],
            "orc_quant_rows": [P, I64, I64, P, ctypes.c_int, P, P, P],
            "orc_gemm_i32": [P, P, I64, I64, I64, P],
            "orc_dequant": [P, P, P, I64, I64, P],
            "orc_geglu_f64": [P, P, I64, P],
            "orc_linear_f64": [P, P, I64, I64, I64, P],
            "orc_rmsnorm_f64": [P, I64, I64, D, P],
            "orc_e4m3_encode_n": [P, I64, P],
            "orc_quant_rows_fp8": [P, I64, I64, P, ctypes.c_int, P, P],
            "orc_gemm_fp8": [P, P, I64, I64, I64, P],
            "orc_dequant_fp8": [P, P, P, I64, I64, P],
            "orc_attn_decode_f64": [P, I64, I64, P, P, I64, D, P],
        }
        for name, args in sigs.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = None
        lib.orc_gemm_i32.restype = ctypes.c_int64
        lib.orc_e4m3_decode.argtypes = [ctypes.c_uint8]
        lib.orc_e4m3_decode.restype = ctypes.c_double
        _lib = lib
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---------------------------------------------------------------- formats

def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    b = _c(b, np.uint16)
    out = np.empty(b.shape, np.float32)
    _L().orc_bf16_to_f32(_p(b), b.size, _p(out))
    return out


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    _L().orc_f32_to_bf16(_p(x), x.size, _p(out))
    return out


def f64_to_bf16(x: np.ndarray) -> np.ndarray:
    x = _c(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    _L().orc_f64_to_bf16(_p(x), x.size, _p(out))
    return out


def as_f32(x: np.ndarray) -> np.ndarray:
    """Exact binary32 view of an input given as float32 or bf16 bits."""
    if x.dtype == np.uint16:
        return bf16_to_f32(x)
    return _c(x, np.float32)


# ---------------------------------------------------------------- a1

def col_absmax(x: np.ndarray, amax: np.ndarray | None = None) -> np.ndarray:
    """Running max_t |X_tj| (eq. delta-attn numerator statistic)."""
    xf = as_f32(x)
    rows, k = xf.shape
    out = np.zeros(k, np.float32) if amax is None else _c(amax, np.float32).copy()
    _L().orc_col_absmax(_p(xf), rows, k, _p(out))
    return out


def smooth_delta(act_amax, w_amax, alpha: float = ALPHA, eps: float = CAL_EPS):
    """delta_j = a_j^alpha / w_j^(1-alpha)  (eq. delta-attn, eq. delta-lmhead)."""
    a = _c(act_amax, np.float32)
    w = _c(w_amax, np.float32)
    out = np.empty(a.shape[0], np.float32)
    _L().orc_smooth_delta(_p(a), _p(w), a.shape[0], float(alpha), float(eps), _p(out))
    return out


def smooth_calibrate(x_cal, weights, alpha: float = ALPHA):
    """delta from calibration activations and every weight that consumes them.

    The weight statistic max_i |W_ij| runs over the rows of all matrices fed by
    this input (gate and up for the FFN input), stacked."""
    a = col_absmax(x_cal)
    w = None
    for wm in weights:
        w = col_absmax(wm, w)
    return smooth_delta(a, w, alpha)


# ---------------------------------------------------------------- a2 / a3

def quant_rows(x, delta=None, mode=MODE_DIV, want_vhat=False):
    """Symmetric per-row int8 codes and scales (eq. si/what-ffn, stx/xint8)."""
    xf = as_f32(x)
    rows, k = xf.shape
    q = np.empty((rows, k), np.int8)
    s = np.empty(rows, np.float32)
    d = None if delta is None else _c(delta, np.float32)
    vhat = np.empty((rows, k), np.float32) if want_vhat else None
    _L().orc_quant_rows(_p(xf), rows, k, _p(d), mode, _p(q), _p(s), _p(vhat))
    return (q, s, vhat) if want_vhat else (q, s)


def quantize_weights(w, delta=None):
    """W_hat = W diag(delta), then per-output-channel codes (a2)."""
    return quant_rows(w, delta, MODE_MUL)


def quantize_act(x, delta=None):
    """x_hat = x / delta, then per-token codes (a3)."""
    return quant_rows(x, delta, MODE_DIV)


# ---------------------------------------------------------------- a4 / a5

def gemm_i32(qa: np.ndarray, qb: np.ndarray) -> np.ndarray:
    qa = _c(qa, np.int8)
    qb = _c(qb, np.int8)
    m, k = qa.shape
    n, k2 = qb.shape
    assert k == k2
    acc = np.empty((m, n), np.int32)
    ovf = _L().orc_gemm_i32(_p(qa), _p(qb), m, n, k, _p(acc))
    if ovf:
        raise OverflowError("int32 accumulator overflow in %d sums" % ovf)
    return acc


def dequant(acc, s_tok, s_ch) -> np.ndarray:
    acc = _c(acc, np.int32)
    m, n = acc.shape
    y = np.empty((m, n), np.float32)
    _L().orc_dequant(_p(acc), _p(_c(s_tok, np.float32)), _p(_c(s_ch, np.float32)),
                     m, n, _p(y))
    return y


def w8a8_linear(x, wq, s_w, delta, out_dtype="f32"):
    """y = s_t s_i sum_j q_x q_w  with x quantised per token after x / delta."""
    qx, sx = quantize_act(x, delta)
    acc = gemm_i32(qx, wq)
    y = dequant(acc, sx, s_w)
    return y if out_dtype == "f32" else f32_to_bf16(y)


# ---------------------------------------------------------------- a6

def geglu(g, u) -> np.ndarray:
    """h = gelu_tanh(g) * u for the binary32 dequantised g, u, evaluated in
    binary64 (the caller rounds once to bf16).  A binary32 evaluation of
    0.5 g (1 + tanh z) loses all relative accuracy for z below about -6, where
    1 + tanh z falls under the rounding error of tanh z near -1."""
    return geglu_f64(_c(g, np.float32), _c(u, np.float32))


def geglu_f64(g, u) -> np.ndarray:
    g = _c(g, np.float64)
    u = _c(u, np.float64)
    h = np.empty(g.shape, np.float64)
    _L().orc_geglu_f64(_p(g), _p(u), g.size, _p(h))
    return h


def w8a8_ffn(x_bf16, q, stages=False):
    """INT8 FFN block: quantise x, gate/up INT8 products, GeGLU, bf16 h,
    requantise h / delta_down per token, down INT8 product, bf16 y.

    ``q`` holds the oracle's quantised weights: wq_gate, s_gate, wq_up, s_up,
    delta_gu, wq_down, s_down, delta_down."""
    qx, sx = quantize_act(x_bf16, q["delta_gu"])
    acc_g = gemm_i32(qx, q["wq_gate"])
    acc_u = gemm_i32(qx, q["wq_up"])
    g = dequant(acc_g, sx, q["s_gate"])
    u = dequant(acc_u, sx, q["s_up"])
    h = f64_to_bf16(geglu(g, u))
    qh, sh = quantize_act(h, q["delta_down"])
    acc_d = gemm_i32(qh, q["wq_down"])
    y = f32_to_bf16(dequant(acc_d, sh, q["s_down"]))
    if stages:
        return y, dict(qx=qx, sx=sx, acc_g=acc_g, acc_u=acc_u, g=g, u=u, h=h,
                       qh=qh, sh=sh, acc_d=acc_d)
    return y


def quantize_ffn(w_gate, w_up, w_down, x_cal, alpha=ALPHA):
    """Offline preparation of one INT8 FFN (a1 + a2): delta for the FFN input
    from the calibration tokens and the stacked gate/up rows; delta for the
    down input from the GeGLU output of the same tokens through the
    unquantised gate/up projections."""
    d_gu = smooth_calibrate(x_cal, [w_gate, w_up], alpha)
    g = linear_f64(x_cal, w_gate)
    u = linear_f64(x_cal, w_up)
    h_cal = f64_to_bf16(geglu(g.astype(np.float32), u.astype(np.float32)))
    d_dn = smooth_calibrate(h_cal, [w_down], alpha)
    wq_g, s_g = quantize_weights(w_gate, d_gu)
    wq_u, s_u = quantize_weights(w_up, d_gu)
    wq_d, s_d = quantize_weights(w_down, d_dn)
    return dict(wq_gate=wq_g, s_gate=s_g, wq_up=wq_u, s_up=s_u, delta_gu=d_gu,
                wq_down=wq_d, s_down=s_d, delta_down=d_dn)


# ---------------------------------------------------------------- bf16 path

def linear_f64(x, w) -> np.ndarray:
    xf = as_f32(x)
    wf = as_f32(w)
    m, k = xf.shape
    n = wf.shape[0]
    y = np.empty((m, n), np.float64)
    _L().orc_linear_f64(_p(xf), _p(wf), m, n, k, _p(y))
    return y


def bf16_linear(x, w) -> np.ndarray:
    """bf16 reference projection: exact products summed in binary64, one
    rounding to bf16."""
    return f64_to_bf16(linear_f64(x, w))


def bf16_ffn(x_bf16, w_gate, w_up, w_down) -> np.ndarray:
    """bf16 FFN block (layers the precision map keeps in bf16): g, u kept
    unrounded, h = bf16(gelu_tanh(g) u), y = bf16(h W_down^T)."""
    g = linear_f64(x_bf16, w_gate).astype(np.float32)
    u = linear_f64(x_bf16, w_up).astype(np.float32)
    h = f64_to_bf16(geglu(g, u))
    return bf16_linear(h, w_down)


def rmsnorm(x) -> np.ndarray:
    """RMSNorm with unit gain, binary64, rounded once to bf16."""
    xf = as_f32(x)
    m, d = xf.shape
    y = np.empty((m, d), np.float64)
    _L().orc_rmsnorm_f64(_p(xf), m, d, RMS_EPS, _p(y))
    return f64_to_bf16(y)


# ---------------------------------------------------------------- a7

def w8a8_lm_head(x_bf16, wq, s_w, delta) -> np.ndarray:
    """Logits in bf16 from the INT8 lm_head (Sec. 6, eq. gemm-final)."""
    return w8a8_linear(x_bf16, wq, s_w, delta, out_dtype="bf16")


# ---------------------------------------------------------------- FP8 variant

# OCP FP8 E4M3 codes as numpy.uint8 (Sec. 4 lists the move from INT8 to FP8
# codes; the scheme keeps smoothing and the per-token / per-channel scales,
# with 448, the largest E4M3 magnitude, in place of 127).
E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    table = np.array([_L().orc_e4m3_decode(c) for c in range(256)], np.float64)
    return table[_c(codes, np.uint8)]


def e4m3_encode(x) -> np.ndarray:
    """Nearest E4M3 code of binary32 values, ties to even, saturating at 448."""
    xf = _c(x, np.float32)
    out = np.empty(xf.shape, np.uint8)
    _L().orc_e4m3_encode_n(_p(xf), xf.size, _p(out))
    return out


def quant_rows_fp8(x, delta=None, mode=MODE_DIV):
    xf = as_f32(x)
    rows, k = xf.shape
    q = np.empty((rows, k), np.uint8)
    s = np.empty(rows, np.float32)
    d = None if delta is None else _c(delta, np.float32)
    _L().orc_quant_rows_fp8(_p(xf), rows, k, _p(d), mode, _p(q), _p(s))
    return q, s


def quantize_weights_fp8(w, delta=None):
    return quant_rows_fp8(w, delta, MODE_MUL)


def quantize_act_fp8(x, delta=None):
    return quant_rows_fp8(x, delta, MODE_DIV)


def gemm_fp8(qa, qb) -> np.ndarray:
    """sum_j dec(qa[t, j]) dec(qb[i, j]) in binary64."""
    qa = _c(qa, np.uint8)
    qb = _c(qb, np.uint8)
    m, k = qa.shape
    n, k2 = qb.shape
    assert k == k2
    acc = np.empty((m, n), np.float64)
    _L().orc_gemm_fp8(_p(qa), _p(qb), m, n, k, _p(acc))
    return acc


def dequant_fp8(acc, s_tok, s_ch) -> np.ndarray:
    acc = _c(acc, np.float64)
    m, n = acc.shape
    y = np.empty((m, n), np.float32)
    _L().orc_dequant_fp8(_p(acc), _p(_c(s_tok, np.float32)), _p(_c(s_ch, np.float32)),
                         m, n, _p(y))
    return y


def fp8_linear(x, wq, s_w, delta, out_dtype="f32"):
    qx, sx = quantize_act_fp8(x, delta)
    y = dequant_fp8(gemm_fp8(qx, wq), sx, s_w)
    return y if out_dtype == "f32" else f32_to_bf16(y)


def quantize_ffn_fp8(w_gate, w_up, w_down, x_cal, alpha=ALPHA):
    """As quantize_ffn, with E4M3 weight codes (same smoothing factors)."""
    q8 = quantize_ffn(w_gate, w_up, w_down, x_cal, alpha)
    out = dict(delta_gu=q8["delta_gu"], delta_down=q8["delta_down"])
    out["wq_gate"], out["s_gate"] = quantize_weights_fp8(w_gate, q8["delta_gu"])
    out["wq_up"], out["s_up"] = quantize_weights_fp8(w_up, q8["delta_gu"])
    out["wq_down"], out["s_down"] = quantize_weights_fp8(w_down, q8["delta_down"])
    return out


def fp8_ffn(x_bf16, q, stages=False):
    """FP8 FFN block, the INT8 block's steps with E4M3 codes."""
    qx, sx = quantize_act_fp8(x_bf16, q["delta_gu"])
    g = dequant_fp8(gemm_fp8(qx, q["wq_gate"]), sx, q["s_gate"])
    u = dequant_fp8(gemm_fp8(qx, q["wq_up"]), sx, q["s_up"])
    h = f64_to_bf16(geglu(g, u))
    qh, sh = quantize_act_fp8(h, q["delta_down"])
    y = f32_to_bf16(dequant_fp8(gemm_fp8(qh, q["wq_down"]), sh, q["s_down"]))
    if stages:
        return y, dict(qx=qx, sx=sx, g=g, u=u, h=h, qh=qh, sh=sh)
    return y


# ---------------------------------------------------------------- a8 / a9

N_LAYERS = 26


def precision_map(name: str, n_layers: int = N_LAYERS) -> np.ndarray:
    """Q_FFN of eq. ffn55 / ffn1010 / ffnall26 as a 0/1 vector (1 = INT8)."""
    p = np.zeros(n_layers, np.uint8)
    if name == "bf16":
        pass
    elif name == "5+5":
        p[0:5] = 1
        p[21:26] = 1
    elif name == "10+10":
        p[0:10] = 1
        p[16:26] = 1
    elif name == "all26":
        p[:] = 1
    else:
        raise ValueError(name)
    return p


def residual_add(x, y) -> np.ndarray:
    return f64_to_bf16(as_f32(x).astype(np.float64) + as_f32(y).astype(np.float64))


def stack_hidden(x_bf16, layers, prec):
    """The token stream after every layer of the FFN stack under a precision
    map (config glue, Sec. 3): x <- bf16(x + bf16(RMSNorm(FFN_l(bf16(RMSNorm(x)))))),
    both norm outputs rounded to bf16 (every activation is a bf16 tensor) and
    the residual sum rounded again; FFN_l the INT8 block for layers in Q_FFN
    and the bf16 block otherwise."""
    x = _c(x_bf16, np.uint16)
    hidden = []
    for l, L in enumerate(layers):
        a = rmsnorm(x)
        if prec[l]:
            f = w8a8_ffn(a, L["int8"])
        else:
            f = bf16_ffn(a, L["w_gate"], L["w_up"], L["w_down"])
        b = rmsnorm(f)
        x = residual_add(x, b)
        hidden.append(x)
    return hidden


def stack(x_bf16, layers, prec, lm_head, lm_head_int8, return_hidden=False):
    """FFN stack under a precision map (stack_hidden), then the final RMSNorm
    and the lm_head (INT8 or bf16)."""
    hidden = stack_hidden(x_bf16, layers, prec)
    x = hidden[-1] if hidden else _c(x_bf16, np.uint16)
    xf = rmsnorm(x)
    if lm_head_int8:
        logits = w8a8_lm_head(xf, lm_head["wq"], lm_head["s_w"], lm_head["delta"])
    else:
        logits = bf16_linear(xf, lm_head["w"])
    return (logits, hidden) if return_hidden else logits


# ---------------------------------------------------------------- metrics

def sqnr_db(clean, dirty) -> float:
    """10 log10(||y_clean||^2 / ||y_clean - y_dirty||^2)  (eq. sqnr-ffn; eq.
    sqnr-block is the same ratio of mean squares over a block's output)."""
    c = np.asarray(clean, np.float64)
    d = np.asarray(dirty, np.float64)
    num = float(np.sum(c * c))
    den = float(np.sum((c - d) ** 2))
    return float("inf") if den == 0.0 else 10.0 * np.log10(num / den)


def stack_sensitivity(x_bf16, layers, prec=None):
    """Per-layer sensitivity (Sec. 3, SA-PTQ by SQNR; Sec. 5 block SQNR).
    isolated[l]: SQNR of layer l's INT8 FFN block output against its bf16 FFN
    block output, both on RMSNorm of layer l's input in the all-bf16 stack.
    propagated[l] (with a map): SQNR of the token stream after layer l under
    the map against the all-bf16 stack.  Parity unpinned against the paper's
    own heatmap (needs Gemma weights)."""
    n = len(layers)
    ref = stack_hidden(x_bf16, layers, np.zeros(n, np.uint8))
    iso = np.zeros(n)
    for l, L in enumerate(layers):
        a = rmsnorm(x_bf16 if l == 0 else ref[l - 1])
        yb = bf16_ffn(a, L["w_gate"], L["w_up"], L["w_down"])
        y8 = w8a8_ffn(a, L["int8"])
        iso[l] = sqnr_db(bf16_to_f32(yb), bf16_to_f32(y8))
    prop = None
    if prec is not None:
        q = stack_hidden(x_bf16, layers, prec)
        prop = np.array([sqnr_db(bf16_to_f32(ref[l]), bf16_to_f32(q[l])) for l in range(n)])
    return iso, prop


def rank_layers(isolated_db) -> np.ndarray:
    """Layers by isolated SQNR, most robust first; NaN last; ties by index."""
    iso = np.asarray(isolated_db, np.float64)
    key = np.where(np.isnan(iso), -np.inf, iso)
    return np.array(sorted(range(iso.size), key=lambda i: (-key[i], i)), np.int64)


def select_map(x_bf16, layers, budget_db, return_trace=False):
    """Automatic precision map under an SQNR budget (Sec. 2: the fastest
    configuration within a quality budget; Sec. 3: the most robust layers are
    quantised first): visit layers by rank_layers of their isolated SQNR, set
    each to INT8, keep it there while the token stream after the last layer has
    at least budget_db SQNR against the all-bf16 stack.  Returns (map, its
    SQNR), and with return_trace the isolated SQNRs and every decision as
    (layer, SQNR with it INT8, kept)."""
    n = len(layers)
    iso, _ = stack_sensitivity(x_bf16, layers)
    ref_last = bf16_to_f32(stack_hidden(x_bf16, layers, np.zeros(n, np.uint8))[-1])
    prec = np.zeros(n, np.uint8)
    best = float("inf")
    trace = []
    for l in rank_layers(iso):
        prec[l] = 1
        db = sqnr_db(ref_last, bf16_to_f32(stack_hidden(x_bf16, layers, prec)[-1]))
        keep = db >= budget_db
        trace.append((int(l), db, keep))
        if keep:
            best = db
        else:
            prec[l] = 0
    if return_trace:
        return prec, best, iso, trace
    return prec, best


# ---------------------------------------------------------------- f4: attention decode with a KV cache

HEAD_DIM = 256      # Sec. 2: four query heads and one key/value head of 256
N_Q_HEADS = 4
ATTN_SCALE = 1.0 / 16.0   # 1 / sqrt(head dim)
GLOBAL_LAYERS = (0, 6, 12, 18)   # Sec. 2: the layers that attend the whole context
LOCAL_WINDOW = 1024              # Sec. 2: sliding window of the other layers


def kv_quantize(kv_bf16):
    """INT8 key/value cache rows: the per-token rule of eq. stx / xint8 with no
    smoothing (delta = 1): s_t = max_d |k_td| / 127, codes rne(k / s_t)
    clamped to [-127, 127]; an all-zero row stores s = 0 and zero codes."""
    return quant_rows(kv_bf16, None, MODE_DIV)


def kv_dequant(codes, scales) -> np.ndarray:
    """k = s_t * code, exact in binary64."""
    return _c(codes, np.int8).astype(np.float64) * _c(scales, np.float32).astype(np.float64)[:, None]


def attn_decode(q, k, v, scale=ATTN_SCALE) -> np.ndarray:
    """One query token with h heads (rows of q) against t cached rows of one
    shared key/value head: softmax(scale q k^T) v per head, binary64."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    h, dh = q.shape
    t = k.shape[0]
    assert k.shape == (t, dh) and v.shape == (t, dh) and t >= 1
    out = np.empty((h, dh), np.float64)
    _L().orc_attn_decode_f64(_p(q), h, dh, _p(k), _p(v), t, float(scale), _p(out))
    return out


def kv_cache(t_max, int8=True, head_dim=HEAD_DIM):
    """An empty key/value cache of t_max rows: INT8 codes with per-row scales,
    or bf16 rows."""
    if int8:
        return dict(int8=True, k=np.zeros((t_max, head_dim), np.int8), sk=np.zeros(t_max, np.float32),
                    v=np.zeros((t_max, head_dim), np.int8), sv=np.zeros(t_max, np.float32))
    return dict(int8=False, k=np.zeros((t_max, head_dim), np.uint16),
                v=np.zeros((t_max, head_dim), np.uint16))


def kv_fill(cache, t0, k_bf16, v_bf16):
    """Write rows t0 .. t0 + n - 1 of the cache from bf16 keys and values."""
    n = k_bf16.shape[0]
    if cache["int8"]:
        cache["k"][t0:t0 + n], cache["sk"][t0:t0 + n] = kv_quantize(k_bf16)
        cache["v"][t0:t0 + n], cache["sv"][t0:t0 + n] = kv_quantize(v_bf16)
    else:
        cache["k"][t0:t0 + n] = k_bf16
        cache["v"][t0:t0 + n] = v_bf16


def kv_rows(cache, t0, t1):
    """Cached keys and values of rows t0 .. t1 - 1 as binary64."""
    if cache["int8"]:
        return (kv_dequant(cache["k"][t0:t1], cache["sk"][t0:t1]),
                kv_dequant(cache["v"][t0:t1], cache["sv"][t0:t1]))
    return (bf16_to_f32(cache["k"][t0:t1]).astype(np.float64),
            bf16_to_f32(cache["v"][t0:t1]).astype(np.float64))


def attn_block_decode(qkv_bf16, cache, pos, window, n_heads=N_Q_HEADS, head_dim=HEAD_DIM):
    """The attention of one decode step: the projection output row [q heads |
    k | v] (bf16) appends its key and value at row pos of the cache, then the
    query heads attend rows max(0, pos + 1 - window) .. pos.  Returns the
    attention output (n_heads x head_dim, concatenated) rounded once to bf16,
    the input of the O projection."""
    qkv = _c(qkv_bf16, np.uint16).reshape(-1)
    nq = n_heads * head_dim
    assert qkv.size == nq + 2 * head_dim
    kv_fill(cache, pos, qkv[nq:nq + head_dim][None, :], qkv[nq + head_dim:][None, :])
    t0 = max(0, pos + 1 - window)
    k, v = kv_rows(cache, t0, pos + 1)
    q = bf16_to_f32(qkv[:nq]).astype(np.float64).reshape(n_heads, head_dim)
    return f64_to_bf16(attn_decode(q, k, v).reshape(-1))


def attn_window(layer: int, context: int) -> int:
    """Rows a layer attends (Sec. 2): the whole context in the global layers,
    the sliding window in the others."""
    return context if layer in GLOBAL_LAYERS else LOCAL_WINDOW


def attn_precision_map(name: str, n_layers: int = N_LAYERS) -> np.ndarray:
    """Q_ATT: the layers whose QKV and O projections run in INT8.  The paper's
    Attn+FFN configurations take Q_ATT = L (eq. attnffn55 / attnffn1010) and
    name blockwise attention subsets by analogy with the FFN ones as a further
    direction (Sec. 4), so the FFN sets of eq. ffn55 / ffn1010 / ffnall26 serve
    for Q_ATT too; "none" keeps every projection in bf16."""
    return precision_map("bf16" if name == "none" else name, n_layers)


def attn_block_proj_decode(x_bf16, xo_bf16, L, int8):
    """The two projections of one attention block at one token: the fused QKV
    projection of the block input and the O projection of the attention
    output, INT8 (eq. gemm-final, one shared quantisation of x for Q, K and V)
    or bf16.  L holds w_qkv, w_o (bf16) and, for INT8, their codes, scales and
    smoothing vectors."""
    if int8:
        qkv = w8a8_linear(x_bf16, L["wq_qkv"], L["s_qkv"], L["delta_qkv"], "bf16")
        o = w8a8_linear(xo_bf16, L["wq_o"], L["s_o"], L["delta_o"], "bf16")
    else:
        qkv = bf16_linear(x_bf16, L["w_qkv"])
        o = bf16_linear(xo_bf16, L["w_o"])
    return qkv, o
