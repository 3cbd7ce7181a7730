"""A rounding-level variant of the oracle's stack, for the tests that bound
how far any other correct implementation may drift from the oracle over many
layers (test code, not a reference).

It computes the same stack as ``oracle.stack_hidden`` with two changes that
any binary32 implementation makes: RMSNorm's sum of squares, root and scaling
in binary32 (a sequential sum) instead of binary64 rounded once, and the bf16
layers' products summed in binary32 (numpy's float32 matrix product) instead
of binary64.  Both differences are below a bf16 rounding step, but the norms
turn every flipped bf16 rounding of a row into a rescaling of the whole row,
so they grow with depth; the GPU may differ from the oracle by about as much
as this variant does.
"""

import numpy as np

import oracle


def rmsnorm32(x_bits):
    xf = oracle.bf16_to_f32(x_bits)
    ss = np.zeros(xf.shape[0], np.float32)
    for j in range(xf.shape[1]):
        ss = (ss + xf[:, j] * xf[:, j]).astype(np.float32)
    inv = np.float32(1.0) / np.sqrt((ss / np.float32(xf.shape[1]) + np.float32(oracle.RMS_EPS))
                                    .astype(np.float32))
    return oracle.f32_to_bf16(xf * inv.astype(np.float32)[:, None])


def bf16_ffn32(a_bits, L):
    af = oracle.bf16_to_f32(a_bits)
    g = af @ oracle.bf16_to_f32(L["w_gate"]).T
    u = af @ oracle.bf16_to_f32(L["w_up"]).T
    h = oracle.f64_to_bf16(oracle.geglu(g, u))
    return oracle.f32_to_bf16(oracle.bf16_to_f32(h) @ oracle.bf16_to_f32(L["w_down"]).T)


def stack_hidden32(x_bits, layers, prec):
    x = x_bits
    out = []
    for l, L in enumerate(layers):
        a = rmsnorm32(x)
        f = oracle.w8a8_ffn(a, L["int8"]) if prec[l] else bf16_ffn32(a, L)
        x = oracle.residual_add(x, rmsnorm32(f))
        out.append(x)
    return out


def rel_l2(a_bits, b_bits):
    a = oracle.bf16_to_f32(a_bits).astype(np.float64)
    b = oracle.bf16_to_f32(b_bits).astype(np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def stack_bars(x_bits, layers, prec, hid_o, base=1e-3, factor=2.0):
    """Per-layer end-to-end bars: base + factor * (variant's rel-L2 from the
    oracle at that layer), and the variant's last token stream."""
    var = stack_hidden32(x_bits, layers, prec)
    return [base + factor * rel_l2(var[l], hid_o[l]) for l in range(len(prec))], var[-1]
