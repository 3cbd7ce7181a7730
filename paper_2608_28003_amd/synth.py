"""Seeded synthetic workloads with the shapes of Gemma-3-1B's FFN and lm_head.

This module only draws inputs.  It holds none of the quantisation arithmetic,
so both the GPU path and the CPU oracle may consume what it produces.

Recipe (numpy PCG64, ``numpy.random.default_rng(seed)``):

* activations ~ N(0, 1); a set of outlier channels, drawn without replacement
  on a separate seed, is multiplied by a constant factor for every token -- the
  channel-wise outliers that motivate smoothing (Sec. 6);
* weights ~ N(0, 0.02^2) (standard deviation 0.02, the usual random init);
* calibration activations: 512 tokens on their own seed with the same outlier
  channels;
* bf16 tensors are stored as uint16 bit patterns, rounded to nearest even from
  the binary32 draw;
* seeds follow ``1000 * config + tensor_id``.

Shapes (Tab. 1, Tab. 2, Sec. 2): hidden d = 1152, FFN intermediate f = 6912,
vocabulary V = 262144, 26 decoder layers.
"""

from __future__ import annotations

import numpy as np

D_MODEL = 1152
D_FF = 6912
VOCAB = 262144
N_LAYERS = 26
N_CAL = 512
W_SIGMA = 0.02


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """binary32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


def normal(seed: int, shape, sigma: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return x


def outlier_channels(seed: int, k: int, count: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(k, size=count, replace=False))


def activations(seed: int, m: int, k: int, channels: np.ndarray,
                factor: float) -> np.ndarray:
    x = normal(seed, (m, k))
    if len(channels):
        x[:, channels] *= np.float32(factor)
    return x


def n_outliers_1pct(k: int) -> int:
    return int(round(0.01 * k))


# ----------------------------------------------------------------- configs

def linear_config(m: int = 16, k: int = D_MODEL, n: int = D_FF, seed_base: int = 1000,
                  n_out: int = 4, factor: float = 50.0, dtype: str = "f32"):
    """Single W8A8 linear: X [m x k] with ``n_out`` outlier channels x factor,
    W [n x k], calibration X_cal [512 x k] with the same channels."""
    ch = outlier_channels(seed_base + 2, k, n_out)
    x = activations(seed_base + 1, m, k, ch, factor)
    w = normal(seed_base + 3, (n, k), W_SIGMA)
    x_cal = activations(seed_base + 4, N_CAL, k, ch, factor)
    if dtype == "bf16":
        x, w, x_cal = to_bf16_bits(x), to_bf16_bits(w), to_bf16_bits(x_cal)
    return dict(x=x, w=w, x_cal=x_cal, channels=ch)


def ffn_weights(seed_gate: int, seed_up: int, seed_down: int, d: int = D_MODEL,
                f: int = D_FF):
    return dict(w_gate=to_bf16_bits(normal(seed_gate, (f, d), W_SIGMA)),
                w_up=to_bf16_bits(normal(seed_up, (f, d), W_SIGMA)),
                w_down=to_bf16_bits(normal(seed_down, (d, f), W_SIGMA)))


def ffn_config(m: int = 128, d: int = D_MODEL, f: int = D_FF, seed_base: int = 2000,
               factor: float = 30.0):
    """Gemma-3-1B-shaped FFN block: bf16 X [m x d] with 1% outlier channels
    x factor, gate/up [f x d], down [d x f], X_cal [512 x d]."""
    ch = outlier_channels(seed_base + 2, d, n_outliers_1pct(d))
    x = to_bf16_bits(activations(seed_base + 1, m, d, ch, factor))
    x_cal = to_bf16_bits(activations(seed_base + 6, N_CAL, d, ch, factor))
    w = ffn_weights(seed_base + 3, seed_base + 4, seed_base + 5, d, f)
    return dict(x=x, x_cal=x_cal, channels=ch, **w)


def lm_head_config(m: int = 64, d: int = D_MODEL, vocab: int = VOCAB,
                   seed_base: int = 3000, factor: float = 30.0):
    """lm_head: bf16 X [m x d] with 1% outlier channels, W [vocab x d].
    Smaller m are prefixes of the m = 64 draw."""
    ch = outlier_channels(seed_base + 2, d, n_outliers_1pct(d))
    x = to_bf16_bits(activations(seed_base + 1, max(m, 64), d, ch, factor))[:m]
    w = to_bf16_bits(normal(seed_base + 3, (vocab, d), W_SIGMA))
    x_cal = to_bf16_bits(activations(seed_base + 4, N_CAL, d, ch, factor))
    return dict(x=np.ascontiguousarray(x), w=w, x_cal=x_cal, channels=ch)


def stack_config(m: int = 512, n_layers: int = N_LAYERS, d: int = D_MODEL,
                 f: int = D_FF, vocab: int = VOCAB, seed_base: int = 4000,
                 factor: float = 30.0):
    """26-layer FFN stack: input X, per-layer gate/up/down weights on seeds
    4100 + 3 l + {0, 1, 2}, lm_head W, calibration tokens."""
    ch = outlier_channels(seed_base + 2, d, n_outliers_1pct(d))
    x = to_bf16_bits(activations(seed_base + 1, m, d, ch, factor))
    x_cal = to_bf16_bits(activations(seed_base + 4, N_CAL, d, ch, factor))
    layers = [ffn_weights(seed_base + 100 + 3 * l, seed_base + 101 + 3 * l,
                          seed_base + 102 + 3 * l, d, f) for l in range(n_layers)]
    w_lm = to_bf16_bits(normal(seed_base + 3, (vocab, d), W_SIGMA))
    return dict(x=x, x_cal=x_cal, layers=layers, w_lm=w_lm, channels=ch)


def attn_config(m: int = 32, d: int = D_MODEL, seed_base: int = 5000,
                factor: float = 30.0, n_q: int = 1024, n_kv: int = 256):
    """Attention projections: fused QKV (d -> n_q + 2 n_kv) and O (n_q -> d)."""
    ch = outlier_channels(seed_base + 2, d, n_outliers_1pct(d))
    x = to_bf16_bits(activations(seed_base + 1, m, d, ch, factor))
    wq = normal(seed_base + 3, (n_q, d), W_SIGMA)
    wk = normal(seed_base + 4, (n_kv, d), W_SIGMA)
    wv = normal(seed_base + 5, (n_kv, d), W_SIGMA)
    wo = normal(seed_base + 6, (d, n_q), W_SIGMA)
    ch_o = outlier_channels(seed_base + 9, n_q, n_outliers_1pct(n_q))
    x_o = to_bf16_bits(activations(seed_base + 7, m, n_q, ch_o, factor))
    x_cal = to_bf16_bits(activations(seed_base + 8, N_CAL, d, ch, factor))
    return dict(x=x, x_o=x_o, x_cal=x_cal,
                w_qkv=to_bf16_bits(np.concatenate([wq, wk, wv], 0)),
                w_o=to_bf16_bits(wo))


HEAD_DIM = 256
KV_SIGMA = 2.0


def kv_decode_inputs(seed: int, t: int, n_heads: int = 4):
    """Cached keys and values of t earlier tokens and the fused QKV row of the
    current token ([n_heads x 256 query | 256 key | 256 value]), bf16.

    Scale: a projection with N(0, 0.02^2) weights of a 1152-wide activation
    whose 12 outlier channels carry 30x has outputs of standard deviation near
    0.02 * sqrt(1140 + 12 * 900) ~ 2.2, so keys, values and queries are drawn
    N(0, 2^2); keys also carry 8 outlier dimensions (x 8, on their own seed),
    the per-channel structure key projections show, which makes the per-token
    INT8 scale of a key row larger than its typical entry.  With this scale
    the scores q.k / 16 have a standard deviation near 7, a peaked softmax."""
    ch = outlier_channels(seed + 1, HEAD_DIM, 8)
    k = normal(seed + 2, (t, HEAD_DIM), KV_SIGMA)
    k[:, ch] *= np.float32(8.0)
    v = normal(seed + 3, (t, HEAD_DIM), KV_SIGMA)
    q = normal(seed + 4, (n_heads * HEAD_DIM,), KV_SIGMA)
    kn = normal(seed + 5, (HEAD_DIM,), KV_SIGMA)
    kn[ch] *= np.float32(8.0)
    vn = normal(seed + 6, (HEAD_DIM,), KV_SIGMA)
    return dict(k=to_bf16_bits(k), v=to_bf16_bits(v),
                qkv=to_bf16_bits(np.concatenate([q, kn, vn])), channels=ch)
